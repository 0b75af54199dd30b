// Device definitions shared by the bf16 attention kernels (attn.hip,
// attn_pipe.hip): MFMA operand types, the LDS tile layouts and the
// direct global->LDS load.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace tsr {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

union Frag {
  uint4 u;
  uint32_t w[4];
  bf16x8 b;
  f16x8 h;
  f16x2 p[4];
};

constexpr int kD = 128;
// Keys per tile of the bf16 kernels.
constexpr int kKT = 32;
// V^T rows (fp16) are 16-byte aligned and hold each 16-key step permuted as
// keys [0..3, 8..11, 4..7, 12..15], so that the eight keys a lane feeds to
// the PV MFMA (4h .. 4h+3 and 8+4h .. 8+4h+3 for half-wave h, the order in
// which the S^T accumulators hand out P^T) are one 16-byte LDS read.
constexpr int kVStr = kKT + 8;         // fp16 elements per V^T row in LDS
// A K tile sits in LDS in the order the QK^T MFMAs consume it: one 1 KB
// block per 16-dim step kst, in which lane l's 16 bytes (at l * 16) are
// K[l % 32][16 kst + 8 (l / 32) .. + 8].  Fragment reads are then
// lane-contiguous (no bank conflicts, immediate offsets), and one direct
// global->LDS load of 16 bytes per lane fills one block.
constexpr int kKBlk = 1024;
constexpr int kKBytes = 8 * kKBlk;
constexpr int kVBytes = kD * kVStr * 2;
// s_waitcnt immediate that waits for every outstanding vector memory
// access (direct global->LDS loads included) and leaves the other counters.
constexpr int kWaitVm0 = 0x0F70;
// Lazy rescale threshold (log2 units): P may grow to 2^kLazy before the
// running max is moved.
constexpr float kLazy = 8.0f;
constexpr float kLazySum = 256.0f;   // 2^kLazy

// Position of key k (0 .. 31) of a tile in its permuted V^T row.
__device__ __forceinline__ int vt_col(int k) {
  const int b = k >> 4, kk = k & 15;
  return 16 * b + ((kk >> 2) & 1) * 8 + ((kk >> 3) & 1) * 4 + (kk & 3);
}

// Direct global->LDS load of 16 bytes per lane: lane l's bytes land at LDS
// address lds + 16 l (lds wave-uniform).  Written as assembly so that the
// compiler does not take the LDS write for a possible alias of the LDS reads
// that follow it (it would wait for the load before each of them); callers
// wait for these loads themselves (s_waitcnt vmcnt) before the barrier that
// hands the buffer to the workgroup.  M0 holds no other value in the
// kernels that use this.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_dma16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(src), "s"(lds) : "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

}  // namespace tsr

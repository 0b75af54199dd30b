// Internal declarations of libtsr: the device image of a plan and the kernel
// launchers.  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <exception>
#include <new>
#include <string>
#include <vector>

#include "../../include/tsr.h"

namespace tsr {

// Rows of one attention row block: consecutive rows of one request (in the
// computed order, or for the three-row-block bf16 kernel in AttnRow order).
constexpr int kTileRows = 32;
// Row blocks per attention item of the MFMA kernels (bf16 and e4m3 KV; one
// workgroup of 4 waves per row block), used when at least
// kMinGroupedRowBlockUse of the items' row-block x key tile slots hold work,
// over rows grouped by first visible key (AttnRow order).  Measured on the
// LOCAL-scope RAG and agent batches (slot use 0.70 and 0.78): three row
// blocks 13 % and 23 % faster than one; at 0.62 (the RAG batch without
// grouping) the two were level.
constexpr int kMaxRowBlocks = 3;
constexpr double kMinGroupedRowBlockUse = 0.6;
// Compute units of the GPU (MI355X).
constexpr int kNumCus = 256;
// Attention launches with at least this many (request, KV head) groups per
// XCD bin issue each bin group by group within thirds of the cost range.
// Measured: Agent-8B (32 groups per bin) 4.6 % faster; fp8 RAG (16) 3 % and
// RAG-8B (8) 1 % slower, the few large groups issued last forming the tail.
constexpr int kGroupMajorMinGroups = 24;
// Row blocks per item of the pipelined bf16 kernel (attn_pipe.hip), and
// the most 16-key blocks an item of it may span (their page ids sit in
// LDS: 65,536 keys).
constexpr int kPipeRowBlocks = 2;
constexpr int kPipeMaxBlocks = 4096;
// Keys per attention KV tile (granularity of the host-tier split of items).
constexpr int kKvTile = 64;
// Keys per tile of the bf16 MFMA attention kernel.
constexpr int kMfmaKeys = 32;
// Set in a V block-table entry whose page is a pool page (V aliasing).
constexpr int32_t kPoolPageFlag = 1 << 30;
// Workgroups of the MFMA attention are dealt round-robin over this many XCDs.
constexpr int kNumXcd = 8;

// A cached token moved by compose: pool slot -> request slot at `pos`.
// Slots are page * page_size + slot-in-page.
struct alignas(16) GatherDesc {
  int32_t src;
  int32_t dst;
  int32_t pos;
  int32_t skip;     // kSkipV / kSkipK: attention reads that half from the pool
};
constexpr int32_t kSkipV = 1, kSkipK = 2;

// A computed row: its request slot and prompt position.
struct alignas(8) RowDesc {
  int32_t dst;
  int32_t pos;
};

// A row of the bf16 row-block attention, in item order: its computed row
// (index of q, out and lse) and prompt position.  Plans of three row blocks
// order each request's rows by their first visible key (positions still
// ascending within each group), so that the rows that see the whole prompt
// (text, recompute windows) form full row blocks even where unit-local
// rows separate them; other plans keep the computed order.
struct alignas(8) AttnRow {
  int32_t row;
  int32_t pos;
};

// A retained token: computed row -> pool slot.
struct alignas(8) RetainDesc {
  int32_t row;
  int32_t dst;
};

// One whole page moved by the e4m3 kernels (each request page of an e4m3
// plan has a single writer, so its scale is computed from its own values).
//   compose: src = pool page, dst = request page, pos = position of slot 0
//   append:  src = first computed row, dst = request page, pos = position
//   retain:  src = first computed row, dst = pool page
// n = valid slots (< page_size only for a unit's or a prompt's last page).
struct alignas(16) PageDesc {
  int32_t src;
  int32_t dst;
  int32_t pos;
  int32_t n;
};

// One attention work item: up to row_blocks x kTileRows consecutive computed
// rows of one request, all with the same first visible key, against one KV head, for
// query heads head0 .. head0+3 of that KV head's group (MFMA kernels; a
// group of G > 4 heads is split over G/4 items).  n_rows == 0 marks padding.
struct alignas(16) AttnItem {
  int32_t row0;      // first computed row (plan order)
  int32_t n_rows;    // rows in the item (<= row_blocks * kTileRows)
  int32_t kv_len;    // keys kv_lo .. kv_len-1 are visible to some row (max pos + 1)
  int32_t min_pos;   // smallest position among the rows
  int32_t kv_head;
  int32_t bt_off;    // offset of the request's block table in the plan
  int32_t n_pages;   // entries of that block table
  int32_t head0;     // first query head of the group handled by the item
  int32_t kv_lo;     // first visible key of every row (0 unless unit-local)
  // -1: the item writes out/lse; else one key range c of a split item of
  // n_parts ranges: row block b's normalized rows and log-sum-exp go to
  // split buffer slot part_slot + b * n_parts (each row block's ranges sit
  // in consecutive slots)
  int32_t part_slot;
  int32_t n_parts;
  // the computed row of the item's first row when its rows are consecutive
  // computed rows at consecutive positions (then row i is crow0 + i at
  // position min_pos + i), else -1; and the K block-table entries of the
  // first key tile's two 16-key blocks: a workgroup can then load its
  // queries and first tile without reading the row table or the block
  // table first
  int32_t crow0;
  int32_t pg[2];
  int32_t pad[3];
};

// A row block of a split item: its rows were computed over n_slots
// consecutive key ranges, slots slot0 .. slot0 + n_slots - 1 of the split
// buffer; the merge kernel writes the rows of AttnRow entries row0 ..
// row0 + n_rows - 1, query heads hq0 .. hq0 + n_heads - 1.
struct alignas(16) CombineDesc {
  int32_t row0;
  int32_t n_rows;
  int32_t hq0;
  int32_t n_heads;
  int32_t slot0;
  int32_t n_slots;
  int32_t pad[2];
};
// Split buffer slot: kTileRows rows x 4 query heads x head_dim fp32
// (normalized output), then kTileRows x 4 fp32 log-sum-exp per slot.
constexpr int kSplitHeads = 4;
// The automatic key-range split caps items at the launch's mean key tiles
// per compute unit (256 on MI355X): a longer item would outlast the launch
// even with a compute unit to itself.  (Capping at the mean per workgroup
// slot, three per unit, split the RAG-8B batch under the LOCAL scope into
// 256 more items and did not shorten it: that launch is bound by its total
// work, not by its longest item.)
constexpr int kSplitSlots = 256;
constexpr int kMinSplitTiles = 32;
// At most this many split buffer slots (64 KiB each at head_dim 128).
constexpr int kMaxSplitSlots = 4096;

// Device-side view of a plan (pointers into the caller's workspace).
struct PlanDev {
  const GatherDesc* gather;
  const RowDesc* rows;
  const AttnRow* attn_rows;   // the rows in item order (row-block bf16 kernel)
  const RetainDesc* retain;
  const AttnItem* items;
  const AttnItem* items_part[2];
  const int32_t* block_tables;
  const int32_t* v_block_tables;  // block_tables, with V-aliased pages flagged
  const int32_t* k_block_tables;  // block_tables, with K-aliased pages flagged
  const PageDesc* gpages;  // e4m3 plans only
  const PageDesc* apages;
  const PageDesc* rpages;
  const float* rope_cos;   // [max_position][d/2]
  const float* rope_sin;   // [max_position][d/2]
  const CombineDesc* combine;   // split items, those of part 0 first
  float* split_o;          // [slots][kTileRows][kSplitHeads][d]
  float* split_lse;        // [slots][kTileRows][kSplitHeads]
};

}  // namespace tsr

struct tsr_plan {
  tsr_model model;
  float scale;              // resolved softmax scale
  int32_t n_pool_pages;
  int32_t n_req_pages;
  int32_t n_req;
  int32_t T;                // computed rows
  int32_t n_gather;
  int32_t n_retain;
  int32_t n_items;          // attention items incl. padding
  // the items split by whether their key tiles hold a gathered position:
  // [0] none (runnable before compose), [1] some; each scheduled on its own
  int32_t n_items_part[2];
  int32_t max_kv_len;
  int32_t row_blocks;       // row blocks per attention item (1, kPipeRowBlocks or kMaxRowBlocks)
  // key-range split items: merge descriptors (part 0's first) and buffer
  int32_t n_combine;
  int32_t n_combine_part[2];
  int32_t n_split_slots;
  int32_t n_split_items;    // items whose key range was split
  size_t off_combine, off_split_o, off_split_lse;
  size_t image_bytes;       // bytes of the image uploaded (the split buffer follows)
  int32_t n_gpages, n_apages, n_rpages;   // e4m3 plans only
  std::vector<int32_t> row_pos, row_req, row_lo;
  std::vector<char> image;  // host copy of the device image
  size_t off_gather, off_rows, off_retain, off_items, off_bt, ws_bytes;
  size_t off_attn_rows;
  bool rows_grouped;          // attn_rows groups rows by first visible key
  size_t off_items_part[2];
  size_t off_vbt;
  bool alias_v;               // V of whole gathered pages read from the pool
  int32_t n_aliased;          // request pages whose V is read from the pool
  bool alias_k;               // K of whole gathered pages rotated on load
  int32_t n_aliased_k;        // request pages whose K is read from the pool
  size_t off_kbt;
  size_t off_gpages, off_apages, off_rpages;
  const void* rope_table;   // device
  void* ws;                 // device, NULL for host-only plans
  // plans made by tsr_plan_create_static: the device and generation of the
  // shared plan area they were written into (0: a workspace plan)
  int32_t static_device = 0;
  uint64_t static_gen = 0;
  tsr::PlanDev dev;
};

namespace tsr {

// Thread-local error text, set by every failing entry point.
void set_error(const std::string& msg);

// A failed HIP call: record its name and message, return TSR_ERR_DEVICE.
inline tsr_status device_fail(const char* what, hipError_t e) {
  set_error(std::string(what) + ": " + hipGetErrorName(e) + " (" +
            hipGetErrorString(e) + ")");
  return TSR_ERR_DEVICE;
}

// Run an entry point's body so that no exception crosses the C ABI.
template <typename F>
tsr_status guarded(F&& f) {
  try {
    return f();
  } catch (const std::bad_alloc&) {
    set_error("host allocation failed");
    return TSR_ERR_INVALID_ARG;
  } catch (const std::exception& e) {
    set_error(std::string("internal error: ") + e.what());
    return TSR_ERR_INVALID_ARG;
  } catch (...) {
    set_error("internal error");
    return TSR_ERR_INVALID_ARG;
  }
}

// TSR_ERR_STATE if p is a static plan whose shared area a later static plan
// on the same device has rewritten.
tsr_status check_static_plan(const tsr_plan* p);

// Validate a model; on failure returns a status and sets the error.
tsr_status check_model(const tsr_model* m);

// Build a plan's host part (validation + descriptors + image layout).
// split_tiles: > 0 split items longer than that many 32-key tiles, 0 the
// automatic threshold, < 0 never (see tsr_plan_options).
tsr_status build_plan(const tsr_model* model, const tsr_request* reqs,
                      int32_t n_req, int32_t n_pool_pages, int32_t n_req_pages,
                      bool alias_v, bool alias_k, int32_t split_tiles, int32_t attn_kernel,
                      tsr_plan* plan);

// tsr_plan_workspace_size_ex / tsr_plan_create_ex; static_plan: the plan
// goes to the static plan area (automatic key-range splitting off).
size_t plan_workspace_size(const tsr_model* model, const tsr_request* reqs, int32_t n_req,
                           int32_t n_pool_pages, int32_t n_req_pages,
                           const tsr_plan_options* options, bool static_plan);
tsr_status create_plan(const tsr_model* model, const tsr_request* reqs, int32_t n_req,
                       int32_t n_pool_pages, int32_t n_req_pages,
                       const tsr_plan_options* options, bool static_plan,
                       const void* dev_rope_table, void* dev_workspace,
                       size_t workspace_bytes, void* stream, tsr_plan** out_plan);

// Kernel launchers (return hipSuccess or the launch error).
hipError_t launch_compose(const tsr_plan* p, const void* pool_k,
                          const void* pool_v, void* req_k, void* req_v,
                          int32_t n_layers, int64_t pool_stride,
                          int64_t req_stride, hipStream_t s);
hipError_t launch_append(const tsr_plan* p, const void* k, const void* v,
                         void* req_k, void* req_v, hipStream_t s);
// compose + append of one layer in one launch
hipError_t launch_assemble(const tsr_plan* p, const void* pool_k, const void* pool_v,
                           const void* k, const void* v, void* req_k, void* req_v,
                           hipStream_t s);
hipError_t launch_assemble_e4m3(const tsr_plan* p, const void* pool_k, const void* pool_v,
                                const float* pool_scale, const void* k, const void* v,
                                void* req_k, void* req_v, float* req_scale, hipStream_t s);
// Attention launchers run `n_items` items from `items` (a plan's full
// schedule or one of its parts); `part` (TSR_ATTN_ALL or one of the two
// parts) selects which split items the merge kernel that follows (bf16
// plans with split items) completes.
hipError_t launch_attn(const tsr_plan* p, int32_t part, const AttnItem* items,
                       int32_t n_items, const void* pool_k, const void* pool_v,
                       const void* q, const void* req_k, const void* req_v, void* out,
                       float* lse, hipStream_t s);
// the pipelined bf16 kernel (plans with row_blocks == kPipeRowBlocks)
hipError_t launch_attn_pipe(const tsr_plan* p, const AttnItem* items, int32_t n_items,
                            const void* pool_v, const void* q, const void* req_k,
                            const void* req_v, void* out, float* lse, hipStream_t s);
hipError_t launch_retain(const tsr_plan* p, const void* k, const void* v,
                         void* pool_k, void* pool_v, hipStream_t s);

// e4m3 pools: codes plus one fp32 scale per (page, K|V), scales [pages][2].
hipError_t launch_compose_e4m3(const tsr_plan* p, const void* pool_k,
                               const void* pool_v, const float* pool_scale,
                               void* req_k, void* req_v, float* req_scale,
                               int32_t n_layers, int64_t pool_stride,
                               int64_t req_stride, int64_t pool_scale_stride,
                               int64_t req_scale_stride, hipStream_t s);
hipError_t launch_append_e4m3(const tsr_plan* p, const void* k, const void* v,
                              void* req_k, void* req_v, float* req_scale,
                              hipStream_t s);
hipError_t launch_retain_e4m3(const tsr_plan* p, const void* k, const void* v,
                              void* pool_k, void* pool_v, float* pool_scale,
                              hipStream_t s);
hipError_t launch_attn_e4m3(const tsr_plan* p, const AttnItem* items, int32_t n_items,
                            const void* q, const void* req_k,
                            const void* req_v, const float* req_scale, void* out,
                            float* lse, hipStream_t s);

}  // namespace tsr

// Context-unit cache directory and block transfers (Sections 5.2-5.4).
//
// The directory is host metadata only: which units hold a complete reusable
// state in a block arena (the node's pinned host-memory cache), in which
// blocks and under which storage epoch, and how many transfers still read
// them.  It never touches the blocks' bytes and makes no HIP call; the bytes
// move with tsr_copy_blocks (copy engines) or the compose/retain kernels.
#include <algorithm>
#include <mutex>
#include <set>
#include <string>
#include <unordered_map>
#include <vector>

#include "tsr_internal.h"

namespace {

struct Entry {
  int32_t state;                 // TSR_ENTRY_PENDING or TSR_ENTRY_READY
  uint64_t epoch;
  std::vector<int32_t> blocks;
  int32_t leases;
};

}  // namespace

struct tsr_cache {
  mutable std::mutex mu;
  int32_t n_blocks = 0;
  // Free blocks, taken lowest id first so that a unit's blocks form long
  // runs (fewer, larger copies) while the arena is not fragmented.
  std::set<int32_t> free_blocks;
  std::unordered_map<uint64_t, Entry> entries;
  // Blocks of cancelled reservations, by epoch: writes may still be in
  // flight, so they return to the free set only on tsr_cache_reclaim.
  std::unordered_map<uint64_t, std::vector<int32_t>> draining;
  uint64_t next_epoch = 1;
};

using tsr::guarded;
using tsr::set_error;

namespace {

std::string unit_str(uint64_t id) { return "unit " + std::to_string(id); }

const char* state_name(int32_t s) {
  return s == TSR_ENTRY_READY ? "READY" : s == TSR_ENTRY_PENDING ? "PENDING" : "ABSENT";
}

// Lookup of an entry that must exist with the given epoch.
tsr_status find_epoch(tsr_cache* c, uint64_t unit, uint64_t epoch, Entry** out) {
  auto it = c->entries.find(unit);
  if (it == c->entries.end()) {
    set_error(unit_str(unit) + " has no entry");
    return TSR_ERR_STATE;
  }
  if (it->second.epoch != epoch) {
    set_error(unit_str(unit) + ": stale storage epoch " + std::to_string(epoch) +
              " (entry holds " + std::to_string(it->second.epoch) + ")");
    return TSR_ERR_STATE;
  }
  *out = &it->second;
  return TSR_OK;
}

}  // namespace

extern "C" {

tsr_status tsr_cache_create(int32_t n_blocks, tsr_cache** out) {
  return guarded([&]() -> tsr_status {
    if (!out || n_blocks < 0) {
      set_error("tsr_cache_create: out is NULL or n_blocks < 0");
      return TSR_ERR_INVALID_ARG;
    }
    *out = nullptr;
    auto* c = new tsr_cache;
    c->n_blocks = n_blocks;
    for (int32_t b = 0; b < n_blocks; ++b) c->free_blocks.insert(c->free_blocks.end(), b);
    *out = c;
    return TSR_OK;
  });
}

void tsr_cache_destroy(tsr_cache* c) { delete c; }

tsr_status tsr_cache_reserve(tsr_cache* c, uint64_t unit, int32_t n_blocks,
                             uint64_t* epoch, int32_t* blocks) {
  return guarded([&]() -> tsr_status {
    if (!c || !epoch || !blocks || n_blocks <= 0) {
      set_error("tsr_cache_reserve: NULL argument or n_blocks <= 0");
      return TSR_ERR_INVALID_ARG;
    }
    std::lock_guard<std::mutex> g(c->mu);
    auto it = c->entries.find(unit);
    if (it != c->entries.end()) {
      set_error(unit_str(unit) + " already has a " + state_name(it->second.state) +
                " entry");
      return TSR_ERR_STATE;
    }
    if ((int64_t)c->free_blocks.size() < n_blocks) {
      set_error(unit_str(unit) + ": " + std::to_string(n_blocks) + " blocks needed, " +
                std::to_string(c->free_blocks.size()) + " free");
      return TSR_ERR_NO_SPACE;
    }
    Entry e{TSR_ENTRY_PENDING, c->next_epoch++, {}, 0};
    e.blocks.reserve(n_blocks);
    auto f = c->free_blocks.begin();
    for (int32_t i = 0; i < n_blocks; ++i) e.blocks.push_back(*f++);
    c->free_blocks.erase(c->free_blocks.begin(), f);
    std::copy(e.blocks.begin(), e.blocks.end(), blocks);
    *epoch = e.epoch;
    c->entries.emplace(unit, std::move(e));
    return TSR_OK;
  });
}

tsr_status tsr_cache_publish(tsr_cache* c, uint64_t unit, uint64_t epoch,
                             const int32_t* blocks, int32_t n_blocks) {
  return guarded([&]() -> tsr_status {
    if (!c || (!blocks && n_blocks > 0) || n_blocks < 0) {
      set_error("tsr_cache_publish: NULL argument or n_blocks < 0");
      return TSR_ERR_INVALID_ARG;
    }
    std::lock_guard<std::mutex> g(c->mu);
    Entry* e = nullptr;
    if (tsr_status s = find_epoch(c, unit, epoch, &e)) return s;
    if (e->state != TSR_ENTRY_PENDING) {
      set_error(unit_str(unit) + " is " + state_name(e->state) + ", not PENDING");
      return TSR_ERR_STATE;
    }
    if ((size_t)n_blocks != e->blocks.size() ||
        !std::equal(e->blocks.begin(), e->blocks.end(), blocks)) {
      set_error(unit_str(unit) + ": block set differs from the reservation");
      return TSR_ERR_STATE;
    }
    e->state = TSR_ENTRY_READY;
    return TSR_OK;
  });
}

tsr_status tsr_cache_cancel(tsr_cache* c, uint64_t unit, uint64_t epoch) {
  return guarded([&]() -> tsr_status {
    if (!c) {
      set_error("tsr_cache_cancel: cache is NULL");
      return TSR_ERR_INVALID_ARG;
    }
    std::lock_guard<std::mutex> g(c->mu);
    Entry* e = nullptr;
    if (tsr_status s = find_epoch(c, unit, epoch, &e)) return s;
    if (e->state != TSR_ENTRY_PENDING) {
      set_error(unit_str(unit) + " is " + state_name(e->state) + ", not PENDING");
      return TSR_ERR_STATE;
    }
    auto& d = c->draining[epoch];
    d.insert(d.end(), e->blocks.begin(), e->blocks.end());
    c->entries.erase(unit);
    return TSR_OK;
  });
}

tsr_status tsr_cache_reclaim(tsr_cache* c, uint64_t epoch) {
  return guarded([&]() -> tsr_status {
    if (!c) {
      set_error("tsr_cache_reclaim: cache is NULL");
      return TSR_ERR_INVALID_ARG;
    }
    std::lock_guard<std::mutex> g(c->mu);
    auto it = c->draining.find(epoch);
    if (it == c->draining.end()) {
      set_error("no cancelled reservation with storage epoch " + std::to_string(epoch));
      return TSR_ERR_STATE;
    }
    c->free_blocks.insert(it->second.begin(), it->second.end());
    c->draining.erase(it);
    return TSR_OK;
  });
}

tsr_status tsr_cache_acquire(tsr_cache* c, uint64_t unit, int32_t max_blocks,
                             uint64_t* epoch, int32_t* blocks, int32_t* n_blocks) {
  return guarded([&]() -> tsr_status {
    if (!c || !epoch || !n_blocks || (!blocks && max_blocks > 0)) {
      set_error("tsr_cache_acquire: NULL argument");
      return TSR_ERR_INVALID_ARG;
    }
    std::lock_guard<std::mutex> g(c->mu);
    auto it = c->entries.find(unit);
    if (it == c->entries.end() || it->second.state != TSR_ENTRY_READY) {
      set_error(unit_str(unit) + " is " +
                state_name(it == c->entries.end() ? TSR_ENTRY_ABSENT : it->second.state) +
                ", not READY");
      return TSR_ERR_STATE;
    }
    Entry& e = it->second;
    *n_blocks = (int32_t)e.blocks.size();
    if ((int32_t)e.blocks.size() > max_blocks) {
      set_error(unit_str(unit) + " holds " + std::to_string(e.blocks.size()) +
                " blocks; the output array has room for " + std::to_string(max_blocks));
      return TSR_ERR_OUT_OF_RANGE;
    }
    std::copy(e.blocks.begin(), e.blocks.end(), blocks);
    *epoch = e.epoch;
    ++e.leases;
    return TSR_OK;
  });
}

tsr_status tsr_cache_release(tsr_cache* c, uint64_t unit, uint64_t epoch) {
  return guarded([&]() -> tsr_status {
    if (!c) {
      set_error("tsr_cache_release: cache is NULL");
      return TSR_ERR_INVALID_ARG;
    }
    std::lock_guard<std::mutex> g(c->mu);
    Entry* e = nullptr;
    if (tsr_status s = find_epoch(c, unit, epoch, &e)) return s;
    if (e->leases <= 0) {
      set_error(unit_str(unit) + " holds no read lease");
      return TSR_ERR_STATE;
    }
    --e->leases;
    return TSR_OK;
  });
}

tsr_status tsr_cache_evict(tsr_cache* c, uint64_t unit) {
  return guarded([&]() -> tsr_status {
    if (!c) {
      set_error("tsr_cache_evict: cache is NULL");
      return TSR_ERR_INVALID_ARG;
    }
    std::lock_guard<std::mutex> g(c->mu);
    auto it = c->entries.find(unit);
    if (it == c->entries.end() || it->second.state != TSR_ENTRY_READY) {
      set_error(unit_str(unit) + " is " +
                state_name(it == c->entries.end() ? TSR_ENTRY_ABSENT : it->second.state) +
                ", not READY");
      return TSR_ERR_STATE;
    }
    if (it->second.leases > 0) {
      set_error(unit_str(unit) + " has " + std::to_string(it->second.leases) +
                " read lease(s) outstanding");
      return TSR_ERR_STATE;
    }
    c->free_blocks.insert(it->second.blocks.begin(), it->second.blocks.end());
    c->entries.erase(it);
    return TSR_OK;
  });
}

tsr_status tsr_cache_query(const tsr_cache* c, uint64_t unit, int32_t* state,
                           uint64_t* epoch, int32_t* n_blocks, int32_t* leases) {
  return guarded([&]() -> tsr_status {
    if (!c || !state) {
      set_error("tsr_cache_query: cache or state is NULL");
      return TSR_ERR_INVALID_ARG;
    }
    std::lock_guard<std::mutex> g(c->mu);
    auto it = c->entries.find(unit);
    const bool found = it != c->entries.end();
    *state = found ? it->second.state : TSR_ENTRY_ABSENT;
    if (epoch) *epoch = found ? it->second.epoch : 0;
    if (n_blocks) *n_blocks = found ? (int32_t)it->second.blocks.size() : 0;
    if (leases) *leases = found ? it->second.leases : 0;
    return TSR_OK;
  });
}

int32_t tsr_cache_free_blocks(const tsr_cache* c) {
  if (!c) return -1;
  std::lock_guard<std::mutex> g(c->mu);
  return (int32_t)c->free_blocks.size();
}

tsr_status tsr_copy_blocks(void* dst, int32_t n_dst_blocks, const int32_t* dst_blocks,
                           const void* src, int32_t n_src_blocks,
                           const int32_t* src_blocks, int32_t n, int64_t block_bytes,
                           int32_t n_layers, int64_t dst_layer_stride,
                           int64_t src_layer_stride, void* stream) {
  return guarded([&]() -> tsr_status {
    if (n < 0 || block_bytes <= 0 || n_layers < 1 || n_dst_blocks < 0 ||
        n_src_blocks < 0) {
      set_error("tsr_copy_blocks: n < 0, block_bytes <= 0, n_layers < 1 or a negative arena size");
      return TSR_ERR_INVALID_ARG;
    }
    if (n == 0) return TSR_OK;
    if (!dst || !src || !dst_blocks || !src_blocks) {
      set_error("tsr_copy_blocks: NULL buffer or block list");
      return TSR_ERR_INVALID_ARG;
    }
    const int64_t arena_d = (int64_t)n_dst_blocks * block_bytes;
    const int64_t arena_s = (int64_t)n_src_blocks * block_bytes;
    if (n_layers > 1 && (dst_layer_stride < arena_d || src_layer_stride < arena_s)) {
      set_error("tsr_copy_blocks: a layer stride is smaller than its arena");
      return TSR_ERR_INVALID_ARG;
    }
    for (int32_t i = 0; i < n; ++i) {
      if (dst_blocks[i] < 0 || dst_blocks[i] >= n_dst_blocks || src_blocks[i] < 0 ||
          src_blocks[i] >= n_src_blocks) {
        set_error("tsr_copy_blocks: pair " + std::to_string(i) + " (" +
                  std::to_string(src_blocks[i]) + " -> " + std::to_string(dst_blocks[i]) +
                  ") is outside its arena");
        return TSR_ERR_OUT_OF_RANGE;
      }
    }
    auto s = static_cast<hipStream_t>(stream);
    auto* d8 = static_cast<char*>(dst);
    auto* s8 = static_cast<const char*>(src);
    // Merge pairs whose ids both continue the previous run; one copy per run
    // (all layers of a run in one strided copy).
    int32_t i = 0;
    while (i < n) {
      int32_t j = i + 1;
      while (j < n && dst_blocks[j] == dst_blocks[j - 1] + 1 &&
             src_blocks[j] == src_blocks[j - 1] + 1)
        ++j;
      const size_t bytes = (size_t)(j - i) * (size_t)block_bytes;
      char* dp = d8 + (int64_t)dst_blocks[i] * block_bytes;
      const char* sp = s8 + (int64_t)src_blocks[i] * block_bytes;
      hipError_t e;
      if (n_layers == 1)
        e = hipMemcpyAsync(dp, sp, bytes, hipMemcpyDefault, s);
      else
        e = hipMemcpy2DAsync(dp, (size_t)dst_layer_stride, sp, (size_t)src_layer_stride,
                             bytes, (size_t)n_layers, hipMemcpyDefault, s);
      if (e != hipSuccess) return tsr::device_fail("tsr_copy_blocks", e);
      i = j;
    }
    return TSR_OK;
  });
}

}  // extern "C"

// Host planner: validates a batch of requests and builds the device image of
// its plan (Section 5.3, placement before preparation: the prompt layout and
// the request's KV slots are fixed before any unit is prepared).
//
// The plan lists
//   * computed rows  -- text tokens, every token of a MISS unit, and the
//                       first min(r, n) tokens of each HIT unit (the fixed
//                       chunk-initial recompute window of the composition
//                       policy, Section 7), by increasing position;
//   * gathered tokens -- the remaining tokens of HIT units, pool slot ->
//                       request slot (Section 5.1 storage blocks: token j of
//                       a unit is in block j / B at slot j % B);
//   * retained tokens -- tokens of MISS units allowed to be retained;
//   * attention items -- tiles of consecutive computed rows x KV heads, in an
//                       XCD-aware, longest-first launch order.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <numeric>
#include <sstream>

#include "tsr_internal.h"

namespace tsr {

namespace {

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

tsr_status fail(tsr_status st, const std::string& msg) {
  set_error(msg);
  return st;
}

struct Seg {
  int32_t start, len;
  int unit;  // -1 for text
};

}  // namespace

tsr_status check_model(const tsr_model* m) {
  if (!m) return fail(TSR_ERR_INVALID_ARG, "model is NULL");
  if (m->n_q_heads <= 0 || m->n_kv_heads <= 0)
    return fail(TSR_ERR_INVALID_ARG, "head counts must be positive");
  if (m->n_q_heads % m->n_kv_heads)
    return fail(TSR_ERR_INVALID_ARG, "n_q_heads must be a multiple of n_kv_heads");
  if (!is_pow2(m->page_size) || m->page_size < 8 || m->page_size > 64)
    return fail(TSR_ERR_UNSUPPORTED, "page_size must be a power of two in [8, 64]");
  if (!(m->rope_theta > 0.0) || !std::isfinite(m->rope_theta))
    return fail(TSR_ERR_INVALID_ARG, "rope_theta must be positive and finite");
  if (m->rope_interleaved != 0 && m->rope_interleaved != 1)
    return fail(TSR_ERR_INVALID_ARG, "rope_interleaved must be 0 or 1");
  if (m->rope_interleaved == 1)
    return fail(TSR_ERR_UNSUPPORTED,
                "interleaved RoPE pairing (2i, 2i+1) is not implemented; only the "
                "half-split pairing (i, i + head_dim/2) is");
  if (m->max_position <= 0 || m->max_position > (1 << 20))
    return fail(TSR_ERR_INVALID_ARG, "max_position must be in [1, 2^20]");
  if (!(m->softmax_scale >= 0.0f) || !std::isfinite(m->softmax_scale))
    return fail(TSR_ERR_INVALID_ARG, "softmax_scale must be >= 0 and finite");
  const int G = m->n_q_heads / m->n_kv_heads;
  if (m->kv_dtype == TSR_F32 && m->act_dtype == TSR_F32) {
    if (m->head_dim != 64 && m->head_dim != 128 && m->head_dim != 256)
      return fail(TSR_ERR_UNSUPPORTED, "fp32 path supports head_dim 64, 128, 256");
    return TSR_OK;
  }
  if (m->kv_dtype == TSR_BF16 && m->act_dtype == TSR_BF16) {
    if (m->head_dim != 128)
      return fail(TSR_ERR_UNSUPPORTED, "bf16 path supports head_dim 128");
    if (m->page_size < 16)
      return fail(TSR_ERR_UNSUPPORTED, "bf16 path needs page_size >= 16");
    if (G != 1 && G != 2 && G != 4 && G != 8)
      return fail(TSR_ERR_UNSUPPORTED, "bf16 path supports GQA group 1, 2, 4, 8");
    return TSR_OK;
  }
  if (m->kv_dtype == TSR_E4M3 && m->act_dtype == TSR_BF16) {
    if (m->head_dim != 128)
      return fail(TSR_ERR_UNSUPPORTED, "e4m3 path supports head_dim 128");
    if (m->page_size != 16)
      return fail(TSR_ERR_UNSUPPORTED, "e4m3 path supports page_size 16");
    if (m->n_kv_heads > 16)
      return fail(TSR_ERR_UNSUPPORTED, "e4m3 path supports at most 16 KV heads");
    if (G != 1 && G != 2 && G != 4 && G != 8)
      return fail(TSR_ERR_UNSUPPORTED, "e4m3 path supports GQA group 1, 2, 4, 8");
    return TSR_OK;
  }
  return fail(TSR_ERR_UNSUPPORTED, "unsupported (kv_dtype, act_dtype) pair");
}

tsr_status build_plan(const tsr_model* model, const tsr_request* reqs,
                      int32_t n_req, int32_t n_pool_pages, int32_t n_req_pages,
                      bool alias_v, bool alias_k, int32_t split_tiles, int32_t attn_kernel,
                      tsr_plan* p) {
  tsr_status st = check_model(model);
  if (st != TSR_OK) return st;
  if (n_req < 0) return fail(TSR_ERR_INVALID_ARG, "n_req < 0");
  if (n_req > 0 && !reqs) return fail(TSR_ERR_INVALID_ARG, "reqs is NULL");
  if (n_pool_pages < 0 || n_req_pages < 0)
    return fail(TSR_ERR_INVALID_ARG, "arena page counts must be >= 0");
  if ((int64_t)n_pool_pages * model->page_size >= INT32_MAX ||
      (int64_t)n_req_pages * model->page_size >= INT32_MAX)
    return fail(TSR_ERR_OUT_OF_RANGE, "arena too large: pages * page_size must fit int32");
  const tsr_model& m = *model;
  const int B = m.page_size;
  const int Hkv = m.n_kv_heads;

  p->model = m;
  p->scale = m.softmax_scale > 0.0f ? m.softmax_scale
                                    : (float)(1.0 / std::sqrt((double)m.head_dim));
  p->n_pool_pages = n_pool_pages;
  p->n_req_pages = n_req_pages;
  p->n_req = n_req;
  p->alias_v = alias_v;
  p->n_aliased = 0;
  if (alias_v && (m.kv_dtype != TSR_BF16 || m.act_dtype != TSR_BF16))
    return fail(TSR_ERR_UNSUPPORTED, "V aliasing is built for bf16 pools only");
  if (alias_v && (int64_t)n_pool_pages >= kPoolPageFlag)
    return fail(TSR_ERR_OUT_OF_RANGE, "V aliasing needs pool page ids below 2^30");
  p->alias_k = alias_k;
  p->n_aliased_k = 0;
  if (alias_k && (m.kv_dtype != TSR_BF16 || m.act_dtype != TSR_BF16))
    return fail(TSR_ERR_UNSUPPORTED, "K rotated on load is built for bf16 pools only");
  if (alias_k && (int64_t)n_pool_pages >= kPoolPageFlag)
    return fail(TSR_ERR_OUT_OF_RANGE, "K aliasing needs pool page ids below 2^30");

  const bool e4m3 = m.kv_dtype == TSR_E4M3;
  std::vector<PageDesc> gpages, apages, rpages;
  std::vector<GatherDesc> gather;
  std::vector<RowDesc> rows;
  std::vector<RetainDesc> retain;
  std::vector<int32_t> bts, vbts, kbts;
  std::vector<int32_t> bt_off(n_req), bt_len(n_req), req_row0(n_req + 1, 0);
  // per request, the position ranges [a, b) that compose fills
  std::vector<std::vector<std::pair<int32_t, int32_t>>> gathered(n_req);
  p->row_pos.clear();
  p->row_req.clear();
  p->row_lo.clear();

  std::vector<uint8_t> req_page_used((size_t)n_req_pages, 0);
  // pool pages: bit 1 = read by a HIT, bit 2 = written by a retained MISS
  std::vector<uint8_t> pool_use((size_t)n_pool_pages, 0);
  std::ostringstream err;

  for (int r = 0; r < n_req; ++r) {
    const tsr_request& q = reqs[r];
    if (q.prompt_len <= 0) {
      err << "request " << r << ": prompt_len must be positive";
      return fail(TSR_ERR_INVALID_ARG, err.str());
    }
    if (q.prompt_len > m.max_position) {
      err << "request " << r << ": prompt_len " << q.prompt_len
          << " exceeds max_position " << m.max_position;
      return fail(TSR_ERR_OUT_OF_RANGE, err.str());
    }
    if (q.miss_scope != TSR_SCOPE_GLOBAL && q.miss_scope != TSR_SCOPE_LOCAL) {
      err << "request " << r << ": miss_scope must be TSR_SCOPE_GLOBAL or TSR_SCOPE_LOCAL";
      return fail(TSR_ERR_INVALID_ARG, err.str());
    }
    const bool local = q.miss_scope == TSR_SCOPE_LOCAL;
    if (q.n_units < 0 || q.n_text < 0 || (q.n_units && !q.units) ||
        (q.n_text && !q.text_segs) || !q.block_table) {
      err << "request " << r << ": null or negative-size member";
      return fail(TSR_ERR_INVALID_ARG, err.str());
    }
    // tiling: segments sorted by start must cover [0, prompt_len) once
    std::vector<Seg> segs;
    segs.reserve(q.n_units + q.n_text);
    for (int t = 0; t < q.n_text; ++t)
      segs.push_back({q.text_segs[2 * t], q.text_segs[2 * t + 1], -1});
    for (int u = 0; u < q.n_units; ++u)
      segs.push_back({q.units[u].position, q.units[u].n_tokens, u});
    std::stable_sort(segs.begin(), segs.end(),
                     [](const Seg& a, const Seg& b) { return a.start < b.start; });
    int32_t expect = 0;
    int last_unit = -1;
    for (const Seg& s : segs) {
      if (s.len <= 0 || s.start != expect) {
        err << "request " << r << ": segments do not tile the prompt (segment at "
            << s.start << " length " << s.len << ", expected start " << expect << ")";
        return fail(TSR_ERR_INVALID_ARG, err.str());
      }
      if (s.unit >= 0) {
        if (s.unit < last_unit) {
          err << "request " << r << ": units are not in prompt order";
          return fail(TSR_ERR_INVALID_ARG, err.str());
        }
        last_unit = s.unit;
      }
      expect += s.len;
    }
    if (expect != q.prompt_len) {
      err << "request " << r << ": segments cover " << expect
          << " tokens but prompt_len is " << q.prompt_len;
      return fail(TSR_ERR_INVALID_ARG, err.str());
    }
    if (e4m3) {
      // every request page must have a single writer (its scale is computed
      // from its own values): segments and recompute windows page aligned
      for (const Seg& sg : segs) {
        const int32_t end = sg.start + sg.len;
        bool ok = sg.start % B == 0 && (end % B == 0 || end == q.prompt_len);
        if (ok && sg.unit >= 0 && q.units[sg.unit].residency == TSR_HIT) {
          const tsr_unit& u = q.units[sg.unit];
          const int32_t rc = std::max(0, std::min(u.n_recompute, u.n_tokens));
          ok = rc % B == 0 || rc == u.n_tokens;
        }
        if (!ok) {
          err << "request " << r << ": e4m3 plans must be page aligned (segment at "
              << sg.start << " length " << sg.len << ")";
          return fail(TSR_ERR_UNSUPPORTED, err.str());
        }
      }
    }
    // block table
    const int npg = (q.prompt_len + B - 1) / B;
    bt_off[r] = (int32_t)bts.size();
    bt_len[r] = npg;
    for (int i = 0; i < npg; ++i) {
      int32_t pg = q.block_table[i];
      if (pg < 0 || pg >= n_req_pages) {
        err << "request " << r << ": block_table[" << i << "] = " << pg
            << " outside the request arena of " << n_req_pages << " pages";
        return fail(TSR_ERR_OUT_OF_RANGE, err.str());
      }
      if (req_page_used[pg]) {
        err << "request " << r << ": request page " << pg << " is used twice";
        return fail(TSR_ERR_INVALID_ARG, err.str());
      }
      req_page_used[pg] = 1;
      bts.push_back(pg);
      vbts.push_back(pg);
      kbts.push_back(pg);
    }
    auto req_slot = [&](int32_t pos) {
      return q.block_table[pos / B] * B + pos % B;
    };
    // walk the prompt in position order
    for (const Seg& s : segs) {
      if (s.unit < 0) {
        if (e4m3)
          for (int32_t j = 0; j < s.len; j += B)
            apages.push_back({(int32_t)rows.size() + j, q.block_table[(s.start + j) / B],
                              s.start + j, std::min(B, s.len - j)});
        for (int32_t j = 0; j < s.len; ++j) {
          rows.push_back({req_slot(s.start + j), s.start + j});
          p->row_pos.push_back(s.start + j);
          p->row_req.push_back(r);
          p->row_lo.push_back(0);
        }
        continue;
      }
      const tsr_unit& u = q.units[s.unit];
      if (u.residency != TSR_HIT && u.residency != TSR_MISS) {
        err << "request " << r << " unit " << s.unit << ": residency must be HIT or MISS";
        return fail(TSR_ERR_INVALID_ARG, err.str());
      }
      if (u.retain != 0 && u.retain != 1) {
        err << "request " << r << " unit " << s.unit << ": retain must be 0 or 1";
        return fail(TSR_ERR_INVALID_ARG, err.str());
      }
      if ((u.residency == TSR_HIT || local) && u.n_recompute < 0) {
        err << "request " << r << " unit " << s.unit << ": n_recompute < 0";
        return fail(TSR_ERR_INVALID_ARG, err.str());
      }
      const bool hit = u.residency == TSR_HIT;
      const bool keep = !hit && u.retain == 1;
      const int upg = (u.n_tokens + B - 1) / B;
      if ((hit || keep) && !u.pool_pages) {
        err << "request " << r << " unit " << s.unit << ": pool_pages is NULL";
        return fail(TSR_ERR_INVALID_ARG, err.str());
      }
      if (hit || keep) {
        for (int i = 0; i < upg; ++i) {
          int32_t pg = u.pool_pages[i];
          if (pg < 0 || pg >= n_pool_pages) {
            err << "request " << r << " unit " << s.unit << ": pool page " << pg
                << " outside the pool arena of " << n_pool_pages << " pages";
            return fail(TSR_ERR_OUT_OF_RANGE, err.str());
          }
          if (keep) {
            if (pool_use[pg] & 2) {
              err << "request " << r << " unit " << s.unit << ": pool page " << pg
                  << " is retained twice in this batch";
              return fail(TSR_ERR_INVALID_ARG, err.str());
            }
            pool_use[pg] |= 2;
          } else {
            pool_use[pg] |= 1;
          }
        }
      }
      const int32_t ncomp = hit ? std::min(u.n_recompute, u.n_tokens) : u.n_tokens;
      const int32_t row0 = (int32_t)rows.size();
      if (e4m3) {
        for (int32_t j = 0; j < ncomp; j += B)
          apages.push_back({row0 + j, q.block_table[(u.position + j) / B], u.position + j,
                            std::min(B, ncomp - j)});
        if (hit)
          for (int32_t j = ncomp; j < u.n_tokens; j += B)
            gpages.push_back({u.pool_pages[j / B], q.block_table[(u.position + j) / B],
                              u.position + j, std::min(B, u.n_tokens - j)});
        else if (keep)
          for (int32_t j = 0; j < u.n_tokens; j += B)
            rpages.push_back({row0 + j, u.pool_pages[j / B], u.position + j,
                              std::min(B, u.n_tokens - j)});
      }
      // under the local scope a MISS unit's tokens past its recompute window
      // see only their own unit
      const int32_t wnd = (!hit && local) ? std::min(u.n_recompute, u.n_tokens) : ncomp;
      for (int32_t j = 0; j < ncomp; ++j) {
        rows.push_back({req_slot(u.position + j), u.position + j});
        p->row_pos.push_back(u.position + j);
        p->row_req.push_back(r);
        p->row_lo.push_back(j < wnd ? 0 : u.position);
      }
      if (hit) {
        if (ncomp < u.n_tokens)
          gathered[r].push_back({u.position + ncomp, u.position + u.n_tokens});
        // Aliasing: a request page that holds B gathered tokens of this
        // unit, slot for slot (the unit starts on a page boundary), reads
        // its V (alias_v) and/or its pre-RoPE K (alias_k, rotated on load)
        // from the pool page; compose then skips that half (both: the
        // tokens are not moved at all)
        int32_t ab0 = 0, ab1 = 0;              // aliasable unit blocks [ab0, ab1)
        if ((alias_v || alias_k) && u.position % B == 0) {
          ab0 = (ncomp + B - 1) / B;
          ab1 = std::max(ab0, u.n_tokens / B);
          for (int32_t b = ab0; b < ab1; ++b) {
            if (alias_v)
              vbts[bt_off[r] + u.position / B + b] = u.pool_pages[b] | kPoolPageFlag;
            if (alias_k)
              kbts[bt_off[r] + u.position / B + b] = u.pool_pages[b] | kPoolPageFlag;
          }
          if (alias_v) p->n_aliased += ab1 - ab0;
          if (alias_k) p->n_aliased_k += ab1 - ab0;
        }
        const int32_t skip = (alias_v ? kSkipV : 0) | (alias_k ? kSkipK : 0);
        for (int32_t j = ncomp; j < u.n_tokens; ++j) {
          const bool aliased = j / B >= ab0 && j / B < ab1;
          if (aliased && skip == (kSkipV | kSkipK)) continue;   // nothing to move
          gather.push_back({u.pool_pages[j / B] * B + j % B, req_slot(u.position + j),
                            u.position + j, aliased ? skip : 0});
        }
      } else if (keep) {
        for (int32_t j = 0; j < u.n_tokens; ++j)
          retain.push_back({row0 + j, u.pool_pages[j / B] * B + j % B});
      }
    }
    req_row0[r + 1] = (int32_t)rows.size();
  }
  for (int32_t pg = 0; pg < n_pool_pages; ++pg) {
    if (pool_use[pg] == 3) {
      err << "pool page " << pg << " is both read by a HIT and written by a retained "
          << "unit in this batch";
      return fail(TSR_ERR_INVALID_ARG, err.str());
    }
  }
  const size_t limit = (size_t)INT32_MAX;
  if (rows.size() >= limit || gather.size() >= limit) {
    return fail(TSR_ERR_OUT_OF_RANGE, "batch too large");
  }

  // attention items: up to rb * kTileRows consecutive rows (in item row
  // order) x KV heads
  // The MFMA kernels give each of their 4 waves per row block one query
  // head; a larger GQA group is split over several items that read the same
  // K/V tiles (adjacent in the launch order, so the repeat reads hit L2).
  const int G = m.n_q_heads / Hkv;
  const int hsplit = (m.act_dtype == TSR_BF16 && G > 4) ? G / 4 : 1;
  // Row order of the items: the computed order, or (grouped) each
  // request's rows stably sorted by first visible key.  Under the LOCAL
  // scope the rows that see the whole prompt (text, recompute windows) come
  // in short runs between the unit-local rows of missed units; grouped,
  // they fill whole row blocks (their positions stay ascending, so an
  // item's first and last rows still bound its positions).
  const int32_t T = (int32_t)rows.size();
  std::vector<int32_t> ord((size_t)T), grouped((size_t)T);
  std::iota(ord.begin(), ord.end(), 0);
  std::iota(grouped.begin(), grouped.end(), 0);
  for (int r = 0; r < n_req; ++r)
    std::stable_sort(grouped.begin() + req_row0[r], grouped.begin() + req_row0[r + 1],
                     [&](int32_t a, int32_t b) { return p->row_lo[a] < p->row_lo[b]; });
  struct Item { AttnItem it; int64_t cost; int group; int part; };
  std::vector<Item> items;
  int32_t max_kv = 0;
  int64_t max_blocks = 0;   // most 16-key blocks an item's key tiles span
  // Builds the items for row blocks of kTileRows rows, rb per item; returns
  // the share of the items' (row block x key tile) slots that hold keys a
  // row block needs (a row block skips the tiles past its last row).
  auto build_items = [&](int rb, bool group_rows = false) -> double {
    if (group_rows) ord = grouped;
    else std::iota(ord.begin(), ord.end(), 0);
    const auto pos_at = [&](int32_t i) { return p->row_pos[ord[i]]; };
    const auto lo_at = [&](int32_t i) { return p->row_lo[ord[i]]; };
    items.clear();
    max_kv = 0;
    max_blocks = 0;
    const int32_t tile_rows = kTileRows * rb;
    int64_t need = 0, slots = 0;
    for (int r = 0; r < n_req; ++r) {
      // runs of consecutive rows with the same first visible key
      for (int32_t a0 = req_row0[r]; a0 < req_row0[r + 1];) {
        int32_t a1 = a0 + 1;
        while (a1 < req_row0[r + 1] && lo_at(a1) == lo_at(a0)) ++a1;
        const int32_t kv_lo = lo_at(a0);
        for (int32_t t0 = a0; t0 < a1; t0 += tile_rows) {
          const int32_t n = std::min(tile_rows, a1 - t0);
          const int32_t lo = pos_at(t0), hi = pos_at(t0 + n - 1);
          int32_t crow0 = ord[t0];
          for (int32_t i = 1; i < n && crow0 >= 0; ++i)
            if (ord[t0 + i] != ord[t0] + i || pos_at(t0 + i) != lo + i) crow0 = -1;
          max_kv = std::max(max_kv, hi + 1);
          const int32_t t_lo = kv_lo / kMfmaKeys;
          max_blocks = std::max<int64_t>(max_blocks, 2 * ((int64_t)hi / kMfmaKeys + 1 - t_lo));
          slots += (int64_t)rb * (hi / kMfmaKeys + 1 - t_lo);
          for (int32_t b0 = 0; b0 < n; b0 += kTileRows)
            need += pos_at(t0 + std::min(n, b0 + kTileRows) - 1) / kMfmaKeys + 1 - t_lo;
          // part 1 if a gathered position lies in the key tiles the kernels
          // load for this item (masked keys included): [tile of kv_lo, end
          // of the tile of hi]
          const int32_t klo = kv_lo / kKvTile * kKvTile;
          const int32_t khi = (hi / kKvTile + 1) * kKvTile;
          int part = 0;
          for (const auto& iv : gathered[r])
            if (iv.first < khi && iv.second > klo) part = 1;
          for (int g = 0; g < Hkv; ++g)
            for (int hs = 0; hs < hsplit; ++hs) {
              AttnItem a{t0, n, hi + 1, lo, g, bt_off[r], bt_len[r], 4 * hs, kv_lo, -1, 0,
                         crow0, {0, 0}, {0, 0, 0}};
              items.push_back({a, (int64_t)(hi + 1 - kv_lo), r * Hkv + g, part});
            }
        }
        a0 = a1;
      }
    }
    return slots ? (double)need / (double)slots : 1.0;
  };
  // The MFMA kernels (bf16 and e4m3 KV) run kMaxRowBlocks row blocks per
  // workgroup (their K/V staging then serves three times the rows) unless
  // short runs of rows (unit-local attention) would leave too many row
  // blocks idle, or the batch has fewer such items than the GPU has compute
  // units (one three-row-block workgroup fills a unit; one-row-block
  // workgroups run three to a unit); the fp32 kernel takes one row block.
  // Both kernels cut their three-row-block items from rows grouped by first
  // visible key (AttnRow order); one-row-block plans keep the computed
  // order.
  // attn_kernel (1 and 2 for bf16 KV only): 1 the pipelined kernel
  // (attn_pipe.hip, two row blocks per item; it cannot rotate K on load and
  // its page-id table bounds an item's keys; measured slower than the
  // row-block kernel on the RAG batches), 2 the row-block kernel under the
  // rule above (as 0), 3 / 4 the row-block kernel (or the e4m3 kernel) with
  // three / one row blocks.
  p->row_blocks = 1;
  const bool bf16_kv = m.act_dtype == TSR_BF16 && m.kv_dtype == TSR_BF16;
  auto split_threshold = [&](int64_t total_tiles) -> int64_t {
    return split_tiles > 0 ? split_tiles
                           : std::max<int64_t>(kMinSplitTiles,
                                               (total_tiles + kSplitSlots - 1) / kSplitSlots);
  };
  const bool mfma = m.act_dtype == TSR_BF16 &&
                    (m.kv_dtype == TSR_BF16 || m.kv_dtype == TSR_E4M3);
  if (bf16_kv && attn_kernel == 1) {
    build_items(kPipeRowBlocks);
    if (alias_k || max_blocks > kPipeMaxBlocks)
      return fail(TSR_ERR_UNSUPPORTED,
                  alias_k ? "the pipelined attention kernel does not rotate K on load"
                          : "an attention item spans more keys than the pipelined kernel takes");
    p->row_blocks = kPipeRowBlocks;
  } else if (mfma && attn_kernel == 3) {
    build_items(kMaxRowBlocks, true);
    p->row_blocks = kMaxRowBlocks;
  } else if (mfma && attn_kernel == 4) {
    build_items(1);
  } else if (mfma && build_items(kMaxRowBlocks, true) >= kMinGroupedRowBlockUse &&
             (int64_t)items.size() >= kNumCus) {
    p->row_blocks = kMaxRowBlocks;
  } else {
    build_items(1);
  }
  p->rows_grouped = !std::is_sorted(ord.begin(), ord.end());
  std::vector<AttnRow> attn_rows((size_t)T);
  for (int32_t i = 0; i < T; ++i) attn_rows[i] = AttnRow{ord[i], p->row_pos[ord[i]]};
  // Key-range split (bf16 plans of the row-block kernel): the launch
  // lasts as long as its longest item, so an item spanning more than S key
  // tiles runs as up to n = ceil(tiles / S) items over consecutive key
  // ranges.  Every range but the first starts on a tile boundary above
  // kv_lo and at or below the smallest row position, so every row sees at
  // least one key of every range and only the last range needs the causal
  // mask; each range writes one split buffer slot per row block (a row
  // block's n ranges in consecutive slots) and the merge kernel combines
  // each row block's n slots.  Ranges inherit the item's part (a part-0
  // item's ranges read no gathered key either).
  std::vector<CombineDesc> combine[2];
  int32_t n_slots = 0, n_split_items = 0;
  // The automatic threshold (split_tiles == 0) applies to one-row-block
  // plans only: on the LOCAL-scope RAG batch at three row blocks it split 64
  // items and the launch plus merge took 4 % longer (one workgroup per
  // compute unit there, so an item's tail is shared by fewer waiting
  // items); split_tiles > 0 splits either.
  const int rb_split = p->row_blocks;
  if ((split_tiles > 0 || (split_tiles == 0 && rb_split == 1)) &&
      (rb_split == 1 || rb_split == kMaxRowBlocks) &&
      m.act_dtype == TSR_BF16 && m.kv_dtype == TSR_BF16 && !items.empty()) {
    auto tiles_of = [](const AttnItem& a) -> int64_t {
      return (a.kv_len + kMfmaKeys - 1) / kMfmaKeys - a.kv_lo / kMfmaKeys;
    };
    int64_t total = 0;
    for (const Item& x : items) total += tiles_of(x.it);
    int64_t S = split_threshold(total);
    auto slots_for = [&](int64_t lim) {
      int64_t n = 0;
      for (const Item& x : items) {
        const int64_t t = tiles_of(x.it);
        if (t > lim) n += rb_split * ((t + lim - 1) / lim);
      }
      return n;
    };
    while (slots_for(S) > kMaxSplitSlots) S *= 2;
    std::vector<Item> split;
    split.reserve(items.size());
    for (const Item& x : items) {
      const AttnItem& a = x.it;
      const int32_t j0 = a.kv_lo / kMfmaKeys;
      const int32_t ntl = (a.kv_len + kMfmaKeys - 1) / kMfmaKeys;
      const int64_t t = ntl - j0;
      // interior boundaries: strictly increasing in (j0, top] with top the
      // tile of the smallest row position, so that every range starts at a
      // key every row sees (no row of a range is left without a visible
      // key) and only the last range holds keys past a row's position
      const int32_t top = std::min(ntl - 1, a.min_pos / kMfmaKeys);
      const int64_t n = std::min<int64_t>((t + S - 1) / S, (int64_t)top - j0 + 1);
      if (t <= S || n < 2) {
        split.push_back(x);
        continue;
      }
      std::vector<int32_t> b((size_t)n + 1);
      b[0] = j0;
      b[n] = ntl;
      for (int64_t c = 1; c < n; ++c)
        b[c] = std::min<int32_t>(top - (int32_t)(n - 1 - c), j0 + (int32_t)((c * t + n / 2) / n));
      for (int64_t c = 1; c < n; ++c) b[c] = std::max(b[c], b[c - 1] + 1);
      for (int64_t c = 0; c < n; ++c) {
        Item y = x;
        y.it.kv_lo = c == 0 ? a.kv_lo : b[c] * kMfmaKeys;
        y.it.kv_len = c == n - 1 ? a.kv_len : b[c + 1] * kMfmaKeys;
        y.it.part_slot = n_slots + (int32_t)c;
        y.it.n_parts = (int32_t)n;
        y.cost = (int64_t)(b[c + 1] - b[c]) * kMfmaKeys;
        split.push_back(y);
      }
      for (int blk = 0; blk < rb_split; ++blk) {
        const int32_t nr = std::min(kTileRows, a.n_rows - kTileRows * blk);
        if (nr > 0)
          combine[x.part].push_back(CombineDesc{a.row0 + kTileRows * blk, nr,
                                                a.kv_head * G + a.head0,
                                                std::min(G, kSplitHeads),
                                                n_slots + blk * (int32_t)n, (int32_t)n, {0, 0}});
      }
      n_slots += rb_split * (int32_t)n;
      ++n_split_items;
    }
    items.swap(split);
  }
  // XCD-aware order: (request, KV head) groups share K/V, so each group is
  // bound to one XCD bin (workgroup w runs on XCD w % kNumXcd); bins are
  // balanced by cost (longest group first onto the lightest bin) and each
  // bin is issued longest item first (measured: issuing a bin group by
  // group for L2 locality lost more to the tail than it gained).  Short bins
  // are padded with empty items.  The full schedule and each part's are
  // built the same way.
  std::stable_sort(items.begin(), items.end(),
                   [](const Item& a, const Item& b) { return a.cost > b.cost; });
  auto schedule = [&](int part) {
    std::vector<int64_t> gcost((size_t)std::max(1, n_req * Hkv), 0);
    for (const Item& x : items)
      if (part < 0 || x.part == part) gcost[x.group] += x.cost;
    std::vector<int> gorder(gcost.size());
    std::iota(gorder.begin(), gorder.end(), 0);
    std::stable_sort(gorder.begin(), gorder.end(),
                     [&](int a, int b) { return gcost[a] > gcost[b]; });
    std::vector<int> gbin(gcost.size(), 0);
    int64_t bin_load[kNumXcd] = {0};
    for (int g : gorder) {
      int best = 0;
      for (int b = 1; b < kNumXcd; ++b)
        if (bin_load[b] < bin_load[best]) best = b;
      gbin[g] = best;
      bin_load[best] += gcost[g];
    }
    std::vector<std::vector<AttnItem>> bins(kNumXcd);
    std::vector<const Item*> sel;
    for (const Item& x : items)
      if (part < 0 || x.part == part) sel.push_back(&x);
    int n_groups = 0;
    for (int64_t c : gcost) n_groups += c > 0;
    if (n_groups >= kGroupMajorMinGroups * kNumXcd && !sel.empty()) {
      // many (request, KV head) groups per bin: within each third of the
      // cost range (longest third first) issue a bin's items group by
      // group, so the compute units of an XCD work on few groups at a time
      // and their K/V stays in the caches; the cost thirds keep the longest
      // items first
      std::vector<int> grank(gcost.size());
      for (size_t i = 0; i < gorder.size(); ++i) grank[gorder[i]] = (int)i;
      std::vector<int64_t> cs;
      for (const Item* x : sel) cs.push_back(x->cost);
      std::sort(cs.begin(), cs.end());
      const int64_t c1 = cs[cs.size() * 2 / 3], c2 = cs[cs.size() / 3];
      auto tier = [&](int64_t c) { return c >= c1 ? 0 : (c >= c2 ? 1 : 2); };
      std::stable_sort(sel.begin(), sel.end(), [&](const Item* a, const Item* b) {
        const int ta = tier(a->cost), tb = tier(b->cost);
        return ta != tb ? ta < tb : grank[a->group] < grank[b->group];
      });
    }
    for (const Item* x : sel) bins[gbin[x->group]].push_back(x->it);
    size_t per_bin = 0;
    for (auto& b : bins) per_bin = std::max(per_bin, b.size());
    std::vector<AttnItem> order;
    order.reserve(per_bin * kNumXcd);
    for (size_t i = 0; i < per_bin; ++i)
      for (int b = 0; b < kNumXcd; ++b)
        order.push_back(i < bins[b].size() ? bins[b][i]
                                           : AttnItem{0, 0, 0, 0, 0, 0, 0, 0, 0, -1, 0, -1,
                                                      {0, 0}, {0, 0, 0}});
    return order;
  };
  std::vector<AttnItem> order = schedule(-1);
  std::vector<AttnItem> order_part[2] = {schedule(0), schedule(1)};
  // first key tile's page ids, from the block table the kernels read for K
  {
    const std::vector<int32_t>& kt = alias_k ? kbts : bts;
    for (std::vector<AttnItem>* list : {&order, &order_part[0], &order_part[1]})
      for (AttnItem& a : *list) {
        if (a.n_rows == 0) continue;
        const int32_t key0 = a.kv_lo / kMfmaKeys * kMfmaKeys;
        for (int b = 0; b < 2; ++b)
          a.pg[b] = kt[a.bt_off + std::min((key0 + 16 * b) / B, a.n_pages - 1)];
      }
  }

  p->T = (int32_t)rows.size();
  p->n_gather = (int32_t)gather.size();
  p->n_retain = (int32_t)retain.size();
  p->n_items = (int32_t)order.size();
  for (int q = 0; q < 2; ++q) p->n_items_part[q] = (int32_t)order_part[q].size();
  p->max_kv_len = max_kv;

  // device image: arrays at 256-byte aligned offsets
  size_t off = 0;
  p->off_gather = off;  off = align_up(off + gather.size() * sizeof(GatherDesc), 256);
  p->off_rows = off;    off = align_up(off + rows.size() * sizeof(RowDesc), 256);
  p->off_attn_rows = off; off = align_up(off + attn_rows.size() * sizeof(AttnRow), 256);
  p->off_retain = off;  off = align_up(off + retain.size() * sizeof(RetainDesc), 256);
  p->off_items = off;   off = align_up(off + order.size() * sizeof(AttnItem), 256);
  for (int q = 0; q < 2; ++q) {
    p->off_items_part[q] = off;
    off = align_up(off + order_part[q].size() * sizeof(AttnItem), 256);
  }
  p->off_bt = off;      off = align_up(off + bts.size() * sizeof(int32_t), 256);
  p->off_vbt = off;     off = align_up(off + vbts.size() * sizeof(int32_t), 256);
  p->off_kbt = off;     off = align_up(off + kbts.size() * sizeof(int32_t), 256);
  p->off_gpages = off;  off = align_up(off + gpages.size() * sizeof(PageDesc), 256);
  p->off_apages = off;  off = align_up(off + apages.size() * sizeof(PageDesc), 256);
  p->off_rpages = off;  off = align_up(off + rpages.size() * sizeof(PageDesc), 256);
  p->n_combine_part[0] = (int32_t)combine[0].size();
  p->n_combine_part[1] = (int32_t)combine[1].size();
  p->n_combine = p->n_combine_part[0] + p->n_combine_part[1];
  p->n_split_slots = n_slots;
  p->n_split_items = n_split_items;
  p->off_combine = off; off = align_up(off + p->n_combine * sizeof(CombineDesc), 256);
  // the split buffer is written by the kernels, not uploaded
  p->image_bytes = std::max<size_t>(off, 256);
  const size_t slot_rows = (size_t)n_slots * kTileRows * kSplitHeads;
  p->off_split_o = off;   off = align_up(off + slot_rows * m.head_dim * sizeof(float), 256);
  p->off_split_lse = off; off = align_up(off + slot_rows * sizeof(float), 256);
  p->n_gpages = (int32_t)gpages.size();
  p->n_apages = (int32_t)apages.size();
  p->n_rpages = (int32_t)rpages.size();
  p->ws_bytes = std::max<size_t>(off, 256);
  p->image.assign(p->image_bytes, 0);
  auto put = [&](size_t o, const void* src, size_t n) {
    if (n) std::memcpy(p->image.data() + o, src, n);
  };
  put(p->off_gather, gather.data(), gather.size() * sizeof(GatherDesc));
  put(p->off_rows, rows.data(), rows.size() * sizeof(RowDesc));
  put(p->off_attn_rows, attn_rows.data(), attn_rows.size() * sizeof(AttnRow));
  put(p->off_retain, retain.data(), retain.size() * sizeof(RetainDesc));
  put(p->off_items, order.data(), order.size() * sizeof(AttnItem));
  for (int q = 0; q < 2; ++q)
    put(p->off_items_part[q], order_part[q].data(), order_part[q].size() * sizeof(AttnItem));
  put(p->off_bt, bts.data(), bts.size() * sizeof(int32_t));
  put(p->off_vbt, vbts.data(), vbts.size() * sizeof(int32_t));
  put(p->off_kbt, kbts.data(), kbts.size() * sizeof(int32_t));
  put(p->off_gpages, gpages.data(), gpages.size() * sizeof(PageDesc));
  put(p->off_apages, apages.data(), apages.size() * sizeof(PageDesc));
  put(p->off_rpages, rpages.data(), rpages.size() * sizeof(PageDesc));
  put(p->off_combine, combine[0].data(), combine[0].size() * sizeof(CombineDesc));
  put(p->off_combine + combine[0].size() * sizeof(CombineDesc), combine[1].data(),
      combine[1].size() * sizeof(CombineDesc));
  return TSR_OK;
}

}  // namespace tsr

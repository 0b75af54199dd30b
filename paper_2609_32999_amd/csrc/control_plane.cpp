// Retrieval-aware cache management and routing (Section 5.2): reuse
// scoring, threshold admission with block-accounted eviction, cache-aware
// routing, and a trace replay of them.  Host code only.
#include <algorithm>
#include <cmath>
#include <deque>
#include <string>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "../../include/tsr_control.h"
#include "tsr_internal.h"

struct tsr_scorer {
  int32_t window = 1;
  double w_recent = 1.0, w_lifetime = 0.05;
  std::deque<std::vector<uint64_t>> last;            // the last `window` requests
  std::unordered_map<uint64_t, int32_t> recent;      // f_W
  std::unordered_map<uint64_t, int64_t> lifetime;    // f_inf
};

struct tsr_admitter {
  int64_t capacity = 0, used = 0;
  double theta = 0.0;
  std::unordered_map<uint64_t, int32_t> resident;    // unit -> blocks
};

using tsr::guarded;
using tsr::set_error;

namespace {

// A request's units in retrieval order, each once.
std::vector<uint64_t> distinct(const uint64_t* ids, int32_t n) {
  std::vector<uint64_t> v;
  std::unordered_set<uint64_t> seen;
  for (int32_t i = 0; i < n; ++i)
    if (seen.insert(ids[i]).second) v.push_back(ids[i]);
  return v;
}

void observe(tsr_scorer* s, std::vector<uint64_t> units) {
  for (uint64_t u : units) {
    ++s->recent[u];
    ++s->lifetime[u];
  }
  s->last.push_back(std::move(units));
  if ((int32_t)s->last.size() > s->window) {
    for (uint64_t u : s->last.front()) {
      auto it = s->recent.find(u);
      if (--it->second == 0) s->recent.erase(it);
    }
    s->last.pop_front();
  }
}

double score(const tsr_scorer* s, uint64_t u) {
  auto r = s->recent.find(u);
  auto l = s->lifetime.find(u);
  const double fr = r == s->recent.end() ? 0.0 : (double)r->second;
  const double fl = l == s->lifetime.end() ? 0.0 : (double)l->second;
  return s->w_recent * fr + s->w_lifetime * fl;
}

// The admission rule; victims are appended to `out` only if admitted.
int32_t decide(tsr_admitter* a, const tsr_scorer* sc, uint64_t u, int32_t nb,
               std::vector<uint64_t>* out) {
  if (a->resident.count(u)) return TSR_ADMIT_RESIDENT;
  const double su = score(sc, u);
  if (su < a->theta) return TSR_ADMIT_BELOW_THRESHOLD;
  if (nb > a->capacity) return TSR_ADMIT_TOO_LARGE;
  int64_t room = a->capacity - a->used;
  if (room < nb) {
    // resident units scoring strictly lower, lowest first (ties by id)
    std::vector<std::pair<double, uint64_t>> lower;
    for (const auto& kv : a->resident) {
      const double sv = score(sc, kv.first);
      if (sv < su) lower.push_back({sv, kv.first});
    }
    std::sort(lower.begin(), lower.end());
    size_t k = 0;
    while (room < nb && k < lower.size()) room += a->resident.at(lower[k++].second);
    if (room < nb) return TSR_ADMIT_NO_ROOM;
    for (size_t i = 0; i < k; ++i) out->push_back(lower[i].second);
  }
  return TSR_ADMIT_ADMITTED;
}

void apply(tsr_admitter* a, uint64_t u, int32_t nb, const std::vector<uint64_t>& victims) {
  for (uint64_t v : victims) {
    a->used -= a->resident.at(v);
    a->resident.erase(v);
  }
  a->resident[u] = nb;
  a->used += nb;
}

int32_t route(const tsr_admitter* const* nodes, const int32_t* inflight, int32_t n,
              const std::vector<uint64_t>& units, uint32_t* rr) {
  int32_t least = inflight[0];
  for (int32_t i = 1; i < n; ++i) least = std::min(least, inflight[i]);
  int32_t best = -1;
  int64_t best_blocks = -1;
  int32_t best_load = 0;
  // scan from the round-robin cursor so that the first of equal nodes wins
  for (int32_t k = 0; k < n; ++k) {
    const int32_t i = (int32_t)((*rr + (uint32_t)k) % (uint32_t)n);
    if (inflight[i] > least + 1) continue;
    int64_t blocks = 0;
    if (nodes && nodes[i])
      for (uint64_t u : units) {
        auto it = nodes[i]->resident.find(u);
        if (it != nodes[i]->resident.end()) blocks += it->second;
      }
    if (blocks > best_blocks || (blocks == best_blocks && inflight[i] < best_load)) {
      best = i;
      best_blocks = blocks;
      best_load = inflight[i];
    }
  }
  *rr = (uint32_t)((best + 1) % n);
  return best;
}

}  // namespace

extern "C" {

tsr_status tsr_scorer_create(int32_t window, double w_recent, double w_lifetime,
                             tsr_scorer** out) {
  return guarded([&]() -> tsr_status {
    if (!out || window < 1 || !std::isfinite(w_recent) || !std::isfinite(w_lifetime)) {
      set_error("tsr_scorer_create: out is NULL, window < 1 or a weight is not finite");
      return TSR_ERR_INVALID_ARG;
    }
    auto* s = new tsr_scorer;
    s->window = window;
    s->w_recent = w_recent;
    s->w_lifetime = w_lifetime;
    *out = s;
    return TSR_OK;
  });
}

void tsr_scorer_destroy(tsr_scorer* s) { delete s; }

tsr_status tsr_scorer_observe(tsr_scorer* s, const uint64_t* unit_ids, int32_t n) {
  return guarded([&]() -> tsr_status {
    if (!s || n < 0 || (n > 0 && !unit_ids)) {
      set_error("tsr_scorer_observe: NULL scorer or unit list, or n < 0");
      return TSR_ERR_INVALID_ARG;
    }
    observe(s, distinct(unit_ids, n));
    return TSR_OK;
  });
}

double tsr_scorer_score(const tsr_scorer* s, uint64_t unit_id) {
  return s ? score(s, unit_id) : 0.0;
}

tsr_status tsr_scorer_counts(const tsr_scorer* s, uint64_t unit_id, int32_t* recent,
                             int64_t* lifetime) {
  if (!s) {
    set_error("tsr_scorer_counts: scorer is NULL");
    return TSR_ERR_INVALID_ARG;
  }
  auto r = s->recent.find(unit_id);
  auto l = s->lifetime.find(unit_id);
  if (recent) *recent = r == s->recent.end() ? 0 : r->second;
  if (lifetime) *lifetime = l == s->lifetime.end() ? 0 : l->second;
  return TSR_OK;
}

int32_t tsr_window_for_capacity(int64_t capacity_blocks, double mean_blocks_per_request) {
  if (!(mean_blocks_per_request > 0.0) || capacity_blocks <= 0) return 1;
  const double w = std::floor((double)capacity_blocks / mean_blocks_per_request);
  return (int32_t)std::max(1.0, std::min(w, 1.0e9));
}

tsr_status tsr_admitter_create(int64_t capacity_blocks, double theta, tsr_admitter** out) {
  return guarded([&]() -> tsr_status {
    if (!out || capacity_blocks < 0 || !std::isfinite(theta)) {
      set_error("tsr_admitter_create: out is NULL, capacity < 0 or theta not finite");
      return TSR_ERR_INVALID_ARG;
    }
    auto* a = new tsr_admitter;
    a->capacity = capacity_blocks;
    a->theta = theta;
    *out = a;
    return TSR_OK;
  });
}

void tsr_admitter_destroy(tsr_admitter* a) { delete a; }

tsr_status tsr_admit(tsr_admitter* a, const tsr_scorer* scorer, uint64_t unit_id,
                     int32_t n_blocks, int32_t* result, uint64_t* victims,
                     int32_t max_victims, int32_t* n_victims) {
  return guarded([&]() -> tsr_status {
    if (!a || !scorer || !result || !n_victims || n_blocks <= 0 || max_victims < 0 ||
        (max_victims > 0 && !victims)) {
      set_error("tsr_admit: NULL argument, n_blocks <= 0 or max_victims < 0");
      return TSR_ERR_INVALID_ARG;
    }
    std::vector<uint64_t> v;
    const int32_t r = decide(a, scorer, unit_id, n_blocks, &v);
    *n_victims = (int32_t)v.size();
    if ((int32_t)v.size() > max_victims) {
      set_error("tsr_admit: " + std::to_string(v.size()) + " victims, room for " +
                std::to_string(max_victims));
      return TSR_ERR_OUT_OF_RANGE;
    }
    if (r == TSR_ADMIT_ADMITTED) apply(a, unit_id, n_blocks, v);
    std::copy(v.begin(), v.end(), victims);
    *result = r;
    return TSR_OK;
  });
}

tsr_status tsr_admitter_remove(tsr_admitter* a, uint64_t unit_id) {
  if (!a) {
    set_error("tsr_admitter_remove: admitter is NULL");
    return TSR_ERR_INVALID_ARG;
  }
  auto it = a->resident.find(unit_id);
  if (it == a->resident.end()) {
    set_error("unit " + std::to_string(unit_id) + " is not resident");
    return TSR_ERR_STATE;
  }
  a->used -= it->second;
  a->resident.erase(it);
  return TSR_OK;
}

int32_t tsr_admitter_blocks(const tsr_admitter* a, uint64_t unit_id) {
  if (!a) return 0;
  auto it = a->resident.find(unit_id);
  return it == a->resident.end() ? 0 : it->second;
}

int64_t tsr_admitter_used_blocks(const tsr_admitter* a) { return a ? a->used : -1; }

int32_t tsr_admitter_num_units(const tsr_admitter* a) {
  return a ? (int32_t)a->resident.size() : -1;
}

tsr_status tsr_route(const tsr_admitter* const* node_caches, const int32_t* inflight,
                     int32_t n_nodes, const uint64_t* unit_ids, int32_t n_units,
                     uint32_t* rr_cursor, int32_t* chosen) {
  return guarded([&]() -> tsr_status {
    if (n_nodes < 1 || !inflight || !rr_cursor || !chosen || n_units < 0 ||
        (n_units > 0 && !unit_ids)) {
      set_error("tsr_route: n_nodes < 1, NULL argument or n_units < 0");
      return TSR_ERR_INVALID_ARG;
    }
    *chosen = route(node_caches, inflight, n_nodes, distinct(unit_ids, n_units), rr_cursor);
    return TSR_OK;
  });
}

tsr_status tsr_replay(const tsr_replay_config* cfg, const int32_t* offsets,
                      const uint64_t* unit_ids, const int32_t* unit_tokens,
                      int32_t n_req, tsr_replay_stats* stats, int32_t* routed) {
  return guarded([&]() -> tsr_status {
    if (!cfg || !offsets || !stats || n_req < 0 || cfg->n_nodes < 1 ||
        cfg->page_size < 1 || cfg->local_capacity_blocks < 0 ||
        cfg->shared_capacity_blocks < 0 || cfg->concurrency < 1 ||
        cfg->local_window < 0 || cfg->shared_window < 0) {
      set_error("tsr_replay: invalid configuration or NULL argument");
      return TSR_ERR_INVALID_ARG;
    }
    if (offsets[0] != 0) {
      set_error("tsr_replay: offsets[0] must be 0");
      return TSR_ERR_INVALID_ARG;
    }
    const int32_t B = cfg->page_size;
    std::unordered_map<uint64_t, int32_t> length;
    int64_t total_blocks = 0;
    for (int32_t i = 0; i < n_req; ++i) {
      if (offsets[i + 1] < offsets[i]) {
        set_error("tsr_replay: offsets must not decrease");
        return TSR_ERR_INVALID_ARG;
      }
      for (int32_t j = offsets[i]; j < offsets[i + 1]; ++j) {
        if (unit_tokens[j] <= 0) {
          set_error("tsr_replay: unit lengths must be positive");
          return TSR_ERR_INVALID_ARG;
        }
        auto ins = length.emplace(unit_ids[j], unit_tokens[j]);
        if (!ins.second && ins.first->second != unit_tokens[j]) {
          set_error("tsr_replay: unit " + std::to_string(unit_ids[j]) +
                    " changes length across the trace");
          return TSR_ERR_INVALID_ARG;
        }
      }
    }
    std::vector<std::vector<uint64_t>> reqs(n_req);
    for (int32_t i = 0; i < n_req; ++i) {
      reqs[i] = distinct(unit_ids + offsets[i], offsets[i + 1] - offsets[i]);
      for (uint64_t u : reqs[i]) total_blocks += (length[u] + B - 1) / B;
    }
    const double mean = n_req ? (double)total_blocks / n_req : 1.0;
    const int32_t n = cfg->n_nodes;
    const int32_t wl = cfg->local_window ? cfg->local_window
                                         : tsr_window_for_capacity(cfg->local_capacity_blocks, mean);
    const int32_t ws = cfg->shared_window ? cfg->shared_window
                                          : tsr_window_for_capacity(cfg->shared_capacity_blocks, mean);
    std::vector<tsr_scorer> local_sc(n);
    std::vector<tsr_admitter> local(n);
    for (int32_t i = 0; i < n; ++i) {
      local_sc[i].window = wl;
      local_sc[i].w_recent = cfg->w_recent;
      local_sc[i].w_lifetime = cfg->w_lifetime;
      local[i].capacity = cfg->local_capacity_blocks;
      local[i].theta = cfg->theta;
    }
    tsr_scorer shared_sc;
    shared_sc.window = ws;
    shared_sc.w_recent = cfg->w_recent;
    shared_sc.w_lifetime = cfg->w_lifetime;
    tsr_admitter shared;
    shared.capacity = cfg->shared_capacity_blocks;
    shared.theta = cfg->theta;
    const bool has_shared = cfg->shared_capacity_blocks > 0;

    std::vector<const tsr_admitter*> node_ptr(n);
    for (int32_t i = 0; i < n; ++i) node_ptr[i] = &local[i];
    std::vector<int32_t> inflight(n, 0);
    std::deque<int32_t> in_flight_order;     // nodes of the requests in flight
    std::vector<int64_t> per_node(n, 0);
    uint32_t rr = 0;
    tsr_replay_stats st{};
    std::vector<uint64_t> victims;
    for (int32_t i = 0; i < n_req; ++i) {
      const auto& units = reqs[i];
      const int32_t node = cfg->cache_aware ? route(node_ptr.data(), inflight.data(), n, units, &rr)
                                            : route(nullptr, inflight.data(), n, units, &rr);
      if (routed) routed[i] = node;
      ++per_node[node];
      ++inflight[node];
      in_flight_order.push_back(node);
      if ((int32_t)in_flight_order.size() > cfg->concurrency) {
        --inflight[in_flight_order.front()];
        in_flight_order.pop_front();
      }
      std::vector<char> in_local(units.size()), in_shared(units.size());
      for (size_t k = 0; k < units.size(); ++k) {
        const uint64_t u = units[k];
        const int64_t nb = (length[u] + B - 1) / B;
        in_local[k] = local[node].resident.count(u) != 0;
        in_shared[k] = has_shared && shared.resident.count(u) != 0;
        ++st.unit_refs;
        st.blocks += nb;
        if (in_local[k]) {
          ++st.local_hit_units;
          st.local_hit_blocks += nb;
        } else if (in_shared[k]) {
          ++st.shared_hit_units;
          st.shared_hit_blocks += nb;
        } else {
          ++st.miss_units;
          st.miss_blocks += nb;
        }
      }
      observe(&local_sc[node], units);
      if (has_shared) observe(&shared_sc, units);
      for (size_t k = 0; k < units.size(); ++k) {
        const uint64_t u = units[k];
        const int32_t nb = (length[u] + B - 1) / B;
        if (!in_local[k]) {
          victims.clear();
          if (decide(&local[node], &local_sc[node], u, nb, &victims) == TSR_ADMIT_ADMITTED) {
            apply(&local[node], u, nb, victims);
            ++st.local_admitted;
            st.local_evicted += (int64_t)victims.size();
          }
        }
        if (has_shared && !in_shared[k]) {
          victims.clear();
          if (decide(&shared, &shared_sc, u, nb, &victims) == TSR_ADMIT_ADMITTED) {
            apply(&shared, u, nb, victims);
            ++st.shared_admitted;
            st.shared_evicted += (int64_t)victims.size();
          }
        }
      }
    }
    st.requests = n_req;
    st.max_node_requests = n_req ? *std::max_element(per_node.begin(), per_node.end()) : 0;
    st.min_node_requests = n_req ? *std::min_element(per_node.begin(), per_node.end()) : 0;
    *stats = st;
    return TSR_OK;
  });
}

}  // extern "C"

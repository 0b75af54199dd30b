/*
 * tsr_control.h -- retrieval-aware cache management and routing
 * (libtsr.so, host code only; Tessera, Section 5.2).
 *
 * The control plane decides which context-unit states a cache retains and
 * which generation node serves a request.  It runs on the CPU and makes no
 * HIP call:
 *
 *   tsr_scorer_*   the reuse score s(u,t) = w_r f_W(u,t) + w_l f_inf(u,t)
 *                  over one request stream (a node's local stream, or every
 *                  request for the shared tier);
 *   tsr_admitter_* threshold admission and eviction of whole units with
 *                  capacity accounted in blocks;
 *   tsr_route      cache-aware routing under a load constraint;
 *   tsr_replay     a trace replay of the above over n nodes with local
 *                  caches and an optional shared tier.
 *
 * Conventions are those of tsr.h: statuses, tsr_last_error(), host
 * pointers, no exception crosses the ABI.  Objects are not thread-safe; a
 * caller serialises access to each one.
 */
#ifndef TSR_CONTROL_H
#define TSR_CONTROL_H

#include "tsr.h"

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------- scoring */

/* Reuse score of Section 5.2 over one request stream: for unit u at
 * request ordinal t (after t requests were observed),
 *   s(u,t) = w_recent * f_W(u,t) + w_lifetime * f_inf(u,t)
 * with f_W the number of the last `window` requests that retrieved u and
 * f_inf the number of all observed requests that did.  A request that lists
 * a unit twice counts once.  The paper fixes w_recent = 1 and
 * w_lifetime = 0.05.  window >= 1. */
typedef struct tsr_scorer tsr_scorer;

tsr_status tsr_scorer_create(int32_t window, double w_recent, double w_lifetime,
                             tsr_scorer** out);
void tsr_scorer_destroy(tsr_scorer* s);
/* One request's retrieved units (host array [n]); t advances by one. */
tsr_status tsr_scorer_observe(tsr_scorer* s, const uint64_t* unit_ids, int32_t n);
/* s(u,t) after the requests observed so far (0 for a unit never seen). */
double tsr_scorer_score(const tsr_scorer* s, uint64_t unit_id);
/* f_W and f_inf of a unit (either pointer may be NULL). */
tsr_status tsr_scorer_counts(const tsr_scorer* s, uint64_t unit_id, int32_t* recent,
                             int64_t* lifetime);
/* W that makes f_W cover the horizon a cache can retain (Section 5.2): the
 * number of requests whose retrieved units fill capacity_blocks, given the
 * mean retrieved blocks per request; at least 1. */
int32_t tsr_window_for_capacity(int64_t capacity_blocks, double mean_blocks_per_request);

/* ----------------------------------------------- admission and eviction */

/* Outcome of an admission decision. */
typedef enum {
  TSR_ADMIT_BELOW_THRESHOLD = 0,  /* s(u,t) < theta: not a candidate        */
  TSR_ADMIT_ADMITTED = 1,         /* admitted (victims, if any, evicted)    */
  TSR_ADMIT_RESIDENT = 2,         /* already resident: nothing changes      */
  TSR_ADMIT_NO_ROOM = 3,          /* candidate, but units with strictly
                                     lower scores cannot free enough blocks */
  TSR_ADMIT_TOO_LARGE = 4         /* the unit exceeds the whole capacity    */
} tsr_admit_result;

/* The resident set of one cache, capacity in blocks (Section 5.2,
 * "Admission and eviction"; Section 5.1, units occupy whole blocks). */
typedef struct tsr_admitter tsr_admitter;

tsr_status tsr_admitter_create(int64_t capacity_blocks, double theta,
                               tsr_admitter** out);
void tsr_admitter_destroy(tsr_admitter* a);
/* Decide for unit_id of n_blocks blocks, scored by `scorer` (which has
 * observed the request that retrieved it):
 *   a unit scoring below theta is not admitted;
 *   if free blocks suffice it is admitted;
 *   otherwise resident units are considered in increasing score order
 *   (ties by unit id) and the candidate is admitted only if units scoring
 *   strictly lower than it free enough blocks; those units are evicted.
 * victims: host array [max_victims] receiving the evicted units in the
 * order they were chosen; n_victims their count.  If more than max_victims
 * would be evicted, returns OUT_OF_RANGE and changes nothing. */
tsr_status tsr_admit(tsr_admitter* a, const tsr_scorer* scorer, uint64_t unit_id,
                     int32_t n_blocks, int32_t* result, uint64_t* victims,
                     int32_t max_victims, int32_t* n_victims);
/* Remove a resident unit (external eviction); STATE if not resident. */
tsr_status tsr_admitter_remove(tsr_admitter* a, uint64_t unit_id);
/* Blocks a unit holds (0 if not resident). */
int32_t tsr_admitter_blocks(const tsr_admitter* a, uint64_t unit_id);
int64_t tsr_admitter_used_blocks(const tsr_admitter* a);
int32_t tsr_admitter_num_units(const tsr_admitter* a);

/* ------------------------------------------------------------- routing */

/* Cache-aware routing (Section 5.2): among the nodes whose in-flight
 * request count is at most one above the least-loaded node's, choose the
 * one whose local cache (node_caches[i]) holds the most blocks of the
 * request's units (each distinct unit counted once); ties go to the lower
 * load, then round-robin from *rr_cursor, which advances past the choice.
 *   node_caches  host array [n_nodes] of admitters (NULL entries hold
 *                nothing); inflight [n_nodes]; unit_ids [n_units]. */
tsr_status tsr_route(const tsr_admitter* const* node_caches, const int32_t* inflight,
                     int32_t n_nodes, const uint64_t* unit_ids, int32_t n_units,
                     uint32_t* rr_cursor, int32_t* chosen);

/* -------------------------------------------------------------- replay */

typedef struct {
  int32_t n_nodes;                  /* generation nodes, >= 1                */
  int64_t local_capacity_blocks;    /* per node                              */
  int64_t shared_capacity_blocks;   /* 0: no shared tier                     */
  int32_t page_size;                /* B, tokens per block                   */
  double theta;                     /* admission threshold                   */
  double w_recent, w_lifetime;      /* score weights                         */
  int32_t local_window;             /* W of the local scorers, 0: derived    */
  int32_t shared_window;            /* W of the shared scorer, 0: derived    */
  int32_t concurrency;              /* a request stays in flight until this
                                       many later requests have arrived     */
  int32_t cache_aware;              /* 1: tsr_route; 0: least loaded, then
                                       round-robin (load-only baseline)     */
} tsr_replay_config;

typedef struct {
  int64_t requests;
  int64_t unit_refs;                /* retrieved units (distinct per request) */
  int64_t blocks;                   /* their blocks                           */
  int64_t local_hit_units, local_hit_blocks;
  int64_t shared_hit_units, shared_hit_blocks;
  int64_t miss_units, miss_blocks;
  int64_t local_admitted, local_evicted;
  int64_t shared_admitted, shared_evicted;
  int64_t max_node_requests, min_node_requests;
} tsr_replay_stats;

/* Replay a trace of n_req requests.  Request i retrieved the units
 * unit_ids[offsets[i] .. offsets[i+1]) with token counts unit_tokens[...]
 * (a unit's length must not change across the trace).  For each request in
 * order: route it (then it is in flight on its node); look each distinct
 * unit up in the node's local cache, else the shared cache (a hit there
 * prepares from the shared tier), else it is a miss; then the node's local
 * scorer and the shared scorer observe the request, and every unit that
 * was not resident in a tier is an admission candidate in that tier
 * (tiers decide independently, Section 5.2).  routed: host [n_req] or NULL,
 * receives each request's node. */
tsr_status tsr_replay(const tsr_replay_config* cfg, const int32_t* offsets,
                      const uint64_t* unit_ids, const int32_t* unit_tokens,
                      int32_t n_req, tsr_replay_stats* stats, int32_t* routed);

#ifdef __cplusplus
}
#endif

#endif /* TSR_CONTROL_H */

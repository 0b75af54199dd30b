/*
 * tsr.h -- C ABI of the composed-prefill hot path (libtsr.so, gfx950).
 *
 * The library composes a request's prefill from per-context-unit KV states,
 * one attention layer at a time (Tessera, Sections 5.1, 5.3 and 5.4):
 *
 *   tsr_compose_kv    cached hits: gather unit KV pages from the pool into
 *                     the request's pages, re-rotating keys cached before
 *                     RoPE to the unit's new prompt positions;
 *   tsr_prefill_attn  the final extend pass: rotate the computed tokens'
 *                     queries and keys at their positions, append their K/V
 *                     to the request pages, and run causal GQA attention of
 *                     those tokens over the whole assembled KV;
 *   tsr_retain_kv     write newly computed units' reusable form (keys before
 *                     RoPE, values) into their pool pages.
 *
 * Conventions
 *   - Every pointer named dev_* or documented as "device" is a HIP device
 *     pointer; every other pointer is host memory.  `stream` is a
 *     hipStream_t passed as void*.  NULL selects the default stream.
 *   - The caller owns every buffer, including the plan workspace and the
 *     RoPE table; the library never allocates device memory.  Host memory
 *     the library allocates lives inside the plan object.
 *   - Inputs are borrowed until the work enqueued on `stream` completes.
 *   - No function throws, aborts or exits.  On failure a status other than
 *     TSR_OK is returned, nothing is enqueued, and tsr_last_error() (a
 *     thread-local string) says why.
 *   - Thread safety: plans are immutable after creation and may be used
 *     from several threads and streams at once.
 *
 * KV page layout (pool and request pages alike), one layer:
 *     [n_pages][n_kv_heads][page_size][head_dim]   (head-major within a page)
 * Token j of a unit lives in its block j / B at slot j % B (Section 5.1);
 * prompt position p of a request lives in request page block_table[p / B]
 * at slot p % B.
 *
 * Row order ("plan order") of the computed tokens: requests in the order
 * given, and within a request the computed tokens by increasing prompt
 * position.  q/k/v inputs and attention outputs use this row order.
 */
#ifndef TSR_H
#define TSR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TSR_ABI_VERSION 7

typedef enum {
  TSR_OK = 0,
  TSR_ERR_INVALID_ARG = 1,   /* malformed request, null pointer, bad size */
  TSR_ERR_UNSUPPORTED = 2,   /* valid but not implemented (dtype, shape)  */
  TSR_ERR_OUT_OF_RANGE = 3,  /* page id, position or arena bound exceeded */
  TSR_ERR_DEVICE = 4,        /* a HIP call failed (message in last error) */
  TSR_ERR_STATE = 5,         /* cache entry not in the state the call needs
                                (exists, absent, PENDING, leased, stale
                                storage epoch, different block set)        */
  TSR_ERR_NO_SPACE = 6       /* not enough free blocks in the cache arena  */
} tsr_status;

typedef enum { TSR_F32 = 0, TSR_BF16 = 1, TSR_E4M3 = 2 } tsr_dtype;

/* Preparation of a unit (Section 5.1, per-unit plan): a state used from a
 * cache tier is a HIT; a state computed from text is a MISS. */
typedef enum { TSR_MISS = 0, TSR_HIT = 1 } tsr_residency;

/* Which keys the rows of a MISS unit see (Section 5.3).
 *   TSR_SCOPE_GLOBAL  every token of a MISS unit is a row of the final pass
 *                     and sees the whole assembled prompt up to itself.
 *   TSR_SCOPE_LOCAL   the paper's preparation of a miss: the unit is
 *                     prefilled on its own and then composed like a hit.
 *                     Its first min(n_recompute, n) tokens (the recompute
 *                     window) are rows of the final pass over the whole
 *                     prompt; its remaining tokens are rows that see only
 *                     the keys of their own unit (evaluated at their final
 *                     positions, which RoPE's relative property makes equal
 *                     to a prefill from position 0). */
typedef enum { TSR_SCOPE_GLOBAL = 0, TSR_SCOPE_LOCAL = 1 } tsr_miss_scope;

/* Shape and numerics of one attention layer.
 *   (kv_dtype, act_dtype) in {(F32, F32), (BF16, BF16), (E4M3, BF16)}.
 *   E4M3 (OCP e4m3fn) pools store codes plus one power-of-two fp32 scale per
 *   (page, K|V); a value is decode(code) * scale.  Scale arrays are
 *   [n_pages][2] fp32 ({K, V}) per layer.  An e4m3 plan must be page aligned
 *   (every request page has one writer: segments start on page boundaries
 *   and end on one or at the prompt's end; recompute windows are whole
 *   pages or the whole unit), else tsr_plan_create returns UNSUPPORTED.
 *   RoPE (Section 2.2 names rotary encoding but not its dimension pairing,
 *   so the pairing is a field):
 *     rope_interleaved = 0  dimension i is paired with i + head_dim/2
 *                           (the half-split pairing of Llama-family
 *                           weights) at frequency rope_theta^(-2i/head_dim);
 *     rope_interleaved = 1  dimensions 2i and 2i+1 are paired (GPT-J
 *                           style).  Not implemented: tsr_plan_create and
 *                           tsr_rope_table_bytes refuse it (UNSUPPORTED /
 *                           0), so such a model is rejected, not run with
 *                           the wrong pairing.
 *     any other value       INVALID_ARG.
 *   Positions must be < max_position (the RoPE table's length).
 *   softmax_scale == 0 selects 1/sqrt(head_dim). */
typedef struct {
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t page_size;
  int32_t kv_dtype;
  int32_t act_dtype;
  double rope_theta;
  int32_t rope_interleaved;
  int32_t max_position;
  float softmax_scale;
} tsr_model;

/* One occurrence of a context unit in a request (Section 5.1).
 *   unit_id      stable identity (opaque to the library).
 *   position     first prompt position of the unit (placement is fixed
 *                before preparation, Section 5.3).
 *   n_tokens     unit length n > 0.
 *   residency    TSR_HIT: its cached state (keys before RoPE, values) is in
 *                pool_pages; TSR_MISS: it is computed in this pass.
 *   n_recompute  the composition policy recomputes the first
 *                min(n_recompute, n) tokens of a HIT (a fixed chunk-initial
 *                window, Section 7); they become computed rows.  Under
 *                TSR_SCOPE_LOCAL the same window applies to a MISS unit.
 *   retain       MISS only: 1 writes the computed state into pool_pages.
 *   pool_pages   host array of ceil(n / page_size) pool page ids: the source
 *                of a HIT, the destination of a retained MISS, else unused
 *                (may be NULL). */
typedef struct {
  uint64_t unit_id;
  int32_t position;
  int32_t n_tokens;
  int32_t residency;
  int32_t n_recompute;
  int32_t retain;
  int32_t reserved;
  const int32_t* pool_pages;
} tsr_unit;

/* One request: an ordered prompt tiled exactly once by its units and text
 * segments (instruction, separators, query), and its request KV pages.
 *   miss_scope   a tsr_miss_scope value; 0 (the global scope) for structs
 *                that are zero-initialised.
 *   text_segs    host array [n_text][2] of {start, length}, length > 0.
 *   block_table  host array of ceil(prompt_len / page_size) request page ids,
 *                not shared with any other request of the batch. */
typedef struct {
  int32_t prompt_len;
  int32_t n_units;
  const tsr_unit* units;
  int32_t n_text;
  int32_t miss_scope;
  const int32_t* text_segs;
  const int32_t* block_table;
} tsr_request;

typedef struct tsr_plan tsr_plan;

/* ---------------------------------------------------------------- RoPE */

/* Bytes of the RoPE table for `model`: cos and sin planes of
 * [max_position][head_dim/2] fp32.  0 if the model is invalid. */
size_t tsr_rope_table_bytes(const tsr_model* model);

/* Fill a caller-owned device buffer with the RoPE table: angles and cos/sin
 * are evaluated in fp64 on the host and rounded to fp32, then copied with
 * hipMemcpyAsync on `stream`.  The table is built once per model and may be
 * shared by every plan of that model. */
tsr_status tsr_rope_table_init(const tsr_model* model, void* dev_table,
                               size_t table_bytes, void* stream);

/* ---------------------------------------------------------------- plan */

/* Device workspace bytes tsr_plan_create needs for this batch, or 0 if the
 * batch fails validation (tsr_last_error says why). */
size_t tsr_plan_workspace_size(const tsr_model* model, const tsr_request* reqs,
                               int32_t n_req, int32_t n_pool_pages,
                               int32_t n_req_pages);

/* Validate a batch and build its plan (Section 5.3, placement before
 * preparation): the computed rows, the gathered tokens, the retained
 * tokens and the attention tile schedule.  The device image of the plan is
 * copied into `dev_workspace` with hipMemcpyAsync on `stream`.
 *   n_pool_pages / n_req_pages  sizes of the pool / request page arenas.
 *   dev_rope_table  a table filled by tsr_rope_table_init for this model.
 *   dev_workspace   NULL builds a host-only plan that can be inspected but
 *                   not executed (no HIP call is made).
 * Checks (all on the host, before anything is enqueued): shapes and dtypes;
 * every request tiled exactly once in order; page ids inside their arena;
 * request pages not shared between requests; positions < max_position; a
 * retained unit's pages neither read by a HIT of the batch nor written by
 * another retained unit. */
tsr_status tsr_plan_create(const tsr_model* model, const tsr_request* reqs,
                           int32_t n_req, int32_t n_pool_pages,
                           int32_t n_req_pages, const void* dev_rope_table,
                           void* dev_workspace, size_t workspace_bytes,
                           void* stream, tsr_plan** out_plan);

/* Plan options (tsr_plan_create_ex; NULL means all zero).
 *   alias_v   1: V aliasing, a zero-copy form of composition.  A request
 *             page that holds B gathered tokens of one HIT unit, slot for
 *             slot (the unit starts on a page boundary), is not filled with
 *             V by tsr_compose_kv (its K still is); attention reads that
 *             page's V from the pool page instead (tsr_attn_aliased).  The
 *             cached V is used as stored, so results equal the composed
 *             path's bit for bit.  The pool pages must stay unchanged until
 *             attention completes.  bf16 pools only (else UNSUPPORTED).
 *   alias_k   1: K rotated on load, the other half of a zero-copy
 *             composition (Section 5.3 places cached keys with RoPE applied
 *             at their new positions; here the placement happens as
 *             attention loads them).  For the same request pages as
 *             alias_v (B gathered tokens of one HIT unit, slot for slot),
 *             tsr_compose_kv does not write K; attention reads the cached
 *             pre-RoPE K from the pool page and rotates it at the key's
 *             prompt position with the same fp32 rotation and bf16 rounding
 *             as compose, so results equal the composed path's bit for bit.
 *             With alias_v too, such pages are not touched by compose at
 *             all.  The pool pages must stay unchanged until attention
 *             completes.  bf16 pools only (else UNSUPPORTED).
 *   split_tiles  key-range splitting of long attention items (plans of
 *             the bf16 row-block kernel; other plans ignore it).
 *             An item whose keys span more than S tiles of 32 keys runs as
 *             ceil(tiles / S) items over consecutive key ranges, each
 *             writing its rows' normalized output and log-sum-exp in fp32
 *             to a buffer in the plan workspace; a second kernel on the
 *             same stream merges them (o = sum_c exp(lse_c - lse) o_c,
 *             lse = log sum_c exp(lse_c)) into out and lse.  Without it a
 *             launch lasts at least as long as its longest item: under
 *             TSR_SCOPE_LOCAL the rows after the units attend to the whole
 *             prompt while most rows attend within a short unit.
 *               0   automatic: for items of one row block, S = the
 *                   launch's mean key tiles per compute unit (256 units,
 *                   32 tiles at least), so only items that would outlast
 *                   the rest of the launch are split; items of three row
 *                   blocks are not split; never for tsr_plan_create_static;
 *               >0  S = split_tiles;
 *               -1  never split.
 *             A plan with split items writes that buffer on every
 *             attention call: calls that use one plan on streams that
 *             run concurrently race there.
 *   attn_kernel  which bf16 attention kernel the plan schedules for
 *             (plans with bf16 activations and bf16 KV; with e4m3 KV only
 *             3 and 4 apply, as noted below; other plans ignore it):
 *               0   automatic: the row-block kernel's rule (2), the faster
 *                   choice on every batch measured;
 *               1   the pipelined kernel: items of up to two 32-row blocks,
 *                   eight waves per workgroup, the QK^T products of the
 *                   next key tile under the softmax of this one.  It
 *                   applies without alias_k and when no item spans more
 *                   than 65,536 keys; otherwise TSR_ERR_UNSUPPORTED;
 *               2   the row-block kernel: items of three 32-row blocks,
 *                   cut from each request's rows grouped by first visible
 *                   key, when at least 60 % of their row-block x key-tile
 *                   slots hold work and there are at least 256 of them
 *                   (one per compute unit); else of one row block;
 *               3   the row-block kernel, three row blocks;
 *               4   the row-block kernel, one row block;
 *             3 and 4 also fix the row blocks of the e4m3 kernel (plans
 *             with bf16 activations and e4m3 KV), which otherwise follows
 *             the rule of 2.
 *             The row-block kernel is the only one for alias_k plans and
 *             for the key-range split.
 *   reserved  must be zero. */
typedef struct {
  int32_t alias_v;
  int32_t alias_k;
  int32_t split_tiles;
  int32_t attn_kernel;
  int32_t reserved[4];
} tsr_plan_options;

/* tsr_plan_workspace_size for a plan made with `options` (NULL: all zero,
 * which is what tsr_plan_workspace_size assumes); the key-range split
 * buffer depends on split_tiles. */
size_t tsr_plan_workspace_size_ex(const tsr_model* model, const tsr_request* reqs,
                                  int32_t n_req, int32_t n_pool_pages, int32_t n_req_pages,
                                  const tsr_plan_options* options);

/* tsr_plan_create with options; tsr_plan_create is this with NULL.  The
 * workspace must hold tsr_plan_workspace_size_ex(..., options) bytes. */
tsr_status tsr_plan_create_ex(const tsr_model* model, const tsr_request* reqs,
                              int32_t n_req, int32_t n_pool_pages, int32_t n_req_pages,
                              const tsr_plan_options* options, const void* dev_rope_table,
                              void* dev_workspace, size_t workspace_bytes, void* stream,
                              tsr_plan** out_plan);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation):
 * tsr_plan_create_ex without a workspace.  The plan's device image is
 * written (hipMemcpyAsync on `stream`) into a plan area the library owns on
 * the current device, a static device array of 16 MiB that each GPU holds
 * until the process ends; the call allocates no device memory.
 *   - A batch whose image exceeds 16 MiB (tsr_plan_workspace_size_ex with
 *     these options; split_tiles = 0 means no key-range splitting here) is
 *     refused with TSR_ERR_OUT_OF_RANGE before any HIP call.
 *   - Every static plan on a device shares that area: creating one rewrites
 *     it, and the plans it replaced are refused from then on
 *     (TSR_ERR_STATE from every entry point that executes a plan).
 *   - Calls that overlap on one GPU race: work of a previous static plan
 *     still running when the next static plan's image is copied reads the
 *     new image.  Order them (one stream, or an event between streams).
 * Other arguments, checks and results as tsr_plan_create_ex; destroy the
 * plan with tsr_plan_destroy. */
tsr_status tsr_plan_create_static(const tsr_model* model, const tsr_request* reqs,
                                  int32_t n_req, int32_t n_pool_pages, int32_t n_req_pages,
                                  const tsr_plan_options* options, const void* dev_rope_table,
                                  void* stream, tsr_plan** out_plan);

/* Number of computed rows T (inputs q/k/v and outputs have T rows). */
int32_t tsr_plan_num_compute_tokens(const tsr_plan* plan);
/* Number of cached tokens gathered by tsr_compose_kv. */
int32_t tsr_plan_num_gather_tokens(const tsr_plan* plan);
/* Number of tokens written by tsr_retain_kv. */
int32_t tsr_plan_num_retain_tokens(const tsr_plan* plan);
/* Number of attention work items (row tile x KV head, plus launch padding).
 * A row tile holds up to 32 consecutive computed rows, or up to 64 (the
 * pipelined bf16 kernel) or 96 (the row-block kernels of bf16 and e4m3 KV)
 * in plans whose runs of rows with a common first visible key are long
 * enough. */
int32_t tsr_plan_num_attn_items(const tsr_plan* plan);
/* Most computed rows an attention item of this plan holds: 32, 64 (the
 * pipelined bf16 kernel) or 96 (three row blocks per workgroup); -1 for a
 * null plan. */
int32_t tsr_plan_attn_rows_per_item(const tsr_plan* plan);
/* Number of attention items whose key range was split (split_tiles), each
 * merged by the second kernel; 0 when none; -1 for a null plan. */
int32_t tsr_plan_num_attn_splits(const tsr_plan* plan);

/* The attention items in two parts, so that attention can start while the
 * cached states are still on their way (Section 5.3: cache hits transfer
 * while missing units are prefilled, and the request completes once every
 * state is ready):
 *   TSR_ATTN_BEFORE_COMPOSE  items none of whose loaded key tiles (masked
 *                            keys included) holds a position tsr_compose_kv
 *                            fills: they read only keys that tsr_append_kv
 *                            writes, so they may run before compose (under
 *                            TSR_SCOPE_LOCAL: the unit-local rows of missing
 *                            units, among others);
 *   TSR_ATTN_AFTER_COMPOSE   every other item.
 * The two parts together compute exactly what TSR_ATTN_ALL computes; each
 * is scheduled over the XCDs on its own.  Items of both parts write
 * disjoint rows and heads of `out` and `lse`. */
typedef enum {
  TSR_ATTN_ALL = 0,
  TSR_ATTN_BEFORE_COMPOSE = 1,
  TSR_ATTN_AFTER_COMPOSE = 2
} tsr_attn_part_id;

/* Items of one part (padding to whole XCD rounds included); -1 for a NULL
 * plan or an unknown part. */
int32_t tsr_plan_num_attn_items_part(const tsr_plan* plan, int32_t part);

/* Request pages whose V attention reads from the pool (alias_v plans; 0
 * otherwise). */
int32_t tsr_plan_num_aliased_pages(const tsr_plan* plan);
/* Request pages whose K attention reads from the pool and rotates on load
 * (alias_k plans; 0 otherwise). */
int32_t tsr_plan_num_aliased_k_pages(const tsr_plan* plan);

/* Prompt position and request index of every computed row, in plan order.
 * host_positions: [T] (required); host_requests: [T] or NULL. */
tsr_status tsr_plan_compute_positions(const tsr_plan* plan,
                                      int32_t* host_positions,
                                      int32_t* host_requests);

/* First visible key position of every computed row, in plan order
 * (host_kv_lo [T]): 0, or under TSR_SCOPE_LOCAL the first position of the
 * unit of a MISS token past its recompute window. */
tsr_status tsr_plan_row_kv_lo(const tsr_plan* plan, int32_t* host_kv_lo);

void tsr_plan_destroy(tsr_plan* plan);

/* ------------------------------------------------------------ hot path */

/* Compose: for every HIT unit u and token j in [min(r_u, n_u), n_u):
 *   V_req[pos_u + j] = V_pool[u's block j/B][slot j%B]        (bit copy)
 *   K_req[pos_u + j] = RoPE(K_pool[...], pos_u + j)  rounded to kv_dtype
 * (Section 5.3, "Preparing cache hits").  The pool is read only.
 * Rotation: fp32 table values, fp32 products and one fp32 add each, no
 * fused multiply-add; bf16 results rounded to nearest even.
 *   pool_k/pool_v  device, [n_pool_pages][H_kv][B][d] of kv_dtype; or, for
 *                  a pool held in host memory (Section 5.2's local tier),
 *                  the device address of pinned host memory
 *                  (hipHostGetDevicePointer), read across the host link.
 *   req_k/req_v    device, [n_req_pages][H_kv][B][d] of kv_dtype.
 *   pool_scale, req_scale  e4m3 only (else NULL): [n_layers][pages][2] fp32.
 *   e4m3: V codes and V scale are copied; K is dequantized, rotated in fp32
 *   and requantized with the smallest power-of-two scale s such that
 *   max |K| / s <= 448 over the request page (nearest even, saturating).
 *   n_layers >= 1 composes that many layers in one launch; layer l uses the
 *   buffers offset by l * pool_layer_stride / req_layer_stride bytes. */
tsr_status tsr_compose_kv(const tsr_plan* plan, const void* pool_k,
                          const void* pool_v, const float* pool_scale,
                          void* req_k, void* req_v, float* req_scale,
                          int32_t n_layers, int64_t pool_layer_stride,
                          int64_t req_layer_stride, void* stream);

/* Final extend pass (Section 5.3, "Completing prefill"):
 *   1. for every computed row t at position p_t: k_rot = RoPE(k_t, p_t) and
 *      v_t are written to the request pages at p_t;
 *   2. o_t,h = softmax(scale * q_rot . K_req[lo_t..p_t, g]^T) V_req[lo_t..p_t, g],
 *      q_rot = RoPE(q_t,h, p_t) rounded to act_dtype, g = h / (H_q / H_kv),
 *      causal by absolute position (a key at p_t itself is visible); lo_t
 *      is 0 except for the unit-local rows of TSR_SCOPE_LOCAL (see
 *      tsr_plan_row_kv_lo).
 *   q    device [T][H_q][d], k/v device [T][H_kv][d]: pre-RoPE, act dtype.
 *   out  device [T][H_q][d] of act_dtype.
 *   lse  device [T][H_q] fp32 natural-log sum of exp(scale * s), or NULL.
 * Must run after tsr_compose_kv of the same plan and layer (stream order).
 * bf16: QK^T in bf16 MFMA with fp32 accumulation; probabilities and values
 * enter the PV product as fp16: V values up to 65280 in magnitude (every
 * bf16 below fp16's maximum) convert exactly; a larger one is staged as NaN
 * (with the values staged beside it) and makes the outputs of the rows whose
 * key tiles hold it non-finite: the input is refused loudly rather than
 * clipped.  e4m3: likewise a V page scale above 2^7 (stored V beyond fp16's
 * range) makes such outputs NaN.
 * e4m3: computed pages are quantized like composed ones (k after rotation);
 * q_rot is quantized per (row, head) to e4m3 with the smallest power-of-two
 * scale covering the row, QK^T runs in fp8 MFMA, PV in fp16 MFMA.
 * Errors: every argument check runs before the first launch, so a status
 * other than TSR_ERR_DEVICE means nothing was enqueued.  The call enqueues
 * two kernels, append then attention; if the HIP runtime reports a failure
 * of the second launch, the append stays enqueued (the request pages
 * receive the computed rows' K/V, out and lse are not written) and
 * TSR_ERR_DEVICE is returned. */
tsr_status tsr_prefill_attn(const tsr_plan* plan, const void* q,
                            const void* k, const void* v, void* req_k,
                            void* req_v, float* req_scale, void* out,
                            float* lse, void* stream);

/* The two halves of tsr_prefill_attn, for callers that schedule them apart
 * (and for timing the attention kernel alone):
 *   tsr_append_kv  step 1 only (rotate computed keys, write k_rot and v to
 *                  the request pages);
 *   tsr_attn       step 2 only; the request pages must already hold every
 *                  position's K/V (compose + append, in stream order).
 * Arguments have the same meaning as in tsr_prefill_attn. */
tsr_status tsr_append_kv(const tsr_plan* plan, const void* k, const void* v,
                         void* req_k, void* req_v, float* req_scale,
                         void* stream);
tsr_status tsr_attn(const tsr_plan* plan, const void* q, const void* req_k,
                    const void* req_v, const float* req_scale, void* out,
                    float* lse, void* stream);

/* Assembly of one layer's request KV in a single launch: exactly
 * tsr_compose_kv (n_layers = 1) followed by tsr_append_kv, with the same
 * results bit for bit, in one kernel whose first workgroups gather the
 * cached tokens and whose others append the computed rows (Section 5.3:
 * hits placed with RoPE at their new positions; computed rows placed before
 * the extend pass).  Both are HBM-bound copies, so one launch spares the
 * second launch and its ramp.  Arguments as in tsr_compose_kv (pool_*,
 * pool_scale, req_*, req_scale) and tsr_append_kv (k, v): pool_k/pool_v may
 * be NULL when the plan gathers nothing, k/v when it computes nothing.
 * Follow with tsr_attn (or tsr_attn_part / tsr_attn_aliased). */
tsr_status tsr_assemble_kv(const tsr_plan* plan, const void* pool_k, const void* pool_v,
                           const float* pool_scale, const void* k, const void* v,
                           void* req_k, void* req_v, float* req_scale, void* stream);

/* tsr_attn restricted to one part of the items (a tsr_attn_part_id);
 * TSR_ATTN_ALL is tsr_attn.  BEFORE_COMPOSE needs tsr_append_kv of the
 * plan in stream order; AFTER_COMPOSE needs append and compose. */
tsr_status tsr_attn_part(const tsr_plan* plan, int32_t part, const void* q,
                         const void* req_k, const void* req_v, const float* req_scale,
                         void* out, float* lse, void* stream);

/* Attention of an alias_v and/or alias_k plan (one part, or TSR_ATTN_ALL):
 * as tsr_attn_part, with the V of V-aliased request pages read from pool_v
 * and the K of K-aliased pages read from pool_k and rotated on load (device,
 * the pool arenas tsr_compose_kv read, [n_pool_pages][H_kv][B][d] bf16).
 * pool_v is required by alias_v plans and pool_k by alias_k plans (NULL
 * otherwise).  The non-aliased entry points refuse aliased plans, and this
 * one refuses the others (INVALID_ARG). */
tsr_status tsr_attn_aliased(const tsr_plan* plan, int32_t part, const void* q,
                            const void* req_k, const void* req_v, const void* pool_k,
                            const void* pool_v, void* out, float* lse, void* stream);

/* Retain (Section 5.4): for every MISS unit with retain = 1 and token j:
 *   K_pool[block j/B][slot j%B] = k (before RoPE), V_pool[...] = v
 * as bit copies from the computed rows (e4m3: quantized per pool page, both
 * scales written).  Slots of a unit's last block
 * beyond n are left untouched.  k/v are the same inputs as
 * tsr_prefill_attn's and must stay alive until the stream reaches this work
 * (Section 5.4: sources stay valid until their copies complete).  A caller
 * may publish the units as HITs only after observing its completion.
 * pool_k/pool_v/pool_scale: as for tsr_compose_kv (device memory, or the
 * device address of pinned host memory). */
tsr_status tsr_retain_kv(const tsr_plan* plan, const void* k, const void* v,
                         void* pool_k, void* pool_v, float* pool_scale,
                         void* stream);

/* -------------------------------------------------- context-unit cache */

/* Directory of a node's context-unit cache (Section 5.2: a cache of unit
 * states in pinned host memory on every generation node; Section 5.4: its
 * entry life cycle).  It records which units hold a complete reusable state
 * in a caller-owned arena of fixed-size blocks (one block = one KV page of
 * every layer), in which blocks and under which storage epoch, and how many
 * transfers still read them.  Host metadata only: the directory never
 * touches the blocks' bytes and makes no HIP call.  Every function is
 * thread-safe (one mutex per directory).
 *
 * Entry life cycle:
 *   reserve  ABSENT -> PENDING.  Takes n free blocks (lowest ids first) and a
 *            new storage epoch, the version that tells successive
 *            allocations of one unit apart; only the holder of that epoch may
 *            publish or cancel.  A PENDING entry is not a hit: acquire fails,
 *            so other requests compute the unit for themselves.
 *   publish  PENDING -> READY, once the writer has observed the completion
 *            of every block write.  The epoch and the exact block list are
 *            checked, so a stale writer or a partial write cannot publish.
 *   cancel   PENDING -> ABSENT for a failed or abandoned writeback.  The
 *            entry is never published; its blocks are "draining" and return
 *            to the free set only when the writer calls tsr_cache_reclaim
 *            for that epoch, after its outstanding transfers completed.
 *   acquire  READY only: takes a read lease and returns the blocks.  This is
 *            the revalidation of a planned hit before its transfer; any
 *            other state returns TSR_ERR_STATE and the caller prepares the
 *            unit from text instead (Section 5.3, preparation failures).
 *   release  drops one lease, after the transfer that read the blocks ended.
 *   evict    READY with no lease -> ABSENT; blocks freed.  A leased entry is
 *            not evicted (TSR_ERR_STATE). */
typedef struct tsr_cache tsr_cache;

typedef enum {
  TSR_ENTRY_ABSENT = 0,
  TSR_ENTRY_PENDING = 1,
  TSR_ENTRY_READY = 2
} tsr_entry_state;

/* A directory over blocks [0, n_blocks), all free. */
tsr_status tsr_cache_create(int32_t n_blocks, tsr_cache** out);
void tsr_cache_destroy(tsr_cache* cache);

/* blocks: host [n_blocks] output; epoch: output.  NO_SPACE if fewer than
 * n_blocks are free; STATE if the unit has an entry. */
tsr_status tsr_cache_reserve(tsr_cache* cache, uint64_t unit_id, int32_t n_blocks,
                             uint64_t* epoch, int32_t* blocks);
/* blocks: host [n_blocks], the list reserve returned, in its order. */
tsr_status tsr_cache_publish(tsr_cache* cache, uint64_t unit_id, uint64_t epoch,
                             const int32_t* blocks, int32_t n_blocks);
tsr_status tsr_cache_cancel(tsr_cache* cache, uint64_t unit_id, uint64_t epoch);
tsr_status tsr_cache_reclaim(tsr_cache* cache, uint64_t epoch);
/* blocks: host [max_blocks] output; n_blocks: the unit's block count (set
 * also when it exceeds max_blocks, which returns OUT_OF_RANGE, no lease). */
tsr_status tsr_cache_acquire(tsr_cache* cache, uint64_t unit_id, int32_t max_blocks,
                             uint64_t* epoch, int32_t* blocks, int32_t* n_blocks);
tsr_status tsr_cache_release(tsr_cache* cache, uint64_t unit_id, uint64_t epoch);
tsr_status tsr_cache_evict(tsr_cache* cache, uint64_t unit_id);
/* state (required), epoch, n_blocks, leases (each may be NULL); an absent
 * unit reads as TSR_ENTRY_ABSENT with zeros. */
tsr_status tsr_cache_query(const tsr_cache* cache, uint64_t unit_id, int32_t* state,
                           uint64_t* epoch, int32_t* n_blocks, int32_t* leases);
/* Blocks neither held by an entry nor draining; -1 for NULL. */
int32_t tsr_cache_free_blocks(const tsr_cache* cache);

/* Copy whole blocks between two block arenas on `stream` with
 * hipMemcpyAsync (between pinned host memory and device memory the copy
 * engines carry it, leaving the compute units to the kernels):
 *   dst block dst_blocks[i] <- src block src_blocks[i] for i < n, in each
 *   of n_layers layers (layer l of an arena starts l * layer_stride bytes
 *   after its base; strides are ignored when n_layers == 1).
 * Pairs whose ids both continue the previous pair's are merged into one
 * copy.  Staging a cached unit into device memory before compose (Section
 * 5.3, local hits copied from the pinned host cache into bounded GPU
 * staging) and writing retained blocks back to the cache (Section 5.4) are
 * both this call.
 *   dst/src      device pointers or pinned host pointers to arenas of
 *                n_dst_blocks / n_src_blocks blocks of block_bytes.
 *   dst_blocks, src_blocks  host arrays [n].
 * Every id is checked against its arena before anything is enqueued
 * (OUT_OF_RANGE).  If a HIP call fails midway (DEVICE), the copies before
 * it stay enqueued.  Source blocks must not be modified, and destination
 * blocks not read, until the stream reaches this work. */
tsr_status tsr_copy_blocks(void* dst, int32_t n_dst_blocks, const int32_t* dst_blocks,
                           const void* src, int32_t n_src_blocks,
                           const int32_t* src_blocks, int32_t n, int64_t block_bytes,
                           int32_t n_layers, int64_t dst_layer_stride,
                           int64_t src_layer_stride, void* stream);

/* Thread-local message of the last failure on this thread ("" if none). */
const char* tsr_last_error(void);

int32_t tsr_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TSR_H */

"""ctypes binding of libtsr.so (include/tsr.h).  Argument marshalling only.

Functions keep the C names.  Pointer arguments accept an int, None, or any
object with `data_ptr()` (a torch tensor); stream arguments accept an int,
None, or an object with `cuda_stream` (a torch stream; on ROCm that handle is
a hipStream_t).  Non-OK statuses raise TsrError carrying the status and the
library's message.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_double, c_float, c_int32, c_int64, c_size_t, c_uint64, c_void_p

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# TSR_LIBRARY overrides the library path (to compare builds side by side).
LIB_PATH = os.environ.get("TSR_LIBRARY") or os.path.join(HERE, "libtsr.so")

(TSR_OK, TSR_ERR_INVALID_ARG, TSR_ERR_UNSUPPORTED, TSR_ERR_OUT_OF_RANGE, TSR_ERR_DEVICE,
 TSR_ERR_STATE, TSR_ERR_NO_SPACE) = range(7)
STATUS_NAMES = {0: "OK", 1: "INVALID_ARG", 2: "UNSUPPORTED", 3: "OUT_OF_RANGE", 4: "DEVICE",
                5: "STATE", 6: "NO_SPACE"}
TSR_ENTRY_ABSENT, TSR_ENTRY_PENDING, TSR_ENTRY_READY = 0, 1, 2
TSR_F32, TSR_BF16, TSR_E4M3 = 0, 1, 2
DTYPE_CODES = {"f32": TSR_F32, "bf16": TSR_BF16, "e4m3": TSR_E4M3}
TSR_MISS, TSR_HIT = 0, 1
TSR_SCOPE_GLOBAL, TSR_SCOPE_LOCAL = 0, 1
TSR_ATTN_ALL, TSR_ATTN_BEFORE_COMPOSE, TSR_ATTN_AFTER_COMPOSE = 0, 1, 2

# Every symbol include/*.h declares.
EXPORTS = (
    "tsr_abi_version", "tsr_last_error", "tsr_rope_table_bytes",
    "tsr_rope_table_init", "tsr_plan_workspace_size", "tsr_plan_workspace_size_ex",
    "tsr_plan_create", "tsr_plan_num_attn_splits",
    "tsr_plan_num_compute_tokens", "tsr_plan_num_gather_tokens",
    "tsr_plan_num_retain_tokens", "tsr_plan_num_attn_items", "tsr_plan_attn_rows_per_item",
    "tsr_plan_num_attn_items_part", "tsr_attn_part", "tsr_plan_create_ex", "tsr_plan_create_static",
    "tsr_plan_num_aliased_pages", "tsr_plan_num_aliased_k_pages", "tsr_attn_aliased",
    "tsr_plan_compute_positions", "tsr_plan_row_kv_lo", "tsr_plan_destroy", "tsr_compose_kv",
    "tsr_prefill_attn", "tsr_append_kv", "tsr_assemble_kv", "tsr_attn", "tsr_retain_kv",
    "tsr_cache_create", "tsr_cache_destroy", "tsr_cache_reserve", "tsr_cache_publish",
    "tsr_cache_cancel", "tsr_cache_reclaim", "tsr_cache_acquire", "tsr_cache_release",
    "tsr_cache_evict", "tsr_cache_query", "tsr_cache_free_blocks", "tsr_copy_blocks",
    "tsr_peak_mfma_flops", "tsr_peak_mfma", "tsr_peak_copy",
    # include/tsr_control.h
    "tsr_scorer_create", "tsr_scorer_destroy", "tsr_scorer_observe", "tsr_scorer_score",
    "tsr_scorer_counts", "tsr_window_for_capacity", "tsr_admitter_create",
    "tsr_admitter_destroy", "tsr_admit", "tsr_admitter_remove", "tsr_admitter_blocks",
    "tsr_admitter_used_blocks", "tsr_admitter_num_units", "tsr_route", "tsr_replay",
)


class TsrError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


class tsr_model(ctypes.Structure):
    _fields_ = [("n_q_heads", c_int32), ("n_kv_heads", c_int32),
                ("head_dim", c_int32), ("page_size", c_int32),
                ("kv_dtype", c_int32), ("act_dtype", c_int32),
                ("rope_theta", c_double), ("rope_interleaved", c_int32),
                ("max_position", c_int32), ("softmax_scale", c_float)]


class tsr_unit(ctypes.Structure):
    _fields_ = [("unit_id", c_uint64), ("position", c_int32),
                ("n_tokens", c_int32), ("residency", c_int32),
                ("n_recompute", c_int32), ("retain", c_int32),
                ("reserved", c_int32), ("pool_pages", POINTER(c_int32))]


class tsr_request(ctypes.Structure):
    _fields_ = [("prompt_len", c_int32), ("n_units", c_int32),
                ("units", POINTER(tsr_unit)), ("n_text", c_int32),
                ("miss_scope", c_int32), ("text_segs", POINTER(c_int32)),
                ("block_table", POINTER(c_int32))]


class tsr_plan_options(ctypes.Structure):
    _fields_ = [("alias_v", c_int32), ("alias_k", c_int32), ("split_tiles", c_int32),
                ("attn_kernel", c_int32), ("reserved", c_int32 * 4)]


class tsr_replay_config(ctypes.Structure):
    _fields_ = [("n_nodes", c_int32), ("local_capacity_blocks", c_int64),
                ("shared_capacity_blocks", c_int64), ("page_size", c_int32),
                ("theta", c_double), ("w_recent", c_double), ("w_lifetime", c_double),
                ("local_window", c_int32), ("shared_window", c_int32),
                ("concurrency", c_int32), ("cache_aware", c_int32)]


class tsr_replay_stats(ctypes.Structure):
    _fields_ = [(n, c_int64) for n in (
        "requests", "unit_refs", "blocks", "local_hit_units", "local_hit_blocks",
        "shared_hit_units", "shared_hit_blocks", "miss_units", "miss_blocks",
        "local_admitted", "local_evicted", "shared_admitted", "shared_evicted",
        "max_node_requests", "min_node_requests")]


_lib = None


def lib():
    """Load libtsr.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2609_32999_amd.build_lib`")
        L = ctypes.CDLL(LIB_PATH)
        P = c_void_p
        sig = {
            "tsr_abi_version": (c_int32, []),
            "tsr_last_error": (ctypes.c_char_p, []),
            "tsr_rope_table_bytes": (c_size_t, [POINTER(tsr_model)]),
            "tsr_rope_table_init": (c_int32, [POINTER(tsr_model), P, c_size_t, P]),
            "tsr_plan_workspace_size": (c_size_t, [POINTER(tsr_model), POINTER(tsr_request),
                                                   c_int32, c_int32, c_int32]),
            "tsr_plan_create": (c_int32, [POINTER(tsr_model), POINTER(tsr_request), c_int32,
                                          c_int32, c_int32, P, P, c_size_t, P,
                                          POINTER(c_void_p)]),
            "tsr_plan_num_compute_tokens": (c_int32, [P]),
            "tsr_plan_num_gather_tokens": (c_int32, [P]),
            "tsr_plan_num_retain_tokens": (c_int32, [P]),
            "tsr_plan_num_attn_items": (c_int32, [P]),
            "tsr_plan_attn_rows_per_item": (c_int32, [P]),
            "tsr_plan_num_attn_items_part": (c_int32, [P, c_int32]),
            "tsr_plan_num_aliased_pages": (c_int32, [P]),
            "tsr_plan_num_aliased_k_pages": (c_int32, [P]),
            "tsr_plan_num_attn_splits": (c_int32, [P]),
            "tsr_plan_workspace_size_ex": (c_size_t, [POINTER(tsr_model), POINTER(tsr_request),
                                                      c_int32, c_int32, c_int32,
                                                      POINTER(tsr_plan_options)]),
            "tsr_plan_create_ex": (c_int32, [POINTER(tsr_model), POINTER(tsr_request), c_int32,
                                             c_int32, c_int32, POINTER(tsr_plan_options), P, P,
                                             c_size_t, P, POINTER(c_void_p)]),
            "tsr_plan_create_static": (c_int32, [POINTER(tsr_model), POINTER(tsr_request),
                                                 c_int32, c_int32, c_int32,
                                                 POINTER(tsr_plan_options), P, P,
                                                 POINTER(c_void_p)]),
            "tsr_attn_aliased": (c_int32, [P, c_int32, P, P, P, P, P, P, P, P]),
            "tsr_plan_compute_positions": (c_int32, [P, POINTER(c_int32), POINTER(c_int32)]),
            "tsr_plan_row_kv_lo": (c_int32, [P, POINTER(c_int32)]),
            "tsr_plan_destroy": (None, [P]),
            "tsr_compose_kv": (c_int32, [P, P, P, P, P, P, P, c_int32, c_int64, c_int64, P]),
            "tsr_prefill_attn": (c_int32, [P, P, P, P, P, P, P, P, P, P]),
            "tsr_retain_kv": (c_int32, [P, P, P, P, P, P, P]),
            "tsr_append_kv": (c_int32, [P, P, P, P, P, P, P]),
            "tsr_assemble_kv": (c_int32, [P, P, P, P, P, P, P, P, P, P]),
            "tsr_attn": (c_int32, [P, P, P, P, P, P, P, P]),
            "tsr_attn_part": (c_int32, [P, c_int32, P, P, P, P, P, P, P]),
            "tsr_cache_create": (c_int32, [c_int32, POINTER(c_void_p)]),
            "tsr_cache_destroy": (None, [P]),
            "tsr_cache_reserve": (c_int32, [P, c_uint64, c_int32, POINTER(c_uint64),
                                            POINTER(c_int32)]),
            "tsr_cache_publish": (c_int32, [P, c_uint64, c_uint64, POINTER(c_int32), c_int32]),
            "tsr_cache_cancel": (c_int32, [P, c_uint64, c_uint64]),
            "tsr_cache_reclaim": (c_int32, [P, c_uint64]),
            "tsr_cache_acquire": (c_int32, [P, c_uint64, c_int32, POINTER(c_uint64),
                                            POINTER(c_int32), POINTER(c_int32)]),
            "tsr_cache_release": (c_int32, [P, c_uint64, c_uint64]),
            "tsr_cache_evict": (c_int32, [P, c_uint64]),
            "tsr_cache_query": (c_int32, [P, c_uint64, POINTER(c_int32), POINTER(c_uint64),
                                          POINTER(c_int32), POINTER(c_int32)]),
            "tsr_cache_free_blocks": (c_int32, [P]),
            "tsr_copy_blocks": (c_int32, [P, c_int32, POINTER(c_int32), P, c_int32,
                                          POINTER(c_int32), c_int32, c_int64, c_int32,
                                          c_int64, c_int64, P]),
            "tsr_peak_mfma_flops": (c_int64, [c_int32, c_int32]),
            "tsr_peak_mfma": (c_int32, [c_int32, c_int32, P, P]),
            "tsr_peak_copy": (c_int32, [P, P, c_size_t, P]),
            "tsr_scorer_create": (c_int32, [c_int32, c_double, c_double, POINTER(c_void_p)]),
            "tsr_scorer_destroy": (None, [P]),
            "tsr_scorer_observe": (c_int32, [P, POINTER(c_uint64), c_int32]),
            "tsr_scorer_score": (c_double, [P, c_uint64]),
            "tsr_scorer_counts": (c_int32, [P, c_uint64, POINTER(c_int32), POINTER(c_int64)]),
            "tsr_window_for_capacity": (c_int32, [c_int64, c_double]),
            "tsr_admitter_create": (c_int32, [c_int64, c_double, POINTER(c_void_p)]),
            "tsr_admitter_destroy": (None, [P]),
            "tsr_admit": (c_int32, [P, P, c_uint64, c_int32, POINTER(c_int32),
                                    POINTER(c_uint64), c_int32, POINTER(c_int32)]),
            "tsr_admitter_remove": (c_int32, [P, c_uint64]),
            "tsr_admitter_blocks": (c_int32, [P, c_uint64]),
            "tsr_admitter_used_blocks": (c_int64, [P]),
            "tsr_admitter_num_units": (c_int32, [P]),
            "tsr_route": (c_int32, [POINTER(c_void_p), POINTER(c_int32), c_int32,
                                    POINTER(c_uint64), c_int32, POINTER(ctypes.c_uint32),
                                    POINTER(c_int32)]),
            "tsr_replay": (c_int32, [POINTER(tsr_replay_config), POINTER(c_int32),
                                     POINTER(c_uint64), POINTER(c_int32), c_int32,
                                     POINTER(tsr_replay_stats), POINTER(c_int32)]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _ptr(x) -> int | None:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s) -> int | None:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(status: int) -> None:
    if status != TSR_OK:
        raise TsrError(status, tsr_last_error())


def tsr_abi_version() -> int:
    return lib().tsr_abi_version()


def tsr_last_error() -> str:
    return lib().tsr_last_error().decode()


def make_model(n_q_heads, n_kv_heads, head_dim, page_size=16, kv_dtype="bf16",
               act_dtype="bf16", rope_theta=500000.0, max_position=65536,
               softmax_scale=0.0, rope_interleaved=0) -> tsr_model:
    return tsr_model(n_q_heads, n_kv_heads, head_dim, page_size,
                     DTYPE_CODES[kv_dtype], DTYPE_CODES[act_dtype],
                     float(rope_theta), int(rope_interleaved), max_position,
                     float(softmax_scale))


class RequestBatch:
    """ctypes arrays for a batch of requests.

    Each request needs `prompt_len`, `units` (objects with unit_id, position,
    n_tokens, residency, n_recompute, retain, pool_pages), `text_segs`
    ([(start, length)]) and `block_table`, and may carry `miss_scope`
    (TSR_SCOPE_GLOBAL when absent).  The arrays stay alive as long as this
    object.
    """

    def __init__(self, requests):
        self._keep = []
        arr = (tsr_request * max(1, len(requests)))()
        for i, r in enumerate(requests):
            units = (tsr_unit * max(1, len(r.units)))()
            for j, u in enumerate(r.units):
                pages = None
                if u.pool_pages is not None:
                    pages = np.ascontiguousarray(u.pool_pages, dtype=np.int32)
                    self._keep.append(pages)
                units[j] = tsr_unit(
                    int(u.unit_id), int(u.position), int(u.n_tokens),
                    int(u.residency), int(u.n_recompute), int(u.retain), 0,
                    pages.ctypes.data_as(POINTER(c_int32)) if pages is not None else None)
            segs = np.ascontiguousarray(np.asarray(r.text_segs, dtype=np.int32).reshape(-1, 2))
            bt = np.ascontiguousarray(r.block_table, dtype=np.int32)
            self._keep += [units, segs, bt]
            arr[i] = tsr_request(int(r.prompt_len), len(r.units), units, len(segs),
                                 int(getattr(r, "miss_scope", TSR_SCOPE_GLOBAL)),
                                 segs.ctypes.data_as(POINTER(c_int32)),
                                 bt.ctypes.data_as(POINTER(c_int32)))
        self.array = arr
        self.n = len(requests)


def tsr_rope_table_bytes(model: tsr_model) -> int:
    return lib().tsr_rope_table_bytes(ctypes.byref(model))


def tsr_rope_table_init(model: tsr_model, dev_table, table_bytes: int, stream=None) -> None:
    _check(lib().tsr_rope_table_init(ctypes.byref(model), _ptr(dev_table),
                                     table_bytes, _stream(stream)))


def tsr_plan_workspace_size(model: tsr_model, batch: RequestBatch, n_pool_pages: int,
                            n_req_pages: int, alias_v: bool = False, alias_k: bool = False,
                            split_tiles: int = 0, attn_kernel: int = 0) -> int:
    opts = tsr_plan_options(alias_v=int(alias_v), alias_k=int(alias_k),
                            split_tiles=split_tiles, attn_kernel=attn_kernel)
    n = lib().tsr_plan_workspace_size_ex(ctypes.byref(model), batch.array, batch.n,
                                         n_pool_pages, n_req_pages, ctypes.byref(opts))
    if n == 0:
        raise TsrError(TSR_ERR_INVALID_ARG, tsr_last_error())
    return n


class Plan:
    """Owner of a tsr_plan handle."""

    def __init__(self, handle: int, model: tsr_model):
        self.handle = handle
        self.model = model

    @property
    def num_compute_tokens(self) -> int:
        return lib().tsr_plan_num_compute_tokens(self.handle)

    @property
    def num_gather_tokens(self) -> int:
        return lib().tsr_plan_num_gather_tokens(self.handle)

    @property
    def num_retain_tokens(self) -> int:
        return lib().tsr_plan_num_retain_tokens(self.handle)

    @property
    def num_attn_items(self) -> int:
        return lib().tsr_plan_num_attn_items(self.handle)

    @property
    def attn_rows_per_item(self) -> int:
        return lib().tsr_plan_attn_rows_per_item(self.handle)

    def num_attn_items_part(self, part: int) -> int:
        return lib().tsr_plan_num_attn_items_part(self.handle, part)

    @property
    def num_aliased_pages(self) -> int:
        return lib().tsr_plan_num_aliased_pages(self.handle)

    @property
    def num_aliased_k_pages(self) -> int:
        return lib().tsr_plan_num_aliased_k_pages(self.handle)

    @property
    def num_attn_splits(self) -> int:
        return lib().tsr_plan_num_attn_splits(self.handle)

    def compute_positions(self):
        T = self.num_compute_tokens
        pos = np.empty(max(T, 1), dtype=np.int32)
        req = np.empty(max(T, 1), dtype=np.int32)
        _check(lib().tsr_plan_compute_positions(
            self.handle, pos.ctypes.data_as(POINTER(c_int32)),
            req.ctypes.data_as(POINTER(c_int32))))
        return pos[:T], req[:T]

    def row_kv_lo(self):
        """First visible key position of every computed row (plan order)."""
        T = self.num_compute_tokens
        lo = np.empty(max(T, 1), dtype=np.int32)
        _check(lib().tsr_plan_row_kv_lo(self.handle, lo.ctypes.data_as(POINTER(c_int32))))
        return lo[:T]

    def destroy(self) -> None:
        if self.handle:
            lib().tsr_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def tsr_plan_create(model: tsr_model, batch: RequestBatch, n_pool_pages: int,
                    n_req_pages: int, dev_rope_table=None, dev_workspace=None,
                    workspace_bytes: int = 0, stream=None, alias_v: bool = False,
                    alias_k: bool = False, split_tiles: int = 0, attn_kernel: int = 0) -> Plan:
    out = c_void_p()
    if alias_v or alias_k or split_tiles or attn_kernel:
        opts = tsr_plan_options(alias_v=int(alias_v), alias_k=int(alias_k),
                                split_tiles=split_tiles, attn_kernel=attn_kernel)
        _check(lib().tsr_plan_create_ex(ctypes.byref(model), batch.array, batch.n,
                                        n_pool_pages, n_req_pages, ctypes.byref(opts),
                                        _ptr(dev_rope_table), _ptr(dev_workspace),
                                        workspace_bytes, _stream(stream), ctypes.byref(out)))
    else:
        _check(lib().tsr_plan_create(ctypes.byref(model), batch.array, batch.n, n_pool_pages,
                                     n_req_pages, _ptr(dev_rope_table), _ptr(dev_workspace),
                                     workspace_bytes, _stream(stream), ctypes.byref(out)))
    plan = Plan(out.value, model)
    plan.alias_v = bool(alias_v)
    plan.alias_k = bool(alias_k)
    return plan


def tsr_plan_create_static(model: tsr_model, batch: RequestBatch, n_pool_pages: int,
                           n_req_pages: int, dev_rope_table, stream=None,
                           alias_v: bool = False, alias_k: bool = False,
                           split_tiles: int = 0, attn_kernel: int = 0) -> Plan:
    """A plan whose device image lives in the library's own plan area (no
    workspace); a later static plan on the same device supersedes it."""
    out = c_void_p()
    opts = tsr_plan_options(alias_v=int(alias_v), alias_k=int(alias_k),
                            split_tiles=split_tiles, attn_kernel=attn_kernel)
    _check(lib().tsr_plan_create_static(ctypes.byref(model), batch.array, batch.n,
                                        n_pool_pages, n_req_pages, ctypes.byref(opts),
                                        _ptr(dev_rope_table), _stream(stream),
                                        ctypes.byref(out)))
    plan = Plan(out.value, model)
    plan.alias_v = bool(alias_v)
    plan.alias_k = bool(alias_k)
    return plan


def tsr_compose_kv(plan: Plan, pool_k, pool_v, pool_scale, req_k, req_v, req_scale,
                   n_layers: int = 1, pool_layer_stride: int = 0,
                   req_layer_stride: int = 0, stream=None) -> None:
    _check(lib().tsr_compose_kv(plan.handle, _ptr(pool_k), _ptr(pool_v), _ptr(pool_scale),
                                _ptr(req_k), _ptr(req_v), _ptr(req_scale), n_layers,
                                pool_layer_stride, req_layer_stride, _stream(stream)))


def tsr_prefill_attn(plan: Plan, q, k, v, req_k, req_v, req_scale, out, lse=None,
                     stream=None) -> None:
    _check(lib().tsr_prefill_attn(plan.handle, _ptr(q), _ptr(k), _ptr(v), _ptr(req_k),
                                  _ptr(req_v), _ptr(req_scale), _ptr(out), _ptr(lse),
                                  _stream(stream)))


def tsr_retain_kv(plan: Plan, k, v, pool_k, pool_v, pool_scale, stream=None) -> None:
    _check(lib().tsr_retain_kv(plan.handle, _ptr(k), _ptr(v), _ptr(pool_k), _ptr(pool_v),
                               _ptr(pool_scale), _stream(stream)))


def tsr_append_kv(plan: Plan, k, v, req_k, req_v, req_scale=None, stream=None) -> None:
    _check(lib().tsr_append_kv(plan.handle, _ptr(k), _ptr(v), _ptr(req_k), _ptr(req_v),
                               _ptr(req_scale), _stream(stream)))


def tsr_assemble_kv(plan: Plan, pool_k, pool_v, pool_scale, k, v, req_k, req_v,
                    req_scale=None, stream=None) -> None:
    _check(lib().tsr_assemble_kv(plan.handle, _ptr(pool_k), _ptr(pool_v), _ptr(pool_scale),
                                 _ptr(k), _ptr(v), _ptr(req_k), _ptr(req_v),
                                 _ptr(req_scale), _stream(stream)))


def tsr_attn(plan: Plan, q, req_k, req_v, req_scale, out, lse=None, stream=None) -> None:
    _check(lib().tsr_attn(plan.handle, _ptr(q), _ptr(req_k), _ptr(req_v), _ptr(req_scale),
                          _ptr(out), _ptr(lse), _stream(stream)))


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _i32p(a: np.ndarray):
    return a.ctypes.data_as(POINTER(c_int32))


class UnitCache:
    """A context-unit cache directory (tsr_cache_*): entries PENDING/READY
    under storage epochs, read leases, draining blocks of cancelled writes."""

    def __init__(self, n_blocks: int):
        out = c_void_p()
        _check(lib().tsr_cache_create(n_blocks, ctypes.byref(out)))
        self.handle = out.value
        self.n_blocks = n_blocks

    def close(self) -> None:
        if self.handle:
            lib().tsr_cache_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def reserve(self, unit_id: int, n_blocks: int) -> tuple[int, np.ndarray]:
        ep = c_uint64()
        blocks = np.empty(max(n_blocks, 0), dtype=np.int32)
        _check(lib().tsr_cache_reserve(self.handle, unit_id, n_blocks, ctypes.byref(ep),
                                       _i32p(blocks)))
        return ep.value, blocks

    def publish(self, unit_id: int, epoch: int, blocks) -> None:
        b = _i32(blocks)
        _check(lib().tsr_cache_publish(self.handle, unit_id, epoch, _i32p(b), len(b)))

    def cancel(self, unit_id: int, epoch: int) -> None:
        _check(lib().tsr_cache_cancel(self.handle, unit_id, epoch))

    def reclaim(self, epoch: int) -> None:
        _check(lib().tsr_cache_reclaim(self.handle, epoch))

    def acquire(self, unit_id: int, max_blocks: int) -> tuple[int, np.ndarray]:
        ep, n = c_uint64(), c_int32()
        blocks = np.empty(max(max_blocks, 0), dtype=np.int32)
        _check(lib().tsr_cache_acquire(self.handle, unit_id, max_blocks, ctypes.byref(ep),
                                       _i32p(blocks), ctypes.byref(n)))
        return ep.value, blocks[:n.value].copy()

    def release(self, unit_id: int, epoch: int) -> None:
        _check(lib().tsr_cache_release(self.handle, unit_id, epoch))

    def evict(self, unit_id: int) -> None:
        _check(lib().tsr_cache_evict(self.handle, unit_id))

    def query(self, unit_id: int) -> dict:
        st, ep, nb, ls = c_int32(), c_uint64(), c_int32(), c_int32()
        _check(lib().tsr_cache_query(self.handle, unit_id, ctypes.byref(st), ctypes.byref(ep),
                                     ctypes.byref(nb), ctypes.byref(ls)))
        return {"state": st.value, "epoch": ep.value, "n_blocks": nb.value,
                "leases": ls.value}

    @property
    def free_blocks(self) -> int:
        return lib().tsr_cache_free_blocks(self.handle)


def tsr_copy_blocks(dst, n_dst_blocks: int, dst_blocks, src, n_src_blocks: int, src_blocks,
                    block_bytes: int, n_layers: int = 1, dst_layer_stride: int = 0,
                    src_layer_stride: int = 0, stream=None) -> None:
    d, sb = _i32(dst_blocks), _i32(src_blocks)
    if len(d) != len(sb):
        raise ValueError("dst_blocks and src_blocks differ in length")
    _check(lib().tsr_copy_blocks(_ptr(dst), n_dst_blocks, _i32p(d), _ptr(src), n_src_blocks,
                                 _i32p(sb), len(d), block_bytes, n_layers, dst_layer_stride,
                                 src_layer_stride, _stream(stream)))


def tsr_peak_mfma_flops(n_workgroups: int, iters: int) -> int:
    return int(lib().tsr_peak_mfma_flops(n_workgroups, iters))


def tsr_peak_mfma(n_workgroups: int, iters: int, dev_out, stream=None) -> None:
    _check(lib().tsr_peak_mfma(n_workgroups, iters, _ptr(dev_out), _stream(stream)))


def tsr_peak_copy(dst, src, nbytes: int, stream=None) -> None:
    _check(lib().tsr_peak_copy(_ptr(dst), _ptr(src), nbytes, _stream(stream)))


def tsr_attn_part(plan: Plan, part: int, q, req_k, req_v, req_scale, out, lse=None,
                  stream=None) -> None:
    _check(lib().tsr_attn_part(plan.handle, part, _ptr(q), _ptr(req_k), _ptr(req_v),
                               _ptr(req_scale), _ptr(out), _ptr(lse), _stream(stream)))


# ------------------------------------------------------------ control plane
TSR_ADMIT_BELOW_THRESHOLD, TSR_ADMIT_ADMITTED, TSR_ADMIT_RESIDENT, TSR_ADMIT_NO_ROOM, \
    TSR_ADMIT_TOO_LARGE = range(5)


def _u64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.uint64))


def _u64p(a: np.ndarray):
    return a.ctypes.data_as(POINTER(c_uint64))


class Scorer:
    """Reuse score s(u,t) = w_recent f_W + w_lifetime f_inf (tsr_scorer_*)."""

    def __init__(self, window: int, w_recent: float = 1.0, w_lifetime: float = 0.05):
        out = c_void_p()
        _check(lib().tsr_scorer_create(window, w_recent, w_lifetime, ctypes.byref(out)))
        self.handle = out.value

    def __del__(self):
        if getattr(self, "handle", None):
            lib().tsr_scorer_destroy(self.handle)
            self.handle = None

    def observe(self, unit_ids) -> None:
        u = _u64(unit_ids)
        _check(lib().tsr_scorer_observe(self.handle, _u64p(u), len(u)))

    def score(self, unit_id: int) -> float:
        return lib().tsr_scorer_score(self.handle, unit_id)

    def counts(self, unit_id: int) -> tuple[int, int]:
        r, l = c_int32(), c_int64()
        _check(lib().tsr_scorer_counts(self.handle, unit_id, ctypes.byref(r), ctypes.byref(l)))
        return r.value, l.value


def tsr_window_for_capacity(capacity_blocks: int, mean_blocks_per_request: float) -> int:
    return lib().tsr_window_for_capacity(capacity_blocks, mean_blocks_per_request)


class Admitter:
    """A cache's resident set with threshold admission (tsr_admitter_*)."""

    def __init__(self, capacity_blocks: int, theta: float):
        out = c_void_p()
        _check(lib().tsr_admitter_create(capacity_blocks, theta, ctypes.byref(out)))
        self.handle = out.value

    def __del__(self):
        if getattr(self, "handle", None):
            lib().tsr_admitter_destroy(self.handle)
            self.handle = None

    def admit(self, scorer: Scorer, unit_id: int, n_blocks: int, max_victims: int = 4096):
        res, nv = c_int32(), c_int32()
        v = np.zeros(max(max_victims, 1), dtype=np.uint64)
        _check(lib().tsr_admit(self.handle, scorer.handle, unit_id, n_blocks, ctypes.byref(res),
                               _u64p(v), max_victims, ctypes.byref(nv)))
        return res.value, [int(x) for x in v[:nv.value]]

    def remove(self, unit_id: int) -> None:
        _check(lib().tsr_admitter_remove(self.handle, unit_id))

    def blocks(self, unit_id: int) -> int:
        return lib().tsr_admitter_blocks(self.handle, unit_id)

    @property
    def used_blocks(self) -> int:
        return lib().tsr_admitter_used_blocks(self.handle)

    @property
    def num_units(self) -> int:
        return lib().tsr_admitter_num_units(self.handle)


def tsr_route(node_caches, inflight, unit_ids, rr_cursor: int = 0) -> tuple[int, int]:
    """Returns (chosen node, next round-robin cursor)."""
    n = len(inflight)
    nodes = (c_void_p * n)(*[(c.handle if c is not None else None) for c in node_caches])
    inf = _i32(inflight)
    u = _u64(unit_ids)
    rr = ctypes.c_uint32(rr_cursor)
    ch = c_int32()
    _check(lib().tsr_route(nodes, _i32p(inf), n, _u64p(u), len(u), ctypes.byref(rr),
                           ctypes.byref(ch)))
    return ch.value, rr.value


def tsr_replay(cfg: tsr_replay_config, requests, return_routes: bool = False):
    """requests: list of (unit_ids, unit_tokens) pairs.  Returns the stats
    as a dict (and the node of every request)."""
    offs = np.zeros(len(requests) + 1, dtype=np.int32)
    offs[1:] = np.cumsum([len(r[0]) for r in requests])
    ids = _u64(np.concatenate([np.asarray(r[0], np.uint64) for r in requests])
               if requests else np.zeros(0, np.uint64))
    toks = _i32(np.concatenate([np.asarray(r[1], np.int32) for r in requests])
                if requests else np.zeros(0, np.int32))
    st = tsr_replay_stats()
    routes = np.zeros(max(len(requests), 1), dtype=np.int32)
    _check(lib().tsr_replay(ctypes.byref(cfg), _i32p(offs), _u64p(ids), _i32p(toks),
                            len(requests), ctypes.byref(st), _i32p(routes)))
    stats = {n: getattr(st, n) for n, _ in tsr_replay_stats._fields_}
    return (stats, routes[:len(requests)].copy()) if return_routes else stats


def tsr_attn_aliased(plan: Plan, part: int, q, req_k, req_v, pool_k, pool_v, out, lse=None,
                     stream=None) -> None:
    _check(lib().tsr_attn_aliased(plan.handle, part, _ptr(q), _ptr(req_k), _ptr(req_v),
                                  _ptr(pool_k), _ptr(pool_v), _ptr(out), _ptr(lse),
                                  _stream(stream)))

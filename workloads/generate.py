"""Seeded generator of composed-prefill workloads.

A workload is a batch of requests.  Each request is an ordered prompt made of
text segments (instruction, query) and context units (retrieved chunks or
memory records).  Every unit occurrence carries what the paper's per-unit plan
carries (Section 5.1): a stable identity, its length, its prompt offset, its
preparation (cached -> HIT, computed -> MISS), the number of leading tokens
the composition policy recomputes, a retention permission, and the ids of the
ceil(n/B) non-adjacent storage blocks that hold (or will hold) its state.

Values are N(0,1) draws rounded (by torch's CPU conversion) to the storage
dtype.  Cached unit states are keyed by unit id; fresh per-token projections
(q, k, v of the tokens that a request computes) are keyed by (request,
position) so that any subset of positions can be drawn on demand.

Nothing in this module implements the method: it does not decide which tokens
are computed, does not rotate, gather, attend or scatter.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable

import numpy as np
import torch

from .configs import ModelShape, WorkloadConfig, get_config

MISS = 0
HIT = 1

_TAG_FRESH = 0x51F
_TAG_UNIT = 0xCAC4E
_TAG_LEN = 0x1E4
_TAG_SCALE = 0x5CA1E
_SCOPES = {"global": 0, "local": 1}


@dataclass
class UnitRef:
    unit_id: int
    n_tokens: int
    position: int
    residency: int          # MISS / HIT
    n_recompute: int
    retain: int             # 1: scatter the computed state to pool_pages
    pool_pages: np.ndarray  # int32 [ceil(n_tokens / B)]


@dataclass
class RequestSpec:
    prompt_len: int
    units: list[UnitRef]
    text_segs: list[tuple[int, int]]   # (start, length), length > 0
    block_table: np.ndarray            # int32 [ceil(prompt_len / B)]
    miss_scope: int = 0                # 0: global, 1: local


def _round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float32 draws to the storage dtype, returned as float32 values."""
    if dtype == "f32":
        return x.astype(np.float32, copy=False)
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
        return t.to(torch.bfloat16).to(torch.float32).numpy()
    raise ValueError(f"no value rounding for dtype {dtype!r}")


@dataclass
class Workload:
    name: str
    seed: int
    model: ModelShape
    requests: list[RequestSpec]
    n_pool_pages: int
    n_req_pages: int
    unit_len: np.ndarray            # int32 [pool_units]
    unit_pages: list[np.ndarray]    # per unit id: its pool page ids
    cfg: WorkloadConfig | None = None
    # test hooks: replace the value draws (used to build invariance cases)
    unit_state_fn: Callable | None = field(default=None, repr=False)
    fresh_fn: Callable | None = field(default=None, repr=False)

    # ------------------------------------------------------------ structure
    @property
    def prompt_tokens(self) -> int:
        return sum(r.prompt_len for r in self.requests)

    def hit_unit_ids(self) -> list[int]:
        ids = {u.unit_id for r in self.requests for u in r.units if u.residency == HIT}
        return sorted(ids)

    # --------------------------------------------------------------- values
    def unit_state(self, unit_id: int) -> tuple[np.ndarray, np.ndarray]:
        """Cached reusable form of a unit: pre-RoPE K and V, [n][H_kv][d].

        Values are float32 holding numbers exactly representable in the
        model's KV dtype.  For e4m3 pools use unit_state_e4m3 instead.
        """
        if self.unit_state_fn is not None:
            return self.unit_state_fn(unit_id)
        m = self.model
        if m.kv_dtype == "e4m3":
            raise ValueError("e4m3 pool: use unit_state_e4m3")
        n = int(self.unit_len[unit_id])
        rng = np.random.default_rng((self.seed, _TAG_UNIT, int(unit_id)))
        shape = (n, m.n_kv_heads, m.head_dim)
        k = rng.standard_normal(shape, dtype=np.float32)
        v = rng.standard_normal(shape, dtype=np.float32)
        return _round_to(k, m.kv_dtype), _round_to(v, m.kv_dtype)

    def unit_state_e4m3(self, unit_id: int):
        """e4m3 cached state: (k_codes, v_codes) uint8 [n][H_kv][d] and
        per-page power-of-two scales (k_scale, v_scale) float32 [pages].

        Codes are torch's e4m3fn encoding of N(0,1)/scale draws clamped to the
        finite range, so code * scale is distributed like N(0,1).  As in any
        pool written by the retention quantizer, each page's scale is the
        smallest power of two that covers the page: one element of every
        page, at a seeded random (slot, head, dim) among its valid slots and
        with a random sign, holds the largest finite magnitude (448).
        """
        m = self.model
        n = int(self.unit_len[unit_id])
        pages = -(-n // m.page_size)
        rng = np.random.default_rng((self.seed, _TAG_UNIT, int(unit_id)))
        srng = np.random.default_rng((self.seed, _TAG_SCALE, int(unit_id)))
        out = []
        for _ in range(2):
            exps = srng.integers(-7, -4, size=pages)          # 2^-7 .. 2^-5
            scale = np.ldexp(np.float32(1.0), exps).astype(np.float32)
            x = rng.standard_normal((n, m.n_kv_heads, m.head_dim), dtype=np.float32)
            tok_scale = np.repeat(scale, m.page_size)[:n]
            x = np.clip(x / tok_scale[:, None, None], -448.0, 448.0)
            codes = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
            B = m.page_size
            for pg in range(pages):
                nv = min(B, n - pg * B)
                j = pg * B + int(srng.integers(nv))
                h = int(srng.integers(m.n_kv_heads))
                d = int(srng.integers(m.head_dim))
                codes[j, h, d] = 0xFE if srng.integers(2) else 0x7E   # -448 / +448
            out.append((codes, scale))
        (kc, ks), (vc, vs) = out
        return kc, vc, ks, vs

    def fresh(self, req: int, positions) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
        """Fresh pre-RoPE projections of request `req` at `positions`.

        Returns q [n][H_q][d], k [n][H_kv][d], v [n][H_kv][d] as float32
        holding values representable in the activation dtype.
        """
        positions = np.asarray(positions, dtype=np.int64)
        if self.fresh_fn is not None:
            return self.fresh_fn(req, positions)
        m = self.model
        nq = m.n_q_heads * m.head_dim
        nk = m.n_kv_heads * m.head_dim
        buf = np.empty((len(positions), nq + 2 * nk), dtype=np.float32)
        for i, p in enumerate(positions):
            rng = np.random.default_rng((self.seed, _TAG_FRESH, int(req), int(p)))
            buf[i] = rng.standard_normal(nq + 2 * nk, dtype=np.float32)
        buf = _round_to(buf, m.act_dtype)
        q = buf[:, :nq].reshape(-1, m.n_q_heads, m.head_dim)
        k = buf[:, nq:nq + nk].reshape(-1, m.n_kv_heads, m.head_dim)
        v = buf[:, nq + nk:].reshape(-1, m.n_kv_heads, m.head_dim)
        return np.ascontiguousarray(q), np.ascontiguousarray(k), np.ascontiguousarray(v)


def _zipf_probs(n: int, s: float) -> np.ndarray:
    w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    return w / w.sum()


def make_workload(cfg: WorkloadConfig) -> Workload:
    m = cfg.model
    B = m.page_size
    rng = np.random.default_rng((cfg.seed, 0))

    # unit lengths are part of a unit's identity
    if isinstance(cfg.unit_tokens, tuple):
        lrng = np.random.default_rng((cfg.seed, _TAG_LEN))
        lo, hi = cfg.unit_tokens
        unit_len = lrng.integers(lo, hi + 1, size=cfg.pool_units).astype(np.int32)
        unit_len *= int(cfg.extra.get("unit_tokens_multiple", 1))
    else:
        unit_len = np.full(cfg.pool_units, cfg.unit_tokens, dtype=np.int32)

    # every unit of the universe owns ceil(n/B) pool pages, scattered at random
    pages_per_unit = -(-unit_len // B)
    n_pool_pages = int(pages_per_unit.sum())
    perm = rng.permutation(n_pool_pages).astype(np.int32)
    offs = np.concatenate([[0], np.cumsum(pages_per_unit)])
    unit_pages = [perm[offs[u]:offs[u + 1]] for u in range(cfg.pool_units)]

    # per request: ordered unit ids and their residency
    probs = _zipf_probs(cfg.pool_units, cfg.zipf_s)
    orders, residencies = [], []
    for r in range(cfg.n_requests):
        if cfg.unit_order is not None:
            ids = np.asarray(cfg.unit_order[r], dtype=np.int64)
        else:
            if isinstance(cfg.units_per_request, tuple):
                lo, hi = cfg.units_per_request
                k = int(rng.integers(lo, hi + 1))
            else:
                k = cfg.units_per_request
            k = min(k, cfg.pool_units)
            ids = rng.choice(cfg.pool_units, size=k, replace=False, p=probs)
        k = len(ids)
        if cfg.residency_pattern is not None:
            res = np.asarray(cfg.residency_pattern[:k], dtype=np.int32)
        elif cfg.n_missing is not None:
            res = np.full(k, HIT, dtype=np.int32)
            res[rng.choice(k, size=min(cfg.n_missing, k), replace=False)] = MISS
        else:
            res = (rng.random(k) < cfg.hit_prob).astype(np.int32)
        orders.append(ids)
        residencies.append(res)

    # retention: a unit cached nowhere in the batch is retained by its first
    # computing occurrence; its pool pages are then read by nobody in the batch
    hit_anywhere = {int(u) for ids, res in zip(orders, residencies)
                    for u, h in zip(ids, res) if h == HIT}
    retained: set[int] = set()

    # prompt construction: instruction, units in retrieval order, query
    requests: list[RequestSpec] = []
    req_page_counts = []
    for r in range(cfg.n_requests):
        units = []
        text = []
        pos = 0
        if cfg.instruction_tokens > 0:
            text.append((0, cfg.instruction_tokens))
            pos = cfg.instruction_tokens
        for uid, h in zip(orders[r], residencies[r]):
            uid = int(uid)
            n = int(unit_len[uid])
            retain = 0
            if (h == MISS and cfg.retain_misses and uid not in hit_anywhere
                    and uid not in retained):
                retain = 1
                retained.add(uid)
            units.append(UnitRef(unit_id=uid, n_tokens=n, position=pos,
                                 residency=int(h), n_recompute=cfg.n_recompute,
                                 retain=retain, pool_pages=unit_pages[uid].copy()))
            pos += n
        if cfg.query_tokens > 0:
            text.append((pos, cfg.query_tokens))
            pos += cfg.query_tokens
        requests.append(RequestSpec(prompt_len=pos, units=units, text_segs=text,
                                    block_table=np.empty(0, dtype=np.int32),
                                    miss_scope=_SCOPES[cfg.miss_scope]))
        req_page_counts.append(-(-pos // B))

    n_req_pages = int(sum(req_page_counts))
    rperm = rng.permutation(n_req_pages).astype(np.int32)
    o = 0
    for req, c in zip(requests, req_page_counts):
        req.block_table = rperm[o:o + c].copy()
        o += c

    return Workload(name=cfg.name, seed=cfg.seed, model=m, requests=requests,
                    n_pool_pages=n_pool_pages, n_req_pages=n_req_pages,
                    unit_len=unit_len, unit_pages=unit_pages, cfg=cfg)


def generate(name_or_cfg) -> Workload:
    cfg = get_config(name_or_cfg) if isinstance(name_or_cfg, str) else name_or_cfg
    return make_workload(cfg)

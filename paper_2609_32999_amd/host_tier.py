"""Host tier of the context-unit cache, with bounded device staging.

A generation node keeps unit states in a cache in pinned host memory
(Section 5.2).  Preparing a request's local hits copies their blocks into a
bounded staging arena in device memory with the copy engines; compose then
places them at the request's positions and re-rotates the keys (Section 5.3,
"Preparing cache hits").  A hit whose entry is no longer READY when it is
revalidated, or that does not fit in staging, falls back to being computed
from text (Section 5.3, "Preparation failures").  A retained unit is written
by the retain kernel into staging blocks, copied back into blocks reserved
under a fresh storage epoch, and published only once that copy has
completed; a failed writeback is cancelled and its blocks are reclaimed once
the copy stream has drained (Section 5.4).

Only bookkeeping and marshalling happen here: the directory is libtsr's
tsr_cache, the transfers are tsr_copy_blocks, and compose, attention and
retain are libtsr's kernels, run through a Session whose pool arena is the
staging arena.

Block layout.  The host arena holds [n_layers][n_blocks][H_kv][B][d] for K
and for V (and [n_layers][n_blocks][2] fp32 scales for e4m3): a block is one
page of every layer.  The staging arena is the Session's pool arena,
[n_layers][n_staging] pages in device memory; a batch's hits and retained
units take consecutive slots of it, and the plan names those slots as their
pool pages.
"""
from __future__ import annotations

import copy
from dataclasses import dataclass, field

import numpy as np
import torch

from . import _binding as B
from .session import Session


@dataclass
class Prepared:
    """One batch's preparation: the requests rewritten for the staging
    arena, and what has to be released or published once transfers end."""
    requests: list
    fallbacks: list = field(default_factory=list)      # (request, unit) downgraded to MISS
    declined: list = field(default_factory=list)       # (request, unit) retention declined
    leases: list = field(default_factory=list)         # (unit_id, epoch)
    stage_src: np.ndarray = None                       # host blocks copied in
    stage_dst: np.ndarray = None                       # staging slots they land in
    # retained units: (unit_id, epoch, host blocks, staging slots)
    reservations: list = field(default_factory=list)
    staged: torch.cuda.Event | None = None
    written: torch.cuda.Event | None = None
    published: list = field(default_factory=list)      # unit ids made READY
    cancelled: list = field(default_factory=list)      # unit ids whose writeback failed
    errors: list = field(default_factory=list)         # messages of failed enqueues
    out_blocks: np.ndarray = None                      # cache blocks written back, in order


class HostTier:
    def __init__(self, shape, n_blocks: int, n_staging: int, n_req_pages: int,
                 n_layers: int = 1, device: str = "cuda"):
        """`shape` as for Session.  n_blocks: host cache arena size in blocks;
        n_staging: staging arena size in pages (the bound on the blocks one
        batch may stage in plus write back)."""
        self.sess = Session(shape, n_staging, n_req_pages, device=device, n_layers=n_layers)
        s = self.sess
        self.cache = B.UnitCache(n_blocks)
        self.n_blocks = n_blocks
        self.n_staging = n_staging
        self.n_layers = n_layers
        self.page_size = shape.page_size
        page = (shape.n_kv_heads, shape.page_size, shape.head_dim)
        # [K|V][layer][block], like the staging arena: one strided copy per
        # run of blocks moves K and V of every layer
        self.host_kv = torch.empty((2, n_layers, n_blocks, *page), dtype=s.kv_dtype,
                                   pin_memory=True)
        self.host_k, self.host_v = self.host_kv[0], self.host_kv[1]
        self.host_scale = self._bounce_in = self._bounce_out = None
        if s.e4m3:
            self.host_scale = torch.empty((n_layers, n_blocks, 2), dtype=torch.float32,
                                          pin_memory=True)
            # page scales are 8 bytes a block: gathered on the host into a
            # pinned bounce buffer and moved in one copy, not one per run
            self._bounce_in = torch.empty((n_layers, n_staging, 2), dtype=torch.float32,
                                          pin_memory=True)
            self._bounce_out = torch.empty_like(self._bounce_in)
        self._bounce_busy = None            # event of the last copy reading _bounce_in
        self._out_pending = None            # batch whose _bounce_out finish() has to scatter
        self.copy_stream = torch.cuda.Stream(device=s.device)

    # ------------------------------------------------------------ copies
    # Slab pitch above which K/V/layers are not folded into one strided copy.
    MAX_PITCH = 1 << 32

    def _copy_kv(self, to_staging: bool, host_blocks, slots, stream) -> None:
        """K and V of every layer for the listed blocks: one strided copy per
        run of consecutive (block, slot) pairs, the 2 * n_layers slabs of an
        arena being its rows."""
        if len(slots) == 0:
            return
        s = self.sess
        blk = self.host_kv[0, 0, 0].nbytes
        hp, sp = self.host_k[0].nbytes, s.pool_k[0].nbytes     # slab pitches
        host = (self.host_kv, self.n_blocks, host_blocks)
        stg = (s.pool_kv, self.n_staging, slots)
        dst, src = (stg, host) if to_staging else (host, stg)
        if max(hp, sp) <= self.MAX_PITCH:
            B.tsr_copy_blocks(*dst, *src, blk, n_layers=2 * self.n_layers,
                              dst_layer_stride=dst[0][0, 0].nbytes,
                              src_layer_stride=src[0][0, 0].nbytes, stream=stream)
            return
        for kv in range(2):
            for l in range(self.n_layers):
                B.tsr_copy_blocks(dst[0][kv, l], dst[1], dst[2], src[0][kv, l], src[1], src[2],
                                  blk, stream=stream)

    def _stage_scales(self, host_blocks, slots, stream) -> None:
        """e4m3: gather the blocks' page scales into the bounce buffer on the
        host, then one copy into the staging slots."""
        n = len(slots)
        if n == 0 or self.host_scale is None:
            return
        if self._bounce_busy is not None:
            self._bounce_busy.synchronize()
        idx = torch.from_numpy(np.asarray(host_blocks, dtype=np.int64))
        for l in range(self.n_layers):
            self._bounce_in[l, :n] = self.host_scale[l, idx]
        st = self.sess.pool_scale
        B.tsr_copy_blocks(st, self.n_staging, slots, self._bounce_in, self.n_staging,
                          np.arange(n, dtype=np.int32), 8, n_layers=self.n_layers,
                          dst_layer_stride=st[0].nbytes,
                          src_layer_stride=self._bounce_in[0].nbytes, stream=stream)
        self._bounce_busy = torch.cuda.Event()
        self._bounce_busy.record(stream)

    def _unstage_scales(self, slots, stream) -> None:
        """e4m3: copy the retained slots' page scales into the outgoing bounce
        buffer (scattered into the cache by finish())."""
        n = len(slots)
        if n == 0 or self.host_scale is None:
            return
        st = self.sess.pool_scale
        B.tsr_copy_blocks(self._bounce_out, self.n_staging, np.arange(n, dtype=np.int32), st,
                          self.n_staging, slots, 8, n_layers=self.n_layers,
                          dst_layer_stride=self._bounce_out[0].nbytes,
                          src_layer_stride=st[0].nbytes, stream=stream)

    # ---------------------------------------------------------- contents
    def insert(self, unit_id: int, k_pages, v_pages, scales=None) -> np.ndarray:
        """Place a unit's state (host tensors [n_layers][pages][H_kv][B][d],
        scales [n_layers][pages][2] for e4m3) into freshly reserved blocks and
        publish it.  A plain host write: nothing is in flight."""
        npg = k_pages.shape[1]
        epoch, blocks = self.cache.reserve(unit_id, npg)
        idx = torch.as_tensor(blocks.astype(np.int64))
        self.host_k[:, idx] = k_pages.to(self.host_k.dtype)
        self.host_v[:, idx] = v_pages.to(self.host_v.dtype)
        if self.host_scale is not None:
            self.host_scale[:, idx] = scales
        self.cache.publish(unit_id, epoch, blocks)
        return blocks

    # ------------------------------------------------------- preparation
    def prepare(self, requests, stream=None, fail_units=(), wait: bool = True) -> Prepared:
        """Revalidate the batch's hits and assign staging (plan_preparation),
        then enqueue the host-to-staging copies on the copy stream.  With
        `wait`, `stream` (the stream compose will run on) waits for them at
        once; otherwise the caller calls wait_staged() before compose and may
        enqueue work that needs no staged state (append, the attention items
        before compose) in between."""
        prep = plan_preparation(self.cache, requests, self.n_staging, self.page_size,
                                fail_units)
        self.stage(prep, stream, wait)
        return prep

    def stage(self, prep: Prepared, stream=None, wait: bool = True) -> None:
        """Enqueue a prepared batch's host-to-staging copies on the copy
        stream, after the work already on `stream`; with `wait`, `stream`
        waits for them."""
        s = stream or self.sess.stream
        # the copies overwrite staging: wait for earlier work that reads it
        self.copy_stream.wait_stream(s)
        try:
            self._copy_kv(True, prep.stage_src, prep.stage_dst, self.copy_stream)
            self._stage_scales(prep.stage_src, prep.stage_dst, self.copy_stream)
        except B.TsrError:
            _undo(self.cache, prep, self.copy_stream)
            raise
        prep.staged = torch.cuda.Event()
        prep.staged.record(self.copy_stream)
        if wait:
            s.wait_event(prep.staged)

    def wait_staged(self, prep: Prepared, stream=None) -> None:
        """Make `stream` wait for the batch's staging copies."""
        (stream or self.sess.stream).wait_event(prep.staged)

    # --------------------------------------------------------- retention
    def writeback(self, prep: Prepared, stream=None, fail_units=()) -> None:
        """After the retain kernel (enqueued on `stream`), copy the retained
        units' staging blocks into their reserved host blocks on the copy
        stream.  `fail_units` marks those units' writeback as failed."""
        s = stream or self.sess.stream
        if self._out_pending is not None:
            raise RuntimeError("finish() the previous batch before the next writeback")
        self.copy_stream.wait_stream(s)
        ok = [(u, e, b, sl) for (u, e, b, sl) in prep.reservations if u not in fail_units]
        prep.cancelled = [u for (u, e, b, sl) in prep.reservations if u in fail_units]
        if ok:
            hb = np.concatenate([b for (_, _, b, _) in ok])
            sl = np.concatenate([x for (_, _, _, x) in ok])
            prep.out_blocks = hb
            if self.host_scale is not None:
                self._out_pending = prep
            try:
                self._copy_kv(False, hb, sl, self.copy_stream)
                self._unstage_scales(sl, self.copy_stream)
            except B.TsrError as e:
                # a failed writeback only loses future reuse: nothing of this
                # batch is published, and finish() reclaims once drained
                prep.cancelled = [u for (u, _, _, _) in prep.reservations]
                prep.errors.append(str(e))
        prep.written = torch.cuda.Event()
        prep.written.record(self.copy_stream)
        s.wait_event(prep.written)

    def finish(self, prep: Prepared) -> None:
        """Once the staged copies have completed, release the read leases;
        once the writeback has completed, publish every retained unit
        (PENDING -> READY under its epoch) and cancel and reclaim the failed
        ones.  Blocks the host until those copies end."""
        if prep.staged is not None:
            prep.staged.synchronize()
        for uid, epoch in prep.leases:
            self.cache.release(uid, epoch)
        prep.leases = []
        if prep.reservations and prep.written is None:
            raise RuntimeError("writeback() was not called for a batch with retained units")
        if prep.written is not None:
            prep.written.synchronize()
        if self._out_pending is prep:
            self._out_pending = None
        if self.host_scale is not None and prep.out_blocks is not None and not prep.errors:
            idx = torch.from_numpy(np.asarray(prep.out_blocks, dtype=np.int64))
            for l in range(self.n_layers):
                self.host_scale[l, idx] = self._bounce_out[l, :len(idx)]
        for uid, epoch, blocks, _ in prep.reservations:
            if uid in prep.cancelled:
                self.cache.cancel(uid, epoch)
                self.cache.reclaim(epoch)     # the copy stream has drained
            else:
                self.cache.publish(uid, epoch, blocks)
                prep.published.append(uid)
        prep.reservations = []


def plan_preparation(cache, requests, n_staging: int, page_size: int,
                     fail_units=()) -> Prepared:
    """Host half of preparing a batch (Section 5.3): no HIP call.

    For every HIT, in request order: revalidate it against the directory by
    taking a read lease (a unit staged once serves every request of the
    batch that hits it).  A hit that is not READY, whose block count
    changed, that does not fit in the staging arena, or that is listed in
    `fail_units` (a stand-in for a failed or timed-out transfer) is released
    and falls back to MISS: its tokens become computed rows and it is not
    retained.
    For every MISS with retain = 1: reserve its cache blocks under a new
    storage epoch.  If an entry exists (another writer holds it PENDING, or
    it is READY), there is no room, or the unit is already reserved in this
    batch, retention is declined (retain = 0) and the request proceeds
    (Section 5.4).
    Staging slots: the staged hits first, ordered by their first cache
    block (so that units adjacent in the cache stay adjacent in staging and
    their copies merge), then the retained units.  Returns the requests
    rewritten so that pool pages name staging slots."""
    prep = Prepared(requests=[])
    staged = {}                 # unit id -> (epoch, cache blocks)
    retained = {}               # unit id -> (epoch, cache blocks)
    used = 0
    rows = []                   # per request: list of (unit copy, kind)
    for ri, r in enumerate(requests):
        units = []
        for ui, u in enumerate(r.units):
            nb = -(-int(u.n_tokens) // page_size)
            nu = copy.copy(u)
            kind = None
            if u.residency == B.TSR_HIT:
                if u.unit_id not in staged:
                    try:
                        got = cache.acquire(u.unit_id, nb)
                    except B.TsrError:
                        got = None                  # not READY any more
                    if got is not None and (len(got[1]) != nb or used + nb > n_staging
                                            or u.unit_id in fail_units):
                        cache.release(u.unit_id, got[0])
                        got = None
                    if got is None:
                        nu.residency = B.TSR_MISS
                        nu.retain = 0
                        nu.pool_pages = np.zeros(0, dtype=np.int32)
                        prep.fallbacks.append((ri, ui))
                        units.append((nu, None))
                        continue
                    staged[u.unit_id] = got
                    prep.leases.append((u.unit_id, got[0]))
                    used += nb
                kind = "hit"
            elif u.retain:
                got = None
                if used + nb <= n_staging and u.unit_id not in retained:
                    try:
                        got = cache.reserve(u.unit_id, nb)
                    except B.TsrError:
                        got = None                  # an entry exists, or no room
                if got is None:
                    nu.retain = 0
                    nu.pool_pages = np.zeros(0, dtype=np.int32)
                    prep.declined.append((ri, ui))
                    units.append((nu, None))
                    continue
                retained[u.unit_id] = got
                used += nb
                kind = "retain"
            units.append((nu, kind))
        rows.append((r, units))
    # slots: staged hits by first cache block, then retained units in order
    slots = {}
    nxt = 0
    src, dst = [], []
    for uid, (epoch, blocks) in sorted(staged.items(), key=lambda kv: int(kv[1][1][0])):
        sl = np.arange(nxt, nxt + len(blocks), dtype=np.int32)
        nxt += len(blocks)
        slots[uid] = sl
        src.append(blocks)
        dst.append(sl)
    for uid, (epoch, blocks) in retained.items():
        sl = np.arange(nxt, nxt + len(blocks), dtype=np.int32)
        nxt += len(blocks)
        slots[("r", uid)] = sl
        prep.reservations.append((uid, epoch, blocks, sl))
    for r, units in rows:
        out = []
        for nu, kind in units:
            if kind == "hit":
                nu.pool_pages = slots[nu.unit_id]
            elif kind == "retain":
                nu.pool_pages = slots[("r", nu.unit_id)]
            out.append(nu)
        nr = copy.copy(r)
        nr.units = out
        prep.requests.append(nr)
    prep.stage_src = np.concatenate(src) if src else np.zeros(0, np.int32)
    prep.stage_dst = np.concatenate(dst) if dst else np.zeros(0, np.int32)
    return prep


def _undo(cache, prep: Prepared, copy_stream) -> None:
    """A copy could not be enqueued: wait for what was, then drop the
    batch's leases and reservations."""
    copy_stream.synchronize()
    for uid, epoch in prep.leases:
        cache.release(uid, epoch)
    for uid, epoch, _, _ in prep.reservations:
        cache.cancel(uid, epoch)
        cache.reclaim(epoch)
    prep.leases, prep.reservations = [], []

"""Benchmark of the composed-prefill hot path on one MI355X.

A step is one attention layer of one batch: compose (gather + RoPE
re-rotation of cached units) -> append + causal GQA prefill attention of the
computed rows (main stream), with retention of computed units running
concurrently on a side stream and joined at the end of the step.  Steps
rotate over --layers distinct layer buffer sets (pool, request KV, inputs),
as consecutive model layers would, so one layer's data is not served from
the previous step's caches.

Prints one JSON line.  `value` is prompt tokens per second per layer.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
PEAK_MFMA_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
# e4m3 KV: QK^T runs in fp8 MFMA (5.0 PFLOP/s dense) and PV in fp16 MFMA
# (2.5 PFLOP/s), half of the FLOPs each: blended peak 1 / (0.5/5.0 + 0.5/2.5).
PEAK_E4M3_BLEND = 1.0 / (0.5 / 5000.0 + 0.5 / 2500.0)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def measured_peaks(torch):
    """Achievable rates on this GPU, as context for the published peaks:
    libtsr's MFMA loop (back-to-back bf16 32x32x16 MFMAs on registers) and
    copy kernel (16-byte loads and stores, 1 GiB), plus a 1 GiB torch
    device copy and a bf16 8192^3 matrix product through torch.matmul (the
    vendor GEMM library).  Copy rates count read + write bytes."""
    import paper_2609_32999_amd as P
    ev = lambda: torch.cuda.Event(enable_timing=True)

    def timed(fn, reps):
        fn()
        t0, t1 = ev(), ev()
        t0.record()
        for _ in range(reps):
            fn()
        t1.record()
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) * 1e-3 / reps

    n_wg, iters = 2048, 2000
    sink = torch.empty(n_wg * 256, dtype=torch.float32, device="cuda")
    t = timed(lambda: P.tsr_peak_mfma(n_wg, iters, sink), 5)
    mfma_loop = P.tsr_peak_mfma_flops(n_wg, iters) / t / 1e12
    a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda").fill_(1)
    b = torch.empty_like(a)
    copy_kernel = 2 * a.numel() / timed(lambda: P.tsr_peak_copy(b, a, a.numel()), 5) / 1e9
    if not torch.equal(a[:1 << 20], b[:1 << 20]):
        raise RuntimeError("tsr_peak_copy produced a wrong copy")
    copy_gbps = 2 * a.numel() / timed(lambda: b.copy_(a), 5) / 1e9
    del a, b, sink
    n = 8192
    x = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    y = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    gemm_tflops = 2.0 * n ** 3 / timed(lambda: x @ y, 5) / 1e12
    del x, y
    torch.cuda.empty_cache()
    log(f"[bench] measured peaks: MFMA loop {mfma_loop:.0f} TFLOP/s, bf16 GEMM "
        f"{gemm_tflops:.0f} TFLOP/s, copy kernel {copy_kernel:.0f} GB/s, torch copy "
        f"{copy_gbps:.0f} GB/s")
    return {"mfma_loop_tflops": mfma_loop, "bf16_gemm_tflops": gemm_tflops,
            "copy_kernel_gbps": copy_kernel, "copy_gbps": copy_gbps,
            "how": "libtsr MFMA loop (2048 workgroups x 2000 x 8 bf16 32x32x16 MFMAs per "
                   "wave) and copy kernel (1 GiB); torch 1 GiB device copy; torch.matmul "
                   "bf16 8192^3; 5 timed repetitions each"}


def kv_elem_bytes(dtype):
    return {"f32": 4, "bf16": 2, "e4m3": 1}[dtype]


def profiled_traffic(workload: str, kernel: str):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary (FETCH_SIZE and WRITE_SIZE scaled against a plain copy), or None
    if there is none or the kernel's source changed since it was taken."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", f"{workload}_kernels.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"```json\n(.*?)\n```", text, re.S)
    if not m:
        return None
    for name, rec in json.loads(m.group(1)).items():
        if name != kernel:
            continue
        src = os.path.join(ROOT, rec["source"])
        digest = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
        return rec["traffic_bytes"] if digest == rec["source_sha256_16"] else None
    return None


def cpu_baseline(wl, n_req):
    """Time the CPU oracle on the first n_req requests of the same batch."""
    import threadpoolctl
    from oracle import pipeline as PL
    from oracle.compose import retained_pages
    info = threadpoolctl.threadpool_info()
    cores = max([i.get("num_threads", 1) for i in info] + [1])
    t0 = time.perf_counter()
    toks = 0
    for r in range(n_req):
        PL.run_request(wl, r)
        toks += wl.requests[r].prompt_len
    sub = type(wl)(**{**vars(wl), "requests": wl.requests[:n_req]})
    retained_pages(sub)
    dt = time.perf_counter() - t0
    return {"value": toks / dt, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"requests 0..{n_req - 1} of the batch ({toks} prompt tokens): "
                      f"compose + append + attention (all heads, fp64) + retain; "
                      f"{dt:.1f} s on {cores} BLAS threads (os.cpu_count()={os.cpu_count()})"}


def host_tier(torch, wl, plan, k, v, row_bytes, reps=5):
    """Compose and retain against a pool held in pinned host memory (the host
    tier): the same kernels read the cached pages, and write the retained
    ones, across the host link.  Reported beside a plain pinned-host <->
    device copy of similar size, the link's achievable rate."""
    from paper_2609_32999_amd import staging
    from paper_2609_32999_amd.session import Session
    m = wl.model
    hs = Session(m, wl.n_pool_pages, wl.n_req_pages, n_layers=1, pool="host")
    staging.upload_pool(hs, wl, layer=0)
    s = torch.cuda.current_stream()
    E = lambda: torch.cuda.Event(enable_timing=True)

    def timed(fn):
        fn()
        a, b = E(), E()
        a.record(s)
        for _ in range(reps):
            fn()
        b.record(s)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    compose_ms = timed(lambda: hs.compose(plan, layer=0, stream=s))
    retain_ms = timed(lambda: hs.retain(plan, k, v, layer=0, stream=s))
    nb = max(plan.num_gather_tokens * row_bytes, 64 << 20)
    h = torch.empty(nb, dtype=torch.uint8, pin_memory=True)
    d = torch.empty(nb, dtype=torch.uint8, device="cuda")
    h2d_ms = timed(lambda: d.copy_(h, non_blocking=True))
    d2h_ms = timed(lambda: h.copy_(d, non_blocking=True))
    read = plan.num_gather_tokens * row_bytes       # crosses the link once
    written = plan.num_retain_tokens * row_bytes
    log(f"[bench] host tier: compose {compose_ms * 1e3:.1f} us, retain {retain_ms * 1e3:.1f} us")
    del hs, h, d
    return {
        "compose_us": compose_ms * 1e3,
        "compose_link_gbps": read / (compose_ms * 1e-3) / 1e9,
        "retain_us": retain_ms * 1e3,
        "retain_link_gbps": written / (retain_ms * 1e-3) / 1e9 if written else None,
        "copy_h2d_gbps": nb / (h2d_ms * 1e-3) / 1e9,
        "copy_d2h_gbps": nb / (d2h_ms * 1e-3) / 1e9,
        "copy_bytes": nb,
    }


def host_tier_staged(torch, wl, reps=5, warmup=2):
    """One layer of a batch through the host tier with device staging (the
    paper's path for local hits): the hits' blocks are copied from the
    pinned host cache into a bounded staging arena by the copy engines,
    compose places them, and retained units are written back to the cache
    through staging.  Timed two ways: in order (stage, then append, compose,
    attention), and overlapped (append and the attention items that read no
    composed key run while the copies are in flight; compose and the other
    items follow).  Retain and the writeback are in both."""
    from paper_2609_32999_amd import TSR_ATTN_AFTER_COMPOSE, TSR_ATTN_BEFORE_COMPOSE, staging
    from paper_2609_32999_amd.host_tier import HostTier, plan_preparation
    m = wl.model
    B = m.page_size
    hits = wl.hit_unit_ids()
    hit_pages = sum(-(-int(wl.unit_len[u]) // B) for u in hits)
    ret_pages = sum(-(-int(u.n_tokens) // B) for r in wl.requests for u in r.units
                    if u.residency == 0 and u.retain)
    n = hit_pages + ret_pages
    # the cache also holds other units: one 32-page entry after every hit
    # unit, so that no two hit units are adjacent and each is its own copy
    gap = 32
    tier = HostTier(m, n + gap * len(hits), n, wl.n_req_pages)
    for i, uid in enumerate(hits):
        if m.kv_dtype == "e4m3":
            kc, vc, ks, vs = wl.unit_state_e4m3(uid)
            sc = torch.from_numpy(np.stack([ks, vs], axis=1))[None]
        else:
            kc, vc = wl.unit_state(uid)
            sc = None
        kp = torch.from_numpy(staging._pages_from_tokens(kc, B))[None]
        vp = torch.from_numpy(staging._pages_from_tokens(vc, B))[None]
        tier.insert(uid, kp, vp, sc)
        ep, blocks = tier.cache.reserve((1 << 40) + i, gap)
        tier.cache.publish((1 << 40) + i, ep, blocks)
    s = tier.sess
    main = s.stream
    prep0 = plan_preparation(tier.cache, wl.requests, n, B)
    tier.stage(prep0, main)
    plan = s.plan(prep0.requests)
    q, k, v = staging.fresh_inputs(s, wl, plan)
    out, lse = s.new_outputs(plan, with_lse=True)
    E = lambda: torch.cuda.Event(enable_timing=True)

    def close(prep):
        tier.finish(prep)
        for uid in prep.published:       # keep every step's directory state alike
            tier.cache.evict(uid)

    n_res0 = len(prep0.reservations)
    tier.writeback(prep0, main)
    torch.cuda.synchronize()
    close(prep0)

    def step(overlap):
        prep = plan_preparation(tier.cache, wl.requests, n, B)
        assert np.array_equal(prep.stage_dst, prep0.stage_dst) and \
            len(prep.reservations) == n_res0
        a, b, c = E(), E(), E()
        a.record(main)
        tier.stage(prep, main, wait=not overlap)
        s.append(plan, k, v, stream=main)
        if overlap:
            s.attn(plan, q, out, lse, stream=main, part=TSR_ATTN_BEFORE_COMPOSE)
            tier.wait_staged(prep, main)
            s.compose(plan, stream=main)
            s.attn(plan, q, out, lse, stream=main, part=TSR_ATTN_AFTER_COMPOSE)
        else:
            s.compose(plan, stream=main)
            s.attn(plan, q, out, lse, stream=main)
        b.record(main)
        s.retain(plan, k, v, stream=main)
        tier.writeback(prep, main)
        c.record(main)
        torch.cuda.synchronize()
        close(prep)
        return a.elapsed_time(b), a.elapsed_time(c)

    def stage_only():
        prep = plan_preparation(tier.cache, wl.requests, n, B)
        a, b = E(), E()
        a.record(main)
        tier.stage(prep, main)
        b.record(main)
        torch.cuda.synchronize()
        for uid, epoch, _, _ in prep.reservations:      # nothing was retained
            tier.cache.cancel(uid, epoch)
            tier.cache.reclaim(epoch)
        prep.reservations = []
        tier.finish(prep)
        return a.elapsed_time(b)

    for _ in range(warmup):
        step(False), step(True), stage_only()
    t_in, t_ov, t_st = [], [], []
    for _ in range(reps):                  # alternate, so neither runs colder
        t_in.append(step(False))
        t_ov.append(step(True))
        t_st.append(stage_only())
    res = {}
    for key, t in (("in_order", np.array(t_in)), ("overlapped", np.array(t_ov))):
        res[key] = {"through_attention_us": float(t[:, 0].mean() * 1e3),
                    "with_writeback_us": float(t[:, 1].mean() * 1e3)}
    src, dst = prep0.stage_src, prep0.stage_dst
    runs = 1 + int(((np.diff(src) != 1) | (np.diff(dst) != 1)).sum()) if len(src) else 0
    res["stage_only_us"] = float(np.mean(t_st) * 1e3)
    res["copies_per_arena"] = runs
    row_bytes = 2 * m.n_kv_heads * m.head_dim * kv_elem_bytes(m.kv_dtype)
    res["staged_bytes"] = int(len(prep0.stage_src)) * B * row_bytes
    res["stage_link_gbps"] = res["staged_bytes"] / (res["stage_only_us"] * 1e-6) / 1e9
    res["written_back_bytes"] = ret_pages * B * row_bytes
    res["items_before_compose"] = plan.num_attn_items_part(TSR_ATTN_BEFORE_COMPOSE)
    res["items_after_compose"] = plan.num_attn_items_part(TSR_ATTN_AFTER_COMPOSE)
    log(f"[bench] host tier staged: {res}")
    del tier
    return res


def alias_v_leg(torch, sess, wl, qs, ks, vs, out, lse, L, steps, warmup):
    """The same step with V aliasing (attention reads V of whole gathered
    pages from the pool; compose writes only their K), timed like the main
    step: compose, append, attention on one stream, layers rotating."""
    plan = sess.plan(wl.requests, alias_v=True)
    main_s = torch.cuda.current_stream()
    E = lambda: torch.cuda.Event(enable_timing=True)
    ev = [[E() for _ in range(4)] for _ in range(steps)]

    def step(i, rec=None):
        l = i % L
        if rec:
            rec[0].record(main_s)
        sess.compose(plan, layer=l, stream=main_s)
        if rec:
            rec[1].record(main_s)
        sess.append(plan, ks[l], vs[l], layer=l, stream=main_s)
        if rec:
            rec[2].record(main_s)
        sess.attn(plan, qs[l], out, lse, layer=l, stream=main_s)
        if rec:
            rec[3].record(main_s)

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    for i in range(steps):
        step(i, ev[i])
    torch.cuda.synchronize()
    t = np.array([[e[0].elapsed_time(e[1]), e[2].elapsed_time(e[3]), e[0].elapsed_time(e[3])]
                  for e in ev])
    res = {"aliased_pages": plan.num_aliased_pages,
           "compose_us": float(t[:, 0].mean() * 1e3), "attention_us": float(t[:, 1].mean() * 1e3),
           "compose_append_attention_us": float(t[:, 2].mean() * 1e3)}
    log(f"[bench] alias_v: {res}")
    return res


def control_plane_replay():
    """Replay of a RAG-shaped retrieval trace through the control plane
    (libtsr's tsr_replay, host code): 6,000 requests of 10 units of 512
    tokens drawn Zipf(1.1) from 2,000 units whose popular set shifts every
    1,500 requests; 4 nodes with 200 units of local cache each; 16 requests
    in flight.  Block hit rates per policy."""
    import paper_2609_32999_amd._binding as B
    from workloads.traces import zipf_trace
    trace = zipf_trace(7, 6000, 2000, 10, zipf_s=1.1, token_range=(512, 512),
                       drift_every=1500, drift_shift=250)
    out = {}
    for name, kw in (("cache_aware", {}), ("load_only", {"cache_aware": 0}),
                     ("cache_aware_shared", {"shared_capacity_blocks": 600 * 32}),
                     ("first_retrieval_admitted", {"theta": 0.0})):
        base = dict(n_nodes=4, local_capacity_blocks=200 * 32, shared_capacity_blocks=0,
                    page_size=16, theta=2.0, w_recent=1.0, w_lifetime=0.05, local_window=0,
                    shared_window=0, concurrency=16, cache_aware=1)
        base.update(kw)
        t0 = time.perf_counter()
        st = B.tsr_replay(B.tsr_replay_config(**base), trace)
        out[name] = {"local_hit": st["local_hit_blocks"] / st["blocks"],
                     "shared_hit": st["shared_hit_blocks"] / st["blocks"],
                     "miss": st["miss_blocks"] / st["blocks"],
                     "local_admitted": st["local_admitted"],
                     "node_requests": [st["min_node_requests"], st["max_node_requests"]],
                     "replay_ms": (time.perf_counter() - t0) * 1e3}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="rag8b")
    ap.add_argument("--layers", type=int, default=8)
    ap.add_argument("--cpu-requests", type=int, default=6)
    ap.add_argument("--scope", choices=["global", "local"], default="global",
                    help="miss scope: global (every missing-unit token attends to the "
                         "whole prompt) or local (missing units attend within themselves "
                         "past their recompute window)")
    ap.add_argument("--no-peaks", dest="peaks", action="store_false",
                    help="skip measuring the achievable copy and bf16 GEMM rates")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-alias-v", dest="alias_v", action="store_false",
                    help="skip timing the step with V aliasing")
    ap.add_argument("--no-host-tier", dest="host_tier", action="store_false",
                    help="skip timing compose and retain against a pool in pinned host memory")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="run one launch of libtsr's plain copy kernel of this size "
                         "first (to scale HBM byte counters against a kernel of known "
                         "traffic)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the path "
              "shards by request or KV head with no exchange, see DESIGN.md", file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads
    from paper_2609_32999_amd import staging
    from paper_2609_32999_amd.session import Session

    measured = measured_peaks(torch) if args.peaks else None

    if args.calib_copy_mib:
        # one launch of libtsr's plain 16-byte copy kernel of known size, for
        # scaling HBM byte counters (FETCH_SIZE, WRITE_SIZE) per byte moved
        from paper_2609_32999_amd import tsr_peak_copy
        n = args.calib_copy_mib << 20
        a = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        tsr_peak_copy(b, a, n)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {args.calib_copy_mib} MiB done")
        del a, b

    wl = workloads.make_workload(workloads.get_config(args.workload).with_(miss_scope=args.scope))
    m = wl.model
    L = args.layers
    log(f"[bench] workload={wl.name} layers={L} prompt_tokens={wl.prompt_tokens}")
    sess = Session(m, wl.n_pool_pages, wl.n_req_pages, n_layers=L)
    staging.upload_pool(sess, wl, layer=0)
    for l in range(1, L):
        sess.pool_k[l].copy_(sess.pool_k[0])
        sess.pool_v[l].copy_(sess.pool_v[0])
    plan = sess.plan(wl.requests)
    q, k, v = staging.fresh_inputs(sess, wl, plan)
    qs = [q] + [q.clone() for _ in range(L - 1)]
    ks = [k] + [k.clone() for _ in range(L - 1)]
    vs = [v] + [v.clone() for _ in range(L - 1)]
    out, lse = sess.new_outputs(plan, with_lse=True)
    pos, _ = plan.compute_positions()
    T = plan.num_compute_tokens
    torch.cuda.synchronize()
    log(f"[bench] plan T={T} gather={plan.num_gather_tokens} retain={plan.num_retain_tokens} "
        f"items={plan.num_attn_items}")

    main_s = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    E = lambda: torch.cuda.Event(enable_timing=True)
    n_ev = args.steps
    evs = [[E() for _ in range(4)] for _ in range(n_ev)]
    evr = [[E(), E()] for _ in range(n_ev)]

    def step(i, rec=None, recr=None):
        # main: compose -> append -> attention.  side: retain, started once
        # append has been issued so that it overlaps the MFMA-bound attention
        # rather than competing with compose for HBM bandwidth.
        l = i % L
        if rec:
            rec[0].record(main_s)
        sess.compose(plan, layer=l, stream=main_s)
        if rec:
            rec[1].record(main_s)
        sess.append(plan, ks[l], vs[l], layer=l, stream=main_s)
        if rec:
            rec[2].record(main_s)
        side.wait_stream(main_s)
        sess.attn(plan, qs[l], out, lse, layer=l, stream=main_s)
        if rec:
            rec[3].record(main_s)
        with torch.cuda.stream(side):
            if recr:
                recr[0].record(side)
            sess.retain(plan, ks[l], vs[l], layer=l, stream=side)
            if recr:
                recr[1].record(side)
        main_s.wait_stream(side)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    log(f"[bench] warmup done ({args.warmup} steps)")
    t_start, t_end = E(), E()
    w0 = time.perf_counter()
    t_start.record(main_s)
    for i in range(args.steps):
        step(i, evs[i], evr[i])
    t_end.record(main_s)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    total_ms = t_start.elapsed_time(t_end)
    ms = total_ms / args.steps
    compose_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    append_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    attn_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
    retain_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evr]))
    log(f"[bench] timed {args.steps} steps: {ms:.3f} ms/step (wall {wall * 1e3 / args.steps:.3f}); "
        f"compose {compose_ms * 1e3:.1f} us, append {append_ms * 1e3:.1f} us, "
        f"attn {attn_ms * 1e3:.1f} us, retain {retain_ms * 1e3:.1f} us")

    # Outside the step: one compose launch over all layer buffer sets (a
    # unit's cached state is placed for every layer at once), the kernel's
    # steady-state bandwidth without the launch ramp of a single layer.
    sess.compose(plan, layer="all", stream=main_s)
    reps = 5
    ev_a, ev_b = E(), E()
    ev_a.record(main_s)
    for _ in range(reps):
        sess.compose(plan, layer="all", stream=main_s)
    ev_b.record(main_s)
    torch.cuda.synchronize()
    compose_all_ms = ev_a.elapsed_time(ev_b) / reps

    alias = alias_v_leg(torch, sess, wl, qs, ks, vs, out, lse, L, args.steps, args.warmup) \
        if m.kv_dtype == "bf16" and args.alias_v else None

    w = kv_elem_bytes(m.kv_dtype)
    row_bytes = 2 * m.n_kv_heads * m.head_dim * w           # K + V of one token
    host = host_tier(torch, wl, plan, ks[0], vs[0], row_bytes) if args.host_tier else None
    if host:
        host["staged"] = host_tier_staged(torch, wl)
    gather_bytes = 2 * plan.num_gather_tokens * row_bytes   # read + write
    append_bytes = 2 * T * row_bytes
    retain_bytes = 2 * plan.num_retain_tokens * row_bytes
    kv_lo = plan.row_kv_lo()
    visible = int((pos.astype(np.int64) - kv_lo + 1).sum())
    attn_flops = 4.0 * m.head_dim * m.n_q_heads * visible
    attn_tflops = attn_flops / (attn_ms * 1e-3) / 1e12
    compose_gbs = gather_bytes / (compose_ms * 1e-3) / 1e9
    peak = PEAK_E4M3_BLEND if m.kv_dtype == "e4m3" else PEAK_MFMA_TFLOPS[m.act_dtype]
    G = m.n_q_heads // m.n_kv_heads
    attn_kernel = (f"attn_fp8_kernel<{G}>" if m.kv_dtype == "e4m3"
                   else f"attn_mfma_kernel<{G}, false, {plan.attn_rows_per_item // 32}>")
    # the e4m3 page kernel is instantiated for 2, 4 or 8 units per thread
    units = m.page_size * m.n_kv_heads * 8
    u = 2 if units <= 512 else 4 if units <= 1024 else 8
    compose_kernel = (f"page_fp8_kernel<0, {u}>" if m.kv_dtype == "e4m3" else
                      f"kv_move_kernel<{m.head_dim}, unsigned short, 0>")
    value = wl.prompt_tokens / (ms * 1e-3)

    rec = {
        "metric": "composed-prefill tokens/s per layer",
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": ("e4m3 KV / bf16 act" if m.kv_dtype == "e4m3" else m.act_dtype),
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: {wl.cfg.description}",
            "requests": len(wl.requests), "prompt_tokens": wl.prompt_tokens,
            "computed_tokens": T, "gathered_tokens": plan.num_gather_tokens,
            "retained_tokens": plan.num_retain_tokens, "layer_buffer_sets": L,
            "miss_scope": args.scope,
            "seed": wl.seed,
        },
        "computed_tokens_per_s": T / (ms * 1e-3),
        "assembly_hbm_gbps": compose_gbs,
        "attention_tflops": attn_tflops,
        "kernel_us": {"compose": compose_ms * 1e3, "append": append_ms * 1e3,
                      "attention": attn_ms * 1e3, "retain_side_stream": retain_ms * 1e3},
        "roofline": {"bound": "mfma", "achieved": attn_tflops, "peak": peak,
                     "unit": "TFLOP/s", "frac": attn_tflops / peak,
                     # the committed profiles are of the GLOBAL scope
                     "traffic": (profiled_traffic(args.workload, attn_kernel)
                                 if args.scope == "global" else None),
                     "kernel": attn_kernel, "flops_per_launch": attn_flops},
        "roofline_compose": {"bound": "hbm", "achieved": compose_gbs, "peak": PEAK_HBM_GBS,
                             "unit": "GB/s", "frac": compose_gbs / PEAK_HBM_GBS,
                             "bytes_per_launch": gather_bytes,
                             "traffic": profiled_traffic(args.workload, compose_kernel),
                             "kernel": compose_kernel},
        "compose_all_layers": {"layers": L, "us": compose_all_ms * 1e3,
                               "gbps": L * gather_bytes / (compose_all_ms * 1e-3) / 1e9,
                               "frac": L * gather_bytes / (compose_all_ms * 1e-3) / 1e9 / PEAK_HBM_GBS},
        "append_gbps": append_bytes / (append_ms * 1e-3) / 1e9,
        "retain_gbps": retain_bytes / (retain_ms * 1e-3) / 1e9 if retain_ms > 0 else None,
    }
    if alias:
        rec["alias_v"] = alias
    if host:
        rec["host_tier"] = host
    rec["control_plane"] = control_plane_replay()
    if measured:
        rec["measured_peaks"] = measured
        mfma_peak = measured["mfma_loop_tflops"]
        if m.kv_dtype == "e4m3":
            mfma_peak *= peak / PEAK_MFMA_TFLOPS["bf16"]   # the blend, at the measured clock
        rec["roofline"]["frac_of_measured"] = attn_tflops / mfma_peak
        rec["roofline_compose"]["frac_of_measured"] = compose_gbs / max(
            measured["copy_kernel_gbps"], measured["copy_gbps"])
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle baseline")
        rec["cpu_baseline"] = cpu_baseline(wl, min(args.cpu_requests, len(wl.requests)))
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()

"""Benchmark of the composed-prefill hot path on one MI355X.

A step is one attention layer of one batch: assembly (compose -- gather +
RoPE re-rotation of cached units -- and append of the computed rows, one
launch) -> causal GQA prefill attention of the computed rows -> retention
of the computed units, in stream order.  Steps
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
PEAK_MFMA_TFLOPS = {"bf16": 2500.0, "f32": 157.3, "fp8": 5000.0}
# e4m3 KV: QK^T runs in fp8 MFMA (5.0 PFLOP/s dense) and PV in fp16 MFMA
# (2.5 PFLOP/s), half of the FLOPs each.  The fraction is reported against
# the fp8 dense peak; the blend 1 / (0.5/5.0 + 0.5/2.5) of the two products'
# peaks is a second, labelled field.
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


def aliasing_leg(torch, sess, wl, qs, ks, vs, out, lse, L, steps, warmup):
    """Zero-copy composition against the composed (materialized) path, each
    timed like the main step without retention: V aliasing (attention reads
    V of whole gathered pages from the pool), K rotated on load (attention
    reads their pre-RoPE K from the pool and rotates it while staging the
    tile), and both (compose leaves those pages alone), under the batch's
    own miss scope and under the LOCAL scope."""
    import workloads
    res = {}
    for scope in ("global", "local"):
        reqs = (wl.requests if wl.cfg.miss_scope == scope else
                workloads.make_workload(wl.cfg.with_(miss_scope=scope)).requests)
        for mode, kw in (("materialized", {}), ("v", dict(alias_v=True)),
                         ("k", dict(alias_k=True)), ("kv", dict(alias_v=True, alias_k=True))):
            plan = sess.plan(reqs, **kw)
            st, asm, att, _, _ = time_path(torch, sess, plan, qs, ks, vs, out, lse, L, steps,
                                           warmup)
            res[f"{scope}_{mode}"] = {
                "aliased_pages_v": plan.num_aliased_pages,
                "aliased_pages_k": plan.num_aliased_k_pages,
                "gathered_tokens_moved": plan.num_gather_tokens,
                "assembly_us": dist(asm), "attention_us": dist(att), "step_us": dist(st)}
    log("[bench] aliasing: " + ", ".join(
        f"{k}: asm {v['assembly_us']['median']:.1f} attn {v['attention_us']['median']:.1f}"
        for k, v in res.items()))
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


def dist(ms_list):
    """Event durations (ms) -> mean, median, p10, p90 in microseconds."""
    a = np.asarray(ms_list, dtype=np.float64) * 1e3
    if a.size == 0:
        return {"mean": 0.0, "median": 0.0, "p10": 0.0, "p90": 0.0}
    return {"mean": float(a.mean()), "median": float(np.median(a)),
            "p10": float(np.percentile(a, 10)), "p90": float(np.percentile(a, 90))}


def attention_flops(plan, m):
    """4 d H_q per visible (row, key) pair: the method's attention work,
    masked-out tile work excluded."""
    pos, _ = plan.compute_positions()
    kv_lo = plan.row_kv_lo()
    visible = int((pos.astype(np.int64) - kv_lo + 1).sum())
    return 4.0 * m.head_dim * m.n_q_heads * visible


def attention_kernel_name(plan, m):
    G = m.n_q_heads // m.n_kv_heads
    if m.kv_dtype == "e4m3":
        return f"attn_fp8_kernel<{G}, {plan.attn_rows_per_item // 32}>"
    if plan.attn_rows_per_item == 64:       # the pipelined kernel
        return f"attn_pipe_kernel<{G}, {str(plan.alias_v).lower()}>"
    return (f"attn_mfma_kernel<{G}, {str(plan.alias_v).lower()}, "
            f"{str(plan.alias_k).lower()}, {plan.attn_rows_per_item // 32}>")


def assembly_kernel_name(m):
    # the e4m3 page kernel is instantiated for 2, 4 or 8 units per thread
    units = m.page_size * m.n_kv_heads * 8
    u = 2 if units <= 512 else 4 if units <= 1024 else 8
    return (f"page_fp8_assemble_kernel<{u}>" if m.kv_dtype == "e4m3" else
            f"kv_assemble_kernel<{m.head_dim}, unsigned short>")


def attention_peaks(m):
    """(peak used for the fraction, blended peak or None)."""
    if m.kv_dtype == "e4m3":
        return PEAK_MFMA_TFLOPS["fp8"], PEAK_E4M3_BLEND
    return PEAK_MFMA_TFLOPS[m.act_dtype], None


def time_path(torch, sess, plan, qs, ks, vs, out, lse, L, steps, warmup):
    """The step, on one stream: one assembly launch (compose + append),
    attention, then retention of the computed units, layers rotating over L
    buffer sets.  (Retention on a second stream beside attention gave the
    same step time: its workgroups wait for compute units the attention
    workgroups hold, and it slowed attention by as much as it saved.)
    Returns per-step durations (ms) of the step, the assembly, attention and
    retention, and the wall time."""
    main_s = torch.cuda.current_stream()
    E = lambda: torch.cuda.Event(enable_timing=True)
    evs = [[E() for _ in range(4)] for _ in range(steps)]

    def step(i, rec=None):
        l = i % L
        if rec:
            rec[0].record(main_s)
        sess.assemble(plan, ks[l], vs[l], layer=l, stream=main_s)
        if rec:
            rec[1].record(main_s)
        sess.attn(plan, qs[l], out, lse, layer=l, stream=main_s)
        if rec:
            rec[2].record(main_s)
        sess.retain(plan, ks[l], vs[l], layer=l, stream=main_s)
        if rec:
            rec[3].record(main_s)

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    end = E()
    w0 = time.perf_counter()
    for i in range(steps):
        step(i, evs[i])
    end.record(main_s)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    # a step lasts from its first event to the next step's; the last one to
    # the event after the loop
    starts = [e[0] for e in evs] + [end]
    step_ms = [starts[i].elapsed_time(starts[i + 1]) for i in range(steps)]
    asm = [e[0].elapsed_time(e[1]) for e in evs]
    att = [e[1].elapsed_time(e[2]) for e in evs]
    ret = [e[2].elapsed_time(e[3]) for e in evs]
    return step_ms, asm, att, ret, wall


def split_leg(torch, sess, plan, ks, vs, L, steps):
    """compose then append as two launches, the unfused form of the
    assembly (same bytes), for reference."""
    main_s = torch.cuda.current_stream()
    E = lambda: torch.cuda.Event(enable_timing=True)
    ev = [[E() for _ in range(3)] for _ in range(steps)]
    for i in range(4):
        sess.compose(plan, layer=i % L, stream=main_s)
        sess.append(plan, ks[i % L], vs[i % L], layer=i % L, stream=main_s)
    for i in range(steps):
        l = i % L
        ev[i][0].record(main_s)
        sess.compose(plan, layer=l, stream=main_s)
        ev[i][1].record(main_s)
        sess.append(plan, ks[l], vs[l], layer=l, stream=main_s)
        ev[i][2].record(main_s)
    torch.cuda.synchronize()
    return {"compose_us": dist([e[0].elapsed_time(e[1]) for e in ev]),
            "append_us": dist([e[1].elapsed_time(e[2]) for e in ev])}


def local_leg(torch, sess, wl, qs, ks, vs, out, lse, L, steps, warmup):
    """The same batch, pool and inputs under the LOCAL miss scope (missing
    units' tokens past their recompute window attend within their unit):
    a second plan, timed like the main step without retention."""
    import workloads
    wl_l = workloads.make_workload(wl.cfg.with_(miss_scope="local"))
    plan = sess.plan(wl_l.requests)
    m = wl.model
    st, asm, att, _, _ = time_path(torch, sess, plan, qs, ks, vs, out, lse, L, steps, warmup)
    flops = attention_flops(plan, m)
    d_att = dist(att)
    tf = flops / (d_att["mean"] * 1e-6) / 1e12
    peak, blend = attention_peaks(m)
    res = {"ms_per_step": float(np.mean(st)),
           "value": wl.prompt_tokens / (np.mean(st) * 1e-3),
           "kernel_us": {"assembly": dist(asm), "attention": d_att},
           "roofline": {"bound": "mfma", "achieved": tf, "peak": peak, "unit": "TFLOP/s",
                        "frac": tf / peak, "kernel": attention_kernel_name(plan, m),
                        "flops_per_launch": flops,
                        # profiles/local_kernels.md is this leg's counter profile
                        "traffic": (profiled_traffic("local", attention_kernel_name(plan, m))
                                    if wl.name == "rag8b" else None)}}
    log(f"[bench] local scope: {res}")
    return res


def workload_leg(torch, name, steps, warmup, L=2):
    """Another workload's assembly + attention step (no retention), with its
    realized counts next to the sizes the configuration names."""
    import workloads
    from paper_2609_32999_amd import staging
    from paper_2609_32999_amd.session import Session
    wl = workloads.generate(name)
    m = wl.model
    sess = Session(m, wl.n_pool_pages, wl.n_req_pages, n_layers=L)
    staging.upload_pool(sess, wl, layer=0)
    for l in range(1, L):
        sess.pool_k[l].copy_(sess.pool_k[0])
        sess.pool_v[l].copy_(sess.pool_v[0])
        if sess.e4m3:
            sess.pool_scale[l].copy_(sess.pool_scale[0])
    plan = sess.plan(wl.requests)
    q, k, v = staging.fresh_inputs(sess, wl, plan)
    qs = [q] + [q.clone() for _ in range(L - 1)]
    ks = [k] + [k.clone() for _ in range(L - 1)]
    vs = [v] + [v.clone() for _ in range(L - 1)]
    out, lse = sess.new_outputs(plan, with_lse=True)
    st, asm, att, _, _ = time_path(torch, sess, plan, qs, ks, vs, out, lse, L, steps, warmup)
    row_bytes = 2 * m.n_kv_heads * m.head_dim * kv_elem_bytes(m.kv_dtype)
    T = plan.num_compute_tokens
    asm_bytes = 2 * (plan.num_gather_tokens + T) * row_bytes
    flops = attention_flops(plan, m)
    d_asm, d_att = dist(asm), dist(att)
    tf = flops / (d_att["mean"] * 1e-6) / 1e12
    gbs = asm_bytes / (d_asm["mean"] * 1e-6) / 1e9
    peak, blend = attention_peaks(m)
    res = {"workload": f"{wl.name}: {wl.cfg.description}",
           "ms_per_step": float(np.mean(st)),
           "value": wl.prompt_tokens / (np.mean(st) * 1e-3),
           "realized": {"requests": len(wl.requests), "prompt_tokens": wl.prompt_tokens,
                        "computed_tokens": T, "gathered_tokens": plan.num_gather_tokens,
                        "visible_pairs": int(flops / (4 * m.head_dim * m.n_q_heads)),
                        "attention_flops": flops,
                        "assembly_bytes": asm_bytes},
           "kernel_us": {"assembly": d_asm, "attention": d_att},
           "roofline": {"bound": "mfma", "achieved": tf, "peak": peak, "unit": "TFLOP/s",
                        "frac": tf / peak, "kernel": attention_kernel_name(plan, m),
                        "flops_per_launch": flops,
                        "traffic": profiled_traffic(name, attention_kernel_name(plan, m))},
           "roofline_assembly": {"bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS,
                                 "unit": "GB/s", "frac": gbs / PEAK_HBM_GBS,
                                 "kernel": assembly_kernel_name(m)}}
    if blend:
        res["roofline"]["frac_of_blend"] = tf / blend
        res["roofline"]["blend_peak"] = blend
    log(f"[bench] leg {name}: {res}")
    del sess
    torch.cuda.empty_cache()
    return res


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
    ap.add_argument("--legs", default="local,fp8rag,agent8b,long70b",
                    help="comma-separated extra legs reported in the same line: local "
                         "(the batch under the LOCAL miss scope), fp8rag, agent8b, long70b "
                         "(those workloads' assembly + attention + retain); '' for none")
    ap.add_argument("--no-peaks", dest="peaks", action="store_false",
                    help="skip measuring the achievable copy and bf16 GEMM rates")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-alias-v", dest="alias_v", action="store_false",
                    help="skip timing the step with zero-copy composition (V aliasing, K "
                         "rotated on load, both)")
    ap.add_argument("--no-host-tier", dest="host_tier", action="store_false",
                    help="skip timing compose and retain against a pool in pinned host memory")
    ap.add_argument("--attn-kernel", type=int, default=0, choices=[0, 1, 2, 3, 4],
                    help="bf16 attention kernel of the main plan: 0 automatic, 1 the "
                         "pipelined kernel, 2 the row-block kernel under its rule, "
                         "3 / 4 the row-block kernel with three / one row blocks")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="run one launch of libtsr's plain copy kernel of this size "
                         "first (to scale HBM byte counters against a kernel of known "
                         "traffic)")
    args = ap.parse_args()
    args.legs = [x for x in args.legs.split(",") if x]
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the path "
              "shards by request or by KV head with no exchange between GPUs, so one GPU's "
              "share is the same kernels on its requests or heads", file=sys.stderr)
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
    plan = sess.plan(wl.requests, attn_kernel=args.attn_kernel)
    q, k, v = staging.fresh_inputs(sess, wl, plan)
    qs = [q] + [q.clone() for _ in range(L - 1)]
    ks = [k] + [k.clone() for _ in range(L - 1)]
    vs = [v] + [v.clone() for _ in range(L - 1)]
    out, lse = sess.new_outputs(plan, with_lse=True)
    pos, _ = plan.compute_positions()
    T = plan.num_compute_tokens
    torch.cuda.synchronize()
    log(f"[bench] plan T={T} gather={plan.num_gather_tokens} retain={plan.num_retain_tokens} "
        f"items={plan.num_attn_items} rows/item={plan.attn_rows_per_item}")

    main_s = torch.cuda.current_stream()
    step_ms, asm_ms, attn_ms, retain_ms, wall = time_path(
        torch, sess, plan, qs, ks, vs, out, lse, L, args.steps, args.warmup)
    ms = float(np.mean(step_ms))
    d_asm, d_attn, d_ret = dist(asm_ms), dist(attn_ms), dist(retain_ms)
    log(f"[bench] timed {args.steps} steps: {ms:.3f} ms/step (wall {wall * 1e3 / args.steps:.3f}); "
        f"assembly {d_asm}, attn {d_attn}, retain {d_ret} (us)")

    # compose and append as two launches (the unfused path), for reference
    split = split_leg(torch, sess, plan, ks, vs, L, args.steps)

    # Outside the step: one compose launch over all layer buffer sets (a
    # unit's cached state is placed for every layer at once), the kernel's
    # steady-state bandwidth without the launch ramp of a single layer.
    sess.compose(plan, layer="all", stream=main_s)
    reps = 5
    E = lambda: torch.cuda.Event(enable_timing=True)
    ev_a, ev_b = E(), E()
    ev_a.record(main_s)
    for _ in range(reps):
        sess.compose(plan, layer="all", stream=main_s)
    ev_b.record(main_s)
    torch.cuda.synchronize()
    compose_all_ms = ev_a.elapsed_time(ev_b) / reps

    alias = aliasing_leg(torch, sess, wl, qs, ks, vs, out, lse, L, args.steps, args.warmup) \
        if m.kv_dtype == "bf16" and args.alias_v else None

    w = kv_elem_bytes(m.kv_dtype)
    row_bytes = 2 * m.n_kv_heads * m.head_dim * w           # K + V of one token
    host = host_tier(torch, wl, plan, ks[0], vs[0], row_bytes) if args.host_tier else None
    if host:
        host["staged"] = host_tier_staged(torch, wl)
    gather_bytes = 2 * plan.num_gather_tokens * row_bytes   # read + write
    append_bytes = 2 * T * row_bytes
    asm_bytes = gather_bytes + append_bytes
    retain_bytes = 2 * plan.num_retain_tokens * row_bytes
    attn_flops = attention_flops(plan, m)
    attn_tflops = attn_flops / (d_attn["mean"] * 1e-6) / 1e12
    asm_gbs = asm_bytes / (d_asm["mean"] * 1e-6) / 1e9
    G = m.n_q_heads // m.n_kv_heads
    attn_kernel = attention_kernel_name(plan, m)
    asm_kernel = assembly_kernel_name(m)
    value = wl.prompt_tokens / (ms * 1e-3)
    peak, blend = attention_peaks(m)

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
        "assembly_hbm_gbps": asm_gbs,
        "attention_tflops": attn_tflops,
        "kernel_us": {"assembly": d_asm, "attention": d_attn, "retain": d_ret,
                      "step": dist(step_ms)},
        "roofline": {"bound": "mfma", "achieved": attn_tflops, "peak": peak,
                     "unit": "TFLOP/s", "frac": attn_tflops / peak,
                     # the committed profiles are of the GLOBAL scope
                     "traffic": (profiled_traffic(args.workload, attn_kernel)
                                 if args.scope == "global" else None),
                     "kernel": attn_kernel, "flops_per_launch": attn_flops,
                     "achieved_from": "mean event duration"},
        "roofline_assembly": {"bound": "hbm", "achieved": asm_gbs, "peak": PEAK_HBM_GBS,
                              "unit": "GB/s", "frac": asm_gbs / PEAK_HBM_GBS,
                              "bytes_per_launch": asm_bytes,
                              "gather_bytes": gather_bytes, "append_bytes": append_bytes,
                              "traffic": profiled_traffic(args.workload, asm_kernel),
                              "kernel": asm_kernel,
                              "frac_at_median": asm_bytes / (d_asm["median"] * 1e-6) / 1e9
                              / PEAK_HBM_GBS},
        "compose_append_split": split,
        "compose_all_layers": {"layers": L, "us": compose_all_ms * 1e3,
                               "gbps": L * gather_bytes / (compose_all_ms * 1e-3) / 1e9,
                               "frac": L * gather_bytes / (compose_all_ms * 1e-3) / 1e9 / PEAK_HBM_GBS},
        "retain_gbps": retain_bytes / (d_ret["mean"] * 1e-6) / 1e9 if d_ret["mean"] > 0 else None,
    }
    if blend:
        rec["roofline"]["frac_of_blend"] = attn_tflops / blend
        rec["roofline"]["blend_peak"] = blend
    if alias:
        rec["zero_copy"] = alias
    if host:
        rec["host_tier"] = host
    rec["control_plane"] = control_plane_replay()
    if args.legs:
        rec["legs"] = {}
        if "local" in args.legs and args.scope == "global" and m.kv_dtype != "f32":
            rec["legs"]["local"] = local_leg(torch, sess, wl, qs, ks, vs, out, lse, L,
                                             args.steps, args.warmup)
        for name in ("fp8rag", "agent8b", "long70b"):
            if name in args.legs and name != args.workload:
                rec["legs"][name] = workload_leg(torch, name, args.steps, args.warmup)
    if measured:
        rec["measured_peaks"] = measured
        mfma_peak = measured["mfma_loop_tflops"]
        if m.kv_dtype == "e4m3":
            mfma_peak *= peak / PEAK_MFMA_TFLOPS["bf16"]   # fp8 peak, at the measured clock
        rec["roofline"]["frac_of_measured"] = attn_tflops / mfma_peak
        rec["roofline_assembly"]["frac_of_measured"] = asm_gbs / max(
            measured["copy_kernel_gbps"], measured["copy_gbps"])
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle baseline")
        rec["cpu_baseline"] = cpu_baseline(wl, min(args.cpu_requests, len(wl.requests)))
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()

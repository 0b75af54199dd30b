"""C-ABI checks that need no GPU: exports, validation, host-only plans."""
import os
import re
from types import SimpleNamespace as NS

import numpy as np
import pytest

import paper_2609_32999_amd as P
import workloads
from oracle import layout as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# rows of a bf16 attention item with several 32-row blocks
MULTI_ROWS = 96


def _model(wl, **kw):
    m = wl.model
    args = dict(n_q_heads=m.n_q_heads, n_kv_heads=m.n_kv_heads, head_dim=m.head_dim,
                page_size=m.page_size, kv_dtype=m.kv_dtype, act_dtype=m.act_dtype,
                rope_theta=m.rope_theta, max_position=m.max_position)
    args.update(kw)
    return P.make_model(**args)


def _plan(wl, reqs=None, **kw):
    reqs = wl.requests if reqs is None else reqs
    return P.tsr_plan_create(_model(wl, **kw), P.RequestBatch(reqs), wl.n_pool_pages,
                             wl.n_req_pages)


def test_library_exports_every_declared_symbol():
    header = ""
    for name in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if name.endswith(".h"):
            with open(os.path.join(ROOT, "include", name)) as f:
                header += f.read()
    declared = set(re.findall(r"^\s*(?:[\w\*]+\s+)+\**(tsr_\w+)\s*\(", header, re.M))
    assert declared == set(P.EXPORTS), declared ^ set(P.EXPORTS)
    lib = P.lib()
    for name in declared:
        assert getattr(lib, name) is not None


def test_abi_version():
    assert P.tsr_abi_version() == 7


@pytest.mark.parametrize("name", ["tiny", "small_bf16", "small_f32", "small_bf16_g8",
                                  "rag8b", "long70b"])
def test_host_plan_matches_oracle_sets(name):
    wl = workloads.generate(name)
    plan = _plan(wl)
    pos, req = plan.compute_positions()
    opos = np.concatenate([L.compute_positions(r) for r in wl.requests])
    oreq = np.concatenate([np.full(len(L.compute_positions(r)), i)
                           for i, r in enumerate(wl.requests)])
    assert np.array_equal(pos, opos) and np.array_equal(req, oreq)
    assert plan.num_gather_tokens == sum(len(L.gather_tokens(r)) for r in wl.requests)
    assert plan.num_retain_tokens == sum(len(L.retain_tokens(r, wl.model.page_size))
                                         for r in wl.requests)
    assert plan.num_attn_items % 8 == 0


def _items_per_kv_head(wl, rows_per_item, grouped=False):
    """Attention items of each KV head (before launch padding) when runs of
    rows with the same first visible key are cut into items of
    rows_per_item rows, and the share of (32-row block x 32-key tile) slots
    of those items that hold keys the block's rows need.  grouped: each
    request's rows first stably sorted by first visible key."""
    n = need = slots = 0
    for req in wl.requests:
        pos, lo = L.compute_positions(req), L.row_kv_lo(req)
        if grouped:
            o = np.argsort(lo, kind="stable")
            pos, lo = pos[o], lo[o]
        a0 = 0
        while a0 < len(pos):
            a1 = a0 + 1
            while a1 < len(pos) and lo[a1] == lo[a0]:
                a1 += 1
            for t0 in range(a0, a1, rows_per_item):
                p = pos[t0:min(a1, t0 + rows_per_item)]
                n += 1
                slots += (rows_per_item // 32) * (p[-1] // 32 + 1 - lo[t0] // 32)
                need += sum(p[b:b + 32].max() // 32 + 1 - lo[t0] // 32
                            for b in range(0, len(p), 32))
            a0 = a1
    return n, need / slots


@pytest.mark.parametrize("name,scope", [("rag8b", "global"), ("rag8b", "local"),
                                        ("agent8b", "local"), ("long70b", "global"),
                                        ("fp8rag", "global"), ("small_f32", "global")])
def test_attention_row_blocks(name, scope):
    """Rows per attention item.  bf16 and e4m3 KV: three 32-row blocks over
    rows grouped by first visible key unless fewer than 60 % of the items'
    block x tile slots would hold work or there would be fewer than 256
    items, then one; fp32: one."""
    cfg = workloads.get_config(name)
    if scope != "global":
        cfg = cfg.with_(miss_scope=scope)
    wl = workloads.make_workload(cfg)
    m = wl.model
    n1, _ = _items_per_kv_head(wl, 32)
    bf16_act = m.act_dtype == "bf16"
    n3, use3 = _items_per_kv_head(wl, 96, grouped=True)
    groups = (m.n_q_heads // m.n_kv_heads) // 4 if bf16_act and \
        m.n_q_heads // m.n_kv_heads > 4 else 1
    per = m.n_kv_heads * groups
    if bf16_act and m.kv_dtype in ("bf16", "e4m3") and use3 >= 0.6 and n3 * per >= 256:
        rows, n = 96, n3
    else:
        rows, n = 32, n1
    plan = _plan(wl)
    # launch padding only adds items: multi-block items give fewer items than
    # one-block items would need, one row block at least that many
    if rows > 32:
        assert n * per <= plan.num_attn_items < n1 * per, (plan.num_attn_items, n1, n, rows)
    else:
        assert plan.num_attn_items >= n1 * per, (plan.num_attn_items, n1, n3, use3)
    assert plan.attn_rows_per_item == rows
    expect = {("rag8b", "global"): 96, ("long70b", "global"): 96, ("fp8rag", "global"): 96,
              ("rag8b", "local"): 96, ("agent8b", "local"): 96}
    assert rows == expect.get((name, scope), 32)


@pytest.mark.parametrize("name", ["rag8b", "small_bf16"])
def test_attention_kernel_option(name):
    """attn_kernel: 1 asks for the pipelined kernel (64-row items, refused
    where it does not apply: K rotated on load), 2 for the row-block
    kernel under its rule (as 0), 3 / 4 for it with three / one row blocks,
    anything else is an invalid argument."""
    wl = workloads.generate(name)
    mk = lambda **kw: P.tsr_plan_create(_model(wl), P.RequestBatch(wl.requests),
                                        wl.n_pool_pages, wl.n_req_pages, **kw)
    assert mk(attn_kernel=1).attn_rows_per_item == 64
    assert mk(attn_kernel=2).attn_rows_per_item in (32, 96)
    assert mk().attn_rows_per_item == mk(attn_kernel=2).attn_rows_per_item
    assert mk(attn_kernel=3).attn_rows_per_item == 96
    assert mk(attn_kernel=4).attn_rows_per_item == 32
    assert mk(attn_kernel=3, alias_k=True).attn_rows_per_item == 96
    with pytest.raises(P.TsrError) as e:
        mk(attn_kernel=1, alias_k=True)
    assert e.value.status == P.TSR_ERR_UNSUPPORTED
    for bad in (-1, 5):
        with pytest.raises(P.TsrError) as e:
            mk(attn_kernel=bad)
        assert e.value.status == P.TSR_ERR_INVALID_ARG


def _tiny_req(**over):
    wl = workloads.generate("tiny")
    req = wl.requests[0]
    units = [NS(**vars(u)) for u in req.units]
    r = NS(prompt_len=req.prompt_len, units=units, text_segs=list(req.text_segs),
           block_table=req.block_table.copy())
    for k, v in over.items():
        setattr(r, k, v)
    return wl, r


def _expect(status, wl, reqs, match, **kw):
    with pytest.raises(P.TsrError) as e:
        _plan(wl, reqs, **kw)
    assert e.value.status == status
    assert re.search(match, e.value.message), e.value.message
    assert re.search(match, P.tsr_last_error())


def test_rejects_gap_and_overlap():
    wl, r = _tiny_req()
    r.units[1].position += 1
    _expect(P._binding.TSR_ERR_INVALID_ARG, wl, [r], "tile")
    wl, r = _tiny_req()
    r.units[1].n_tokens += 1
    _expect(P._binding.TSR_ERR_INVALID_ARG, wl, [r], "tile")
    wl, r = _tiny_req(prompt_len=300)
    _expect(P._binding.TSR_ERR_INVALID_ARG, wl, [r], "prompt_len")


def test_rejects_out_of_range_pages():
    wl, r = _tiny_req()
    r.units[1].pool_pages = r.units[1].pool_pages.copy()
    r.units[1].pool_pages[0] = wl.n_pool_pages
    _expect(P._binding.TSR_ERR_OUT_OF_RANGE, wl, [r], "pool page")
    wl, r = _tiny_req()
    r.block_table[3] = -1
    _expect(P._binding.TSR_ERR_OUT_OF_RANGE, wl, [r], "block_table")


def test_rejects_shared_request_pages():
    wl, r = _tiny_req()
    r2 = NS(**vars(r))
    _expect(P._binding.TSR_ERR_INVALID_ARG, wl, [r, r2], "used twice")


def test_rejects_retain_into_pages_read_by_a_hit():
    wl, r = _tiny_req()
    # unit 0 is a retained MISS; point it at the pages of the HIT unit 1
    assert r.units[0].residency == 0 and r.units[0].retain == 1
    r.units[0].pool_pages = r.units[1].pool_pages
    _expect(P._binding.TSR_ERR_INVALID_ARG, wl, [r], "both read")


def test_rejects_double_retain():
    wl, r = _tiny_req()
    r.units[2].retain = 1
    r.units[2].pool_pages = r.units[0].pool_pages
    _expect(P._binding.TSR_ERR_INVALID_ARG, wl, [r], "retained twice")


def test_rejects_unsupported_shapes():
    wl, r = _tiny_req()
    _expect(P._binding.TSR_ERR_UNSUPPORTED, wl, [r], "e4m3", kv_dtype="e4m3", act_dtype="bf16")
    _expect(P._binding.TSR_ERR_UNSUPPORTED, wl, [r], "head_dim", head_dim=96)
    _expect(P._binding.TSR_ERR_UNSUPPORTED, wl, [r], "bf16 path", kv_dtype="bf16",
            act_dtype="bf16")           # tiny has head_dim 64
    _expect(P._binding.TSR_ERR_OUT_OF_RANGE, wl, [r], "max_position", max_position=100)
    _expect(P._binding.TSR_ERR_INVALID_ARG, wl, [r], "multiple", n_q_heads=6)


def test_rope_pairing_field():
    """The model names its RoPE pairing (Section 2.2 leaves it open): the
    half-split pairing runs, the interleaved one is refused rather than run
    with the wrong pairing, and any other value is malformed."""
    wl, r = _tiny_req()
    _plan(wl, [r], rope_interleaved=0)
    _expect(P._binding.TSR_ERR_UNSUPPORTED, wl, [r], "interleaved", rope_interleaved=1)
    _expect(P._binding.TSR_ERR_INVALID_ARG, wl, [r], "rope_interleaved", rope_interleaved=2)
    _expect(P._binding.TSR_ERR_INVALID_ARG, wl, [r], "rope_interleaved", rope_interleaved=-1)
    assert P.tsr_rope_table_bytes(_model(wl, rope_interleaved=1)) == 0
    with pytest.raises(P.TsrError, match="interleaved"):     # size 0: refused
        P.tsr_plan_workspace_size(_model(wl, rope_interleaved=1), P.RequestBatch([r]),
                                  wl.n_pool_pages, wl.n_req_pages)


def test_rejects_bad_unit_fields():
    wl, r = _tiny_req()
    r.units[1].residency = 2
    _expect(P._binding.TSR_ERR_INVALID_ARG, wl, [r], "residency")
    wl, r = _tiny_req()
    r.units[1].n_recompute = -1
    _expect(P._binding.TSR_ERR_INVALID_ARG, wl, [r], "n_recompute")
    wl, r = _tiny_req()
    r.units[1].pool_pages = None
    _expect(P._binding.TSR_ERR_INVALID_ARG, wl, [r], "pool_pages")


def test_host_only_plan_cannot_execute():
    wl = workloads.generate("tiny")
    plan = _plan(wl)
    with pytest.raises(P.TsrError) as e:
        P.tsr_compose_kv(plan, 1, 1, None, 1, 1, None)
    assert e.value.status == P._binding.TSR_ERR_INVALID_ARG
    assert "host-only" in e.value.message


def test_workspace_size_and_rope_table_size():
    wl = workloads.generate("rag8b")
    m = _model(wl)
    ws = P.tsr_plan_workspace_size(m, P.RequestBatch(wl.requests), wl.n_pool_pages,
                                   wl.n_req_pages)
    assert ws > 0 and ws % 256 == 0
    assert P.tsr_rope_table_bytes(m) == 2 * 4 * m.max_position * (m.head_dim // 2)


def test_edge_requests_plan():
    # a prompt made only of reused units with no window: nothing to compute
    wl, r = _tiny_req()
    for u in r.units:
        u.residency, u.n_recompute, u.retain = 1, 0, 0
    r.units[-1].n_tokens += 16
    r.units[-1].pool_pages = np.append(r.units[-1].pool_pages, 0).astype(np.int32)
    r.text_segs = []
    plan = _plan(wl, [r])
    assert plan.num_compute_tokens == 0 and plan.num_gather_tokens == 272
    # single-token prompt of text only
    r1 = NS(prompt_len=1, units=[], text_segs=[(0, 1)], block_table=np.array([5], np.int32))
    plan = _plan(wl, [r1])
    assert plan.num_compute_tokens == 1 and plan.num_attn_items == 8


@pytest.mark.parametrize("name", ["tiny", "small_bf16", "rag8b", "agent8b"])
def test_host_plan_row_kv_lo_matches_oracle_local_scope(name):
    cfg = workloads.get_config(name).with_(miss_scope="local")
    wl = workloads.make_workload(cfg)
    plan = _plan(wl)
    want = np.concatenate([L.row_kv_lo(r) for r in wl.requests])
    got = plan.row_kv_lo()
    assert np.array_equal(got, want)
    assert (got > 0).any()
    # the global scope of the same batch: every row sees the whole prefix
    assert not _plan(workloads.make_workload(cfg.with_(miss_scope="global"))).row_kv_lo().any()


def test_bad_miss_scope_and_negative_local_window_are_rejected():
    wl = workloads.generate("tiny")
    req = wl.requests[0]
    bad = NS(**{**vars(req), "miss_scope": 2})
    with pytest.raises(P.TsrError) as e:
        _plan(wl, [bad])
    assert e.value.status == P.TSR_ERR_INVALID_ARG
    units = [NS(**vars(u)) for u in req.units]
    units[0].n_recompute = -1                     # a MISS unit
    assert units[0].residency == 0
    loc = NS(**{**vars(req), "units": units, "miss_scope": 1})
    with pytest.raises(P.TsrError) as e:
        _plan(wl, [loc])
    assert e.value.status == P.TSR_ERR_INVALID_ARG
    # under the global scope a MISS unit's n_recompute is not used
    glob = NS(**{**vars(req), "units": units, "miss_scope": 0})
    _plan(wl, [glob]).destroy()


def _expected_aliased_pages(wl):
    """Request pages whose B positions are all cached tokens of one HIT unit,
    held in the same slots of one pool page (counted from the oracle's
    gather set)."""
    B = wl.model.page_size
    n = 0
    for req in wl.requests:
        by_page = {}
        for ui, j, p in L.gather_tokens(req):
            u = req.units[ui]
            src = (int(u.pool_pages[j // B]), j % B)
            by_page.setdefault(p // B, []).append((ui, src, p % B))
        for pg, toks in by_page.items():
            units = {t[0] for t in toks}
            if len(toks) == B and len(units) == 1 and len({t[1][0] for t in toks}) == 1 \
                    and all(t[1][1] == t[2] for t in toks):
                n += 1
    return n


@pytest.mark.parametrize("name", ["rag8b", "small_bf16", "small_bf16_g8", "agent8b"])
def test_alias_v_pages_match_the_gather_set(name):
    wl = workloads.generate(name)
    plan = P.tsr_plan_create(_model(wl), P.RequestBatch(wl.requests), wl.n_pool_pages,
                             wl.n_req_pages, alias_v=True)
    assert plan.num_aliased_pages == _expected_aliased_pages(wl)
    plain = _plan(wl)
    assert plain.num_aliased_pages == 0
    assert plan.num_gather_tokens == plain.num_gather_tokens
    if name == "rag8b":
        assert plan.num_aliased_pages > 0


@pytest.mark.parametrize("name", ["rag8b", "small_bf16", "agent8b"])
def test_alias_k_pages_and_zero_copy_gather_set(name):
    """K rotated on load aliases the same request pages as V aliasing; with
    both, compose moves none of those pages' tokens."""
    wl = workloads.generate(name)
    mk = lambda **kw: P.tsr_plan_create(_model(wl), P.RequestBatch(wl.requests),
                                        wl.n_pool_pages, wl.n_req_pages, **kw)
    plain, k_only, both = mk(), mk(alias_k=True), mk(alias_k=True, alias_v=True)
    n = _expected_aliased_pages(wl)
    assert k_only.num_aliased_k_pages == n and k_only.num_aliased_pages == 0
    assert both.num_aliased_k_pages == n and both.num_aliased_pages == n
    assert plain.num_aliased_k_pages == 0
    assert k_only.num_gather_tokens == plain.num_gather_tokens
    B = wl.model.page_size
    assert both.num_gather_tokens == plain.num_gather_tokens - B * n
    if name == "rag8b":
        assert n > 0 and both.num_gather_tokens < plain.num_gather_tokens


def test_alias_v_is_bf16_only_and_options_are_checked():
    for name in ("small_f32", "small_fp8"):
        wl = workloads.generate(name)
        with pytest.raises(P.TsrError) as e:
            P.tsr_plan_create(_model(wl), P.RequestBatch(wl.requests), wl.n_pool_pages,
                              wl.n_req_pages, alias_v=True)
        assert e.value.status == P.TSR_ERR_UNSUPPORTED
    import ctypes
    from paper_2609_32999_amd._binding import tsr_plan_options
    wl = workloads.generate("small_bf16")
    batch = P.RequestBatch(wl.requests)
    for field, value in (("reserved", 3), ("alias_k", 2), ("alias_v", -1)):
        opts = tsr_plan_options(alias_v=0)
        if field == "reserved":
            opts.reserved[value] = 1
        else:
            setattr(opts, field, value)
        out = ctypes.c_void_p()
        st = P.lib().tsr_plan_create_ex(ctypes.byref(_model(wl)), batch.array,
                                        len(wl.requests), wl.n_pool_pages, wl.n_req_pages,
                                        ctypes.byref(opts), None, None, 0, None,
                                        ctypes.byref(out))
        assert st == P.TSR_ERR_INVALID_ARG, field
    for name in ("small_f32", "small_fp8"):
        wl = workloads.generate(name)
        with pytest.raises(P.TsrError) as e:
            P.tsr_plan_create(_model(wl), P.RequestBatch(wl.requests), wl.n_pool_pages,
                              wl.n_req_pages, alias_k=True)
        assert e.value.status == P.TSR_ERR_UNSUPPORTED


def test_peak_kernels_validate_before_launch():
    # measurement aids: sizes and alignment are checked on the host, nothing
    # is launched for a rejected call
    assert P.tsr_peak_mfma_flops(2, 3) == 2 * 4 * 3 * 8 * 2 * 32 * 32 * 16
    assert P.tsr_peak_mfma_flops(0, 3) == 0 and P.tsr_peak_mfma_flops(2, -1) == 0
    for args in [(0, 10, 1 << 12), (4, 0, 1 << 12), (4, 10, 0)]:
        with pytest.raises(P.TsrError) as e:
            P.tsr_peak_mfma(*args)
        assert e.value.status == P.TSR_ERR_INVALID_ARG
    for dst, src, n in [(0, 1 << 12, 64), (1 << 12, 0, 64), (1 << 12, 1 << 13, 0),
                        (1 << 12, 1 << 13, 24), (1 << 12 | 8, 1 << 13, 64)]:
        with pytest.raises(P.TsrError) as e:
            P.tsr_peak_copy(dst, src, n)
        assert e.value.status == P.TSR_ERR_INVALID_ARG


def _split_plans(name, scope, *splits):
    wl = workloads.make_workload(workloads.get_config(name).with_(miss_scope=scope))
    m, batch = _model(wl), P.RequestBatch(wl.requests)
    plans = [P.tsr_plan_create(m, batch, wl.n_pool_pages, wl.n_req_pages, split_tiles=s)
             for s in splits]
    sizes = [P.tsr_plan_workspace_size(m, batch, wl.n_pool_pages, wl.n_req_pages,
                                       split_tiles=s) for s in splits]
    return wl, plans, sizes


def test_split_option_counts_and_workspace():
    """Forced key-range splitting adds items and split-buffer slots (at
    least two 64 KiB slots per split item at head_dim 128); -1 never splits;
    values below -1 are refused."""
    wl, (never, forced), (ws_never, ws_forced) = _split_plans("small_bf16", "local", -1, 2)
    assert never.num_attn_splits == 0
    assert forced.num_attn_splits > 0
    assert forced.num_attn_items > never.num_attn_items
    slot = 32 * 4 * wl.model.head_dim * 4
    assert ws_forced >= ws_never + 2 * slot * forced.num_attn_splits
    with pytest.raises(P.TsrError):
        _split_plans("small_bf16", "local", -2)


@pytest.mark.parametrize("name", ["small_fp8", "small_f32"])
def test_split_ignored_outside_bf16(name):
    _, (plan,), _ = _split_plans(name, "local", 2)
    assert plan.num_attn_splits == 0


def test_split_automatic_threshold():
    """Automatic splitting caps one-row-block items at the launch's mean key
    tiles per compute unit.  With one row block per item (attn_kernel 4:
    3,664 items, a mean of 288 tiles per unit) the RAG batch under the
    LOCAL scope splits none; one request alone splits (its suffix rows then
    far exceed the mean).  Three-row-block plans are not split
    automatically: the RAG LOCAL batch's grouped items (1,344 items, 31,680
    tiles, 124 per unit) hold 64 longer than the mean, and splitting them
    measured slower; an explicit threshold still splits them.  Under the
    GLOBAL scope none exceeds the mean either way."""
    wl, (local, forced), _ = _split_plans("rag8b", "local", 0, 124)
    assert local.attn_rows_per_item == 96 and local.num_attn_splits == 0
    assert forced.attn_rows_per_item == 96 and forced.num_attn_splits == 64
    mk = lambda reqs: P.tsr_plan_create(_model(wl), P.RequestBatch(reqs), wl.n_pool_pages,
                                        wl.n_req_pages, attn_kernel=4)
    one_rb = mk(wl.requests)
    assert one_rb.attn_rows_per_item == 32 and one_rb.num_attn_splits == 0
    one = mk(wl.requests[:1])
    assert one.attn_rows_per_item == 32 and one.num_attn_splits > 0
    _, (glob,), _ = _split_plans("rag8b", "global", 0)
    assert glob.attn_rows_per_item == 96 and glob.num_attn_splits == 0

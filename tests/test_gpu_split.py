"""Key-range split of long attention items (plan option split_tiles): the
split ranges and their merge against the CPU oracle, against the unsplit
plan, and run as the two attention parts."""
import numpy as np
import pytest
import torch

import paper_2609_32999_amd as P
import workloads
from gpu_harness import GpuRun, check_request, check_request_sentinels, check_retained, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    P.lib()   # fail loudly if the library is missing


def _local(name, **model_kw):
    cfg = workloads.get_config(name).with_(miss_scope="local")
    if model_kw:
        cfg = cfg.with_(model=cfg.model.__class__(**{**vars(cfg.model), **model_kw}))
    return workloads.make_workload(cfg)


def _check_all(run, expect_split=True):
    if expect_split:
        assert run.plan.num_attn_splits > 0, "no item was split"
    assert run.pool_after_compose_ok and run.pool_after_attn_ok, "pool modified"
    for r in range(len(run.wl.requests)):
        check_request(run, r)
        check_request_sentinels(run, r)
    check_retained(run)


@pytest.mark.parametrize("kernel", [4, 3])
@pytest.mark.parametrize("name,split", [("small_bf16", 1), ("small_bf16", 2),
                                        ("small_bf16", 5), ("small_bf16_g8", 2)])
def test_split_local_matches_oracle(name, split, kernel):
    """Every row of every request against the oracle with items split every
    `split` key tiles (one-tile ranges included; the first range holds the
    unit's first key off the tile grid, the last the causal diagonal), for
    items of one row block (attn_kernel 4) and of three row blocks over rows
    grouped by first visible key (3: a slot per row block and range)."""
    run = GpuRun(_local(name), split_tiles=split, attn_kernel=kernel)
    assert run.plan.attn_rows_per_item == (96 if kernel == 3 else 32)
    # range boundaries stay at or below an item's smallest position: the
    # small batch's grouped three-block items reach at most 4 tiles past it,
    # so 5-tile ranges split none of them
    _check_all(run, expect_split=not (kernel == 3 and split == 5))


@pytest.mark.parametrize("G", [1, 2])
def test_split_local_small_groups(G):
    """Fewer query heads than the four head slots of a split buffer slot."""
    wl = _local("small_bf16", n_q_heads=8 * G)
    _check_all(GpuRun(wl, split_tiles=2))


def _attn(sess, plan, q, part=P.TSR_ATTN_ALL, out=None, lse=None):
    if out is None:
        out, lse = sess.new_outputs(plan, with_lse=True)
    P.tsr_attn_part(plan, part, q, sess.req_k[0], sess.req_v[0], None, out, lse)
    return out, lse


@pytest.mark.parametrize("kernel", [4, 3])
def test_split_against_unsplit_and_parts(kernel):
    """The same batch planned without splitting and with two-tile ranges:
    outputs agree to bf16 rounding and lse to fp32 rounding (the merge sums
    the ranges in fp32); the two attention parts together reproduce the
    split plan's full launch bit for bit."""
    wl = _local("small_bf16")
    run = GpuRun(wl, split_tiles=-1, attn_kernel=kernel)
    s = run.sess
    assert run.plan.num_attn_splits == 0
    plan = s.plan(wl.requests, split_tiles=2, attn_kernel=kernel)
    assert plan.num_attn_splits > 0
    out1, lse1 = _attn(s, plan, run.q)
    torch.cuda.synchronize()
    a, b = run.out.float(), out1.float()
    den = a.norm(dim=-1).clamp_min(1e-30)
    row_err = float(((a - b).norm(dim=-1) / den).max())
    lse_err = float((run.lse - lse1).abs().max())
    say(f"[split] unsplit vs split: worst row rel {row_err:.3e}, lse abs {lse_err:.3e}")
    assert row_err <= 8e-3 and lse_err <= 2e-5
    out2, lse2 = s.new_outputs(plan, with_lse=True)
    out2.fill_(float("nan"))
    lse2.fill_(float("nan"))
    for part in (P.TSR_ATTN_BEFORE_COMPOSE, P.TSR_ATTN_AFTER_COMPOSE):
        _attn(s, plan, run.q, part, out2, lse2)
    torch.cuda.synchronize()
    assert torch.equal(out1.view(torch.int16), out2.view(torch.int16))
    assert torch.equal(lse1, lse2)


@pytest.mark.slow
def test_split_automatic_single_request_local():
    """The automatic threshold splits one full-size RAG request under the
    LOCAL scope (its suffix rows attend to the whole prompt, far beyond the
    launch's mean work per compute unit); every KV head against the oracle."""
    cfg = workloads.get_config("rag8b").with_(miss_scope="local", n_requests=1)
    wl = workloads.make_workload(cfg)
    run = GpuRun(wl)
    assert run.plan.attn_rows_per_item == 32 and run.plan.num_attn_splits > 0
    check_request(run, 0)
    check_request_sentinels(run, 0)


@pytest.mark.slow
def test_grouped_split_full_local_batch():
    """The full RAG batch under the LOCAL scope: three-row-block items over
    rows grouped by first visible key (the automatic choice), the longest
    split by key range at 124 tiles (the launch's mean per compute unit; the
    automatic threshold leaves three-row-block items whole).  The first and
    last requests against the oracle on every KV head."""
    wl = _local("rag8b")
    run = GpuRun(wl, split_tiles=124)
    assert run.plan.attn_rows_per_item == 96 and run.plan.num_attn_splits > 0
    assert run.pool_after_compose_ok and run.pool_after_attn_ok, "pool modified"
    for r in (0, len(wl.requests) - 1):
        check_request(run, r)
        check_request_sentinels(run, r)

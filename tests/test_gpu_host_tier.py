"""GPU tests of the host tier with device staging: hits staged from a
pinned host cache by the copy engines, compose/attention/retain against the
staging arena, writeback and publication, and the fallbacks (through the C
ABI; parity against the oracle)."""
import dataclasses

import numpy as np
import pytest
import torch

import workloads
from gpu_harness import StagedRun, check_request, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2609_32999_amd as P
    P.lib()   # fail loudly if the library is missing


def _hits(wl):
    return wl.hit_unit_ids()


@pytest.mark.parametrize("name,over", [
    ("small_bf16", {}), ("small_fp8", {}), ("small_fp8", {"hit_prob": 0.3}),
    ("small_f32", {}), ("small_bf16", {"miss_scope": "local"})])
def test_staged_hits_match_the_oracle(name, over):
    wl = workloads.make_workload(workloads.get_config(name).with_(**over))
    run = StagedRun(wl, n_layers=2)
    assert not run.prep.fallbacks and not run.prep.declined
    run.check_staged_bytes()
    for r in range(len(wl.requests)):
        check_request(run, r)
    n_ret = sum(len(b) for (_, _, b, _) in run.reservations)
    assert run.check_published() == n_ret
    assert n_ret > 0 or name == "small_fp8" and not over
    for uid in _hits(wl):
        q = run.tier.cache.query(uid)
        assert q["state"] == 2 and q["leases"] == 0, (uid, q)


@pytest.mark.slow
def test_staged_hits_full_size_rag8b():
    """The full RAG-8B batch through the host tier: every hit staged from
    the pinned host cache by the copy engines, then compose, attention and
    retain against the staging arena; every request's K/V and attention
    (every head) against the oracle, retained units written back and
    published."""
    wl = workloads.generate("rag8b")
    run = StagedRun(wl, n_layers=1)
    assert not run.prep.fallbacks and not run.prep.declined
    run.check_staged_bytes()
    for r in range(len(wl.requests)):
        check_request(run, r)
    n_ret = sum(len(b) for (_, _, b, _) in run.reservations)
    assert n_ret > 0 and run.check_published() == n_ret


@pytest.mark.parametrize("name", ["small_bf16", "small_fp8"])
def test_failed_and_overflowing_hits_fall_back_to_text(name):
    wl = workloads.generate(name)
    hits = _hits(wl)
    from gpu_harness import staged_pages_needed
    need = staged_pages_needed(wl.requests, wl.model.page_size)
    run = StagedRun(wl, n_layers=1, n_staging=need // 2, fail_units={hits[0]})
    down = {wl.requests[ri].units[ui].unit_id for ri, ui in run.prep.fallbacks}
    assert hits[0] in down and len(down) > 1
    run.check_staged_bytes()
    for r in range(len(wl.requests)):
        check_request(run, r)
    run.check_published()
    for uid in hits:
        q = run.tier.cache.query(uid)
        assert q["state"] == 2 and q["leases"] == 0, (uid, q)


@pytest.mark.parametrize("name,over", [("small_f32", {}), ("small_fp8", {"hit_prob": 0.3})])
def test_failed_writeback_is_never_published(name, over):
    wl = workloads.make_workload(workloads.get_config(name).with_(**over))
    ret = [u.unit_id for r in wl.requests for u in r.units if u.residency == 0 and u.retain]
    assert len(ret) >= 2
    run = StagedRun(wl, n_layers=1, fail_retain={ret[0]})
    assert run.prep.cancelled == [ret[0]]
    assert run.tier.cache.query(ret[0])["state"] == 0
    assert run.check_published() > 0
    B = wl.model.page_size
    held = sum(-(-int(wl.unit_len[u]) // B) for u in _hits(wl))
    held += sum(-(-int(u.n_tokens) // B) for r in wl.requests for u in r.units
                if u.residency == 0 and u.retain and u.unit_id in run.prep.published)
    assert run.tier.cache.free_blocks == run.tier.n_blocks - held


@pytest.mark.parametrize("name", ["small_bf16", "small_f32"])
def test_retained_unit_is_a_hit_for_the_next_batch(name):
    """A unit computed and retained by one batch is published, then composed
    from the host cache by the next batch at its positions there."""
    wl = workloads.generate(name)
    run1 = StagedRun(wl, n_layers=1)
    assert run1.prep.published
    uid = run1.prep.published[0]
    r1 = next(ri for ri, r in enumerate(wl.requests)
              if any(u.unit_id == uid and u.residency == 0 for u in r.units))
    ui = next(i for i, u in enumerate(wl.requests[r1].units) if u.unit_id == uid)
    u1 = wl.requests[r1].units[ui]
    # the retained state: the fresh pre-RoPE k, v of that unit in batch 1
    pos = np.arange(u1.position, u1.position + u1.n_tokens)
    _, kf, vf = wl.fresh(r1, pos)
    base = workloads.generate(name)

    def state(u):
        return (kf, vf) if u == uid else base.unit_state(u)

    req = dataclasses.replace(wl.requests[r1])
    units = []
    win = max([u.n_recompute for u in req.units if u.residency == 1] + [0])
    for u in req.units:
        nu = dataclasses.replace(u, retain=0)
        if u.unit_id == uid:
            nu = dataclasses.replace(nu, residency=1, n_recompute=win)
        units.append(nu)
    req.units = units
    wl2 = dataclasses.replace(wl, requests=[req], unit_state_fn=state)
    say(f"[gpu] second batch hits unit {uid} retained by request {r1}")
    run2 = StagedRun(wl2, tier=run1.tier, insert=False)
    assert not run2.prep.fallbacks
    assert uid in {u.unit_id for u in run2.prep.requests[0].units if u.residency == 1}
    check_request(run2, 0)


@pytest.mark.parametrize("direction", ["h2d", "d2h", "d2d"])
@pytest.mark.parametrize("n_layers", [1, 3])
def test_copy_blocks_runs_and_layers(direction, n_layers):
    """tsr_copy_blocks moves exactly the listed blocks, merged runs and
    single blocks alike, in every layer, and nothing else."""
    import paper_2609_32999_amd as P
    g = torch.Generator().manual_seed(7)
    nsrc, ndst, blk = 37, 29, 96          # bytes per block
    src_cpu = torch.randint(0, 256, (n_layers, nsrc, blk), dtype=torch.uint8, generator=g)
    dst_cpu = torch.randint(0, 256, (n_layers, ndst, blk), dtype=torch.uint8, generator=g)
    src = src_cpu.clone().pin_memory() if direction == "h2d" else src_cpu.cuda()
    dst = dst_cpu.clone().pin_memory() if direction == "d2h" else dst_cpu.cuda()
    sb = [3, 4, 5, 6, 20, 21, 0, 36, 10, 11, 12]
    db = [0, 1, 2, 3, 10, 11, 28, 5, 15, 16, 27]      # 10,11,12 -> 15,16,27 breaks a run
    P.tsr_copy_blocks(dst, ndst, db, src, nsrc, sb, blk, n_layers=n_layers,
                      dst_layer_stride=dst[0].nbytes, src_layer_stride=src[0].nbytes,
                      stream=torch.cuda.current_stream())
    torch.cuda.synchronize()
    want = dst_cpu.clone()
    want[:, db] = src_cpu[:, sb]
    assert torch.equal(dst.cpu(), want)

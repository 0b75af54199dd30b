"""GPU tests of zero-copy composition: V aliasing (attention reads V of whole
gathered pages from the pool), K rotated on load (attention reads their
pre-RoPE K from the pool and rotates it as it stages the tile), and both
(compose does not touch those pages).  The result equals the composed path
bit for bit and matches the oracle."""
import numpy as np
import pytest
import torch

import workloads
from gpu_harness import check_request, fill_sentinel, is_sentinel, say
from oracle import layout as L
from paper_2609_32999_amd import staging
from paper_2609_32999_amd.session import Session

pytestmark = pytest.mark.gpu

ALIGNED = dict(instruction_tokens=64, extra={"unit_tokens_multiple": 64}, unit_tokens=(1, 3))
CASES = [("small_bf16", ALIGNED), ("small_bf16", {**ALIGNED, "miss_scope": "local"}),
         ("small_bf16_g8", ALIGNED), ("small_bf16", {**ALIGNED, "n_recompute": 0})]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2609_32999_amd as P
    P.lib()


def aliased_pages(wl):
    """(request, prompt page) of every request page whose B positions are
    cached tokens of one HIT unit in the same slots of one pool page."""
    B = wl.model.page_size
    out = []
    for r, req in enumerate(wl.requests):
        by_page = {}
        for ui, j, p in L.gather_tokens(req):
            u = req.units[ui]
            by_page.setdefault(p // B, []).append((ui, int(u.pool_pages[j // B]), j % B == p % B))
        for pg, toks in by_page.items():
            if len(toks) == B and len({t[0] for t in toks}) == 1 and \
                    len({t[1] for t in toks}) == 1 and all(t[2] for t in toks):
                out.append((r, pg))
    return out


MODES = {"v": dict(alias_v=True), "k": dict(alias_k=True),
         "kv": dict(alias_v=True, alias_k=True)}


class Run:
    def __init__(self, wl, mode=None, assemble=False, split_tiles=0, attn_kernel=0):
        m = wl.model
        self.wl = wl
        s = self.sess = Session(m, wl.n_pool_pages, wl.n_req_pages)
        for t in (s.pool_k, s.pool_v, s.req_k, s.req_v):
            fill_sentinel(t)
        staging.upload_pool(s, wl)
        self.plan = p = s.plan(wl.requests, split_tiles=split_tiles, attn_kernel=attn_kernel,
                               **(MODES[mode] if mode else {}))
        q, k, v = staging.fresh_inputs(s, wl, p)
        self.pos, self.req = p.compute_positions()
        self.out, self.lse = s.new_outputs(p, True)
        if assemble:
            s.assemble(p, k, v)
            s.attn(p, q, self.out, self.lse)
        else:
            s.compose(p)
            s.prefill_attn(p, q, k, v, self.out, self.lse)
        torch.cuda.synchronize()

    def request_kv(self, r):
        return staging.request_kv(self.sess, self.wl, r)

    def rows_of(self, r):
        return np.nonzero(self.req == r)[0]


def _check_against_composed(wl, run, ref, mode, pages):
    assert torch.equal(run.out.view(torch.int16), ref.out.view(torch.int16))
    assert torch.equal(run.lse.view(torch.int32), ref.lse.view(torch.int32))
    aliased = {int(wl.requests[r].block_table[pg]) for r, pg in pages}
    # the aliased halves of aliased pages are never written; everything else
    # equals the composed request pages
    for arena, ref_arena, half in ((run.sess.req_k, ref.sess.req_k, "k"),
                                   (run.sess.req_v, ref.sess.req_v, "v")):
        skipped = half in mode
        for rp in range(arena.shape[1]):
            if skipped and rp in aliased:
                assert bool(is_sentinel(arena[0, rp]).all()), (half, rp)
            else:
                assert torch.equal(arena[0, rp].view(torch.int16),
                                   ref_arena[0, rp].view(torch.int16)), (half, rp)


@pytest.mark.parametrize("mode", ["v", "k", "kv"])
@pytest.mark.parametrize("name,over", CASES)
def test_aliasing_equals_composed_path(name, over, mode):
    wl = workloads.make_workload(workloads.get_config(name).with_(**over))
    pages = aliased_pages(wl)
    say(f"[gpu] aliasing {mode}: workload={wl.name} seed={wl.seed} aliased pages={len(pages)}")
    # the same kernel on both sides (K rotated on load runs on the row-block
    # kernel only)
    kern = 2 if "k" in mode else 0
    ref = Run(wl, attn_kernel=kern)
    run = Run(wl, mode, assemble=(mode == "kv"), attn_kernel=kern)
    assert len(pages) > 0
    assert run.plan.num_aliased_pages == (len(pages) if "v" in mode else 0)
    assert run.plan.num_aliased_k_pages == (len(pages) if "k" in mode else 0)
    _check_against_composed(wl, run, ref, mode, pages)
    for r in range(len(wl.requests)):
        check_request(run, r, check_kv=False)


@pytest.mark.slow
@pytest.mark.parametrize("mode", ["v", "k", "kv"])
def test_aliasing_three_row_blocks(mode):
    """Aliasing under the twelve-wave attention (96-row items): a two-request
    RAG-shaped batch, bit-equal to the composed path, one sampled KV head of
    each request against the oracle."""
    wl = workloads.make_workload(workloads.get_config("rag8b").with_(n_requests=2))
    pages = aliased_pages(wl)
    say(f"[gpu] aliasing {mode}: workload={wl.name} seed={wl.seed} aliased pages={len(pages)}")
    ref = Run(wl, attn_kernel=2)
    run = Run(wl, mode, assemble=True, attn_kernel=2)
    assert run.plan.attn_rows_per_item > 32
    assert len(pages) > 0
    _check_against_composed(wl, run, ref, mode, pages)
    rng = np.random.default_rng(43)
    for r in range(len(wl.requests)):
        check_request(run, r, kv_heads=[int(rng.integers(wl.model.n_kv_heads))], check_kv=False)


@pytest.mark.parametrize("mode", ["v", "k", "kv"])
def test_aliasing_with_key_range_split(mode):
    """Aliased plans whose items are split by key range (two-tile ranges
    under the LOCAL scope): bit-equal to the composed plan split the same
    way, and the oracle."""
    wl = workloads.make_workload(workloads.get_config("small_bf16").with_(
        **{**ALIGNED, "miss_scope": "local"}))
    pages = aliased_pages(wl)
    ref = Run(wl, split_tiles=2, attn_kernel=2)
    run = Run(wl, mode, assemble=(mode == "kv"), split_tiles=2, attn_kernel=2)
    assert run.plan.num_attn_splits > 0 and run.plan.num_attn_splits == ref.plan.num_attn_splits
    _check_against_composed(wl, run, ref, mode, pages)
    for r in range(len(wl.requests)):
        check_request(run, r, check_kv=False)

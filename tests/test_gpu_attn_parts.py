"""GPU tests of the attention split around compose (tsr_attn_part): the
items that read no composed key run before compose, the rest after; the
two together equal the whole launch bit for bit and match the oracle."""
import numpy as np
import pytest
import torch

import workloads
from gpu_harness import check_request, fill_sentinel, say
from paper_2609_32999_amd import (TSR_ATTN_AFTER_COMPOSE, TSR_ATTN_ALL,
                                  TSR_ATTN_BEFORE_COMPOSE, staging)
from paper_2609_32999_amd.session import Session

pytestmark = pytest.mark.gpu

ALIGNED = dict(instruction_tokens=64, extra={"unit_tokens_multiple": 64}, unit_tokens=(1, 3))
CASES = [
    ("tiny", {}), ("tiny", {"miss_scope": "local"}), ("small_f32", {"miss_scope": "local"}),
    ("small_fp8", {"miss_scope": "local"}),
    ("small_bf16", {**ALIGNED, "miss_scope": "local"}),
    ("small_bf16", {**ALIGNED}),
    ("small_bf16_g8", {**ALIGNED, "miss_scope": "local"}),
]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2609_32999_amd as P
    P.lib()


class PartsRun:
    def __init__(self, wl):
        m = wl.model
        self.wl = wl
        s = self.sess = Session(m, wl.n_pool_pages, wl.n_req_pages)
        for t in (s.pool_k, s.pool_v, s.req_k, s.req_v):
            fill_sentinel(t)
        if s.e4m3:
            s.pool_scale.fill_(float("nan"))
            s.req_scale.fill_(float("nan"))
        staging.upload_pool(s, wl)
        self.plan = p = s.plan(wl.requests)
        self.n1 = p.num_attn_items_part(TSR_ATTN_BEFORE_COMPOSE)
        self.n2 = p.num_attn_items_part(TSR_ATTN_AFTER_COMPOSE)
        say(f"[gpu] parts: workload={wl.name} seed={wl.seed} items={p.num_attn_items} "
            f"before={self.n1} after={self.n2}")
        q, k, v = staging.fresh_inputs(s, wl, p)
        self.pos, self.req = p.compute_positions()
        self.out, self.lse = s.new_outputs(p, True)
        s.append(p, k, v)
        s.attn(p, q, self.out, self.lse, part=TSR_ATTN_BEFORE_COMPOSE)
        s.compose(p)
        s.attn(p, q, self.out, self.lse, part=TSR_ATTN_AFTER_COMPOSE)
        self.out0, self.lse0 = s.new_outputs(p, True)
        s.attn(p, q, self.out0, self.lse0, part=TSR_ATTN_ALL)
        torch.cuda.synchronize()

    def request_kv(self, r):
        return staging.request_kv(self.sess, self.wl, r)

    def rows_of(self, r):
        return np.nonzero(self.req == r)[0]


@pytest.mark.parametrize("name,over", CASES)
def test_parts_around_compose(name, over):
    wl = workloads.make_workload(workloads.get_config(name).with_(**over))
    run = PartsRun(wl)
    assert run.n1 > 0 and run.n2 > 0
    a = run.out.view(torch.int16) if run.out.dtype == torch.bfloat16 else run.out.view(torch.int32)
    b = run.out0.view(torch.int16) if run.out0.dtype == torch.bfloat16 else run.out0.view(torch.int32)
    assert torch.equal(a, b), "the two parts differ from the whole launch"
    assert torch.equal(run.lse.view(torch.int32), run.lse0.view(torch.int32))
    for r in range(len(wl.requests)):
        check_request(run, r)

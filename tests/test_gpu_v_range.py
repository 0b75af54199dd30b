"""V beyond fp16's range (the P V product runs in fp16): refused loudly.

A bf16 V of magnitude 65536 or more is staged as NaN and an e4m3 page whose
V scale exceeds 2^7 dequantizes to NaN, so the outputs of rows that read
such a value are non-finite instead of silently clipped.
The oracle (fp64) stays finite on the same input; the test checks that the
kernel's output is non-finite where the value is read (rows at or after
its position, heads of its KV head -- every head for e4m3, whose page
scale covers all KV heads of a page) and finite for the other KV heads and
requests.  (Earlier rows of a row block that loads the value's key tile
may turn non-finite too: a masked probability of 0 times NaN is NaN.)"""
import numpy as np
import pytest
import torch

import paper_2609_32999_amd as P
import workloads
from gpu_harness import say
from paper_2609_32999_amd import staging
from paper_2609_32999_amd.session import Session

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    P.lib()


@pytest.mark.parametrize("name,big", [("small_bf16", 1.0e6), ("small_bf16", 65536.0),
                                      ("small_fp8", 1.0e6)])
def test_out_of_range_v_gives_non_finite_outputs(name, big):
    wl = workloads.generate(name)
    m = wl.model
    s = Session(m, wl.n_pool_pages, wl.n_req_pages)
    staging.upload_pool(s, wl)
    plan = s.plan(wl.requests)
    q, k, v = staging.fresh_inputs(s, wl, plan)
    pos, req = plan.compute_positions()
    rows0 = np.nonzero(req == 0)[0]
    t = int(rows0[len(rows0) // 2])          # a computed row in the middle of request 0
    g, d = 1, 5
    v[t, g, d] = big
    s.compose(plan)
    out, lse = s.new_outputs(plan, with_lse=True)
    s.prefill_attn(plan, q, k, v, out, lse)
    torch.cuda.synchronize()
    o = out.float().cpu().numpy()
    G = m.n_q_heads // m.n_kv_heads
    # an e4m3 page has one V scale for all its KV heads: every head reads it
    heads = (np.arange(m.n_q_heads) if m.kv_dtype == "e4m3"
             else np.arange(g * G, (g + 1) * G))
    later = rows0[pos[rows0] >= pos[t]]
    say(f"[vrange] {name} big={big} row {t} pos {pos[t]}: {len(later)} later rows")
    hit = o[np.ix_(later, heads)][..., d]
    assert not np.isfinite(hit).any(), "an output that reads the value stayed finite"
    others = np.setdiff1d(np.arange(m.n_q_heads), heads)
    assert np.isfinite(o[:, others]).all(), "heads of other KV heads became non-finite"
    assert np.isfinite(o[np.nonzero(req != 0)[0]]).all(), "other requests became non-finite"

"""The allocation-free plan entry point, tsr_plan_create_static (the plan's
device image in the library's own plan area), against tsr_plan_create with
a caller workspace: identical request pages, outputs and lse through the
assembly and attention, on two static plans in a row (the second for a
smaller batch); the superseded plan is refused; an oversized batch is
refused before any device call."""
import dataclasses
from types import SimpleNamespace as NS

import numpy as np
import pytest
import torch

import paper_2609_32999_amd as P
import workloads
from paper_2609_32999_amd import staging
from paper_2609_32999_amd.session import Session


def _subset(wl, n):
    return dataclasses.replace(wl, requests=wl.requests[:n])


def _run(sess, plan, wl):
    """assembly + attention of one layer; returns request pages, out, lse."""
    q, k, v = staging.fresh_inputs(sess, wl, plan)
    sess.req_k.zero_()
    sess.req_v.zero_()
    if sess.e4m3:
        sess.req_scale.zero_()
    sess.assemble(plan, k, v)
    out, lse = sess.new_outputs(plan, with_lse=True)
    sess.attn(plan, q, out, lse)
    torch.cuda.synchronize()
    res = [sess.req_k.clone(), sess.req_v.clone(), out, lse]
    if sess.e4m3:
        res.append(sess.req_scale.clone())
    return res


def _same(a, b):
    assert len(a) == len(b)
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.uint8), y.view(torch.uint8))


@pytest.mark.gpu
@pytest.mark.parametrize("name", ["small_bf16", "small_fp8", "small_f32"])
def test_static_plan_equals_workspace_plan_twice(name):
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    wl = workloads.generate(name)
    assert len(wl.requests) >= 2
    sess = Session(wl.model, wl.n_pool_pages, wl.n_req_pages)
    staging.upload_pool(sess, wl)
    print(f"[no-alloc] {name}: {len(wl.requests)} requests", flush=True)

    first = sess.plan_static(wl.requests)
    _same(_run(sess, first, wl), _run(sess, sess.plan(wl.requests), wl))

    small = _subset(wl, 1)                      # second call: a smaller batch
    print(f"[no-alloc] {name}: second static plan, 1 request", flush=True)
    second = sess.plan_static(small.requests)
    assert second.num_compute_tokens < first.num_compute_tokens
    _same(_run(sess, second, small), _run(sess, sess.plan(small.requests), small))

    with pytest.raises(P.TsrError) as e:         # superseded by `second`
        _run(sess, first, wl)
    assert e.value.status == P.TSR_ERR_STATE and "superseded" in e.value.message
    # the owning plan still runs
    _same(_run(sess, second, small), _run(sess, sess.plan(small.requests), small))


def test_static_plan_refuses_oversized_batch():
    """Two requests gathering one 600,000-token unit: 1.2 M gather
    descriptors (about 19 MiB of plan image) exceed the 16 MiB area."""
    B, n = 16, 600_000
    pages = np.arange(n // B, dtype=np.int32)
    reqs = []
    for r in range(2):
        u = NS(unit_id=1, position=0, n_tokens=n, residency=P.TSR_HIT, n_recompute=0,
               retain=0, pool_pages=pages)
        reqs.append(NS(prompt_len=n + 16, units=[u], text_segs=[(n, 16)],
                       block_table=np.arange(r * (n // B + 1), (r + 1) * (n // B + 1),
                                             dtype=np.int32)))
    model = P.make_model(32, 8, 128, page_size=B, max_position=1 << 20)
    batch = P.RequestBatch(reqs)
    ws = P.tsr_plan_workspace_size(model, batch, n // B, 2 * (n // B + 1))
    assert ws > 16 << 20
    with pytest.raises(P.TsrError) as e:
        P._binding.tsr_plan_create_static(model, batch, n // B, 2 * (n // B + 1), None)
    assert e.value.status == P.TSR_ERR_OUT_OF_RANGE and "static plan area" in e.value.message

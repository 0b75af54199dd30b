"""GPU parity of each bf16 attention kernel shape against the oracle, on
every request and query head: the pipelined kernel (attn_kernel 1: items of
two 32-row blocks, eight waves, the next tile's QK^T under this tile's
softmax) and the row-block kernel with three row blocks over rows grouped
by first visible key (3) and with one row block (4).  Cases: GQA groups of
1, 2, 4 and 8, pages of 32 keys, the LOCAL scope (a first visible key inside
a tile; grouped rows out of computed order), rows past an item's last, no
recompute window or no text, all hits, all misses, duplicate units and V
aliasing."""
import numpy as np
import pytest
import torch

import workloads
from gpu_harness import GpuRun, check_request, check_request_sentinels, check_retained, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2609_32999_amd as P
    P.lib()


def _shape(cfg, **over):
    return cfg.model.__class__(**{**vars(cfg.model), **over})


def _case(name):
    base = workloads.get_config("small_bf16")
    if name == "small_bf16":
        return base
    if name == "g1":
        return base.with_(model=_shape(base, n_q_heads=8))
    if name == "g2":
        return base.with_(model=_shape(base, n_q_heads=16))
    if name == "g8":
        return workloads.get_config("small_bf16_g8")
    if name == "page32":
        return base.with_(model=_shape(base, page_size=32), n_recompute=0)
    if name == "local":
        return base.with_(miss_scope="local")
    if name == "local_g8":
        return workloads.get_config("small_bf16_g8").with_(miss_scope="local")
    if name == "all_hit":
        return base.with_(hit_prob=1.0, n_recompute=0, instruction_tokens=0, query_tokens=3)
    if name == "all_miss":
        return base.with_(hit_prob=0.0)
    if name == "dup_units":
        # unit 2 a HIT then a MISS, unit 5 a MISS then a HIT, unit 7 a MISS twice
        return base.with_(unit_order=((2, 5, 2, 7, 5, 7), (7, 2, 7)),
                          residency_pattern=(1, 0, 0, 0, 1, 0), n_requests=2)
    if name == "long_rows":
        # long runs of rows (several 64-row items per request, the fast loop)
        return base.with_(unit_tokens=(300, 700), hit_prob=0.3, n_requests=2)
    raise KeyError(name)


CASES = ["small_bf16", "g1", "g2", "g8", "page32", "local", "local_g8", "all_hit",
         "all_miss", "dup_units", "long_rows"]


@pytest.mark.parametrize("kernel", [1, 3, 4])
@pytest.mark.parametrize("name", CASES)
def test_attention_kernel_against_oracle(name, kernel):
    wl = workloads.make_workload(_case(name))
    run = GpuRun(wl, attn_kernel=kernel)
    assert run.plan.attn_rows_per_item == {1: 64, 3: 96, 4: 32}[kernel]
    assert run.pool_after_compose_ok and run.pool_after_attn_ok, "pool modified"
    for r in range(len(wl.requests)):
        check_request(run, r)
        check_request_sentinels(run, r)
    check_retained(run)


@pytest.mark.parametrize("name", ["small_bf16", "g8", "long_rows"])
def test_pipelined_v_aliasing_equals_composed(name):
    """V read from whole gathered pool pages (alias_v) under the pipelined
    kernel: outputs and lse equal the composed plan's bit for bit."""
    cfg = _case(name).with_(instruction_tokens=64, extra={"unit_tokens_multiple": 64},
                            unit_tokens=(1, 3) if name != "long_rows" else (5, 9))
    wl = workloads.make_workload(cfg)
    ref = GpuRun(wl, attn_kernel=1)
    run = GpuRun(wl, attn_kernel=1, alias_v=True)
    say(f"[gpu] aliased V pages: {run.plan.num_aliased_pages}")
    assert run.plan.num_aliased_pages > 0
    assert torch.equal(run.out.view(torch.int16), ref.out.view(torch.int16))
    assert torch.equal(run.lse.view(torch.int32), ref.lse.view(torch.int32))
    for r in range(len(wl.requests)):
        check_request(run, r, check_kv=False)


def test_pipelined_is_deterministic():
    """Two launches of one plan give the same bits (no order-dependent
    reduction across waves)."""
    wl = workloads.make_workload(_case("long_rows"))
    run = GpuRun(wl, attn_kernel=1)
    out2, lse2 = run.sess.new_outputs(run.plan, True)
    run.sess.attn(run.plan, run.q, out2, lse2)
    torch.cuda.synchronize()
    assert torch.equal(out2.view(torch.int16), run.out.view(torch.int16))
    assert torch.equal(lse2.view(torch.int32), run.lse.view(torch.int32))

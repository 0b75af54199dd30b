"""GPU parity of the HIP path against the CPU oracle (through the C ABI)."""
import itertools

import numpy as np
import pytest
import torch

import workloads
from gpu_harness import (GpuRun, check_request, check_request_sentinels, check_retained,
                         say)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2609_32999_amd as P
    P.lib()   # fail loudly if the library is missing


def _full_check(wl):
    run = GpuRun(wl)
    assert run.pool_after_compose_ok and run.pool_after_attn_ok, "pool modified"
    for r in range(len(wl.requests)):
        check_request(run, r)
        check_request_sentinels(run, r)
    check_retained(run)
    return run


def test_tiny_fp32():
    _full_check(workloads.generate("tiny"))


@pytest.mark.parametrize("pattern", list(itertools.product([0, 1], repeat=4)))
def test_tiny_all_residency_patterns(pattern):
    cfg = workloads.get_config("tiny").with_(residency_pattern=tuple(pattern))
    _full_check(workloads.make_workload(cfg))


@pytest.mark.parametrize("name", ["small_f32", "small_bf16", "small_bf16_g8"])
def test_small_configs(name):
    _full_check(workloads.generate(name))


@pytest.mark.parametrize("G", [1, 2])
def test_bf16_small_groups(G):
    cfg = workloads.get_config("small_bf16")
    shape = cfg.model.__class__(**{**vars(cfg.model), "n_q_heads": 8 * G})
    _full_check(workloads.make_workload(cfg.with_(model=shape)))


def test_bf16_page_size_32_and_recompute_edges():
    cfg = workloads.get_config("small_bf16")
    shape = cfg.model.__class__(**{**vars(cfg.model), "page_size": 32})
    _full_check(workloads.make_workload(cfg.with_(model=shape, n_recompute=0)))
    _full_check(workloads.make_workload(cfg.with_(n_recompute=1000)))


def test_bf16_all_hit_no_window_no_text():
    cfg = workloads.get_config("small_bf16").with_(hit_prob=1.0, n_recompute=0,
                                                   instruction_tokens=0, query_tokens=3)
    _full_check(workloads.make_workload(cfg))


def test_bf16_all_miss():
    cfg = workloads.get_config("small_bf16").with_(hit_prob=0.0)
    _full_check(workloads.make_workload(cfg))


@pytest.mark.slow
def test_rag8b_full_size():
    """The 8B RAG batch at full size, in the launch configuration the
    benchmark times: K/V of every request bit-exact; attention for every
    request on two sampled KV heads (all their query heads and rows)."""
    wl = workloads.generate("rag8b")
    run = GpuRun(wl)
    assert run.pool_after_compose_ok and run.pool_after_attn_ok
    heads = np.random.default_rng(101).choice(wl.model.n_kv_heads, 2, replace=False)
    for r in range(len(wl.requests)):
        check_request(run, r, kv_heads=sorted(heads.tolist()))
        check_request_sentinels(run, r)
    assert check_retained(run) > 0


@pytest.mark.slow
@pytest.mark.parametrize("name,n_req", [("agent8b", 3), ("long70b", 1)])
def test_large_configs_sampled(name, n_req):
    wl = workloads.generate(name)
    run = GpuRun(wl, with_lse=False)
    rng = np.random.default_rng(7)
    for r in sorted(rng.choice(len(wl.requests), n_req, replace=False).tolist()):
        check_request(run, r, kv_heads=[int(rng.integers(wl.model.n_kv_heads))])
    assert run.pool_after_attn_ok


def test_fp8_small():
    _full_check(workloads.generate("small_fp8"))


def test_fp8_small_all_miss_and_g8():
    _full_check(workloads.make_workload(workloads.get_config("small_fp8").with_(hit_prob=0.0)))
    cfg = workloads.get_config("small_fp8")
    shape = cfg.model.__class__(**{**vars(cfg.model), "n_q_heads": 64})
    _full_check(workloads.make_workload(cfg.with_(model=shape)))


@pytest.mark.slow
def test_fp8rag_full_size():
    """The fp8 RAG batch at full size: every request's codes and page scales
    bit-exact; attention on two sampled KV heads of every request."""
    wl = workloads.generate("fp8rag")
    run = GpuRun(wl)
    assert run.pool_after_compose_ok and run.pool_after_attn_ok
    heads = np.random.default_rng(202).choice(wl.model.n_kv_heads, 2, replace=False)
    for r in range(0, len(wl.requests), 3):
        check_request(run, r, kv_heads=sorted(heads.tolist()))
    assert check_retained(run) > 0

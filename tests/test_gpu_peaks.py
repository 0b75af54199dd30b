"""The measurement-aid kernels the benchmark uses for achievable peaks."""
import pytest

torch = pytest.importorskip("torch")

import paper_2609_32999_amd as P

pytestmark = pytest.mark.gpu


def test_peak_copy_copies_exactly():
    n = (5 << 20) + 48                       # not a multiple of the grid's stride
    src = torch.randint(0, 256, (n,), dtype=torch.uint8, device="cuda")
    buf = torch.full((n + 256,), 7, dtype=torch.uint8, device="cuda")
    P.tsr_peak_copy(buf, src, n)
    torch.cuda.synchronize()
    assert torch.equal(buf[:n], src)
    assert torch.all(buf[n:] == 7)           # nothing written past the end


def test_peak_mfma_runs_and_counts_flops():
    n_wg, iters = 16, 4
    out = torch.full((n_wg * 256,), float("nan"), dtype=torch.float32, device="cuda")
    P.tsr_peak_mfma(n_wg, iters, out)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()
    assert P.tsr_peak_mfma_flops(n_wg, iters) == n_wg * 4 * iters * 8 * 32768

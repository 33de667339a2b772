"""The comparison point through its C-ABI (include/rg_baseline.h): the transient FP32 copy is
the exact widening of W, and y agrees with the binary64 product within the FP32 GEMM bound.
Its bits are not the documented order's (vendor GEMM), so no bitwise claim is made."""
import numpy as np
import pytest

from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M,N,K", [(1, 4096, 4096), (4, 1000, 1000), (16, 257, 8200)])
def test_cast_baseline_matches_fp64_within_bound(M, N, K):
    import torch
    import oracle
    from paper_2609_25624_amd import baseline
    x, w = gu.layer(M, N, K, seed=M + N + K)
    xd, wd = gu.to_dev(x, w)
    wt = torch.full((N, K), float("nan"), dtype=torch.float32, device=gu.dev())
    y = torch.full((M, N), float("nan"), dtype=torch.float32, device=gu.dev())
    baseline.rg_linear_cast_baseline(xd, wd, wt, y)
    torch.cuda.synchronize()
    assert np.array_equal(wt.cpu().numpy().view(np.uint32), w.astype(np.uint32) << 16)
    y64, asum = oracle.ref_fp64(x, w)
    err = np.abs(y.cpu().numpy().astype(np.float64) - y64)
    # any FP32 summation order: |err| <= K u / (1 - K u) * sum |x w|
    u = 2.0 ** -24
    assert np.all(err <= K * u / (1 - K * u) * asum + 1e-30)

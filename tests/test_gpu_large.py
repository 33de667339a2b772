"""Weights beyond 4 GiB: 64-bit addressing in every kernel family.

W is a seeded block of R = 1021 rows repeated down N rows on the GPU, so every output
must equal the oracle's output for row n mod R.  The shapes put rows past the 4 GiB
mark: for K = 2304, 2^32 bytes is not a whole number of rows, and for K = 4096 it is
524288 rows, which is not a multiple of R.  A 32-bit offset that wrapped would read
other weights and change the bits.  Every output is compared, not a sample.
"""
import numpy as np
import pytest

from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

_R = 1021


@pytest.mark.parametrize("M,N,K,kernel", [(1, 1048579, 2304, "decode_xs"), (1, 524309, 4096, "gemv"),
                                          (3, 1048579, 2304, "decode"), (16, 1048579, 2304, "ktile"),
                                          (70, 1048579, 2304, "tiled")])
def test_weights_beyond_4_gib(M, N, K, kernel):
    import torch
    import paper_2609_25624_amd as rg
    assert 2 * N * K > (1 << 32)
    plan = rg.rg_plan(M, N, K)
    assert plan["kernel_name"] == kernel
    gu.log(f"large W: M={M} N={N} K={K} ({2 * N * K / 2**30:.2f} GiB) kernel={kernel}")
    x, wblock = gu.layer(M, _R, K, seed=77 + M)
    want_block = gu.oracle_full(x, wblock)
    xd, wb = gu.to_dev(x, wblock)
    reps = (N + _R - 1) // _R
    wbig = wb.repeat(reps, 1)[:N]
    assert wbig.is_contiguous() and wbig.shape == (N, K)
    y = torch.empty((M, N), dtype=torch.float32, device=gu.dev())
    rg.rg_linear(xd, wbig, y)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    del wbig, y
    torch.cuda.empty_cache()
    want = np.tile(want_block, (1, reps))[:, :N]
    gu.assert_bitwise(got, want, f"large W ({M},{N},{K}) {kernel}")

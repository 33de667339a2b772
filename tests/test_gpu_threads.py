"""Calls from several host threads at once, each on its own stream, through the C-ABI.

Every output must equal the oracle bit for bit, also while another thread changes the
process-wide scheduling override (the workgroup order), since launch settings never
change the arithmetic.
"""
import threading
import time

import pytest

from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

_SHAPES = [(1, 1030, 4096), (3, 300, 1000), (16, 515, 4104), (1, 777, 14336), (70, 130, 1000)]
_REPEATS = 12


@pytest.fixture(autouse=True)
def _reset_launch():
    import paper_2609_25624_amd as rg
    rg.rg_linear_set_launch(None)
    yield
    rg.rg_linear_set_launch(None)


def _cases():
    cases = []
    for i, (M, N, K) in enumerate(_SHAPES):
        x, w = gu.layer(M, N, K, seed=40 + i)
        xd, wd = gu.to_dev(x, w)
        cases.append((xd, wd, gu.oracle_full(x, w), M, N))
    return cases


def _run_threads(cases, toggle):
    import torch
    import paper_2609_25624_amd as rg
    torch.cuda.synchronize()                      # inputs are ready before other streams read them
    outs = [[] for _ in cases]
    errors = []
    done = threading.Event()

    def worker(i):
        try:
            xd, wd, _, M, N = cases[i]
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                for _ in range(_REPEATS):
                    y = torch.empty((M, N), dtype=torch.float32, device=xd.device)
                    rg.rg_linear(xd, wd, y, stream=s)
                    outs[i].append(y)
            s.synchronize()
        except Exception as e:                    # reported by the main thread
            errors.append((i, repr(e)))

    def toggler():
        k = 0
        while not done.is_set():
            rg.rg_linear_set_launch(grid_order=1) if k % 2 else rg.rg_linear_set_launch(None)
            k += 1
            time.sleep(0.0002)

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(cases))]
    tog = threading.Thread(target=toggler) if toggle else None
    if tog:
        tog.start()
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    done.set()
    if tog:
        tog.join(timeout=30)
    torch.cuda.synchronize()
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors
    for i, (_, _, want, M, N) in enumerate(cases):
        assert len(outs[i]) == _REPEATS
        for r, y in enumerate(outs[i]):
            gu.assert_bitwise(y.cpu().numpy(), want, f"shape {_SHAPES[i]} repeat {r}")


def test_concurrent_calls_on_separate_streams():
    gu.log("threads: concurrent rg_linear on separate streams")
    _run_threads(_cases(), toggle=False)


def test_concurrent_calls_while_the_launch_order_changes():
    gu.log("threads: concurrent rg_linear while another thread flips the workgroup order")
    _run_threads(_cases(), toggle=True)

"""Helpers for the GPU tests: device copies of seeded inputs, C-ABI calls, bitwise comparison."""
import numpy as np

import oracle
import synth

_oracle_cache = {}


def dev():
    import torch
    return torch.device("cuda:0")


def to_dev(x, w):
    import torch
    xd = torch.from_numpy(np.array(x, dtype=np.float32, copy=True)).to(dev())
    wd = torch.from_numpy(np.array(w, dtype=np.uint16, copy=True).view(np.int16)).to(dev())
    return xd, wd


def run(xd, wd, stream=None, out=None):
    import torch
    import paper_2609_25624_amd as rg
    M, N = xd.shape[0], wd.shape[0]
    y = out if out is not None else torch.empty((M, N), dtype=torch.float32, device=xd.device)
    rg.rg_linear(xd, wd, y, stream=stream)
    return y


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def assert_bitwise(got, want, what):
    g, w = bits(got), bits(want)
    assert g.shape == w.shape, (what, g.shape, w.shape)
    bad = np.flatnonzero(g.ravel() != w.ravel())
    if bad.size:
        i = bad[0]
        raise AssertionError(f"{what}: {bad.size}/{g.size} outputs differ; first at flat {i}: "
                             f"gpu 0x{g.ravel()[i]:08x} oracle 0x{w.ravel()[i]:08x}")


_layer_cache = {}


def layer(M, N, K, seed=0, w_std=0.02, layer_id=0):
    """Seeded (x, W) for one layer; cached, returned read-only (copy before editing)."""
    key = (M, N, K, seed, w_std, layer_id)
    if key not in _layer_cache:
        if len(_layer_cache) > 6:
            _layer_cache.clear()
        x, w = synth.layer_inputs(M, N, K, seed=seed, w_std=w_std, layer=layer_id)
        x.flags.writeable = False
        w.flags.writeable = False
        _layer_cache[key] = (x, w)
    return _layer_cache[key]


def oracle_full(x, w, key=None):
    if key is not None and key in _oracle_cache:
        return _oracle_cache[key]
    y = oracle.linear(x, w)
    if key is not None:
        _oracle_cache[key] = y
    return y


def sample_indices(M, N, count, seed=0):
    rng = np.random.default_rng(seed)
    rows = rng.integers(0, M, count)
    cols = rng.integers(0, N, count)
    # always include the corners and the last rows/columns (tails)
    rows = np.concatenate([rows, [0, M - 1, 0, M - 1]])
    cols = np.concatenate([cols, [0, 0, N - 1, N - 1]])
    return rows, cols


def log(msg):
    print(msg, flush=True)


def stored_digest(case):
    """The oracle-written full-output digest of a case of tests/golden/config_digests.json."""
    import json
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "config_digests.json")
    return json.load(open(path))["cases"][case]


def assert_full_output(got, x, w, case):
    """Every output of `got` against the stored oracle digest of `case`; on a mismatch the
    oracle output is recomputed to name the first differing element."""
    import hashlib
    from tests.golden import make_config_digests as mk
    c = stored_digest(case)
    assert got.shape == (c["M"], c["N"]), (got.shape, case)
    d = hashlib.sha256(np.ascontiguousarray(got, dtype=np.float32).tobytes()).hexdigest()[:16]
    if d != c["sha256_16"]:
        want = mk.oracle_output(dict(c, name=case), x, w)
        assert_bitwise(got, want, f"{case} full output")
        raise AssertionError(f"{case}: digest {d} != stored {c['sha256_16']} but the outputs match the oracle")

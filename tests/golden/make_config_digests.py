"""Writes config_digests.json beside this file: full-output digests of the batched and large workloads.

For every case below it records the first 16 hex digits of the SHA-256 of the oracle's output
bytes (float32 [M][N], row-major) on the seeded synthetic inputs the GPU tests use: seed 0,
x ~ N(0, 1) float32 (an M-row batch is the first M rows of the 64-row one), W ~ N(0, std)
rounded to bfloat16, input stream = the layer id below.

  batched 8B layers (QKV 6144x4096, O 4096x4096, gate+up 28672x4096, down 4096x14336) at
    M = 4, 16, 64, std 0.02, layer ids 0..3;
  LM head 128256x4096 at M = 1 and 16, std 0.02, layer id 7;
  70B layers (gate+up 57344x8192, down 8192x28672) at M = 1 and 2048, std 0.01, layer id 9.

Outputs up to 2e10 multiply-adds come from the definitional oracle (oracle.linear); larger ones
from the same-order vectorised oracle (oracle.linear_fast), which the CPU tests pin bit for bit
against it.  Calls only the oracle and the input generator:
    python tests/golden/make_config_digests.py
"""
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import synth  # noqa: E402

L8B = [("qkv", 6144, 4096), ("o", 4096, 4096), ("gate_up", 28672, 4096), ("down", 4096, 14336)]
CASES = ([dict(name=f"{n}_m{M}", M=M, N=N, K=K, std=0.02, layer=li, xrows=64)
          for M in (4, 16, 64) for li, (n, N, K) in enumerate(L8B)]
         + [dict(name=f"lm_head_m{M}", M=M, N=128256, K=4096, std=0.02, layer=7, xrows=16) for M in (1, 16)]
         + [dict(name=f"70b_{n}_m{M}", M=M, N=N, K=K, std=0.01, layer=9, xrows=M)
            for n, N, K in (("gate_up", 57344, 8192), ("down", 8192, 28672)) for M in (1, 2048)])
DEFINITIONAL_MAX_FMAS = 2e10


def digest(y):
    return hashlib.sha256(np.ascontiguousarray(y, dtype=np.float32).tobytes()).hexdigest()[:16]


def inputs(c):
    """The case's (x, w): x is the first M rows of an xrows-row seeded batch."""
    x, w = synth.layer_inputs(c["xrows"], c["N"], c["K"], seed=0, w_std=c["std"], layer=c["layer"])
    return np.ascontiguousarray(x[:c["M"]]), w


def oracle_output(c, x, w):
    if c["M"] * c["N"] * c["K"] <= DEFINITIONAL_MAX_FMAS:
        return oracle.linear(x, w)
    return oracle.linear_fast(x, w)


def case_digest(c):
    x, w = inputs(c)
    return digest(oracle_output(c, x, w))


if __name__ == "__main__":
    doc = {"what": "SHA-256 (first 16 hex digits) of y = x * up(W)^T in RG-ORDER-1 over the full output, "
                   "seed 0, x ~ N(0, 1) float32 (first M rows of an xrows-row batch), W ~ N(0, std) bfloat16, "
                   "input stream = layer",
           "cases": {}}
    for c in CASES:
        d = case_digest(c)
        doc["cases"][c["name"]] = dict({k: c[k] for k in ("M", "N", "K", "std", "layer", "xrows")}, sha256_16=d)
        print(c["name"], d, flush=True)
    with open(os.path.join(HERE, "config_digests.json"), "w") as f:
        json.dump(doc, f, indent=1)
        f.write("\n")

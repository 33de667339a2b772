"""Writes m1_step_digests.json beside this file.

For each layer of the M = 1 Llama-3-8B-shaped decode step (QKV 6144x4096, O 4096x4096,
gate+up 28672x4096, down 4096x14336) it records the first 16 hex digits of the SHA-256 of the
oracle's output bytes (float32, row-major) on the seeded synthetic inputs of that step: seed 0,
input stream = the layer's index, x ~ N(0, 1) in float32 and W ~ N(0, 0.02) rounded to bfloat16.
Any implementation that follows the documented order produces these digests on any device.
It also records the digest of the fixed-order decode attention (RG-ATTN-1) on a
Llama-3-8B-shaped batch: 16 sequences, 32 query heads, 8 kv heads, head dim 128,
Lmax 4096, lengths 4096 - 241 b for sequence b, seed 0, scale = float32(1 / sqrt(128)).

Calls only the oracle and the input generator:  python tests/golden/make_step_digests.py
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

LAYERS = [("qkv", 6144, 4096), ("o", 4096, 4096), ("gate_up", 28672, 4096), ("down", 4096, 14336)]


def digest(y):
    return hashlib.sha256(np.ascontiguousarray(y, dtype=np.float32).tobytes()).hexdigest()[:16]


ATTN = {"B": 16, "H": 32, "Hkv": 8, "Lmax": 4096, "D": 128, "seed": 0}


def attn_case():
    a = ATTN
    q, kc, vc = synth.attn_inputs(a["B"], a["H"], a["Hkv"], a["Lmax"], a["D"], seed=a["seed"])
    lens = np.array([a["Lmax"] - 241 * b for b in range(a["B"])], np.int32)
    scale = np.float32(1.0 / np.sqrt(a["D"]))
    return q, kc, vc, lens, scale


def attn_digest():
    q, kc, vc, lens, scale = attn_case()
    return dict(ATTN, lens="Lmax - 241 b", sha256_16=digest(oracle.attn_decode(q, kc, vc, lens, scale)))


def step_digests():
    out = {}
    for li, (name, N, K) in enumerate(LAYERS):
        x, w = synth.layer_inputs(1, N, K, seed=0, w_std=0.02, layer=li)
        out[name] = {"N": N, "K": K, "layer": li, "sha256_16": digest(oracle.linear(x, w))}
    return out


if __name__ == "__main__":
    doc = {"what": "SHA-256 (first 16 hex digits) of y = x * up(W)^T in RG-ORDER-1, M = 1, seed 0, "
                   "x ~ N(0, 1) float32, W ~ N(0, 0.02) bfloat16, input stream = layer index",
           "layers": step_digests(),
           "attention": attn_digest()}
    with open(os.path.join(HERE, "m1_step_digests.json"), "w") as f:
        json.dump(doc, f, indent=1)
        f.write("\n")
    print(json.dumps(doc["layers"]), json.dumps(doc["attention"]))

"""Benchmark of the fused-upcast, fixed-order linear layer on one MI355X.

One step = the four decode-time linear layers of a Llama-3-8B-shaped decoder
block at batch M = 1 (QKV 6144x4096, O 4096x4096, gate+up 28672x4096,
down 4096x14336), each y = x * up(W_bf16)^T through rg_linear.  Inputs are
seeded synthetic data resident in HBM; every layer rotates over enough
distinct weight copies (>= 640 MB per layer) that each call reads its weights
cold from HBM rather than from the 256 MB last-level cache.

value = BF16 weight bytes moved per step / step time (TB/s).  Also printed:
per-layer us/call, the roofline of the dominant kernel (gate+up), the
bit-exactness of the last step against the CPU oracle, the scheme the paper
improves on (cast W to an FP32 temporary, then an FP32 GEMM), and the CPU
oracle's own throughput on a bounded sample.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "µs/call + achieved HBM TB/s (BF16 weight bytes) at M=1; bit-exact vs oracle"
LAYERS = [("qkv", 6144, 4096), ("o", 4096, 4096), ("gate_up", 28672, 4096), ("down", 4096, 14336)]
HBM_PEAK_GBS = 8000.0
ROTATE_BYTES = 640e6


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--per-layer-calls", type=int, default=200)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-baseline-scheme", action="store_true")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: this build has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import synth
    import paper_2609_25624_amd as rg

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    torch.backends.cuda.matmul.allow_tf32 = False
    stream = torch.cuda.current_stream()

    # ---- inputs: seeded on the host, copied once, rotated copies made on the device ----
    layers = []
    for li, (name, N, K) in enumerate(LAYERS):
        x, w = synth.layer_inputs(1, N, K, seed=0, w_std=0.02, layer=li)
        xd = torch.from_numpy(x).to(dev)
        w0 = torch.from_numpy(w.view(np.int16)).to(dev)
        nrot = max(1, int(np.ceil(ROTATE_BYTES / (2.0 * N * K))))
        ws = [w0] + [w0.clone() for _ in range(nrot - 1)]
        y = torch.empty((1, N), dtype=torch.float32, device=dev)
        plan = rg.rg_plan(1, N, K)
        layers.append(dict(name=name, N=N, K=K, x=x, w=w, xd=xd, ws=ws, y=y, plan=plan,
                           wbytes=2.0 * N * K, algo_bytes=2.0 * N * K + 4.0 * K + 4.0 * N))
    torch.cuda.synchronize()
    step_wbytes = sum(L["wbytes"] for L in layers)

    def step(i):
        for L in layers:
            rg.rg_linear(L["xd"], L["ws"][i % len(L["ws"])], L["y"], stream=stream)

    # ---- warmup, then exactly K timed steps ----
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for i in range(args.steps):
        step(i)
    t1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t0.elapsed_time(t1) / args.steps
    value_tbs = step_wbytes / (ms_per_step * 1e-3) / 1e12

    # ---- per-layer us/call (same rotation, same stream) ----
    per_layer = {}
    for L in layers:
        R = args.per_layer_calls
        for i in range(10):
            rg.rg_linear(L["xd"], L["ws"][i % len(L["ws"])], L["y"], stream=stream)
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for i in range(R):
            rg.rg_linear(L["xd"], L["ws"][i % len(L["ws"])], L["y"], stream=stream)
        b.record(stream)
        torch.cuda.synchronize()
        us = a.elapsed_time(b) * 1e3 / R
        per_layer[L["name"]] = dict(
            N=L["N"], K=L["K"], us_per_call=round(us, 3),
            weight_TBs=round(L["wbytes"] / (us * 1e-6) / 1e12, 4),
            frac_of_8TBs=round(L["wbytes"] / (us * 1e-6) / (HBM_PEAK_GBS * 1e9), 4),
            kernel=L["plan"]["kernel_name"], waves_per_wg=L["plan"]["waves_per_wg"],
            grid_wgs=L["plan"]["grid_wgs"], rotated_copies=len(L["ws"]))

    # ---- bit-exactness of the last outputs against the CPU oracle ----
    import oracle
    exact = {}
    for L in layers:
        rg.rg_linear(L["xd"], L["ws"][0], L["y"], stream=stream)
    torch.cuda.synchronize()
    for L in layers:
        want = oracle.linear(L["x"], L["w"])
        got = L["y"].cpu().numpy()
        exact[L["name"]] = bool(np.array_equal(got.view(np.uint32), want.view(np.uint32)))

    # ---- roofline of the dominant kernel: the gate+up launch ----
    dom = next(L for L in layers if L["name"] == "gate_up")
    dom_us = per_layer["gate_up"]["us_per_call"]
    achieved = dom["algo_bytes"] / (dom_us * 1e-6) / 1e9
    traffic = None
    tfile = os.path.join(ROOT, "profiles", "decode_gate_up_m1_traffic.json")
    if os.path.exists(tfile):
        try:
            t = json.load(open(tfile))
            if t.get("kernel_source_hash") == _kernel_hash():
                traffic = t.get("bytes_per_launch")
        except Exception:
            traffic = None
    roofline = dict(bound="hbm", achieved=round(achieved, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=round(achieved / HBM_PEAK_GBS, 4), traffic=traffic,
                    kernel=f"decode (gate+up 28672x4096, M=1, {dom['plan']['waves_per_wg']} waves/WG)",
                    algorithmic_bytes_per_launch=int(dom["algo_bytes"]))

    # ---- the scheme the paper improves on: cast to an FP32 temporary, then FP32 GEMM ----
    scheme = None
    if not args.no_baseline_scheme:
        tmp = {L["name"]: torch.empty((L["N"], L["K"]), dtype=torch.float32, device=dev) for L in layers}

        def scheme_step(i):
            for L in layers:
                wt = tmp[L["name"]]
                rg.rg_cast_bf16_f32(L["ws"][i % len(L["ws"])], wt, stream=stream)
                torch.matmul(L["xd"], wt.t(), out=L["y"])

        R = max(20, args.steps // 3)
        for i in range(5):
            scheme_step(i)
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for i in range(R):
            scheme_step(i)
        b.record(stream)
        torch.cuda.synchronize()
        sms = a.elapsed_time(b) / R
        scheme = dict(ms_per_step=round(sms, 4), speedup_of_fused=round(sms / ms_per_step, 3),
                      transient_fp32_bytes=int(max(4 * L["N"] * L["K"] for L in layers)),
                      gemm="torch.matmul float32 (vendor BLAS)")
        del tmp

    # ---- CPU oracle on the host: bounded sample of the same step ----
    cpu = None
    if not args.no_cpu:
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        t_start = time.perf_counter()
        reps = 0
        while True:
            for L in layers:
                oracle.linear(L["x"], L["w"], nthreads=threads)
            reps += 1
            el = time.perf_counter() - t_start
            if el >= args.cpu_seconds or reps >= 200:
                break
        cpu = dict(value=round(reps * step_wbytes / el / 1e12, 6), unit="TB/s", cores=threads, kind="oracle",
                   sample=f"{reps} full steps (4 layers, M=1) in {el:.1f} s")

    out = {
        "metric": METRIC,
        "value": round(value_tbs, 4),
        "unit": "TB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "llama3-8b-decode-linears-m1", "M": 1, "weight_dtype": "bf16",
                   "layers": {n: [N, K] for n, N, K in LAYERS}, "cold_weights": True},
        "bitexact_vs_oracle": all(exact.values()),
        "bitexact_layers": exact,
        "layers": per_layer,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "baseline_scheme": scheme,
    }
    print(json.dumps(out), flush=True)


def _kernel_hash():
    import hashlib
    h = hashlib.sha256()
    for f in ("rg_kernels.hip", "rg_kernels.h"):
        h.update(open(os.path.join(ROOT, "paper_2609_25624_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


if __name__ == "__main__":
    main()

#!/usr/bin/env python3
"""Benchmark of the sparse forward/backward path on one MI355X.

Default workload (one "step"): forward and backward of the transformer-FFN
shaped sparse pair -- W1 768->3072 and W2 3072->768, each 95% unstructured
sparse, 8192 tokens -- chained X -> W1 -> W2, then backward through W2 and W1
(input gradient and weight gradient of each).  Six sparse ops per step.

Metric: effective GFLOP/s = sum over ops of 2 * nnz * tokens, divided by the
step time.  Inputs live in HBM before the timed region; the mask structure
(plan) is prepared once outside it, as the method prescribes (masks change
rarely), and its preparation time is reported separately.

Prints ONE JSON line.  Extra fields: `roofline` (dominant kernel: algorithmic
bytes / FLOPs per launch over its event-timed duration), `cpu_baseline` (the
CPU oracle timed on a bounded token sample on the host), `ops` (per-op times).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "effective GFLOP/s (2·nnz·batch) fwd+bwd per layer at 90–98% sparsity; HBM GB/s"
HBM_PEAK_GBS = 8000.0
# FP32 FMA on the vector ALUs, one FMA per lane per clock (packed FP32 is not
# used): 256 CUs x 4 SIMD x 16 lanes x 2 flop x 2.4 GHz.
VALU_FP32_PEAK_TFLOPS = 256 * 4 * 16 * 2 * 2.4e9 / 1e12


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-tokens", type=int, default=1024,
                    help="token sample for the CPU oracle baseline")
    return ap.parse_args()


def linear_alg_bytes(op, B, in_f, out_f, nnz):
    """Minimum bytes an op must move: dense operands once, values+indices once."""
    if op == "fwd":
        return 4 * B * in_f + 4 * B * out_f + 8 * nnz + 4 * (out_f + 1)
    if op == "bwd_input":
        return 4 * B * out_f + 4 * B * in_f + 8 * nnz + 4 * (in_f + 1)
    return 4 * B * (in_f + out_f) + 8 * nnz + 4 * (out_f + 1)


class Layer:
    def __init__(self, sp, torch, d):
        self.out_f, self.in_f = d["mask"].shape
        dev = "cuda"
        m = torch.from_numpy(d["mask"]).to(dev)
        w = torch.from_numpy(d["W"]).to(dev)
        self.row_ptr = torch.empty(self.out_f + 1, dtype=torch.int32, device=dev)
        sp.sp_linear_encode_rows(self.out_f, self.in_f, m, self.row_ptr)
        self.nnz = int(self.row_ptr[-1].item())
        self.col_idx = torch.empty(self.nnz, dtype=torch.int32, device=dev)
        self.vals = torch.empty(self.nnz, dtype=torch.float32, device=dev)
        sp.sp_linear_encode_fill(self.out_f, self.in_f, m, w, self.row_ptr, self.col_idx, self.vals)
        self.plan = torch.empty(sp.sp_linear_plan_bytes(self.in_f, self.out_f, self.nnz), dtype=torch.uint8,
                                device=dev)
        torch.cuda.synchronize()
        t = time.perf_counter()
        sp.sp_linear_plan(self.in_f, self.out_f, self.row_ptr, self.col_idx, self.nnz, self.plan)
        torch.cuda.synchronize()
        self.plan_ms = (time.perf_counter() - t) * 1e3
        self.dW = torch.empty(self.nnz, dtype=torch.float32, device=dev)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(data-parallel sharding is described in DESIGN.md); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2302_04852_amd as sp
    from synth import linear_layer, FFN_PAIR, seed_for

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)

    layers_np = []
    for li, (name, out_f, in_f, B, s) in enumerate(FFN_PAIR):
        layers_np.append(linear_layer(seed_for(2, li), out_f, in_f, B, s))
    B = FFN_PAIR[0][3]
    L1 = Layer(sp, torch, layers_np[0])
    L2 = Layer(sp, torch, layers_np[1])
    X = torch.from_numpy(layers_np[0]["X"]).cuda()
    dY2 = torch.from_numpy(layers_np[1]["dY"]).cuda()
    Y1 = torch.empty(B, L1.out_f, device="cuda")
    Y2 = torch.empty(B, L2.out_f, device="cuda")
    dX2 = torch.empty(B, L2.in_f, device="cuda")
    dX1 = torch.empty(B, L1.in_f, device="cuda")
    ws_bytes = max(sp.sp_linear_bwd_weight_ws(B, L.in_f, L.out_f, L.nnz) for L in (L1, L2))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")

    ops = [
        ("W1.fwd", lambda: sp.sp_linear_fwd(X, B, L1.in_f, L1.out_f, L1.vals, L1.nnz, L1.plan, Y1), L1, "fwd"),
        ("W2.fwd", lambda: sp.sp_linear_fwd(Y1, B, L2.in_f, L2.out_f, L2.vals, L2.nnz, L2.plan, Y2), L2, "fwd"),
        ("W2.bwd_input", lambda: sp.sp_linear_bwd_input(dY2, B, L2.in_f, L2.out_f, L2.vals, L2.nnz, L2.plan, dX2),
         L2, "bwd_input"),
        ("W2.bwd_weight", lambda: sp.sp_linear_bwd_weight(dY2, Y1, B, L2.in_f, L2.out_f, L2.nnz, L2.plan, L2.dW, ws),
         L2, "bwd_weight"),
        ("W1.bwd_input", lambda: sp.sp_linear_bwd_input(dX2, B, L1.in_f, L1.out_f, L1.vals, L1.nnz, L1.plan, dX1),
         L1, "bwd_input"),
        ("W1.bwd_weight", lambda: sp.sp_linear_bwd_weight(dX2, X, B, L1.in_f, L1.out_f, L1.nnz, L1.plan, L1.dW, ws),
         L1, "bwd_weight"),
    ]
    flops_step = sum(2.0 * L.nnz * B for _, _, L, _ in ops)

    def step():
        for _, f, _, _ in ops:
            f()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # Timed region: K whole steps between two events on the launch stream.
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    total_ms = e0.elapsed_time(e1)
    ms_per_step = total_ms / args.steps

    # Per-op durations: events around each op over the same number of steps.
    per_op = {name: 0.0 for name, _, _, _ in ops}
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in ops]
    for _ in range(args.steps):
        for (name, f, _, _), (a, b) in zip(ops, evs):
            a.record(stream)
            f()
            b.record(stream)
        torch.cuda.synchronize()
        for (name, _, _, _), (a, b) in zip(ops, evs):
            per_op[name] += a.elapsed_time(b)
    op_rows = {}
    for name, _, L, kind in ops:
        ms = per_op[name] / args.steps
        fl = 2.0 * L.nnz * B
        by = linear_alg_bytes(kind, B, L.in_f, L.out_f, L.nnz)
        op_rows[name] = {"ms": round(ms, 5), "tflops": round(fl / ms / 1e9, 3),
                         "alg_GBps": round(by / ms / 1e6, 1), "hbm_frac": round(by / ms / 1e6 / HBM_PEAK_GBS, 4)}

    # Dominant kernel: the SpMM kernel serves fwd and bwd_input (4 launches
    # of equal algorithmic work per step); the SDDMM kernel serves bwd_weight.
    spmm_ms = np.mean([per_op[n] / args.steps for n, _, _, k in ops if k in ("fwd", "bwd_input")])
    sddmm_ms = np.mean([per_op[n] / args.steps for n, _, _, k in ops if k == "bwd_weight"])
    if sddmm_ms >= spmm_ms:
        dom, dom_ms, kind = "k_sddmm (+reduce)", sddmm_ms, "bwd_weight"
    else:
        dom, dom_ms, kind = "k_spmm", spmm_ms, "fwd"
    fl = 2.0 * L1.nnz * B
    by = linear_alg_bytes(kind, B, L1.in_f, L1.out_f, L1.nnz)
    achieved_tf = fl / (dom_ms * 1e-3) / 1e12
    roof = {"kernel": dom, "bound": "alu", "achieved": round(achieved_tf, 3), "peak": round(VALU_FP32_PEAK_TFLOPS, 1),
            "unit": "TFLOP/s", "frac": round(achieved_tf / VALU_FP32_PEAK_TFLOPS, 4), "traffic": None,
            "alg_bytes_per_launch": by, "flops_per_launch": fl, "ms_per_launch": round(float(dom_ms), 5),
            "hbm_achieved_GBps": round(by / (dom_ms * 1e-3) / 1e9, 1), "hbm_peak_GBps": HBM_PEAK_GBS,
            "hbm_frac": round(by / (dom_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}

    step_bytes = sum(linear_alg_bytes(k, B, L.in_f, L.out_f, L.nnz) for _, _, L, k in ops)
    out = {
        "metric": METRIC,
        "value": round(flops_step / (ms_per_step * 1e-3) / 1e9, 1),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "FFN pair W1 768->3072 + W2 3072->768, 95% unstructured sparse, 8192 tokens, "
                               "fwd+bwd (input and weight gradient) of both layers",
                   "tokens": B, "sparsity": 0.95, "nnz_per_layer": L1.nnz},
        "hbm": {"alg_GB_per_step": round(step_bytes / 1e9, 4),
                "achieved_GBps": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
                "frac_of_8TBps": round(step_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
        "roofline": roof,
        "ops": op_rows,
        "plan_ms": {"W1": round(L1.plan_ms, 3), "W2": round(L2.plan_ms, 3)},
    }

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(layers_np, args.cpu_tokens)
    print(json.dumps(out), flush=True)


def cpu_baseline(layers_np, ntok):
    """The CPU oracle (as it stands) on the same step, restricted to the first
    `ntok` tokens; reported in the same effective-GFLOP/s unit."""
    import oracle
    t_total = 0.0
    flops = 0.0
    X = layers_np[0]["X"][:ntok]
    dY2 = layers_np[1]["dY"][:ntok]
    enc = [oracle.linear_encode(d["mask"], d["W"]) for d in layers_np]
    t = time.perf_counter()
    (rp1, ci1, v1), (rp2, ci2, v2) = enc
    o1, i1 = layers_np[0]["mask"].shape
    o2, i2 = layers_np[1]["mask"].shape
    Y1, _ = oracle.linear_fwd(X, rp1, ci1, v1, o1)
    Y1f = Y1.astype(np.float32)
    oracle.linear_fwd(Y1f, rp2, ci2, v2, o2)
    dX2, _ = oracle.linear_bwd_input(dY2, rp2, ci2, v2, i2)
    oracle.linear_bwd_weight(dY2, Y1f, rp2, ci2)
    dX2f = dX2.astype(np.float32)
    oracle.linear_bwd_input(dX2f, rp1, ci1, v1, i1)
    oracle.linear_bwd_weight(dX2f, X, rp1, ci1)
    t_total = time.perf_counter() - t
    flops = 3 * 2.0 * (len(v1) + len(v2)) * ntok
    cpu_model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": round(flops / t_total / 1e9, 3), "unit": "GFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle", "seconds": round(t_total, 2), "cpu": cpu_model,
            "sample": "same six-op FFN step on the first %d of 8192 tokens (fp64-accumulating plain loops, "
                      "OpenMP over independent outputs)" % ntok}


if __name__ == "__main__":
    main()

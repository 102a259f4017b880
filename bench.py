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
CPU oracle timed on the host over whole repeated steps, about 10 s), `ops` (per-op times).
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
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum CPU time of the oracle baseline (whole steps are repeated)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run only a plain device-to-device copy of COPY_BYTES (counter calibration)")
    return ap.parse_args()


COPY_BYTES = 1 << 30
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_spmm2_k_sddmm2_ffn_pair_hbm_traffic.txt")
KERNEL_SOURCES = ["sp_common.h", "sp_common.hip", "sp_spmm2.h", "sp_slots.hip", "sp_linear.hip"]


def kernel_source_hash():
    """sha256 over the sources of the kernels the bench launches."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2302_04852_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary, or
    None when it is absent or was taken on different kernel sources."""
    try:
        lines = open(TRAFFIC_FILE).read().splitlines()
    except OSError:
        return None
    for line in lines:
        if line.startswith("TRAFFIC "):
            rec = json.loads(line[len("TRAFFIC "):])
            if rec.get("source_hash") == kernel_source_hash() and kernel in rec.get("bytes_per_launch", {}):
                return rec["bytes_per_launch"][kernel]
    return None


def calibrate_copy():
    """A plain copy of COPY_BYTES, 5 times: under rocprofv3 --pmc its
    FETCH_SIZE / WRITE_SIZE per dispatch give the counters' scale."""
    import torch
    a = torch.ones(COPY_BYTES // 4, device="cuda")
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": COPY_BYTES, "copy_bytes_written": COPY_BYTES, "launches": 5}), flush=True)


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
        print("bench.py measures one GPU only (the library has no multi-GPU path); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.calibrate_copy:
        calibrate_copy()
        return

    import paper_2302_04852_amd as sp
    from synth import linear_layer, FFN_PAIR, seed_for

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

    # Timed region: K whole steps between two events on the launch stream,
    # with an event pair around every op inside it (per-op durations).
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in ops]
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    e0.record(stream)
    for k in range(args.steps):
        for (name, f, _, _), (a, b) in zip(ops, evs[k]):
            a.record(stream)
            f()
            b.record(stream)
    e1.record(stream)
    torch.cuda.synchronize()
    total_ms = e0.elapsed_time(e1)
    ms_per_step = total_ms / args.steps
    per_op = {name: 0.0 for name, _, _, _ in ops}
    for k in range(args.steps):
        for (name, _, _, _), (a, b) in zip(ops, evs[k]):
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
    if 2 * sddmm_ms >= 4 * spmm_ms:
        dom, dom_ms, kind = "k_sddmm2+k_slot_reduce", sddmm_ms, "bwd_weight"
    else:
        dom, dom_ms, kind = "k_spmm2", spmm_ms, "fwd"
    fl = 2.0 * L1.nnz * B
    by = linear_alg_bytes(kind, B, L1.in_f, L1.out_f, L1.nnz)
    achieved_tf = fl / (dom_ms * 1e-3) / 1e12
    traffic = measured_traffic(dom)
    roof = {"kernel": dom, "bound": "alu", "achieved": round(achieved_tf, 3), "peak": round(VALU_FP32_PEAK_TFLOPS, 1),
            "unit": "TFLOP/s", "frac": round(achieved_tf / VALU_FP32_PEAK_TFLOPS, 4), "traffic": traffic,
            "source_hash": kernel_source_hash(),
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
        out["cpu_baseline"] = cpu_baseline(layers_np, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def cpu_baseline(layers_np, min_seconds):
    """The CPU oracle (as it stands) on the same six-op step over all tokens,
    repeated until at least `min_seconds` have passed; reported in the same
    effective-GFLOP/s unit."""
    import oracle
    X = layers_np[0]["X"]
    dY2 = layers_np[1]["dY"]
    ntok = X.shape[0]
    (rp1, ci1, v1), (rp2, ci2, v2) = [oracle.linear_encode(d["mask"], d["W"]) for d in layers_np]
    o1, i1 = layers_np[0]["mask"].shape
    o2, i2 = layers_np[1]["mask"].shape
    reps = 0
    t = time.perf_counter()
    while True:
        Y1, _ = oracle.linear_fwd(X, rp1, ci1, v1, o1)
        Y1f = Y1.astype(np.float32)
        oracle.linear_fwd(Y1f, rp2, ci2, v2, o2)
        dX2, _ = oracle.linear_bwd_input(dY2, rp2, ci2, v2, i2)
        oracle.linear_bwd_weight(dY2, Y1f, rp2, ci2)
        dX2f = dX2.astype(np.float32)
        oracle.linear_bwd_input(dX2f, rp1, ci1, v1, i1)
        oracle.linear_bwd_weight(dX2f, X, rp1, ci1)
        reps += 1
        t_total = time.perf_counter() - t
        if t_total >= min_seconds:
            break
    flops = reps * 3 * 2.0 * (len(v1) + len(v2)) * ntok
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
            "sample": "the same six-op FFN step over all %d tokens, repeated %d times (fp64-accumulating "
                      "plain loops, OpenMP over independent outputs; conversions between ops included)"
                      % (ntok, reps)}


if __name__ == "__main__":
    main()

#!/usr/bin/env python3
"""Benchmark of the sparse forward/backward path on one MI355X.

Default workload (one "step"): forward and backward of the transformer-FFN
shaped sparse pair -- W1 768->3072 and W2 3072->768, each 95% unstructured
sparse, 8192 tokens -- chained X -> W1 -> W2, then backward through W2 and W1
(input gradient and weight gradient of each).  Six sparse ops per step.

Other workloads (``--workload``), each timed the same way:
  linear_small  a 256x256 linear layer at 90%, 16 tokens (latency-bound);
  conv3x3_56    a 3x3 64->64 convolution on 32x64x56x56 at 90%;
  conv_sweep    3x3 128@28x28, 3x3 256@14x14 and 1x1 256->1024@14x14 at batch 32,
                each at 80/90/95/98%;
  resnet18      the 20 convolutions and the FC layer of a ResNet-18 at batch 64,
                224x224, 95% (sparse passes only; activations drawn per layer).
A step is the forward, input gradient and weight gradient of every layer; the
two gradients of a layer come from one sp_linear_bwd / sp_conv_bwd call.

Metric: effective GFLOP/s = sum over ops of 2 * nnz * tokens (linear) or
2 * nnz * B * OH * OW (conv), divided by the step time.  Inputs live in HBM
before the timed region; the mask structure (plan) is prepared once outside
it, as the method prescribes (masks change rarely), and its preparation time
is reported separately.

Timing: W untimed steps; then K steps with an event pair around every op for
the per-op times and the roofline (event records between ops add gaps of
their own; that pass's step time is reported as `ms_per_step_with_op_events`);
then K steps between two HIP events with nothing recorded in between: the
step time and `value`.

Prints ONE JSON line.  Extra fields: `roofline` (dominant kernel: algorithmic
bytes / FLOPs per launch over its event-timed duration), `cpu_baseline` (the
CPU oracle timed on the host over a bounded sample, about 10 s), `ops`
(per-op times, warm caches: consecutive steps), `cold` (per-op medians with
the caches evicted before every launch, and the achievable HBM rate of a
1 GiB copy).
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
# FP32 on the matrix cores (v_mfma_f32_32x32x2_f32), MI355X's published dense peak.
MFMA_FP32_PEAK_TFLOPS = 157.3
WORKLOADS = ("ffn", "linear_small", "conv3x3_56", "conv_sweep", "resnet18")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", choices=WORKLOADS, default="ffn")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--variant", choices=("auto", "sparse", "dense"), default="auto",
                    help="auto = the paper's choice per layer (dense below 80%% sparsity, else the faster of "
                         "one timed step each); sparse/dense force one variant for every layer")
    ap.add_argument("--sparsity", type=float, default=None,
                    help="linear workloads: override the layers' sparsity (default: the workload's own)")
    ap.add_argument("--cold-reps", type=int, default=10,
                    help="launches per op for the cold-cache per-op medians (0: skip)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum CPU time of the oracle baseline (whole sample passes are repeated)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run only a plain device-to-device copy of COPY_BYTES (counter calibration)")
    return ap.parse_args()


COPY_BYTES = 1 << 30
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_spmm2_k_bwd_fused_ffn_pair_hbm_traffic.txt")
FLUSH_BYTES = 1 << 30
KERNEL_SOURCES = ["sp_common.h", "sp_common.hip", "sp_spmm2.h", "sp_slots.hip", "sp_linear.hip"]
# The 3x3 64@56 convolution's counters (its backward dominates its step).
CONV_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_conv_bwd_fused_conv3x3_56_hbm_traffic.txt")
CONV_KERNEL_SOURCES = ["sp_common.h", "sp_common.hip", "sp_spmm2.h", "sp_slots.hip", "sp_conv.hip"]


def kernel_source_hash(sources=None):
    """sha256 over the sources of the kernels a workload launches (default:
    the FFN bench's)."""
    import hashlib
    h = hashlib.sha256()
    for f in (KERNEL_SOURCES if sources is None else sources):
        with open(os.path.join(ROOT, "paper_2302_04852_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, path=None, sources=None):
    """HBM bytes per launch of `kernel` from a committed counter summary, or
    None when it is absent or was taken on different kernel sources."""
    try:
        lines = open(TRAFFIC_FILE if path is None else path).read().splitlines()
    except OSError:
        return None
    for line in lines:
        if line.startswith("TRAFFIC "):
            rec = json.loads(line[len("TRAFFIC "):])
            if rec.get("source_hash") == kernel_source_hash(sources) and kernel in rec.get("bytes_per_launch", {}):
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


# ------------------------------------------------------------ algorithmic cost

def linear_alg_bytes(op, B, in_f, out_f, nnz):
    """Minimum bytes an op must move: dense operands once, values+indices once.
    "bwd" is both gradients in one pass: dY, X and dX once, values, indices
    and dW once."""
    if op == "fwd":
        return 4 * B * in_f + 4 * B * out_f + 8 * nnz + 4 * (out_f + 1)
    if op == "bwd_input":
        return 4 * B * out_f + 4 * B * in_f + 8 * nnz + 4 * (in_f + 1)
    if op == "bwd":
        return 4 * B * out_f + 8 * B * in_f + 12 * nnz + 4 * (in_f + 1) + 4 * (out_f + 1)
    return 4 * B * (in_f + out_f) + 8 * nnz + 4 * (out_f + 1)


def conv_alg_bytes(B, IC, H, W, OC, OH, OW, nnz):
    """Activations once, then per stored entry a 4-byte value (forward, input
    gradient) or a 4-byte gradient (weight gradient) plus its two 1-byte
    taps, and the two index arrays of the format.  The same for all three
    passes."""
    return 4 * B * IC * H * W + 4 * B * OC * OH * OW + 6 * nnz + 2 * OC * (IC + 1) + 4 * (OC + 1)


def conv_bwd_alg_bytes(B, IC, H, W, OC, OH, OW, nnz):
    """Both gradients in one pass: X read and dX written, dY read once; per
    stored entry its value read, its gradient written and its two taps; the
    two index arrays."""
    return 8 * B * IC * H * W + 4 * B * OC * OH * OW + 10 * nnz + 2 * OC * (IC + 1) + 4 * (OC + 1)


def bound_of(flops, nbytes):
    """Roofline bound of an op: HBM when its arithmetic intensity is below the
    ridge point (peak FLOP/s over peak B/s), else the FP32 ALU."""
    return "hbm" if flops / nbytes * HBM_PEAK_GBS * 1e9 < VALU_FP32_PEAK_TFLOPS * 1e12 else "alu"


# --------------------------------------------------------------------- layers

def select_flags(sp, sparsity):
    """The paper applies its 80% rule to a layer's pruning target.  A mask
    pruned to 80% holds round(0.2 * numel) entries, which the rounding can put
    a fraction of an entry above 20% density, i.e. below 80% sparsity by the
    library's count.  Layers pruned to 80% or more are therefore always timed;
    below that the library's rule (dense, untimed) applies."""
    return sp.SP_SELECT_ALWAYS_TIME if sparsity >= 0.8 else 0


class LinearLayer:
    def __init__(self, sp, torch, d, name):
        self.name = name
        self.out_f, self.in_f = d["mask"].shape
        dev = "cuda"
        m = torch.from_numpy(d["mask"]).to(dev)
        w = torch.from_numpy(d["W"]).to(dev)
        self.row_ptr = torch.empty(self.out_f + 1, dtype=torch.int32, device=dev)
        sp.sp_linear_encode_rows(self.out_f, self.in_f, m, self.row_ptr)
        self.nnz = int(self.row_ptr[-1].item())
        self.col_idx = torch.empty(max(self.nnz, 1), dtype=torch.int32, device=dev)
        self.vals = torch.empty(max(self.nnz, 1), dtype=torch.float32, device=dev)
        sp.sp_linear_encode_fill(self.out_f, self.in_f, m, w, self.row_ptr, self.col_idx, self.vals)
        self.plan = torch.empty(sp.sp_linear_plan_bytes(self.in_f, self.out_f, self.nnz), dtype=torch.uint8,
                                device=dev)
        torch.cuda.synchronize()
        t = time.perf_counter()
        sp.sp_linear_plan(self.in_f, self.out_f, self.row_ptr, self.col_idx, self.nnz, self.plan)
        torch.cuda.synchronize()
        self.plan_ms = (time.perf_counter() - t) * 1e3
        self.dW = torch.empty(max(self.nnz, 1), dtype=torch.float32, device=dev)


class ConvLayer:
    def __init__(self, sp, torch, spec, seed):
        from synth import conv_layer
        name, B, IC, H, W, OC, KH, KW, s, p, sparsity = spec
        self.name = name
        self.sparsity = sparsity
        self.dims = (B, IC, H, W, OC, KH, KW)
        self.shape = sp.conv_shape(B, IC, H, W, OC, KH, KW, (s, s), (p, p))
        self.OH, self.OW = sp.sp_conv_out_hw(self.shape)
        d = conv_layer(seed, B, IC, H, W, OC, KH, KW, (self.OH, self.OW), sparsity)
        dev = "cuda"
        m = torch.from_numpy(d["mask"]).to(dev)
        w = torch.from_numpy(d["W"]).to(dev)
        self.w_oc = torch.empty(OC + 1, dtype=torch.int32, device=dev)
        self.w_ic = torch.empty(OC * (IC + 1), dtype=torch.int16, device=dev)
        sp.sp_conv_encode_rows(OC, IC, KH, KW, m, self.w_oc, self.w_ic)
        self.nnz = int(self.w_oc[-1].item())
        n1 = max(self.nnz, 1)
        self.w_x = torch.empty(n1, dtype=torch.uint8, device=dev)
        self.w_y = torch.empty(n1, dtype=torch.uint8, device=dev)
        self.w_vals = torch.empty(n1, dtype=torch.float32, device=dev)
        sp.sp_conv_encode_fill(OC, IC, KH, KW, m, w, self.w_oc, self.w_ic, self.w_x, self.w_y, self.w_vals)
        self.plan = torch.empty(sp.sp_conv_plan_bytes(self.shape, self.nnz), dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()
        t = time.perf_counter()
        sp.sp_conv_plan(self.shape, self.w_oc, self.w_ic, self.w_x, self.w_y, self.nnz, self.plan)
        torch.cuda.synchronize()
        self.plan_ms = (time.perf_counter() - t) * 1e3
        self.X = torch.from_numpy(d["X"]).to(dev)
        self.dY = torch.from_numpy(d["dY"]).to(dev)
        self.Y = torch.empty(B, OC, self.OH, self.OW, device=dev)
        self.dX = torch.empty(B, IC, H, W, device=dev)
        self.dW = torch.empty(n1, device=dev)
        self.ws = torch.empty(max(sp.sp_conv_bwd_weight_ws(self.shape, self.nnz), 1), dtype=torch.uint8,
                              device=dev)
        self.mask_np, self.W_np = d["mask"], d["W"]

    def select(self, sp, torch, mode):
        """The paper's per-layer choice (sp_conv_select), or a forced variant."""
        if mode != "auto":
            self.variant = sp.SP_VARIANT_DENSE if mode == "dense" else sp.SP_VARIANT_SPARSE
            self.choice = {"variant": mode, "forced": True}
        else:
            ws = torch.empty(max(sp.sp_conv_select_ws(self.shape, self.nnz), 1), dtype=torch.uint8, device="cuda")
            v, ms = sp.sp_conv_select(self.X, self.dY, self.shape, self.w_oc, self.w_ic, self.w_x, self.w_y,
                                      self.w_vals, self.nnz, self.plan, self.Y, self.dX, self.dW, ws, 3,
                                      select_flags(sp, self.sparsity))
            del ws
            self.variant = v
            self.choice = {"variant": "dense" if v == sp.SP_VARIANT_DENSE else "sparse",
                           "ms_sparse_step": round(ms[0], 4), "ms_dense_step": round(ms[1], 4)}
        if self.variant == sp.SP_VARIANT_DENSE:
            B, IC, H, W, OC, KH, KW = self.dims
            self.Wd = torch.empty(OC, IC, KH, KW, device="cuda")
            self.dws = torch.empty(max(sp.sp_conv_dense_ws(self.shape), 1), dtype=torch.uint8, device="cuda")

    def ops(self, sp):
        B, IC, H, W, OC, KH, KW = self.dims
        fl = 2.0 * self.nnz * B * self.OH * self.OW
        by = conv_alg_bytes(B, IC, H, W, OC, self.OH, self.OW, self.nnz)
        by_b = conv_bwd_alg_bytes(B, IC, H, W, OC, self.OH, self.OW, self.nnz)
        if self.variant == sp.SP_VARIANT_DENSE:
            def fwd():
                sp.sp_conv_densify(self.shape, self.w_oc, self.w_ic, self.w_x, self.w_y, self.w_vals, self.nnz,
                                   self.Wd)
                sp.sp_conv_dense_fwd(self.X, self.shape, self.Wd, self.Y, self.dws)

            def bwd():
                sp.sp_conv_dense_bwd_input(self.dY, self.shape, self.Wd, self.dX, self.dws)
                sp.sp_conv_dense_bwd_weight(self.dY, self.X, self.shape, self.w_oc, self.w_ic, self.w_x, self.w_y,
                                            self.nnz, self.dW, self.dws)
            return [(self.name + ".fwd", fwd, "dense_fwd", fl, by, self),
                    (self.name + ".bwd", bwd, "dense_bwd", 2 * fl, by_b, self)]
        # the backward is one sp_conv_bwd call: input and weight gradient
        return [
            (self.name + ".fwd", lambda: sp.sp_conv_fwd(self.X, self.shape, self.w_vals, self.nnz, self.plan, self.Y),
             "fwd", fl, by, self),
            (self.name + ".bwd",
             lambda: sp.sp_conv_bwd(self.dY, self.X, self.shape, self.w_vals, self.nnz, self.plan, self.dX, self.dW,
                                    self.ws),
             "bwd", 2 * fl, by_b, self),
        ]

    def dense_flops(self):
        B, IC, H, W, OC, KH, KW = self.dims
        return 2.0 * B * self.OH * self.OW * OC * IC * KH * KW


# --------------------------------------------------------------------- timing

def time_ops(torch, ops, steps, warmup):
    """W untimed steps; then K steps with an event pair around every op (the
    per-op times; the event records between the ops add gaps of their own);
    then K steps between two events on the launch stream with nothing
    recorded in between (the step time).  Returns the step time (ms), the
    mean time of every op (ms) and the step time of the instrumented pass
    (ms)."""
    def step():
        for op in ops:
            op[1]()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in ops]
           for _ in range(steps)]
    torch.cuda.synchronize()
    e0.record(stream)
    for k in range(steps):
        for op, (a, b) in zip(ops, evs[k]):
            a.record(stream)
            op[1]()
            b.record(stream)
    e1.record(stream)
    torch.cuda.synchronize()
    per_op = [0.0] * len(ops)
    for k in range(steps):
        for i, (a, b) in enumerate(evs[k]):
            per_op[i] += a.elapsed_time(b)
    ms_instr = e0.elapsed_time(e1) / steps

    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps, [t / steps for t in per_op], ms_instr


def cold_ops(torch, ops, reps):
    """Per-op times with cold caches: before every timed launch a 1 GiB fill
    (more than the L2s and the 256 MB last-level cache together) evicts the
    operands.  Median over `reps` launches of each op."""
    scratch = torch.empty(FLUSH_BYTES // 4, device="cuda")
    stream = torch.cuda.current_stream()
    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
           for _ in ops]
    for op, ev in zip(ops, evs):
        for a, b in ev:
            scratch.fill_(1.0)
            a.record(stream)
            op[1]()
            b.record(stream)
    torch.cuda.synchronize()
    return [float(np.median([a.elapsed_time(b) for a, b in ev])) for ev in evs]


def copy_rate_GBps(torch):
    """Achievable HBM rate: a 1 GiB device-to-device copy (read + write
    counted), best of 5."""
    a = torch.ones(FLUSH_BYTES // 4, device="cuda")
    b = torch.empty_like(a)
    stream = torch.cuda.current_stream()
    best = None
    for _ in range(5):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        b.copy_(a)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    return 2.0 * FLUSH_BYTES / (best * 1e-3) / 1e9


def cold_record(torch, args, ops):
    """Cold-cache per-op medians and the achievable HBM rate, or None."""
    if args.cold_reps <= 0:
        return None
    t = cold_ops(torch, ops, args.cold_reps)
    rate = copy_rate_GBps(torch)
    return {"method": "median of %d launches per op, each after a 1 GiB fill that evicts L2 and the "
                      "last-level cache" % args.cold_reps,
            "hbm_copy_GBps": round(rate, 1),
            "step_ms": round(sum(t), 5),
            "ops": {o[0]: dict(op_row(ms, o[3], o[4]), hbm_frac_of_copy=round(o[4] / (ms * 1e-3) / 1e9 / rate, 4))
                    for o, ms in zip(ops, t)}}


def op_row(ms, fl, by):
    return {"ms": round(ms, 5), "tflops": round(fl / ms / 1e9, 3), "alg_GBps": round(by / ms / 1e6, 1),
            "hbm_frac": round(by / ms / 1e6 / HBM_PEAK_GBS, 4), "bound": bound_of(fl, by)}


def roofline(kernel, kind, fl, by, ms, traffic=None, extra=None, mfma_flops=None):
    """Roofline record of one kernel from its algorithmic flops/bytes per
    launch and its mean event-timed launch duration (ms).  mfma_flops: the
    dense matrix-core flops of a dense-variant launch, priced against the
    fp32 matrix-core peak."""
    bound = "mfma" if mfma_flops else bound_of(fl, by)
    if bound == "mfma":
        achieved, peak, unit = mfma_flops / (ms * 1e-3) / 1e12, MFMA_FP32_PEAK_TFLOPS, "TFLOP/s"
    elif bound == "alu":
        achieved, peak, unit = fl / (ms * 1e-3) / 1e12, VALU_FP32_PEAK_TFLOPS, "TFLOP/s"
    else:
        achieved, peak, unit = by / (ms * 1e-3) / 1e9, HBM_PEAK_GBS, "GB/s"
    r = {"kernel": kernel, "op": kind, "bound": bound, "achieved": round(achieved, 3), "peak": round(peak, 1),
         "unit": unit, "frac": round(achieved / peak, 4), "traffic": traffic,
         "alg_bytes_per_launch": int(by), "flops_per_launch": fl, "ms_per_launch": round(float(ms), 5),
         "hbm_achieved_GBps": round(by / (ms * 1e-3) / 1e9, 1), "hbm_peak_GBps": HBM_PEAK_GBS,
         "hbm_frac": round(by / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
         "tflops": round(fl / (ms * 1e-3) / 1e12, 3), "alu_peak_TFLOPs": round(VALU_FP32_PEAK_TFLOPS, 1)}
    if extra:
        r.update(extra)
    return r


def base_record(args, value, ms_per_step, config):
    return {
        "metric": METRIC, "value": round(value, 1), "unit": "GFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic", "config": config,
    }


def hbm_record(bytes_step, ms_per_step):
    return {"alg_GB_per_step": round(bytes_step / 1e9, 4),
            "achieved_GBps": round(bytes_step / (ms_per_step * 1e-3) / 1e9, 1),
            "frac_of_8TBps": round(bytes_step / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}


# ------------------------------------------------------------------ workloads

def run_linear(args, sp, torch, which):
    from synth import FFN_PAIR, LINEAR_SMALL, linear_layer, seed_for

    spec = FFN_PAIR if which == "ffn" else LINEAR_SMALL
    sparsity = spec[0][4] if args.sparsity is None else args.sparsity
    if which == "ffn":
        layers_np = [linear_layer(seed_for(2, li), o, i, B, sparsity) for li, (_, o, i, B, _) in enumerate(spec)]
    else:
        layers_np = [linear_layer(seed_for(1, 0), o, i, B, sparsity) for (_, o, i, B, _) in spec]
    B = spec[0][3]
    L1 = LinearLayer(sp, torch, layers_np[0], "W1")
    X = torch.from_numpy(layers_np[0]["X"]).cuda()
    Y1 = torch.empty(B, L1.out_f, device="cuda")
    dX1 = torch.empty(B, L1.in_f, device="cuda")
    if which == "ffn":
        L2 = LinearLayer(sp, torch, layers_np[1], "W2")
        dY2 = torch.from_numpy(layers_np[1]["dY"]).cuda()
        Y2 = torch.empty(B, L2.out_f, device="cuda")
        dX2 = torch.empty(B, L2.in_f, device="cuda")
        layers = (L1, L2)
    else:
        dY1 = torch.from_numpy(layers_np[0]["dY"]).cuda()
        layers = (L1,)
    ws_bytes = max(max(sp.sp_linear_bwd_weight_ws(B, L.in_f, L.out_f, L.nnz) for L in layers), 1)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")

    # The paper's end-to-end protocol: a layer below 80% sparsity runs dense;
    # from 80% on one forward+backward step of each variant is timed and the
    # faster is kept (sp_linear_select).  Selection runs once, before the
    # timed region, on the layer's own synthetic inputs.
    choice = {}
    for L, d in zip(layers, layers_np):
        if args.variant != "auto":
            L.variant = sp.SP_VARIANT_DENSE if args.variant == "dense" else sp.SP_VARIANT_SPARSE
            choice[L.name] = {"variant": args.variant, "forced": True}
            if args.variant == "dense":
                L.Wd = torch.empty(L.out_f, L.in_f, device="cuda")
            continue
        xs = torch.from_numpy(d["X"]).cuda()
        dys = torch.from_numpy(d["dY"]).cuda()
        sws = torch.empty(max(sp.sp_linear_select_ws(B, L.in_f, L.out_f, L.nnz), 1), dtype=torch.uint8,
                          device="cuda")
        v, ms = sp.sp_linear_select(xs, dys, B, L.in_f, L.out_f, L.row_ptr, L.col_idx, L.vals, L.nnz, L.plan,
                                    torch.empty(B, L.out_f, device="cuda"), torch.empty(B, L.in_f, device="cuda"),
                                    L.dW, sws, 3, select_flags(sp, sparsity))
        L.variant = v
        choice[L.name] = {"variant": "dense" if v == sp.SP_VARIANT_DENSE else "sparse",
                          "ms_sparse_step": round(ms[0], 4), "ms_dense_step": round(ms[1], 4)}
        del sws
        if v == sp.SP_VARIANT_DENSE:
            L.Wd = torch.empty(L.out_f, L.in_f, device="cuda")
    dws_bytes = max([sp.sp_linear_dense_ws(B, L.in_f, L.out_f) for L in layers
                     if L.variant == sp.SP_VARIANT_DENSE] + [1])
    dws = torch.empty(dws_bytes, dtype=torch.uint8, device="cuda")

    def fwd_op(name, L, x, y):
        if L.variant == sp.SP_VARIANT_DENSE:
            def f():
                sp.sp_linear_densify(L.out_f, L.in_f, L.row_ptr, L.col_idx, L.vals, L.nnz, L.Wd)
                sp.sp_linear_dense_fwd(x, B, L.in_f, L.out_f, L.Wd, y, dws)
            return (name, f, "dense_fwd", 2.0 * L.nnz * B, linear_alg_bytes("fwd", B, L.in_f, L.out_f, L.nnz), L)
        return (name, lambda: sp.sp_linear_fwd(x, B, L.in_f, L.out_f, L.vals, L.nnz, L.plan, y), "fwd",
                2.0 * L.nnz * B, linear_alg_bytes("fwd", B, L.in_f, L.out_f, L.nnz), L)

    # The backward of a sparse layer is one sp_linear_bwd call: the input
    # gradient and the weight gradient in one launch (plus the fixed-order
    # reduction).
    def bwd_op(name, L, dy, x, dx):
        by = linear_alg_bytes("bwd", B, L.in_f, L.out_f, L.nnz)
        if L.variant == sp.SP_VARIANT_DENSE:
            def f():
                sp.sp_linear_dense_bwd_input(dy, B, L.in_f, L.out_f, L.Wd, dx, dws)
                sp.sp_linear_dense_bwd_weight(dy, x, B, L.in_f, L.out_f, L.row_ptr, L.col_idx, L.nnz, L.dW, dws)
            return (name, f, "dense_bwd", 4.0 * L.nnz * B, by, L)
        return (name, lambda: sp.sp_linear_bwd(dy, x, B, L.in_f, L.out_f, L.vals, L.nnz, L.plan, dx, L.dW, ws),
                "bwd", 4.0 * L.nnz * B, by, L)

    if which == "ffn":
        ops = [fwd_op("W1.fwd", L1, X, Y1), fwd_op("W2.fwd", L2, Y1, Y2),
               bwd_op("W2.bwd", L2, dY2, Y1, dX2), bwd_op("W1.bwd", L1, dX2, X, dX1)]
    else:
        ops = [fwd_op("fwd", L1, X, Y1), bwd_op("bwd", L1, dY1, X, dX1)]
    ms_per_step, per_op, ms_instr = time_ops(torch, ops, args.steps, args.warmup)
    flops_step = sum(o[3] for o in ops)
    bytes_step = sum(o[4] for o in ops)

    # Dominant kernel: the kind of op with the largest share of the step.  The
    # SpMM kernel serves the sparse forward passes; the fused backward kernel
    # (input-gradient SpMM and weight-gradient SDDMM in one launch, then the
    # split reduction) the sparse backward passes; the matrix-core GEMM the
    # dense ones.  Per launch: the mean over the launches of that kind (the
    # two layers' backward passes move different dense bytes).
    kinds = sorted({o[2] for o in ops})
    share = {k: sum(t for o, t in zip(ops, per_op) if o[2] == k) for k in kinds}
    kind = max(kinds, key=lambda k: share[k])
    dom_ms = float(np.mean([t for o, t in zip(ops, per_op) if o[2] == kind]))
    dom = {"fwd": "k_spmm2", "bwd": "k_bwd_fused+k_slot_reduce", "dense_fwd": "k_gemm (after k_scatter_rows)",
           "dense_bwd": "k_gemm x2 + k_sample_rows"}[kind]
    fl = float(np.mean([o[3] for o in ops if o[2] == kind]))
    by = float(np.mean([o[4] for o in ops if o[2] == kind]))
    traffic = measured_traffic(dom) if which == "ffn" and not kind.startswith("dense") else None
    if which == "ffn":
        config = {"workload": "FFN pair W1 768->3072 + W2 3072->768, %g%% unstructured sparse, 8192 tokens, "
                              % (100 * sparsity) +
                              "fwd+bwd (input and weight gradient) of both layers",
                  "tokens": B, "sparsity": sparsity, "nnz_per_layer": L1.nnz}
    else:
        config = {"workload": "linear 256->256, %g%% unstructured sparse, 16 tokens, fwd+bwd" % (100 * sparsity),
                  "tokens": B, "sparsity": sparsity, "nnz": L1.nnz}
    if args.variant != "auto":
        config["variant"] = args.variant
    out = base_record(args, flops_step / (ms_per_step * 1e-3) / 1e9, ms_per_step, config)
    out["hbm"] = hbm_record(bytes_step, ms_per_step)
    out["ms_per_step_with_op_events"] = round(ms_instr, 5)
    mf = None
    if kind.startswith("dense"):
        mf = float(np.mean([(2.0 if kind == "dense_fwd" else 4.0) * B * o[5].in_f * o[5].out_f
                            for o in ops if o[2] == kind]))
    out["roofline"] = roofline(dom, kind, fl, by, dom_ms, traffic, {"source_hash": kernel_source_hash()}, mf)
    out["ops"] = {o[0]: op_row(t, o[3], o[4]) for o, t in zip(ops, per_op)}
    out["variant_choice"] = choice
    cold = cold_record(torch, args, ops)
    if cold:
        out["cold"] = cold
    out["plan_ms"] = {L.name: round(L.plan_ms, 3) for L in layers}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_linear(layers_np, args.cpu_seconds, which)
    return out


def conv_specs(which):
    from synth import CONV_3X3_56, conv_sweep, resnet18_convs, seed_for
    if which == "conv3x3_56":
        return [(s, seed_for(3, i)) for i, s in enumerate(CONV_3X3_56)]
    if which == "conv_sweep":
        return [(s, seed_for(4, i)) for i, s in enumerate(conv_sweep())]
    return [(s, seed_for(5, i)) for i, s in enumerate(resnet18_convs())]


CONV_DESC = {
    "conv3x3_56": "sparse 3x3 conv 64->64, stride 1, pad 1, input 32x64x56x56, 90% unstructured; fwd, bwd_input, "
                  "bwd_weight",
    "conv_sweep": "sparse conv sweep at batch 32: 3x3 128->128 @28x28, 3x3 256->256 @14x14, 1x1 256->1024 @14x14, "
                  "each at 80/90/95/98%; fwd, bwd_input, bwd_weight of every layer",
    "resnet18": "ResNet-18 sparse layers at batch 64, 224x224, 95%: the 20 convolutions and the FC 512->1000; "
                "fwd, bwd_input, bwd_weight of every layer (BN/ReLU/pooling not included)",
}
CONV_KERNEL = {"fwd": "k_spmm2<ConvGeo<0>>",
               "bwd": "k_conv_bwd_fused+k_slot_reduce (<= 8 input channels: k_fewrows, then the SDDMM)",
               "dense_fwd": "k_gemm<ConvTokens> (after k_conv_scatter)",
               "dense_bwd": "k_conv_wt + k_gemm<ConvTokens> + k_gemm<PlaneRows, ConvCols> + k_conv_sample"}


def run_conv(args, sp, torch, which):
    from synth import RESNET18_FC, linear_layer, seed_for
    layers = []
    for spec, seed in conv_specs(which):
        layers.append(ConvLayer(sp, torch, spec, seed))
    # The paper's end-to-end protocol, per layer, before the timed region:
    # dense below 80% sparsity, else the faster of one timed step each.
    choice = {}
    for L in layers:
        L.select(sp, torch, args.variant)
        choice[L.name] = L.choice
    ops = []
    for L in layers:
        ops += L.ops(sp)
    fc = None
    if which == "resnet18":
        _, o_f, i_f, B, s = RESNET18_FC
        d = linear_layer(seed_for(5, 20), o_f, i_f, B, s)
        fc = LinearLayer(sp, torch, d, "fc")
        X = torch.from_numpy(d["X"]).cuda()
        dY = torch.from_numpy(d["dY"]).cuda()
        Y = torch.empty(B, o_f, device="cuda")
        dX = torch.empty(B, i_f, device="cuda")
        ws = torch.empty(max(sp.sp_linear_bwd_weight_ws(B, i_f, o_f, fc.nnz), 1), dtype=torch.uint8, device="cuda")
        if args.variant == "auto":
            sws = torch.empty(max(sp.sp_linear_select_ws(B, i_f, o_f, fc.nnz), 1), dtype=torch.uint8, device="cuda")
            v, ms = sp.sp_linear_select(X, dY, B, i_f, o_f, fc.row_ptr, fc.col_idx, fc.vals, fc.nnz, fc.plan, Y, dX,
                                        fc.dW, sws, 3, select_flags(sp, s))
            del sws
            choice["fc"] = {"variant": "dense" if v == sp.SP_VARIANT_DENSE else "sparse",
                            "ms_sparse_step": round(ms[0], 4), "ms_dense_step": round(ms[1], 4)}
        else:
            v = sp.SP_VARIANT_DENSE if args.variant == "dense" else sp.SP_VARIANT_SPARSE
            choice["fc"] = {"variant": args.variant, "forced": True}
        if v == sp.SP_VARIANT_DENSE:
            Wd = torch.empty(o_f, i_f, device="cuda")
            dws = torch.empty(max(sp.sp_linear_dense_ws(B, i_f, o_f), 1), dtype=torch.uint8, device="cuda")

            def fc_fwd():
                sp.sp_linear_densify(o_f, i_f, fc.row_ptr, fc.col_idx, fc.vals, fc.nnz, Wd)
                sp.sp_linear_dense_fwd(X, B, i_f, o_f, Wd, Y, dws)

            def fc_bwd():
                sp.sp_linear_dense_bwd_input(dY, B, i_f, o_f, Wd, dX, dws)
                sp.sp_linear_dense_bwd_weight(dY, X, B, i_f, o_f, fc.row_ptr, fc.col_idx, fc.nnz, fc.dW, dws)
            fc_ops = (("dense_fwd", fc_fwd), ("dense_bwd", fc_bwd))
        else:
            fc_ops = (("fwd", lambda: sp.sp_linear_fwd(X, B, i_f, o_f, fc.vals, fc.nnz, fc.plan, Y)),
                      ("bwd", lambda: sp.sp_linear_bwd(dY, X, B, i_f, o_f, fc.vals, fc.nnz, fc.plan, dX, fc.dW,
                                                       ws)))
        for kind, f in fc_ops:
            ops.append(("fc." + kind.replace("dense_", ""), f, kind,
                        (4.0 if kind.endswith("bwd") else 2.0) * fc.nnz * B,
                        linear_alg_bytes(kind.replace("dense_", ""), B, i_f, o_f, fc.nnz), fc))
    ms_per_step, per_op, ms_instr = time_ops(torch, ops, args.steps, args.warmup)
    flops_step = sum(o[3] for o in ops)
    bytes_step = sum(o[4] for o in ops)
    # Dominant kernel: the conv op kind with the largest total time; its
    # roofline is taken per launch as total work over total time of its launches.
    kinds = {}
    for o, t in zip(ops, per_op):
        if isinstance(o[5], ConvLayer):
            k = kinds.setdefault(o[2], [0.0, 0.0, 0.0, 0])
            k[0] += t
            k[1] += o[3]
            k[2] += o[4]
            k[3] += 1
    kind = max(kinds, key=lambda k: kinds[k][0])
    t, fl, by, n = kinds[kind]
    config = {"workload": CONV_DESC[which], "layers": len(layers) + (1 if fc else 0),
              "nnz_total": int(sum(L.nnz for L in layers) + (fc.nnz if fc else 0))}
    if args.variant != "auto":
        config["variant"] = args.variant
    out = base_record(args, flops_step / (ms_per_step * 1e-3) / 1e9, ms_per_step, config)
    out["hbm"] = hbm_record(bytes_step, ms_per_step)
    out["ms_per_step_with_op_events"] = round(ms_instr, 5)
    mf = None
    if kind.startswith("dense"):
        dl = [o[5] for o in ops if o[2] == kind and isinstance(o[5], ConvLayer)]
        mf = sum(L.dense_flops() * (2 if kind == "dense_bwd" else 1) for L in dl) / len(dl)
    traffic = None
    if which == "conv3x3_56" and not kind.startswith("dense"):
        traffic = measured_traffic(CONV_KERNEL[kind], CONV_TRAFFIC_FILE, CONV_KERNEL_SOURCES)
    out["roofline"] = roofline(CONV_KERNEL[kind], kind, fl / n, by / n, t / n, traffic,
                               {"launches_per_step": n, "note": "per-launch means over the workload's layers",
                                "source_hash": kernel_source_hash(CONV_KERNEL_SOURCES)}, mf)
    out["by_op"] = {k: {"ms": round(v[0], 4), "tflops": round(v[1] / v[0] / 1e9, 3),
                        "alg_GBps": round(v[2] / v[0] / 1e6, 1), "bound": bound_of(v[1], v[2])}
                    for k, v in kinds.items()}
    out["ops"] = {o[0]: op_row(t, o[3], o[4]) for o, t in zip(ops, per_op)}
    out["variant_choice"] = choice
    cold = cold_record(torch, args, ops)
    if cold:
        out["cold"] = cold
    out["plan_ms"] = {L.name: round(L.plan_ms, 3) for L in layers}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_conv(layers, args.cpu_seconds)
    return out


# --------------------------------------------------------------- CPU baseline

def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def cpu_baseline_linear(layers_np, min_seconds, which):
    """The CPU oracle (as it stands) on the same step over all tokens,
    repeated until at least `min_seconds` have passed; reported in the same
    effective-GFLOP/s unit."""
    import oracle
    X = layers_np[0]["X"]
    ntok = X.shape[0]
    enc = [oracle.linear_encode(d["mask"], d["W"]) for d in layers_np]
    reps = 0
    t = time.perf_counter()
    while True:
        if which == "ffn":
            (rp1, ci1, v1), (rp2, ci2, v2) = enc
            o1, i1 = layers_np[0]["mask"].shape
            o2, i2 = layers_np[1]["mask"].shape
            dY2 = layers_np[1]["dY"]
            Y1, _ = oracle.linear_fwd(X, rp1, ci1, v1, o1)
            Y1f = Y1.astype(np.float32)
            oracle.linear_fwd(Y1f, rp2, ci2, v2, o2)
            dX2, _ = oracle.linear_bwd_input(dY2, rp2, ci2, v2, i2)
            oracle.linear_bwd_weight(dY2, Y1f, rp2, ci2)
            dX2f = dX2.astype(np.float32)
            oracle.linear_bwd_input(dX2f, rp1, ci1, v1, i1)
            oracle.linear_bwd_weight(dX2f, X, rp1, ci1)
        else:
            (rp1, ci1, v1), = enc
            o1, i1 = layers_np[0]["mask"].shape
            oracle.linear_fwd(X, rp1, ci1, v1, o1)
            oracle.linear_bwd_input(layers_np[0]["dY"], rp1, ci1, v1, i1)
            oracle.linear_bwd_weight(layers_np[0]["dY"], X, rp1, ci1)
        reps += 1
        t_total = time.perf_counter() - t
        if t_total >= min_seconds:
            break
    flops = reps * 3 * 2.0 * sum(len(e[2]) for e in enc) * ntok
    return {"value": round(flops / t_total / 1e9, 3), "unit": "GFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle", "seconds": round(t_total, 2), "cpu": _cpu_model(),
            "sample": "the same %d-op step over all %d tokens, repeated %d times (fp64-accumulating plain loops, "
                      "OpenMP over independent outputs; conversions between ops included)"
                      % (3 * len(enc), ntok, reps)}


def cpu_baseline_conv(layers, min_seconds):
    """The CPU oracle on one image per layer (forward, input gradient and
    weight gradient of that image), cycling over the layers until at least
    `min_seconds` have passed and every layer has run once."""
    import oracle
    from synth import conv_layer
    samples = []
    for i, L in enumerate(layers):
        B, IC, H, W, OC, KH, KW = L.dims
        s = L.shape
        d1 = conv_layer(777 + i, 1, IC, H, W, OC, KH, KW, (L.OH, L.OW), 0.5)
        enc = oracle.conv_encode(L.mask_np, L.W_np)
        osh = oracle.conv_shape(1, IC, H, W, OC, KH, KW, (s.stride_h, s.stride_w), (s.pad_h, s.pad_w))
        samples.append((d1["X"], d1["dY"], osh, enc, 3 * 2.0 * L.nnz * L.OH * L.OW))
    flops, n = 0.0, 0
    t = time.perf_counter()
    while True:
        X1, dY1, osh, enc, fl = samples[n % len(samples)]
        oracle.conv_fwd(X1, osh, *enc)
        oracle.conv_bwd_input(dY1, osh, *enc)
        oracle.conv_bwd_weight(dY1, X1, osh, *enc[:4])
        flops += fl
        n += 1
        t_total = time.perf_counter() - t
        if t_total >= min_seconds and n >= len(samples):
            break
    return {"value": round(flops / t_total / 1e9, 3), "unit": "GFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle", "seconds": round(t_total, 2), "cpu": _cpu_model(),
            "sample": "forward, input gradient and weight gradient of one image per layer, %d layer passes over "
                      "%d layers (fp64-accumulating plain loops, OpenMP over independent outputs)"
                      % (n, len(samples))}


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
    if args.workload in ("ffn", "linear_small"):
        out = run_linear(args, sp, torch, args.workload)
    else:
        out = run_conv(args, sp, torch, args.workload)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

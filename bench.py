#!/usr/bin/env python3
"""Benchmark of the mixed-adapter LoRA layer on one MI355X.

One step = one pass of the whole hot path over one batch: the device-built row
grouping (plan) followed by the forward residual (lora_apply), or, for the
masked-backward workload, the plan followed by lora_grad.  The headline line is
the decode workload (256 single-token rows over 64 rank-16 adapters, hidden
4096 -> 4096, bf16): tokens/s of whole steps.  The other four workloads are
measured the same way and reported under "extra"; for the masked-backward
workload the input gradient (lora_grad_x, over the same plan), both gradients in
one call (lora_backward), the AdamW step
over its adapters' tensors (lora_adamw_step) and the PPO-style token loss over
logits [n, 32768] with its action mask (lora_token_loss) are also timed alone;
for the prefill workload the whole adapted layer (lora_linear: the base
projection X W^T plus the residual, one GEMM) is timed too, with torch's own
X W^T (hipBLASLt) beside it for context.

Measurement protocol
  * inputs are resident in HBM before timing; each workload keeps R copies of its
    inputs and weights at distinct addresses and step i uses copy i % R, with
    R * working set >= 576 MB, so every step reads cold (no Infinity Cache hits
    left over from the previous step);
  * the timed region is enqueued behind a GPU-side start gate (a bounded sleep
    kernel), so the GPU runs the K steps back to back without waiting on the
    host; HIP events on the compute stream bracket the region and each op;
  * achieved bandwidth = algorithmic bytes (each tensor counted once at its
    minimum: touched rows of X and Y, touched adapters' weights, ids) divided by
    the average op duration; the peak is MI355X's 8 TB/s HBM; durations are
    also reported as the median and p10 / p90 of block averages (8 blocks);
  * calibration on the same box: a plain 1 GiB device copy (achievable HBM)
    and a register-only matrix-core loop (achievable bf16 MFMA rate); every
    fraction is given against both the datasheet peak and the calibrated one.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--configs 1,2,3,4,5]
"""
import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # dense bf16 matrix cores
FP32_PEAK_TFLOPS = 157.3       # vector fp32
ROTATE_BYTES = 576 << 20       # >= 2 x 288 MB of rotating working set
HEADLINE = 2
IDS_MAX_ROWS = 1024            # lora_apply_ids row limit (LORA_APPLY_IDS_MAX_ROWS)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--configs", default="1,2,3,4,5")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy", action="store_true",
                    help="(kept for old command lines: the calibrations always run)")
    ap.add_argument("--pmc-summary", nargs="+", metavar="CSV",
                    help="print the per-kernel table of rocprofv3 --pmc counter CSVs of bench "
                         "runs (no GPU needed) and exit")
    ap.add_argument("--stats-summary", metavar="CSV",
                    help="print the markdown table of a rocprofv3 --kernel-trace --stats "
                         "kernel_stats.csv (no GPU needed) and exit")
    return ap.parse_args()


# sources the decode batch's kernels are built from (the forward kernels, their
# launch code and the entry points' dispatch); the gradient and vector-path
# files do not affect them
HEADLINE_SOURCES = ("fwd_mfma.hip", "api.cpp", "device_common.h", "lora_internal.h")


def source_digest(files=HEADLINE_SOURCES):
    """Digest of the native sources the headline kernels come from (None: every
    source file of the library)."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2601_07376_amd", "csrc")
    if files is None:
        files = [f for f in os.listdir(csrc) if f.endswith((".hip", ".cpp", ".h"))]
    for f in sorted(files):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


# ----------------------------------------------------------------------------
# algorithmic bytes and flops (each tensor once, at its minimum)
# ----------------------------------------------------------------------------

def workload_counts(case):
    idx = case.idx
    act = idx >= 0
    touched = np.unique(idx[act])
    xs = 2 if case.x_dtype == "bf16" else 4
    ws = 2 if case.w_dtype == "bf16" else 4
    ys = 2 if case.y_dtype == "bf16" else 4
    d_in, d_out = case.d_in, case.d_out
    ranks = case.ranks.astype(np.int64)
    if case.mask is None:                  # forward
        n_act = int(act.sum())
        w_bytes = int(np.sum(ranks[touched]) * (d_in + d_out) * ws)
        op_bytes = n_act * d_in * xs + 2 * n_act * d_out * ys + w_bytes
        plan_bytes = case.n * 4
        flops = int(np.sum(2 * ranks[idx[act]] * (d_in + d_out)))
        return dict(n=case.n, n_act=n_act, adapters=len(touched), op_bytes=op_bytes,
                    plan_bytes=plan_bytes, flops=flops)
    m = act & (case.mask != 0)
    n_m = int(m.sum())
    live = np.nonzero(ranks > 0)[0]
    op_bytes = (n_m * (d_in + d_out) * xs
                + int(np.sum(ranks[live]) * (d_in + d_out) * (ws + 4)))
    flops = int(np.sum(4 * ranks[idx[m]] * (d_in + d_out)))
    return dict(n=case.n, n_act=int(act.sum()), n_masked=n_m, adapters=len(live),
                op_bytes=op_bytes, plan_bytes=case.n * 5, flops=flops)


# ----------------------------------------------------------------------------
# one workload on the GPU
# ----------------------------------------------------------------------------

class Rig:
    """R device copies of one workload, each with its own table and workspaces."""

    def __init__(self, case, copies):
        import torch
        import paper_2601_07376_amd as L
        from workloads.device import case_to_device
        self.case, self.L, self.torch = case, L, torch
        # small bf16 forward batches run plan-free (lora_apply_ids: the kernels
        # group the rows by adapter themselves, two launches per step)
        self.plan_free = (case.mask is None and case.x_dtype == "bf16" and case.w_dtype == "bf16"
                          and case.n <= IDS_MAX_ROWS and case.seg_offsets is None)
        base = case_to_device(case, "cuda")
        wdt = torch.bfloat16 if case.w_dtype == "bf16" else torch.float32
        self.sets = []
        for r in range(copies):
            if r == 0:
                d = dict(base)
            else:
                d = {k: ([t.clone() if t is not None else None for t in v]
                         if isinstance(v, list) else (v.clone() if v is not None else None))
                     for k, v in base.items()}
            table = L.Table(case.num_slots, case.d_in, case.d_out, w_dtype=wdt, device="cuda")
            for a in range(case.num_slots):
                if case.ranks[a] > 0:
                    table.set(a, d["A"][a], d["B"][a], float(case.scales[a]))
            table.upload()
            n = case.n
            d["table"] = table
            d["plan_ws"] = torch.empty(max(L.lib().lora_plan_workspace_bytes(n, case.num_slots), 16),
                                       dtype=torch.uint8, device="cuda")
            # a plan object only to size the op workspaces
            if "seg_offsets" in d:
                probe = L.Plan(table, seg_offsets=d["seg_offsets"], seg_adapter=d["seg_adapter"],
                               n=n, mask=d["mask"])
            else:
                probe = L.Plan(table, idx=d["idx"], mask=d["mask"])
            if case.mask is None:
                d["op_ws"] = L.apply_workspace(probe)
                if self.plan_free:
                    d["ids_ws"] = L.apply_ids_workspace(table, n)
            else:
                d["op_ws"] = L.grad_workspace(probe)
                d["dA"] = [torch.zeros(int(r_), case.d_in, dtype=torch.float32, device="cuda")
                           if r_ > 0 else None for r_ in case.ranks]
                d["dB"] = [torch.zeros(case.d_out, int(r_), dtype=torch.float32, device="cuda")
                           if r_ > 0 else None for r_ in case.ranks]
                S = case.num_slots
                d["pA"] = (ctypes.c_void_p * S)(*[t.data_ptr() if t is not None else None
                                                   for t in d["dA"]])
                d["pB"] = (ctypes.c_void_p * S)(*[t.data_ptr() if t is not None else None
                                                   for t in d["dB"]])
                d["dX"] = torch.zeros(n, case.d_in, dtype=torch.float32, device="cuda")
                d["gx_ws"] = L.grad_x_workspace(probe)
                d["bw_ws"] = L.backward_workspace(probe)
                # optimizer state of every adapter tensor: fp32 master, moments,
                # the gradient buffers above, and the table's bf16 weights as the
                # rounded copy
                keep, recs = [], []
                for a in range(case.num_slots):
                    if case.ranks[a] <= 0:
                        continue
                    for w, g in ((d["A"][a], d["dA"][a]), (d["B"][a], d["dB"][a])):
                        pm = w.float().reshape(-1).clone()
                        mm, vv = torch.zeros_like(pm), torch.zeros_like(pm)
                        keep += [pm, mm, vv]
                        recs.append(L.AdamWTensor(pm.data_ptr(), mm.data_ptr(), vv.data_ptr(),
                                                  g.data_ptr(), w.data_ptr(), pm.numel(), 10,
                                                  1e-4, 0.9, 0.999, 1e-8, 0.01))
                d["adam_keep"] = keep
                d["adam_recs"] = (L.AdamWTensor * len(recs))(*recs)
                d["adam_elems"] = sum(int(r.n) for r in recs)
            del probe
            self.sets.append(d)
        torch.cuda.synchronize()

    def build_plan(self, d):
        """Enqueue the plan build for one copy; returns the host handle."""
        L, case = self.L, self.case
        lib = L.lib()
        stream = ctypes.c_void_p(self.torch.cuda.current_stream().cuda_stream)
        h = ctypes.c_void_p()
        mask = d["mask"].data_ptr() if d["mask"] is not None else None
        if "seg_offsets" in d:
            st = lib.lora_plan_build_segments(d["table"].handle, case.n, d["seg_adapter"].numel(),
                                              d["seg_offsets"].data_ptr(),
                                              d["seg_adapter"].data_ptr(), mask,
                                              d["plan_ws"].data_ptr(), d["plan_ws"].numel(),
                                              stream, ctypes.byref(h))
        else:
            st = lib.lora_plan_build(d["table"].handle, case.n, d["idx"].data_ptr(), mask,
                                     d["plan_ws"].data_ptr(), d["plan_ws"].numel(), stream,
                                     ctypes.byref(h))
        assert st == 0, lib.lora_last_error()
        return h

    def run_op(self, d, h):
        """Enqueue the forward residual (or the masked gradients) for one copy."""
        L, case = self.L, self.case
        lib = L.lib()
        stream = ctypes.c_void_p(self.torch.cuda.current_stream().cuda_stream)
        X = d["X"]
        xdt = 1 if case.x_dtype == "bf16" else 0
        if case.mask is None:
            Y = d["Y"]
            st = lib.lora_apply(h, X.data_ptr(), xdt, X.stride(0), Y.data_ptr(),
                                1 if case.y_dtype == "bf16" else 0, Y.stride(0),
                                d["op_ws"].data_ptr(), d["op_ws"].numel(), stream)
        else:
            dY = d["dY"]
            st = lib.lora_grad(h, X.data_ptr(), xdt, X.stride(0), dY.data_ptr(), xdt,
                               dY.stride(0), None, 0, d["pA"], d["pB"], 0,
                               d["op_ws"].data_ptr(), d["op_ws"].numel(), stream)
        assert st == 0, lib.lora_last_error()

    def run_ids(self, d):
        """Enqueue lora_apply_ids (no plan) for one copy."""
        lib = self.L.lib()
        stream = ctypes.c_void_p(self.torch.cuda.current_stream().cuda_stream)
        X, Y = d["X"], d["Y"]
        st = lib.lora_apply_ids(d["table"].handle, self.case.n, d["idx"].data_ptr(), X.data_ptr(), 1,
                                X.stride(0), Y.data_ptr(), 1 if self.case.y_dtype == "bf16" else 0,
                                Y.stride(0), d["ids_ws"].data_ptr(), d["ids_ws"].numel(), stream)
        assert st == 0, lib.lora_last_error()

    def step_with_plan(self, i):
        """Enqueue one step through a plan: plan build, then the op."""
        d = self.sets[i % len(self.sets)]
        h = self.build_plan(d)
        self.run_op(d, h)
        self.L.lib().lora_plan_destroy(h)   # host object only; enqueued work keeps its arguments

    def run_grad_x(self, d, h):
        """Enqueue the input gradient dX += s dY B A over the masked rows for one copy."""
        lib = self.L.lib()
        stream = ctypes.c_void_p(self.torch.cuda.current_stream().cuda_stream)
        dY, dX = d["dY"], d["dX"]
        st = lib.lora_grad_x(h, dY.data_ptr(), 1 if self.case.x_dtype == "bf16" else 0,
                             dY.stride(0), dX.data_ptr(), 0, dX.stride(0),
                             d["gx_ws"].data_ptr(), d["gx_ws"].numel(), stream)
        assert st == 0, lib.lora_last_error()

    def run_backward(self, d, h):
        """Enqueue lora_backward (adapter gradients and input gradient) for one copy."""
        lib = self.L.lib()
        stream = ctypes.c_void_p(self.torch.cuda.current_stream().cuda_stream)
        X, dY, dX = d["X"], d["dY"], d["dX"]
        st = lib.lora_backward(h, X.data_ptr(), 1, X.stride(0), dY.data_ptr(), 1, dY.stride(0), None, 0,
                               d["pA"], d["pB"], 0, dX.data_ptr(), 0, dX.stride(0),
                               d["bw_ws"].data_ptr(), d["bw_ws"].numel(), stream)
        assert st == 0, lib.lora_last_error()

    def run_adamw(self, d):
        """Enqueue one AdamW step over every adapter tensor of one copy."""
        lib = self.L.lib()
        stream = ctypes.c_void_p(self.torch.cuda.current_stream().cuda_stream)
        st = lib.lora_adamw_step(ctypes.cast(d["adam_recs"], ctypes.c_void_p),
                                 len(d["adam_recs"]), stream)
        assert st == 0, lib.lora_last_error()

    def step(self, i):
        """Enqueue one step on the current stream: lora_apply_ids for a
        plan-free batch, else plan build then the op."""
        if self.plan_free:
            self.run_ids(self.sets[i % len(self.sets)])
        else:
            self.step_with_plan(i)


LOSS_VOCAB = 32768


def token_loss_leg(case, timed, steps):
    """The PPO-style token loss on logits [n, LOSS_VOCAB] (bf16 in and out) with
    the batch's action mask: the active rows' logits are read once (rows up to
    32768 stay in registers) and every gradient row is written."""
    import torch
    import paper_2601_07376_amd as L
    n, V = case.n, LOSS_VOCAB
    g = torch.Generator(device="cuda").manual_seed(5)
    z = (torch.randn(n, V, device="cuda", generator=g) * 2.0).to(torch.bfloat16)
    dz = torch.empty_like(z)
    target = torch.randint(0, V, (n,), device="cuda", generator=g, dtype=torch.int32)
    mask = torch.from_numpy(np.asarray(case.mask, np.uint8)).cuda()
    old = torch.randn(n, device="cuda", generator=g) - 10.0
    adv = torch.randn(n, device="cuda", generator=g)
    loss = torch.empty(n, device="cuda")
    logp = torch.empty(n, device="cuda")
    lib = L.lib()
    args = [2, n, V, z.data_ptr(), 1, V, target.data_ptr(), None, mask.data_ptr(), old.data_ptr(),
            adv.data_ptr(), None, 0.2, 0.2, loss.data_ptr(), logp.data_ptr(), dz.data_ptr(), 1, V]

    def enqueue(i):
        st = lib.lora_token_loss(*args, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        assert st == 0, lib.lora_last_error()
    for i in range(3):
        enqueue(i)
    us = timed(enqueue, max(20, steps // 4)) * 1e3
    act = int(np.count_nonzero(case.mask))
    nbytes = act * V * 2 + n * V * 2 + n * 4 * 6      # active logits read, gradient written, per-row vectors
    del z, dz
    torch.cuda.empty_cache()
    return dict(op="lora_token_loss", kind="ppo", rows=n, active_rows=act, vocab=V, us_mean=us,
                bytes=nbytes, GBps=nbytes / (us * 1e-6) / 1e9,
                hbm_frac=nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS)


def linear_leg(case, rig, h, timed, steps):
    """The whole adapted layer on the prefill batch: lora_linear writes
    Y = X W^T + s_a (X A_a^T) B_a^T (bf16 Y) with W [d_out, d_in] bf16 ~
    N(0, 1/d_in).  X, W and Y (1.1 GB together) exceed the Infinity Cache, so
    every call streams them from HBM.  torch.matmul of X W^T alone (hipBLASLt)
    is timed on the same tensors for context."""
    import torch
    import workloads
    import paper_2601_07376_amd as L
    d = rig.sets[0]
    X = d["X"]
    W = torch.from_numpy(workloads.base_weight(case).view(np.int16)).cuda().view(torch.bfloat16)
    Y = torch.empty(case.n, case.d_out, dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(max(L.lib().lora_linear_workspace_bytes(h), 16), dtype=torch.uint8, device="cuda")
    lib = L.lib()

    def enqueue(i):
        st = lib.lora_linear(h, X.data_ptr(), 1, X.stride(0), W.data_ptr(), 1, W.stride(0),
                             Y.data_ptr(), 1, Y.stride(0), ws.data_ptr(), ws.numel(),
                             ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        assert st == 0, lib.lora_last_error()
    for i in range(2):
        enqueue(i)
    k = max(10, steps // 10)
    us = timed(enqueue, k, "linear_us") * 1e3
    Wt = W.t()
    for i in range(2):
        torch.matmul(X, Wt, out=Y)
    t_us = timed(lambda i: torch.matmul(X, Wt, out=Y), k, "torch_xwt_us") * 1e3
    idx = case.idx
    act = idx >= 0
    ranks = case.ranks.astype(np.int64)
    touched = np.unique(idx[act])
    base_flops = 2 * case.n * case.d_in * case.d_out
    lora_flops = int(np.sum(2 * ranks[idx[act]] * (case.d_in + case.d_out)))
    nbytes = (case.n * case.d_in * 2 + case.d_out * case.d_in * 2 + case.n * case.d_out * 2
              + int(np.sum(ranks[touched]) * (case.d_in + case.d_out) * 2))
    fl = base_flops + lora_flops
    del W, Y, ws
    torch.cuda.empty_cache()
    return dict(op="lora_linear", us_mean=us, flops=fl, base_flops=base_flops, lora_flops=lora_flops,
                bytes=nbytes, TFLOPs=fl / (us * 1e-6) / 1e12,
                mfma_frac=fl / (us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS,
                GBps=nbytes / (us * 1e-6) / 1e9, torch_xwt_us=t_us,
                torch_xwt_TFLOPs=base_flops / (t_us * 1e-6) / 1e12)


def sleep_rate(torch):
    """GPU sleep-kernel cycles per millisecond (for the start gate)."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    torch.cuda._sleep(2_000_000)
    e1.record()
    torch.cuda.synchronize()
    return 2_000_000 / max(e0.elapsed_time(e1), 1e-3)


def run_workload(cfg, steps, warmup, rate):
    import torch
    import workloads
    import paper_2601_07376_amd as L
    t0 = time.time()
    case = workloads.make_config(cfg)
    counts = workload_counts(case)
    ws_bytes = counts["op_bytes"] + counts["plan_bytes"]
    copies = 1 if cfg == 1 else max(1, min(64, -(-ROTATE_BYTES // max(ws_bytes, 1))))
    rig = Rig(case, copies)
    log(f"[bench] workload {cfg} {case.name}: n={case.n} copies={copies} "
        f"(setup {time.time() - t0:.1f}s)")

    # warmup, and the host's enqueue cost per step (sizes the start gate)
    c0 = time.perf_counter()
    for i in range(warmup):
        rig.step(i)
    host_ms = (time.perf_counter() - c0) * 1e3 / max(warmup, 1)
    torch.cuda.synchronize()

    dist = {}

    def timed(enqueue, k, key=None, blocks=8, warm=0):
        """Average GPU time (ms) per call of enqueue(i) over k back-to-back calls:
        the calls are queued behind a GPU-side start gate, so the GPU never waits
        on the host, and events on the compute stream bracket them; an event
        after each of `blocks` blocks gives the spread of block averages
        (median, p10, p90 in us, stored under `key`).  warm > 0: that many
        untimed calls first, whose host cost also sizes the gate."""
        leg_ms = host_ms
        if warm > 0:
            torch.cuda.synchronize()
            c1 = time.perf_counter()
            for i in range(warm):
                enqueue(i)
            leg_ms = max(host_ms, (time.perf_counter() - c1) * 1e3 / warm)
            torch.cuda.synchronize()
        nb = max(1, min(blocks, k // 8))
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(nb + 1)]
        gate_ms = min(500.0, 2.0 + 2.0 * leg_ms * k)
        torch.cuda.synchronize()
        torch.cuda._sleep(int(gate_ms * rate))
        ev[0].record()
        bounds = [round(j * k / nb) for j in range(nb + 1)]
        for j in range(nb):
            for i in range(bounds[j], bounds[j + 1]):
                enqueue(i)
            ev[j + 1].record()
        torch.cuda.synchronize()
        per = [ev[j].elapsed_time(ev[j + 1]) * 1e3 / max(bounds[j + 1] - bounds[j], 1) for j in range(nb)]
        if key is not None:
            dist[key] = dict(median=float(np.median(per)), p10=float(np.percentile(per, 10)),
                             p90=float(np.percentile(per, 90)), blocks=nb)
        return ev[0].elapsed_time(ev[nb]) / k

    # whole steps (plan + op), the measured quantity
    w0 = time.perf_counter()
    ms_step = timed(rig.step, steps, "step_us")
    wall_ms = (time.perf_counter() - w0) * 1e3
    # each kernel stage alone, back to back over the same rotating copies
    handles = [rig.build_plan(d) for d in rig.sets]
    torch.cuda.synchronize()
    nc = len(rig.sets)
    if rig.plan_free:
        op_mean = timed(lambda i: rig.run_ids(rig.sets[i % nc]), steps, "op_us") * 1e3
        # the same batch through a plan (plan build + lora_apply), for context
        with_plan = dict(
            step_us=timed(rig.step_with_plan, steps, "plan_path_step_us") * 1e3,
            op_us=timed(lambda i: rig.run_op(rig.sets[i % nc], handles[i % nc]), steps,
                        "plan_path_op_us") * 1e3)
    else:
        op_mean = timed(lambda i: rig.run_op(rig.sets[i % nc], handles[i % nc]), steps, "op_us") * 1e3
        with_plan = None
    gx_us = adam_us = bw_us = None
    if case.mask is not None and case.x_dtype == "bf16":
        # the other legs: a few untimed calls each first, and at least 50 timed
        kl = max(steps, 50)
        gx_us = timed(lambda i: rig.run_grad_x(rig.sets[i % nc], handles[i % nc]), kl, "grad_x_us",
                      warm=4) * 1e3
        bw_us = timed(lambda i: rig.run_backward(rig.sets[i % nc], handles[i % nc]), kl, "backward_us",
                      warm=4) * 1e3
    if case.mask is not None:
        adam_us = timed(lambda i: rig.run_adamw(rig.sets[i % nc]), max(steps, 50), "adamw_us",
                        warm=4) * 1e3
    loss_r = token_loss_leg(case, timed, steps) if case.mask is not None else None
    lin_r = linear_leg(case, rig, handles[0], timed, steps) if cfg == 3 else None
    for h in handles:
        L.lib().lora_plan_destroy(h)
    plan_us = timed(lambda i: L.lib().lora_plan_destroy(rig.build_plan(rig.sets[i % nc])),
                    steps, "plan_us") * 1e3
    r = dict(workload=case.name, config=cfg, copies=copies, steps=steps,
             ms_per_step=ms_step, tokens_per_s=case.n / (ms_step * 1e-3),
             op_us_mean=op_mean, plan_us_mean=plan_us,
             op=("lora_grad" if case.mask is not None
                 else "lora_apply_ids" if rig.plan_free else "lora_apply"),
             wall_ms_incl_gate=wall_ms, host_enqueue_ms_per_step=host_ms,
             **counts)
    r["op_GBps"] = counts["op_bytes"] / (op_mean * 1e-6) / 1e9
    r["op_hbm_frac"] = r["op_GBps"] / HBM_PEAK_GBS
    r["op_TFLOPs"] = counts["flops"] / (op_mean * 1e-6) / 1e12
    peak_f = BF16_PEAK_TFLOPS if case.x_dtype == "bf16" else FP32_PEAK_TFLOPS
    r["op_mfma_frac"] = r["op_TFLOPs"] / peak_f
    # the matrix-core fraction an HBM-bound op can reach at this intensity
    r["mfma_frac_ceiling"] = min(1.0, (counts["flops"] / counts["op_bytes"]) * HBM_PEAK_GBS
                                 / 1e3 / peak_f)
    r["step_GBps"] = ws_bytes / (ms_step * 1e-3) / 1e9
    r["timing_spread_us"] = dict(dist)
    if with_plan is not None:
        with_plan["plan_us"] = plan_us
        r["plan_path"] = with_plan
        log(f"[bench]   through a plan: plan {plan_us:.2f} us + lora_apply {with_plan['op_us']:.2f} us; "
            f"step {with_plan['step_us']:.2f} us")
    if lin_r is not None:
        r["linear"] = lin_r
        log(f"[bench]   lora_linear (X W^T + residual, {case.n} x {case.d_in} -> {case.d_out}): "
            f"{lin_r['us_mean']:.1f} us, {lin_r['TFLOPs']:.0f} TFLOP/s = "
            f"{100 * lin_r['mfma_frac']:.1f}% of bf16 peak; torch X W^T alone "
            f"{lin_r['torch_xwt_us']:.1f} us")
    if loss_r is not None:
        r["token_loss"] = loss_r
        log(f"[bench]   lora_token_loss (PPO, {loss_r['rows']} rows, {loss_r['active_rows']} active, "
            f"vocab {loss_r['vocab']}): {loss_r['us_mean']:.2f} us, {loss_r['GBps']:.0f} GB/s = "
            f"{100 * loss_r['hbm_frac']:.1f}% HBM")
    if gx_us is not None:
        # input gradient: dY rows read, f32 dX rows read and written, both
        # factors of every touched adapter read once
        n_m = counts["n_masked"]
        ranks = case.ranks.astype(np.int64)
        m = (case.idx >= 0) & (case.mask != 0)
        touched = np.unique(case.idx[m])
        gx_bytes = (n_m * (case.d_out * 2 + case.d_in * 8)
                    + int(np.sum(ranks[touched]) * (case.d_in + case.d_out) * 2))
        gx_flops = int(np.sum(2 * ranks[case.idx[m]] * (case.d_in + case.d_out)))
        r["grad_x"] = dict(op="lora_grad_x", us_mean=gx_us, bytes=gx_bytes, flops=gx_flops,
                           GBps=gx_bytes / (gx_us * 1e-6) / 1e9,
                           hbm_frac=gx_bytes / (gx_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                           TFLOPs=gx_flops / (gx_us * 1e-6) / 1e12)
        log(f"[bench]   lora_grad_x: {gx_us:.2f} us, {r['grad_x']['GBps']:.0f} GB/s = "
            f"{100 * r['grad_x']['hbm_frac']:.1f}% HBM")
    if bw_us is not None:
        bb = counts["op_bytes"] + r["grad_x"]["bytes"]
        r["backward"] = dict(op="lora_backward", us_mean=bw_us, bytes=bb,
                             GBps=bb / (bw_us * 1e-6) / 1e9,
                             hbm_frac=bb / (bw_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                             separate_us=op_mean + gx_us)
        log(f"[bench]   lora_backward (grad + grad_x): {bw_us:.2f} us against "
            f"{op_mean + gx_us:.2f} us as two calls")
    if adam_us is not None:
        # per element: p, m, v, g read (16 bytes), p, m, v written (12), bf16 copy (2)
        el = rig.sets[0]["adam_elems"]
        ab = 30 * el
        r["adamw"] = dict(op="lora_adamw_step", us_mean=adam_us, tensors=len(rig.sets[0]["adam_recs"]),
                          elements=el, bytes=ab, GBps=ab / (adam_us * 1e-6) / 1e9,
                          hbm_frac=ab / (adam_us * 1e-6) / 1e9 / HBM_PEAK_GBS)
        log(f"[bench]   lora_adamw_step ({r['adamw']['tensors']} tensors, {el} elements): "
            f"{adam_us:.2f} us, {r['adamw']['GBps']:.0f} GB/s = {100 * r['adamw']['hbm_frac']:.1f}% HBM")
    log(f"[bench]   {'(no plan)' if rig.plan_free else f'plan {plan_us:.2f} us;'} {r['op']}: {op_mean:.2f} us, "
        f"{r['op_GBps']:.0f} GB/s = {100 * r['op_hbm_frac']:.1f}% HBM, "
        f"{r['op_TFLOPs']:.1f} TFLOP/s; step {ms_step * 1e3:.2f} us, "
        f"{r['tokens_per_s']:.3e} tokens/s")
    del rig
    torch.cuda.empty_cache()
    return r, case


def calib_copy():
    """A plain elementwise copy kernel of known size (read 1 GiB, write 1 GiB): the
    achievable HBM rate on this machine, and the reading that scales the FETCH_SIZE
    / WRITE_SIZE counters to bytes.  Best of 5."""
    import torch
    a = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1.0)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    best = None
    for _ in range(5):
        e0.record()
        torch.neg(a, out=b)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    gbps = 2 * (1 << 30) / best / 1e6
    log(f"[bench] calibration copy (neg) 1 GiB: {best:.3f} ms = {gbps:.0f} GB/s")
    del a, b
    torch.cuda.empty_cache()
    return dict(bytes_read=1 << 30, bytes_written=1 << 30, ms=best, GBps=gbps)


def calib_mfma():
    """The library's register-only matrix-core loop (lora_calibrate_mfma), one
    workgroup of 4 waves per CU: the achievable bf16 MFMA rate on this machine
    (clock under a matrix-core load included).  Best of 3."""
    import torch
    import paper_2601_07376_amd as L
    wgs, iters = 256, 20000
    out = torch.empty(wgs * 256, dtype=torch.float32, device="cuda")
    lib = L.lib()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    best = None
    for _ in range(3):
        e0.record()
        st = lib.lora_calibrate_mfma(wgs, iters, out.data_ptr(),
                                     ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        assert st == 0, lib.lora_last_error()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    flops = wgs * 4 * iters * 16 * 32768.0
    tf = flops / (best * 1e-3) / 1e12
    log(f"[bench] calibration matrix cores (register-only bf16 loop): {tf:.0f} TFLOP/s")
    return dict(flops=flops, ms=best, TFLOPs=tf)


def _oracle_pass(case):
    """One pass of the float64 oracle over a whole batch: the plan and the
    residual (forward workloads) or the masked gradients (backward workload)."""
    import oracle
    import workloads
    dec = workloads.decode
    X = dec(case.X, case.x_dtype)
    A = [dec(a, case.w_dtype) if a is not None else None for a in case.A]
    B = [dec(b, case.w_dtype) if b is not None else None for b in case.B]
    if case.mask is None:
        Y = dec(case.Y, case.y_dtype)

        def run():
            eff, _ = oracle.effective_ids(case.idx, case.num_slots, case.ranks)
            oracle.canonical_plan(case.idx, case.num_slots, ranks=case.ranks)
            oracle.apply(eff, X, Y, A, B, case.scales)
    else:
        dY = dec(case.dY, case.x_dtype)

        def run():
            eff, _ = oracle.effective_ids(case.idx, case.num_slots, case.ranks)
            oracle.canonical_plan(case.idx, case.num_slots, mask=case.mask, ranks=case.ranks)
            oracle.grad(eff, case.mask, X, dY, A, B, case.scales)
    return run


def _time_passes(run, seconds, min_reps=3):
    times, t0 = [], time.perf_counter()
    while len(times) < min_reps or time.perf_counter() - t0 < seconds:
        a = time.perf_counter()
        run()
        times.append(time.perf_counter() - a)
    return times


def cpu_baseline(case, seconds):
    """The float64 oracle on the host (plan + residual) on the whole headline
    batch, for about `seconds` on every core BLAS uses; tokens/s from the median
    pass (p10 / p90 beside it).  Then single-thread runs (BLAS limited to one
    thread) of the tiny, decode and masked-backward workloads, about 2 s each."""
    import workloads
    from threadpoolctl import threadpool_info, threadpool_limits
    blas = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    affinity = len(os.sched_getaffinity(0))
    times = _time_passes(_oracle_pass(case), seconds)
    med = float(np.median(times))
    one = {}
    with threadpool_limits(limits=1):
        for c in (1, 2, 5):
            cs = case if c == HEADLINE else workloads.make_config(c)
            t = _time_passes(_oracle_pass(cs), 2.0)
            one[cs.name] = dict(tokens_per_s=cs.n / float(np.median(t)), passes=len(t),
                                median_s=float(np.median(t)))
    return dict(value=case.n / med, unit="tokens/s", cores=int(min(blas, affinity)), kind="oracle",
                sample=f"{len(times)} passes of the full {case.name} batch ({case.n} rows): "
                       f"plan + float64 residual, {sum(times):.1f} s; median pass",
                blas_threads=int(blas), affinity_cores=int(affinity),
                p10_tokens_per_s=case.n / float(np.percentile(times, 90)),
                p90_tokens_per_s=case.n / float(np.percentile(times, 10)),
                single_thread=one)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "all_workloads.counters.txt")
# kernels of one call of the headline op (lora_apply_ids on the decode batch)
HEADLINE_KERNELS = ("ids_shrink_kernel", "ids_expand_kernel")
# kernels of one call of each measured op, per workload (each launched once per
# call; names as the counter summary prints them)
OP_KERNELS = {
    ("tiny_sgmv_fp32", "lora_apply"): ("shrink_valu_kernel<false, false, 32>(ValuArgs)",
                                        "expand_valu_kernel<false, false>(ValuArgs)"),
    ("decode_bgmv", "lora_apply_ids"): ("ids_shrink_kernel<1, 8>", "ids_expand_kernel<true, 1, true>"),
    ("prefill_sgmv", "lora_apply"): ("shrink_kernel<4, 1>", "expand_kernel<true, true, 2, 1>"),
    ("prefill_sgmv", "lora_linear"): ("shrink_kernel<4, 1>", "linear_hpack_kernel(LinArgs)",
                                      "linear_kernel<true, true, 64, 2, true, true>(LinArgs)"),
    ("skewed_hetero", "lora_apply"): ("shrink_fine_kernel<4, false>",
                                      "expand_fine_kernel<true, true, 2, 2, false>",
                                      "small_shrink_kernel<4, 2>", "small_expand_kernel<true, 4, true>"),
    ("masked_backward", "lora_grad"): ("hg_kernel<2>(GradArgs)", "hgsum_kernel(GradArgs)",
                                       "dadb_kernel<2>(GradArgs)"),
    ("masked_backward", "lora_grad_x"): ("shrink_fine_kernel<2, true>",
                                         "expand_fine_kernel<false, true, 1, 1, true>"),
    ("masked_backward", "lora_token_loss"): ("token_loss_kernel<true, true>(LossArgs)",),
    ("masked_backward", "lora_adamw_step"): ("adamw_kernel(AdamArgs)",),
}
# the calibration copy (torch's elementwise negation of 1 GiB float32 into a new
# tensor): reads and writes exactly 1 GiB, which scales FETCH_SIZE / WRITE_SIZE
CALIB_KERNEL = "neg_kernel"


def _short_kernel(name):
    n = name.replace("void ", "").replace("lora::(anonymous namespace)::", "")
    n = n.split("(lora::")[0].split("(FwdArgs")[0]
    if CALIB_KERNEL in n:
        return "calibration copy (" + n[:60] + ")"
    return n[:70]


def pmc_summary(paths):
    """Per-kernel means of rocprofv3 --pmc counter CSVs (one row per kernel, one
    column per counter, dispatch durations under counters), the FETCH/WRITE
    scale from the calibration copy, and the headline op's traffic per call."""
    import csv
    import collections
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    dur = collections.defaultdict(list)
    for path in paths:
        with open(path) as f:
            for r in csv.DictReader(f):
                k = _short_kernel(r["Kernel_Name"])
                vals[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
                dur[k].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3)
    counters = sorted({c for d in vals.values() for c in d})
    mean = {k: {c: (sum(v) / len(v)) for c, v in d.items()} for k, d in vals.items()}
    calib = next((k for k in mean if k.startswith("calibration copy")), None)
    fs = ws = None
    if calib is not None:
        if mean[calib].get("FETCH_SIZE"):
            fs = (1 << 20) / mean[calib]["FETCH_SIZE"]
        if mean[calib].get("WRITE_SIZE"):
            ws = (1 << 20) / mean[calib]["WRITE_SIZE"]
    out = [f"source_digest: {source_digest()}", f"source_digest_all: {source_digest(None)}"]
    if fs is not None:
        out.append(f"fetch_scale: {fs:.4f}")
    if ws is not None:
        out.append(f"write_scale: {ws:.4f}")
    head = [k for k in mean if k.startswith(HEADLINE_KERNELS)]
    hb = lambda k: (mean[k].get("FETCH_SIZE", 0) * fs + mean[k].get("WRITE_SIZE", 0) * ws) * 1024
    if fs is not None and ws is not None and head:
        out.append(f"traffic_bytes_per_launch: {int(round(sum(hb(k) for k in head)))}")
        out.append("headline_kernels: " + " + ".join(sorted(head)))
    if fs is not None and ws is not None:
        # every op whose kernels all appear: bytes per call
        for (wl, op), ks in OP_KERNELS.items():
            if all(k in mean for k in ks):
                out.append(f"traffic {wl} {op}: {int(round(sum(hb(k) for k in ks)))}")
    out.append("")
    cols = ["kernel", "dispatches"] + counters + ["us/dispatch (under counters)"]
    if fs is not None and ws is not None:
        cols.insert(2 + len(counters), "HBM MB/dispatch (scaled)")
    out.append("| " + " | ".join(cols) + " |")
    out.append("|" + "---|" * len(cols))
    order = sorted(mean, key=lambda k: -sum(dur[k]))
    for k in order:
        n = max(len(v) for v in vals[k].values())
        row = [k, str(n)] + [f"{mean[k][c]:.1f}" if c in mean[k] else "" for c in counters]
        if fs is not None and ws is not None:
            row.append(f"{(mean[k].get('FETCH_SIZE', 0) * fs + mean[k].get('WRITE_SIZE', 0) * ws) * 1024 / 1e6:.2f}"
                       if "FETCH_SIZE" in mean[k] or "WRITE_SIZE" in mean[k] else "")
        row.append(f"{sum(dur[k]) / len(dur[k]):.2f}")
        out.append("| " + " | ".join(row) + " |")
    print("\n".join(out))


def _traffic_kv():
    kv = {}
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            for ln in f:
                if ":" in ln and not ln.startswith((" ", "#", "|")):
                    k, v = ln.split(":", 1)
                    kv[k.strip()] = v.strip()
    return kv


def traffic_for(result):
    """HBM bytes per call of the headline op (the sum over its kernels) from the
    committed rocprofv3 counter summary, if its counters were taken on the
    current kernel sources; otherwise None."""
    kv = _traffic_kv()
    if kv.get("source_digest") != source_digest() or kv.get("workload") != result["workload"] \
            or kv.get("op") != result["op"]:
        return None
    try:
        return int(kv["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def op_traffic(workload, op):
    """HBM bytes per call of any measured op from the same summary, gated on a
    digest of every native source; None when the summary is stale or lacks it."""
    kv = _traffic_kv()
    if kv.get("source_digest_all") != source_digest(None):
        return None
    try:
        return int(kv[f"traffic {workload} {op}"])
    except (KeyError, ValueError):
        return None


def stats_summary(path):
    """rocprofv3 --stats kernel table: calls, average / min / max us, share."""
    import csv
    rows = list(csv.DictReader(open(path)))
    print("| kernel | calls | avg us | min us | max us | share |")
    print("|---|---|---|---|---|---|")
    for r in rows:
        print(f"| {_short_kernel(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
              f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
              f"{float(r['Percentage']):.2f}% |")


def main():
    args = parse()
    if args.pmc_summary:
        pmc_summary(args.pmc_summary)
        return
    if args.stats_summary:
        stats_summary(args.stats_summary)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    import paper_2601_07376_amd as L
    L.lib()
    cfgs = [int(c) for c in args.configs.split(",") if c]
    if HEADLINE not in cfgs:
        cfgs = [HEADLINE] + cfgs
    rate = sleep_rate(torch)
    calib = calib_copy()
    calib_m = calib_mfma()
    results, head_case = {}, None
    for c in cfgs:
        r, case = run_workload(c, args.steps, args.warmup, rate)
        results[c] = r
        if c == HEADLINE:
            head_case = case
    for r in results.values():
        t = op_traffic(r["workload"], r["op"])
        r["traffic"] = t
        r["traffic_over_algorithmic"] = None if t is None else round(t / r["op_bytes"], 4)
        for leg in ("linear", "grad_x", "token_loss", "adamw"):
            if leg in r:
                t = op_traffic(r["workload"], r[leg]["op"])
                r[leg]["traffic"] = t
                r[leg]["traffic_over_algorithmic"] = None if t is None else round(t / r[leg]["bytes"], 4)
        r["op_hbm_frac_of_copy"] = r["op_GBps"] / calib["GBps"]
        r["op_mfma_frac_of_calibrated"] = r["op_TFLOPs"] / calib_m["TFLOPs"]
        if "linear" in r:
            r["linear"]["mfma_frac_of_calibrated"] = r["linear"]["TFLOPs"] / calib_m["TFLOPs"]
    h = results[HEADLINE]
    traffic = traffic_for(h)
    roof = dict(bound="hbm",
                kernel=("lora_apply_ids on the decode batch (ids_shrink_kernel + ids_expand_kernel)"
                        if h["op"] == "lora_apply_ids" else
                        "lora_apply on the decode batch (small_shrink_kernel + small_expand_kernel)"),
                achieved=round(h["op_GBps"], 1), peak=HBM_PEAK_GBS, unit="GB/s",
                frac=round(h["op_hbm_frac"], 4), traffic=traffic,
                frac_of_copy=round(h["op_hbm_frac_of_copy"], 4), copy_GBps=round(calib["GBps"], 1),
                bytes_per_launch=h["op_bytes"], avg_launch_us=round(h["op_us_mean"], 3))
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(head_case, args.cpu_seconds)
        log(f"[bench] cpu baseline (oracle): {cpu['value']:.3e} tokens/s on {cpu['cores']} threads")
    line = {
        "metric": "mixed-adapter LoRA tokens/s; decode HBM GB/s and prefill/bwd TFLOP/s vs peak",
        "value": round(h["tokens_per_s"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(h["ms_per_step"], 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "decode_bgmv", "tokens": h["n"], "active_rows": h["n_act"],
                   "adapters": 64, "rank": 16, "d_in": 4096, "d_out": 4096,
                   "y_dtype": "bf16", "parallelism": "none (1 GPU)"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "extra": {"workloads": [results[c] for c in cfgs], "calibration_copy": calib,
                  "calibration_mfma": calib_m, "source_digest": source_digest()},
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()

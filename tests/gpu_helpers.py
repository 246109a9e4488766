"""Helpers for the GPU parity tests: run the HIP path through the binding and
compare with the float64 oracle.  No LoRA arithmetic lives here."""
import sys

import numpy as np
import torch

import oracle
import workloads
from workloads.device import case_to_device, from_torch
from helpers import f64_case

import paper_2601_07376_amd as L

DEV = "cuda"

# spec tolerance: bf16 inputs, float32 accumulation
REL_FRO = 5e-3
MAX_ABS = 3e-2


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def torch_wdtype(case):
    return torch.bfloat16 if case.w_dtype == "bf16" else torch.float32


def make_table(case, dev, debug=False):
    """debug: bind the table (and its plans and ops) to the debug library."""
    t = L.Table(case.num_slots, case.d_in, case.d_out, w_dtype=torch_wdtype(case), device=DEV,
                debug=debug)
    for a in range(case.num_slots):
        if case.ranks[a] > 0:
            t.set(a, dev["A"][a], dev["B"][a], float(case.scales[a]))
    t.upload()
    return t


def make_plan(case, dev, table, segments=False, mask=True, policy=None):
    """policy: dict of lora_policy fields (path selection) or None."""
    m = dev["mask"] if mask else None
    if segments:
        assert policy is None, "path policies apply to plans built from ids"
        return L.Plan(table, seg_offsets=dev["seg_offsets"], seg_adapter=dev["seg_adapter"],
                      n=case.n, mask=m)
    return L.Plan(table, idx=dev["idx"], mask=m, policy=policy)


def compare_plan(got, ref):
    """Bit-exact comparison of exported plan arrays with the oracle's."""
    for k in ("counts", "offsets", "perm", "run_start", "run_len", "run_adapter",
              "m_counts", "m_offsets", "m_perm"):
        g = np.asarray(got[k], np.int64)
        r = np.asarray(ref[k], np.int64)
        assert g.shape == r.shape and np.array_equal(g, r), f"plan array {k} differs"
    assert got["n_runs"] == ref["n_runs"]


def half_ulp_bf16(x):
    x = np.abs(np.asarray(x, np.float64))
    e = np.floor(np.log2(np.maximum(x, 2.0 ** -126)))
    return 2.0 ** (e - 8)


def check_forward(case, Y_out_raw, eff, rows=None, ref_delta=None):
    """Compare Y_out with the oracle on active rows (or the given sample of rows).
    Rows with no adapter must be bit-identical to the input."""
    X, A, B, Y, _ = f64_case(case)
    Yo = workloads.decode(Y_out_raw, case.y_dtype)
    if rows is None:
        rows = np.arange(case.n)
    rows = np.asarray(rows)
    none = rows[eff[rows] < 0]
    assert Y_out_raw[none].tobytes() == case.Y[none].tobytes(), "rows with id -1 changed"
    act = rows[eff[rows] >= 0]
    if act.size == 0:
        return 0.0, 0.0
    if ref_delta is None:
        ref_delta = oracle.delta_rows(eff, X, A, B, case.scales, act)
    got_delta = Yo[act] - Y[act]
    rel = oracle.rel_fro(got_delta, ref_delta)
    if case.y_dtype == "f32":
        mx = oracle.max_abs(got_delta, ref_delta)
        assert rel <= REL_FRO and mx <= MAX_ABS, f"relF {rel:.3g} maxabs {mx:.3g}"
    else:
        # bf16 Y: compare with the exact result rounded to bf16 (the closest
        # storable value); a last-bit flip near a rounding tie is one ulp.
        ref_y = workloads.decode(workloads.encode(Y[act] + ref_delta, "bf16"), "bf16")
        err = Yo[act] - ref_y
        rel = float(np.linalg.norm(err) / max(np.linalg.norm(ref_delta), 1e-300))
        mx = float(np.max(np.abs(err)))
        allow = MAX_ABS + 2.0 * half_ulp_bf16(ref_y)
        assert rel <= REL_FRO, f"relF {rel:.3g}"
        assert np.all(np.abs(err) <= allow), f"max excess {float(np.max(np.abs(err) - allow)):.3g}"
    return rel, mx


def run_apply(case, segments=False, ws=None, policy=None):
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, segments=segments, mask=False, policy=policy)
    Y = dev["Y"].clone()
    L.apply(plan, dev["X"], Y, ws=ws)
    torch.cuda.synchronize()
    return from_torch(Y), plan


def effective(case):
    eff, _ = oracle.effective_ids(case.idx, case.num_slots, case.ranks)
    return eff


def check_grads(case, dA, dB, eff, mask, H_saved=None, tol=(REL_FRO, MAX_ABS)):
    """dA / dB against the oracle, concatenated over slots and per slot (each
    slot's dA and dB together): relF and max-abs within the bar.  A slot with
    no trainable row must hold exact zeros."""
    X, A, B, _, dY = f64_case(case)
    rA, rB = oracle.grad(eff, mask, X, dY, A, B, case.scales, H_saved=H_saved)
    got, ref = [], []
    for a in range(case.num_slots):
        if A[a] is None:
            continue
        ga = dA[a].detach().cpu().double().numpy()
        gb = dB[a].detach().cpu().double().numpy()
        sg = np.concatenate([ga.ravel(), gb.ravel()])
        sr = np.concatenate([rA[a].ravel(), rB[a].ravel()])
        srel, smx = oracle.rel_fro(sg, sr), oracle.max_abs(sg, sr)
        assert srel <= tol[0] and smx <= tol[1], f"slot {a}: grad relF {srel:.3g} maxabs {smx:.3g}"
        if not np.any(sr):
            assert not np.any(sg), f"slot {a} has no trainable row but nonzero gradients"
        got.append(sg)
        ref.append(sr)
    g = np.concatenate(got)
    r = np.concatenate(ref)
    rel, mx = oracle.rel_fro(g, r), oracle.max_abs(g, r)
    assert rel <= tol[0] and mx <= tol[1], f"grad relF {rel:.3g} maxabs {mx:.3g}"
    return rel, mx

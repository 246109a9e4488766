"""The header's limits (GPU): LORA_MAX_SLOTS table slots with ranks 1 to
LORA_MAX_RANK, and LORA_MAX_DIM-wide rows, through every op that takes them,
against the float64 oracle."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_helpers import (DEV, check_forward, check_grads, effective, make_plan, make_table,
                         say)
from helpers import f64_case
from test_gpu_grad_x import check_grad_x
from workloads.device import case_to_device, from_torch, to_torch

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu

MAX_SLOTS, MAX_RANK, MAX_DIM = 1024, 128, 65536


def forward(case, dev, table, policy=None):
    plan = make_plan(case, dev, table, mask=False, policy=policy)
    Y = dev["Y"].clone()
    L.apply(plan, dev["X"], Y)
    torch.cuda.synchronize()
    return from_torch(Y)


@pytest.mark.parametrize("ydt", ["f32", "bf16"])
def test_max_slots(ydt):
    """All 1024 slots live, ranks 1, 8, 24, 64 and 128, about six rows per
    slot (small groups beside a few grouped ones): lora_apply, lora_apply_ids
    on the first 1024 rows, and the masked gradients of every slot."""
    say(f"limits: {MAX_SLOTS} slots, y={ydt}")
    case = workloads.random_case(91, 6000, 256, 264, MAX_SLOTS, rank_choices=(1, 8, 24, 64, MAX_RANK),
                                 frac_none=0.05, mask_p=0.5, want_dy=True, y_dtype=ydt)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    eff = effective(case)
    rel, mx = check_forward(case, forward(case, dev, table), eff)
    say(f"  apply relF {rel:.3g} maxabs {mx:.3g}")
    m = 1024
    Yi = dev["Y"][:m].clone()
    L.apply_ids(table, dev["idx"][:m], dev["X"][:m], Yi)
    torch.cuda.synchronize()
    check_forward(case, np.concatenate([from_torch(Yi), case.Y[m:]]), eff, rows=np.arange(m))
    if ydt == "f32":
        plan = make_plan(case, dev, table, mask=True)
        dA, dB = L.grad(plan, dev["X"], dev["dY"])
        torch.cuda.synchronize()
        rel, mx = check_grads(case, dA, dB, eff, case.mask)
        say(f"  grad relF {rel:.3g} maxabs {mx:.3g}")


def wide_case(seed, d_in, d_out, n=48, y_dtype="f32"):
    return workloads.random_case(seed, n, d_in, d_out, 3, rank_choices=(16, MAX_RANK), frac_none=0.1,
                                 mask_p=0.6, want_dy=True, y_dtype=y_dtype)


@pytest.mark.parametrize("policy", [None, dict(small_max=0)], ids=["small_groups", "grouped"])
def test_max_dim_forward(policy):
    """d_in = d_out = 65536: the small-group kernels (the library's choice
    here) and the grouped 64-row kernels, then lora_apply_ids."""
    say(f"limits: d_in = d_out = {MAX_DIM}, policy {policy}")
    case = wide_case(92, MAX_DIM, MAX_DIM)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    eff = effective(case)
    rel, mx = check_forward(case, forward(case, dev, table, policy), eff)
    say(f"  apply relF {rel:.3g} maxabs {mx:.3g}")
    if policy is None:
        Yi = dev["Y"].clone()
        L.apply_ids(table, dev["idx"], dev["X"], Yi)
        torch.cuda.synchronize()
        check_forward(case, from_torch(Yi), eff)


def test_max_dim_backward():
    """d_in = d_out = 65536: masked adapter gradients and the input gradient."""
    say(f"limits: gradients at d = {MAX_DIM}")
    case = wide_case(93, MAX_DIM, MAX_DIM)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=True)
    dA, dB = L.grad(plan, dev["X"], dev["dY"])
    dx0 = torch.zeros(case.n, case.d_in, dtype=torch.float32, device=DEV)
    dX = dx0.clone()
    L.grad_x(plan, dev["dY"], dX)
    torch.cuda.synchronize()
    rel, mx = check_grads(case, dA, dB, effective(case), case.mask)
    say(f"  grad relF {rel:.3g} maxabs {mx:.3g}")
    check_grad_x(case, dx0.cpu(), dX.cpu())


@pytest.mark.parametrize("d_in,d_out", [(256, MAX_DIM), (MAX_DIM, 264)])
def test_max_dim_linear(d_in, d_out):
    """lora_linear with one side at 65536 (the other small, so W stays 32 MB)."""
    say(f"limits: lora_linear {d_in} -> {d_out}")
    case = workloads.random_case(94, 300, d_in, d_out, 3, rank_choices=(16, 64), layout="segments",
                                 seg_len=(20, 150), frac_none=0.1, y_dtype="bf16")
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=False)
    W_raw = workloads.base_weight(case, dtype="bf16")
    W = to_torch(W_raw, "bf16", DEV)
    Y = torch.empty(case.n, d_out, dtype=torch.bfloat16, device=DEV)
    L.linear(plan, dev["X"], W, Y)
    torch.cuda.synchronize()
    X, A, B, _, _ = f64_case(case)
    Wd = workloads.decode(W_raw, "bf16")
    eff = effective(case)
    ref = oracle.linear(eff, X, Wd, A, B, case.scales)
    got = workloads.decode(from_torch(Y), "bf16")
    rel = oracle.rel_fro(got, ref)
    say(f"  relF {rel:.3g}")
    assert rel <= 5e-3
    assert np.max(np.abs(got - ref)) <= 3e-2 + np.max(np.abs(ref)) * 2.0 ** -8

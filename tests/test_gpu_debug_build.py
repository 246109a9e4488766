"""The debug build (liblora_mi355x_debug.so) on the GPU.

* Clean inputs: every op gives the release library's bytes, and no data flag
  is raised (the kernels' bounds checks have no false positives).
* Overlapping buffers: the op is refused with LORA_ERR_ALIAS and nothing is
  enqueued (the buffers keep their bytes).
* A plan row id out of range (written into the plan with the test hook
  lora_debug_plan_poke): the kernels that read it set LORA_DATA_BOUNDS, which
  lora_plan_check reports.  Every buffer such a case indexes by row has spare
  rows past n, so the planted row n + 3 lies inside its allocation even if a
  check were missing.
"""
import pytest
import torch

import workloads
from gpu_helpers import DEV, make_table, say
from workloads.device import case_to_device, to_torch

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu

ALIAS = 11
SPARE = 16          # rows past n in the poked cases' buffers


def mixed_case():
    """Decode-sized groups beside segments of up to 120 rows, ranks 8-64, a
    loss mask: the small-group and grouped kernels, both gradient stages."""
    return workloads.random_case(41, 600, 512, 384, 9, rank_choices=(8, 16, 32, 64),
                                 layout="segments", seg_len=(1, 120), mask_p=0.4, want_dy=True,
                                 y_dtype="bf16")


def run_all(case, debug, policy):
    dev = case_to_device(case, DEV)
    table = make_table(case, dev, debug=debug)
    plan = L.Plan(table, idx=dev["idx"], mask=dev["mask"], policy=policy)
    out = {}
    Y = dev["Y"].clone()
    L.apply(plan, dev["X"], Y)
    out["apply"] = Y
    Yi = dev["Y"].clone()
    L.apply_ids(table, dev["idx"], dev["X"], Yi)
    out["apply_ids"] = Yi
    H = L.shrink(plan, dev["X"])
    out["shrink"] = H
    Ye = dev["Y"].clone()
    L.expand(plan, H, Ye)
    out["expand"] = Ye
    W = to_torch(workloads.base_weight(case), "bf16", DEV)
    Yl = torch.empty_like(dev["Y"])
    L.linear(plan, dev["X"], W, Yl)
    out["linear"] = Yl
    dA, dB = L.grad(plan, dev["X"], dev["dY"])
    out["grad"] = torch.cat([g.flatten() for g in dA + dB if g is not None])
    dX = torch.zeros(case.n, case.d_in, dtype=torch.float32, device=DEV)
    L.grad_x(plan, dev["dY"], dX)
    out["grad_x"] = dX
    dX2 = torch.zeros_like(dX)
    bA, bB, _ = L.backward(plan, dev["X"], dev["dY"], dX2)
    out["backward"] = torch.cat([g.flatten() for g in bA + bB if g is not None] + [dX2.flatten()])
    torch.cuda.synchronize()
    return out, plan.check()


# every group small (the library's choice at 600 rows), small groups beside
# grouped ones (with and without the second stream), every group grouped
POLICIES = [None, dict(small_max=16), dict(small_max=16, fork=1), dict(small_max=0)]


@pytest.mark.parametrize("policy", POLICIES, ids=["default", "mixed", "mixed_fork", "grouped"])
def test_debug_build_matches_release(policy):
    say(f"debug build: every op against the release library, no flag, policy {policy}")
    case = mixed_case()
    rel, rflags = run_all(case, False, policy)
    dbg, dflags = run_all(case, True, policy)
    assert rflags == 0 and dflags == 0, (rflags, dflags)
    for k in rel:
        assert torch.equal(rel[k].view(torch.uint8) if rel[k].dtype == torch.bfloat16 else rel[k],
                           dbg[k].view(torch.uint8) if dbg[k].dtype == torch.bfloat16 else dbg[k]), k


def test_debug_build_refuses_overlaps():
    say("debug build: overlapping outputs refused, nothing enqueued")
    case = mixed_case()
    dev = case_to_device(case, DEV)
    table = make_table(case, dev, debug=True)
    plan = L.Plan(table, idx=dev["idx"], mask=dev["mask"])
    X0 = dev["X"].clone()
    with pytest.raises(L.LoraError) as e:               # Y over X's first columns
        L.apply(plan, dev["X"], dev["X"][:, :case.d_out])
    assert e.value.status == ALIAS and "Y overlaps X" in str(e.value)
    with pytest.raises(L.LoraError) as e:
        L.apply_ids(table, dev["idx"], dev["X"], dev["X"][:, :case.d_out])
    assert e.value.status == ALIAS
    live = [a for a in range(case.num_slots) if case.ranks[a] > 0]
    a, b = live[0], live[1]
    buf = torch.zeros(4 << 20, dtype=torch.float32, device=DEV)
    dA = [None] * case.num_slots
    dB = [None] * case.num_slots
    dA[a] = buf[:case.ranks[a] * case.d_in].view(case.ranks[a], case.d_in)
    dB[b] = buf[:case.d_out * case.ranks[b]].view(case.d_out, case.ranks[b])   # over dA[a]
    with pytest.raises(L.LoraError) as e:
        L.grad(plan, dev["X"], dev["dY"], dA=dA, dB=dB)
    assert e.value.status == ALIAS and "of slot" in str(e.value)
    # dX and the backward's workspace in one buffer, the workspace 4 KB in
    need = L.backward_workspace(plan).numel()
    big = torch.zeros(case.n * case.d_in + (need + 4096) // 4 + 4, dtype=torch.float32, device=DEV)
    dXw = big[:case.n * case.d_in].view(case.n, case.d_in)
    ws = big.view(torch.uint8)[4096:4096 + need]
    with pytest.raises(L.LoraError) as e:
        L.backward(plan, dev["X"], dev["dY"], dXw, ws=ws)
    assert e.value.status == ALIAS and "dX" in str(e.value)
    torch.cuda.synchronize()
    assert torch.equal(dev["X"].view(torch.uint8), X0.view(torch.uint8))
    assert float(buf.abs().sum()) == 0.0 and float(big.abs().sum()) == 0.0
    assert plan.check() == 0


def padded(t, rows):
    """t's rows at the top of a buffer with `rows` spare rows (zeros) after them."""
    p = torch.zeros(t.shape[0] + rows, t.shape[1], dtype=t.dtype, device=t.device)
    p[:t.shape[0]] = t
    return p


def grouped_case(seed=43):
    """Three adapters in segments of 100-300 rows: every group on the grouped
    (plan-indexed) kernels."""
    return workloads.random_case(seed, 600, 256, 256, 3, rank_choices=(16,), layout="segments",
                                 seg_len=(100, 300), mask_p=0.5, want_dy=True, y_dtype="f32")


def poked(case, array, policy=None):
    """A debug-library plan of `case` whose row id 0 of `array` is n + 3, and
    the case's buffers with SPARE spare rows."""
    dev = case_to_device(case, DEV)
    table = make_table(case, dev, debug=True)
    plan = L.Plan(table, idx=dev["idx"], mask=dev["mask"], policy=policy)
    torch.cuda.synchronize()
    assert plan.check() == 0
    plan.debug_poke(array, 0, case.n + 3)
    bufs = {k: padded(dev[k], SPARE) for k in ("X", "Y", "dY") if dev[k] is not None}
    return dev, table, plan, bufs


@pytest.mark.parametrize("op", ["apply", "shrink", "expand", "linear"])
def test_bounds_flag_on_bad_perm(op):
    say(f"debug build: perm[0] = n + 3 through {op}")
    case = grouped_case()
    n = case.n
    dev, table, plan, b = poked(case, L.LORA_PLAN_PERM, policy=dict(small_max=0))
    X, Y = b["X"][:n], b["Y"][:n]
    if op == "apply":
        L.apply(plan, X, Y)
    elif op == "shrink":
        H = torch.zeros(n + SPARE, 16, dtype=torch.float32, device=DEV)
        L.shrink(plan, X, H=H[:n])
    elif op == "expand":
        H = torch.zeros(n + SPARE, 16, dtype=torch.float32, device=DEV)
        L.expand(plan, H[:n], Y)
    else:
        W = to_torch(workloads.base_weight(case, dtype="bf16"), "bf16", DEV)
        Yb = torch.zeros(n + SPARE, case.d_out, dtype=torch.bfloat16, device=DEV)
        L.linear(plan, X, W, Yb[:n])
    torch.cuda.synchronize()
    assert plan.check() & L.LORA_DATA_BOUNDS


@pytest.mark.parametrize("op", ["grad", "grad_x", "backward"])
def test_bounds_flag_on_bad_m_perm(op):
    say(f"debug build: m_perm[0] = n + 3 through {op}")
    case = grouped_case(44)
    n = case.n
    dev, table, plan, b = poked(case, L.LORA_PLAN_M_PERM)
    X, dY = b["X"][:n], b["dY"][:n]
    dX = torch.zeros(n + SPARE, case.d_in, dtype=torch.float32, device=DEV)
    if op == "grad":
        L.grad(plan, X, dY)
    elif op == "grad_x":
        L.grad_x(plan, dY, dX[:n])
    else:
        L.backward(plan, X, dY, dX[:n])
    torch.cuda.synchronize()
    assert plan.check() & L.LORA_DATA_BOUNDS


@pytest.mark.parametrize("split", [0, 1])
def test_bounds_flag_on_bad_small_record_row(split):
    say(f"debug build: small record row 0 = n + 3, small_split {split}")
    case = workloads.random_case(45, 64, 1024, 512, 8, rank_choices=(16,), y_dtype="f32")
    n = case.n
    dev, table, plan, b = poked(case, L.LORA_PLAN_SMALL_ROW,
                                policy=dict(small_max=16, small_split=split))
    L.apply(plan, b["X"][:n], b["Y"][:n])
    torch.cuda.synchronize()
    assert plan.check() & L.LORA_DATA_BOUNDS

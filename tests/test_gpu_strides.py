"""Leading dimensions wider than the rows (GPU).

Every op takes its matrices as row-major with a leading dimension of its own
(a multiple of 8).  Here each op runs twice on the same values: once on
contiguous tensors, once on column views of wider buffers (each matrix with its
own padding), and the two results must be the same bits, since the arithmetic
does not depend on where the rows start.  The padding columns of inputs hold
NaN (an op that read them would spread it) and those of outputs hold a sentinel
that must come back unchanged.  One result per op family is also held to the
oracle bar, so the pair cannot agree on a wrong answer.  The widths are
ragged (multiples of 8, not of the kernels' 32- or 64-wide steps), so every
tail path runs next to the NaN padding.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_helpers import DEV, MAX_ABS, REL_FRO, check_forward, check_grads, effective, make_plan, \
    make_table, say
from helpers import f64_case
from workloads.device import case_to_device, from_torch

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu

# extra columns per matrix (multiples of 8, all different)
PAD = dict(X=24, Y=40, dY=16, dX=56, H=8, W=32)
SENTINEL = 7.0


def wide(t, pad, fill):
    """(buffer, view): t as the left columns of a buffer `pad` columns wider
    whose other columns hold `fill`."""
    buf = torch.full((t.shape[0], t.shape[1] + pad), fill, dtype=t.dtype, device=t.device)
    buf[:, :t.shape[1]] = t
    view = buf[:, :t.shape[1]]
    assert view.stride(0) == t.shape[1] + pad and view.stride(1) == 1
    return buf, view


def bits(t):
    t = t.detach().cpu().contiguous()
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).numpy()


def same_bits(a, b, what):
    assert np.array_equal(bits(a), bits(b)), f"{what}: strided result differs from the contiguous one"


def pad_intact(buf, cols, fill, what):
    rest = buf[:, cols:]
    assert bool(torch.all(rest == fill)), f"{what}: a padding column was written"


def fwd_case(seed, n, y_dtype, seg_len=(1, 400)):
    return workloads.random_case(seed, n, 1032, 776, 12, rank_choices=(8, 16, 32, 64),
                                 layout="segments", seg_len=seg_len, y_dtype=y_dtype)


APPLY = [
    # (name, n, segment lengths, policy): every forward kernel family
    ("small_split", 700, (1, 12), None),
    ("small_fused", 700, (1, 12), dict(small_split=0)),
    ("mixed_fork_fine", 3000, (1, 300), dict(small_max=32, fork=1)),
    ("coarse", 3000, (200, 800), dict(small_max=0, block_rows=256)),
]


@pytest.mark.parametrize("ydt", ["f32", "bf16"])
@pytest.mark.parametrize("name,n,seg,policy", APPLY, ids=[a[0] for a in APPLY])
def test_apply_strided(name, n, seg, policy, ydt):
    say(f"strided apply {name} y={ydt}")
    case = fwd_case(11, n, ydt, seg)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=False, policy=policy)
    Yc = dev["Y"].clone()
    L.apply(plan, dev["X"], Yc)
    _, Xv = wide(dev["X"], PAD["X"], float("nan"))
    Yb, Yv = wide(dev["Y"], PAD["Y"], SENTINEL)
    L.apply(plan, Xv, Yv)
    torch.cuda.synchronize()
    same_bits(Yv, Yc, "Y")
    pad_intact(Yb, case.d_out, SENTINEL, "Y")
    rel, mx = check_forward(case, from_torch(Yv.contiguous()), effective(case))
    say(f"  relF {rel:.3g} maxabs {mx:.3g}")


def test_shrink_expand_strided():
    say("strided shrink / expand")
    case = fwd_case(12, 3000, "f32", (200, 800))
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=False)
    Hc = L.shrink(plan, dev["X"])                 # H starts as zeros
    _, Xv = wide(dev["X"], PAD["X"], float("nan"))
    Hb, Hv = wide(torch.zeros_like(Hc), PAD["H"], SENTINEL)
    L.shrink(plan, Xv, H=Hv)
    torch.cuda.synchronize()
    same_bits(Hv, Hc, "H")
    pad_intact(Hb, Hc.shape[1], SENTINEL, "H")
    Yc = dev["Y"].clone()
    L.expand(plan, Hc, Yc)
    Yb, Yv = wide(dev["Y"], PAD["Y"], SENTINEL)
    _, Hv2 = wide(Hc, PAD["H"], float("nan"))
    L.expand(plan, Hv2, Yv)
    torch.cuda.synchronize()
    same_bits(Yv, Yc, "Y")
    pad_intact(Yb, case.d_out, SENTINEL, "Y")
    check_forward(case, from_torch(Yv.contiguous()), effective(case))


@pytest.mark.parametrize("ydt", ["f32", "bf16"])
def test_apply_ids_strided(ydt):
    say(f"strided apply_ids y={ydt}")
    case = workloads.random_case(13, 256, 1032, 776, 24, rank_choices=(8, 16, 32), y_dtype=ydt)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    Yc = dev["Y"].clone()
    L.apply_ids(table, dev["idx"], dev["X"], Yc)
    _, Xv = wide(dev["X"], PAD["X"], float("nan"))
    Yb, Yv = wide(dev["Y"], PAD["Y"], SENTINEL)
    L.apply_ids(table, dev["idx"], Xv, Yv)
    torch.cuda.synchronize()
    same_bits(Yv, Yc, "Y")
    pad_intact(Yb, case.d_out, SENTINEL, "Y")
    check_forward(case, from_torch(Yv.contiguous()), effective(case))


@pytest.mark.parametrize("ydt", ["f32", "bf16"])
def test_linear_strided(ydt):
    say(f"strided linear y={ydt}")
    case = workloads.random_case(14, 600, 520, 776, 6, rank_choices=(16, 32), layout="segments",
                                 seg_len=(40, 200), y_dtype=ydt)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=False)
    W = torch.from_numpy(workloads.base_weight(case, dtype="bf16").view(np.int16)).to(DEV) \
        .view(torch.bfloat16)
    Yc = torch.zeros_like(dev["Y"])
    L.linear(plan, dev["X"], W, Yc)
    _, Xv = wide(dev["X"], PAD["X"], float("nan"))
    _, Wv = wide(W, PAD["W"], float("nan"))
    Yb, Yv = wide(torch.zeros_like(dev["Y"]), PAD["Y"], SENTINEL)
    L.linear(plan, Xv, Wv, Yv)
    torch.cuda.synchronize()
    same_bits(Yv, Yc, "Y")
    pad_intact(Yb, case.d_out, SENTINEL, "Y")
    # against X W^T + Delta in float64
    X, A, B, _, _ = f64_case(case)
    Wd = workloads.decode(workloads.base_weight(case, dtype="bf16"), "bf16")
    eff = effective(case)
    ref = X @ Wd.T
    act = np.nonzero(eff >= 0)[0]
    ref[act] += oracle.delta_rows(eff, X, A, B, case.scales, act)
    got = Yv.float().cpu().double().numpy()
    rel = oracle.rel_fro(got, ref)
    assert rel <= REL_FRO, rel


def grad_case(seed):
    return workloads.random_case(seed, 2000, 776, 1032, 6, rank_choices=(8, 16, 32),
                                 layout="segments", seg_len=(50, 500), mask_p=0.4, want_dy=True)


@pytest.mark.parametrize("h_saved", [False, True])
def test_grad_strided(h_saved):
    say(f"strided grad h_saved={h_saved}")
    case = grad_case(15)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=True)
    Hc = L.shrink(plan, dev["X"]) if h_saved else None
    dA0, dB0 = L.grad(plan, dev["X"], dev["dY"], H_saved=Hc)
    _, Xv = wide(dev["X"], PAD["X"], float("nan"))
    _, dYv = wide(dev["dY"], PAD["dY"], float("nan"))
    Hv = None
    if h_saved:
        _, Hv = wide(Hc, PAD["H"], float("nan"))
    dA1, dB1 = L.grad(plan, Xv, dYv, H_saved=Hv)
    torch.cuda.synchronize()
    for a in range(case.num_slots):
        if dA0[a] is not None:
            same_bits(dA1[a], dA0[a], f"dA of slot {a}")
            same_bits(dB1[a], dB0[a], f"dB of slot {a}")
    H64 = Hc.double().cpu().numpy() if h_saved else None
    check_grads(case, dA1, dB1, effective(case), case.mask, H_saved=H64)


@pytest.mark.parametrize("dxt", [torch.float32, torch.bfloat16])
def test_grad_x_and_backward_strided(dxt):
    say(f"strided grad_x / backward dX={dxt}")
    case = grad_case(16)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=True)
    g = torch.Generator().manual_seed(3)
    dx0 = torch.randn(case.n, case.d_in, generator=g).to(dxt).to(DEV)
    _, dYv = wide(dev["dY"], PAD["dY"], float("nan"))
    _, Xv = wide(dev["X"], PAD["X"], float("nan"))
    # input gradient alone
    dXc = dx0.clone()
    L.grad_x(plan, dev["dY"], dXc)
    dXb, dXv = wide(dx0, PAD["dX"], SENTINEL)
    L.grad_x(plan, dYv, dXv)
    torch.cuda.synchronize()
    same_bits(dXv, dXc, "dX")
    pad_intact(dXb, case.d_in, SENTINEL, "dX")
    # both gradients in one call
    dXc2 = dx0.clone()
    dA0, dB0, _ = L.backward(plan, dev["X"], dev["dY"], dXc2)
    dXb2, dXv2 = wide(dx0, PAD["dX"], SENTINEL)
    dA1, dB1, _ = L.backward(plan, Xv, dYv, dXv2)
    torch.cuda.synchronize()
    same_bits(dXv2, dXc2, "dX (backward)")
    same_bits(dXv2, dXc, "dX (backward against grad_x)")
    pad_intact(dXb2, case.d_in, SENTINEL, "dX (backward)")
    for a in range(case.num_slots):
        if dA0[a] is not None:
            same_bits(dA1[a], dA0[a], f"dA of slot {a}")
            same_bits(dB1[a], dB0[a], f"dB of slot {a}")
    # the strided input gradient against the oracle
    X, A, B, _, dY = f64_case(case)
    eff = effective(case)
    base = dx0.double().cpu().numpy()
    ref = oracle.grad_x(eff, case.mask, dY, A, B, case.scales, base)
    sel = (eff >= 0) & (np.asarray(case.mask) != 0)
    got = dXv.double().cpu().numpy()
    d_got, d_ref = got[sel] - base[sel], ref[sel] - base[sel]
    rel = oracle.rel_fro(d_got, d_ref)
    assert rel <= REL_FRO, rel
    if dxt == torch.float32:
        assert oracle.max_abs(d_got, d_ref) <= MAX_ABS

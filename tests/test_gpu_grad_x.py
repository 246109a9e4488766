"""Input gradient lora_grad_x vs the float64 oracle (GPU).

dX[t] += s_a (dY_t B_a) A_a over the masked rows T_a^m; every other row must
come back bit-identical.  Parity bar as for the forward: relF <= 5e-3 and
max-abs <= 3e-2 on the update over T_a^m (float32 dX), bit-exact on
integer-valued inputs.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_helpers import DEV, MAX_ABS, REL_FRO, effective, make_plan, make_table, say
from helpers import f64_case
from workloads.device import case_to_device

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu


def _dx0(case, dtype=torch.float32, seed=0):
    g = torch.Generator().manual_seed(seed)
    return torch.randn(case.n, case.d_in, generator=g).to(dtype)


def _bits(t):
    return (t.view(torch.int16) if t.dtype == torch.bfloat16 else t).numpy()


def run_grad_x(case, dx0, segments=False, dY=None):
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, segments=segments, mask=True)
    dX = dx0.to(DEV).clone()
    L.grad_x(plan, dev["dY"] if dY is None else dY.to(DEV), dX)
    torch.cuda.synchronize()
    return dX.cpu()


def check_grad_x(case, dx0, got, dY64=None, exact=False):
    X, A, B, _, dY = f64_case(case)
    if dY64 is not None:
        dY = dY64
    eff = effective(case)
    base = dx0.double().numpy()
    ref = oracle.grad_x(eff, case.mask, dY, A, B, case.scales, base)
    sel = eff >= 0
    if case.mask is not None:
        sel = sel & (np.asarray(case.mask) != 0)
    g = got.double().numpy()
    # rows outside T_a^m: bit-identical
    assert _bits(got)[~sel].tobytes() == _bits(dx0)[~sel].tobytes()
    if exact:
        assert np.array_equal(g[sel], ref[sel])
        return 0.0, 0.0
    d_got, d_ref = g[sel] - base[sel], ref[sel] - base[sel]
    rel, mx = oracle.rel_fro(d_got, d_ref), oracle.max_abs(d_got, d_ref)
    if got.dtype == torch.bfloat16:
        ulp = np.abs(ref[sel]) * 2.0 ** -8            # half a bf16 ulp of the result, generously
        assert np.all(np.abs(g[sel] - ref[sel]) <= MAX_ABS + ulp)
        assert rel <= REL_FRO
    else:
        assert rel <= REL_FRO and mx <= MAX_ABS, (rel, mx)
    return rel, mx


def test_grad_x_config5_full():
    say("grad_x config 5")
    case = workloads.make_config(5)
    dx0 = _dx0(case)
    got = run_grad_x(case, dx0)
    rel, mx = check_grad_x(case, dx0, got)
    say(f"  relF {rel:.3g} maxabs {mx:.3g}")
    again = run_grad_x(case, dx0, segments=True)   # deterministic, and segments == indices
    assert _bits(got).tobytes() == _bits(again).tobytes()


FUZZ = [
    ("ragged", dict(n=1000, d_in=264, d_out=136, num_slots=5, rank_choices=(8, 16, 32),
                    layout="segments", seg_len=(1, 150), mask_p=0.4)),
    ("odd_ranks", dict(n=700, d_in=128, d_out=200, num_slots=6, rank_choices=(1, 5, 12, 33),
                       mask_p=0.7)),
    ("rank128", dict(n=900, d_in=1024, d_out=1024, num_slots=3, rank_choices=(128,),
                     layout="segments", seg_len=(40, 300), mask_p=0.3)),
    ("rank64_mixed", dict(n=1500, d_in=520, d_out=264, num_slots=9, rank_choices=(8, 40, 64),
                          layout="segments", seg_len=(1, 200), mask_p=0.5)),
    ("sparse_mask", dict(n=2000, d_in=512, d_out=512, num_slots=40, rank_choices=(16, 64),
                         mask_p=0.02)),
    ("many_slots", dict(n=3000, d_in=256, d_out=256, num_slots=150, rank_choices=(8, 16),
                        mask_p=0.5)),
    ("decode_like", dict(n=256, d_in=4096, d_out=4096, num_slots=64, rank_choices=(16,),
                         mask_p=0.9)),
    ("no_mask_rows", dict(n=300, d_in=64, d_out=72, num_slots=4, rank_choices=(16,),
                          mask_p=0.0)),
]


@pytest.mark.parametrize("name", [f[0] for f in FUZZ])
def test_grad_x_fuzz(name):
    kw = next(f[1] for f in FUZZ if f[0] == name)
    say(f"grad_x fuzz {name}")
    case = workloads.random_case(31, want_dy=True, want_y=False, **kw)
    dx0 = _dx0(case, seed=1)
    got = run_grad_x(case, dx0)
    rel, mx = check_grad_x(case, dx0, got)
    say(f"  relF {rel:.3g} maxabs {mx:.3g}")


def test_grad_x_bf16_dx():
    say("grad_x bf16 dX")
    case = workloads.random_case(32, 1200, 384, 520, 7, rank_choices=(16, 32), layout="segments",
                                 seg_len=(1, 300), mask_p=0.5, want_dy=True, want_y=False)
    dx0 = _dx0(case, dtype=torch.bfloat16, seed=2)
    got = run_grad_x(case, dx0)
    check_grad_x(case, dx0, got)


def test_grad_x_integer_exact():
    """{-1, 0, 1} inputs and power-of-two scales: every partial sum is an exact
    float32 integer, so any summation order gives the oracle's bits."""
    say("grad_x integer exact")
    case = workloads.random_case(33, 600, 128, 256, 4, rank_choices=(8, 16, 48), mask_p=0.6,
                                 want_dy=True, want_y=False, int_values=True,
                                 scales=[0.25, 0.5, 1.0, 2.0])
    dx0 = torch.from_numpy(np.random.default_rng(3).integers(-4, 5, (case.n, case.d_in))
                           .astype(np.float32))
    got = run_grad_x(case, dx0)
    check_grad_x(case, dx0, got, exact=True)


def test_grad_x_masked_rows_never_read():
    """NaN / Inf in the dY rows of masked-out and id -1 rows change nothing."""
    say("grad_x masked rows")
    case = workloads.random_case(34, 500, 256, 128, 5, rank_choices=(16,), mask_p=0.5,
                                 frac_none=0.2, want_dy=True, want_y=False)
    dx0 = _dx0(case, seed=4)
    clean = run_grad_x(case, dx0)
    eff = effective(case)
    out = (np.asarray(case.mask) == 0) | (eff < 0)
    dev = case_to_device(case, DEV)
    dY = dev["dY"].clone()
    rows = torch.from_numpy(np.nonzero(out)[0]).to(DEV)
    dY[rows] = torch.tensor(float("nan"), dtype=dY.dtype, device=DEV)
    dY[rows[::2]] = torch.tensor(float("inf"), dtype=dY.dtype, device=DEV)
    junk = run_grad_x(case, dx0, dY=dY)
    assert _bits(junk).tobytes() == _bits(clean).tobytes()


def test_grad_x_table_reupload():
    """The input gradient follows the table as last uploaded: empty slots
    between live ones, then a re-upload with other ranks, weights and scales
    on the same table object, each checked against the oracle."""
    say("grad_x table re-upload")
    kw = dict(mask_p=0.5, want_dy=True, want_y=False, layout="segments", seg_len=(1, 120))
    c1 = workloads.random_case(37, 800, 200, 136, 6, ranks=[16, 0, 64, 8, 0, 33], **kw)
    dev1 = case_to_device(c1, DEV)
    table = make_table(c1, dev1)
    dx0 = _dx0(c1, seed=5)
    dX = dx0.to(DEV).clone()
    L.grad_x(make_plan(c1, dev1, table), dev1["dY"], dX)
    torch.cuda.synchronize()
    check_grad_x(c1, dx0, dX.cpu())
    c2 = workloads.random_case(38, 800, 200, 136, 6, ranks=[128, 24, 0, 8, 40, 0], **kw)
    dev2 = case_to_device(c2, DEV)
    for a in range(c2.num_slots):
        if c2.ranks[a] > 0:
            table.set(a, dev2["A"][a], dev2["B"][a], float(c2.scales[a]))
        else:
            table.clear(a)
    table.upload()
    dX = dx0.to(DEV).clone()
    L.grad_x(make_plan(c2, dev2, table), dev2["dY"], dX)
    torch.cuda.synchronize()
    check_grad_x(c2, dx0, dX.cpu())


def test_grad_x_empty_batch_and_dtype_errors():
    case = workloads.random_case(35, 0, 64, 64, 3, rank_choices=(8,), mask_p=0.5, want_dy=True,
                                 want_y=False)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=True)
    dX = torch.empty(0, case.d_in, device=DEV)
    L.grad_x(plan, dev["dY"], dX)                 # n = 0: nothing to do
    case = workloads.random_case(36, 40, 64, 64, 3, rank_choices=(8,), mask_p=0.5,
                                 want_dy=True, want_y=False)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=True)
    dX = torch.zeros(case.n, case.d_in, device=DEV)
    with pytest.raises(L.LoraError):
        L.grad_x(plan, dev["dY"].float(), dX)     # float32 dY: the matrix-core path only

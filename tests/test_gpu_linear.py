"""The whole adapted layer, lora_linear: Y = X W^T + s_a (X A_a^T) B_a^T (rows
with no adapter: X W^T), against the float64 oracle (GPU).

Graded parity uses float32 Y: relative Frobenius error <= 5e-3 and max-abs
<= 3e-2 over the whole output (bf16 X, W and adapter weights, float32
accumulation).  bfloat16 Y is compared with the exact result rounded to
bfloat16, within 3e-2 plus one bf16 ulp.  Integer-valued inputs must match bit
for bit.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_helpers import DEV, MAX_ABS, REL_FRO, effective, half_ulp_bf16, make_plan, make_table, say
from helpers import f64_case
from workloads.device import case_to_device, from_torch

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu


def run_linear(case, W_raw, y_dtype, segments=False, policy=None):
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, segments=segments, mask=False, policy=policy)
    W = torch.from_numpy(W_raw.view(np.int16)).to(DEV).view(torch.bfloat16)
    tdt = torch.float32 if y_dtype == "f32" else torch.bfloat16
    Y = torch.full((case.n, case.d_out), float("nan"), dtype=tdt, device=DEV)
    L.linear(plan, dev["X"], W, Y)
    torch.cuda.synchronize()
    return Y.cpu()


def check_linear(case, W_raw, Y, rows=None):
    X, A, B, _, _ = f64_case(case)
    W = workloads.decode(W_raw, "bf16")
    eff = effective(case)
    if rows is None:
        ref = oracle.linear(eff, X, W, A, B, case.scales)
        got = Y.double().numpy()
    else:
        ref = oracle.linear_rows(eff, X, W, A, B, case.scales, rows)
        got = Y.double().numpy()[rows]
    if Y.dtype == torch.float32:
        rel, mx = oracle.rel_fro(got, ref), oracle.max_abs(got, ref)
        assert rel <= REL_FRO and mx <= MAX_ABS, f"relF {rel:.3g} maxabs {mx:.3g}"
    else:
        ref_b = workloads.decode(workloads.encode(ref, "bf16"), "bf16")
        err = got - ref_b
        rel = float(np.linalg.norm(err) / max(np.linalg.norm(ref), 1e-300))
        mx = float(np.max(np.abs(err))) if err.size else 0.0
        assert rel <= REL_FRO, f"relF {rel:.3g}"
        allow = MAX_ABS + 2.0 * half_ulp_bf16(ref_b)
        assert np.all(np.abs(err) <= allow), f"max excess {float(np.max(np.abs(err) - allow)):.3g}"
    return rel, mx


def test_linear_config3_every_row_f32():
    """The prefill workload's layer (15.8k rows, 4096 -> 14336, 32 adapters of
    rank 64) in float32 Y, every element against the oracle."""
    say("linear config 3 f32, every row")
    case = workloads.make_config(3, y_dtype="f32")
    W = workloads.base_weight(case)
    Y = run_linear(case, W, "f32", segments=True)
    rel, mx = check_linear(case, W, Y)
    say(f"  relF {rel:.3g} maxabs {mx:.3g}")


def test_linear_config3_sampled_bf16():
    say("linear config 3 bf16, sampled rows")
    case = workloads.make_config(3, y_dtype="bf16")
    W = workloads.base_weight(case)
    Y = run_linear(case, W, "bf16", segments=True)
    rng = np.random.default_rng(4)
    rows = np.unique(np.concatenate([rng.choice(case.n, 300, replace=False),
                                     case.seg_offsets[:-1], case.seg_offsets[1:] - 1,
                                     np.arange(case.n - 40, case.n)]))
    rel, mx = check_linear(case, W, Y, rows=rows)
    say(f"  relF {rel:.3g} maxabs {mx:.3g}")


FUZZ = [
    # ragged in every dimension: n, d_in (K tail), d_out (column tail)
    ("ragged_segments", dict(n=1000, d_in=1032, d_out=520, num_slots=7,
                             rank_choices=(8, 16, 32, 64), layout="segments", seg_len=(1, 300))),
    ("odd_ranks", dict(n=777, d_in=264, d_out=296, num_slots=5, rank_choices=(1, 5, 12, 33),
                       layout="segments", seg_len=(20, 200))),
    ("rank128", dict(n=600, d_in=512, d_out=768, num_slots=3, rank_choices=(128,),
                     layout="segments", seg_len=(50, 300))),
    ("decode_ids", dict(n=300, d_in=256, d_out=264, num_slots=20, rank_choices=(16,))),
    ("single_adapter", dict(n=513, d_in=128, d_out=256, num_slots=1, rank_choices=(64,),
                            layout="single", frac_none=0.0)),
    ("all_none", dict(n=257, d_in=200, d_out=136, num_slots=3, frac_none=1.0)),
    ("tiny", dict(n=5, d_in=8, d_out=8, num_slots=2, rank_choices=(8,))),
]


@pytest.mark.parametrize("ydt", ["f32", "bf16"])
@pytest.mark.parametrize("name", [f[0] for f in FUZZ])
def test_linear_fuzz(name, ydt):
    kw = dict(FUZZ)[name]
    say(f"linear fuzz {name} y={ydt}")
    case = workloads.random_case(41, y_dtype=ydt, **kw)
    W = workloads.base_weight(case)
    Y = run_linear(case, W, ydt)
    check_linear(case, W, Y)


@pytest.mark.parametrize("small", [None, 0])
def test_linear_integer_exact(small):
    """Values in {-1, 0, 1}: every partial sum is an exact float32 integer and
    s_a H splits exactly into hi + lo, so Y must equal the oracle bit for bit."""
    say(f"linear integer small={small}")
    case = workloads.random_case(43, 1100, 264, 136, 7, rank_choices=(8, 16, 40, 64),
                                 layout="segments", seg_len=(1, 90), y_dtype="f32",
                                 int_values=True, scales=[0.25, 0.5, 1, 2, 2, 1, 0.5])
    W = workloads.base_weight(case, int_values=True)
    Y = run_linear(case, W, "f32", policy=None if small is None else dict(small_max=small))
    X, A, B, _, _ = f64_case(case)
    ref = oracle.linear(effective(case), X, workloads.decode(W, "bf16"), A, B, case.scales)
    assert np.array_equal(Y.double().numpy(), ref)


def test_linear_zero_base_equals_residual():
    """W = 0: the layer is the residual alone, which lora_apply adds to Y = 0."""
    say("linear W = 0")
    case = workloads.random_case(44, 900, 512, 264, 6, rank_choices=(16, 32, 64),
                                 layout="segments", seg_len=(1, 200), y_dtype="f32")
    W = np.zeros((case.d_out, case.d_in), np.uint16)
    Y = run_linear(case, W, "f32")
    check_linear(case, W, Y)
    eff = effective(case)
    assert np.all(Y.numpy()[eff < 0] == 0.0)


def test_linear_rejects_and_empty():
    say("linear argument errors and n = 0")
    case = workloads.random_case(45, 0, 64, 64, 2, rank_choices=(8,), y_dtype="f32")
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=False)
    W = torch.zeros(64, 64, dtype=torch.bfloat16, device=DEV)
    L.linear(plan, dev["X"], W, torch.empty(0, 64, device=DEV))      # n = 0: nothing to do
    case = workloads.random_case(46, 40, 64, 64, 2, rank_choices=(8,), y_dtype="f32")
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=False)
    Y = torch.full((40, 64), 3.0, device=DEV)
    with pytest.raises(L.LoraError):                                   # float32 W
        L.linear(plan, dev["X"], W.float(), Y)
    with pytest.raises(L.LoraError):                                   # ldw 32 < d_in 64
        L.linear(plan, dev["X"], torch.zeros(64, 32, dtype=torch.bfloat16, device=DEV), Y)
    torch.cuda.synchronize()
    assert torch.all(Y == 3.0)

"""Plan-free small batches: lora_apply_ids vs the float64 oracle and vs
lora_apply's split small-group path (GPU).

lora_apply_ids finds each slot's rows inside its kernels, with the same 16-row
tiles, d-slices and column chunks as the split path of lora_apply, so the two
must agree bit for bit; the oracle bounds are those of the forward tests.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_helpers import DEV, check_forward, effective, make_plan, make_table, say
from helpers import f64_case
from workloads.device import case_to_device, from_torch

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu


def run_ids(case, dev=None):
    dev = dev or case_to_device(case, DEV)
    table = make_table(case, dev)
    Y = dev["Y"].clone()
    L.apply_ids(table, dev["idx"], dev["X"], Y)
    torch.cuda.synchronize()
    return from_torch(Y), table, dev


def run_split(case, dev, table):
    plan = make_plan(case, dev, table, mask=False, policy=dict(small_max=100000, small_split=1))
    Y = dev["Y"].clone()
    L.apply(plan, dev["X"], Y)
    torch.cuda.synchronize()
    return from_torch(Y)


def with_bad_ids(case, seed):
    """Ids past the table and below -1 on a few rows (they must be ignored)."""
    rng = np.random.default_rng(seed)
    idx = case.idx.copy()
    k = max(1, case.n // 16)
    rows = rng.choice(case.n, size=min(k, case.n), replace=False)
    idx[rows[::2]] = case.num_slots + rng.integers(0, 5, size=len(rows[::2]))
    idx[rows[1::2]] = -2 - rng.integers(0, 5, size=len(rows[1::2]))
    case.idx = idx
    return case


@pytest.mark.parametrize("ydt", ["f32", "bf16"])
def test_apply_ids_decode_workload(ydt):
    """The decode workload (256 rows, 64 slots of rank 16, 4096 -> 4096): every
    row against the oracle, and equal to lora_apply bit for bit."""
    say(f"apply_ids config 2 y={ydt}")
    case = workloads.make_config(2, y_dtype=ydt)
    Yo, table, dev = run_ids(case)
    rel, mx = check_forward(case, Yo, effective(case))
    say(f"  relF {rel:.3g} maxabs {mx:.3g}")
    assert Yo.tobytes() == run_split(case, dev, table).tobytes()


FUZZ = [
    # name, random_case kwargs
    ("ragged_dims", dict(n=300, d_in=264, d_out=136, num_slots=20, rank_choices=(8, 16, 32))),
    ("odd_ranks", dict(n=200, d_in=128, d_out=200, num_slots=9, rank_choices=(1, 5, 12, 20, 33))),
    ("rank64_128", dict(n=180, d_in=1024, d_out=520, num_slots=5, rank_choices=(64, 128))),
    ("rank100", dict(n=90, d_in=512, d_out=256, num_slots=3, rank_choices=(100,))),
    ("long_groups", dict(n=700, d_in=512, d_out=1032, num_slots=4, rank_choices=(16, 32),
                         layout="segments", seg_len=(30, 200))),
    ("max_rows", dict(n=1024, d_in=256, d_out=264, num_slots=64, rank_choices=(8, 16))),
    ("one_row", dict(n=1, d_in=256, d_out=128, num_slots=3, rank_choices=(16,), frac_none=0.0)),
    ("all_none", dict(n=100, d_in=64, d_out=64, num_slots=3, frac_none=1.0)),
]


@pytest.mark.parametrize("ydt", ["f32", "bf16"])
@pytest.mark.parametrize("name", [f[0] for f in FUZZ])
def test_apply_ids_fuzz(name, ydt):
    """Ragged widths, ranks not a multiple of 8, ranks 64-128, slots with more
    than one 16-row tile, 1024 rows (the limit), one row, no adapter rows; ids
    past the table, below -1 and of empty slots leave their rows unchanged."""
    kw = next(f[1] for f in FUZZ if f[0] == name)
    say(f"apply_ids fuzz {name} y={ydt}")
    case = workloads.random_case(17, y_dtype=ydt, empty_slots=(1,), **kw)
    if case.n > 4:
        case = with_bad_ids(case, 3)
    Yo, table, dev = run_ids(case)
    check_forward(case, Yo, effective(case))
    assert Yo.tobytes() == run_split(case, dev, table).tobytes()


def test_apply_ids_integer_exact():
    """Values in {-1, 0, 1}: the oracle's result bit for bit."""
    say("apply_ids integer-exact")
    case = workloads.random_case(4, 500, 256, 136, 12, rank_choices=(8, 16, 40, 64),
                                 y_dtype="f32", int_values=True,
                                 scales=[0.25, 0.5, 1, 2] * 3)
    Yo, _, _ = run_ids(case)
    X, A, B, Y, _ = f64_case(case)
    ref = oracle.apply(effective(case), X, Y, A, B, case.scales)
    assert np.array_equal(workloads.decode(Yo, "f32"), ref)


def test_apply_ids_empty_batch_and_table():
    """n = 0 enqueues nothing; a table with no adapter leaves Y unchanged."""
    say("apply_ids n=0 and empty table")
    case = workloads.random_case(2, 64, 128, 128, 4, rank_choices=(16,))
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    Y = dev["Y"].clone()
    L.apply_ids(table, dev["idx"][:0], dev["X"][:0], Y[:0])
    empty = L.Table(4, 128, 128, device=DEV)
    empty.upload()
    L.apply_ids(empty, dev["idx"], dev["X"], Y)
    torch.cuda.synchronize()
    assert torch.equal(Y, dev["Y"])


def test_apply_ids_repeated_calls_reuse_workspace():
    """Two calls in a row on one workspace, the second on a smaller batch:
    each call writes every plane entry it reads."""
    say("apply_ids workspace reuse")
    big = workloads.random_case(8, 400, 512, 512, 10, rank_choices=(16, 32))
    dev = case_to_device(big, DEV)
    table = make_table(big, dev)
    ws = L.apply_ids_workspace(table, big.n)
    Y1 = dev["Y"].clone()
    L.apply_ids(table, dev["idx"], dev["X"], Y1, ws=ws)
    m = 150
    Y2 = dev["Y"][:m].clone()
    L.apply_ids(table, dev["idx"][:m], dev["X"][:m], Y2, ws=ws)
    torch.cuda.synchronize()
    check_forward(big, from_torch(Y1), effective(big))
    small = workloads.random_case(8, 400, 512, 512, 10, rank_choices=(16, 32))
    small.n, small.idx, small.X, small.Y = m, small.idx[:m], small.X[:m], small.Y[:m]
    check_forward(small, from_torch(Y2), effective(small))

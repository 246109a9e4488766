"""Forward parity: lora_apply / lora_shrink / lora_expand vs the float64 oracle (GPU).

Graded parity uses float32 Y (relative Frobenius <= 5e-3, max-abs <= 3e-2 on the
LoRA delta of active rows, bf16 inputs, float32 accumulation).  bfloat16 Y is
checked with the same relF and max-abs plus half a bf16 ulp of |Y| (the store
rounding).  Rows with id -1 must come back bit-identical.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_helpers import (DEV, check_forward, effective, make_plan, make_table, run_apply,
                         say)
from helpers import f64_case
from workloads.device import case_to_device, from_torch

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("ydt", ["f32", "bf16"])
@pytest.mark.parametrize("cfg", [1, 2, 4])
def test_apply_config_full(cfg, ydt):
    if cfg == 1 and ydt == "bf16":
        pytest.skip("the tiny workload is float32 end to end")
    say(f"apply config {cfg} y={ydt}")
    case = workloads.make_config(cfg, y_dtype=ydt)
    Yo, _ = run_apply(case)
    rel, mx = check_forward(case, Yo, effective(case))
    say(f"  relF {rel:.3g} maxabs {mx:.3g}")


def test_apply_config3_every_row():
    """The full prefill workload (launch shape of the benchmark) in float32 Y,
    every row against the oracle."""
    say("apply config 3 y=f32, every row")
    case = workloads.make_config(3, y_dtype="f32")
    Yo, _ = run_apply(case, segments=True)
    rel, mx = check_forward(case, Yo, effective(case))
    say(f"  relF {rel:.3g} maxabs {mx:.3g}")


def test_apply_config3_sampled_rows():
    """The full prefill workload in bfloat16 Y; the oracle checks a sample of
    rows one by one, including every segment's first and last row."""
    ydt = "bf16"
    say(f"apply config 3 y={ydt}")
    case = workloads.make_config(3, y_dtype=ydt)
    Yo, _ = run_apply(case, segments=True)
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([rng.choice(case.n, 384, replace=False),
                                     case.seg_offsets[:-1], case.seg_offsets[1:] - 1]))
    rel, mx = check_forward(case, Yo, effective(case), rows=rows)
    say(f"  relF {rel:.3g} maxabs {mx:.3g}")


FUZZ = [
    # name, kwargs for random_case, small_max override
    ("decode_r16", dict(n=300, d_in=512, d_out=768, num_slots=20, rank_choices=(16,)), None),
    ("decode_hetero", dict(n=257, d_in=264, d_out=136, num_slots=33,
                           rank_choices=(8, 16, 32, 64, 128)), None),
    ("odd_ranks", dict(n=200, d_in=128, d_out=200, num_slots=9, rank_choices=(1, 5, 12, 20, 33)), None),
    ("segments_mixed", dict(n=3000, d_in=512, d_out=1032, num_slots=12,
                            rank_choices=(8, 32, 64), layout="segments", seg_len=(1, 300)), None),
    ("segments_force_grouped", dict(n=700, d_in=256, d_out=520, num_slots=6,
                                    rank_choices=(16, 48), layout="segments", seg_len=(20, 200)), 0),
    ("single_adapter", dict(n=2500, d_in=384, d_out=256, num_slots=1, rank_choices=(64,),
                            layout="single", frac_none=0.0), None),
    ("alternating", dict(n=1500, d_in=256, d_out=256, num_slots=4, rank_choices=(32,),
                         layout="alternating"), None),
    ("rank128", dict(n=1200, d_in=1024, d_out=512, num_slots=3, rank_choices=(128,),
                     layout="segments", seg_len=(50, 400)), None),
    ("all_none", dict(n=100, d_in=64, d_out=64, num_slots=3, frac_none=1.0), None),
]


@pytest.mark.parametrize("ydt", ["f32", "bf16"])
@pytest.mark.parametrize("name", [f[0] for f in FUZZ])
def test_apply_fuzz(name, ydt):
    kw, small = next((f[1], f[2]) for f in FUZZ if f[0] == name)
    say(f"apply fuzz {name} y={ydt}")
    case = workloads.random_case(11, y_dtype=ydt, **kw)
    Yo, _ = run_apply(case, policy=None if small is None else dict(small_max=small))
    check_forward(case, Yo, effective(case))


@pytest.mark.parametrize("small", [None, 0, 100000])
def test_apply_integer_exact(small):
    """Values in {-1, 0, 1}: every partial sum is an exact float32 integer and H
    fits bf16 exactly, so the result must equal the oracle bit for bit."""
    say(f"apply integer small={small}")
    case = workloads.random_case(3, 1100, 256, 136, 7, rank_choices=(8, 16, 40, 64),
                                 layout="segments", seg_len=(1, 90), y_dtype="f32",
                                 int_values=True, scales=[0.25, 0.5, 1, 2, 2, 1, 0.5])
    Yo, _ = run_apply(case, policy=None if small is None else dict(small_max=small))
    X, A, B, Y, _ = f64_case(case)
    ref = oracle.apply(effective(case), X, Y, A, B, case.scales)
    assert np.array_equal(workloads.decode(Yo, "f32"), ref)


@pytest.mark.parametrize("small", [None, 16])
@pytest.mark.parametrize("block_rows", [64, 256])
def test_apply_block_rows(block_rows, small):
    """Both large-group block sizes (the host picks one and launches only its
    kernels) give the oracle's result bit for bit on integer-exact values, with
    and without a small-group path beside them; ragged groups span several
    blocks of either size."""
    say(f"apply block_rows={block_rows} small={small}")
    case = workloads.random_case(5, 3000, 256, 520, 40, rank_choices=(8, 16, 32, 64),
                                 layout="segments", seg_len=(1, 700), y_dtype="f32",
                                 int_values=True)
    Yo, _ = run_apply(case, policy=dict(block_rows=block_rows, small_max=small))
    X, A, B, Y, _ = f64_case(case)
    ref = oracle.apply(effective(case), X, Y, A, B, case.scales)
    assert np.array_equal(workloads.decode(Yo, "f32"), ref)


def test_segments_plan_equals_index_plan():
    say("segments == indices")
    case = workloads.make_config(5)        # segment layout, 8 adapters
    case.Y = workloads.encode(np.random.default_rng(1).standard_normal((case.n, case.d_out)), "bf16")
    y1, _ = run_apply(case, segments=False)
    y2, _ = run_apply(case, segments=True)
    assert y1.tobytes() == y2.tobytes()


def test_apply_deterministic():
    say("determinism")
    case = workloads.make_config(4)
    y1, _ = run_apply(case)
    y2, _ = run_apply(case)
    assert y1.tobytes() == y2.tobytes()


def test_zero_B_leaves_Y():
    say("zero B")
    case = workloads.random_case(4, 900, 256, 256, 5, rank_choices=(16, 32), y_dtype="bf16")
    case.B = [np.zeros_like(b) if b is not None else None for b in case.B]
    case.Y[case.Y == 0x8000] = 0               # -0.0 + 0.0 would become +0.0
    Yo, _ = run_apply(case)
    assert Yo.tobytes() == case.Y.tobytes()


@pytest.mark.parametrize("xdt,wdt", [("f32", "f32"), ("bf16", "bf16"), ("f32", "bf16"),
                                     ("bf16", "f32")])
def test_shrink_then_expand(xdt, wdt):
    say(f"shrink/expand x={xdt} w={wdt}")
    case = workloads.random_case(8, 1300, 256, 264, 6, rank_choices=(8, 24, 64),
                                 layout="segments", seg_len=(1, 200), x_dtype=xdt,
                                 w_dtype=wdt, y_dtype="f32")
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=False)
    H = torch.full((case.n, 72), 7.0, dtype=torch.float32, device=DEV)
    L.shrink(plan, dev["X"], H)
    Y = dev["Y"].clone()
    L.expand(plan, H, Y)
    torch.cuda.synchronize()
    X, A, B, Yr, _ = f64_case(case)
    eff = effective(case)
    Href = oracle.shrink(eff, X, A, H=np.full((case.n, 72), 7.0))
    Hg = H.cpu().double().numpy()
    assert oracle.rel_fro(Hg, Href) <= 1e-5
    assert oracle.max_abs(Hg, Href) <= 1e-3
    assert np.array_equal(Hg[eff < 0], Href[eff < 0])       # untouched rows
    for a in range(case.num_slots):                          # untouched columns
        rows = eff == a
        assert np.all(Hg[rows, case.ranks[a]:] == 7.0)
    check_forward(case, from_torch(Y), eff)


def test_fp32_tiny_workload_all_entry_points():
    say("fp32 tiny")
    case = workloads.make_config(1)
    Yo, plan = run_apply(case, segments=True)
    check_forward(case, Yo, effective(case))


SMALL_PATH_CASES = ["decode_r16", "decode_hetero", "odd_ranks", "segments_mixed", "rank128"]


@pytest.mark.parametrize("path", ["fused", "split1", "split3", "split8"])
@pytest.mark.parametrize("name", SMALL_PATH_CASES)
def test_apply_small_group_paths(name, path):
    """Both small-group paths (the fused kernel, and the split shrink per d-slice
    + expand with 1, 3 or 8 slices) against the oracle."""
    kw = next(f[1] for f in FUZZ if f[0] == name)
    say(f"apply small path {path} {name}")
    case = workloads.random_case(12, y_dtype="f32", **kw)
    split = 0 if path == "fused" else 1
    slices = None if path == "fused" else int(path[5:])
    Yo, _ = run_apply(case, policy=dict(small_split=split, split_slices=slices))
    check_forward(case, Yo, effective(case))


@pytest.mark.parametrize("path", ["fused", "split"])
@pytest.mark.parametrize("cfg", [2, 4])
def test_apply_configs_both_small_paths(cfg, path):
    say(f"apply config {cfg} small path {path}")
    case = workloads.make_config(cfg, y_dtype="bf16")
    Yo, _ = run_apply(case, policy=dict(small_split=0 if path == "fused" else 1))
    rel, mx = check_forward(case, Yo, effective(case))
    say(f"  relF {rel:.3g} maxabs {mx:.3g}")


def _permuted(case, perm):
    """The same batch with its rows reordered: row i of the result is row perm[i]."""
    import copy
    c = copy.copy(case)
    c.idx = case.idx[perm]
    c.X = case.X[perm]
    c.Y = case.Y[perm]
    c.seg_offsets = c.seg_adapter = None
    if case.mask is not None:
        c.mask = case.mask[perm]
    return c


@pytest.mark.parametrize("cfg", [2, 4])
def test_apply_row_permutation_invariance(cfg):
    """Each row's result depends only on that row (grouping is by adapter
    identity, Section 3.4): reordering the batch reorders the output rows, bit
    for bit."""
    say(f"row permutation invariance, config {cfg}")
    case = workloads.make_config(cfg, y_dtype="bf16")
    perm = np.random.default_rng(5).permutation(case.n)
    y1, _ = run_apply(case)
    y2, _ = run_apply(_permuted(case, perm))
    assert y2.tobytes() == y1[perm].tobytes()


def test_apply_adapter_isolation():
    """Changing one adapter's weights changes no row of any other adapter."""
    say("adapter isolation")
    case = workloads.make_config(4, y_dtype="bf16")
    eff = effective(case)
    counts = np.bincount(eff[eff >= 0], minlength=case.num_slots)
    b = int(np.argmax(counts))           # the busiest adapter (large-group path)
    small = int(np.nonzero((counts > 0) & (counts <= 16))[0][0])   # and a small one
    y1, _ = run_apply(case)
    import copy
    c2 = copy.copy(case)
    rng = np.random.default_rng(9)
    c2.A = list(case.A)
    c2.B = list(case.B)
    for a in (b, small):
        c2.A[a] = workloads.encode(rng.standard_normal(case.A[a].shape), "bf16")
        c2.B[a] = workloads.encode(rng.standard_normal(case.B[a].shape), "bf16")
    y2, _ = run_apply(c2)
    keep = (eff != b) & (eff != small)
    assert y2[keep].tobytes() == y1[keep].tobytes()
    assert y2[eff == b].tobytes() != y1[eff == b].tobytes()
    check_forward(c2, y2, eff)


def test_apply_empty_batch():
    """n = 0: every entry point returns OK and touches nothing."""
    say("empty batch")
    case = workloads.random_case(3, 0, 128, 64, 4, rank_choices=(16,), y_dtype="f32")
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=False)
    L.apply(plan, dev["X"], dev["Y"])
    H = torch.zeros((0, 16), dtype=torch.float32, device=DEV)
    L.shrink(plan, dev["X"], H)
    L.expand(plan, H, dev["Y"])
    torch.cuda.synchronize()


def _grouped_case(seed, sizes, pad_none, ranks, d_in=256, d_out=136, y_dtype="f32"):
    """A batch whose adapter groups have exactly the given sizes (rows shuffled),
    plus pad_none rows without an adapter."""
    S = len(sizes)
    case = workloads.random_case(seed, n=sum(sizes) + pad_none, d_in=d_in, d_out=d_out,
                                 num_slots=S, ranks=ranks, frac_none=0.0, y_dtype=y_dtype)
    idx = np.concatenate([np.full(c, a, np.int32) for a, c in enumerate(sizes)] +
                         [np.full(pad_none, -1, np.int32)])
    case.idx = np.random.default_rng(seed).permutation(idx).astype(np.int32)
    return case


def _coarse_blocks(case):
    """Large-group blocks of 256 rows the plan counts (groups above 16 rows when
    n > 1024)."""
    eff = effective(case)
    cnt = np.bincount(eff[eff >= 0], minlength=case.num_slots)
    small_max = 16 if case.n > 1024 else np.iinfo(np.int32).max
    return int(sum((c + 255) // 256 for c in cnt if c > small_max))


BLOCK_MODE_CASES = {
    # 47 coarse blocks: the batch takes 64-row blocks
    "fine_47": (dict(sizes=[17] * 47, pad_none=400, ranks=[8, 16, 32, 64, 128] * 9 + [16, 8]), False),
    # 48: 256-row blocks
    "coarse_48": (dict(sizes=[17] * 48, pad_none=400, ranks=[8, 16, 32, 64, 128] * 9 + [16, 8, 24]), True),
    # ragged fine blocks: 1, 63, 64, 65, 255, 256, 257 rows and a long group
    "fine_ragged": (dict(sizes=[257, 256, 255, 65, 64, 63, 1000, 17, 3, 1],
                         pad_none=200, ranks=[64, 32, 16, 8, 48, 128, 40, 24, 16, 8]), False),
    # long groups: many 256-row blocks with ragged ends
    "coarse_long": (dict(sizes=[2900, 3100, 1, 2500, 3333, 1800], pad_none=500,
                         ranks=[64, 16, 8, 32, 128, 40]), True),
}


@pytest.mark.parametrize("ydt", ["f32", "bf16"])
@pytest.mark.parametrize("name", list(BLOCK_MODE_CASES))
def test_apply_large_block_sizes(name, ydt):
    """The plan cuts large groups into 256-row blocks, or into 64-row blocks when
    that gives fewer than 48 of them; both grouped kernel pairs against the
    oracle, on each side of the threshold and with ragged group ends."""
    kw, coarse = BLOCK_MODE_CASES[name]
    case = _grouped_case(31, y_dtype=ydt, **kw)
    nb = _coarse_blocks(case)
    assert (nb >= 48) == coarse, nb
    say(f"apply block mode {name} ({nb} coarse blocks) y={ydt}")
    Yo, _ = run_apply(case)
    rel, mx = check_forward(case, Yo, effective(case))
    say(f"  relF {rel:.3g} maxabs {mx:.3g}")
    # the standalone shrink and expand take the same kernels
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=False)
    H = L.shrink(plan, dev["X"])
    Y = dev["Y"].clone()
    L.expand(plan, H, Y)
    torch.cuda.synchronize()
    check_forward(case, from_torch(Y), effective(case))

"""Heterogeneous ranks side by side (Section 3.4, rank-aware scheduling: one
launch carries adapters of different ranks, each tile padded to its own rank).

Every pairing of the rank classes 8, 16, 32, 64 and 128 (a class beside itself
too) goes through each kernel family at ragged sizes: the grouped 64-row and
256-row pairs, the small-group split and fused kernels, the plan-free pair of
lora_apply_ids, the adapter gradients and the input gradient.  Each kernel is instantiated for the batch's largest
rank, so a pairing (a, b) runs the rank-a tiles inside the rank-b instance.
A missing wait between a matrix-core result and its first reader shows up
here as a wrong tile of the smaller rank.
"""
import itertools

import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_helpers import (DEV, MAX_ABS, REL_FRO, check_forward, check_grads, effective,
                         make_plan, make_table, run_apply, say)
from helpers import f64_case
from workloads.device import case_to_device, from_torch

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu

CLASSES = (8, 16, 32, 64, 128)
PAIRS = list(itertools.combinations_with_replacement(CLASSES, 2))


def _case(seed, sizes, pad_none, ranks, d_in, d_out, mask_p=None):
    """Adapter groups of exactly `sizes` rows (shuffled), plus pad_none rows
    with no adapter."""
    n = sum(sizes) + pad_none
    case = workloads.random_case(seed, n=n, d_in=d_in, d_out=d_out, num_slots=len(sizes),
                                 ranks=ranks, frac_none=0.0, y_dtype="f32", mask_p=mask_p,
                                 want_dy=mask_p is not None)
    idx = np.concatenate([np.full(c, a, np.int32) for a, c in enumerate(sizes)] +
                         [np.full(pad_none, -1, np.int32)])
    case.idx = np.random.default_rng(seed).permutation(idx).astype(np.int32)
    return case


def _ranks(ra, rb, S):
    return [ra if a % 2 == 0 else rb for a in range(S)]


FINE_SIZES = [1, 16, 17, 63, 200, 5, 340, 9]      # small (<= 16) and large groups
COARSE_SIZES = [3000, 2900, 17, 3100, 2600, 12, 2000, 1]   # >= 48 blocks of 256 rows

FINE_PATHS = {
    "split+grouped64": dict(small_max=16, small_split=1),
    "fused+grouped64": dict(small_max=16, small_split=0),
    "grouped64_only": dict(small_max=0),
    "small_only": None,                          # n <= 1024: every group small
}


@pytest.mark.parametrize("ra,rb", PAIRS, ids=lambda v: str(v))
def test_rank_pair_forward_and_backward(ra, rb):
    seed = 100 + 7 * ra + rb
    case = _case(seed, FINE_SIZES, 120, _ranks(ra, rb, 8), d_in=1032, d_out=264, mask_p=0.5)
    eff = effective(case)
    for name, pol in FINE_PATHS.items():
        say(f"ranks ({ra}, {rb}) apply {name}")
        Yo, _ = run_apply(case, policy=pol)
        check_forward(case, Yo, eff)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    say(f"ranks ({ra}, {rb}) apply_ids")
    Yi = dev["Y"].clone()
    L.apply_ids(table, dev["idx"], dev["X"], Yi)
    torch.cuda.synchronize()
    check_forward(case, from_torch(Yi), eff)
    say(f"ranks ({ra}, {rb}) grad and grad_x")
    plan = make_plan(case, dev, table, mask=True)
    dA, dB = L.grad(plan, dev["X"], dev["dY"])
    dX = torch.zeros(case.n, case.d_in, dtype=torch.float32, device=DEV)
    L.grad_x(plan, dev["dY"], dX)
    torch.cuda.synchronize()
    check_grads(case, dA, dB, eff, case.mask)
    X, A, B, _, dY = f64_case(case)
    ref = oracle.grad_x(eff, case.mask, dY, A, B, case.scales, np.zeros((case.n, case.d_in)))
    got = dX.cpu().double().numpy()
    sel = (eff >= 0) & (np.asarray(case.mask) != 0)
    assert np.all(got[~sel] == 0)
    rel, mx = oracle.rel_fro(got[sel], ref[sel]), oracle.max_abs(got[sel], ref[sel])
    assert rel <= REL_FRO and mx <= MAX_ABS, f"grad_x relF {rel:.3g} maxabs {mx:.3g}"


@pytest.mark.parametrize("ra,rb", PAIRS, ids=lambda v: str(v))
def test_rank_pair_coarse_blocks(ra, rb):
    seed = 300 + 7 * ra + rb
    case = _case(seed, COARSE_SIZES, 333, _ranks(ra, rb, 8), d_in=264, d_out=136)
    say(f"ranks ({ra}, {rb}) apply 256-row blocks")
    Yo, _ = run_apply(case)
    check_forward(case, Yo, effective(case))

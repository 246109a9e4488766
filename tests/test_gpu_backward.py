"""lora_backward (adapter gradients and input gradient in one call) vs the two
separate calls (GPU).  The same kernels run with the same arguments, the input
gradient on a second stream beside the adapter gradients, so every output must
match the separate calls bit for bit."""
import numpy as np
import pytest
import torch

import workloads
from gpu_helpers import DEV, make_plan, make_table, say
from workloads.device import case_to_device

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu


def _bits(ts):
    return [t.view(torch.int32).cpu() if t is not None else None for t in ts]


def _same(a, b):
    return all((x is None and y is None) or torch.equal(x, y) for x, y in zip(_bits(a), _bits(b)))


@pytest.mark.parametrize("which", ["config5", "fuzz_accumulate"])
def test_backward_matches_separate_calls(which):
    say(f"backward {which}")
    if which == "config5":
        case = workloads.make_config(5)
        accumulate = False
    else:
        case = workloads.random_case(61, 1500, 520, 264, 9, rank_choices=(8, 40, 64), layout="segments",
                                     seg_len=(1, 200), mask_p=0.5, want_dy=True, want_y=False)
        accumulate = True
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=True)
    g = torch.Generator(device=DEV).manual_seed(62)

    def fresh():
        dA = [torch.randn(int(r), case.d_in, device=DEV, generator=g) if r > 0 else None for r in case.ranks]
        dB = [torch.randn(case.d_out, int(r), device=DEV, generator=g) if r > 0 else None for r in case.ranks]
        dX = torch.randn(case.n, case.d_in, device=DEV, generator=g)
        return dA, dB, dX

    dA1, dB1, dX1 = fresh()
    dA2, dB2, dX2 = [t.clone() if t is not None else None for t in dA1], \
        [t.clone() if t is not None else None for t in dB1], dX1.clone()
    L.grad(plan, dev["X"], dev["dY"], dA1, dB1, accumulate=accumulate)
    L.grad_x(plan, dev["dY"], dX1)
    L.backward(plan, dev["X"], dev["dY"], dX2, dA2, dB2, accumulate=accumulate)
    torch.cuda.synchronize()
    assert _same(dA1, dA2) and _same(dB1, dB2)
    assert torch.equal(dX1.view(torch.int32), dX2.view(torch.int32))


def test_backward_empty_batch_and_rejects():
    case = workloads.random_case(63, 0, 64, 64, 3, rank_choices=(8,), mask_p=0.5, want_dy=True,
                                 want_y=False)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=True)
    dA, dB, dX = L.backward(plan, dev["X"], dev["dY"], torch.empty(0, 64, device=DEV))
    torch.cuda.synchronize()
    assert all(torch.all(t == 0) for t in dA + dB if t is not None)   # overwrite mode: zeros
    case = workloads.random_case(64, 40, 64, 64, 3, rank_choices=(8,), mask_p=0.5, want_dy=True,
                                 want_y=False)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=True)
    sentinel = [torch.full((8, 64), 7.0, device=DEV) for _ in range(3)]
    dX = torch.zeros(case.n, case.d_in, device=DEV)
    with pytest.raises(L.LoraError):           # float32 dY: no input gradient, nothing enqueued
        L.backward(plan, dev["X"].float(), dev["dY"].float(), dX, dA=sentinel)
    tiny = torch.empty(16, dtype=torch.uint8, device=DEV)
    with pytest.raises(L.LoraError):
        L.backward(plan, dev["X"], dev["dY"], dX, dA=sentinel, ws=tiny)
    torch.cuda.synchronize()
    assert all(torch.all(t == 7.0) for t in sentinel)

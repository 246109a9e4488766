"""Calls on a stream other than torch's current one (GPU).

The binding allocates plan, workspace and output buffers on torch's current
stream; the kernels run on the stream passed in.  Those buffers must not be
handed out again while that stream still uses them.  The test runs a plan
build, lora_apply and lora_backward on a side stream, then fills fresh
allocations on the current stream before the side stream has finished, and
checks every result against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_helpers import (DEV, MAX_ABS, REL_FRO, check_forward, check_grads, effective,
                         make_table, say)
from helpers import f64_case
from workloads.device import case_to_device, from_torch

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu


def _scribble(n_bytes, rounds=8):
    """Allocate and fill memory on the current stream (reuses freed blocks)."""
    junk = []
    for i in range(rounds):
        t = torch.empty(n_bytes // 4, dtype=torch.float32, device=DEV)
        t.fill_(float("nan") if i % 2 else 1e30)
        junk.append(t)
    return junk


def test_side_stream_apply_and_backward(monkeypatch):
    say("side stream: plan, apply, backward")
    made = []
    for name in ("apply_workspace", "backward_workspace"):
        real = getattr(L.lora, name)

        def wrapped(plan, _real=real):
            ws = _real(plan)
            made.append(ws)
            return ws
        monkeypatch.setattr(L.lora, name, wrapped)
    case = workloads.random_case(71, 3000, 1024, 768, 12, rank_choices=(8, 16, 32, 64),
                                 layout="segments", seg_len=(1, 300), mask_p=0.5, want_dy=True,
                                 y_dtype="f32")
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    # one pass on the current stream first: the first launch of a kernel loads
    # its code, which can take longer on the host than the spin below on the GPU
    warm = L.Plan(table, idx=dev["idx"], mask=dev["mask"])
    L.apply(warm, dev["X"], dev["Y"].clone())
    L.backward(warm, dev["X"], dev["dY"], torch.zeros_like(dev["X"], dtype=torch.float32))
    torch.cuda.synchronize()
    made.clear()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    # a long queue on the side stream first (200 passes over 256 MB, about
    # 20 ms), so the later kernels run after the current stream's allocations
    spin = torch.empty(64 << 20, dtype=torch.float32, device=DEV)
    with torch.cuda.stream(side):
        for _ in range(200):
            spin.mul_(1.0)
    Y = dev["Y"].clone()
    dX = torch.zeros(case.n, case.d_in, dtype=torch.float32, device=DEV)
    side.wait_stream(torch.cuda.current_stream())
    plan = L.Plan(table, idx=dev["idx"], mask=dev["mask"], stream=side)
    L.apply(plan, dev["X"], Y, stream=side)
    dA, dB, _ = L.backward(plan, dev["X"], dev["dY"], dX, stream=side)
    # the workspaces the binding made have been dropped, but the side stream
    # (still behind the spin) has not used them yet: fresh allocations of the
    # same sizes on the current stream must get other memory
    ptrs = [w.data_ptr() for w in made]
    sizes = [w.numel() for w in made]
    made.clear()
    assert len(ptrs) == 2
    fresh = [torch.empty(n, dtype=torch.uint8, device=DEV) for n in sizes]
    # the check only means something while the side stream still has work queued
    assert not side.query(), "side stream drained before the check: lengthen the spin"
    assert not set(ptrs) & {f.data_ptr() for f in fresh}, "workspace reused while in use"
    junk = _scribble(32 << 20)
    side.synchronize()
    torch.cuda.synchronize()
    del junk
    eff = effective(case)
    check_forward(case, from_torch(Y), eff)
    check_grads(case, dA, dB, eff, case.mask)
    X, A, B, _, dY = f64_case(case)
    ref = oracle.grad_x(eff, case.mask, dY, A, B, case.scales, np.zeros((case.n, case.d_in)))
    got = dX.cpu().double().numpy()
    sel = (eff >= 0) & (np.asarray(case.mask) != 0)
    rel, mx = oracle.rel_fro(got[sel], ref[sel]), oracle.max_abs(got[sel], ref[sel])
    assert rel <= REL_FRO and mx <= MAX_ABS, f"grad_x relF {rel:.3g} maxabs {mx:.3g}"
    assert np.all(got[~sel] == 0)

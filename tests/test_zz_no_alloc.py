"""lora_apply_noalloc (the fixed per-GPU scratch instead of a workspace) against
lora_apply on the same inputs (GPU).  Both run the same kernels, so the
outputs must match bit for bit; each is also checked against the oracle.  Two
calls in a row, the second on a smaller batch, share the one scratch array."""
import numpy as np
import pytest
import torch

import workloads
from gpu_helpers import DEV, check_forward, effective, make_plan, make_table, say
from workloads.device import case_to_device, from_torch

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu


def _both(case, segments=False):
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, segments=segments, mask=False)
    Y1 = dev["Y"].clone()
    L.apply(plan, dev["X"], Y1)
    Y2 = dev["Y"].clone()
    torch.cuda.synchronize()
    before = torch.cuda.memory_allocated()
    L.apply_noalloc(plan, dev["X"], Y2)
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == before
    return from_torch(Y1), from_torch(Y2)


@pytest.mark.parametrize("first,second", [(4, 2), (3, 1)])
def test_noalloc_matches_apply_two_calls(first, second):
    for cfg in (first, second):                 # the second batch is the smaller one
        say(f"apply_noalloc config {cfg}")
        case = workloads.make_config(cfg, y_dtype="f32")
        y_ws, y_static = _both(case, segments=(cfg == 3))
        assert y_ws.tobytes() == y_static.tobytes()
        if cfg != 3:
            check_forward(case, y_static, effective(case))


def test_noalloc_mixed_batch_fuzz_then_decode():
    """A mixed batch with small and large groups and ragged sizes, then a
    decode batch: the second call sees the first call's leftovers."""
    a = workloads.random_case(91, 3000, 1032, 520, 12, rank_choices=(8, 16, 32, 64, 128),
                              layout="segments", seg_len=(1, 300), y_dtype="f32")
    b = workloads.random_case(92, 200, 264, 136, 40, rank_choices=(8, 16, 40), y_dtype="bf16")
    for case in (a, b):
        say(f"apply_noalloc fuzz n={case.n}")
        y_ws, y_static = _both(case)
        assert y_ws.tobytes() == y_static.tobytes()
        check_forward(case, y_static, effective(case))


def test_noalloc_rejects_a_plan_beyond_its_scratch():
    say("apply_noalloc size limit")
    case = workloads.random_case(93, 70000, 256, 128, 2, rank_choices=(128,), y_dtype="f32",
                                 layout="segments", seg_len=(5000, 30000))
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    plan = make_plan(case, dev, table, mask=False)
    assert L.lib().lora_apply_workspace_bytes(plan.handle) > (32 << 20)
    Y = dev["Y"].clone()
    with pytest.raises(L.LoraError, match="scratch"):
        L.apply_noalloc(plan, dev["X"], Y)
    torch.cuda.synchronize()
    assert torch.equal(Y, dev["Y"])

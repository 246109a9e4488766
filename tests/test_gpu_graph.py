"""lora_apply captured into a HIP graph (GPU).

A mixed batch (small and large groups) runs its small-group path on a second
stream forked from the caller's with events, so a capture records both
streams into the caller's graph.  Each of three replays, with eager work and
synchronisation between them, must give the eager call's bytes.
"""
import numpy as np
import pytest
import torch

import workloads
from gpu_helpers import DEV, say
from workloads.device import case_to_device

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu


def test_apply_graph_replays_match_eager():
    say("graph capture of a mixed apply")
    case = workloads.random_case(88, 2048, 512, 768, 96, rank_choices=(8, 16, 32), layout="segments",
                                 seg_len=(1, 300), y_dtype="f32", want_y=True)
    counts = np.bincount(case.idx[case.idx >= 0], minlength=case.num_slots)
    assert np.any((counts > 0) & (counts <= 16)) and np.any(counts > 16)   # both paths have work
    dev = case_to_device(case, DEV)
    table = L.Table(case.num_slots, case.d_in, case.d_out, w_dtype=torch.bfloat16, device=DEV)
    for a in range(case.num_slots):
        if case.ranks[a] > 0:
            table.set(a, dev["A"][a], dev["B"][a], float(case.scales[a]))
    table.upload()
    plan = L.Plan(table, idx=dev["idx"])
    ws = L.apply_workspace(plan)
    Y0 = dev["Y"].clone()
    eager = Y0.clone()
    L.apply(plan, dev["X"], eager, ws=ws)          # eager call (also creates the second stream)
    torch.cuda.synchronize()
    Y = Y0.clone()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            L.apply(plan, dev["X"], Y, ws=ws)
    torch.cuda.synchronize()
    for rep in range(3):
        Y.copy_(Y0)                                   # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y.view(torch.int32), eager.view(torch.int32)), f"replay {rep}"

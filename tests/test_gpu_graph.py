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
    assert np.any((counts > 0) & (counts <= 32)) and np.any(counts > 32)   # both paths have work
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


def _decode_ids(rng, n, S):
    ids = rng.integers(0, S, size=n).astype(np.int32)
    ids[rng.random(n) < 0.1] = -1
    return torch.from_numpy(ids).to(DEV)


def test_decode_step_graph_new_ids_each_replay():
    """A decode step captured once and replayed with other ids, as a serving
    loop does: the ids live in one device buffer that the caller rewrites
    before each replay.  Two graphs on the decode workload (256 rows, 64
    slots of rank 16, 4096 -> 4096): plan build + lora_apply, and
    lora_apply_ids.  Every replay must give the bytes of eager calls on that
    replay's ids (a plan built from them, and lora_apply_ids)."""
    say("graph capture of a decode step, new ids each replay")
    case = workloads.make_config(2, y_dtype="bf16")
    dev = case_to_device(case, DEV)
    table = L.Table(case.num_slots, case.d_in, case.d_out, w_dtype=torch.bfloat16, device=DEV)
    for a in range(case.num_slots):
        table.set(a, dev["A"][a], dev["B"][a], float(case.scales[a]))
    table.upload()
    n, S = case.n, case.num_slots
    ids = dev["idx"].clone()
    Y0 = dev["Y"].clone()
    Yp, Yi = Y0.clone(), Y0.clone()
    ws_ids = L.apply_ids_workspace(table, n)
    # eager calls first (they also create anything the library makes once)
    warm = L.Plan(table, idx=ids)
    ws_apply = L.apply_workspace(warm)
    L.apply(warm, dev["X"], Yp.clone(), ws=ws_apply)
    L.apply_ids(table, ids, dev["X"], Yi.clone(), ws=ws_ids)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g_plan, g_ids = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g_plan, stream=s):
            plan = L.Plan(table, idx=ids)                # workspace from the graph's pool
            L.apply(plan, dev["X"], Yp, ws=ws_apply)
        with torch.cuda.graph(g_ids, stream=s):
            L.apply_ids(table, ids, dev["X"], Yi, ws=ws_ids)
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    for rep in range(3):
        ids.copy_(_decode_ids(rng, n, S))              # the next step's ids, eager
        Yp.copy_(Y0)
        Yi.copy_(Y0)
        torch.cuda.synchronize()
        g_plan.replay()
        g_ids.replay()
        torch.cuda.synchronize()
        ep, ei = Y0.clone(), Y0.clone()
        L.apply(L.Plan(table, idx=ids), dev["X"], ep)
        L.apply_ids(table, ids, dev["X"], ei)
        torch.cuda.synchronize()
        assert torch.equal(Yp.view(torch.int16), ep.view(torch.int16)), f"plan + apply, replay {rep}"
        assert torch.equal(Yi.view(torch.int16), ei.view(torch.int16)), f"apply_ids, replay {rep}"
        assert not torch.equal(Yp.view(torch.int16), Y0.view(torch.int16))
    del plan

"""Device row grouping vs the oracle's canonical plan: bit-exact (GPU)."""
import zlib

import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_helpers import DEV, compare_plan, make_plan, make_table, say
from workloads.device import case_to_device

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_plan_configs(cfg):
    say(f"plan config {cfg}")
    case = workloads.make_config(cfg)
    dev = case_to_device(case, DEV)
    table = make_table(case, dev)
    ref = oracle.canonical_plan(case.idx, case.num_slots, mask=case.mask, ranks=case.ranks)
    got = make_plan(case, dev, table).export()
    compare_plan(got, ref)
    assert got["data_flags"] == 0
    if case.seg_offsets is not None:
        got_s = make_plan(case, dev, table, segments=True).export()
        compare_plan(got_s, ref)


def _plan_case(idx, S, mask=None, ranks=None, seed=0):
    ranks = np.full(S, 8, np.int32) if ranks is None else np.asarray(ranks, np.int32)
    c = workloads.random_case(seed, 1, 8, 8, S, ranks=ranks, frac_none=0.0)
    table = L.Table(S, 8, 8, device=DEV)
    w = torch.zeros(8, 8, dtype=torch.bfloat16, device=DEV)
    for a in range(S):
        if ranks[a] > 0:
            r = int(ranks[a])
            table.set(a, w[:r].contiguous(), torch.zeros(8, r, dtype=torch.bfloat16, device=DEV), 1.0)
    table.upload()
    idx_t = torch.from_numpy(np.asarray(idx, np.int32)).to(DEV)
    m_t = None if mask is None else torch.from_numpy(np.asarray(mask, np.uint8)).to(DEV)
    got = L.Plan(table, idx=idx_t, mask=m_t).export()
    ref = oracle.canonical_plan(np.asarray(idx), S, mask=mask, ranks=ranks)
    return got, ref


FUZZ = [
    ("all_none", lambda r: (np.full(300, -1), 7, None)),
    ("single_adapter", lambda r: (np.zeros(777, np.int64), 1, None)),
    ("alternating", lambda r: (np.arange(1000) % 5, 5, r.integers(0, 2, 1000))),
    ("empty", lambda r: (np.zeros(0, np.int64), 3, None)),
    ("one_row", lambda r: (np.array([2]), 3, np.array([1]))),
    ("ragged_65", lambda r: (r.integers(-1, 9, 65), 9, r.integers(0, 2, 65))),
    # edges of the 256-thread grouping (n <= 256 and slots <= 256) and of the
    # 1024-thread one
    ("t256_full", lambda r: (r.integers(-1, 256, 256), 256, r.integers(0, 2, 256))),
    ("t256_slots_past", lambda r: (r.integers(-1, 300, 200), 300, r.integers(0, 2, 200))),
    ("t256_rows_past", lambda r: (r.integers(-1, 64, 257), 64, r.integers(0, 2, 257))),
    ("t1024_full", lambda r: (r.integers(-1, 1024, 1024), 1024, r.integers(0, 2, 1024))),
    ("long_runs", lambda r: (np.repeat(r.integers(-1, 12, 400), 37)[:13001], 12,
                             r.integers(0, 2, 13001))),
    ("large_n", lambda r: (r.integers(-1, 50, 70001), 50, r.integers(0, 2, 70001))),
    ("max_slots", lambda r: (r.integers(-1, 1024, 20000), 1024, None)),
    ("zipf_1024", lambda r: (np.minimum(r.zipf(1.3, 9000) - 1, 1023), 1024, r.integers(0, 2, 9000))),
    # chunk edges of the chunked grouping: one row past a chunk, whole chunks,
    # and one run spanning several chunks
    ("chunk_plus_one", lambda r: (r.integers(-1, 4, 1025), 4, r.integers(0, 2, 1025))),
    ("two_chunks", lambda r: (r.integers(-1, 3, 2048), 3, None)),
    ("run_across_chunks", lambda r: (np.concatenate([np.full(3000, 2), np.full(100, -1),
                                                     np.full(2500, 1)]), 4, r.integers(0, 2, 5600))),
    ("chunked_limit", lambda r: (r.integers(-1, 40, 65536), 40, r.integers(0, 2, 65536))),
]


@pytest.mark.parametrize("name", [f[0] for f in FUZZ])
def test_plan_fuzz(name):
    say(f"plan fuzz {name}")
    rng = np.random.default_rng(zlib.crc32(name.encode()))   # stable across processes
    idx, S, mask = dict(FUZZ)[name](rng)
    got, ref = _plan_case(idx, S, mask)
    compare_plan(got, ref)
    assert got["data_flags"] == 0


def test_plan_bad_ids_and_empty_slots():
    say("plan bad ids")
    rng = np.random.default_rng(5)
    idx = rng.integers(-3, 12, 3000)
    ranks = np.full(10, 8)
    ranks[[2, 7]] = 0
    got, ref = _plan_case(idx, 10, rng.integers(0, 2, 3000), ranks=ranks)
    compare_plan(got, ref)
    assert got["data_flags"] == (L.LORA_DATA_BAD_ID | L.LORA_DATA_EMPTY_SLOT)


def test_plan_segments_edge_cases():
    say("plan segments")
    S = 4
    table = L.Table(S, 8, 8, device=DEV)
    w = torch.zeros(8, 8, dtype=torch.bfloat16, device=DEV)
    for a in range(S):
        table.set(a, w, w, 1.0)
    table.upload()
    dv = lambda x: torch.tensor(x, dtype=torch.int32, device=DEV)
    # empty segments and adjacent segments of one adapter
    off, ad = [0, 3, 3, 7, 12, 12, 20], [2, 0, 2, 2, 1, 3]
    n = 20
    got = L.Plan(table, seg_offsets=dv(off), seg_adapter=dv(ad), n=n).export()
    ids = oracle.segments_to_ids(off, ad, n)
    compare_plan(got, oracle.canonical_plan(ids, S))
    assert got["n_runs"] == 2 and got["data_flags"] == 0
    # malformed tables: not starting at 0, decreasing, not ending at n
    for off in ([1, 5, 20], [0, 12, 9, 20], [0, 5, 19]):
        ad = [1] * (len(off) - 1)
        got = L.Plan(table, seg_offsets=dv(off), seg_adapter=dv(ad), n=n).export()
        assert got["data_flags"] == L.LORA_DATA_BAD_SEGMENTS
        assert got["offsets"].tolist() == [0] * (S + 1) and got["n_runs"] == 0
    # longer batches (grouped in chunks): empty segments, runs across chunk edges
    r = np.random.default_rng(5)
    lens = r.integers(0, 180, 60)
    n = int(lens.sum())
    off = np.concatenate([[0], np.cumsum(lens)]).tolist()
    ad = r.integers(-1, S, 60).tolist()
    got = L.Plan(table, seg_offsets=dv(off), seg_adapter=dv(ad), n=n).export()
    compare_plan(got, oracle.canonical_plan(oracle.segments_to_ids(off, ad, n), S))
    bad = list(off)
    bad[30] = bad[31] + 1
    got = L.Plan(table, seg_offsets=dv(bad), seg_adapter=dv(ad), n=n).export()
    assert got["data_flags"] == L.LORA_DATA_BAD_SEGMENTS and got["n_runs"] == 0


def test_plan_check_reports_flags():
    say("plan check")
    S = 3
    table = L.Table(S, 8, 8, device=DEV)
    w = torch.zeros(8, 8, dtype=torch.bfloat16, device=DEV)
    table.set(0, w, w, 1.0)
    table.upload()
    p = L.Plan(table, idx=torch.tensor([0, 1, -1, 5], dtype=torch.int32, device=DEV))
    assert p.check() == (L.LORA_DATA_BAD_ID | L.LORA_DATA_EMPTY_SLOT)
    p2 = L.Plan(table, idx=torch.tensor([0, -1, 0], dtype=torch.int32, device=DEV))
    assert p2.check() == 0

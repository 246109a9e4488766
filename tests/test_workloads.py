"""The seeded input generators: encodings and the five workload recipes (CPU)."""
import numpy as np
import pytest
import torch

import oracle
import workloads


def test_bf16_rne_matches_torch_on_f32_values():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
                        np.array([0.0, -0.0, 1.0, -1.5, 3.0e38, -3.0e38, 1e-39])])
    x32 = x.astype(np.float32)
    ours = workloads.bf16_bits_from_f64(x32.astype(np.float64))
    ref = torch.from_numpy(x32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_bf16_round_trip_and_specials():
    vals = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, np.inf, -np.inf, np.nan, 1e39])
    bits = workloads.bf16_bits_from_f64(vals)
    back = workloads.f64_from_bf16_bits(bits)
    assert back[0] == 1.0
    assert back[1] == 1.0                       # tie -> even
    assert back[2] == 1.0 + 2 ** -6             # tie -> even (up)
    assert np.isposinf(back[3]) and np.isneginf(back[4]) and np.isnan(back[5])
    assert np.isposinf(back[6])                 # overflow
    b = np.arange(0, 65536, dtype=np.uint16)
    f = workloads.f64_from_bf16_bits(b)
    finite = np.isfinite(f)
    assert np.array_equal(workloads.bf16_bits_from_f64(f[finite]), b[finite])


def test_direct_rounding_avoids_double_rounding():
    # 1 + 2^-8 + 2^-40 is above the bf16 tie: direct RNE rounds up; going through
    # binary32 first would land exactly on the tie and round to even (down).
    x = np.array([1.0 + 2 ** -8 + 2 ** -40])
    assert workloads.f64_from_bf16_bits(workloads.bf16_bits_from_f64(x))[0] == 1.0 + 2 ** -7


def test_config1_recipe():
    c = workloads.make_config(1)
    assert (c.n, c.d_in, c.d_out, c.num_slots) == (64, 256, 256, 4)
    assert c.idx.tolist() == sum([[a] * 16 for a in range(4)], [])
    assert c.X.dtype == np.float32 and c.Y.dtype == np.float32
    assert all(a.shape == (8, 256) for a in c.A) and all(b.shape == (256, 8) for b in c.B)


def test_config2_recipe():
    c = workloads.make_config(2)
    assert c.n == 256 and int((c.idx == -1).sum()) == 26
    live = c.idx[c.idx >= 0]
    assert live.min() >= 0 and live.max() < 64
    X = workloads.decode(c.X, "bf16")
    assert abs(X.std() - 1.0) < 0.02
    A = workloads.decode(c.A[0], "bf16")
    assert abs(A.std() * 64 - 1.0) < 0.05


def test_config5_recipe():
    c = workloads.make_config(5)
    assert c.n == 8192 and c.num_slots == 8 and (c.ranks == 32).all()
    lens = np.diff(c.seg_offsets)
    assert sorted(lens.tolist()) == sorted([512, 768, 1024, 1280, 1536, 256, 1792, 1024])
    assert abs(c.mask.mean() - 0.3) < 0.02
    p = oracle.canonical_plan(c.idx, 8, mask=c.mask)
    assert p["n_runs"] == 8


@pytest.fixture(scope="module")
def cfg4():
    return workloads.make_config(4)


def test_config4_recipe(cfg4):
    c = cfg4
    assert c.n == 4096 and c.num_slots == 256 and c.d_in == 5120
    assert set(np.unique(c.ranks).tolist()) <= {8, 16, 32, 64}
    assert np.allclose(c.scales * c.ranks, 16.0)
    counts = np.bincount(c.idx, minlength=256)
    assert counts[0] == counts.max()            # Zipf head
    assert (counts > 0).sum() > 150


def test_config3_structure():
    # the structure is drawn before any value, so a fresh generator reproduces it
    rng = np.random.Generator(np.random.PCG64(2))
    lens = np.clip(np.rint(rng.lognormal(np.log(1024) - 0.18, 0.6, 16)), 128, 4096)
    assert 128 <= lens.min() and lens.max() <= 4096
    assert 8000 < lens.sum() < 30000


def test_random_case_int_values_exact():
    c = workloads.random_case(3, 20, 16, 8, 3, int_values=True, x_dtype="bf16",
                              w_dtype="bf16", y_dtype="bf16")
    X = workloads.decode(c.X, "bf16")
    assert set(np.unique(X).tolist()) <= {-1.0, 0.0, 1.0}

"""The five seeded workloads of the mixed-adapter LoRA layer, plus fuzz cases.

Every case is drawn with ``numpy.random.Generator(PCG64(seed))`` in a fixed
order: structure (ids, segment lengths, ranks, mask, advantages), then X, then
A per slot in slot order, then B per slot in slot order, then Y, then dY.
Values are drawn in float64 and stored in the case's dtypes (see ``encode``).

Shapes follow the paper's LoRA definition (Section 3.4, the adapted linear
layer): ``A_a`` is ``[r_a, d_in]`` and ``B_a`` is ``[d_out, r_a]``, both row-major;
``X`` is ``[n, d_in]``, ``Y`` and ``dY`` are ``[n, d_out]``.  An id of -1 marks a
row with no adapter.  A slot with rank 0 is empty.
"""
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from .encode import encode

CONFIG_NAMES = {
    1: "tiny_sgmv_fp32",
    2: "decode_bgmv",
    3: "prefill_sgmv",
    4: "skewed_hetero",
    5: "masked_backward",
}

_ROW_CHUNK = 2048          # rows drawn per call; the stream is identical to one call


@dataclass
class Case:
    name: str
    seed: int
    n: int
    d_in: int
    d_out: int
    num_slots: int
    ranks: np.ndarray                      # int32 [S]; 0 = empty slot
    scales: np.ndarray                     # float32 [S]
    idx: np.ndarray                        # int32 [n]; -1 = no adapter
    x_dtype: str
    w_dtype: str
    y_dtype: str
    X: np.ndarray                          # storage [n, d_in]
    A: List[Optional[np.ndarray]]          # storage [r_a, d_in] per slot
    B: List[Optional[np.ndarray]]          # storage [d_out, r_a] per slot
    Y: Optional[np.ndarray] = None         # storage [n, d_out]
    dY: Optional[np.ndarray] = None        # storage [n, d_out]
    mask: Optional[np.ndarray] = None      # uint8 [n]; nonzero = trainable
    seg_offsets: Optional[np.ndarray] = None   # int32 [num_segs + 1]
    seg_adapter: Optional[np.ndarray] = None   # int32 [num_segs]
    meta: dict = field(default_factory=dict)

    @property
    def r_max(self):
        return int(self.ranks.max()) if self.ranks.size else 0


def segments_to_idx(seg_offsets, seg_adapter, n):
    """Expand contiguous segments into a per-row adapter id array (rows not
    covered by any segment get -1)."""
    idx = np.full(n, -1, dtype=np.int32)
    for s in range(len(seg_adapter)):
        idx[seg_offsets[s]:seg_offsets[s + 1]] = seg_adapter[s]
    return idx


def _normal(rng, shape, std, dtype):
    """Draw N(0, std^2) values row-chunk by row-chunk and encode them."""
    shape = tuple(int(s) for s in shape)
    if len(shape) == 1:
        return encode(rng.standard_normal(shape[0]) * std, dtype)
    rows, cols = shape
    out = np.empty(shape, dtype=np.uint16 if dtype == "bf16" else np.float32)
    for r0 in range(0, rows, _ROW_CHUNK):
        r1 = min(rows, r0 + _ROW_CHUNK)
        out[r0:r1] = encode(rng.standard_normal((r1 - r0, cols)) * std, dtype)
    return out


def _draw_values(rng, case_kw, x_std, a_std, b_std, *, want_y, want_dy, dy_row_scale=None):
    """Draw X, A (slot order), B (slot order), Y, dY in that order."""
    n, d_in, d_out = case_kw["n"], case_kw["d_in"], case_kw["d_out"]
    ranks = case_kw["ranks"]
    xd, wd, yd = case_kw["x_dtype"], case_kw["w_dtype"], case_kw["y_dtype"]
    X = _normal(rng, (n, d_in), x_std, xd)
    A, B = [], []
    for a, r in enumerate(ranks):
        A.append(_normal(rng, (int(r), d_in), a_std, wd) if r > 0 else None)
    for a, r in enumerate(ranks):
        std = b_std(int(r)) if callable(b_std) else b_std
        B.append(_normal(rng, (d_out, int(r)), std, wd) if r > 0 else None)
    Y = _normal(rng, (n, d_out), 1.0, yd) if want_y else None
    dY = None
    if want_dy:
        if dy_row_scale is None:
            dY = _normal(rng, (n, d_out), 1.0, xd)
        else:
            dY = np.empty((n, d_out), dtype=np.uint16 if xd == "bf16" else np.float32)
            for r0 in range(0, n, _ROW_CHUNK):
                r1 = min(n, r0 + _ROW_CHUNK)
                z = rng.standard_normal((r1 - r0, d_out))
                dY[r0:r1] = encode(z * dy_row_scale[r0:r1, None], xd)
    return X, A, B, Y, dY


def _config1(seed, y_dtype=None):
    rng = np.random.Generator(np.random.PCG64(seed))
    n, d, S, r = 64, 256, 4, 8
    seg_offsets = np.arange(0, n + 1, 16, dtype=np.int32)
    seg_adapter = np.arange(S, dtype=np.int32)
    kw = dict(n=n, d_in=d, d_out=d, ranks=np.full(S, r, np.int32),
              x_dtype="f32", w_dtype="f32", y_dtype=y_dtype or "f32")
    X, A, B, Y, _ = _draw_values(rng, kw, 1 / np.sqrt(d), 1 / np.sqrt(d),
                                 1 / np.sqrt(r), want_y=True, want_dy=False)
    return Case(name=CONFIG_NAMES[1], seed=seed, num_slots=S,
                scales=np.full(S, 2.0, np.float32),
                idx=segments_to_idx(seg_offsets, seg_adapter, n),
                X=X, A=A, B=B, Y=Y, seg_offsets=seg_offsets, seg_adapter=seg_adapter,
                **kw)


def _config2(seed, y_dtype=None):
    rng = np.random.Generator(np.random.PCG64(seed))
    n, d, S, r = 256, 4096, 64, 16
    idx = rng.integers(0, S, size=n).astype(np.int32)
    none_rows = rng.choice(n, size=int(round(0.1 * n)), replace=False)
    idx[none_rows] = -1
    kw = dict(n=n, d_in=d, d_out=d, ranks=np.full(S, r, np.int32),
              x_dtype="bf16", w_dtype="bf16", y_dtype=y_dtype or "bf16")
    X, A, B, Y, _ = _draw_values(rng, kw, 1.0, 1 / np.sqrt(d), 1 / np.sqrt(r),
                                 want_y=True, want_dy=False)
    return Case(name=CONFIG_NAMES[2], seed=seed, num_slots=S,
                scales=np.full(S, 2.0, np.float32), idx=idx, X=X, A=A, B=B, Y=Y, **kw)


def _config3(seed, y_dtype=None):
    rng = np.random.Generator(np.random.PCG64(seed))
    d_in, d_out, S, r, nseq = 4096, 14336, 32, 64, 16
    mu = np.log(1024.0) - 0.5 * 0.6 ** 2     # unclipped mean length 1024
    lens = np.clip(np.rint(rng.lognormal(mean=mu, sigma=0.6, size=nseq)), 128, 4096)
    lens = lens.astype(np.int32)
    seg_adapter = rng.integers(0, S, size=nseq).astype(np.int32)
    seg_offsets = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    n = int(seg_offsets[-1])
    kw = dict(n=n, d_in=d_in, d_out=d_out, ranks=np.full(S, r, np.int32),
              x_dtype="bf16", w_dtype="bf16", y_dtype=y_dtype or "bf16")
    X, A, B, Y, _ = _draw_values(rng, kw, 1.0, 1 / np.sqrt(d_in), 1 / np.sqrt(r),
                                 want_y=True, want_dy=False)
    return Case(name=CONFIG_NAMES[3], seed=seed, num_slots=S,
                scales=np.full(S, 2.0, np.float32),
                idx=segments_to_idx(seg_offsets, seg_adapter, n), X=X, A=A, B=B, Y=Y,
                seg_offsets=seg_offsets, seg_adapter=seg_adapter, **kw)


def _config4(seed, y_dtype=None):
    rng = np.random.Generator(np.random.PCG64(seed))
    d, S = 5120, 256
    ranks = rng.choice(np.array([8, 16, 32, 64]), size=S).astype(np.int32)
    pop = (np.arange(S) + 1.0) ** -1.1
    pop /= pop.sum()
    n_decode, n_prefill = 2048, 2048
    decode_ids = rng.choice(S, size=n_decode, p=pop)
    seg_lens, seg_ids, total = [], [], 0
    while total < n_prefill:
        L = int(rng.integers(64, 513))
        seg_lens.append(min(L, n_prefill - total))
        seg_ids.append(int(rng.choice(S, p=pop)))
        total += seg_lens[-1]
    units = [("d", int(a)) for a in decode_ids] + list(zip(seg_lens, seg_ids))
    order = rng.permutation(len(units))
    idx_parts = []
    for u in order:
        kind, val = units[u]
        if kind == "d":
            idx_parts.append(np.array([val], np.int32))
        else:
            idx_parts.append(np.full(kind, val, np.int32))
    idx = np.concatenate(idx_parts).astype(np.int32)
    n = idx.size
    kw = dict(n=n, d_in=d, d_out=d, ranks=ranks,
              x_dtype="bf16", w_dtype="bf16", y_dtype=y_dtype or "bf16")
    X, A, B, Y, _ = _draw_values(rng, kw, 1.0, 1 / np.sqrt(d), lambda r: 1 / np.sqrt(r),
                                 want_y=True, want_dy=False)
    return Case(name=CONFIG_NAMES[4], seed=seed, num_slots=S,
                scales=(16.0 / ranks).astype(np.float32), idx=idx, X=X, A=A, B=B, Y=Y,
                meta=dict(n_segments=len(seg_lens)), **kw)


def _config5(seed, y_dtype=None):
    rng = np.random.Generator(np.random.PCG64(seed))
    d, S, r = 4096, 8, 32
    lens = rng.permutation(np.array([512, 768, 1024, 1280, 1536, 256, 1792, 1024]))
    seg_offsets = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    seg_adapter = np.arange(S, dtype=np.int32)
    n = int(seg_offsets[-1])
    mask = (rng.random(n) < 0.3).astype(np.uint8)
    adv = rng.standard_normal(S)
    idx = segments_to_idx(seg_offsets, seg_adapter, n)
    row_adv = adv[idx]
    kw = dict(n=n, d_in=d, d_out=d, ranks=np.full(S, r, np.int32),
              x_dtype="bf16", w_dtype="bf16", y_dtype=y_dtype or "bf16")
    X, A, B, _, dY = _draw_values(rng, kw, 1.0, 1 / np.sqrt(d), 1 / np.sqrt(r),
                                  want_y=False, want_dy=True, dy_row_scale=row_adv)
    return Case(name=CONFIG_NAMES[5], seed=seed, num_slots=S,
                scales=np.full(S, 2.0, np.float32), idx=idx, X=X, A=A, B=B, dY=dY,
                mask=mask, seg_offsets=seg_offsets, seg_adapter=seg_adapter,
                meta=dict(advantages=adv), **kw)


_MAKERS = {1: _config1, 2: _config2, 3: _config3, 4: _config4, 5: _config5}


def make_config(k, seed=None, y_dtype=None):
    """Draw workload ``k`` (1..5).  The default seed is ``k - 1``."""
    return _MAKERS[k](k - 1 if seed is None else seed, y_dtype=y_dtype)


def base_weight(case, seed=None, dtype=None, int_values=False):
    """The base layer's weight W [d_out, d_in] for a case (the shared
    projection of the adapted layer): N(0, 1/d_in) so that x W^T has unit
    variance for unit-variance x, drawn from its own generator (seed defaults
    to 1000 + the case's seed) so the case's other draws are unchanged.
    ``int_values`` draws values in {-1, 0, 1}."""
    seed = 1000 + case.seed if seed is None else seed
    dtype = dtype or case.w_dtype
    rng = np.random.Generator(np.random.PCG64(seed))
    if int_values:
        return encode(rng.integers(-1, 2, (case.d_out, case.d_in)).astype(np.float64), dtype)
    return _normal(rng, (case.d_out, case.d_in), 1.0 / np.sqrt(case.d_in), dtype)


def random_case(seed, n, d_in, d_out, num_slots, *, ranks=None, rank_choices=(16,),
                frac_none=0.1, layout="random", seg_len=(1, 64), mask_p=None,
                x_dtype="bf16", w_dtype="bf16", y_dtype="f32", scales=None,
                empty_slots=(), want_y=True, want_dy=False, int_values=False):
    """A fuzz case.  ``layout`` is 'random' (iid ids), 'segments' (contiguous
    runs of one adapter with lengths in ``seg_len``), 'alternating' or 'single'
    (every row on slot 0).  ``int_values`` draws values in {-1, 0, 1} so that
    every product and sum is exactly representable."""
    rng = np.random.Generator(np.random.PCG64(seed))
    S = num_slots
    if ranks is None:
        ranks = rng.choice(np.asarray(rank_choices), size=S).astype(np.int32)
    ranks = np.asarray(ranks, np.int32).copy()
    for e in empty_slots:
        ranks[e] = 0
    live = np.nonzero(ranks > 0)[0]
    if layout == "random":
        idx = rng.choice(live, size=n).astype(np.int32) if live.size else np.full(n, -1, np.int32)
    elif layout == "segments":
        parts, total = [], 0
        while total < n:
            L = min(int(rng.integers(seg_len[0], seg_len[1] + 1)), n - total)
            parts.append(np.full(L, rng.choice(live), np.int32))
            total += L
        idx = np.concatenate(parts) if parts else np.zeros(0, np.int32)
    elif layout == "alternating":
        idx = live[np.arange(n) % max(1, live.size)].astype(np.int32)
    elif layout == "single":
        idx = np.zeros(n, np.int32)
    else:
        raise ValueError(layout)
    idx = idx.astype(np.int32)
    if frac_none > 0 and n > 0:
        none_rows = rng.choice(n, size=int(round(frac_none * n)), replace=False)
        idx[none_rows] = -1
    mask = None
    if mask_p is not None:
        mask = (rng.random(n) < mask_p).astype(np.uint8)
    if scales is None:
        scales = rng.choice(np.array([0.25, 0.5, 1.0, 2.0]), size=S)
    scales = np.asarray(scales, np.float32)
    kw = dict(n=n, d_in=d_in, d_out=d_out, ranks=ranks,
              x_dtype=x_dtype, w_dtype=w_dtype, y_dtype=y_dtype)
    if int_values:
        def ints(shape, dt):
            return encode(rng.integers(-1, 2, size=shape).astype(np.float64), dt)
        X = ints((n, d_in), x_dtype)
        A = [ints((int(r), d_in), w_dtype) if r > 0 else None for r in ranks]
        B = [ints((d_out, int(r)), w_dtype) if r > 0 else None for r in ranks]
        Y = encode(rng.integers(-8, 9, size=(n, d_out)).astype(np.float64), y_dtype) if want_y else None
        dY = ints((n, d_out), x_dtype) if want_dy else None
    else:
        X, A, B, Y, dY = _draw_values(
            rng, kw, 1.0, 1 / np.sqrt(d_in), lambda r: 1 / np.sqrt(max(r, 1)),
            want_y=want_y, want_dy=want_dy)
    return Case(name=f"fuzz_s{seed}", seed=seed, num_slots=S, scales=scales, idx=idx,
                X=X, A=A, B=B, Y=Y, dY=dY, mask=mask, **kw)

"""Pins of the float64 oracle against things other than itself (CPU only).

* hand-derived worked examples (tests/golden/*.txt),
* scalar brute force on tiny inputs (a different evaluation order and no
  grouping / gather / scatter),
* exact linearity of the masked loss in A and in B, which ties the backward to
  the forward without restating the gradient formula,
* closed forms (permutation x diagonal adapters, rank-1 adapters),
* integer-valued inputs checked with exact Python integer arithmetic,
* invariants (id -1 rows bit-identical, zero B, permutation, mask exactness),
* planted mistakes: each plausible bug in the oracle must make a pin fail.
"""
import fractions
import types

import numpy as np
import pytest

import oracle
import workloads
from helpers import f64_case, load_golden

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


# ----------------------------------------------------------------------------
# pin checks, parameterised by the implementation so planted mistakes can be run
# ----------------------------------------------------------------------------

def check_plan_golden(impl):
    g = load_golden("plan_worked_example.txt")
    p = impl.canonical_plan(g["idx"].astype(np.int64), int(g["num_slots"][0]),
                            mask=g["mask"].astype(np.uint8))
    for k in ("counts", "offsets", "perm", "run_start", "run_len", "run_adapter",
              "m_counts", "m_offsets", "m_perm"):
        if not np.array_equal(np.asarray(p[k]), g[k].astype(np.int64)):
            return False
    return p["n_runs"] == int(g["n_runs"][0]) and p["error"] == bool(g["error"][0])


def check_plan_empty_slot_golden(impl):
    """Rows naming an empty slot (rank 0) carry no adapter and raise the flag."""
    g = load_golden("plan_empty_slot_example.txt")
    p = impl.canonical_plan(g["idx"].astype(np.int64), int(g["num_slots"][0]),
                            mask=g["mask"].astype(np.uint8), ranks=g["ranks"].astype(np.int64))
    for k in ("counts", "offsets", "perm", "run_start", "run_len", "run_adapter",
              "m_counts", "m_offsets", "m_perm", "eff"):
        if not np.array_equal(np.asarray(p[k]), g[k].astype(np.int64)):
            return False
    return p["n_runs"] == int(g["n_runs"][0]) and p["error"] == bool(g["error"][0])


def _plan_fuzz_cases():
    """(idx, S, mask, ranks): ranks hold zeros (empty slots) in half the cases."""
    rng = np.random.default_rng(1234)
    cases = [
        (np.full(37, -1), 5, None, None),
        (np.zeros(50, np.int64), 1, None, None),
        (np.arange(40) % 7, 7, rng.integers(0, 2, 40), None),
        (np.zeros(0, np.int64), 3, None, None),
        (np.array([3, 3, 3, -1, 3, 9, -7, 0]), 4, np.array([1, 0, 1, 1, 1, 1, 1, 0]), None),
        (np.array([0, 1, 1, 2, 0, 1]), 3, None, np.array([4, 0, 8])),
        (np.arange(30) % 5, 5, rng.integers(0, 2, 30), np.zeros(5, np.int64)),
    ]
    for s in range(40):
        n = int(rng.integers(1, 300))
        S = int(rng.integers(1, 40))
        idx = rng.integers(-2, S + 1, n)
        seg = rng.random() < 0.5
        if seg:
            idx = np.repeat(rng.integers(-1, S, n // 9 + 1), 9)[:n]
        mask = rng.integers(0, 2, n) if rng.random() < 0.6 else None
        ranks = None
        if s % 2 == 0:
            ranks = rng.integers(1, 65, S)
            ranks[rng.random(S) < 0.3] = 0
        cases.append((idx, S, mask, ranks))
    return cases


def check_plan_bruteforce(impl):
    for idx, S, mask, ranks in _plan_fuzz_cases():
        if ranks is None:
            ranks = np.ones(S, np.int64)
        p = impl.canonical_plan(idx, S, mask=mask, ranks=ranks)
        b = oracle.plan_bruteforce(list(idx), S, mask=None if mask is None else list(mask),
                                   ranks=list(ranks))
        for k in ("counts", "offsets", "perm", "run_start", "run_len", "run_adapter",
                  "m_counts", "m_offsets", "m_perm"):
            if not np.array_equal(np.asarray(p[k], np.int64), np.asarray(b[k], np.int64)):
                return False
        if p["n_runs"] != b["n_runs"] or p["error"] != b["error"]:
            return False
    return True


def _golden_forward():
    g = load_golden("forward_worked_example.txt")
    d_in, d_out = int(g["d_in"][0]), int(g["d_out"][0])
    r = g["rank"].astype(int)
    A = [g["A0"].reshape(r[0], d_in), g["A1"].reshape(r[1], d_in)]
    B = [g["B0"].reshape(d_out, r[0]), g["B1"].reshape(d_out, r[1])]
    X = g["X"].reshape(-1, d_in)
    Y = g["Y"].reshape(-1, d_out)
    return g, A, B, X, Y, g["idx"].astype(np.int64), g["scale"]


def check_forward_golden(impl):
    g, A, B, X, Y, idx, s = _golden_forward()
    out = impl.apply(idx, X, Y, A, B, s)
    return np.array_equal(out, g["Y_out"].reshape(Y.shape))


def _tiny_case(seed, n=13, d_in=7, d_out=5, S=3, mask_p=None, frac_none=0.2):
    c = workloads.random_case(seed, n, d_in, d_out, S, rank_choices=(1, 2, 3, 4),
                              frac_none=frac_none, x_dtype="f32", w_dtype="f32",
                              y_dtype="f32", mask_p=mask_p, want_dy=mask_p is not None)
    X, A, B, Y, dY = f64_case(c)
    eff, _ = oracle.effective_ids(c.idx, S, c.ranks)
    return c, eff, X, A, B, Y, dY


def check_forward_bruteforce(impl):
    for seed in range(6):
        c, eff, X, A, B, Y, _ = _tiny_case(seed)
        ref = oracle.apply_bruteforce(eff, X, Y, A, B, c.scales)
        out = impl.apply(eff, X, Y, A, B, c.scales)
        if not np.allclose(out, ref, rtol=1e-12, atol=1e-12):
            return False
    return True


def check_forward_closed_form(impl):
    """A = permutation matrix, B = diagonal: Delta[t, o] = s * d_o * X[t, pi(o)]."""
    rng = np.random.default_rng(7)
    n, d = 9, 6
    pi = rng.permutation(d)
    P = np.zeros((d, d))
    P[np.arange(d), pi] = 1.0                    # (X P^T)[t, j] = X[t, pi(j)]
    diag = rng.integers(1, 9, d).astype(np.float64)
    X = rng.integers(-5, 6, (n, d)).astype(np.float64)
    Y = rng.integers(-5, 6, (n, d)).astype(np.float64)
    idx = np.zeros(n, np.int64)
    out = impl.apply(idx, X, Y, [P], [np.diag(diag)], np.array([0.5]))
    expect = Y + 0.5 * diag[None, :] * X[:, pi]
    if not np.array_equal(out, expect):
        return False
    # rank-1: A = u^T, B = v  ->  Delta[t] = s (X[t] . u) v
    u = rng.integers(-3, 4, d).astype(np.float64)
    v = rng.integers(-3, 4, d + 2).astype(np.float64)
    Y2 = np.zeros((n, d + 2))
    out = impl.apply(idx, X, Y2, [u[None, :]], [v[:, None]], np.array([2.0]))
    expect = np.array([[2.0 * sum(X[t, k] * u[k] for k in range(d)) * v[o]
                        for o in range(d + 2)] for t in range(n)])
    return np.array_equal(out, expect)


def check_forward_integer_exact(impl):
    """Integer inputs, power-of-two scales: compare with exact rational arithmetic."""
    c = workloads.random_case(21, 40, 24, 20, 4, rank_choices=(1, 3, 8), frac_none=0.25,
                              x_dtype="f32", w_dtype="f32", y_dtype="f32", int_values=True)
    X, A, B, Y, _ = f64_case(c)
    eff, _ = oracle.effective_ids(c.idx, c.num_slots, c.ranks)
    out = impl.apply(eff, X, Y, A, B, c.scales)
    for t in range(c.n):
        a = int(eff[t])
        for o in range(c.d_out):
            exp = fractions.Fraction(int(Y[t, o]))
            if a >= 0:
                h = [sum(int(X[t, k]) * int(A[a][j, k]) for k in range(c.d_in))
                     for j in range(A[a].shape[0])]
                exp += fractions.Fraction(float(c.scales[a])) * sum(
                    h[j] * int(B[a][o, j]) for j in range(len(h)))
            if fractions.Fraction(out[t, o]) != exp:
                return False
    return True


def check_grad_golden(impl):
    g, A, B, X, _, idx, s = _golden_forward()
    gg = load_golden("grad_worked_example.txt")
    dY = gg["dY"].reshape(X.shape[0], -1)
    for tag in ("a", "b"):
        mask = gg["mask_" + tag].astype(np.uint8)
        dA, dB = impl.grad(idx, mask, X, dY, A, B, s)
        for a in range(2):
            if not np.array_equal(dA[a].ravel(), gg[f"dA{a}_{tag}"]):
                return False
            if not np.array_equal(dB[a].ravel(), gg[f"dB{a}_{tag}"]):
                return False
        if impl.masked_loss(idx, mask, X, dY, A, B, s) != gg["loss_" + tag][0]:
            return False
    return True


def check_grad_linearity(impl):
    """L(A + eps E) - L(A) = eps <dA, E> and the same for B, exactly up to f64
    rounding, because the masked loss is linear in A (B fixed) and in B (A fixed).
    The loss uses the forward oracle, so this ties the backward to the forward."""
    for seed in range(4):
        c, eff, X, A, B, Y, dY = _tiny_case(100 + seed, n=17, mask_p=0.6)
        dA, dB = impl.grad(eff, c.mask, X, dY, A, B, c.scales)
        L0 = oracle.masked_loss(eff, c.mask, X, dY, A, B, c.scales)
        rng = np.random.default_rng(seed)
        for a in range(c.num_slots):
            if A[a] is None:
                continue
            for which in ("A", "B"):
                W = A if which == "A" else B
                E = rng.standard_normal(W[a].shape)
                eps = 0.37
                W2 = [w.copy() if w is not None else None for w in W]
                W2[a] = W[a] + eps * E
                L1 = oracle.masked_loss(eff, c.mask, X, dY, W2 if which == "A" else A,
                                        B if which == "A" else W2, c.scales)
                g = dA[a] if which == "A" else dB[a]
                pred = eps * float(np.sum(g * E))
                if abs((L1 - L0) - pred) > 1e-10 * max(1.0, abs(pred), abs(L0)):
                    return False
    return True


def check_grad_bruteforce(impl):
    for seed in range(3):
        c, eff, X, A, B, Y, dY = _tiny_case(200 + seed, n=11, d_in=5, d_out=4, mask_p=0.5)
        dA, dB = impl.grad(eff, c.mask, X, dY, A, B, c.scales)
        rA, rB = oracle.grad_bruteforce(eff, c.mask, X, dY, A, B, c.scales)
        for a in range(c.num_slots):
            if A[a] is None:
                continue
            if not (np.allclose(dA[a], rA[a], rtol=1e-12, atol=1e-12)
                    and np.allclose(dB[a], rB[a], rtol=1e-12, atol=1e-12)):
                return False
    return True


def check_grad_mask_exact(impl):
    """Masked-out rows hold NaN / Inf / 1e30 in X and dY: dA, dB are byte-identical
    to the run where those rows are zero."""
    c, eff, X, A, B, Y, dY = _tiny_case(300, n=19, mask_p=0.5)
    out = c.mask == 0
    X0, dY0 = X.copy(), dY.copy()
    X0[out] = 0.0
    dY0[out] = 0.0
    X1, dY1 = X.copy(), dY.copy()
    junk = np.array([np.nan, np.inf, -np.inf, 1e30])
    X1[out] = junk[np.arange(X1[out].size) % 4].reshape(X1[out].shape)
    dY1[out] = junk[np.arange(dY1[out].size) % 4].reshape(dY1[out].shape)
    a0, b0 = impl.grad(eff, c.mask, X0, dY0, A, B, c.scales)
    a1, b1 = impl.grad(eff, c.mask, X1, dY1, A, B, c.scales)
    for a in range(c.num_slots):
        if A[a] is None:
            continue
        if a0[a].tobytes() != a1[a].tobytes() or b0[a].tobytes() != b1[a].tobytes():
            return False
    return True


def check_grad_x_linearity(impl):
    """L(X + eps E) - L(X) = eps <dX, E> exactly up to f64 rounding: the masked
    loss is linear in X, and it is evaluated by the forward oracle."""
    for seed in range(4):
        c, eff, X, A, B, Y, dY = _tiny_case(400 + seed, n=17, mask_p=0.6)
        dX = impl.grad_x(eff, c.mask, dY, A, B, c.scales, np.zeros_like(X))
        L0 = oracle.masked_loss(eff, c.mask, X, dY, A, B, c.scales)
        E = np.random.default_rng(seed).standard_normal(X.shape)
        eps = 0.29
        L1 = oracle.masked_loss(eff, c.mask, X + eps * E, dY, A, B, c.scales)
        pred = eps * float(np.sum(dX * E))
        if abs((L1 - L0) - pred) > 1e-10 * max(1.0, abs(pred), abs(L0)):
            return False
    return True


def check_grad_x_bruteforce(impl):
    for seed in range(3):
        c, eff, X, A, B, Y, dY = _tiny_case(500 + seed, n=11, d_in=5, d_out=4, mask_p=0.5)
        dX0 = np.random.default_rng(seed).standard_normal(X.shape)
        got = impl.grad_x(eff, c.mask, dY, A, B, c.scales, dX0)
        ref = oracle.grad_x_bruteforce(eff, c.mask, dY, A, B, c.scales, dX0)
        if not np.allclose(got, ref, rtol=1e-12, atol=1e-12):
            return False
    return True


def check_grad_x_dense_and_untouched(impl):
    """One adapter, no mask: dX + s dY (B A) by numpy in the other association.
    Rows with id -1 or mask 0 come back bit-identical, whatever their dY holds."""
    c, eff, X, A, B, Y, dY = _tiny_case(600, n=9, S=1, frac_none=0.0, mask_p=0.5)
    dX0 = np.random.default_rng(1).standard_normal(X.shape)
    got = impl.grad_x(eff, None, dY, A, B, c.scales, dX0)
    ref = dX0 + float(c.scales[0]) * (dY @ (B[0] @ A[0]))
    if not np.allclose(got, ref, rtol=1e-12, atol=1e-12):
        return False
    c, eff, X, A, B, Y, dY = _tiny_case(601, n=19, mask_p=0.5, frac_none=0.3)
    out = (c.mask == 0) | (eff < 0)
    dYj = dY.copy()
    junk = np.array([np.nan, np.inf, -np.inf, 1e30])
    dYj[out] = junk[np.arange(dYj[out].size) % 4].reshape(dYj[out].shape)
    dX0 = np.random.default_rng(2).standard_normal(X.shape)
    got = impl.grad_x(eff, c.mask, dYj, A, B, c.scales, dX0)
    clean = impl.grad_x(eff, c.mask, np.where(out[:, None], 0.0, dY), A, B, c.scales, dX0)
    return got[out].tobytes() == dX0[out].tobytes() and got.tobytes() == clean.tobytes()


ADAMW_SETS = [  # (lr, beta1, beta2, eps, weight_decay)
    (1e-3, 0.9, 0.999, 1e-8, 0.01),
    (3e-2, 0.8, 0.95, 1e-3, 0.1),
    (1e-2, 0.0, 0.5, 1e-6, 0.0),
    (5e-4, 0.95, 0.9999, 1e-8, 1.0),
]


def check_adamw_torch(impl):
    """Six steps against torch.optim.AdamW in float64 (an independent
    implementation of the published algorithm), the state carried across steps."""
    import torch
    for k, (lr, b1, b2, eps, wd) in enumerate(ADAMW_SETS):
        rng = np.random.default_rng(700 + k)
        p0 = rng.standard_normal(37) * 0.3
        tp = torch.nn.Parameter(torch.from_numpy(p0.copy()))
        opt = torch.optim.AdamW([tp], lr=lr, betas=(b1, b2), eps=eps, weight_decay=wd)
        p, m, v = p0.copy(), np.zeros(37), np.zeros(37)
        for t in range(1, 7):
            g = rng.standard_normal(37) * (0.1 if t % 2 else 2.0)
            g[::5] = 0.0
            tp.grad = torch.from_numpy(g.copy())
            opt.step()
            p, m, v = impl.adamw(p, m, v, g, t, lr, b1, b2, eps, wd)
            if not np.allclose(p, tp.detach().numpy(), rtol=1e-12, atol=1e-15):
                return False
            st = opt.state[tp]
            if not (np.allclose(m, st["exp_avg"].numpy(), rtol=1e-12, atol=1e-300) and
                    np.allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-12, atol=1e-300)):
                return False
    return True


def check_adamw_closed_forms(impl):
    """From zero moments: the first step is p - lr (g / (|g| + eps) + wd p); a
    zero gradient only decays, p (1 - lr wd)^t; a constant gradient with no
    decay moves every step by lr g / (|g| + eps) (the bias corrections make
    mhat = g and vhat = g^2 at every t)."""
    rng = np.random.default_rng(800)
    p0 = rng.standard_normal(50)
    g = rng.standard_normal(50)
    g[3] = 0.0
    z = np.zeros(50)
    for lr, b1, b2, eps, wd in ADAMW_SETS:
        p1, m1, v1 = impl.adamw(p0, z, z, g, 1, lr, b1, b2, eps, wd)
        if not np.allclose(p1, p0 - lr * (g / (np.abs(g) + eps) + wd * p0), rtol=1e-12, atol=1e-15):
            return False
        p, m, v = p0, z, z
        for t in range(1, 6):
            p, m, v = impl.adamw(p, m, v, z, t, lr, b1, b2, eps, wd)
        if not np.allclose(p, p0 * (1.0 - lr * wd) ** 5, rtol=1e-12, atol=1e-15):
            return False
        p, m, v = p0, z, z
        for t in range(1, 8):
            p, m, v = impl.adamw(p, m, v, g, t, lr, b1, b2, eps, 0.0)
        if not np.allclose(p, p0 - 7 * lr * g / (np.abs(g) + eps), rtol=1e-10, atol=1e-13):
            return False
    return True


def _loss_case(seed, n=9, V=13, kind=0):
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((n, V)) * 2.0
    z[1] += 800.0                           # large logits: exp overflows unless shifted
    z[2, 3] = -700.0
    y = rng.integers(0, V, n)
    w = rng.uniform(0.5, 2.0, n)
    w[[0, 4]] = 0.0
    mask = (rng.random(n) < 0.7).astype(np.uint8)
    mask[1] = 1
    adv = rng.standard_normal(n)
    corr = rng.uniform(0.5, 1.5, n)
    old = rng.standard_normal(n) - 2.0
    return z, y, w, mask, old, adv, corr


def check_loss_ce_torch(impl):
    """Cross-entropy, its log-probabilities and gradient against torch in float64
    (reduction 'none', weighted sum differentiated by autograd)."""
    import torch
    import torch.nn.functional as F
    for seed in range(3):
        z, y, w, *_ = _loss_case(900 + seed)
        L, lp, dz = impl.token_loss(oracle.LOSS_CE, z, y, weight=w)
        tz = torch.tensor(z, requires_grad=True)
        ce = F.cross_entropy(tz, torch.tensor(y), reduction="none")
        (torch.tensor(w) * ce).sum().backward()
        act = w != 0
        if not (np.allclose(L, w * ce.detach().numpy(), rtol=1e-12, atol=1e-12) and
                np.allclose(lp[act], -ce.detach().numpy()[act], rtol=1e-12, atol=1e-12) and
                np.all(lp[~act] == 0) and
                np.allclose(dz, tz.grad.numpy(), rtol=1e-10, atol=1e-14)):
            return False
    return True


def check_loss_finite_differences(impl):
    """dz against central differences of the summed loss, every kind (rows kept
    away from the PPO clip edges, where the loss has a kink)."""
    h = 1e-6
    for kind in (oracle.LOSS_CE, oracle.LOSS_IS, oracle.LOSS_PPO):
        z, y, w, mask, old, adv, corr = _loss_case(950 + kind, n=5, V=6)
        z[1] -= 800.0
        _, lp0, _ = oracle.token_loss(oracle.LOSS_CE, z, y, weight=np.ones(5))
        rho = np.array([0.5, 0.95, 1.05, 1.6, 0.7])
        old = lp0 - np.log(rho)
        kw = dict(weight=w, mask=mask, old_logp=old, adv=adv, corr=corr, clip_lo=0.2, clip_hi=0.25)
        _, _, dz = impl.token_loss(kind, z, y, **kw)
        num = np.zeros_like(z)
        for t in range(z.shape[0]):
            for v in range(z.shape[1]):
                zp, zm = z.copy(), z.copy()
                zp[t, v] += h
                zm[t, v] -= h
                num[t, v] = (impl.token_loss(kind, zp, y, **kw)[0].sum() -
                             impl.token_loss(kind, zm, y, **kw)[0].sum()) / (2 * h)
        if not np.allclose(dz, num, rtol=1e-6, atol=1e-8):
            return False
    return True


def check_loss_closed_forms(impl):
    """Equal logits give logp = -log V; at rho = 1 the IS loss is -m c A; PPO at
    chosen ratios: clipped above / below (loss at the clip bound, no gradient)
    and unclipped (loss and gradient of the ratio term); inactive rows with NaN
    logits give zero loss, zero logp and a zero gradient row."""
    V = 11
    z = np.full((6, V), 0.37)
    y = np.array([0, 3, 5, 7, 10, 2])
    _, lp, _ = impl.token_loss(oracle.LOSS_CE, z, y, weight=np.ones(6))
    if not np.allclose(lp, -np.log(V), rtol=0, atol=1e-14):
        return False
    rng = np.random.default_rng(990)
    z = rng.standard_normal((6, V))
    _, lp, _ = impl.token_loss(oracle.LOSS_CE, z, y, weight=np.ones(6))
    soft = np.exp(z - z.max(1, keepdims=True))
    soft /= soft.sum(1, keepdims=True)
    onehot = np.eye(V)[y]
    c = np.array([1.0, 0.5, 2.0, 1.5, 0.8, 1.0])
    A = np.array([0.7, -1.3, 0.9, -0.4, 1.1, 0.6])
    m = np.array([1, 1, 1, 1, 1, 0], np.uint8)
    L, _, dz = impl.token_loss(oracle.LOSS_IS, z, y, mask=m, old_logp=lp, adv=A, corr=c)
    g = m * c * A
    if not (np.allclose(L, -g, rtol=1e-12, atol=1e-15) and
            np.allclose(dz, g[:, None] * (soft - onehot), rtol=1e-10, atol=1e-15)):
        return False
    #            A>0 rho>1+hi   A<0 rho<1-lo   A>0 rho<1-lo   A<0 rho>1+hi   inside  masked
    rho = np.array([1.5, 0.5, 0.5, 1.5, 1.1, 1.0])
    A = np.array([0.8, -0.6, 0.9, -0.7, 0.5, 0.3])
    zz = z.copy()
    zz[5] = np.nan
    L, lpp, dz = impl.token_loss(oracle.LOSS_PPO, zz, y, mask=m, old_logp=lp - np.log(rho), adv=A,
                                 corr=c, clip_lo=0.2, clip_hi=0.2)
    want_L = -c * np.array([1.2 * 0.8, 0.8 * -0.6, 0.5 * 0.9, 1.5 * -0.7, 1.1 * 0.5, 0.0])
    want_g = c * A * rho * np.array([0, 0, 1, 1, 1, 0])
    return bool(np.allclose(L, want_L, rtol=1e-12, atol=1e-15) and
                np.allclose(dz[:5], want_g[:5, None] * (soft[:5] - onehot[:5]), rtol=1e-10, atol=1e-15)
                and np.all(dz[5] == 0) and lpp[5] == 0 and L[5] == 0)


def check_metrics(impl):
    """The comparison metrics against hand-computed values: relative Frobenius
    error ||out - ref||_F / ||ref||_F and the largest absolute difference, with
    the zero-reference cases and NaN (a NaN output is never within tolerance)."""
    ref = np.array([[1.0, 2.0], [2.0, 4.0]])            # ||ref||_F = 5
    out = ref + np.array([[0.0, 3.0], [-4.0, 0.0]])     # ||out - ref||_F = 5
    if impl.rel_fro(out, ref) != 1.0 or impl.max_abs(out, ref) != 4.0:
        return False
    out = ref - np.array([[0.0, 0.0], [0.0, 0.5]])      # ||diff|| = 0.5, of 5
    if abs(impl.rel_fro(out, ref) - 0.1) > 1e-15 or impl.max_abs(out, ref) != 0.5:
        return False
    if impl.rel_fro(2.0 * ref, ref) != 1.0:              # normalised by ref, not out
        return False
    z = np.zeros((3, 2))
    if impl.rel_fro(z, z) != 0.0 or impl.max_abs(z, z) != 0.0:
        return False
    if impl.rel_fro(z + 1e-3, z) != float("inf"):
        return False
    if impl.max_abs(np.zeros(0), np.zeros(0)) != 0.0:
        return False
    bad = ref.copy()
    bad[0, 1] = np.nan
    if not (np.isnan(impl.rel_fro(bad, ref)) and np.isnan(impl.max_abs(bad, ref))):
        return False
    return True


def check_linear_golden(impl):
    g = load_golden("linear_worked_example.txt")
    d_in, d_out = int(g["d_in"][0]), int(g["d_out"][0])
    r = g["rank"].astype(int)
    X = g["X"].reshape(-1, d_in)
    W = g["W"].reshape(d_out, d_in)
    A = [g["A0"].reshape(r[0], d_in), g["A1"].reshape(r[1], d_in)]
    B = [g["B0"].reshape(d_out, r[0]), g["B1"].reshape(d_out, r[1])]
    out = impl.linear(g["idx"].astype(np.int64), X, W, A, B, g["scale"])
    return np.array_equal(out, g["Y_out"].reshape(-1, d_out))


def _linear_case(seed, n=11, d_in=7, d_out=5, S=3):
    c, eff, X, A, B, Y, _ = _tiny_case(seed, n=n, d_in=d_in, d_out=d_out, S=S)
    W = np.random.default_rng(seed + 500).standard_normal((d_out, d_in))
    return c, eff, X, W, A, B


def check_linear_bruteforce(impl):
    for seed in range(5):
        c, eff, X, W, A, B = _linear_case(seed)
        ref = oracle.linear_bruteforce(eff, X, W, A, B, c.scales)
        if not np.allclose(impl.linear(eff, X, W, A, B, c.scales), ref, rtol=1e-12, atol=1e-12):
            return False
    return True


def check_linear_merged_weights(impl):
    """Each row of adapter a equals x (W + s_a B_a A_a)^T (the adapter merged
    into the base weight, a different association of the same products); a
    row with no adapter equals x W^T."""
    for seed in range(4):
        c, eff, X, W, A, B = _linear_case(seed + 20, n=17, d_in=9, d_out=6, S=3)
        out = impl.linear(eff, X, W, A, B, c.scales)
        for t in range(c.n):
            a = int(eff[t])
            Wm = W if a < 0 else W + float(c.scales[a]) * (B[a] @ A[a])
            if not np.allclose(out[t], Wm @ X[t], rtol=1e-12, atol=1e-12):
                return False
    return True


def check_linear_zero_base_is_apply(impl):
    """W = 0 leaves the residual alone: the forward oracle applied to Y = 0."""
    c, eff, X, W, A, B = _linear_case(41)
    out = impl.linear(eff, X, np.zeros_like(W), A, B, c.scales)
    return np.allclose(out, oracle.apply(eff, X, np.zeros((c.n, W.shape[0])), A, B, c.scales),
                       rtol=1e-13, atol=1e-13)


def check_linear_integer_exact(impl):
    """Integer inputs and power-of-two scales: the result is exact, compared
    with exact rational arithmetic."""
    rng = np.random.default_rng(77)
    n, d_in, d_out, S = 9, 6, 4, 3
    X = rng.integers(-2, 3, (n, d_in)).astype(np.float64)
    W = rng.integers(-2, 3, (d_out, d_in)).astype(np.float64)
    ranks = [2, 1, 3]
    A = [rng.integers(-2, 3, (r, d_in)).astype(np.float64) for r in ranks]
    B = [rng.integers(-2, 3, (d_out, r)).astype(np.float64) for r in ranks]
    scale = np.array([0.5, 2.0, 0.25])
    eff = np.array([0, -1, 2, 1, 1, -1, 0, 2, 2])
    out = impl.linear(eff, X, W, A, B, scale)
    for t in range(n):
        for o in range(d_out):
            y = sum(fractions.Fraction(int(X[t, k]) * int(W[o, k])) for k in range(d_in))
            a = int(eff[t])
            if a >= 0:
                h = [sum(int(X[t, k]) * int(A[a][j, k]) for k in range(d_in)) for j in range(ranks[a])]
                y += fractions.Fraction(scale[a]) * sum(h[j] * int(B[a][o, j]) for j in range(ranks[a]))
            if fractions.Fraction(out[t, o]) != y:
                return False
    return True


ALL_CHECKS = [check_linear_golden, check_linear_bruteforce, check_linear_merged_weights,
              check_linear_zero_base_is_apply, check_linear_integer_exact, check_plan_golden, check_plan_empty_slot_golden, check_metrics, check_plan_bruteforce, check_forward_golden,
              check_forward_bruteforce, check_forward_closed_form,
              check_forward_integer_exact, check_grad_golden, check_grad_linearity,
              check_grad_bruteforce, check_grad_mask_exact, check_grad_x_linearity,
              check_grad_x_bruteforce, check_grad_x_dense_and_untouched, check_adamw_torch,
              check_adamw_closed_forms, check_loss_ce_torch, check_loss_finite_differences,
              check_loss_closed_forms]


# ----------------------------------------------------------------------------
# the oracle passes every pin
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    assert check(oracle)


def test_none_rows_bit_identical():
    """Rows with id -1 are copied bit for bit, including -0.0 and NaN payloads."""
    c, eff, X, A, B, Y, _ = _tiny_case(5)
    Y = Y.copy()
    none = np.nonzero(eff < 0)[0]
    Y[none[0], 0] = -0.0
    Y[none[-1], 1] = np.nan
    out = oracle.apply(eff, X, Y, A, B, c.scales)
    assert out[none].tobytes() == Y[none].tobytes()


def test_zero_B_or_A_leaves_Y():
    c, eff, X, A, B, Y, _ = _tiny_case(6)
    zB = [np.zeros_like(b) if b is not None else None for b in B]
    zA = [np.zeros_like(a) if a is not None else None for a in A]
    assert np.array_equal(oracle.apply(eff, X, Y, A, zB, c.scales), Y)
    assert np.array_equal(oracle.apply(eff, X, Y, zA, B, c.scales), Y)


def test_permutation_invariance():
    """Permuting rows permutes the output; gradients do not change."""
    c, eff, X, A, B, Y, dY = _tiny_case(8, n=31, mask_p=0.5)
    p = np.random.default_rng(3).permutation(c.n)
    out = oracle.apply(eff, X, Y, A, B, c.scales)
    outp = oracle.apply(eff[p], X[p], Y[p], A, B, c.scales)
    assert np.allclose(outp, out[p], rtol=1e-13, atol=1e-13)
    dA, dB = oracle.grad(eff, c.mask, X, dY, A, B, c.scales)
    dAp, dBp = oracle.grad(eff[p], c.mask[p], X[p], dY[p], A, B, c.scales)
    for a in range(c.num_slots):
        if A[a] is not None:
            assert np.allclose(dAp[a], dA[a], rtol=1e-12, atol=1e-12)
            assert np.allclose(dBp[a], dB[a], rtol=1e-12, atol=1e-12)


def test_shrink_then_expand_is_apply():
    c, eff, X, A, B, Y, _ = _tiny_case(9)
    H = oracle.shrink(eff, X, A)
    assert np.allclose(oracle.expand(eff, H, Y, B, c.scales),
                       oracle.apply(eff, X, Y, A, B, c.scales), rtol=1e-13, atol=1e-13)


def test_delta_rows_matches_apply():
    c, eff, X, A, B, Y, _ = _tiny_case(10)
    rows = np.arange(c.n)
    assert np.allclose(oracle.delta_rows(eff, X, A, B, c.scales, rows),
                       oracle.apply(eff, X, Y, A, B, c.scales) - Y, rtol=1e-12, atol=1e-12)


def test_segments_equal_ids():
    seg_offsets = np.array([0, 3, 3, 7, 12])
    seg_adapter = np.array([2, 0, 2, 1])
    ids = oracle.segments_to_ids(seg_offsets, seg_adapter, 14)
    assert ids.tolist() == [2, 2, 2, 2, 2, 2, 2, 1, 1, 1, 1, 1, -1, -1]
    p = oracle.canonical_plan(ids, 3)
    assert p["n_runs"] == 2                       # adjacent same-adapter segments merge


def test_h_saved_equals_recompute():
    c, eff, X, A, B, Y, dY = _tiny_case(11, mask_p=0.7)
    H = oracle.shrink(eff, X, A)
    dA0, dB0 = oracle.grad(eff, c.mask, X, dY, A, B, c.scales)
    dA1, dB1 = oracle.grad(eff, c.mask, X, dY, A, B, c.scales, H_saved=H)
    for a in range(c.num_slots):
        if A[a] is not None:
            assert np.allclose(dA0[a], dA1[a], rtol=1e-13, atol=1e-13)
            assert np.allclose(dB0[a], dB1[a], rtol=1e-13, atol=1e-13)


def test_explicit_mask_not_inferred_from_zero_dy():
    """A trainable row whose dY is zero is still counted as trainable (Section 3.3:
    the span comes from the mask, not from a nonzero learning signal)."""
    idx = np.array([0, 0, 1])
    mask = np.array([1, 0, 1])
    p = oracle.canonical_plan(idx, 2, mask=mask)
    assert p["m_counts"].tolist() == [1, 1]


# ----------------------------------------------------------------------------
# planted mistakes: each must be rejected by at least one pin
# ----------------------------------------------------------------------------

def _mutant(**overrides):
    ns = types.SimpleNamespace(canonical_plan=oracle.canonical_plan, apply=oracle.apply,
                               linear=oracle.linear,
                               grad=oracle.grad, grad_x=oracle.grad_x,
                               masked_loss=oracle.masked_loss, adamw=oracle.adamw,
                               token_loss=oracle.token_loss, rel_fro=oracle.rel_fro,
                               max_abs=oracle.max_abs)
    for k, v in overrides.items():
        setattr(ns, k, v)
    return ns


def _apply_transposed_B(eff, X, Y, A, B, scale):
    out = np.array(Y, dtype=np.float64, copy=True)
    for a in range(len(A)):
        rows = np.nonzero(eff == a)[0]
        if rows.size == 0 or A[a] is None:
            continue
        Bt = B[a].T if B[a].shape[0] == B[a].shape[1] else B[a][::-1]
        out[rows] += float(scale[a]) * ((X[rows] @ A[a].T) @ Bt.T)
    return out


def _apply_no_scale(eff, X, Y, A, B, scale):
    return oracle.apply(eff, X, Y, A, B, np.ones_like(scale))


def _apply_wrong_rows(eff, X, Y, A, B, scale):
    return oracle.apply(np.roll(eff, 1), X, Y, A, B, scale)


def _apply_touches_none_rows(eff, X, Y, A, B, scale):
    return oracle.apply(np.where(eff < 0, 0, eff), X, Y, A, B, scale)


def _grad_mask_ignored(eff, mask, X, dY, A, B, scale, H_saved=None):
    return oracle.grad(eff, None, X, dY, A, B, scale)


def _grad_swapped(eff, mask, X, dY, A, B, scale, H_saved=None):
    dA, dB = oracle.grad(eff, mask, X, dY, A, B, scale)
    # dA computed from H instead of G (a wrong chain-rule term)
    out = []
    for a in range(len(A)):
        if A[a] is None:
            out.append(None)
            continue
        sel = (eff == a) & (np.asarray(mask) != 0)
        rows = np.nonzero(sel)[0]
        H = X[rows] @ A[a].T
        out.append(float(scale[a]) * (H.T @ X[rows]))
    return out, dB


def _grad_sign(eff, mask, X, dY, A, B, scale, H_saved=None):
    dA, dB = oracle.grad(eff, mask, X, dY, A, B, scale)
    return dA, [(-b if b is not None else None) for b in dB]


def _grad_no_scale(eff, mask, X, dY, A, B, scale, H_saved=None):
    return oracle.grad(eff, mask, X, dY, A, B, np.ones_like(scale))


def _grad_mask_multiplied(eff, mask, X, dY, A, B, scale, H_saved=None):
    m = np.asarray(mask, np.float64)[:, None]
    return oracle.grad(eff, None, X * m, dY * m, A, B, scale)


def _grad_x_mask_ignored(eff, mask, dY, A, B, scale, dX):
    return oracle.grad_x(eff, None, dY, A, B, scale, dX)


def _grad_x_no_scale(eff, mask, dY, A, B, scale, dX):
    return oracle.grad_x(eff, mask, dY, A, B, np.ones_like(scale), dX)


def _grad_x_sign(eff, mask, dY, A, B, scale, dX):
    return 2 * np.asarray(dX, np.float64) - oracle.grad_x(eff, mask, dY, A, B, scale, dX)


def _grad_x_overwrites(eff, mask, dY, A, B, scale, dX):
    # the delta stored instead of added
    d = oracle.grad_x(eff, mask, dY, A, B, scale, np.zeros_like(dX))
    sel = np.any(d != 0, axis=1)
    out = np.array(dX, dtype=np.float64, copy=True)
    out[sel] = d[sel]
    return out


def _grad_x_wrong_weight(eff, mask, dY, A, B, scale, dX):
    # A reversed along d_in (a transposed or mis-indexed operand)
    return oracle.grad_x(eff, mask, dY, [a[:, ::-1] if a is not None else None for a in A], B,
                         scale, dX)


def _adamw_coupled_decay(p, m, v, g, step, lr, b1, b2, eps, wd):
    # L2 added to the gradient (Adam with L2), not decoupled
    return oracle.adamw(p, m, v, np.asarray(g) + wd * np.asarray(p), step, lr, b1, b2, eps, 0.0)


def _adamw_no_bias_correction(p, m, v, g, step, lr, b1, b2, eps, wd):
    p = np.asarray(p, np.float64)
    m_t = b1 * np.asarray(m) + (1 - b1) * np.asarray(g)
    v_t = b2 * np.asarray(v) + (1 - b2) * np.asarray(g) ** 2
    return p - lr * (m_t / (np.sqrt(v_t) + eps) + wd * p), m_t, v_t


def _adamw_eps_inside_sqrt(p, m, v, g, step, lr, b1, b2, eps, wd):
    p = np.asarray(p, np.float64)
    m_t = b1 * np.asarray(m) + (1 - b1) * np.asarray(g)
    v_t = b2 * np.asarray(v) + (1 - b2) * np.asarray(g) ** 2
    mh, vh = m_t / (1 - b1 ** step), v_t / (1 - b2 ** step)
    return p - lr * (mh / np.sqrt(vh + eps) + wd * p), m_t, v_t


def _adamw_beta1_in_v(p, m, v, g, step, lr, b1, b2, eps, wd):
    return oracle.adamw(p, m, v, g, step, lr, b1, b1, eps, wd)


def _adamw_step_off_by_one(p, m, v, g, step, lr, b1, b2, eps, wd):
    return oracle.adamw(p, m, v, g, step + 1, lr, b1, b2, eps, wd)


def _adamw_decay_after_step(p, m, v, g, step, lr, b1, b2, eps, wd):
    p_t, m_t, v_t = oracle.adamw(p, m, v, g, step, lr, b1, b2, eps, 0.0)
    return p_t * (1 - lr * wd), m_t, v_t


def _loss_variant(change):
    """The token loss with one planted mistake (the definition retyped with a switch)."""
    def f(kind, logits, target, weight=None, mask=None, old_logp=None, adv=None, corr=None,
          clip_lo=0.2, clip_hi=0.2):
        z = np.asarray(logits, np.float64)
        n, V = z.shape
        if kind == oracle.LOSS_CE:
            act = np.asarray(weight) != 0
        else:
            act = np.ones(n, bool) if (mask is None or change == "mask_ignored") else np.asarray(mask) != 0
        L, lp, dz = np.zeros(n), np.zeros(n), np.zeros((n, V))
        for t in np.nonzero(act)[0]:
            mx = 0.0 if change == "no_shift" else np.max(z[t])
            e = np.exp(z[t] - mx)
            logp = z[t, target[t]] - (mx + np.log(e.sum()))
            soft = e / e.sum()
            if kind == oracle.LOSS_CE:
                L[t], g = -weight[t] * logp, weight[t]
            else:
                c = 1.0 if (corr is None or change == "corr_ignored") else corr[t]
                rho = np.exp((old_logp[t] - logp) if change == "ratio_inverted" else (logp - old_logp[t]))
                A = adv[t]
                un, cl = rho * A, min(max(rho, 1 - clip_lo), 1 + clip_hi) * A
                pick = max if change == "ppo_max" else min
                if kind == oracle.LOSS_IS or pick(un, cl) == un:
                    L[t], g = -c * un, c * A * rho
                else:
                    L[t], g = -c * cl, 0.0
            lp[t] = logp
            dz[t] = (-g if change == "grad_sign" else g) * soft
            if change != "no_onehot":
                dz[t, target[t]] -= (-g if change == "grad_sign" else g)
        return L, lp, dz
    return f


def _plan_unstable(idx, num_slots, mask=None, ranks=None):
    p = oracle.canonical_plan(idx, num_slots, mask=mask, ranks=ranks)
    p = dict(p)
    perm = np.array(p["perm"])
    off = p["offsets"]
    for a in range(num_slots):
        perm[off[a]:off[a + 1]] = perm[off[a]:off[a + 1]][::-1]
    p["perm"] = perm
    return p


def _plan_inclusive_offsets(idx, num_slots, mask=None, ranks=None):
    p = dict(oracle.canonical_plan(idx, num_slots, mask=mask, ranks=ranks))
    p["offsets"] = np.concatenate([p["offsets"][1:], p["offsets"][-1:]])
    return p


def _plan_mask_ignored(idx, num_slots, mask=None, ranks=None):
    return oracle.canonical_plan(idx, num_slots, mask=None, ranks=ranks)


def _plan_no_validation(idx, num_slots, mask=None, ranks=None):
    p = dict(oracle.canonical_plan(np.clip(idx, -1, num_slots - 1), num_slots, mask=mask,
                                   ranks=ranks))
    return p


def _plan_ranks_ignored(idx, num_slots, mask=None, ranks=None):
    # empty slots treated as live (no flag, their rows grouped)
    return oracle.canonical_plan(idx, num_slots, mask=mask, ranks=None)


def _rel_fro_zero(out, ref):
    return 0.0


def _rel_fro_by_out(out, ref):
    d = np.linalg.norm(np.asarray(out, np.float64))
    return float(np.linalg.norm(np.asarray(out, np.float64) - np.asarray(ref, np.float64)) / d) if d else 0.0


def _rel_fro_squared(out, ref):
    r = oracle.rel_fro(out, ref)
    return r * r


def _max_abs_signed(out, ref):
    d = np.asarray(out, np.float64) - np.asarray(ref, np.float64)
    return float(np.max(d)) if d.size else 0.0


def _max_abs_nan_blind(out, ref):
    d = np.abs(np.asarray(out, np.float64) - np.asarray(ref, np.float64))
    return float(np.nanmax(d)) if d.size else 0.0


def _linear_no_base_on_none(eff, X, W, A, B, scale):
    out = oracle.linear(eff, X, W, A, B, scale)
    out[np.asarray(eff) < 0] = 0.0
    return out


def _linear_lora_on_none(eff, X, W, A, B, scale):
    return oracle.linear(np.where(np.asarray(eff) < 0, 0, eff), X, W, A, B, scale)


def _linear_base_reversed(eff, X, W, A, B, scale):
    # the base weight read with a reversed d_in axis (a mis-indexed operand)
    return oracle.linear(eff, X, W[:, ::-1], A, B, scale)


def _linear_no_scale(eff, X, W, A, B, scale):
    return oracle.linear(eff, X, W, A, B, np.ones_like(scale))


def _linear_base_twice(eff, X, W, A, B, scale):
    return oracle.linear(eff, X, W, A, B, scale) + X @ W.T


def _linear_scale_on_base(eff, X, W, A, B, scale):
    out = oracle.linear(eff, X, W, A, B, scale)
    for t in range(X.shape[0]):
        if eff[t] >= 0:
            out[t] += (float(scale[eff[t]]) - 1.0) * (W @ X[t])
    return out


MUTANTS = {
    "linear_no_base_on_none": _mutant(linear=_linear_no_base_on_none),
    "linear_lora_on_none": _mutant(linear=_linear_lora_on_none),
    "linear_base_reversed": _mutant(linear=_linear_base_reversed),
    "linear_no_scale": _mutant(linear=_linear_no_scale),
    "linear_base_twice": _mutant(linear=_linear_base_twice),
    "linear_scale_on_base": _mutant(linear=_linear_scale_on_base),
    "plan_ranks_ignored": _mutant(canonical_plan=_plan_ranks_ignored),
    "rel_fro_zero": _mutant(rel_fro=_rel_fro_zero),
    "rel_fro_by_out": _mutant(rel_fro=_rel_fro_by_out),
    "rel_fro_squared": _mutant(rel_fro=_rel_fro_squared),
    "max_abs_signed": _mutant(max_abs=_max_abs_signed),
    "max_abs_nan_blind": _mutant(max_abs=_max_abs_nan_blind),
    "apply_transposed_B": _mutant(apply=_apply_transposed_B),
    "apply_no_scale": _mutant(apply=_apply_no_scale),
    "apply_wrong_rows": _mutant(apply=_apply_wrong_rows),
    "apply_touches_none_rows": _mutant(apply=_apply_touches_none_rows),
    "grad_mask_ignored": _mutant(grad=_grad_mask_ignored),
    "grad_wrong_chain_term": _mutant(grad=_grad_swapped),
    "grad_sign": _mutant(grad=_grad_sign),
    "grad_no_scale": _mutant(grad=_grad_no_scale),
    "grad_mask_multiplied": _mutant(grad=_grad_mask_multiplied),
    "grad_x_mask_ignored": _mutant(grad_x=_grad_x_mask_ignored),
    "grad_x_no_scale": _mutant(grad_x=_grad_x_no_scale),
    "grad_x_sign": _mutant(grad_x=_grad_x_sign),
    "grad_x_overwrites": _mutant(grad_x=_grad_x_overwrites),
    "grad_x_wrong_weight": _mutant(grad_x=_grad_x_wrong_weight),
    "adamw_coupled_decay": _mutant(adamw=_adamw_coupled_decay),
    "adamw_no_bias_correction": _mutant(adamw=_adamw_no_bias_correction),
    "adamw_eps_inside_sqrt": _mutant(adamw=_adamw_eps_inside_sqrt),
    "adamw_beta1_in_v": _mutant(adamw=_adamw_beta1_in_v),
    "adamw_step_off_by_one": _mutant(adamw=_adamw_step_off_by_one),
    "adamw_decay_after_step": _mutant(adamw=_adamw_decay_after_step),
    "loss_no_shift": _mutant(token_loss=_loss_variant("no_shift")),
    "loss_grad_sign": _mutant(token_loss=_loss_variant("grad_sign")),
    "loss_no_onehot": _mutant(token_loss=_loss_variant("no_onehot")),
    "loss_ppo_max": _mutant(token_loss=_loss_variant("ppo_max")),
    "loss_ratio_inverted": _mutant(token_loss=_loss_variant("ratio_inverted")),
    "loss_mask_ignored": _mutant(token_loss=_loss_variant("mask_ignored")),
    "loss_corr_ignored": _mutant(token_loss=_loss_variant("corr_ignored")),
    "plan_unstable": _mutant(canonical_plan=_plan_unstable),
    "plan_inclusive_offsets": _mutant(canonical_plan=_plan_inclusive_offsets),
    "plan_mask_ignored": _mutant(canonical_plan=_plan_mask_ignored),
    "plan_no_validation": _mutant(canonical_plan=_plan_no_validation),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    impl = MUTANTS[name]
    failed = []
    for check in ALL_CHECKS:
        try:
            ok = check(impl)
        except Exception:
            ok = False
        if not ok:
            failed.append(check.__name__)
    assert failed, f"planted mistake {name} passed every pin"

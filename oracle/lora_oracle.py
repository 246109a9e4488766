"""Float64 CPU oracle for the mixed-adapter LoRA layer.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, links or runs
this module; only the tests, the smoke check and the benchmark's CPU-baseline
leg do.  It shares no code with the HIP library.

What it computes (all arithmetic in float64 on the exact stored input values;
widening bfloat16 or binary32 to float64 is exact):

* ``canonical_plan``  -- grouping of token rows by adapter identity, the
  gather step of the paper's gather-group-compute-scatter structure
  (Section 3.4, the rollout kernel paragraph and Figure 2) and the routing of
  trainable rows by adapter identity (Section 3.5, "Batch routing").
* ``apply`` / ``shrink`` / ``expand`` -- the adapter residual of the LoRA layer
  equation in Section 3.4, y = x W^T + s_a (x A_a^T) B_a^T, evaluated per adapter
  group as Delta_a = s_a (X_a A_a^T) B_a^T and added back to the original rows.
* ``linear`` -- the whole adapted layer of Section 3.4, the shared base
  projection x W^T of every row plus the adapter residual of its group (rows
  with no adapter get the base projection alone).
* ``grad`` -- the adapter-local gradients dA_a, dB_a of the loss through that
  residual, restricted to rows whose explicit loss mask is nonzero (Section 3.3
  for the mask, Section 3.5 for adapter-local gradients).  The paper does not
  write the backward; it is the chain rule on the LoRA equation:
  with H = X_m A_a^T and G = dY_m B_a,  dB_a = s_a dY_m^T H  and
  dA_a = s_a G^T X_m.
* ``grad_x`` -- the input gradient through the same residual over the same
  masked rows, dX_t += s_a (dY_t B_a) A_a (the chain rule on the LoRA equation
  with respect to x; rows outside T_a^m are left as they are).
* ``adamw`` -- one optimizer step of one adapter tensor's own state (the
  paper keeps gradients, optimizer moments and step counters local to the
  owning policy and issues the optimizer step per policy, Section 3.5; it
  names no optimizer, and the update is the published AdamW: Adam's moment
  estimates with bias correction (Kingma and Ba) and weight decay decoupled
  from the gradient (Loshchilov and Hutter), with the learning rate scaling
  both the Adam step and the decay).
* ``token_loss`` -- the masked token-level objectives that produce the
  gradient at the logits, summed over target positions: cross-entropy with
  SFT weights w_t, and the importance-sampling and PPO-style policy-gradient
  losses with the action mask m_t, rollout log-probabilities, advantages and
  optional correction weights on the same target axis (Section 3.3, the SFT
  and RL data path; Section 3.5, "Forward/backward path", for the objectives).
  The paper names the objectives without writing them; the forms are the
  standard ones (see the function).
* ``*_bruteforce`` -- scalar Python loops over the same definitions, used only
  as an independent pin on tiny inputs.

Conventions: ``A[a]`` is ``[r_a, d_in]``, ``B[a]`` is ``[d_out, r_a]`` (the paper's
shapes), ``None`` for an empty slot.  Ids are in ``[-1, S)``; -1 means no
adapter.  An id outside that range, or naming an empty slot, is a data error:
the row is treated as -1 and the plan's error flag is set.
"""
import numpy as np


# ----------------------------------------------------------------------------
# grouping (the gather / routing step)
# ----------------------------------------------------------------------------

def effective_ids(idx, num_slots, ranks=None):
    """Ids after validation: invalid ids and ids naming an empty slot become -1.

    Returns ``(eff_ids int64[n], error bool)``.
    """
    idx = np.asarray(idx, dtype=np.int64)
    bad = (idx < -1) | (idx >= num_slots)
    eff = np.where(bad, -1, idx)
    if ranks is not None:
        ranks = np.asarray(ranks)
        live = eff >= 0
        empty = np.zeros_like(live)
        empty[live] = ranks[eff[live]] <= 0
        bad = bad | empty
        eff = np.where(empty, -1, eff)
    return eff, bool(bad.any())


def _group(eff, num_slots):
    """counts, exclusive offsets and the stable per-adapter row order."""
    live = eff >= 0
    counts = np.bincount(eff[live], minlength=num_slots).astype(np.int64)
    offsets = np.zeros(num_slots + 1, dtype=np.int64)
    np.cumsum(counts, out=offsets[1:])
    key = np.where(live, eff, num_slots)          # rows with no adapter sort last
    order = np.argsort(key, kind="stable")
    perm = order[: offsets[-1]]
    return counts, offsets, perm


def _runs(eff):
    """Maximal runs [start, start+len) of one adapter id >= 0, ascending start."""
    n = eff.size
    if n == 0:
        z = np.zeros(0, np.int64)
        return z, z, z
    live = eff >= 0
    prev = np.concatenate([[-2], eff[:-1]])
    starts = np.nonzero(live & (eff != prev))[0]
    nxt = np.concatenate([eff[1:], [-2]])
    ends = np.nonzero(live & (eff != nxt))[0]
    return starts, ends - starts + 1, eff[starts]


def canonical_plan(idx, num_slots, mask=None, ranks=None):
    """The canonical grouping arrays (all int64 numpy arrays).

    counts[a]   number of rows with id a
    offsets     exclusive prefix sum of counts, length S+1
    perm        row indices grouped by adapter, ascending row order inside a group
    run_start, run_len, run_adapter   maximal runs of one adapter id
    m_counts, m_offsets, m_perm       the same grouping over rows with mask != 0
    error       True if any id was invalid or named an empty slot
    """
    eff, error = effective_ids(idx, num_slots, ranks)
    counts, offsets, perm = _group(eff, num_slots)
    rs, rl, ra = _runs(eff)
    if mask is None:
        eff_m = eff
    else:
        eff_m = np.where(np.asarray(mask) != 0, eff, -1)
    m_counts, m_offsets, m_perm = _group(eff_m, num_slots)
    return dict(counts=counts, offsets=offsets, perm=perm, n_runs=rs.size,
                run_start=rs, run_len=rl, run_adapter=ra, m_counts=m_counts,
                m_offsets=m_offsets, m_perm=m_perm, error=error, eff=eff)


def plan_bruteforce(idx, num_slots, mask=None, ranks=None):
    """Scalar enumeration of the same arrays (independent pin for the plan)."""
    n = len(idx)
    eff, error = [], False
    for t in range(n):
        a = int(idx[t])
        ok = -1 <= a < num_slots and (a < 0 or ranks is None or ranks[a] > 0)
        if not ok:
            error = True
            a = -1
        eff.append(a)
    counts = [0] * num_slots
    perm_lists = [[] for _ in range(num_slots)]
    m_lists = [[] for _ in range(num_slots)]
    for t in range(n):
        if eff[t] >= 0:
            counts[eff[t]] += 1
            perm_lists[eff[t]].append(t)
            if mask is None or mask[t] != 0:
                m_lists[eff[t]].append(t)
    offsets = [0]
    for a in range(num_slots):
        offsets.append(offsets[-1] + counts[a])
    m_offsets = [0]
    for a in range(num_slots):
        m_offsets.append(m_offsets[-1] + len(m_lists[a]))
    rs, rl, ra = [], [], []
    t = 0
    while t < n:
        if eff[t] < 0:
            t += 1
            continue
        u = t
        while u + 1 < n and eff[u + 1] == eff[t]:
            u += 1
        rs.append(t)
        rl.append(u - t + 1)
        ra.append(eff[t])
        t = u + 1
    return dict(counts=counts, offsets=offsets,
                perm=[t for a in range(num_slots) for t in perm_lists[a]],
                n_runs=len(rs), run_start=rs, run_len=rl, run_adapter=ra,
                m_counts=[len(m) for m in m_lists], m_offsets=m_offsets,
                m_perm=[t for a in range(num_slots) for t in m_lists[a]], error=error)


def segments_to_ids(seg_offsets, seg_adapter, n):
    """Per-row ids from contiguous segments [seg_offsets[s], seg_offsets[s+1]).
    Rows outside every segment get -1."""
    idx = np.full(n, -1, dtype=np.int64)
    for s in range(len(seg_adapter)):
        idx[int(seg_offsets[s]):int(seg_offsets[s + 1])] = int(seg_adapter[s])
    return idx


# ----------------------------------------------------------------------------
# forward: shrink, expand, apply (Section 3.4, LoRA equation and Delta_a)
# ----------------------------------------------------------------------------

def shrink(eff, X, A, H=None):
    """H[t, :r_a] = X[t] A_a^T for every row t with adapter a (unscaled).

    ``H`` (float64 [n, >= r_max]) is updated in place if given; rows with no
    adapter and columns >= r_a are left as they were.
    """
    n = X.shape[0]
    r_max = max([a.shape[0] for a in A if a is not None] + [0])
    if H is None:
        H = np.zeros((n, r_max))
    for a, Aa in enumerate(A):
        rows = np.nonzero(eff == a)[0]
        if rows.size == 0 or Aa is None:
            continue
        H[rows, : Aa.shape[0]] = X[rows] @ Aa.T
    return H


def expand(eff, H, Y, B, scale):
    """Y[t] += s_a H[t, :r_a] B_a^T for every row t with adapter a; returns a new
    float64 array, rows with no adapter copied unchanged."""
    out = np.array(Y, dtype=np.float64, copy=True)
    for a, Ba in enumerate(B):
        rows = np.nonzero(eff == a)[0]
        if rows.size == 0 or Ba is None:
            continue
        r = Ba.shape[1]
        out[rows] += float(scale[a]) * (H[rows, :r] @ Ba.T)
    return out


def apply(eff, X, Y, A, B, scale):
    """Y_out = Y + Delta with Delta_a = s_a (X_a A_a^T) B_a^T scattered back to
    the rows of group a.  Rows with no adapter are copied bit for bit."""
    out = np.array(Y, dtype=np.float64, copy=True)
    for a in range(len(A)):
        if A[a] is None:
            continue
        rows = np.nonzero(eff == a)[0]
        if rows.size == 0:
            continue
        Ha = X[rows] @ A[a].T
        out[rows] += float(scale[a]) * (Ha @ B[a].T)
    return out


def delta_rows(eff, X, A, B, scale, rows):
    """The residual Delta[t] for the listed rows only (zero for rows with no
    adapter); used to check large cases on sampled rows."""
    rows = np.asarray(rows, dtype=np.int64)
    d_out = next(b.shape[0] for b in B if b is not None)
    out = np.zeros((rows.size, d_out))
    for i, t in enumerate(rows):
        a = int(eff[t])
        if a < 0:
            continue
        h = A[a] @ X[t]
        out[i] = float(scale[a]) * (B[a] @ h)
    return out


def apply_bruteforce(eff, X, Y, A, B, scale):
    """Scalar loops over the LoRA equation, row by row (tiny inputs only)."""
    n, d_in = X.shape
    d_out = Y.shape[1]
    out = [[float(Y[t][o]) for o in range(d_out)] for t in range(n)]
    for t in range(n):
        a = int(eff[t])
        if a < 0:
            continue
        r = A[a].shape[0]
        h = []
        for j in range(r):
            acc = 0.0
            for k in range(d_in):
                acc += float(X[t][k]) * float(A[a][j][k])
            h.append(acc)
        for o in range(d_out):
            acc = 0.0
            for j in range(r):
                acc += h[j] * float(B[a][o][j])
            out[t][o] += float(scale[a]) * acc
    return np.array(out)


# ----------------------------------------------------------------------------
# the whole adapted layer: shared base projection plus the adapter residual
# (Section 3.4, LoRA layer equation)
# ----------------------------------------------------------------------------

def linear(eff, X, W, A, B, scale):
    """Y = X W^T + Delta: the base projection of every row (W is [d_out, d_in],
    the same for all rows), plus s_a (X_a A_a^T) B_a^T on the rows of each
    adapter group a.  Rows with no adapter get the base projection alone.

    Section 3.4 writes the adapted layer as y = x W^T + s_a (x A_a^T) B_a^T and
    computes the base term once over all active rows, the residual per group.
    """
    out = X @ W.T
    for a in range(len(A)):
        if A[a] is None:
            continue
        rows = np.nonzero(eff == a)[0]
        if rows.size == 0:
            continue
        out[rows] += float(scale[a]) * ((X[rows] @ A[a].T) @ B[a].T)
    return out


def linear_rows(eff, X, W, A, B, scale, rows):
    """linear() for the listed rows only (large cases checked on samples)."""
    rows = np.asarray(rows, dtype=np.int64)
    out = X[rows] @ W.T
    for i, t in enumerate(rows):
        a = int(eff[t])
        if a >= 0:
            out[i] += float(scale[a]) * (B[a] @ (A[a] @ X[t]))
    return out


def linear_bruteforce(eff, X, W, A, B, scale):
    """Scalar loops over the layer equation, row by row (tiny inputs only)."""
    n, d_in = X.shape
    d_out = W.shape[0]
    out = []
    for t in range(n):
        row = []
        a = int(eff[t])
        h = []
        if a >= 0:
            for j in range(A[a].shape[0]):
                h.append(sum(float(X[t][k]) * float(A[a][j][k]) for k in range(d_in)))
        for o in range(d_out):
            y = sum(float(X[t][k]) * float(W[o][k]) for k in range(d_in))
            if a >= 0:
                y += float(scale[a]) * sum(h[j] * float(B[a][o][j]) for j in range(len(h)))
            row.append(y)
        out.append(row)
    return np.array(out).reshape(n, d_out)


# ----------------------------------------------------------------------------
# backward: masked, adapter-local gradients (Sections 3.3 and 3.5)
# ----------------------------------------------------------------------------

def grad(eff, mask, X, dY, A, B, scale, H_saved=None):
    """dA_a, dB_a over rows T_a^m = {t : eff[t] = a and mask[t] != 0}.

    dB_a = s_a dY_m^T (X_m A_a^T)     [d_out, r_a]
    dA_a = s_a (dY_m B_a)^T X_m       [r_a, d_in]

    Rows outside T_a^m are never read.  A slot with no such row gets exact
    zeros.  ``H_saved`` (float64 [n, >= r_a]) replaces X_m A_a^T when given.
    Returns two lists indexed by slot (None for empty slots).
    """
    dA, dB = [], []
    for a in range(len(A)):
        if A[a] is None:
            dA.append(None)
            dB.append(None)
            continue
        r = A[a].shape[0]
        sel = eff == a
        if mask is not None:
            sel = sel & (np.asarray(mask) != 0)
        rows = np.nonzero(sel)[0]
        if rows.size == 0:
            dA.append(np.zeros_like(A[a], dtype=np.float64))
            dB.append(np.zeros_like(B[a], dtype=np.float64))
            continue
        Xm = X[rows]
        dYm = dY[rows]
        Ha = H_saved[rows, :r] if H_saved is not None else Xm @ A[a].T
        Ga = dYm @ B[a]
        s = float(scale[a])
        dB.append(s * (dYm.T @ Ha))
        dA.append(s * (Ga.T @ Xm))
    return dA, dB


def grad_bruteforce(eff, mask, X, dY, A, B, scale):
    """Scalar loops for dA, dB (tiny inputs only)."""
    n, d_in = X.shape
    d_out = dY.shape[1]
    dA, dB = [], []
    for a in range(len(A)):
        if A[a] is None:
            dA.append(None)
            dB.append(None)
            continue
        r = A[a].shape[0]
        s = float(scale[a])
        gA = [[0.0] * d_in for _ in range(r)]
        gB = [[0.0] * r for _ in range(d_out)]
        for t in range(n):
            if int(eff[t]) != a or (mask is not None and mask[t] == 0):
                continue
            h = [sum(float(X[t][k]) * float(A[a][j][k]) for k in range(d_in)) for j in range(r)]
            g = [sum(float(dY[t][o]) * float(B[a][o][j]) for o in range(d_out)) for j in range(r)]
            for o in range(d_out):
                for j in range(r):
                    gB[o][j] += s * float(dY[t][o]) * h[j]
            for j in range(r):
                for k in range(d_in):
                    gA[j][k] += s * g[j] * float(X[t][k])
        dA.append(np.array(gA))
        dB.append(np.array(gB))
    return dA, dB


def grad_x(eff, mask, dY, A, B, scale, dX):
    """dX_out = dX + s_a (dY_t B_a) A_a for every row t in T_a^m = {t : eff[t] = a
    and mask[t] != 0}; every other row of dX is returned unchanged (bit-identical).
    dY is [n, d_out], dX [n, d_in]; returns a new float64 array.
    """
    out = np.array(dX, dtype=np.float64, copy=True)
    for a in range(len(A)):
        if A[a] is None:
            continue
        sel = eff == a
        if mask is not None:
            sel = sel & (np.asarray(mask) != 0)
        rows = np.nonzero(sel)[0]
        if rows.size == 0:
            continue
        out[rows] = out[rows] + float(scale[a]) * ((dY[rows] @ B[a]) @ A[a])
    return out


def grad_x_bruteforce(eff, mask, dY, A, B, scale, dX):
    """Scalar loops for the input gradient (tiny inputs only)."""
    n, d_out = dY.shape
    out = [[float(v) for v in row] for row in np.asarray(dX, np.float64)]
    for t in range(n):
        a = int(eff[t])
        if a < 0 or A[a] is None or (mask is not None and mask[t] == 0):
            continue
        r, d_in = A[a].shape
        s = float(scale[a])
        g = [sum(float(dY[t][o]) * float(B[a][o][j]) for o in range(d_out)) for j in range(r)]
        for k in range(d_in):
            out[t][k] = out[t][k] + s * sum(g[j] * float(A[a][j][k]) for j in range(r))
    return np.array(out)


def masked_loss(eff, mask, X, dY, A, B, scale):
    """L = sum over masked rows t with an adapter of <dY_t, Delta_t>.

    L is linear in each A_a (B fixed), in each B_a (A fixed) and in X, and its
    partial derivatives are exactly dA_a, dB_a and dX; the tests use this to pin
    ``grad`` and ``grad_x``.
    """
    total = 0.0
    for a in range(len(A)):
        if A[a] is None:
            continue
        sel = eff == a
        if mask is not None:
            sel = sel & (np.asarray(mask) != 0)
        rows = np.nonzero(sel)[0]
        if rows.size == 0:
            continue
        D = float(scale[a]) * ((X[rows] @ A[a].T) @ B[a].T)
        total += float(np.sum(dY[rows] * D))
    return total


# ----------------------------------------------------------------------------
# comparison metrics
# ----------------------------------------------------------------------------

# ----------------------------------------------------------------------------
# adapter-local optimizer step
# ----------------------------------------------------------------------------

def adamw(p, m, v, g, step, lr, beta1, beta2, eps, weight_decay):
    """AdamW step number ``step`` (t >= 1) of one tensor, elementwise in float64.

    With the tensor's own moments m, v and step count t:
        m_t = beta1 m + (1 - beta1) g
        v_t = beta2 v + (1 - beta2) g^2
        mhat = m_t / (1 - beta1^t),   vhat = v_t / (1 - beta2^t)
        p_t = p - lr (mhat / (sqrt(vhat) + eps) + weight_decay p)
    The decay term uses the value before the step (decoupled weight decay: it
    never enters the moments).  Returns (p_t, m_t, v_t); the inputs are not
    modified."""
    if step < 1:
        raise ValueError("AdamW step numbers start at 1")
    p = np.asarray(p, np.float64)
    m = np.asarray(m, np.float64)
    v = np.asarray(v, np.float64)
    g = np.asarray(g, np.float64)
    m_t = beta1 * m + (1.0 - beta1) * g
    v_t = beta2 * v + (1.0 - beta2) * g * g
    mhat = m_t / (1.0 - beta1 ** step)
    vhat = v_t / (1.0 - beta2 ** step)
    p_t = p - lr * (mhat / (np.sqrt(vhat) + eps) + weight_decay * p)
    return p_t, m_t, v_t


# ----------------------------------------------------------------------------
# masked token-level losses -> gradient at the logits
# ----------------------------------------------------------------------------

LOSS_CE, LOSS_IS, LOSS_PPO = 0, 1, 2


def token_loss(kind, logits, target, weight=None, mask=None, old_logp=None, adv=None,
               corr=None, clip_lo=0.2, clip_hi=0.2):
    """Per-token loss L_t, log-probability logp_t and dL_t/dz_t for logits z [n, V].

    logp_t = z_t[y_t] - log sum_v exp(z_t[v])
    CE  (kind 0): L_t = -w_t logp_t                                  (row active when w_t != 0)
    IS  (kind 1): L_t = -m_t c_t A_t rho_t,  rho_t = exp(logp_t - l_old_t)
    PPO (kind 2): L_t = -m_t c_t min(rho_t A_t, clip(rho_t, 1 - clip_lo, 1 + clip_hi) A_t)
    (for IS / PPO a row is active when m_t != 0; mask None = every row; c_t = 1
    when corr is None.)  With g_t = -dL_t/dlogp_t the gradient is
    dL_t/dz_t = g_t (softmax(z_t) - onehot(y_t)); for PPO, g_t = m_t c_t A_t rho_t
    where the unclipped term is the minimum (ties included), else 0.
    Inactive rows: L_t = 0, logp_t = 0, a zero gradient row; their logits are
    never read.  Returns (L [n], logp [n], dz [n, V]) in float64."""
    z = np.asarray(logits, np.float64)
    n, V = z.shape
    y = np.asarray(target, np.int64)
    if kind == LOSS_CE:
        act = np.asarray(weight, np.float64) != 0
    else:
        act = np.ones(n, bool) if mask is None else (np.asarray(mask) != 0)
    L = np.zeros(n)
    lp = np.zeros(n)
    dz = np.zeros((n, V))
    for t in np.nonzero(act)[0]:
        zt = z[t]
        mx = np.max(zt)
        e = np.exp(zt - mx)
        s = np.sum(e)
        logp = zt[y[t]] - (mx + np.log(s))
        soft = e / s
        if kind == LOSS_CE:
            w = float(weight[t])
            L[t] = -w * logp
            g = w
        else:
            c = 1.0 if corr is None else float(corr[t])
            A = float(adv[t])
            rho = np.exp(logp - float(old_logp[t]))
            if kind == LOSS_IS:
                L[t] = -c * A * rho
                g = c * A * rho
            else:
                unclipped = rho * A
                clipped = min(max(rho, 1.0 - clip_lo), 1.0 + clip_hi) * A
                if unclipped <= clipped:
                    L[t] = -c * unclipped
                    g = c * A * rho
                else:
                    L[t] = -c * clipped
                    g = 0.0
        lp[t] = logp
        dz[t] = g * soft
        dz[t, y[t]] -= g
    return L, lp, dz


def rel_fro(out, ref):
    """||out - ref||_F / ||ref||_F (0 when both are zero)."""
    out = np.asarray(out, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(out - ref)
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return float(num / den)


def max_abs(out, ref):
    out = np.asarray(out, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.max(np.abs(out - ref))) if out.size else 0.0

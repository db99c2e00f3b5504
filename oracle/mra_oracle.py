"""Plain float64 CPU oracle of MRA-2 approximate self-attention.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call or
execute this module; only the tests, the smoke check and the benchmark's
CPU-baseline leg use it. It shares no code with the HIP kernels.

It computes, slowly and literally, what the paper defines for the
two-resolution scheme R = {b, 1} ("MRA-2", Sec. 5, b = 32):

* block means of Q, K, V (Sec. 4.1, eq. recursive_pooling; Sec. 4.3,
  eq. recursive_pooling_V), taken here as the direct mean of each b-row block,
  which is what b/2-fold pairwise averaging gives in exact arithmetic;
* coarse logits mu_{b,x,y} = exp(<B^b_{x,y}, P>/b^2) = exp(Q~_x . K~_y)
  (Sec. 4.1, eq. exp_of_average), with P = Q K^T / sqrt(d);
* per block-row selection of the `m` coarse blocks with the largest score
  (Sec. 4.2, Alg. 1, applied row by row; ties go to the lower block index);
* the approximation A^ of eq. actual_approx_mat_form: inside a selected block
  every entry is exp(P_ij) (the scale-1 components), every other block is the
  constant exp(S~_xy) (the scale-b component it was not replaced by);
* Z = D^ A^ V with D^ the diagonal that makes every row of A^ sum to one
  (Sec. 2.1, eq. softmax-attention, applied to A^).

Readings of points the paper leaves open (scale 1/sqrt(d) kept in both fine and
coarse logits, per-row budget, replacement rather than addition, factor b on
the coarse term in Alg. 2, ties to the lower index, ascending index lists) are
listed with their reasons in the design notes.

The sparse-only variant MRA-2-s (Sec. 5: only the scale-1 components over the
selected blocks, normalised by their own row sums) is ``mra2s_rows``.

Three resolutions R = {s0, b, 1} (Alg. 1 with two refinement levels, budgets
per block-row at each level) are ``select_multilevel``,
``mra_multilevel_dense`` and ``mra_multilevel_factored``; any number of
resolutions R = {s_0 > s_1 > ... > s_{L-1}, 1} (Alg. 1 refining level by
level) are ``select_levels``, ``mra_levels_dense`` and
``mra_levels_factored``.

Gradients with the selection held fixed (``mra_grads``) differentiate the
factored form written with torch float64 CPU operations (``mra_torch``, which
can also leave out the coarse part: MRA-2-s); ``mra_lse`` gives each query's
log normaliser, the natural log of its row sum of A^.

Two forms of the output are provided: the dense definition over the full
logit slab of each block-row (``mra_dense``) and the factored form of Alg. 2
(``mra_factored``), where the unselected blocks contribute b*exp(S~)*V~_y.
The tests check that they agree.

Conventions: single-head functions take 2-D arrays [n, d]; batched wrappers
take [B, H, n, d]. Every array is converted to float64 on entry.
"""
from __future__ import annotations

import math
import numpy as np


# --------------------------------------------------------------------------
# Sec. 4.1 / 4.3: block means (eq. recursive_pooling, eq. recursive_pooling_V)
# --------------------------------------------------------------------------
def block_mean(x, b):
    """Rows of x averaged over consecutive blocks of b rows: [n, d] -> [n/b, d]."""
    x = np.asarray(x, dtype=np.float64)
    n, d = x.shape
    if n % b:
        raise ValueError("sequence length must be a multiple of the block size")
    return x.reshape(n // b, b, d).sum(axis=1) / b


# --------------------------------------------------------------------------
# Sec. 4.1, eq. exp_of_average: coarse logits S~ = Q~ K~^T / sqrt(d)
# --------------------------------------------------------------------------
def coarse_logits(qp, kp):
    """S~[x, y] = Q~_x . K~_y / sqrt(d); mu_{b,x,y} = exp(S~[x, y])."""
    qp = np.asarray(qp, dtype=np.float64)
    kp = np.asarray(kp, dtype=np.float64)
    return (qp @ kp.T) / math.sqrt(qp.shape[1])


# --------------------------------------------------------------------------
# Sec. 4.2, Alg. 1: pop the blocks with the largest mu, per block-row
# --------------------------------------------------------------------------
def select_blocks(S, m):
    """For every block-row x, the m column blocks with the largest S~[x, .]
    (equivalently the largest mu, exp being increasing); among equal scores
    the lower index wins. Each row of the result is in ascending order."""
    S = np.asarray(S, dtype=np.float64)
    nb = S.shape[1]
    if not 0 <= m <= nb:
        raise ValueError("budget out of range")
    out = np.empty((S.shape[0], m), dtype=np.int64)
    cols = np.arange(nb)
    for x in range(S.shape[0]):
        order = np.lexsort((cols, -S[x]))      # primary: -score, then index
        out[x] = np.sort(order[:m])
    return out


# --------------------------------------------------------------------------
# Sec. 4.2, Alg. 1 with one budget for the whole head (R = {b, 1}): pop the
# m_1 blocks with the largest mu over all (x, y); J may start with priors
# --------------------------------------------------------------------------
def select_global(S, budget, prior_diagonal=False):
    """The blocks refined for one head when Alg. 1 pops `budget` blocks over
    all nb x nb coarse blocks at once: the `budget` largest S~[x, y] (equal
    scores: the lower flat index x*nb + y first) among the blocks that are not
    priors, plus the priors (with prior_diagonal, every diagonal block (x, x)
    is refined from the start and does not count against the budget).

    Returns an int64 array [nb, nb]: row x lists its refined column blocks in
    ascending order, followed by -1 up to nb entries."""
    S = np.asarray(S, dtype=np.float64)
    nb = S.shape[0]
    assert S.shape == (nb, nb)
    prior = np.eye(nb, dtype=bool) if prior_diagonal else np.zeros((nb, nb), dtype=bool)
    free = np.flatnonzero(~prior.ravel())
    if not 0 <= budget <= free.size:
        raise ValueError("budget out of range")
    order = free[np.lexsort((free, -S.ravel()[free]))]   # primary: -score, then flat index
    keep = prior.ravel().copy()
    keep[order[:budget]] = True
    keep = keep.reshape(nb, nb)
    out = np.full((nb, nb), -1, dtype=np.int64)
    for x in range(nb):
        ys = np.flatnonzero(keep[x])
        out[x, :ys.size] = ys
    return out


def rows_of(idx):
    """The valid entries (0 <= y < nb) of every row of a padded selection."""
    idx = np.asarray(idx, dtype=np.int64)
    nb = idx.shape[0]
    return [r[(r >= 0) & (r < nb)] for r in idx]


def mra_global(q, k, v, b, budget, prior_diagonal=False, idx=None):
    """MRA-2 for one head with the head-wide budget of select_global: Z and the
    padded selection. The approximation and its normalisation are those of
    mra_factored_rows (scale-1 entries on refined blocks, b*exp(S~) V~ on the
    others)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    if idx is None:
        S = coarse_logits(block_mean(q, b), block_mean(k, b))
        idx = select_global(S, budget, prior_diagonal)
    Z, _, _ = mra_factored_rows(q, k, v, b, 0, idx=rows_of(idx))
    return Z, idx


# --------------------------------------------------------------------------
# eq. actual_approx_mat_form: the logits of A^ for one block-row
# --------------------------------------------------------------------------
def approx_logits_slab(q, k, S, sel, b, x):
    """log A^ restricted to the b query rows of block-row x: an array [b, n].

    Inside a selected column block the entry is the fine logit P_ij (scale-1
    component, mu_{1,i,j} = exp(P_ij)); every other column of block y holds the
    coarse logit S~[x, y] (scale-b component, mu_{b,x,y})."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    n, d = k.shape
    nb = n // b
    rows = q[x * b:(x + 1) * b]
    slab = np.repeat(S[x], b)[None, :].repeat(b, axis=0)      # coarse everywhere
    for y in sel:
        cols = slice(y * b, (y + 1) * b)
        slab[:, cols] = rows @ k[cols].T / math.sqrt(d)         # replace by fine
    assert slab.shape == (b, nb * b)
    return slab


def approx_matrix(q, k, b, idx):
    """Dense A^ (n x n) for a single head with the given selection. Tiny n only."""
    qp, kp = block_mean(q, b), block_mean(k, b)
    S = coarse_logits(qp, kp)
    nb = S.shape[0]
    return np.vstack([np.exp(approx_logits_slab(q, k, S, idx[x], b, x)) for x in range(nb)])


def _normalised_rows(logits, v):
    """Rows of exp(logits) normalised to sum 1, times v; shifted by the row max
    (the normalised result does not depend on the shift)."""
    z = logits - logits.max(axis=1, keepdims=True)
    w = np.exp(z)
    return (w @ v) / w.sum(axis=1, keepdims=True)


def mra_dense(q, k, v, b, m, idx=None):
    """Z = D^ A^ V for one head from the dense slab of each block-row.

    If idx is given it replaces the selection of Alg. 1 (used to evaluate the
    output under another, equally valid, tie choice). Returns (Z, idx)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    qp, kp = block_mean(q, b), block_mean(k, b)
    S = coarse_logits(qp, kp)
    if idx is None:
        idx = select_blocks(S, m)
    Z = np.empty((q.shape[0], v.shape[1]))
    for x in range(S.shape[0]):
        slab = approx_logits_slab(q, k, S, idx[x], b, x)
        Z[x * b:(x + 1) * b] = _normalised_rows(slab, v)
    return Z, idx


# --------------------------------------------------------------------------
# Sec. 4.3, Alg. 2 at s = b: the low-resolution term of one block-row
# --------------------------------------------------------------------------
def coarse_term(S_row, sel, vp, b):
    """For the unselected blocks y of one block-row, with M the largest
    unselected S~: returns (M, c, L) where c = sum_y b*exp(S~_y - M) and
    L = sum_y b*exp(S~_y - M) * V~_y. With no unselected block, M = -inf and
    c, L are zero. The factor b counts the b columns each block spans."""
    S_row = np.asarray(S_row, dtype=np.float64)
    vp = np.asarray(vp, dtype=np.float64)
    mask = np.ones(S_row.shape[0], dtype=bool)
    mask[np.asarray(sel, dtype=np.int64)] = False
    if not mask.any():
        return -np.inf, 0.0, np.zeros(vp.shape[1])
    M = S_row[mask].max()
    w = b * np.exp(S_row[mask] - M)
    return M, w.sum(), w @ vp[mask]


def mra_factored_rows(q, k, v, b, m, rows=None, idx=None):
    """Z for the given block-rows of one head, computed as in Alg. 2:
    fine products exp(P) V over the selected blocks plus the coarse term
    b*exp(S~_xy) V~_y over the rest, divided by the matching row sums.

    Returns (Z_rows [len(rows)*b, d], idx_rows [len(rows), m], S [nb, nb] rows)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    n, d = q.shape
    nb = n // b
    rows = list(range(nb)) if rows is None else list(rows)
    qp, kp, vp = block_mean(q, b), block_mean(k, b), block_mean(v, b)
    S = coarse_logits(qp[rows], kp)
    sel_all = select_blocks(S, m) if idx is None else idx   # rows may differ in length
    out = np.empty((len(rows) * b, v.shape[1]))
    for r, x in enumerate(rows):
        sel = np.asarray(sel_all[r], dtype=np.int64)
        M, c, L = coarse_term(S[r], sel, vp, b)
        qx = q[x * b:(x + 1) * b]
        if len(sel):
            cols = np.concatenate([np.arange(y * b, (y + 1) * b) for y in sel])
            P = qx @ k[cols].T / math.sqrt(d)
            mf = P.max(axis=1, keepdims=True)
        else:
            cols = np.zeros(0, dtype=np.int64)
            P = np.zeros((b, 0))
            mf = np.full((b, 1), -np.inf)
        top = np.maximum(mf, M)
        wf = np.exp(P - top)
        wc = np.exp(M - top) if np.isfinite(M) else np.zeros_like(top)
        num = wf @ v[cols] + wc * L[None, :]
        den = wf.sum(axis=1, keepdims=True) + wc * c
        out[r * b:(r + 1) * b] = num / den
    return out, sel_all, S


def mra_factored(q, k, v, b, m, idx=None):
    Z, idx, _ = mra_factored_rows(q, k, v, b, m, idx=idx)
    return Z, idx


# --------------------------------------------------------------------------
# Sec. 5, MRA-2-s: only the scale-1 part A^_1 over the selected blocks J,
# normalised by its own row sums (D^ applied to A^_1)
# --------------------------------------------------------------------------
def mra2s_rows(q, k, v, b, m, idx=None, rows=None):
    """Z = D^ A^_1 V for one head: for query i in block-row x, the softmax of
    the fine logits P_ij = q_i . k_j / sqrt(d) over the columns j of the
    selected blocks T_x only, times V. Needs m >= 1. With `rows`, only those
    block-rows (idx then lists their selections in the same order). Returns
    (Z [len(rows)*b, d], idx)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    n, d = q.shape
    nb = n // b
    rows = list(range(nb)) if rows is None else list(rows)
    if idx is None:
        if m < 1:
            raise ValueError("MRA-2-s needs at least one selected block per row")
        S = coarse_logits(block_mean(q, b)[rows], block_mean(k, b))
        idx = select_blocks(S, m)
    Z = np.empty((len(rows) * b, v.shape[1]))
    for r, x in enumerate(rows):
        cols = np.concatenate([np.arange(y * b, (y + 1) * b) for y in np.asarray(idx[r], dtype=np.int64)])
        P = q[x * b:(x + 1) * b] @ k[cols].T / math.sqrt(d)
        Z[r * b:(r + 1) * b] = _normalised_rows(P, v[cols])
    return Z, idx


def mra2s_batched(q, k, v, b, m, idx=None):
    """MRA-2-s Z and idx for every head of [B, H, n, d] inputs."""
    B, H, n, d = q.shape
    Z = np.empty((B, H, n, v.shape[-1]))
    I = np.empty((B, H, n // b, m), dtype=np.int64)
    for bb in range(B):
        for h in range(H):
            Z[bb, h], I[bb, h] = mra2s_rows(q[bb, h], k[bb, h], v[bb, h], b, m,
                                            idx=None if idx is None else idx[bb, h])
    return Z, I


# --------------------------------------------------------------------------
# Sec. 4.2 Alg. 1 and Sec. 4.3 Alg. 2 with three resolutions R = {s0, b, 1}
# (s0 a multiple of b), budgets per block-row at every scale
# --------------------------------------------------------------------------
def select_multilevel(q, k, s0, b, m1, m2):
    """Alg. 1 for R = {s0, b, 1}, applied row by row: every s0-block-row X
    keeps the m1 s0-blocks Y with the largest S~0[X, Y] (its refined coarse
    blocks); every b-block-row x then keeps, among the b-blocks inside its
    parent row's refined s0-blocks (m1 * s0/b candidates), the m2 with the
    largest S~[x, y] (those become exact). Ties: lower index first. Returns
    (idx1 [n/s0, m1], idx2 [n/b, m2]), rows ascending."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    n = q.shape[0]
    r = s0 // b
    S0 = coarse_logits(block_mean(q, s0), block_mean(k, s0))
    idx1 = select_blocks(S0, m1)
    S1 = coarse_logits(block_mean(q, b), block_mean(k, b))
    nb = n // b
    if not 0 <= m2 <= m1 * r:
        raise ValueError("second-level budget out of range")
    idx2 = np.empty((nb, m2), dtype=np.int64)
    for x in range(nb):
        cand = [int(Y) * r + t for Y in idx1[x // r] for t in range(r)]
        best = sorted(cand, key=lambda y: (-S1[x, y], y))[:m2]
        idx2[x] = sorted(best)
    return idx1, idx2


def multilevel_logits_slab(q, k, s0, b, idx1, idx2, x):
    """The b x n logits of block-row x under eq. actual_approx_mat_form with
    three scales: exact P_ij inside its refined b-blocks, S~[x, y] inside the
    other b-blocks of its parent's refined s0-blocks, S~0[X, Y] in the
    s0-blocks its parent row did not refine."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    n, d = q.shape
    r = s0 // b
    X = x // r
    S0 = coarse_logits(block_mean(q, s0), block_mean(k, s0))
    S1 = coarse_logits(block_mean(q, b), block_mean(k, b))
    P = q[x * b:(x + 1) * b] @ k.T / math.sqrt(d)
    refined0 = set(int(Y) for Y in idx1[X])
    refined1 = set(int(y) for y in idx2[x])
    slab = np.empty((b, n))
    for j in range(n):
        Y, y = j // s0, j // b
        if Y not in refined0:
            slab[:, j] = S0[X, Y]
        elif y not in refined1:
            slab[:, j] = S1[x, y]
        else:
            slab[:, j] = P[:, j]
    return slab


def mra_multilevel_dense(q, k, v, s0, b, m1, m2, idx1=None, idx2=None):
    """Z = D^ A^ V for one head with R = {s0, b, 1} (dense slab per
    block-row). Returns (Z, idx1, idx2)."""
    if idx1 is None:
        idx1, idx2 = select_multilevel(q, k, s0, b, m1, m2)
    v = np.asarray(v, dtype=np.float64)
    nb = q.shape[0] // b
    Z = np.vstack([_normalised_rows(multilevel_logits_slab(q, k, s0, b, idx1, idx2, x), v) for x in range(nb)])
    return Z, idx1, idx2


def multilevel_coarse_term(q, k, v, s0, b, idx1, idx2, x):
    """Alg. 2's low-resolution part of block-row x with three scales, shifted
    by its largest coarse logit M: (M, c, L) with c = sum of s0 e^{S~0 - M}
    over the parent row's unrefined s0-blocks plus b e^{S~ - M} over the
    unrefined b-blocks inside its refined s0-blocks, and L the same sums
    weighting V~0_Y and V~_y (each coarse block counts the columns it spans)."""
    return _multilevel_term(_multilevel_means(q, k, v, s0, b), s0, b, idx1, idx2, x)


def _multilevel_means(q, k, v, s0, b):
    """(S~0, S~, V~0, V~) of one head: the coarse logits and pooled values at
    both scales."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    S0 = coarse_logits(block_mean(q, s0), block_mean(k, s0))
    S1 = coarse_logits(block_mean(q, b), block_mean(k, b))
    return S0, S1, block_mean(v, s0), block_mean(v, b)


def _multilevel_term(means, s0, b, idx1, idx2, x):
    """multilevel_coarse_term from the head's precomputed means."""
    S0, S1, vp0, vp1 = means
    r = s0 // b
    X = x // r
    refined0 = set(int(Y) for Y in idx1[X])
    refined1 = set(int(y) for y in idx2[x])
    terms = [(S0[X, Y], s0, vp0[Y]) for Y in range(S0.shape[1]) if Y not in refined0]
    terms += [(S1[x, Y * r + t], b, vp1[Y * r + t]) for Y in sorted(refined0) for t in range(r)
              if Y * r + t not in refined1]
    if not terms:
        return -np.inf, 0.0, np.zeros(vp1.shape[1])
    M = max(t[0] for t in terms)
    c = sum(w * math.exp(lg - M) for lg, w, _ in terms)
    L = sum(w * math.exp(lg - M) * vv for lg, w, vv in terms)
    return M, c, L


def mra_multilevel_factored(q, k, v, s0, b, m1, m2, idx1=None, idx2=None, rows=None):
    """The same Z computed as in Alg. 2: exact tiles exp(P) V over the
    refined b-blocks merged with multilevel_coarse_term. With `rows`, only
    those block-rows (stacked). Returns (Z, idx1, idx2)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    n, d = q.shape
    if idx1 is None:
        idx1, idx2 = select_multilevel(q, k, s0, b, m1, m2)
    rows = list(range(n // b)) if rows is None else list(rows)
    out = np.empty((len(rows) * b, v.shape[1]))
    means = _multilevel_means(q, k, v, s0, b)
    for i, x in enumerate(rows):
        M, c, L = _multilevel_term(means, s0, b, idx1, idx2, x)
        sel = [int(y) for y in idx2[x]]
        qx = q[x * b:(x + 1) * b]
        if sel:
            cols = np.concatenate([np.arange(y * b, (y + 1) * b) for y in sel])
            P = qx @ k[cols].T / math.sqrt(d)
            mf = P.max(axis=1, keepdims=True)
        else:
            cols = np.zeros(0, dtype=np.int64)
            P = np.zeros((b, 0))
            mf = np.full((b, 1), -np.inf)
        top = np.maximum(mf, M)
        wf = np.exp(P - top)
        wc = np.exp(M - top) if np.isfinite(M) else np.zeros_like(top)
        out[i * b:(i + 1) * b] = (wf @ v[cols] + wc * L[None, :]) / (wf.sum(axis=1, keepdims=True) + wc * c)
    return out, idx1, idx2


# --------------------------------------------------------------------------
# Sec. 4.2 Alg. 1 and Sec. 4.3 Alg. 2 with any number of resolutions
# R = {s_0 > s_1 > ... > s_{L-1}, 1}: the blocks popped at scale s_l are
# replaced by their s_{l+1}-blocks, whose block-rows then pop their own budget
# among those; the blocks popped at the last coarse scale become exact
# --------------------------------------------------------------------------
def _check_levels(n, scales, budgets):
    scales = [int(s) for s in scales]
    budgets = [int(m) for m in budgets]
    if not scales or len(scales) != len(budgets):
        raise ValueError("one budget per coarse scale")
    for l, s in enumerate(scales):
        if s < 1 or n % s:
            raise ValueError("every scale must divide the sequence length")
        if l > 0 and (s >= scales[l - 1] or scales[l - 1] % s):
            raise ValueError("scales must decrease, each dividing the one before")
    return scales, budgets


def select_levels(q, k, scales, budgets):
    """Alg. 1 refined level by level, per block-row: every s_0-block-row keeps
    the budgets[0] s_0-blocks with the largest S~_0; at level l every
    s_l-block-row keeps, among the s_l-blocks inside its parent row's (scale
    s_{l-1}) kept blocks, the budgets[l] with the largest S~_l. Ties: lower
    index first. Returns [idx_0, ..., idx_{L-1}], idx_l [n/s_l, budgets[l]]
    with rows ascending."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    n = q.shape[0]
    scales, budgets = _check_levels(n, scales, budgets)
    idx = []
    for l, (s, m) in enumerate(zip(scales, budgets)):
        S = coarse_logits(block_mean(q, s), block_mean(k, s))
        if l == 0:
            idx.append(select_blocks(S, m))
            continue
        p = scales[l - 1] // s
        if not 0 <= m <= budgets[l - 1] * p:
            raise ValueError("budget out of range")
        out = np.empty((n // s, m), dtype=np.int64)
        for x in range(n // s):
            cand = [int(Y) * p + t for Y in idx[l - 1][x // p] for t in range(p)]
            out[x] = sorted(sorted(cand, key=lambda y: (-S[x, y], y))[:m])
        idx.append(out)
    return idx


def levels_logits_slab(q, k, scales, idx, x):
    """The s_{L-1} x n logits of finest block-row x under eq.
    actual_approx_mat_form: column j takes the coarse logit S~_l of the first
    level l whose block around j the row's ancestor at that level did not
    keep, and the exact P_ij if every level kept it."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    n, d = q.shape
    b = scales[-1]
    S = [coarse_logits(block_mean(q, s), block_mean(k, s)) for s in scales]
    kept = [set(int(Y) for Y in idx[l][x * b // s]) for l, s in enumerate(scales)]
    P = q[x * b:(x + 1) * b] @ k.T / math.sqrt(d)
    slab = np.empty((b, n))
    for j in range(n):
        for l, s in enumerate(scales):
            if j // s not in kept[l]:
                slab[:, j] = S[l][x * b // s, j // s]
                break
        else:
            slab[:, j] = P[:, j]
    return slab


def mra_levels_dense(q, k, v, scales, budgets, idx=None):
    """Z = D^ A^ V for one head with R = {scales..., 1} (dense slab per finest
    block-row). Returns (Z, idx list)."""
    if idx is None:
        idx = select_levels(q, k, scales, budgets)
    v = np.asarray(v, dtype=np.float64)
    nb = q.shape[0] // scales[-1]
    Z = np.vstack([_normalised_rows(levels_logits_slab(q, k, scales, idx, x), v) for x in range(nb)])
    return Z, idx


def levels_coarse_term(q, k, v, scales, idx, x):
    """Alg. 2's low-resolution part of finest block-row x, shifted by its
    largest coarse logit M: (M, c, L), c summing s_l e^{S~_l - M} and L
    s_l e^{S~_l - M} V~_l over, at every level l, the s_l-blocks inside the
    ancestor's kept blocks of level l - 1 (all blocks at level 0) that the
    ancestor at level l did not keep."""
    return _levels_term(_levels_means(q, k, v, scales), scales, idx, x)


def _levels_means(q, k, v, scales):
    """[(S~_l, V~_l)] of one head: coarse logits and pooled values per scale."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    return [(coarse_logits(block_mean(q, s), block_mean(k, s)), block_mean(v, s)) for s in scales]


def _levels_term(means, scales, idx, x):
    """levels_coarse_term from the head's precomputed means."""
    b = scales[-1]
    terms = []
    for l, s in enumerate(scales):
        S, vp = means[l]
        X = x * b // s
        if l == 0:
            cand = range(S.shape[1])
        else:
            p = scales[l - 1] // s
            cand = [int(Y) * p + t for Y in idx[l - 1][x * b // scales[l - 1]] for t in range(p)]
        kept = set(int(Y) for Y in idx[l][X])
        terms += [(S[X, Y], s, vp[Y]) for Y in cand if Y not in kept]
    if not terms:
        return -np.inf, 0.0, np.zeros(means[0][1].shape[1])
    M = max(t[0] for t in terms)
    c = sum(w * math.exp(lg - M) for lg, w, _ in terms)
    L = sum(w * math.exp(lg - M) * vv for lg, w, vv in terms)
    return M, c, L


def mra_levels_factored(q, k, v, scales, budgets, idx=None, rows=None):
    """The same Z computed as in Alg. 2: exact tiles exp(P) V over the blocks
    kept at the finest level merged with levels_coarse_term. With `rows`, only
    those finest block-rows (stacked). Returns (Z, idx list)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    n, d = q.shape
    if idx is None:
        idx = select_levels(q, k, scales, budgets)
    b = scales[-1]
    rows = list(range(n // b)) if rows is None else list(rows)
    out = np.empty((len(rows) * b, v.shape[1]))
    means = _levels_means(q, k, v, scales)
    for i, x in enumerate(rows):
        M, c, L = _levels_term(means, scales, idx, x)
        sel = [int(y) for y in idx[-1][x]]
        qx = q[x * b:(x + 1) * b]
        if sel:
            cols = np.concatenate([np.arange(y * b, (y + 1) * b) for y in sel])
            P = qx @ k[cols].T / math.sqrt(d)
            mf = P.max(axis=1, keepdims=True)
        else:
            cols = np.zeros(0, dtype=np.int64)
            P = np.zeros((b, 0))
            mf = np.full((b, 1), -np.inf)
        top = np.maximum(mf, M)
        wf = np.exp(P - top)
        wc = np.exp(M - top) if np.isfinite(M) else np.zeros_like(top)
        out[i * b:(i + 1) * b] = (wf @ v[cols] + wc * L[None, :]) / (wf.sum(axis=1, keepdims=True) + wc * c)
    return out, idx


# --------------------------------------------------------------------------
# Gradients of the MRA-2 output (the selection held fixed): the factored form
# written with torch float64 CPU operations and differentiated by autograd
# --------------------------------------------------------------------------
def mra_torch(q, k, v, b, idx, coarse=True, rows=None):
    """Z for one head as a differentiable function of q, k, v (torch float64
    tensors [n, d]) for a fixed selection `idx` (rows of block ids; entries
    outside [0, nb) ignored). Block-row x's queries take the softmax over the
    fine logits of its refined blocks' columns and the coarse logits
    S~[x, y] + log b of the others (b e^{S~} is e^{S~ + log b}), applied to
    the rows of V and the pooled rows V~ respectively (Alg. 2, eq.
    actual_approx_mat_form). With coarse=False the coarse part is left out:
    the sparse-only variant MRA-2-s (Sec. 5). With `rows`, only those
    block-rows' outputs, stacked in that order."""
    import torch
    n, d = q.shape
    nb = n // b
    qp = q.reshape(nb, b, d).mean(dim=1)
    kp = k.reshape(nb, b, d).mean(dim=1)
    vp = v.reshape(nb, b, v.shape[1]).mean(dim=1)
    S = qp @ kp.T / math.sqrt(d)
    out = []
    for x in (range(nb) if rows is None else rows):
        sel = [int(y) for y in idx[x] if 0 <= int(y) < nb]
        chosen = set(sel)
        rest = [y for y in range(nb) if y not in chosen] if coarse else []
        cols = [j for y in sel for j in range(y * b, (y + 1) * b)]
        parts_l, parts_v = [], []
        if cols:
            parts_l.append(q[x * b:(x + 1) * b] @ k[cols].T / math.sqrt(d))
            parts_v.append(v[cols])
        if rest:
            parts_l.append((S[x, rest] + math.log(b)).expand(b, len(rest)))
            parts_v.append(vp[rest])
        w = torch.softmax(torch.cat(parts_l, dim=1), dim=1)
        out.append(w @ torch.cat(parts_v, dim=0))
    return torch.cat(out, dim=0)


def mra_grads(q, k, v, g, b, idx, coarse=True, rows=None):
    """(dq, dk, dv) = the gradient of sum(g * Z) for one head, Z = mra_torch
    under the fixed selection idx. Arrays in, float64 numpy arrays out. With
    `rows`, the loss covers only those block-rows (g still [n, d]; its other
    rows unused); block-row x's output depends on Q only through Q's rows in
    block x, so dq on those rows is then the full gradient's."""
    import torch
    tq, tk, tv = (torch.tensor(np.asarray(a, dtype=np.float64), requires_grad=True) for a in (q, k, v))
    Z = mra_torch(tq, tk, tv, b, idx, coarse, rows)
    gt = torch.tensor(np.asarray(g, dtype=np.float64))
    if rows is not None:
        gt = torch.cat([gt[x * b:(x + 1) * b] for x in rows], dim=0)
    Z.backward(gt)
    return tq.grad.numpy(), tk.grad.numpy(), tv.grad.numpy()


def mra_grad_terms(q, k, v, g, b, idx, coarse=True, absolute=False):
    """The gradients of sum(g * Z) for one head under the fixed selection idx,
    written out by the chain rule in numpy (an independent formulation of
    mra_grads), or with absolute=True the sums of the magnitudes of the terms
    each gradient element is a sum of: the size against which a rounding of
    those terms is measured (a first-order error bound).

    Per block-row x (queries i, softmax p over the fine logits c Q_i.K_j of
    the refined columns and the coarse logits S~[x,y] + ln b of the other
    blocks, delta_i = g_i . Z_i):
      logit gradient  dl = p (g_i . value - delta_i)
      dq_i += c sum_j dl_ij k_j,  dk_j += c sum_i dl_ij q_i,  dv_j += sum_i p_ij g_i
      dS~[x,y] = sum_i dl_iy (the 32 queries share S~[x,y]),  dV~_y += sum_i p_iy g_i
    then dQ~ = c dS~ K~, dK~ = c dS~^T Q~, each reaching the b rows of its
    block divided by b (the pooled rows are block means). With
    absolute=True every sum is taken over the magnitudes of its terms, down to
    the inputs (|Z| = p |v|, |delta| = |g| . |Z|, |g . v| = |g| . |v|, and the
    difference in dl becomes a sum), so each element bounds what rounding
    any of the intermediate terms can move it by, relative to that
    rounding."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    f = np.abs if absolute else (lambda a: a)
    n, d = q.shape
    nb = n // b
    c = 1.0 / math.sqrt(d)
    qp, kp, vp = block_mean(q, b), block_mean(k, b), block_mean(v, b)
    S = coarse_logits(qp, kp)
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    dS = np.zeros((nb, nb))
    dvp = np.zeros_like(vp)
    for x in range(nb):
        sel = [int(y) for y in idx[x] if 0 <= int(y) < nb]
        chosen = set(sel)
        rest = [y for y in range(nb) if y not in chosen] if coarse else []
        cols = np.array([j for y in sel for j in range(y * b, (y + 1) * b)], dtype=np.int64)
        rows = slice(x * b, (x + 1) * b)
        logits = np.concatenate([q[rows] @ k[cols].T * c,
                                 np.broadcast_to(S[x, rest] + math.log(b), (b, len(rest)))], axis=1)
        e = np.exp(logits - logits.max(axis=1, keepdims=True))
        p = e / e.sum(axis=1, keepdims=True)
        pf, pc = p[:, :len(cols)], p[:, len(cols):]
        Z = pf @ f(v[cols]) + pc @ f(vp[rest])
        delta = (f(g[rows]) * Z).sum(axis=1, keepdims=True)
        gvf, gvc = f(g[rows]) @ f(v[cols]).T, f(g[rows]) @ f(vp[rest]).T
        # absolute: every factor is already a magnitude, and the difference
        # of the two sums becomes their sum
        sgn = 1.0 if absolute else -1.0
        af, ac = pf * (gvf + sgn * delta), pc * (gvc + sgn * delta)
        dq[rows] += c * af @ f(k[cols])
        dk[cols] += c * af.T @ f(q[rows])
        dv[cols] += pf.T @ f(g[rows])
        dS[x, rest] += ac.sum(axis=0)
        dvp[rest] += pc.T @ f(g[rows])
    dq += np.repeat(c * dS @ f(kp), b, axis=0) / b
    dk += np.repeat(c * dS.T @ f(qp), b, axis=0) / b
    dv += np.repeat(dvp, b, axis=0) / b
    return dq, dk, dv


def mra_lse(q, k, b, idx, coarse=True):
    """Each query's log normaliser L_i = ln(sum of row i of A^): the fine
    terms exp(P_ij) of its refined blocks plus, with coarse=True, b exp(S~)
    for every other block (eq. actual_approx_mat_form; the row sums that
    D^ of Sec. 2.1 divides by). Taken with a max shift; float64 [n]."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    n, d = q.shape
    nb = n // b
    S = coarse_logits(block_mean(q, b), block_mean(k, b))
    L = np.empty(n)
    for x in range(nb):
        sel = [int(y) for y in idx[x] if 0 <= int(y) < nb]
        chosen = set(sel)
        rest = [y for y in range(nb) if y not in chosen] if coarse else []
        cols = [j for y in sel for j in range(y * b, (y + 1) * b)]
        parts = []
        if cols:
            parts.append(q[x * b:(x + 1) * b] @ k[cols].T / math.sqrt(d))
        if rest:
            parts.append(np.broadcast_to(S[x, rest] + math.log(b), (b, len(rest))))
        logits = np.concatenate(parts, axis=1)
        mx = logits.max(axis=1)
        L[x * b:(x + 1) * b] = mx + np.log(np.exp(logits - mx[:, None]).sum(axis=1))
    return L


# --------------------------------------------------------------------------
# Sec. 2.1, eq. softmax-attention: exact attention (scale 1/sqrt(d))
# --------------------------------------------------------------------------
def exact_attention(q, k, v):
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    return _normalised_rows(q @ k.T / math.sqrt(q.shape[1]), v)


def exact_attention_rows(q, k, v, i0, i1):
    """Rows i0 .. i1-1 of exact_attention(q, k, v), without forming the other
    rows' logits (for long sequences)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    return _normalised_rows(q[i0:i1] @ k.T / math.sqrt(q.shape[1]), v)


# --------------------------------------------------------------------------
# batched wrappers over [B, H, n, d]
# --------------------------------------------------------------------------
def pool_batched(x, b):
    x = np.asarray(x, dtype=np.float64)
    B, H, n, d = x.shape
    return x.reshape(B, H, n // b, b, d).sum(axis=3) / b


def coarse_batched(qp, kp):
    qp = np.asarray(qp, dtype=np.float64)
    kp = np.asarray(kp, dtype=np.float64)
    return np.einsum("bhxd,bhyd->bhxy", qp, kp) / math.sqrt(qp.shape[-1])


def select_batched(S, m):
    B, H, nb, _ = S.shape
    out = np.empty((B, H, nb, m), dtype=np.int64)
    for bb in range(B):
        for h in range(H):
            out[bb, h] = select_blocks(S[bb, h], m)
    return out


def coarse_term_batched(S, idx, vp, b):
    """(M, c, L) arrays [B,H,nb], [B,H,nb], [B,H,nb,d] for all block-rows."""
    B, H, nb, _ = S.shape
    d = vp.shape[-1]
    M = np.empty((B, H, nb)); c = np.empty((B, H, nb)); L = np.empty((B, H, nb, d))
    for bb in range(B):
        for h in range(H):
            for x in range(nb):
                M[bb, h, x], c[bb, h, x], L[bb, h, x] = coarse_term(S[bb, h, x], idx[bb, h, x], vp[bb, h], b)
    return M, c, L


def mra_batched(q, k, v, b, m, idx=None, form="factored"):
    """Z and idx for every head of [B, H, n, d] inputs."""
    fn = mra_factored if form == "factored" else mra_dense
    B, H, n, d = q.shape
    Z = np.empty((B, H, n, v.shape[-1]))
    I = np.empty((B, H, n // b, m), dtype=np.int64)
    for bb in range(B):
        for h in range(H):
            Z[bb, h], I[bb, h] = fn(q[bb, h], k[bb, h], v[bb, h], b, m,
                                    idx=None if idx is None else idx[bb, h])
    return Z, I

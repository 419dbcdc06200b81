"""COBS decode-step method, written out in float64 (oracle side).

One (batch, KV head) unit at a time: K, V are [T, d] (the cached keys and
values of one KV head), q is [G, d] (the G query heads sharing it).  The
attention scale c multiplies q inside every exponent (the paper absorbs it
into q, Sec. 2 "Notation").

Readings of passages the paper leaves open (kept identical in the HIP path):
  * n_b = min(L, T - b L): a partial tail block scores with ln n_b (Sec. 5.2).
  * The normaliser of eq. (gqa-secondorder) sums over all ceil(T/L) blocks.
  * A block whose tokens all lie in the sliding window is not a candidate;
    the kept token set is the union of the window and the selected blocks,
    each token once, attended with one softmax (Sec. 2 window branch, eq.
    (oracle-true)).
  * Top-s ties go to the lower block index; the set is returned ascending,
    padded with -1.
  * A partial block (n_b < L) stores zero factors; its factors are computed
    when it fills (Sec. 5.6: a block's statistics are rebuilt as it fills).
  * The sign of a stored eigenvector is chosen so that its largest-magnitude
    entry (lowest index on ties) is positive; the score does not depend on it.

This module is test infrastructure (see the package docstring).
"""

import math

import numpy as np

from . import records as rec


# ----------------------------------------------------------------- blocks --

def num_blocks(T, L):
    """ceil(T/L) contiguous, non-overlapping blocks of L tokens (Sec. 2)."""
    return -(-int(T) // int(L))


def block_count(T, L, b):
    """Tokens held by block b: min(L, T - b L)."""
    return min(int(L), int(T) - int(b) * int(L))


def block_mean(Kb):
    """First cumulant of the block's key distribution, eq. (cgf-cumulants)."""
    Kb = np.asarray(Kb, dtype=np.float64)
    return Kb.sum(axis=0) / Kb.shape[0]


def block_covariance(Kb):
    """Second cumulant, the population (1/n) covariance, eq. (cgf-cumulants), App. B."""
    Kb = np.asarray(Kb, dtype=np.float64)
    Kc = Kb - block_mean(Kb)
    return Kc.T @ Kc / Kb.shape[0]


def canonical_sign(xi):
    """Flip each row so its largest-|.| entry (lowest index on ties) is positive."""
    xi = np.array(xi, dtype=np.float64, copy=True)
    for i in range(xi.shape[0]):
        j = int(np.argmax(np.abs(xi[i])))          # argmax returns the first maximum
        if xi[i, j] < 0:
            xi[i] = -xi[i]
    return xi


def scaled_eigenvectors(Sigma, r):
    """Top-r scaled eigenvectors xi_i = sqrt(lambda_i) u_i of Sigma, eq. (lowrank).

    Eigenvalues in descending order; negative rounding noise is clipped to 0.
    Rows i >= d are zero.  Returns [r, d].
    """
    Sigma = np.asarray(Sigma, dtype=np.float64)
    d = Sigma.shape[0]
    lam, U = np.linalg.eigh(Sigma)                 # ascending
    lam, U = lam[::-1], U[:, ::-1]
    xi = np.zeros((r, d))
    k = min(r, d)
    lam_k = np.clip(lam[:k], 0.0, None)
    xi[:k] = (np.sqrt(lam_k)[:, None] * U[:, :k].T)
    return canonical_sign(xi)


def scaled_eigenvectors_gram(Kb, r):
    """Same factors through the Gram trick of Sec. 5.6.

    With centred keys Kc (n x d), the unit eigenpairs (lambda_i, w_i) of the
    n x n Gram matrix Kc Kc^T / n give xi_i = Kc^T w_i / sqrt(n).
    """
    Kb = np.asarray(Kb, dtype=np.float64)
    n, d = Kb.shape
    Kc = Kb - block_mean(Kb)
    Gm = Kc @ Kc.T / n
    lam, W = np.linalg.eigh(Gm)
    lam, W = lam[::-1], W[:, ::-1]
    xi = np.zeros((r, d))
    k = min(r, n)
    xi[:k] = (Kc.T @ W[:, :k]).T / np.sqrt(n)
    # directions with eigenvalue <= 0 carry no energy
    xi[:k][lam[:k] <= 0] = 0.0
    return canonical_sign(xi)


def query_subspace(Q, s):
    """U_Q of Sec. 5.4: the top-s eigenvectors of the query second moment
    E[q q^T], estimated from a sample Q [N, d] as (1/N) sum q q^T; [d, s],
    orthonormal columns, eigenvalues descending."""
    Q = np.asarray(Q, dtype=np.float64)
    M2 = Q.T @ Q / Q.shape[0]
    lam, U = np.linalg.eigh(M2)
    return U[:, ::-1][:, :int(s)]


def energy_rank(Q, frac=0.9):
    """Smallest k whose top-k eigenvalues of the query second moment hold at
    least `frac` of its trace (the rank capturing 90 % of the query spectral
    energy, Sec. 5.4 and Sec. 7.6.2)."""
    Q = np.asarray(Q, dtype=np.float64)
    lam = np.sort(np.linalg.eigvalsh(Q.T @ Q / Q.shape[0]))[::-1]
    cum = np.cumsum(np.clip(lam, 0.0, None))
    return int(np.searchsorted(cum, frac * cum[-1] * (1 - 1e-12)) + 1)


def subspace_covariance(Sigma, U):
    """B_b = U_Q^T Sigma_b U_Q, eq. (subspace)."""
    U = np.asarray(U, dtype=np.float64)
    return U.T @ np.asarray(Sigma, dtype=np.float64) @ U


def subspace_factors(Kb, U, r):
    """Top-r scaled eigenvectors xi^ss of B_b (eq. subspace-lowrank), [r, s]:
    the Gram trick of Sec. 5.6 on the projected centred keys Kc U_Q (the
    paper's route), with eigenvalues of the n x n Gram matrix; sign fixed as
    for the full-space factors."""
    Kb = np.asarray(Kb, dtype=np.float64)
    return scaled_eigenvectors_gram(Kb @ np.asarray(U, dtype=np.float64), r)


def block_statistics(K, T, L, r, U=None):
    """Counts, means and factors of every block of one KV head (Sec. 5.3).

    K [>=T, d].  Returns counts [NB], means [NB, d], factors [NB, r, d], or
    with a query subspace U [d, s] (Sec. 5.4) the subspace factors [NB, r, s]
    of B_b = U^T Sigma_b U.  A partial block stores zero factors.
    """
    K = np.asarray(K, dtype=np.float64)
    d = K.shape[1]
    fd = d if U is None else np.asarray(U).shape[1]
    nb = num_blocks(T, L)
    counts = np.zeros(nb, dtype=np.int64)
    means = np.zeros((nb, d))
    factors = np.zeros((nb, r, fd))
    for b in range(nb):
        n = block_count(T, L, b)
        Kb = K[b * L:b * L + n]
        counts[b] = n
        means[b] = block_mean(Kb)
        if n == L and r > 0:
            if U is None:
                factors[b] = scaled_eigenvectors(block_covariance(Kb), r)
            else:
                factors[b] = scaled_eigenvectors(subspace_covariance(block_covariance(Kb), U), r)
    return counts, means, factors


def skew_coefficients(Kb, xi):
    """Diagonal third cumulant along each stored direction (Sec. 7.7), per factor.

    With u_i = xi_i / |xi_i| and lambda_i = |xi_i|^2, the paper's scalar is
    g_i = (1/n) sum_t (u_i . (k_t - kbar))^3 and its cubic score term is
    (1/6) (u_i . q)^3 g_i.  Stored here: gamma_i = g_i / lambda_i^(3/2) (the
    standardised skewness of the block along u_i), so that the same term is
    (1/6) gamma_i (xi_i . q)^3 from the stored xi_i.  A zero factor gives 0.
    Kb [n, d] keys, xi [r, d] factors  ->  [r].
    """
    Kb = np.asarray(Kb, dtype=np.float64)
    xi = np.asarray(xi, dtype=np.float64)
    Kc = Kb - block_mean(Kb)
    out = np.zeros(xi.shape[0])
    for i in range(xi.shape[0]):
        lam = float(xi[i] @ xi[i])
        if lam > 0.0:
            u = xi[i] / math.sqrt(lam)
            g = float(np.mean((Kc @ u) ** 3))
            out[i] = g / lam ** 1.5
    return out


def block_extras(K, V, T, L, factors, skew, value_mean):
    """Optional record parts of every block: skew coefficients [NB, r] of its
    factors (zero for a partial block, whose factors are zero) and the mean
    value [NB, d] of its tokens (the pooled value of the compression branch).
    Either is None when not asked for."""
    K = np.asarray(K, dtype=np.float64)
    nb, r = factors.shape[0], factors.shape[1]
    skews = np.zeros((nb, r)) if skew else None
    vmeans = np.zeros((nb, K.shape[1])) if value_mean else None
    for b in range(nb):
        n = block_count(T, L, b)
        if skew:
            skews[b] = skew_coefficients(K[b * L:b * L + n], factors[b])
        if value_mean:
            vmeans[b] = block_mean(np.asarray(V, dtype=np.float64)[b * L:b * L + n])
    return skews, vmeans


def stored_statistics(counts, means, factors, mean_dtype, factor_dtype, skews=None, vmeans=None):
    """Round-trip through the descriptor storage format (bf16 / fp32 / E2M1).
    With skew coefficients or value means, returns them too (5-tuple)."""
    d = means.shape[1]
    r, fdim = factors.shape[1], factors.shape[2]
    buf = rec.encode(counts, means, factors, mean_dtype, factor_dtype, skews, vmeans)
    return rec.decode(buf, d, r, mean_dtype, factor_dtype, skews is not None, vmeans is not None, fdim)


# ---------------------------------------------------------------- scoring --

def log_mass_estimate(q, counts, means, factors, c, skews=None, U=None):
    """Second-order log-mass estimate of every block for every query head.

    eq. (trunc) with q <- c q and L <- n_b, curvature through eq. (gram):
        l_b^g = ln n_b + c q_g . kbar_b + (c^2 / 2) sum_i (xi_{b,i} . q_g)^2
    With skew coefficients gamma (Sec. 7.7, see skew_coefficients) the
    diagonal third-order term (c^3 / 6) sum_i gamma_{b,i} (xi_{b,i} . q_g)^3
    is added.  With a query subspace U [d, s] the factors are subspace factors
    [NB, r, s] and meet the projected query U^T q (eq. subspace-quad, eq. gram);
    the mean term keeps the full q.
    q [G, d], counts [NB], means [NB, d], factors [NB, r, d or s]  ->  [NB, G].
    """
    q = np.asarray(q, dtype=np.float64)
    lin = means @ q.T                                   # [NB, G]
    qf = q if U is None else q @ np.asarray(U, dtype=np.float64)
    if factors.shape[1] > 0:
        proj = np.einsum("brd,gd->bgr", factors, qf)    # [NB, G, r]
        quad = (proj ** 2).sum(axis=2)
    else:
        proj = None
        quad = np.zeros_like(lin)
    ell = np.log(np.asarray(counts, dtype=np.float64))[:, None] + c * lin + 0.5 * c * c * quad
    if skews is not None and proj is not None:
        cub = (np.asarray(skews, dtype=np.float64)[:, None, :] * proj ** 3).sum(axis=2)
        ell = ell + (c ** 3 / 6.0) * cub
    return ell


def logsumexp(x, axis):
    x = np.asarray(x, dtype=np.float64)
    m = np.max(x, axis=axis, keepdims=True)
    m = np.where(np.isfinite(m), m, 0.0)
    return np.squeeze(m, axis=axis) + np.log(np.sum(np.exp(x - m), axis=axis))


def group_scores(ell):
    """Log of the GQA group score of eq. (gqa-secondorder).

    Z^g = sum_b exp(l_b^g) over all blocks; score_b = sum_g exp(l_b^g) / Z^g.
    Returns sigma_b = ln score_b (same order as the score).  ell [NB, G].
    """
    lse = logsumexp(ell, axis=0)                        # [G]
    return logsumexp(ell - lse[None, :], axis=1)        # [NB]


def candidate_count(T, L, w):
    """Blocks with at least one token before the window: b L < T - w."""
    ws = max(0, int(T) - int(w))
    return -(-ws // int(L))


def select_top(sigma, nc, s):
    """The min(s, nc) candidates with the largest score, ties to the lower index.

    Returned ascending, padded with -1 to length s.
    """
    k = min(int(s), int(nc))
    order = sorted(range(int(nc)), key=lambda b: (-float(sigma[b]), b))[:k]
    out = -np.ones(int(s), dtype=np.int64)
    out[:k] = sorted(order)
    return out


def union_tokens(T, L, w, sel):
    """Kept tokens: the last w tokens plus every token of a selected block, once each."""
    ws = max(0, int(T) - int(w))
    keep = np.zeros(int(T), dtype=bool)
    keep[ws:T] = True
    for b in np.asarray(sel).tolist():
        if b >= 0:
            keep[b * L:min(b * L + L, T)] = True
    return np.nonzero(keep)[0]


def sparse_attention(q, K, V, U, c):
    """Softmax attention renormalised over the kept tokens U, eq. (oracle-true).

    Returns out [G, d] and lse [G] = ln sum_{t in U} exp(c q_g . k_t).
    An empty U gives out = 0 and lse = -inf.
    """
    q = np.asarray(q, dtype=np.float64)
    G, d = q.shape
    if len(U) == 0:
        return np.zeros((G, d)), np.full(G, -np.inf)
    Ku = np.asarray(K, dtype=np.float64)[U]
    Vu = np.asarray(V, dtype=np.float64)[U]
    s = c * (q @ Ku.T)                                  # [G, |U|]
    m = s.max(axis=1, keepdims=True)
    p = np.exp(s - m)
    l = p.sum(axis=1, keepdims=True)
    return (p @ Vu) / l, (m + np.log(l))[:, 0]


def branch_tokens(T, L, w, sel):
    """The two disjoint token sets of the union: tokens of the selected blocks
    before the window start, and the last w tokens (the selection and window
    branches of the NSA layout of Sec. 2)."""
    ws = max(0, int(T) - int(w))
    sel_set = set()
    for b in np.asarray(sel).tolist():
        if b >= 0:
            sel_set.update(range(b * L, min(b * L + L, ws)))
    return np.array(sorted(sel_set), dtype=np.int64), np.arange(ws, int(T), dtype=np.int64)


def branch_attention(q, K, V, T, L, w, sel, c):
    """Softmax attention of each branch on its own: (out, lse) over the selected
    blocks' tokens and (out, lse) over the window, eq. (oracle-true) on each set."""
    Us, Uw = branch_tokens(T, L, w, sel)
    o_s, l_s = sparse_attention(q, K, V, Us, c)
    o_w, l_w = sparse_attention(q, K, V, Uw, c)
    return o_s, l_s, o_w, l_w


def compression_attention(q, counts, key_means, value_means, c):
    """The mean-pool compression branch (Sec. 2 branch (i); Sec. 5.2 keeps it
    beside the covariance selector): softmax attention of each query head over
    the pooled blocks, block b entering as one key kbar_b (its mean key) with
    one value vbar_b (its mean value), for every block holding a token.
    Returns out [G, d] and lse [G] = ln sum_b exp(c q_g . kbar_b); no blocks
    give 0 and -inf."""
    live = np.asarray(counts) > 0
    return sparse_attention(q, np.asarray(key_means)[live], np.asarray(value_means)[live],
                            np.arange(int(live.sum())), c)


def decode_unit(q, K, V, T, L, r, s, w, c, mean_dtype, factor_dtype, stats=None, skew=False):
    """One decode step of one (batch, KV head) unit, every stage in order.

    stats: optional (counts, means, factors[, skews, vmeans]) already in
    storage precision; otherwise they are built from K (with skew coefficients
    when `skew`) and round-tripped through storage.
    Returns dict(ell, sigma, nc, sel, out, lse, stats).
    """
    if stats is None:
        counts, means, factors = block_statistics(K, T, L, r)
        skews, _ = block_extras(K, V, T, L, factors, skew, False)
        stats = stored_statistics(counts, means, factors, mean_dtype, factor_dtype, skews)
    counts, means, factors = stats[:3]
    skews = stats[3] if len(stats) > 3 else None
    ell = log_mass_estimate(q, counts, means, factors, c, skews)
    sigma = group_scores(ell)
    nc = candidate_count(T, L, w)
    sel = select_top(sigma, nc, s)
    U = union_tokens(T, L, w, sel)
    out, lse = sparse_attention(q, K, V, U, c)
    return dict(ell=ell, sigma=sigma, nc=nc, sel=sel, out=out, lse=lse, stats=stats)


# ------------------------------------------------------------ diagnostics --

def exact_block_log_mass(q, K, T, L, c):
    """ln m_b^g, m_b = sum_{t in b} exp(c q_g . k_t), eq. (bg-defs).  [NB, G]."""
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    nb = num_blocks(T, L)
    out = np.zeros((nb, q.shape[0]))
    for b in range(nb):
        Kb = K[b * L:min(b * L + L, T)]
        out[b] = logsumexp(c * (q @ Kb.T), axis=1)
    return out


def osa_group_scores(q, K, T, L, c):
    """Exact-mass GQA score of eq. (prop-gqa) in log form (OSA, Sec. 3.5)."""
    return group_scores(exact_block_log_mass(q, K, T, L, c))


def quest_block_scores(q, K, T, L):
    """Quest's box score of eq. (rw-quest-score): per block the element-wise
    minimum and maximum of its keys (eq. rw-quest-box), and per query head the
    largest inner product a point of that box attains.  [NB, G]."""
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    nb = num_blocks(T, L)
    out = np.zeros((nb, q.shape[0]))
    for b in range(nb):
        Kb = K[b * L:min(b * L + L, T)]
        kmin, kmax = Kb.min(axis=0), Kb.max(axis=0)
        out[b] = np.maximum(q * kmin[None, :], q * kmax[None, :]).sum(axis=1)
    return out


def quest_group_scores(q, K, T, L, c):
    """Reading for a GQA group: c times the box score stands in for ln m_b^g in
    the group score of eq. (gqa-secondorder) (log form, as for the other
    selectors)."""
    return group_scores(c * quest_block_scores(q, K, T, L))


def block_mixture(q1, K, V, T, L, c):
    """Block probabilities P_b and value centroids v^c_b of one query head.

    eq. (bg-defs) and eq. (oracle-true): o* = sum_b P_b v^c_b.
    q1 [d].  Returns P [NB], centroids [NB, d].
    """
    q1 = np.asarray(q1, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    sc = c * (K[:T] @ q1)
    M = sc.max()
    e = np.exp(sc - M)
    Z = e.sum()
    nb = num_blocks(T, L)
    P = np.zeros(nb)
    cent = np.zeros((nb, K.shape[1]))
    for b in range(nb):
        sl = slice(b * L, min(b * L + L, T))
        mb = e[sl].sum()
        P[b] = mb / Z
        cent[b] = (e[sl][:, None] * V[sl]).sum(axis=0) / mb
    return P, cent


def kept_output(P, cent, kept):
    """o_hat_S = sum_{b in S} P_b v^c_b / (1 - tau), eq. (oracle-true)."""
    kept = np.asarray(kept, dtype=bool)
    tau = P[~kept].sum()
    return (P[kept][:, None] * cent[kept]).sum(axis=0) / (1.0 - tau), tau


def drop_error(P, cent, kept):
    """(1 / (1 - tau)) sum_{b not in S} P_b (v^c_b - o*), eq. (oracle-exact)."""
    kept = np.asarray(kept, dtype=bool)
    o_star = (P[:, None] * cent).sum(axis=0)
    tau = P[~kept].sum()
    return ((P[~kept][:, None] * (cent[~kept] - o_star)).sum(axis=0)) / (1.0 - tau)

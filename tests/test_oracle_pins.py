"""Pins of the fp64 oracle against what the paper and the mathematics fix.

CPU only.  Each test names the passage it pins and the closed form, identity,
brute force or library routine that is independent of the oracle's own code.
"""

import itertools
import math
import os

import numpy as np
import pytest
import torch

from oracle import method as M
from oracle import numerics as nx
from oracle import records as R
from oracle import traffic as TR
import synth


# ------------------------------------------------------------ cumulants --

def test_mean_and_population_covariance_match_library():
    """eq. (cgf-cumulants) and App. B: kappa_1 is the mean, kappa_2 the 1/n covariance."""
    Kb = synth.make_keys_block(64, 64, "gauss", 7).astype(np.float64)
    np.testing.assert_allclose(M.block_mean(Kb), np.mean(Kb, axis=0), rtol=0, atol=1e-14)
    np.testing.assert_allclose(M.block_covariance(Kb), np.cov(Kb.T, bias=True), rtol=0, atol=1e-13)
    # and not the 1/(n-1) estimator
    assert not np.allclose(M.block_covariance(Kb), np.cov(Kb.T, bias=False), atol=1e-6)


def test_zero_variance_block_estimate_is_exact():
    """eq. (trunc): Sigma_b = 0 makes the second-order estimate exact, ln m_b = ln n + c q.k."""
    d, L, c = 64, 64, 1.0 / 8.0
    rng = np.random.default_rng(3)
    K = np.concatenate([synth.make_keys_block(L, d, "const", 11 + i) for i in range(4)]).astype(np.float64)
    q = rng.standard_normal((2, d))
    T = 4 * L - 5                                           # partial tail block too
    counts, means, factors = M.block_statistics(K, T, L, r=3)
    est = M.log_mass_estimate(q, counts, means, factors, c)
    exact = M.exact_block_log_mass(q, K, T, L, c)
    np.testing.assert_allclose(est, exact, rtol=0, atol=1e-12)
    closed = np.log(counts)[:, None] + c * (K[::L][: len(counts)] @ q.T)
    np.testing.assert_allclose(est, closed, rtol=0, atol=1e-12)


@pytest.mark.parametrize("n,d,r", [(64, 64, 64), (64, 128, 63), (32, 16, 16)])
def test_full_rank_factors_reproduce_quadratic_form(n, d, r):
    """eq. (gram) with r >= rank(Sigma_b): sum_i (xi_i . q)^2 = q^T Sigma_b q."""
    Kb = synth.make_keys_block(n, d, "gauss", 5).astype(np.float64)
    Sigma = np.cov(Kb.T, bias=True)                         # library, not the oracle
    q = np.random.default_rng(9).standard_normal((3, d))
    for xi in (M.scaled_eigenvectors(M.block_covariance(Kb), r), M.scaled_eigenvectors_gram(Kb, r)):
        quad = ((xi @ q.T) ** 2).sum(axis=0)
        ref = np.einsum("gd,de,ge->g", q, Sigma, q)
        np.testing.assert_allclose(quad, ref, rtol=1e-11, atol=0)


def test_gram_trick_equals_covariance_eigh():
    """Sec. 5.6 Gram trick: same nonzero eigenvalues, same scaled eigenvectors (sign fixed)."""
    for seed in range(5):
        Kb = synth.make_keys_block(64, 128, "gauss", 100 + seed).astype(np.float64)
        a = M.scaled_eigenvectors(M.block_covariance(Kb), 8)
        b = M.scaled_eigenvectors_gram(Kb, 8)
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-10)
        lam_cov = np.sort(np.linalg.eigvalsh(np.cov(Kb.T, bias=True)))[::-1][:63]
        Kc = Kb - Kb.mean(0)
        lam_gram = np.sort(np.linalg.eigvalsh(Kc @ Kc.T / 64))[::-1][:63]
        np.testing.assert_allclose(lam_cov, lam_gram, rtol=1e-9, atol=1e-12)
        np.testing.assert_allclose((a ** 2).sum(1), lam_cov[:8], rtol=1e-10)


def test_rank_cap_is_n_minus_one():
    """Sec. 7.6.1: a block of L keys has covariance rank at most L - 1; factors beyond are 0."""
    Kb = synth.make_keys_block(16, 64, "gauss", 21).astype(np.float64)
    xi = M.scaled_eigenvectors(M.block_covariance(Kb), 20)
    norms = np.linalg.norm(xi, axis=1)
    assert np.all(norms[:15] > 1e-3)
    assert np.all(norms[15:] < 1e-6)


def test_low_rank_factors_are_best_rank_r():
    """eq. (lowrank): sum_i xi_i xi_i^T is the best rank-r approximation (Eckart-Young via SVD)."""
    Kb = synth.make_keys_block(64, 128, "spiked", 31).astype(np.float64)
    Kc = Kb - Kb.mean(0)
    U, S, Vt = np.linalg.svd(Kc / math.sqrt(64), full_matrices=False)    # library SVD
    best = (Vt[:4].T * S[:4] ** 2) @ Vt[:4]
    xi = M.scaled_eigenvectors(M.block_covariance(Kb), 4)
    np.testing.assert_allclose(xi.T @ xi, best, rtol=0, atol=1e-11)


def test_sign_rule_on_hand_worked_vectors():
    """Reading of the stored eigenvector's sign (the paper leaves it open; the score
    q^T xi xi^T q does not depend on it): each vector is flipped so that its
    largest-magnitude entry is positive, the lowest index winning a tie."""
    xi = np.array([[0.1, -0.5, 0.3],        # largest |.| at index 1, negative: flip
                   [0.2, 0.7, -0.1],        # largest positive already: keep
                   [-0.5, 0.5, 0.0],        # tie between 0 and 1: index 0 decides, flip
                   [0.5, -0.5, 0.25],       # tie, index 0 positive: keep
                   [0.0, 0.0, 0.0]])        # zero vector stays zero
    want = np.array([[-0.1, 0.5, -0.3],
                     [0.2, 0.7, -0.1],
                     [0.5, -0.5, -0.0],
                     [0.5, -0.5, 0.25],
                     [0.0, 0.0, 0.0]])
    np.testing.assert_array_equal(M.canonical_sign(xi), want)
    # every stored factor of a real block obeys the rule (checked entry by entry)
    Kb = synth.make_keys_block(64, 128, "gauss", 41).astype(np.float64)
    for fac in (M.scaled_eigenvectors(M.block_covariance(Kb), 6), M.scaled_eigenvectors_gram(Kb, 6)):
        for row in fac:
            mags = np.abs(row)
            first = int(np.nonzero(mags == mags.max())[0][0])
            assert row[first] > 0


def test_partial_tail_block_stores_zero_factors_until_it_fills():
    """Sec. 5.6 rebuilds a block's factors as the block fills; the reading here: a
    partial block (n_b < L) stores its exact count and mean and zero factors, and
    the same block gets the top-r eigen-factors of its population covariance once
    it holds L keys."""
    L, d, r = 64, 32, 3
    K = synth.make_keys_block(4 * L, d, "gauss", 77).astype(np.float64)
    for m in (1, 17, 63):
        T = 3 * L + m
        counts, means, factors = M.block_statistics(K, T, L, r)
        assert counts.tolist() == [L, L, L, m]
        np.testing.assert_allclose(means[3], np.mean(K[3 * L:T], axis=0), rtol=0, atol=1e-14)
        assert np.all(factors[3] == 0.0)
        for b in range(3):
            assert np.all(np.linalg.norm(factors[b], axis=1) > 0.1)
    counts, means, factors = M.block_statistics(K, 4 * L, L, r)
    assert counts.tolist() == [L] * 4
    # the filled block: top-r eigenpairs of the library's 1/n covariance (up to sign)
    lam, U = np.linalg.eigh(np.cov(K[3 * L:].T, bias=True))
    ref = (np.sqrt(lam[::-1][:r])[:, None] * U[:, ::-1][:, :r].T)
    for i in range(r):
        assert min(np.abs(factors[3, i] - ref[i]).max(), np.abs(factors[3, i] + ref[i]).max()) < 1e-10


def test_gaussian_cgf_has_no_higher_cumulants():
    """eq. (cgf-expansion): for Gaussian keys ln E[exp(c q.x)] = c q.mu + c^2/2 q^T Sigma q.

    The estimate is fed the population mean and a factorisation of Sigma; the
    reference is a Monte-Carlo average over 2^18 samples (CLT error ~2e-3).
    """
    rng = np.random.default_rng(12)
    d, c = 64, 1.0 / 8.0
    A = rng.standard_normal((d, 6)) * 0.35
    Sigma = A @ A.T + 0.05 * np.eye(d)
    mu = rng.standard_normal(d) * 0.3
    q = rng.standard_normal((1, d))
    scale = math.sqrt(0.5 / (c * c * float(q[0] @ Sigma @ q[0])))   # c^2 q^T Sigma q = 0.5
    q = q * scale
    xi = np.linalg.cholesky(Sigma).T                      # Sigma = xi^T xi, d rows
    est = M.log_mass_estimate(q, np.array([1]), mu[None], xi[None], c)[0, 0]
    x = rng.multivariate_normal(mu, Sigma, size=1 << 18)
    mc = math.log(np.mean(np.exp(c * (x @ q[0]))))
    assert abs(est - mc) < 1e-2
    assert abs(est - (c * q[0] @ mu + 0.25)) < 1e-12


def test_second_order_estimate_unbiased_on_gaussian_blocks():
    """Sec. 5.2: on Gaussian blocks the truncated estimate tracks the exact log-mass in expectation.

    Mean of (estimate - exact ln m_b) over 4096 blocks of 64 keys is O(1/n) (~1e-3);
    a dropped or mis-signed term would move it by >= 0.25.
    """
    rng = np.random.default_rng(13)
    d, L, c, nblk = 32, 64, 1.0 / math.sqrt(32), 4096
    A = rng.standard_normal((d, 4)) * 0.5
    Sigma = A @ A.T + 0.1 * np.eye(d)
    q = rng.standard_normal((1, d))
    q = q * math.sqrt(0.5 / (c * c * float(q[0] @ Sigma @ q[0])))
    Lc = np.linalg.cholesky(Sigma)
    K = (rng.standard_normal((nblk * L, d)) @ Lc.T) + rng.standard_normal(d) * 0.2
    T = nblk * L
    counts, means, factors = M.block_statistics(K, T, L, r=d)
    est = M.log_mass_estimate(q, counts, means, factors, c)[:, 0]
    exact = M.exact_block_log_mass(q, K, T, L, c)[:, 0]
    gap = float(np.mean(est - exact))
    assert abs(gap) < 1e-2, gap
    # the first-order (mean-pool) score misses the curvature by ~0.25 on average
    first = M.log_mass_estimate(q, counts, means, factors[:, :0], c)[:, 0]
    assert float(np.mean(exact - first)) > 0.2


# -------------------------------------------------------- selection rule --

def _brute_force_best(P_list, nc, s):
    best, best_set = None, None
    for S in itertools.combinations(range(nc), s):
        kept = np.zeros(len(P_list[0]), dtype=bool)
        kept[list(S)] = True
        loss = sum(P[~kept].sum() for P in P_list)
        if best is None or loss < best - 1e-15:
            best, best_set = loss, S
    return best, best_set


def test_mha_topk_by_mass_minimises_dropped_mass():
    """App. A, MHA case: keeping the top-k blocks by mass minimises tau (brute force over C(15,4))."""
    L, d, c = 8, 16, 0.5
    rng = np.random.default_rng(41)
    K = rng.standard_normal((15 * L, d))
    V = rng.standard_normal((15 * L, d))
    q = rng.standard_normal((1, d))
    T = 15 * L
    P, _ = M.block_mixture(q[0], K, V, T, L, c)
    _, best = _brute_force_best([P], 15, 4)
    sigma = M.osa_group_scores(q, K, T, L, c)
    sel = M.select_top(sigma, 15, 4)
    assert tuple(sel.tolist()) == tuple(sorted(best))
    # same set as sorting the exact log-masses directly
    lm = M.exact_block_log_mass(q, K, T, L, c)[:, 0]
    assert set(sel.tolist()) == set(np.argsort(-lm)[:4].tolist())


def test_gqa_additive_score_minimises_summed_dropped_mass():
    """eq. (prop-gqa) under A3: top-k by sum_g m_b^g / Z^g minimises sum_g tau_g (C(8,3) subsets)."""
    L, d, c, G = 8, 16, 0.6, 2
    rng = np.random.default_rng(42)
    K = rng.standard_normal((8 * L, d))
    V = rng.standard_normal((8 * L, d))
    q = rng.standard_normal((G, d))
    T = 8 * L
    Ps = [M.block_mixture(q[g], K, V, T, L, c)[0] for g in range(G)]
    _, best = _brute_force_best(Ps, 8, 3)
    sel = M.select_top(M.osa_group_scores(q, K, T, L, c), 8, 3)
    assert tuple(sel.tolist()) == tuple(sorted(best))
    # group score equals the normalised mass sum of eq. (prop-gqa)
    np.testing.assert_allclose(np.exp(M.osa_group_scores(q, K, T, L, c)), sum(Ps), rtol=1e-12)


def test_select_top_ties_padding_and_candidates():
    """Reading of the top-s rule: ties to the lower index, ascending output, -1 padding."""
    sigma = np.array([0.5, 1.0, 1.0, 0.2, 1.0, -3.0])
    assert M.select_top(sigma, 6, 2).tolist() == [1, 2]
    assert M.select_top(sigma, 6, 4).tolist() == [0, 1, 2, 4]
    assert M.select_top(sigma, 3, 5).tolist() == [0, 1, 2, -1, -1]
    assert M.select_top(sigma, 0, 3).tolist() == [-1, -1, -1]
    assert M.candidate_count(1024, 64, 64) == 15
    assert M.candidate_count(1000, 64, 64) == 15            # block 14 straddles the window start
    assert M.candidate_count(1000, 64, 0) == 16             # w = 0: the partial tail is a candidate
    assert M.candidate_count(500, 64, 512) == 0             # T <= w: dense window only
    U = M.union_tokens(1000, 64, 100, [3, 14])
    expect = sorted(set(range(900, 1000)) | set(range(192, 256)) | set(range(896, 900)))
    assert U.tolist() == expect


def test_planted_block_is_top_by_exact_and_estimated_mass(golden_dir):
    """Tiny single-head workload: the planted block is the argmax of the exact and estimated masses."""
    with open(os.path.join(golden_dir, "c1_seed.txt")) as f:
        seed = int(f.read().split()[0])
    prob = synth.make_problem("c1", seed=seed)
    cfg = prob["cfg"]
    q = prob["q"][0].numpy().astype(np.float64)
    K = prob["k"][0, 0].numpy().astype(np.float64)
    c = 1.0 / math.sqrt(cfg["d"])
    exact = M.exact_block_log_mass(q, K, cfg["T"], cfg["L"], c)[:15, 0]
    stats = M.block_statistics(K, cfg["T"], cfg["L"], cfg["r"])
    est = M.log_mass_estimate(q, *stats, c)[:15, 0]
    planted = prob["planted"][(0, 0)]
    assert int(np.argmax(exact)) == planted
    assert int(np.argmax(est)) == planted


# ---------------------------------------------------- attention identities --

def _sdpa(q, K, V, c):
    """Dense attention by torch's library routine, float64 on the CPU."""
    qt = torch.from_numpy(q)[None, :, None, :]              # [1, G, 1, d]
    G = q.shape[0]
    Kt = torch.from_numpy(K)[None, None].expand(1, G, -1, -1)
    Vt = torch.from_numpy(V)[None, None].expand(1, G, -1, -1)
    o = torch.nn.functional.scaled_dot_product_attention(qt, Kt, Vt, scale=c)
    return o[0, :, 0].numpy()


def test_full_selection_is_dense_attention():
    """eq. (oracle-true) with tau = 0: s >= #candidates keeps every token -> dense attention."""
    rng = np.random.default_rng(51)
    T, L, d, G, c = 700, 64, 32, 3, 1.0 / math.sqrt(32)
    K = rng.standard_normal((T, d))
    V = rng.standard_normal((T, d))
    q = rng.standard_normal((G, d))
    for w in (0, 64, 100, 1000):
        res = M.decode_unit(q, K, V, T, L, r=2, s=20, w=w, c=c, mean_dtype="f32", factor_dtype="f32")
        np.testing.assert_allclose(res["out"], _sdpa(q, K, V, c), rtol=0, atol=1e-12)
        s = c * q @ K.T
        np.testing.assert_allclose(res["lse"], np.log(np.exp(s).sum(1)), rtol=1e-13)


def test_kept_output_two_ways_and_exact_error_identity():
    """eq. (oracle-true) and eq. (oracle-exact) at w = 0.

    The union softmax equals sum_{b in S} P_b v^c_b / (1 - tau), and
    o* - o_hat_S equals (1/(1 - tau)) sum_{b not in S} P_b (v^c_b - o*).
    """
    rng = np.random.default_rng(52)
    T, L, d, c = 10 * 16, 16, 24, 0.4
    K = rng.standard_normal((T, d))
    V = rng.standard_normal((T, d))
    q = rng.standard_normal((1, d))
    S = [1, 4, 5, 9]
    kept = np.zeros(10, dtype=bool)
    kept[S] = True
    P, cent = M.block_mixture(q[0], K, V, T, L, c)
    o_hat, tau = M.kept_output(P, cent, kept)
    U = M.union_tokens(T, L, 0, S)
    out, _ = M.sparse_attention(q, K, V, U, c)
    np.testing.assert_allclose(out[0], o_hat, rtol=0, atol=1e-12)
    o_star = _sdpa(q, K, V, c)[0]
    np.testing.assert_allclose(o_star - o_hat, M.drop_error(P, cent, kept), rtol=0, atol=1e-12)
    assert 0 < tau < 1


def test_empty_union_gives_zero_and_minus_inf():
    out, lse = M.sparse_attention(np.ones((2, 4)), np.ones((3, 4)), np.ones((3, 4)), np.array([], int), 1.0)
    assert np.all(out == 0) and np.all(np.isneginf(lse))


# --------------------------------------------------------- traffic tables --

def _read_table(path):
    rows = {}
    with open(path) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            parts = line.split()
            rows[parts[0]] = [None if p == "-" else float(p) for p in parts[1:]]
    return rows


def test_bandwidth_table_reproduces(golden_dir):
    """Table "bandwidth": every branch, total and ratio of every row."""
    rows = _read_table(os.path.join(golden_dir, "bandwidth_table.txt"))
    args = dict(T=32768, H=4, D=128, L=32, k=16, w=256)
    spec = {
        "dense": ("dense", {}), "osa": ("osa", {}),
        "nsa_mlp": ("nsa_mlp", {}), "nsa_meanpool": ("nsa_meanpool", {}), "nsa_quest": ("nsa_quest", {}),
        "cobs_full_r4_bf16": ("cobs_full", dict(r=4, quant="bf16")),
        "cobs_full_r6_bf16": ("cobs_full", dict(r=6, quant="bf16")),
        "cobs_full_r4_fp4": ("cobs_full", dict(r=4, quant="fp4")),
        "cobs_full_r6_fp4": ("cobs_full", dict(r=6, quant="fp4")),
        "cobs_sub85_r4_fp4": ("cobs_subspace", dict(r=4, quant="fp4", sub_dim=84.875)),
    }
    dense = TR.per_layer_traffic("dense", **args)["total"] / TR.KIB
    nsa = TR.per_layer_traffic("nsa_mlp", **args)["total"] / TR.KIB
    for name, (meth, kw) in spec.items():
        t = TR.per_layer_traffic(meth, **args, **kw)
        keys, vals, win, fine, tot, less, more = rows[name]
        got = [t[k] / TR.KIB for k in ("summary_keys", "summary_values", "window", "fine", "total")]
        want = [0 if v is None else v for v in (keys, vals, win, fine, tot)]
        assert [round(x) for x in got] == [round(x) for x in want], name
        if less is not None:
            assert round(dense / got[4], 2) == less, name
        if more is not None:
            assert round(got[4] / nsa, 2) == more, name


def test_quant_table_bytes(golden_dir):
    """Table "quant": factor bytes per descriptor and the reduction versus bf16."""
    with open(os.path.join(golden_dir, "quant_bytes.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            r, dim, b16, b4, red = line.split()
            assert TR.factor_bytes(int(r), int(dim), "bf16") == int(b16)
            assert TR.factor_bytes(int(r), int(dim), "fp4") == int(b4)
            assert round(int(b16) / int(b4), 1) == float(red)


def test_subspace_dimension_averages(golden_dir):
    """Figure "subspace-perlayer": averages 68 and 84.875 (about 1.25x)."""
    dark, full = [], []
    with open(os.path.join(golden_dir, "subspace_dims.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            _, a, b = line.split()
            dark.append(int(a))
            full.append(int(a) + int(b))
    assert sum(dark) / 16 == 68
    assert sum(full) / 16 == 84.875
    assert abs(84.875 / 68 - 1.25) < 0.01


def test_record_algorithmic_bytes_match_descriptor_accounting():
    """Table "quant" byte rule applied to the record: count + mean + factors (+ scales)."""
    assert R.algorithmic_bytes(128, 4, "f32", "f32") == 2564
    assert R.algorithmic_bytes(128, 4, "bf16", "bf16") == 1284
    assert R.algorithmic_bytes(128, 4, "bf16", "e2m1") == 4 + 256 + 272
    assert R.algorithmic_bytes(128, 4, "e2m1", "e2m1") == 4 + 68 + 272
    assert R.algorithmic_bytes(64, 2, "f32", "f32") == 772
    for md in R.DTYPES:
        for fd in R.DTYPES:
            lay = R.layout(128, 4, md, fd)
            assert lay["total"] % 16 == 0
            assert lay["total"] - R.algorithmic_bytes(128, 4, md, fd) < 16


def test_branch_outputs_merge_to_the_union_attention():
    """The selection and window branches partition the union: their log-sum-exp
    merge is the union attention, an empty branch is (0, -inf), and a selection
    reaching into the window is cut at the window start."""
    rng = np.random.default_rng(91)
    T, L, d, G, c = 700, 64, 32, 3, 0.2
    K, V, q = rng.standard_normal((T, d)), rng.standard_normal((T, d)), rng.standard_normal((G, d))
    for w, sel in [(100, [0, 3, 9, -1]), (0, [2, 5]), (700, [1]), (150, [-1, -1]), (90, [8, 10])]:
        o_s, l_s, o_w, l_w = M.branch_attention(q, K, V, T, L, w, sel, c)
        o_u, l_u = M.sparse_attention(q, K, V, M.union_tokens(T, L, w, sel), c)
        m = np.maximum(l_s, l_w)
        a, b = np.exp(l_s - m), np.exp(l_w - m)
        np.testing.assert_allclose(m + np.log(a + b), l_u, rtol=0, atol=1e-12)
        np.testing.assert_allclose((a[:, None] * o_s + b[:, None] * o_w) / (a + b)[:, None], o_u, rtol=0, atol=1e-12)
        Us, Uw = M.branch_tokens(T, L, w, sel)
        assert len(np.intersect1d(Us, Uw)) == 0 and np.all(Us < T - w)
    # empty selection branch
    o_s, l_s, _, _ = M.branch_attention(q, K, V, T, L, 100, [-1], c)
    assert np.all(o_s == 0) and np.all(np.isneginf(l_s))


def test_quest_box_score_bounds_and_forms():
    """Box score (eq. rw-quest-score): an upper bound of every key's inner product
    in the block, exact for a one-token block, equal to its second printed form,
    and a bound the box's own corners attain."""
    rng = np.random.default_rng(92)
    T, L, d, G = 200, 64, 16, 3
    K, q = rng.standard_normal((T, d)), rng.standard_normal((G, d))
    sb = M.quest_block_scores(q, K, T, L)
    for b in range(M.num_blocks(T, L)):
        Kb = K[b * L:min(b * L + L, T)]
        assert np.all(sb[b] >= (q @ Kb.T).max(axis=1) - 1e-12)
        kmin, kmax = Kb.min(0), Kb.max(0)
        second = (np.maximum(q, 0) * kmax + np.minimum(q, 0) * kmin).sum(1)
        np.testing.assert_allclose(sb[b], second, rtol=0, atol=1e-12)
        corner = np.where(q > 0, kmax, kmin)            # the maximising corner, per head
        np.testing.assert_allclose(sb[b], (q * corner).sum(1), rtol=0, atol=1e-12)
    # a block of one token: the bound is that token's inner product
    one = M.quest_block_scores(q, K, 1, L)
    np.testing.assert_allclose(one[0], q @ K[0], rtol=0, atol=1e-12)
    # brute force over the box's corners on a tiny case
    Kt, qt = rng.standard_normal((5, 3)), rng.standard_normal((1, 3))
    lo, hi = Kt.min(0), Kt.max(0)
    corners = np.array([[lo[0] if a else hi[0], lo[1] if b_ else hi[1], lo[2] if c_ else hi[2]]
                        for a in (0, 1) for b_ in (0, 1) for c_ in (0, 1)])
    np.testing.assert_allclose(M.quest_block_scores(qt, Kt, 5, 8)[0, 0], (corners @ qt[0]).max(), atol=1e-12)


# ------------------------------------------------- diagonal skew (Sec. 7.7) --

def _rank1_skewed_block(n, d, seed):
    """Keys varying along one unit direction u with exponential (skewed) weights."""
    rng = np.random.default_rng(seed)
    u = rng.standard_normal(d)
    u /= np.linalg.norm(u)
    m = rng.standard_normal(d)
    a = rng.exponential(1.0, n)
    return m[None, :] + a[:, None] * u[None, :], u


def test_skew_term_is_the_exact_third_cumulant_for_a_rank_one_block():
    """For keys along one direction the third cumulant tensor is g u (x) u (x) u,
    so the diagonal term equals (c^3 / 6) (1/n) sum_t (q . (k_t - kbar))^3,
    computed here from the keys by brute force."""
    Kb, u = _rank1_skewed_block(64, 32, 5)
    counts, means, factors = M.block_statistics(Kb, 64, 64, 2)
    skews, _ = M.block_extras(Kb, None, 64, 64, factors, True, False)
    q = np.random.default_rng(6).standard_normal((3, 32))
    c = 0.2
    l2 = M.log_mass_estimate(q, counts, means, factors, c)
    l3 = M.log_mass_estimate(q, counts, means, factors, c, skews)
    Kc = Kb - Kb.mean(axis=0)
    brute = c ** 3 / 6.0 * np.mean((Kc @ q.T) ** 3, axis=0)
    np.testing.assert_allclose((l3 - l2)[0], brute, rtol=1e-10, atol=1e-13)
    assert abs(skews[0, 0]) > 0.5                 # an exponential law is strongly skewed
    assert np.max(np.abs(brute)) > 1e-3


def test_skew_term_vanishes_for_symmetric_blocks_and_ignores_the_sign():
    """A block symmetric about its mean has no third cumulant; flipping a stored
    vector's sign flips its coefficient, leaving the score unchanged."""
    rng = np.random.default_rng(8)
    half = rng.standard_normal((32, 48)) * np.linspace(3, 0.2, 48)
    Kb = np.concatenate([1.0 + half, 1.0 - half])
    counts, means, factors = M.block_statistics(Kb, 64, 64, 4)
    skews, _ = M.block_extras(Kb, None, 64, 64, factors, True, False)
    np.testing.assert_allclose(skews, 0.0, atol=1e-12)
    Ks, _ = _rank1_skewed_block(64, 48, 9)
    Ks = Ks + 0.3 * rng.standard_normal(Ks.shape)
    xi = M.scaled_eigenvectors(M.block_covariance(Ks), 3)
    q = rng.standard_normal((2, 48))
    g = M.skew_coefficients(Ks, xi)
    gf = M.skew_coefficients(Ks, -xi)
    np.testing.assert_allclose(gf, -g, rtol=1e-12)
    a = M.log_mass_estimate(q, [64], Ks.mean(0)[None], xi[None], 0.3, g[None])
    b = M.log_mass_estimate(q, [64], Ks.mean(0)[None], -xi[None], 0.3, gf[None])
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_third_order_estimate_has_a_fourth_order_remainder():
    """eq. (cgf-expansion) truncated after kappa_3: on a rank-one block the error
    of the third-order estimate against the exact ln m_b shrinks 16-fold when q
    halves, that of the second-order estimate 8-fold."""
    Kb, u = _rank1_skewed_block(64, 16, 12)
    counts, means, factors = M.block_statistics(Kb, 64, 64, 1)
    skews, _ = M.block_extras(Kb, None, 64, 64, factors, True, False)
    errs = []
    for scale in (0.08, 0.04):
        q = (scale * u)[None, :]
        exact = M.exact_block_log_mass(q, Kb, 64, 64, 1.0)[0, 0]
        l2 = M.log_mass_estimate(q, counts, means, factors, 1.0)[0, 0]
        l3 = M.log_mass_estimate(q, counts, means, factors, 1.0, skews)[0, 0]
        errs.append((abs(l2 - exact), abs(l3 - exact)))
    (e2a, e3a), (e2b, e3b) = errs
    assert e3a < e2a and e3b < e2b
    assert 6.5 < e2a / e2b < 9.5, e2a / e2b
    assert 13.0 < e3a / e3b < 19.0, e3a / e3b


# ---------------------------------------- compression branch (Sec. 2, 5.2) --

def test_compression_branch_of_one_token_blocks_is_dense_attention():
    """With one token per block the pooled keys and values are the tokens
    themselves: the branch is softmax attention over every token, written out
    here directly."""
    rng = np.random.default_rng(21)
    K, V, q = rng.standard_normal((40, 16)), rng.standard_normal((40, 16)), rng.standard_normal((3, 16))
    counts, means, factors = M.block_statistics(K, 40, 1, 0)
    _, vmeans = M.block_extras(K, V, 40, 1, factors, False, True)
    out, lse = M.compression_attention(q, counts, means, vmeans, 0.25)
    s = 0.25 * q @ K.T
    p = np.exp(s - s.max(axis=1, keepdims=True))
    np.testing.assert_allclose(out, (p @ V) / p.sum(axis=1, keepdims=True), rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, np.log(np.exp(s).sum(axis=1)), rtol=0, atol=1e-12)


def test_compression_branch_pools_blocks_by_their_means():
    """Blocks of L copies of one (key, value) pool to that pair; a partial tail
    block pools its own tokens; no blocks give 0 and -inf."""
    rng = np.random.default_rng(22)
    reps_k, reps_v = rng.standard_normal((5, 8)), rng.standard_normal((5, 8))
    K = np.repeat(reps_k, 4, axis=0)[:19]
    V = np.repeat(reps_v, 4, axis=0)[:19]
    q = rng.standard_normal((2, 8))
    counts, means, factors = M.block_statistics(K, 19, 4, 0)
    _, vmeans = M.block_extras(K, V, 19, 4, factors, False, True)
    assert counts.tolist() == [4, 4, 4, 4, 3]
    out, lse = M.compression_attention(q, counts, means, vmeans, 0.5)
    s = 0.5 * q @ reps_k.T
    p = np.exp(s)
    np.testing.assert_allclose(out, (p @ reps_v) / p.sum(axis=1, keepdims=True), rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, np.log(p.sum(axis=1)), rtol=0, atol=1e-12)
    o0, l0 = M.compression_attention(q, np.zeros(3, int), np.zeros((3, 8)), np.zeros((3, 8)), 0.5)
    assert np.all(o0 == 0) and np.all(np.isneginf(l0))


def test_records_with_skew_and_value_means_round_trip():
    """fp32 storage of every part is exact; the optional parts sit where the
    layout says, the rest of the record is unchanged."""
    rng = np.random.default_rng(23)
    nb, d, r = 5, 64, 3
    counts = np.array([64, 64, 64, 64, 9])
    means, vmeans = rng.standard_normal((nb, d)), rng.standard_normal((nb, d))
    factors, skews = rng.standard_normal((nb, r, d)), rng.standard_normal((nb, r))
    f32 = lambda x: np.asarray(x).astype(np.float32).astype(np.float64)
    buf = R.encode(counts, means, factors, "f32", "f32", skews, vmeans)
    c2, m2, x2, s2, v2 = R.decode(buf, d, r, "f32", "f32", True, True)
    assert c2.tolist() == counts.tolist()
    for a, b in ((m2, means), (x2, factors), (s2, skews), (v2, vmeans)):
        np.testing.assert_array_equal(a, f32(b))
    plain = R.encode(counts, means, factors, "f32", "f32")
    lay, lay0 = R.layout(d, r, "f32", "f32", True, True), R.layout(d, r, "f32", "f32")
    np.testing.assert_array_equal(buf[:, lay["mean_off"]:lay["vmean_off"]], plain[:, lay0["mean_off"]:lay0["total"]])
    assert lay["total"] == lay0["total"] + 16 + 4 * d


# ------------------------------------------------- subspace COBS (Sec. 5.4) --

def _queries_with_spectrum(lam, seed):
    """A query sample whose second moment (1/N) Q^T Q is exactly V diag(lam) V^T."""
    d = len(lam)
    rng = np.random.default_rng(seed)
    V, _ = np.linalg.qr(rng.standard_normal((d, d)))
    Z, _ = np.linalg.qr(rng.standard_normal((d, d)))       # orthonormal rows: Z^T Z = I
    Q = math.sqrt(d) * Z @ np.diag(np.sqrt(lam)) @ V.T
    return Q, V


def test_query_subspace_and_energy_rank_on_a_known_spectrum():
    """U_Q spans the top-s eigenvectors of E[q q^T]; the rank capturing 90 % of
    the spectral energy is where the cumulative eigenvalue sum first reaches it."""
    lam = np.concatenate([np.full(10, 8.0), np.full(54, 0.1)])   # top 10 hold 80/85.4 = 93.7 %
    Q, V = _queries_with_spectrum(lam, 3)
    np.testing.assert_allclose(Q.T @ Q / len(Q), V @ np.diag(lam) @ V.T, atol=1e-12)
    U = M.query_subspace(Q, 10)
    np.testing.assert_allclose(U.T @ U, np.eye(10), atol=1e-12)
    np.testing.assert_allclose(U @ U.T, V[:, :10] @ V[:, :10].T, atol=1e-10)
    assert M.energy_rank(Q, 0.9) == 10
    lam2 = np.linspace(2.0, 0.02, 64)
    Q2, _ = _queries_with_spectrum(lam2, 4)
    cum = np.cumsum(lam2) / lam2.sum()
    assert M.energy_rank(Q2, 0.9) == int(np.argmax(cum >= 0.9)) + 1


def test_subspace_dimension_rule_matches_the_figure(golden_dir):
    """Figure "subspace-perlayer": each layer's full bar is 1.25 times the rank
    capturing 90 % of the query energy (averaged over heads), to the unit."""
    with open(os.path.join(golden_dir, "subspace_dims.txt")) as f:
        rows = [l.split() for l in f if l.strip() and not l.startswith("#")]
    for _, dark, extra in rows:
        dark, full = int(dark), int(dark) + int(extra)
        assert abs(full - 1.25 * dark) <= 1.0, (dark, full)


def test_subspace_factors_with_the_whole_space_are_the_full_factors():
    """U_Q = I (s = d): B_b = Sigma_b, the subspace factors are the full-space
    factors and the scores agree."""
    Kb = synth.make_keys_block(64, 32, "spiked", 61).astype(np.float64)
    I = np.eye(32)
    c1, m1, f1 = M.block_statistics(Kb, 64, 64, 4)
    c2, m2, f2 = M.block_statistics(Kb, 64, 64, 4, U=I)
    np.testing.assert_allclose(f2, f1, atol=1e-10)
    q = np.random.default_rng(62).standard_normal((3, 32))
    np.testing.assert_allclose(M.log_mass_estimate(q, c2, m2, f2, 0.3, U=I),
                               M.log_mass_estimate(q, c1, m1, f1, 0.3), atol=1e-12)


def test_subspace_quadratic_form_is_exact_inside_the_subspace():
    """eq. (subspace-quad): with every direction of B_b kept (r = s), the
    subspace score's curvature equals q^T Sigma_b q for q in the span of U_Q,
    and only the in-subspace part of q otherwise (Sigma from the library)."""
    rng = np.random.default_rng(63)
    d, s = 48, 12
    Kb = synth.make_keys_block(64, d, "gauss", 64).astype(np.float64)
    U, _ = np.linalg.qr(rng.standard_normal((d, s)))
    Sigma = np.cov(Kb.T, bias=True)
    _, _, f = M.block_statistics(Kb, 64, 64, s, U=U)
    q_in = (U @ rng.standard_normal((s, 2))).T
    quad = ((f[0] @ (q_in @ U).T) ** 2).sum(axis=0)
    np.testing.assert_allclose(quad, np.einsum("gd,de,ge->g", q_in, Sigma, q_in), rtol=1e-10)
    q = rng.standard_normal((2, d))
    quad = ((f[0] @ (q @ U).T) ** 2).sum(axis=0)
    Pq = q @ U @ U.T
    np.testing.assert_allclose(quad, np.einsum("gd,de,ge->g", Pq, Sigma, Pq), rtol=1e-10)
    assert not np.allclose(quad, np.einsum("gd,de,ge->g", q, Sigma, q), rtol=1e-3)


def test_subspace_gram_trick_equals_eigh_of_the_projected_covariance():
    """Sec. 5.6 applied to Kc U_Q: the same factors as eigh(U^T Sigma U), with
    the rank-r truncation of eq. (subspace-lowrank) the best one (Eckart-Young)."""
    rng = np.random.default_rng(65)
    Kb = synth.make_keys_block(64, 128, "spiked", 66).astype(np.float64)
    U, _ = np.linalg.qr(rng.standard_normal((128, 40)))
    a = M.subspace_factors(Kb, U, 4)
    _, _, b = M.block_statistics(Kb, 64, 64, 4, U=U)
    np.testing.assert_allclose(a, b[0], atol=1e-10)
    B = U.T @ np.cov(Kb.T, bias=True) @ U
    lam, W = np.linalg.eigh(B)
    best = (W[:, ::-1][:, :4] * lam[::-1][:4]) @ W[:, ::-1][:, :4].T
    np.testing.assert_allclose(a.T @ a, best, atol=1e-10)


def test_subspace_records_store_s_element_factors():
    """Record layout with factors of s elements (Table "quant": subspace r = 4,
    s = 64 takes 512 B in bf16 and 144 B in E2M1, without the mean)."""
    assert R.layout(128, 4, "bf16", "bf16", fdim=64)["vec_bytes"] * 4 == 512
    lay = R.layout(128, 4, "bf16", "e2m1", fdim=64)
    assert lay["vec_bytes"] * 4 + 4 * 4 == 144
    assert R.algorithmic_bytes(128, 4, "bf16", "e2m1", fdim=64) == 4 + 256 + 144
    rng = np.random.default_rng(67)
    f = rng.standard_normal((3, 4, 64))
    buf = R.encode(np.array([64, 64, 5]), rng.standard_normal((3, 128)), f, "f32", "f32")
    _, _, f2 = R.decode(buf, 128, 4, "f32", "f32", fdim=64)
    np.testing.assert_array_equal(f2, f.astype(np.float32).astype(np.float64))

"""Helpers for the GPU parity tests: oracle per (batch row, KV head) unit and
the comparison rules.  Oracle inputs are only generator outputs (never GPU
results)."""

import math

import numpy as np
import torch

from oracle import method as M
from oracle import records as R
from paper_2607_09052_amd import cobs

DEV = "cuda:0"

# Tolerances fixed by the decode-step requirements: relative L2 of the output,
# 2e-3 for bf16 K/V and 1e-5 for fp32 K/V; |sigma| within 2e-5; selection
# bit-exact unless the oracle's score gap at the s-th boundary is below 1e-4.
OUT_TOL = {"bf16": 2e-3, "f32": 1e-5}
LSE_TOL = 1e-5
SIGMA_TOL = 2e-5
BAND = 1e-4


def say(msg):
    print(msg, flush=True)


def config_from(cfg_dict, **over):
    c = dict(batch=cfg_dict["B"], num_q_heads=cfg_dict["Hq"], num_kv_heads=cfg_dict["Hkv"],
             head_dim=cfg_dict["d"], max_seq_len=cfg_dict["T_max"], rank=cfg_dict["r"],
             budget=cfg_dict["s"], window=cfg_dict["w"], kv_dtype=cfg_dict["kv_dtype"],
             mean_dtype=cfg_dict["mean_dtype"], factor_dtype=cfg_dict["factor_dtype"],
             block_size=cfg_dict.get("L", 64))
    c.update(over)
    return cobs.Config(**c)


def f64(t):
    return t.detach().to("cpu").to(torch.float64).numpy()


def oracle_select(rec_unit, q_unit, T, cfg, U=None):
    """Oracle sigma, candidate count and selection of one unit from record bytes.
    A row with no tokens has no blocks, no candidates and no selection.  U: the
    unit's query basis for subspace factors."""
    if T <= 0:
        return np.zeros(0), 0, []
    parts = R.decode(rec_unit, cfg.head_dim, cfg.rank, cfg.mean_dtype, cfg.factor_dtype, cfg.skew, cfg.value_mean,
                     cfg.subspace_dim or None)
    counts, means, factors = parts[:3]
    skews = parts[3] if cfg.skew else None
    nb = M.num_blocks(T, cfg.block_size)
    ell = M.log_mass_estimate(q_unit, counts[:nb], means[:nb], factors[:nb], cfg.scale,
                              None if skews is None else skews[:nb], U)
    sigma = M.group_scores(ell)
    nc = M.candidate_count(T, cfg.block_size, cfg.window)
    return sigma, nc, M.select_top(sigma, nc, cfg.budget)


def check_selection(sel_gpu, sigma, nc, s, band=BAND):
    """Set rule: exact unless the oracle's boundary gap is below `band`; else the
    GPU set has k entries, contains every sure-in block and no sure-out block."""
    k = min(s, nc)
    sel_gpu = np.asarray(sel_gpu)
    assert np.all(sel_gpu[k:] == -1), sel_gpu
    got = sel_gpu[:k]
    assert np.all(np.diff(got) > 0), got
    assert np.all((got >= 0) & (got < nc)), got
    if k == 0:
        return True
    cand = np.asarray(sigma[:nc], dtype=np.float64)
    order = sorted(range(nc), key=lambda b: (-cand[b], b))
    want = np.sort(order[:k])
    kth = cand[order[k - 1]]
    nxt = cand[order[k]] if k < nc else -np.inf
    if kth - nxt >= band:
        assert np.array_equal(got, want), (got, want)
        return True
    sure_in = np.nonzero(cand >= kth + band)[0]
    sure_out = np.nonzero(cand <= nxt - band)[0]
    assert set(sure_in) <= set(got.tolist()), (sure_in, got)
    assert not (set(sure_out) & set(got.tolist())), (sure_out, got)
    return np.array_equal(got, want)


def rel_l2(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def valid_prefix(sel_row, nc):
    """Entries the library uses: the longest strictly ascending prefix of ids in [0, nc)."""
    out = []
    for x in np.asarray(sel_row).tolist():
        if x < 0 or x >= nc or (out and x <= out[-1]):
            break
        out.append(x)
    return out


def oracle_decode(q_unit, K_unit, V_unit, T, sel, cfg):
    U = M.union_tokens(T, cfg.block_size, cfg.window, sel)
    return M.sparse_attention(q_unit, K_unit, V_unit, U, cfg.scale)


def score_slack(q_unit, K_unit, T, sel, cfg):
    """Per query head, the largest error the bf16 score products allow in a
    score of the attended tokens, and so in the lse: the query reaches the
    matrix cores as two bf16 parts, each rounded to nearest at 2^-9 relative,
    so q_hi + q_lo is within 2^-18 |q_e| of every element, the bf16 products
    are exact in fp32, and a score c q.k moves by at most
    2^-18 c sum_e |q_e| |k_e|; taken at 2^-17 for margin."""
    U = M.union_tokens(T, cfg.block_size, cfg.window, sel)
    if len(U) == 0:
        return np.zeros(np.asarray(q_unit).shape[0])
    qa = np.abs(np.asarray(q_unit, dtype=np.float64))
    ka = np.abs(np.asarray(K_unit, dtype=np.float64)[U])
    return 2.0 ** -17 * cfg.scale * (qa @ ka.T).max(axis=1)


def check_out(out_gpu, lse_gpu, out_ora, lse_ora, kv_dtype, slack=None):
    """Attention against the oracle: relative L2 of out per head and over the
    heads; |lse diff| <= 1e-5 max(1, |lse|) plus, for bf16 K/V, `slack`
    (score_slack: the bf16 split of the query)."""
    tol = OUT_TOL[kv_dtype]
    if np.all(np.isneginf(lse_ora)):
        assert np.all(out_gpu == 0) and np.all(np.isneginf(lse_gpu))
        return
    for g in range(out_ora.shape[0]):
        e = rel_l2(out_gpu[g], out_ora[g])
        assert e <= tol, (g, e)
    assert rel_l2(out_gpu, out_ora) <= tol
    atol = LSE_TOL * max(1.0, float(np.max(np.abs(lse_ora))))
    extra = np.zeros(np.asarray(lse_ora).shape) if slack is None or kv_dtype != "bf16" else np.asarray(slack)
    err = np.abs(np.asarray(lse_gpu, dtype=np.float64) - np.asarray(lse_ora, dtype=np.float64))
    assert np.all(err <= atol + extra), (err, atol, extra)


def cuda(x):
    return x.to(DEV) if isinstance(x, torch.Tensor) else torch.as_tensor(x).to(DEV)


def qscale(cfg):
    return cfg.scale if cfg.softmax_scale == 0 else cfg.softmax_scale


def sync():
    torch.cuda.synchronize()


def unit_slices(cfg, b, h):
    G = cfg.num_q_heads // cfg.num_kv_heads
    return b, slice(h * G, (h + 1) * G)


def ky_fan_checks(xi, K, n, r, U=None):
    """Block statistics of the GPU (fp32 factors xi [r, d] of the n keys K) against
    the oracle: Ky-Fan energy, orthogonality and, where the eigengap allows,
    closeness of the rank-r covariance.  With a query basis U [d, s'] the
    factors are subspace factors [r, s'] of B_b = U^T Sigma_b U (Sec. 5.4)."""
    Sig = M.block_covariance(K)
    if U is not None:
        Sig = M.subspace_covariance(Sig, U)
    lam = np.sort(np.clip(np.linalg.eigvalsh(Sig), 0, None))[::-1]
    etop = lam[:r].sum()
    e = float((xi ** 2).sum())
    if etop <= 1e-12:
        assert np.all(xi == 0), "zero-variance block must store exact zeros"
        return
    assert (1 - 1e-3) * etop <= e <= (1 + 1e-5) * etop + 1e-6, (e, etop)
    nrm = np.linalg.norm(xi, axis=1)
    for i in range(r):
        for j in range(i + 1, r):
            if nrm[i] > 0 and nrm[j] > 0:
                assert abs(xi[i] @ xi[j]) <= 1e-4 * nrm[i] * nrm[j] + 1e-7
    if lam[r - 1] > 0 and (lam[r - 1] - lam[r]) / lam[r - 1] >= 0.05:
        ref = M.scaled_eigenvectors(Sig, r)
        A, Bm = xi.T @ xi, ref.T @ ref
        assert np.linalg.norm(A - Bm) <= 1e-3 * np.linalg.norm(Bm), np.linalg.norm(A - Bm) / np.linalg.norm(Bm)


def check_records(cfg, rec_unit, rec32_unit, K_unit, T, blocks=None, V_unit=None, U=None):
    """GPU block records of one unit against the oracle.

    rec32_unit: the unit's records built with fp32 mean and factors from the
    same keys; rec_unit: the configured storage.  Counts exact, means within
    fp32 rounding of the oracle's, zero factors for a partial block, Ky-Fan
    energy / orthogonality / rank-r subspace for full blocks, and the configured
    record byte-identical to the oracle's encoding of the fp32 statistics (the
    storage rounding of Sec. 5.5).  `blocks`: block indices to check (default all).
    U: the unit's query basis [d, s'] for subspace factors."""
    L, d, r = cfg.block_size, cfg.head_dim, cfg.rank
    nb = M.num_blocks(T, L)
    if nb == 0:
        return
    fdim = cfg.subspace_dim or None
    parts = R.decode(rec32_unit[:nb], d, r, "f32", "f32", cfg.skew, cfg.value_mean, fdim)
    counts, means, factors = parts[:3]
    skews, vmeans = (parts[3], parts[4]) if (cfg.skew or cfg.value_mean) else (None, None)
    K = np.asarray(K_unit, dtype=np.float64)
    blocks = range(nb) if blocks is None else [j for j in blocks if j < nb]
    for j in blocks:
        n = M.block_count(T, L, j)
        Kb = K[j * L:j * L + n]
        assert counts[j] == n, (j, counts[j], n)
        np.testing.assert_allclose(means[j], M.block_mean(Kb), rtol=0, atol=1e-6 * max(np.abs(Kb).max(), 1e-30))
        if n < L or r == 0:
            assert np.all(factors[j] == 0), j
        else:
            ky_fan_checks(factors[j], Kb, n, r, U)
        if skews is not None:
            Kp = Kb if U is None else Kb @ U
            np.testing.assert_allclose(skews[j], M.skew_coefficients(Kp, factors[j]), rtol=1e-4, atol=2e-4)
        if vmeans is not None and V_unit is not None:
            Vb = np.asarray(V_unit, dtype=np.float64)[j * L:j * L + n]
            np.testing.assert_allclose(vmeans[j], M.block_mean(Vb), rtol=0, atol=1e-6 * max(np.abs(Vb).max(), 1e-30))
    want = R.encode(counts, means, factors, cfg.mean_dtype, cfg.factor_dtype, skews, vmeans)
    got = np.asarray(rec_unit[:nb])
    for j in blocks:
        np.testing.assert_array_equal(got[j], want[j], err_msg=f"block {j}")


def subspace_sigma_bound(ell, qg, U, factors, skews, c):
    """Bound on |sigma_gpu - sigma_oracle| per block from the GPU's fp32
    arithmetic: l_b^g summed in fp32 (a few ulps of |l|), and each
    t = c xi . U^T q off by up to 1e-6 c |xi| |U^T q| (the projection and the
    dot product in fp32), which moves (1/2) sum t^2 by sum |t| dt and the skew
    term by sum |gamma| t^2 dt / 2; sigma_b takes the error of its own l_b^g
    and of the normaliser ln Z^g, a weighted mean over all blocks."""
    qf = qg @ U                                               # [G, s']
    t = c * np.einsum("brf,gf->bgr", factors, qf)
    dt = 1e-6 * c * np.linalg.norm(factors, axis=2)[:, None, :] * np.linalg.norm(qf, axis=1)[None, :, None]
    dl = 4e-7 * np.abs(ell) + (np.abs(t) * dt).sum(axis=2)
    if skews is not None:
        dl += (np.abs(skews)[:, None, :] * t * t * dt).sum(axis=2) / 2
    return SIGMA_TOL + dl.max(axis=1) + dl.max()


def f32_config(cfg):
    """The same problem with fp32 mean and factor storage."""
    import dataclasses
    return dataclasses.replace(cfg, mean_dtype="f32", factor_dtype="f32")


def block_statistics_gpu(cfg, k, v, seq_lens):
    rec = cobs.new_summaries(cfg, DEV)
    cobs.cobs_build_block_stats(cfg, k, v, seq_lens, rec)
    return rec


__all__ = [n for n in dir() if not n.startswith("_")] + ["math"]

"""Optional record parts on the GPU against the oracle: the diagonal skew
coefficients of Sec. 7.7 and the block value means, the skew term in the
selector, the decode step with both, and the mean-pool compression branch
(Sec. 2, Sec. 5.2).  Shared-bytes rule as elsewhere: the oracle scores and
attends over the records the GPU built."""

import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle import method as M
from oracle import records as R
from paper_2607_09052_amd import cobs
from tests.gpu_util import (DEV, LSE_TOL, SIGMA_TOL, check_selection, f64, ky_fan_checks, rel_l2, say,
                            sync)

pytestmark = pytest.mark.gpu


def _problem(d, kv, T, seed, B=2, Hkv=2, G=4):
    prob = synth.make_problem("c5", seed=seed, B=B, Hq=G * Hkv, Hkv=Hkv, d=d, T=T, steps=0, kv_dtype=kv)
    return prob


def _cfg(d, r, kv, md, fd, T, G=4, B=2, Hkv=2, s=8, w=128, **kw):
    return cobs.Config(batch=B, num_q_heads=G * Hkv, num_kv_heads=Hkv, head_dim=d, max_seq_len=T, rank=r,
                       budget=s, window=w, kv_dtype=kv, mean_dtype=md, factor_dtype=fd, **kw)


BUILD_CASES = [
    # d, r, K/V, mean, factor
    (128, 4, "f32", "f32", "f32"),
    (128, 4, "bf16", "bf16", "e2m1"),
    (64, 2, "bf16", "e2m1", "e2m1"),
    (128, 6, "bf16", "f32", "bf16"),
]


@pytest.mark.parametrize("d,r,kv,md,fd", BUILD_CASES)
def test_build_with_skew_and_value_means(d, r, kv, md, fd):
    """Records with both optional parts: the plain parts byte-identical to a
    plain build; the value means within fp32 rounding of the oracle's; the skew
    coefficients equal to the oracle's on the GPU's own fp32 factors; every
    stored part the oracle's storage encoding of the GPU's fp32 statistics."""
    T = 1024
    prob = _problem(d, kv, T, seed=400 + d + r)
    k, v = prob["k"].to(DEV), prob["v"].to(DEV)
    seq = torch.tensor([T, 700], dtype=torch.int32, device=DEV)
    plain = _cfg(d, r, kv, md, fd, T)
    opt = dataclasses.replace(plain, skew=True, value_mean=True)
    opt32 = dataclasses.replace(opt, mean_dtype="f32", factor_dtype="f32")
    recs = {}
    for name, c in (("plain", plain), ("opt", opt), ("opt32", opt32)):
        recs[name] = cobs.new_summaries(c, DEV)
        say(f"build with options: {name} d={d} r={r} {kv} {c.mean_dtype}/{c.factor_dtype}")
        cobs.cobs_build_block_stats(c, k, v, seq, recs[name])
    sync()
    lp, lo = R.layout(d, r, md, fd), R.layout(d, r, md, fd, True, True)
    for b, Tb in enumerate([T, 700]):
        nb = -(-Tb // 64)
        for h in range(2):
            po, pp = recs["opt"][b, h, :nb].cpu().numpy(), recs["plain"][b, h, :nb].cpu().numpy()
            np.testing.assert_array_equal(po[:, 0:4], pp[:, 0:4])
            np.testing.assert_array_equal(po[:, 16:16 + (lp["mean_off"] - 16)], pp[:, 16:lp["mean_off"]])
            np.testing.assert_array_equal(po[:, lo["mean_off"]:lo["vmean_off"]], pp[:, lp["mean_off"]:lp["fac_off"] + r * lp["vec_bytes"]])
            cnt, mns, fac, skw, vmn = R.decode(recs["opt32"][b, h, :nb].cpu().numpy(), d, r, "f32", "f32", True, True)
            Kh, Vh = f64(prob["k"][b, h, :Tb]), f64(prob["v"][b, h, :Tb])
            for j in range(nb):
                n = min(64, Tb - 64 * j)
                Kb, Vb = Kh[64 * j:64 * j + n], Vh[64 * j:64 * j + n]
                np.testing.assert_allclose(vmn[j], M.block_mean(Vb), rtol=0, atol=1e-6 * np.abs(Vb).max())
                if n < 64:
                    assert np.all(skw[j] == 0) and np.all(fac[j] == 0)
                    continue
                ky_fan_checks(fac[j], Kb, n, r)
                want = M.skew_coefficients(Kb, fac[j])
                np.testing.assert_allclose(skw[j], want, rtol=1e-4, atol=2e-4)
            # stored parts: the oracle's encoding of the fp32 statistics
            enc = R.encode(cnt, mns, fac, md, fd, skw, vmn)
            np.testing.assert_array_equal(po, enc)


SELECT_CASES = [
    # d, G, r, K/V, mean, factor
    (128, 4, 4, "bf16", "f32", "f32"),
    (128, 8, 4, "bf16", "bf16", "e2m1"),
    (128, 4, 6, "bf16", "e2m1", "e2m1"),
    (64, 2, 2, "f32", "f32", "bf16"),
    (128, 16, 12, "bf16", "f32", "f32"),
]


@pytest.mark.parametrize("d,G,r,kv,md,fd", SELECT_CASES)
def test_select_with_skew_term_matches_oracle(d, G, r, kv, md, fd):
    """The skew term of Sec. 7.7 in the selector, on the GPU's own records:
    |sigma| within 2e-5 of the oracle's third-order scores and the set rule."""
    T, B, Hkv, s, w = 2048, 3, 2, 12, 200
    prob = _problem(d, kv, T, seed=500 + G + r, B=B, Hkv=Hkv, G=G)
    cfg = _cfg(d, r, kv, md, fd, T, G=G, B=B, Hkv=Hkv, s=s, w=w, skew=True)
    k, v, q = prob["k"].to(DEV), prob["v"].to(DEV), prob["q"].to(DEV)
    lens = [T, 1500, 333]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    rec = cobs.new_summaries(cfg, DEV)
    say(f"select with skew d={d} G={G} r={r} {md}/{fd}")
    cobs.cobs_build_block_stats(cfg, k, v, seq, rec)
    sel = torch.empty((B, Hkv, s), dtype=torch.int32, device=DEV)
    scores = torch.empty((B, Hkv, cfg.num_blocks), dtype=torch.float32, device=DEV)
    cobs.cobs_select(cfg, q, rec, seq, sel, cobs.new_workspace(cfg, cobs.OP_SELECT, DEV), scores=scores)
    sync()
    moved = 0.0
    for b, Tb in enumerate(lens):
        nb = -(-Tb // 64)
        for h in range(Hkv):
            cnt, mns, fac, skw, _ = R.decode(rec[b, h, :nb].cpu().numpy(), d, r, md, fd, True, False)
            qg = f64(prob["q"][b, h * G:(h + 1) * G])
            ell = M.log_mass_estimate(qg, cnt, mns, fac, cfg.scale, skw)
            sigma = M.group_scores(ell)
            nc = M.candidate_count(Tb, 64, w)
            got = scores[b, h].cpu().numpy()
            assert np.all(np.abs(got[:nc] - sigma[:nc]) <= SIGMA_TOL), np.max(np.abs(got[:nc] - sigma[:nc]))
            assert np.all(np.isneginf(got[nc:]))
            check_selection(sel[b, h].cpu().numpy(), sigma, nc, s)
            # the term is really there: the second-order scores differ
            s2 = M.group_scores(M.log_mass_estimate(qg, cnt, mns, fac, cfg.scale))
            moved = max(moved, float(np.max(np.abs(s2[:nc] - sigma[:nc]))) if nc else 0.0)
    assert moved > 1e-3, moved


@pytest.mark.parametrize("t0,rank", [(3000, 4), (3008, 4), (3008, 6)])
def test_decode_step_with_options_is_build_select_decode(t0, rank):
    """With skew coefficients and value means in the records, the step's
    refresh of the newest block writes both, and the step equals the three
    entry points bitwise."""
    d, kv, G, Hkv = 128, "bf16", 4, 4
    prob = synth.make_problem("c3", seed=37, B=2, Hq=G * Hkv, Hkv=Hkv, T=3000, s=10, w=300, kv_dtype=kv)
    cfg = cobs.Config(batch=2, num_q_heads=G * Hkv, num_kv_heads=Hkv, head_dim=d, max_seq_len=3008, rank=rank,
                      budget=10, window=300, kv_dtype=kv, mean_dtype="bf16", factor_dtype="e2m1",
                      skew=True, value_mean=True)
    k, v, q = prob["k"].to(DEV), prob["v"].to(DEV), prob["q"].to(DEV)
    lens = [t0, 2049]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    rec0 = cobs.new_summaries(cfg, DEV)
    say(f"step with options: T={t0} r={rank}")
    cobs.cobs_build_block_stats(cfg, k, v, seq, rec0)
    rec1 = rec0.clone()
    for b, T in enumerate(lens):
        rec1[b, :, (T - 1) // 64] = 0
    out1 = torch.empty((2, G * Hkv, d), dtype=torch.float32, device=DEV)
    lse1 = torch.empty((2, G * Hkv), dtype=torch.float32, device=DEV)
    sel1 = torch.empty((2, Hkv, 10), dtype=torch.int32, device=DEV)
    cobs.cobs_decode_step(cfg, q, k, v, seq, rec1, out1, cobs.new_workspace(cfg, cobs.OP_STEP, DEV), sel=sel1,
                          lse=lse1)
    sel2, out2, lse2 = torch.empty_like(sel1), torch.empty_like(out1), torch.empty_like(lse1)
    cobs.cobs_select(cfg, q, rec0, seq, sel2, cobs.new_workspace(cfg, cobs.OP_SELECT, DEV))
    cobs.cobs_sparse_decode(cfg, q, k, v, seq, sel2, out2, cobs.new_workspace(cfg, cobs.OP_DECODE, DEV), lse=lse2)
    sync()
    assert torch.equal(rec1, rec0)
    assert torch.equal(sel1, sel2) and torch.equal(out1, out2) and torch.equal(lse1, lse2)


COMPRESS_CASES = [
    # d, G, K/V, mean dtype
    (128, 4, "bf16", "f32"),
    (128, 8, "bf16", "bf16"),
    (128, 16, "bf16", "e2m1"),
    (64, 1, "f32", "f32"),
    (64, 2, "bf16", "e2m1"),
]


@pytest.mark.parametrize("d,G,kv,md", COMPRESS_CASES)
def test_compression_branch_matches_oracle(d, G, kv, md):
    """Attention over the pooled (mean key, mean value) blocks of the GPU's
    records against the oracle's compression_attention on the same bytes,
    rows of several lengths including an empty one."""
    T, B, Hkv = 4096, 4, 2
    prob = _problem(d, kv, T, seed=600 + G, B=B, Hkv=Hkv, G=G)
    cfg = _cfg(d, 4, kv, md, "e2m1", T, G=G, B=B, Hkv=Hkv, value_mean=True)
    k, v, q = prob["k"].to(DEV), prob["v"].to(DEV), prob["q"].to(DEV)
    lens = [T, 2500, 63, 0]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    rec = cobs.new_summaries(cfg, DEV)
    say(f"compression branch d={d} G={G} {kv} mean {md}")
    cobs.cobs_build_block_stats(cfg, k, v, seq, rec)
    out = torch.full((B, G * Hkv, d), 7.0, dtype=torch.float32, device=DEV)
    lse = torch.full((B, G * Hkv), 7.0, dtype=torch.float32, device=DEV)
    cobs.cobs_compression_branch(cfg, q, rec, seq, out, lse)
    sync()
    for b, Tb in enumerate(lens):
        nb = -(-Tb // 64)
        for h in range(Hkv):
            gs = slice(h * G, (h + 1) * G)
            got_o, got_l = out[b, gs].cpu().numpy(), lse[b, gs].cpu().numpy()
            if nb == 0:
                assert np.all(got_o == 0) and np.all(np.isneginf(got_l))
                continue
            cnt, mns, _, _, vmn = R.decode(rec[b, h, :nb].cpu().numpy(), d, 4, md, "e2m1", False, True)
            o, l = M.compression_attention(f64(prob["q"][b, gs]), cnt, mns, vmn, cfg.scale)
            for g in range(G):
                assert rel_l2(got_o[g], o[g]) <= 1e-5, (b, h, g, rel_l2(got_o[g], o[g]))
            np.testing.assert_allclose(got_l, l, rtol=0, atol=LSE_TOL * max(1.0, float(np.max(np.abs(l)))))

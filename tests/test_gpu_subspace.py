"""Subspace factors (Sec. 5.4) on the GPU against the oracle.

The query basis U_Q of each KV head is the oracle's estimate (top eigenvectors
of the second moment of a calibration sample of the group's queries, drawn from
the subspace query law); both sides take it as an input.  The build is checked
on fp32 records through the invariants of the eigenproblem of
B_b = U_Q^T Sigma_b U_Q, the stored records against the oracle's storage
encoding of the GPU's fp32 statistics; the selector on the GPU's own record
bytes (sigma within 2e-5 of the oracle's subspace scores, the set rule); the
decode step bitwise against build + select + decode.
"""

import numpy as np
import pytest
import torch

import synth
from oracle import method as M
from oracle import records as R
from paper_2607_09052_amd import cobs
from tests.gpu_util import (DEV, check_records, check_selection, f32_config, f64, oracle_select, say,
                            subspace_sigma_bound, sync)

pytestmark = pytest.mark.gpu


def _basis(Hkv, d, sd, G, seed):
    """U_Q per KV head [Hkv, d, sd] (oracle estimate from 512 query rows) and
    the rotation of the query law."""
    rot, sig = synth.query_rotation(Hkv, d, seed)
    cal = synth.subspace_queries(rot, sig, 512, G, seed + 1)
    U = np.stack([M.query_subspace(f64(cal[:, h * G:(h + 1) * G].reshape(-1, d)), sd) for h in range(Hkv)])
    return U, rot, sig


def _cfg(d, sd, L, kv, r, md, fd, T, basis, G=4, B=2, Hkv=2, s=8, w=128, **kw):
    return cobs.Config(batch=B, num_q_heads=G * Hkv, num_kv_heads=Hkv, head_dim=d, max_seq_len=T, rank=r,
                       budget=s, window=w, kv_dtype=kv, mean_dtype=md, factor_dtype=fd, block_size=L,
                       subspace_dim=sd, query_basis=basis, **kw)


BUILD_CASES = [
    # d, s', L, K/V, r, mean, factor, skew, key law, value means
    (128, 96, 64, "bf16", 4, "bf16", "e2m1", False, "c4", False),
    (128, 32, 32, "f32", 2, "e2m1", "bf16", True, "c5", False),
    (64, 32, 128, "bf16", 4, "bf16", "bf16", False, "c5", False),
    (128, 64, 128, "bf16", 3, "e2m1", "e2m1", True, "c3", False),
    (128, 96, 64, "f32", 1, "bf16", "e2m1", True, "c2", False),
    (128, 64, 64, "bf16", 4, "e2m1", "e2m1", True, "c4", True),
    (128, 64, 32, "bf16", 3, "bf16", "bf16", False, "c3", True),
    (64, 32, 64, "bf16", 2, "f32", "e2m1", False, "c5", True),
]


@pytest.mark.parametrize("d,sd,L,kv,r,md,fd,skew,law,vm", BUILD_CASES)
def test_subspace_build_matches_oracle(d, sd, L, kv, r, md, fd, skew, law, vm):
    T, B, Hkv, G = 2048, 2, 2, 4
    U, _, _ = _basis(Hkv, d, sd, G, seed=700 + sd + L)
    basis = torch.from_numpy(U.astype(np.float32)).contiguous().to(DEV)
    prob = synth.make_problem(law, seed=710 + d + L, B=B, Hq=G * Hkv, Hkv=Hkv, d=d, T=T, L=L, steps=0,
                              kv_dtype=kv)
    k, v = prob["k"].to(DEV), prob["v"].to(DEV)
    lens = [T, T - L - 5]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    cfg = _cfg(d, sd, L, kv, r, md, fd, T, basis, G=G, B=B, Hkv=Hkv, skew=skew, value_mean=vm)
    cfg32 = f32_config(cfg)
    rec, rec32 = cobs.new_summaries(cfg, DEV), cobs.new_summaries(cfg32, DEV)
    say(f"subspace build d={d} s'={sd} L={L} {kv} r={r} {md}/{fd} skew={skew} law={law} value means={vm}")
    cobs.cobs_build_block_stats(cfg, k, v, seq, rec)
    cobs.cobs_build_block_stats(cfg32, k, v, seq, rec32)
    sync()
    for b, Tb in enumerate(lens):
        for h in range(Hkv):
            check_records(cfg, rec[b, h].cpu().numpy(), rec32[b, h].cpu().numpy(), f64(prob["k"][b, h]), Tb,
                          V_unit=f64(prob["v"][b, h]) if vm else None, U=U[h])


SELECT_CASES = [
    # d, s', G, L, mean, factor, skew, subspace-law queries
    (128, 96, 4, 64, "bf16", "e2m1", False, True),
    (128, 96, 8, 64, "e2m1", "e2m1", True, True),
    (128, 32, 16, 32, "bf16", "bf16", False, False),
    (128, 64, 1, 128, "e2m1", "bf16", False, True),
    (64, 32, 2, 64, "bf16", "e2m1", True, True),
]


@pytest.mark.parametrize("d,sd,G,L,md,fd,skew,ssq", SELECT_CASES)
def test_subspace_select_matches_oracle(d, sd, G, L, md, fd, skew, ssq):
    """The selector on subspace records: the curvature term meets U_Q^T q,
    the mean term the full q; rows of several lengths, one empty."""
    T, B, Hkv, s, w, r = 4096, 4, 2, 12, 256, 4
    U, rot, sig = _basis(Hkv, d, sd, G, seed=800 + sd + G)
    basis = torch.from_numpy(U.astype(np.float32)).contiguous().to(DEV)
    prob = synth.make_problem("c4", seed=810 + G, B=B, Hq=G * Hkv, Hkv=Hkv, d=d, T=T, L=L, steps=0)
    q = synth.subspace_queries(rot, sig, B, G, seed=820 + G) if ssq else prob["q"]
    q = (q * 2.0).contiguous()           # a curvature term of the size of the mean term
    cfg = _cfg(d, sd, L, "bf16", r, md, fd, T, basis, G=G, B=B, Hkv=Hkv, s=s, w=w, skew=skew)
    k, v = prob["k"].to(DEV), prob["v"].to(DEV)
    lens = [T, 3000, 900, 0]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    rec = cobs.new_summaries(cfg, DEV)
    say(f"subspace select d={d} s'={sd} G={G} L={L} {md}/{fd} skew={skew}")
    cobs.cobs_build_block_stats(cfg, k, v, seq, rec)
    sel = torch.empty((B, Hkv, s), dtype=torch.int32, device=DEV)
    scores = torch.empty((B, Hkv, cfg.num_blocks), dtype=torch.float32, device=DEV)
    cobs.cobs_select(cfg, q.to(DEV), rec, seq, sel, cobs.new_workspace(cfg, cobs.OP_SELECT, DEV), scores=scores)
    sync()
    moved = 0.0
    for b, Tb in enumerate(lens):
        for h in range(Hkv):
            qg = f64(q[b, h * G:(h + 1) * G])
            sigma, nc, _ = oracle_select(rec[b, h].cpu().numpy(), qg, Tb, cfg, U[h])
            got = scores[b, h].cpu().numpy()
            assert np.all(np.isneginf(got[nc:]))
            check_selection(sel[b, h].cpu().numpy(), sigma, nc, s)
            if not nc:
                continue
            nb = M.num_blocks(Tb, L)
            parts = R.decode(rec[b, h, :nb].cpu().numpy(), d, r, md, fd, skew, False, sd)
            ell = M.log_mass_estimate(qg, parts[0], parts[1], parts[2], cfg.scale, parts[3] if skew else None, U[h])
            tol = subspace_sigma_bound(ell, qg, U[h], parts[2], parts[3] if skew else None, cfg.scale)[:nc]
            err = np.abs(got[:nc] - sigma[:nc])
            assert np.all(err <= tol), float((err - tol).max())
            # the curvature term moves the scores: the first-order scores differ
            first = M.group_scores(M.log_mass_estimate(qg, parts[0], parts[1], parts[2][:, :0], cfg.scale))
            moved = max(moved, float(np.max(np.abs(first[:nc] - sigma[:nc]))))
    assert moved > 1e-2, moved


STEP_CASES = [
    # L, newest length, s', K/V, skew, value means
    (64, 3000, 96, "bf16", False, False),
    (64, 3008, 96, "bf16", False, False),
    (32, 2999, 96, "bf16", False, False),
    (64, 2999, 64, "bf16", True, True),
    (32, 3008, 64, "bf16", False, True),
    (64, 3001, 32, "f32", True, False),
    (32, 2976, 32, "f32", False, True),
]


@pytest.mark.parametrize("L,t0,sd,kv,skew,vm", STEP_CASES)
def test_subspace_decode_step_is_build_select_decode(L, t0, sd, kv, skew, vm):
    """The step with subspace factors (build of the newest block, query
    projection, selection, attention) equals the separate calls bitwise, for a
    partial or a full newest block."""
    d, G, Hkv, B, s, w = 128, 4, 4, 2, 10, 300
    U, rot, sig = _basis(Hkv, d, sd, G, seed=900 + L + sd)
    basis = torch.from_numpy(U.astype(np.float32)).contiguous().to(DEV)
    prob = synth.make_problem("c3", seed=910 + L, B=B, Hq=G * Hkv, Hkv=Hkv, T=3000, s=s, w=w, L=L)
    T_max = 3008
    cfg = _cfg(d, sd, L, kv, 4, "bf16", "e2m1", T_max, basis, G=G, B=B, Hkv=Hkv, s=s, w=w, skew=skew,
               value_mean=vm)
    dt = torch.bfloat16 if kv == "bf16" else torch.float32
    k = torch.zeros((B, Hkv, T_max, d), dtype=dt)
    v = torch.zeros_like(k)
    k[:, :, :3000], v[:, :, :3000] = prob["k"][:, :, :3000].to(dt), prob["v"][:, :, :3000].to(dt)
    k, v = k.to(DEV), v.to(DEV)
    q = synth.subspace_queries(rot, sig, B, G, seed=920).to(DEV)
    lens = [t0, 2049]
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    rec0 = cobs.new_summaries(cfg, DEV)
    say(f"subspace step L={L} T={t0} s'={sd} {kv} skew={skew} value means={vm}")
    cobs.cobs_build_block_stats(cfg, k, v, seq, rec0)
    rec1 = rec0.clone()
    for b, T in enumerate(lens):
        rec1[b, :, (T - 1) // L] = 0
    out1 = torch.empty((B, G * Hkv, d), dtype=torch.float32, device=DEV)
    lse1 = torch.empty((B, G * Hkv), dtype=torch.float32, device=DEV)
    sel1 = torch.empty((B, Hkv, s), dtype=torch.int32, device=DEV)
    cobs.cobs_decode_step(cfg, q, k, v, seq, rec1, out1, cobs.new_workspace(cfg, cobs.OP_STEP, DEV), sel=sel1,
                          lse=lse1)
    sel2, out2, lse2 = torch.empty_like(sel1), torch.empty_like(out1), torch.empty_like(lse1)
    cobs.cobs_select(cfg, q, rec0, seq, sel2, cobs.new_workspace(cfg, cobs.OP_SELECT, DEV))
    cobs.cobs_sparse_decode(cfg, q, k, v, seq, sel2, out2, cobs.new_workspace(cfg, cobs.OP_DECODE, DEV), lse=lse2)
    sync()
    assert torch.equal(rec1, rec0)
    assert torch.equal(sel1, sel2) and torch.equal(out1, out2) and torch.equal(lse1, lse2)

"""Randomised GPU parity: seeded draws over the configuration space (batch,
heads, group size, head dim, rank, budget, window, descriptor and K/V types,
ragged lengths including T < L and T <= w), each checked end to end against the
oracle: the selector on the GPU's own records, the attention on the GPU's
selection, and the decode step against the three entry points.  A second draw
takes contexts of up to 64k tokens (many selector chunks and decode workgroups
per unit), a third checks the exact-mass and Quest selectors and the two-branch
decode, and a fourth checks that a paged cache is bitwise the contiguous one.
A fifth puts rows of length 0 beside the others, a sixth draws subspace
factors (Sec. 5.4).  COBS_RANDOM_SEEDS sets the number of seeds of each draw
(default 24, 6, 8, 6, 6 and 8) for a longer sweep."""

import os

import numpy as np
import pytest
import torch

import synth
from oracle import method as M
from oracle import records as R
from paper_2607_09052_amd import cobs
from tests.gpu_util import (DEV, SIGMA_TOL, check_out, check_records, check_selection, f32_config, f64,
                            oracle_decode, oracle_select, say, score_slack, subspace_sigma_bound, sync)

pytestmark = pytest.mark.gpu

DTYPES = ["f32", "bf16", "e2m1"]


def _draw(seed):
    rng = np.random.default_rng(seed)
    G = int(rng.choice([1, 2, 4, 8, 16]))
    d = int(rng.choice([64, 128]))
    Hkv = int(rng.integers(1, 4))
    B = int(rng.integers(1, 5))
    tmax = 64 * int(rng.integers(4, 40))
    kv = "f32" if rng.random() < 0.25 else "bf16"
    md, fd = DTYPES[int(rng.integers(3))], DTYPES[int(rng.integers(3))]
    r = int(rng.integers(0, 7))
    s = int(rng.integers(0, 21))
    w = int(rng.choice([0, 64, int(rng.integers(1, 600))]))
    seq = rng.integers(1, tmax + 1, size=B).astype(np.int32)
    seq[0] = tmax
    if B > 1:
        seq[1] = int(rng.integers(1, 64))           # a row shorter than one block
    # optional record parts (skew coefficients, value means) and the block
    # length, drawn last so the other draws of a seed are unchanged; T_max is
    # rounded up to whole blocks
    skew, vmean = bool(rng.random() < 0.3), bool(rng.random() < 0.3)
    L = int(rng.choice([32, 64, 64, 128]))
    tmax = -(-tmax // L) * L
    seq[0] = tmax
    return dict(G=G, d=d, Hkv=Hkv, B=B, tmax=tmax, kv=kv, md=md, fd=fd, r=r, s=s, w=w, seq=seq,
                skew=skew, vmean=vmean, L=L)


def _draw_long(seed):
    """As _draw, with T_max up to 1024 blocks, budgets up to 119 and windows up to 3000."""
    c = _draw(seed)
    rng = np.random.default_rng(seed + 777)
    tmax = c["L"] * int(rng.integers(40, 1025) * 64 // c["L"])
    seq = rng.integers(1, tmax + 1, size=c["B"]).astype(np.int32)
    seq[0] = tmax
    if c["B"] > 1:
        seq[1] = int(rng.integers(1, 64))
    c.update(tmax=tmax, seq=seq, s=int(rng.integers(0, 120)),
             w=int(rng.choice([0, 512, 1024, int(rng.integers(1, 3000))])))
    return c


_N = os.environ.get("COBS_RANDOM_SEEDS")


@pytest.mark.parametrize("seed", list(range(int(_N) if _N else 24)))
def test_random_configuration_end_to_end(seed):
    _check(_draw(1000 + seed), 2000 + seed, f"random config {seed}")


@pytest.mark.parametrize("seed", list(range(int(_N) if _N else 6)))
def test_random_long_context_end_to_end(seed):
    _check(_draw_long(3000 + seed), 4000 + seed, f"random long-context config {seed}")


@pytest.mark.parametrize("seed", list(range(int(_N) if _N else 6)))
def test_random_configuration_with_empty_rows(seed):
    """Rows of length 0 beside full and ragged ones: no candidates, all -1
    selections, scores -inf, out 0 and lse -inf for the empty rows, no record
    written for them, and the other rows unaffected.  A length above T_max
    counts as T_max and a negative one as 0."""
    c = _draw(11000 + seed)
    rng = np.random.default_rng(12000 + seed)
    B = max(c["B"], 4)
    seq = rng.integers(0, c["tmax"] + 1, size=B).astype(np.int32)
    seq[0], seq[1] = c["tmax"], 0
    seq[2] = c["tmax"] + int(rng.integers(1, 500))
    seq[3] = -int(rng.integers(1, 100))
    c.update(B=B, seq=seq)
    _check(c, 13000 + seed, f"random config with empty rows {seed}")


@pytest.mark.parametrize("seed", list(range(int(_N) if _N else 8)))
def test_random_subspace_end_to_end(seed):
    """Subspace factors: s' in {32, 64, 96} below d, U_Q the oracle's estimate
    from a calibration sample of the subspace query law, queries of that law
    (or i.i.d. Gaussian), bf16 / E2M1 descriptors, r in [1, 4]."""
    c = _draw(14000 + seed)
    rng = np.random.default_rng(15000 + seed)
    c.update(md=["bf16", "e2m1"][int(rng.integers(2))], fd=["bf16", "e2m1"][int(rng.integers(2))],
             r=int(rng.integers(1, 5)), sd=int(rng.choice([32, 64, 96] if c["d"] == 128 else [32])),
             ssq=bool(rng.random() < 0.7))
    _check(c, 16000 + seed, f"random subspace config {seed}")


def _check(c, data_seed, tag):
    G, d, Hkv, B, tmax = c["G"], c["d"], c["Hkv"], c["B"], c["tmax"]
    say(f"{tag}: {c}")
    L = c.get("L", 64)
    prob = synth.make_problem("c2", seed=data_seed, B=B, Hq=G * Hkv, Hkv=Hkv, d=d, T=tmax, kv_dtype=c["kv"], L=L)
    sub, U = {}, None
    if c.get("sd"):
        # U_Q per KV head: the oracle's estimate from 256 rows of the subspace law
        rot, sig = synth.query_rotation(Hkv, d, data_seed + 1)
        cal = synth.subspace_queries(rot, sig, 256, G, data_seed + 2)
        U = np.stack([M.query_subspace(f64(cal[:, h * G:(h + 1) * G].reshape(-1, d)), c["sd"]) for h in range(Hkv)])
        sub = dict(subspace_dim=c["sd"], query_basis=torch.from_numpy(U.astype(np.float32)).to(DEV))
        if c["ssq"]:
            prob["q"] = synth.subspace_queries(rot, sig, B, G, data_seed + 3)
    cfg = cobs.Config(batch=B, num_q_heads=G * Hkv, num_kv_heads=Hkv, head_dim=d, max_seq_len=tmax,
                      rank=c["r"], budget=c["s"], window=c["w"], kv_dtype=c["kv"], mean_dtype=c["md"],
                      factor_dtype=c["fd"], skew=c.get("skew", False), value_mean=c.get("vmean", False),
                      block_size=L, **sub)
    q, k, v = prob["q"], prob["k"], prob["v"]
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    seq_d = torch.from_numpy(c["seq"]).to(DEV)
    rec = cobs.new_summaries(cfg, DEV)
    cobs.cobs_build_block_stats(cfg, kd, vd, seq_d, rec)
    cfg32 = f32_config(cfg)
    rec32 = cobs.new_summaries(cfg32, DEV)
    cobs.cobs_build_block_stats(cfg32, kd, vd, seq_d, rec32)
    s_alloc = max(c["s"], 1)
    sel = torch.full((B, Hkv, s_alloc), -7, dtype=torch.int32, device=DEV)
    scores = torch.empty((B, Hkv, cfg.num_blocks), dtype=torch.float32, device=DEV)
    cobs.cobs_select(cfg, qd, rec, seq_d, sel, cobs.new_workspace(cfg, cobs.OP_SELECT, DEV), scores=scores)
    out = torch.empty((B, G * Hkv, d), dtype=torch.float32, device=DEV)
    lse = torch.empty((B, G * Hkv), dtype=torch.float32, device=DEV)
    sel_c = sel[:, :, :c["s"]].contiguous()
    cobs.cobs_sparse_decode(cfg, qd, kd, vd, seq_d, sel_c, out, cobs.new_workspace(cfg, cobs.OP_DECODE, DEV),
                            lse=lse)
    # the step on a copy whose newest-block records are stale
    rec1 = rec.clone()
    seq_c = np.clip(c["seq"], 0, tmax)                 # lengths as the library reads them
    for b in range(B):
        if int(seq_c[b]) > 0:
            rec1[b, :, (int(seq_c[b]) - 1) // L] = 0
    sel1 = torch.empty_like(sel_c)
    out1, lse1 = torch.empty_like(out), torch.empty_like(lse)
    cobs.cobs_decode_step(cfg, qd, kd, vd, seq_d, rec1, out1, cobs.new_workspace(cfg, cobs.OP_STEP, DEV),
                          sel=sel1 if c["s"] > 0 else None, lse=lse1)
    if cfg.value_mean:
        out_c, lse_c = torch.empty_like(out), torch.empty_like(lse)
        cobs.cobs_compression_branch(cfg, qd, rec, seq_d, out_c, lse_c)
    sync()
    rec_h, sc_h, rec32_h = rec.cpu().numpy(), scores.cpu().numpy(), rec32.cpu().numpy()
    sel_h, out_h, lse_h = sel_c.cpu().numpy(), out.cpu().numpy(), lse.cpu().numpy()
    for b in range(B):
        T = int(seq_c[b])
        nb = -(-T // L)
        # block statistics of this row: every block of short contexts, else a
        # stride of them plus the last two
        blocks = None if nb <= 64 else sorted(set(range(0, nb, nb // 32)) | {nb - 2, nb - 1})
        for h in range(Hkv):
            gs = slice(h * G, (h + 1) * G)
            Uh = None if U is None else U[h]
            check_records(cfg, rec_h[b, h], rec32_h[b, h], f64(k[b, h]), T, blocks, f64(v[b, h]), Uh)
            sigma, nc, _ = oracle_select(rec_h[b, h], q[b, gs].double().numpy(), T, cfg, Uh)
            tol = SIGMA_TOL
            if Uh is not None and nc:
                parts = R.decode(rec_h[b, h, :nb], d, cfg.rank, c["md"], c["fd"], cfg.skew, cfg.value_mean, c["sd"])
                qg = q[b, gs].double().numpy()
                ell = M.log_mass_estimate(qg, parts[0], parts[1], parts[2], cfg.scale,
                                          parts[3] if cfg.skew else None, Uh)
                tol = subspace_sigma_bound(ell, qg, Uh, parts[2], parts[3] if cfg.skew else None, cfg.scale)[:nc]
            assert np.all(np.abs(sc_h[b, h, :nc] - sigma[:nc]) <= tol)
            assert np.all(np.isneginf(sc_h[b, h, nc:]))
            if c["s"] > 0:
                check_selection(sel_h[b, h], sigma, nc, c["s"])
            o, l = oracle_decode(q[b, gs].double().numpy(), f64(k[b, h]), f64(v[b, h]), T, sel_h[b, h], cfg)
            check_out(out_h[b, gs], lse_h[b, gs], o, l, c["kv"],
                      score_slack(q[b, gs].double().numpy(), f64(k[b, h]), T, sel_h[b, h], cfg))
            if cfg.value_mean:
                nb = -(-T // L)
                parts = R.decode(rec_h[b, h, :nb], d, cfg.rank, c["md"], c["fd"], cfg.skew, True, c.get("sd") or None)
                o, l = M.compression_attention(q[b, gs].double().numpy(), parts[0], parts[1], parts[4], cfg.scale)
                check_out(out_c[b, gs].cpu().numpy(), lse_c[b, gs].cpu().numpy(), o, l, "f32")
    assert torch.equal(rec1, rec)
    if c["s"] > 0:
        assert torch.equal(sel1, sel_c)
    assert torch.equal(out1, out) and torch.equal(lse1, lse)


@pytest.mark.parametrize("seed", list(range(int(_N) if _N else 8)))
def test_random_diagnostic_entry_points(seed):
    """The exact-mass and Quest selectors and the two-branch decode on random
    bf16-cache draws: scores and selections against the oracle's, each branch
    against the oracle's attention on its own token set (on the exact-mass
    selection the GPU made)."""
    c = _draw(5000 + seed)
    c["kv"] = "bf16"
    G, d, Hkv, B, tmax, s, w = c["G"], c["d"], c["Hkv"], c["B"], c["tmax"], c["s"], c["w"]
    say(f"random diagnostic config {seed}: {c}")
    L = c["L"]
    prob = synth.make_problem("c2", seed=6000 + seed, B=B, Hq=G * Hkv, Hkv=Hkv, d=d, T=tmax, kv_dtype="bf16", L=L)
    cfg = cobs.Config(batch=B, num_q_heads=G * Hkv, num_kv_heads=Hkv, head_dim=d, max_seq_len=tmax,
                      rank=c["r"], budget=s, window=w, kv_dtype="bf16", block_size=L)
    q, k, v = prob["q"], prob["k"], prob["v"]
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    seq_d = torch.from_numpy(c["seq"]).to(DEV)
    ws = cobs.new_workspace(cfg, cobs.OP_SELECT_EXACT, DEV)
    outs = {}
    for name, fn in (("exact", cobs.cobs_select_exact), ("quest", cobs.cobs_select_quest)):
        sel = torch.full((B, Hkv, max(s, 1)), -7, dtype=torch.int32, device=DEV)
        scores = torch.empty((B, Hkv, cfg.num_blocks), dtype=torch.float32, device=DEV)
        fn(cfg, qd, kd, vd, seq_d, sel, ws, scores=scores)
        outs[name] = (sel, scores)
    sel_e = outs["exact"][0][:, :, :s].contiguous()
    shp = (B, G * Hkv, d)
    o_s, o_w = (torch.empty(shp, dtype=torch.float32, device=DEV) for _ in range(2))
    l_s, l_w = (torch.empty(shp[:2], dtype=torch.float32, device=DEV) for _ in range(2))
    cobs.cobs_sparse_decode_branches(cfg, qd, kd, vd, seq_d, sel_e, o_s, o_w,
                                     cobs.new_workspace(cfg, cobs.OP_DECODE, DEV), lse_sel=l_s, lse_win=l_w)
    sync()
    hs, hw, ls, lw = o_s.cpu().numpy(), o_w.cpu().numpy(), l_s.cpu().numpy(), l_w.cpu().numpy()
    oracles = {"exact": M.osa_group_scores, "quest": M.quest_group_scores}
    for b in range(B):
        T = int(c["seq"][b])
        nc = M.candidate_count(T, L, w)
        for h in range(Hkv):
            gs = slice(h * G, (h + 1) * G)
            qg, Kg = q[b, gs].double().numpy(), f64(k[b, h])
            for name, (sel, scores) in outs.items():
                sigma = oracles[name](qg, Kg, T, L, cfg.scale)
                got = scores[b, h].cpu().numpy()
                assert np.all(np.abs(got[:nc] - sigma[:nc]) <= SIGMA_TOL), (name, b, h)
                assert np.all(np.isneginf(got[nc:])), (name, b, h)
                if s > 0:
                    check_selection(sel[b, h, :s].cpu().numpy(), sigma, nc, s)
            ref = M.branch_attention(qg, Kg, f64(v[b, h]), T, L, w, sel_e[b, h].cpu().numpy(), cfg.scale)
            slack = score_slack(qg, Kg, T, sel_e[b, h].cpu().numpy(), cfg)
            check_out(hs[b, gs], ls[b, gs], ref[0], ref[1], "bf16", slack)
            check_out(hw[b, gs], lw[b, gs], ref[2], ref[3], "bf16", slack)


@pytest.mark.parametrize("seed", list(range(int(_N) if _N else 6)))
def test_random_paged_cache_is_bitwise_contiguous(seed):
    """The same cache stored as pages of one block in a shuffled pool (with
    unused pages) gives bitwise the contiguous results: block statistics,
    attention, the decode step and, for bf16 caches, the exact-mass selector and
    the two-branch decode."""
    c = _draw(7000 + seed)
    G, d, Hkv, B, tmax, s, w = c["G"], c["d"], c["Hkv"], c["B"], c["tmax"], c["s"], c["w"]
    say(f"random paged config {seed}: {c}")
    L = c["L"]
    prob = synth.make_problem("c2", seed=8000 + seed, B=B, Hq=G * Hkv, Hkv=Hkv, d=d, T=tmax, kv_dtype=c["kv"], L=L)
    cfg = cobs.Config(batch=B, num_q_heads=G * Hkv, num_kv_heads=Hkv, head_dim=d, max_seq_len=tmax,
                      rank=c["r"], budget=s, window=w, kv_dtype=c["kv"], mean_dtype=c["md"],
                      factor_dtype=c["fd"], skew=c["skew"], value_mean=c["vmean"], block_size=L)
    q, k, v = prob["q"].to(DEV), prob["k"].to(DEV), prob["v"].to(DEV)
    nbm = tmax // L
    pages = B * nbm + 3
    perm = torch.randperm(pages, generator=torch.Generator().manual_seed(9000 + seed))[:B * nbm]
    table = perm.view(B, nbm).to(torch.int32)
    kp = torch.zeros((pages, Hkv, L, d), dtype=k.dtype, device=DEV)
    vp = torch.zeros_like(kp)
    for b in range(B):
        for j in range(nbm):
            kp[table[b, j]] = k[b, :, j * L:(j + 1) * L]
            vp[table[b, j]] = v[b, :, j * L:(j + 1) * L]
    tab = table.to(DEV)
    seq_d = torch.from_numpy(c["seq"]).to(DEV)

    def run(paged):
        kw = dict(block_table=tab, num_pages=pages) if paged else {}
        kk, vv = (kp, vp) if paged else (k, v)
        res = {}
        rec = cobs.new_summaries(cfg, DEV)
        cobs.cobs_build_block_stats(cfg, kk, vv, seq_d, rec, **kw)
        res["rec"] = rec
        sel = synth.make_selection(B, Hkv, c["seq"], L, w, max(s, 1), seed=seed, fill="random")[:, :, :s]
        sel = sel.contiguous().to(DEV)
        res["out"] = torch.empty((B, G * Hkv, d), dtype=torch.float32, device=DEV)
        res["lse"] = torch.empty((B, G * Hkv), dtype=torch.float32, device=DEV)
        cobs.cobs_sparse_decode(cfg, q, kk, vv, seq_d, sel, res["out"], cobs.new_workspace(cfg, cobs.OP_DECODE, DEV),
                                lse=res["lse"], **kw)
        res["rec1"] = rec.clone()
        res["out1"], res["lse1"] = torch.empty_like(res["out"]), torch.empty_like(res["lse"])
        res["sel1"] = torch.empty((B, Hkv, max(s, 1)), dtype=torch.int32, device=DEV)
        cobs.cobs_decode_step(cfg, q, kk, vv, seq_d, res["rec1"], res["out1"],
                              cobs.new_workspace(cfg, cobs.OP_STEP, DEV), sel=res["sel1"] if s > 0 else None,
                              lse=res["lse1"], **kw)
        if c["kv"] == "bf16":
            res["sx"] = torch.full((B, Hkv, max(s, 1)), -7, dtype=torch.int32, device=DEV)
            res["scx"] = torch.empty((B, Hkv, cfg.num_blocks), dtype=torch.float32, device=DEV)
            cobs.cobs_select_exact(cfg, q, kk, vv, seq_d, res["sx"], cobs.new_workspace(cfg, cobs.OP_SELECT_EXACT, DEV),
                                   scores=res["scx"], **kw)
            for nm in ("os", "ow"):
                res[nm] = torch.empty_like(res["out"])
            for nm in ("ls", "lw"):
                res[nm] = torch.empty_like(res["lse"])
            cobs.cobs_sparse_decode_branches(cfg, q, kk, vv, seq_d, sel, res["os"], res["ow"],
                                             cobs.new_workspace(cfg, cobs.OP_DECODE, DEV), lse_sel=res["ls"],
                                             lse_win=res["lw"], **kw)
        sync()
        return res

    a, b_ = run(False), run(True)
    assert sorted(a) == sorted(b_)
    for key in a:
        if key == "sel1" and s == 0:
            continue
        assert torch.equal(a[key], b_[key]), key

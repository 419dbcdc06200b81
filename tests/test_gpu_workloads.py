"""End-to-end decode steps of the five workloads against the fp64 oracle.

Two comparisons per checked (batch row, KV head) unit:

* Shared record bytes (the decode-step rule): the oracle scores the records the
  GPU built, so |sigma_gpu - sigma_oracle| <= 2e-5 on every candidate, the
  selection is bit-exact unless the oracle's gap at the s-th boundary is below
  1e-4 (then the set rule), and the step's output matches the oracle's
  attention on the GPU's selection (relative L2 2e-3 for bf16 K/V, 1e-5 for
  fp32).  The GPU's records themselves are checked against the oracle's block
  statistics (counts, means, Ky-Fan energy, orthogonality, rank-r covariance)
  and byte for byte against the oracle's storage encoding of the GPU's fp32
  statistics.
* Independent descriptors (build quality): the oracle also builds its own
  descriptors from K by exact fp64 eigendecomposition.  The two sides' fp32
  statistics, scored alike, agree within 2e-3 on every candidate (the solver's
  accuracy, free of the storage rounding, whose encoding is checked byte for
  byte above); at the configured storage the selections follow the set rule at
  twice a band per factor storage type (DECISION_BAND), the share of selected
  block ids that differ is bounded, and attention on the oracle's selection
  matches the oracle.
"""

import numpy as np
import pytest
import torch

import synth
from oracle import method as M
from paper_2607_09052_amd import cobs
from tests.gpu_util import (DEV, SIGMA_TOL, check_out, check_records, check_selection, config_from, f32_config,
                            f64, oracle_decode, oracle_select, say, score_slack, sync)

pytestmark = pytest.mark.gpu

# |sigma_gpu - sigma_oracle| band for independently built descriptors, by the
# factor storage type.  fp32 factors: the fixed-count iteration meets the
# Ky-Fan energy bound to ~1e-6 and the rank-r covariance to 1e-3 (relative
# Frobenius) where the eigengap is >= 5 %, which moves (c^2/2) q^T Sigma_r q by
# well under 2e-3 at these query norms; the scores of the fp32 statistics are
# held to this band.  Stored bf16 / E2M1 factors: a solver difference of ~1e-6
# can move an element across a rounding boundary of the storage format, one
# code step (for E2M1 up to max|xi|/3), which moved one c4 block's sigma by
# 3.2e-2; these bands apply to the selections (set rule at twice the band) and
# to the share of differing block ids.
DECISION_BAND = {"f32": 2e-3, "bf16": 4e-3, "e2m1": 2e-2}
# Largest share of selected block ids allowed to differ between the GPU's and
# the oracle's independently built descriptors (boundary blocks whose scores
# lie within the band above).
ID_DIFF_BOUND = {"f32": 0.01, "bf16": 0.01, "e2m1": 0.02}


def _oracle_stats(K, T, cfg):
    return M.stored_statistics(*M.block_statistics(K, T, cfg.block_size, cfg.rank), cfg.mean_dtype,
                               cfg.factor_dtype)


def _id_diff(a, b):
    a = {x for x in np.asarray(a).tolist() if x >= 0}
    b = {x for x in np.asarray(b).tolist() if x >= 0}
    return len(a - b), max(len(a), 1)


def _shared_bytes_check(cfg, rec_u, q_u, K_u, V_u, T, sel_u, out_u, lse_u, scores_u=None):
    """The decode-step rule on the GPU's own records: oracle scores of the same
    bytes, the set rule at 1e-4, attention on the GPU's selection."""
    sigma, nc, _ = oracle_select(rec_u, q_u, T, cfg)
    if scores_u is not None:
        assert np.all(np.abs(scores_u[:nc] - sigma[:nc]) <= SIGMA_TOL), float(np.max(np.abs(scores_u[:nc] - sigma[:nc])))
    exact = check_selection(sel_u, sigma, nc, cfg.budget)
    o, l = oracle_decode(q_u, K_u, V_u, T, sel_u, cfg)
    check_out(out_u, lse_u, o, l, cfg.kv_dtype, score_slack(q_u, K_u, T, sel_u, cfg))
    return exact


def _sample_blocks(nb, want=48):
    return sorted(set(range(0, nb, max(1, nb // want))) | {nb - 1})


def _run_case(name, seed, units=None, **over):
    prob = synth.make_problem(name, seed=seed, device=DEV, **over)
    c = prob["cfg"]
    cfg = config_from(c)
    B, Hkv, G, d = c["B"], c["Hkv"], c["Hq"] // c["Hkv"], c["d"]
    q, k, v, seq = prob["q"], prob["k"], prob["v"], prob["seq_lens"]
    rec = cobs.new_summaries(cfg, DEV)
    say(f"{name}: build {B}x{Hkv}x{cfg.num_blocks} blocks")
    cobs.cobs_build_block_stats(cfg, k, v, seq, rec)
    cfg32 = f32_config(cfg)
    if (cfg.mean_dtype, cfg.factor_dtype) == ("f32", "f32"):
        rec32 = rec
    else:
        rec32 = cobs.new_summaries(cfg32, DEV)
        cobs.cobs_build_block_stats(cfg32, k, v, seq, rec32)
    out = torch.empty((B, c["Hq"], d), dtype=torch.float32, device=DEV)
    lse = torch.empty((B, c["Hq"]), dtype=torch.float32, device=DEV)
    sel = torch.empty((B, Hkv, c["s"]), dtype=torch.int32, device=DEV)
    ws = cobs.new_workspace(cfg, cobs.OP_STEP, DEV)
    say(f"{name}: decode step")
    cobs.cobs_decode_step(cfg, q, k, v, seq, rec, out, ws, sel=sel, lse=lse)
    scores = torch.empty((B, Hkv, cfg.num_blocks), dtype=torch.float32, device=DEV)
    sel2 = torch.empty_like(sel)
    cobs.cobs_select(cfg, q, rec, seq, sel2, cobs.new_workspace(cfg, cobs.OP_SELECT, DEV), scores=scores)
    sync()
    assert torch.equal(sel, sel2)
    if units is None:
        units = [(b, h) for b in range(B) for h in range(Hkv)]
    band = DECISION_BAND[cfg.factor_dtype]
    # the oracle's selections, fed to the GPU's sparse decode
    ora = {}
    sel_o = torch.full_like(sel, -1)
    worst = 0.0
    same = shared_exact = 0
    ndiff = ntot = 0
    T = int(c["T"])
    L = cfg.block_size
    nb = -(-T // L)
    for (b, h) in units:
        K, V = f64(k[b, h, :T]), f64(v[b, h, :T])
        qu = f64(q[b, h * G:(h + 1) * G])
        sl = slice(h * G, (h + 1) * G)
        rec_u = rec[b, h].cpu().numpy()
        check_records(cfg, rec_u, rec32[b, h].cpu().numpy(), K, T, _sample_blocks(nb))
        shared_exact += _shared_bytes_check(cfg, rec_u, qu, K, V, T, sel[b, h].cpu().numpy(),
                                            out[b, sl].cpu().numpy(), lse[b, sl].cpu().numpy(),
                                            scores[b, h].cpu().numpy())
        raw = M.block_statistics(K, T, L, cfg.rank)
        res = M.decode_unit(qu, K, V, T, L, cfg.rank, cfg.budget, cfg.window, cfg.scale,
                            cfg.mean_dtype, cfg.factor_dtype,
                            stats=M.stored_statistics(*raw, cfg.mean_dtype, cfg.factor_dtype))
        ora[(b, h)] = res
        nc = res["nc"]
        # the solver: both sides' fp32 statistics, scored alike
        sg = oracle_select(rec32[b, h].cpu().numpy(), qu, T, cfg32)[0]
        so = M.group_scores(M.log_mass_estimate(qu, *M.stored_statistics(*raw, "f32", "f32")[:3], cfg.scale))
        dev_ = float(np.max(np.abs(sg[:nc] - so[:nc]))) if nc else 0.0
        worst = max(worst, dev_)
        assert dev_ <= DECISION_BAND["f32"], (b, h, dev_)
        same += check_selection(sel[b, h].cpu().numpy(), res["sigma"], nc, cfg.budget, band=2 * band)
        nd, nt = _id_diff(sel[b, h].cpu().numpy(), res["sel"])
        ndiff, ntot = ndiff + nd, ntot + nt
        sel_o[b, h] = torch.from_numpy(res["sel"].astype(np.int32))
    say(f"{name}: shared bytes: exact selections {shared_exact}/{len(units)}; independent descriptors: "
        f"max |sigma_gpu - sigma_oracle| at fp32 storage = {worst:.2e}, identical selections {same}/{len(units)}, "
        f"differing block ids {ndiff}/{ntot}")
    assert ndiff <= ID_DIFF_BOUND[cfg.factor_dtype] * ntot, (ndiff, ntot)
    out_o = torch.empty_like(out)
    lse_o = torch.empty_like(lse)
    cobs.cobs_sparse_decode(cfg, q, k, v, seq, sel_o, out_o, cobs.new_workspace(cfg, cobs.OP_DECODE, DEV), lse=lse_o)
    sync()
    for (b, h), res in ora.items():
        sl = slice(h * G, (h + 1) * G)
        qu = f64(q[b, h * G:(h + 1) * G])
        check_out(out_o[b, sl].cpu().numpy(), lse_o[b, sl].cpu().numpy(), res["out"], res["lse"], cfg.kv_dtype,
                  score_slack(qu, f64(k[b, h, :T]), T, res["sel"], cfg))
    return prob, sel, ora


def test_c1_tiny_single_head(golden_dir):
    import os
    with open(os.path.join(golden_dir, "c1_seed.txt")) as f:
        seed = int(f.read().split()[0])
    prob, sel, ora = _run_case("c1", seed)
    res = ora[(0, 0)]
    assert sel[0, 0].cpu().tolist() == res["sel"].tolist()
    assert prob["planted"][(0, 0)] in res["sel"].tolist()


@pytest.mark.parametrize("name,over", [
    ("c2", dict(B=1, Hq=8, Hkv=2, T=4096)),
    ("c3", dict(B=2, Hq=8, Hkv=2, T=4096, s=16)),
    ("c4", dict(B=1, Hq=16, Hkv=2, T=8192, s=20)),
    ("c5", dict(B=2, Hq=8, Hkv=2, T=3000, s=16, steps=0)),
    # the paper's block length (Sec. 7.1: L = 32) and L = 128
    ("c2", dict(B=1, Hq=8, Hkv=2, T=4096, s=32, L=32)),
    ("c3", dict(B=2, Hq=8, Hkv=2, T=4096, s=10, L=128)),
    ("c5", dict(B=2, Hq=8, Hkv=2, T=3000, s=24, steps=0, L=32)),
])
def test_reduced_workloads(name, over):
    _run_case(name, 2000 + len(name) + over["T"] + over.get("L", 64), **over)


def test_c2_full_size_every_unit():
    _run_case("c2", None)


@pytest.mark.parametrize("name,units", [("c3", [(0, 0), (13, 5), (31, 7)]), ("c4", [(0, 0), (7, 6)])])
def test_full_size_sampled_units(name, units):
    _run_case(name, None, units=units)
    torch.cuda.empty_cache()


def test_c5_build_then_256_appending_steps():
    """Prefill build, then 256 decode steps that each append one token (c5 shapes).

    Every 8th step, every block-fill step and the last: on two units, the step's
    selection and output against the oracle on the step's own records (the
    decode-step rule), and against the oracle's independently maintained
    records (band rule; the differing selected ids are counted and bounded).
    On block-fill steps the newly filled block's record is also checked against
    the oracle's statistics of its keys."""
    prob = synth.make_problem("c5", device=DEV)
    c = prob["cfg"]
    cfg = config_from(c)
    cfg32 = f32_config(cfg)
    B, Hkv, G, d, T0 = c["B"], c["Hkv"], c["Hq"] // c["Hkv"], c["d"], c["T"]
    k, v = prob["k"], prob["v"]
    seq = torch.full((B,), T0, dtype=torch.int32, device=DEV)
    rec = cobs.new_summaries(cfg, DEV)
    rec32 = cobs.new_summaries(cfg32, DEV)
    say("c5: prefill build")
    cobs.cobs_build_block_stats(cfg, k, v, seq, rec)
    ws = cobs.new_workspace(cfg, cobs.OP_STEP, DEV)
    out = torch.empty((B, c["Hq"], d), dtype=torch.float32, device=DEV)
    lse = torch.empty((B, c["Hq"]), dtype=torch.float32, device=DEV)
    sel = torch.empty((B, Hkv, c["s"]), dtype=torch.int32, device=DEV)
    units = [(0, 0), (3, 5)]
    Kf = {u: f64(k[u[0], u[1]]) for u in units}
    Vf = {u: f64(v[u[0], u[1]]) for u in units}
    stats = {u: [np.array(x) for x in _oracle_stats(Kf[u], T0, cfg)] for u in units}
    band = DECISION_BAND[cfg.factor_dtype]
    checked = shared_exact = indep_same = ndiff = ntot = fills = 0
    for step in range(c["steps"]):
        T = T0 + step + 1
        seq.fill_(T)
        q = prob["q_steps"][step].contiguous()
        cobs.cobs_decode_step(cfg, q, k, v, seq, rec, out, ws, sel=sel, lse=lse)
        fill = T % 64 == 0
        if step % 8 == 0 or step == c["steps"] - 1 or fill:
            j = (T - 1) // 64
            if fill:
                # the filled block once more with fp32 storage, for its statistics
                cobs.cobs_build_block_stats(cfg32, k, v, seq, rec32, first_block=j, num_blocks=1)
            sync()
            say(f"c5: step {step} T={T}")
            for (b, h) in units:
                qu = f64(q[b, h * G:(h + 1) * G])
                sl = slice(h * G, (h + 1) * G)
                rec_u = rec[b, h].cpu().numpy()
                if fill:
                    check_records(cfg, rec_u, rec32[b, h].cpu().numpy(), Kf[(b, h)][:T], T, [j])
                    fills += 1
                shared_exact += _shared_bytes_check(cfg, rec_u, qu, Kf[(b, h)], Vf[(b, h)], T,
                                                    sel[b, h].cpu().numpy(), out[b, sl].cpu().numpy(),
                                                    lse[b, sl].cpu().numpy())
                # oracle tail update (the block holding token T-1), then the step
                # on the oracle's own records
                cnt, mns, fac = stats[(b, h)]
                tail = M.stored_statistics(*M.block_statistics(Kf[(b, h)][j * 64:T], T - j * 64, 64, cfg.rank),
                                           cfg.mean_dtype, cfg.factor_dtype)
                if j >= len(cnt):
                    cnt = np.concatenate([cnt, tail[0]])
                    mns = np.concatenate([mns, tail[1]])
                    fac = np.concatenate([fac, tail[2]])
                else:
                    cnt[j], mns[j], fac[j] = tail[0][0], tail[1][0], tail[2][0]
                stats[(b, h)] = [cnt, mns, fac]
                res = M.decode_unit(qu, Kf[(b, h)], Vf[(b, h)], T, 64, cfg.rank, cfg.budget, cfg.window,
                                    cfg.scale, cfg.mean_dtype, cfg.factor_dtype, stats=(cnt, mns, fac))
                indep_same += check_selection(sel[b, h].cpu().numpy(), res["sigma"], res["nc"], cfg.budget,
                                              band=2 * band)
                nd, nt = _id_diff(sel[b, h].cpu().numpy(), res["sel"])
                ndiff, ntot = ndiff + nd, ntot + nt
                checked += 1
    say(f"c5: {checked} unit-steps checked ({fills} on block fills); shared bytes: exact selections "
        f"{shared_exact}/{checked}; independent descriptors: identical selections {indep_same}/{checked}, "
        f"differing block ids {ndiff}/{ntot}")
    assert fills >= 2 * 4
    assert ndiff <= ID_DIFF_BOUND[cfg.factor_dtype] * ntot, (ndiff, ntot)

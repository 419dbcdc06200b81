"""cobs_decode_step_noalloc (the library's own per-GPU workspace) against
cobs_decode_step with a caller workspace: bitwise equal selections, outputs,
log-sum-exps and refreshed records, on two calls in a row whose second has a
smaller problem (a different workspace layout over the same array), on both
dispatch paths of the step (the refresh inside the selector launch, rank <= 4
with bf16 K/V; and the separate refresh launch, rank 6)."""

import numpy as np
import pytest
import torch

import synth
from paper_2607_09052_amd import cobs
from tests.gpu_util import DEV, say, sync

pytestmark = pytest.mark.gpu


def _case(B, Hq, Hkv, d, T, r, s, w, md, fd, seed):
    prob = synth.make_problem("c2", seed=seed, B=B, Hq=Hq, Hkv=Hkv, d=d, T=T, kv_dtype="bf16")
    cfg = cobs.Config(batch=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, max_seq_len=T, rank=r, budget=s,
                      window=w, kv_dtype="bf16", mean_dtype=md, factor_dtype=fd)
    q, k, v = prob["q"].to(DEV), prob["k"].to(DEV), prob["v"].to(DEV)
    rng = np.random.default_rng(seed)
    seq = rng.integers(1, T + 1, size=B).astype(np.int32)
    seq[0] = T - 1
    seq_d = torch.from_numpy(seq).to(DEV)
    rec = cobs.new_summaries(cfg, DEV)
    cobs.cobs_build_block_stats(cfg, k, v, seq_d, rec)
    # the newest block of each row is stale: the step must recompute it
    for b in range(B):
        rec[b, :, (int(seq[b]) - 1) // 64] = 0
    return cfg, q, k, v, seq_d, rec


def _both(cfg, q, k, v, seq_d, rec):
    B, Hq, d, Hkv, s = cfg.batch, cfg.num_q_heads, cfg.head_dim, cfg.num_kv_heads, cfg.budget
    res = []
    for noalloc in (False, True):
        r = rec.clone()
        out = torch.full((B, Hq, d), 7.0, dtype=torch.float32, device=DEV)
        lse = torch.full((B, Hq), 7.0, dtype=torch.float32, device=DEV)
        sel = torch.full((B, Hkv, s), -7, dtype=torch.int32, device=DEV)
        if noalloc:
            cobs.cobs_decode_step_noalloc(cfg, q, k, v, seq_d, r, out, sel=sel, lse=lse)
        else:
            cobs.cobs_decode_step(cfg, q, k, v, seq_d, r, out, cobs.new_workspace(cfg, cobs.OP_STEP, DEV),
                                  sel=sel, lse=lse)
        res.append((r, out, lse, sel))
    sync()
    for a, b in zip(*res):
        assert torch.equal(a, b)
    assert bool(torch.all(res[1][3][0, :, 0] >= 0))      # row 0 has candidates


@pytest.mark.parametrize("rank", [4, 6])
def test_noalloc_step_matches_workspace_step_twice(rank):
    big = _case(B=4, Hq=32, Hkv=8, d=128, T=8192, r=rank, s=24, w=300, md="bf16", fd="e2m1", seed=31 + rank)
    say(f"noalloc: rank {rank}, first call B=4 Hq=32 Hkv=8 T=8192")
    _both(*big)
    small = _case(B=2, Hq=8, Hkv=2, d=64, T=1536, r=rank, s=5, w=64, md="f32", fd="f32", seed=41 + rank)
    say(f"noalloc: rank {rank}, second call B=2 Hq=8 Hkv=2 d=64 T=1536")
    _both(*small)

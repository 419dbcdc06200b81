"""Seeded synthetic inputs for the COBS decode-step path.

Shared by the tests, the benchmark and the smoke check; it serves both the HIP
path and the oracle and therefore holds none of the method's arithmetic: it
only draws random numbers with the shapes and distributions of the decode
workloads and lays them out in memory.

Workloads (B batch, Hq query heads, Hkv KV heads, d head dim, T context, L block,
r factor rank, s block budget, w window):

  c1  tiny single head      1,  1, 1,  64,   1024, 64, 2,  4,   64   fp32 K/V
  c2  single-layer GQA      1, 32, 8, 128,  32768, 64, 4, 16,  512   bf16 K/V
  c3  batched GQA          32, 32, 8, 128,  32768, 64, 4, 85,  512   bf16 K/V
  c4  long-context FP4      8, 64, 8, 128, 131072, 64, 4, 85, 1024   bf16 K/V
  c5  build + 256 steps     4, 32, 8, 128,  65536, 64, 4, 64,  512   bf16 K/V

Key laws (per KV head):
  c1  q, K, V i.i.d. N(0,1); one planted block p ~ U{0..14} gets
      k += 0.5 q / |q|.
  c2  per-block mean mu_b ~ N(0, 0.09 I); k = mu_b + N(0, I).
  c3  mu_b ~ N(0, 0.09 I); A_b in R^{d x 8} with N(0, 1/8) entries;
      k = mu_b + A_b z + sqrt(0.1) eps (block covariance A A^T + 0.1 I);
      5 needle blocks among the candidates, u = normalised sum_g q_g/|q_g|:
      3 mean-shift needles k += 2 u, 2 curvature needles k += a_t u with
      a_t ~ N(0, 4).
  c4  sigma_j = 4 (1/16)^(j/63) on channel pair j; mu_b ~ N(0, 0.09) * sigma;
      k = mu_b + sigma * t3 with i.i.d. Student-t (nu = 3) entries.
  c5  16 component means m_j ~ N(0, I); each token picks a component
      uniformly; k = m_z + 0.5 eps.
  V ~ N(0, 1) and q ~ N(0, 1) everywhere.
"""

import math

import numpy as np
import torch

CONFIGS = {
    "c1": dict(B=1, Hq=1, Hkv=1, d=64, T=1024, L=64, r=2, s=4, w=64,
               kv_dtype="f32", mean_dtype="f32", factor_dtype="f32", law="c1"),
    "c2": dict(B=1, Hq=32, Hkv=8, d=128, T=32768, L=64, r=4, s=16, w=512,
               kv_dtype="bf16", mean_dtype="f32", factor_dtype="f32", law="c2"),
    "c3": dict(B=32, Hq=32, Hkv=8, d=128, T=32768, L=64, r=4, s=85, w=512,
               kv_dtype="bf16", mean_dtype="f32", factor_dtype="f32", law="c3"),
    "c4": dict(B=8, Hq=64, Hkv=8, d=128, T=131072, L=64, r=4, s=85, w=1024,
               kv_dtype="bf16", mean_dtype="e2m1", factor_dtype="e2m1", law="c4"),
    "c5": dict(B=4, Hq=32, Hkv=8, d=128, T=65536, L=64, r=4, s=64, w=512,
               kv_dtype="bf16", mean_dtype="bf16", factor_dtype="e2m1", law="c5",
               steps=256),
}

SEED_BASE = 1000


def config(name, **over):
    """A copy of a workload description, with optional overrides (smaller B, T, ...)."""
    cfg = dict(CONFIGS[name])
    cfg.update(over)
    cfg.setdefault("steps", 0)
    # cache capacity: the tokens of the workload rounded up to whole blocks
    cfg.setdefault("T_max", -(-(cfg["T"] + cfg["steps"]) // cfg["L"]) * cfg["L"])
    return cfg


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def _randn(shape, g, device, std=1.0):
    return torch.randn(*shape, generator=g, device=device, dtype=torch.float32) * std


def _store(x, kv_dtype):
    return x.to(torch.bfloat16) if kv_dtype == "bf16" else x.to(torch.float32)


def _unit(x, dim=-1):
    return x / x.norm(dim=dim, keepdim=True)


def _keys_c1(cfg, q, g, device):
    B, Hkv, Tm, d, L = cfg["B"], cfg["Hkv"], cfg["T_max"], cfg["d"], cfg["L"]
    K = _randn((B, Hkv, Tm, d), g, device)
    G = cfg["Hq"] // Hkv
    nb = cfg["T"] // L
    planted = {}
    for b in range(B):
        for h in range(Hkv):
            p = int(torch.randint(0, max(1, nb - 1), (1,), generator=g, device=device).item())
            u = _unit(q[b, h * G:(h + 1) * G].sum(0))
            K[b, h, p * L:(p + 1) * L] += 0.5 * u
            planted[(b, h)] = p
    return K, planted


def _keys_c2(cfg, g, device):
    B, Hkv, Tm, d, L = cfg["B"], cfg["Hkv"], cfg["T_max"], cfg["d"], cfg["L"]
    nb = -(-Tm // L)
    mu = _randn((B, Hkv, nb, 1, d), g, device, 0.3)
    K = _randn((B, Hkv, nb, L, d), g, device) + mu
    return K.reshape(B, Hkv, nb * L, d)[:, :, :Tm]


def _keys_c3(cfg, q, g, device):
    B, Hkv, Tm, d, L, T, w = (cfg[k] for k in ("B", "Hkv", "T_max", "d", "L", "T", "w"))
    G = cfg["Hq"] // Hkv
    nb = -(-Tm // L)
    K = torch.empty((B, Hkv, nb, L, d), device=device, dtype=torch.float32)
    for b in range(B):                               # one batch row at a time bounds memory
        mu = _randn((Hkv, nb, 1, d), g, device, 0.3)
        A = _randn((Hkv, nb, d, 8), g, device, 1.0 / math.sqrt(8.0))
        z = _randn((Hkv, nb, 8, L), g, device)
        eps = _randn((Hkv, nb, L, d), g, device, math.sqrt(0.1))
        K[b] = mu + torch.matmul(A, z).transpose(-1, -2) + eps
    K = K.reshape(B, Hkv, nb * L, d)
    nc = -(-max(0, T - w) // L)
    needles, kinds = {}, {}
    if nc >= 5:
        for b in range(B):
            for h in range(Hkv):
                qs = q[b, h * G:(h + 1) * G]
                u = _unit((qs / qs.norm(dim=1, keepdim=True)).sum(0))
                pick = torch.randperm(nc, generator=g, device=device)[:5].tolist()
                for j, blk in enumerate(pick):
                    sl = slice(blk * L, (blk + 1) * L)
                    if j < 3:
                        K[b, h, sl] += 2.0 * u
                    else:
                        a = _randn((L, 1), g, device, 2.0)
                        K[b, h, sl] += a * u
                needles[(b, h)] = sorted(pick)
                kinds[(b, h)] = {blk: ("mean" if j < 3 else "curvature") for j, blk in enumerate(pick)}
    return K[:, :, :Tm], needles, kinds


def _keys_c4(cfg, g, device):
    B, Hkv, Tm, d, L = cfg["B"], cfg["Hkv"], cfg["T_max"], cfg["d"], cfg["L"]
    nb = -(-Tm // L)
    j = torch.arange(d // 2, device=device, dtype=torch.float32)
    sig = (4.0 * (1.0 / 16.0) ** (j / 63.0)).repeat_interleave(2)          # [d]
    K = torch.empty((B, Hkv, nb, L, d), device=device, dtype=torch.float32)
    for b in range(B):
        mu = _randn((Hkv, nb, 1, d), g, device, 0.3) * sig
        z = _randn((Hkv, nb, L, d), g, device)
        chi2 = (_randn((3, Hkv, nb, L, d), g, device) ** 2).sum(0)
        K[b] = mu + sig * (z / torch.sqrt(chi2 / 3.0))
    return K.reshape(B, Hkv, nb * L, d)[:, :, :Tm]


def _keys_c5(cfg, g, device):
    B, Hkv, Tm, d = cfg["B"], cfg["Hkv"], cfg["T_max"], cfg["d"]
    m = _randn((B, Hkv, 16, d), g, device)
    z = torch.randint(0, 16, (B, Hkv, Tm), generator=g, device=device)
    K = torch.gather(m, 2, z[..., None].expand(B, Hkv, Tm, d)) + _randn((B, Hkv, Tm, d), g, device, 0.5)
    return K


def make_problem(name, seed=None, device="cpu", **over):
    """Seeded decode problem of a workload.

    Returns dict(cfg, q [B,Hq,d] fp32, k, v [B,Hkv,T_max,d] in the K/V dtype,
    seq_lens [B] int32 (all T), and for c5 q_steps [steps,B,Hq,d]; for c1 the
    planted block and for c3 the needle blocks, per (b, h), and their kinds).
    """
    cfg = config(name, **over)
    seed = SEED_BASE + int(name[1:]) if seed is None else seed
    g = _gen(device, seed)
    B, Hq, Hkv, d, Tm = cfg["B"], cfg["Hq"], cfg["Hkv"], cfg["d"], cfg["T_max"]
    q = _randn((B, Hq, d), g, device)
    law = cfg["law"]
    extra = {}
    if law == "c1":
        K, extra["planted"] = _keys_c1(cfg, q, g, device)
    elif law == "c2":
        K = _keys_c2(cfg, g, device)
    elif law == "c3":
        K, extra["needles"], extra["needle_kinds"] = _keys_c3(cfg, q, g, device)
    elif law == "c4":
        K = _keys_c4(cfg, g, device)
    elif law == "c5":
        K = _keys_c5(cfg, g, device)
    else:
        raise ValueError(law)
    V = _randn((B, Hkv, Tm, d), g, device)
    out = dict(cfg=cfg, q=q, k=_store(K, cfg["kv_dtype"]).contiguous(),
               v=_store(V, cfg["kv_dtype"]).contiguous(),
               seq_lens=torch.full((B,), cfg["T"], dtype=torch.int32, device=device))
    if cfg["steps"]:
        out["q_steps"] = _randn((cfg["steps"], B, Hq, d), g, device)
    out.update(extra)
    return out


# ------------------------------------------------------- descriptor records --
# Random records laid out in the documented record format (see include/cobs.h):
# 16-byte header {int32 n, f32 mean scale, 8 zero bytes}, E2M1 factor scales
# padded to 16 bytes, the mean, the r factors, total padded to 16 bytes.

def _vec_bytes(d, dt):
    return {"f32": 4 * d, "bf16": 2 * d, "e2m1": d // 2}[dt]


def record_bytes(d, r, mean_dtype, factor_dtype):
    fs = ((4 * r + 15) // 16 * 16) if factor_dtype == "e2m1" else 0
    tot = 16 + fs + _vec_bytes(d, mean_dtype) + r * _vec_bytes(d, factor_dtype)
    return (tot + 15) // 16 * 16


def _random_vectors(rng, n, d, dt, std):
    """(raw bytes [n, vec_bytes], scales or None) of random vectors drawn in storage format."""
    if dt == "f32":
        return (rng.standard_normal((n, d)) * std).astype(np.float32).view(np.uint8), None
    if dt == "bf16":
        x = torch.from_numpy((rng.standard_normal((n, d)) * std).astype(np.float32)).to(torch.bfloat16)
        return x.view(torch.int16).numpy().view(np.uint8).reshape(n, -1), None
    nib = rng.integers(0, 16, size=(n, d), dtype=np.uint8)
    raw = (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)
    scales = (std / 3.0 * np.exp(rng.normal(0.0, 0.3, size=n))).astype(np.float32)
    return raw, scales


def make_records(B, Hkv, T_max, L, d, r, mean_dtype, factor_dtype, seq_lens, seed,
                 mean_std=0.3, factor_std=0.5):
    """Random descriptor records [B, Hkv, ceil(T_max/L), record_bytes] (uint8, CPU).

    Counts follow each sequence length: n_b = min(L, T - bL) for b < ceil(T/L),
    0 beyond.  Means and factors are random numbers drawn directly in the
    storage dtype (random codes and scales for E2M1).
    """
    rng = np.random.default_rng(seed)
    nbm = -(-T_max // L)
    rb = record_bytes(d, r, mean_dtype, factor_dtype)
    fs = ((4 * r + 15) // 16 * 16) if factor_dtype == "e2m1" else 0
    moff = 16 + fs
    mb = _vec_bytes(d, mean_dtype)
    vb = _vec_bytes(d, factor_dtype)
    out = np.zeros((B, Hkv, nbm, rb), dtype=np.uint8)
    for b in range(B):
        T = int(seq_lens[b])
        nb = -(-T // L)
        for h in range(Hkv):
            cnt = np.array([min(L, T - i * L) for i in range(nb)], dtype=np.int32)
            rec = out[b, h, :nb]
            rec[:, 0:4] = cnt.view(np.uint8).reshape(nb, 4)
            raw, sc = _random_vectors(rng, nb, d, mean_dtype, mean_std)
            rec[:, moff:moff + mb] = raw
            if sc is not None:
                rec[:, 4:8] = sc.view(np.uint8).reshape(nb, 4)
            for i in range(r):
                raw, sc = _random_vectors(rng, nb, d, factor_dtype, factor_std)
                off = moff + mb + i * vb
                rec[:, off:off + vb] = raw
                if sc is not None:
                    rec[:, 16 + 4 * i:20 + 4 * i] = sc.view(np.uint8).reshape(nb, 4)
    return torch.from_numpy(out)


def make_selection(B, Hkv, seq_lens, L, w, s, seed, fill="random"):
    """Random block selections [B, Hkv, s] int32: ascending candidate ids, -1 padded.

    fill="random": a random count in [0, min(s, nc)]; fill="full": min(s, nc).
    """
    rng = np.random.default_rng(seed)
    sel = -np.ones((B, Hkv, s), dtype=np.int32)
    for b in range(B):
        T = int(seq_lens[b])
        nc = -(-max(0, T - w) // L)
        kmax = min(s, nc)
        for h in range(Hkv):
            k = kmax if fill == "full" else int(rng.integers(0, kmax + 1))
            pick = np.sort(rng.choice(nc, size=k, replace=False)) if k else np.zeros(0, np.int64)
            sel[b, h, :k] = pick
    return torch.from_numpy(sel)


def make_keys_block(n, d, law, seed, rank=None):
    """Keys of single blocks for statistics tests: [nblk, n, d] float32 (CPU).

    law "gauss": i.i.d. N(0,1); "lowrank": rank-`rank` plus tiny noise;
    "const": every token equal; "spiked": the c3 law.
    """
    return np.ascontiguousarray(_keys_block(n, d, law, seed, rank))


def _keys_block(n, d, law, seed, rank):
    rng = np.random.default_rng(seed)
    if law == "gauss":
        return rng.standard_normal((n, d)).astype(np.float32)
    if law == "lowrank":
        A = rng.standard_normal((d, rank))
        z = rng.standard_normal((rank, n))
        return (A @ z).T.astype(np.float32)
    if law == "const":
        return np.repeat(rng.standard_normal((1, d)), n, axis=0).astype(np.float32)
    if law == "spiked":
        A = rng.standard_normal((d, 8)) / math.sqrt(8.0)
        return ((A @ rng.standard_normal((8, n))).T + math.sqrt(0.1) * rng.standard_normal((n, d))
                + 0.3 * rng.standard_normal((1, d))).astype(np.float32)
    raise ValueError(law)


# ------------------------------------------------- queries in a subspace --
# Query law for the subspace factors: per KV head a random orthogonal d x d
# matrix R_h (Gaussian matrix, QR, columns signed so diag of the triangular
# factor is positive) and a decaying spectrum, q = R_h (sigma * z) with z
# i.i.d. N(0, 1) and sigma_j^2 = exp(-j / tau): with tau = 30 at d = 128 the
# leading 66 directions carry 90 % of the energy.  The first s' columns of R_h
# span the top-s' directions of the population second moment.

def query_rotation(Hkv, d, seed, tau=30.0):
    """(R [Hkv, d, d] float32, sigma [d] float32) of the subspace query law."""
    g = _gen("cpu", seed)
    rot = torch.empty((Hkv, d, d), dtype=torch.float64)
    for h in range(Hkv):
        a = torch.randn(d, d, generator=g, dtype=torch.float64)
        qm, rm = torch.linalg.qr(a)
        rot[h] = qm * torch.sign(torch.diagonal(rm))[None, :]
    sigma = torch.exp(-torch.arange(d, dtype=torch.float64) / (2.0 * tau))
    return rot.to(torch.float32), sigma.to(torch.float32)


def subspace_queries(rot, sigma, n, G, seed):
    """n query rows [n, Hkv * G, d] float32 of the subspace law (head h * G + g
    of row i draws from R_h)."""
    Hkv, d, _ = rot.shape
    g = _gen("cpu", seed)
    z = torch.randn(n, Hkv, G, d, generator=g, dtype=torch.float32) * sigma
    q = torch.einsum("hde,nhge->nhgd", rot, z)
    return q.reshape(n, Hkv * G, d).contiguous()

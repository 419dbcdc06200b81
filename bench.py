"""Decode-step benchmark of the COBS path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload c2] [--copies M] [--no-cpu-baseline]

One step = one cobs_decode_step call on one layer: refresh of the record of the
block holding the newest token, block scoring + top-s selection, and sparse
attention over the selected blocks plus the window, for every batch row and
KV head.  Inputs are seeded synthetic tensors resident in HBM before timing.
To measure HBM rather than the 256 MB last-level cache, the timed steps rotate
over M independent copies of the layer (K/V cache, descriptors, queries) whose
combined footprint read per step exceeds 2 GB.

Prints one JSON line: the metric (us per decode step per layer), achieved
GB/s on the step's algorithmic bytes, the roofline of the dominant kernel
(timed on its own with HIP events on the launch stream) and the fp64 oracle's
time on the host cores as a baseline.
"""

import argparse
import json
import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402
from paper_2607_09052_amd import cobs  # noqa: E402

HBM_PEAK_GBPS = 8000.0
METRIC = "µs per decode step per layer and achieved HBM GB/s (fraction of peak) at 32k ctx"
ESZ = {"f32": 4, "bf16": 2}


def vec_bytes(d, dt):
    return {"f32": 4 * d, "bf16": 2 * d, "e2m1": d // 2}[dt]


def descriptor_bytes(cfg):
    """Bytes a scorer must read per block: count, mean (+scale), r factors (+scales)."""
    d, r = cfg.head_dim, cfg.rank
    b = 4 + vec_bytes(d, cfg.mean_dtype) + (4 if cfg.mean_dtype == "e2m1" else 0)
    return b + r * vec_bytes(d, cfg.factor_dtype) + (4 * r if cfg.factor_dtype == "e2m1" else 0)


def union_tokens(T, w, sel_row, L=64):
    ws = max(0, T - w)
    nc = -(-ws // L)
    n = T - ws
    prev = -1
    for x in sel_row:
        if x < 0 or x >= nc or x <= prev:
            break
        n += min(x * L + L, ws) - x * L
        prev = x
    return n


def algorithmic_bytes(cfg, seq_lens, sel):
    """Per-kernel algorithmic bytes of one decode step, from the actual selection."""
    B, Hkv, Hq, d = cfg.batch, cfg.num_kv_heads, cfg.num_q_heads, cfg.head_dim
    kv = ESZ[cfg.kv_dtype]
    q_bytes = B * Hq * d * 4
    sel_bytes = B * Hkv * cfg.budget * 4
    out_bytes = B * Hq * (d + 1) * 4
    score = 0
    dec = 0
    tail = 0
    for b in range(B):
        T = int(seq_lens[b])
        nb = -(-T // 64)
        score += Hkv * nb * descriptor_bytes(cfg)
        n_tail = T - (T - 1) // 64 * 64
        tail += Hkv * (n_tail * d * kv + cobs.record_bytes(cfg))
        for h in range(Hkv):
            dec += union_tokens(T, cfg.window, sel[b, h].tolist()) * d * kv * 2
    return dict(select=score + q_bytes + sel_bytes, decode=dec + q_bytes + sel_bytes + out_bytes,
                tail=tail, step=score + dec + tail + q_bytes + sel_bytes + out_bytes)


def time_launches(fn, n, stream):
    """Average duration per call of `fn(i)`, HIP events on the launch stream."""
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(n):
        fn(i)
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end) * 1e3 / n          # microseconds


def cpu_baseline(prob, cfg, budget_s=12.0):
    """The fp64 oracle's decode step on the host cores, on a bounded sample.

    Untimed: the oracle builds its own descriptors for the sampled units.
    Timed per unit: refresh of the tail block's statistics, scoring, top-s
    and sparse attention.  Scaled to one full step (all units of the layer).
    """
    from oracle import method as M
    c = prob["cfg"]
    G = c["Hq"] // c["Hkv"]
    units = [(b, h) for b in range(c["B"]) for h in range(c["Hkv"])]
    T = c["T"]
    r, L = cfg.rank, 64
    prepared = []
    t_prep = time.time()
    for (b, h) in units[:2]:
        K = prob["k"][b, h, :T].to("cpu", torch.float64).numpy()
        V = prob["v"][b, h, :T].to("cpu", torch.float64).numpy()
        q = prob["q"][b, h * G:(h + 1) * G].to("cpu", torch.float64).numpy()
        stats = M.stored_statistics(*M.block_statistics(K, T, L, r), cfg.mean_dtype, cfg.factor_dtype)
        prepared.append((q, K, V, [np.array(x) for x in stats]))
    prep_s = time.time() - t_prep
    n = 0
    t0 = time.time()
    while time.time() - t0 < budget_s:
        q, K, V, stats = prepared[n % len(prepared)]
        j = (T - 1) // L
        tail = M.stored_statistics(*M.block_statistics(K[j * L:T], T - j * L, L, r),
                                   cfg.mean_dtype, cfg.factor_dtype)
        for arr, x in zip(stats, tail):
            arr[j] = x[0]
        M.decode_unit(q, K, V, T, L, r, cfg.budget, cfg.window, cfg.scale, cfg.mean_dtype,
                      cfg.factor_dtype, stats=tuple(stats))
        n += 1
    per_unit = (time.time() - t0) / n
    cores = len(os.sched_getaffinity(0))
    return {"value": per_unit * len(units) * 1e6, "unit": "us/step/layer", "cores": cores,
            "kind": "oracle",
            "sample": f"{n} unit-steps of 2 (batch row, KV head) units at T={T} in {per_unit * n:.1f} s, "
                      f"scaled x{len(units)} units; descriptor prefill ({prep_s:.1f} s) untimed; "
                      f"numpy BLAS threads = {cores} host cores"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="c2", choices=sorted(synth.CONFIGS))
    ap.add_argument("--copies", type=int, default=0, help="layer copies to rotate (0: >= 2 GB read)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--traffic", default="", help="JSON file with rocprofv3 FETCH/WRITE bytes per launch")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the decode step shards "
              "by KV head or batch row with no communication; see the design notes)", file=sys.stderr)
        sys.exit(2)

    dev = "cuda:0"
    torch.cuda.set_device(0)
    name = args.workload
    prob = synth.make_problem(name, device=dev, steps=0)
    c = prob["cfg"]
    cfg = cobs.Config(batch=c["B"], num_q_heads=c["Hq"], num_kv_heads=c["Hkv"], head_dim=c["d"],
                      max_seq_len=c["T_max"], rank=c["r"], budget=c["s"], window=c["w"],
                      kv_dtype=c["kv_dtype"], mean_dtype=c["mean_dtype"], factor_dtype=c["factor_dtype"])
    seq = prob["seq_lens"]
    rec = cobs.new_summaries(cfg, dev)
    cobs.cobs_build_block_stats(cfg, prob["k"], prob["v"], seq, rec)
    torch.cuda.synchronize()

    # bytes one step reads, then the number of independent copies to rotate
    sel0 = torch.empty((c["B"], c["Hkv"], c["s"]), dtype=torch.int32, device=dev)
    out = torch.empty((c["B"], c["Hq"], c["d"]), dtype=torch.float32, device=dev)
    lse = torch.empty((c["B"], c["Hq"]), dtype=torch.float32, device=dev)
    ws = cobs.new_workspace(cfg, cobs.OP_STEP, dev)
    cobs.cobs_decode_step(cfg, prob["q"], prob["k"], prob["v"], seq, rec, out, ws, sel=sel0, lse=lse)
    torch.cuda.synchronize()
    ab = algorithmic_bytes(cfg, seq.tolist(), sel0.cpu())
    copies = args.copies or max(2, math.ceil(2e9 / ab["step"]))
    layers = [(prob["q"], prob["k"], prob["v"], rec)]
    for _ in range(copies - 1):
        layers.append(tuple(x.clone() for x in layers[0]))
    sels = [torch.empty_like(sel0) for _ in layers]
    wss = [cobs.new_workspace(cfg, cobs.OP_STEP, dev) for _ in layers]
    stream = torch.cuda.current_stream()

    def step(i):
        q, k, v, r_ = layers[i % copies]
        cobs.cobs_decode_step(cfg, q, k, v, seq, r_, out, wss[i % copies], sel=sels[i % copies], lse=lse)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for i in range(args.steps):
        step(i)
    end.record(stream)
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / args.steps
    us_step = ms_step * 1e3

    # per-kernel durations: each entry point alone, rotating copies the same way
    sel_ws = [cobs.new_workspace(cfg, cobs.OP_SELECT, dev) for _ in layers]
    dec_ws = [cobs.new_workspace(cfg, cobs.OP_DECODE, dev) for _ in layers]
    n_k = max(args.steps, 50)

    def k_select(i):
        q, k, v, r_ = layers[i % copies]
        cobs.cobs_select(cfg, q, r_, seq, sels[i % copies], sel_ws[i % copies])

    def k_decode(i):
        q, k, v, r_ = layers[i % copies]
        cobs.cobs_sparse_decode(cfg, q, k, v, seq, sels[i % copies], out, dec_ws[i % copies], lse=lse)

    def k_tail(i):
        q, k, v, r_ = layers[i % copies]
        cobs.cobs_build_block_stats(cfg, k, v, seq, r_, first_block=cfg.num_blocks - 1, num_blocks=1)

    for fn in (k_select, k_decode, k_tail):
        for i in range(5):
            fn(i)
    kern = {"select_kernel": (time_launches(k_select, n_k, stream), ab["select"]),
            "decode_kernel": (time_launches(k_decode, n_k, stream), ab["decode"]),
            "build_stats_kernel (tail)": (time_launches(k_tail, n_k, stream), ab["tail"])}
    dom = max(kern, key=lambda k_: kern[k_][0])
    dom_us, dom_bytes = kern[dom]
    traffic = None
    if args.traffic and os.path.exists(args.traffic):
        with open(args.traffic) as f:
            traffic = json.load(f).get(dom.split()[0])

    gbps = ab["step"] / (us_step * 1e-6) / 1e9
    res = {
        "metric": METRIC,
        "value": round(us_step, 3),
        "unit": "us/step/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "achieved_gbps": round(gbps, 1),
        "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4),
        "config": {
            "workload": f"{name}: B={c['B']} Hq={c['Hq']} Hkv={c['Hkv']} d={c['d']} T={c['T']} L=64 "
                        f"r={c['r']} s={c['s']} w={c['w']} K/V {c['kv_dtype']}, descriptors "
                        f"{c['mean_dtype']} mean / {c['factor_dtype']} factors",
            "bytes_per_step": ab["step"],
            "layer_copies_rotated": copies,
            "kernels_us": {k_: round(v_[0], 3) for k_, v_ in kern.items()},
        },
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(dom_bytes / (dom_us * 1e-6) / 1e9, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(dom_bytes / (dom_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                     "traffic": traffic},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(prob, cfg)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

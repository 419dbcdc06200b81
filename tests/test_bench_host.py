"""Host-side logic of bench.py, CPU only.

The roofline figure divides algorithmic bytes by the measured kernel time, so
the byte counts are checked here against the oracle's own accounting.  The
oracle's accounting is pinned to Table "quant" and Table "bandwidth" in
test_oracle_pins.py.  The counter-summary lookup must drop a stale entry, and
the one-GPU guard must refuse several GPUs without touching a device.
"""

import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from oracle import method as M  # noqa: E402
from oracle import traffic as TR  # noqa: E402
from paper_2607_09052_amd import cobs  # noqa: E402


def _cfg(**over):
    base = dict(batch=1, num_q_heads=4, num_kv_heads=1, head_dim=128, max_seq_len=4096, rank=4,
                budget=8, window=128, kv_dtype="bf16", mean_dtype="f32", factor_dtype="f32")
    base.update(over)
    return cobs.Config(**base)


@pytest.mark.parametrize("d,r", [(128, 4), (128, 8), (64, 2), (128, 16)])
def test_descriptor_bytes_follow_the_quant_table(d, r):
    """bf16 mean with bf16 or E2M1 factors: the oracle's per-block key-summary
    bytes (mean plus factors, Table "quant"), plus the 4-byte token count."""
    for fdt, quant in (("bf16", "bf16"), ("e2m1", "fp4")):
        c = _cfg(head_dim=d, rank=r, mean_dtype="bf16", factor_dtype=fdt)
        assert bench.descriptor_bytes(c) == TR.summary_key_bytes("cobs_full", d, r, quant) + 4, (d, r, fdt)


def test_descriptor_bytes_of_the_workload_records():
    """fp32 and all-E2M1 records at d = 128, r = 4, and the d = 64, r = 2 fp32
    record: count, mean (plus its scale) and r factors (plus theirs)."""
    assert bench.descriptor_bytes(_cfg()) == 4 + 128 * 4 + 4 * 128 * 4 == 2564
    assert bench.descriptor_bytes(_cfg(mean_dtype="e2m1", factor_dtype="e2m1")) == 4 + 68 + 4 * 68 == 344
    assert bench.descriptor_bytes(_cfg(head_dim=64, rank=2)) == 4 + 256 + 2 * 256 == 772
    # a record as stored is at least as large as what the scorer reads
    for md, fd in (("f32", "f32"), ("bf16", "bf16"), ("bf16", "e2m1"), ("e2m1", "e2m1")):
        c = _cfg(mean_dtype=md, factor_dtype=fd)
        assert cobs.record_bytes(c) >= bench.descriptor_bytes(c)


def test_attended_token_count_matches_the_oracle_union():
    """The decode's byte count uses the number of tokens in window ∪ selected
    blocks; on valid selections (ascending candidates, -1 padded) it equals the
    size of the oracle's token union."""
    rng = np.random.default_rng(7)
    L, s = 64, 12
    for _ in range(400):
        T = int(rng.integers(1, 6000))
        w = int(rng.choice([0, 1, 63, 64, 100, 512, 7000]))
        nc = -(-max(0, T - w) // L)
        k = int(rng.integers(0, min(s, nc) + 1))
        row = np.full(s, -1, np.int64)
        row[:k] = np.sort(rng.choice(nc, size=k, replace=False)) if k else []
        want = len(M.union_tokens(T, L, w, row))
        assert bench.union_tokens(T, w, row.tolist()) == want, (T, w, row)


def test_traffic_lookup_drops_stale_counters(tmp_path):
    """Counter bytes are used only while the kernel sources hash as recorded."""
    good, bad = tmp_path / "good.txt", tmp_path / "bad.txt"
    body = "traffic c9 some_kernel 1000 24\n"
    good.write_text(f"source_sha256 {bench.kernel_source_hash()}\n{body}")
    bad.write_text("source_sha256 " + "0" * 64 + "\n" + body)
    assert bench.measured_traffic(str(good), "c9", "some_kernel") == 1024
    assert bench.measured_traffic(str(good), "c9", "other_kernel") is None
    assert bench.measured_traffic(str(good), "c8", "some_kernel") is None
    assert bench.measured_traffic(str(bad), "c9", "some_kernel") is None
    assert bench.measured_traffic(str(tmp_path / "missing.txt"), "c9", "some_kernel") is None


def test_bench_refuses_several_gpus():
    env = dict(os.environ, HIP_VISIBLE_DEVICES="")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, env=env, cwd=ROOT)
    assert r.returncode == 2, r.stderr[-500:]
    assert "measures one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_prefill_flops_count_the_method_not_the_iteration():
    """Sec. 5.6: Gram matrix 2 L^2 d, a dense symmetric eigenproblem (its
    tridiagonal reduction, 4 L^3 / 3) and the factors 2 L d r per full block."""
    c = _cfg(rank=4)
    ms = 1.0
    out = bench.prefill_summary(c, 1, 64 * 10, ms)
    per = 2 * 64 * 64 * 128 + 4 * 64 ** 3 / 3 + 2 * 64 * 128 * 4
    assert out["full_blocks"] == 10 and out["blocks"] == 10
    assert abs(out["method_mflop_per_block"] - per / 1e6) < 1e-3
    assert abs(out["gflops"] - 10 * per / 1e-3 / 1e9) < 0.1
    assert out["executed_mflop_per_block"] > out["method_mflop_per_block"]

"""The C-ABI library loads, exports every declared symbol, sizes records and
workspaces consistently with the documented layout, and rejects invalid
arguments on the host before touching the GPU.  CPU only: no kernel launches.
"""

import ctypes
import os
import re
import subprocess

import pytest

from oracle import records as R
from paper_2607_09052_amd import cobs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    with open(os.path.join(ROOT, "include", "cobs.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:size_t|cobs_status_t|const char\*)\s+(cobs_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    declared = _declared_functions()
    assert len(declared) == 13, declared
    lib = cobs.lib()
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(cobs.EXPORTS) == declared
    nm = subprocess.run(["nm", "-D", "--defined-only", cobs.LIB_PATH], capture_output=True, text=True)
    exported = set(re.findall(r" T (cobs_\w+)", nm.stdout))
    assert set(declared) <= exported


def _cfg(**over):
    base = dict(batch=2, num_q_heads=8, num_kv_heads=2, head_dim=128, max_seq_len=4096, rank=4,
                budget=8, window=128, kv_dtype="bf16", mean_dtype="f32", factor_dtype="f32")
    base.update(over)
    return cobs.Config(**base)


@pytest.mark.parametrize("md", ["f32", "bf16", "e2m1"])
@pytest.mark.parametrize("fd", ["f32", "bf16", "e2m1"])
@pytest.mark.parametrize("d,r", [(64, 2), (128, 4), (128, 16), (64, 0)])
@pytest.mark.parametrize("skew,vmean", [(False, False), (True, False), (False, True), (True, True)])
def test_record_bytes_match_oracle_layout(md, fd, d, r, skew, vmean):
    assert cobs.record_bytes(_cfg(head_dim=d, rank=r, mean_dtype=md, factor_dtype=fd, skew=skew,
                                  value_mean=vmean)) == R.layout(d, r, md, fd, skew, vmean)["total"]


def _basis_struct(d=128, sd=96, hkv=2, **over):
    """A config struct with subspace factors and a host stand-in basis address
    (validation only dereferences nothing)."""
    cfg = _cfg(head_dim=d, num_kv_heads=hkv, num_q_heads=4 * hkv, mean_dtype="bf16", factor_dtype="e2m1",
               **over).c_struct()
    cfg.subspace_dim = sd
    cfg.query_basis = 1 << 20
    return cfg


@pytest.mark.parametrize("md", ["bf16", "e2m1"])
@pytest.mark.parametrize("fd", ["bf16", "e2m1"])
@pytest.mark.parametrize("d,sd", [(128, 32), (128, 64), (128, 96), (64, 32)])
@pytest.mark.parametrize("skew", [False, True])
def test_subspace_record_bytes_match_oracle_layout(md, fd, d, sd, skew):
    cfg = _basis_struct(d=d, sd=sd, skew=skew)
    cfg.mean_dtype = cobs.DTYPES[md]
    cfg.factor_dtype = cobs.DTYPES[fd]
    lay = R.layout(d, 4, md, fd, skew, False, fdim=sd)
    assert cobs.lib().cobs_record_bytes(ctypes.byref(cfg)) == lay["total"]
    assert lay["vec_bytes"] == {"bf16": 2, "e2m1": 0.5}[fd] * sd


@pytest.mark.parametrize("edit,code", [
    (dict(query_basis=None), 1),          # a dimension without a basis
    (dict(subspace_dim=0), 1),            # a basis without a dimension
    (dict(subspace_dim=-32), 1),
    (dict(subspace_dim=48), 2),           # not a multiple of 32
    (dict(subspace_dim=128), 2),          # s' = d is the full space
    (dict(rank=0), 1),
    (dict(rank=8), 2),
    (dict(query_basis=(1 << 20) + 4), 1), # misaligned basis
])
def test_invalid_subspace_configs_are_rejected(edit, code):
    cfg = _basis_struct()
    for k, v in edit.items():
        setattr(cfg, k, v)
    lib = cobs.lib()
    assert lib.cobs_record_bytes(ctypes.byref(cfg)) == 0
    fake = ctypes.c_void_p(1 << 20)
    assert lib.cobs_select(ctypes.byref(cfg), fake, fake, fake, fake, None, ctypes.c_void_p(256), 1 << 30,
                           None) == code


@pytest.mark.parametrize("edit", [dict(factor_dtype=0), dict(mean_dtype=0)])
def test_subspace_scoring_needs_bf16_or_e2m1_descriptors(edit):
    """fp32 subspace records are built (record size > 0) but not scored."""
    cfg = _basis_struct()
    for k, v in edit.items():
        setattr(cfg, k, v)
    lib = cobs.lib()
    assert lib.cobs_record_bytes(ctypes.byref(cfg)) > 0
    fake = ctypes.c_void_p(1 << 20)
    assert lib.cobs_select(ctypes.byref(cfg), fake, fake, fake, fake, None, ctypes.c_void_p(256), 1 << 30,
                           None) == 2
    kv = cobs._KV(fake.value, fake.value, 0, 0, 128, None, 0)
    assert lib.cobs_decode_step(ctypes.byref(cfg), fake, ctypes.byref(kv), fake, fake, None, fake, None,
                                ctypes.c_void_p(256), 1 << 30, None) == 2


def test_binding_checks_the_basis_shape():
    import torch
    cfg = _cfg(mean_dtype="bf16", factor_dtype="e2m1", subspace_dim=96,
               query_basis=torch.zeros(2, 128, 64))
    with pytest.raises(cobs.CobsError):
        cfg.c_struct()
    ok = _cfg(mean_dtype="bf16", factor_dtype="e2m1", subspace_dim=96, query_basis=torch.zeros(2, 128, 96))
    assert cobs.record_bytes(ok) == R.layout(128, 4, "bf16", "e2m1", fdim=96)["total"]


def test_subspace_select_workspace_holds_the_projected_queries():
    full = _cfg(mean_dtype="bf16", factor_dtype="e2m1")
    sub = _basis_struct(hkv=full.num_kv_heads)
    lib = cobs.lib()
    extra = lib.cobs_workspace_bytes(ctypes.byref(sub), 1) - cobs.workspace_bytes(full, 1)
    need = 4 * full.batch * full.num_q_heads * 96
    assert need <= extra < need + 256


def test_unknown_options_and_compression_without_value_means_are_rejected():
    lib = cobs.lib()
    cfg = _cfg().c_struct()
    cfg.options = 4
    assert lib.cobs_record_bytes(ctypes.byref(cfg)) == 0
    fake = ctypes.c_void_p(1 << 20)
    plain = _cfg().c_struct()
    assert lib.cobs_compression_branch(ctypes.byref(plain), fake, fake, fake, fake, None, None) == 1
    vm = _cfg(value_mean=True).c_struct()
    assert lib.cobs_compression_branch(ctypes.byref(vm), None, fake, fake, fake, None, None) == 1


def test_workspace_sizes_are_aligned_and_ordered():
    cfg = _cfg()
    sel, dec, step = (cobs.workspace_bytes(cfg, op) for op in (1, 2, 3))
    assert cobs.workspace_bytes(cfg, 0) == 0
    assert sel % 256 == 0 and dec % 256 == 0 and step % 256 == 0
    assert step >= sel + dec
    exact = cobs.workspace_bytes(cfg, 4)
    # the exact-mass selector's scores and chunk partials (chunks of >= 4 blocks)
    assert exact % 256 == 0 and exact >= 4 * cfg.batch * cfg.num_kv_heads * 4 * cfg.num_blocks


@pytest.mark.parametrize("over,code", [
    (dict(num_q_heads=7), 1),          # Hq not a multiple of Hkv
    (dict(num_q_heads=6, num_kv_heads=2), 2),   # G = 3
    (dict(head_dim=96), 2),
    (dict(block_size=256), 2),         # L in {32, 64, 128}
    (dict(rank=17), 2),
    (dict(rank=-1), 1),
    (dict(max_seq_len=4000), 1),       # not a multiple of L
    (dict(budget=-1), 1),
    (dict(softmax_scale=-1.0), 1),
    (dict(max_seq_len=64 * 8193), 2),
])
def test_invalid_configs_are_rejected(over, code):
    cfg = _cfg(**over).c_struct()
    lib = cobs.lib()
    assert lib.cobs_record_bytes(ctypes.byref(cfg)) == 0
    st = lib.cobs_select(ctypes.byref(cfg), ctypes.c_void_p(16), ctypes.c_void_p(16), ctypes.c_void_p(16),
                         ctypes.c_void_p(16), None, ctypes.c_void_p(256), 1 << 30, None)
    assert st == code


def test_null_and_workspace_errors_on_host():
    lib = cobs.lib()
    cfg = _cfg().c_struct()
    fake = ctypes.c_void_p(1 << 20)
    # null q
    assert lib.cobs_select(ctypes.byref(cfg), None, fake, fake, fake, None, fake, 1 << 30, None) == 1
    # workspace too small / misaligned
    assert lib.cobs_select(ctypes.byref(cfg), fake, fake, fake, fake, None, fake, 16, None) == 3
    assert lib.cobs_select(ctypes.byref(cfg), fake, fake, fake, fake, None, ctypes.c_void_p((1 << 20) + 8),
                           1 << 30, None) == 3
    # misaligned KV / bad strides
    kv = cobs._KV(fake.value + 2, fake.value, 0, 0, 128, None, 0)
    assert lib.cobs_sparse_decode(ctypes.byref(cfg), fake, ctypes.byref(kv), fake, fake, fake, None, fake,
                                  1 << 30, None) == 1
    kv = cobs._KV(fake.value, fake.value, 0, 0, 100, None, 0)       # stride_t < d
    assert lib.cobs_sparse_decode(ctypes.byref(cfg), fake, ctypes.byref(kv), fake, fake, fake, None, fake,
                                  1 << 30, None) == 1
    # block range outside the cache
    kv = cobs._KV(fake.value, fake.value, 0, 0, 128, None, 0)
    assert lib.cobs_build_block_stats(ctypes.byref(cfg), ctypes.byref(kv), fake, 60, 10, fake, None, 0,
                                      None) == 1
    assert lib.cobs_pack_e2m1(fake, 4, 3, fake, fake, None) == 1
    # exact-mass selector: fp32 keys unsupported, null selection, small workspace
    kv = cobs._KV(fake.value, fake.value, 0, 0, 128, None, 0)
    cfg32 = _cfg(kv_dtype="f32").c_struct()
    assert lib.cobs_select_exact(ctypes.byref(cfg32), fake, ctypes.byref(kv), fake, fake, None, fake,
                                 1 << 30, None) == 2
    assert lib.cobs_select_exact(ctypes.byref(cfg), fake, ctypes.byref(kv), fake, None, None, fake,
                                 1 << 30, None) == 1
    assert lib.cobs_select_exact(ctypes.byref(cfg), fake, ctypes.byref(kv), fake, fake, None, fake,
                                 16, None) == 3
    assert lib.cobs_select_quest(ctypes.byref(cfg32), fake, ctypes.byref(kv), fake, fake, None, fake,
                                 1 << 30, None) == 2
    assert lib.cobs_select_quest(ctypes.byref(cfg), fake, ctypes.byref(kv), fake, fake, None, fake,
                                 16, None) == 3
    # branch outputs: fp32 K/V unsupported, a missing branch output rejected
    assert lib.cobs_sparse_decode_branches(ctypes.byref(cfg32), fake, ctypes.byref(kv), fake, fake, fake, None,
                                           fake, None, fake, 1 << 30, None) == 2
    assert lib.cobs_sparse_decode_branches(ctypes.byref(cfg), fake, ctypes.byref(kv), fake, fake, fake, None,
                                           None, None, fake, 1 << 30, None) == 1
    assert lib.cobs_status_string(3).startswith(b"COBS_ERR_WORKSPACE")


def test_binding_rejects_tensors_the_kernels_would_misread():
    """The Python binding checks dtype, contiguity, size and device of every
    tensor before calling the library (CPU tensors: the device check fires last)."""
    import torch
    cfg = _cfg(batch=2, num_q_heads=8, num_kv_heads=2, head_dim=128, max_seq_len=1024, budget=4)
    B, Hq, Hkv, d, T = 2, 8, 2, 128, 1024
    q = torch.zeros((B, Hq, d), dtype=torch.float32)
    k = torch.zeros((B, Hkv, T, d), dtype=torch.bfloat16)
    seq = torch.zeros(B, dtype=torch.int32)
    sel = torch.zeros((B, Hkv, 4), dtype=torch.int32)
    out = torch.zeros((B, Hq, d), dtype=torch.float32)
    ws = torch.zeros(1 << 20, dtype=torch.uint8)

    def rejects(fn, *a, match, **kw):
        with pytest.raises(cobs.CobsError, match=match):
            fn(*a, **kw)

    dec = cobs.cobs_sparse_decode
    rejects(dec, cfg, q.to(torch.bfloat16), k, k, seq, sel, out, ws, match="q must be")
    rejects(dec, cfg, q[:, :4].contiguous(), k, k, seq, sel, out, ws, match="q holds")
    rejects(dec, cfg, q.transpose(0, 1), k, k, seq, sel, out, ws, match="contiguous")
    rejects(dec, cfg, q, k, k, seq.to(torch.int64), sel, out, ws, match="seq_lens must be")
    rejects(dec, cfg, q, k, k, seq, sel.to(torch.int64), out, ws, match="sel must be")
    rejects(dec, cfg, q, k, k, seq, None, out, ws, match="sel is required")
    rejects(dec, cfg, q, k, k, seq, sel, out.to(torch.bfloat16), ws, match="out must be")
    rejects(dec, cfg, q, k, k, seq, sel, out, ws, lse=torch.zeros(B * Hq, dtype=torch.float64),
            match="lse must be")
    rejects(dec, cfg, q, k, k, seq, sel, out, ws, match="q must be on a GPU")
    rejects(cobs.cobs_select, cfg, q, torch.zeros(8, dtype=torch.uint8), seq, sel, ws, match="summaries holds")
    rejects(cobs.cobs_decode_step, cfg, q, k, k, seq, torch.zeros(8, dtype=torch.uint8), out, ws,
            match="summaries holds")
    rejects(cobs.cobs_pack_e2m1, torch.zeros((4, 8), dtype=torch.float64), torch.zeros((4, 4), dtype=torch.uint8),
            torch.zeros(4), match="x must be")
    rejects(dec, cfg, q, k.to(torch.float32), k.to(torch.float32), seq, sel, out, ws, match="kv_dtype")
    rejects(dec, cfg, q, k[..., :64], k[..., :64], seq, sel, out, ws, match="dense head dimension")
    rejects(dec, cfg, q, k[:, :, :512], k[:, :, :512], seq, sel, out, ws, match="smaller than")
    rejects(dec, cfg, q, k, k, seq, sel, out, ws, block_table=torch.zeros((B, 16), dtype=torch.int32),
            num_pages=4, match="paged k must be")


def test_noalloc_step_rejects_problems_beyond_its_scratch():
    """cobs_decode_step_noalloc refuses, on the host, a problem whose step
    workspace exceeds the library's per-GPU array."""
    lib = cobs.lib()
    fake = ctypes.c_void_p(1 << 20)
    kv = cobs._KV(fake.value, fake.value, 1 << 24, 1 << 21, 128, None, 0)
    big = _cfg(batch=64, num_q_heads=64, num_kv_heads=8, max_seq_len=131072, budget=85, window=1024,
               mean_dtype="e2m1", factor_dtype="e2m1")
    assert cobs.workspace_bytes(big, cobs.OP_STEP) > 32 << 20
    assert lib.cobs_decode_step_noalloc(ctypes.byref(big.c_struct()), fake, ctypes.byref(kv), fake, fake, None,
                                        fake, None, None) == 3
    assert lib.cobs_decode_step_noalloc(ctypes.byref(_cfg().c_struct()), None, ctypes.byref(kv), fake, fake,
                                        None, fake, None, None) == 1


@pytest.mark.parametrize("L,s,w", [(32, 1, 64), (32, 1, 1), (64, 1, 1), (128, 1, 1), (32, 0, 64), (32, 5, 0)])
def test_decode_workspace_holds_a_partial_per_branch(L, s, w):
    """The two-branch decode needs one partial per non-empty branch: the decode
    workspace holds at least two per unit whenever both budget and window are
    positive, at every block length."""
    cfg = _cfg(batch=1, num_q_heads=8, num_kv_heads=1, max_seq_len=2048, block_size=L, budget=s, window=w)
    G, d = 8, cfg.head_dim
    least = 2 if (s > 0 and w > 0) else 1
    assert cobs.workspace_bytes(cfg, cobs.OP_DECODE) >= least * G * (d + 2) * 4 + 4

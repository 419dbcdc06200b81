"""Thin Python binding of libcobs.so (the COBS decode-step C ABI, include/cobs.h).

Argument marshalling only: every stage runs in the library's HIP kernels.
Tensors are torch tensors on the GPU; torch supplies device memory and the
stream (the current stream of the tensors' device, unless one is passed).
A missing library raises at import of this module's functions' first use -
there is no other implementation to fall back to.
"""

import ctypes
import dataclasses
import math
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcobs.so")

F32, BF16, E2M1 = 0, 1, 2
DTYPES = {"f32": F32, "bf16": BF16, "e2m1": E2M1}
OP_BUILD, OP_SELECT, OP_DECODE, OP_STEP, OP_SELECT_EXACT = 0, 1, 2, 3, 4
OPT_SKEW, OPT_VALUE_MEAN = 1, 2
BLOCK = 64


class CobsError(RuntimeError):
    pass


class _Config(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("max_seq_len", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("rank", ctypes.c_int32), ("budget", ctypes.c_int32), ("window", ctypes.c_int32),
                ("kv_dtype", ctypes.c_int), ("mean_dtype", ctypes.c_int),
                ("factor_dtype", ctypes.c_int), ("softmax_scale", ctypes.c_float),
                ("options", ctypes.c_int32), ("subspace_dim", ctypes.c_int32),
                ("query_basis", ctypes.c_void_p)]


class _KV(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("stride_b", ctypes.c_int64),
                ("stride_h", ctypes.c_int64), ("stride_t", ctypes.c_int64),
                ("block_table", ctypes.c_void_p), ("num_pages", ctypes.c_int64)]


_P = ctypes.c_void_p
_SIGS = {
    "cobs_record_bytes": (ctypes.c_size_t, [_P]),
    "cobs_workspace_bytes": (ctypes.c_size_t, [_P, ctypes.c_int]),
    "cobs_build_block_stats": (ctypes.c_int, [_P, _P, _P, ctypes.c_int32, ctypes.c_int32, _P, _P,
                                              ctypes.c_size_t, _P]),
    "cobs_select": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "cobs_select_exact": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "cobs_select_quest": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "cobs_sparse_decode": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "cobs_sparse_decode_branches": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "cobs_decode_step": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "cobs_decode_step_noalloc": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "cobs_compression_branch": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P]),
    "cobs_pack_e2m1": (ctypes.c_int, [_P, ctypes.c_int64, ctypes.c_int32, _P, _P, _P]),
    "cobs_status_string": (ctypes.c_char_p, [ctypes.c_int]),
}
EXPORTS = tuple(_SIGS)

_lib = None


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise CobsError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_09052_amd.build`")
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        _lib = h
    return _lib


@dataclasses.dataclass
class Config:
    """Problem description (cobs_config_t)."""
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    max_seq_len: int
    rank: int
    budget: int
    window: int
    kv_dtype: str = "bf16"
    mean_dtype: str = "f32"
    factor_dtype: str = "f32"
    softmax_scale: float = 0.0
    block_size: int = BLOCK
    skew: bool = False           # records carry the diagonal third-cumulant coefficients
    value_mean: bool = False     # records carry the block's mean value (compression branch)
    subspace_dim: int = 0        # subspace factors of this many elements (Sec. 5.4); 0: full space
    # U_Q of every KV head for subspace factors: fp32 [Hkv, d, subspace_dim] on the GPU
    query_basis: object = dataclasses.field(default=None, compare=False, repr=False)

    @property
    def options(self):
        return (OPT_SKEW if self.skew else 0) | (OPT_VALUE_MEAN if self.value_mean else 0)

    def c_struct(self):
        basis = None
        if self.query_basis is not None:
            want = (self.num_kv_heads, self.head_dim, self.subspace_dim)
            _need("query_basis", self.query_basis, torch.float32, math.prod(want))
            if tuple(self.query_basis.shape) != want:
                raise CobsError(f"query_basis must have shape {list(want)}, got {list(self.query_basis.shape)}")
            basis = self.query_basis.data_ptr()
        return _Config(self.batch, self.num_q_heads, self.num_kv_heads, self.head_dim,
                       self.max_seq_len, self.block_size, self.rank, self.budget, self.window,
                       DTYPES[self.kv_dtype], DTYPES[self.mean_dtype], DTYPES[self.factor_dtype],
                       float(self.softmax_scale), self.options, int(self.subspace_dim), basis)

    @property
    def num_blocks(self):
        return self.max_seq_len // self.block_size

    @property
    def scale(self):
        return self.softmax_scale if self.softmax_scale > 0 else 1.0 / math.sqrt(self.head_dim)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream, dev_tensor):
    if stream is not None:
        return ctypes.c_void_p(stream if isinstance(stream, int) else stream.cuda_stream)
    return ctypes.c_void_p(torch.cuda.current_stream(dev_tensor.device).cuda_stream)


def _check(status):
    if status != 0:
        msg = lib().cobs_status_string(status).decode()
        raise CobsError(msg)


_TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}


def _need(name, t, dtype, numel):
    """Reject a tensor the kernels would misread: wrong dtype, not contiguous,
    or fewer elements than the call reads or writes.  Returns it."""
    if t is None:
        raise CobsError(f"{name} is required")
    if t.dtype != dtype:
        raise CobsError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise CobsError(f"{name} must be contiguous")
    if t.numel() < numel:
        raise CobsError(f"{name} holds {t.numel()} elements, the call needs {numel}")
    return t


def _opt(name, t, dtype, numel):
    return None if t is None else _need(name, t, dtype, numel)


def _same_gpu(**tensors):
    """Every given tensor on one GPU (checked after the shapes and types)."""
    dev = None
    for name, t in tensors.items():
        if t is None:
            continue
        if not t.is_cuda:
            raise CobsError(f"{name} must be on a GPU")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise CobsError(f"{name} is on {t.device}, the call runs on {dev}")


def _kv(cfg, k, v, block_table=None, num_pages=0):
    """Validated K/V view (contiguous [>=B, >=Hkv, >=T_max, d] with the head
    dimension dense, or pages [num_pages, Hkv, L, d] with a [B, T_max/L] table)."""
    want = _TORCH_DTYPE[cfg.kv_dtype]
    for name, t in (("k", k), ("v", v)):
        if t is None or t.dtype != want:
            raise CobsError(f"{name} must be {want} (kv_dtype {cfg.kv_dtype})")
        if t.dim() != 4 or t.shape[-1] != cfg.head_dim or t.stride(-1) != 1:
            raise CobsError(f"{name} must be 4-D with a dense head dimension of {cfg.head_dim}")
    if block_table is not None:
        for name, t in (("k", k), ("v", v)):
            if tuple(t.shape[1:]) != (cfg.num_kv_heads, cfg.block_size, cfg.head_dim) or not t.is_contiguous():
                raise CobsError(f"paged {name} must be a contiguous [pages, Hkv, L, d] pool")
            if not 1 <= int(num_pages) <= t.shape[0]:
                raise CobsError(f"num_pages must lie in [1, {t.shape[0]}]")
        _need("block_table", block_table, torch.int32, cfg.batch * cfg.num_blocks)
        return _KV(k.data_ptr(), v.data_ptr(), 0, 0, 0, block_table.data_ptr(), int(num_pages))
    if k.stride() != v.stride() or k.shape != v.shape:
        raise CobsError("K and V must share shape and strides")
    if k.shape[0] < cfg.batch or k.shape[1] < cfg.num_kv_heads or k.shape[2] < cfg.max_seq_len:
        raise CobsError(f"K/V of shape {tuple(k.shape)} is smaller than "
                        f"[{cfg.batch}, {cfg.num_kv_heads}, {cfg.max_seq_len}, {cfg.head_dim}]")
    return _KV(k.data_ptr(), v.data_ptr(), k.stride(0), k.stride(1), k.stride(2), None, 0)


def _units(cfg):
    return cfg.batch * cfg.num_kv_heads


def _ws(ws):
    """Workspace tensor (any element type, contiguous) and its size in bytes."""
    if ws is None:
        raise CobsError("ws is required")
    if not ws.is_contiguous():
        raise CobsError("ws must be contiguous")
    return ws.numel() * ws.element_size()


def _summaries(cfg, summaries):
    return _need("summaries", summaries, torch.uint8, _units(cfg) * cfg.num_blocks * record_bytes(cfg))


def record_bytes(cfg):
    return int(lib().cobs_record_bytes(ctypes.byref(cfg.c_struct())))


def workspace_bytes(cfg, op):
    return int(lib().cobs_workspace_bytes(ctypes.byref(cfg.c_struct()), int(op)))


def new_workspace(cfg, op, device):
    """Zero-filled workspace for `op` (the library requires zeros before first use)."""
    n = workspace_bytes(cfg, op)
    return torch.zeros(max(n, 256), dtype=torch.uint8, device=device)


def new_summaries(cfg, device):
    return torch.zeros((cfg.batch, cfg.num_kv_heads, cfg.num_blocks, record_bytes(cfg)),
                       dtype=torch.uint8, device=device)


def cobs_build_block_stats(cfg, k, v, seq_lens, summaries, first_block=0, num_blocks=None,
                           ws=None, block_table=None, num_pages=0, stream=None):
    if num_blocks is None:
        num_blocks = cfg.num_blocks - first_block
    _need("seq_lens", seq_lens, torch.int32, cfg.batch)
    _summaries(cfg, summaries)
    kv = _kv(cfg, k, v, block_table, num_pages)
    _same_gpu(seq_lens=seq_lens, summaries=summaries, k=k, v=v, block_table=block_table,
              query_basis=cfg.query_basis)
    _check(lib().cobs_build_block_stats(ctypes.byref(cfg.c_struct()), ctypes.byref(kv),
                                        _ptr(seq_lens), int(first_block), int(num_blocks),
                                        _ptr(summaries), _ptr(ws),
                                        0 if ws is None else ws.numel() * ws.element_size(),
                                        _stream(stream, summaries)))


def _select_io(cfg, q, seq_lens, sel, scores):
    _need("q", q, torch.float32, cfg.batch * cfg.num_q_heads * cfg.head_dim)
    _need("seq_lens", seq_lens, torch.int32, cfg.batch)
    _need("sel", sel, torch.int32, _units(cfg) * cfg.budget)
    _opt("scores", scores, torch.float32, _units(cfg) * cfg.num_blocks)


def cobs_select(cfg, q, summaries, seq_lens, sel, ws, scores=None, stream=None):
    _select_io(cfg, q, seq_lens, sel, scores)
    _summaries(cfg, summaries)
    nws = _ws(ws)
    _same_gpu(q=q, summaries=summaries, seq_lens=seq_lens, sel=sel, scores=scores, ws=ws,
              query_basis=cfg.query_basis)
    _check(lib().cobs_select(ctypes.byref(cfg.c_struct()), _ptr(q), _ptr(summaries),
                             _ptr(seq_lens), _ptr(sel), _ptr(scores), _ptr(ws), nws, _stream(stream, q)))


def _dense_key_select(fn, cfg, q, k, v, seq_lens, sel, ws, scores, block_table, num_pages, stream):
    _select_io(cfg, q, seq_lens, sel, scores)
    kv = _kv(cfg, k, v, block_table, num_pages)
    nws = _ws(ws)
    _same_gpu(q=q, k=k, v=v, seq_lens=seq_lens, sel=sel, scores=scores, ws=ws, block_table=block_table)
    _check(fn(ctypes.byref(cfg.c_struct()), _ptr(q), ctypes.byref(kv), _ptr(seq_lens), _ptr(sel), _ptr(scores),
              _ptr(ws), nws, _stream(stream, q)))


def cobs_select_exact(cfg, q, k, v, seq_lens, sel, ws, scores=None, block_table=None, num_pages=0,
                      stream=None):
    _dense_key_select(lib().cobs_select_exact, cfg, q, k, v, seq_lens, sel, ws, scores, block_table, num_pages,
                      stream)


def cobs_select_quest(cfg, q, k, v, seq_lens, sel, ws, scores=None, block_table=None, num_pages=0,
                      stream=None):
    _dense_key_select(lib().cobs_select_quest, cfg, q, k, v, seq_lens, sel, ws, scores, block_table, num_pages,
                      stream)


def _decode_io(cfg, q, seq_lens, sel, outs, lses, sel_required=True):
    _need("q", q, torch.float32, cfg.batch * cfg.num_q_heads * cfg.head_dim)
    _need("seq_lens", seq_lens, torch.int32, cfg.batch)
    if (sel_required and cfg.budget > 0) or sel is not None:
        _need("sel", sel, torch.int32, _units(cfg) * cfg.budget)
    for name, o in outs.items():
        _need(name, o, torch.float32, cfg.batch * cfg.num_q_heads * cfg.head_dim)
    for name, l in lses.items():
        _opt(name, l, torch.float32, cfg.batch * cfg.num_q_heads)


def cobs_sparse_decode(cfg, q, k, v, seq_lens, sel, out, ws, lse=None, block_table=None,
                       num_pages=0, stream=None):
    _decode_io(cfg, q, seq_lens, sel, dict(out=out), dict(lse=lse))
    kv = _kv(cfg, k, v, block_table, num_pages)
    nws = _ws(ws)
    _same_gpu(q=q, k=k, v=v, seq_lens=seq_lens, sel=sel, out=out, lse=lse, ws=ws, block_table=block_table)
    _check(lib().cobs_sparse_decode(ctypes.byref(cfg.c_struct()), _ptr(q), ctypes.byref(kv),
                                    _ptr(seq_lens), _ptr(sel), _ptr(out), _ptr(lse), _ptr(ws), nws,
                                    _stream(stream, q)))


def cobs_sparse_decode_branches(cfg, q, k, v, seq_lens, sel, out_sel, out_win, ws, lse_sel=None, lse_win=None,
                                block_table=None, num_pages=0, stream=None):
    _decode_io(cfg, q, seq_lens, sel, dict(out_sel=out_sel, out_win=out_win), dict(lse_sel=lse_sel, lse_win=lse_win))
    kv = _kv(cfg, k, v, block_table, num_pages)
    nws = _ws(ws)
    _same_gpu(q=q, k=k, v=v, seq_lens=seq_lens, sel=sel, out_sel=out_sel, out_win=out_win, lse_sel=lse_sel,
              lse_win=lse_win, ws=ws, block_table=block_table)
    _check(lib().cobs_sparse_decode_branches(ctypes.byref(cfg.c_struct()), _ptr(q), ctypes.byref(kv),
                                             _ptr(seq_lens), _ptr(sel), _ptr(out_sel), _ptr(lse_sel),
                                             _ptr(out_win), _ptr(lse_win), _ptr(ws), nws, _stream(stream, q)))


def cobs_decode_step(cfg, q, k, v, seq_lens, summaries, out, ws, sel=None, lse=None,
                     block_table=None, num_pages=0, stream=None):
    _decode_io(cfg, q, seq_lens, sel, dict(out=out), dict(lse=lse), sel_required=False)
    _summaries(cfg, summaries)
    kv = _kv(cfg, k, v, block_table, num_pages)
    nws = _ws(ws)
    _same_gpu(q=q, k=k, v=v, seq_lens=seq_lens, summaries=summaries, sel=sel, out=out, lse=lse, ws=ws,
              block_table=block_table, query_basis=cfg.query_basis)
    _check(lib().cobs_decode_step(ctypes.byref(cfg.c_struct()), _ptr(q), ctypes.byref(kv),
                                  _ptr(seq_lens), _ptr(summaries), _ptr(sel), _ptr(out), _ptr(lse),
                                  _ptr(ws), nws, _stream(stream, q)))


def cobs_decode_step_noalloc(cfg, q, k, v, seq_lens, summaries, out, sel=None, lse=None,
                             block_table=None, num_pages=0, stream=None):
    """cobs_decode_step on the library's own per-GPU workspace (no ws argument)."""
    _decode_io(cfg, q, seq_lens, sel, dict(out=out), dict(lse=lse), sel_required=False)
    _summaries(cfg, summaries)
    kv = _kv(cfg, k, v, block_table, num_pages)
    _same_gpu(q=q, k=k, v=v, seq_lens=seq_lens, summaries=summaries, sel=sel, out=out, lse=lse,
              block_table=block_table, query_basis=cfg.query_basis)
    _check(lib().cobs_decode_step_noalloc(ctypes.byref(cfg.c_struct()), _ptr(q), ctypes.byref(kv),
                                          _ptr(seq_lens), _ptr(summaries), _ptr(sel), _ptr(out), _ptr(lse),
                                          _stream(stream, q)))


def cobs_compression_branch(cfg, q, summaries, seq_lens, out, lse=None, stream=None):
    """The mean-pool compression branch over value-mean records (cfg.value_mean)."""
    _need("q", q, torch.float32, cfg.batch * cfg.num_q_heads * cfg.head_dim)
    _need("seq_lens", seq_lens, torch.int32, cfg.batch)
    _summaries(cfg, summaries)
    _need("out", out, torch.float32, cfg.batch * cfg.num_q_heads * cfg.head_dim)
    _opt("lse", lse, torch.float32, cfg.batch * cfg.num_q_heads)
    _same_gpu(q=q, summaries=summaries, seq_lens=seq_lens, out=out, lse=lse)
    _check(lib().cobs_compression_branch(ctypes.byref(cfg.c_struct()), _ptr(q), _ptr(summaries), _ptr(seq_lens),
                                         _ptr(out), _ptr(lse), _stream(stream, q)))


def cobs_pack_e2m1(x, codes, scales, stream=None):
    if x is None or x.dim() != 2:
        raise CobsError("x must be a 2-D [num_vectors, dim] tensor")
    n, dim = x.shape
    _need("x", x, torch.float32, n * dim)
    _need("codes", codes, torch.uint8, n * (dim // 2))
    _need("scales", scales, torch.float32, n)
    _same_gpu(x=x, codes=codes, scales=scales)
    _check(lib().cobs_pack_e2m1(_ptr(x), int(n), int(dim), _ptr(codes), _ptr(scales),
                                _stream(stream, x)))

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
BLOCK = 64


class CobsError(RuntimeError):
    pass


class _Config(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("max_seq_len", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("rank", ctypes.c_int32), ("budget", ctypes.c_int32), ("window", ctypes.c_int32),
                ("kv_dtype", ctypes.c_int), ("mean_dtype", ctypes.c_int),
                ("factor_dtype", ctypes.c_int), ("softmax_scale", ctypes.c_float)]


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

    def c_struct(self):
        return _Config(self.batch, self.num_q_heads, self.num_kv_heads, self.head_dim,
                       self.max_seq_len, self.block_size, self.rank, self.budget, self.window,
                       DTYPES[self.kv_dtype], DTYPES[self.mean_dtype], DTYPES[self.factor_dtype],
                       float(self.softmax_scale))

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


def _kv(k, v, block_table=None, num_pages=0):
    if block_table is not None:
        return _KV(k.data_ptr(), v.data_ptr(), 0, 0, 0, block_table.data_ptr(), int(num_pages))
    if k.stride() != v.stride():
        raise CobsError("K and V must share strides")
    if k.stride(-1) != 1:
        raise CobsError("the head dimension of K/V must be contiguous")
    return _KV(k.data_ptr(), v.data_ptr(), k.stride(0), k.stride(1), k.stride(2), None, 0)


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
    kv = _kv(k, v, block_table, num_pages)
    _check(lib().cobs_build_block_stats(ctypes.byref(cfg.c_struct()), ctypes.byref(kv),
                                        _ptr(seq_lens), int(first_block), int(num_blocks),
                                        _ptr(summaries), _ptr(ws),
                                        0 if ws is None else ws.numel() * ws.element_size(),
                                        _stream(stream, summaries)))


def cobs_select(cfg, q, summaries, seq_lens, sel, ws, scores=None, stream=None):
    _check(lib().cobs_select(ctypes.byref(cfg.c_struct()), _ptr(q), _ptr(summaries),
                             _ptr(seq_lens), _ptr(sel), _ptr(scores), _ptr(ws),
                             ws.numel() * ws.element_size(), _stream(stream, q)))


def cobs_select_exact(cfg, q, k, v, seq_lens, sel, ws, scores=None, block_table=None, num_pages=0,
                      stream=None):
    kv = _kv(k, v, block_table, num_pages)
    _check(lib().cobs_select_exact(ctypes.byref(cfg.c_struct()), _ptr(q), ctypes.byref(kv),
                                   _ptr(seq_lens), _ptr(sel), _ptr(scores), _ptr(ws),
                                   ws.numel() * ws.element_size(), _stream(stream, q)))


def cobs_select_quest(cfg, q, k, v, seq_lens, sel, ws, scores=None, block_table=None, num_pages=0,
                      stream=None):
    kv = _kv(k, v, block_table, num_pages)
    _check(lib().cobs_select_quest(ctypes.byref(cfg.c_struct()), _ptr(q), ctypes.byref(kv),
                                   _ptr(seq_lens), _ptr(sel), _ptr(scores), _ptr(ws),
                                   ws.numel() * ws.element_size(), _stream(stream, q)))


def cobs_sparse_decode(cfg, q, k, v, seq_lens, sel, out, ws, lse=None, block_table=None,
                       num_pages=0, stream=None):
    kv = _kv(k, v, block_table, num_pages)
    _check(lib().cobs_sparse_decode(ctypes.byref(cfg.c_struct()), _ptr(q), ctypes.byref(kv),
                                    _ptr(seq_lens), _ptr(sel), _ptr(out), _ptr(lse), _ptr(ws),
                                    ws.numel() * ws.element_size(), _stream(stream, q)))


def cobs_sparse_decode_branches(cfg, q, k, v, seq_lens, sel, out_sel, out_win, ws, lse_sel=None, lse_win=None,
                                block_table=None, num_pages=0, stream=None):
    kv = _kv(k, v, block_table, num_pages)
    _check(lib().cobs_sparse_decode_branches(ctypes.byref(cfg.c_struct()), _ptr(q), ctypes.byref(kv),
                                             _ptr(seq_lens), _ptr(sel), _ptr(out_sel), _ptr(lse_sel),
                                             _ptr(out_win), _ptr(lse_win), _ptr(ws),
                                             ws.numel() * ws.element_size(), _stream(stream, q)))


def cobs_decode_step(cfg, q, k, v, seq_lens, summaries, out, ws, sel=None, lse=None,
                     block_table=None, num_pages=0, stream=None):
    kv = _kv(k, v, block_table, num_pages)
    _check(lib().cobs_decode_step(ctypes.byref(cfg.c_struct()), _ptr(q), ctypes.byref(kv),
                                  _ptr(seq_lens), _ptr(summaries), _ptr(sel), _ptr(out), _ptr(lse),
                                  _ptr(ws), ws.numel() * ws.element_size(), _stream(stream, q)))


def cobs_pack_e2m1(x, codes, scales, stream=None):
    n, dim = x.shape
    _check(lib().cobs_pack_e2m1(_ptr(x), int(n), int(dim), _ptr(codes), _ptr(scales),
                                _stream(stream, x)))

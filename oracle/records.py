"""Per-block descriptor record byte layout (oracle side).

The cached, query-independent block summary of Sec. 5.3/5.5 is the token
count, the mean key and the r scaled eigenvectors xi_i.  Two optional parts
extend it: the diagonal third-cumulant coefficients of Sec. 7.7 (one fp32
scalar per factor), and the mean value of the block's tokens (the pooled value
of the mean-pool compression branch, Sec. 2 and Sec. 5.2).  One record per
block, all offsets in bytes, little-endian, every record 16-byte aligned:

  0              int32    n_b, tokens in the block
  4              float32  scale of the mean (E2M1 mean only, else 0)
  8              float32  scale of the value mean (E2M1 value mean only, else 0)
  12             4 bytes  zero
  16             float32  scale of factor i, i < r (E2M1 factors only),
                          zero-padded to a multiple of 16 bytes
  S              float32  skew coefficient of factor i, i < r (skew records
                          only), zero-padded to a multiple of 16 bytes
  M              mean, d elements of the mean dtype
  F = M + |mean| factors, r vectors of d elements of the factor dtype (of s
                          elements for subspace factors, Sec. 5.4), vector i
                          at F + i * |vector|
  V = F + r|vec| value mean, d elements of the mean dtype (value-mean
                          records only)
  total          rounded up to a multiple of 16 bytes

Element sizes: f32 4 B, bf16 2 B, e2m1 half a byte (element 2j in the low
nibble of byte j).  The HIP library implements the same layout independently.
This module is test infrastructure (see the package docstring).
"""

import numpy as np

from . import numerics as nx

DTYPES = ("f32", "bf16", "e2m1")


def _vec_bytes(d, dtype):
    return {"f32": 4 * d, "bf16": 2 * d, "e2m1": d // 2}[dtype]


def _round16(x):
    return (x + 15) // 16 * 16


def layout(d, r, mean_dtype, factor_dtype, skew=False, value_mean=False, fdim=None):
    """Offsets and total size of one record (factor vectors of fdim elements,
    d unless given)."""
    assert mean_dtype in DTYPES and factor_dtype in DTYPES
    fscale_bytes = _round16(4 * r) if factor_dtype == "e2m1" else 0
    skew_off = 16 + fscale_bytes
    mean_off = skew_off + (_round16(4 * r) if skew else 0)
    mean_bytes = _vec_bytes(d, mean_dtype)
    fac_off = mean_off + mean_bytes
    vec_bytes = _vec_bytes(d if fdim is None else fdim, factor_dtype)
    vmean_off = fac_off + r * vec_bytes
    total = _round16(vmean_off + (mean_bytes if value_mean else 0))
    return dict(mean_off=mean_off, mean_bytes=mean_bytes, fac_off=fac_off,
                vec_bytes=vec_bytes, skew_off=skew_off, vmean_off=vmean_off, total=total)


def algorithmic_bytes(d, r, mean_dtype, factor_dtype, skew=False, fdim=None):
    """Bytes a scorer must read per block, without layout padding.

    int32 count, the mean (plus its fp32 scale if E2M1) and the r factors
    (plus one fp32 scale each if E2M1), as counted by Table "quant"; with the
    skew term, one more fp32 scalar per factor.
    """
    b = 4 + _vec_bytes(d, mean_dtype) + (4 if mean_dtype == "e2m1" else 0)
    b += r * _vec_bytes(d if fdim is None else fdim, factor_dtype) + (4 * r if factor_dtype == "e2m1" else 0)
    return b + (4 * r if skew else 0)


def _encode_vectors(v, dtype):
    """Return (bytes [..., vec_bytes], scales or None) for float64 vectors v [..., d]."""
    if dtype == "f32":
        return v.astype(np.float32).view(np.uint8).reshape(v.shape[:-1] + (-1,)), None
    if dtype == "bf16":
        bits = nx.bf16_bits(nx.round_bf16(v))
        return bits.view(np.uint8).reshape(v.shape[:-1] + (-1,)), None
    codes, scales = nx.e2m1_encode(v)
    return nx.pack_nibbles(codes), scales


def _decode_vectors(raw, d, dtype, scales=None):
    lead = raw.shape[:-1]
    if dtype == "f32":
        return np.ascontiguousarray(raw).view(np.float32).reshape(lead + (d,)).astype(np.float64)
    if dtype == "bf16":
        return nx.bf16_from_bits(np.ascontiguousarray(raw).view(np.uint16).reshape(lead + (d,)))
    codes = nx.unpack_nibbles(raw)
    return nx.e2m1_decode(codes, scales)


def encode(counts, means, factors, mean_dtype, factor_dtype, skews=None, vmeans=None):
    """Encode float64 statistics into records.

    counts [NB], means [NB, d], factors [NB, r, d], optional skew coefficients
    [NB, r] and value means [NB, d]  ->  uint8 [NB, total].
    """
    counts = np.asarray(counts)
    means = np.asarray(means, dtype=np.float64)
    factors = np.asarray(factors, dtype=np.float64)
    nb, d = means.shape
    r, fdim = factors.shape[1], factors.shape[2]
    lay = layout(d, r, mean_dtype, factor_dtype, skews is not None, vmeans is not None, fdim)
    out = np.zeros((nb, lay["total"]), dtype=np.uint8)
    out[:, 0:4] = counts.astype(np.int32).view(np.uint8).reshape(nb, 4)
    mraw, mscale = _encode_vectors(means, mean_dtype)
    out[:, lay["mean_off"]:lay["mean_off"] + lay["mean_bytes"]] = mraw
    if mscale is not None:
        out[:, 4:8] = mscale.astype(np.float32).view(np.uint8).reshape(nb, 4)
    if r > 0:
        fraw, fscale = _encode_vectors(factors, factor_dtype)
        out[:, lay["fac_off"]:lay["fac_off"] + r * lay["vec_bytes"]] = fraw.reshape(nb, -1)
        if fscale is not None:
            out[:, 16:16 + 4 * r] = fscale.astype(np.float32).view(np.uint8).reshape(nb, 4 * r)
    if skews is not None and r > 0:
        sk = np.ascontiguousarray(np.asarray(skews, dtype=np.float64).astype(np.float32))
        out[:, lay["skew_off"]:lay["skew_off"] + 4 * r] = sk.view(np.uint8).reshape(nb, 4 * r)
    if vmeans is not None:
        vraw, vscale = _encode_vectors(np.asarray(vmeans, dtype=np.float64), mean_dtype)
        out[:, lay["vmean_off"]:lay["vmean_off"] + lay["mean_bytes"]] = vraw
        if vscale is not None:
            out[:, 8:12] = vscale.astype(np.float32).view(np.uint8).reshape(nb, 4)
    return out


def decode(buf, d, r, mean_dtype, factor_dtype, skew=False, value_mean=False, fdim=None):
    """Decode records uint8 [NB, total] -> (counts int64 [NB], means [NB, d], factors [NB, r, d]),
    followed by the skew coefficients [NB, r] and the value means [NB, d] (None
    where absent) when either optional part is asked for."""
    buf = np.ascontiguousarray(np.asarray(buf, dtype=np.uint8))
    lay = layout(d, r, mean_dtype, factor_dtype, skew, value_mean, fdim)
    fd = d if fdim is None else fdim
    assert buf.shape[-1] == lay["total"], (buf.shape, lay)
    nb = buf.shape[0]
    counts = np.ascontiguousarray(buf[:, 0:4]).view(np.int32).reshape(nb).astype(np.int64)
    mscale = np.ascontiguousarray(buf[:, 4:8]).view(np.float32).reshape(nb)
    mraw = buf[:, lay["mean_off"]:lay["mean_off"] + lay["mean_bytes"]]
    means = _decode_vectors(mraw, d, mean_dtype, mscale)
    if r == 0:
        factors = np.zeros((nb, 0, fd))
    else:
        fraw = buf[:, lay["fac_off"]:lay["fac_off"] + r * lay["vec_bytes"]].reshape(nb, r, lay["vec_bytes"])
        fscale = None
        if factor_dtype == "e2m1":
            fscale = np.ascontiguousarray(buf[:, 16:16 + 4 * r]).view(np.float32).reshape(nb, r)
        factors = _decode_vectors(fraw, fd, factor_dtype, fscale)
    if not (skew or value_mean):
        return counts, means, factors
    skews = vmeans = None
    if skew:
        skews = np.ascontiguousarray(buf[:, lay["skew_off"]:lay["skew_off"] + 4 * r]).view(np.float32)
        skews = skews.reshape(nb, r).astype(np.float64)
    if value_mean:
        vscale = np.ascontiguousarray(buf[:, 8:12]).view(np.float32).reshape(nb)
        vmeans = _decode_vectors(buf[:, lay["vmean_off"]:lay["vmean_off"] + lay["mean_bytes"]], d, mean_dtype,
                                 vscale)
    return counts, means, factors, skews, vmeans

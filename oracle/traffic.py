"""KV-cache read traffic per decode step and layer (oracle side).

Written from the accounting of Sec. 7.5 (Table "bandwidth") and the
descriptor sizes of Table "quant": per layer, H KV heads of dimension D, a
context of T tokens in blocks of L, top-k selected blocks, a window of w
tokens, bf16 K/V (2 bytes per element).  Each branch reads

  summary keys     T/L * H * (per-block key-summary bytes)
  summary values   T/L * H * D * 2          (bf16 mean of the values)
  window           w * H * D * 2 * 2        (K and V)
  fine grained     k * L * H * D * 2 * 2    (K and V of the selected blocks)

Dense reads T * H * D * 2 * 2; OSA additionally re-reads every key.
This module is test infrastructure (see the package docstring).
"""

KIB = 1024


def factor_bytes(r, dim, quant):
    """Covariance-factor bytes per block: r vectors of `dim` entries (Table "quant").

    bf16: 2 bytes per entry.  fp4 (E2M1): half a byte per entry plus one fp32
    scale per vector (Sec. 5.5).
    """
    if quant == "bf16":
        return r * dim * 2
    if quant == "fp4":
        return r * dim / 2 + 4 * r
    raise ValueError(quant)


def summary_key_bytes(method, D, r=None, quant=None, sub_dim=None):
    """Per-block key-summary bytes read by each selector of Table "bandwidth"."""
    mean = D * 2                                   # bf16 mean key
    if method in ("nsa_mlp", "nsa_meanpool"):
        return mean
    if method == "nsa_quest":                      # mean + per-channel min and max
        return 3 * mean
    if method == "cobs_full":
        return mean + factor_bytes(r, D, quant)
    if method == "cobs_subspace":
        return mean + factor_bytes(r, sub_dim, quant)
    raise ValueError(method)


def per_layer_traffic(method, T, H, D, L, k, w, r=None, quant=None, sub_dim=None):
    """Dict of branch bytes and their sum for one decode step of one layer."""
    nb = T // L
    kv = 2 * 2                                     # K and V, bf16
    if method == "dense":
        fine = T * H * D * kv
        return dict(summary_keys=0, summary_values=0, window=0, fine=fine, total=fine)
    values = nb * H * D * 2
    window = w * H * D * kv
    fine = k * L * H * D * kv
    if method == "osa":
        keys = T * H * D * 2 + nb * H * summary_key_bytes("nsa_meanpool", D)
    else:
        keys = nb * H * summary_key_bytes(method, D, r, quant, sub_dim)
    return dict(summary_keys=keys, summary_values=values, window=window, fine=fine,
                total=keys + values + window + fine)

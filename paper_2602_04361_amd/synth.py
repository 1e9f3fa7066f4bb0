"""Seeded synthetic inputs shaped like a next-scale-prediction VAR KV cache.

This module only draws numbers. It holds none of the attention, selection or
index-mapping arithmetic: the oracle and the HIP path both receive the arrays
it returns and compute independently from them.

Token layout (the cache layout of the paper's cross-scale attention, Eq. (1)):
scales are concatenated in ascending order and each scale is stored row-major,
so token (x, y) of scale l sits at flat index offset(l) + x * w_l + y.

Recipe (one generator for every workload):
  * Q, K, V ~ N(0, 1) in float32, shape [B, H, N_total, d], drawn in that
    order from numpy's PCG64 seeded with ``seed``; then a unit vector u ~ N(0, I_d)
    normalised to length 1.
  * 2-D sinusoidal position features of each token's normalised position on its
    own scale, px = (x + 0.5) / h_l, py = (y + 0.5) / w_l, with frequencies
    omega_f = pi * (f + 1), f = 0..F-1. Features for frequency f occupy dims
    4f..4f+3 as [sin(omega px), cos(omega px), sin(omega py), cos(omega py)]
    and are added with amplitude 1 to Q and K. The same location on different
    scales gets the same features, which gives the data cross-scale similarity
    and spatial locality.
  * Sinks: keys of the first ``n_sink_scales`` scales get +3u, every query +u.
  * Optional round-to-nearest-even to bfloat16 (values stay float32 arrays that
    are exactly representable in bfloat16).
"""
from __future__ import annotations

import numpy as np

__all__ = ["token_table", "make_qkv", "round_to_bf16", "scale_offsets"]


def scale_offsets(h, w):
    """Start index of each scale in the concatenated cache, plus the total."""
    off = [0]
    for hh, ww in zip(h, w):
        off.append(off[-1] + int(hh) * int(ww))
    return off


def token_table(h, w):
    """Per token: (scale index 0-based, row x, column y, h_l, w_l) as int arrays."""
    sc, xs, ys, hs, ws = [], [], [], [], []
    for l, (hh, ww) in enumerate(zip(h, w)):
        x, y = np.meshgrid(np.arange(hh), np.arange(ww), indexing="ij")
        n = hh * ww
        sc.append(np.full(n, l))
        xs.append(x.reshape(-1))
        ys.append(y.reshape(-1))
        hs.append(np.full(n, hh))
        ws.append(np.full(n, ww))
    return tuple(np.concatenate(a).astype(np.int64) for a in (sc, xs, ys, hs, ws))


def round_to_bf16(x):
    """Round float32 values to the nearest bfloat16 (ties to even); float32 out."""
    a = np.ascontiguousarray(x, dtype=np.float32)
    bits = a.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    bits = ((bits + 0x7FFF + lsb) & 0xFFFF0000).astype(np.uint32)
    return bits.view(np.float32).reshape(a.shape)


def make_qkv(h, w, batch, heads, head_dim, n_freq, n_sink_scales, seed=0, bf16=True):
    """Return float32 arrays Q, K, V of shape [batch, heads, N_total, head_dim].

    Q rows of scale k are Q[..., offset(k-1):offset(k), :]; K and V prefixes are
    the append-only cache seen at step k.
    """
    if 4 * n_freq > head_dim:
        raise ValueError("4 * n_freq must not exceed head_dim")
    off = scale_offsets(h, w)
    n_total = off[-1]
    rng = np.random.default_rng(seed)
    shape = (batch, heads, n_total, head_dim)
    q = rng.standard_normal(shape, dtype=np.float32)
    k = rng.standard_normal(shape, dtype=np.float32)
    v = rng.standard_normal(shape, dtype=np.float32)
    u = rng.standard_normal(head_dim)
    u = (u / np.linalg.norm(u)).astype(np.float32)

    if n_freq > 0:
        _, xs, ys, hs, ws = token_table(h, w)
        px = (xs + 0.5) / hs
        py = (ys + 0.5) / ws
        feats = np.empty((n_total, 4 * n_freq), dtype=np.float64)
        for f in range(n_freq):
            om = np.pi * (f + 1)
            feats[:, 4 * f + 0] = np.sin(om * px)
            feats[:, 4 * f + 1] = np.cos(om * px)
            feats[:, 4 * f + 2] = np.sin(om * py)
            feats[:, 4 * f + 3] = np.cos(om * py)
        feats = feats.astype(np.float32)
        q[..., : 4 * n_freq] += feats
        k[..., : 4 * n_freq] += feats

    n_sink_tok = off[min(n_sink_scales, len(h))]
    k[:, :, :n_sink_tok, :] += 3.0 * u
    q += u
    if bf16:
        q, k, v = round_to_bf16(q), round_to_bf16(k), round_to_bf16(v)
    return q, k, v

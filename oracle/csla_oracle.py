"""Plain fp64 CPU oracle for SparVAR's Cross-Scale Local Sparse Attention
(CSLA) in the paper's own form: a token-wise sink-plus-local mask, reduced to
1-D blocks of B contiguous tokens on both axes.

TEST INFRASTRUCTURE ONLY, like the rest of this package: only the test suite,
the smoke check and the benchmark's CPU-baseline leg may import it. It shares
no code with the HIP library.

It follows Sec. 3.3 (Cross-Scale Local Mapping; Block-wise Sparse Mask,
Eq. block_mask) and the CSLA paragraph of the complexity appendix:
  * a query at (x, y) of scale k is aligned to historical scale h at
    (round(x H_h / H_k), round(y W_h / W_k));
  * it keeps the keys of scale h inside the square of radius r_h around that
    centre (Chebyshev distance), r_h = floor(w_h / 2) for window size w_h;
  * it keeps every key of the sink region (the early scales) as well;
  * the token mask M^(k) is the OR of the sink mask and the local masks of all
    historical scales, and the block mask keeps key block v for query block u
    when any query of u keeps any key of v; every query of u then attends to
    every key of every kept block.

Readings taken where the paper leaves a choice open (collected in the design
notes as well):
  * round() rounds half up, evaluated in exact integers:
    round(x H_h / H_k) = floor((2 x H_h + H_k) / (2 H_k));
  * window sizes are given per historical scale; a scale without a window
    (w_h = 0) contributes no local keys; the default "[3, 5, 7] for the last
    three scales" assigns 3, 5 and 7 to scales k - 2, k - 1 and k, ascending
    with the scale;
  * the sink region is every token of scales 1..n_sink (the first five scales
    hold 121 tokens on the Infinity schedule);
  * query blocks cover the N_k queries of scale k from its first token and key
    blocks the N_<=k keys of the cache from token 0, the last block of each
    axis ragged; the softmax scale 1/sqrt(d) is kept.
"""
from __future__ import annotations

import numpy as np

from .cs4a_oracle import token_attention
from .sparvar_oracle import Geometry

__all__ = [
    "compact_schedule",
    "kv_compact",
    "aligned_centre",
    "default_windows",
    "csla_token_mask",
    "csla_block_rows",
    "csla_block_mask",
    "csla_attention",
]


def aligned_centre(x, n_k, n_h):
    """round(x * n_h / n_k) with halves rounded up, in exact integers (the aligned
    coordinate of the Cross-Scale Local Mapping on one axis)."""
    return (2 * x * n_h + n_k) // (2 * n_k)


def default_windows(k, sizes=(3, 5, 7)):
    """Window size per historical scale h = 1..k (index h - 1): the given sizes on
    the last len(sizes) scales up to k, ascending with the scale; 0 elsewhere."""
    w = [0] * k
    for i, s in enumerate(reversed(sizes)):
        if k - 1 - i >= 0:
            w[k - 1 - i] = int(s)
    return w


def csla_token_mask(geom: Geometry, k, n_sink_scales, windows):
    """Token-wise mask M^(k) [N_k, N_<=k]: query (x, y) of scale k keeps key j when
    j is a sink token (scales 1..n_sink_scales) or j = (x', y') of a scale h with
    window w_h > 0 and max(|cx - x'|, |cy - y'|) <= floor(w_h / 2), where (cx, cy)
    is the query aligned to scale h."""
    if len(windows) != k:
        raise ValueError("one window size per historical scale 1..k is required")
    if min(windows) < 0:
        raise ValueError("window sizes must be non-negative")
    Hk, Wk = geom.hh(k), geom.ww(k)
    mask = np.zeros((Hk * Wk, geom.C(k)), dtype=bool)
    n_sink_tok = geom.C(min(max(n_sink_scales, 0), k))
    mask[:, :n_sink_tok] = True
    qx = np.repeat(np.arange(Hk), Wk)  # query coordinates, row-major
    qy = np.tile(np.arange(Wk), Hk)
    for h in range(1, k + 1):
        if windows[h - 1] == 0:
            continue
        r = windows[h - 1] // 2
        Hh, Wh = geom.hh(h), geom.ww(h)
        cx = aligned_centre(qx, Hk, Hh)
        cy = aligned_centre(qy, Wk, Wh)
        kx = np.repeat(np.arange(Hh), Wh)  # key coordinates of scale h
        ky = np.tile(np.arange(Wh), Hh)
        near = (np.abs(cx[:, None] - kx[None, :]) <= r) & (np.abs(cy[:, None] - ky[None, :]) <= r)
        mask[:, geom.C(h - 1):geom.C(h)] |= near
    return mask


def csla_block_rows(token_mask, B):
    """Eq. block_mask: for each query block u (queries [u B, u B + B)), the ascending
    ids of the key blocks v (keys [v B, v B + B)) holding at least one kept pair."""
    token_mask = np.asarray(token_mask, dtype=bool)
    if B < 1:
        raise ValueError("block size must be positive")
    n_q, n_kv = token_mask.shape
    rows = []
    for u in range(-(-n_q // B)):
        any_key = token_mask[u * B:(u + 1) * B].any(axis=0)
        rows.append([v for v in range(-(-n_kv // B)) if any_key[v * B:(v + 1) * B].any()])
    return rows


def csla_block_mask(rows, n_q, n_kv, B):
    """Token-level mask of the kept blocks: query i sees key j when block j // B is
    in the row of block i // B (the OR semantics of Eq. block_mask)."""
    mask = np.zeros((n_q, n_kv), dtype=bool)
    for u, row in enumerate(rows):
        for v in row:
            mask[u * B:(u + 1) * B, v * B:(v + 1) * B] = True
    return mask


def csla_attention(q_k, k_lek, v_lek, rows, B, scale):
    """Block-sparse attention of scale k: each query block of B queries attends to
    every key of its kept key blocks. Returns (O [N_k, d], LSE [N_k])."""
    n_kv = np.asarray(k_lek).shape[0]
    tok_rows = [[t for v in row for t in range(v * B, min(v * B + B, n_kv))] for row in rows]
    return token_attention(q_k, k_lek, v_lek, tok_rows, B, scale)


def compact_schedule(geom: Geometry, keep):
    """Scale sides of the compressed cache that keeps scales `keep` (ascending,
    1-based): the kept scales in their order (the sink and local scales of the
    paper's KV compression)."""
    keep = [int(l) for l in keep]
    if not keep or keep != sorted(set(keep)) or keep[0] < 1 or keep[-1] > geom.L:
        raise ValueError("kept scales must be ascending, distinct and within the schedule")
    return [geom.hh(l) for l in keep], [geom.ww(l) for l in keep]


def kv_compact(x_all, geom: Geometry, keep):
    """The tokens of the kept scales of one cache plane [N_total, d], in scale order."""
    x_all = np.asarray(x_all)
    return np.concatenate([x_all[geom.C(l - 1):geom.C(l)] for l in keep], axis=0)

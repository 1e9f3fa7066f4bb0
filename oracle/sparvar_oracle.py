"""Plain fp64 CPU oracle for SparVAR's block-sparse cross-scale attention path.

TEST INFRASTRUCTURE ONLY. This module is the checker, not the product: only the
test suite, the smoke check and the benchmark's CPU-baseline leg may import it.
It shares no code with the HIP library and imports nothing from it.

Everything here is written for a reader holding the paper (SparVAR, "Exploring
Sparsity in Visual AutoRegressive Modeling for Training-Free Acceleration").
Each function names the passage it follows. Floating point is fp64 throughout;
inputs are the exact values handed to the GPU (bfloat16 values upcast).

Where the paper leaves a choice open, the reading taken here is stated at the
function and collected in the design notes:
  * blocks are 2-D b x b spatial tiles of each scale (a scale smaller than b
    along an axis is one tile along that axis), not 1-D runs of the flattened
    sequence;
  * the decision-scale score of a (query tile, key block) pair is the softmax
    mass summed over the tile's queries and the block's keys;
  * top-k keeps min(k, #candidates) blocks, ties to the lower block id, output
    ascending and padded with -1;
  * the query homography rounds half up, evaluated in exact integers;
  * Decompose-Align-Project maps a tile through its origin token and takes the
    tile that contains the projected token;
  * the local window is a Chebyshev radius of r tiles in scale k plus every
    scale-(k-1) tile overlapping the query tile's footprint (optionally dilated).

Parity status: every function below is pinned by the CPU tests
(brute force, closed forms, printed geometry, invariants) except where a
docstring says "parity unpinned".
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "Geometry",
    "dense_attention",
    "masked_attention",
    "pooled_scores",
    "topk_blocks",
    "homography",
    "map_block",
    "map_block_cover",
    "sink_blocks",
    "local_blocks",
    "build_rows",
    "rows_to_csr",
    "longest_first",
    "block_mask",
    "block_sparse_attention",
    "block_sparse_attention_gather",
]


# --------------------------------------------------------------------------
# Geometry of the multi-scale cache
# --------------------------------------------------------------------------
@dataclass
class Geometry:
    """Scale schedule and its tiling into b x b blocks.

    Scales are 1-based as in the paper. C(l) is the paper's prefix count
    C_l = N_1 + ... + N_l with C(0) = 0 (appendix, Decompose step of the
    Relative Scale Alignment). Tokens of a scale are row-major, so token (x, y)
    of scale l has flat index C(l-1) + x * w_l + y (the re-linearisation
    delta' = u' * w_l' + v' of the Spatial Projection step).

    Tiling: along the rows of scale l the tile edge is e_h(l) = h_l if h_l < b,
    else b, and there are T_h(l) = ceil(h_l / e_h(l)) tile rows (likewise for
    columns). Block ids run scale-major, tiles row-major within a scale, so
    sorting block ids sorts blocks by their first token.
    """

    h: list
    w: list
    b: int
    n_sink: int
    _base: list = field(init=False, repr=False)

    def __post_init__(self):
        self.h = [int(x) for x in self.h]
        self.w = [int(x) for x in self.w]
        if len(self.h) != len(self.w) or not self.h:
            raise ValueError("h and w must be non-empty and of equal length")
        if self.b < 1 or min(self.h) < 1 or min(self.w) < 1:
            raise ValueError("sizes must be positive")
        base = [0]
        for l in range(1, self.L + 1):
            base.append(base[-1] + self.tiles(l))
        self._base = base

    @property
    def L(self):
        return len(self.h)

    def hh(self, l):
        return self.h[l - 1]

    def ww(self, l):
        return self.w[l - 1]

    def N(self, l):
        return self.hh(l) * self.ww(l)

    def C(self, l):
        return sum(self.N(i) for i in range(1, l + 1))

    def eh(self, l):
        return self.hh(l) if self.hh(l) < self.b else self.b

    def ew(self, l):
        return self.ww(l) if self.ww(l) < self.b else self.b

    def Th(self, l):
        return -(-self.hh(l) // self.eh(l))

    def Tw(self, l):
        return -(-self.ww(l) // self.ew(l))

    def tiles(self, l):
        return self.Th(l) * self.Tw(l)

    def base(self, l):
        """Block id of the first tile of scale l."""
        return self._base[l - 1]

    def nb_le(self, l):
        """Number of blocks in scales 1..l."""
        return self._base[l]

    def block_id(self, l, tu, tv):
        return self.base(l) + tu * self.Tw(l) + tv

    def decompose_block(self, v):
        """Block id -> (scale l, tile row tu, tile column tv)."""
        if not 0 <= v < self._base[-1]:
            raise ValueError(f"block id {v} out of range")
        l = 1
        while self._base[l] <= v:
            l += 1
        t = v - self._base[l - 1]
        return l, t // self.Tw(l), t % self.Tw(l)

    def tile_extent(self, l, tu, tv):
        """Row range and column range (half-open) of tile (tu, tv) of scale l."""
        r0 = tu * self.eh(l)
        c0 = tv * self.ew(l)
        return (r0, min(r0 + self.eh(l), self.hh(l))), (c0, min(c0 + self.ew(l), self.ww(l)))

    def tile_local_tokens(self, l, tu, tv):
        """Within-scale offsets x * w_l + y of the tile's tokens, row-major."""
        (r0, r1), (c0, c1) = self.tile_extent(l, tu, tv)
        return np.array([x * self.ww(l) + y for x in range(r0, r1) for y in range(c0, c1)], dtype=np.int64)

    def block_tokens(self, v):
        """Flat cache indices of the tokens of block v."""
        l, tu, tv = self.decompose_block(v)
        return self.C(l - 1) + self.tile_local_tokens(l, tu, tv)


# --------------------------------------------------------------------------
# Attention: the plain definitions
# --------------------------------------------------------------------------
def dense_attention(q, k, v, scale):
    """Cross-scale attention of the Background section, Eq. (1).

    O = softmax(scale * Q K^T) V over all keys, computed with the row maximum
    subtracted. Also returns LSE = m + ln(sum exp(scale * s - m)), the natural
    log of the softmax denominator. Shapes: q [n_q, d], k and v [n_kv, d].
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    s = float(scale) * (q @ k.T)
    m = s.max(axis=1, keepdims=True)
    p = np.exp(s - m)
    den = p.sum(axis=1, keepdims=True)
    o = (p @ v) / den
    lse = (m + np.log(den))[:, 0]
    return o, lse


def masked_attention(q, k, v, mask, scale):
    """Softmax attention where query i sees only keys j with mask[i, j].

    This is Eq. (1) with the softmax restricted to the kept keys, i.e. the
    sparse update Delta O of the Cross-Scale Sparse Computation paragraph and
    the masked attention of the CSLA section. A row with no kept key returns
    O = 0 and LSE = -inf.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    mask = np.asarray(mask, dtype=bool)
    s = float(scale) * (q @ k.T)
    s = np.where(mask, s, -np.inf)
    o = np.zeros((q.shape[0], v.shape[1]))
    lse = np.full(q.shape[0], -np.inf)
    for i in range(q.shape[0]):
        if not mask[i].any():
            continue
        m = s[i].max()
        p = np.exp(s[i] - m)
        den = p.sum()
        o[i] = (p @ v) / den
        lse[i] = m + math.log(den)
    return o, lse


# --------------------------------------------------------------------------
# Decision scale: pooled scores and top-k
# --------------------------------------------------------------------------
def pooled_scores(q_S, k_leS, scale, geom, S):
    """Block scores at the sparse decision scale S.

    Follows the Sparse Decision Scale paragraph: P = softmax(scale * Q_S K^T)
    over all N_<=S keys; the column-sum D sums P over the queries of a query
    block; here a query block is a b x b tile of scale S and the key axis is
    also pooled, score[g, v] = sum over keys j of block v of D[g, j].
    The scale factor is kept (the paper drops 1/sqrt(d) from its notation only).
    Returns float64 [G_S, NB_<=S].
    """
    n_le = geom.C(S)
    q_S = np.asarray(q_S, dtype=np.float64)
    k_leS = np.asarray(k_leS, dtype=np.float64)
    assert q_S.shape[0] == geom.N(S) and k_leS.shape[0] == n_le
    s = float(scale) * (q_S @ k_leS.T)
    m = s.max(axis=1, keepdims=True)
    p = np.exp(s - m)
    p /= p.sum(axis=1, keepdims=True)
    G = geom.tiles(S)
    NB = geom.nb_le(S)
    out = np.zeros((G, NB))
    for g in range(G):
        rows = geom.tile_local_tokens(S, g // geom.Tw(S), g % geom.Tw(S))
        D = p[rows].sum(axis=0)  # column sum over the query block
        for vb in range(NB):
            out[g, vb] = D[geom.block_tokens(vb)].sum()
    return out


def topk_blocks(scores_row, topk):
    """TopK over one query block's scores (Sparse Decision Scale paragraph).

    Keeps the min(topk, len) highest scores; among equal scores the lower block
    id wins. Returns the kept ids ascending, padded with -1 to length topk.
    """
    if topk <= 0:
        raise ValueError("topk must be positive")
    vals = [float(x) for x in scores_row]
    order = sorted(range(len(vals)), key=lambda i: (-vals[i], i))
    keep = sorted(order[: min(topk, len(vals))])
    return keep + [-1] * (topk - len(keep))


# --------------------------------------------------------------------------
# Cross-scale index mapping (appendix: Cross-Scale Sparse Index Mapping)
# --------------------------------------------------------------------------
def homography(a, T_k, T_S):
    """Query Block Homography along one axis.

    The paper's nearest-neighbour map, round((a + 0.5) / T_k * T_S - 0.5)
    clipped to [0, T_S), with rounding half up, equals floor((2a + 1) T_S /
    (2 T_k)) for 0 <= a < T_k: the source tile whose span contains the centre
    of target tile a. Evaluated here in exact integers; the clip never acts.
    """
    if not 0 <= a < T_k:
        raise ValueError("tile index out of range")
    return ((2 * a + 1) * T_S) // (2 * T_k)


def map_block(geom, v, S, k):
    """Decompose-Align-Project of one selected block from step S to step k.

    Decompose: block v of the cache at step S -> (scale l, tile row, tile col).
    Align: l' = k - (S - l), keeping the relative scale distance.
    Project: the tile's origin token (u, w0) = (tu e_h(l), tv e_w(l)) goes to
    (floor(u h_l' / h_l), floor(w0 w_l' / w_l)) on scale l'; the mapped block is
    the scale-l' tile containing it.
    """
    l, tu, tv = geom.decompose_block(v)
    if l > S:
        raise ValueError("block is not in the cache at step S")
    lp = k - (S - l)
    u = tu * geom.eh(l)
    w0 = tv * geom.ew(l)
    up = (u * geom.hh(lp)) // geom.hh(l)
    wp = (w0 * geom.ww(lp)) // geom.ww(l)
    return geom.block_id(lp, up // geom.eh(lp), wp // geom.ew(lp))


def _upsampled_tiles(geom, l, lp, t, axis):
    """Scale-lp tile range along one axis covered by the upsampled span of tile t of scale l."""
    if axis == 0:
        e, n, e_p, n_p = geom.eh(l), geom.hh(l), geom.eh(lp), geom.hh(lp)
    else:
        e, n, e_p, n_p = geom.ew(l), geom.ww(l), geom.ew(lp), geom.ww(lp)
    x0, x1 = t * e, min((t + 1) * e, n)         # the tile's tokens along the axis, [x0, x1)
    lo = (x0 * n_p) // n                        # first target token of the span x0 n_p / n ...
    hi = -(-(x1 * n_p) // n)                    # ... and the end of x1 n_p / n, rounded up (exclusive)
    return lo // e_p, (hi - 1) // e_p


def map_block_cover(geom, v, S, k):
    """Decompose-Align-Project of one selected block, covering form.

    Decompose and Align as in map_block (scale l -> l' = k - (S - l)). Project
    follows the Spatial Projection step token by token, u -> floor(u h_l'/h_l):
    the tile's tokens [x0, x1) x [y0, y1) of scale l occupy the upsampled span
    [x0 h_l'/h_l, x1 h_l'/h_l) x [y0 w_l'/w_l, y1 w_l'/w_l) of scale l', and the
    mapped blocks are every scale-l' tile overlapping that span. A selected
    region thus keeps its share of its scale's area on the larger scale (the
    kept keys stay about alpha of the cache, as the complexity appendix
    assumes), where the point form keeps the count of blocks. The point form's
    tile is always among them. Returns the ascending block ids.
    """
    l, tu, tv = geom.decompose_block(v)
    if l > S:
        raise ValueError("block is not in the cache at step S")
    lp = k - (S - l)
    r0, r1 = _upsampled_tiles(geom, l, lp, tu, 0)
    c0, c1 = _upsampled_tiles(geom, l, lp, tv, 1)
    return [geom.block_id(lp, a, c) for a in range(r0, r1 + 1) for c in range(c0, c1 + 1)]


def sink_blocks(geom):
    """Every block of the first n_sink scales (the Attention Sink paragraph:
    the first N_sink tokens stay visible to all queries)."""
    return list(range(geom.nb_le(min(geom.n_sink, geom.L)))) if geom.n_sink > 0 else []


def _footprint_tiles(geom, k, a, axis):
    """Scale-(k-1) tile range along one axis overlapping tile a of scale k."""
    if axis == 0:
        e_k, n_k, n_p, e_p, T_p = geom.eh(k), geom.hh(k), geom.hh(k - 1), geom.eh(k - 1), geom.Th(k - 1)
    else:
        e_k, n_k, n_p, e_p, T_p = geom.ew(k), geom.ww(k), geom.ww(k - 1), geom.ew(k - 1), geom.Tw(k - 1)
    lo = (a * e_k * n_p) // n_k
    hi = -(-(min((a + 1) * e_k, n_k) * n_p) // n_k)  # ceiling, exclusive end
    return lo // e_p, (hi - 1) // e_p, T_p


def local_blocks(geom, k, radius, prev_dilation=0):
    """Block-level cross-scale local window for every query tile of scale k.

    Block form of the CSLA local mapping (the unified mask M = M_sink OR the
    local masks, and its block aggregation Eq. (3)): for query tile (a, c) the
    row keeps the sink blocks, the scale-k tiles within Chebyshev distance
    ``radius`` and the scale-(k-1) tiles overlapping the footprint of (a, c),
    widened by ``prev_dilation`` tiles. Returns one ascending list per tile,
    tiles row-major.
    """
    if radius < 0 or prev_dilation < 0:
        raise ValueError("radius and dilation must be non-negative")
    sinks = set(sink_blocks(geom))
    rows = []
    for a in range(geom.Th(k)):
        for c in range(geom.Tw(k)):
            s = set(sinks)
            for ap in range(max(0, a - radius), min(geom.Th(k), a + radius + 1)):
                for cp in range(max(0, c - radius), min(geom.Tw(k), c + radius + 1)):
                    s.add(geom.block_id(k, ap, cp))
            if k >= 2:
                r0, r1, Tr = _footprint_tiles(geom, k, a, 0)
                c0, c1, Tc = _footprint_tiles(geom, k, c, 1)
                r0, r1 = max(0, r0 - prev_dilation), min(Tr - 1, r1 + prev_dilation)
                c0, c1 = max(0, c0 - prev_dilation), min(Tc - 1, c1 + prev_dilation)
                for ap in range(r0, r1 + 1):
                    for cp in range(c0, c1 + 1):
                        s.add(geom.block_id(k - 1, ap, cp))
            rows.append(sorted(s))
    return rows


def build_rows(geom, S, k, topk_idx, local_rows, projection="point"):
    """Kept-block lists at step k for every (batch*head, query tile).

    inds^(k) = A_sink U M_{S->k}(inds^(S)) (Attention Sink paragraph), united
    with the local window. The source tile of target tile (a, c) is
    (homography(a), homography(c)); each of its selected blocks goes through
    map_block (projection "point") or map_block_cover ("cover").
    ``topk_idx`` is int [BH, G_S, topk] with -1 padding.
    Returns rows[bh][g] as ascending unique lists.
    """
    if projection not in ("point", "cover"):
        raise ValueError("projection is 'point' or 'cover'")
    topk_idx = np.asarray(topk_idx)
    BH = topk_idx.shape[0]
    out = []
    for bh in range(BH):
        per = []
        for a in range(geom.Th(k)):
            for c in range(geom.Tw(k)):
                g = a * geom.Tw(k) + c
                gs = homography(a, geom.Th(k), geom.Th(S)) * geom.Tw(S) + homography(c, geom.Tw(k), geom.Tw(S))
                s = set(local_rows[g])
                for vb in topk_idx[bh, gs]:
                    if vb >= 0:
                        if projection == "point":
                            s.add(map_block(geom, int(vb), S, k))
                        else:
                            s.update(map_block_cover(geom, int(vb), S, k))
                per.append(sorted(s))
        out.append(per)
    return out


def rows_to_csr(rows_flat):
    """Lists -> (row_ptr int64 [R+1], col_idx int64 [nnz])."""
    ptr = [0]
    col = []
    for r in rows_flat:
        col.extend(r)
        ptr.append(len(col))
    return np.array(ptr, dtype=np.int64), np.array(col, dtype=np.int64)


def longest_first(row_ptr):
    """Rows ordered by length, longest first; equal lengths keep row order."""
    n = np.diff(np.asarray(row_ptr))
    return sorted(range(len(n)), key=lambda i: (-int(n[i]), i))


# --------------------------------------------------------------------------
# Block-sparse attention (Eq. (3) and the sparse update Delta O)
# --------------------------------------------------------------------------
def block_mask(geom, k, rows_g):
    """Token mask [N_k, N_<=k] of one head: query tile g sees exactly the tokens
    of the blocks in rows_g[g] (OR-aggregation of Eq. (3): a kept block is kept
    whole)."""
    M = np.zeros((geom.N(k), geom.C(k)), dtype=bool)
    for g, row in enumerate(rows_g):
        qs = geom.tile_local_tokens(k, g // geom.Tw(k), g % geom.Tw(k))
        for vb in row:
            M[np.ix_(qs, geom.block_tokens(vb))] = True
    return M


def block_sparse_attention(q_k, k_lek, v_lek, geom, k, rows_g, scale):
    """Block-sparse attention of one head at step k, by the plain definition.

    Builds the token mask of Eq. (3) and evaluates the masked softmax attention.
    q_k [N_k, d], k_lek and v_lek [N_<=k, d]. Returns (O [N_k, d], LSE [N_k]).
    """
    return masked_attention(q_k, k_lek, v_lek, block_mask(geom, k, rows_g), scale)


def block_sparse_attention_gather(q_k, k_lek, v_lek, geom, k, rows_g, scale, tiles=None):
    """Same result as block_sparse_attention, computed per query tile by
    gathering the kept keys (the natural sparse form; used where the full mask
    would be too large). ``tiles`` limits the work to a subset of query tiles;
    rows of other tiles are returned as NaN."""
    q_k = np.asarray(q_k, dtype=np.float64)
    k_lek = np.asarray(k_lek, dtype=np.float64)
    v_lek = np.asarray(v_lek, dtype=np.float64)
    o = np.full((geom.N(k), v_lek.shape[1]), np.nan)
    lse = np.full(geom.N(k), np.nan)
    it = range(len(rows_g)) if tiles is None else tiles
    for g in it:
        qs = geom.tile_local_tokens(k, g // geom.Tw(k), g % geom.Tw(k))
        if rows_g[g]:
            keys = np.concatenate([geom.block_tokens(vb) for vb in rows_g[g]])
        else:
            keys = np.zeros(0, dtype=np.int64)
        if keys.size == 0:
            o[qs] = 0.0
            lse[qs] = -np.inf
            continue
        og, lg = dense_attention(q_k[qs], k_lek[keys], v_lek[keys], scale)
        o[qs] = og
        lse[qs] = lg
    return o, lse

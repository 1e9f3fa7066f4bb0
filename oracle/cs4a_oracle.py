"""Plain fp64 CPU oracle for SparVAR's token-granular CS^4A path.

TEST INFRASTRUCTURE ONLY, like the rest of this package: only the test suite,
the smoke check and the benchmark's CPU-baseline leg may import it. It shares
no code with the HIP library.

It follows Sec. 3.2 (Cross-Scale Self-Similar Sparse Attention) and the
appendix (Hardware-Efficient Sparse Computation; Cross-Scale Sparse Index
Mapping) at the granularity the paper describes: 1-D query blocks of C
contiguous queries of the flattened scale, and individual key tokens.
  * column sums at the decision scale S: D[i, j] = sum over the queries q of
    block i of P[q, j], with P = softmax(scale * Q_S K_<=S^T);
  * inds^(S)[i] = TopK over D[i, :] (ties to the lower token index, output
    ascending, padded with -1);
  * O_cache^(S) = O_dense^(S) - Softmax(Q K_inds^T) V_inds, the attention of
    each query block restricted to its own top-K tokens;
  * for a later scale k: the target query block g_k takes the tokens of source
    block phi(g_k) (Query Block Homography on the block index), each mapped by
    Decompose-Align-Project at token level, together with the sink tokens
    (every token of scales 1..n_sink);
  * Delta O^(k) = the attention of each query block restricted to its mapped
    tokens, and O^(k) = upsample(O_cache^(S)) + Delta O^(k).

Readings taken where the paper leaves a choice open (collected in the design
notes as well):
  * the softmax scale 1/sqrt(d) is kept (the paper drops it from notation only);
  * the homography's round-half-up is evaluated in exact integers,
    phi(g) = floor((2g + 1) G_S / (2 G_k));
  * "upsampled cache prediction" is read as nearest-neighbour upsampling of the
    scale-S grid onto the scale-k grid by token centres,
    (x, y) -> (floor((2x + 1) h_S / (2 h_k)), floor((2y + 1) w_S / (2 w_k)));
  * the sink set is every token of scales 1..n_sink, and a mapped token already
    in it is kept once.
"""
from __future__ import annotations

import numpy as np

from .sparvar_oracle import Geometry, dense_attention

__all__ = [
    "query_blocks",
    "column_sums",
    "topk_tokens",
    "block_homography",
    "map_token",
    "cs4a_rows",
    "token_attention",
    "o_cache",
    "upsample_nearest",
    "cs4a_output",
]


def query_blocks(n, C):
    """Query block i of a scale of n tokens: flat offsets [i C, min((i+1) C, n))
    (reshape of the query axis into G = ceil(n / C) blocks, Sec. 3.2)."""
    if C < 1:
        raise ValueError("block size must be positive")
    return [np.arange(i * C, min((i + 1) * C, n)) for i in range(-(-n // C))]


def column_sums(q_S, k_leS, scale, C):
    """Column-sum tensor D of the Sparse Decision Scale paragraph.

    P = softmax(scale * Q_S K_<=S^T) over all keys (row maximum subtracted),
    D[i, j] = sum of P[q, j] over the queries q of query block i.
    Returns float64 [G_S, N_<=S].
    """
    q_S = np.asarray(q_S, dtype=np.float64)
    k_leS = np.asarray(k_leS, dtype=np.float64)
    s = float(scale) * (q_S @ k_leS.T)
    s -= s.max(axis=1, keepdims=True)
    p = np.exp(s)
    p /= p.sum(axis=1, keepdims=True)
    return np.stack([p[rows].sum(axis=0) for rows in query_blocks(q_S.shape[0], C)])


def topk_tokens(d_row, K):
    """inds^(S) for one query block: the min(K, len) largest column sums, ties to
    the lower token index; returned ascending and padded with -1 to length K."""
    if K <= 0:
        raise ValueError("K must be positive")
    vals = [float(x) for x in d_row]
    order = sorted(range(len(vals)), key=lambda j: (-vals[j], j))
    keep = sorted(order[: min(K, len(vals))])
    return keep + [-1] * (K - len(keep))


def block_homography(g_k, G_k, G_S):
    """Query Block Homography on 1-D block indices: the paper's
    round((g_k + 0.5) / G_k * G_S - 0.5), rounding half up and clipped to
    [0, G_S), equals floor((2 g_k + 1) G_S / (2 G_k)) in exact integers."""
    if not 0 <= g_k < G_k:
        raise ValueError("block index out of range")
    return ((2 * g_k + 1) * G_S) // (2 * G_k)


def map_token(geom: Geometry, j, S, k):
    """Decompose-Align-Project of one key token from step S to step k.

    Decompose: j -> (l, delta) with C_{l-1} <= j < C_l, delta = j - C_{l-1}.
    Align: l' = k - (S - l).
    Project: delta -> (u, v) = (delta // w_l, delta % w_l) -> (floor(u h_l' / h_l),
    floor(v w_l' / w_l)) -> delta' = u' w_l' + v'; j' = C_{l'-1} + delta'.
    """
    if not 0 <= j < geom.C(S):
        raise ValueError("token is not in the cache at step S")
    l = 1
    while geom.C(l) <= j:
        l += 1
    delta = j - geom.C(l - 1)
    lp = k - (S - l)
    u, v = divmod(delta, geom.ww(l))
    up = (u * geom.hh(lp)) // geom.hh(l)
    vp = (v * geom.ww(lp)) // geom.ww(l)
    return geom.C(lp - 1) + up * geom.ww(lp) + vp


def cs4a_rows(geom: Geometry, S, k, inds_S, C):
    """Kept key tokens of every query block of scale k: the sink tokens (all of
    scales 1..n_sink) and the mapped tokens of source block phi(g_k), ascending
    without repeats. inds_S: per source block, ascending ids padded with -1."""
    G_S = -(-geom.N(S) // C)
    G_k = -(-geom.N(k) // C)
    if len(inds_S) != G_S:
        raise ValueError("one index row per query block of scale S is required")
    n_sink_tok = geom.C(min(geom.n_sink, geom.L)) if geom.n_sink > 0 else 0
    rows = []
    for g in range(G_k):
        src = block_homography(g, G_k, G_S)
        mapped = {map_token(geom, int(j), S, k) for j in inds_S[src] if j >= 0}
        rows.append(sorted(set(range(n_sink_tok)) | mapped))
    return rows


def token_attention(q, k_all, v_all, rows, C, scale):
    """Attention of each query block restricted to its own key tokens
    (Softmax(Q K_inds^T) V_inds of Sec. 3.2). A block with no token gives O = 0
    and LSE = -inf. Returns (O [n_q, d], LSE [n_q])."""
    q = np.asarray(q, dtype=np.float64)
    k_all = np.asarray(k_all, dtype=np.float64)
    v_all = np.asarray(v_all, dtype=np.float64)
    o = np.zeros((q.shape[0], v_all.shape[1]))
    lse = np.full(q.shape[0], -np.inf)
    blocks = query_blocks(q.shape[0], C)
    if len(rows) != len(blocks):
        raise ValueError("one token row per query block is required")
    for qs, toks in zip(blocks, rows):
        toks = [t for t in toks if t >= 0]
        if not toks:
            continue
        o[qs], lse[qs] = dense_attention(q[qs], k_all[toks], v_all[toks], scale)
    return o, lse


def o_cache(q_S, k_leS, v_leS, inds_S, C, scale):
    """O_cache^(S) = O_dense^(S) - Softmax(Q K_inds^T) V_inds, with the dense
    attention over all keys of scales 1..S and the sparse one over each query
    block's own top-K tokens (Sec. 3.2)."""
    o_dense, _ = dense_attention(q_S, k_leS, v_leS, scale)
    o_sparse, _ = token_attention(q_S, k_leS, v_leS, inds_S, C, scale)
    return o_dense - o_sparse


def upsample_nearest(x_S, h_S, w_S, h_k, w_k):
    """Nearest-neighbour upsampling of a scale-S token grid [h_S * w_S, d] to
    scale k [h_k * w_k, d] by token centres (the reading of the paper's
    "upsampled cache prediction")."""
    x_S = np.asarray(x_S, dtype=np.float64)
    out = np.empty((h_k * w_k, x_S.shape[1]))
    for x in range(h_k):
        xs = ((2 * x + 1) * h_S) // (2 * h_k)
        for y in range(w_k):
            ys = ((2 * y + 1) * w_S) // (2 * w_k)
            out[x * w_k + y] = x_S[xs * w_S + ys]
    return out


def cs4a_output(q_k, k_lek, v_lek, rows_k, C, scale, o_cache_S, geom: Geometry, S, k):
    """O^(k) = upsample(O_cache^(S)) + Delta O^(k) (Cross-Scale Sparse
    Computation paragraph); pass o_cache_S=None for Delta O^(k) alone."""
    delta, _ = token_attention(q_k, k_lek, v_lek, rows_k, C, scale)
    if o_cache_S is None:
        return delta
    return upsample_nearest(o_cache_S, geom.hh(S), geom.ww(S), geom.hh(k), geom.ww(k)) + delta

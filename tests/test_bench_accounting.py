"""The bench's algorithmic accounting (FLOPs, bytes, density of a block-sparse
launch) against a brute-force count over the oracle's own rows: every kept
(query, key) pair of a row is counted once per query of its tile, the bytes are
Q + O plus the K and V of the distinct tokens a (b, h) plane keeps, and -1
padding or out-of-range ids count nothing. Host only (the geometry comes from
the library's host-side sparvar_scale_info)."""
import numpy as np
import pytest

import bench
import oracle as O
from paper_2602_04361_amd import sparvar as sv


def padded_csr(rows, extra, nb, rng):
    """Rows at a fixed stride with -1 padding; a few padding slots hold ids out of range."""
    M = max(len(r) for r in rows) + extra
    ci = np.full(len(rows) * M, -1, dtype=np.int32)
    for i, r in enumerate(rows):
        ci[i * M:i * M + len(r)] = r
        if extra and rng.random() < 0.3:
            ci[i * M + len(r)] = nb + 5  # out of range: skipped by the kernels and by the accounting
    return np.arange(len(rows) + 1, dtype=np.int32) * M, ci


@pytest.mark.parametrize("sides,b,ns,S,k,B,H,topk,r,d", [
    ([1, 2, 4, 6, 8, 12], 4, 2, 4, 6, 1, 2, 3, 1, 64),
    ([1, 2, 3, 5, 7, 10, 13], 4, 1, 5, 7, 2, 1, 4, 1, 128),
    ([1, 2, 4, 6, 8, 12, 16, 20, 24, 32, 40], 8, 4, 10, 11, 1, 2, 8, 1, 128),
])
def test_sparse_accounting_matches_brute_force(sides, b, ns, S, k, B, H, topk, r, d):
    og = O.Geometry(sides, sides, b, ns)
    g = sv.Geometry(sides, sides, b, ns)
    info = {l: g.scale_info(l) for l in range(1, len(sides) + 1)}
    rng = np.random.default_rng(len(sides) * 100 + k)
    BH, G_S, NB_S = B * H, og.tiles(S), og.nb_le(S)
    sel = np.sort(np.stack([rng.choice(NB_S, min(topk, NB_S), replace=False) for _ in range(BH * G_S)]), axis=1)
    rows_bh = O.build_rows(og, S, k, sel.reshape(BH, G_S, -1), O.local_blocks(og, k, r))
    rows = [row for per in rows_bh for row in per]
    rp, ci = padded_csr(rows, 2, og.nb_le(k), rng)
    flops, bytes_, density, keys = bench.sparse_accounting(rp, ci, info, k, BH, d)

    G_k = og.tiles(k)
    n_k, n_le = og.C(k) - og.C(k - 1), og.C(k)
    pairs, uniq = 0, 0
    for bh in range(BH):
        kept = set()
        for t in range(G_k):
            row = rows_bh[bh][t]
            toks = [x for v in row for x in og.block_tokens(v)]
            assert len(toks) == len(set(toks))  # a row lists disjoint blocks
            n_q = len(og.block_tokens(og.nb_le(k - 1) + t))  # query tile t of scale k is block NB_<k + t
            pairs += n_q * len(toks)
            assert keys[bh * G_k + t] == len(toks)
            kept.update(toks)
        uniq += len(kept)
    assert flops == 4.0 * d * pairs
    assert bytes_ == BH * n_k * d * 2 * 2 + uniq * d * 2 * 2
    assert density == pytest.approx(pairs / (BH * n_k * n_le), rel=1e-12)


def test_dense_rows_give_density_one():
    # every block of scales 1..k in every row: the sparse accounting equals dense attention
    sides, b, ns, k, d = [1, 2, 4, 6, 8, 12], 4, 2, 6, 64
    og = O.Geometry(sides, sides, b, ns)
    g = sv.Geometry(sides, sides, b, ns)
    info = {l: g.scale_info(l) for l in range(1, len(sides) + 1)}
    rows = [list(range(og.nb_le(k))) for _ in range(og.tiles(k))]
    rp, ci = padded_csr(rows, 0, og.nb_le(k), np.random.default_rng(0))
    flops, bytes_, density, _ = bench.sparse_accounting(rp, ci, info, k, 1, d)
    n_k, n_le = og.C(k) - og.C(k - 1), og.C(k)
    assert density == 1.0
    assert flops == 4.0 * d * n_k * n_le
    assert bytes_ == n_k * d * 4 + n_le * d * 4

"""Pins of the token-granular CS^4A oracle against what the paper and the
mathematics fix: hand-derived index maps (tests/golden/cs4a_hand.json), the
paper's homography formula in exact rationals, brute-force loops, closed forms
(uniform attention, every-token rows), invariants (rows of D sum to the block
size, injective and monotone maps) and agreement with the block-level mapping,
which is pinned by its own hand tables."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))
HAND = json.load(open(os.path.join(HERE, "golden", "cs4a_hand.json")))
INF = HAND["sides"]


def rng_qkv(n_q, n_k, d, seed):
    r = np.random.default_rng(seed)
    return r.standard_normal((n_q, d)), r.standard_normal((n_k, d)), r.standard_normal((n_k, d))


def test_query_blocks_cover_the_scale_once():
    for n, C in [(64, 16), (100, 32), (7, 3), (5, 8)]:
        blocks = O.query_blocks(n, C)
        assert len(blocks) == -(-n // C)
        assert np.concatenate(blocks).tolist() == list(range(n))
        assert all(len(b) == C for b in blocks[:-1])


def test_column_sums_brute_force_and_row_sums():
    q, k, _ = rng_qkv(10, 13, 4, 1)
    sc = 0.7
    D = O.column_sums(q, k, sc, 4)
    ref = np.zeros((3, 13))
    for i in range(10):
        w = [np.exp(sc * float(q[i] @ k[j])) for j in range(13)]
        tot = sum(w)
        for j in range(13):
            ref[i // 4, j] += w[j] / tot
    assert np.allclose(D, ref, atol=1e-13)
    # each query's probabilities sum to one, so a block's sums add up to its size
    assert np.allclose(D.sum(axis=1), [4, 4, 2])


def test_column_sums_uniform_when_queries_are_zero():
    _, k, _ = rng_qkv(1, 9, 5, 2)
    D = O.column_sums(np.zeros((6, 5)), k, 1.0, 4)
    assert np.allclose(D[0], 4 / 9) and np.allclose(D[1], 2 / 9)


def test_topk_tokens_against_repeated_argmax_with_ties():
    r = np.random.default_rng(3)
    for trial in range(50):
        row = r.integers(0, 5, size=int(r.integers(1, 30))).astype(float)  # many ties
        K = int(r.integers(1, 35))
        got = O.topk_tokens(row, K)
        vals = row.copy()
        picked = []
        for _ in range(min(K, len(row))):
            j = int(np.argmax(vals))  # first maximum: the lower index on ties
            picked.append(j)
            vals[j] = -np.inf
        assert got == sorted(picked) + [-1] * (K - len(picked))


def test_block_homography_equals_the_papers_rounding_in_rationals():
    for G_k in range(1, 41):
        for G_S in range(1, 41):
            for g in range(G_k):
                x = (Fraction(2 * g + 1, 2 * G_k)) * G_S - Fraction(1, 2)
                want = int(x + Fraction(1, 2)) if x >= 0 else 0  # round half up, x > -1/2 always
                want = min(max(want, 0), G_S - 1)
                assert O.block_homography(g, G_k, G_S) == want
    for case in HAND["block_homography"]:
        assert O.block_homography(case["g"], case["G_k"], case["G_S"]) == case["expect"], case


def test_map_token_hand_values():
    g = O.Geometry(INF, INF, 8, 4)
    for case in HAND["token_map"]:
        assert O.map_token(g, case["j"], case["S"], case["k"]) == case["expect"], case


def test_map_token_identity_injective_monotone():
    g = O.Geometry(INF, INF, 8, 4)
    assert all(O.map_token(g, j, 10, 10) == j for j in range(g.C(10)))
    for k in (11, 12, 13):
        m = [O.map_token(g, j, 10, k) for j in range(g.C(10))]
        assert all(a < b for a, b in zip(m, m[1:])), k  # strictly increasing: injective and monotone
        assert 0 <= m[0] and m[-1] < g.C(k)
        # scale l lands in scale l + (k - S)
        for l in range(1, 11):
            lo, hi = O.map_token(g, g.C(l - 1), 10, k), O.map_token(g, g.C(l) - 1, 10, k)
            assert g.C(l + k - 10 - 1) <= lo <= hi < g.C(l + k - 10)


def test_map_token_agrees_with_the_block_mapping_at_tile_origins():
    for h, w, b in [(INF, INF, 8), ([1, 2, 3, 5, 8, 11], [1, 3, 4, 7, 9, 14], 4)]:
        g = O.Geometry(h, w, b, 2)
        L = g.L
        for S in range(2, L):
            for k in range(S + 1, L + 1):
                for v in range(g.nb_le(S)):
                    origin = int(g.block_tokens(v)[0])
                    assert O.map_token(g, origin, S, k) in set(g.block_tokens(O.map_block(g, v, S, k)).tolist())


def test_rows_hold_sinks_and_mapped_tokens():
    g = O.Geometry(INF, INF, 8, 4)
    C, K = 128, 20
    r = np.random.default_rng(4)
    G_S = -(-g.N(10) // C)
    inds = [sorted(r.choice(g.C(10), size=K, replace=False).tolist()) for _ in range(G_S)]
    rows = O.cs4a_rows(g, 10, 13, inds, C)
    assert len(rows) == -(-g.N(13) // C)
    for gk, row in enumerate(rows):
        assert row == sorted(set(row))
        assert set(range(57)) <= set(row)
        src = O.block_homography(gk, len(rows), G_S)
        assert set(row) - set(range(57)) <= {O.map_token(g, j, 10, 13) for j in inds[src]}
        assert len(row) <= 57 + K


def test_token_attention_every_token_is_dense_and_empty_is_zero():
    q, k, v = rng_qkv(20, 11, 6, 5)
    sc = 0.4
    o, lse = O.token_attention(q, k, v, [list(range(11))] * 3, 8, sc)
    od, ld = O.dense_attention(q, k, v, sc)
    assert np.allclose(o, od, atol=1e-12) and np.allclose(lse, ld, atol=1e-12)
    o, lse = O.token_attention(q, k, v, [[], [3, 5], [-1, -1]], 8, sc)
    assert (o[:8] == 0).all() and np.isneginf(lse[:8]).all() and (o[16:] == 0).all()
    mask = np.zeros((20, 11), dtype=bool)
    mask[8:16, [3, 5]] = True
    om, _ = O.masked_attention(q, k, v, mask, sc)
    assert np.allclose(o[8:16], om[8:16], atol=1e-12)


def test_o_cache_closed_forms():
    q, k, v = rng_qkv(16, 9, 4, 6)
    sc = 0.5
    assert np.allclose(O.o_cache(q, k, v, [list(range(9))] * 2, 8, sc), 0, atol=1e-12)
    od, _ = O.dense_attention(q, k, v, sc)
    assert np.allclose(O.o_cache(q, k, v, [[-1, -1]] * 2, 8, sc), od, atol=1e-12)


def test_upsample_nearest_hand_rows_identity_and_constants():
    for case in HAND["upsample_rows"]:
        n_S, n_k = case["n_S"], case["n_k"]
        x = np.arange(n_S * n_S, dtype=float)[:, None]
        up = O.upsample_nearest(x, n_S, n_S, n_k, n_k)[:, 0].reshape(n_k, n_k)
        rows = case["expect"]
        for a in range(n_k):
            for c in range(n_k):
                assert up[a, c] == rows[a] * n_S + rows[c]
    # non-square with unequal ratios: a 2 x 3 grid onto 4 x 9 (rows doubled, columns tripled)
    x = np.arange(6, dtype=float)[:, None]
    up = O.upsample_nearest(x, 2, 3, 4, 9)[:, 0].reshape(4, 9)
    assert all(up[a, c] == (a // 2) * 3 + c // 3 for a in range(4) for c in range(9))
    x = np.random.default_rng(7).standard_normal((12, 3))
    assert np.array_equal(O.upsample_nearest(x, 3, 4, 3, 4), x)
    assert np.allclose(O.upsample_nearest(np.full((6, 2), 2.5), 2, 3, 5, 7), 2.5)


def test_output_with_every_token_and_zero_cache_is_dense():
    g = O.Geometry([1, 2, 4], [1, 2, 4], 2, 1)
    q, k, v = rng_qkv(16, 21, 4, 8)
    rows = [list(range(21))] * 2
    out = O.cs4a_output(q, k, v, rows, 8, 0.5, np.zeros((4, 4)), g, 2, 3)
    od, _ = O.dense_attention(q, k, v, 0.5)
    assert np.allclose(out, od, atol=1e-12)
    with pytest.raises(ValueError):
        O.map_token(g, 5, 2, 3)  # token 5 is not in the cache at step 2 (C_2 = 5)

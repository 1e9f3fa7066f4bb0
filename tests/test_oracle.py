"""CPU pins of the fp64 oracle against what the paper and the mathematics fix.

Every test here is independent of the oracle's own code: printed numbers,
hand-derived tables, closed forms, brute force on tiny inputs written as plain
Python loops, exact rational evaluation of the paper's formulas, and invariants.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import (
    Geometry,
    block_mask,
    block_sparse_attention,
    block_sparse_attention_gather,
    build_rows,
    dense_attention,
    homography,
    local_blocks,
    longest_first,
    map_block,
    map_block_cover,
    masked_attention,
    pooled_scores,
    rows_to_csr,
    sink_blocks,
    topk_blocks,
)
from paper_2602_04361_amd.synth import make_qkv

INF_SIDES = [1, 2, 4, 6, 8, 12, 16, 20, 24, 32, 40, 48, 64]


def load(golden_dir, name):
    with open(os.path.join(golden_dir, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- geometry
def test_printed_infinity_geometry(golden_dir):
    gj = load(golden_dir, "paper_geometry.json")
    g = Geometry(gj["sides"], gj["sides"], 8, 4)
    assert g.N(13) == gj["q_len_last_scale"]
    assert g.C(13) == gj["kv_len_last_scale"]
    assert g.C(5) == gj["tokens_first_5_scales"]


def test_hand_block_table(golden_dir):
    t = load(golden_dir, "hand_tables.json")["infinity_b8_tiles_per_scale"]
    g = Geometry(INF_SIDES, INF_SIDES, 8, 4)
    assert [g.tiles(l) for l in range(1, 14)] == t["tiles"]
    assert [g.nb_le(l) for l in range(1, 14)] == t["blocks_le"]


def test_blocks_partition_tokens():
    # Every token of the cache belongs to exactly one block, and ids sort by first token.
    for sides_h, sides_w, b in [(INF_SIDES, INF_SIDES, 8), ([1, 2, 3, 5, 7, 10, 13], [1, 3, 2, 5, 9, 10, 6], 4),
                                (INF_SIDES, INF_SIDES, 16)]:
        g = Geometry(sides_h, sides_w, b, 2)
        n = g.C(g.L)
        seen = np.zeros(n, dtype=int)
        firsts = []
        for v in range(g.nb_le(g.L)):
            toks = g.block_tokens(v)
            seen[toks] += 1
            firsts.append(int(toks[0]))
            assert len(toks) <= b * b
        assert (seen == 1).all()
        assert firsts == sorted(firsts)


def test_block_tokens_brute_force():
    # A block's tokens are exactly those whose (row // e_h, col // e_w) is its tile.
    g = Geometry([3, 5, 10], [2, 7, 9], 4, 1)
    for v in range(g.nb_le(3)):
        l, tu, tv = g.decompose_block(v)
        off = sum(g.h[i] * g.w[i] for i in range(l - 1))
        eh = g.h[l - 1] if g.h[l - 1] < 4 else 4
        ew = g.w[l - 1] if g.w[l - 1] < 4 else 4
        want = [off + x * g.w[l - 1] + y for x in range(g.h[l - 1]) for y in range(g.w[l - 1])
                if x // eh == tu and y // ew == tv]
        assert list(g.block_tokens(v)) == want


# ---------------------------------------------------------------- attention
def brute_attention(q, k, v, scale):
    """Textbook softmax attention as pure-Python loops."""
    out, lses = [], []
    for qi in q:
        s = [scale * sum(a * b for a, b in zip(qi, kj)) for kj in k]
        m = max(s)
        e = [math.exp(x - m) for x in s]
        den = sum(e)
        out.append([sum(e[j] * v[j][c] for j in range(len(k))) / den for c in range(len(v[0]))])
        lses.append(m + math.log(den))
    return np.array(out), np.array(lses)


def test_dense_matches_brute_force():
    rng = np.random.default_rng(1)
    q, k, v = rng.standard_normal((4, 3)), rng.standard_normal((6, 3)), rng.standard_normal((6, 5))
    o, lse = dense_attention(q, k, v, 0.7)
    ob, lb = brute_attention(q.tolist(), k.tolist(), v.tolist(), 0.7)
    assert np.abs(o - ob).max() < 1e-13
    assert np.abs(lse - lb).max() < 1e-13


def test_dense_closed_forms():
    rng = np.random.default_rng(2)
    k, v = rng.standard_normal((9, 8)), rng.standard_normal((9, 4))
    # Q = 0: uniform weights, output = mean of V, LSE = ln(n).
    o, lse = dense_attention(np.zeros((3, 8)), k, v, 0.5)
    assert np.abs(o - v.mean(axis=0)).max() < 1e-14
    assert np.abs(lse - math.log(9)).max() < 1e-14
    # One key: output is that value, LSE the scaled score.
    q = rng.standard_normal((2, 8))
    o, lse = dense_attention(q, k[:1], v[:1], 0.5)
    assert np.abs(o - v[0]).max() < 1e-14
    assert np.abs(lse - 0.5 * q @ k[0]).max() < 1e-12
    # Two keys: sigmoid of the score difference.
    o, _ = dense_attention(q, k[:2], v[:2], 0.5)
    d = 0.5 * (q @ k[0] - q @ k[1])
    p0 = 1.0 / (1.0 + np.exp(-d))
    assert np.abs(o - (p0[:, None] * v[0] + (1 - p0[:, None]) * v[1])).max() < 1e-13
    # Rows sum to one: an all-ones value channel returns exactly 1.
    o, _ = dense_attention(q, k, np.ones((9, 1)), 0.5)
    assert np.abs(o - 1.0).max() < 1e-12


def test_dense_key_permutation_equivariance():
    rng = np.random.default_rng(3)
    q, k, v = rng.standard_normal((5, 6)), rng.standard_normal((11, 6)), rng.standard_normal((11, 3))
    perm = rng.permutation(11)
    o1, l1 = dense_attention(q, k, v, 0.3)
    o2, l2 = dense_attention(q, k[perm], v[perm], 0.3)
    assert np.abs(o1 - o2).max() < 1e-13 and np.abs(l1 - l2).max() < 1e-13


def test_masked_attention_brute_force_and_empty_row():
    rng = np.random.default_rng(4)
    q, k, v = rng.standard_normal((4, 3)), rng.standard_normal((7, 3)), rng.standard_normal((7, 2))
    mask = rng.random((4, 7)) < 0.5
    mask[0] = False
    mask[1, :] = False
    mask[1, 3] = True
    o, lse = masked_attention(q, k, v, mask, 0.9)
    assert (o[0] == 0).all() and lse[0] == -np.inf
    assert np.abs(o[1] - v[3]).max() < 1e-14
    for i in range(2, 4):
        keep = [j for j in range(7) if mask[i, j]]
        if not keep:
            continue
        ob, lb = brute_attention([q[i].tolist()], [k[j].tolist() for j in keep], [v[j].tolist() for j in keep], 0.9)
        assert np.abs(o[i] - ob[0]).max() < 1e-13 and abs(lse[i] - lb[0]) < 1e-13
    full, fl = masked_attention(q, k, v, np.ones((4, 7), bool), 0.9)
    d, dl = dense_attention(q, k, v, 0.9)
    assert np.abs(full - d).max() < 1e-14 and np.abs(fl - dl).max() < 1e-14


# ---------------------------------------------------------------- pooled scores and top-k
def tiny_geom():
    return Geometry([1, 2, 4, 8], [1, 2, 4, 8], 4, 2)


def test_pooled_scores_brute_force():
    g = Geometry([1, 2, 3, 5], [1, 3, 2, 6], 2, 1)
    S = 4
    rng = np.random.default_rng(5)
    q = rng.standard_normal((g.N(S), 4))
    k = rng.standard_normal((g.C(S), 4))
    sc = pooled_scores(q, k, 0.8, g, S)
    # Brute force: softmax per query via loops, then add P[q, j] over (q in tile, j in block)
    # with tile membership decided from coordinates.
    off = [0]
    for i in range(4):
        off.append(off[-1] + g.h[i] * g.w[i])
    P = []
    for qi in q:
        s = [0.8 * sum(a * b for a, b in zip(qi, kj)) for kj in k]
        m = max(s)
        e = [math.exp(x - m) for x in s]
        P.append([x / sum(e) for x in e])

    def tile_of(l, x, y):
        eh = g.h[l] if g.h[l] < 2 else 2
        ew = g.w[l] if g.w[l] < 2 else 2
        tw = -(-g.w[l] // ew)
        return (x // eh) * tw + y // ew

    blk_of_tok = []
    base = 0
    for l in range(4):
        for x in range(g.h[l]):
            for y in range(g.w[l]):
                blk_of_tok.append(base + tile_of(l, x, y))
        eh = g.h[l] if g.h[l] < 2 else 2
        ew = g.w[l] if g.w[l] < 2 else 2
        base += (-(-g.h[l] // eh)) * (-(-g.w[l] // ew))
    want = np.zeros_like(sc)
    for x in range(g.h[3]):
        for y in range(g.w[3]):
            qi = x * g.w[3] + y
            for j in range(g.C(S)):
                want[tile_of(3, x, y), blk_of_tok[j]] += P[qi][j]
    assert np.abs(sc - want).max() < 1e-13


def test_pooled_scores_closed_forms():
    g = tiny_geom()
    S = 3
    rng = np.random.default_rng(6)
    k = rng.standard_normal((g.C(S), 5))
    q = rng.standard_normal((g.N(S), 5))
    sc = pooled_scores(q, k, 0.4, g, S)
    # Softmax rows sum to one: a tile's scores add up to its query count.
    for gi in range(g.tiles(S)):
        assert abs(sc[gi].sum() - len(g.tile_local_tokens(S, gi // g.Tw(S), gi % g.Tw(S)))) < 1e-12
    # Q = 0: uniform softmax, score = |tile| * |block| / N_<=S.
    sc0 = pooled_scores(np.zeros_like(q), k, 0.4, g, S)
    for gi in range(g.tiles(S)):
        nq = len(g.tile_local_tokens(S, gi // g.Tw(S), gi % g.Tw(S)))
        for vb in range(g.nb_le(S)):
            assert abs(sc0[gi, vb] - nq * len(g.block_tokens(vb)) / g.C(S)) < 1e-14


def brute_topk(vals, k):
    """Repeated argmax; a strictly larger value wins, a tie keeps the earlier index."""
    left = list(range(len(vals)))
    chosen = []
    for _ in range(min(k, len(vals))):
        best = left[0]
        for i in left[1:]:
            if vals[i] > vals[best]:
                best = i
        chosen.append(best)
        left.remove(best)
    return sorted(chosen) + [-1] * (k - len(chosen))


def test_topk_against_brute_force_with_ties():
    rng = np.random.default_rng(7)
    for trial in range(300):
        n = int(rng.integers(1, 40))
        vals = rng.integers(0, 6, size=n).astype(np.float32)  # many ties
        if trial % 3 == 0:
            vals = rng.random(n).astype(np.float32)
        k = int(rng.integers(1, 45))
        assert topk_blocks(vals, k) == brute_topk(vals.tolist(), k)


def test_topk_padding_and_all_equal():
    assert topk_blocks([1.0, 1.0, 1.0], 2) == [0, 1]
    assert topk_blocks([0.5, 2.0], 5) == [0, 1, -1, -1, -1]
    with pytest.raises(ValueError):
        topk_blocks([1.0], 0)


# ---------------------------------------------------------------- index mapping
def test_homography_hand_tables(golden_dir):
    for case in load(golden_dir, "hand_tables.json")["homography"]["cases"]:
        assert [homography(a, case["T_k"], case["T_S"]) for a in range(case["T_k"])] == case["map"]


def test_homography_equals_paper_formula_exactly():
    # round((a + 1/2)/T_k * T_S - 1/2), round half up, clipped to [0, T_S), in exact rationals.
    for T_k in range(1, 40):
        for T_S in range(1, 40):
            for a in range(T_k):
                x = Fraction(2 * a + 1, 2 * T_k) * T_S - Fraction(1, 2)
                r = math.floor(x + Fraction(1, 2))
                r = min(max(r, 0), T_S - 1)
                assert homography(a, T_k, T_S) == r


def test_homography_identity_and_monotone():
    for T in range(1, 30):
        assert [homography(a, T, T) for a in range(T)] == list(range(T))
    for T_k in range(1, 30):
        for T_S in range(1, T_k + 1):
            m = [homography(a, T_k, T_S) for a in range(T_k)]
            assert all(x <= y for x, y in zip(m, m[1:]))
            assert m[0] >= 0 and m[-1] < T_S


def test_projection_hand_tables(golden_dir):
    for case in load(golden_dir, "hand_tables.json")["projection"]["cases"]:
        # scale l = 2 of a 3-scale schedule at step S=2, mapped to step k=3 (l' = 3)
        g = Geometry([1, case["h_l"], case["h_lp"]], [1, case["h_l"], case["h_lp"]], 8, 0)
        assert g.eh(2) == case["e_l"] and g.eh(3) == case["e_lp"]
        got = []
        for tu in case["tiles"]:
            mapped = map_block(g, g.block_id(2, tu, 0), 2, 3)
            l, mu, mv = g.decompose_block(mapped)
            assert l == 3 and mv == 0
            got.append(mu)
        assert got == case["mapped"]


def test_map_block_alignment_identity_monotone_injective():
    g = Geometry(INF_SIDES, INF_SIDES, 8, 4)
    S = 10
    for v in range(g.nb_le(S)):
        assert map_block(g, v, S, S) == v  # ratio one: identity
    for k in (11, 12, 13):
        mapped = [map_block(g, v, S, k) for v in range(g.nb_le(S))]
        for v, mv in zip(range(g.nb_le(S)), mapped):
            l, _, _ = g.decompose_block(v)
            assert g.decompose_block(mv)[0] == l + (k - S)  # Align: l' = k - (S - l)
        assert len(set(mapped)) == len(mapped)  # injective (every h_l' >= h_l here)
        assert mapped == sorted(mapped)  # monotone in block id


def test_local_blocks_invariants_and_footprint(golden_dir):
    g = Geometry(INF_SIDES, INF_SIDES, 8, 4)
    k = 13
    fp = load(golden_dir, "hand_tables.json")["footprint_64_on_48_b8"]["tile_ranges"]
    for r in (0, 1, 2):
        rows = local_blocks(g, k, r)
        assert len(rows) == 64
        for gi, row in enumerate(rows):
            a, c = divmod(gi, 8)
            assert row == sorted(set(row))
            assert g.block_id(k, a, c) in row  # every tile keeps its own block
            assert set(sink_blocks(g)) <= set(row)
            win = [v for v in row if g.decompose_block(v)[0] == k]
            na = min(7, a + r) - max(0, a - r) + 1
            nc = min(7, c + r) - max(0, c - r) + 1
            assert len(win) == na * nc
            prev = [g.decompose_block(v)[1:] for v in row if g.decompose_block(v)[0] == k - 1]
            want = [(x, y) for x in range(fp[a][0], fp[a][1] + 1) for y in range(fp[c][0], fp[c][1] + 1)]
            assert sorted(prev) == want
            assert len(row) == len(sink_blocks(g)) + len(win) + len(prev)


def test_config0_keeps_every_block():
    g = tiny_geom()
    rows = local_blocks(g, 4, 1)
    assert all(r == list(range(7)) for r in rows)


# ---------------------------------------------------------------- rows, CSR, sparse attention
def test_build_rows_and_csr():
    g = Geometry(INF_SIDES, INF_SIDES, 8, 4)
    S, k, topk = 10, 13, 8
    rng = np.random.default_rng(8)
    topk_idx = np.stack([[sorted(rng.choice(g.nb_le(S), topk, replace=False)) for _ in range(g.tiles(S))]
                         for _ in range(3)])
    local = local_blocks(g, k, 1)
    rows = build_rows(g, S, k, topk_idx, local)
    for bh in range(3):
        for gi, row in enumerate(rows[bh]):
            a, c = divmod(gi, 8)
            gs = (a // 2) * 4 + c // 2  # 64 -> 32 tiles: the homography halves
            want = set(local[gi]) | {map_block(g, int(v), S, k) for v in topk_idx[bh, gs]}
            assert row == sorted(want)
    ptr, col = rows_to_csr([r for per in rows for r in per])
    assert ptr[0] == 0 and ptr[-1] == len(col) and (np.diff(ptr) > 0).all()
    order = longest_first(ptr)
    n = np.diff(ptr)
    assert sorted(order) == list(range(len(n)))
    for x, y in zip(order, order[1:]):
        assert n[x] > n[y] or (n[x] == n[y] and x < y)


def test_sparse_equals_dense_when_every_block_kept():
    # The tiny schedule 1,2,4,8 with b=4, sinks 1-2 and r=1 keeps all 7 blocks.
    g = tiny_geom()
    q, k, v = make_qkv(g.h, g.w, 1, 1, 64, 8, 2, seed=0, bf16=False)
    sc = 1 / 8
    qs = q[0, 0, g.C(3):g.C(4)]
    rows = [[0, 1, 2, 3, 4, 5, 6]] * 4
    o, lse = block_sparse_attention(qs, k[0, 0, :g.C(4)], v[0, 0, :g.C(4)], g, 4, rows, sc)
    od, ld = dense_attention(qs, k[0, 0, :g.C(4)], v[0, 0, :g.C(4)], sc)
    assert np.abs(o - od).max() < 1e-13 and np.abs(lse - ld).max() < 1e-12


def test_block_mass_indicator():
    # V[j, c] = 1 if token j is in block c: output channel c is the attention mass on block c.
    g = Geometry([1, 2, 4, 8, 16], [1, 2, 4, 8, 16], 4, 2)
    k = 5
    rng = np.random.default_rng(9)
    local = local_blocks(g, k, 0)
    NB = g.nb_le(k)
    V = np.zeros((g.C(k), NB))
    for c in range(NB):
        V[g.block_tokens(c), c] = 1.0
    q = rng.standard_normal((g.N(k), 6))
    kk = rng.standard_normal((g.C(k), 6))
    o, _ = block_sparse_attention(q, kk, V, g, k, local, 0.5)
    for gi, row in enumerate(local):
        qs = g.tile_local_tokens(k, gi // g.Tw(k), gi % g.Tw(k))
        dropped = [c for c in range(NB) if c not in row]
        assert (o[np.ix_(qs, dropped)] == 0).all()
        assert np.abs(o[qs].sum(axis=1) - 1).max() < 1e-12
        assert (o[np.ix_(qs, row)] > 0).all()


def test_gather_form_equals_mask_form():
    g = Geometry([1, 2, 3, 5, 7, 10, 13], [1, 2, 3, 5, 7, 10, 13], 4, 2)
    S, k = 6, 7
    q, kk, v = make_qkv(g.h, g.w, 1, 2, 16, 2, 2, seed=3, bf16=True)
    local = local_blocks(g, k, 1)
    sc = pooled_scores(q[0, 0, g.C(S - 1):g.C(S)], kk[0, 0, :g.C(S)], 0.25, g, S)
    topk_idx = np.array([[topk_blocks(r, 3) for r in sc]])
    rows = build_rows(g, S, k, topk_idx, local)[0]
    M = block_mask(g, k, rows)
    assert M.any(axis=1).all()
    o1, l1 = block_sparse_attention(q[0, 0, g.C(k - 1):g.C(k)], kk[0, 0, :g.C(k)], v[0, 0, :g.C(k)], g, k, rows, 0.25)
    o2, l2 = block_sparse_attention_gather(q[0, 0, g.C(k - 1):g.C(k)], kk[0, 0, :g.C(k)], v[0, 0, :g.C(k)], g, k, rows, 0.25)
    assert np.abs(o1 - o2).max() < 1e-13 and np.abs(l1 - l2).max() < 1e-12


def test_synth_generator_is_seeded_and_shaped():
    h = [1, 2, 4]
    a = make_qkv(h, h, 2, 3, 16, 2, 1, seed=5)
    b = make_qkv(h, h, 2, 3, 16, 2, 1, seed=5)
    for x, y in zip(a, b):
        assert x.shape == (2, 3, 21, 16) and x.dtype == np.float32
        assert (x == y).all()
        # bf16-representable: low 16 bits of every float are zero
        assert (x.view(np.uint32) & 0xFFFF == 0).all()


def test_projection_nonsquare_hand_table(golden_dir):
    c = load(golden_dir, "hand_tables.json")["projection_nonsquare"]
    g = Geometry([1, c["h_l"], c["h_lp"]], [1, c["w_l"], c["w_lp"]], c["b"], 0)
    for (tu, tv), want in zip(c["tiles"], c["mapped"]):
        l, mu, mv = g.decompose_block(map_block(g, g.block_id(2, tu, tv), 2, 3))
        assert (l, mu, mv) == (3, want[0], want[1])


def test_footprint_hand_table_with_ceiling(golden_dir):
    fp = load(golden_dir, "hand_tables.json")["footprint_7_on_5_b2"]["tile_ranges"]
    g = Geometry([1, 5, 7], [1, 5, 7], 2, 0)
    rows = local_blocks(g, 3, 0)
    for gi, row in enumerate(rows):
        a, c = divmod(gi, g.Tw(3))
        prev = sorted(g.decompose_block(v)[1:] for v in row if g.decompose_block(v)[0] == 2)
        assert prev == [(x, y) for x in range(fp[a][0], fp[a][1] + 1) for y in range(fp[c][0], fp[c][1] + 1)]


def test_footprint_is_positive_measure_overlap():
    # A scale-(k-1) tile is in the footprint iff its span overlaps, with positive
    # length, the query tile's span rescaled to scale k-1 (exact rationals).
    for n_k in range(1, 26):
        for n_p in range(1, n_k + 1):
            for b in (1, 2, 3, 4, 8):
                g = Geometry([n_p, n_k], [1, 1], b, 0)
                rows = local_blocks(g, 2, 0)
                e_k, e_p = g.eh(2), g.eh(1)
                for a in range(g.Th(2)):
                    lo = Fraction(a * e_k * n_p, n_k)
                    hi = Fraction(min((a + 1) * e_k, n_k) * n_p, n_k)
                    want = [t for t in range(g.Th(1)) if t * e_p < hi and min((t + 1) * e_p, n_p) > lo]
                    got = sorted(g.decompose_block(v)[1] for v in rows[a] if g.decompose_block(v)[0] == 1)
                    assert got == want, (n_k, n_p, b, a)


# ---------------------------------------------------------------- covering projection
def test_cover_projection_hand_tables(golden_dir):
    for case in load(golden_dir, "hand_tables.json")["projection_cover"]["cases"]:
        # scale l = 2 of a square 3-scale schedule at step S=2, mapped to step k=3 (l' = 3), b = 8
        g = Geometry([1, case["h_l"], case["h_lp"]], [1, case["h_l"], case["h_lp"]], 8, 0)
        c_lo, c_hi = case["tile_ranges"][0]  # column span of the source column tile 0
        for tu, (lo, hi) in zip(case["tiles"], case["tile_ranges"]):
            want = [g.block_id(3, a, c) for a in range(lo, hi + 1) for c in range(c_lo, c_hi + 1)]
            assert map_block_cover(g, g.block_id(2, tu, 0), 2, 3) == want, (case, tu)


def _cover_geometries():
    inf = [1, 2, 4, 6, 8, 12, 16, 20, 24, 32, 40, 48, 64]
    return [Geometry(inf, inf, 8, 4), Geometry(inf, inf, 16, 4), Geometry(inf + [80, 96, 128], inf + [80, 96, 128], 8, 4),
            Geometry([1, 2, 3, 5, 7, 10, 13], [1, 3, 4, 7, 9, 14, 21], 3, 1),
            Geometry([1, 2, 3, 5, 7, 10, 13], [1, 3, 4, 7, 9, 14, 21], 2, 0)]


def test_cover_contains_point_map_identity_and_monotone():
    for g in _cover_geometries():
        for S in range(1, g.L + 1):
            for v in range(g.nb_le(S)):
                assert map_block_cover(g, v, S, S) == [v]  # no scale change: the tile itself
            for k in range(S + 1, g.L + 1):
                for v in range(g.nb_le(S)):
                    cov = map_block_cover(g, v, S, k)
                    assert cov == sorted(set(cov)) and map_block(g, v, S, k) in cov
                    l, tu, tv = g.decompose_block(v)
                    assert all(g.decompose_block(x)[0] == k - (S - l) for x in cov)
                # tile ranges move forward with the source tile, per axis
                for l in range(1, S + 1):
                    lp = k - (S - l)
                    firsts = [g.decompose_block(map_block_cover(g, g.block_id(l, tu, 0), S, k)[0])[1]
                              for tu in range(g.Th(l))]
                    lasts = [g.decompose_block(map_block_cover(g, g.block_id(l, tu, 0), S, k)[-1])[1]
                             for tu in range(g.Th(l))]
                    assert firsts == sorted(firsts) and lasts == sorted(lasts) and lasts[-1] == g.Th(lp) - 1


def test_cover_is_positive_area_overlap_of_the_upsampled_tile():
    # brute force in exact rationals: a scale-l' tile is covered iff its extent meets
    # the upsampled span of the source tile with positive area
    for h, w, b in [([1, 2, 3, 5, 7, 10, 13], [1, 3, 4, 7, 9, 14, 21], 3), ([1, 2, 4, 6, 9, 12], [1, 2, 4, 6, 9, 12], 4),
                    ([1, 3, 5, 8, 11], [2, 3, 7, 10, 16], 2)]:
        g = Geometry(h, w, b, 1)
        for S in range(1, g.L):
            for k in range(S + 1, g.L + 1):
                for v in range(g.nb_le(S)):
                    l, tu, tv = g.decompose_block(v)
                    lp = k - (S - l)
                    rh, rw = Fraction(g.hh(lp), g.hh(l)), Fraction(g.ww(lp), g.ww(l))
                    x0, x1 = tu * g.eh(l), min((tu + 1) * g.eh(l), g.hh(l))
                    y0, y1 = tv * g.ew(l), min((tv + 1) * g.ew(l), g.ww(l))
                    want = []
                    for a in range(g.Th(lp)):
                        for c in range(g.Tw(lp)):
                            a0, a1 = a * g.eh(lp), min((a + 1) * g.eh(lp), g.hh(lp))
                            c0, c1 = c * g.ew(lp), min((c + 1) * g.ew(lp), g.ww(lp))
                            if max(a0, x0 * rh) < min(a1, x1 * rh) and max(c0, y0 * rw) < min(c1, y1 * rw):
                                want.append(g.block_id(lp, a, c))
                    assert map_block_cover(g, v, S, k) == want, (h, w, b, S, k, v)


def test_cover_keeps_the_selected_share_of_each_scale():
    # the blocks of a scale cover the aligned scale exactly, and any selection keeps at
    # least its share of its scale's tokens on the larger scale (kept keys stay about
    # alpha of the cache), while the point form keeps only the count of blocks
    rng = np.random.default_rng(3)
    for g in _cover_geometries():
        for S in range(2, g.L):
            for k in range(S + 1, g.L + 1):
                for l in range(1, S + 1):
                    lp = k - (S - l)
                    blocks = [g.block_id(l, a, c) for a in range(g.Th(l)) for c in range(g.Tw(l))]
                    every = set()
                    for v in blocks:
                        every.update(map_block_cover(g, v, S, k))
                    assert every == set(range(g.base(lp), g.base(lp) + g.tiles(lp)))
                    for _ in range(3):
                        sel = [v for v in blocks if rng.random() < 0.3] or blocks[:1]
                        cov = set()
                        for v in sel:
                            cov.update(map_block_cover(g, v, S, k))
                        share_src = Fraction(sum(len(g.block_tokens(v)) for v in sel), g.N(l))
                        share_dst = Fraction(sum(len(g.block_tokens(v)) for v in cov), g.N(lp))
                        assert share_dst >= share_src


def test_build_rows_cover_is_a_superset_of_point():
    inf = [1, 2, 4, 6, 8, 12, 16, 20, 24, 32, 40, 48, 64]
    g = Geometry(inf, inf, 8, 4)
    rng = np.random.default_rng(11)
    topk = np.sort(np.stack([rng.choice(g.nb_le(10), 8, replace=False) for _ in range(2 * g.tiles(10))]), axis=1)
    topk = topk.reshape(2, g.tiles(10), 8)
    for k in (11, 12, 13):
        loc = local_blocks(g, k, 1)
        point = build_rows(g, 10, k, topk, loc)
        cover = build_rows(g, 10, k, topk, loc, projection="cover")
        for bh in range(2):
            for t in range(g.tiles(k)):
                assert set(point[bh][t]) <= set(cover[bh][t]) and cover[bh][t] == sorted(set(cover[bh][t]))
        with pytest.raises(ValueError):
            build_rows(g, 10, k, topk, loc, projection="area")

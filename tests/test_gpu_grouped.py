"""GPU parity of every launch form of the block-sparse kernel against the fp64
oracle: one query tile per workgroup, and groups of 2, 4 or 8 neighbouring
tiles per workgroup walking the union of their rows (each tile still attends
to exactly its own blocks). The form is chosen through the library's launch
knobs, read at every call.

Rows are seeded random ascending block subsets with out-of-range ids mixed in
(skipped by definition), empty rows, and rows longer than a group's merge
capacity (those groups are served tile by tile).
"""
import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import INF_SIDES, assert_close, make_case, note, oracle_geometry, scale_of, to_dev
from paper_2602_04361_amd import sparvar as sv
from test_gpu_parity import run_case

pytestmark = pytest.mark.gpu

FORMS = {
    "per_tile": {"SPARSE_GROUP_WAVES": "0"},
    "group4": {"SPARSE_GROUP_WAVES": "4"},
    "group8": {"SPARSE_GROUP_WAVES": "8"},
    "group8_kc32": {"SPARSE_GROUP_WAVES": "8", "SPARSE_GROUP_CHUNK": "32"},
}


def random_rows(nb, n_rows, rng, long_every, long_len, short_len):
    rows, clean = [], []
    for g in range(n_rows):
        if g % 11 == 5:
            n = 0
        elif long_every and g % long_every == 0:
            n = min(long_len, nb)
        else:
            n = int(rng.integers(1, short_len + 1))
        ids = sorted(rng.choice(nb, size=n, replace=False).tolist())
        row = list(ids)
        for _ in range(int(rng.integers(0, 3))):
            row.insert(int(rng.integers(0, len(row) + 1)), int(rng.choice([-1, -5, nb, nb + 7])))
        rows.append(row)
        clean.append(ids)
    return rows, clean


def run_rows(launch_option, form, h, w, b, ns, k, B, H, d, seed, long_every, long_len, short_len):
    for key, val in FORMS[form].items():
        launch_option(key, val)
    note(f"[grouped] form={form} h={h} w={w} b={b} k={k} B={B} H={H} d={d} seed={seed}")
    q, kk, v = make_case(h, w, B, H, d, 8, ns, seed, "bf16")
    og = oracle_geometry(h, w, b, ns)
    g = sv.Geometry(h, w, b, ns)
    Q, K, V = to_dev(q, "bf16"), to_dev(kk, "bf16"), to_dev(v, "bf16")
    rng = np.random.default_rng(seed)
    BH, G_k, nb = B * H, og.tiles(k), og.nb_le(k)
    rows, clean = random_rows(nb, BH * G_k, rng, long_every, long_len, short_len)
    ptr, col = O.rows_to_csr(rows)
    rp = torch.tensor(ptr, dtype=torch.int32, device="cuda")
    ci = torch.tensor(col, dtype=torch.int32, device="cuda")
    o = torch.full((B, H, og.N(k), d), 3.0, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(B, H, og.N(k), device="cuda")
    C0, C1 = og.C(k - 1), og.C(k)
    sv.sparvar_block_sparse_attn_fwd(g, k, Q[:, :, C0:C1], K[:, :, :C1], V[:, :, :C1], o, rp, ci, lse=lse,
                                     softmax_scale=scale_of(d))
    torch.cuda.synchronize()
    got = o.float().cpu().numpy().reshape(BH, -1, d)
    gl = lse.cpu().numpy().reshape(BH, -1)
    qf, kf, vf = q.reshape(BH, -1, d), kk.reshape(BH, -1, d), v.reshape(BH, -1, d)
    for bh in range(BH):
        per = clean[bh * G_k:(bh + 1) * G_k]
        o_ref, l_ref = O.block_sparse_attention_gather(qf[bh, C0:C1], kf[bh, :C1], vf[bh, :C1], og, k, per,
                                                       scale_of(d))
        assert_close(got[bh], o_ref, "bf16", f"{form} O head {bh}")
        fin = np.isfinite(l_ref)
        assert (np.isneginf(gl[bh]) == ~fin).all(), f"{form} empty rows head {bh}"
        assert np.abs(gl[bh][fin] - l_ref[fin]).max() <= 2e-4, f"{form} LSE head {bh}"
    return got


@pytest.mark.parametrize("form", list(FORMS))
def test_forms_infinity_last_scale(launch_option, form):
    # 8x8 tiles at 64x64 (2 waves a tile); every 9th row longer than 128 blocks
    run_rows(launch_option, form, INF_SIDES, INF_SIDES, 8, 4, 13, 1, 2, 128, 21, 9, 140, 40)


@pytest.mark.parametrize("form", ["per_tile", "group4", "group8"])
def test_forms_small_tiles_partial_groups(launch_option, form):
    # 4x4 tiles (16 queries, one wave a tile) on a 27x27 scale: edge tiles 3 wide
    # and groups hanging over the scale's edge; rows of 70 blocks exceed the
    # merge capacity of 64 entries per tile
    h = [1, 2, 3, 5, 7, 10, 13, 20, 27]
    run_rows(launch_option, form, h, h, 4, 2, 9, 1, 2, 64, 22, 7, 70, 20)


@pytest.mark.parametrize("form", ["group4", "group8"])
def test_forms_nonsquare_d64(launch_option, form):
    h = [1, 2, 3, 5, 8, 11, 17]
    w = [1, 3, 4, 7, 9, 14, 21]
    run_rows(launch_option, form, h, w, 8, 2, 7, 2, 2, 64, 23, 0, 0, 12)


@pytest.mark.parametrize("form", ["per_tile", "group4"])
def test_forms_on_pipeline_rows(launch_option, form):
    # The whole path (decision, mapping, attention at 40/48/64) with the rows the
    # mapping step writes; the automatic form is covered by the parity suite.
    for key, val in FORMS[form].items():
        launch_option(key, val)
    run_case(INF_SIDES, INF_SIDES, 8, 4, 10, [11, 12, 13], 1, 4, 128, 32, 8, 1, "bf16", seed=12,
             tiles_per_step=16)


def check_order(order, lengths, n_items, grouped, item_len):
    """order: launch positions -> items (rows, or -2 - group); a permutation of the
    items, each half of each XCD share of positions holding its own items,
    longest first (ties in item order)."""
    per = -(-n_items // 8)
    got = order[:n_items].tolist()
    items = [(-2 - v) if grouped else v for v in got]
    assert sorted(items) == list(range(n_items))
    for x in range(8):
        lo, hi = x * per, min((x + 1) * per, n_items)
        if hi <= lo:
            continue
        n = hi - lo
        w = min(((n + 1) // 2 + 3) & ~3, n)
        for a, b in ((lo, lo + w), (lo + w, hi)):
            window = items[a:b]
            assert sorted(window) == list(range(a, b))
            keys = [(-item_len(i), i) for i in window]
            assert keys == sorted(keys)


@pytest.mark.parametrize("form", ["per_tile", "group4"])
def test_launch_order_from_the_mapping(launch_option, form):
    # one mapping launch writes every step's order; the attention gives the same
    # bits with and without it, and ignores an order of the other form
    for key, val in FORMS[form].items():
        launch_option(key, val)
    from paper_2602_04361_amd.pipeline import SparsePath

    h, b, ns, S, steps, B, H, d = INF_SIDES, 8, 4, 10, [11, 12, 13], 1, 4, 128
    note(f"[order] form={form}")
    q, kk, v = make_case(h, h, B, H, d, 8, ns, 70, "bf16")
    Q, K, V = to_dev(q, "bf16"), to_dev(kk, "bf16"), to_dev(v, "bf16")
    g = sv.Geometry(h, h, b, ns)
    og = oracle_geometry(h, h, b, ns)
    path = SparsePath(g, S, steps, B, H, d, 8, 1, use_schedule=True)
    path.decision(Q, K, V)
    path.map_all(orders=True)
    torch.cuda.synchronize()
    grouped = form != "per_tile"
    for k in steps:
        rp, ci, _ = path.csr[k]
        ci_h = ci.cpu().numpy()
        M = int(rp[1].item() - rp[0].item())
        n_rows = B * H * og.tiles(k)
        lens = [int((ci_h[r * M:(r + 1) * M] >= 0).sum()) for r in range(n_rows)]
        Th, Tw = og.Th(k), og.Tw(k)
        if grouped:
            ngc, ngr = -(-Tw // 2), Th
            n_items = B * H * ngr * ngc

            def item_len(i):
                bh, gi = divmod(i, ngr * ngc)
                A, Cg = divmod(gi, ngc)
                return sum(lens[bh * Th * Tw + A * Tw + c] for c in (2 * Cg, 2 * Cg + 1) if c < Tw)
        else:
            n_items = n_rows

            def item_len(i):
                return lens[i]
        check_order(path.orders[k].cpu().numpy(), lens, n_items, grouped, item_len)
        path.attn_step(k, Q, K, V, use_schedule=False)
        torch.cuda.synchronize()
        ref = path.out[k].clone()
        path.out[k].zero_()
        path.attn_step(k, Q, K, V, use_order=True)
        torch.cuda.synchronize()
        assert torch.equal(path.out[k], ref), f"step {k}: results depend on the launch order"
        # the other kind of order is ignored: a row permutation for groups, a group order for tiles
        other = torch.arange(n_rows, dtype=torch.int32, device="cuda").flip(0) if grouped else \
            -2 - torch.arange(n_rows, dtype=torch.int32, device="cuda")
        path.out[k].zero_()
        sv.sparvar_block_sparse_attn_fwd(g, k, path.q_slice(Q, k), path.kv_prefix(K, k), path.kv_prefix(V, k),
                                         path.out[k], rp, ci, schedule=other, softmax_scale=path.scale)
        torch.cuda.synchronize()
        assert torch.equal(path.out[k], ref), f"step {k}: an order of the other form changed the results"

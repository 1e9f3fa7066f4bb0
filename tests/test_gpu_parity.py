"""GPU parity: the HIP path (called through the C ABI) against the fp64 oracle.

Block lists, top-k and schedules must match bit for bit (top-k given the GPU's
own pooled scores); pooled scores within 1e-4 after dividing by the query-tile
size; attention within max-abs 2e-2 / mean-abs 2e-3 (bf16) or 1e-5 (fp32).
"""
import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import (INF_SIDES, assert_close, csr_rows, make_case, note, oracle_geometry, scale_of,
                         to_dev, torch_dtype)
from paper_2602_04361_amd import sparvar as sv
from paper_2602_04361_amd.pipeline import SparsePath

pytestmark = pytest.mark.gpu

LSE_TOL = {"bf16": 2e-4, "f32": 1e-5}


def run_case(h, w, b, ns, S, steps, B, H, d, F, topk, r, dtype, seed=0, dil=0, heads=None, tiles_per_step=None,
             check_schedule=True, projection="point"):
    note(f"[case] h={h} w={w} b={b} ns={ns} S={S} steps={steps} B={B} H={H} d={d} topk={topk} r={r} "
         f"dil={dil} {dtype} seed={seed} projection={projection}")
    q, k, v = make_case(h, w, B, H, d, F, ns, seed, dtype)
    Qd, Kd, Vd = to_dev(q, dtype), to_dev(k, dtype), to_dev(v, dtype)
    g = sv.Geometry(h, w, b, ns)
    og = oracle_geometry(h, w, b, ns)
    path = SparsePath(g, S, steps, B, H, d, topk, r, dil, dtype=torch_dtype(dtype), use_schedule=True,
                      local_lists=True, projection=projection)
    path.build_local()
    path.decision(Qd, Kd, Vd)
    lse_k = {}
    for kk in steps:
        path.map_step(kk)
        lse_k[kk] = torch.empty(B, H, og.N(kk), dtype=torch.float32, device="cuda")
        path.attn_step(kk, Qd, Kd, Vd, lse=lse_k[kk])
    torch.cuda.synchronize()
    sc = scale_of(d)
    BH = B * H
    heads = list(range(BH)) if heads is None else heads
    qf = q.reshape(BH, -1, d)
    kf = k.reshape(BH, -1, d)
    vf = v.reshape(BH, -1, d)

    # decision scale: dense attention + LSE
    oS = path.o_S.float().cpu().numpy().reshape(BH, -1, d)
    lS = path.lse_S.cpu().numpy().reshape(BH, -1)
    scores = path.scores.cpu().numpy().reshape(BH, og.tiles(S), og.nb_le(S))
    for bh in heads:
        o_ref, l_ref = O.dense_attention(qf[bh, og.C(S - 1):og.C(S)], kf[bh, :og.C(S)], vf[bh, :og.C(S)], sc)
        assert_close(oS[bh], o_ref, dtype, f"dense O at S, head {bh}")
        assert np.abs(lS[bh] - l_ref).max() <= LSE_TOL[dtype], f"dense LSE at S, head {bh}"
        # pooled scores, normalised by the query-tile size
        s_ref = O.pooled_scores(qf[bh, og.C(S - 1):og.C(S)], kf[bh, :og.C(S)], sc, og, S)
        nq = np.array([len(og.tile_local_tokens(S, t // og.Tw(S), t % og.Tw(S))) for t in range(og.tiles(S))])
        err = np.abs(scores[bh] - s_ref) / nq[:, None]
        assert err.max() <= 1e-4, f"pooled scores head {bh}: {err.max():.3e}"

    # top-k: bit-exact given the GPU's scores
    tk = path.topk_idx.cpu().numpy().reshape(BH, og.tiles(S), topk)
    for bh in range(BH):
        for t in range(og.tiles(S)):
            assert tk[bh, t].tolist() == O.topk_blocks(scores[bh, t], topk), (bh, t)

    merged = {}
    for kk in steps:
        # local rows: bit-exact
        loc = O.local_blocks(og, kk, r, dil)
        assert csr_rows(*path.local[kk]) == loc, f"local rows step {kk}"
        # merged rows: bit-exact
        rows = O.build_rows(og, S, kk, tk, loc, projection=projection)
        rp, ci, sch = path.csr[kk]
        got = csr_rows(rp, ci, padded=True)
        assert got == [r_ for per in rows for r_ in per], f"CSR rows step {kk}"
        stride = rp[1].item() - rp[0].item()
        assert (np.diff(rp.cpu().numpy()) == stride).all()
        # the mapping call generating the local rows itself gives the same rows
        path.local_lists = False
        path.map_step(kk)
        torch.cuda.synchronize()
        assert csr_rows(rp, ci, padded=True) == got, f"CSR rows (in-call local rows) step {kk}"
        path.local_lists = True
        merged[kk] = got
        if check_schedule and sch is not None:
            compact_ptr, _ = O.rows_to_csr(got)
            assert sch.cpu().numpy().tolist() == O.longest_first(compact_ptr), f"schedule step {kk}"
        # attention
        ok = path.out[kk].float().cpu().numpy().reshape(BH, -1, d)
        lk = lse_k[kk].cpu().numpy().reshape(BH, -1)
        for bh in heads:
            if tiles_per_step is None:
                tiles = list(range(og.tiles(kk)))
            else:
                rng = np.random.default_rng(1000 * kk + bh)
                tiles = sorted(rng.choice(og.tiles(kk), size=min(tiles_per_step, og.tiles(kk)), replace=False))
            o_ref, l_ref = O.block_sparse_attention_gather(qf[bh, og.C(kk - 1):og.C(kk)], kf[bh, :og.C(kk)],
                                                           vf[bh, :og.C(kk)], og, kk, rows[bh], sc, tiles=tiles)
            qs = np.concatenate([og.tile_local_tokens(kk, t // og.Tw(kk), t % og.Tw(kk)) for t in tiles])
            mx, mean = assert_close(ok[bh][qs], o_ref[qs], dtype, f"sparse O step {kk} head {bh}")
            assert np.abs(lk[bh][qs] - l_ref[qs]).max() <= LSE_TOL[dtype], f"sparse LSE step {kk} head {bh}"
        note(f"  step {kk}: ok (last head max {mx:.2e} mean {mean:.2e})")
    # every step's rows from one multi-step mapping launch: the same rows
    for kk in steps:
        path.csr[kk][1].fill_(-7)
    path.map_all()
    torch.cuda.synchronize()
    for kk in steps:
        assert csr_rows(path.csr[kk][0], path.csr[kk][1], padded=True) == merged[kk], f"multi-step rows {kk}"
    return path, (Qd, Kd, Vd)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tiny_config_every_block_kept(dtype):
    # Schedule 1,2,4,8, b=4, sinks 1-2, top-2, r=1: all 7 blocks are kept, so
    # the sparse result must equal dense attention over the whole cache.
    h = [1, 2, 4, 8]
    path, (Qd, Kd, Vd) = run_case(h, h, 4, 2, 3, [4], 1, 1, 64, 8, 2, 1, dtype)
    og = oracle_geometry(h, h, 4, 2)
    q, k, v = make_case(h, h, 1, 1, 64, 8, 2, 0, dtype)
    o_ref, _ = O.dense_attention(q[0, 0, og.C(3):og.C(4)], k[0, 0], v[0, 0], scale_of(64))
    assert_close(path.out[4].float().cpu().numpy()[0, 0], o_ref, dtype, "sparse == dense")
    assert all(len(r) == 7 for r in csr_rows(*path.csr[4][:2], padded=True))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("r", [0, 1])
def test_tiny_sparse_square(dtype, r):
    h = [1, 2, 4, 8, 16]
    run_case(h, h, 4, 2, 4, [5], 1, 2, 64, 4, 2, r, dtype, seed=1)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_odd_sides_partial_tiles(dtype):
    h = [1, 2, 3, 5, 7, 10, 13]
    run_case(h, h, 4, 2, 5, [6, 7], 2, 2, 128, 8, 3, 1, dtype, seed=2)


def test_nonsquare_scales_and_dilation():
    h = [1, 2, 3, 5, 8, 11]
    w = [1, 3, 4, 7, 9, 14]
    run_case(h, w, 4, 2, 4, [5, 6], 1, 3, 128, 8, 3, 1, "bf16", seed=3, dil=1)


def test_topk_larger_than_candidates():
    h = [1, 2, 4, 8, 16]
    run_case(h, h, 4, 2, 3, [4, 5], 1, 2, 64, 4, 9, 1, "bf16", seed=4)


def test_block_edge_16_multiwave_tiles():
    # 256-query tiles (8 waves) and 256-token blocks split into 64-key chunks.
    run_case(INF_SIDES, INF_SIDES, 16, 4, 10, [13], 1, 2, 128, 32, 8, 1, "bf16", seed=5, tiles_per_step=6)


def test_infinity_config_full_size():
    # B=2, H=16, d=128, S=32x32, top-8, r=1, steps 40/48/64: every index list
    # bit-exact; attention sampled on three heads.
    run_case(INF_SIDES, INF_SIDES, 8, 4, 10, [11, 12, 13], 2, 16, 128, 32, 8, 1, "bf16", seed=0,
             heads=[0, 17, 31], tiles_per_step=12)


def test_schedule_2048_sampled():
    # 2048x2048-shaped schedule: scales up to 128x128 (42521 keys), decision at
    # 64x64 with 172 candidate blocks, top-16, steps 80/96/128. Every index list
    # bit-exact on all 16 heads; attention and decision outputs sampled on two heads.
    sides = INF_SIDES + [80, 96, 128]
    run_case(sides, sides, 8, 4, 13, [14, 15, 16], 1, 16, 128, 32, 16, 1, "bf16", seed=6, heads=[0, 9],
             tiles_per_step=12)


def test_infinity_wide_32_heads_full_size():
    # the wider variant: B=2, H=32 (64 planes), same schedule and sparsity rules.
    # Every index list bit-exact on all heads; attention sampled on three heads.
    run_case(INF_SIDES, INF_SIDES, 8, 4, 10, [11, 12, 13], 2, 32, 128, 32, 8, 1, "bf16", seed=2,
             heads=[0, 45, 63], tiles_per_step=8)


@pytest.mark.parametrize("b,topk,r", [(b, t, r) for b in (8, 16) for r in (1, 2) for t in (4, 8, 16, 32)])
def test_sparsity_sweep_settings_full_size(b, topk, r):
    # all 16 settings of the sparsity sweep on the Infinity layer (B=2, H=16,
    # d=128): top-k 4, 8, 16 and 32, blocks of 8x8 and 16x16 tokens, local radius
    # 1 and 2. Index lists bit-exact on all heads; attention sampled on two heads.
    run_case(INF_SIDES, INF_SIDES, b, 4, 10, [11, 12, 13], 2, 16, 128, 32, topk, r, "bf16", seed=40 + topk + r,
             heads=[3, 26], tiles_per_step=6)


def test_cover_projection_infinity_full_size():
    # covering projection of the mapped blocks on the Infinity layer (B=2, H=16,
    # d=128, S=32x32, top-8, r=1): every index list bit-exact on all heads,
    # attention sampled on three heads
    run_case(INF_SIDES, INF_SIDES, 8, 4, 10, [11, 12, 13], 2, 16, 128, 32, 8, 1, "bf16", seed=90,
             heads=[0, 17, 31], tiles_per_step=12, projection="cover")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_cover_projection_odd_nonsquare(dtype):
    # non-square scales with odd sides and a non-integer ratio between aligned scales
    h = [1, 2, 3, 5, 8, 11]
    w = [1, 3, 4, 7, 9, 14]
    run_case(h, w, 4, 1, 3, [4, 5, 6], 1, 2, 64, 8, 3, 1, dtype, seed=91, dil=1, projection="cover")


def test_cover_projection_2048_schedule_sampled():
    # the 2048x2048-shaped schedule, decision at 64x64, top-16, covering projection
    sides = INF_SIDES + [80, 96, 128]
    run_case(sides, sides, 8, 4, 13, [14, 15, 16], 1, 16, 128, 32, 16, 1, "bf16", seed=92, heads=[0, 9],
             tiles_per_step=8, projection="cover")


# ---------------------------------------------------------------- dense kernel edge cases
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n_q,n_kv,d", [(1, 1, 64), (33, 65, 64), (100, 333, 128), (257, 129, 128)])
def test_dense_ragged(dtype, n_q, n_kv, d):
    note(f"[dense] n_q={n_q} n_kv={n_kv} d={d} {dtype}")
    rng = np.random.default_rng(n_q * 1000 + n_kv)
    q = rng.standard_normal((2, 3, n_q, d)).astype(np.float32)
    k = rng.standard_normal((2, 3, n_kv, d)).astype(np.float32)
    v = rng.standard_normal((2, 3, n_kv, d)).astype(np.float32)
    if dtype == "bf16":
        from paper_2602_04361_amd.synth import round_to_bf16
        q, k, v = round_to_bf16(q), round_to_bf16(k), round_to_bf16(v)
    Q, K, V = to_dev(q, dtype), to_dev(k, dtype), to_dev(v, dtype)
    o = torch.empty_like(Q)
    lse = torch.empty(2, 3, n_q, dtype=torch.float32, device="cuda")
    sv.sparvar_dense_attn_fwd(Q, K, V, o, lse, softmax_scale=scale_of(d))
    torch.cuda.synchronize()
    for b in range(2):
        for hh in range(3):
            o_ref, l_ref = O.dense_attention(q[b, hh], k[b, hh], v[b, hh], scale_of(d))
            assert_close(o[b, hh].float().cpu().numpy(), o_ref, dtype, f"dense {b},{hh}")
            assert np.abs(lse[b, hh].cpu().numpy() - l_ref).max() <= LSE_TOL[dtype]


def test_dense_full_64_scale_sampled():
    # Dense baseline at the 64x64 step of the Infinity schedule (B=2, H=16):
    # 4096 queries against 10521 keys, rows sampled.
    B, H, d = 2, 16, 128
    note("[dense] 64x64 step of the Infinity schedule, B=2 H=16 d=128")
    q, k, v = make_case(INF_SIDES, INF_SIDES, B, H, d, 32, 4, 0, "bf16")
    og = oracle_geometry(INF_SIDES, INF_SIDES, 8, 4)
    Q, K, V = to_dev(q, "bf16"), to_dev(k, "bf16"), to_dev(v, "bf16")
    qk = Q[:, :, og.C(12):og.C(13)]
    o = torch.empty(B, H, og.N(13), d, dtype=torch.bfloat16, device="cuda")
    sv.sparvar_dense_attn_fwd(qk, K, V, o, None, softmax_scale=scale_of(d))
    torch.cuda.synchronize()
    rng = np.random.default_rng(7)
    for bh in (0, 9, 31):
        b, hh = divmod(bh, H)
        rows = rng.choice(og.N(13), 256, replace=False)
        o_ref, _ = O.dense_attention(q[b, hh, og.C(12) + rows], k[b, hh], v[b, hh], scale_of(d))
        assert_close(o[b, hh].float().cpu().numpy()[rows], o_ref, "bf16", f"dense 64x64 head {bh}")


# ---------------------------------------------------------------- CSR edge cases
def test_empty_and_invalid_csr_entries():
    h = [1, 2, 4, 8]
    d = 64
    q, k, v = make_case(h, h, 1, 1, d, 8, 2, 9, "f32")
    g = sv.Geometry(h, h, 4, 2)
    og = oracle_geometry(h, h, 4, 2)
    Q, K, V = to_dev(q, "f32"), to_dev(k, "f32"), to_dev(v, "f32")
    # rows: tile 0 empty; tile 1 with out-of-range ids mixed in; tile 2 one block; tile 3 all blocks
    rows = [[], [-1, 2, 5, 7, 99], [6], [0, 1, 2, 3, 4, 5, 6]]
    clean = [[], [2, 5], [6], [0, 1, 2, 3, 4, 5, 6]]
    ptr, col = O.rows_to_csr(rows)
    rp = torch.tensor(ptr, dtype=torch.int32, device="cuda")
    ci = torch.tensor(col, dtype=torch.int32, device="cuda")
    o = torch.full((1, 1, 64, d), 7.0, device="cuda")
    lse = torch.empty(1, 1, 64, device="cuda")
    sv.sparvar_block_sparse_attn_fwd(g, 4, Q[:, :, og.C(3):], K, V, o, rp, ci, lse=lse, softmax_scale=scale_of(d))
    torch.cuda.synchronize()
    o_ref, l_ref = O.block_sparse_attention(q[0, 0, og.C(3):], k[0, 0], v[0, 0], og, 4, clean, scale_of(d))
    got = o[0, 0].cpu().numpy()
    t0 = og.tile_local_tokens(4, 0, 0)
    assert (got[t0] == 0).all() and np.isneginf(lse[0, 0].cpu().numpy()[t0]).all()
    rest = np.setdiff1d(np.arange(64), t0)
    assert_close(got[rest], o_ref[rest], "f32", "rows with invalid ids skipped")


def test_deterministic_and_schedule_invariant():
    h = INF_SIDES
    B, H, d = 1, 4, 128
    q, k, v = make_case(h, h, B, H, d, 32, 4, 11, "bf16")
    Q, K, V = to_dev(q, "bf16"), to_dev(k, "bf16"), to_dev(v, "bf16")
    g = sv.Geometry(h, h, 8, 4)
    path = SparsePath(g, 10, [13], B, H, d, 8, 1, use_schedule=True)
    path.build_local()
    path.run(Q, K, V)
    torch.cuda.synchronize()
    first = path.out[13].clone()
    csr_first = [t.clone() for t in path.csr[13]]
    path.run(Q, K, V)
    torch.cuda.synchronize()
    assert torch.equal(first, path.out[13])
    for a, b_ in zip(csr_first, path.csr[13]):
        assert torch.equal(a, b_)
    path.attn_step(13, Q, K, V, use_schedule=False)
    torch.cuda.synchronize()
    assert torch.equal(first, path.out[13])


@pytest.mark.parametrize("group_waves", ["0", "4"])
def test_full_rows_past_the_chunk_table(launch_option, group_waves):
    # every 8x8 tile of the 64x64 scale lists all 172 blocks of the Infinity cache:
    # 344 chunks of 32 keys per row, past the 256-entry chunk table (refills), and
    # for pairs of tiles past the row-merge capacity (served tile by tile); the
    # result is dense attention over the 10521-token cache
    launch_option("SPARSE_GROUP_WAVES", group_waves)
    h, d = INF_SIDES, 128
    note(f"[parity] full rows at 64x64, group waves {group_waves}")
    g = sv.Geometry(h, h, 8, 4)
    og = oracle_geometry(h, h, 8, 4)
    q, k, v = make_case(h, h, 1, 2, d, 32, 4, 64, "bf16")
    NB, G = og.nb_le(13), og.tiles(13)
    rows = 2 * G
    rp = torch.arange(0, (rows + 1) * NB, NB, dtype=torch.int32, device="cuda")
    ci = torch.arange(NB, dtype=torch.int32, device="cuda").repeat(rows)
    n0, n1 = og.C(12), og.C(13)
    Q = to_dev(q[:, :, n0:n1], "bf16")
    K, V = to_dev(k, "bf16"), to_dev(v, "bf16")
    o = torch.empty_like(Q)
    sv.sparvar_block_sparse_attn_fwd(g, 13, Q, K, V, o, rp, ci, softmax_scale=scale_of(d))
    torch.cuda.synchronize()
    got = o.float().cpu().numpy()
    for bh in range(2):
        ref, _ = O.dense_attention(q[0, bh, n0:n1], k[0, bh], v[0, bh], scale_of(d))
        assert_close(got[0, bh], ref, "bf16", f"full rows head {bh}")

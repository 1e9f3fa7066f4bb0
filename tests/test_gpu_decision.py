"""GPU parity of the fused decision step (dense attention + LSE, pooled block
scores and top-k at the decision scale in one call) against the fp64 oracle,
and against the two-call path on the same seeded inputs.

O_S within the bf16 attention tolerance, LSE within 2e-4, pooled scores within
1e-4 after dividing by the query-tile size, top-k bit-exact given the call's own
scores (ties to the lower id, -1 padding past the candidate count).
"""
import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import INF_SIDES, assert_close, make_case, note, oracle_geometry, scale_of, to_dev
from paper_2602_04361_amd import sparvar as sv

pytestmark = pytest.mark.gpu


def decision_case(h, w, b, ns, S, B, H, d, F, topk, seed, heads=None):
    note(f"[decision] h={h} w={w} b={b} S={S} B={B} H={H} d={d} topk={topk} seed={seed}")
    q, k, v = make_case(h, w, B, H, d, F, ns, seed, "bf16")
    og = oracle_geometry(h, w, b, ns)
    g = sv.Geometry(h, w, b, ns)
    Q, K, V = to_dev(q, "bf16"), to_dev(k, "bf16"), to_dev(v, "bf16")
    C0, C1 = og.C(S - 1), og.C(S)
    NS, G_S, NB = og.N(S), og.tiles(S), og.nb_le(S)
    o = torch.empty(B, H, NS, d, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(B, H, NS, device="cuda")
    scores = torch.empty(B, H, G_S, NB, device="cuda")
    idx = torch.empty(B, H, G_S, topk, dtype=torch.int32, device="cuda")
    sv.sparvar_decision_step(g, S, Q[:, :, C0:C1], K[:, :, :C1], V[:, :, :C1], o, lse, scores, topk, idx,
                             softmax_scale=scale_of(d))
    torch.cuda.synchronize()
    BH = B * H
    qf, kf, vf = q.reshape(BH, -1, d), k.reshape(BH, -1, d), v.reshape(BH, -1, d)
    got_o = o.float().cpu().numpy().reshape(BH, NS, d)
    got_l = lse.cpu().numpy().reshape(BH, NS)
    got_s = scores.cpu().numpy().reshape(BH, G_S, NB)
    got_i = idx.cpu().numpy().reshape(BH, G_S, topk)
    nq = np.array([len(og.tile_local_tokens(S, t // og.Tw(S), t % og.Tw(S))) for t in range(G_S)])
    for bh in (range(BH) if heads is None else heads):
        o_ref, l_ref = O.dense_attention(qf[bh, C0:C1], kf[bh, :C1], vf[bh, :C1], scale_of(d))
        assert_close(got_o[bh], o_ref, "bf16", f"O_S head {bh}")
        assert np.abs(got_l[bh] - l_ref).max() <= 2e-4, f"LSE head {bh}"
        s_ref = O.pooled_scores(qf[bh, C0:C1], kf[bh, :C1], scale_of(d), og, S)
        err = np.abs(got_s[bh] - s_ref) / nq[:, None]
        assert err.max() <= 1e-4, f"scores head {bh}: {err.max():.3e}"
    for bh in range(BH):
        for t in range(G_S):
            assert got_i[bh, t].tolist() == O.topk_blocks(got_s[bh, t], topk), (bh, t)
    return (Q, K, V), (o, lse, scores, idx), g


def test_infinity_decision_scale_and_two_call_agreement():
    # 32x32 decision scale of the Infinity schedule, 8x8 tiles (two key splits per workgroup)
    S, B, H, d, topk = 10, 1, 4, 128, 8
    (Q, K, V), (o, lse, scores, idx), g = decision_case(INF_SIDES, INF_SIDES, 8, 4, S, B, H, d, 32, topk, 31)
    og = oracle_geometry(INF_SIDES, INF_SIDES, 8, 4)
    C0, C1 = og.C(S - 1), og.C(S)
    o2, l2 = torch.empty_like(o), torch.empty_like(lse)
    s2, i2 = torch.empty_like(scores), torch.empty_like(idx)
    sv.sparvar_dense_attn_fwd(Q[:, :, C0:C1], K[:, :, :C1], V[:, :, :C1], o2, l2, softmax_scale=scale_of(d))
    sv.sparvar_select_blocks(g, S, Q[:, :, C0:C1], K[:, :, :C1], l2, topk, i2, scores_out=s2,
                             softmax_scale=scale_of(d))
    torch.cuda.synchronize()
    assert (o.float() - o2.float()).abs().max().item() <= 2e-2
    assert (lse - l2).abs().max().item() <= 2e-4
    assert (scores - s2).abs().max().item() / 64 <= 1e-4
    # the fused call is deterministic
    o3, l3, s3, i3 = torch.empty_like(o), torch.empty_like(lse), torch.empty_like(scores), torch.empty_like(idx)
    sv.sparvar_decision_step(g, S, Q[:, :, C0:C1], K[:, :, :C1], V[:, :, :C1], o3, l3, s3, topk, i3,
                             softmax_scale=scale_of(d))
    torch.cuda.synchronize()
    assert torch.equal(o, o3) and torch.equal(lse, l3) and torch.equal(scores, s3) and torch.equal(idx, i3)


def test_small_tiles_d64_partial_tiles_topk_padding():
    # 4x4 tiles (one wave a tile), 13x13 decision scale with 1-wide edge tiles,
    # top-40 of 36 candidates: all kept, padded with -1
    h = [1, 2, 3, 5, 7, 10, 13]
    decision_case(h, h, 4, 2, 7, 2, 2, 64, 8, 40, 32)


def test_nonsquare_d128_topk3():
    h = [1, 2, 3, 5, 8, 11, 17]
    w = [1, 3, 4, 7, 9, 14, 21]
    decision_case(h, w, 8, 2, 7, 1, 3, 128, 8, 3, 33)


def test_block_edge_16_single_split():
    # 16x16 tiles (256 queries, 8 waves, one key split)
    decision_case(INF_SIDES, INF_SIDES, 16, 4, 10, 1, 2, 128, 32, 8, 34)


def test_fallback_shapes_give_the_same_definitions():
    # d=64 with 256-query tiles runs the two-call sequence inside the entry point
    decision_case(INF_SIDES[:10], INF_SIDES[:10], 16, 4, 10, 1, 2, 64, 16, 4, 35)

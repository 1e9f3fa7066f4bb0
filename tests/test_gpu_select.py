"""GPU parity of block selection under ties (Sec. 3.2, TopK; ties go to the lower
block id) and of the mapping call's status word, through the C ABI.

Random fp32 scores essentially never tie, so the tie rule is forced here: with
integer-valued scores given to sparvar_select_blocks (scores_in), and through
the fused decision kernel with Q = 0 at the decision scale, where every key has
probability exactly 1/N and blocks of equal size get bit-identical masses."""
import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import INF_SIDES, csr_rows, make_case, note, oracle_geometry, scale_of, to_dev
from paper_2602_04361_amd import sparvar as sv
from paper_2602_04361_amd.pipeline import SparsePath

pytestmark = pytest.mark.gpu


def tie_crossing_rows(scores, topk):
    """Rows whose topk-th and (topk+1)-th largest scores are equal (a tie group cut by the selection)."""
    n = 0
    for r in scores.reshape(-1, scores.shape[-1]):
        if topk < len(r):
            s = np.sort(r)[::-1]
            n += int(s[topk - 1] == s[topk])
    return n


@pytest.mark.parametrize("sides,b,ns,S,B,H", [(INF_SIDES, 8, 4, 10, 2, 3), ([1, 2, 4, 8], 4, 2, 3, 1, 2),
                                            (INF_SIDES + [80, 96, 128], 8, 4, 13, 1, 2)])
def test_select_from_given_scores_with_forced_ties(sides, b, ns, S, B, H):
    og = oracle_geometry(sides, sides, b, ns)
    g = sv.Geometry(sides, sides, b, ns)
    G_S, NB = og.tiles(S), og.nb_le(S)
    rng = np.random.default_rng(NB)
    for topk in sorted({1, 3, 8, 16, NB - 1, NB, NB + 5}):
        if topk < 1:
            continue
        note(f"[select ties] NB={NB} G_S={G_S} topk={topk}")
        # small integers: heavy ties; a few constant rows; one row of zeros
        sc = rng.integers(0, 4, size=(B, H, G_S, NB)).astype(np.float32)
        sc[0, 0, 0] = 2.0
        sc[-1, -1, -1] = 0.0
        scores = torch.from_numpy(sc).cuda()
        idx = torch.full((B, H, G_S, topk), 9, dtype=torch.int32, device="cuda")
        sv.sparvar_select_blocks(g, S, None, None, None, topk, idx, scores_in=scores)
        torch.cuda.synchronize()
        got = idx.cpu().numpy().reshape(-1, topk)
        for row, want in zip(sc.reshape(-1, NB), got):
            assert want.tolist() == O.topk_blocks(row, topk)
        if topk < NB:
            assert tie_crossing_rows(sc, topk) > 0  # the cut went through a tie group somewhere
        else:
            assert (got[:, NB:] == -1).all() and (got[:, :NB] == np.arange(NB)).all()


def test_fused_decision_tie_rule_on_equal_block_masses():
    # Q = 0 at the 32x32 decision scale of the Infinity schedule: every score is 0,
    # every probability 1/2521, and the 64-token blocks (most of the 47) tie
    h, b, ns, S, B, H, d = INF_SIDES, 8, 4, 10, 1, 2, 128
    note("[decision ties] Q = 0 at 32x32")
    og = oracle_geometry(h, h, b, ns)
    g = sv.Geometry(h, h, b, ns)
    q, k, v = make_case(h, h, B, H, d, 32, ns, 81, "bf16")
    q[:] = 0.0
    Q, K, V = to_dev(q, "bf16"), to_dev(k, "bf16"), to_dev(v, "bf16")
    for topk in (8, 30):
        path = SparsePath(g, S, [13], B, H, d, topk, 1)
        path.decision(Q, K, V)
        torch.cuda.synchronize()
        scores = path.scores.cpu().numpy().reshape(B * H, og.tiles(S), og.nb_le(S))
        tk = path.topk_idx.cpu().numpy().reshape(B * H, og.tiles(S), topk)
        assert tie_crossing_rows(scores, topk) == B * H * og.tiles(S)  # every row cuts a tie group
        sizes = np.array([len(og.block_tokens(v_)) for v_ in range(og.nb_le(S))])
        for bh in range(B * H):
            # equal-size blocks have bit-identical scores on the GPU
            for t in range(og.tiles(S)):
                for sz in np.unique(sizes):
                    assert len(np.unique(scores[bh, t][sizes == sz])) == 1
                assert tk[bh, t].tolist() == O.topk_blocks(scores[bh, t], topk)
            # and the oracle's exact scores select the same blocks
            qS, kS = q.reshape(B * H, -1, d)[bh, og.C(S - 1):og.C(S)], k.reshape(B * H, -1, d)[bh, :og.C(S)]
            s_ref = O.pooled_scores(qS, kS, scale_of(d), og, S)
            for t in range(og.tiles(S)):
                assert tk[bh, t].tolist() == O.topk_blocks(s_ref[t], topk)


def test_map_status_word_reports_cut_local_rows():
    # local rows built with radius 2 handed to a mapping call told radius 1: they are
    # longer than the call's bound, so it cuts them and sets the status word
    h, b, ns, S, k, B, H, topk = INF_SIDES, 8, 4, 10, 13, 1, 2, 8
    og = oracle_geometry(h, h, b, ns)
    g = sv.Geometry(h, h, b, ns)
    note("[map status] radius-2 local rows against a radius-1 bound")
    G_S, G_k = og.tiles(S), og.tiles(k)
    rng = np.random.default_rng(5)
    sel = np.sort(np.stack([rng.choice(og.nb_le(S), topk, replace=False) for _ in range(B * H * G_S)]), axis=1)
    topk_idx = torch.from_numpy(sel.astype(np.int32)).cuda()
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    for radius_rows, radius_call, want in ((1, 1, sv.OK), (2, 1, sv.ERR_CAPACITY)):
        n_loc = sv.sparvar_local_blocks_capacity(g, k, radius_rows)
        lrp = torch.empty(G_k + 1, dtype=torch.int32, device="cuda")
        lci = torch.empty(n_loc, dtype=torch.int32, device="cuda")
        sv.sparvar_local_blocks(g, k, radius_rows, lrp, lci)
        cap = sv.sparvar_map_index_capacity(g, S, k, B, H, topk, radius_call)
        rp = torch.empty(B * H * G_k + 1, dtype=torch.int32, device="cuda")
        ci = torch.empty(cap, dtype=torch.int32, device="cuda")
        status.zero_()
        sv.sparvar_map_index(g, S, k, B, H, topk, topk_idx, lrp, lci, radius_call, rp, ci, status=status)
        torch.cuda.synchronize()
        assert status.item() == want, (radius_rows, radius_call, status.item())
        if want == sv.OK:
            loc = O.local_blocks(og, k, radius_rows)
            rows = O.build_rows(og, S, k, sel.reshape(B * H, G_S, topk), loc)
            assert csr_rows(rp, ci, padded=True) == [r for per in rows for r in per]

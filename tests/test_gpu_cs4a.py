"""GPU parity of the token-granular CS^4A path (called through the C ABI)
against the fp64 oracle on the same seeded inputs.

Column sums within 1e-4 after dividing by the query-block size; top-K tokens
bit-exact given the GPU's own column sums; token rows bit-exact given the GPU's
top-K; O_cache at S and the outputs of the later steps within the bf16
attention tolerance (max-abs 2e-2, mean-abs 2e-3), the steps checked against
the oracle fed with the GPU's own O_cache so that each stage is judged alone.
"""
import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import INF_SIDES, assert_close, make_case, note, oracle_geometry, scale_of, to_dev
from paper_2602_04361_amd import sparvar as sv
from paper_2602_04361_amd.pipeline import Cs4aPath

pytestmark = pytest.mark.gpu


def strip(row):
    row = [int(x) for x in row]
    n = next((i for i, x in enumerate(row) if x < 0), len(row))
    assert all(x < 0 for x in row[n:])
    return row[:n]


def cs4a_case(h, b, ns, S, steps, B, H, d, F, C, K, seed, heads=None, with_cache=True):
    note(f"[cs4a] h={h} S={S} steps={steps} B={B} H={H} d={d} C={C} K={K} cache={with_cache} seed={seed}")
    q, k, v = make_case(h, h, B, H, d, F, ns, seed, "bf16")
    Qd, Kd, Vd = to_dev(q, "bf16"), to_dev(k, "bf16"), to_dev(v, "bf16")
    g = sv.Geometry(h, h, b, ns)
    og = oracle_geometry(h, h, b, ns)
    path = Cs4aPath(g, S, steps, B, H, d, C, K, with_cache=with_cache)
    path.run(Qd, Kd, Vd)
    torch.cuda.synchronize()
    sc = scale_of(d)
    BH = B * H
    heads = list(range(BH)) if heads is None else heads
    qf, kf, vf = q.reshape(BH, -1, d), k.reshape(BH, -1, d), v.reshape(BH, -1, d)
    G_S = -(-og.N(S) // C)
    colsum = path.colsum.cpu().numpy().reshape(BH, G_S, og.C(S))
    inds = path.inds.cpu().numpy().reshape(BH, G_S, K)
    o_cache = path.o_cache.float().cpu().numpy().reshape(BH, og.N(S), d)
    sizes = np.array([len(r) for r in O.query_blocks(og.N(S), C)])
    for bh in heads:
        qS, kS, vS = qf[bh, og.C(S - 1):og.C(S)], kf[bh, :og.C(S)], vf[bh, :og.C(S)]
        D = O.column_sums(qS, kS, sc, C)
        err = np.abs(colsum[bh] - D) / sizes[:, None]
        assert err.max() <= 1e-4, f"column sums head {bh}: {err.max():.3e}"
        if with_cache:
            ref = O.o_cache(qS, kS, vS, [r.tolist() for r in inds[bh]], C, sc)
            assert_close(o_cache[bh], ref, "bf16", f"O_cache head {bh}")
    for bh in range(BH):
        for i in range(G_S):
            assert inds[bh, i].tolist() == O.topk_tokens(colsum[bh, i], K), (bh, i)
    for kk in steps:
        rows = O.cs4a_rows(og, S, kk, [r.tolist() for r in inds[0]], C)
        got_rows = path.tokens[kk].cpu().numpy().reshape(BH, -1, path.M)
        for bh in range(BH):
            rows_bh = rows if bh == 0 else O.cs4a_rows(og, S, kk, [r.tolist() for r in inds[bh]], C)
            assert [strip(r) for r in got_rows[bh]] == rows_bh, f"token rows step {kk} head {bh}"
        out = path.out[kk].float().cpu().numpy().reshape(BH, og.N(kk), d)
        for bh in heads:
            rows_bh = O.cs4a_rows(og, S, kk, [r.tolist() for r in inds[bh]], C)
            ref = O.cs4a_output(qf[bh, og.C(kk - 1):og.C(kk)], kf[bh, :og.C(kk)], vf[bh, :og.C(kk)], rows_bh, C, sc,
                                o_cache[bh] if with_cache else None, og, S, kk)
            mx, mean = assert_close(out[bh], ref, "bf16", f"step {kk} head {bh}")
        note(f"  step {kk}: ok (last head max {mx:.2e} mean {mean:.2e})")
    return path


def test_infinity_schedule_blocks_of_128():
    # decision 32x32 (8 blocks of 128 queries), top-256 tokens, steps 40/48/64
    cs4a_case(INF_SIDES, 8, 4, 10, [11, 12, 13], 1, 2, 128, 32, 128, 256, 41)


def test_infinity_layer_full_size_sampled_heads():
    # the swept token-path workload: B = 2, H = 16, d = 128, query blocks of 128,
    # top-1024 tokens, steps 40/48/64 (automatic chunk shapes); every index list
    # and top-K bit-exact, attention checked on two heads
    cs4a_case(INF_SIDES, 8, 4, 10, [11, 12, 13], 2, 16, 128, 32, 128, 1024, 49, heads=[0, 31])


@pytest.mark.parametrize("chunk", ["32", "64"])
@pytest.mark.parametrize("C", [64, 128])
def test_gather_chunks_of_32_and_64_keys(launch_option, chunk, C):
    # both chunk shapes of the gather attention at d = 128 (two and four waves),
    # for the O_cache pass at S and the later steps
    launch_option("CS4A_CHUNK", chunk)
    cs4a_case(INF_SIDES, 8, 4, 10, [11, 13], 1, 2, 128, 32, C, 200, 46 + C, heads=[1])


def test_blocks_of_64_without_cache_and_d64():
    h = [1, 2, 3, 5, 7, 10, 13, 20]
    cs4a_case(h, 4, 2, 6, [7, 8], 2, 2, 64, 8, 64, 40, 42, with_cache=False)


def test_topk_above_candidates_and_blocks_of_32():
    # K larger than the 85 keys at S: every token kept, rows padded with -1;
    # with every token kept, O_cache is dense minus dense (close to zero)
    h = [1, 2, 4, 8, 16]
    path = cs4a_case(h, 4, 2, 4, [5], 1, 2, 64, 8, 32, 100, 43)
    assert (path.inds[..., 85:] == -1).all()
    assert path.o_cache.float().abs().max().item() <= 2e-2


def test_blocks_of_256_ragged_last_block():
    # 40x40 = 1600 queries: six full blocks of 256 and one of 64
    cs4a_case(INF_SIDES[:11], 8, 4, 10, [11], 1, 1, 128, 32, 256, 128, 44)


def test_select_tokens_ties_and_rows():
    # integer-valued rows with many ties, several row lengths around the radix passes
    r = np.random.default_rng(45)
    # 9000 > 8192: the row is read from global memory on every pass instead of LDS
    for n, K in [(1, 1), (7, 3), (300, 257), (2521, 256), (4096, 1000), (9000, 700), (9000, 9000)]:
        vals = r.integers(0, 6, size=(5, n)).astype(np.float32)
        vals[0] = -vals[0]  # negative values order correctly too
        d_vals = torch.from_numpy(vals).cuda()
        inds = torch.empty(5, K, dtype=torch.int32, device="cuda")
        sv.sparvar_cs4a_select_tokens(d_vals, K, inds)
        torch.cuda.synchronize()
        got = inds.cpu().numpy()
        for i in range(5):
            assert got[i].tolist() == O.topk_tokens(vals[i], K), (n, K, i)

"""GPU parity of the CSLA block path (called through the C ABI) against the fp64
oracle on the same seeded inputs: block rows bit-exact; attention outputs within
the bf16 tolerance (max-abs 2e-2, mean-abs 2e-3) and LSE within 2e-4, the bar of
the same attention core on the 2-D block path."""
import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import INF_SIDES, assert_close, make_case, note, scale_of, to_dev
from paper_2602_04361_amd import sparvar as sv

pytestmark = pytest.mark.gpu


def gpu_rows(g, k, windows, block):
    M = sv.sparvar_csla_row_stride(g, k, block)
    n_rows = -(-g.scale_info(k)["n_tokens"] // block)
    rows = torch.full((n_rows, M), 7, dtype=torch.int32, device="cuda")  # padding must be overwritten
    sv.sparvar_csla_block_rows(g, k, windows, block, rows)
    torch.cuda.synchronize()
    got = rows.cpu().numpy()
    out = []
    for r in got:
        n = int(np.argmax(r < 0)) if (r < 0).any() else len(r)
        assert (r[n:] == -1).all()
        out.append(r[:n].tolist())
    return rows, out


def check_rows(h, w, ns, k, windows, block):
    note(f"[csla rows] sides={h}x{w} sinks={ns} k={k} windows={windows} block={block}")
    g = sv.Geometry(h, w, 8, ns)
    og = O.Geometry(h, w, 8, ns)
    rows, got = gpu_rows(g, k, windows, block)
    want = O.csla_block_rows(O.csla_token_mask(og, k, ns, windows), block)
    assert got == want
    return rows, want


@pytest.mark.parametrize("block", [32, 64, 128, 256])
def test_rows_infinity_last_scales(block):
    for k in (11, 12, 13):
        check_rows(INF_SIDES, INF_SIDES, 5, k, O.default_windows(k), block)


def test_rows_ablation_windows_and_sinks():
    # the sink and window settings of the paper's CSLA ablation, at the last scale
    for ns, sizes in [(5, (1, 3, 5)), (5, (3, 3, 3)), (5, (7, 9, 11)), (8, (3, 5, 7)), (0, (3, 5, 7))]:
        check_rows(INF_SIDES, INF_SIDES, ns, 13, O.default_windows(13, sizes), 128)


def test_rows_odd_shapes_wide_history_and_no_keys():
    h, w = [1, 2, 3, 5, 7], [1, 6, 2, 4, 9]  # scale 2 is wider than scales 3 and 4
    r = np.random.default_rng(50)
    for trial in range(4):
        k = int(r.integers(2, 6))
        windows = [int(x) for x in r.integers(0, 6, size=k)]
        for block in (32, 64):
            check_rows(h, w, int(r.integers(0, 3)), k, windows, block)
    check_rows(h, w, 0, 4, [0, 0, 0, 0], 32)           # nothing kept: every row empty
    check_rows(h, w, 1, 5, [99, 99, 99, 99, 99], 32)   # windows covering every grid: every block


def attn_case(h, ns, k, windows, block, B, H, d, seed, heads=None):
    note(f"[csla attn] k={k} block={block} B={B} H={H} d={d} windows={windows} sinks={ns} seed={seed}")
    g = sv.Geometry(h, h, 8, ns)
    og = O.Geometry(h, h, 8, ns)
    q, kk, v = make_case(h, h, B, H, d, 16, ns, seed, "bf16")
    n_kv, n0, n1 = og.C(k), og.C(k - 1), og.C(k)
    Q = to_dev(q[:, :, n0:n1], "bf16")
    Kd, Vd = to_dev(kk[:, :, :n_kv], "bf16"), to_dev(v[:, :, :n_kv], "bf16")
    rows, want_rows = gpu_rows(g, k, windows, block)
    o = torch.empty_like(Q)
    lse = torch.empty(B, H, n1 - n0, dtype=torch.float32, device="cuda")
    sv.sparvar_csla_attn_fwd(g, k, block, Q, Kd, Vd, o, rows, lse=lse)
    torch.cuda.synchronize()
    o = o.float().cpu().numpy().reshape(B * H, n1 - n0, d)
    lse = lse.cpu().numpy().reshape(B * H, n1 - n0)
    qf, kf, vf = (x.reshape(B * H, -1, d) for x in (q, kk, v))
    sc = scale_of(d)
    heads = range(B * H) if heads is None else heads
    for bh in heads:
        ref, ref_lse = O.csla_attention(qf[bh, n0:n1], kf[bh, :n_kv], vf[bh, :n_kv], want_rows, block, sc)
        mx, mean = assert_close(o[bh], ref, "bf16", f"head {bh}")
        fin = np.isfinite(ref_lse)
        assert (np.isneginf(lse[bh]) == ~fin).all()
        assert np.abs(lse[bh][fin] - ref_lse[fin]).max(initial=0) <= 2e-4
    note(f"  ok (last head max {mx:.2e} mean {mean:.2e})")
    return rows


def test_attention_scale_24x24_blocks_of_64_and_128():
    for block in (64, 128):
        attn_case(INF_SIDES[:9], 5, 9, O.default_windows(9), block, 2, 2, 128, 51)


def test_attention_d64_blocks_of_32_and_256():
    attn_case(INF_SIDES[:10], 4, 10, O.default_windows(10), 32, 1, 2, 64, 52)
    attn_case(INF_SIDES[:10], 4, 10, O.default_windows(10), 256, 1, 2, 64, 53)


def test_attention_table1_shape_sampled_heads():
    # 24 heads, 4096 queries against 10521 keys, d = 128, sinks = scales 1-5,
    # windows 3, 5, 7 on scales 11-13, blocks of 128
    attn_case(INF_SIDES, 5, 13, O.default_windows(13), 128, 1, 24, 128, 54, heads=[0, 23])


def test_attention_empty_rows_give_zero_and_stop_at_first_invalid_id():
    h = INF_SIDES[:8]
    g = sv.Geometry(h, h, 8, 0)
    og = O.Geometry(h, h, 8, 0)
    k, block, d = 8, 64, 128
    q, kk, v = make_case(h, h, 1, 1, d, 16, 0, 55, "bf16")
    Q = to_dev(q[:, :, og.C(7):og.C(8)], "bf16")
    Kd, Vd = to_dev(kk, "bf16"), to_dev(v, "bf16")
    rows, _ = gpu_rows(g, k, [0] * k, block)  # no sink, no window: every row empty
    o = torch.full_like(Q, 3.0)
    lse = torch.zeros(1, 1, og.N(8), dtype=torch.float32, device="cuda")
    sv.sparvar_csla_attn_fwd(g, k, block, Q, Kd, Vd, o, rows, lse=lse)
    torch.cuda.synchronize()
    assert (o == 0).all() and torch.isneginf(lse).all()
    # a row ending with ids after an invalid entry: only the ids before it count
    M = rows.shape[1]
    n_rows = rows.shape[0]
    hand = np.full((n_rows, M), -1, dtype=np.int32)
    hand[:, 0], hand[:, 1], hand[:, 2], hand[:, 3] = 0, 3, -5, 4
    sv.sparvar_csla_attn_fwd(g, k, block, Q, Kd, Vd, o, torch.from_numpy(hand).cuda(), lse=lse)
    torch.cuda.synchronize()
    got = o.float().cpu().numpy()[0, 0]
    ref, _ = O.csla_attention(q[0, 0, og.C(7):og.C(8)], kk[0, 0], v[0, 0], [[0, 3]] * n_rows, block, scale_of(d))
    assert_close(got, ref, "bf16", "rows cut at the first invalid id")


@pytest.mark.parametrize("stages", [2, 3, 4])
def test_attention_chunks_of_32(launch_option, stages):
    # the 32-key chunk shapes (d = 128, two to eight waves)
    launch_option("CSLA_CHUNK", "32")
    launch_option("CSLA_STAGES", str(stages))
    for block in (64, 128, 256):
        attn_case(INF_SIDES[:10], 5, 10, O.default_windows(10), block, 1, 2, 128, 56 + block)


def test_rows_longer_than_the_lds_table():
    # every scale a sink: each of the 200 query blocks of the 80x80 scale lists all
    # 529 key blocks of 32, past the ids staged in LDS
    h = INF_SIDES + [80]
    k = 14
    rows, want = check_rows(h, h, k, k, [0] * k, 32)
    assert all(len(r) == 529 for r in want)
    g = sv.Geometry(h, h, 8, k)
    og = O.Geometry(h, h, 8, k)
    q, kk, v = make_case(h, h, 1, 1, 128, 16, 4, 57, "bf16")
    n0, n1 = og.C(k - 1), og.C(k)
    Q, Kd, Vd = to_dev(q[:, :, n0:n1], "bf16"), to_dev(kk, "bf16"), to_dev(v, "bf16")
    o = torch.empty_like(Q)
    sv.sparvar_csla_attn_fwd(g, k, 32, Q, Kd, Vd, o, rows)
    torch.cuda.synchronize()
    ref, _ = O.dense_attention(q[0, 0, n0:n1], kk[0, 0], v[0, 0], scale_of(128))
    assert_close(o.float().cpu().numpy()[0, 0], ref, "bf16", "every block kept")


def test_pipeline_last_three_scales():
    from paper_2602_04361_amd.pipeline import CslaPath

    h, ns, block, d = INF_SIDES, 5, 128, 128
    steps = [11, 12, 13]
    note(f"[csla pipeline] steps={steps} block={block}")
    g = sv.Geometry(h, h, 8, ns)
    og = O.Geometry(h, h, 8, ns)
    q, kk, v = make_case(h, h, 1, 2, d, 16, ns, 58, "bf16")
    Qd, Kd, Vd = to_dev(q, "bf16"), to_dev(kk, "bf16"), to_dev(v, "bf16")
    path = CslaPath(g, steps, {k: O.default_windows(k) for k in steps}, block, 1, 2, d)
    path.rows()
    outs = {k: path.step(k, Qd, Kd, Vd) for k in steps}
    torch.cuda.synchronize()
    for k in steps:
        rows = O.csla_block_rows(O.csla_token_mask(og, k, ns, O.default_windows(k)), block)
        ref, _ = O.csla_attention(q[0, 1, og.C(k - 1):og.C(k)], kk[0, 1, :og.C(k)], v[0, 1, :og.C(k)], rows, block,
                                  scale_of(d))
        assert_close(outs[k].float().cpu().numpy()[0, 1], ref, "bf16", f"step {k}")

"""GPU parity of KV compression (called through the C ABI): the compact cache is
bit-exact against the oracle's copy of the kept scales, and the CSLA block path
on the compact schedule matches the oracle on that schedule (rows bit-exact,
outputs within the bf16 tolerance)."""
import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import INF_SIDES, assert_close, make_case, note, scale_of, to_dev
from paper_2602_04361_amd import sparvar as sv

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_compact_copy_is_exact_with_strided_planes(dtype):
    h = INF_SIDES[:10]
    og = O.Geometry(h, h, 8, 4)
    g = sv.Geometry(h, h, 8, 4)
    keep = [1, 2, 3, 4, 8, 9, 10]
    B, H, d = 2, 3, 64 if dtype == "f32" else 128
    note(f"[kv] compact {dtype} keep={keep} B={B} H={H} d={d}")
    r = np.random.default_rng(60)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    n = og.C(10)
    # source planes padded to n + 24 rows (plane stride larger than the plane)
    Ksrc = torch.from_numpy(r.standard_normal((B, H, n + 24, d)).astype(np.float32)).to(tdt).cuda()[:, :, :n]
    Vsrc = torch.from_numpy(r.standard_normal((B, H, n + 24, d)).astype(np.float32)).to(tdt).cuda()[:, :, :n]
    m = sum(og.N(l) for l in keep)
    Kd = torch.full((B, H, m, d), 7.0, dtype=tdt, device="cuda")
    Vd = torch.full((B, H, m, d), 7.0, dtype=tdt, device="cuda")
    sv.sparvar_kv_compact(g, keep, Ksrc, Vsrc, Kd, Vd)
    torch.cuda.synchronize()
    ks, vs = Ksrc.cpu().float().numpy(), Vsrc.cpu().float().numpy()
    for b in range(B):
        for hh in range(H):
            assert np.array_equal(Kd[b, hh].cpu().float().numpy(), O.kv_compact(ks[b, hh], og, keep))
            assert np.array_equal(Vd[b, hh].cpu().float().numpy(), O.kv_compact(vs[b, hh], og, keep))


def test_csla_on_the_compressed_cache():
    # the paper's setting: sinks = scales 1-5, windows 3/5/7 on the last three
    # scales; the compressed cache keeps exactly those scales
    h, ns, k, block, d = INF_SIDES, 5, 13, 128, 128
    keep = [1, 2, 3, 4, 5, 11, 12, 13]
    note(f"[kv] csla on the compressed cache keep={keep} block={block}")
    g = sv.Geometry(h, h, 8, ns)
    og = O.Geometry(h, h, 8, ns)
    q, kk, v = make_case(h, h, 1, 2, d, 16, ns, 61, "bf16")
    Kf, Vf = to_dev(kk, "bf16"), to_dev(v, "bf16")
    m = sum(og.N(l) for l in keep)
    Kc = torch.empty(1, 2, m, d, dtype=torch.bfloat16, device="cuda")
    Vc = torch.empty_like(Kc)
    sv.sparvar_kv_compact(g, keep, Kf, Vf, Kc, Vc)
    gc = sv.compact_geometry(g, keep)
    hc, wc = O.compact_schedule(og, keep)
    ogc = O.Geometry(hc, wc, 8, ns)
    kc = len(keep)
    M = sv.sparvar_csla_row_stride(gc, kc, block)
    rows = torch.empty(-(-og.N(k) // block), M, dtype=torch.int32, device="cuda")
    sv.sparvar_csla_block_rows(gc, kc, O.default_windows(kc), block, rows)
    Q = to_dev(q[:, :, og.C(k - 1):og.C(k)], "bf16")
    o = torch.empty_like(Q)
    sv.sparvar_csla_attn_fwd(gc, kc, block, Q, Kc, Vc, o, rows)
    torch.cuda.synchronize()
    want_rows = O.csla_block_rows(O.csla_token_mask(ogc, kc, ns, O.default_windows(kc)), block)
    got = rows.cpu().numpy()
    assert [r_[r_ >= 0].tolist() for r_ in got] == want_rows
    for bh in range(2):
        kcmp = O.kv_compact(kk[0, bh], og, keep)
        vcmp = O.kv_compact(v[0, bh], og, keep)
        ref, _ = O.csla_attention(q[0, bh, og.C(k - 1):og.C(k)], kcmp, vcmp, want_rows, block, scale_of(d))
        assert_close(o.float().cpu().numpy()[0, bh], ref, "bf16", f"compressed cache head {bh}")


def test_compact_full_size_24_heads():
    # the measured workload: batch 1, 24 heads, d = 128, the 10521-token cache of
    # the Infinity schedule compressed to its sink and windowed scales (8121 tokens)
    h, d, H = INF_SIDES, 128, 24
    keep = [1, 2, 3, 4, 5, 11, 12, 13]
    og = O.Geometry(h, h, 8, 5)
    g = sv.Geometry(h, h, 8, 5)
    note(f"[kv] compact full size H={H} keep={keep}")
    r = np.random.default_rng(63)
    n = og.C(13)
    Ks = torch.from_numpy(r.standard_normal((1, H, n, d)).astype(np.float32)).to(torch.bfloat16).cuda()
    Vs = torch.from_numpy(r.standard_normal((1, H, n, d)).astype(np.float32)).to(torch.bfloat16).cuda()
    m = sum(og.N(l) for l in keep)
    assert m == 8121
    Kd = torch.empty(1, H, m, d, dtype=torch.bfloat16, device="cuda")
    Vd = torch.empty_like(Kd)
    sv.sparvar_kv_compact(g, keep, Ks, Vs, Kd, Vd)
    torch.cuda.synchronize()
    ks, vs = Ks.view(torch.int16).cpu().numpy(), Vs.view(torch.int16).cpu().numpy()
    kd, vd = Kd.view(torch.int16).cpu().numpy(), Vd.view(torch.int16).cpu().numpy()
    for hh in range(H):
        assert np.array_equal(kd[0, hh], O.kv_compact(ks[0, hh], og, keep))
        assert np.array_equal(vd[0, hh], O.kv_compact(vs[0, hh], og, keep))

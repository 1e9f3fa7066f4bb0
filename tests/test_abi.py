"""Host-only checks of the C ABI: the library loads, exports every declared
symbol, and validates arguments before touching the GPU."""
import ctypes
import os
import re

import pytest

from oracle import Geometry as OGeom
from oracle import local_blocks as o_local_blocks
from paper_2602_04361_amd import sparvar as sv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INF = [1, 2, 4, 6, 8, 12, 16, 20, 24, 32, 40, 48, 64]


def declared_symbols():
    with open(os.path.join(ROOT, "include", "sparvar.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+char\s*\*|int64_t|int32_t|int)\s+(sparvar_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    lib = sv.load_library()
    names = declared_symbols()
    assert set(names) == set(sv.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    lib = sv.load_library()
    for st in (0, -1, -2, -3, -4):
        assert lib.sparvar_status_string(st)
    assert lib.sparvar_status_string(7) == b"unknown status"


def test_scale_info_matches_oracle_geometry():
    for sides, b, ns in [(INF, 8, 4), (INF, 16, 4), ([1, 2, 3, 5, 7, 10, 13], 4, 2)]:
        g = sv.Geometry(sides, sides, b, ns)
        o = OGeom(sides, sides, b, ns)
        for l in range(1, len(sides) + 1):
            info = g.scale_info(l)
            assert info["n_tokens"] == o.N(l)
            assert info["token_offset"] == o.C(l - 1) and info["n_tokens_le"] == o.C(l)
            assert (info["tile_h"], info["tile_w"]) == (o.eh(l), o.ew(l))
            assert (info["tiles_h"], info["tiles_w"]) == (o.Th(l), o.Tw(l))
            assert info["block_offset"] == o.base(l) and info["n_blocks_le"] == o.nb_le(l)


def test_local_capacity_matches_oracle():
    for sides, b, ns, k, r, dil in [(INF, 8, 4, 13, 1, 0), (INF, 8, 4, 11, 2, 1), (INF, 16, 4, 13, 1, 0),
                                    ([1, 2, 3, 5, 7, 10, 13], 4, 2, 7, 1, 0), ([1, 2, 4, 8], 4, 2, 4, 1, 0),
                                    ([1, 2, 4, 8], 4, 4, 4, 0, 0), ([1, 5, 7], 2, 0, 3, 0, 2)]:
        g = sv.Geometry(sides, sides, b, ns)
        rows = o_local_blocks(OGeom(sides, sides, b, ns), k, r, dil)
        assert sv.sparvar_local_blocks_capacity(g, k, r, dil) == sum(map(len, rows))


def test_map_capacity_bound():
    g = sv.Geometry(INF, INF, 8, 4)
    rows = o_local_blocks(OGeom(INF, INF, 8, 4), 13, 1)
    # every row at its longest (local + top-k), plus one length slot per row
    rows_n = 2 * 16 * 64
    assert sv.sparvar_map_index_capacity(g, 10, 13, 2, 16, 8, 1) == rows_n * (max(map(len, rows)) + 8) + rows_n


def test_map_capacity_bound_cover():
    # covering projection: each selected block takes as many slots as the largest
    # cover box of a block of scales 1..S (from the oracle's cover map)
    from oracle import map_block_cover
    for sides, b, S, k, topk in [(INF, 8, 10, 13, 8), (INF, 8, 10, 11, 8), (INF, 16, 10, 12, 4),
                                 (INF + [80, 96, 128], 8, 13, 16, 16), ([1, 2, 3, 5, 7, 10, 13], 3, 4, 7, 3)]:
        og = OGeom(sides, sides, b, 4)
        g = sv.Geometry(sides, sides, b, 4)
        mx_cover = max(len(map_block_cover(og, v, S, k)) for v in range(og.nb_le(S)))
        mx_local = max(map(len, o_local_blocks(og, k, 1)))
        rows_n = 2 * 3 * og.tiles(k)
        want = rows_n * (mx_local + topk * mx_cover) + rows_n
        assert sv.sparvar_map_index_capacity(g, S, k, 2, 3, topk, 1, projection="cover") == want
    assert max(len(map_block_cover(OGeom(INF, INF, 8, 4), v, 10, 13)) for v in range(47)) == 9


@pytest.mark.parametrize("args,status", [
    (dict(S=13, k=13), sv.ERR_INVALID),
    (dict(S=0, k=13), sv.ERR_INVALID),
    (dict(topk=0), sv.ERR_INVALID),
    (dict(topk=2000), sv.ERR_INVALID),
    (dict(radius=-1), sv.ERR_INVALID),
    (dict(projection=2), sv.ERR_INVALID),
])
def test_map_capacity_rejects(args, status):
    g = sv.Geometry(INF, INF, 8, 4)
    a = dict(S=10, k=13, B=2, H=16, topk=8, radius=1)
    a.update(args)
    n = sv.load_library().sparvar_map_index_capacity(g.ref, a["S"], a["k"], a["B"], a["H"], a["topk"],
                                                     a["radius"], 0, a.get("projection", 0))
    assert n == status
    assert sv.load_library().sparvar_last_error()


def test_geometry_validation():
    lib = sv.load_library()
    info = sv._CScaleInfo()
    assert lib.sparvar_scale_info(None, 1, ctypes.byref(info)) == sv.ERR_INVALID
    for h, b in [([0, 2], 8), ([1, 2], 0), ([1, 2], 65), (list(range(1, 40)), 8)]:
        g = sv.Geometry(h, h, b, 1)
        assert lib.sparvar_scale_info(g.ref, 1, ctypes.byref(info)) == sv.ERR_INVALID
    # a side over 65535 (the chunk descriptors keep a row pitch in 16 bits)
    g = sv.Geometry([1, 1], [1, 65536], 8, 1)
    assert lib.sparvar_scale_info(g.ref, 1, ctypes.byref(info)) == sv.ERR_INVALID
    g = sv.Geometry([1, 1], [1, 65535], 8, 1)
    assert lib.sparvar_scale_info(g.ref, 2, ctypes.byref(info)) == sv.OK
    g = sv.Geometry([1, 2], [1, 2], 8, 1)
    assert lib.sparvar_scale_info(g.ref, 3, ctypes.byref(info)) == sv.ERR_INVALID


def test_attention_validation_before_launch():
    lib = sv.load_library()
    vp = ctypes.c_void_p
    fake = vp(1 << 20)  # never dereferenced: validation fails first
    # unsupported head dim
    assert lib.sparvar_dense_attn_fwd(1, 1, 4, 4, 96, sv.BF16, fake, 4 * 96, fake, fake, 4 * 96, fake, None,
                                      0.1, None) == sv.ERR_UNSUPPORTED
    # unsupported dtype
    assert lib.sparvar_dense_attn_fwd(1, 1, 4, 4, 64, 7, fake, 256, fake, fake, 256, fake, None, 0.1,
                                      None) == sv.ERR_UNSUPPORTED
    # null pointer, bad stride, misaligned pointer, non-finite scale
    assert lib.sparvar_dense_attn_fwd(1, 1, 4, 4, 64, sv.BF16, None, 256, fake, fake, 256, fake, None, 0.1,
                                      None) == sv.ERR_INVALID
    assert lib.sparvar_dense_attn_fwd(1, 1, 4, 4, 64, sv.BF16, fake, 100, fake, fake, 256, fake, None, 0.1,
                                      None) == sv.ERR_INVALID
    assert lib.sparvar_dense_attn_fwd(1, 1, 4, 4, 64, sv.BF16, vp((1 << 20) + 2), 256, fake, fake, 256, fake,
                                      None, 0.1, None) == sv.ERR_INVALID
    assert lib.sparvar_dense_attn_fwd(1, 1, 4, 4, 64, sv.BF16, fake, 256, fake, fake, 256, fake, None,
                                      float("nan"), None) == sv.ERR_INVALID
    g = sv.Geometry(INF, INF, 8, 4)
    # scale out of range, missing CSR
    assert lib.sparvar_block_sparse_attn_fwd(g.ref, 14, 1, 1, 128, sv.BF16, fake, 4096 * 128, fake, fake,
                                             10521 * 128, fake, None, 0.1, fake, fake, None, None) == sv.ERR_INVALID
    assert lib.sparvar_block_sparse_attn_fwd(g.ref, 13, 1, 1, 128, sv.BF16, fake, 4096 * 128, fake, fake,
                                             10521 * 128, fake, None, 0.1, None, fake, None, None) == sv.ERR_INVALID
    # select: scores_out required without scores_in; local: capacity too small
    assert lib.sparvar_select_blocks(g.ref, 10, 1, 1, 128, sv.BF16, fake, 1024 * 128, fake, 2521 * 128, fake, 0.1,
                                     None, None, 8, fake, None) == sv.ERR_INVALID
    assert lib.sparvar_local_blocks(g.ref, 13, 1, 0, fake, fake, 10, None) == sv.ERR_CAPACITY
    assert lib.sparvar_map_index(g.ref, 10, 13, 1, 1, 8, fake, fake, fake, 1, 0, 0, fake, fake, 10, None, None,
                                 None) == sv.ERR_CAPACITY
    assert b"capacity" in lib.sparvar_last_error()


def test_decision_step_validation_before_launch():
    lib = sv.load_library()
    vp = ctypes.c_void_p
    fake = vp(1 << 20)
    g = sv.Geometry(INF, INF, 8, 4)
    args = lambda **kw: dict(dict(S=10, B=1, H=1, d=128, dt=sv.BF16, q=fake, qs=1024 * 128, k=fake, v=fake,
                                  kvs=2521 * 128, o=fake, lse=fake, scale=0.1, scores=fake, topk=8, idx=fake), **kw)

    def call(a):
        return lib.sparvar_decision_step(g.ref, a["S"], a["B"], a["H"], a["d"], a["dt"], a["q"], a["qs"], a["k"],
                                         a["v"], a["kvs"], a["o"], a["lse"], a["scale"], a["scores"], a["topk"],
                                         a["idx"], None)
    assert call(args(S=14)) == sv.ERR_INVALID          # scale out of range
    assert call(args(d=96)) == sv.ERR_UNSUPPORTED      # head dim
    assert call(args(topk=0)) == sv.ERR_INVALID        # top-k range
    assert call(args(lse=None)) == sv.ERR_INVALID      # LSE, scores and ids are required
    assert call(args(scores=None)) == sv.ERR_INVALID
    assert call(args(v=None)) == sv.ERR_INVALID
    assert call(args(kvs=100)) == sv.ERR_INVALID       # plane stride shorter than the plane
    assert call(args(scale=float("inf"))) == sv.ERR_INVALID


def test_csla_validation_before_launch():
    lib = sv.load_library()
    vp = ctypes.c_void_p
    fake = vp(1 << 20)
    g = sv.Geometry(INF, INF, 8, 5)
    # row stride = key blocks of the cache at step k
    assert sv.sparvar_csla_row_stride(g, 13, 128) == 83 and sv.sparvar_csla_row_stride(g, 13, 64) == 165
    assert sv.sparvar_csla_row_stride(g, 11, 32) == -(-4121 // 32)
    assert lib.sparvar_csla_row_stride(g.ref, 13, 48) == sv.ERR_UNSUPPORTED   # block size
    assert lib.sparvar_csla_row_stride(g.ref, 14, 64) == sv.ERR_INVALID       # scale out of range
    big = sv.Geometry([256, 300], [256, 300], 8, 1)                            # more than 2048 key blocks of 32
    assert lib.sparvar_csla_row_stride(big.ref, 2, 32) == sv.ERR_UNSUPPORTED
    win = (ctypes.c_int32 * 13)(*([0] * 10 + [3, 5, 7]))
    neg = (ctypes.c_int32 * 13)(*([0] * 12 + [-1]))
    wp = ctypes.cast(win, vp)
    assert lib.sparvar_csla_block_rows(g.ref, 13, wp, 128, fake, 82, None) == sv.ERR_CAPACITY
    assert lib.sparvar_csla_block_rows(g.ref, 13, ctypes.cast(neg, vp), 128, fake, 83, None) == sv.ERR_INVALID
    assert lib.sparvar_csla_block_rows(g.ref, 13, None, 128, fake, 83, None) == sv.ERR_INVALID
    assert lib.sparvar_csla_block_rows(g.ref, 13, wp, 128, None, 83, None) == sv.ERR_INVALID

    def attn(**kw):
        a = dict(k=13, block=128, B=1, H=24, d=128, dt=sv.BF16, q=fake, qs=4096 * 128, kk=fake, v=fake,
                 kvs=10521 * 128, o=fake, scale=0.1, rows=fake, M=83)
        a.update(kw)
        return lib.sparvar_csla_attn_fwd(g.ref, a["k"], a["block"], a["B"], a["H"], a["d"], a["dt"], a["q"], a["qs"],
                                         a["kk"], a["v"], a["kvs"], a["o"], None, a["scale"], a["rows"], a["M"], None)
    assert attn(block=96) == sv.ERR_UNSUPPORTED
    assert attn(dt=sv.F32) == sv.ERR_UNSUPPORTED
    assert attn(d=96) == sv.ERR_UNSUPPORTED
    assert attn(rows=None) == sv.ERR_INVALID
    assert attn(M=0) == sv.ERR_INVALID
    assert attn(kvs=100) == sv.ERR_INVALID
    assert attn(scale=float("nan")) == sv.ERR_INVALID
    assert attn(k=0) == sv.ERR_INVALID


def test_map_steps_validation_before_launch():
    lib = sv.load_library()
    vp = ctypes.c_void_p
    fake = 1 << 20
    g = sv.Geometry(INF, INF, 8, 4)
    cap = [sv.sparvar_map_index_capacity(g, 10, k, 2, 16, 8, 1) for k in (11, 12, 13)]

    def call(n, ks, caps, S=10, topk=8, rp=fake):
        k_arr = (ctypes.c_int32 * 3)(*ks)
        p_arr = (ctypes.c_void_p * 3)(rp, fake, fake)
        c_arr = (ctypes.c_int64 * 3)(*caps)
        return lib.sparvar_map_index_steps(g.ref, S, n, ctypes.cast(k_arr, vp), 2, 16, topk, vp(fake), 1, 0, 0,
                                           ctypes.cast(p_arr, vp), ctypes.cast(p_arr, vp), ctypes.cast(c_arr, vp), None,
                                           None)
    assert call(0, (11, 12, 13), cap) == sv.ERR_INVALID            # no step
    assert call(9, (11, 12, 13), cap) == sv.ERR_INVALID            # more than eight
    assert call(3, (11, 12, 10), cap) == sv.ERR_INVALID            # k <= S
    assert call(3, (11, 12, 13), cap, topk=0) == sv.ERR_INVALID
    assert call(3, (11, 12, 13), cap, rp=0) == sv.ERR_INVALID      # NULL row_ptr of step 0
    assert call(3, (11, 12, 13), (cap[0], cap[1] - 1, cap[2])) == sv.ERR_CAPACITY
    assert b"step 1" in lib.sparvar_last_error()


def test_kv_compact_validation_before_launch():
    lib = sv.load_library()
    vp = ctypes.c_void_p
    fake = vp(1 << 20)
    g = sv.Geometry(INF, INF, 8, 5)

    def call(keep, d=128, dt=sv.BF16, src=10521 * 128, dst=8121 * 128):
        arr = (ctypes.c_int32 * max(len(keep), 1))(*keep)
        return lib.sparvar_kv_compact(g.ref, len(keep), ctypes.cast(arr, vp), 1, 24, d, dt, fake, fake, src, fake,
                                      fake, dst, None)
    keep = [1, 2, 3, 4, 5, 11, 12, 13]
    assert call([]) == sv.ERR_INVALID
    assert call([1, 3, 2]) == sv.ERR_INVALID               # not ascending
    assert call([0, 1]) == sv.ERR_INVALID                  # scale out of range
    assert call([1, 14]) == sv.ERR_INVALID
    assert call(keep, d=96) == sv.ERR_UNSUPPORTED
    assert call(keep, dst=8120 * 128) == sv.ERR_INVALID    # compact plane too short
    assert call(keep, src=10520 * 128) == sv.ERR_INVALID   # source plane too short for scale 13
    assert sv.compact_geometry(g, keep).h == [1, 2, 4, 6, 8, 40, 48, 64]


def test_softmax_scale_must_be_positive():
    # the bf16 kernels take the running max of the raw scores, so scale <= 0 is refused everywhere
    lib = sv.load_library()
    vp = ctypes.c_void_p
    fake = vp(1 << 20)
    g = sv.Geometry(INF, INF, 8, 4)
    for scale in (0.0, -0.1, float("-inf")):
        assert lib.sparvar_dense_attn_fwd(1, 1, 4, 4, 64, sv.BF16, fake, 256, fake, fake, 256, fake, None, scale,
                                          None) == sv.ERR_INVALID
        assert lib.sparvar_block_sparse_attn_fwd(g.ref, 13, 1, 1, 128, sv.BF16, fake, 4096 * 128, fake, fake,
                                                 10521 * 128, fake, None, scale, fake, fake, None,
                                                 None) == sv.ERR_INVALID
        assert lib.sparvar_decision_step(g.ref, 10, 1, 1, 128, sv.BF16, fake, 1024 * 128, fake, fake, 2521 * 128,
                                         fake, fake, scale, fake, 8, fake, None) == sv.ERR_INVALID
        assert lib.sparvar_csla_attn_fwd(g.ref, 13, 128, 1, 1, 128, sv.BF16, fake, 4096 * 128, fake, fake,
                                         10521 * 128, fake, None, scale, fake, 83, None) == sv.ERR_INVALID
        assert lib.sparvar_select_blocks(g.ref, 10, 1, 1, 128, sv.BF16, fake, 1024 * 128, fake, 2521 * 128, fake,
                                         scale, None, fake, 8, fake, None) == sv.ERR_INVALID
        assert b"softmax_scale" in lib.sparvar_last_error()


def test_bf16_plane_offsets_limited_to_32_bits():
    # the bf16 HBM -> LDS copies use 32-bit byte offsets inside a (b, h) plane
    lib = sv.load_library()
    vp = ctypes.c_void_p
    fake = vp(1 << 20)
    n_kv = 1 << 24  # x 128 x 2 bytes = 2^32
    assert lib.sparvar_dense_attn_fwd(1, 1, 4, n_kv, 128, sv.BF16, fake, 4 * 128, fake, fake, n_kv * 128, fake,
                                      None, 0.1, None) == sv.ERR_INVALID
    assert b"2^32" in lib.sparvar_last_error()
    side = [1, 4097]  # 16785410 cache tokens at step 2
    g = sv.Geometry(side, side, 8, 1)
    nq = 4097 * 4097
    assert lib.sparvar_block_sparse_attn_fwd(g.ref, 2, 1, 1, 128, sv.BF16, fake, nq * 128, fake, fake,
                                             (nq + 1) * 128, fake, None, 0.1, fake, fake, None,
                                             None) == sv.ERR_INVALID
    assert b"2^32" in lib.sparvar_last_error()


def test_decision_step_fallback_validates_before_any_launch():
    # 32x32-token tiles at the 32x32 decision scale: the fused kernel does not take
    # them and the scoring kernel of the two-call sequence serves at most 256-token
    # tiles, so the call must fail before it enqueues the dense attention (on this
    # GPU-less host an enqueued launch would report a HIP error instead)
    lib = sv.load_library()
    vp = ctypes.c_void_p
    fake = vp(1 << 20)
    g = sv.Geometry(INF, INF, 32, 4)
    st = lib.sparvar_decision_step(g.ref, 10, 1, 1, 128, sv.BF16, fake, 1024 * 128, fake, fake, 2521 * 128, fake,
                                   fake, 0.1, fake, 8, fake, None)
    assert st == sv.ERR_UNSUPPORTED, lib.sparvar_last_error()
    assert b"256 tokens" in lib.sparvar_last_error()


def test_launch_options_set_get_reset():
    lib = sv.load_library()
    defaults = {n: sv.sparvar_get_launch_option(n) for n in sv.LAUNCH_OPTIONS}
    assert defaults["SWIZZLE"] == 1 and defaults["SPARSE_CHUNK"] == 32 and defaults["SPARSE_GROUP_WAVES"] == -1
    with sv.launch_options(SPARSE_CHUNK=64, SWIZZLE=0):
        assert sv.sparvar_get_launch_option("SPARSE_CHUNK") == 64 and sv.sparvar_get_launch_option("SWIZZLE") == 0
    assert {n: sv.sparvar_get_launch_option(n) for n in sv.LAUNCH_OPTIONS} == defaults
    sv.sparvar_set_launch_option("DENSE_WAVES", 4)
    sv.sparvar_set_launch_option("DENSE_WAVES", None)  # back to the default
    assert sv.sparvar_get_launch_option("DENSE_WAVES") == defaults["DENSE_WAVES"]
    v = ctypes.c_int32()
    assert lib.sparvar_set_launch_option(len(sv.LAUNCH_OPTIONS), 1) == sv.ERR_INVALID
    assert lib.sparvar_get_launch_option(-1, ctypes.byref(v)) == sv.ERR_INVALID
    assert lib.sparvar_get_launch_option(0, None) == sv.ERR_INVALID


def test_launch_option_names_follow_the_header():
    with open(os.path.join(ROOT, "include", "sparvar.h")) as f:
        text = f.read()
    body = text[text.index("typedef enum sparvar_launch_option"):text.index("} sparvar_launch_option_t;")]
    names = re.findall(r"SPARVAR_OPT_(\w+)", body)
    assert names[-1] == "COUNT" and names[0] == "SWIZZLE"
    assert names[:-1] == sv.LAUNCH_OPTIONS


def test_noalloc_mapping_validation_before_launch():
    # the allocation-free mapping call: capacities need only the row slots, and the
    # steps' rows together must fit the fixed scratch of SPARVAR_NOALLOC_MAX_ROWS
    lib = sv.load_library()
    vp = ctypes.c_void_p
    fake = 1 << 20
    g = sv.Geometry(INF, INF, 8, 4)

    def call(B, H, cap):
        k_arr = (ctypes.c_int32 * 1)(13)
        p_arr = (ctypes.c_void_p * 1)(fake)
        c_arr = (ctypes.c_int64 * 1)(cap)
        return lib.sparvar_map_index_steps_noalloc(g.ref, 10, 1, ctypes.cast(k_arr, vp), B, H, 8, vp(fake), 1, 0, 0,
                                                   ctypes.cast(p_arr, vp), ctypes.cast(p_arr, vp),
                                                   ctypes.cast(c_arr, vp), None, None)
    H = sv.NOALLOC_MAX_ROWS // 64 + 1  # 64 tiles per plane at 64x64: one plane past the scratch
    rows = H * 64
    slots = sv.sparvar_map_index_capacity(g, 10, 13, 1, H, 8, 1) - rows
    assert call(1, H, slots) == sv.ERR_CAPACITY
    assert b"fixed scratch" in lib.sparvar_last_error()
    rows = 2 * 16 * 64
    slots = sv.sparvar_map_index_capacity(g, 10, 13, 2, 16, 8, 1) - rows
    assert call(2, 16, slots - 1) == sv.ERR_CAPACITY           # the row slots are still required
    assert b"capacity" in lib.sparvar_last_error()
    with open(os.path.join(ROOT, "include", "sparvar.h")) as f:
        assert f"#define SPARVAR_NOALLOC_MAX_ROWS (1 << {sv.NOALLOC_MAX_ROWS.bit_length() - 1})" in f.read()

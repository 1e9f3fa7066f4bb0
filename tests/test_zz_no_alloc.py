"""The allocation-free mapping entry point (sparvar_map_index_steps_noalloc)
against sparvar_map_index_steps, through the C ABI: same rows and launch
orders bit for bit, on two calls in a row, the second with a smaller input
(the fixed scratch keeps the first call's row lengths, which must not leak
into the second)."""
import numpy as np
import pytest
import torch

from gpu_helpers import INF_SIDES, make_case, note, to_dev
from paper_2602_04361_amd import sparvar as sv
from paper_2602_04361_amd.pipeline import SparsePath

pytestmark = pytest.mark.gpu


def map_both(g, S, steps, B, H, d, topk, radius, projection, seed):
    note(f"[noalloc] S={S} steps={steps} B={B} H={H} topk={topk} r={radius} projection={projection} seed={seed}")
    q, k, v = make_case(g.h, g.w, B, H, d, 32, g.num_sink_scales, seed, "bf16")
    Q, K, V = to_dev(q, "bf16"), to_dev(k, "bf16"), to_dev(v, "bf16")
    path = SparsePath(g, S, steps, B, H, d, topk, radius, projection=projection)
    path.decision(Q, K, V)
    path.map_all(orders=True)  # the existing entry point: row lengths after the row slots
    i32 = dict(dtype=torch.int32, device="cuda")
    rps, cis, ords = [], [], []
    for kk in steps:
        info = path.info[kk]
        rows = B * H * info["tiles_h"] * info["tiles_w"]
        cap = sv.sparvar_map_index_capacity(g, S, kk, B, H, topk, radius, 0, projection) - rows  # row slots only
        rps.append(torch.full((rows + 1,), -9, **i32))
        cis.append(torch.full((cap,), -9, **i32))
        ords.append(torch.full((rows,), -9, **i32))
    sv.sparvar_map_index_steps(g, S, steps, B, H, topk, path.topk_idx, radius, rps, cis, orders=ords,
                               projection=projection, noalloc=True)
    torch.cuda.synchronize()
    for i, kk in enumerate(steps):
        rp, ci, _ = path.csr[kk]
        n = cis[i].numel()
        assert torch.equal(rps[i], rp), f"row_ptr step {kk}"
        assert torch.equal(cis[i], ci[:n]), f"col_idx step {kk}"
        assert torch.equal(ords[i], path.orders[kk]), f"launch order step {kk}"
        assert (ci[:n] >= -1).all() and int((ci[:n] >= 0).sum()) > 0


def test_noalloc_mapping_matches_the_workspace_form_twice():
    g = sv.Geometry(INF_SIDES, INF_SIDES, 8, 4)
    # first call: the Infinity layer, three steps, 4000 rows
    map_both(g, 10, [11, 12, 13], 2, 16, 128, 8, 1, "point", seed=3)
    # second call, smaller: fewer heads and one step, with the covering projection
    map_both(g, 10, [12], 1, 3, 128, 4, 2, "cover", seed=4)

"""GPU check that a whole layer of the hot path (fused decision step, one mapping
launch with launch orders, three block-sparse steps), captured once per input
set into a HIP graph, replays bit-identically to eager launches: several replays
of each graph, with eager launches of the other input set and synchronisations
between them, each compared with the eager result of its own inputs."""
import pytest
import torch

from gpu_helpers import INF_SIDES, make_case, note, to_dev
from paper_2602_04361_amd import sparvar as sv
from paper_2602_04361_amd.pipeline import SparsePath

pytestmark = pytest.mark.gpu


def test_layer_graph_replays_match_eager():
    h, B, H, d = INF_SIDES, 1, 4, 128
    g = sv.Geometry(h, h, 8, 4)
    sets = []
    for seed in (71, 72):
        q, k, v = make_case(h, h, B, H, d, 32, 4, seed, "bf16")
        sets.append((to_dev(q, "bf16"), to_dev(k, "bf16"), to_dev(v, "bf16")))
    path = SparsePath(g, 10, [11, 12, 13], B, H, d, 8, 1)

    def layer(s):
        Q, K, V = sets[s]
        path.decision(Q, K, V)
        path.map_all(orders=True)
        for kk in (11, 12, 13):
            path.attn_step(kk, Q, K, V, use_order=True)

    def outputs():
        return [path.o_S, path.lse_S, path.topk_idx] + [path.out[kk] for kk in (11, 12, 13)]

    eager = []
    for s in range(2):
        layer(s)
        torch.cuda.synchronize()
        eager.append([t.clone() for t in outputs()])
    graphs = []
    for s in range(2):
        gph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gph):
            layer(s)
        graphs.append(gph)
    for rep in range(3):
        for s in range(2):
            note(f"[graph] replay {rep} of set {s}")
            layer(1 - s)  # eager work on the other inputs in between
            torch.cuda.synchronize()
            for t in outputs():
                t.zero_()
            graphs[s].replay()
            torch.cuda.synchronize()
            for a, b in zip(eager[s], outputs()):
                assert torch.equal(a, b)

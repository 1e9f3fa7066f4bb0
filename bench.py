"""Benchmark of the SparVAR sparse path on one MI355X.

One step = one layer of the whole hot path on the Infinity 1024x1024 schedule
(scales 1,2,4,6,8,12,16,20,24,32,40,48,64; B=2 CFG pair, H=16, d=128, bf16):
  decision scale 32x32: dense attention + LSE, pooled block scores and top-8
  (one fused call);
  index mapping into CSR for the three sparse steps in one call (their rows
  depend only on the selection at 32x32; the sink and local rows are generated
  inside the mapping call), which also writes each step's launch order;
  for each sparse step 40x40, 48x48, 64x64: block-sparse attention (8x8-token
  blocks, sinks = scales 1-4, 3x3 window).
Inputs are seeded synthetic tensors resident in HBM; four input sets rotate so
no step finds its K/V in cache from the previous one.

Prints one JSON line. `value` is the algorithmic TFLOP/s of the block-sparse
attention at the 64x64 step (4 d * kept query-key pairs over its measured
duration inside the step), the metric's subject; `ms_per_layer` is the whole
step and `layer_tflops` its algorithmic rate (the dense decision scale plus the
kept pairs of the three sparse steps).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

SIDES = [1, 2, 4, 6, 8, 12, 16, 20, 24, 32, 40, 48, 64]
CFG = dict(B=2, H=16, d=128, b=8, n_sink=4, S=10, steps=[11, 12, 13], topk=8, radius=1, n_freq=32)
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
N_SETS = 4


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=200,
                    help="untimed steps first; about 70 ms of work, which brings the clocks up to speed")
    ap.add_argument("--ramp-seconds", type=float, default=0.5,
                    help="untimed whole steps for this long before the warm-up steps: the GPU reaches its "
                         "steady clock after about 0.25 s of sustained work (0 = none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU time of the oracle sample")
    ap.add_argument("--sets", type=int, default=N_SETS)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="finish with three plain device copies of 256 MiB (reference for HBM byte counters)")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the step line: one JSON line per setting of the wider-head, 2048x2048 and "
                         "sparsity-sweep workloads (per-layer times, TFLOP/s, density, speedup)")
    ap.add_argument("--csla", action="store_true",
                    help="instead of the step line: the CSLA block-path settings only")
    ap.add_argument("--only", default=None,
                    help="with --sweep: only the block-path workloads whose name contains this string")
    return ap.parse_args()


# ---------------------------------------------------------------- accounting
def block_sizes(info):
    """Token count of every block id, from the library's per-scale geometry."""
    sizes = []
    for l in sorted(info):
        i = info[l]
        for tu in range(i["tiles_h"]):
            nr = min(i["tile_h"], i["h"] - tu * i["tile_h"])
            for tv in range(i["tiles_w"]):
                nc = min(i["tile_w"], i["w"] - tv * i["tile_w"])
                sizes.append(nr * nc)
    return np.array(sizes, dtype=np.int64)


def query_tile_sizes(i):
    out = []
    for tu in range(i["tiles_h"]):
        for tv in range(i["tiles_w"]):
            out.append(min(i["tile_h"], i["h"] - tu * i["tile_h"]) * min(i["tile_w"], i["w"] - tv * i["tile_w"]))
    return np.array(out, dtype=np.int64)


def sparse_accounting(row_ptr, col_idx, info, k, BH, d, elem=2):
    """Algorithmic FLOPs and bytes of one block-sparse attention launch."""
    bs = block_sizes(info)
    qsz = query_tile_sizes(info[k])
    G = len(qsz)
    rp = row_ptr.astype(np.int64)
    nk = info[k]["n_tokens"]
    nb_k = info[k]["n_blocks_le"]
    col_idx = col_idx[:rp[-1]]
    valid = (col_idx >= 0) & (col_idx < nb_k)
    tok = np.where(valid, bs[np.where(valid, col_idx, 0)], 0)  # -1 padding and skipped ids count 0
    keys = np.add.reduceat(tok, rp[:-1]) if len(tok) else np.zeros(len(rp) - 1)
    keys = np.where(np.diff(rp) > 0, keys, 0)
    pairs = (keys * np.tile(qsz, BH)).sum()
    flops = 4.0 * d * pairs
    uniq_tokens = 0
    for bh in range(BH):
        seg = col_idx[rp[bh * G]:rp[(bh + 1) * G]]
        uniq_tokens += bs[np.unique(seg[(seg >= 0) & (seg < nb_k)])].sum()
    bytes_ = BH * nk * d * elem * 2 + uniq_tokens * d * elem * 2  # Q + O + unique K and V
    density = pairs / (BH * nk * info[k]["n_tokens_le"])
    return flops, bytes_, density, keys


# ---------------------------------------------------------------- CPU baseline (oracle)
def cpu_baseline(q, k, v, target_s):
    """Time the fp64 oracle on a bounded sample of heads of the same step."""
    import oracle as O

    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    affinity = len(os.sched_getaffinity(0))
    B, H, d = CFG["B"], CFG["H"], CFG["d"]
    g = O.Geometry(SIDES, SIDES, CFG["b"], CFG["n_sink"])
    S = CFG["S"]
    sc = float(np.float32(1.0 / math.sqrt(d)))
    BH = B * H
    qf, kf, vf = (x.reshape(BH, -1, d) for x in (q, k, v))
    flops_done = 0.0
    heads = 0
    t0 = time.perf_counter()
    local = {kk: O.local_blocks(g, kk, CFG["radius"]) for kk in CFG["steps"]}
    for bh in range(BH):
        # decision scale: dense + pooled scores + top-k for one head
        qS, kS, vS = qf[bh, g.C(S - 1):g.C(S)], kf[bh, :g.C(S)], vf[bh, :g.C(S)]
        O.dense_attention(qS, kS, vS, sc)
        scores = O.pooled_scores(qS, kS, sc, g, S)
        tk = np.array([[O.topk_blocks(r, CFG["topk"]) for r in scores]])
        flops_done += 4.0 * d * g.N(S) * g.C(S)
        for kk in CFG["steps"]:
            rows = O.build_rows(g, S, kk, tk, local[kk])[0]
            O.block_sparse_attention_gather(qf[bh, g.C(kk - 1):g.C(kk)], kf[bh, :g.C(kk)], vf[bh, :g.C(kk)], g, kk,
                                            rows, sc)
            kept = sum(len(g.tile_local_tokens(kk, t // g.Tw(kk), t % g.Tw(kk))) *
                       sum(len(g.block_tokens(vb)) for vb in rows[t]) for t in range(len(rows)))
            flops_done += 4.0 * d * kept
        heads += 1
        if time.perf_counter() - t0 >= target_s:
            break
    dt = time.perf_counter() - t0
    return {"value": flops_done / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "blas_threads": int(threads), "affinity_cores": affinity,
            "sample": f"whole step (decision + 3 sparse steps) for {heads} of {BH} (batch, head) planes, "
                      f"fp64 NumPy, {dt:.1f} s; {threads} BLAS threads on {affinity} cores in the affinity mask"}


def profile_value(name, key, kernel_hash):
    """A per-launch figure of the 64x64 sparse kernel from a committed rocprofv3
    PMC summary under profiles/, if it was taken on the current kernel source;
    else None."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k_, val = line.split("=", 1)
                vals[k_.strip()] = val.strip()
    if vals.get("kernel_source_sha256") != kernel_hash:
        return None
    try:
        return float(vals[key])
    except (KeyError, ValueError):
        return None


def own_block_rows(info, k, BH):
    """CSR in which every query tile of scale k lists only its own block: each
    K/V token of scale k is read by exactly one workgroup (no re-reads), so the
    launch's compulsory HBM bytes are known exactly (Q + K/V of scale k + O)."""
    G = info[k]["tiles_h"] * info[k]["tiles_w"]
    base = info[k]["block_offset"]
    rows = BH * G
    row_ptr = np.arange(rows + 1, dtype=np.int32)
    col_idx = (base + np.tile(np.arange(G, dtype=np.int32), BH)).astype(np.int32)
    return row_ptr, col_idx


def kernel_source_hash():
    h = hashlib.sha256()
    for name in ("csrc/attention.hip", "csrc/device_common.h", "csrc/geometry.h", "build.py"):  # build.py: the flags
        with open(os.path.join(ROOT, "paper_2602_04361_amd", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


# ---------------------------------------------------------------- sweep of the other workloads
SWEEP = ([dict(name="heads32", sides=SIDES, B=2, H=32, b=8, S=10, steps=[11, 12, 13], topk=8, radius=1, sets=4),
          dict(name="cover_projection", sides=SIDES, B=2, H=16, b=8, S=10, steps=[11, 12, 13], topk=8, radius=1,
               sets=4, projection="cover"),
          dict(name="schedule2048", sides=SIDES + [80, 96, 128], B=1, H=16, b=8, S=13, steps=[14, 15, 16], topk=16,
               radius=1, sets=2)] +
         [dict(name=f"last_step_b{b}_r{r}_top{t}", sides=SIDES, B=2, H=16, b=b, S=10, steps=[13], topk=t, radius=r,
               sets=4) for b in (8, 16) for r in (1, 2) for t in (4, 8, 16, 32)])


def sweep(args, dev, only=None):
    import torch

    from paper_2602_04361_amd import sparvar as sv
    from paper_2602_04361_amd.pipeline import SparsePath
    from paper_2602_04361_amd.synth import make_qkv

    d, nf, ns = CFG["d"], CFG["n_freq"], CFG["n_sink"]
    cache = {}
    ramp_left = args.ramp_seconds  # the first workload also brings the clocks up
    for st in SWEEP:
        if only is not None and only not in st["name"]:
            continue
        key = (tuple(st["sides"]), st["B"], st["H"], st["sets"])
        if key not in cache:
            cache.clear()
            sets = []
            for s in range(st["sets"]):
                q, k, v = make_qkv(st["sides"], st["sides"], st["B"], st["H"], d, nf, ns, seed=s, bf16=True)
                sets.append(tuple(torch.from_numpy(x).to(dev).to(torch.bfloat16) for x in (q, k, v)))
                del q, k, v
            cache[key] = sets
        sets = cache[key]
        B, H = st["B"], st["H"]
        g = sv.Geometry(st["sides"], st["sides"], st["b"], ns)
        path = SparsePath(g, st["S"], st["steps"], B, H, d, st["topk"], st["radius"],
                          projection=st.get("projection", "point"))
        info = path.info
        stream = torch.cuda.current_stream()
        n_ev = 3 + len(st["steps"])

        def one(i, ev=None):
            Q, K, V = sets[i % len(sets)]
            if ev is not None:
                ev[0].record(stream)
            path.decision(Q, K, V)
            if ev is not None:
                ev[1].record(stream)
            path.map_all(orders=True)
            if ev is not None:
                ev[2].record(stream)
            for j, kk in enumerate(st["steps"]):
                path.attn_step(kk, Q, K, V, use_order=True)
                if ev is not None:
                    ev[3 + j].record(stream)

        for i in range(5):
            one(i)
        torch.cuda.synchronize()
        t_ramp, i = time.perf_counter(), 5
        while time.perf_counter() - t_ramp < ramp_left:
            one(i)
            i += 1
            if i % 10 == 0:
                torch.cuda.synchronize()
        torch.cuda.synchronize()
        ramp_left = 0.0
        n = 20
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(n_ev)] for _ in range(n)]
        for i in range(n):
            one(i, evs[i])
        torch.cuda.synchronize()
        med = lambda a, b: float(np.median([evs[i][a].elapsed_time(evs[i][b]) for i in range(n)]))
        out = {"sweep": st["name"], "B": B, "H": H, "block": st["b"], "topk": st["topk"], "radius": st["radius"],
               "projection": st.get("projection", "point"),
               "decision_scale": st["sides"][st["S"] - 1], "decision_ms": med(0, 1),
               "map_all_steps_ms": med(1, 2), "steps": {}}
        BH = B * H
        for j, kk in enumerate(st["steps"]):
            rp, ci, _ = path.csr[kk]
            f, b_, dens, _ = sparse_accounting(rp.cpu().numpy(), ci.cpu().numpy(), info, kk, BH, d)
            t_attn = med(2 + j, 3 + j)
            out["steps"][str(info[kk]["h"])] = {"attn_ms": t_attn, "gflop": f / 1e9,
                                                "tflops": f / t_attn / 1e9,
                                                "frac_bf16_peak": f / t_attn / 1e9 / PEAK_BF16_TFLOPS,
                                                "density": dens}
        # our dense kernel at the last step, same buffers
        kl = st["steps"][-1]
        il = info[kl]
        o = torch.empty(B, H, il["n_tokens"], d, dtype=torch.bfloat16, device=dev)

        def dense(i):
            Q, K, V = sets[i % len(sets)]
            sv.sparvar_dense_attn_fwd(path.q_slice(Q, kl), path.kv_prefix(K, kl), path.kv_prefix(V, kl), o, None,
                                      softmax_scale=path.scale)

        for i in range(2):
            dense(i)
        torch.cuda.synchronize()
        de = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(5)]
        for i, (a, b_) in enumerate(de):
            a.record(stream)
            dense(i)
            b_.record(stream)
        torch.cuda.synchronize()
        t_dense = float(np.median([a.elapsed_time(b_) for a, b_ in de]))
        last = out["steps"][str(il["h"])]
        out["dense_last_ms"] = t_dense
        out["dense_last_tflops"] = 4.0 * d * BH * il["n_tokens"] * il["n_tokens_le"] / t_dense / 1e9
        out["speedup_last_vs_own_dense"] = t_dense / last["attn_ms"]
        print(json.dumps(out), flush=True)
        del path


CS4A_SWEEP = [dict(C=128, K=1024), dict(C=128, K=512), dict(C=64, K=1024), dict(C=256, K=1024)]


def sweep_cs4a(dev):
    """Token-granular CS^4A path on the Infinity layer: per-stage times and the
    gather attention's algorithmic TFLOP/s (4 d * queries * kept tokens)."""
    import torch

    from paper_2602_04361_amd import sparvar as sv
    from paper_2602_04361_amd.pipeline import Cs4aPath
    from paper_2602_04361_amd.synth import make_qkv

    B, H, d = CFG["B"], CFG["H"], CFG["d"]
    sets = []
    for s in range(N_SETS):
        q, k, v = make_qkv(SIDES, SIDES, B, H, d, CFG["n_freq"], CFG["n_sink"], seed=s, bf16=True)
        sets.append(tuple(torch.from_numpy(x).to(dev).to(torch.bfloat16) for x in (q, k, v)))
    g = sv.Geometry(SIDES, SIDES, CFG["b"], CFG["n_sink"])
    stream = torch.cuda.current_stream()
    for st in CS4A_SWEEP:
        path = Cs4aPath(g, CFG["S"], CFG["steps"], B, H, d, st["C"], st["K"])
        names = ["dense_S", "colsum", "topk", "cache"] + [f"{n}_{k}" for k in CFG["steps"] for n in ("map", "attn")]

        def one(i, ev=None):
            Q, K, V = sets[i % len(sets)]
            S = CFG["S"]
            q, kk, vv = path.q_slice(Q, S), path.kv_prefix(K, S), path.kv_prefix(V, S)
            rec = (lambda j: ev[j].record(stream)) if ev is not None else (lambda j: None)
            rec(0)
            sv.sparvar_dense_attn_fwd(q, kk, vv, path.o_S, path.lse_S, softmax_scale=path.scale)
            rec(1)
            sv.sparvar_cs4a_column_sums(g, S, path.C, q, kk, path.lse_S, path.colsum, softmax_scale=path.scale)
            rec(2)
            sv.sparvar_cs4a_select_tokens(path.colsum, path.K, path.inds)
            rec(3)
            sv.sparvar_cs4a_attn_fwd(g, S, path.C, q, kk, vv, path.o_cache, path.inds, path.K, mode=1, base=path.o_S,
                                     softmax_scale=path.scale)
            rec(4)
            j = 5
            for kk_ in CFG["steps"]:
                sv.sparvar_cs4a_map_tokens(g, S, kk_, path.C, B, H, path.K, path.inds, path.tokens[kk_], path.M)
                rec(j)
                sv.sparvar_cs4a_attn_fwd(g, kk_, path.C, path.q_slice(Q, kk_), path.kv_prefix(K, kk_),
                                         path.kv_prefix(V, kk_), path.out[kk_], path.tokens[kk_], path.M, mode=2,
                                         base=path.o_cache, base_scale=S, softmax_scale=path.scale)
                rec(j + 1)
                j += 2

        for i in range(5):
            one(i)
        torch.cuda.synchronize()
        n = 20
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)] for _ in range(n)]
        for i in range(n):
            one(i, evs[i])
        torch.cuda.synchronize()
        med = {nm: float(np.median([evs[i][j].elapsed_time(evs[i][j + 1]) for i in range(n)]))
               for j, nm in enumerate(names)}
        out = {"sweep": f"cs4a_C{st['C']}_K{st['K']}", "B": B, "H": H, "C": st["C"], "K": st["K"],
               "stages_ms": {nm: med[nm] for nm in ("dense_S", "colsum", "topk", "cache")}, "steps": {}}
        for kk_ in CFG["steps"]:
            toks = path.tokens[kk_].cpu().numpy().reshape(B * H, -1, path.M)
            n_q = path.info[kk_]["n_tokens"]
            blocks = -(-n_q // st["C"])
            qsz = np.array([min(st["C"], n_q - i * st["C"]) for i in range(blocks)])
            kept = ((toks >= 0) & (toks < path.info[kk_]["n_tokens_le"])).sum(axis=2)
            flops = 4.0 * d * float((kept * qsz[None, :]).sum())
            t = med[f"attn_{kk_}"]
            out["steps"][str(path.info[kk_]["h"])] = {
                "map_ms": med[f"map_{kk_}"], "attn_ms": t, "gflop": flops / 1e9, "tflops": flops / t / 1e9,
                "frac_bf16_peak": flops / t / 1e9 / PEAK_BF16_TFLOPS,
                "density": float((kept * qsz[None, :]).sum()) / (B * H * n_q * path.info[kk_]["n_tokens_le"])}
        print(json.dumps(out), flush=True)
        del path


# Block form of Cross-Scale Local Sparse Attention at the last Infinity scale with
# 24 heads (4096 queries against 10521 keys, d = 128, batch 1): sink scales and
# window sizes on the last three scales, 1-D blocks on both axes.
CSLA_SWEEP = ([dict(block=64, n_sink=5, sizes=(3, 5, 7)), dict(block=128, n_sink=5, sizes=(3, 5, 7))]
              + [dict(block=128, n_sink=5, sizes=z) for z in ((1, 3, 5), (3, 3, 3), (5, 5, 5), (5, 7, 9),
                                                             (7, 7, 7), (7, 9, 11))]
              + [dict(block=128, n_sink=n, sizes=(3, 5, 7)) for n in (6, 7, 8, 0)])


def sweep_csla(dev, only=None):
    """CSLA block path: block-row build and attention times, kept density and the
    attention's algorithmic TFLOP/s (4 d * kept query-key pairs), against our
    dense kernel at the same shape."""
    import torch

    from paper_2602_04361_amd import sparvar as sv
    from paper_2602_04361_amd.synth import make_qkv

    B, H, d, k = 1, 24, 128, 13
    n0 = sum(x * x for x in SIDES[:k - 1])
    n_q, n_kv = SIDES[k - 1] ** 2, n0 + SIDES[k - 1] ** 2
    sets = []
    for s in range(2):
        q, kk, v = make_qkv(SIDES, SIDES, B, H, d, CFG["n_freq"], 5, seed=100 + s, bf16=True)
        sets.append((torch.from_numpy(q[:, :, n0:n_kv]).to(dev).to(torch.bfloat16),
                     torch.from_numpy(kk).to(dev).to(torch.bfloat16), torch.from_numpy(v).to(dev).to(torch.bfloat16)))
    o = torch.empty(B, H, n_q, d, dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream()
    scale = 1.0 / math.sqrt(d)

    def timed(fn, n=20):
        for i in range(3):
            fn(i)
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        for i in range(n):
            evs[i][0].record(stream)
            fn(i)
            evs[i][1].record(stream)
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in evs]))

    t_dense = timed(lambda i: sv.sparvar_dense_attn_fwd(*sets[i % 2], o, None, softmax_scale=scale))
    dense_flops = 4.0 * d * B * H * n_q * n_kv
    for st in CSLA_SWEEP if only is None else only:
        g = sv.Geometry(SIDES, SIDES, CFG["b"], st["n_sink"])
        blk = st["block"]
        wins = [0] * (k - len(st["sizes"])) + list(st["sizes"])
        M = sv.sparvar_csla_row_stride(g, k, blk)
        rows = torch.empty(-(-n_q // blk), M, dtype=torch.int32, device=dev)
        t_rows = timed(lambda i: sv.sparvar_csla_block_rows(g, k, wins, blk, rows))
        t_attn = timed(lambda i: sv.sparvar_csla_attn_fwd(g, k, blk, *sets[i % 2], o, rows, softmax_scale=scale))
        r = rows.cpu().numpy()
        pairs = 0
        for u in range(r.shape[0]):
            ids = r[u][r[u] >= 0]
            nq = min(blk, n_q - u * blk)
            pairs += nq * int(sum(min(blk, n_kv - v * blk) for v in ids))
        flops = 4.0 * d * B * H * pairs
        print(json.dumps({"sweep": f"csla_b{blk}_sink{st['n_sink']}_w{'-'.join(map(str, st['sizes']))}",
                          "B": B, "H": H, "n_q": n_q, "n_kv": n_kv, "block": blk, "n_sink_scales": st["n_sink"],
                          "windows_last3": list(st["sizes"]), "rows_ms": t_rows, "attn_ms": t_attn,
                          "density": pairs / (n_q * n_kv), "sparsity": 1.0 - pairs / (n_q * n_kv),
                          "gflop": flops / 1e9, "tflops": flops / t_attn / 1e9,
                          "frac_bf16_peak": flops / t_attn / 1e9 / PEAK_BF16_TFLOPS,
                          "dense_ms": t_dense, "dense_tflops": dense_flops / t_dense / 1e9,
                          "speedup_vs_own_dense": t_dense / t_attn}), flush=True)


def sweep_kv_compression(dev):
    """KV compression at the 24-head last-scale shape: keep the sink scales 1-5 and
    the windowed scales 11-13, copy them into a compact cache (HBM-bound gather:
    GB/s against 8 TB/s), and run the CSLA block path (blocks of 128) on it."""
    import torch

    from paper_2602_04361_amd import sparvar as sv
    from paper_2602_04361_amd.synth import make_qkv

    B, H, d, k, blk = 1, 24, 128, 13, 128
    keep = [1, 2, 3, 4, 5, 11, 12, 13]
    n0 = sum(x * x for x in SIDES[:k - 1])
    n_q, n_kv = SIDES[k - 1] ** 2, n0 + SIDES[k - 1] ** 2
    q, kk, v = make_qkv(SIDES, SIDES, B, H, d, CFG["n_freq"], 5, seed=100, bf16=True)
    Q = torch.from_numpy(q[:, :, n0:n_kv]).to(dev).to(torch.bfloat16)
    K = torch.from_numpy(kk).to(dev).to(torch.bfloat16)
    V = torch.from_numpy(v).to(dev).to(torch.bfloat16)
    g = sv.Geometry(SIDES, SIDES, CFG["b"], 5)
    gc = sv.compact_geometry(g, keep)
    m = sum(SIDES[l - 1] ** 2 for l in keep)
    Kc = torch.empty(B, H, m, d, dtype=torch.bfloat16, device=dev)
    Vc = torch.empty_like(Kc)
    o = torch.empty_like(Q)
    stream = torch.cuda.current_stream()

    def timed(fn, n=20):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        for a, b in evs:
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in evs]))

    t_copy = timed(lambda: sv.sparvar_kv_compact(g, keep, K, V, Kc, Vc))
    copy_bytes = 2.0 * 2 * B * H * m * d * 2  # K and V, read and written
    kc = len(keep)
    wins = [0] * (kc - 3) + [3, 5, 7]
    M = sv.sparvar_csla_row_stride(gc, kc, blk)
    rows = torch.empty(-(-n_q // blk), M, dtype=torch.int32, device=dev)
    sv.sparvar_csla_block_rows(gc, kc, wins, blk, rows)
    t_attn = timed(lambda: sv.sparvar_csla_attn_fwd(gc, kc, blk, Q, Kc, Vc, o, rows))
    r = rows.cpu().numpy()
    pairs = sum(min(blk, n_q - u * blk) * sum(min(blk, m - x * blk) for x in r[u][r[u] >= 0]) for u in range(len(r)))
    flops = 4.0 * d * B * H * pairs
    print(json.dumps({"sweep": "kv_compression_sink5_local3_b128", "B": B, "H": H, "kept_scales": keep,
                      "kv_tokens_full": n_kv, "kv_tokens_kept": m,
                      "kv_bytes_full": 2 * B * H * n_kv * d * 2, "kv_bytes_kept": 2 * B * H * m * d * 2,
                      "compact_ms": t_copy, "compact_gbs": copy_bytes / t_copy / 1e6,
                      "compact_frac_hbm_peak": copy_bytes / t_copy / 1e6 / 8000.0,
                      "attn_ms": t_attn, "tflops": flops / t_attn / 1e9,
                      "frac_bf16_peak": flops / t_attn / 1e9 / PEAK_BF16_TFLOPS,
                      "density_of_compact": pairs / (n_q * m)}), flush=True)


# ---------------------------------------------------------------- main
def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the path shards by (batch, head) "
              f"with no exchange inside attention, and the benchmark measures one GPU's share.", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2602_04361_amd import sparvar as sv
    from paper_2602_04361_amd.pipeline import SparsePath
    from paper_2602_04361_amd.synth import make_qkv

    sv.load_library()
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    if args.sweep and args.only:
        sweep(args, dev, only=args.only)
        return
    if args.sweep:
        sweep(args, dev)
        sweep_cs4a(dev)
        sweep_csla(dev)
        sweep_kv_compression(dev)
        return
    if args.csla:
        sweep_csla(dev)
        sweep_kv_compression(dev)
        return
    B, H, d = CFG["B"], CFG["H"], CFG["d"]
    BH = B * H
    g = sv.Geometry(SIDES, SIDES, CFG["b"], CFG["n_sink"])
    sets, host0 = [], None
    for s in range(args.sets):
        q, k, v = make_qkv(SIDES, SIDES, B, H, d, CFG["n_freq"], CFG["n_sink"], seed=s, bf16=True)
        if s == 0:
            host0 = (q, k, v)
        sets.append(tuple(torch.from_numpy(x).to(dev).to(torch.bfloat16) for x in (q, k, v)))
        print(f"[bench] input set {s} resident", file=sys.stderr, flush=True)
    path = SparsePath(g, CFG["S"], CFG["steps"], B, H, d, CFG["topk"], CFG["radius"])
    info = path.info
    stream = torch.cuda.current_stream()

    names = ["decision", "map", "attn_11", "attn_12", "attn_13"]

    def one_step(i, ev=None):
        Q, K, V = sets[i % len(sets)]
        if ev is not None:
            ev[0].record(stream)
        path.decision(Q, K, V)
        if ev is not None:
            ev[1].record(stream)
        # the rows of all three steps depend only on the selection at S; with them,
        # each step's launch order (longest first inside each XCD's share)
        path.map_all(orders=True)
        if ev is not None:
            ev[2].record(stream)
        for j, kk in enumerate(CFG["steps"]):
            path.attn_step(kk, Q, K, V, use_order=True)
            if ev is not None:
                ev[3 + j].record(stream)

    # clock ramp: whole steps for a fixed time, so that the warm-up and timed steps
    # run at the steady clock (after 5 steps a layer takes about 18% longer than
    # after 0.25 s of sustained work); nothing it computes is reused
    t_ramp = time.perf_counter()
    n_ramp = 0
    while time.perf_counter() - t_ramp < args.ramp_seconds:
        for _ in range(10):
            one_step(n_ramp)
            n_ramp += 1
        torch.cuda.synchronize()
    ramp_s = time.perf_counter() - t_ramp
    for i in range(args.warmup):
        one_step(i)
    torch.cuda.synchronize()

    # accounting from the CSR built on set 0 (outside the timed region)
    one_step(0)
    torch.cuda.synchronize()
    acct = {}
    for kk in CFG["steps"]:
        rp, ci, _ = path.csr[kk]
        acct[kk] = sparse_accounting(rp.cpu().numpy(), ci.cpu().numpy(), info, kk, BH, d)
    iS = info[CFG["S"]]
    dense_S_flops = 4.0 * d * BH * iS["n_tokens"] * iS["n_tokens_le"]
    step_flops = dense_S_flops + sum(a[0] for a in acct.values())

    # timed region
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(args.steps):
        one_step(i, evs[i])
        evs[i][-1].record(stream)
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    step_ms = np.array([evs[i][0].elapsed_time(evs[i][-1]) for i in range(args.steps)])
    ms_step = total_ms / args.steps
    samples = {n: np.array([evs[i][j].elapsed_time(evs[i][j + 1]) for i in range(args.steps)])
               for j, n in enumerate(names)}
    per = {n: float(np.mean(x)) for n, x in samples.items()}
    spread = {n: {"median": float(np.median(x)), "p10": float(np.percentile(x, 10)), "p90": float(np.percentile(x, 90))}
              for n, x in samples.items()}

    # our dense kernel at the 64x64 step (speedup denominator), same buffers and rotation
    i13 = info[13]
    o_dense = torch.empty(B, H, i13["n_tokens"], d, dtype=torch.bfloat16, device=dev)
    for i in range(3):
        Q, K, V = sets[i % len(sets)]
        sv.sparvar_dense_attn_fwd(path.q_slice(Q, 13), path.kv_prefix(K, 13), path.kv_prefix(V, 13), o_dense, None,
                                  softmax_scale=path.scale)
    torch.cuda.synchronize()
    dn = max(3, min(args.steps, 10))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(dn):
        Q, K, V = sets[i % len(sets)]
        sv.sparvar_dense_attn_fwd(path.q_slice(Q, 13), path.kv_prefix(K, 13), path.kv_prefix(V, 13), o_dense, None,
                                  softmax_scale=path.scale)
    e1.record(stream)
    torch.cuda.synchronize()
    dense64_ms = e0.elapsed_time(e1) / dn
    dense64_flops = 4.0 * d * BH * i13["n_tokens"] * i13["n_tokens_le"]

    # warm number, labelled as such: the 64x64 sparse attention repeated on one
    # input set (its K/V partly cache-resident from the previous launch)
    Q0, K0, V0 = sets[0]
    one_step(0)  # the rows of set 0, which the accounting used
    torch.cuda.synchronize()
    wn = 20
    we = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(wn)]
    for a_, b_ in we:
        a_.record(stream)
        path.attn_step(13, Q0, K0, V0, use_order=True)
        b_.record(stream)
    torch.cuda.synchronize()
    warm13_ms = float(np.median([a_.elapsed_time(b_) for a_, b_ in we]))

    f13, b13, dens13, _ = acct[13]
    attn13_ms = per["attn_13"]
    kernels = {"decision": {"ms": per["decision"], "tflops": dense_S_flops / per["decision"] / 1e9,
                            **{"ms_" + q: v for q, v in spread["decision"].items()}},
               "map_all_steps": {"ms": per["map"], **{"ms_" + q: v for q, v in spread["map"].items()}}}
    for kk in CFG["steps"]:
        f, b_, dens, keys = acct[kk]
        side = info[kk]["h"]
        kernels[f"attn_{side}"] = {"ms": per[f"attn_{kk}"], **{"ms_" + q: v for q, v in spread[f"attn_{kk}"].items()},
                                   "gflop": f / 1e9,
                                   "tflops": f / per[f"attn_{kk}"] / 1e9,
                                   "frac_bf16_peak": f / per[f"attn_{kk}"] / 1e9 / PEAK_BF16_TFLOPS,
                                   "hbm_gbs_algorithmic": b_ / per[f"attn_{kk}"] / 1e6,
                                   "density": dens, "kept_keys_per_row_mean": float(np.mean(keys))}
    dominant = max(kernels, key=lambda n: kernels[n]["ms"])
    khash = kernel_source_hash()
    traffic = profile_value("sparse_attn_64_traffic.txt", "hbm_bytes_per_launch", khash)
    issued = profile_value("sparse_attn_64_mfma.txt", "mfma_flops_per_launch", khash)
    achieved = f13 / attn13_ms / 1e9
    # the roof that bounds the kernel at its algorithmic intensity: MFMA above the
    # ridge (peak FLOP/s over peak bytes/s), HBM below it
    intensity = f13 / b13
    ridge = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    roofline = {"kernel": "block-sparse attention, 64x64 step", "bound": "mfma" if intensity >= ridge else "hbm",
                "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                "traffic": traffic, "algorithmic_bytes": b13, "algorithmic_flops": f13,
                "intensity_flop_per_byte": intensity, "ridge_flop_per_byte": ridge,
                "hbm_frac_algorithmic": b13 / attn13_ms / 1e6 / PEAK_HBM_GBS,
                "dominant_kernel_in_step": dominant}

    if args.copy_calibration:
        # plain device copies of known size: the reference that scales the HBM byte
        # counters (FETCH_SIZE, WRITE_SIZE) of the kernels above
        src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] copy calibration: 3 x {src.numel() * 4} bytes read and written", file=sys.stderr, flush=True)
        del src, dst
        # the same check on the attention kernel itself: every tile of the 64x64 step
        # lists only its own block, so each K/V token is read once (last dispatches of
        # the sparse kernel in the run)
        rp_np, ci_np = own_block_rows(info, 13, BH)
        rp_c = torch.from_numpy(rp_np).to(dev)
        ci_c = torch.from_numpy(ci_np).to(dev)
        o_c = torch.empty(B, H, i13["n_tokens"], d, dtype=torch.bfloat16, device=dev)
        for i in range(2):
            Q, K, V = sets[(i + 1) % len(sets)]
            sv.sparvar_block_sparse_attn_fwd(g, 13, path.q_slice(Q, 13), path.kv_prefix(K, 13),
                                             path.kv_prefix(V, 13), o_c, rp_c, ci_c, softmax_scale=path.scale)
        torch.cuda.synchronize()
        cb = BH * i13["n_tokens"] * d * 2
        print(f"[bench] attention calibration: 2 launches, each reading {3 * cb} bytes (Q + K + V of scale 13) and "
              f"writing {cb} bytes (O)", file=sys.stderr, flush=True)
        del o_c

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(*host0, args.cpu_seconds)

    line = {
        "metric": "ms/layer + effective TFLOP/s (% bf16 MFMA peak) sparse attn at 64x64 scale",
        "value": achieved,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) Q/K/V + 2-D sinusoidal position features + sink bias), 4 rotating sets",
        "config": {"workload": "Infinity 1024x1024 schedule, one layer: dense attention + selection at 32x32, "
                               "block-sparse steps 40x40/48x48/64x64", "batch": B, "heads": H, "head_dim": d,
                   "block": "8x8 tokens", "topk": CFG["topk"], "window_radius": CFG["radius"],
                   "sink_scales": CFG["n_sink"], "kv_tokens_last_step": info[13]["n_tokens_le"]},
        "value_is": "algorithmic TFLOP/s of the block-sparse attention at the 64x64 step, timed inside the step",
        "clock_ramp": {"seconds": ramp_s, "steps": n_ramp},
        "ms_per_layer": ms_step,
        "layer_tflops": step_flops / ms_step / 1e9,
        "ms_per_step_spread": {"median": float(np.median(step_ms)), "p10": float(np.percentile(step_ms, 10)),
                               "p90": float(np.percentile(step_ms, 90))},
        "sparse_64": {"ms": attn13_ms, "tflops": achieved, "frac_bf16_peak": achieved / PEAK_BF16_TFLOPS,
                      "dense_equivalent_tflops": dense64_flops / attn13_ms / 1e9,
                      "mfma_issued_flops": issued,
                      "mfma_padding_efficiency": (f13 / issued) if issued else None,
                      "warm_same_buffers_ms": warm13_ms,
                      "warm_same_buffers_tflops": f13 / warm13_ms / 1e9,
                      "density": dens13, "dense_ms": dense64_ms,
                      "dense_tflops": dense64_flops / dense64_ms / 1e9,
                      "dense_frac_bf16_peak": dense64_flops / dense64_ms / 1e9 / PEAK_BF16_TFLOPS,
                      "speedup_vs_own_dense": dense64_ms / attn13_ms},
        "kernels": kernels,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line, default=lambda o: o.item() if hasattr(o, "item") else str(o)))


if __name__ == "__main__":
    main()

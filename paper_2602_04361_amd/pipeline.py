"""One layer of the SparVAR sparse path on the GPU, as a sequence of C-ABI calls.

SparsePath owns the device buffers (allocated with torch) and issues, on the
current stream:
  decision(): dense attention with LSE at the decision scale S, pooled block
              scores and per-query-tile top-k in one sparvar_decision_step
              call (or, with fused=False, sparvar_dense_attn_fwd followed by
              sparvar_select_blocks);
  step(k):    sparvar_map_index (mapped + local blocks -> CSR + schedule), then
              sparvar_block_sparse_attn_fwd at scale k;
  map_all():  the rows of every step in one sparvar_map_index_steps launch
              (they depend only on the selection at S).
Local rows are geometry-only and built once per step by build_local().
All arithmetic runs in libsparvar.so; this module only allocates and calls.
"""
from __future__ import annotations

import math

import torch

from . import sparvar as sv


class SparsePath:
    def __init__(self, geom: sv.Geometry, S, steps, B, H, d, topk, radius, prev_dilation=0,
                 dtype=torch.bfloat16, device="cuda", use_schedule=False, softmax_scale=None, local_lists=False,
                 fused_decision=True, projection="point"):
        self.g = geom
        self.S, self.steps = int(S), [int(k) for k in steps]
        self.B, self.H, self.d = B, H, d
        self.topk, self.radius, self.dil = topk, radius, prev_dilation
        self.dtype, self.device = dtype, device
        # local_lists: build the sink + local rows once with sparvar_local_blocks and
        # pass them to the mapping; otherwise the mapping generates them itself.
        self.local_lists = local_lists
        self.fused_decision = fused_decision
        # projection of the mapped blocks: "point" (tile origin) or "cover" (every tile of the upsampled span)
        self.projection = sv.PROJECTIONS[projection]
        self.scale = float(torch.tensor(1.0 / math.sqrt(d), dtype=torch.float32)) if softmax_scale is None \
            else float(softmax_scale)
        info = {l: geom.scale_info(l) for l in range(1, len(geom.h) + 1)}
        self.info = info
        iS = info[S]
        G_S, NB_S = iS["tiles_h"] * iS["tiles_w"], iS["n_blocks_le"]
        i32 = dict(dtype=torch.int32, device=device)
        self.o_S = torch.empty(B, H, iS["n_tokens"], d, dtype=dtype, device=device)
        self.lse_S = torch.empty(B, H, iS["n_tokens"], dtype=torch.float32, device=device)
        self.scores = torch.empty(B, H, G_S, NB_S, dtype=torch.float32, device=device)
        self.topk_idx = torch.empty(B, H, G_S, topk, **i32)
        self.local, self.csr, self.out = {}, {}, {}
        for k in self.steps:
            ik = info[k]
            G_k = ik["tiles_h"] * ik["tiles_w"]
            cap_l = sv.sparvar_local_blocks_capacity(geom, k, radius, prev_dilation)
            self.local[k] = (torch.empty(G_k + 1, **i32), torch.empty(max(cap_l, 1), **i32))
            cap = sv.sparvar_map_index_capacity(geom, S, k, B, H, topk, radius, prev_dilation, self.projection)
            rows = B * H * G_k
            self.csr[k] = (torch.empty(rows + 1, **i32), torch.empty(cap, **i32),
                           torch.empty(rows, **i32) if use_schedule else None)
            self.out[k] = torch.empty(B, H, ik["n_tokens"], d, dtype=dtype, device=device)
        self.orders = {}

    # ------------------------------------------------------------------ calls
    def build_local(self):
        for k in self.steps:
            rp, ci = self.local[k]
            sv.sparvar_local_blocks(self.g, k, self.radius, rp, ci, prev_dilation=self.dil)

    def q_slice(self, Q_all, l):
        i = self.info[l]
        return Q_all[:, :, i["token_offset"]:i["n_tokens_le"]]

    def kv_prefix(self, X_all, l):
        return X_all[:, :, :self.info[l]["n_tokens_le"]]

    def decision(self, Q_all, K_all, V_all):
        S = self.S
        q, kk, vv = self.q_slice(Q_all, S), self.kv_prefix(K_all, S), self.kv_prefix(V_all, S)
        if self.fused_decision:
            sv.sparvar_decision_step(self.g, S, q, kk, vv, self.o_S, self.lse_S, self.scores, self.topk,
                                     self.topk_idx, softmax_scale=self.scale)
            return
        sv.sparvar_dense_attn_fwd(q, kk, vv, self.o_S, self.lse_S, softmax_scale=self.scale)
        sv.sparvar_select_blocks(self.g, S, q, kk, self.lse_S, self.topk, self.topk_idx, scores_out=self.scores,
                                 softmax_scale=self.scale)

    def map_step(self, k):
        rp_l, ci_l = self.local[k] if self.local_lists else (None, None)
        rp, ci, sch = self.csr[k]
        sv.sparvar_map_index(self.g, self.S, k, self.B, self.H, self.topk, self.topk_idx, rp_l, ci_l, self.radius,
                             rp, ci, schedule=sch, prev_dilation=self.dil, projection=self.projection)

    def map_all(self, orders=False):
        """The rows of every sparse step in one launch (generated local rows); with orders, also each step's
        attention launch order (longest first inside each XCD's share), used by attn_step(use_order=True)."""
        if orders and not self.orders:
            i32 = dict(dtype=torch.int32, device=self.device)
            self.orders = {k: torch.empty(self.B * self.H * self.info[k]["tiles_h"] * self.info[k]["tiles_w"], **i32)
                           for k in self.steps}
        sv.sparvar_map_index_steps(self.g, self.S, self.steps, self.B, self.H, self.topk, self.topk_idx, self.radius,
                                   [self.csr[k][0] for k in self.steps], [self.csr[k][1] for k in self.steps],
                                   prev_dilation=self.dil, projection=self.projection,
                                   orders=[self.orders[k] for k in self.steps] if orders else None)

    def attn_step(self, k, Q_all, K_all, V_all, lse=None, use_schedule=True, use_order=False):
        rp, ci, sch = self.csr[k]
        if use_order:
            sch, use_schedule = self.orders[k], True
        sv.sparvar_block_sparse_attn_fwd(self.g, k, self.q_slice(Q_all, k), self.kv_prefix(K_all, k),
                                         self.kv_prefix(V_all, k), self.out[k], rp, ci, lse=lse,
                                         schedule=sch if use_schedule else None, softmax_scale=self.scale)

    def step(self, k, Q_all, K_all, V_all):
        self.map_step(k)
        self.attn_step(k, Q_all, K_all, V_all)

    def run(self, Q_all, K_all, V_all):
        """Decision step plus every sparse step (with local_lists, build_local() first)."""
        self.decision(Q_all, K_all, V_all)
        for k in self.steps:
            self.step(k, Q_all, K_all, V_all)


class Cs4aPath:
    """One layer of the token-granular CS^4A path (Sec. 3.2) as C-ABI calls.

    decision(): dense attention with LSE at S, column sums over 1-D query blocks
                of C queries, the top-K tokens of each block, and O_cache at S
                (O_dense minus the attention restricted to those tokens);
    step(k):    the token rows of scale k (sinks + mapped tokens), then the
                gather attention, adding the upsampled O_cache unless
                with_cache is False.
    """

    def __init__(self, geom: sv.Geometry, S, steps, B, H, d, C, K, device="cuda", softmax_scale=None,
                 with_cache=True):
        self.g = geom
        self.S, self.steps = int(S), [int(k) for k in steps]
        self.B, self.H, self.d, self.C, self.K = B, H, d, C, K
        self.with_cache = with_cache
        self.scale = float(torch.tensor(1.0 / math.sqrt(d), dtype=torch.float32)) if softmax_scale is None \
            else float(softmax_scale)
        info = {l: geom.scale_info(l) for l in range(1, len(geom.h) + 1)}
        self.info = info
        iS = info[S]
        G_S = -(-iS["n_tokens"] // C)
        bf = dict(dtype=torch.bfloat16, device=device)
        self.o_S = torch.empty(B, H, iS["n_tokens"], d, **bf)
        self.lse_S = torch.empty(B, H, iS["n_tokens"], dtype=torch.float32, device=device)
        self.colsum = torch.empty(B, H, G_S, iS["n_tokens_le"], dtype=torch.float32, device=device)
        self.inds = torch.empty(B, H, G_S, K, dtype=torch.int32, device=device)
        self.o_cache = torch.empty(B, H, iS["n_tokens"], d, **bf)
        self.M = sv.sparvar_cs4a_row_stride(geom, K)
        self.tokens, self.out = {}, {}
        for k in self.steps:
            G_k = -(-info[k]["n_tokens"] // C)
            self.tokens[k] = torch.empty(B, H, G_k, self.M, dtype=torch.int32, device=device)
            self.out[k] = torch.empty(B, H, info[k]["n_tokens"], d, **bf)

    def q_slice(self, Q_all, l):
        i = self.info[l]
        return Q_all[:, :, i["token_offset"]:i["n_tokens_le"]]

    def kv_prefix(self, X_all, l):
        return X_all[:, :, :self.info[l]["n_tokens_le"]]

    def decision(self, Q_all, K_all, V_all):
        S = self.S
        q, kk, vv = self.q_slice(Q_all, S), self.kv_prefix(K_all, S), self.kv_prefix(V_all, S)
        sv.sparvar_dense_attn_fwd(q, kk, vv, self.o_S, self.lse_S, softmax_scale=self.scale)
        sv.sparvar_cs4a_column_sums(self.g, S, self.C, q, kk, self.lse_S, self.colsum, softmax_scale=self.scale)
        sv.sparvar_cs4a_select_tokens(self.colsum, self.K, self.inds)
        if self.with_cache:
            sv.sparvar_cs4a_attn_fwd(self.g, S, self.C, q, kk, vv, self.o_cache, self.inds, self.K, mode=1,
                                     base=self.o_S, softmax_scale=self.scale)

    def step(self, k, Q_all, K_all, V_all):
        sv.sparvar_cs4a_map_tokens(self.g, self.S, k, self.C, self.B, self.H, self.K, self.inds, self.tokens[k],
                                   self.M)
        sv.sparvar_cs4a_attn_fwd(self.g, k, self.C, self.q_slice(Q_all, k), self.kv_prefix(K_all, k),
                                 self.kv_prefix(V_all, k), self.out[k], self.tokens[k], self.M,
                                 mode=2 if self.with_cache else 0, base=self.o_cache if self.with_cache else None,
                                 base_scale=self.S, softmax_scale=self.scale)

    def run(self, Q_all, K_all, V_all):
        self.decision(Q_all, K_all, V_all)
        for k in self.steps:
            self.step(k, Q_all, K_all, V_all)


class CslaPath:
    """One layer of the paper-literal CSLA block path (Sec. 3.3) as C-ABI calls.

    The block rows of each sparse scale depend only on the geometry, the window
    sizes and the block size, so they are built once (rows()) and reused by every
    layer and head; step(k) runs the block-sparse attention of scale k.
    windows[k] lists one window size per scale 1..k (0: no local keys there).
    """

    def __init__(self, geom: sv.Geometry, steps, windows, block, B, H, d, device="cuda", softmax_scale=None):
        self.g = geom
        self.steps = [int(k) for k in steps]
        self.windows = {int(k): [int(w) for w in windows[k]] for k in self.steps}
        self.block, self.B, self.H, self.d = int(block), B, H, d
        self.scale = float(torch.tensor(1.0 / math.sqrt(d), dtype=torch.float32)) if softmax_scale is None \
            else float(softmax_scale)
        self.info = {l: geom.scale_info(l) for l in range(1, len(geom.h) + 1)}
        self.block_rows, self.out = {}, {}
        for k in self.steps:
            M = sv.sparvar_csla_row_stride(geom, k, self.block)
            G_k = -(-self.info[k]["n_tokens"] // self.block)
            self.block_rows[k] = torch.empty(G_k, M, dtype=torch.int32, device=device)
            self.out[k] = torch.empty(B, H, self.info[k]["n_tokens"], d, dtype=torch.bfloat16, device=device)

    def rows(self):
        for k in self.steps:
            sv.sparvar_csla_block_rows(self.g, k, self.windows[k], self.block, self.block_rows[k])

    def step(self, k, Q_all, K_all, V_all):
        i = self.info[k]
        sv.sparvar_csla_attn_fwd(self.g, k, self.block, Q_all[:, :, i["token_offset"]:i["n_tokens_le"]],
                                 K_all[:, :, :i["n_tokens_le"]], V_all[:, :, :i["n_tokens_le"]], self.out[k],
                                 self.block_rows[k], softmax_scale=self.scale)
        return self.out[k]

// Fused decision step at scale S (Sec. 3.2): dense attention of the scale-S
// queries over the keys of scales 1..S with its LSE, the pooled block scores
// (softmax mass summed over a query tile and a key block) and the per-tile
// top-k, in one launch and without a second S = Q K^T pass.
//
// A workgroup owns one query tile g of one (b, h) plane: WPT waves of 32 queries
// per key split, KS key splits (contiguous ranges of block ids, balanced by
// chunk count), NW = WPT * KS waves. The waves of a split walk its blocks one
// tile-row band (<= 32 keys) at a time through their own two LDS stages, with
// the attention core of attn_chunk.h, and keep for every query the probability
// mass of each block relative to the running max (rescaled with the
// accumulator whenever the max moves): the current block's in a register, each
// finished block's in LDS. After the walk the splits are merged in
// LDS (max, sum, output), and a block's score is sum over the tile's queries of
// its mass divided by that query's softmax sum: exactly the sum of the
// normalised probabilities. Top-k follows in the same workgroup: a block is
// kept iff fewer than topk blocks beat it (higher score, or equal score and
// lower id), and kept ids are written ascending, -1 after them.
#include <type_traits>

#include "attn_chunk.h"
#include "device_common.h"
#include "launch.h"

namespace sparvar {

constexpr int kMaxSplits = 2;

struct DecisionIO {
  GeoTable G;
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;
  float* scores;      // nullable, [B,H,G_S,NB]
  int32_t* topk_idx;  // [B,H,G_S,topk]
  int64_t q_bh_stride, kv_bh_stride;
  int32_t S, G_S, NB, topk;
  int32_t vb[kMaxSplits + 1];  // block range of each key split
  int32_t steps;               // chunks of the longest split
  int32_t pstride;             // partial-mass row length (>= longest split in blocks, odd)
  int32_t n_items, swizzle;
  float scale_log2;
};

// Dynamic LDS layout (floats): mass [KS][WQ][pstride], ml [KS][WQ][2],
// fac [KS][WQ], scores [NB], keep [NB] (int).
template <int D, int WPT, int KS>
__global__ __launch_bounds__(WPT * KS * 64) void decision_kernel(DecisionIO io) {
  constexpr int KC = 32;
  constexpr int NW = WPT * KS;
  constexpr int NT = NW * 64;
  constexpr int WQ = WPT * kQPerWave;  // query slots of the tile
  constexpr int U = D / 8;
  constexpr int kRow = D * 2;
  constexpr int kTile = KC * kRow;
  constexpr int kStage = 2 * kTile;
  constexpr int kLoads = KC * U / (WPT * 64);  // direct loads per thread per tensor (one split's waves)
  static_assert((KC * U) % (WPT * 64) == 0, "chunk must split evenly over a split's waves");
  static_assert(KS >= 1 && KS <= kMaxSplits, "key splits");
  static_assert(KS == 1 || WPT * kQPerWave * D * 4 <= 2 * kStage, "split outputs must fit the stages they merge through");
  // stages of split s: s_0 (stage 0) and s_1 (stage 1), each its own array
  __shared__ __attribute__((aligned(16))) char st00[kStage];
  __shared__ __attribute__((aligned(16))) char st01[kStage];
  __shared__ __attribute__((aligned(16))) char st10[KS > 1 ? kStage : 16];
  __shared__ __attribute__((aligned(16))) char st11[KS > 1 ? kStage : 16];
  extern __shared__ float dyn[];

  const int32_t item = swizzled_item(blockIdx.x, gridDim.x, io.swizzle);
  if (item >= io.n_items) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int split = __builtin_amdgcn_readfirstlane(wave / WPT);
  const int slab = __builtin_amdgcn_readfirstlane(wave % WPT);
  const GeoTable& G = io.G;
  const int S = io.S;

  const int32_t bh = item / io.G_S;
  const int32_t g = item - bh * io.G_S;
  const int32_t tw = G.Tw[S - 1];
  const Tile qt = tile_at(G, S, g / tw, g % tw);
  const int32_t nq = qt.nr * qt.nc;
  const int32_t qslot = slab * kQPerWave + l32;
  const bool qvalid = qslot < nq;
  const int32_t qi = qvalid ? qslot : 0;
  const int32_t qrow = (qt.base - G.C[S - 1]) + (qi / qt.nc) * qt.stride + (qi % qt.nc);

  const bf16_bits* qplane = static_cast<const bf16_bits*>(io.q) + (int64_t)bh * io.q_bh_stride;
  const char* kbytes = reinterpret_cast<const char*>(static_cast<const bf16_bits*>(io.k) + (int64_t)bh * io.kv_bh_stride);
  const char* vbytes = reinterpret_cast<const char*>(static_cast<const bf16_bits*>(io.v) + (int64_t)bh * io.kv_bh_stride);
  QFragBF16<D> qf;
  qf.load(qplane + (int64_t)qrow * D, half);

  const int32_t ps = io.pstride;
  float* mass = dyn;                         // [KS][WQ][ps]
  float* ml = mass + KS * WQ * ps;           // [KS][WQ][2]
  float* fac = ml + KS * WQ * 2;             // [KS][WQ]
  float* sc_out = fac + KS * WQ;             // [NB]
  int32_t* keep = reinterpret_cast<int32_t*>(sc_out + io.NB);  // [NB]
  for (int32_t i = tid; i < KS * WQ * ps; i += NT) mass[i] = 0.f;
  float* my_mass = mass + (split * WQ + qslot) * ps;  // this query's row of block masses (half 0 writes)

  f32x16 acc[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) acc[i] = zero16();
  float m_run = -INFINITY, l_run = 0.f;
  const float sl2 = io.scale_log2;

  int ld_row[kLoads], ld_unit[kLoads];
#pragma unroll
  for (int j = 0; j < kLoads; ++j) {
    const int slot = (j * WPT + slab) * 64 + lane;
    ld_row[j] = slot / U;
    ld_unit[j] = (slot % U) ^ (unit_swizzle(ld_row[j]) & (U - 1));
  }
  FragOffsets<D, KC> fo;
  fo.init(l32, half, lane);
  const int32_t v0 = io.vb[split];

  // The walk of one split over its two stages (compile-time arrays, so every LDS
  // address is a lane register plus an immediate). Every wave runs io.steps
  // barriers whatever its split's chunk count.
  auto walk_split = [&](auto sp_c) {
    constexpr int SP = decltype(sp_c)::value;
    char* const s0 = SP == 0 ? st00 : st10;
    char* const s1 = SP == 0 ? st01 : st11;
    auto issue = [&](const Chunk& c, char* stg) {
#pragma unroll
      for (int j = 0; j < kLoads; ++j) {
        const int first = (j * WPT + slab) * 64;
        const int r = ld_row[j];
        const uint32_t off = (uint32_t)(chunk_token(c, chunk_slot(r, c.count)) * D + 8 * ld_unit[j]) * 2u;
        dma16(kbytes + off, stg + first * 16);
        dma16(vbytes + off, stg + kTile + first * 16);
      }
    };
    BlockWalker<KC> walk;
    walk.start(&G, v0, io.vb[split + 1]);
    Chunk cur;
    int32_t blk = 0;
    bool last = false;
    bool have = walk.next(cur, blk, last);
    if (have) issue(cur, s0);
    float cur_mass = 0.f;  // the current block's mass, stored when its last chunk is done
    auto step = [&](auto st_c) {
      constexpr int ST = decltype(st_c)::value;
      char* const stg = ST == 0 ? s0 : s1;
      char* const nstg = ST == 0 ? s1 : s0;
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
      __syncthreads();
      Chunk nxt;
      int32_t nblk = 0;
      bool nlast = false;
      const bool have_n = have && walk.next(nxt, nblk, nlast);
      if (have_n) issue(nxt, nstg);
      if (have) {
        f32x16 sc[KC / 32];
        bf16x8 pf[KC / 16];
        qk_chunk<D, KC>(stg, fo, qf, sc);
        if (cur.count < KC) mask_tail<KC>(sc, cur.count, half);
        const float mx = row_max<KC>(sc, sl2);
        if (__builtin_amdgcn_ballot_w64(mx > m_run + 8.f)) {
          const float m_new = fmaxf(m_run, mx);
          const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
          l_run *= alpha;
#pragma unroll
          for (int i = 0; i < D / 32; ++i) acc[i] *= alpha;
          if (half == 0)
            for (int32_t u = 0; u < blk - v0; ++u) my_mass[u] *= alpha;
          cur_mass *= alpha;
          m_run = m_new;
        }
        const float p = exp_pack<KC>(sc, sl2, m_run, pf);
        l_run += p;
        pv_chunk<D, KC>(stg, fo, pf, acc);
        cur_mass += sum_halves(p);
        if (last) {
          if (half == 0) my_mass[blk - v0] = cur_mass;
          cur_mass = 0.f;
        }
      }
      cur = nxt;
      blk = nblk;
      last = nlast;
      have = have_n;
    };
    for (int32_t s = 0; s < io.steps; s += 2) {
      step(std::integral_constant<int, 0>{});
      if (s + 1 < io.steps) step(std::integral_constant<int, 1>{});
    }
  };
  if (KS == 1 || split == 0) walk_split(std::integral_constant<int, 0>{});
  else walk_split(std::integral_constant<int, 1>{});

  // ---- merge the splits: max, sum, output
  const float l_tot = sum_halves(l_run);
  if (half == 0) {
    ml[(split * WQ + qslot) * 2 + 0] = m_run;
    ml[(split * WQ + qslot) * 2 + 1] = l_tot;
  }
  __syncthreads();
  float m_g = -INFINITY;
#pragma unroll
  for (int s = 0; s < KS; ++s) m_g = fmaxf(m_g, ml[(s * WQ + qslot) * 2]);
  float l_g = 0.f;
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const float ms = ml[(s * WQ + qslot) * 2];
    l_g += ms == -INFINITY ? 0.f : ml[(s * WQ + qslot) * 2 + 1] * __builtin_amdgcn_exp2f(ms - m_g);
  }
  const float own = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - m_g);
  const float inv = l_g > 0.f ? 1.f / l_g : 0.f;
  // fraction of the softmax that a unit of this split's masses stands for
  if (half == 0) fac[split * WQ + qslot] = qvalid ? own * inv : 0.f;
  if constexpr (KS > 1) {
    // split 1 hands its scaled accumulator to split 0 through its own stages
    float* ob = reinterpret_cast<float*>(slab == 0 ? st10 : st11);
    if (split == 1) {
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) ob[(dt * 16 + r) * 64 + lane] = acc[dt][r] * own;
    }
    __syncthreads();
    if (split == 0) {
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[dt][r] = acc[dt][r] * own + ob[(dt * 16 + r) * 64 + lane];
    }
  } else {
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) acc[dt] *= own;
  }
  if (split == 0 && qvalid) {
    const int64_t orow = (int64_t)bh * G.h[S - 1] * G.w[S - 1] + qrow;
    bf16_bits* op = static_cast<bf16_bits*>(io.o) + orow * D;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int d = 32 * dt + 8 * j + 4 * half;
        uint2 w;
        w.x = pack_bf16x2(acc[dt][4 * j + 0] * inv, acc[dt][4 * j + 1] * inv);
        w.y = pack_bf16x2(acc[dt][4 * j + 2] * inv, acc[dt][4 * j + 3] * inv);
        *reinterpret_cast<uint2*>(op + d) = w;
      }
    }
    if (io.lse && half == 0) io.lse[orow] = l_g > 0.f ? (m_g + __builtin_log2f(l_g)) * kLn2 : -INFINITY;
  }
  __syncthreads();

  // ---- pooled scores: score[v] = sum over the tile's queries of mass * fac
  const int32_t NB = io.NB;
  for (int32_t v = tid; v < NB; v += NT) {
    int s = 0;
#pragma unroll
    for (int t = 1; t < KS; ++t) s += v >= io.vb[t];
    const float* mrow = mass + s * WQ * ps + (v - io.vb[s]);
    const float* frow = fac + s * WQ;
    float acc_s = 0.f;
    for (int32_t q = 0; q < nq; ++q) acc_s += mrow[q * ps] * frow[q];
    sc_out[v] = acc_s;
  }
  __syncthreads();
  const int64_t row = (int64_t)bh * io.G_S + g;
  if (io.scores)
    for (int32_t v = tid; v < NB; v += NT) io.scores[row * NB + v] = sc_out[v];
  // ---- top-k
  const int32_t topk = io.topk;
  for (int32_t v = tid; v < NB; v += NT) {
    const float x = sc_out[v];
    int32_t better = 0;
    for (int32_t u = 0; u < NB; ++u) {
      const float y = sc_out[u];
      better += (y > x) || (y == x && u < v);
    }
    keep[v] = better < topk;
  }
  __syncthreads();
  int32_t* orow_k = io.topk_idx + row * topk;
  for (int32_t v = tid; v < NB; v += NT) {
    if (keep[v]) {
      int32_t pos = 0;
      for (int32_t u = 0; u < v; ++u) pos += keep[u];
      if (pos < topk) orow_k[pos] = v;
    }
  }
  const int32_t nsel = topk < NB ? topk : NB;
  for (int32_t p = nsel + tid; p < topk; p += NT) orow_k[p] = -1;
}

namespace {

// chunks of the blocks [v0, v1) at KC keys per chunk (bands of whole tile rows)
int32_t block_chunks(const GeoTable& G, int32_t v0, int32_t v1, int kc) {
  int32_t n = 0;
  for (int32_t v = v0; v < v1; ++v) {
    int l = 1;
    while (l < G.L && G.NB[l] <= v) ++l;
    const int32_t t = v - G.NB[l - 1];
    const int32_t tu = t / G.Tw[l - 1], tv = t % G.Tw[l - 1];
    const int32_t nr = (tu * G.eh[l - 1] + G.eh[l - 1] < G.h[l - 1] ? G.eh[l - 1] : G.h[l - 1] - tu * G.eh[l - 1]);
    const int32_t nc = (tv * G.ew[l - 1] + G.ew[l - 1] < G.w[l - 1] ? G.ew[l - 1] : G.w[l - 1] - tv * G.ew[l - 1]);
    const int32_t rpc = kc / nc;
    n += (nr + rpc - 1) / rpc;
  }
  return n;
}

template <int D, int WPT, int KS>
hipError_t launch_decision_t(DecisionIO io, int32_t BH, hipStream_t stream) {
  constexpr int WQ = WPT * kQPerWave;
  io.n_items = BH * io.G_S;
  const int32_t grid = io.swizzle ? (io.n_items + 7) / 8 * 8 : io.n_items;
  if (grid == 0) return hipSuccess;
  const size_t dyn = ((size_t)KS * WQ * io.pstride + (size_t)KS * WQ * 3 + 2 * (size_t)io.NB) * 4;
  hipLaunchKernelGGL((decision_kernel<D, WPT, KS>), dim3(grid), dim3(WPT * KS * 64), dyn, stream, io);
  return hipGetLastError();
}

}  // namespace

// Launch plan: waves per query tile WPT in {1, 2, 4, 8}; two key splits for
// tiles of at most 64 queries (so that B*H*G_S workgroups still fill the chip),
// one above; the split point balances the two splits' chunk counts.
struct DecisionPlan {
  bool ok;
  int wpt, ks;
  int32_t vb[kMaxSplits + 1], steps, pstride;
  size_t lds;
};

DecisionPlan plan_decision(const GeoTable& G, int S, int d) {
  DecisionPlan p{};
  p.ok = false;
  if (d != 64 && d != 128) return p;
  for (int l = 1; l <= S; ++l)
    if (G.ew[l - 1] > 32) return p;  // tile widths <= 32 keys per chunk
  const int32_t tq = G.eh[S - 1] * G.ew[S - 1];
  if (tq > 256) return p;
  p.wpt = tq <= 32 ? 1 : tq <= 64 ? 2 : tq <= 128 ? 4 : 8;
  if (d == 64 && p.wpt == 8) return p;  // a 32-key chunk of d = 64 is too small for 8 waves of loads
  p.ks = p.wpt <= 2 ? 2 : 1;
  const int32_t NB = G.NB[S];
  p.vb[0] = 0;
  p.vb[1] = NB;
  p.vb[2] = NB;
  int32_t steps = block_chunks(G, 0, NB, 32);
  if (p.ks == 2) {
    int32_t best = steps, best_v = NB, left = 0;
    for (int32_t v = 0; v <= NB; ++v) {
      const int32_t right = steps - left;
      const int32_t m = left > right ? left : right;
      if (m < best) {
        best = m;
        best_v = v;
      }
      if (v < NB) left += block_chunks(G, v, v + 1, 32);
    }
    p.vb[1] = best_v;
    steps = best;
  }
  p.steps = steps;
  int32_t longest = p.vb[1] - p.vb[0];
  if (p.ks == 2 && p.vb[2] - p.vb[1] > longest) longest = p.vb[2] - p.vb[1];
  p.pstride = (longest > 0 ? longest : 1) | 1;
  const size_t wq = (size_t)p.wpt * 32;
  const size_t dyn = ((size_t)p.ks * wq * p.pstride + (size_t)p.ks * wq * 3 + 2 * (size_t)NB) * 4;
  const size_t stages = (size_t)p.ks * 2 * 2 * 32 * d * 2;
  p.lds = dyn + stages;
  p.ok = p.lds <= 150 * 1024;
  return p;
}

bool decision_supported(const GeoTable& G, int S, int d, int32_t, size_t* lds_bytes) {
  const DecisionPlan p = plan_decision(G, S, d);
  if (lds_bytes) *lds_bytes = p.lds;
  return p.ok;
}

hipError_t launch_decision(const DecisionArgs& a, hipStream_t stream) {
  const GeoTable& G = *a.G;
  const int S = a.S;
  const DecisionPlan p = plan_decision(G, S, a.d);
  if (!p.ok) return hipErrorInvalidValue;
  DecisionIO io;
  io.G = G;
  io.q = a.q;
  io.k = a.k;
  io.v = a.v;
  io.o = a.o;
  io.lse = a.lse;
  io.scores = a.scores;
  io.topk_idx = a.topk_idx;
  io.q_bh_stride = a.q_bh_stride;
  io.kv_bh_stride = a.kv_bh_stride;
  io.S = S;
  io.G_S = tiles_of(G, S);
  io.NB = G.NB[S];
  io.topk = a.topk;
  io.swizzle = a.swizzle;
  io.scale_log2 = a.softmax_scale * kLog2e;
  for (int i = 0; i <= kMaxSplits; ++i) io.vb[i] = p.vb[i];
  io.steps = p.steps;
  io.pstride = p.pstride;
#define SV_DEC(DD, WW, KK) \
  if (a.d == DD && p.wpt == WW && p.ks == KK) return launch_decision_t<DD, WW, KK>(io, a.BH, stream);
  SV_DEC(128, 1, 2) SV_DEC(128, 2, 2) SV_DEC(128, 4, 1) SV_DEC(128, 8, 1)
  SV_DEC(64, 1, 2) SV_DEC(64, 2, 2) SV_DEC(64, 4, 1)
#undef SV_DEC
  return hipErrorInvalidValue;
}

}  // namespace sparvar

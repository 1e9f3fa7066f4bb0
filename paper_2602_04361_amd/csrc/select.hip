// Decision-scale block selection (Sec. 3.2: column-sum D and TopK).
//
// pooled_scores_kernel: one workgroup per (b, h, group of query tiles of
//   scale S). For every block v of scales 1..S it recomputes the S^T = K Q^T
//   tile with MFMA and adds P = exp(scale * s - lse) over each tile's queries and
//   the block's keys. Sums run in a fixed order (lane, shuffle tree, waves in
//   order), so results are deterministic.
// topk_kernel: one wave per (b, h, g) row; candidate v is kept iff fewer than
//   topk candidates beat it (higher score, or equal score and lower id); kept
//   ids are written ascending.
#include <type_traits>

#include "device_common.h"
#include "launch.h"

namespace sparvar {

struct ScoreIO {
  GeoTable G;
  const void* q;
  const void* k;
  const float* lse;
  float* scores;
  int64_t q_bh_stride, k_bh_stride;
  int32_t S, G_S, NB;
  int32_t per;  // blocks per workgroup along grid.y (bf16 scoring)
  float scale_log2;
};

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

// fp32 (parity-grade) scoring: K rows read straight from memory, one reduction per block.
template <typename T, int D, int NW>
__global__ __launch_bounds__(NW * 64) void pooled_scores_f32_kernel(ScoreIO io) {
  constexpr bool kBF16 = std::is_same<T, bf16_bits>::value;
  __shared__ float red[NW];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int32_t row = blockIdx.x;  // (b*H + h) * G_S + g
  const int32_t bh = row / io.G_S, g = row - bh * io.G_S;
  const GeoTable& G = io.G;
  const int S = io.S;
  const int32_t tw = G.Tw[S - 1];
  const Tile qt = tile_at(G, S, g / tw, g % tw);
  const int32_t nq = qt.nr * qt.nc;

  const int32_t qslot = wave * kQPerWave + l32;
  const bool qvalid = qslot < nq;
  const int32_t qi = qvalid ? qslot : 0;
  const int32_t qrow = (qt.base - G.C[S - 1]) + (qi / qt.nc) * qt.stride + (qi % qt.nc);

  const T* qplane = static_cast<const T*>(io.q) + (int64_t)bh * io.q_bh_stride;
  const T* kplane = static_cast<const T*>(io.k) + (int64_t)bh * io.k_bh_stride;
  using QFrag = typename std::conditional<kBF16, QFragBF16<D>, QFragF32<D>>::type;
  QFrag qf;
  qf.load(qplane + (int64_t)qrow * D, half);
  const float lse2 = io.lse[(int64_t)bh * G.h[S - 1] * G.w[S - 1] + qrow] * kLog2e;

  float* out = io.scores + (int64_t)row * io.NB;
  for (int32_t v = 0; v < io.NB; ++v) {
    const Tile t = block_tile(G, v);
    const int32_t rpc = kChunk / t.nc;
    float acc = 0.f;
    for (int32_t r0 = 0; r0 < t.nr; r0 += rpc) {
      const int32_t rows = (t.nr - r0 < rpc) ? t.nr - r0 : rpc;
      const Chunk c = make_chunk(t.base + r0 * t.stride, t.nc, t.stride, rows * t.nc);
      f32x16 st[2];
      chunk_scores<D>(kplane, c, qf, l32, half, st);
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const bool ok = qvalid && key_of(kt, r, half) < c.count;
          acc += ok ? __builtin_amdgcn_exp2f(st[kt][r] * io.scale_log2 - lse2) : 0.f;
        }
      }
    }
    acc = wave_sum(acc);
    if (lane == 0) red[wave] = acc;
    __syncthreads();
    if (tid == 0) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += red[w];
      out[v] = s;
    }
    __syncthreads();
  }
}


// bf16 scoring: one workgroup per (b, h, group of TPW query tiles of scale S),
// WPT waves per tile. Every query of a head scores against all keys of scales
// 1..S, so the tiles of a group share each K chunk: chunks stream HBM -> LDS
// (direct 16-byte loads, swizzled rows, double buffered) once per group.
// S^T = K Q^T on MFMA; each lane accumulates exp2(scale*log2e*s - lse*log2e) over
// its keys and its query; at the end of a block the wave sum goes to LDS, and a
// tile's score is the sum over its waves in order (deterministic). Blocks of a
// row are split over grid.y.
template <int D, int WPT, int TPW>
__global__ __launch_bounds__(WPT * TPW * 64) void pooled_scores_kernel(ScoreIO io) {
  constexpr int NW = WPT * TPW;
  constexpr int KC = 64, NT = NW * 64, U = D / 8, kRow = D * 2, kTile = KC * kRow;
  constexpr int kLoads = KC * U / NT;
  static_assert((KC * U) % NT == 0, "chunk must split evenly over the workgroup");
  // two K stages as separate arrays, so the compiler can tell that copies into
  // one stage never touch the stage being read
  __shared__ __attribute__((aligned(16))) char kstage0[kTile];
  __shared__ __attribute__((aligned(16))) char kstage1[kTile];
  extern __shared__ float red[];  // [NW][per] per-wave block sums

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const int32_t groups = (io.G_S + TPW - 1) / TPW;
  const int32_t bh = blockIdx.x / groups;
  const int32_t g0 = (blockIdx.x - bh * groups) * TPW;
  const GeoTable& G = io.G;
  const int S = io.S;
  const int32_t tw = G.Tw[S - 1];
  const int32_t g = g0 + wave / WPT;  // this wave's query tile
  const bool gvalid = g < io.G_S;
  const Tile qt = tile_at(G, S, gvalid ? g / tw : 0, gvalid ? g % tw : 0);
  const int32_t nq = qt.nr * qt.nc;
  const int32_t qslot = (wave % WPT) * kQPerWave + l32;
  const bool qvalid = gvalid && qslot < nq;
  const int32_t qi = qvalid ? qslot : 0;
  const int32_t qrow = (qt.base - G.C[S - 1]) + (qi / qt.nc) * qt.stride + (qi % qt.nc);
  const bf16_bits* qplane = static_cast<const bf16_bits*>(io.q) + (int64_t)bh * io.q_bh_stride;
  const char* kbytes = reinterpret_cast<const char*>(static_cast<const bf16_bits*>(io.k) + (int64_t)bh * io.k_bh_stride);
  QFragBF16<D> qf;
  qf.load(qplane + (int64_t)qrow * D, half);
  const float lse2 = io.lse[(int64_t)bh * G.h[S - 1] * G.w[S - 1] + qrow] * kLog2e;

  int ld_row[kLoads], ld_unit[kLoads];
#pragma unroll
  for (int j = 0; j < kLoads; ++j) {
    const int slot = (j * NW + wave) * 64 + lane;
    ld_row[j] = slot / U;
    ld_unit[j] = (slot % U) ^ (unit_swizzle(ld_row[j]) & (U - 1));
  }
  int k_off[2][D / 16];
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) {
    const int r = 32 * kt + l32;
#pragma unroll
    for (int s2 = 0; s2 < D / 16; ++s2) k_off[kt][s2] = r * kRow + 16 * ((2 * s2 + half) ^ (unit_swizzle(r) & (U - 1)));
  }
  auto issue = [&](const Chunk& c, auto stage_c) {
    constexpr int SG = decltype(stage_c)::value;
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int first = (j * NW + wave_s) * 64;
      const int r = ld_row[j];
      const uint32_t off = (uint32_t)(chunk_token(c, chunk_slot(r, c.count)) * D + 8 * ld_unit[j]) * 2u;
      dma16(kbytes + off, (SG == 0 ? kstage0 : kstage1) + first * 16);
    }
  };

  // this workgroup scores blocks [v0, v1)
  const int32_t per = io.per;
  const int32_t v0 = blockIdx.y * per;
  const int32_t v1 = (v0 + per < io.NB) ? v0 + per : io.NB;
  BlockWalker<KC> walk;
  walk.start(&G, v0, v1);
  Chunk c0;
  int32_t b0 = 0;
  bool last0 = false;
  bool have = walk.next(c0, b0, last0);
  if (have) issue(c0, std::integral_constant<int, 0>{});
  float psum = 0.f;

  auto step = [&](auto stage_c) -> bool {
    constexpr int SG = decltype(stage_c)::value;
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();
    Chunk cn;
    int32_t bn = 0;
    bool lastn = false;
    const bool have_n = walk.next(cn, bn, lastn);
    if (have_n) issue(cn, std::integral_constant<int, SG ^ 1>{});
    const char* kst = SG == 0 ? kstage0 : kstage1;
    f32x16 st[2];
    st[0] = zero16();
    st[1] = zero16();
#pragma unroll
    for (int s2 = 0; s2 < D / 16; ++s2) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(kst + k_off[kt][s2]);
        st[kt] = mfma_bf16(as_bf16x8(a), qf.f[s2], st[kt]);
      }
    }
    float part = 0.f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(st[kt][r], io.scale_log2, -lse2));
        part += key_of(kt, r, half) < c0.count ? p : 0.f;
      }
    }
    psum += qvalid ? part : 0.f;
    if (last0) {
      const float sw = wave_sum(psum);
      if (lane == 0) red[wave * per + (b0 - v0)] = sw;
      psum = 0.f;
    }
    c0 = cn;
    b0 = bn;
    last0 = lastn;
    return have_n;
  };
  while (have) {
    if (!step(std::integral_constant<int, 0>{})) break;
    if (!step(std::integral_constant<int, 1>{})) break;
  }
  __syncthreads();
  const int32_t nv = v1 - v0;
  for (int32_t i = tid; i < TPW * nv; i += NT) {
    const int t = i / nv;
    const int32_t v = v0 + (i - t * nv);
    if (g0 + t >= io.G_S) continue;
    float sc = 0.f;
#pragma unroll
    for (int w = 0; w < WPT; ++w) sc += red[(t * WPT + w) * per + (v - v0)];
    io.scores[((int64_t)bh * io.G_S + g0 + t) * io.NB + v] = sc;
  }
}

__global__ __launch_bounds__(64) void topk_kernel(const float* __restrict__ scores, int32_t nb,
                                                  int32_t topk, int32_t* __restrict__ out) {
  extern __shared__ float s_sc[];
  int32_t* s_sel = reinterpret_cast<int32_t*>(s_sc + nb);
  const int tid = threadIdx.x;
  const int64_t row = blockIdx.x;
  const float* sr = scores + row * nb;
  for (int32_t i = tid; i < nb; i += 64) s_sc[i] = sr[i];
  __syncthreads();
  for (int32_t v = tid; v < nb; v += 64) {
    const float x = s_sc[v];
    int32_t better = 0;
    for (int32_t u = 0; u < nb; ++u) {
      const float y = s_sc[u];
      better += (y > x) || (y == x && u < v);
    }
    s_sel[v] = better < topk;
  }
  __syncthreads();
  int32_t* orow = out + row * topk;
  for (int32_t v = tid; v < nb; v += 64) {
    if (s_sel[v]) {
      int32_t pos = 0;
      for (int32_t u = 0; u < v; ++u) pos += s_sel[u];
      if (pos < topk) orow[pos] = v;  // a strict total order selects exactly min(topk, nb)
    }
  }
  const int32_t nsel = topk < nb ? topk : nb;
  for (int32_t p = nsel + tid; p < topk; p += 64) orow[p] = -1;
}

namespace {
template <typename T, int D>
hipError_t launch_scores_f32(const ScoreIO& io, int nw, int32_t grid, hipStream_t stream) {
  switch (nw) {
    case 1: hipLaunchKernelGGL((pooled_scores_f32_kernel<T, D, 1>), dim3(grid), dim3(64), 0, stream, io); break;
    case 2: hipLaunchKernelGGL((pooled_scores_f32_kernel<T, D, 2>), dim3(grid), dim3(128), 0, stream, io); break;
    case 4: hipLaunchKernelGGL((pooled_scores_f32_kernel<T, D, 4>), dim3(grid), dim3(256), 0, stream, io); break;
    default: hipLaunchKernelGGL((pooled_scores_f32_kernel<T, D, 8>), dim3(grid), dim3(512), 0, stream, io); break;
  }
  return hipGetLastError();
}
// Query tiles of a head are grouped (TPW per workgroup) and the blocks of a row
// split over grid.y so that about 1024 workgroups run.
template <int D, int WPT, int TPW>
hipError_t launch_scores_bf16(const ScoreIO& io, int32_t BH, hipStream_t stream) {
  const int32_t grid = BH * ((io.G_S + TPW - 1) / TPW);
  int32_t splits = (1024 + grid - 1) / grid;
  if (splits > io.NB) splits = io.NB;
  if (splits < 1) splits = 1;
  const int32_t per = (io.NB + splits - 1) / splits;
  splits = (io.NB + per - 1) / per;
  ScoreIO io2 = io;
  io2.per = per;
  const size_t red = (size_t)WPT * TPW * per * sizeof(float);
  hipLaunchKernelGGL((pooled_scores_kernel<D, WPT, TPW>), dim3(grid, splits), dim3(WPT * TPW * 64), red, stream, io2);
  return hipGetLastError();
}

template <int D>
hipError_t launch_scores_bf16_d(const ScoreIO& io, int32_t BH, int wpt, hipStream_t stream) {
  switch (wpt) {
    case 1: return launch_scores_bf16<D, 1, 4>(io, BH, stream);
    case 2: return launch_scores_bf16<D, 2, 4>(io, BH, stream);
    case 4: return launch_scores_bf16<D, 4, 1>(io, BH, stream);
    default: return launch_scores_bf16<D, 8, 1>(io, BH, stream);
  }
}
}  // namespace

hipError_t launch_pooled_scores(const ScoreArgs& a, hipStream_t stream) {
  const GeoTable& G = *a.G;
  const int S = a.S;
  ScoreIO io;
  io.G = G;
  io.q = a.q;
  io.k = a.k;
  io.lse = a.lse;
  io.scores = a.scores;
  io.q_bh_stride = a.q_bh_stride;
  io.k_bh_stride = a.k_bh_stride;
  io.S = S;
  io.G_S = tiles_of(G, S);
  io.NB = G.NB[S];
  io.per = io.NB;
  io.scale_log2 = a.softmax_scale * kLog2e;
  const int32_t tile_q = G.eh[S - 1] * G.ew[S - 1];
  const int nw = tile_q <= 32 ? 1 : tile_q <= 64 ? 2 : tile_q <= 128 ? 4 : 8;
  const int32_t grid = a.BH * io.G_S;
  if (grid == 0) return hipSuccess;
  // per-wave block sums in LDS: at most 8 waves x NB floats
  if (a.bf16 && (size_t)8 * io.NB * sizeof(float) <= 32 * 1024)
    return a.d == 64 ? launch_scores_bf16_d<64>(io, a.BH, nw, stream) : launch_scores_bf16_d<128>(io, a.BH, nw, stream);
  if (a.bf16) return a.d == 64 ? launch_scores_f32<bf16_bits, 64>(io, nw, grid, stream)
                               : launch_scores_f32<bf16_bits, 128>(io, nw, grid, stream);
  return a.d == 64 ? launch_scores_f32<float, 64>(io, nw, grid, stream) : launch_scores_f32<float, 128>(io, nw, grid, stream);
}

hipError_t launch_topk(const float* scores, int32_t rows, int32_t nb, int32_t topk, int32_t* out,
                       hipStream_t stream) {
  if (rows == 0) return hipSuccess;
  const size_t shmem = (size_t)nb * 8;
  hipLaunchKernelGGL(topk_kernel, dim3(rows), dim3(64), shmem, stream, scores, nb, topk, out);
  return hipGetLastError();
}

}  // namespace sparvar

// Decision-scale block selection (Sec. 3.2: column-sum D and TopK).
//
// pooled_scores_kernel: one workgroup per (b, h, query tile g of scale S).
//   For every block v of scales 1..S it recomputes the S^T = K Q^T tile with
//   MFMA and adds P = exp(scale * s - lse) over the tile's queries and the
//   block's keys. Sums run in a fixed order (lane, shuffle tree, waves in
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
  float scale_log2;
};

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

template <typename T, int D, int NW>
__global__ __launch_bounds__(NW * 64) void pooled_scores_kernel(ScoreIO io) {
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
hipError_t launch_scores_t(const ScoreIO& io, int nw, int32_t grid, hipStream_t stream) {
  switch (nw) {
    case 1: hipLaunchKernelGGL((pooled_scores_kernel<T, D, 1>), dim3(grid), dim3(64), 0, stream, io); break;
    case 2: hipLaunchKernelGGL((pooled_scores_kernel<T, D, 2>), dim3(grid), dim3(128), 0, stream, io); break;
    case 4: hipLaunchKernelGGL((pooled_scores_kernel<T, D, 4>), dim3(grid), dim3(256), 0, stream, io); break;
    default: hipLaunchKernelGGL((pooled_scores_kernel<T, D, 8>), dim3(grid), dim3(512), 0, stream, io); break;
  }
  return hipGetLastError();
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
  io.scale_log2 = a.softmax_scale * kLog2e;
  const int32_t tile_q = G.eh[S - 1] * G.ew[S - 1];
  const int nw = tile_q <= 32 ? 1 : tile_q <= 64 ? 2 : tile_q <= 128 ? 4 : 8;
  const int32_t grid = a.BH * io.G_S;
  if (grid == 0) return hipSuccess;
  if (a.bf16) return a.d == 64 ? launch_scores_t<bf16_bits, 64>(io, nw, grid, stream)
                               : launch_scores_t<bf16_bits, 128>(io, nw, grid, stream);
  return a.d == 64 ? launch_scores_t<float, 64>(io, nw, grid, stream) : launch_scores_t<float, 128>(io, nw, grid, stream);
}

hipError_t launch_topk(const float* scores, int32_t rows, int32_t nb, int32_t topk, int32_t* out,
                       hipStream_t stream) {
  if (rows == 0) return hipSuccess;
  const size_t shmem = (size_t)nb * 8;
  hipLaunchKernelGGL(topk_kernel, dim3(rows), dim3(64), shmem, stream, scores, nb, topk, out);
  return hipGetLastError();
}

}  // namespace sparvar

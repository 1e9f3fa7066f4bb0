// Token-granular CS^4A (Sec. 3.2; appendix: Hardware-Efficient Sparse
// Computation, Cross-Scale Sparse Index Mapping) with 1-D query blocks of C
// contiguous queries of the flattened scale:
//   cs4a_colsum_kernel  column sums D[b,h,i,j] = sum over the queries q of block
//                       i of P[q,j], P = softmax(scale * Q_S K_<=S^T), from the
//                       decision pass's LSE;
//   cs4a_topk_kernel    inds^(S) = the top-K tokens of each row of D (ties to the
//                       lower token index), ascending, -1 padding;
//   cs4a_map_kernel     rows of scale k: sink tokens, then the tokens of source
//                       block phi(g) mapped by Decompose-Align-Project.
// The gather attention over those rows is the attention kernel's token source.
#include "device_common.h"
#include "launch.h"

namespace sparvar {

// ---------------------------------------------------------------- column sums
// One workgroup per (b, h, key range, query block): NW = C / 32 waves of 32
// queries. The key axis is cut into n_splits ranges of whole chunks; the column
// sums of different keys are independent, so the ranges need no reduction
// between workgroups and only add parallelism (a plane has few query blocks).
// Work items run (b, h)-major, then key range, then query block, so the
// workgroups that share a range's K on one XCD run together. Keys stream through
// LDS in 64-key chunks (direct loads, two stages in separate arrays). Each wave computes S = Q K^T with MFMA (A = Q rows from registers,
// B = K rows from LDS), so a lane's accumulator column is one key and its 16
// registers are 16 of the wave's queries: P = exp2(s * scale * log2e - LSE *
// log2e), the sum over the registers and one half-wave exchange give the key's
// sum over the wave's queries; the waves' sums are added in a fixed order.
struct ColsumIO {
  const void* q;
  const void* k;
  const float* lse;
  float* out;  // [planes, n_blocks, n_kv]
  int64_t q_bh_stride, k_bh_stride;
  int32_t n_q, n_kv, C, n_blocks, n_items, swizzle;
  int32_t n_splits, split_chunks;  // key ranges, chunks per range
  float scale_log2;
};

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void cs4a_colsum_kernel(ColsumIO io) {
  constexpr int KC = 64, NT = NW * 64, U = D / 8, kRow = D * 2, kTile = KC * kRow;
  constexpr int kLoads = KC * U / NT;
  static_assert((KC * U) % NT == 0, "chunk must split evenly over the workgroup");
  __shared__ __attribute__((aligned(16))) char ks0[kTile];
  __shared__ __attribute__((aligned(16))) char ks1[kTile];
  __shared__ float red[2][NW * KC];  // per-wave sums of a chunk, by chunk parity

  const int32_t item = swizzled_item(blockIdx.x, gridDim.x, io.swizzle);
  if (item >= io.n_items) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const int32_t per_bh = io.n_splits * io.n_blocks;
  const int32_t bh = item / per_bh;
  const int32_t split = (item - bh * per_bh) / io.n_blocks;
  const int32_t g = item - bh * per_bh - split * io.n_blocks;
  const int32_t q_end = (g + 1) * io.C < io.n_q ? (g + 1) * io.C : io.n_q;
  const int32_t q_first = g * io.C + wave * kQPerWave;

  const bf16_bits* qplane = static_cast<const bf16_bits*>(io.q) + (int64_t)bh * io.q_bh_stride;
  const char* kbytes = reinterpret_cast<const char*>(static_cast<const bf16_bits*>(io.k) + (int64_t)bh * io.k_bh_stride);
  const int32_t my_q = q_first + l32 < q_end ? q_first + l32 : g * io.C;
  QFragBF16<D> qf;
  qf.load(qplane + (int64_t)my_q * D, half);
  // LSE (exp2 domain) of the queries of this lane's accumulator registers; +inf
  // for query slots past the block, whose probabilities are then 0
  float lse2[16];
  const float* lrow = io.lse + (int64_t)bh * io.n_q;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int32_t qq = q_first + 8 * (r >> 2) + 4 * half + (r & 3);
    lse2[r] = qq < q_end ? lrow[qq] * kLog2e : INFINITY;
  }

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
  const int32_t n_kv = io.n_kv;
  auto issue = [&](int32_t p0, char* stg) {
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int first = (j * NW + wave_s) * 64;
      const int32_t tok = p0 + ld_row[j] < n_kv ? p0 + ld_row[j] : 0;
      dma16(kbytes + (uint32_t)(tok * D + 8 * ld_unit[j]) * 2u, stg + first * 16);
    }
  };
  float* orow = io.out + ((int64_t)bh * io.n_blocks + g) * n_kv;
  const int32_t all_chunks = (n_kv + KC - 1) / KC;
  const int32_t c_begin = split * io.split_chunks;
  const int32_t c_end = c_begin + io.split_chunks < all_chunks ? c_begin + io.split_chunks : all_chunks;
  // the sums of chunk c - 1 are reduced after the barrier of step c (their LDS
  // row alternates with the chunk's parity), so a step has one barrier
  auto reduce = [&](int32_t c) {
    if (tid < KC) {
      const float* rr = red[c & 1];
      float t = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) t += rr[w * KC + tid];
      const int32_t key = c * KC + tid;
      if (key < n_kv) orow[key] = t;
    }
  };
  if (c_begin < c_end) issue(c_begin * KC, ks0);
  auto step = [&](int32_t c, auto st_c) {
    constexpr int ST = decltype(st_c)::value;
    char* const stg = ST == 0 ? ks0 : ks1;
    char* const nstg = ST == 0 ? ks1 : ks0;
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();
    if (c + 1 < c_end) issue((c + 1) * KC, nstg);
    if (c > c_begin) reduce(c - 1);
    f32x16 st[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) st[kt] = zero16();
#pragma unroll
    for (int s2 = 0; s2 < D / 16; ++s2) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const u32x4 b = *reinterpret_cast<const u32x4*>(stg + k_off[kt][s2]);
        st[kt] = mfma_bf16(qf.f[s2], as_bf16x8(b), st[kt]);
      }
    }
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      float cs = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) cs += __builtin_amdgcn_exp2f(__builtin_fmaf(st[kt][r], io.scale_log2, -lse2[r]));
      cs = sum_halves(cs);
      if (half == 0) red[c & 1][wave * KC + 32 * kt + l32] = cs;
    }
  };
  for (int32_t c = c_begin; c < c_end; c += 2) {
    step(c, std::integral_constant<int, 0>{});
    if (c + 1 < c_end) step(c + 1, std::integral_constant<int, 1>{});
  }
  if (c_begin < c_end) {
    __syncthreads();
    reduce(c_end - 1);
  }
}

// ---------------------------------------------------------------- token top-K
// One workgroup per row. Radix select over order-preserving 32-bit keys (8 bits
// per pass, most significant first) finds the K-th largest value T and how many
// of the values equal to T are taken; then, in index order, a token is kept if
// its value is above T or it is among the first of those equal to T, and kept
// tokens are written ascending.
__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int kTopkThreads = 256;
constexpr int32_t kTopkStageMax = 8192;  // rows up to this length are staged in LDS (32 KB)

// STAGED: the row's order keys are read from global memory once into LDS
// (dynamic, n words); otherwise every pass reads them from global memory.
template <bool STAGED>
__global__ __launch_bounds__(kTopkThreads) void cs4a_topk_kernel(const float* __restrict__ in, int32_t n, int32_t K,
                                                                  int32_t* __restrict__ out) {
  constexpr int NT = kTopkThreads;
  extern __shared__ uint32_t staged[];
  __shared__ int32_t hist[256];
  __shared__ int32_t wt[NT / 64];
  __shared__ uint32_t sel_prefix;
  __shared__ int32_t sel_remaining;
  const int tid = threadIdx.x;
  const int64_t row = blockIdx.x;
  const float* x = in + row * n;
  int32_t* o = out + row * K;
  const int32_t nsel = K < n ? K : n;
  if constexpr (STAGED) {
    for (int32_t i = tid; i < n; i += NT) staged[i] = order_key(x[i]);
  }
  auto key = [&](int32_t i) -> uint32_t {
    if constexpr (STAGED) return staged[i];
    else return order_key(x[i]);
  };
  uint32_t prefix = 0, mask = 0;
  int32_t remaining = nsel;
  if (K < n) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      hist[tid] = 0;  // NT == 256 bins
      __syncthreads();
      for (int32_t i = tid; i < n; i += NT) {
        const uint32_t u = key(i);
        if ((u & mask) == prefix) atomicAdd(&hist[(u >> shift) & 255], 1);
      }
      __syncthreads();
      // thread t owns bin 255 - t: counts of the bins above it and of it
      const int32_t mine = hist[255 - tid];
      int32_t total;
      const int32_t above = block_excl_scan<NT>(mine, wt, total);
      if (above < remaining && above + mine >= remaining) {
        sel_prefix = (uint32_t)(255 - tid);
        sel_remaining = remaining - above;
      }
      __syncthreads();
      prefix |= sel_prefix << shift;
      mask |= 255u << shift;
      remaining = sel_remaining;
      __syncthreads();
    }
  }
  // prefix: the K-th largest key; remaining: how many keys equal to it to keep.
  // Thread t owns the contiguous indices [t seg, (t + 1) seg): one scan ranks the
  // keys equal to the threshold in index order, a second places the kept ones.
  const bool all = K >= n;
  const int32_t seg = (n + NT - 1) / NT;
  const int32_t i0 = tid * seg, i1 = i0 + seg < n ? i0 + seg : n;
  int32_t n_eq = 0;
  if (!all)
    for (int32_t i = i0; i < i1; ++i) n_eq += key(i) == prefix ? 1 : 0;
  int32_t eq_total;
  const int32_t eq_before = block_excl_scan<NT>(n_eq, wt, eq_total);
  int32_t n_keep = 0;
  {
    int32_t e = eq_before;
    for (int32_t i = i0; i < i1; ++i) {
      const uint32_t u = key(i);
      const bool eq = !all && u == prefix;
      n_keep += (all || u > prefix || (eq && e < remaining)) ? 1 : 0;
      e += eq ? 1 : 0;
    }
  }
  int32_t keep_total;
  int32_t pos = block_excl_scan<NT>(n_keep, wt, keep_total);
  {
    int32_t e = eq_before;
    for (int32_t i = i0; i < i1; ++i) {
      const uint32_t u = key(i);
      const bool eq = !all && u == prefix;
      if (all || u > prefix || (eq && e < remaining)) {
        if (pos < K) o[pos] = i;
        ++pos;
      }
      e += eq ? 1 : 0;
    }
  }
  for (int32_t p = nsel + tid; p < K; p += NT) o[p] = -1;
}

// ---------------------------------------------------------------- token mapping
// One workgroup per target row r = (b*H + h) * G_k + g: the sink tokens
// 0 .. n_sink - 1, then every listed token j of source row phi(g) mapped to step
// k (tokens that land among the sinks are dropped), kept in list order by a
// workgroup prefix count, then -1 up to the row stride M. Listed tokens
// ascending give ascending rows (the map is increasing in j).
struct MapTokIO {
  GeoTable G;
  const int32_t* inds;  // [planes, G_S, K]
  int32_t* tokens;      // [planes, G_k, M]
  int32_t S, k, K, M, G_S, G_k, n_sink_tok, rows;
};

constexpr int kMapThreads = 256;

__device__ __forceinline__ int32_t map_token(const GeoTable& G, int32_t j, int S, int k) {
  int l = 1;
  while (l < S && G.C[l] <= j) ++l;
  const int32_t delta = j - G.C[l - 1];
  const int lp = k - (S - l);
  const int32_t u = delta / G.w[l - 1], v = delta - (delta / G.w[l - 1]) * G.w[l - 1];
  const int32_t up = (int32_t)(((int64_t)u * G.h[lp - 1]) / G.h[l - 1]);
  const int32_t vp = (int32_t)(((int64_t)v * G.w[lp - 1]) / G.w[l - 1]);
  return G.C[lp - 1] + up * G.w[lp - 1] + vp;
}

__global__ __launch_bounds__(kMapThreads) void cs4a_map_kernel(MapTokIO io) {
  constexpr int NT = kMapThreads;
  __shared__ int32_t wt[NT / 64];
  // the geometry table in LDS: map_token indexes it per lane (scale search),
  // which on the kernel-argument copy is a chain of dependent global loads
  __shared__ GeoTable s_geo;
  const int32_t r = blockIdx.x;
  if (r >= io.rows) return;
  const int tid = threadIdx.x;
  {
    const int32_t* src = reinterpret_cast<const int32_t*>(&io.G);
    int32_t* dst = reinterpret_cast<int32_t*>(&s_geo);
    for (int i = tid; i < (int)(sizeof(GeoTable) / 4); i += NT) dst[i] = src[i];
  }
  __syncthreads();
  const int32_t bh = r / io.G_k;
  const int32_t g = r - bh * io.G_k;
  const int32_t src = (int32_t)(((int64_t)(2 * g + 1) * io.G_S) / (2 * (int64_t)io.G_k));
  const int32_t* in = io.inds + ((int64_t)bh * io.G_S + src) * io.K;
  int32_t* out = io.tokens + (int64_t)r * io.M;
  const int32_t ns = io.n_sink_tok;
  const int32_t n_le_S = io.G.C[io.S];
  for (int32_t i = tid; i < ns; i += NT) out[i] = i;
  int32_t pos = ns;
  for (int32_t base = 0; base < io.K; base += NT) {
    const int32_t i = base + tid;
    const int32_t j = i < io.K ? in[i] : -1;
    int32_t m = -1;
    if (j >= 0 && j < n_le_S) m = map_token(s_geo, j, io.S, io.k);
    const int32_t keep = m >= ns ? 1 : 0;
    int32_t total;
    const int32_t before = block_excl_scan<NT>(keep, wt, total);
    if (keep) out[pos + before] = m;
    pos += total;
  }
  for (int32_t i = pos + tid; i < io.M; i += NT) out[i] = -1;
}

// ---------------------------------------------------------------- launchers
namespace {

template <int D, int NW>
hipError_t launch_colsum_t(const ColsumIO& io, hipStream_t stream) {
  const int32_t grid = io.swizzle ? (io.n_items + 7) / 8 * 8 : io.n_items;
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL((cs4a_colsum_kernel<D, NW>), dim3(grid), dim3(NW * 64), 0, stream, io);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_cs4a_colsum(const Cs4aColsumArgs& a, hipStream_t stream) {
  ColsumIO io;
  io.q = a.q;
  io.k = a.k;
  io.lse = a.lse;
  io.out = a.out;
  io.q_bh_stride = a.q_bh_stride;
  io.k_bh_stride = a.k_bh_stride;
  io.n_q = a.n_q;
  io.n_kv = a.n_kv;
  io.C = a.C;
  io.n_blocks = (a.n_q + a.C - 1) / a.C;
  // key ranges: enough workgroups for about four per CU, at least 8 chunks each
  const int32_t all_chunks = (a.n_kv + 63) / 64;
  const int64_t base = (int64_t)a.BH * io.n_blocks;
  const int64_t want = base > 0 ? (4 * (int64_t)(a.num_cu > 0 ? a.num_cu : 256) + base - 1) / base : 1;
  int32_t splits = (int32_t)(want < all_chunks / 8 ? want : all_chunks / 8);
  splits = splits < 1 ? 1 : splits;
  io.split_chunks = (all_chunks + splits - 1) / splits;
  io.n_splits = all_chunks > 0 ? (all_chunks + io.split_chunks - 1) / io.split_chunks : 1;
  io.n_items = (int32_t)(base * io.n_splits);
  io.swizzle = a.swizzle;
  io.scale_log2 = a.softmax_scale * kLog2e;
  const int nw = a.C / kQPerWave;
#define SV_CS(DD, NN) \
  if (a.d == DD && nw == NN) return launch_colsum_t<DD, NN>(io, stream);
  SV_CS(128, 1) SV_CS(128, 2) SV_CS(128, 4) SV_CS(128, 8) SV_CS(64, 1) SV_CS(64, 2) SV_CS(64, 4) SV_CS(64, 8)
#undef SV_CS
  return hipErrorInvalidValue;
}

hipError_t launch_cs4a_topk(const float* in, int32_t rows, int32_t n, int32_t K, int32_t* out, hipStream_t stream) {
  if (rows == 0) return hipSuccess;
  if (n <= kTopkStageMax)
    hipLaunchKernelGGL(cs4a_topk_kernel<true>, dim3(rows), dim3(kTopkThreads), (size_t)n * 4, stream, in, n, K, out);
  else
    hipLaunchKernelGGL(cs4a_topk_kernel<false>, dim3(rows), dim3(kTopkThreads), 0, stream, in, n, K, out);
  return hipGetLastError();
}

hipError_t launch_cs4a_map(const GeoTable& G, int S, int k, int32_t BH, int32_t C, int32_t K, const int32_t* inds,
                           int32_t* tokens, int32_t M, hipStream_t stream) {
  MapTokIO io;
  io.G = G;
  io.inds = inds;
  io.tokens = tokens;
  io.S = S;
  io.k = k;
  io.K = K;
  io.M = M;
  io.G_S = (G.h[S - 1] * G.w[S - 1] + C - 1) / C;
  io.G_k = (G.h[k - 1] * G.w[k - 1] + C - 1) / C;
  io.n_sink_tok = G.C[G.n_sink];
  io.rows = BH * io.G_k;
  if (io.rows == 0) return hipSuccess;
  hipLaunchKernelGGL(cs4a_map_kernel, dim3(io.rows), dim3(kMapThreads), 0, stream, io);
  return hipGetLastError();
}

}  // namespace sparvar

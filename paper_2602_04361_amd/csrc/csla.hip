// Cross-Scale Local Sparse Attention (Sec. 3.3) in the paper's own form: the
// token-wise sink-plus-local mask reduced to 1-D blocks of B contiguous tokens
// on both axes (Eq. block_mask). csla_rows_kernel lists, for every query block
// of scale k, the key blocks that hold at least one kept (query, key) pair; the
// attention over those rows is the attention kernel's 1-D block source.
//
// A query (x, y) of scale k is aligned to historical scale h at
// (round(x H_h / H_k), round(y W_h / W_k)), halves rounded up, and keeps the keys
// of scale h within Chebyshev distance r_h = floor(w_h / 2) of that centre; the
// tokens of scales 1..n_sink are kept by every query.
#include "device_common.h"
#include "launch.h"

namespace sparvar {

struct CslaRowsIO {
  GeoTable G;
  int32_t win[kMaxScales];  // window size of historical scale h at index h - 1 (0: none)
  int32_t* rows_out;  // [n_rows, M]
  int32_t k, B, M, n_rows, n_kv_blocks;
};

// round(x * n_h / n_k) with halves rounded up (x >= 0).
__device__ __forceinline__ int32_t aligned_centre(int32_t x, int32_t n_k, int32_t n_h) {
  return (int32_t)(((int64_t)2 * x * n_h + n_k) / (2 * (int64_t)n_k));
}

// Sets the bits of the key blocks holding tokens [s, e] (s <= e).
__device__ __forceinline__ void mark_blocks(uint32_t* bits, int32_t s, int32_t e, int32_t B) {
  for (int32_t v = s / B; v <= e / B; ++v) atomicOr(&bits[v >> 5], 1u << (v & 31));
}

// One workgroup per query block u (queries [u B, min(u B + B, N_k)) of scale k).
// Work items are (windowed scale h, query row x of the block, row offset dx in
// [-r_h, r_h]); each marks the key blocks of one key row's column span. Query
// columns of one row are contiguous, and when W_h <= W_k their centres step by
// at most one, so the union of their windows on a key row is one span; a wider
// historical scale is walked query column by query column. The bitmask is then
// compacted into ascending ids and padded with -1 to the row stride M.
constexpr int kCslaThreads = 256;

__global__ __launch_bounds__(kCslaThreads) void csla_rows_kernel(CslaRowsIO io) {
  constexpr int NT = kCslaThreads;
  __shared__ uint32_t bits[kCslaMaxBlocks / 32];
  __shared__ int32_t wt[NT / 64];
  const int32_t u = blockIdx.x;
  const GeoTable& G = io.G;
  const int k = io.k;
  const int32_t B = io.B;
  const int32_t Hk = G.h[k - 1], Wk = G.w[k - 1];
  const int32_t Nk = Hk * Wk;
  const int32_t nwords = (io.n_kv_blocks + 31) >> 5;
  for (int32_t i = threadIdx.x; i < nwords; i += NT) bits[i] = 0u;
  __syncthreads();

  const int32_t q0 = u * B, q1 = (q0 + B < Nk ? q0 + B : Nk) - 1;  // first and last query
  const int32_t x0 = q0 / Wk, x1 = q1 / Wk;
  const int32_t nx = x1 - x0 + 1;
  const int32_t n_sink_tok = G.C[G.n_sink < k ? G.n_sink : k];
  if (threadIdx.x == 0 && n_sink_tok > 0) mark_blocks(bits, 0, n_sink_tok - 1, B);

  for (int h = 1; h <= k; ++h) {
    const int32_t w = io.win[h - 1];
    if (w <= 0) continue;
    const int32_t r = w / 2;
    const int32_t Hh = G.h[h - 1], Wh = G.w[h - 1];
    const int32_t base = G.C[h - 1];
    const int32_t span = 2 * r + 1;
    const int32_t items = nx * span;
    for (int32_t it = threadIdx.x; it < items; it += NT) {
      const int32_t xi = it / span;
      const int32_t x = x0 + xi;
      const int32_t kx = aligned_centre(x, Hk, Hh) + (it - xi * span) - r;  // key row
      if (kx < 0 || kx >= Hh) continue;
      const int32_t ya = x == x0 ? q0 - x0 * Wk : 0;
      const int32_t yb = x == x1 ? q1 - x1 * Wk : Wk - 1;
      const int32_t row = base + kx * Wh;
      if (Wh <= Wk) {
        int32_t lo = aligned_centre(ya, Wk, Wh) - r, hi = aligned_centre(yb, Wk, Wh) + r;
        lo = lo < 0 ? 0 : lo;
        hi = hi >= Wh ? Wh - 1 : hi;
        if (lo <= hi) mark_blocks(bits, row + lo, row + hi, B);
      } else {
        for (int32_t y = ya; y <= yb; ++y) {
          const int32_t c = aligned_centre(y, Wk, Wh);
          int32_t lo = c - r, hi = c + r;
          lo = lo < 0 ? 0 : lo;
          hi = hi >= Wh ? Wh - 1 : hi;
          if (lo <= hi) mark_blocks(bits, row + lo, row + hi, B);
        }
      }
    }
  }
  __syncthreads();

  // compaction: thread t owns words [t * per, (t + 1) * per)
  const int32_t per = (nwords + NT - 1) / NT;
  const int32_t w0 = threadIdx.x * per;
  int32_t cnt = 0;
  for (int32_t i = 0; i < per; ++i)
    if (w0 + i < nwords) cnt += __builtin_popcount(bits[w0 + i]);
  int32_t total;
  int32_t pos = block_excl_scan<NT>(cnt, wt, total);
  int32_t* out = io.rows_out + (int64_t)u * io.M;
  for (int32_t i = 0; i < per; ++i) {
    if (w0 + i >= nwords) break;
    uint32_t m = bits[w0 + i];
    while (m) {
      const int b = __builtin_ctz(m);
      out[pos++] = (w0 + i) * 32 + b;
      m &= m - 1;
    }
  }
  for (int32_t i = total + threadIdx.x; i < io.M; i += NT) out[i] = -1;
}

hipError_t launch_csla_rows(const GeoTable& G, int k, const int32_t* windows, int32_t B, int32_t* rows, int32_t M,
                            hipStream_t stream) {
  CslaRowsIO io;
  io.G = G;
  for (int i = 0; i < kMaxScales; ++i) io.win[i] = i < k ? windows[i] : 0;
  io.k = k;
  io.B = B;
  io.M = M;
  io.rows_out = rows;
  io.n_rows = (G.h[k - 1] * G.w[k - 1] + B - 1) / B;
  io.n_kv_blocks = (G.C[k] + B - 1) / B;
  if (io.n_rows == 0) return hipSuccess;
  hipLaunchKernelGGL(csla_rows_kernel, dim3(io.n_rows), dim3(kCslaThreads), 0, stream, io);
  return hipGetLastError();
}

}  // namespace sparvar

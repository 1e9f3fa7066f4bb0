// Integer kernels building the kept-block lists.
//
// local_blocks_kernel (one workgroup): row lengths -> prefix sum -> entries of
//   the sink + cross-scale local rows (block form of the CSLA window, Sec. 3.3).
// map_rows_kernel (one wave per CSR row, two passes): candidates are the local
//   row of the target tile plus the Decompose-Align-Project image of every
//   block selected for the source tile given by the Query Block Homography
//   (appendix, Cross-Scale Sparse Index Mapping). Pass 0 counts distinct
//   candidates; pass 1 writes each distinct candidate at its rank, giving an
//   ascending duplicate-free row.
// scan_schedule_kernel (one workgroup): row lengths -> row_ptr (clamped to the
//   index capacity) and, optionally, a longest-first stable row order.
#include "device_common.h"
#include "launch.h"

namespace sparvar {

constexpr int kScanThreads = 1024;

// In-place inclusive prefix sum of x[0..n) by one workgroup of kScanThreads.
// Values are clamped to `cap` after summation when cap >= 0.
__device__ void block_inclusive_scan(int32_t* x, int32_t n, int64_t cap, int32_t* lds) {
  const int tid = threadIdx.x;
  int64_t carry = 0;
  for (int32_t c0 = 0; c0 < n; c0 += kScanThreads) {
    const int32_t i = c0 + tid;
    int32_t v = i < n ? x[i] : 0;
    lds[tid] = v;
    __syncthreads();
    for (int off = 1; off < kScanThreads; off <<= 1) {
      const int32_t add = tid >= off ? lds[tid - off] : 0;
      __syncthreads();
      lds[tid] += add;
      __syncthreads();
    }
    int64_t s = carry + lds[tid];
    if (i < n) x[i] = (int32_t)((cap >= 0 && s > cap) ? cap : s);
    carry += lds[kScanThreads - 1];
    __syncthreads();
  }
}

__global__ __launch_bounds__(kScanThreads) void local_blocks_kernel(GeoTable G, int k, int32_t radius,
                                                                    int32_t dil, int32_t* row_ptr,
                                                                    int32_t* col_idx) {
  __shared__ int32_t lds[kScanThreads];
  const int32_t n = tiles_of(G, k);
  for (int32_t g = threadIdx.x; g < n; g += kScanThreads)
    row_ptr[g + 1] = local_row_len(local_row(G, k, radius, dil, g));
  if (threadIdx.x == 0) row_ptr[0] = 0;
  __syncthreads();
  block_inclusive_scan(row_ptr + 1, n, -1, lds);
  __syncthreads();
  for (int32_t g = threadIdx.x; g < n; g += kScanThreads) {
    const LocalRow r = local_row(G, k, radius, dil, g);
    const int32_t start = row_ptr[g], len = local_row_len(r);
    for (int32_t i = 0; i < len; ++i) col_idx[start + i] = local_row_entry(G, k, r, i);
  }
}

struct MapIO {
  GeoTable G;
  const int32_t* topk_idx;
  const int32_t* local_row_ptr;
  const int32_t* local_col;
  int32_t* row_ptr;
  int32_t* col_idx;
  int32_t S, k, G_k, G_S, topk, rows, max_cand;
};

constexpr int kMapWaves = 4;
constexpr int32_t kInvalid = 0x7fffffff;

template <int PASS>
__global__ __launch_bounds__(kMapWaves * 64) void map_rows_kernel(MapIO io) {
  extern __shared__ int32_t s_cand[];  // [kMapWaves][2][max_cand]: candidates, first occurrences
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t r = blockIdx.x * kMapWaves + wave;
  const bool active = r < io.rows;
  int32_t* cand = s_cand + wave * 2 * io.max_cand;
  int32_t* uniq = cand + io.max_cand;
  const GeoTable& G = io.G;
  const int32_t bh = r / io.G_k, g = r - bh * io.G_k;
  const int32_t twk = G.Tw[io.k - 1];
  const int32_t a = g / twk, c = g - a * twk;
  const int32_t gs = homography(a, G.Th[io.k - 1], G.Th[io.S - 1]) * G.Tw[io.S - 1] +
                     homography(c, twk, G.Tw[io.S - 1]);
  int32_t lp = 0, n_loc = 0;
  if (active) {
    lp = io.local_row_ptr[g];
    n_loc = io.local_row_ptr[g + 1] - lp;
    if (n_loc < 0) n_loc = 0;
    if (n_loc > io.max_cand - io.topk) n_loc = io.max_cand - io.topk;
  }
  const int32_t n = active ? n_loc + io.topk : 0;
  const int32_t* sel = io.topk_idx + ((int64_t)bh * io.G_S + gs) * io.topk;
  const int32_t nb_S = G.NB[io.S], nb_k = G.NB[io.k];

  for (int32_t i = lane; i < n; i += 64) {
    int32_t v;
    if (i < n_loc) {
      v = io.local_col[lp + i];
      if (v < 0 || v >= nb_k) v = kInvalid;
    } else {
      const int32_t s = sel[i - n_loc];
      v = (s >= 0 && s < nb_S) ? map_block(G, s, io.S, io.k) : kInvalid;
    }
    cand[i] = v;
  }
  __syncthreads();
  int32_t kept = 0;
  for (int32_t i = lane; i < n; i += 64) {
    const int32_t v = cand[i];
    bool keep = v != kInvalid;
    for (int32_t j = 0; j < i && keep; ++j) keep = cand[j] != v;
    uniq[i] = keep ? v : kInvalid;
    kept += keep;
  }
  if (PASS == 0) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) kept += __shfl_xor(kept, off, 64);
    if (active && lane == 0) io.row_ptr[r + 1] = kept;
    if (r == 0 && lane == 0) io.row_ptr[0] = 0;
    return;
  }
  __syncthreads();
  if (!active) return;
  const int32_t start = io.row_ptr[r], stop = io.row_ptr[r + 1];
  for (int32_t i = lane; i < n; i += 64) {
    const int32_t v = uniq[i];
    if (v == kInvalid) continue;
    int32_t rank = 0;  // distinct kept values below v
    for (int32_t j = 0; j < n; ++j) rank += uniq[j] < v;
    if (start + rank < stop) io.col_idx[start + rank] = v;
  }
}

// Longest-first stable order of rows given row_ptr. Counting sort by length
// (descending); ties keep row order: within a chunk of kScanThreads rows,
// waves are placed one after another, and inside a wave a row's rank among
// equal lengths comes from ballots.
__global__ __launch_bounds__(kScanThreads) void scan_schedule_kernel(int32_t* row_ptr, int32_t rows,
                                                                     int64_t capacity,
                                                                     int32_t* schedule,
                                                                     int32_t max_len) {
  __shared__ int32_t lds[kScanThreads];
  extern __shared__ int32_t s_hist[];  // [max_len + 1] start offsets, then running counts
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  block_inclusive_scan(row_ptr + 1, rows, capacity, lds);
  __syncthreads();
  if (!schedule) return;
  int32_t* hist = s_hist;
  for (int32_t i = tid; i <= max_len; i += kScanThreads) hist[i] = 0;
  __syncthreads();
  for (int32_t r = tid; r < rows; r += kScanThreads) {
    int32_t len = row_ptr[r + 1] - row_ptr[r];
    len = len > max_len ? max_len : len;
    atomicAdd(&hist[len], 1);
  }
  __syncthreads();
  if (tid == 0) {  // exclusive offsets, longest first
    int32_t run = 0;
    for (int32_t len = max_len; len >= 0; --len) {
      const int32_t h = hist[len];
      hist[len] = run;
      run += h;
    }
  }
  __syncthreads();
  int nbits = 1;
  while ((1 << nbits) <= max_len) ++nbits;
  for (int32_t c0 = 0; c0 < rows; c0 += kScanThreads) {
    const int32_t r = c0 + tid;
    const bool live = r < rows;
    int32_t len = live ? row_ptr[r + 1] - row_ptr[r] : 0;
    len = len > max_len ? max_len : len;
    uint64_t same = __ballot(live);
    for (int b = 0; b < nbits; ++b) {
      const uint64_t bit = __ballot(live && ((len >> b) & 1));
      same &= ((len >> b) & 1) ? bit : ~bit;
    }
    const uint64_t below = same & ((1ull << lane) - 1ull);
    const int rank = __popcll(below);
    const bool last = (same >> lane) == 1ull;  // highest lane with this length
    for (int w = 0; w < kScanThreads / 64; ++w) {
      if (wave == w && live) {
        schedule[hist[len] + rank] = r;
      }
      __syncthreads();
      if (wave == w && live && last) hist[len] += rank + 1;
      __syncthreads();
    }
  }
}

hipError_t launch_local_blocks(const GeoTable& G, int k, int32_t radius, int32_t dil, int32_t* row_ptr,
                               int32_t* col_idx, hipStream_t stream) {
  hipLaunchKernelGGL(local_blocks_kernel, dim3(1), dim3(kScanThreads), 0, stream, G, k, radius, dil, row_ptr,
                     col_idx);
  return hipGetLastError();
}

hipError_t launch_map_index(const GeoTable& G, int S, int k, int32_t BH, int32_t topk,
                            const int32_t* topk_idx, const int32_t* local_row_ptr,
                            const int32_t* local_col_idx, int32_t max_local, int32_t* row_ptr,
                            int32_t* col_idx, int64_t capacity, int32_t* schedule, hipStream_t stream) {
  MapIO io;
  io.G = G;
  io.topk_idx = topk_idx;
  io.local_row_ptr = local_row_ptr;
  io.local_col = local_col_idx;
  io.row_ptr = row_ptr;
  io.col_idx = col_idx;
  io.S = S;
  io.k = k;
  io.G_k = tiles_of(G, k);
  io.G_S = tiles_of(G, S);
  io.topk = topk;
  io.rows = BH * io.G_k;
  io.max_cand = max_local + topk;
  if (io.rows == 0) return hipSuccess;
  const int32_t grid = (io.rows + kMapWaves - 1) / kMapWaves;
  const size_t shmem = (size_t)kMapWaves * 2 * io.max_cand * sizeof(int32_t);
  hipLaunchKernelGGL(map_rows_kernel<0>, dim3(grid), dim3(kMapWaves * 64), shmem, stream, io);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int32_t max_len = io.max_cand;
  hipLaunchKernelGGL(scan_schedule_kernel, dim3(1), dim3(kScanThreads), (size_t)(max_len + 1) * sizeof(int32_t),
                     stream, row_ptr, io.rows, capacity, schedule, max_len);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(map_rows_kernel<1>, dim3(grid), dim3(kMapWaves * 64), shmem, stream, io);
  return hipGetLastError();
}

}  // namespace sparvar

// Integer kernels building the kept-block lists.
//
// local_blocks_kernel (one workgroup): row lengths -> prefix sum -> entries of
//   the sink + cross-scale local rows (block form of the CSLA window, Sec. 3.3).
// map_rows_kernel (one wave per row): candidates are the local row of the
//   target tile plus the Decompose-Align-Project image of every block selected
//   for the source tile given by the Query Block Homography (appendix,
//   Cross-Scale Sparse Index Mapping). Each distinct candidate is written at its
//   rank, so the row is ascending and duplicate-free; rows sit at a fixed stride
//   (the largest possible row) and end with -1 padding, so no prefix sum and a
//   single launch build them.
// schedule_kernel (optional): the rows' longest-first stable order.
#include <mutex>

#include "device_common.h"
#include "launch.h"
#include "sparvar.h"

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

// One target scale of a map launch; its rows are grid blocks [block0, block0 + ceil(rows / kMapWaves)).
struct MapStep {
  const int32_t* local_row_ptr;  // NULL: local rows come from (radius, dil)
  const int32_t* local_col;
  int32_t* row_ptr;
  int32_t* col_idx;
  int32_t* counts;  // [rows] row lengths
  int32_t* status;  // nullable: receives kStatusCut when a supplied local row is cut
  int32_t k, G_k, rows, max_cand, block0;
  int32_t cover;  // 0: point projection; else the largest cover box (candidates per selected block)
};

struct MapIO {
  GeoTable G;
  const int32_t* topk_idx;
  int32_t* schedule;  // nullable; single-step launches only
  int32_t S, G_S, topk, radius, dil, n_steps;
  MapStep st[kMaxMapSteps];
};

constexpr int kMapWaves = 4;
constexpr int32_t kInvalid = 0x7fffffff;
constexpr int32_t kStatusCut = SPARVAR_ERR_CAPACITY;

// One wave per row: candidates (local row + mapped selection) in LDS, first
// occurrences kept, each kept id written at its rank; the row occupies
// col_idx[r * max_cand, (r + 1) * max_cand) with -1 after its last id. The
// grid covers the rows of every step of the launch, step after step.
__global__ __launch_bounds__(kMapWaves * 64) void map_rows_kernel(MapIO io) {
  extern __shared__ int32_t s_cand[];  // [kMapWaves][2][max_cand of the step]
  // The geometry table in LDS: the per-lane decode of local and mapped blocks
  // indexes it per lane, which on the kernel-argument copy is a chain of
  // dependent global loads.
  __shared__ GeoTable s_geo;
  {
    const int32_t* src = reinterpret_cast<const int32_t*>(&io.G);
    int32_t* dst = reinterpret_cast<int32_t*>(&s_geo);
    for (int i = threadIdx.x; i < (int)(sizeof(GeoTable) / 4); i += kMapWaves * 64) dst[i] = src[i];
  }
  __syncthreads();
  int si = 0;
  while (si + 1 < io.n_steps && (int32_t)blockIdx.x >= io.st[si + 1].block0) ++si;
  const MapStep& ms = io.st[si];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t r = ((int32_t)blockIdx.x - ms.block0) * kMapWaves + wave;
  const bool active = r < ms.rows;
  const int k = ms.k;
  int32_t* cand = s_cand + wave * 2 * ms.max_cand;
  int32_t* uniq = cand + ms.max_cand;
  const GeoTable& G = s_geo;
  const int32_t bh = r / ms.G_k, g = r - bh * ms.G_k;
  const int32_t twk = G.Tw[k - 1];
  const int32_t a = g / twk, c = g - a * twk;
  const int32_t gs = homography(a, G.Th[k - 1], G.Th[io.S - 1]) * G.Tw[io.S - 1] +
                     homography(c, twk, G.Tw[io.S - 1]);
  int32_t lp = 0, n_loc = 0;
  const LocalRow lr = local_row(G, k, io.radius, io.dil, active ? g : 0);
  if (active) {
    if (ms.local_row_ptr) {
      lp = ms.local_row_ptr[g];
      n_loc = ms.local_row_ptr[g + 1] - lp;
    } else {
      n_loc = local_row_len(lr);
    }
    if (n_loc < 0) n_loc = 0;
    const int32_t loc_cap = ms.max_cand - io.topk * (ms.cover > 0 ? ms.cover : 1);
    if (n_loc > loc_cap) {
      // a supplied local row longer than the (radius, dilation) bound: cut to
      // the bound, and reported through the caller's status word
      n_loc = loc_cap;
      if (ms.status && lane == 0) *ms.status = kStatusCut;
    }
  }
  const int32_t per_sel = ms.cover > 0 ? ms.cover : 1;
  const int32_t n = active ? n_loc + io.topk * per_sel : 0;
  const int32_t* sel = io.topk_idx + ((int64_t)bh * io.G_S + gs) * io.topk;
  const int32_t nb_S = G.NB[io.S], nb_k = G.NB[k];
  for (int32_t i = lane; i < n; i += 64) {
    int32_t v;
    if (i < n_loc) {
      v = ms.local_row_ptr ? ms.local_col[lp + i] : local_row_entry(G, k, lr, i);
      if (v < 0 || v >= nb_k) v = kInvalid;
    } else if (ms.cover == 0) {
      const int32_t s = sel[i - n_loc];
      v = (s >= 0 && s < nb_S) ? map_block(G, s, io.S, k) : kInvalid;
    } else {
      // covering projection: slot j of selected block i / cover is the j-th tile
      // of its cover box, if the box has that many
      const int32_t q = (i - n_loc) / ms.cover, j = (i - n_loc) - q * ms.cover;
      const int32_t s = sel[q];
      v = kInvalid;
      if (s >= 0 && s < nb_S) {
        const CoverBox b = map_block_cover(G, s, io.S, k);
        if (j < cover_size(b)) v = cover_entry(b, j);
      }
    }
    cand[i] = v;
  }
  __syncthreads();
  // first occurrences (branch-free scan so the LDS reads pipeline)
  for (int32_t i = lane; i < n; i += 64) {
    const int32_t v = cand[i];
    int32_t dup = 0;
#pragma unroll 8
    for (int32_t j = 0; j < n; ++j) dup |= (j < i) & (cand[j] == v);
    uniq[i] = (dup || v == kInvalid) ? kInvalid : v;
  }
  __syncthreads();
  int32_t kept = 0;
  if (active) {
    int32_t* out = ms.col_idx + (int64_t)r * ms.max_cand;
    for (int32_t i = lane; i < n; i += 64) {
      const int32_t v = uniq[i];
      int32_t rank = 0;  // distinct kept values below v
#pragma unroll 8
      for (int32_t j = 0; j < n; ++j) rank += uniq[j] < v;
      if (v != kInvalid) {
        out[rank] = v;
        ++kept;
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) kept += __shfl_xor(kept, off, 64);
    for (int32_t i = kept + lane; i < ms.max_cand; i += 64) out[i] = -1;
    if (lane == 0) {
      ms.row_ptr[r] = r * ms.max_cand;
      if (r == ms.rows - 1) ms.row_ptr[ms.rows] = ms.rows * ms.max_cand;
      ms.counts[r] = kept;
    }
  }
}

// Longest-first stable order: rank of row r = rows that are longer, plus rows
// of equal length with a smaller index.
__global__ __launch_bounds__(kMapWaves * 64) void schedule_kernel(const int32_t* counts, int32_t rows,
                                                                  int32_t* schedule) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t r = blockIdx.x * kMapWaves + wave;
  if (r >= rows) return;
  const int32_t len = counts[r];
  int32_t before = 0;
  for (int32_t i = lane; i < rows; i += 64) {
    const int32_t li = counts[i];
    before += (li > len) || (li == len && i < r);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) before += __shfl_xor(before, off, 64);
  if (lane == 0) schedule[before] = r;
}

hipError_t launch_local_blocks(const GeoTable& G, int k, int32_t radius, int32_t dil, int32_t* row_ptr,
                               int32_t* col_idx, hipStream_t stream) {
  hipLaunchKernelGGL(local_blocks_kernel, dim3(1), dim3(kScanThreads), 0, stream, G, k, radius, dil, row_ptr,
                     col_idx);
  return hipGetLastError();
}

// Launch order of the block-sparse kernel's work items (query tiles, or groups
// of neighbouring tiles) at one step: inside each half of each XCD's share of
// the launch positions (the items the XCD-aware order gives that XCD), items go
// longest first (length = the rows' entries, summed over a group's tiles; ties
// keep the item order), so the workgroups that start last are the short ones.
struct OrderStep {
  int32_t* order;
  const int32_t* counts;
  int32_t n_items, per;                      // items, and positions per XCD share
  int32_t G_k, Th, Tw, gh, gw, ngc, n_groups;  // gh = 0: items are rows
};

struct OrderIO {
  OrderStep st[kMaxMapSteps];
};

constexpr int kOrderThreads = 256;
constexpr int kOrderMaxPer = 4096;

// Grid (8 XCD shares x 2 windows, steps); one workgroup ranks one window. The
// two windows of a share are ranked separately: the first half of the share's
// positions keeps the first half of its items (the XCD works on about as many
// (b, h) planes at a time as in natural order, so its L2 keeps their K/V). The
// split is rounded up to a multiple of 4.
__global__ __launch_bounds__(kOrderThreads) void order_kernel(OrderIO io) {
  __shared__ __attribute__((aligned(16))) int32_t key[kOrderMaxPer + 4];
  const OrderStep& s = io.st[blockIdx.y];
  const int32_t share = (int32_t)blockIdx.x >> 1, second = (int32_t)blockIdx.x & 1;
  const int32_t s_lo = share * s.per;
  const int32_t s_hi = s_lo + s.per < s.n_items ? s_lo + s.per : s.n_items;
  const int32_t n_share = s_hi - s_lo;
  if (n_share <= 0) return;
  const int32_t half = (n_share + 1) / 2;
  const int32_t w = ((half + 3) & ~3) < n_share ? ((half + 3) & ~3) : n_share;
  const int32_t lo = s_lo + (second ? w : 0), hi = second ? s_hi : s_lo + w;
  const int32_t n = hi - lo;
  if (n <= 0) return;
  const bool grouped = s.gh > 0;
  if (n > kOrderMaxPer) {  // beyond the LDS table: the natural order
    for (int32_t i = lo + (int32_t)threadIdx.x; i < hi; i += kOrderThreads) s.order[i] = grouped ? -2 - i : i;
    return;
  }
  for (int32_t i = threadIdx.x; i < n; i += kOrderThreads) {
    const int32_t it = lo + i;
    int32_t len;
    if (!grouped) {
      len = s.counts[it];
    } else {
      const int32_t bh = it / s.n_groups, gi = it - bh * s.n_groups;
      const int32_t A = gi / s.ngc, Cg = gi - A * s.ngc;
      len = 0;
      for (int t = 0; t < s.gh * s.gw; ++t) {
        const int32_t a = A * s.gh + t / s.gw, c = Cg * s.gw + t % s.gw;
        if (a < s.Th && c < s.Tw) len += s.counts[bh * s.G_k + a * s.Tw + c];
      }
    }
    key[i] = len;
  }
  if (threadIdx.x < 4) key[n + threadIdx.x] = INT32_MIN;  // padding: never ahead of a real length
  __syncthreads();
  const int4* key4 = reinterpret_cast<const int4*>(key);
  for (int32_t i = threadIdx.x; i < n; i += kOrderThreads) {
    const int32_t ki = key[i];
    int32_t rank = 0;
    for (int32_t j4 = 0; j4 < (n + 3) >> 2; ++j4) {
      const int4 kk = key4[j4];
      const int32_t j = j4 << 2;
      rank += (kk.x > ki) | ((kk.x == ki) & (j < i));
      rank += (kk.y > ki) | ((kk.y == ki) & (j + 1 < i));
      rank += (kk.z > ki) | ((kk.z == ki) & (j + 2 < i));
      rank += (kk.w > ki) | ((kk.w == ki) & (j + 3 < i));
    }
    s.order[lo + rank] = grouped ? -2 - (lo + i) : lo + i;
  }
}

hipError_t launch_map_order(const GeoTable& G, int32_t BH, int32_t topk, int n_steps, const MapStepArgs* steps,
                            int32_t* const* orders, int num_cu, int group_waves, hipStream_t stream) {
  OrderIO io;
  int used = 0;
  for (int i = 0; i < n_steps; ++i) {
    OrderStep& o = io.st[i];
    const int k = steps[i].k;
    const SparseForm f = sparse_form(G, k, BH, num_cu, group_waves);
    const int32_t rows = BH * tiles_of(G, k);
    o.order = orders ? orders[i] : nullptr;
    const int32_t per_sel = steps[i].cover > 0 ? steps[i].cover : 1;
    // row lengths: after the row slots, or where the step's counts pointer says
    o.counts = steps[i].counts ? steps[i].counts : steps[i].col_idx + (int64_t)rows * (steps[i].max_local + topk * per_sel);
    o.n_items = o.order ? f.n_items : 0;
    o.per = (o.n_items + 7) / 8;
    o.G_k = tiles_of(G, k);
    o.Th = G.Th[k - 1];
    o.Tw = G.Tw[k - 1];
    o.gh = f.gh;
    o.gw = f.gw;
    o.ngc = f.gw > 0 ? (G.Tw[k - 1] + f.gw - 1) / f.gw : 1;
    o.n_groups = f.gh > 0 ? ((G.Th[k - 1] + f.gh - 1) / f.gh) * o.ngc : 1;
    if (o.order) ++used;
  }
  if (used == 0) return hipSuccess;
  hipLaunchKernelGGL(order_kernel, dim3(16, n_steps), dim3(kOrderThreads), 0, stream, io);
  return hipGetLastError();
}

hipError_t launch_map_index(const GeoTable& G, int S, int32_t BH, int32_t topk, const int32_t* topk_idx,
                            int32_t radius, int32_t dil, int n_steps, const MapStepArgs* steps, int32_t* schedule,
                            hipStream_t stream) {
  MapIO io;
  io.G = G;
  io.topk_idx = topk_idx;
  io.schedule = n_steps == 1 ? schedule : nullptr;
  io.S = S;
  io.G_S = tiles_of(G, S);
  io.topk = topk;
  io.radius = radius;
  io.dil = dil;
  io.n_steps = n_steps;
  int32_t blocks = 0, max_cand = 1;
  for (int i = 0; i < n_steps; ++i) {
    MapStep& m = io.st[i];
    const MapStepArgs& a = steps[i];
    m.local_row_ptr = a.local_row_ptr;
    m.local_col = a.local_col_idx;
    m.row_ptr = a.row_ptr;
    m.col_idx = a.col_idx;
    m.k = a.k;
    m.G_k = tiles_of(G, a.k);
    m.rows = BH * m.G_k;
    m.cover = a.cover;
    m.max_cand = a.max_local + topk * (a.cover > 0 ? a.cover : 1);
    m.counts = a.counts ? a.counts : a.col_idx + (int64_t)m.rows * m.max_cand;  // default: past the last row slot
    m.status = a.status;
    m.block0 = blocks;
    blocks += (m.rows + kMapWaves - 1) / kMapWaves;
    max_cand = m.max_cand > max_cand ? m.max_cand : max_cand;
  }
  if (blocks == 0) return hipSuccess;
  const size_t shmem = (size_t)kMapWaves * 2 * max_cand * sizeof(int32_t);
  hipLaunchKernelGGL(map_rows_kernel, dim3(blocks), dim3(kMapWaves * 64), shmem, stream, io);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !io.schedule) return e;
  const int32_t grid = (io.st[0].rows + kMapWaves - 1) / kMapWaves;
  hipLaunchKernelGGL(schedule_kernel, dim3(grid), dim3(kMapWaves * 64), 0, stream, io.st[0].counts, io.st[0].rows,
                     schedule);
  return hipGetLastError();
}

// ---------------------------------------------------------------- fixed scratch
// Row lengths of the allocation-free mapping call: a fixed array in device
// memory, one copy per device, held until the process ends. In host code the
// array's name only stands for it; kernels get its device address, looked up
// once per device.
static __device__ __align__(256) int32_t scratch[kNoAllocMaxRows];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
int32_t* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t noalloc_row_lengths(int32_t** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = static_cast<int32_t*>(p);
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace sparvar

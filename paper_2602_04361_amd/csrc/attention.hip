// Dense and block-sparse cross-scale attention forward for gfx950.
//
// One kernel body serves both: a workgroup owns up to 32 * NW queries of one
// (batch, head) plane (a query tile of scale k for the sparse path, a run of
// rows for the dense path) and walks a sequence of key chunks of <= 64 keys
// (the kept blocks of its CSR row, or the whole cache). Per chunk and wave:
//   S^T = K Q^T      bf16 MFMA 32x32x16 (K rows gathered straight from HBM),
//   online softmax   exp2 domain, fp32, lane-local + one half-wave exchange,
//   O^T += V^T P^T   bf16 MFMA; V^T is staged in LDS, double buffered, by a
//                    register transpose of 8 keys x 8 dims per thread.
// The fp32 variant uses the 32x32x2 fp32 MFMA with the same accumulator
// layout and keeps V untransposed in LDS.
#include <type_traits>

#include "device_common.h"
#include "launch.h"

namespace sparvar {

struct AttnIO {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;
  int64_t q_bh_stride;   // elements between (b,h) planes of q
  int64_t kv_bh_stride;  // elements between (b,h) planes of k and v
  int32_t o_rows;        // rows of an output plane
  int32_t n_items;       // workgroups doing work
  int32_t swizzle;       // remap workgroups so consecutive items share an XCD
  float scale_log2;      // softmax_scale * log2(e)
};

// Queries of one workgroup: slot i in [q0, q1) is plane row
// qbase + (i / qnc) * qstride + i % qnc.
struct QuerySet {
  int32_t bh, qbase, qnc, qstride, q0, q1;
};

// ---------------------------------------------------------------- sources
struct DenseCursor {
  int32_t pos, n;
  __device__ __forceinline__ bool next(Chunk& c) {
    if (pos >= n) return false;
    const int32_t cnt = (n - pos < kChunk) ? n - pos : kChunk;
    c = run_chunk(pos, cnt);
    pos += cnt;
    return true;
  }
};

struct DenseSrc {
  int32_t n_q, n_kv, slabs, q_per_wg;
  __device__ __forceinline__ QuerySet queries(int32_t item) const {
    QuerySet s;
    s.bh = item / slabs;
    const int32_t slab = item - s.bh * slabs;
    s.qbase = 0;
    s.qnc = n_q;
    s.qstride = 0;
    s.q0 = slab * q_per_wg;
    s.q1 = (s.q0 + q_per_wg < n_q) ? s.q0 + q_per_wg : n_q;
    return s;
  }
  __device__ __forceinline__ DenseCursor cursor(int32_t) const { return DenseCursor{0, n_kv}; }
};

// Walks the kept blocks of one CSR row. Consecutive blocks whose tokens are
// contiguous in the cache (whole small scales, e.g. the sink scales) are packed
// into one chunk of up to 64 keys; blocks larger than 64 tokens are cut into
// row bands of at most 64 keys.
struct CsrCursor {
  const GeoTable* G;
  const int32_t* __restrict__ col;
  int32_t pos, end, nb;
  Tile big;
  int32_t big_row, big_rpc;

  __device__ __forceinline__ bool fetch(int32_t& v) {
    while (pos < end) {
      v = col[pos++];
      if (v >= 0 && v < nb) return true;
    }
    return false;
  }

  __device__ __forceinline__ bool next(Chunk& c) {
    if (big_row < big.nr) {
      const int32_t rows = (big.nr - big_row < big_rpc) ? big.nr - big_row : big_rpc;
      c = make_chunk(big.base + big_row * big.stride, big.nc, big.stride, rows * big.nc);
      big_row += rows;
      return true;
    }
    int32_t v;
    if (!fetch(v)) return false;
    const Tile t = block_tile(*G, v);
    const int32_t cnt = t.nr * t.nc;
    if (cnt > kChunk) {
      big = t;
      big_rpc = kChunk / t.nc;
      big_row = 0;
      return next(c);
    }
    if (!(t.nr == 1 || t.nc == t.stride)) {
      c = make_chunk(t.base, t.nc, t.stride, cnt);
      return true;
    }
    int32_t total = cnt;
    while (pos < end) {
      const int32_t v2 = col[pos];
      if (v2 < 0 || v2 >= nb) break;
      const Tile t2 = block_tile(*G, v2);
      const int32_t c2 = t2.nr * t2.nc;
      if (!(t2.nr == 1 || t2.nc == t2.stride) || t2.base != t.base + total || total + c2 > kChunk) break;
      total += c2;
      ++pos;
    }
    c = run_chunk(t.base, total);
    return true;
  }
};

struct SparseSrc {
  GeoTable G;
  const int32_t* row_ptr;
  const int32_t* col_idx;
  const int32_t* schedule;
  int32_t k, G_k, slabs, q_per_wg;

  __device__ __forceinline__ int32_t row_of(int32_t item) const {
    const int32_t r = item / slabs;
    return schedule ? schedule[r] : r;
  }
  __device__ __forceinline__ QuerySet queries(int32_t item) const {
    const int32_t r = row_of(item);
    const int32_t slab = item - (item / slabs) * slabs;
    QuerySet s;
    s.bh = r / G_k;
    const int32_t g = r - s.bh * G_k;
    const int32_t tw = G.Tw[k - 1];
    const Tile t = tile_at(G, k, g / tw, g % tw);
    s.qbase = t.base - G.C[k - 1];  // row inside the scale-k query plane
    s.qnc = t.nc;
    s.qstride = t.stride;
    const int32_t nq = t.nr * t.nc;
    s.q0 = slab * q_per_wg;
    s.q1 = (s.q0 + q_per_wg < nq) ? s.q0 + q_per_wg : nq;
    return s;
  }
  __device__ __forceinline__ CsrCursor cursor(int32_t item) const {
    const int32_t r = row_of(item);
    CsrCursor c;
    c.G = &G;
    c.col = col_idx;
    c.pos = row_ptr[r];
    c.end = row_ptr[r + 1];
    c.nb = G.NB[k];
    c.big.nr = 0;
    c.big_row = 0;
    c.big_rpc = 1;
    return c;
  }
};

__device__ __forceinline__ int32_t swizzled_item(int32_t wg, int32_t n_wg, int32_t on) {
  if (!on) return wg;
  // Workgroups are dealt round-robin to the 8 XCDs; give each XCD a contiguous
  // range of items so neighbouring query tiles share that XCD's L2.
  const int32_t per = n_wg >> 3;  // n_wg is a multiple of 8 when swizzling
  return (wg & 7) * per + (wg >> 3);
}

// ---------------------------------------------------------------- kernel
template <typename T, int D, int NW, class Src>
__global__ __launch_bounds__(NW * 64) void attn_fwd_kernel(AttnIO io, Src src) {
  constexpr bool kBF16 = std::is_same<T, bf16_bits>::value;
  constexpr int NT = NW * 64;
  // bf16: V^T[d][72] (64 key slots + pad; row = 144 B keeps 16-lane reads conflict free)
  // fp32: V[64][D + 8]
  constexpr int kVtRow = kChunk + 8;
  constexpr int kBufBytes = kBF16 ? D * kVtRow * 2 : kChunk * (D + 8) * 4;
  __shared__ __attribute__((aligned(16))) char smem[2 * kBufBytes];

  const int32_t item = swizzled_item(blockIdx.x, gridDim.x, io.swizzle);
  if (item >= io.n_items) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;

  const QuerySet qs = src.queries(item);
  const T* qplane = static_cast<const T*>(io.q) + (int64_t)qs.bh * io.q_bh_stride;
  const T* kplane = static_cast<const T*>(io.k) + (int64_t)qs.bh * io.kv_bh_stride;
  const T* vplane = static_cast<const T*>(io.v) + (int64_t)qs.bh * io.kv_bh_stride;

  const int32_t qslot = qs.q0 + wave * kQPerWave + l32;
  const bool qvalid = qslot < qs.q1;
  const int32_t qi = qvalid ? qslot : qs.q0;
  const int32_t qrow = qs.qbase + (qi / qs.qnc) * qs.qstride + (qi % qs.qnc);

  using QFrag = typename std::conditional<kBF16, QFragBF16<D>, QFragF32<D>>::type;
  QFrag qf;
  qf.load(qplane + (int64_t)qrow * D, half);

  f32x16 acc[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) acc[i] = zero16();
  float m_run = -INFINITY, l_run = 0.f;

  // ---- V staging (global -> registers -> LDS)
  constexpr int kGroups = kBF16 ? D : kChunk * D / 4;  // bf16: 8x8 blocks; fp32: 16-byte pieces
  constexpr int kGPT = (kGroups + NT - 1) / NT;
  u32x4 vreg[kBF16 ? kGPT * 8 : kGPT];

  auto stage_load = [&](const Chunk& c) {
#pragma unroll
    for (int j = 0; j < kGPT; ++j) {
      const int gi = tid + j * NT;
      if (gi < kGroups) {
        if constexpr (kBF16) {
          const int kg = gi & 7, dg = gi >> 3;
          const int k0 = 16 * (kg >> 1) + 4 * (kg & 1);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int key = k0 + (e < 4 ? e : e + 4);
            const int32_t tok = chunk_token(c, key < c.count ? key : 0);
            vreg[j * 8 + e] = ldg16(vplane + (int64_t)tok * D + 8 * dg);
          }
        } else {
          const int slot = gi / (D / 4), c4 = gi % (D / 4);
          const int32_t tok = chunk_token(c, slot < c.count ? slot : 0);
          vreg[j] = ldg16(vplane + (int64_t)tok * D + 4 * c4);
        }
      }
    }
  };

  auto stage_store = [&](int buf) {
    char* base = smem + buf * kBufBytes;
#pragma unroll
    for (int j = 0; j < kGPT; ++j) {
      const int gi = tid + j * NT;
      if (gi < kGroups) {
        if constexpr (kBF16) {
          const int kg = gi & 7, dg = gi >> 3;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
#pragma unroll
            for (int e2 = 0; e2 < 2; ++e2) {
              const uint32_t sel = e2 ? 0x07060302u : 0x05040100u;
              u32x4 w;
#pragma unroll
              for (int u = 0; u < 4; ++u)
                w[u] = __builtin_amdgcn_perm(vreg[j * 8 + 2 * u + 1][i], vreg[j * 8 + 2 * u][i], sel);
              const int d = 8 * dg + 2 * i + e2;
              *reinterpret_cast<u32x4*>(base + (d * kVtRow + 8 * kg) * 2) = w;
            }
          }
        } else {
          const int slot = gi / (D / 4), c4 = gi % (D / 4);
          *reinterpret_cast<u32x4*>(base + (slot * (D + 8) + 4 * c4) * 4) = vreg[j];
        }
      }
    }
  };

  auto cur = src.cursor(item);
  Chunk c;
  bool have = cur.next(c);
  if (have) {
    stage_load(c);
    stage_store(0);
  }
  __syncthreads();
  int buf = 0;

  while (have) {
    Chunk cn;
    const bool have_n = cur.next(cn);
    if (have_n) stage_load(cn);

    f32x16 st[2];
    chunk_scores<D>(kplane, c, qf, l32, half, st);

    // online softmax over this chunk (exp2 domain)
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float x = key_of(kt, r, half) < c.count ? st[kt][r] * io.scale_log2 : -INFINITY;
        st[kt][r] = x;
        mx = fmaxf(mx, x);
      }
    }
    mx = fmaxf(mx, xor32(mx));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    float ps = 0.f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(st[kt][r] - m_new);
        st[kt][r] = p;
        ps += p;
      }
    }
    l_run = l_run * alpha + ps;
    m_run = m_new;
#pragma unroll
    for (int i = 0; i < D / 32; ++i) acc[i] *= alpha;

    const char* vb = smem + buf * kBufBytes;
    if constexpr (kBF16) {
      bf16x8 pf[4];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        u32x4 w;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          w[u] = pack_bf16x2(st[ks >> 1][8 * (ks & 1) + 2 * u], st[ks >> 1][8 * (ks & 1) + 2 * u + 1]);
        pf[ks] = as_bf16x8(w);
      }
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const u32x4 a = *reinterpret_cast<const u32x4*>(vb + ((32 * dt + l32) * kVtRow + 16 * ks + 8 * half) * 2);
          acc[dt] = mfma_bf16(as_bf16x8(a), pf[ks], acc[dt]);
        }
      }
    } else {
      const float* vs = reinterpret_cast<const float*>(vb);
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = key_of(kt, r, half);
            acc[dt] = mfma_f32(vs[key * (D + 8) + 32 * dt + l32], st[kt][r], acc[dt]);
          }
        }
      }
    }

    if (have_n) stage_store(buf ^ 1);
    __syncthreads();
    c = cn;
    have = have_n;
    buf ^= 1;
  }

  // ---- epilogue
  const float l_tot = l_run + xor32(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (qvalid) {
    const int64_t orow = (int64_t)qs.bh * io.o_rows + qrow;
    T* op = static_cast<T*>(io.o) + orow * D;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int d = 32 * dt + 8 * j + 4 * half;
        if constexpr (kBF16) {
          uint2 w;
          w.x = pack_bf16x2(acc[dt][4 * j + 0] * inv, acc[dt][4 * j + 1] * inv);
          w.y = pack_bf16x2(acc[dt][4 * j + 2] * inv, acc[dt][4 * j + 3] * inv);
          *reinterpret_cast<uint2*>(op + d) = w;
        } else {
          float4 w = make_float4(acc[dt][4 * j + 0] * inv, acc[dt][4 * j + 1] * inv,
                                 acc[dt][4 * j + 2] * inv, acc[dt][4 * j + 3] * inv);
          *reinterpret_cast<float4*>(op + d) = w;
        }
      }
    }
    if (io.lse && half == 0) io.lse[orow] = l_tot > 0.f ? (m_run + __builtin_log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

// ---------------------------------------------------------------- launchers
namespace {

template <typename T, int D, int NW, class Src>
hipError_t launch_one(const AttnIO& io_in, const Src& src, hipStream_t stream) {
  AttnIO io = io_in;
  int32_t grid = io.n_items;
  if (io.swizzle) grid = (grid + 7) / 8 * 8;
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL((attn_fwd_kernel<T, D, NW, Src>), dim3(grid), dim3(NW * 64), 0, stream, io, src);
  return hipGetLastError();
}

template <typename T, int D, class Src>
hipError_t launch_nw(int nw, const AttnIO& io, const Src& src, hipStream_t stream) {
  switch (nw) {
    case 1: return launch_one<T, D, 1>(io, src, stream);
    case 2: return launch_one<T, D, 2>(io, src, stream);
    case 4: return launch_one<T, D, 4>(io, src, stream);
    default: return launch_one<T, D, 8>(io, src, stream);
  }
}

template <class Src>
hipError_t launch_typed(bool bf16, int d, int nw, const AttnIO& io, const Src& src, hipStream_t stream) {
  if (bf16) return d == 64 ? launch_nw<bf16_bits, 64>(nw, io, src, stream) : launch_nw<bf16_bits, 128>(nw, io, src, stream);
  return d == 64 ? launch_nw<float, 64>(nw, io, src, stream) : launch_nw<float, 128>(nw, io, src, stream);
}

int waves_for(int32_t queries) {
  if (queries <= 32) return 1;
  if (queries <= 64) return 2;
  if (queries <= 128) return 4;
  return 8;
}

}  // namespace

hipError_t launch_dense_attn(const DenseAttnArgs& a, hipStream_t stream) {
  const int nw = a.waves > 0 ? a.waves : 4;
  const int32_t qpw = nw * kQPerWave;
  DenseSrc src;
  src.n_q = a.n_q;
  src.n_kv = a.n_kv;
  src.q_per_wg = qpw;
  src.slabs = (a.n_q + qpw - 1) / qpw;
  AttnIO io;
  io.q = a.q;
  io.k = a.k;
  io.v = a.v;
  io.o = a.o;
  io.lse = a.lse;
  io.q_bh_stride = a.q_bh_stride;
  io.kv_bh_stride = a.kv_bh_stride;
  io.o_rows = a.n_q;
  io.n_items = a.BH * src.slabs;
  io.swizzle = a.swizzle;
  io.scale_log2 = a.softmax_scale * kLog2e;
  return launch_typed(a.bf16, a.d, nw, io, src, stream);
}

hipError_t launch_sparse_attn(const SparseAttnArgs& a, hipStream_t stream) {
  const GeoTable& G = *a.G;
  const int k = a.k;
  const int32_t tile_q = G.eh[k - 1] * G.ew[k - 1];
  const int nw = a.waves > 0 ? a.waves : waves_for(tile_q);
  const int32_t qpw = nw * kQPerWave;
  SparseSrc src;
  src.G = G;
  src.row_ptr = a.row_ptr;
  src.col_idx = a.col_idx;
  src.schedule = a.schedule;
  src.k = k;
  src.G_k = tiles_of(G, k);
  src.q_per_wg = qpw;
  src.slabs = (tile_q + qpw - 1) / qpw;
  AttnIO io;
  io.q = a.q;
  io.k = a.k_cache;
  io.v = a.v_cache;
  io.o = a.o;
  io.lse = a.lse;
  io.q_bh_stride = a.q_bh_stride;
  io.kv_bh_stride = a.kv_bh_stride;
  io.o_rows = G.h[k - 1] * G.w[k - 1];
  io.n_items = a.BH * src.G_k * src.slabs;
  io.swizzle = a.swizzle;
  io.scale_log2 = a.softmax_scale * kLog2e;
  return launch_typed(a.bf16, a.d, nw, io, src, stream);
}

}  // namespace sparvar

// Dense and block-sparse cross-scale attention forward for gfx950.
//
// A workgroup owns up to 32 * NW queries of one (batch, head) plane (a query
// tile of scale k for the sparse path, a slab of rows for the dense path) and
// walks a sequence of key chunks of at most KC keys: the kept blocks of its CSR
// row, or the whole cache. Per chunk and wave (32 queries):
//   S^T = K Q^T      bf16 MFMA 32x32x16, K from LDS, Q^T held in registers;
//   online softmax   exp2 domain, fp32; the running max is only moved (and the
//                    accumulator rescaled) when some row max grows by more than
//                    2^8, which keeps the result exact and skips most rescales;
//   O^T += V^T P^T   bf16 MFMA; V^T fragments come from the row-major V tile in
//                    LDS through the gfx950 transposing LDS read.
// K and V chunks are copied HBM -> LDS with 16-byte direct loads (no VGPR
// staging), XOR-swizzled by row so MFMA-fragment reads are bank-conflict free,
// and double buffered: the next chunk streams in while the current one is
// computed, with one workgroup barrier per chunk.
// The fp32 variant (parity-grade tiny cases) uses the 32x32x2 fp32 MFMA with the
// same accumulator layout and a simpler register-staged V.
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

// ---------------------------------------------------------------- key sources
template <int KC>
struct DenseCursor {
  int32_t pos, n;
  __device__ __forceinline__ bool next(Chunk& c) {
    if (pos >= n) return false;
    const int32_t cnt = (n - pos < KC) ? n - pos : KC;
    c = run_chunk(pos, cnt);
    pos += cnt;
    return true;
  }
};

template <int KC>
struct DenseSrc {
  static constexpr bool kSparse = false;
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
  __device__ __forceinline__ DenseCursor<KC> cursor(int32_t) const { return DenseCursor<KC>{0, n_kv}; }
};

// Walks the kept blocks of one CSR row as chunks of at most KC keys.
// Consecutive blocks whose tokens are contiguous in the cache (whole small
// scales such as the sink scales) are merged into one run and cut at KC;
// other tiles are emitted as bands of whole tile rows (or row pieces when a
// tile row is longer than KC).
template <int KC>
struct CsrCursor {
  const GeoTable* G;
  const int32_t* __restrict__ col;
  int32_t pos, end, nb;
  int32_t run_base, run_left;
  Tile t;
  int32_t t_row, t_col;

  __device__ __forceinline__ bool fetch(int32_t& v) {
    while (pos < end) {
      v = col[pos++];
      if (v >= 0 && v < nb) return true;
    }
    return false;
  }

  __device__ __forceinline__ static bool contiguous(const Tile& x) { return x.nr == 1 || x.nc == x.stride; }

  __device__ __forceinline__ bool next(Chunk& c) {
    for (;;) {
      if (run_left > 0) {
        const int32_t n = run_left < KC ? run_left : KC;
        c = run_chunk(run_base, n);
        run_base += n;
        run_left -= n;
        return true;
      }
      if (t_row < t.nr) {
        if (t.nc <= KC) {
          const int32_t rpc = KC / t.nc;
          const int32_t rows = (t.nr - t_row < rpc) ? t.nr - t_row : rpc;
          c = make_chunk(t.base + t_row * t.stride, t.nc, t.stride, rows * t.nc);
          t_row += rows;
        } else {
          const int32_t n = (t.nc - t_col < KC) ? t.nc - t_col : KC;
          c = run_chunk(t.base + t_row * t.stride + t_col, n);
          t_col += n;
          if (t_col >= t.nc) {
            t_col = 0;
            ++t_row;
          }
        }
        return true;
      }
      int32_t v;
      if (!fetch(v)) return false;
      const Tile x = block_tile(*G, v);
      if (contiguous(x)) {
        run_base = x.base;
        run_left = x.nr * x.nc;
        while (pos < end) {
          const int32_t v2 = col[pos];
          if (v2 < 0 || v2 >= nb) break;
          const Tile y = block_tile(*G, v2);
          if (!contiguous(y) || y.base != run_base + run_left) break;
          run_left += y.nr * y.nc;
          ++pos;
        }
      } else {
        t = x;
        t_row = 0;
        t_col = 0;
      }
    }
  }
};

// Chunk list of one CSR row, decoded in parallel by the whole workgroup into an
// LDS table: each refill decodes up to `group` blocks (one per thread), merges
// runs of contiguous blocks, splits everything into chunks of at most KC keys
// and writes 8-byte descriptors; the main loop then only reads descriptors.
// Descriptor: x = first token, y = stride << 16 | nc << 8 | count.
constexpr int kTableCap = 256;

template <int KC, int NT>
struct TableCursor {
  const GeoTable* G;
  const int32_t* __restrict__ col;
  int32_t pos, end, nb, group;
  int32_t tn, ti;
  uint2* tbl;    // [kTableCap]
  int4* info;    // [NT] decoded tiles of the current group (nr = 0: skipped id)
  int32_t* cnt;  // [NT + 1] chunk counts, then exclusive offsets

  __device__ __forceinline__ static bool contiguous(const int4& x) { return x.y == 1 || x.z == x.w; }

  __device__ static int32_t chunks_of(const int4& x, int32_t total_if_run) {
    if (contiguous(x)) return (total_if_run + KC - 1) / KC;
    if (x.z <= KC) {
      const int32_t rpc = KC / x.z;
      return (x.y + rpc - 1) / rpc;
    }
    return x.y * ((x.z + KC - 1) / KC);
  }

  __device__ void refill() {
    const int tid = threadIdx.x;
    __syncthreads();
    const int32_t nblk = (end - pos < group) ? end - pos : group;
    if (tid < nblk) {
      const int32_t v = col[pos + tid];
      int4 x = make_int4(0, 0, 1, 1);
      if (v >= 0 && v < nb) {
        const Tile t = block_tile(*G, v);
        x = make_int4(t.base, t.nr, t.nc, t.stride);
      }
      info[tid] = x;
    }
    __syncthreads();
    int32_t n = 0, run_total = 0;
    int4 x = make_int4(0, 0, 1, 1);
    if (tid < nblk) {
      x = info[tid];
      if (x.y > 0) {
        bool cont = false;
        if (contiguous(x) && tid > 0) {
          const int4 p = info[tid - 1];
          cont = p.y > 0 && contiguous(p) && p.x + p.y * p.z == x.x;
        }
        if (!cont) {
          run_total = x.y * x.z;
          if (contiguous(x)) {
            for (int32_t u = tid + 1; u < nblk; ++u) {
              const int4 y = info[u];
              if (y.y > 0 && contiguous(y) && y.x == x.x + run_total) run_total += y.y * y.z;
              else break;
            }
          }
          n = chunks_of(x, run_total);
        }
      }
    }
    // exclusive scan of n over the workgroup
    cnt[tid] = n;
    __syncthreads();
    for (int off = 1; off < NT; off <<= 1) {
      const int32_t add = tid >= off ? cnt[tid - off] : 0;
      __syncthreads();
      cnt[tid] += add;
      __syncthreads();
    }
    const int32_t incl = cnt[tid];
    const int32_t total = cnt[NT - 1];
    int32_t o = incl - n;
    if (n > 0) {
      if (contiguous(x)) {
        for (int32_t done = 0; done < run_total; done += KC, ++o) {
          const int32_t m = (run_total - done < KC) ? run_total - done : KC;
          tbl[o] = make_uint2((uint32_t)(x.x + done), (uint32_t)((kChunk << 16) | (kChunk << 8) | m));
        }
      } else if (x.z <= KC) {
        const int32_t rpc = KC / x.z;
        for (int32_t r0 = 0; r0 < x.y; r0 += rpc, ++o) {
          const int32_t rows = (x.y - r0 < rpc) ? x.y - r0 : rpc;
          tbl[o] = make_uint2((uint32_t)(x.x + r0 * x.w), (uint32_t)((x.w << 16) | (x.z << 8) | (rows * x.z)));
        }
      } else {
        for (int32_t r0 = 0; r0 < x.y; ++r0)
          for (int32_t c0 = 0; c0 < x.z; c0 += KC, ++o) {
            const int32_t m = (x.z - c0 < KC) ? x.z - c0 : KC;
            tbl[o] = make_uint2((uint32_t)(x.x + r0 * x.w + c0), (uint32_t)((kChunk << 16) | (kChunk << 8) | m));
          }
      }
    }
    __syncthreads();
    tn = __builtin_amdgcn_readfirstlane(total);
    ti = 0;
    pos += nblk;
  }

  __device__ __forceinline__ bool next(Chunk& c) {
    while (ti >= tn) {
      if (pos >= end) return false;
      refill();
    }
    const uint2 e = tbl[ti++];
    const uint32_t y = __builtin_amdgcn_readfirstlane(e.y);
    c.base = __builtin_amdgcn_readfirstlane(e.x);
    c.stride = (int32_t)(y >> 16);
    c.nc = (int32_t)((y >> 8) & 0xff);
    c.count = (int32_t)(y & 0xff);
    c.magic = kNcMagic[c.nc];
    return true;
  }
};

template <int KC>
struct SparseSrc {
  static constexpr bool kSparse = true;
  GeoTable G;
  const int32_t* row_ptr;
  const int32_t* col_idx;
  const int32_t* schedule;
  int32_t k, G_k, slabs, q_per_wg;
  int32_t max_chunks_per_block;  // bound used to size a table refill

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
  __device__ __forceinline__ CsrCursor<KC> cursor(int32_t item) const {
    const int32_t r = row_of(item);
    CsrCursor<KC> c;
    c.G = &G;
    c.col = col_idx;
    c.pos = row_ptr[r];
    c.end = row_ptr[r + 1];
    c.nb = G.NB[k];
    c.run_base = 0;
    c.run_left = 0;
    c.t.nr = 0;
    c.t_row = 0;
    c.t_col = 0;
    return c;
  }
  template <int NT>
  __device__ __forceinline__ TableCursor<KC, NT> table_cursor(int32_t item, uint2* tbl, int4* info,
                                                              int32_t* cnt) const {
    const int32_t r = row_of(item);
    TableCursor<KC, NT> c;
    c.G = &G;
    c.col = col_idx;
    c.pos = row_ptr[r];
    c.end = row_ptr[r + 1];
    c.nb = G.NB[k];
    const int32_t g = kTableCap / (max_chunks_per_block > 0 ? max_chunks_per_block : 1);
    c.group = g < NT ? (g > 0 ? g : 1) : NT;
    c.tn = 0;
    c.ti = 0;
    c.tbl = tbl;
    c.info = info;
    c.cnt = cnt;
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

// ---------------------------------------------------------------- bf16 kernel
template <int D, int NW, int KC, int NS, class Src>
__global__ __launch_bounds__(NW * 64) void attn_bf16_kernel(AttnIO io, Src src) {
  constexpr int NT = NW * 64;
  constexpr int U = D / 8;                 // 16-byte units per row
  constexpr int kRow = D * 2;              // bytes per K/V row
  constexpr int kTile = KC * kRow;         // bytes of one K (or V) chunk
  constexpr int kStage = 2 * kTile;        // K then V
  constexpr int kLoads = KC * U / NT;      // direct loads per thread per tensor
  static_assert(KC % 32 == 0 && (KC * U) % NT == 0, "chunk must split evenly over the workgroup");
  static_assert(NS >= 2 && NS <= 4, "pipeline depth");
  static_assert(2 * kLoads * (NS - 2) < 64, "vmcnt range");
  __shared__ __attribute__((aligned(16))) char smem[NS * kStage];
  // chunk table of the sparse path (unused by the dense path)
  constexpr int kTblBytes = Src::kSparse ? kTableCap * 8 + NT * 16 + (NT + 1) * 4 : 16;
  __shared__ __attribute__((aligned(16))) char tsmem[kTblBytes];

  const int32_t item = swizzled_item(blockIdx.x, gridDim.x, io.swizzle);
  if (item >= io.n_items) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;

  const QuerySet qs = src.queries(item);
  const bf16_bits* qplane = static_cast<const bf16_bits*>(io.q) + (int64_t)qs.bh * io.q_bh_stride;
  const bf16_bits* kplane = static_cast<const bf16_bits*>(io.k) + (int64_t)qs.bh * io.kv_bh_stride;
  const bf16_bits* vplane = static_cast<const bf16_bits*>(io.v) + (int64_t)qs.bh * io.kv_bh_stride;

  const int32_t qslot = qs.q0 + wave * kQPerWave + l32;
  const bool qvalid = qslot < qs.q1;
  const int32_t qi = qvalid ? qslot : qs.q0;
  const int32_t qrow = qs.qbase + (qi / qs.qnc) * qs.qstride + (qi % qs.qnc);
  QFragBF16<D> qf;
  qf.load(qplane + (int64_t)qrow * D, half);

  f32x16 acc[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) acc[i] = zero16();
  float m_run = -INFINITY, l_run = 0.f;

  // ---- lane-constant layout offsets (bytes inside one stage)
  // direct loads: wave instruction j covers LDS units [first_j, first_j + 64); lane i
  // fetches the logical unit the swizzle stores at unit first_j + i.
  int ld_row[kLoads], ld_unit[kLoads];
#pragma unroll
  for (int j = 0; j < kLoads; ++j) {
    const int slot = (j * NW + wave) * 64 + lane;
    ld_row[j] = slot / U;
    ld_unit[j] = (slot % U) ^ (unit_swizzle(ld_row[j]) & (U - 1));
  }
  // K fragment reads: key row r = 32 kt + l32, logical unit 2 s + half.
  int k_off[KC / 32][D / 16];
#pragma unroll
  for (int kt = 0; kt < KC / 32; ++kt) {
    const int r = 32 * kt + l32;
#pragma unroll
    for (int s2 = 0; s2 < D / 16; ++s2) k_off[kt][s2] = r * kRow + 16 * ((2 * s2 + half) ^ (unit_swizzle(r) & (U - 1)));
  }
  // V^T fragment reads through the transposing LDS read: within each group of 16
  // lanes, lane j receives element t of its 4-element result from the 8-byte
  // piece addressed by lane 4t + j/4 of the group, at position j % 4. Part p
  // covers keys 16 ks + 4 half + 8 p + (0..3); the swizzle term does not depend on ks.
  const int tr_g = lane >> 4, tr_t = (lane & 15) >> 2, tr_q = lane & 3;
  int v_off[2][D / 32];
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const int key = 4 * half + 8 * p + tr_t;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
      v_off[p][dt] = kTile + key * kRow +
                     16 * ((4 * dt + 2 * (tr_g & 1) + (tr_q >> 1)) ^ (unit_swizzle(key) & (U - 1))) + (tr_q & 1) * 8;
  }

  // Direct loads of a chunk into LDS stage S: 32-bit unsigned byte offsets from the
  // scalar plane bases, wave-uniform LDS destinations.
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const char* kbytes = reinterpret_cast<const char*>(kplane);
  const char* vbytes = reinterpret_cast<const char*>(vplane);
  auto issue = [&](const Chunk& c, auto stage_c) {
    constexpr int S = decltype(stage_c)::value;
    char* kb = smem + S * kStage;
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int first = (j * NW + wave_s) * 64;
      const int r = ld_row[j];
      const uint32_t off = (uint32_t)(chunk_token(c, r < c.count ? r : 0) * D + 8 * ld_unit[j]) * 2u;
      dma16(kbytes + off, kb + first * 16);
      dma16(vbytes + off, kb + kTile + first * 16);
    }
  };

  auto cur = [&]() {
    if constexpr (Src::kSparse) {
      return src.template table_cursor<NT>(item, reinterpret_cast<uint2*>(tsmem),
                                           reinterpret_cast<int4*>(tsmem + kTableCap * 8),
                                           reinterpret_cast<int32_t*>(tsmem + kTableCap * 8 + NT * 16));
    } else {
      return src.cursor(item);
    }
  }();
  // ring of chunk descriptors: ring[0] is being computed, ring[1..] are in flight
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;
  using S3 = std::integral_constant<int, 3>;
  Chunk ring[NS - 1];
  int ahead = 0;  // chunks issued beyond the one being computed
  bool have = cur.next(ring[0]);
  if (have) issue(ring[0], S0{});
  if constexpr (NS > 2) {
    if (have && cur.next(ring[1])) {
      issue(ring[1], S1{});
      ++ahead;
    }
  }
  if constexpr (NS > 3) {
    if (have && ahead == 1 && cur.next(ring[2])) {
      issue(ring[2], S2{});
      ++ahead;
    }
  }

  // One pipeline step on LDS stage S (a compile-time constant, so every LDS
  // address below is a lane-constant register plus an immediate).
  auto step = [&](auto stage_c) -> bool {
    constexpr int S = decltype(stage_c)::value;
    if (NS > 2 && ahead > 0) {
      if (ahead >= NS - 2) __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * kLoads * (NS - 2)));
      else __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    } else {
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    }
    __syncthreads();
    const Chunk c = ring[0];
    Chunk cn;
    const bool have_n = ahead == NS - 2 && cur.next(cn);
    if (have_n) issue(cn, std::integral_constant<int, (S + NS - 1) % NS>{});

    const char* kst = smem + S * kStage;

    // ---- S^T = K Q^T
    f32x16 st[KC / 32];
#pragma unroll
    for (int kt = 0; kt < KC / 32; ++kt) st[kt] = zero16();
#pragma unroll
    for (int s2 = 0; s2 < D / 16; ++s2) {
#pragma unroll
      for (int kt = 0; kt < KC / 32; ++kt) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(kst + k_off[kt][s2]);
        st[kt] = mfma_bf16(as_bf16x8(a), qf.f[s2], st[kt]);
      }
    }

    // ---- online softmax (exp2 domain)
    if (c.count < KC) {
#pragma unroll
      for (int kt = 0; kt < KC / 32; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (key_of(kt, r, half) >= c.count) st[kt][r] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < KC / 32; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, st[kt][r]);
    mx = max_halves(mx) * io.scale_log2;
    if (__builtin_amdgcn_ballot_w64(mx > m_run + 8.f)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int i = 0; i < D / 32; ++i) acc[i] *= alpha;
      m_run = m_new;
    }
    float ps = 0.f;
#pragma unroll
    for (int kt = 0; kt < KC / 32; ++kt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(st[kt][r], io.scale_log2, -m_run));
        st[kt][r] = p;
        ps += p;
      }
    }
    l_run += ps;

    // ---- O^T += V^T P^T
#pragma unroll
    for (int ks = 0; ks < KC / 16; ++ks) {
      u32x4 w;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        w[u] = pack_bf16x2(st[ks >> 1][8 * (ks & 1) + 2 * u], st[ks >> 1][8 * (ks & 1) + 2 * u + 1]);
      const bf16x8 pf = as_bf16x8(w);
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) {
        const i16x4 lo = lds_read_tr(kst + v_off[0][dt] + ks * 16 * kRow);
        const i16x4 hi = lds_read_tr(kst + v_off[1][dt] + ks * 16 * kRow);
        u32x4 av;
        av[0] = __builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 0, 1));
        av[1] = __builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 2, 3));
        av[2] = __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 0, 1));
        av[3] = __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 2, 3));
        acc[dt] = mfma_bf16(as_bf16x8(av), pf, acc[dt]);
      }
    }

    // ---- advance the ring
#pragma unroll
    for (int p = 0; p < NS - 2; ++p) ring[p] = ring[p + 1];
    if (have_n) ring[NS - 2] = cn;
    else --ahead;
    return ahead >= 0;
  };

  while (have) {
    if (!step(S0{})) break;
    if (!step(S1{})) break;
    if constexpr (NS > 2) {
      if (!step(S2{})) break;
    }
    if constexpr (NS > 3) {
      if (!step(S3{})) break;
    }
  }

  // ---- epilogue
  const float l_tot = sum_halves(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (qvalid) {
    const int64_t orow = (int64_t)qs.bh * io.o_rows + qrow;
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
    if (io.lse && half == 0) io.lse[orow] = l_tot > 0.f ? (m_run + __builtin_log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

// ---------------------------------------------------------------- fp32 kernel
// Parity-grade fp32 path: 32x32x2 fp32 MFMA, V staged through registers into a
// row-major LDS tile (double buffered), eager rescaling.
template <int D, int NW, class Src>
__global__ __launch_bounds__(NW * 64) void attn_f32_kernel(AttnIO io, Src src) {
  constexpr int NT = NW * 64;
  constexpr int KC = 64;
  constexpr int kBufBytes = KC * (D + 8) * 4;
  __shared__ __attribute__((aligned(16))) char smem[2 * kBufBytes];

  const int32_t item = swizzled_item(blockIdx.x, gridDim.x, io.swizzle);
  if (item >= io.n_items) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;

  const QuerySet qs = src.queries(item);
  const float* qplane = static_cast<const float*>(io.q) + (int64_t)qs.bh * io.q_bh_stride;
  const float* kplane = static_cast<const float*>(io.k) + (int64_t)qs.bh * io.kv_bh_stride;
  const float* vplane = static_cast<const float*>(io.v) + (int64_t)qs.bh * io.kv_bh_stride;
  const int32_t qslot = qs.q0 + wave * kQPerWave + l32;
  const bool qvalid = qslot < qs.q1;
  const int32_t qi = qvalid ? qslot : qs.q0;
  const int32_t qrow = qs.qbase + (qi / qs.qnc) * qs.qstride + (qi % qs.qnc);
  QFragF32<D> qf;
  qf.load(qplane + (int64_t)qrow * D, half);

  f32x16 acc[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) acc[i] = zero16();
  float m_run = -INFINITY, l_run = 0.f;

  constexpr int kGroups = KC * D / 4;
  constexpr int kGPT = (kGroups + NT - 1) / NT;
  u32x4 vreg[kGPT];
  auto stage_load = [&](const Chunk& c) {
#pragma unroll
    for (int j = 0; j < kGPT; ++j) {
      const int gi = tid + j * NT;
      if (gi < kGroups) {
        const int slot = gi / (D / 4), c4 = gi % (D / 4);
        const int32_t tok = chunk_token(c, slot < c.count ? slot : 0);
        vreg[j] = ldg16(vplane + (int64_t)tok * D + 4 * c4);
      }
    }
  };
  auto stage_store = [&](int buf) {
    char* base = smem + buf * kBufBytes;
#pragma unroll
    for (int j = 0; j < kGPT; ++j) {
      const int gi = tid + j * NT;
      if (gi < kGroups) {
        const int slot = gi / (D / 4), c4 = gi % (D / 4);
        *reinterpret_cast<u32x4*>(base + (slot * (D + 8) + 4 * c4) * 4) = vreg[j];
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
    const float* vs = reinterpret_cast<const float*>(smem + buf * kBufBytes);
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
    if (have_n) stage_store(buf ^ 1);
    __syncthreads();
    c = cn;
    have = have_n;
    buf ^= 1;
  }

  const float l_tot = l_run + xor32(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (qvalid) {
    const int64_t orow = (int64_t)qs.bh * io.o_rows + qrow;
    float* op = static_cast<float*>(io.o) + orow * D;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int d = 32 * dt + 8 * j + 4 * half;
        *reinterpret_cast<float4*>(op + d) = make_float4(acc[dt][4 * j + 0] * inv, acc[dt][4 * j + 1] * inv,
                                                         acc[dt][4 * j + 2] * inv, acc[dt][4 * j + 3] * inv);
      }
    }
    if (io.lse && half == 0) io.lse[orow] = l_tot > 0.f ? (m_run + __builtin_log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

// ---------------------------------------------------------------- launchers
namespace {

int32_t grid_for(const AttnIO& io) { return io.swizzle ? (io.n_items + 7) / 8 * 8 : io.n_items; }

template <int D, int NW, int KC, int NS, class Src>
hipError_t launch_bf16(const AttnIO& io, const Src& src, hipStream_t stream) {
  const int32_t grid = grid_for(io);
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL((attn_bf16_kernel<D, NW, KC, NS, Src>), dim3(grid), dim3(NW * 64), 0, stream, io, src);
  return hipGetLastError();
}

template <int D, int NW, class Src>
hipError_t launch_f32(const AttnIO& io, const Src& src, hipStream_t stream) {
  const int32_t grid = grid_for(io);
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL((attn_f32_kernel<D, NW, Src>), dim3(grid), dim3(NW * 64), 0, stream, io, src);
  return hipGetLastError();
}

// bf16 launch shapes (d, waves, keys per chunk, pipeline stages) that are instantiated.
#define SV_BF16_SHAPES(X)                                                                          \
  X(128, 1, 64, 2) X(128, 2, 32, 2) X(128, 2, 32, 3) X(128, 2, 32, 4) X(128, 2, 64, 2)            \
  X(128, 2, 64, 3) X(128, 4, 32, 2) X(128, 4, 32, 3) X(128, 4, 64, 2) X(128, 4, 64, 3)            \
  X(128, 8, 64, 2) X(64, 1, 64, 2) X(64, 2, 32, 2) X(64, 2, 32, 3) X(64, 2, 64, 2) X(64, 4, 64, 2) \
  X(64, 4, 64, 3) X(64, 8, 64, 2)

bool bf16_shape_exists(int d, int nw, int kc, int ns) {
#define SV_HAS(DD, NN, KK, SS) \
  if (d == DD && nw == NN && kc == KK && ns == SS) return true;
  SV_BF16_SHAPES(SV_HAS)
#undef SV_HAS
  return false;
}

// Dispatch on (dtype, d, waves, chunk, stages) for a source template family.
template <template <int> class SrcT, class Make>
hipError_t dispatch(bool bf16, int d, int nw, int kc, int ns, const AttnIO& io, Make make, hipStream_t stream) {
#define SV_BF16(DD, NN, KK, SS) \
  if (d == DD && nw == NN && kc == KK && ns == SS) return launch_bf16<DD, NN, KK, SS>(io, make(SrcT<KK>{}), stream);
#define SV_F32(DD, NN) \
  if (d == DD && nw == NN) return launch_f32<DD, NN>(io, make(SrcT<64>{}), stream);
  if (bf16) {
    SV_BF16_SHAPES(SV_BF16)
  } else {
    SV_F32(128, 1) SV_F32(128, 2) SV_F32(128, 4) SV_F32(128, 8) SV_F32(64, 1) SV_F32(64, 2) SV_F32(64, 4)
    SV_F32(64, 8)
  }
#undef SV_BF16
#undef SV_F32
  return hipErrorInvalidValue;
}

int waves_for(int32_t queries) {
  if (queries <= 32) return 1;
  if (queries <= 64) return 2;
  if (queries <= 128) return 4;
  return 8;
}

// (chunk, stages) for a bf16 launch: the requested shape if instantiated, else a
// fallback that is (64 keys, 2 stages).
void shape_for(int d, int nw, int want_kc, int want_ns, int* kc, int* ns) {
  if (bf16_shape_exists(d, nw, want_kc, want_ns)) {
    *kc = want_kc;
    *ns = want_ns;
  } else {
    *kc = 64;
    *ns = 2;
  }
}

}  // namespace

hipError_t launch_dense_attn(const DenseAttnArgs& a, hipStream_t stream) {
  // Widest workgroup (most queries sharing each K/V chunk) that still gives every
  // one of the 256 CUs a workgroup: 8 waves, else 4 waves, else 2 waves with
  // 32-key chunks.
  auto wgs = [&](int w) { return (int64_t)a.BH * ((a.n_q + 32 * w - 1) / (32 * w)); };
  int nw = a.waves;
  int want_kc = a.chunk;
  if (nw <= 0) {
    if (wgs(8) >= 256) nw = 8;
    else if (wgs(4) >= 256) nw = 4;
    else {
      nw = 2;
      want_kc = 32;
    }
  }
  int kc = 64, ns = 2;
  if (a.bf16) shape_for(a.d, nw, want_kc, a.stages, &kc, &ns);
  const int32_t qpw = nw * kQPerWave;
  AttnIO io;
  io.q = a.q;
  io.k = a.k;
  io.v = a.v;
  io.o = a.o;
  io.lse = a.lse;
  io.q_bh_stride = a.q_bh_stride;
  io.kv_bh_stride = a.kv_bh_stride;
  io.o_rows = a.n_q;
  const int32_t slabs = (a.n_q + qpw - 1) / qpw;
  io.n_items = a.BH * slabs;
  io.swizzle = a.swizzle;
  io.scale_log2 = a.softmax_scale * kLog2e;
  auto make = [&](auto proto) {
    auto s = proto;
    s.n_q = a.n_q;
    s.n_kv = a.n_kv;
    s.q_per_wg = qpw;
    s.slabs = slabs;
    return s;
  };
  return dispatch<DenseSrc>(a.bf16, a.d, nw, kc, ns, io, make, stream);
}

hipError_t launch_sparse_attn(const SparseAttnArgs& a, hipStream_t stream) {
  const GeoTable& G = *a.G;
  const int k = a.k;
  const int32_t tile_q = G.eh[k - 1] * G.ew[k - 1];
  const int nw = a.waves > 0 ? a.waves : waves_for(tile_q);
  int kc = 64, ns = 2;
  if (a.bf16) shape_for(a.d, nw, a.chunk, a.stages, &kc, &ns);
  const int32_t qpw = nw * kQPerWave;
  const int32_t slabs = (tile_q + qpw - 1) / qpw;
  const int32_t G_k = tiles_of(G, k);
  AttnIO io;
  io.q = a.q;
  io.k = a.k_cache;
  io.v = a.v_cache;
  io.o = a.o;
  io.lse = a.lse;
  io.q_bh_stride = a.q_bh_stride;
  io.kv_bh_stride = a.kv_bh_stride;
  io.o_rows = G.h[k - 1] * G.w[k - 1];
  io.n_items = a.BH * G_k * slabs;
  io.swizzle = a.swizzle;
  io.scale_log2 = a.softmax_scale * kLog2e;
  // largest chunk count of any block of scales 1..k (full and edge tiles)
  int32_t maxc = 1;
  for (int l = 1; l <= k; ++l) {
    const int32_t eh = G.eh[l - 1], ew = G.ew[l - 1];
    const int32_t rh[2] = {eh, G.h[l - 1] - (G.Th[l - 1] - 1) * eh};
    const int32_t rw[2] = {ew, G.w[l - 1] - (G.Tw[l - 1] - 1) * ew};
    for (int i = 0; i < 2; ++i)
      for (int j = 0; j < 2; ++j) {
        const int32_t nr = rh[i], nc = rw[j];
        int32_t c;
        if (nr == 1 || nc == G.w[l - 1]) c = (nr * nc + kc - 1) / kc;
        else if (nc <= kc) c = (nr + kc / nc - 1) / (kc / nc);
        else c = nr * ((nc + kc - 1) / kc);
        maxc = c > maxc ? c : maxc;
      }
  }
  auto make = [&](auto proto) {
    auto s = proto;
    s.max_chunks_per_block = maxc;
    s.G = G;
    s.row_ptr = a.row_ptr;
    s.col_idx = a.col_idx;
    s.schedule = a.schedule;
    s.k = k;
    s.G_k = G_k;
    s.q_per_wg = qpw;
    s.slabs = slabs;
    return s;
  };
  return dispatch<SparseSrc>(a.bf16, a.d, nw, kc, ns, io, make, stream);
}

}  // namespace sparvar

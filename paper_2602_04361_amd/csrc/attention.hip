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

#include "attn_chunk.h"
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
  // Epilogue (bf16 kernel): 0 writes the attention output A; 1 writes base - A
  // (base: [planes, o_rows, D], same layout as o); 2 writes up(base) + A, where
  // up() takes for output row (x, y) of an up_hk x up_wk grid the base row
  // (floor((2x+1) up_hs / (2 up_hk)), floor((2y+1) up_ws / (2 up_wk))) of an
  // up_hs x up_ws grid (base: [planes, up_hs * up_ws, D]).
  int32_t epi_mode = 0;
  const void* epi_base = nullptr;
  int32_t up_hs = 1, up_ws = 1, up_hk = 1, up_wk = 1;
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
  static constexpr bool kGrouped = false;
  static constexpr bool kTokens = false;
  int32_t n_q, n_kv, slabs, q_per_wg;
  template <int NT>
  static constexpr int table_bytes() { return 16; }
  __device__ __forceinline__ int tile_of(int) const { return 0; }
  __device__ __forceinline__ QuerySet queries(int32_t item, int wave) const {
    QuerySet s;
    s.bh = item / slabs;
    const int32_t slab = item - s.bh * slabs;
    s.qbase = 0;
    s.qnc = n_q;
    s.qstride = 0;
    const int32_t q0 = slab * q_per_wg;
    s.q1 = (q0 + q_per_wg < n_q) ? q0 + q_per_wg : n_q;
    s.q0 = q0 + wave * kQPerWave;
    return s;
  }
  __device__ __forceinline__ DenseCursor<KC> cursor(int32_t) const { return DenseCursor<KC>{0, n_kv}; }
};

// Key tokens listed one by one (token-granular rows): chunk slot r holds the
// token tokens[base + r].
template <int KC>
struct TokenCursor {
  int32_t pos, len, row_off;
  __device__ __forceinline__ bool next(Chunk& c) {
    if (pos >= len) return false;
    const int32_t cnt = (len - pos < KC) ? len - pos : KC;
    c = run_chunk(row_off + pos, cnt);
    pos += cnt;
    return true;
  }
};

// Rows of key tokens for 1-D query blocks of C contiguous queries (C = 32 NW):
// row r = (b*H + h) * n_blocks + g lists, for the queries [g C, g C + C) of the
// plane, ascending token ids in [0, n_kv) followed by padding (any id outside
// that range), at a fixed stride M.
template <int KC>
struct TokenSrc {
  static constexpr bool kSparse = false;
  static constexpr bool kGrouped = false;
  static constexpr bool kTokens = true;
  const int32_t* tokens;
  int32_t M, C, n_q, n_kv, n_blocks;
  template <int NT>
  static constexpr int table_bytes() { return 64; }
  __device__ __forceinline__ int tile_of(int) const { return 0; }
  __device__ __forceinline__ QuerySet queries(int32_t item, int wave) const {
    QuerySet s;
    s.bh = item / n_blocks;
    const int32_t g = item - s.bh * n_blocks;
    s.qbase = g * C;
    s.qnc = 1 << 30;  // contiguous rows
    s.qstride = 0;
    s.q0 = wave * kQPerWave;
    s.q1 = (n_q - g * C < C) ? n_q - g * C : C;
    return s;
  }
  // The row's token count (its ids up to the first padding entry), by the whole workgroup.
  template <int NT>
  __device__ __forceinline__ TokenCursor<KC> token_cursor(int32_t item, char* lds) const {
    const int32_t* row = tokens + (int64_t)item * M;
    int32_t cnt = 0;
    for (int32_t i = threadIdx.x; i < M; i += NT) {
      const int32_t t = row[i];
      cnt += (t >= 0 && t < n_kv) ? 1 : 0;
    }
    int32_t total;
    block_excl_scan<NT>(cnt, reinterpret_cast<int32_t*>(lds), total);
    TokenCursor<KC> c;
    c.pos = 0;
    c.len = __builtin_amdgcn_readfirstlane(total);
    c.row_off = item * M;
    return c;
  }
};

// Listed 1-D key blocks of B contiguous tokens: consecutive ids are merged into
// one run of the cache, cut into chunks of at most KC keys. The first kRunTable
// entries of the row are staged in LDS; later ones are read from global memory.
// The walk ends at the first id outside [0, nkb).
constexpr int kRunTable = 512;

template <int KC>
struct RunCursor {
  const int32_t* ids;  // LDS
  const int32_t* row;  // global
  int32_t pos, len, B, n_kv, nkb, run_base, run_left;
  __device__ __forceinline__ int32_t id_at(int32_t p) const {
    return __builtin_amdgcn_readfirstlane(p < kRunTable ? ids[p] : row[p]);
  }
  __device__ __forceinline__ bool next(Chunk& c) {
    if (run_left == 0) {
      if (pos >= len) return false;
      int32_t v = id_at(pos);
      if ((uint32_t)v >= (uint32_t)nkb) {
        pos = len;
        return false;
      }
      ++pos;
      run_base = v * B;
      while (pos < len && id_at(pos) == v + 1) {
        ++v;
        ++pos;
      }
      const int32_t end = v * B + B;
      run_left = (end < n_kv ? end : n_kv) - run_base;
    }
    const int32_t cnt = run_left < KC ? run_left : KC;
    c = run_chunk(run_base, cnt);
    run_base += cnt;
    run_left -= cnt;
    return true;
  }
};

// 1-D query blocks of C = 32 NW contiguous queries, each with a row of 1-D key
// blocks of C tokens (the CSLA block mask). Row g of rows, shared by every
// (b, h), lists ascending ids in [0, ceil(n_kv / C)) followed by padding (any id
// outside that range), at a fixed stride M.
template <int KC>
struct BlockRowSrc {
  static constexpr bool kSparse = false;
  static constexpr bool kGrouped = false;
  static constexpr bool kTokens = false;
  static constexpr bool kRuns = true;
  const int32_t* rows;
  int32_t M, C, n_q, n_kv, n_blocks;
  template <int NT>
  static constexpr int table_bytes() { return 4 * kRunTable; }
  __device__ __forceinline__ int tile_of(int) const { return 0; }
  __device__ __forceinline__ QuerySet queries(int32_t item, int wave) const {
    QuerySet s;
    s.bh = item / n_blocks;
    const int32_t g = item - s.bh * n_blocks;
    s.qbase = g * C;
    s.qnc = 1 << 30;  // contiguous rows
    s.qstride = 0;
    s.q0 = wave * kQPerWave;
    s.q1 = (n_q - g * C < C) ? n_q - g * C : C;
    return s;
  }
  // Stages the head of the row in LDS, by the whole workgroup.
  template <int NT>
  __device__ __forceinline__ RunCursor<KC> run_cursor(int32_t item, char* lds) const {
    const int32_t g = item % n_blocks;
    const int32_t* row = rows + (int64_t)g * M;
    int32_t* ids = reinterpret_cast<int32_t*>(lds);
    const int32_t lim = M < kRunTable ? M : kRunTable;
    for (int32_t i = threadIdx.x; i < lim; i += NT) ids[i] = row[i];
    __syncthreads();
    RunCursor<KC> c;
    c.ids = ids;
    c.row = row;
    c.pos = 0;
    c.len = M;
    c.B = C;
    c.n_kv = n_kv;
    c.nkb = (n_kv + C - 1) / C;
    c.run_base = 0;
    c.run_left = 0;
    return c;
  }
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

// Chunk list of a block list, decoded in parallel by the whole workgroup into an
// LDS table: each refill decodes up to `group` blocks (one per thread), merges
// runs of contiguous blocks that have the same tile mask, splits everything into
// chunks of at most KC keys and writes 8-byte descriptors plus the mask; the main
// loop then only reads descriptors. Descriptor: x = first token,
// y = stride << 16 | nc << 8 | count.
// Blocks supplies the ids: id(i) and mask(i) for i in the current segment
// [pos, end), and segment(pos, end), which moves to the next segment (false when
// there is none). Every thread of the workgroup calls next() in the same order.
constexpr int kTableCap = 256;

template <int NT>
struct TableLds {  // byte offsets inside the table region
  static constexpr int kTbl = 0;
  static constexpr int kTmask = kTbl + kTableCap * 8;
  static constexpr int kInfo = kTmask + kTableCap * 4;
  static constexpr int kImask = kInfo + NT * 16;
  static constexpr int kWt = kImask + NT * 4;
  static constexpr int kGeo = kWt + 16 * 4;  // LDS copy of the geometry table
  static constexpr int kBytes = kGeo + (int)((sizeof(GeoTable) + 15) / 16 * 16);
};

// Copies the geometry table from the kernel arguments into LDS, where the
// per-thread block decode of a refill reads it: indexed per lane, the
// kernel-argument copy is read with a chain of dependent global loads (one per
// scale searched), which made the first refill of every workgroup take
// microseconds. Visible after the next workgroup barrier.
template <int NT>
__device__ __forceinline__ const GeoTable* stage_geometry(const GeoTable& G, char* lds) {
  static_assert(sizeof(GeoTable) % 4 == 0, "geometry table is 32-bit words");
  constexpr int kWords = (int)(sizeof(GeoTable) / 4);
  const int32_t* s = reinterpret_cast<const int32_t*>(&G);
  int32_t* d = reinterpret_cast<int32_t*>(lds + TableLds<NT>::kGeo);
  for (int i = threadIdx.x; i < kWords; i += NT) d[i] = s[i];
  return reinterpret_cast<const GeoTable*>(lds + TableLds<NT>::kGeo);
}

template <int KC, int NT, class Blocks>
struct TableCursor {
  const GeoTable* G;
  Blocks blocks;
  int32_t nb, group;
  int32_t pos, end;  // entries of the current segment not yet decoded
  int32_t tn, ti;    // table fill and read position
  char* lds;         // TableLds<NT> region

  __device__ __forceinline__ static bool contiguous(const int4& x) { return x.y == 1 || x.z == x.w; }

  __device__ static int32_t chunks_of(const int4& x, int32_t total_if_run) {
    if (contiguous(x)) return (total_if_run + KC - 1) / KC;
    if (x.z <= KC) {
      const int32_t rpc = KC / x.z;
      return (x.y + rpc - 1) / rpc;
    }
    return x.y * ((x.z + KC - 1) / KC);
  }

  __device__ __forceinline__ void refill() {
    using L = TableLds<NT>;
    uint2* tbl = reinterpret_cast<uint2*>(lds + L::kTbl);
    uint32_t* tmask = reinterpret_cast<uint32_t*>(lds + L::kTmask);
    int4* info = reinterpret_cast<int4*>(lds + L::kInfo);
    uint32_t* imask = reinterpret_cast<uint32_t*>(lds + L::kImask);
    int32_t* wt = reinterpret_cast<int32_t*>(lds + L::kWt);
    const int tid = threadIdx.x;
    __syncthreads();
    const int32_t nblk = (end - pos < group) ? end - pos : group;
    if (tid < nblk) {
      const int32_t v = blocks.id(pos + tid);
      int4 x = make_int4(0, 0, 1, 1);
      if (v >= 0 && v < nb) {
        const Tile t = block_tile(*G, v);
        x = make_int4(t.base, t.nr, t.nc, t.stride);
      }
      info[tid] = x;
      imask[tid] = blocks.mask(pos + tid);
    }
    __syncthreads();
    int32_t n = 0, run_total = 0;
    int4 x = make_int4(0, 0, 1, 1);
    uint32_t m = 0;
    if (tid < nblk) {
      x = info[tid];
      m = imask[tid];
      if (x.y > 0) {
        bool cont = false;
        if (contiguous(x) && tid > 0) {
          const int4 p = info[tid - 1];
          cont = p.y > 0 && contiguous(p) && p.x + p.y * p.z == x.x && imask[tid - 1] == m;
        }
        if (!cont) {
          run_total = x.y * x.z;
          if (contiguous(x)) {
            for (int32_t u = tid + 1; u < nblk; ++u) {
              const int4 y = info[u];
              if (y.y > 0 && contiguous(y) && y.x == x.x + run_total && imask[u] == m) run_total += y.y * y.z;
              else break;
            }
          }
          n = chunks_of(x, run_total);
        }
      }
    }
    int32_t total;
    int32_t o = block_excl_scan<NT>(n, wt, total);
    if (n > 0) {
      if (contiguous(x)) {
        for (int32_t done = 0; done < run_total; done += KC, ++o) {
          const int32_t cnt = (run_total - done < KC) ? run_total - done : KC;
          tbl[o] = make_uint2((uint32_t)(x.x + done), (uint32_t)((kChunk << 16) | (kChunk << 8) | cnt));
          tmask[o] = m;
        }
      } else if (x.z <= KC) {
        const int32_t rpc = KC / x.z;
        for (int32_t r0 = 0; r0 < x.y; r0 += rpc, ++o) {
          const int32_t rows = (x.y - r0 < rpc) ? x.y - r0 : rpc;
          tbl[o] = make_uint2((uint32_t)(x.x + r0 * x.w), (uint32_t)((x.w << 16) | (x.z << 8) | (rows * x.z)));
          tmask[o] = m;
        }
      } else {
        for (int32_t r0 = 0; r0 < x.y; ++r0)
          for (int32_t c0 = 0; c0 < x.z; c0 += KC, ++o) {
            const int32_t cnt = (x.z - c0 < KC) ? x.z - c0 : KC;
            tbl[o] = make_uint2((uint32_t)(x.x + r0 * x.w + c0), (uint32_t)((kChunk << 16) | (kChunk << 8) | cnt));
            tmask[o] = m;
          }
      }
    }
    __syncthreads();
    tn = __builtin_amdgcn_readfirstlane(total);
    ti = 0;
    pos += nblk;
  }

  __device__ __forceinline__ bool next(Chunk& c) {
    using L = TableLds<NT>;
    while (ti >= tn) {
      if (pos >= end) {
        if (!blocks.segment(pos, end)) return false;
        continue;
      }
      refill();
    }
    const uint2 e = reinterpret_cast<const uint2*>(lds + L::kTbl)[ti];
    const uint32_t m = reinterpret_cast<const uint32_t*>(lds + L::kTmask)[ti];
    ++ti;
    const uint32_t y = __builtin_amdgcn_readfirstlane(e.y);
    c.base = __builtin_amdgcn_readfirstlane(e.x);
    c.stride = (int32_t)(y >> 16);
    c.nc = (int32_t)((y >> 8) & 0xff);
    c.count = (int32_t)(y & 0xff);
    c.magic = kNcMagic[c.nc];
    c.mask = __builtin_amdgcn_readfirstlane(m);
    return true;
  }
};

// Block list of one CSR row in global memory (a single segment, every tile).
struct CsrBlocks {
  const int32_t* __restrict__ col;
  int32_t p0, p1;
  bool done;
  __device__ __forceinline__ int32_t id(int32_t i) const { return col[i]; }
  __device__ __forceinline__ uint32_t mask(int32_t) const { return ~0u; }
  __device__ __forceinline__ bool segment(int32_t& pos, int32_t& end) {
    if (done) return false;
    done = true;
    pos = p0;
    end = p1;
    return true;
  }
};

template <int KC>
struct SparseSrc {
  static constexpr bool kSparse = true;
  static constexpr bool kGrouped = false;
  static constexpr bool kTokens = false;
  GeoTable G;
  const int32_t* row_ptr;
  const int32_t* col_idx;
  const int32_t* schedule;  // nullable launch order of rows; ignored when schedule[0] < 0 (an order of groups)
  int32_t k, G_k, slabs, q_per_wg, n_rows;
  int32_t max_chunks_per_block;  // bound used to size a table refill

  template <int NT>
  static constexpr int table_bytes() { return TableLds<NT>::kBytes; }
  __device__ __forceinline__ int tile_of(int) const { return 0; }
  __device__ __forceinline__ int32_t row_of(int32_t item) const {
    const int32_t r = item / slabs;
    if (!schedule || schedule[0] < 0) return r;
    const int32_t v = schedule[r];
    return (v >= 0 && v < n_rows) ? v : r;
  }
  __device__ __forceinline__ QuerySet queries(int32_t item, int wave) const {
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
    const int32_t q0 = slab * q_per_wg;
    s.q1 = (q0 + q_per_wg < nq) ? q0 + q_per_wg : nq;
    s.q0 = q0 + wave * kQPerWave;
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
  __device__ __forceinline__ TableCursor<KC, NT, CsrBlocks> table_cursor(int32_t item, char* lds) const {
    const int32_t r = row_of(item);
    TableCursor<KC, NT, CsrBlocks> c;
    c.G = stage_geometry<NT>(G, lds);  // the first refill starts with a barrier
    c.blocks.col = col_idx;
    c.blocks.p0 = row_ptr[r];
    c.blocks.p1 = row_ptr[r + 1];
    c.blocks.done = false;
    c.nb = G.NB[k];
    const int32_t g = kTableCap / (max_chunks_per_block > 0 ? max_chunks_per_block : 1);
    c.group = g < NT ? (g > 0 ? g : 1) : NT;
    c.pos = 0;
    c.end = 0;
    c.tn = 0;
    c.ti = 0;
    c.lds = lds;
    return c;
  }
};

// ------------------------------------------------------- grouped query tiles
// A workgroup serves a group of T neighbouring query tiles of scale k (T = 2,
// 4 or 8; gh x gw tiles) and walks the union of their CSR rows once: every
// staged chunk carries the mask of the group's tiles whose row lists the block,
// and the waves of the other tiles skip it. Each tile still attends to exactly
// its own blocks; the union only lets tiles share each HBM -> LDS copy.
//
// Union of sorted rows, built in parallel (thread = row entry): each row's
// valid ids are compacted; an entry is the owner of its id when no lower row and
// no earlier entry of its own row holds the id; its place in the union is the
// number of owners with smaller ids, found by a binary search in every other
// row; its mask has a bit for every row holding the id. Rows longer than
// NT / T entries are served tile by tile instead, in windows of NT entries.
template <int NT>
struct GroupLds {
  static constexpr int kIds = 0;
  static constexpr int kOwnp = kIds + NT * 4;
  static constexpr int kUid = kOwnp + NT * 4;
  static constexpr int kUmask = kUid + NT * 4;
  static constexpr int kRowP = kUmask + NT * 4;
  static constexpr int kRowN = kRowP + 8 * 4;
  static constexpr int kRowC = kRowN + 8 * 4;
  static constexpr int kWt = kRowC + 8 * 4;
  static constexpr int kBytes = kWt + 16 * 4;
};

template <int NT>
struct GroupBlocks {
  static constexpr int kLgNT = NT == 512 ? 9 : NT == 256 ? 8 : NT == 128 ? 7 : 6;
  const int32_t* __restrict__ col;
  int32_t nb, T, lgT;
  bool by_tile, started;
  int32_t seg_t, seg_off;  // next window of the tile-by-tile mode
  char* lds;               // GroupLds<NT> region

  __device__ __forceinline__ int32_t* arr(int off) const { return reinterpret_cast<int32_t*>(lds + off); }
  __device__ __forceinline__ int32_t id(int32_t i) const { return arr(GroupLds<NT>::kUid)[i]; }
  __device__ __forceinline__ uint32_t mask(int32_t i) const {
    return (uint32_t)arr(GroupLds<NT>::kUmask)[i];
  }

  __device__ __forceinline__ int32_t build_union() {
    using L = GroupLds<NT>;
    int32_t* ids = arr(L::kIds);
    int32_t* ownp = arr(L::kOwnp);
    const int32_t* rowp = arr(L::kRowP);
    const int32_t* rown = arr(L::kRowN);
    int32_t* rowc = arr(L::kRowC);
    int32_t* wt = arr(L::kWt);
    const int tid = threadIdx.x;
    const int lgRC = kLgNT - lgT;
    const int32_t RC = 1 << lgRC;
    const int t = tid >> lgRC;
    const int32_t i = tid & (RC - 1);
    int32_t raw = -1;
    if (i < rown[t]) raw = col[rowp[t] + i];
    const bool valid = raw >= 0 && raw < nb;
    int32_t total;
    const int32_t e = block_excl_scan<NT>(valid ? 1 : 0, wt, total);
    ownp[tid] = e;
    __syncthreads();
    const int32_t row0 = ownp[t * RC];
    if (valid) ids[t * RC + (e - row0)] = raw;
    if (i == 0) rowc[t] = ((t + 1) * RC < NT ? ownp[(t + 1) * RC] : total) - row0;
    __syncthreads();

    const int32_t nt = rowc[t];
    int32_t v = 0;
    uint32_t m = 0;
    bool own = false;
    if (i < nt) {
      v = ids[t * RC + i];
      own = !(i > 0 && ids[t * RC + i - 1] == v);
      m = 1u << t;
    }
    int32_t lb[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      lb[u] = 0;
      if (u < T && i < nt) {
        if (u == t) {
          lb[u] = i;
        } else {
          const int32_t* r = ids + u * RC;
          const int32_t n = rowc[u];
          int32_t lo = 0, hi = n;
          while (lo < hi) {
            const int32_t mid = (lo + hi) >> 1;
            if (r[mid] < v) lo = mid + 1;
            else hi = mid;
          }
          lb[u] = lo;
          if (lo < n && r[lo] == v) {
            m |= 1u << u;
            if (u < t) own = false;
          }
        }
      }
    }
    int32_t owners;
    const int32_t e2 = block_excl_scan<NT>(own ? 1 : 0, wt, owners);
    ownp[tid] = e2;
    __syncthreads();
    if (own) {
      int32_t rank = 0;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (u < T) {
          const int32_t base = ownp[u * RC];
          const int32_t j = lb[u];
          const int32_t at = j < RC ? ownp[u * RC + j] : ((u + 1) * RC < NT ? ownp[(u + 1) * RC] : owners);
          rank += at - base;
        }
      }
      arr(L::kUid)[rank] = v;
      arr(L::kUmask)[rank] = (int32_t)m;
    }
    __syncthreads();
    return __builtin_amdgcn_readfirstlane(owners);
  }

  __device__ __forceinline__ int32_t build_window() {
    using L = GroupLds<NT>;
    const int tid = threadIdx.x;
    const int32_t n = arr(L::kRowN)[seg_t] - seg_off;
    int32_t raw = -1;
    if (tid < n) raw = col[arr(L::kRowP)[seg_t] + seg_off + tid];
    const bool valid = raw >= 0 && raw < nb;
    int32_t total;
    const int32_t e = block_excl_scan<NT>(valid ? 1 : 0, arr(L::kWt), total);
    if (valid) {
      arr(L::kUid)[e] = raw;
      arr(L::kUmask)[e] = 1 << seg_t;
    }
    __syncthreads();
    return __builtin_amdgcn_readfirstlane(total);
  }

  __device__ __forceinline__ bool segment(int32_t& pos, int32_t& end) {
    if (!by_tile) {
      if (started) return false;
      started = true;
      end = build_union();
      pos = 0;
      return true;
    }
    const int32_t* rown = arr(GroupLds<NT>::kRowN);
    while (seg_t < T && seg_off >= rown[seg_t]) {
      ++seg_t;
      seg_off = 0;
    }
    if (seg_t >= T) return false;
    end = build_window();
    pos = 0;
    seg_off += NT;
    return true;
  }
};

template <int KC>
struct GroupSrc {
  static constexpr bool kSparse = true;
  static constexpr bool kGrouped = true;
  static constexpr bool kTokens = false;
  GeoTable G;
  const int32_t* row_ptr;
  const int32_t* col_idx;
  int32_t k, G_k;
  int32_t gh, gw, lgT;   // group of gh x gw tiles, T = gh * gw = 1 << lgT
  int32_t ngc, n_groups;  // groups per group row, groups per (b, h)
  uint32_t wave_tile, wave_slab;  // 4 bits per wave: the wave's tile in the group and its 32-query slab
  int32_t max_chunks_per_block;
  // Nullable launch order: order[p] = -2 - (group item launched at position p),
  // as the mapping call writes it; a row permutation (non-negative entries) is
  // not an order of groups and is ignored.
  const int32_t* order;
  static constexpr bool kRemap = true;

  __device__ __forceinline__ int32_t remap(int32_t p, int32_t n_items) const {
    if (!order || order[0] >= 0) return p;
    const int32_t v = -2 - order[p];
    return (v >= 0 && v < n_items) ? v : p;
  }

  template <int NT>
  static constexpr int table_bytes() { return TableLds<NT>::kBytes + GroupLds<NT>::kBytes; }
  __device__ __forceinline__ int tile_of(int wave) const { return (int)((wave_tile >> (4 * wave)) & 15u); }

  // Tile t of the group of item; false when it lies outside the scale.
  __device__ __forceinline__ bool group_tile(int32_t item, int t, int32_t& bh, int32_t& a, int32_t& c) const {
    bh = item / n_groups;
    const int32_t gi = item - bh * n_groups;
    const int32_t A = gi / ngc, Cg = gi - A * ngc;
    a = A * gh + t / gw;
    c = Cg * gw + t % gw;
    return a < G.Th[k - 1] && c < G.Tw[k - 1];
  }
  __device__ __forceinline__ QuerySet queries(int32_t item, int wave) const {
    QuerySet s;
    int32_t a, c;
    const bool ok = group_tile(item, tile_of(wave), s.bh, a, c);
    const Tile t = tile_at(G, k, ok ? a : 0, ok ? c : 0);
    s.qbase = t.base - G.C[k - 1];
    s.qnc = t.nc;
    s.qstride = t.stride;
    s.q0 = (int32_t)((wave_slab >> (4 * wave)) & 15u) * kQPerWave;
    s.q1 = ok ? t.nr * t.nc : 0;
    return s;
  }
  template <int NT>
  __device__ __forceinline__ TableCursor<KC, NT, GroupBlocks<NT>> table_cursor(int32_t item, char* lds) const {
    using L = GroupLds<NT>;
    char* glds = lds + TableLds<NT>::kBytes;
    const int T = 1 << lgT;
    const int tid = threadIdx.x;
    const GeoTable* geo = stage_geometry<NT>(G, lds);  // published by the barrier below
    if (tid < T) {
      int32_t bh, a, c;
      int32_t p = 0, n = 0;
      if (group_tile(item, tid, bh, a, c)) {
        const int32_t r = bh * G_k + a * G.Tw[k - 1] + c;
        p = row_ptr[r];
        n = row_ptr[r + 1] - p;
      }
      reinterpret_cast<int32_t*>(glds + L::kRowP)[tid] = p;
      reinterpret_cast<int32_t*>(glds + L::kRowN)[tid] = n;
    }
    __syncthreads();
    const int32_t RC = NT >> lgT;
    bool long_row = false;
    for (int t = 0; t < T; ++t) long_row |= reinterpret_cast<const int32_t*>(glds + L::kRowN)[t] > RC;
    TableCursor<KC, NT, GroupBlocks<NT>> cur;
    cur.G = geo;
    cur.blocks.col = col_idx;
    cur.blocks.nb = G.NB[k];
    cur.blocks.T = T;
    cur.blocks.lgT = lgT;
    cur.blocks.by_tile = long_row;
    cur.blocks.started = false;
    cur.blocks.seg_t = 0;
    cur.blocks.seg_off = 0;
    cur.blocks.lds = glds;
    cur.nb = G.NB[k];
    const int32_t g = kTableCap / (max_chunks_per_block > 0 ? max_chunks_per_block : 1);
    cur.group = g < NT ? (g > 0 ? g : 1) : NT;
    cur.pos = 0;
    cur.end = 0;
    cur.tn = 0;
    cur.ti = 0;
    cur.lds = lds;
    return cur;
  }
};


// LDS pipeline stages as separate arrays: alias analysis then sees that the
// direct HBM -> LDS copies into one stage cannot touch the stage being read,
// and the compiler does not wait for those copies before every LDS read.
#define SV_STAGE_ARRAYS(NSX, BYTES)                                              \
  __shared__ __attribute__((aligned(16))) char sv_stage0[BYTES];                 \
  __shared__ __attribute__((aligned(16))) char sv_stage1[BYTES];                 \
  __shared__ __attribute__((aligned(16))) char sv_stage2[(NSX) > 2 ? (BYTES) : 16]; \
  __shared__ __attribute__((aligned(16))) char sv_stage3[(NSX) > 3 ? (BYTES) : 16];

template <int S>
__device__ __forceinline__ char* stage_ptr(char* s0, char* s1, char* s2, char* s3) {
  if constexpr (S == 0) return s0;
  else if constexpr (S == 1) return s1;
  else if constexpr (S == 2) return s2;
  else return s3;
}

// Sources with a kRuns member walk listed 1-D key blocks (BlockRowSrc).
template <class Src, class = void>
constexpr bool kRunsOf = false;
template <class Src>
constexpr bool kRunsOf<Src, std::void_t<decltype(Src::kRuns)>> = Src::kRuns;
// Sources with a kRemap member map a launch position to a work item (GroupSrc).
template <class Src, class = void>
constexpr bool kRemapOf = false;
template <class Src>
constexpr bool kRemapOf<Src, std::void_t<decltype(Src::kRemap)>> = Src::kRemap;

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
  SV_STAGE_ARRAYS(NS, kStage)
#define SV_STAGE(S) stage_ptr<S>(sv_stage0, sv_stage1, sv_stage2, sv_stage3)
  // chunk table of the sparse paths (unused by the dense path)
  constexpr int kTblBytes = Src::template table_bytes<NT>();
  __shared__ __attribute__((aligned(16))) char tsmem[kTblBytes];

  int32_t item = swizzled_item(blockIdx.x, gridDim.x, io.swizzle);
  if (item >= io.n_items) return;
  if constexpr (kRemapOf<Src>) item = __builtin_amdgcn_readfirstlane(src.remap(item, io.n_items));

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;

  const QuerySet qs = src.queries(item, wave);
  const int my_tile = src.tile_of(wave);  // bit of this wave's query tile in chunk masks
  const bf16_bits* qplane = static_cast<const bf16_bits*>(io.q) + (int64_t)qs.bh * io.q_bh_stride;
  const bf16_bits* kplane = static_cast<const bf16_bits*>(io.k) + (int64_t)qs.bh * io.kv_bh_stride;
  const bf16_bits* vplane = static_cast<const bf16_bits*>(io.v) + (int64_t)qs.bh * io.kv_bh_stride;

  const int32_t qslot = qs.q0 + l32;
  const bool qvalid = qslot < qs.q1;
  const int32_t qi = qvalid ? qslot : 0;
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
  // MFMA fragment offsets: K rows 32 kt + l32 (key tile kt is an immediate
  // 32 kt rows further) and V^T pieces through the transposing LDS read.
  FragOffsets<D, KC> fo;
  fo.init(l32, half, lane);

  // Direct loads of a chunk into LDS stage S: 32-bit unsigned byte offsets from the
  // scalar plane bases, wave-uniform LDS destinations.
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const char* kbytes = reinterpret_cast<const char*>(kplane);
  const char* vbytes = reinterpret_cast<const char*>(vplane);
  auto issue = [&](const Chunk& c, auto stage_c) {
    constexpr int S = decltype(stage_c)::value;
    char* kb = SV_STAGE(S);
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int first = (j * NW + wave_s) * 64;
      const int r = ld_row[j];
      int32_t tok;
      if constexpr (Src::kTokens) tok = src.tokens[c.base + (r < c.count ? r : 0)];
      else tok = chunk_token(c, chunk_slot(r, c.count));
      const uint32_t off = (uint32_t)(tok * D + 8 * ld_unit[j]) * 2u;
      dma16(kbytes + off, kb + first * 16);
      dma16(vbytes + off, kb + kTile + first * 16);
    }
  };

  auto cur = [&]() {
    if constexpr (Src::kSparse) {
      return src.template table_cursor<NT>(item, tsmem);
    } else if constexpr (kRunsOf<Src>) {
      return src.template run_cursor<NT>(item, tsmem);
    } else if constexpr (Src::kTokens) {
      return src.template token_cursor<NT>(item, tsmem);
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
    const char* kst = SV_STAGE(S);
    // waves of a grouped launch skip chunks their query tile does not list
    const bool active = !Src::kGrouped || ((c.mask >> my_tile) & 1u);
    // Sparse sources with 32-key chunks read the whole K chunk first, then look up
    // and copy the next chunk while those reads land, and issue the V^T reads
    // under the S^T products: no read waits behind a product or behind the next
    // chunk's descriptor (left to itself the compiler pairs each two K reads with a
    // full wait, after the descriptor lookup). The other shapes keep the
    // compiler's order: the extra registers would cost them a wave per SIMD.
    constexpr bool kHoist = KC == 32 && Src::kSparse;
    u32x4 kf[D / 16];
    if constexpr (kHoist) {
      if (active) {
#pragma unroll
        for (int s2 = 0; s2 < D / 16; ++s2) kf[s2] = *reinterpret_cast<const u32x4*>(kst + fo.k_off[s2]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    Chunk cn;
    const bool have_n = ahead == NS - 2 && cur.next(cn);
    if (have_n) issue(cn, std::integral_constant<int, (S + NS - 1) % NS>{});

    if (active) {
    // ---- S^T = K Q^T
    f32x16 st[KC / 32];
#pragma unroll
    for (int kt = 0; kt < KC / 32; ++kt) st[kt] = zero16();
    i16x4 vlo[KC / 16][D / 32], vhi[KC / 16][D / 32];
    if constexpr (kHoist) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int s2 = 0; s2 < D / 16; ++s2) st[0] = mfma_bf16(as_bf16x8(kf[s2]), qf.f[s2], st[0]);
#pragma unroll
      for (int ks = 0; ks < KC / 16; ++ks)
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) {
          vlo[ks][dt] = lds_read_tr(kst + fo.v_off[0][dt] + ks * 16 * kRow);
          vhi[ks][dt] = lds_read_tr(kst + fo.v_off[1][dt] + ks * 16 * kRow);
        }
      __builtin_amdgcn_sched_barrier(0);
    } else {
#pragma unroll
      for (int s2 = 0; s2 < D / 16; ++s2) {
#pragma unroll
        for (int kt = 0; kt < KC / 32; ++kt) {
          const u32x4 a = *reinterpret_cast<const u32x4*>(kst + fo.k_off[s2] + kt * 32 * kRow);
          st[kt] = mfma_bf16(as_bf16x8(a), qf.f[s2], st[kt]);
        }
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
        i16x4 lo, hi;
        if constexpr (kHoist) {
          lo = vlo[ks][dt];
          hi = vhi[ks][dt];
        } else {
          lo = lds_read_tr(kst + fo.v_off[0][dt] + ks * 16 * kRow);
          hi = lds_read_tr(kst + fo.v_off[1][dt] + ks * 16 * kRow);
        }
        u32x4 av;
        av[0] = __builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 0, 1));
        av[1] = __builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 2, 3));
        av[2] = __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 0, 1));
        av[3] = __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 2, 3));
        acc[dt] = mfma_bf16(as_bf16x8(av), pf, acc[dt]);
      }
    }
    }  // active

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
    const bf16_bits* bp = nullptr;  // epilogue base row
    float sgn = 1.f;
    if (io.epi_mode == 1) {
      bp = static_cast<const bf16_bits*>(io.epi_base) + orow * D;
      sgn = -1.f;
    } else if (io.epi_mode == 2) {
      const int32_t x = qrow / io.up_wk, y = qrow - (qrow / io.up_wk) * io.up_wk;
      const int32_t xs = ((2 * x + 1) * io.up_hs) / (2 * io.up_hk);
      const int32_t ys = ((2 * y + 1) * io.up_ws) / (2 * io.up_wk);
      bp = static_cast<const bf16_bits*>(io.epi_base) +
           ((int64_t)qs.bh * io.up_hs * io.up_ws + xs * io.up_ws + ys) * D;
    }
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int d = 32 * dt + 8 * j + 4 * half;
        float r[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) r[e] = acc[dt][4 * j + e] * inv * sgn;
        if (bp) {
          const uint2 b = *reinterpret_cast<const uint2*>(bp + d);
          r[0] += __uint_as_float(b.x << 16);
          r[1] += __uint_as_float(b.x & 0xffff0000u);
          r[2] += __uint_as_float(b.y << 16);
          r[3] += __uint_as_float(b.y & 0xffff0000u);
        }
        uint2 w;
        w.x = pack_bf16x2(r[0], r[1]);
        w.y = pack_bf16x2(r[2], r[3]);
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

  const QuerySet qs = src.queries(item, wave);
  const float* qplane = static_cast<const float*>(io.q) + (int64_t)qs.bh * io.q_bh_stride;
  const float* kplane = static_cast<const float*>(io.k) + (int64_t)qs.bh * io.kv_bh_stride;
  const float* vplane = static_cast<const float*>(io.v) + (int64_t)qs.bh * io.kv_bh_stride;
  const int32_t qslot = qs.q0 + l32;
  const bool qvalid = qslot < qs.q1;
  const int32_t qi = qvalid ? qslot : 0;
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
        const int32_t tok = chunk_token(c, chunk_slot(slot, c.count));
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

namespace {
// Workgroups that fit a CU at once for the two bf16 dense shapes compared below
// (register-bound: about 240 VGPRs for 8 waves with 64-key chunks give one
// workgroup; about 160 VGPRs for 4 waves with 32-key chunks (64 at d = 64) give
// three).
constexpr int kDenseWgsPerCu8 = 1;
constexpr int kDenseWgsPerCu4 = 3;

// Share of the launch's last round of workgroups that is busy: n workgroups over
// cus * per_cu slots.
double last_round_fill(int64_t n, int64_t cus, int per_cu) {
  const int64_t slots = cus * per_cu;
  const int64_t rounds = (n + slots - 1) / slots;
  return rounds == 0 ? 1.0 : (double)n / (double)(rounds * slots);
}
}  // namespace

hipError_t launch_dense_attn(const DenseAttnArgs& a, hipStream_t stream) {
  // Widest workgroup (most queries sharing each K/V chunk) that still gives every
  // CU a workgroup: 8 waves, else 4 waves, else 2 waves with 32-key chunks. In
  // bf16, 4 waves with 32-key chunks (several workgroups per CU) replace 8 waves
  // when they fill the CUs' slots more evenly.
  auto wgs = [&](int w) { return (int64_t)a.BH * ((a.n_q + 32 * w - 1) / (32 * w)); };
  int nw = a.waves;
  int want_kc = a.chunk;
  if (nw <= 0) {
    const int64_t cus = a.num_cu > 0 ? a.num_cu : 256;
    if (wgs(8) >= cus) {
      nw = 8;
      if (a.bf16 && a.stages == 2 && want_kc == 64) {
        const double f8 = last_round_fill(wgs(8), cus, kDenseWgsPerCu8);
        const double f4 = last_round_fill(wgs(4), cus, kDenseWgsPerCu4);
        if (f4 > f8 + 0.05) {
          nw = 4;
          want_kc = a.d == 128 ? 32 : 64;
        }
      }
    } else if (wgs(4) >= cus) {
      nw = 4;
    } else {
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

// token-row launch shapes (d, waves = C / 32, keys per chunk), two stages
#define SV_TOKEN_SHAPES(X) \
  X(128, 1, 64) X(128, 2, 64) X(128, 4, 64) X(128, 8, 64) X(64, 1, 64) X(64, 2, 64) X(64, 4, 64) X(64, 8, 64)

hipError_t launch_token_attn(const TokenAttnArgs& a, hipStream_t stream) {
  const int nw = a.C / kQPerWave;
  AttnIO io;
  io.q = a.q;
  io.k = a.k;
  io.v = a.v;
  io.o = a.o;
  io.lse = a.lse;
  io.q_bh_stride = a.q_bh_stride;
  io.kv_bh_stride = a.kv_bh_stride;
  io.o_rows = a.n_q;
  const int32_t n_blocks = (a.n_q + a.C - 1) / a.C;
  io.n_items = a.BH * n_blocks;
  io.swizzle = a.swizzle;
  io.scale_log2 = a.softmax_scale * kLog2e;
  io.epi_mode = a.epi_mode;
  io.epi_base = a.epi_base;
  io.up_hs = a.up_hs;
  io.up_ws = a.up_ws;
  io.up_hk = a.up_hk;
  io.up_wk = a.up_wk;
  auto make = [&](auto proto) {
    auto s = proto;
    s.tokens = a.tokens;
    s.M = a.M;
    s.C = a.C;
    s.n_q = a.n_q;
    s.n_kv = a.n_kv;
    s.n_blocks = n_blocks;
    return s;
  };
#define SV_TOK(DD, NN, KK) \
  if (a.d == DD && nw == NN && kc == KK) return launch_bf16<DD, NN, KK, 2>(io, make(TokenSrc<KK>{}), stream);
  // 32-key chunks (d = 128) halve the LDS of a workgroup: four 2-wave workgroups
  // per CU instead of two, three 4-wave ones instead of two. Automatic choice:
  // always for 2 waves, for 4 waves when it takes fewer rounds of workgroups.
  int kc = 64;
  if (a.d == 128 && nw >= 2 && nw <= 4) {
    const int64_t r64 = (io.n_items + 2LL * a.num_cu - 1) / (2LL * a.num_cu);
    const int64_t r32 = (io.n_items + (nw == 2 ? 4LL : 3LL) * a.num_cu - 1) / ((nw == 2 ? 4LL : 3LL) * a.num_cu);
    if (a.chunk == 32 || (a.chunk < 0 && (nw == 2 || r32 < r64))) kc = 32;
  } else if (a.d == 128 && nw == 8 && a.chunk == 32) {
    kc = 32;
  }
  SV_TOKEN_SHAPES(SV_TOK)
  SV_TOK(128, 2, 32) SV_TOK(128, 4, 32) SV_TOK(128, 8, 32)
#undef SV_TOK
  return hipErrorInvalidValue;
}

hipError_t launch_block_row_attn(const BlockRowAttnArgs& a, hipStream_t stream) {
  const int nw = a.block / kQPerWave;
  AttnIO io;
  io.q = a.q;
  io.k = a.k;
  io.v = a.v;
  io.o = a.o;
  io.lse = a.lse;
  io.q_bh_stride = a.q_bh_stride;
  io.kv_bh_stride = a.kv_bh_stride;
  io.o_rows = a.n_q;
  const int32_t n_blocks = (a.n_q + a.block - 1) / a.block;
  io.n_items = a.BH * n_blocks;
  io.swizzle = a.swizzle;
  io.scale_log2 = a.softmax_scale * kLog2e;
  auto make = [&](auto proto) {
    auto s = proto;
    s.rows = a.block_rows;
    s.M = a.M;
    s.C = a.block;
    s.n_q = a.n_q;
    s.n_kv = a.n_kv;
    s.n_blocks = n_blocks;
    return s;
  };
  int kc = a.chunk, ns = a.stages;
  if (!(a.d == 128 && nw >= 2 && kc == 32 && ns >= 2 && ns <= 4)) kc = 64, ns = 2;
#define SV_BLK(DD, NN, KK, SS) \
  if (a.d == DD && nw == NN && kc == KK && ns == SS) \
    return launch_bf16<DD, NN, KK, SS>(io, make(BlockRowSrc<KK>{}), stream);
#define SV_BLK2(DD, NN, KK) SV_BLK(DD, NN, KK, 2)
  SV_TOKEN_SHAPES(SV_BLK2)
  SV_BLK(128, 2, 32, 2) SV_BLK(128, 4, 32, 2) SV_BLK(128, 8, 32, 2)
  SV_BLK(128, 2, 32, 3) SV_BLK(128, 4, 32, 3) SV_BLK(128, 8, 32, 3)
  SV_BLK(128, 2, 32, 4) SV_BLK(128, 4, 32, 4) SV_BLK(128, 8, 32, 4)
#undef SV_BLK2
#undef SV_BLK
  return hipErrorInvalidValue;
}

namespace {

// Largest chunk count of any block of scales 1..k (full and edge tiles) at kc keys per chunk.
int32_t max_chunks_per_block(const GeoTable& G, int k, int kc) {
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
  return maxc;
}

// bf16 grouped launch shapes (d, waves, keys per chunk, pipeline stages).
#define SV_GROUP_SHAPES(X) \
  X(128, 8, 64, 2) X(128, 8, 32, 2) X(128, 4, 64, 2) X(128, 4, 32, 2) X(64, 8, 64, 2) X(64, 4, 64, 2) \
  X(128, 4, 32, 3) X(128, 4, 32, 4)

bool group_shape_exists(int d, int nw, int kc, int ns) {
#define SV_HAS(DD, NN, KK, SS) \
  if (d == DD && nw == NN && kc == KK && ns == SS) return true;
  SV_GROUP_SHAPES(SV_HAS)
#undef SV_HAS
  return false;
}

// Waves to (tile, slab): tiles in order for the first four waves, then in
// reverse tile order, so that when waves are dealt to the four SIMDs in turn a
// SIMD holds waves of tiles far apart in the group and a chunk listed by only
// some of the tiles still keeps several SIMDs busy.
void wave_map(int nw, int T, int wpt, uint32_t* wave_tile, uint32_t* wave_slab) {
  int tile[8], slab[8], n = 0;
  for (int t = 0; t < T; ++t)
    for (int s = 0; s < wpt; ++s) {
      tile[n] = t;
      slab[n] = s;
      ++n;
    }
  int order[8];
  for (int w = 0; w < nw; ++w) order[w] = w;
  if (nw > 4) {
    // waves 4.. take the remaining pairs by descending tile, ascending slab
    int m = 4;
    for (int t = T - 1; t >= 0; --t)
      for (int p = 4; p < nw; ++p)
        if (tile[p] == t) order[m++] = p;
  }
  *wave_tile = 0;
  *wave_slab = 0;
  for (int w = 0; w < nw; ++w) {
    *wave_tile |= (uint32_t)tile[order[w]] << (4 * w);
    *wave_slab |= (uint32_t)slab[order[w]] << (4 * w);
  }
}

hipError_t launch_grouped(const SparseAttnArgs& a, int nw, int wpt, int kc, int ns, hipStream_t stream) {
  const GeoTable& G = *a.G;
  const int k = a.k;
  const int T = nw / wpt;
  int gh = 1, gw = 2, lgT = 1;
  if (T == 4) {
    gh = 2;
    gw = 2;
    lgT = 2;
  } else if (T == 8) {
    gh = 2;
    gw = 4;
    lgT = 3;
  }
  const int32_t ngr = (G.Th[k - 1] + gh - 1) / gh, ngc = (G.Tw[k - 1] + gw - 1) / gw;
  AttnIO io;
  io.q = a.q;
  io.k = a.k_cache;
  io.v = a.v_cache;
  io.o = a.o;
  io.lse = a.lse;
  io.q_bh_stride = a.q_bh_stride;
  io.kv_bh_stride = a.kv_bh_stride;
  io.o_rows = G.h[k - 1] * G.w[k - 1];
  io.n_items = a.BH * ngr * ngc;
  io.swizzle = a.swizzle;
  io.scale_log2 = a.softmax_scale * kLog2e;
  GroupSrc<64> proto;
  proto.G = G;
  proto.row_ptr = a.row_ptr;
  proto.col_idx = a.col_idx;
  proto.k = k;
  proto.G_k = tiles_of(G, k);
  proto.gh = gh;
  proto.gw = gw;
  proto.lgT = lgT;
  proto.ngc = ngc;
  proto.n_groups = ngr * ngc;
  wave_map(nw, T, wpt, &proto.wave_tile, &proto.wave_slab);
  proto.max_chunks_per_block = max_chunks_per_block(G, k, kc);
  proto.order = a.schedule;
  auto as = [&](auto tag) {
    decltype(tag) s;
    s.G = proto.G;
    s.row_ptr = proto.row_ptr;
    s.col_idx = proto.col_idx;
    s.k = proto.k;
    s.G_k = proto.G_k;
    s.gh = proto.gh;
    s.gw = proto.gw;
    s.lgT = proto.lgT;
    s.ngc = proto.ngc;
    s.n_groups = proto.n_groups;
    s.wave_tile = proto.wave_tile;
    s.wave_slab = proto.wave_slab;
    s.max_chunks_per_block = proto.max_chunks_per_block;
    s.order = proto.order;
    return s;
  };
#define SV_GROUP(DD, NN, KK, SS) \
  if (a.d == DD && nw == NN && kc == KK && ns == SS) return launch_bf16<DD, NN, KK, SS>(io, as(GroupSrc<KK>{}), stream);
  SV_GROUP_SHAPES(SV_GROUP)
#undef SV_GROUP
  return hipErrorInvalidValue;
}

}  // namespace

int group_waves_for(const GeoTable& G, int k, int32_t BH, int num_cu, int group_waves) {
  if (group_waves >= 0) return group_waves;
  // Automatic choice. With the launch order of the mapping call (longest first
  // inside each XCD's share), one tile per workgroup is the faster form up to
  // about two rounds of workgroups (Infinity 64x64 step, 2048 tiles: 105 against
  // 111 us for pairs of tiles); from 16 tiles per CU on (2048x2048 schedule,
  // 128x128 step: 4096 tiles), pairs of 64-query tiles (quads of 32-query tiles)
  // sharing each staged chunk are faster (285 against 307 us).
  const int wpt = waves_for(G.eh[k - 1] * G.ew[k - 1]);
  if (wpt > 2) return 0;
  return (int64_t)BH * tiles_of(G, k) >= 16 * (int64_t)num_cu ? 4 : 0;
}

SparseForm sparse_form(const GeoTable& G, int k, int32_t BH, int num_cu, int group_waves) {
  SparseForm f;
  const int wpt = waves_for(G.eh[k - 1] * G.ew[k - 1]);
  const int gwv = group_waves_for(G, k, BH, num_cu, group_waves);
  f.gh = f.gw = 0;
  f.n_items = BH * tiles_of(G, k);
  if (gwv > wpt) {
    const int T = gwv / wpt;
    f.gh = T == 2 ? 1 : 2;
    f.gw = T == 8 ? 4 : 2;
    f.n_items = BH * ((G.Th[k - 1] + f.gh - 1) / f.gh) * ((G.Tw[k - 1] + f.gw - 1) / f.gw);
  }
  return f;
}

hipError_t launch_sparse_attn(const SparseAttnArgs& a, hipStream_t stream) {
  const GeoTable& G = *a.G;
  const int k = a.k;
  const int32_t tile_q = G.eh[k - 1] * G.ew[k - 1];
  const int wpt = waves_for(tile_q);
  // grouped path: several query tiles per workgroup share each staged chunk
  // (pairs of 64-query tiles or quads of 32-query tiles in 4-wave workgroups,
  // or 8-wave groups), when group_waves asks for it.
  const int gwv = group_waves_for(G, k, a.BH, a.num_cu, a.group_waves);
  if (a.bf16 && a.waves <= 0 && gwv > wpt) {
    int kc = a.group_chunk, ns = a.group_stages;
    if (!group_shape_exists(a.d, gwv, kc, ns)) {
      kc = 64;
      ns = 2;
    }
    if (group_shape_exists(a.d, gwv, kc, ns)) return launch_grouped(a, gwv, wpt, kc, ns, stream);
  }
  const int nw = a.waves > 0 ? a.waves : wpt;
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
  const int32_t maxc = max_chunks_per_block(G, k, kc);
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
    s.n_rows = a.BH * G_k;
    return s;
  };
  return dispatch<SparseSrc>(a.bf16, a.d, nw, kc, ns, io, make, stream);
}

}  // namespace sparvar

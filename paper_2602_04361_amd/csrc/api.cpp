// C ABI entry points: host-side validation, geometry tables, launches.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

#include "geometry.h"
#include "launch.h"
#include "sparvar.h"

using namespace sparvar;

namespace {

thread_local char g_last_error[512] = "";

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

int ok() {
  g_last_error[0] = '\0';
  return SPARVAR_OK;
}

int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(SPARVAR_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Compute units of the current device (queried once per device; concurrent
// first calls store the same value).
int device_cus() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// Launch options (sparvar_set_launch_option): process-wide, read at each call.
// The defaults are the tuned automatic choices.
constexpr int32_t kOptionDefaults[SPARVAR_OPT_COUNT] = {
    1,   // SPARVAR_OPT_SWIZZLE
    0,   // SPARVAR_OPT_DENSE_WAVES
    64,  // SPARVAR_OPT_DENSE_CHUNK
    2,   // SPARVAR_OPT_DENSE_STAGES
    0,   // SPARVAR_OPT_SPARSE_WAVES
    32,  // SPARVAR_OPT_SPARSE_CHUNK
    2,   // SPARVAR_OPT_SPARSE_STAGES
    -1,  // SPARVAR_OPT_SPARSE_GROUP_WAVES
    64,  // SPARVAR_OPT_SPARSE_GROUP_CHUNK
    2,   // SPARVAR_OPT_SPARSE_GROUP_STAGES
    32,  // SPARVAR_OPT_CSLA_CHUNK
    2,   // SPARVAR_OPT_CSLA_STAGES
    -1,  // SPARVAR_OPT_CS4A_CHUNK
    -1,  // SPARVAR_OPT_DECISION_FUSED
};

std::atomic<int32_t> g_options[SPARVAR_OPT_COUNT] = {
    kOptionDefaults[0], kOptionDefaults[1], kOptionDefaults[2],  kOptionDefaults[3],  kOptionDefaults[4],
    kOptionDefaults[5], kOptionDefaults[6], kOptionDefaults[7],  kOptionDefaults[8],  kOptionDefaults[9],
    kOptionDefaults[10], kOptionDefaults[11], kOptionDefaults[12], kOptionDefaults[13]};
static_assert(SPARVAR_OPT_COUNT == 14, "one default and one slot per launch option");

int32_t opt(sparvar_launch_option_t o) { return g_options[o].load(std::memory_order_relaxed); }

// softmax_scale must be finite and positive: the bf16 kernels take the running
// maximum of the raw scores and scale it afterwards.
int check_softmax_scale(float s) {
  if (!std::isfinite(s) || !(s > 0.f)) return fail(SPARVAR_ERR_INVALID, "softmax_scale %g is not finite and > 0", s);
  return SPARVAR_OK;
}

// The bf16 HBM -> LDS copies address a (b, h) plane of K/V with 32-bit byte
// offsets: every key row must start below 2^32 bytes into its plane.
int check_kv_offsets(int64_t n_kv, int32_t d, int elem) {
  if (elem == 2 && n_kv * d * elem >= (int64_t(1) << 32))
    return fail(SPARVAR_ERR_INVALID, "K/V plane of %lld tokens x %d exceeds 2^32 bytes (bf16 copy offsets are 32-bit)",
                (long long)n_kv, d);
  return SPARVAR_OK;
}

int build_table(const sparvar_geometry_t* g, GeoTable* T) {
  if (!g) return fail(SPARVAR_ERR_INVALID, "geometry is NULL");
  if (g->num_scales < 1 || g->num_scales > kMaxScales)
    return fail(SPARVAR_ERR_INVALID, "num_scales %d outside [1, %d]", g->num_scales, kMaxScales);
  if (!g->h || !g->w) return fail(SPARVAR_ERR_INVALID, "geometry h/w is NULL");
  if (g->block_edge < 1 || g->block_edge > 64)
    return fail(SPARVAR_ERR_INVALID, "block_edge %d outside [1, 64]", g->block_edge);
  if (g->num_sink_scales < 0) return fail(SPARVAR_ERR_INVALID, "num_sink_scales < 0");
  std::memset(T, 0, sizeof(*T));
  T->L = g->num_scales;
  T->b = g->block_edge;
  T->n_sink = g->num_sink_scales < g->num_scales ? g->num_sink_scales : g->num_scales;
  int64_t tok = 0, blk = 0;
  for (int i = 0; i < T->L; ++i) {
    const int32_t h = g->h[i], w = g->w[i];
    if (h < 1 || w < 1) return fail(SPARVAR_ERR_INVALID, "scale %d has size %dx%d", i + 1, h, w);
    // chunk descriptors keep a tile's row pitch (the scale width) in 16 bits
    if (h > SPARVAR_MAX_SIDE || w > SPARVAR_MAX_SIDE)
      return fail(SPARVAR_ERR_INVALID, "scale %d has a side over %d (%dx%d)", i + 1, SPARVAR_MAX_SIDE, h, w);
    T->h[i] = h;
    T->w[i] = w;
    T->eh[i] = h < T->b ? h : T->b;
    T->ew[i] = w < T->b ? w : T->b;
    T->Th[i] = (h + T->eh[i] - 1) / T->eh[i];
    T->Tw[i] = (w + T->ew[i] - 1) / T->ew[i];
    tok += (int64_t)h * w;
    blk += (int64_t)T->Th[i] * T->Tw[i];
    if (tok >= (int64_t(1) << 31) || blk >= (int64_t(1) << 31))
      return fail(SPARVAR_ERR_INVALID, "cache longer than 2^31 tokens");
    T->C[i + 1] = (int32_t)tok;
    T->NB[i + 1] = (int32_t)blk;
    if ((uint64_t)T->Th[i] * T->Tw[i] * T->Tw[i] >= (uint64_t(1) << 32))
      return fail(SPARVAR_ERR_INVALID, "scale %d has too many tiles", i + 1);
    T->mTw[i] = magic_for((uint32_t)T->Tw[i]);
  }
  return SPARVAR_OK;
}

int check_dtype_d(sparvar_dtype_t dt, int32_t d) {
  if (dt != SPARVAR_BF16 && dt != SPARVAR_F32) return fail(SPARVAR_ERR_UNSUPPORTED, "dtype %d not supported", (int)dt);
  if (d != 64 && d != 128) return fail(SPARVAR_ERR_UNSUPPORTED, "head dim %d not supported (64 or 128)", d);
  return SPARVAR_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

int check_plane(const void* p, int64_t stride, int64_t rows, int32_t d, int elem, const char* name) {
  if (!p) return fail(SPARVAR_ERR_INVALID, "%s is NULL", name);
  if (!aligned16(p)) return fail(SPARVAR_ERR_INVALID, "%s is not 16-byte aligned", name);
  if (stride < rows * d) return fail(SPARVAR_ERR_INVALID, "%s plane stride %lld < rows*d = %lld", name,
                                     (long long)stride, (long long)(rows * d));
  if ((stride * elem) % 16 != 0) return fail(SPARVAR_ERR_INVALID, "%s plane stride is not a multiple of 16 bytes", name);
  return SPARVAR_OK;
}

int32_t local_max_len(const GeoTable& T, int k, int32_t r, int32_t dil, int64_t* total) {
  int32_t mx = 0;
  int64_t sum = 0;
  for (int32_t g = 0; g < tiles_of(T, k); ++g) {
    const int32_t n = local_row_len(local_row(T, k, r, dil, g));
    mx = n > mx ? n : mx;
    sum += n;
  }
  if (total) *total = sum;
  return mx;
}

// Limits of the selection kernels (sparvar_select_blocks; the two-call form of
// sparvar_decision_step): the top-k kernel holds a row of NB scores and ids in
// 64 KiB of LDS, and the scoring kernel serves query tiles of at most 256 tokens.
int check_select_limits(const GeoTable& T, int S, bool scoring) {
  const int32_t NB = T.NB[S];
  if ((int64_t)NB * 8 > 64 * 1024) return fail(SPARVAR_ERR_UNSUPPORTED, "%d candidate blocks exceed the selection kernel's LDS", NB);
  if (scoring && T.eh[S - 1] * T.ew[S - 1] > 256)
    return fail(SPARVAR_ERR_UNSUPPORTED, "query tiles above 256 tokens are not supported by the scoring kernel");
  return SPARVAR_OK;
}

// Row slots of a mapping step: the longest local row plus topk selected blocks,
// each of which maps to one block (point projection) or to a cover box of at
// most `cover` blocks. Validates the shared mapping arguments.
struct MapSlots {
  int32_t max_local, cover, per_row;
  int64_t rows, need;  // rows, and the capacity they need (row slots, then one length per row)
};

int map_slots(const GeoTable& T, int32_t S, int32_t k, int32_t B, int32_t H, int32_t topk, int32_t radius,
              int32_t dil, int32_t projection, MapSlots* m) {
  if (S < 1 || k > T.L || S >= k) return fail(SPARVAR_ERR_INVALID, "need 1 <= S < k <= %d (S=%d, k=%d)", T.L, S, k);
  if (B < 1 || H < 1) return fail(SPARVAR_ERR_INVALID, "B and H must be >= 1");
  if (topk < 1 || topk > 1024) return fail(SPARVAR_ERR_INVALID, "topk %d outside [1, 1024]", topk);
  if (radius < 0 || dil < 0) return fail(SPARVAR_ERR_INVALID, "radius and dilation must be >= 0");
  if (projection != SPARVAR_PROJECT_POINT && projection != SPARVAR_PROJECT_COVER)
    return fail(SPARVAR_ERR_INVALID, "projection %d is not SPARVAR_PROJECT_POINT or SPARVAR_PROJECT_COVER", projection);
  m->max_local = local_max_len(T, k, radius, dil, nullptr);
  m->cover = projection == SPARVAR_PROJECT_COVER ? max_cover_size(T, S, k) : 0;
  const int64_t per_row = (int64_t)m->max_local + (int64_t)topk * (m->cover > 0 ? m->cover : 1);
  m->rows = (int64_t)B * H * tiles_of(T, k);
  m->need = m->rows * per_row + m->rows;
  if (m->rows >= (int64_t(1) << 31) || m->need >= (int64_t(1) << 31))
    return fail(SPARVAR_ERR_INVALID, "index lists too large for int32 offsets");
  if (per_row * 2 * 4 * 4 > 64 * 1024)
    return fail(SPARVAR_ERR_UNSUPPORTED, "rows of %lld candidates exceed the merge kernel's LDS", (long long)per_row);
  m->per_row = (int32_t)per_row;
  return SPARVAR_OK;
}

// Mapping of several steps in one launch (sparvar_map_index_steps). With
// noalloc, the per-row lengths the map kernel writes (and the order kernel
// reads) go to the library's fixed per-device scratch instead of the tail of
// each col_idxs[i], so the capacities only need the row slots.
int map_steps(const sparvar_geometry_t* g, int32_t S, int32_t n_steps, const int32_t* ks, int32_t B, int32_t H,
              int32_t topk, const int32_t* topk_idx, int32_t radius, int32_t prev_dilation, int32_t projection,
              int32_t* const* row_ptrs, int32_t* const* col_idxs, const int64_t* capacities, int32_t* const* orders,
              bool noalloc, hipStream_t stream) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if (n_steps < 1 || n_steps > kMaxMapSteps)
    return fail(SPARVAR_ERR_INVALID, "n_steps %d outside [1, %d]", n_steps, kMaxMapSteps);
  if (!ks || !row_ptrs || !col_idxs || !capacities) return fail(SPARVAR_ERR_INVALID, "a step array is NULL");
  if (!topk_idx) return fail(SPARVAR_ERR_INVALID, "topk_idx is NULL");
  MapStepArgs sa[kMaxMapSteps];
  int64_t blocks = 0, all_rows = 0;
  for (int i = 0; i < n_steps; ++i) {
    const int32_t k = ks[i];
    MapSlots m;
    if ((st = map_slots(T, S, k, B, H, topk, radius, prev_dilation, projection, &m)))
      return fail(st, "step %d: %s", i, std::string(g_last_error).c_str());
    if (!row_ptrs[i] || !col_idxs[i]) return fail(SPARVAR_ERR_INVALID, "step %d: row_ptr/col_idx is NULL", i);
    const int64_t need = noalloc ? m.need - m.rows : m.need;
    if (capacities[i] < need)
      return fail(SPARVAR_ERR_CAPACITY, "step %d: capacity %lld < bound %lld", i, (long long)capacities[i],
                  (long long)need);
    blocks += (m.rows + 3) / 4;
    sa[i].k = k;
    sa[i].max_local = m.max_local;
    sa[i].cover = m.cover;
    sa[i].local_row_ptr = nullptr;
    sa[i].local_col_idx = nullptr;
    sa[i].row_ptr = row_ptrs[i];
    sa[i].col_idx = col_idxs[i];
    sa[i].status = nullptr;
    sa[i].counts = nullptr;
    all_rows += m.rows;
  }
  if (blocks >= (int64_t(1) << 31)) return fail(SPARVAR_ERR_INVALID, "too many rows for one launch");
  if (noalloc) {
    if (all_rows > kNoAllocMaxRows)
      return fail(SPARVAR_ERR_CAPACITY, "%lld rows exceed the %d row lengths of the fixed scratch",
                  (long long)all_rows, kNoAllocMaxRows);
    int32_t* lengths = nullptr;
    if ((st = hip_status(noalloc_row_lengths(&lengths), "fixed scratch lookup"))) return st;
    int64_t off = 0;
    for (int i = 0; i < n_steps; ++i) {
      sa[i].counts = lengths + off;
      off += (int64_t)B * H * tiles_of(T, sa[i].k);
    }
  }
  st = hip_status(launch_map_index(T, S, B * H, topk, topk_idx, radius, prev_dilation, n_steps, sa, nullptr, stream),
                  "map index launch");
  if (st || !orders) return st;
  return hip_status(launch_map_order(T, B * H, topk, n_steps, sa, orders, device_cus(),
                                     opt(SPARVAR_OPT_SPARSE_GROUP_WAVES), stream),
                    "launch order launch");
}

}  // namespace

extern "C" {

const char* sparvar_status_string(int status) {
  switch (status) {
    case SPARVAR_OK: return "ok";
    case SPARVAR_ERR_INVALID: return "invalid argument";
    case SPARVAR_ERR_UNSUPPORTED: return "unsupported dtype or head dimension";
    case SPARVAR_ERR_CAPACITY: return "index capacity too small";
    case SPARVAR_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* sparvar_last_error(void) { return g_last_error; }

int sparvar_set_launch_option(int32_t option, int32_t value) {
  if (option < 0 || option >= SPARVAR_OPT_COUNT) return fail(SPARVAR_ERR_INVALID, "launch option %d unknown", option);
  g_options[option].store(value == SPARVAR_OPT_DEFAULT ? kOptionDefaults[option] : value, std::memory_order_relaxed);
  return ok();
}

int sparvar_get_launch_option(int32_t option, int32_t* value) {
  if (option < 0 || option >= SPARVAR_OPT_COUNT) return fail(SPARVAR_ERR_INVALID, "launch option %d unknown", option);
  if (!value) return fail(SPARVAR_ERR_INVALID, "value is NULL");
  *value = g_options[option].load(std::memory_order_relaxed);
  return ok();
}

int sparvar_scale_info(const sparvar_geometry_t* g, int32_t l, sparvar_scale_info_t* out) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if (!out) return fail(SPARVAR_ERR_INVALID, "out is NULL");
  if (l < 1 || l > T.L) return fail(SPARVAR_ERR_INVALID, "scale %d outside [1, %d]", l, T.L);
  out->h = T.h[l - 1];
  out->w = T.w[l - 1];
  out->n_tokens = T.h[l - 1] * T.w[l - 1];
  out->token_offset = T.C[l - 1];
  out->n_tokens_le = T.C[l];
  out->tile_h = T.eh[l - 1];
  out->tile_w = T.ew[l - 1];
  out->tiles_h = T.Th[l - 1];
  out->tiles_w = T.Tw[l - 1];
  out->block_offset = T.NB[l - 1];
  out->n_blocks_le = T.NB[l];
  return ok();
}

int sparvar_dense_attn_fwd(int32_t B, int32_t H, int32_t n_q, int32_t n_kv, int32_t d,
                           sparvar_dtype_t dtype, const void* q, int64_t q_bh_stride,
                           const void* k, const void* v, int64_t kv_bh_stride, void* o,
                           float* lse, float softmax_scale, hipStream_t stream) {
  int st = check_dtype_d(dtype, d);
  if (st) return st;
  if (B < 1 || H < 1 || n_q < 1 || n_kv < 1) return fail(SPARVAR_ERR_INVALID, "B, H, n_q, n_kv must be >= 1");
  if ((int64_t)B * H * n_q >= (int64_t(1) << 31)) return fail(SPARVAR_ERR_INVALID, "B*H*n_q too large");
  if ((st = check_softmax_scale(softmax_scale))) return st;
  const int elem = dtype == SPARVAR_BF16 ? 2 : 4;
  if ((st = check_plane(q, q_bh_stride, n_q, d, elem, "q"))) return st;
  if ((st = check_plane(k, kv_bh_stride, n_kv, d, elem, "k"))) return st;
  if ((st = check_plane(v, kv_bh_stride, n_kv, d, elem, "v"))) return st;
  if ((st = check_kv_offsets(n_kv, d, elem))) return st;
  if ((st = check_plane(o, (int64_t)n_q * d, n_q, d, elem, "o"))) return st;
  DenseAttnArgs a;
  a.BH = B * H;
  a.n_q = n_q;
  a.n_kv = n_kv;
  a.d = d;
  a.bf16 = dtype == SPARVAR_BF16;
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = o;
  a.lse = lse;
  a.q_bh_stride = q_bh_stride;
  a.kv_bh_stride = kv_bh_stride;
  a.softmax_scale = softmax_scale;
  a.waves = opt(SPARVAR_OPT_DENSE_WAVES);
  a.chunk = opt(SPARVAR_OPT_DENSE_CHUNK);
  a.stages = opt(SPARVAR_OPT_DENSE_STAGES);
  a.swizzle = opt(SPARVAR_OPT_SWIZZLE);
  a.num_cu = device_cus();
  return hip_status(launch_dense_attn(a, stream), "dense attention launch");
}

int sparvar_select_blocks(const sparvar_geometry_t* g, int32_t S, int32_t B, int32_t H,
                          int32_t d, sparvar_dtype_t dtype, const void* q_S,
                          int64_t q_bh_stride, const void* k_leS, int64_t k_bh_stride,
                          const float* lse_S, float softmax_scale, const float* scores_in,
                          float* scores_out, int32_t topk, int32_t* topk_idx,
                          hipStream_t stream) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if (S < 1 || S > T.L) return fail(SPARVAR_ERR_INVALID, "decision scale %d outside [1, %d]", S, T.L);
  if (B < 1 || H < 1) return fail(SPARVAR_ERR_INVALID, "B and H must be >= 1");
  if (topk < 1 || topk > 1024) return fail(SPARVAR_ERR_INVALID, "topk %d outside [1, 1024]", topk);
  if (!topk_idx) return fail(SPARVAR_ERR_INVALID, "topk_idx is NULL");
  const int32_t NB = T.NB[S];
  if ((st = check_select_limits(T, S, !scores_in))) return st;
  const int64_t rows = (int64_t)B * H * tiles_of(T, S);
  if (rows * (NB > topk ? NB : topk) >= (int64_t(1) << 31)) return fail(SPARVAR_ERR_INVALID, "score tensor too large");
  const float* sel_in = scores_in;
  if (!scores_in) {
    if (!scores_out) return fail(SPARVAR_ERR_INVALID, "scores_out is required when scores_in is NULL");
    if ((st = check_dtype_d(dtype, d))) return st;
    if (!lse_S) return fail(SPARVAR_ERR_INVALID, "lse_S is NULL");
    if ((st = check_softmax_scale(softmax_scale))) return st;
    const int elem = dtype == SPARVAR_BF16 ? 2 : 4;
    const int32_t NS = T.h[S - 1] * T.w[S - 1];
    if ((st = check_plane(q_S, q_bh_stride, NS, d, elem, "q_S"))) return st;
    if ((st = check_plane(k_leS, k_bh_stride, T.C[S], d, elem, "k_leS"))) return st;
    if ((st = check_kv_offsets(T.C[S], d, elem))) return st;
    ScoreArgs a;
    a.G = &T;
    a.S = S;
    a.BH = B * H;
    a.d = d;
    a.bf16 = dtype == SPARVAR_BF16;
    a.q = q_S;
    a.k = k_leS;
    a.q_bh_stride = q_bh_stride;
    a.k_bh_stride = k_bh_stride;
    a.lse = lse_S;
    a.softmax_scale = softmax_scale;
    a.scores = scores_out;
    hipError_t e = launch_pooled_scores(a, stream);
    if (e != hipSuccess) return hip_status(e, "pooled score launch");
    sel_in = scores_out;
  }
  return hip_status(launch_topk(sel_in, (int32_t)rows, NB, topk, topk_idx, stream), "top-k launch");
}

int sparvar_decision_step(const sparvar_geometry_t* g, int32_t S, int32_t B, int32_t H, int32_t d,
                          sparvar_dtype_t dtype, const void* q_S, int64_t q_bh_stride,
                          const void* k_leS, const void* v_leS, int64_t kv_bh_stride, void* o_S,
                          float* lse_S, float softmax_scale, float* scores_out, int32_t topk,
                          int32_t* topk_idx, hipStream_t stream) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if (S < 1 || S > T.L) return fail(SPARVAR_ERR_INVALID, "decision scale %d outside [1, %d]", S, T.L);
  if (B < 1 || H < 1) return fail(SPARVAR_ERR_INVALID, "B and H must be >= 1");
  if ((st = check_dtype_d(dtype, d))) return st;
  if (topk < 1 || topk > 1024) return fail(SPARVAR_ERR_INVALID, "topk %d outside [1, 1024]", topk);
  if (!lse_S || !scores_out || !topk_idx) return fail(SPARVAR_ERR_INVALID, "lse_S, scores_out and topk_idx are required");
  if ((st = check_softmax_scale(softmax_scale))) return st;
  const int elem = dtype == SPARVAR_BF16 ? 2 : 4;
  const int32_t NS = T.h[S - 1] * T.w[S - 1];
  const int32_t NB = T.NB[S];
  if ((st = check_plane(q_S, q_bh_stride, NS, d, elem, "q_S"))) return st;
  if ((st = check_plane(k_leS, kv_bh_stride, T.C[S], d, elem, "k_leS"))) return st;
  if ((st = check_plane(v_leS, kv_bh_stride, T.C[S], d, elem, "v_leS"))) return st;
  if ((st = check_kv_offsets(T.C[S], d, elem))) return st;
  if ((st = check_plane(o_S, (int64_t)NS * d, NS, d, elem, "o_S"))) return st;
  const int64_t rows = (int64_t)B * H * tiles_of(T, S);
  if ((int64_t)B * H * NS >= (int64_t(1) << 31) || rows * (NB > topk ? NB : topk) >= (int64_t(1) << 31))
    return fail(SPARVAR_ERR_INVALID, "tensors too large");
  // The fused kernel keeps every query's per-block mass in LDS; when that leaves
  // room for only one workgroup per CU (many candidate blocks), the two-call
  // sequence is faster. SPARVAR_DECISION_FUSED: 1 = whenever supported, 0 = never.
  size_t lds = 0;
  const int fused = opt(SPARVAR_OPT_DECISION_FUSED);
  const bool can_fuse = dtype == SPARVAR_BF16 && decision_supported(T, S, d, NB, &lds);
  if (can_fuse && (fused == 1 || (fused < 0 && lds <= 80 * 1024))) {
    DecisionArgs a;
    a.G = &T;
    a.S = S;
    a.BH = B * H;
    a.d = d;
    a.q = q_S;
    a.k = k_leS;
    a.v = v_leS;
    a.o = o_S;
    a.lse = lse_S;
    a.q_bh_stride = q_bh_stride;
    a.kv_bh_stride = kv_bh_stride;
    a.softmax_scale = softmax_scale;
    a.scores = scores_out;
    a.topk = topk;
    a.topk_idx = topk_idx;
    a.swizzle = opt(SPARVAR_OPT_SWIZZLE);
    return hip_status(launch_decision(a, stream), "decision step launch");
  }
  // the two-call sequence: every limit of both calls is checked before the first enqueues work
  if ((st = check_select_limits(T, S, true))) return st;
  if ((st = sparvar_dense_attn_fwd(B, H, NS, T.C[S], d, dtype, q_S, q_bh_stride, k_leS, v_leS, kv_bh_stride, o_S,
                                   lse_S, softmax_scale, stream)))
    return st;
  return sparvar_select_blocks(g, S, B, H, d, dtype, q_S, q_bh_stride, k_leS, kv_bh_stride, lse_S, softmax_scale,
                               nullptr, scores_out, topk, topk_idx, stream);
}

namespace {
int check_query_block(int32_t C) {
  if (C != 32 && C != 64 && C != 128 && C != 256)
    return fail(SPARVAR_ERR_UNSUPPORTED, "query block size %d is not 32, 64, 128 or 256", C);
  return SPARVAR_OK;
}
}  // namespace

int sparvar_cs4a_column_sums(const sparvar_geometry_t* g, int32_t S, int32_t C, int32_t B, int32_t H,
                             int32_t d, sparvar_dtype_t dtype, const void* q_S, int64_t q_bh_stride,
                             const void* k_leS, int64_t k_bh_stride, const float* lse_S,
                             float softmax_scale, float* colsum, hipStream_t stream) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if (S < 1 || S > T.L) return fail(SPARVAR_ERR_INVALID, "decision scale %d outside [1, %d]", S, T.L);
  if (B < 1 || H < 1) return fail(SPARVAR_ERR_INVALID, "B and H must be >= 1");
  if ((st = check_dtype_d(dtype, d))) return st;
  if (dtype != SPARVAR_BF16) return fail(SPARVAR_ERR_UNSUPPORTED, "token-granular paths take bf16 inputs");
  if ((st = check_query_block(C))) return st;
  if (!lse_S || !colsum) return fail(SPARVAR_ERR_INVALID, "lse_S and colsum are required");
  if ((st = check_softmax_scale(softmax_scale))) return st;
  const int32_t NS = T.h[S - 1] * T.w[S - 1];
  if ((st = check_plane(q_S, q_bh_stride, NS, d, 2, "q_S"))) return st;
  if ((st = check_plane(k_leS, k_bh_stride, T.C[S], d, 2, "k_leS"))) return st;
  if ((st = check_kv_offsets(T.C[S], d, 2))) return st;
  const int64_t G = (NS + C - 1) / C;
  if ((int64_t)B * H * G * T.C[S] >= (int64_t(1) << 31)) return fail(SPARVAR_ERR_INVALID, "column-sum tensor too large");
  Cs4aColsumArgs a;
  a.BH = B * H;
  a.n_q = NS;
  a.n_kv = T.C[S];
  a.d = d;
  a.C = C;
  a.q = q_S;
  a.k = k_leS;
  a.lse = lse_S;
  a.out = colsum;
  a.q_bh_stride = q_bh_stride;
  a.k_bh_stride = k_bh_stride;
  a.softmax_scale = softmax_scale;
  a.swizzle = opt(SPARVAR_OPT_SWIZZLE);
  a.num_cu = device_cus();
  return hip_status(launch_cs4a_colsum(a, stream), "column-sum launch");
}

int sparvar_cs4a_select_tokens(const float* values, int32_t rows, int32_t n, int32_t K, int32_t* inds,
                               hipStream_t stream) {
  if (!values || !inds) return fail(SPARVAR_ERR_INVALID, "values and inds are required");
  if (rows < 0 || n < 1) return fail(SPARVAR_ERR_INVALID, "rows must be >= 0 and n >= 1");
  if (K < 1 || K > 65536) return fail(SPARVAR_ERR_INVALID, "K %d outside [1, 65536]", K);
  if ((int64_t)rows * n >= (int64_t(1) << 31) || (int64_t)rows * K >= (int64_t(1) << 31))
    return fail(SPARVAR_ERR_INVALID, "tensors too large");
  return hip_status(launch_cs4a_topk(values, rows, n, K, inds, stream), "token top-K launch");
}

int32_t sparvar_cs4a_row_stride(const sparvar_geometry_t* g, int32_t K) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if (K < 1 || K > 65536) return fail(SPARVAR_ERR_INVALID, "K %d outside [1, 65536]", K);
  ok();
  return T.C[T.n_sink] + K;
}

int sparvar_cs4a_map_tokens(const sparvar_geometry_t* g, int32_t S, int32_t k, int32_t C, int32_t B,
                            int32_t H, int32_t K, const int32_t* inds_S, int32_t* tokens, int32_t M,
                            hipStream_t stream) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if (!(1 <= S && S < k && k <= T.L)) return fail(SPARVAR_ERR_INVALID, "need 1 <= S < k <= %d", T.L);
  if (B < 1 || H < 1) return fail(SPARVAR_ERR_INVALID, "B and H must be >= 1");
  if ((st = check_query_block(C))) return st;
  if (K < 1 || K > 65536) return fail(SPARVAR_ERR_INVALID, "K %d outside [1, 65536]", K);
  if (!inds_S || !tokens) return fail(SPARVAR_ERR_INVALID, "inds_S and tokens are required");
  if (M < T.C[T.n_sink] + K) return fail(SPARVAR_ERR_CAPACITY, "row stride %d < %d", M, T.C[T.n_sink] + K);
  const int64_t Gk = (T.h[k - 1] * T.w[k - 1] + C - 1) / C;
  if ((int64_t)B * H * Gk * M >= (int64_t(1) << 31)) return fail(SPARVAR_ERR_INVALID, "token rows too large");
  return hip_status(launch_cs4a_map(T, S, k, B * H, C, K, inds_S, tokens, M, stream), "token mapping launch");
}

int sparvar_cs4a_attn_fwd(const sparvar_geometry_t* g, int32_t k, int32_t C, int32_t B, int32_t H,
                          int32_t d, sparvar_dtype_t dtype, const void* q_k, int64_t q_bh_stride,
                          const void* k_lek, const void* v_lek, int64_t kv_bh_stride, void* o,
                          float* lse, float softmax_scale, const int32_t* tokens, int32_t M,
                          int32_t mode, const void* base, int32_t base_scale, hipStream_t stream) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if (k < 1 || k > T.L) return fail(SPARVAR_ERR_INVALID, "scale %d outside [1, %d]", k, T.L);
  if (B < 1 || H < 1) return fail(SPARVAR_ERR_INVALID, "B and H must be >= 1");
  if ((st = check_dtype_d(dtype, d))) return st;
  if (dtype != SPARVAR_BF16) return fail(SPARVAR_ERR_UNSUPPORTED, "token-granular paths take bf16 inputs");
  if ((st = check_query_block(C))) return st;
  if (!tokens || M < 1) return fail(SPARVAR_ERR_INVALID, "tokens and a row stride >= 1 are required");
  if (mode < 0 || mode > 2) return fail(SPARVAR_ERR_INVALID, "mode %d is not 0, 1 or 2", mode);
  if ((st = check_softmax_scale(softmax_scale))) return st;
  const int32_t Nk = T.h[k - 1] * T.w[k - 1];
  if ((int64_t)B * H * Nk >= (int64_t(1) << 31)) return fail(SPARVAR_ERR_INVALID, "B*H*N_k too large");
  if ((st = check_plane(q_k, q_bh_stride, Nk, d, 2, "q_k"))) return st;
  if ((st = check_plane(k_lek, kv_bh_stride, T.C[k], d, 2, "k_lek"))) return st;
  if ((st = check_plane(v_lek, kv_bh_stride, T.C[k], d, 2, "v_lek"))) return st;
  if ((st = check_kv_offsets(T.C[k], d, 2))) return st;
  if ((st = check_plane(o, (int64_t)Nk * d, Nk, d, 2, "o"))) return st;
  const int64_t Gk = (Nk + C - 1) / C;
  if ((int64_t)B * H * Gk * M >= (int64_t(1) << 31)) return fail(SPARVAR_ERR_INVALID, "token rows too large");
  TokenAttnArgs a;
  a.up_hs = a.up_ws = a.up_hk = a.up_wk = 1;
  if (mode == 1) {
    if ((st = check_plane(base, (int64_t)Nk * d, Nk, d, 2, "base"))) return st;
  } else if (mode == 2) {
    if (base_scale < 1 || base_scale > k) return fail(SPARVAR_ERR_INVALID, "base scale %d outside [1, %d]", base_scale, k);
    const int32_t NS = T.h[base_scale - 1] * T.w[base_scale - 1];
    if ((st = check_plane(base, (int64_t)NS * d, NS, d, 2, "base"))) return st;
    a.up_hs = T.h[base_scale - 1];
    a.up_ws = T.w[base_scale - 1];
    a.up_hk = T.h[k - 1];
    a.up_wk = T.w[k - 1];
  }
  a.BH = B * H;
  a.n_q = Nk;
  a.n_kv = T.C[k];
  a.d = d;
  a.C = C;
  a.M = M;
  a.q = q_k;
  a.k = k_lek;
  a.v = v_lek;
  a.o = o;
  a.lse = lse;
  a.q_bh_stride = q_bh_stride;
  a.kv_bh_stride = kv_bh_stride;
  a.softmax_scale = softmax_scale;
  a.tokens = tokens;
  a.epi_mode = mode;
  a.epi_base = mode == 0 ? nullptr : base;
  a.swizzle = opt(SPARVAR_OPT_SWIZZLE);
  a.chunk = opt(SPARVAR_OPT_CS4A_CHUNK);
  a.num_cu = device_cus();
  return hip_status(launch_token_attn(a, stream), "token attention launch");
}

namespace {
int check_csla(const GeoTable& T, int32_t k, int32_t block) {
  if (k < 1 || k > T.L) return fail(SPARVAR_ERR_INVALID, "scale %d outside [1, %d]", k, T.L);
  if (block != 32 && block != 64 && block != 128 && block != 256)
    return fail(SPARVAR_ERR_UNSUPPORTED, "block size %d is not 32, 64, 128 or 256", block);
  if ((T.C[k] + (int64_t)block - 1) / block > kCslaMaxBlocks)
    return fail(SPARVAR_ERR_UNSUPPORTED, "%d cache tokens make more than %d blocks of %d", T.C[k], kCslaMaxBlocks,
                block);
  return SPARVAR_OK;
}
}  // namespace

int32_t sparvar_csla_row_stride(const sparvar_geometry_t* g, int32_t k, int32_t block) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if ((st = check_csla(T, k, block))) return st;
  ok();
  return (T.C[k] + block - 1) / block;
}

int sparvar_csla_block_rows(const sparvar_geometry_t* g, int32_t k, const int32_t* windows, int32_t block,
                            int32_t* rows, int32_t M, hipStream_t stream) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if ((st = check_csla(T, k, block))) return st;
  if (!windows || !rows) return fail(SPARVAR_ERR_INVALID, "windows and rows are required");
  for (int h = 0; h < k; ++h)
    if (windows[h] < 0 || windows[h] > (1 << 20)) return fail(SPARVAR_ERR_INVALID, "window %d of scale %d", windows[h], h + 1);
  const int32_t need = (T.C[k] + block - 1) / block;
  if (M < need) return fail(SPARVAR_ERR_CAPACITY, "row stride %d < %d", M, need);
  const int64_t Gk = ((int64_t)T.h[k - 1] * T.w[k - 1] + block - 1) / block;
  if (Gk * M >= (int64_t(1) << 31)) return fail(SPARVAR_ERR_INVALID, "block rows too large");
  return hip_status(launch_csla_rows(T, k, windows, block, rows, M, stream), "CSLA block rows launch");
}

int sparvar_csla_attn_fwd(const sparvar_geometry_t* g, int32_t k, int32_t block, int32_t B, int32_t H, int32_t d,
                          sparvar_dtype_t dtype, const void* q_k, int64_t q_bh_stride, const void* k_lek,
                          const void* v_lek, int64_t kv_bh_stride, void* o, float* lse, float softmax_scale,
                          const int32_t* rows, int32_t M, hipStream_t stream) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if ((st = check_csla(T, k, block))) return st;
  if (B < 1 || H < 1) return fail(SPARVAR_ERR_INVALID, "B and H must be >= 1");
  if ((st = check_dtype_d(dtype, d))) return st;
  if (dtype != SPARVAR_BF16) return fail(SPARVAR_ERR_UNSUPPORTED, "the CSLA block path takes bf16 inputs");
  if (!rows || M < 1) return fail(SPARVAR_ERR_INVALID, "rows and a row stride >= 1 are required");
  if ((st = check_softmax_scale(softmax_scale))) return st;
  const int32_t Nk = T.h[k - 1] * T.w[k - 1];
  if ((int64_t)B * H * Nk >= (int64_t(1) << 31)) return fail(SPARVAR_ERR_INVALID, "B*H*N_k too large");
  if ((st = check_plane(q_k, q_bh_stride, Nk, d, 2, "q_k"))) return st;
  if ((st = check_plane(k_lek, kv_bh_stride, T.C[k], d, 2, "k_lek"))) return st;
  if ((st = check_plane(v_lek, kv_bh_stride, T.C[k], d, 2, "v_lek"))) return st;
  if ((st = check_kv_offsets(T.C[k], d, 2))) return st;
  if ((st = check_plane(o, (int64_t)Nk * d, Nk, d, 2, "o"))) return st;
  const int64_t Gk = (Nk + block - 1) / block;
  if (Gk * M >= (int64_t(1) << 31)) return fail(SPARVAR_ERR_INVALID, "block rows too large");
  BlockRowAttnArgs a;
  a.BH = B * H;
  a.n_q = Nk;
  a.n_kv = T.C[k];
  a.d = d;
  a.block = block;
  a.M = M;
  a.q = q_k;
  a.k = k_lek;
  a.v = v_lek;
  a.o = o;
  a.lse = lse;
  a.q_bh_stride = q_bh_stride;
  a.kv_bh_stride = kv_bh_stride;
  a.softmax_scale = softmax_scale;
  a.block_rows = rows;
  // 32-key chunks in two stages (d = 128): three 4-wave or four 2-wave
  // workgroups per CU; 2-5% ahead of three stages at blocks of 64 and 128
  a.chunk = opt(SPARVAR_OPT_CSLA_CHUNK);
  a.stages = opt(SPARVAR_OPT_CSLA_STAGES);
  a.swizzle = opt(SPARVAR_OPT_SWIZZLE);
  return hip_status(launch_block_row_attn(a, stream), "CSLA attention launch");
}

int sparvar_kv_compact(const sparvar_geometry_t* g, int32_t n_keep, const int32_t* keep, int32_t B, int32_t H,
                       int32_t d, sparvar_dtype_t dtype, const void* k_src, const void* v_src, int64_t src_bh_stride,
                       void* k_dst, void* v_dst, int64_t dst_bh_stride, hipStream_t stream) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if ((st = check_dtype_d(dtype, d))) return st;
  if (B < 1 || H < 1) return fail(SPARVAR_ERR_INVALID, "B and H must be >= 1");
  if (!keep || n_keep < 1 || n_keep > T.L) return fail(SPARVAR_ERR_INVALID, "n_keep %d outside [1, %d]", n_keep, T.L);
  for (int i = 0; i < n_keep; ++i) {
    if (keep[i] < 1 || keep[i] > T.L || (i > 0 && keep[i] <= keep[i - 1]))
      return fail(SPARVAR_ERR_INVALID, "kept scales must be strictly ascending within [1, %d]", T.L);
  }
  const int elem = dtype == SPARVAR_BF16 ? 2 : 4;
  int64_t kept = 0;
  for (int i = 0; i < n_keep; ++i) kept += T.C[keep[i]] - T.C[keep[i] - 1];
  const int32_t need_src = T.C[keep[n_keep - 1]];
  if ((st = check_plane(k_src, src_bh_stride, need_src, d, elem, "k_src"))) return st;
  if ((st = check_plane(v_src, src_bh_stride, need_src, d, elem, "v_src"))) return st;
  if ((st = check_plane(k_dst, dst_bh_stride, kept, d, elem, "k_dst"))) return st;
  if ((st = check_plane(v_dst, dst_bh_stride, kept, d, elem, "v_dst"))) return st;
  if (kept * d * elem / 16 >= (int64_t(1) << 31)) return fail(SPARVAR_ERR_INVALID, "compact plane too large");
  if ((int64_t)B * H > 65535) return fail(SPARVAR_ERR_INVALID, "B*H above 65535");
  KvCompactArgs a;
  a.G = &T;
  a.n_keep = n_keep;
  a.keep = keep;
  a.planes = B * H;
  a.d = d;
  a.elem = elem;
  a.k_src = k_src;
  a.v_src = v_src;
  a.k_dst = k_dst;
  a.v_dst = v_dst;
  a.src_bh_stride = src_bh_stride;
  a.dst_bh_stride = dst_bh_stride;
  return hip_status(launch_kv_compact(a, stream), "KV compaction launch");
}

int64_t sparvar_local_blocks_capacity(const sparvar_geometry_t* g, int32_t k, int32_t radius,
                                      int32_t prev_dilation) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if (k < 1 || k > T.L) return fail(SPARVAR_ERR_INVALID, "scale %d outside [1, %d]", k, T.L);
  if (radius < 0 || prev_dilation < 0) return fail(SPARVAR_ERR_INVALID, "radius and dilation must be >= 0");
  int64_t total = 0;
  local_max_len(T, k, radius, prev_dilation, &total);
  ok();
  return total;
}

int sparvar_local_blocks(const sparvar_geometry_t* g, int32_t k, int32_t radius,
                         int32_t prev_dilation, int32_t* row_ptr, int32_t* col_idx,
                         int64_t capacity, hipStream_t stream) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if (k < 1 || k > T.L) return fail(SPARVAR_ERR_INVALID, "scale %d outside [1, %d]", k, T.L);
  if (radius < 0 || prev_dilation < 0) return fail(SPARVAR_ERR_INVALID, "radius and dilation must be >= 0");
  if (!row_ptr || !col_idx) return fail(SPARVAR_ERR_INVALID, "row_ptr/col_idx is NULL");
  int64_t total = 0;
  local_max_len(T, k, radius, prev_dilation, &total);
  if (total >= (int64_t(1) << 31)) return fail(SPARVAR_ERR_INVALID, "local lists too large");
  if (capacity < total)
    return fail(SPARVAR_ERR_CAPACITY, "capacity %lld < %lld entries", (long long)capacity, (long long)total);
  return hip_status(launch_local_blocks(T, k, radius, prev_dilation, row_ptr, col_idx, stream), "local blocks launch");
}

int64_t sparvar_map_index_capacity(const sparvar_geometry_t* g, int32_t S, int32_t k, int32_t B,
                                   int32_t H, int32_t topk, int32_t radius,
                                   int32_t prev_dilation, int32_t projection) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  MapSlots m;
  if ((st = map_slots(T, S, k, B, H, topk, radius, prev_dilation, projection, &m))) return st;
  ok();
  return m.need;
}

int sparvar_map_index(const sparvar_geometry_t* g, int32_t S, int32_t k, int32_t B, int32_t H,
                      int32_t topk, const int32_t* topk_idx, const int32_t* local_row_ptr,
                      const int32_t* local_col_idx, int32_t radius, int32_t prev_dilation,
                      int32_t projection, int32_t* row_ptr, int32_t* col_idx, int64_t capacity,
                      int32_t* schedule, int32_t* status, hipStream_t stream) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  MapSlots m;
  if ((st = map_slots(T, S, k, B, H, topk, radius, prev_dilation, projection, &m))) return st;
  if (!topk_idx || !row_ptr || !col_idx || (!local_row_ptr) != (!local_col_idx))
    return fail(SPARVAR_ERR_INVALID, "a required pointer is NULL");
  if (capacity < m.need)
    return fail(SPARVAR_ERR_CAPACITY, "capacity %lld < bound %lld", (long long)capacity, (long long)m.need);
  MapStepArgs sa;
  sa.k = k;
  sa.max_local = m.max_local;
  sa.cover = m.cover;
  sa.local_row_ptr = local_row_ptr;
  sa.local_col_idx = local_col_idx;
  sa.row_ptr = row_ptr;
  sa.col_idx = col_idx;
  sa.status = local_row_ptr ? status : nullptr;
  return hip_status(launch_map_index(T, S, B * H, topk, topk_idx, radius, prev_dilation, 1, &sa, schedule, stream),
                    "map index launch");
}

int sparvar_map_index_steps(const sparvar_geometry_t* g, int32_t S, int32_t n_steps, const int32_t* ks, int32_t B,
                            int32_t H, int32_t topk, const int32_t* topk_idx, int32_t radius, int32_t prev_dilation,
                            int32_t projection, int32_t* const* row_ptrs, int32_t* const* col_idxs,
                            const int64_t* capacities, int32_t* const* orders, hipStream_t stream) {
  return map_steps(g, S, n_steps, ks, B, H, topk, topk_idx, radius, prev_dilation, projection, row_ptrs, col_idxs,
                   capacities, orders, false, stream);
}

int sparvar_map_index_steps_noalloc(const sparvar_geometry_t* g, int32_t S, int32_t n_steps, const int32_t* ks,
                                    int32_t B, int32_t H, int32_t topk, const int32_t* topk_idx, int32_t radius,
                                    int32_t prev_dilation, int32_t projection, int32_t* const* row_ptrs,
                                    int32_t* const* col_idxs, const int64_t* capacities, int32_t* const* orders,
                                    hipStream_t stream) {
  return map_steps(g, S, n_steps, ks, B, H, topk, topk_idx, radius, prev_dilation, projection, row_ptrs, col_idxs,
                   capacities, orders, true, stream);
}

int sparvar_block_sparse_attn_fwd(const sparvar_geometry_t* g, int32_t k, int32_t B, int32_t H,
                                  int32_t d, sparvar_dtype_t dtype, const void* q_k,
                                  int64_t q_bh_stride, const void* k_lek, const void* v_lek,
                                  int64_t kv_bh_stride, void* o, float* lse,
                                  float softmax_scale, const int32_t* row_ptr,
                                  const int32_t* col_idx, const int32_t* schedule,
                                  hipStream_t stream) {
  GeoTable T;
  int st = build_table(g, &T);
  if (st) return st;
  if ((st = check_dtype_d(dtype, d))) return st;
  if (k < 1 || k > T.L) return fail(SPARVAR_ERR_INVALID, "scale %d outside [1, %d]", k, T.L);
  if (B < 1 || H < 1) return fail(SPARVAR_ERR_INVALID, "B and H must be >= 1");
  if (!row_ptr || !col_idx) return fail(SPARVAR_ERR_INVALID, "row_ptr/col_idx is NULL");
  if ((st = check_softmax_scale(softmax_scale))) return st;
  const int32_t Nk = T.h[k - 1] * T.w[k - 1];
  if ((int64_t)B * H * Nk >= (int64_t(1) << 31)) return fail(SPARVAR_ERR_INVALID, "B*H*N_k too large");
  const int elem = dtype == SPARVAR_BF16 ? 2 : 4;
  if ((st = check_plane(q_k, q_bh_stride, Nk, d, elem, "q_k"))) return st;
  if ((st = check_plane(k_lek, kv_bh_stride, T.C[k], d, elem, "k_lek"))) return st;
  if ((st = check_plane(v_lek, kv_bh_stride, T.C[k], d, elem, "v_lek"))) return st;
  if ((st = check_kv_offsets(T.C[k], d, elem))) return st;
  if ((st = check_plane(o, (int64_t)Nk * d, Nk, d, elem, "o"))) return st;
  SparseAttnArgs a;
  a.G = &T;
  a.k = k;
  a.BH = B * H;
  a.d = d;
  a.bf16 = dtype == SPARVAR_BF16;
  a.q = q_k;
  a.k_cache = k_lek;
  a.v_cache = v_lek;
  a.o = o;
  a.lse = lse;
  a.q_bh_stride = q_bh_stride;
  a.kv_bh_stride = kv_bh_stride;
  a.softmax_scale = softmax_scale;
  a.row_ptr = row_ptr;
  a.col_idx = col_idx;
  a.schedule = schedule;
  a.waves = opt(SPARVAR_OPT_SPARSE_WAVES);
  a.chunk = opt(SPARVAR_OPT_SPARSE_CHUNK);
  a.stages = opt(SPARVAR_OPT_SPARSE_STAGES);
  a.swizzle = opt(SPARVAR_OPT_SWIZZLE);
  a.group_waves = opt(SPARVAR_OPT_SPARSE_GROUP_WAVES);
  a.group_chunk = opt(SPARVAR_OPT_SPARSE_GROUP_CHUNK);
  a.group_stages = opt(SPARVAR_OPT_SPARSE_GROUP_STAGES);
  a.num_cu = device_cus();
  return hip_status(launch_sparse_attn(a, stream), "block-sparse attention launch");
}

}  // extern "C"

// Internal launchers called by the C ABI after host-side validation.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "geometry.h"
#include "sparvar.h"

namespace sparvar {

struct DenseAttnArgs {
  int32_t BH, n_q, n_kv, d;
  bool bf16;
  const void *q, *k, *v;
  void* o;
  float* lse;
  int64_t q_bh_stride, kv_bh_stride;
  float softmax_scale;
  int waves;    // 0 = default
  int chunk;    // keys per chunk (32 or 64)
  int stages;   // LDS pipeline depth
  int swizzle;  // XCD-aware workgroup order
  int num_cu;   // compute units of the device (automatic launch choices)
};

struct SparseAttnArgs {
  const GeoTable* G;
  int32_t k, BH, d;
  bool bf16;
  const void *q, *k_cache, *v_cache;
  void* o;
  float* lse;
  int64_t q_bh_stride, kv_bh_stride;
  float softmax_scale;
  const int32_t *row_ptr, *col_idx, *schedule;
  int waves;    // 0 = from the tile size
  int chunk;    // keys per chunk (32 or 64)
  int stages;   // LDS pipeline depth
  int swizzle;
  int group_waves;  // grouped path: waves per workgroup (4 or 8), 0 = one tile per workgroup, < 0 = auto
  int group_chunk;  // grouped path: keys per chunk (32 or 64)
  int group_stages; // grouped path: LDS pipeline depth
  int num_cu;       // compute units of the device (automatic launch choices)
};

struct ScoreArgs {
  const GeoTable* G;
  int32_t S, BH, d;
  bool bf16;
  const void *q, *k;
  int64_t q_bh_stride, k_bh_stride;
  const float* lse;
  float softmax_scale;
  float* scores;
};

hipError_t launch_dense_attn(const DenseAttnArgs& a, hipStream_t stream);
struct DecisionArgs {
  const GeoTable* G;
  int32_t S, BH, d;
  const void *q, *k, *v;
  void* o;
  float* lse;
  int64_t q_bh_stride, kv_bh_stride;
  float softmax_scale;
  float* scores;
  int32_t topk;
  int32_t* topk_idx;
  int swizzle;
};

struct Cs4aColsumArgs {
  int32_t BH, n_q, n_kv, d, C;
  const void *q, *k;
  const float* lse;
  float* out;
  int64_t q_bh_stride, k_bh_stride;
  float softmax_scale;
  int swizzle;
  int num_cu;  // compute units of the device (key-range split)
};

struct TokenAttnArgs {
  int32_t BH, n_q, n_kv, d, C, M;
  const void *q, *k, *v;
  void* o;
  float* lse;
  int64_t q_bh_stride, kv_bh_stride;
  float softmax_scale;
  const int32_t* tokens;
  int epi_mode;
  const void* epi_base;
  int32_t up_hs, up_ws, up_hk, up_wk;
  int swizzle;
  int chunk = -1;  // keys per chunk: 32 or 64 (32 only for d = 128), < 0 = automatic
  int num_cu = 256;
};

// 1-D key blocks of the CSLA block mask: row g (shared by every (b, h)) of
// block_rows lists, ascending, the key blocks [v B, min(v B + B, n_kv)) of
// query block g (queries [g B, min(g B + B, n_q))), then padding.
struct BlockRowAttnArgs {
  int32_t BH, n_q, n_kv, d, block, M;
  const void *q, *k, *v;
  void* o;
  float* lse;
  int64_t q_bh_stride, kv_bh_stride;
  float softmax_scale;
  const int32_t* block_rows;
  int chunk;   // keys per chunk: 64 (two stages), or 32 with 3 or 4 stages (d = 128, >= 2 waves)
  int stages;
  int swizzle;
};

// Key blocks a 1-D block row may list (LDS bitmask of the row builder).
constexpr int32_t kCslaMaxBlocks = 2048;

// Copy of the kept scales' K/V tokens (in scale order) into a compact cache.
struct KvCompactArgs {
  const GeoTable* G;
  int32_t n_keep;
  const int32_t* keep;  // host, 1-based, ascending
  int32_t planes, d, elem;
  const void *k_src, *v_src;
  void *k_dst, *v_dst;
  int64_t src_bh_stride, dst_bh_stride;  // elements
};
hipError_t launch_kv_compact(const KvCompactArgs& a, hipStream_t stream);

// Work items of the bf16 block-sparse launch at scale k (with the default
// waves, chunk and stages): one query tile per workgroup (gh = gw = 0), or groups
// of gh x gw neighbouring tiles per workgroup. group_waves: as in SparseAttnArgs.
struct SparseForm {
  int gh, gw;
  int32_t n_items;
};
int group_waves_for(const GeoTable& G, int k, int32_t BH, int num_cu, int group_waves);
SparseForm sparse_form(const GeoTable& G, int k, int32_t BH, int num_cu, int group_waves);

hipError_t launch_sparse_attn(const SparseAttnArgs& a, hipStream_t stream);
hipError_t launch_block_row_attn(const BlockRowAttnArgs& a, hipStream_t stream);
hipError_t launch_csla_rows(const GeoTable& G, int k, const int32_t* windows, int32_t B, int32_t* rows, int32_t M,
                            hipStream_t stream);
hipError_t launch_token_attn(const TokenAttnArgs& a, hipStream_t stream);
hipError_t launch_cs4a_colsum(const Cs4aColsumArgs& a, hipStream_t stream);
hipError_t launch_cs4a_topk(const float* in, int32_t rows, int32_t n, int32_t K, int32_t* out, hipStream_t stream);
hipError_t launch_cs4a_map(const GeoTable& G, int S, int k, int32_t BH, int32_t C, int32_t K, const int32_t* inds,
                           int32_t* tokens, int32_t M, hipStream_t stream);
// fused dense attention + LSE + pooled scores + top-k at the decision scale (bf16)
bool decision_supported(const GeoTable& G, int S, int d, int32_t NB, size_t* lds_bytes);
hipError_t launch_decision(const DecisionArgs& a, hipStream_t stream);
hipError_t launch_pooled_scores(const ScoreArgs& a, hipStream_t stream);
hipError_t launch_topk(const float* scores, int32_t rows, int32_t nb, int32_t topk, int32_t* out,
                       hipStream_t stream);
hipError_t launch_local_blocks(const GeoTable& G, int k, int32_t radius, int32_t dil, int32_t* row_ptr,
                               int32_t* col_idx, hipStream_t stream);
// One target scale of a map launch. max_local bounds its local rows; row slots
// are max_local + topk * max(cover, 1) wide, and the row lengths follow the last slot.
struct MapStepArgs {
  int32_t k, max_local;
  const int32_t *local_row_ptr, *local_col_idx;  // both NULL: generated
  int32_t *row_ptr, *col_idx;
  int32_t* status;  // nullable: set to SPARVAR_ERR_CAPACITY when a supplied local row is cut to max_local
  int32_t cover = 0;  // 0: point projection; else covering, with boxes of at most `cover` tiles
  int32_t* counts = nullptr;  // row lengths; nullptr: after the last row slot of col_idx
};
// Rows whose lengths the allocation-free mapping call can hold (its fixed scratch).
constexpr int32_t kNoAllocMaxRows = SPARVAR_NOALLOC_MAX_ROWS;
// Device address of this device's fixed row-length scratch (looked up on first use).
hipError_t noalloc_row_lengths(int32_t** out);
constexpr int kMaxMapSteps = 8;
// Rows of every listed step in one launch; the schedule (single step only) is
// the longest-first order of that step's rows.
hipError_t launch_map_index(const GeoTable& G, int S, int32_t BH, int32_t topk, const int32_t* topk_idx,
                            int32_t radius, int32_t dil, int n_steps, const MapStepArgs* steps, int32_t* schedule,
                            hipStream_t stream);
// Launch order of the block-sparse kernel at each step with a non-NULL orders[i]
// (from the row lengths the map launch wrote): XCD-local longest first, over the
// work items of the form sparse_form() gives; group items are stored as -2 - item.
hipError_t launch_map_order(const GeoTable& G, int32_t BH, int32_t topk, int n_steps, const MapStepArgs* steps,
                            int32_t* const* orders, int num_cu, int group_waves, hipStream_t stream);

}  // namespace sparvar

/*
 * sparvar.h -- C ABI of the SparVAR block-sparse cross-scale attention library
 * for AMD Instinct MI355X (gfx950).
 *
 * The library implements the sparse hot path of SparVAR (arXiv 2602.04361):
 * queries of scale k of a next-scale-prediction VAR model attend to the
 * concatenated key/value cache of scales 1..k (Sec. 3.1, Eq. (1)), restricted
 * to kept b x b blocks: sink blocks on the early scales, a pattern selected at
 * a decision scale S and carried to scale k by the cross-scale index mapping
 * (Sec. 3.2 and the appendix "Cross-Scale Sparse Index Mapping"), and
 * cross-scale local windows (Sec. 3.3).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Scales are 1-based, as in the paper. The geometry struct is host memory
 *    read during the call only.
 *  - Tensors are [B, H, rows, d] with d contiguous and rows contiguous inside a
 *    (batch, head) plane; consecutive planes (b-major, then h) are
 *    `*_bh_stride` elements apart (>= rows * d), so a prefix of a preallocated
 *    cache, or a slice of one scale's queries out of it, is passed without a
 *    copy. Output tensors (o, lse, scores) are fully contiguous.
 *  - Cache tokens are concatenated in scale order; inside a scale they are
 *    row-major, token (x, y) of scale l at index C_{l-1} + x * w_l + y, where
 *    C_l = N_1 + ... + N_l (appendix, Decompose step).
 *  - Blocks are b x b spatial tiles of each scale; along an axis where the
 *    scale is shorter than b the whole axis is one tile. Block ids run
 *    scale-major and row-major over tiles inside a scale. Query tiles of
 *    scale k use the same tiling ("query blocks" of the paper).
 *  - Every pointer except the geometry is device memory owned by the caller.
 *    The library allocates no device memory (the allocation-free mapping call
 *    uses a fixed array that is part of the library's device code, one per
 *    device) and never synchronises: work is
 *    enqueued on `stream` (NULL = the default stream) and results are valid
 *    once the caller has synchronised that stream.
 *  - Process-wide state: the message of the last failure (one per calling
 *    thread), the compute-unit count of each device (queried once, used by the
 *    automatic launch shapes) and the launch options of
 *    sparvar_set_launch_option. Calls are safe from several threads and
 *    streams; a launch option changed while another thread launches takes
 *    effect for that call or the next.
 *  - Every call validates its arguments on the host before enqueueing any
 *    work; on error nothing is written. Device data (index lists, block ids)
 *    is not read on the host; kernels skip block ids that are out of range.
 *  - Inputs must be finite and softmax_scale finite and > 0 (the bf16 kernels
 *    take the running maximum of the raw scores and scale it afterwards).
 *    Outputs are bitwise deterministic for fixed inputs, launch arguments
 *    and launch options.
 *  - Supported: d in {64, 128}; dtype bf16 (bf16 MFMA, fp32 softmax and
 *    accumulation, bf16 output rounded to nearest even) or fp32 (fp32 MFMA).
 *  - Limits: 1 <= num_scales <= SPARVAR_MAX_SCALES, 1 <= block_edge <= 64,
 *    scale sides <= SPARVAR_MAX_SIDE, total cache tokens < 2^31,
 *    B * H * rows < 2^31; for bf16, one (b, h) plane of K or V (cache tokens
 *    x d x 2 bytes) below 2^32 bytes, i.e. fewer than 2^24 cache tokens at
 *    d = 128 (the HBM -> LDS copies use 32-bit offsets into a plane).
 *
 * Return value: SPARVAR_OK (0) or a negative status; a message for the last
 * failure on the calling thread is available from sparvar_last_error().
 *
 * Launch shapes are chosen automatically; sparvar_set_launch_option overrides
 * them process-wide (for measurements and tests).
 */
#ifndef SPARVAR_H_
#define SPARVAR_H_

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPARVAR_MAX_SCALES 32
#define SPARVAR_MAX_SIDE 65535

enum sparvar_status {
  SPARVAR_OK = 0,
  SPARVAR_ERR_INVALID = -1,     /* null pointer, bad shape, S >= k, topk <= 0, ... */
  SPARVAR_ERR_UNSUPPORTED = -2, /* dtype or head dimension not supported */
  SPARVAR_ERR_CAPACITY = -3,    /* output index buffer too small */
  SPARVAR_ERR_HIP = -4          /* a HIP launch or runtime call failed */
};

typedef enum sparvar_dtype { SPARVAR_BF16 = 0, SPARVAR_F32 = 1 } sparvar_dtype_t;

/* Launch options: process-wide overrides of the automatic launch shapes. A
 * shape that is not built falls back to the default; results depend on the
 * options only through floating-point summation order (index lists never). */
typedef enum sparvar_launch_option {
  SPARVAR_OPT_SWIZZLE = 0,         /* 1 (default): XCD-aware workgroup order; 0: natural order */
  SPARVAR_OPT_DENSE_WAVES,         /* dense attention: waves per workgroup, 0 (default) = automatic */
  SPARVAR_OPT_DENSE_CHUNK,         /* keys per staged chunk, 64 (default) or 32 */
  SPARVAR_OPT_DENSE_STAGES,        /* LDS pipeline stages, 2 (default) to 4 */
  SPARVAR_OPT_SPARSE_WAVES,        /* block-sparse attention: waves, 0 (default) = from the tile size */
  SPARVAR_OPT_SPARSE_CHUNK,        /* 32 (default) or 64 */
  SPARVAR_OPT_SPARSE_STAGES,       /* 2 (default) to 4 */
  SPARVAR_OPT_SPARSE_GROUP_WAVES,  /* -1 (default) = automatic, 0 = one query tile per workgroup, 4 or 8 */
  SPARVAR_OPT_SPARSE_GROUP_CHUNK,  /* 64 (default) or 32 */
  SPARVAR_OPT_SPARSE_GROUP_STAGES, /* 2 (default) to 4 */
  SPARVAR_OPT_CSLA_CHUNK,          /* CSLA block path: 32 (default) or 64 */
  SPARVAR_OPT_CSLA_STAGES,         /* 2 (default) to 4 */
  SPARVAR_OPT_CS4A_CHUNK,          /* token gather attention: -1 (default) = automatic, 32 or 64 */
  SPARVAR_OPT_DECISION_FUSED,      /* sparvar_decision_step: -1 (default) = automatic, 1 = fused whenever
                                      supported, 0 = two-call sequence */
  SPARVAR_OPT_COUNT
} sparvar_launch_option_t;
#define SPARVAR_OPT_DEFAULT INT32_MIN /* value that restores an option's default */

/* Set (or, with SPARVAR_OPT_DEFAULT, reset) one launch option; read one. */
int sparvar_set_launch_option(int32_t option, int32_t value);
int sparvar_get_launch_option(int32_t option, int32_t* value);

/* Scale schedule and tiling. h[l-1], w[l-1] are the rows and columns of scale
 * l; the first num_sink_scales scales are the attention sink (appendix,
 * Attention Sink paragraph). */
typedef struct sparvar_geometry {
  int32_t num_scales;
  const int32_t* h;
  const int32_t* w;
  int32_t block_edge;
  int32_t num_sink_scales;
} sparvar_geometry_t;

/* Derived geometry of one scale (host-only query). */
typedef struct sparvar_scale_info {
  int32_t h, w;            /* rows, columns */
  int32_t n_tokens;        /* N_l = h * w */
  int32_t token_offset;    /* C_{l-1}: first cache index of the scale */
  int32_t n_tokens_le;     /* C_l = N_<=l: cache length at step l */
  int32_t tile_h, tile_w;  /* tile edge e_h, e_w */
  int32_t tiles_h, tiles_w;/* tiles per axis T_h, T_w; query tiles G_l = T_h * T_w */
  int32_t block_offset;    /* id of the scale's first block */
  int32_t n_blocks_le;     /* blocks in scales 1..l */
} sparvar_scale_info_t;

/* Fill *out for scale l (1-based) of geometry g. Host only, no GPU work. */
int sparvar_scale_info(const sparvar_geometry_t* g, int32_t l, sparvar_scale_info_t* out);

/*
 * Dense cross-scale attention, Sec. 3.1 Eq. (1):
 *   O[b,h,i,:] = sum_j softmax_j(softmax_scale * <Q[b,h,i,:], K[b,h,j,:]>) V[b,h,j,:]
 * over all n_kv keys. q: [B,H,n_q,d] (plane stride q_bh_stride); k, v:
 * [B,H,n_kv,d] (plane stride kv_bh_stride); o: [B,H,n_q,d] contiguous, same
 * dtype as q. lse (nullable): [B,H,n_q] fp32, natural log of the softmax
 * denominator of the scaled scores. Used at the decision scale (Sec. 3.2,
 * dense attention at S) and as the dense baseline at every scale.
 */
int sparvar_dense_attn_fwd(int32_t B, int32_t H, int32_t n_q, int32_t n_kv, int32_t d,
                           sparvar_dtype_t dtype, const void* q, int64_t q_bh_stride,
                           const void* k, const void* v, int64_t kv_bh_stride, void* o,
                           float* lse, float softmax_scale, hipStream_t stream);

/*
 * Decision-scale block selection, Sec. 3.2 (column-sum D and TopK) and the
 * appendix "Hardware-Efficient Sparse Computation".
 * Scores: P = softmax(softmax_scale * Q_S K_<=S^T) using lse_S from
 * sparvar_dense_attn_fwd at scale S; score[b,h,g,v] = sum of P over the
 * queries of query tile g of scale S and the keys of block v < NB_<=S.
 * Selection: per row (b,h,g), the min(topk, NB_<=S) highest scores, ties to
 * the lower block id, written ascending to topk_idx[b,h,g,0..topk) and padded
 * with -1.
 *   q_S: [B,H,N_S,d] (plane stride q_bh_stride); k_leS: [B,H,N_<=S,d] (plane
 *   stride k_bh_stride); lse_S: [B,H,N_S] fp32.
 *   scores_in (nullable): if set, selection runs on these fp32
 *   [B,H,G_S,NB_<=S] scores and q_S, k_leS, lse_S are ignored (may be NULL).
 *   scores_out (nullable): receives the computed scores; required when
 *   scores_in is NULL.
 *   topk_idx: int32 [B,H,G_S,topk]. 1 <= topk <= 1024.
 */
int sparvar_select_blocks(const sparvar_geometry_t* g, int32_t S, int32_t B, int32_t H,
                          int32_t d, sparvar_dtype_t dtype, const void* q_S,
                          int64_t q_bh_stride, const void* k_leS, int64_t k_bh_stride,
                          const float* lse_S, float softmax_scale, const float* scores_in,
                          float* scores_out, int32_t topk, int32_t* topk_idx,
                          hipStream_t stream);

/*
 * The whole decision step at scale S in one call (Sec. 3.2): dense attention
 * of the scale-S queries over the keys of scales 1..S (O_S, LSE_S), the pooled
 * block scores and the per-tile top-k -- the results of sparvar_dense_attn_fwd
 * followed by sparvar_select_blocks, but for bf16 in one fused launch that
 * takes each block's probability mass from the attention pass itself (no
 * second S = Q K^T pass). fp32 inputs, tiles wider than 32 tokens, and
 * candidate sets large enough that the per-query block masses crowd the LDS
 * (e.g. 172 blocks at a 64x64 decision scale) run the two-call sequence.
 *   q_S: [B,H,N_S,d] (plane stride q_bh_stride); k_leS, v_leS: [B,H,N_<=S,d]
 *   (plane stride kv_bh_stride); o_S: [B,H,N_S,d] contiguous; lse_S: [B,H,N_S]
 *   fp32; scores_out: fp32 [B,H,G_S,NB_<=S]; topk_idx: int32 [B,H,G_S,topk]
 *   (ascending ids, -1 padding when topk > NB_<=S). All required.
 *   Scores and ids follow sparvar_select_blocks' definitions; the scores are
 *   computed in a different order, so equal-score ties may resolve
 *   differently from the two-call path at the last bit.
 * Requires 1 <= S <= num_scales, 1 <= topk <= 1024.
 */
int sparvar_decision_step(const sparvar_geometry_t* g, int32_t S, int32_t B, int32_t H, int32_t d,
                          sparvar_dtype_t dtype, const void* q_S, int64_t q_bh_stride,
                          const void* k_leS, const void* v_leS, int64_t kv_bh_stride, void* o_S,
                          float* lse_S, float softmax_scale, float* scores_out, int32_t topk,
                          int32_t* topk_idx, hipStream_t stream);

/*
 * ---- Token-granular CS^4A (Sec. 3.2; appendix, Hardware-Efficient Sparse
 * Computation and Cross-Scale Sparse Index Mapping). Query blocks are 1-D:
 * block i of a scale holds its queries [i C, min(i C + C, N)) in flattened
 * order, C in {32, 64, 128, 256}; G = ceil(N / C). bf16 only, d in {64, 128}.
 *
 * Column sums at the decision scale S: colsum[b,h,i,j] = sum over the queries
 * q of block i of P[q,j], P = softmax(scale * Q_S K_<=S^T), using lse_S from
 * sparvar_dense_attn_fwd (or sparvar_decision_step) at S.
 *   q_S: [B,H,N_S,d]; k_leS: [B,H,N_<=S,d]; lse_S: [B,H,N_S] fp32;
 *   colsum: fp32 [B,H,G_S,N_<=S].
 */
int sparvar_cs4a_column_sums(const sparvar_geometry_t* g, int32_t S, int32_t C, int32_t B, int32_t H,
                             int32_t d, sparvar_dtype_t dtype, const void* q_S, int64_t q_bh_stride,
                             const void* k_leS, int64_t k_bh_stride, const float* lse_S,
                             float softmax_scale, float* colsum, hipStream_t stream);

/*
 * inds^(S) = TopK over each of `rows` rows of n fp32 values: the min(K, n)
 * largest, ties to the lower index, written ascending and padded with -1.
 *   values: [rows, n]; inds: int32 [rows, K]. 1 <= K <= 65536.
 */
int sparvar_cs4a_select_tokens(const float* values, int32_t rows, int32_t n, int32_t K, int32_t* inds,
                               hipStream_t stream);

/*
 * Row stride M of the token rows of sparvar_cs4a_map_tokens: the sink tokens
 * (all of scales 1..num_sink_scales) plus K. Host-only; < 0 on error.
 */
int32_t sparvar_cs4a_row_stride(const sparvar_geometry_t* g, int32_t K);

/*
 * Key tokens of every query block g of scale k (1 <= S < k <= num_scales):
 * the sink tokens 0 .. N_sink - 1, then each token of row phi(g) of inds_S
 * (phi(g) = floor((2g + 1) G_S / (2 G_k)), the Query Block Homography)
 * mapped by Decompose-Align-Project -- scale l -> l' = k - (S - l), offset
 * (u, v) -> (floor(u h_l'/h_l), floor(v w_l'/w_l)) -- dropping mapped tokens
 * that fall among the sinks; then -1 up to the stride M. Ascending inds_S rows
 * give ascending token rows.
 *   inds_S: int32 [B,H,G_S,K] (sparvar_cs4a_select_tokens; -1 entries skipped);
 *   tokens: int32 [B,H,G_k,M], M = sparvar_cs4a_row_stride(g, K).
 */
int sparvar_cs4a_map_tokens(const sparvar_geometry_t* g, int32_t S, int32_t k, int32_t C, int32_t B,
                            int32_t H, int32_t K, const int32_t* inds_S, int32_t* tokens, int32_t M,
                            hipStream_t stream);

/*
 * Gather attention over token rows at scale k: every query of block g of
 * (b,h) attends, with one softmax, to the tokens of row (b*H + h) * G_k + g --
 * its ids in [0, N_<=k) up to the first id outside that range (ascending ids,
 * then padding) -- giving A; then, by mode:
 *   0: o = A (the sparse update Delta O^(k));
 *   1: o = base - A, base [B,H,N_k,d] (O_cache^(S) = O_dense - A at k = S);
 *   2: o = up(base) + A, base [B,H,N_S,d] a scale-S grid (O_cache^(S)),
 *      up() the nearest-neighbour upsampling by token centres: output token
 *      (x, y) of scale k reads base token (floor((2x+1) h_S / (2 h_k)),
 *      floor((2y+1) w_S / (2 w_k))) (Sec. 3.2: O^(k) = O_cache^(k) + Delta O^(k)).
 *   q_k: [B,H,N_k,d]; k_lek, v_lek: [B,H,N_<=k,d]; o: [B,H,N_k,d] contiguous;
 *   lse (nullable): [B,H,N_k] fp32 of A (-inf for an empty row, where A = 0);
 *   tokens: int32 [B*H*G_k, M]. base_scale: S for mode 2, ignored otherwise.
 */
int sparvar_cs4a_attn_fwd(const sparvar_geometry_t* g, int32_t k, int32_t C, int32_t B, int32_t H,
                          int32_t d, sparvar_dtype_t dtype, const void* q_k, int64_t q_bh_stride,
                          const void* k_lek, const void* v_lek, int64_t kv_bh_stride, void* o,
                          float* lse, float softmax_scale, const int32_t* tokens, int32_t M,
                          int32_t mode, const void* base, int32_t base_scale, hipStream_t stream);

/*
 * Sink + cross-scale local blocks of every query tile of scale k (block form
 * of the CSLA mask, Sec. 3.3, and the sink set of the appendix). Row g
 * (query tile (a,c) = (g / T_w(k), g % T_w(k))) lists ascending:
 *   - every block of scales 1..num_sink_scales;
 *   - the scale-k tiles (a',c') with max(|a'-a|, |c'-c|) <= radius;
 *   - the scale-(k-1) tiles overlapping the footprint of (a,c) rescaled to
 *     scale k-1, widened by prev_dilation tiles per side.
 * Head independent; compute once per (geometry, k, radius, dilation).
 * row_ptr: int32 [G_k + 1]; col_idx: int32 [capacity], capacity >=
 * sparvar_local_blocks_capacity(...). 1 <= k <= num_scales.
 */
int64_t sparvar_local_blocks_capacity(const sparvar_geometry_t* g, int32_t k, int32_t radius,
                                      int32_t prev_dilation); /* exact nnz, < 0 on error */
int sparvar_local_blocks(const sparvar_geometry_t* g, int32_t k, int32_t radius,
                         int32_t prev_dilation, int32_t* row_ptr, int32_t* col_idx,
                         int64_t capacity, hipStream_t stream);

/* Projection step of Decompose-Align-Project (appendix, Relative Scale
 * Alignment, Spatial Projection), at block granularity. */
typedef enum sparvar_projection {
  /* the tile origin (x,y) -> (floor(x h_l'/h_l), floor(y w_l'/w_l)), and the
   * scale-l' tile containing it: one block per selected block */
  SPARVAR_PROJECT_POINT = 0,
  /* every scale-l' tile overlapping the upsampled span [x0 h_l'/h_l,
   * x1 h_l'/h_l) x [y0 w_l'/w_l, y1 w_l'/w_l) of the tile's tokens [x0, x1) x
   * [y0, y1): a selection keeps its share of its scale's area */
  SPARVAR_PROJECT_COVER = 1
} sparvar_projection_t;

/*
 * Cross-scale index mapping and merge into CSR (appendix "Cross-Scale Sparse
 * Index Mapping" and "Attention Sink"). For target query tile (a,c) of scale
 * k and every (b,h): the source tile is the Query Block Homography
 * (floor((2a+1) T_h(S) / (2 T_h(k))), same for c); each selected block of
 * topk_idx[b,h,source,:] (skipping -1) goes through Decompose-Align-Project:
 * scale l -> l' = k - (S - l), then the projection (sparvar_projection_t).
 * The row is the ascending, duplicate-free union of the mapped blocks and
 * local row (a,c). Row index r = (b*H + h) * G_k + g.
 * Output layout (padded CSR): rows have a fixed stride M = (longest local row)
 * + topk * P, with P = 1 for the point projection and P = the largest cover
 * box of any block of scales 1..S for the covering one (9 at the Infinity
 * steps 40/48/64 from 32x32): row_ptr[r] = r * M, and col_idx[r*M .. r*M + M)
 * holds the row's ids followed by -1 up to the stride
 * (sparvar_block_sparse_attn_fwd skips them).
 *   topk_idx: int32 [B,H,G_S,topk] (from sparvar_select_blocks).
 *   local_row_ptr / local_col_idx: output of sparvar_local_blocks for k, or
 *   both NULL: the local rows are then generated from radius and
 *   prev_dilation inside this call (same lists, no extra launch).
 *   row_ptr: int32 [B*H*G_k + 1]; col_idx: int32 [capacity].
 *   radius, prev_dilation: the values the local rows are built with; they
 *   bound the local row length. A supplied local row longer than that bound
 *   is cut to it, and the call sets *status (below) to SPARVAR_ERR_CAPACITY.
 *   capacity: >= sparvar_map_index_capacity(...) with the same arguments
 *   (B*H*G_k * M row slots, plus B*H*G_k entries the call uses for row lengths
 *   when a schedule is asked for).
 *   schedule (nullable): int32 [B*H*G_k], the rows ordered longest first,
 *   equal lengths in row order.
 *   status (nullable): one device int32 that the caller clears beforehand; the
 *   kernel stores SPARVAR_ERR_CAPACITY there when it cut a supplied local row,
 *   and writes nothing otherwise (generated local rows always fit).
 * Requires 1 <= S < k <= num_scales.
 */
int64_t sparvar_map_index_capacity(const sparvar_geometry_t* g, int32_t S, int32_t k, int32_t B,
                                   int32_t H, int32_t topk, int32_t radius,
                                   int32_t prev_dilation, int32_t projection); /* upper bound, < 0 on error */
int sparvar_map_index(const sparvar_geometry_t* g, int32_t S, int32_t k, int32_t B, int32_t H,
                      int32_t topk, const int32_t* topk_idx, const int32_t* local_row_ptr,
                      const int32_t* local_col_idx, int32_t radius, int32_t prev_dilation,
                      int32_t projection, int32_t* row_ptr, int32_t* col_idx, int64_t capacity,
                      int32_t* schedule, int32_t* status, hipStream_t stream);

/*
 * Index mapping for several target scales in one launch: for each i <
 * n_steps (1 <= n_steps <= 8), the rows of scale ks[i] exactly as
 * sparvar_map_index(g, S, ks[i], B, H, topk, topk_idx, NULL, NULL, radius,
 * prev_dilation, projection, row_ptrs[i], col_idxs[i], capacities[i], NULL,
 * NULL, stream) writes them (local rows generated in the call). The mapping of every later scale
 * depends only on the selection at S, so all of them can be built right after
 * the decision step.
 *   ks, row_ptrs, col_idxs, capacities: host arrays of n_steps entries, read
 *   during the call; row_ptrs[i], col_idxs[i] are device buffers sized as for
 *   sparvar_map_index, capacities[i] >= sparvar_map_index_capacity(g, S,
 *   ks[i], B, H, topk, radius, prev_dilation, projection).
 *   orders (nullable host array of n_steps nullable device pointers, each
 *   int32 [B*H*G_k of ks[i]]): a launch order for sparvar_block_sparse_attn_fwd
 *   at ks[i] (its schedule argument), written from the row lengths by a second
 *   launch: the work items of the form that call uses by default on this
 *   device (one query tile per workgroup, or groups of neighbouring tiles),
 *   longest first inside each XCD's share of the launch. Tile items are stored
 *   as row ids, group items g as -2 - g; the attention call uses an order only
 *   for the form it belongs to and launches in natural order otherwise. The
 *   order never changes results.
 */
int sparvar_map_index_steps(const sparvar_geometry_t* g, int32_t S, int32_t n_steps, const int32_t* ks,
                            int32_t B, int32_t H, int32_t topk, const int32_t* topk_idx,
                            int32_t radius, int32_t prev_dilation, int32_t projection,
                            int32_t* const* row_ptrs, int32_t* const* col_idxs,
                            const int64_t* capacities, int32_t* const* orders, hipStream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * call and results as sparvar_map_index_steps, but the per-row lengths that
 * call keeps after the row slots of each col_idxs[i] (and that its launch
 * orders are ranked from) live in a fixed array of SPARVAR_NOALLOC_MAX_ROWS
 * int32 inside the library, one per device, held until the process ends. So
 * capacities[i] only need the row slots: sparvar_map_index_capacity(...) minus
 * B*H*G_k of ks[i]. The call allocates nothing; the first call on a device
 * looks up that device's array. The array is shared by every call on a
 * device: calls that overlap on one device race (serialise them, e.g. on one
 * stream). Fails with SPARVAR_ERR_CAPACITY when the steps' rows (B*H*G_k
 * summed over the steps) exceed SPARVAR_NOALLOC_MAX_ROWS.
 */
#define SPARVAR_NOALLOC_MAX_ROWS (1 << 20) /* 4 MiB of row lengths per device */
int sparvar_map_index_steps_noalloc(const sparvar_geometry_t* g, int32_t S, int32_t n_steps,
                                    const int32_t* ks, int32_t B, int32_t H, int32_t topk,
                                    const int32_t* topk_idx, int32_t radius, int32_t prev_dilation,
                                    int32_t projection, int32_t* const* row_ptrs,
                                    int32_t* const* col_idxs, const int64_t* capacities,
                                    int32_t* const* orders, hipStream_t stream);

/*
 * Block-sparse cross-scale attention at scale k (the sparse update
 * Delta O of Sec. 3.2 and the block-masked attention of Sec. 3.3, Eq. (3)):
 * every query of query tile g of (b,h) attends, with one softmax, to exactly
 * the tokens of the blocks listed in CSR row r = (b*H + h) * G_k + g.
 *   q_k: [B,H,N_k,d] (plane stride q_bh_stride); k_lek, v_lek: [B,H,N_<=k,d]
 *   (plane stride kv_bh_stride); o: [B,H,N_k,d] contiguous; lse (nullable):
 *   [B,H,N_k] fp32. A row with no valid block yields o = 0, lse = -inf.
 *   row_ptr / col_idx: CSR over B*H*G_k rows; ids outside [0, NB_<=k) are
 *   skipped wherever they appear, and the remaining ids of a row must be
 *   strictly ascending (as written by sparvar_map_index). A row that repeats
 *   an id or lists ids out of order gives unspecified values (never an access
 *   outside the inputs and outputs).
 *   schedule (nullable): a launch order; it changes only the order of work,
 *   never the results. Either a permutation of the B*H*G_k rows (non-negative
 *   entries: sparvar_map_index's longest-first schedule, or an order from
 *   sparvar_map_index_steps), used by the one-tile-per-workgroup form, or an
 *   order of groups of neighbouring tiles (entries -2 - group, from
 *   sparvar_map_index_steps), used by the grouped form; each form launches in
 *   natural order when given the other kind (told apart by schedule[0]).
 */
int sparvar_block_sparse_attn_fwd(const sparvar_geometry_t* g, int32_t k, int32_t B, int32_t H,
                                  int32_t d, sparvar_dtype_t dtype, const void* q_k,
                                  int64_t q_bh_stride, const void* k_lek, const void* v_lek,
                                  int64_t kv_bh_stride, void* o, float* lse,
                                  float softmax_scale, const int32_t* row_ptr,
                                  const int32_t* col_idx, const int32_t* schedule,
                                  hipStream_t stream);

/*
 * Cross-Scale Local Sparse Attention in the paper's block form (Sec. 3.3:
 * Cross-Scale Local Mapping, sink mask, Eq. block_mask), with 1-D blocks of
 * `block` contiguous tokens on both axes: query block u holds queries
 * [u*block, min((u+1)*block, N_k)) of scale k, key block v holds cache tokens
 * [v*block, min((v+1)*block, N_<=k)). block is 32, 64, 128 or 256;
 * ceil(N_<=k / block) <= 2048.
 *
 * Row stride of the block rows: ceil(N_<=k / block). Host-only; < 0 on error.
 */
int32_t sparvar_csla_row_stride(const sparvar_geometry_t* g, int32_t k, int32_t block);

/*
 * Block rows of scale k (1 <= k <= num_scales). A query (x, y) of scale k is
 * aligned to historical scale h at (round(x h_h / h_k), round(y w_h / w_k)),
 * halves rounded up and not clipped, and keeps the keys (x', y') of scale h
 * with max(|cx - x'|, |cy - y'|) <= windows[h-1] / 2 (integer division; a
 * window of 0 keeps no key of that scale); every token of scales
 * 1..num_sink_scales is kept as well. Row u lists, ascending, the key blocks
 * holding at least one kept (query of u, key) pair, then -1 up to the stride.
 * Head independent: compute once per (geometry, k, windows, block).
 *   windows: host int32 [k], window sizes w_h >= 0 (read during the call).
 *   rows: int32 [G_k, M], G_k = ceil(N_k / block),
 *   M >= sparvar_csla_row_stride(g, k, block).
 */
int sparvar_csla_block_rows(const sparvar_geometry_t* g, int32_t k, const int32_t* windows,
                            int32_t block, int32_t* rows, int32_t M, hipStream_t stream);

/*
 * Block-sparse attention over the rows of sparvar_csla_block_rows: every
 * query of block u of (b,h) attends, with one softmax, to every key of the
 * key blocks of row u (shared by all (b,h)), up to its first id outside
 * [0, ceil(N_<=k / block)). A row with no valid block yields o = 0 and
 * lse = -inf. bf16 only.
 *   q_k: [B,H,N_k,d] (plane stride q_bh_stride); k_lek, v_lek: [B,H,N_<=k,d]
 *   (plane stride kv_bh_stride); o: [B,H,N_k,d] contiguous; lse (nullable):
 *   [B,H,N_k] fp32; rows: int32 [G_k, M]. Ids of a row must be strictly
 *   ascending before the first invalid one; otherwise values are unspecified
 *   (never an access outside the inputs and outputs).
 */
int sparvar_csla_attn_fwd(const sparvar_geometry_t* g, int32_t k, int32_t block, int32_t B,
                          int32_t H, int32_t d, sparvar_dtype_t dtype, const void* q_k,
                          int64_t q_bh_stride, const void* k_lek, const void* v_lek,
                          int64_t kv_bh_stride, void* o, float* lse, float softmax_scale,
                          const int32_t* rows, int32_t M, hipStream_t stream);

/*
 * KV compression, the memory side of the paper's "+ KV comp." setting (memory
 * consumption paragraph of the additional experiments: keep only the KV cache
 * of the sink scales and of the local scales). For every (b,h) plane, copies
 * the K and V tokens of the scales keep[0..n_keep) (1-based, strictly
 * ascending), in that order, into a compact cache: the cache of the schedule
 * made of the kept scales' sides, on which every call above runs unchanged.
 * With the sink scales and the scales that carry CSLA windows kept, the CSLA
 * token mask of the compact schedule is exactly the full mask restricted to the
 * kept tokens (dropped scales hold no kept key). The 2-D block path is not
 * served by a compact cache in general: its rows at step k read the sink
 * scales, scales k - 1 and k (local windows) and every scale the mapping
 * aligns a selected block to (l + k - S for l <= S, i.e. scales k - S + 1
 * .. k), which at the Infinity steps is every scale.
 *   keep: host int32 [n_keep], read during the call.
 *   k_src, v_src: [B,H,>= C_{keep[n_keep-1]},d] (plane stride src_bh_stride);
 *   k_dst, v_dst: [B,H,>= sum of N_l over the kept scales,d] (plane stride
 *   dst_bh_stride); element strides are multiples of 16 bytes. B*H <= 65535.
 */
int sparvar_kv_compact(const sparvar_geometry_t* g, int32_t n_keep, const int32_t* keep, int32_t B,
                       int32_t H, int32_t d, sparvar_dtype_t dtype, const void* k_src,
                       const void* v_src, int64_t src_bh_stride, void* k_dst, void* v_dst,
                       int64_t dst_bh_stride, hipStream_t stream);

/* Static description of a status code. */
const char* sparvar_status_string(int status);
/* Message of the last failed call on this thread ("" if none). */
const char* sparvar_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SPARVAR_H_ */

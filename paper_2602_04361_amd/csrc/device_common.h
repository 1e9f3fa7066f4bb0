// Device-side building blocks shared by the attention and scoring kernels:
// MFMA fragment types, key chunks, and the S^T = K Q^T tile product.
//
// Layout choice (CDNA MFMA 32x32): the score tile is computed transposed,
// S^T[key][query] = K Q^T, so that a lane owns one query column and 16 keys.
// Row-wise softmax statistics are then lane-local plus one exchange between
// the two 32-lane halves, and the probabilities leave the accumulator already
// in the B-operand layout of the P V^T product (O^T = V^T P^T).
//
// Accumulator layout of a 32x32 MFMA tile: register r of lane
// (col = lane % 32, half = lane / 32) holds row 8 * (r / 4) + 4 * half + r % 4.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "geometry.h"

namespace sparvar {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef uint16_t bf16_bits;

constexpr int kChunk = 64;     // keys per chunk
constexpr int kQPerWave = 32;  // queries per wave (MFMA N)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Keys of a chunk: slot s < count is token base + (s / nc) * stride + s % nc.
// mask: query tiles of a workgroup's tile group that attend to the chunk (bit t for tile t).
struct Chunk {
  int32_t base, nc, stride, count, magic;  // magic = ceil(65536 / nc): s / nc == (s * magic) >> 16 for s < 64
  uint32_t mask;
};

// Both products must use the 24-bit multiplier, which issues at full rate where
// a 32-bit integer multiply issues at quarter rate. Every factor fits (s < 64,
// magic <= 65536, 0 <= stride - nc < 65536); the row advance is masked to 16
// bits so that the compiler can see it too.
__device__ __forceinline__ int32_t chunk_token(const Chunk& c, int32_t s) {
  const uint32_t q = __umul24((uint32_t)s, (uint32_t)c.magic) >> 16;
  const uint32_t adv = (uint32_t)(c.stride - c.nc) & 0xffffu;
  return c.base + s + (int32_t)(q * adv);
}

// Slot a copying lane reads: slots past the chunk's count read its last key
// (their scores are masked), so every lane issues the same copies. One unsigned
// minimum against a wave-uniform bound below 64 (count <= 64), which also tells
// the compiler that the slot fits the 24-bit multiplier.
__device__ __forceinline__ int32_t chunk_slot(int32_t s, int32_t count) {
  const uint32_t last = (uint32_t)(count > 1 ? count - 1 : 0) & 63u;
  const uint32_t u = (uint32_t)s;
  return (int32_t)(u < last ? u : last);
}

// ceil(65536 / n) for n = 0..64 (entry 0 unused).
__constant__ const uint32_t kNcMagic[65] = {
    0, 65536, 32768, 21846, 16384, 13108, 10923, 9363, 8192, 7282, 6554, 5958, 5462,
    5042, 4682, 4370, 4096, 3856, 3641, 3450, 3277, 3121, 2979, 2850, 2731, 2622,
    2521, 2428, 2341, 2260, 2185, 2115, 2048, 1986, 1928, 1873, 1821, 1772, 1725,
    1681, 1639, 1599, 1561, 1525, 1490, 1457, 1425, 1395, 1366, 1338, 1311, 1286,
    1261, 1237, 1214, 1192, 1171, 1150, 1130, 1111, 1093, 1075, 1058, 1041, 1024};

__device__ __forceinline__ int32_t div_magic(int32_t nc) { return kNcMagic[nc]; }

__device__ __forceinline__ Chunk make_chunk(int32_t base, int32_t nc, int32_t stride, int32_t count) {
  Chunk c;
  c.base = base;
  c.nc = nc;
  c.stride = stride;
  c.count = count;
  c.magic = div_magic(nc);
  c.mask = ~0u;
  return c;
}

// Contiguous run of count tokens starting at base.
__device__ __forceinline__ Chunk run_chunk(int32_t base, int32_t count) {
  return make_chunk(base, kChunk, kChunk, count);
}

__device__ __forceinline__ u32x4 ldg16(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ f32x16 mfma_bf16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 mfma_f32(float a, float b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

// Round to nearest even fp32 -> bf16 (hardware conversion on gfx950).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
  bf16x2 v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

// Cross-half exchange between lanes l and l ^ 32 with the gfx950 permlane32 swap:
// after swapping x with itself, operand 0 holds the lower half's values in every
// lane and operand 1 the upper half's. (The builtin exists only in the device
// pass; the host pass sees a placeholder and never runs it.)
struct HalfPair {
  float lo, hi;
};
__device__ __forceinline__ HalfPair halves(float x) {
#if defined(__HIP_DEVICE_COMPILE__)
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return HalfPair{__uint_as_float(r[0]), __uint_as_float(r[1])};
#else
  return HalfPair{x, x};
#endif
}
__device__ __forceinline__ float xor32(float x) {
  const HalfPair p = halves(x);
  return (threadIdx.x & 32) ? p.lo : p.hi;
}
__device__ __forceinline__ float max_halves(float x) {
  const HalfPair p = halves(x);
  return fmaxf(p.lo, p.hi);
}
__device__ __forceinline__ float sum_halves(float x) {
  const HalfPair p = halves(x);
  return p.lo + p.hi;
}

// Query fragments (B operand of S^T = K Q^T) for the lane's query row.
// bf16: step s holds d in [16 s + 8 half, +8). fp32: step s holds d = 2 s + half.
template <int D>
struct QFragBF16 {
  bf16x8 f[D / 16];
  __device__ __forceinline__ void load(const bf16_bits* row, int half) {
#pragma unroll
    for (int s = 0; s < D / 16; ++s) f[s] = as_bf16x8(ldg16(row + 16 * s + 8 * half));
  }
};

template <int D>
struct QFragF32 {
  float f[D / 2];
  __device__ __forceinline__ void load(const float* row, int half) {
#pragma unroll
    for (int s = 0; s < D / 2; ++s) f[s] = row[2 * s + half];
  }
};

// S^T for one 64-key chunk and the wave's 32 queries: st[kt] covers keys
// 32 kt .. 32 kt + 31 (rows) x 32 queries (columns). Key slots past the chunk's
// count load a valid token (slot 0) and must be masked by the caller.
template <int D>
__device__ __forceinline__ void chunk_scores(const bf16_bits* kplane, const Chunk& c,
                                             const QFragBF16<D>& q, int l32, int half,
                                             f32x16 st[2]) {
  const bf16_bits* krow[2];
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) {
    const int32_t s = 32 * kt + l32;
    krow[kt] = kplane + (int64_t)chunk_token(c, chunk_slot(s, c.count)) * D + 8 * half;
    st[kt] = zero16();
  }
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) st[kt] = mfma_bf16(as_bf16x8(ldg16(krow[kt] + 16 * s)), q.f[s], st[kt]);
  }
}

template <int D>
__device__ __forceinline__ void chunk_scores(const float* kplane, const Chunk& c,
                                             const QFragF32<D>& q, int l32, int half,
                                             f32x16 st[2]) {
  const float* krow[2];
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) {
    const int32_t s = 32 * kt + l32;
    krow[kt] = kplane + (int64_t)chunk_token(c, chunk_slot(s, c.count)) * D + half;
    st[kt] = zero16();
  }
#pragma unroll
  for (int s = 0; s < D / 2; ++s) {
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) st[kt] = mfma_f32(krow[kt][2 * s], q.f[s], st[kt]);
  }
}

// Key index (within the chunk) of accumulator register r of key tile kt.
__device__ __forceinline__ int key_of(int kt, int r, int half) {
  return 32 * kt + 8 * (r >> 2) + 4 * half + (r & 3);
}

// Blocks [first, end) in id order, each cut into bands of whole tile rows of at
// most KC keys (a block never shares a chunk with another block). Tiles must be
// at most KC tokens wide.
template <int KC>
struct BlockWalker {
  const GeoTable* G;
  int32_t l, tu, tv, r0, v, nb;
  Tile t;
  // walk blocks [first, end)
  __device__ __forceinline__ void start(const GeoTable* g, int32_t first, int32_t end) {
    G = g;
    nb = end;
    v = first;
    r0 = 0;
    if (v < nb) {
      l = block_scale(*G, v);
      const int32_t t0 = v - G->NB[l - 1];
      tu = (int32_t)div_by_magic((uint32_t)t0, G->mTw[l - 1]);
      tv = t0 - tu * G->Tw[l - 1];
      t = tile_at(*G, l, tu, tv);
    }
  }
  // Next chunk; `blk` is its block id and `last` tells whether it ends that block.
  __device__ __forceinline__ bool next(Chunk& c, int32_t& blk, bool& last) {
    if (v >= nb) return false;
    const int32_t rpc = KC / t.nc;  // t.nc <= block edge <= 64 = KC
    const int32_t rows = (t.nr - r0 < rpc) ? t.nr - r0 : rpc;
    c = make_chunk(t.base + r0 * t.stride, t.nc, t.stride, rows * t.nc);
    blk = v;
    r0 += rows;
    last = r0 >= t.nr;
    if (last) {
      ++v;
      r0 = 0;
      if (++tv == G->Tw[l - 1]) {
        tv = 0;
        if (++tu == G->Th[l - 1]) {
          tu = 0;
          ++l;
        }
      }
      if (v < nb) t = tile_at(*G, l, tu, tv);
    }
    return true;
  }
};

__device__ __forceinline__ int32_t swizzled_item(int32_t wg, int32_t n_wg, int32_t on) {
  if (!on) return wg;
  // Workgroups are dealt round-robin to the 8 XCDs; give each XCD a contiguous
  // range of items so neighbouring query tiles share that XCD's L2.
  const int32_t per = n_wg >> 3;  // n_wg is a multiple of 8 when swizzling
  return (wg & 7) * per + (wg >> 3);
}

// Uniform (wave-invariant) value hint.
__device__ __forceinline__ int32_t uniform(int32_t x) { return __builtin_amdgcn_readfirstlane(x); }

// Row r's 16-byte unit u lives at unit u ^ unit_swizzle(r) (bijection on 0..15).
// Sixteen consecutive rows read at one logical unit hit sixteen different
// units, and four consecutive rows x two adjacent units (a transposing read)
// hit eight different units.
__device__ __forceinline__ int unit_swizzle(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

typedef __attribute__((ext_vector_type(4))) short i16x4;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) void lds_void;

// 16-byte direct copy HBM -> LDS: lane i of the wave writes lds + 16 i (lds is
// wave-uniform). Kept out of lambdas: a target builtin inside a lambda voids the
// host-side instantiation of the kernel.
__device__ __forceinline__ void dma16(const void* g, char* lds) {
  __builtin_amdgcn_global_load_lds(g, (lds_void*)lds, 16, 0, 0);
}

// p points into __shared__ memory.
__device__ __forceinline__ i16x4 lds_read_tr(const char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(const_cast<char*>(p)));
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ int32_t wave_incl_scan(int32_t x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int32_t y = __shfl_up(x, off, 64);
    x += lane >= off ? y : 0;
  }
  return x;
}

// Exclusive prefix sum of x over the NT threads of the workgroup; total receives
// the sum. wt: NT / 64 ints of LDS. Holds barriers: every thread must call it.
template <int NT>
__device__ __forceinline__ int32_t block_excl_scan(int32_t x, int32_t* wt, int32_t& total) {
  constexpr int NW = NT / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t inc = wave_incl_scan(x);
  if (lane == 63) wt[wave] = inc;
  __syncthreads();
  int32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int32_t t = wt[w];
    before += w < wave ? t : 0;
    all += t;
  }
  __syncthreads();
  total = all;
  return before + inc - x;
}

// s_waitcnt immediate for "vmcnt <= n" (gfx9 encoding; expcnt and lgkmcnt left at max).
__host__ __device__ constexpr int waitcnt_vm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

}  // namespace sparvar

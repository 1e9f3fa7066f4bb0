// One key chunk of the attention core as functions over LDS-staged K/V tiles:
// fragment offsets, S^T = K Q^T, the exp2-domain softmax pieces and
// O^T += V^T P^T. The layout conventions are those of device_common.h (row-major
// K and V tiles of KC rows, 16-byte units XOR-swizzled by unit_swizzle).
#pragma once

#include "device_common.h"

namespace sparvar {

// Lane-constant LDS byte offsets of the MFMA fragments inside one stage.
// Key row r and r + 32 share the unit swizzle, so key tile kt adds 32 kt rows
// as an immediate offset.
template <int D, int KC>
struct FragOffsets {
  static constexpr int U = D / 8, kRow = D * 2, kTile = KC * kRow;
  int k_off[D / 16];
  int v_off[2][D / 32];
  __device__ __forceinline__ void init(int l32, int half, int lane) {
#pragma unroll
    for (int s2 = 0; s2 < D / 16; ++s2) k_off[s2] = l32 * kRow + 16 * ((2 * s2 + half) ^ (unit_swizzle(l32) & (U - 1)));
    const int tr_g = lane >> 4, tr_t = (lane & 15) >> 2, tr_q = lane & 3;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int key = 4 * half + 8 * p + tr_t;
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt)
        v_off[p][dt] = kTile + key * kRow +
                       16 * ((4 * dt + 2 * (tr_g & 1) + (tr_q >> 1)) ^ (unit_swizzle(key) & (U - 1))) + (tr_q & 1) * 8;
    }
  }
};

// S^T = K Q^T for one chunk held in LDS stage kst.
template <int D, int KC>
__device__ __forceinline__ void qk_chunk(const char* kst, const FragOffsets<D, KC>& f, const QFragBF16<D>& q,
                                         f32x16 (&st)[KC / 32]) {
#pragma unroll
  for (int kt = 0; kt < KC / 32; ++kt) st[kt] = zero16();
#pragma unroll
  for (int s2 = 0; s2 < D / 16; ++s2) {
#pragma unroll
    for (int kt = 0; kt < KC / 32; ++kt) {
      const u32x4 a = *reinterpret_cast<const u32x4*>(kst + f.k_off[s2] + kt * 32 * (D * 2));
      st[kt] = mfma_bf16(as_bf16x8(a), q.f[s2], st[kt]);
    }
  }
}

// O^T += V^T P^T for one chunk held in LDS stage kst (V at kst + kTile).
template <int D, int KC>
__device__ __forceinline__ void pv_chunk(const char* kst, const FragOffsets<D, KC>& f, const bf16x8 (&pf)[KC / 16],
                                         f32x16 (&acc)[D / 32]) {
  constexpr int kRow = D * 2;
#pragma unroll
  for (int ks = 0; ks < KC / 16; ++ks) {
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
      const i16x4 lo = lds_read_tr(kst + f.v_off[0][dt] + ks * 16 * kRow);
      const i16x4 hi = lds_read_tr(kst + f.v_off[1][dt] + ks * 16 * kRow);
      u32x4 av;
      av[0] = __builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 0, 1));
      av[1] = __builtin_bit_cast(uint32_t, __builtin_shufflevector(lo, lo, 2, 3));
      av[2] = __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 0, 1));
      av[3] = __builtin_bit_cast(uint32_t, __builtin_shufflevector(hi, hi, 2, 3));
      acc[dt] = mfma_bf16(as_bf16x8(av), pf[ks], acc[dt]);
    }
  }
}

// P = exp2(s * scale_log2 - m) packed to bf16 B-operand fragments; returns the lane's sum.
template <int KC>
__device__ __forceinline__ float exp_pack(const f32x16 (&st)[KC / 32], float scale_log2, float m,
                                          bf16x8 (&pf)[KC / 16]) {
  float ps = 0.f;
#pragma unroll
  for (int ks = 0; ks < KC / 16; ++ks) {
    u32x4 w;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(st[ks >> 1][8 * (ks & 1) + 2 * u], scale_log2, -m));
      const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(st[ks >> 1][8 * (ks & 1) + 2 * u + 1], scale_log2, -m));
      ps += p0;
      ps += p1;
      w[u] = pack_bf16x2(p0, p1);
    }
    pf[ks] = as_bf16x8(w);
  }
  return ps;
}

// Row maximum of a score chunk in the exp2 domain (both halves of the wave).
template <int KC>
__device__ __forceinline__ float row_max(const f32x16 (&st)[KC / 32], float scale_log2) {
  float mx = -INFINITY;
#pragma unroll
  for (int kt = 0; kt < KC / 32; ++kt)
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, st[kt][r]);
  return max_halves(mx) * scale_log2;
}

// Keys at or past count get -inf. The lane part of the key index (4 * half) is
// folded into the limit so that every comparison is against an immediate.
template <int KC>
__device__ __forceinline__ void mask_tail(f32x16 (&st)[KC / 32], int32_t count, int half) {
  const int32_t lim = count - 4 * half;
#pragma unroll
  for (int kt = 0; kt < KC / 32; ++kt)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (32 * kt + 8 * (r >> 2) + (r & 3) >= lim) st[kt][r] = -INFINITY;
}

}  // namespace sparvar

// KV compression: the memory side of SparVAR's "+ KV comp." setting (additional
// experiments, memory consumption paragraph), which keeps only the KV cache of
// the sink scales and of the local scales. kv_compact_kernel copies, for every
// (b, h) plane, the cache tokens of the kept scales, in scale order, into a
// compact cache: the cache of the schedule made of the kept scales. A plain
// HBM-bound gather of contiguous runs in 16-byte units.
#include "device_common.h"
#include "launch.h"

namespace sparvar {

struct KvCompactIO {
  const uint4* k_src;
  const uint4* v_src;
  uint4* k_dst;
  uint4* v_dst;
  int64_t src_stride, dst_stride;  // plane strides, 16-byte units
  int32_t n_keep;
  int32_t block0[kMaxScales + 1];  // first grid block of each kept scale; block0[n_keep] = blocks
  int32_t units[kMaxScales];       // 16-byte units of each kept scale
  int32_t dst_off[kMaxScales];     // its first unit in the compact plane
  int32_t src_off[kMaxScales];     // its first unit in the source plane
};

constexpr int kKvThreads = 256;
constexpr int kKvUnitsPerThread = 8;
constexpr int kKvUnitsPerBlock = kKvThreads * kKvUnitsPerThread;

// Grid: x walks the blocks of every kept scale, scale after scale (so a block's
// scale is uniform), y the (b, h) planes.
__global__ __launch_bounds__(kKvThreads) void kv_compact_kernel(KvCompactIO io) {
  // the block's kept scale, selected with constant indices (a runtime index into
  // the argument arrays would copy them to private memory)
  const int32_t bx = blockIdx.x;
  int32_t b0 = 0, units = io.units[0], so = io.src_off[0], dof = io.dst_off[0];
#pragma unroll
  for (int j = 1; j < kMaxScales; ++j) {
    if (j < io.n_keep && bx >= io.block0[j]) {
      b0 = io.block0[j];
      units = io.units[j];
      so = io.src_off[j];
      dof = io.dst_off[j];
    }
  }
  const int64_t plane = blockIdx.y;
  const uint4* ks = io.k_src + plane * io.src_stride + so;
  const uint4* vs = io.v_src + plane * io.src_stride + so;
  uint4* kd = io.k_dst + plane * io.dst_stride + dof;
  uint4* vd = io.v_dst + plane * io.dst_stride + dof;
  const int32_t u0 = (bx - b0) * kKvUnitsPerBlock + threadIdx.x;
  // all loads first (clamped into the scale, so none is conditional), then the
  // stores of the units inside it
  u32x4 kr[kKvUnitsPerThread], vr[kKvUnitsPerThread];
#pragma unroll
  for (int j = 0; j < kKvUnitsPerThread; ++j) {
    const int32_t u = u0 + j * kKvThreads;
    const int32_t uc = u < units ? u : units - 1;
    kr[j] = *reinterpret_cast<const u32x4*>(ks + uc);
    vr[j] = *reinterpret_cast<const u32x4*>(vs + uc);
  }
#pragma unroll
  for (int j = 0; j < kKvUnitsPerThread; ++j) {
    const int32_t u = u0 + j * kKvThreads;
    if (u < units) {
      *reinterpret_cast<u32x4*>(kd + u) = kr[j];
      *reinterpret_cast<u32x4*>(vd + u) = vr[j];
    }
  }
}

hipError_t launch_kv_compact(const KvCompactArgs& a, hipStream_t stream) {
  KvCompactIO io;
  const int32_t upt = a.d * a.elem / 16;  // units per token
  io.k_src = static_cast<const uint4*>(a.k_src);
  io.v_src = static_cast<const uint4*>(a.v_src);
  io.k_dst = static_cast<uint4*>(a.k_dst);
  io.v_dst = static_cast<uint4*>(a.v_dst);
  io.src_stride = a.src_bh_stride * a.elem / 16;
  io.dst_stride = a.dst_bh_stride * a.elem / 16;
  io.n_keep = a.n_keep;
  int32_t off = 0, blocks = 0;
  for (int i = 0; i < a.n_keep; ++i) {
    const int l = a.keep[i];
    io.units[i] = (a.G->C[l] - a.G->C[l - 1]) * upt;
    io.dst_off[i] = off;
    io.src_off[i] = a.G->C[l - 1] * upt;
    io.block0[i] = blocks;
    off += io.units[i];
    blocks += (io.units[i] + kKvUnitsPerBlock - 1) / kKvUnitsPerBlock;
  }
  io.block0[a.n_keep] = blocks;
  if (blocks == 0 || a.planes == 0) return hipSuccess;
  hipLaunchKernelGGL(kv_compact_kernel, dim3(blocks, a.planes), dim3(kKvThreads), 0, stream, io);
  return hipGetLastError();
}

}  // namespace sparvar

// Geometry of the multi-scale cache and its b x b tiling, usable on host and
// device. A GeoTable is built once on the host from sparvar_geometry_t and
// passed to kernels by value (kernel argument segment).
//
// Notation follows the paper: scales l = 1..L of h_l x w_l tokens,
// C_l = N_1 + ... + N_l (appendix, Decompose step). Tile edges e_h(l), e_w(l)
// equal b unless the scale is shorter than b along that axis, in which case the
// whole axis is one tile.
#pragma once

#include <stdint.h>

#include "sparvar.h"

#if defined(__HIPCC__)
#define SV_HD __host__ __device__ __forceinline__
#else
#define SV_HD inline
#endif

namespace sparvar {

constexpr int kMaxScales = SPARVAR_MAX_SCALES;

struct GeoTable {
  int32_t L;       // number of scales
  int32_t b;       // block edge
  int32_t n_sink;  // sink scales, clamped to [0, L]
  int32_t h[kMaxScales], w[kMaxScales];    // index l-1
  int32_t eh[kMaxScales], ew[kMaxScales];  // tile edges
  int32_t Th[kMaxScales], Tw[kMaxScales];  // tiles per axis
  int32_t C[kMaxScales + 1];               // C[l] = tokens of scales 1..l
  int32_t NB[kMaxScales + 1];              // NB[l] = blocks of scales 1..l
  uint32_t mTw[kMaxScales];                // ceil(2^32 / Tw): t / Tw == mulhi(t, mTw) for t * Tw < 2^32
};

// t / d for 0 <= t with t * d < 2^32, given m = ceil(2^32 / d) (d >= 1; m = 0 encodes d = 1).
SV_HD uint32_t div_by_magic(uint32_t t, uint32_t m) {
  return m == 0 ? t : (uint32_t)(((uint64_t)t * m) >> 32);
}

inline uint32_t magic_for(uint32_t d) {
  return d <= 1 ? 0u : (uint32_t)(((uint64_t(1) << 32) + d - 1) / d);
}

// A tile of the cache: tokens base + x * stride + y for x < nr, y < nc.
struct Tile {
  int32_t base, nr, nc, stride;
};

SV_HD int32_t tiles_of(const GeoTable& G, int l) { return G.Th[l - 1] * G.Tw[l - 1]; }

// Scale (1-based) holding block id v; v must be in [0, NB[L]).
SV_HD int block_scale(const GeoTable& G, int32_t v) {
  int l = 1;
  while (l < G.L && G.NB[l] <= v) ++l;
  return l;
}

SV_HD Tile tile_at(const GeoTable& G, int l, int32_t tu, int32_t tv) {
  const int32_t eh = G.eh[l - 1], ew = G.ew[l - 1], hl = G.h[l - 1], wl = G.w[l - 1];
  const int32_t r0 = tu * eh, c0 = tv * ew;
  Tile t;
  t.nr = (r0 + eh < hl ? r0 + eh : hl) - r0;
  t.nc = (c0 + ew < wl ? c0 + ew : wl) - c0;
  t.stride = wl;
  t.base = G.C[l - 1] + r0 * wl + c0;
  return t;
}

SV_HD Tile block_tile(const GeoTable& G, int32_t v) {
  const int l = block_scale(G, v);
  const int32_t t = v - G.NB[l - 1];
  const int32_t tu = (int32_t)div_by_magic((uint32_t)t, G.mTw[l - 1]);
  return tile_at(G, l, tu, t - tu * G.Tw[l - 1]);
}

// Query Block Homography along one axis (appendix): nearest source tile of the
// target tile's centre, rounding half up, in exact integers.
SV_HD int32_t homography(int32_t a, int32_t T_k, int32_t T_S) {
  return (int32_t)(((int64_t)(2 * a + 1) * T_S) / (2 * (int64_t)T_k));
}

// Decompose-Align-Project of block v from step S to step k (appendix,
// Relative Scale Alignment): l' = k - (S - l); the tile origin is projected by
// floor(x * h_l' / h_l), floor(y * w_l' / w_l); the result is the scale-l'
// tile containing the projected token.
SV_HD int32_t map_block(const GeoTable& G, int32_t v, int S, int k) {
  const int l = block_scale(G, v);
  const int lp = k - (S - l);
  const int32_t t = v - G.NB[l - 1];
  const int32_t tu = t / G.Tw[l - 1], tv = t % G.Tw[l - 1];
  const int64_t x = (int64_t)tu * G.eh[l - 1], y = (int64_t)tv * G.ew[l - 1];
  const int32_t xp = (int32_t)((x * G.h[lp - 1]) / G.h[l - 1]);
  const int32_t yp = (int32_t)((y * G.w[lp - 1]) / G.w[l - 1]);
  return G.NB[lp - 1] + (xp / G.eh[lp - 1]) * G.Tw[lp - 1] + (yp / G.ew[lp - 1]);
}

// Scale-(k-1) tile range [lo, hi] along one axis overlapping target tile a of
// scale k, widened by dil and clipped.
SV_HD void footprint(int32_t a, int32_t e_k, int32_t n_k, int32_t n_p, int32_t e_p, int32_t T_p,
                     int32_t dil, int32_t* lo, int32_t* hi) {
  const int64_t r0 = (int64_t)a * e_k;
  const int64_t r1 = (r0 + e_k < n_k) ? r0 + e_k : n_k;
  const int64_t plo = (r0 * n_p) / n_k;
  const int64_t phi = (r1 * n_p + n_k - 1) / n_k;  // exclusive, rounded up
  int32_t t0 = (int32_t)(plo / e_p) - dil;
  int32_t t1 = (int32_t)((phi - 1) / e_p) + dil;
  *lo = t0 < 0 ? 0 : t0;
  *hi = t1 > T_p - 1 ? T_p - 1 : t1;
}

// Covering form of Decompose-Align-Project (appendix, Spatial Projection applied
// token by token): the tile's tokens [x0, x1) of scale l span
// [x0 h_l'/h_l, x1 h_l'/h_l) on scale l' = k - (S - l), and every scale-l' tile
// overlapping that span (along both axes) is mapped: the box [r0, r1] x [c0, c1]
// of tiles of scale l'. The span is the footprint above, taken upwards.
struct CoverBox {
  int32_t base, Tw;    // first block id of scale l', tiles per row of scale l'
  int32_t r0, r1, c0, c1;
};

SV_HD CoverBox map_block_cover(const GeoTable& G, int32_t v, int S, int k) {
  const int l = block_scale(G, v);
  const int lp = k - (S - l);
  const int32_t t = v - G.NB[l - 1];
  const int32_t tu = t / G.Tw[l - 1], tv = t % G.Tw[l - 1];
  CoverBox b;
  b.base = G.NB[lp - 1];
  b.Tw = G.Tw[lp - 1];
  footprint(tu, G.eh[l - 1], G.h[l - 1], G.h[lp - 1], G.eh[lp - 1], G.Th[lp - 1], 0, &b.r0, &b.r1);
  footprint(tv, G.ew[l - 1], G.w[l - 1], G.w[lp - 1], G.ew[lp - 1], G.Tw[lp - 1], 0, &b.c0, &b.c1);
  return b;
}

SV_HD int32_t cover_size(const CoverBox& b) { return (b.r1 - b.r0 + 1) * (b.c1 - b.c0 + 1); }

// i-th block (ascending) of a cover box, i < cover_size(b).
SV_HD int32_t cover_entry(const CoverBox& b, int32_t i) {
  const int32_t wc = b.c1 - b.c0 + 1;
  return b.base + (b.r0 + i / wc) * b.Tw + b.c0 + i % wc;
}

// Largest cover box of any block of scales 1..S mapped to step k (host).
inline int32_t max_cover_size(const GeoTable& G, int S, int k) {
  int32_t mx = 1;
  for (int l = 1; l <= S; ++l) {
    const int lp = k - (S - l);
    int32_t mr = 0, mc = 0, lo, hi;
    for (int32_t t = 0; t < G.Th[l - 1]; ++t) {
      footprint(t, G.eh[l - 1], G.h[l - 1], G.h[lp - 1], G.eh[lp - 1], G.Th[lp - 1], 0, &lo, &hi);
      mr = hi - lo + 1 > mr ? hi - lo + 1 : mr;
    }
    for (int32_t t = 0; t < G.Tw[l - 1]; ++t) {
      footprint(t, G.ew[l - 1], G.w[l - 1], G.w[lp - 1], G.ew[lp - 1], G.Tw[lp - 1], 0, &lo, &hi);
      mc = hi - lo + 1 > mc ? hi - lo + 1 : mc;
    }
    mx = mr * mc > mx ? mr * mc : mx;
  }
  return mx;
}

// Parts of local row g of scale k (block form of the CSLA window):
// [0, n_sink_blocks) sinks; scale-(k-1) footprint tiles; scale-k window tiles.
struct LocalRow {
  int32_t n_sink_blocks;
  int32_t pr0, pr1, pc0, pc1;  // footprint tiles in scale k-1 (empty if pr1 < pr0)
  int32_t wr0, wr1, wc0, wc1;  // window tiles in scale k (empty if wr1 < wr0)
};

SV_HD LocalRow local_row(const GeoTable& G, int k, int32_t radius, int32_t dil, int32_t g) {
  LocalRow r;
  const int ns = G.n_sink;
  r.n_sink_blocks = G.NB[ns];
  const int32_t Tw = G.Tw[k - 1], Th = G.Th[k - 1];
  const int32_t a = g / Tw, c = g % Tw;
  r.pr0 = 0; r.pr1 = -1; r.pc0 = 0; r.pc1 = -1;
  if (k >= 2 && k - 1 > ns) {
    footprint(a, G.eh[k - 1], G.h[k - 1], G.h[k - 2], G.eh[k - 2], G.Th[k - 2], dil, &r.pr0, &r.pr1);
    footprint(c, G.ew[k - 1], G.w[k - 1], G.w[k - 2], G.ew[k - 2], G.Tw[k - 2], dil, &r.pc0, &r.pc1);
  }
  r.wr0 = 0; r.wr1 = -1; r.wc0 = 0; r.wc1 = -1;
  if (k > ns) {
    r.wr0 = a - radius < 0 ? 0 : a - radius;
    r.wr1 = a + radius > Th - 1 ? Th - 1 : a + radius;
    r.wc0 = c - radius < 0 ? 0 : c - radius;
    r.wc1 = c + radius > Tw - 1 ? Tw - 1 : c + radius;
  }
  return r;
}

SV_HD int32_t local_row_len(const LocalRow& r) {
  return r.n_sink_blocks + (r.pr1 - r.pr0 + 1) * (r.pc1 - r.pc0 + 1) +
         (r.wr1 - r.wr0 + 1) * (r.wc1 - r.wc0 + 1);
}

// i-th entry (ascending) of a local row.
SV_HD int32_t local_row_entry(const GeoTable& G, int k, const LocalRow& r, int32_t i) {
  if (i < r.n_sink_blocks) return i;
  i -= r.n_sink_blocks;
  const int32_t fc = r.pc1 - r.pc0 + 1;
  const int32_t nf = (r.pr1 - r.pr0 + 1) * fc;
  if (i < nf) return G.NB[k - 2] + (r.pr0 + i / fc) * G.Tw[k - 2] + r.pc0 + i % fc;
  i -= nf;
  const int32_t wc = r.wc1 - r.wc0 + 1;
  return G.NB[k - 1] + (r.wr0 + i / wc) * G.Tw[k - 1] + r.wc0 + i % wc;
}

}  // namespace sparvar

// tiles.h -- output-row tiles of the 3x3x3 conv kernels (tile -> rows, the
// staged input footprint, the XCD-aware tile order).  See Tiling in
// internal.h for the two modes.
#pragma once

#include "internal.h"

namespace pd {

// Row r (0..255) of tile `tile`: false if the row is outside the volume,
// else its padded output index (pidx) and its column j (col).  Also the LDS
// voxel of the row's (0,0,0) tap (lds_base) and the staging origin: the
// line-space index of staged voxel 0 (mode 0) or its padded index (mode 1).
// 32-bit voxel counts: the host guarantees max_batch * V < 2^31.  Divisions
// by the run-time sizes use the Tiling's precomputed multipliers (a plain
// integer division costs tens of instructions per lane, which small
// batches, with one tile per workgroup, pay in full).
__host__ __device__ inline bool tile_row(const Geom& g, const Tiling& tl, int tile, int r, int batch,
                                         long long* pidx, int* lds_base, long long* stage_origin,
                                         int* col = nullptr) {
  const int HH = g.H * g.H;
  if (tl.mode == 0) {
    const int seg = (int)fdiv((uint32_t)tile, tl.dv_tps);
    const int k0 = (tile - seg * tl.tiles_per_seg) * kTileRows;
    const int u0 = seg * (int)tl.seg_len + k0;
    const int b0 = (int)fdiv((uint32_t)u0, tl.dv_V);
    const int v0 = u0 - b0 * g.V;
    const int t0 = (int)fdiv((uint32_t)v0, tl.dv_HH), s0 = v0 - t0 * HH;
    const int i0 = (int)fdiv((uint32_t)s0, tl.dv_H);
    const long long l0 = line_index(g, b0, t0, i0, s0 - i0 * g.H);
    *stage_origin = l0 - (line_plane(g) + g.H + 1);
    const int u = u0 + r;
    if (k0 + r >= tl.seg_len || u >= batch * g.V) {
      *lds_base = 0;
      if (col) *col = -1;
      return false;
    }
    const int b = (int)fdiv((uint32_t)u, tl.dv_V);
    const int v = u - b * g.V;
    const int t = (int)fdiv((uint32_t)v, tl.dv_HH), s = v - t * HH;
    const int i = (int)fdiv((uint32_t)s, tl.dv_H), j = s - i * g.H;
    *pidx = padded_index(g, b, t, i, j);
    *lds_base = (int)(line_index(g, b, t, i, j) - l0);
    if (col) *col = j;
    return true;
  } else {
    const int per = tl.ntT * tl.ntI * tl.ntJ, ntij = tl.ntI * tl.ntJ;
    const int b = (int)fdiv((uint32_t)tile, tl.dv_per);
    const int rem = tile - b * per;
    const int tt = (int)fdiv((uint32_t)rem, tl.dv_ntij), rem2 = rem - tt * ntij;
    const int ti = (int)fdiv((uint32_t)rem2, tl.dv_ntj), tj = rem2 - ti * tl.ntJ;
    const int t0 = tt * tl.BT, i0 = ti * tl.BI, j0 = tj * tl.BJ;
    *stage_origin = (long long)b * g.S + (long long)t0 * g.P + (long long)i0 * g.Wp + j0;
    const int bij = tl.BI * tl.BJ;
    const int a = (int)fdiv((uint32_t)r, tl.dv_bij), ra = r - a * bij;
    const int c = (int)fdiv((uint32_t)ra, tl.dv_bj), e = ra - c * tl.BJ;
    const int t = t0 + a, i = i0 + c, j = j0 + e;
    const bool ok = (r < tl.BT * bij) && t < g.T && i < g.H && j < g.H;
    *lds_base = ok ? (a * (tl.BI + 2 * g.pad) + c) * (tl.BJ + 2 * g.pad) + e : 0;
    if (col) *col = ok ? j : -1;
    if (!ok) return false;
    *pidx = padded_index(g, b, t, i, j);
    return true;
  }
}

// Sample and grid coordinates (b, t, i, j) of row r of tile `tile`; false if
// the row is outside the volume.  32-bit arithmetic (max_batch * V < 2^31).
__host__ __device__ inline bool tile_row_coords(const Geom& g, const Tiling& tl, int tile, int r, int batch,
                                                int* b, int* t, int* i, int* j) {
  const int HH = g.H * g.H;
  if (tl.mode == 0) {
    const int seg = (int)fdiv((uint32_t)tile, tl.dv_tps);
    const int k0 = (tile - seg * tl.tiles_per_seg) * kTileRows;
    const int u = seg * (int)tl.seg_len + k0 + r;
    if (k0 + r >= tl.seg_len || u >= batch * g.V) return false;
    *b = (int)fdiv((uint32_t)u, tl.dv_V);
    const int v = u - *b * g.V;
    *t = (int)fdiv((uint32_t)v, tl.dv_HH);
    const int s = v - *t * HH;
    *i = (int)fdiv((uint32_t)s, tl.dv_H);
    *j = s - *i * g.H;
    return true;
  }
  const int per = tl.ntT * tl.ntI * tl.ntJ, ntij = tl.ntI * tl.ntJ;
  *b = (int)fdiv((uint32_t)tile, tl.dv_per);
  const int rem = tile - *b * per;
  const int tt = (int)fdiv((uint32_t)rem, tl.dv_ntij), rem2 = rem - tt * ntij;
  const int ti = (int)fdiv((uint32_t)rem2, tl.dv_ntj), tj = rem2 - ti * tl.ntJ;
  const int bij = tl.BI * tl.BJ;
  const int a = (int)fdiv((uint32_t)r, tl.dv_bij), ra = r - a * bij;
  const int c = (int)fdiv((uint32_t)ra, tl.dv_bj), e = ra - c * tl.BJ;
  *t = tt * tl.BT + a;
  *i = ti * tl.BI + c;
  *j = tj * tl.BJ + e;
  return r < tl.BT * bij && *t < g.T && *i < g.H && *j < g.H;
}

// Padded (t, i, j) of a box-mode tile's staging origin.
struct BoxOrigin {
  int t0, i0, j0;
};

__host__ __device__ inline BoxOrigin box_origin(const Geom& g, const Tiling& tl, long long origin) {
  BoxOrigin bo{0, 0, 0};
  if (tl.mode == 1) {
    const long long rem = origin % g.S;
    bo.t0 = (int)(rem / g.P);
    const int r2 = (int)(rem - (long long)bo.t0 * g.P);
    bo.i0 = r2 / g.Wp;
    bo.j0 = r2 - bo.i0 * g.Wp;
  }
  return bo;
}

// Global padded voxel of staged voxel vv (clamped to voxel 0, a zero halo
// voxel, when outside the batch or outside the sample's padded box).
__host__ __device__ inline long long staged_voxel(const Geom& g, const Tiling& tl, long long origin,
                                                  const BoxOrigin& bo, int vv, long long limit) {
  if (tl.mode == 0) {
    const long long p = line_to_padded(g, origin + vv);
    return (p < limit) ? p : 0;
  }
  const int bj2 = tl.BJ + 2 * g.pad, bij2 = (tl.BI + 2 * g.pad) * bj2;
  const int a = vv / bij2;
  const int rem = vv - a * bij2;
  const int c = rem / bj2;
  const int e = rem - c * bj2;
  if (bo.t0 + a >= g.T + 2 * g.pad || bo.i0 + c >= g.Wp || bo.j0 + e >= g.Wp) return 0;
  return origin + (long long)a * g.P + (long long)c * g.Wp + e;
}

// Tile handled by persistent workgroup `wg` at iteration `it`: the 8 XCDs
// receive workgroups round-robin, so workgroup wg runs on XCD wg % 8; each
// XCD gets a contiguous range of tiles (neighbouring tiles share halo voxels
// in its L2) and its workgroups stride through it.  -1 when done.
__host__ __device__ inline int tile_of(int wg, int nwg, int it, int ntiles) {
  const int xcd = wg & 7, k = wg >> 3, per_xcd_wg = nwg >> 3;
  const int per_xcd = (ntiles + 7) >> 3;
  const int idx = k + it * per_xcd_wg;
  if (idx >= per_xcd) return -1;
  const int t = xcd * per_xcd + idx;
  return t < ntiles ? t : -1;
}

// Staging source of a tile: its staging origin (see tile_row) and box origin.
struct StageSrc {
  long long origin;
  BoxOrigin bo;
};

// The staging source of tile `tile` (mode 1: the box origin in padded
// coordinates is the tile's first interior voxel, (t0, i0, j0) = (tt BT,
// ti BI, tj BJ), shifted by the halo).
__host__ __device__ inline StageSrc tile_source(const Geom& g, const Tiling& tl, int tile, int batch) {
  StageSrc src;
  long long p;
  int lb;
  tile_row(g, tl, tile, 0, batch, &p, &lb, &src.origin);
  src.bo = BoxOrigin{0, 0, 0};
  if (tl.mode == 1) {
    const int per = tl.ntT * tl.ntI * tl.ntJ, ntij = tl.ntI * tl.ntJ;
    const int b = (int)fdiv((uint32_t)tile, tl.dv_per);
    const int rem = tile - b * per;
    const int tt = (int)fdiv((uint32_t)rem, tl.dv_ntij), rem2 = rem - tt * ntij;
    const int ti = (int)fdiv((uint32_t)rem2, tl.dv_ntj), tj = rem2 - ti * tl.ntJ;
    src.bo = BoxOrigin{tt * tl.BT, ti * tl.BI, tj * tl.BJ};
  }
  return src;
}

// Global padded voxel of staged voxel vv; -1 when it is outside the batch or
// the sample's padded box (such voxels only feed rows that are discarded).
template <int MODE>
__host__ __device__ inline long long staged_voxel_fast(const Geom& g, const Tiling& tl, const StageSrc& src,
                                                       int vv, long long limit) {
  if constexpr (MODE == 0) {
    const uint32_t u = (uint32_t)(src.origin + vv);  // < 2^31 (host check)
    const uint32_t tp = fastdiv(u, tl.div_a);
    const uint32_t rem = u - tp * (uint32_t)tl.sa;
    const uint32_t ip = fastdiv(rem, tl.div_b);
    const uint32_t jj = rem - ip * (uint32_t)g.H;
    const long long p = (long long)tp * g.P + (long long)ip * g.Wp + jj + 1;
    return p < limit ? p : -1;
  } else {
  const int a = (int)fastdiv((uint32_t)vv, tl.div_a);
  const int rem = vv - a * tl.sa;
  const int c = (int)fastdiv((uint32_t)rem, tl.div_b);
  const int e = rem - c * tl.sb;
  if (src.bo.t0 + a >= g.T + 2 * g.pad || src.bo.i0 + c >= g.Wp || src.bo.j0 + e >= g.Wp) return -1;
  return src.origin + (long long)a * g.P + (long long)c * g.Wp + e;
  }
}

}  // namespace pd

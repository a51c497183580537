// Fused point filter: one streaming pass over all points.
//
// Per point (Alg. 1 keep loop with out-of-ROI rate zero): load x, y, z and
// the sweep id, move the point into the current frame (Eq. 6), find the
// candidate ROIs of its coarse BEV cell that admit its sweep, run the exact
// oriented-box test on those candidates only, quantise (Alg. 1 Voxelize:
// range check and voxel indices) and emit (voxel key, point index).
//
// Two phases keep the pass bandwidth-bound:
//   A. for every point of the thread: compensate, take an approximate cell
//      index (multiplication by the reciprocal voxel size; the cell
//      rectangles of the ROIs are padded by cell_pad voxels, more than the
//      approximation can be off), and issue all cell-mask loads back to back;
//   B. only for points whose cell has a candidate ROI (a few percent): the
//      exact test, the exact quantisation (correctly rounded division) and
//      the key.  The keep decision is therefore exactly the definition's.
// The tile's poses, budget masks, ROI records and frame offsets are staged
// in LDS.
//
// Kept points are written as (key, point index) pairs in point order: wave
// ballots give the rank inside a wave, LDS gives the rank inside the tile,
// and each persistent workgroup appends to its own region (its chunk of
// tiles' first point index onwards), so no workgroup waits on another: a
// chained scan across workgroups costs one memory round trip per
// predecessor when many publish together.  The regions are compacted for
// free by the first radix pass, which reads them in place using the per-
// workgroup counts and first-digit histograms left here.
//
// Layout: each thread owns G groups of 4 consecutive points; group g of
// thread t starts at point tile*T + 4*(t + 256 g), so each float4 load of a
// column is coalesced across the wave.
#include "launch.hpp"

namespace mmbev {

namespace {

struct FilterLds {
  uint32_t hist[kMaxPasses][kSortBins];
  float pose[kMaxPoseLds][12];
  float roi[6][kMaxLdsRois];  // cx, cy, cos, sin, ext_x, ext_y
  uint32_t bm[kMaxLdsBudgetWords];
  int64_t off[kMaxLdsFrames + 1];
  int32_t roff[kMaxLdsFrames + 1];
  uint32_t wave_tot[kFilterGroups][kWaves];
  uint32_t prefix, run;
  int32_t f0, f1, roi_lo, roi_n;
  int32_t off_lds, pose_lds, bm_lds, chunk_staged;
};

__device__ __forceinline__ int32_t tile_frame(const Config& c, const FilterLds& L, int64_t i) {
  if (L.f0 == L.f1) return L.f0;
  int32_t lo = L.f0, hi = L.f1;
  if (L.off_lds) {
    while (lo < hi) {
      int32_t mid = (lo + hi + 1) >> 1;
      if (L.off[mid - L.f0] <= i)
        lo = mid;
      else
        hi = mid - 1;
    }
  } else {
    while (lo < hi) {
      int32_t mid = (lo + hi + 1) >> 1;
      if (c.frame_off[mid] <= i)
        lo = mid;
      else
        hi = mid - 1;
    }
  }
  return lo;
}

__device__ __forceinline__ void load_pose(const Config& c, const FilterLds& L, int32_t b, uint32_t s, float* P) {
  if (L.pose_lds) {
    const float* src = L.pose[(b - L.f0) * c.S + s];
#pragma unroll
    for (int k = 0; k < 12; ++k) P[k] = src[k];
  } else {
    const float* src = c.poses + ((int64_t)b * c.S + s) * 12;
#pragma unroll
    for (int k = 0; k < 12; ++k) P[k] = src[k];
  }
}

__device__ __forceinline__ uint32_t budget_word(const Config& c, const FilterLds& L, int32_t b, uint32_t s, int w) {
  if (L.bm_lds) return L.bm[((b - L.f0) * c.S + s) * c.W + w];
  return c.budgetmask[((int64_t)b * c.S + s) * c.W + w];
}

__device__ __forceinline__ bool roi_hit(const Config& c, const FilterLds& L, int32_t gj, float px, float py) {
  const int32_t lj = gj - L.roi_lo;
  mmbev_roi_t r;
  if (L.roi_n >= 0 && lj >= 0 && lj < L.roi_n) {
    r.cx = L.roi[0][lj];
    r.cy = L.roi[1][lj];
    r.cos_yaw = L.roi[2][lj];
    r.sin_yaw = L.roi[3][lj];
    r.ext_x = L.roi[4][lj];
    r.ext_y = L.roi[5][lj];
  } else {
    r = c.rois[gj];
  }
  return inside_roi(r, px, py);
}

// Phase B: exact decision for a point with candidate ROIs, given p'.
__device__ __forceinline__ bool exact_keep(const Config& c, const FilterLds& L, int32_t b, uint32_t s, float px,
                                           float py, float pz, uint32_t cand, uint32_t& key) {
  int32_t ix, iy, iz;
  bool in = quantize_axis(px, c.mn[0], c.vs[0], c.Df[0], ix);
  in &= quantize_axis(py, c.mn[1], c.vs[1], c.Df[1], iy);
  in &= quantize_axis(pz, c.mn[2], c.vs[2], c.Df[2], iz);
  if (!in) return false;
  const int32_t r0 = L.off_lds ? L.roff[b - L.f0] : min(max(c.roi_off[b], 0), c.R);
  bool hit = false;
  if (c.W == 1) {
    uint32_t m = cand;
    while (m && !hit) {
      const int k = __builtin_ctz(m);
      m &= m - 1;
      hit = roi_hit(c, L, r0 + k, px, py);
    }
  } else {
    const int32_t cell = (iy >> c.cell_shift) * c.ncx + (ix >> c.cell_shift);
    const uint32_t* cm = c.cellmask + ((int64_t)b * c.ncells + cell) * c.W;
    for (int w = 0; w < c.W && !hit; ++w) {
      uint32_t m = cm[w] & budget_word(c, L, b, s, w);
      while (m && !hit) {
        const int k = __builtin_ctz(m);
        m &= m - 1;
        hit = roi_hit(c, L, r0 + w * 32 + k, px, py);
      }
    }
  }
  if (!hit) return false;
  const uint32_t kl = ((uint32_t)iz * c.Dy + (uint32_t)iy) * c.Dx + (uint32_t)ix;
  key = (c.key_has_frame && c.fb > 0) ? (((uint32_t)b << c.kb) | kl) : kl;
  return true;
}

// Point data of one tile held in registers: G groups of 4 points per thread.
template <int G>
struct TileData {
  float x[G][4], y[G][4], z[G][4];
  uint32_t s[G];  // four sweep ids per group, one byte each (0xff: no point)
};

template <int G, bool VEC>
__device__ __forceinline__ void load_tile(const Config& c, int64_t base, TileData<G>& d) {
  const int tid = threadIdx.x;
  const int64_t N = c.N;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int64_t i0 = base + 4 * (int64_t)(tid + kBlock * g);
    if (VEC && i0 + 3 < N) {
      const float4 x4 = *reinterpret_cast<const float4*>(c.feat + i0);
      const float4 y4 = *reinterpret_cast<const float4*>(c.feat + c.stride + i0);
      const float4 z4 = *reinterpret_cast<const float4*>(c.feat + 2 * c.stride + i0);
      d.s[g] = *reinterpret_cast<const uint32_t*>(c.sweep + i0);
      d.x[g][0] = x4.x; d.x[g][1] = x4.y; d.x[g][2] = x4.z; d.x[g][3] = x4.w;
      d.y[g][0] = y4.x; d.y[g][1] = y4.y; d.y[g][2] = y4.z; d.y[g][3] = y4.w;
      d.z[g][0] = z4.x; d.z[g][1] = z4.y; d.z[g][2] = z4.z; d.z[g][3] = z4.w;
    } else {
      d.s[g] = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t i = i0 + q;
        const bool ok = i < N;
        d.x[g][q] = ok ? c.feat[i] : 0.0f;
        d.y[g][q] = ok ? c.feat[c.stride + i] : 0.0f;
        d.z[g][q] = ok ? c.feat[2 * c.stride + i] : 0.0f;
        d.s[g] |= (ok ? (uint32_t)c.sweep[i] : 0xffu) << (8 * q);
      }
    }
  }
}

// Frame/ROI range of LDS staging (thread 0), from tile info of [t0, t1].
__device__ __forceinline__ void plan_staging(const Config& c, FilterLds& L, const TileInfo& a, const TileInfo& b) {
  const int32_t f0 = a.f0, f1 = max(b.f1, a.f0);
  const int32_t nf = f1 - f0 + 1;
  L.f0 = f0;
  L.f1 = f1;
  L.off_lds = nf <= kMaxLdsFrames;
  L.pose_lds = nf * c.S <= kMaxPoseLds;
  L.bm_lds = nf * c.S * c.W <= kMaxLdsBudgetWords;
  L.roi_lo = a.r_lo;
  const int32_t r_hi = max(b.r_hi, a.r_lo);
  L.roi_n = (r_hi - a.r_lo <= kMaxLdsRois) ? r_hi - a.r_lo : -1;
}

__device__ __forceinline__ void do_staging(const Config& c, FilterLds& L) {
  const int tid = threadIdx.x;
  const int32_t nf = L.f1 - L.f0 + 1;
  if (L.off_lds)
    for (int e = tid; e <= nf; e += kBlock) {
      L.off[e] = c.frame_off[L.f0 + e];
      L.roff[e] = min(max(c.roi_off[L.f0 + e], 0), c.R);
    }
  if (L.pose_lds)
    for (int e = tid; e < nf * c.S * 12; e += kBlock) (&L.pose[0][0])[e] = c.poses[(int64_t)L.f0 * c.S * 12 + e];
  if (L.bm_lds)
    for (int e = tid; e < nf * c.S * c.W; e += kBlock) L.bm[e] = c.budgetmask[(int64_t)L.f0 * c.S * c.W + e];
  if (L.roi_n > 0)
    for (int e = tid; e < L.roi_n; e += kBlock) {
      const mmbev_roi_t r = c.rois[L.roi_lo + e];
      L.roi[0][e] = r.cx;
      L.roi[1][e] = r.cy;
      L.roi[2][e] = r.cos_yaw;
      L.roi[3][e] = r.sin_yaw;
      L.roi[4][e] = r.ext_x;
      L.roi[5][e] = r.ext_y;
    }
}

// Keep test of one tile already in registers; kept pairs appended to this
// workgroup's region at out_base + L.run, in point order.
template <int G>
__device__ __forceinline__ void process_tile(const Config& c, FilterLds& L, int64_t base, TileData<G>& d,
                                             uint32_t out_base) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int64_t N = c.N;
  // phase A: p' (overwrites the raw coordinates) and the candidate cell, or -1
  int32_t cidx[G][4];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int64_t i0 = base + 4 * (int64_t)(tid + kBlock * g);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t s = (d.s[g] >> (8 * q)) & 0xffu;
      cidx[g][q] = -1;
      if (s < (uint32_t)c.S && i0 + q < N) {
        const int32_t b = tile_frame(c, L, i0 + q);
        float P[12];
        load_pose(c, L, b, s, P);
        float px, py, pz;
        compensate(P, d.x[g][q], d.y[g][q], d.z[g][q], px, py, pz);
        d.x[g][q] = px;
        d.y[g][q] = py;
        d.z[g][q] = pz;
        const float fx = (px - c.mn[0]) * c.inv_vs[0];
        const float fy = (py - c.mn[1]) * c.inv_vs[1];
        const float fz = (pz - c.mn[2]) * c.inv_vs[2];
        const bool near = fx >= -2.0f && fx < c.Df[0] + 2.0f && fy >= -2.0f && fy < c.Df[1] + 2.0f &&
                          fz >= -2.0f && fz < c.Df[2] + 2.0f;
        if (near) {
          const int32_t ax = min(max((int32_t)floorf(fx), 0), (int32_t)c.Dx - 1) >> c.cell_shift;
          const int32_t ay = min(max((int32_t)floorf(fy), 0), (int32_t)c.Dy - 1) >> c.cell_shift;
          cidx[g][q] = b * c.ncells + ay * c.ncx + ax;
        }
      }
    }
  }
  // all cell-mask loads of the thread in flight together (always in bounds)
  uint32_t cand[G][4];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int q = 0; q < 4; ++q) cand[g][q] = c.cellany[max(cidx[g][q], 0)];

  // phase B: exact test for points with candidates
  uint32_t keys[G][4];
  uint32_t keepm[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int64_t i0 = base + 4 * (int64_t)(tid + kBlock * g);
    keepm[g] = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      keys[g][q] = 0;
      uint32_t m = cidx[g][q] >= 0 ? cand[g][q] : 0u;
      if (m) {
        const uint32_t s = (d.s[g] >> (8 * q)) & 0xffu;
        const int32_t b = tile_frame(c, L, i0 + q);
        if (c.W == 1) m &= budget_word(c, L, b, s, 0);
        if (m && exact_keep(c, L, b, s, d.x[g][q], d.y[g][q], d.z[g][q], m, keys[g][q])) keepm[g] |= 1u << q;
      }
    }
  }

  // rank of each kept point inside the tile: order (group, wave, lane, q)
  uint32_t excl[G];
  const uint64_t lt = lanemask_lt();
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint32_t cnt = __popc(keepm[g]);
    const uint64_t b0 = __ballot(cnt & 1u), b1 = __ballot(cnt & 2u), b2 = __ballot(cnt & 4u);
    excl[g] = __popcll(b0 & lt) + 2u * __popcll(b1 & lt) + 4u * __popcll(b2 & lt);
    if (lane == 0) L.wave_tot[g][wave] = __popcll(b0) + 2u * __popcll(b1) + 4u * __popcll(b2);
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t run = 0;
    for (int g = 0; g < G; ++g)
      for (int w = 0; w < kWaves; ++w) {
        const uint32_t t = L.wave_tot[g][w];
        L.wave_tot[g][w] = run;
        run += t;
      }
    L.prefix = L.run;
    L.run += run;
  }
  __syncthreads();

  const uint32_t dmask = (1u << c.dbits) - 1u;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    uint32_t pos = out_base + L.prefix + L.wave_tot[g][wave] + excl[g];
    const int64_t i0 = base + 4 * (int64_t)(tid + kBlock * g);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (keepm[g] & (1u << q)) {
        c.keys[0][pos] = keys[g][q];
        c.vals[0][pos] = (uint32_t)(i0 + q);
        ++pos;
        uint64_t comp = keys[g][q];
        if (!c.key_has_frame) comp |= (uint64_t)tile_frame(c, L, i0 + q) << c.kb;
        atomicAdd(&L.hist[0][comp & dmask], 1u);  // first radix pass: this chunk's digit counts
      }
    }
  }
}

// Persistent: workgroup w owns the contiguous tiles
// [w*chunk_tiles, (w+1)*chunk_tiles) and appends its kept pairs to its own
// region starting at point index w*chunk_tiles*T, so no workgroup ever waits
// on another.  The next tile's points are loaded while the current one is
// processed.  Per workgroup it leaves the number of kept pairs and their
// digit counts for the first radix pass.
template <int G, bool VEC>
__global__ __launch_bounds__(kBlock) void filter_kernel(Config c) {
  constexpr int kTile = kBlock * 4 * G;
  __shared__ FilterLds L;
  const int tid = threadIdx.x;
  const int64_t t_begin = (int64_t)blockIdx.x * c.filter_chunk_tiles;
  const int64_t t_end = min(t_begin + (int64_t)c.filter_chunk_tiles, (int64_t)c.filter_tiles);
  const uint32_t out_base = blockIdx.x * (uint32_t)c.filter_chunk_points;
  const uint32_t nbins = 1u << c.dbits;

  for (int e = tid; e < kSortBins; e += kBlock) L.hist[0][e] = 0;
  if (tid == 0) {
    L.run = 0;
    L.chunk_staged = 0;
    if (t_begin < t_end) {
      const TileInfo a = c.tinfo[t_begin], b = c.tinfo[t_end - 1];
      plan_staging(c, L, a, b);
      L.chunk_staged = L.off_lds && L.pose_lds && L.bm_lds && L.roi_n >= 0;
    }
  }
  __syncthreads();
  if (L.chunk_staged) do_staging(c, L);

  TileData<G> cur, nxt;
  if (t_begin < t_end) load_tile<G, VEC>(c, t_begin * kTile, cur);
  for (int64_t t = t_begin; t < t_end; t += 2) {
    // tile t (in cur), prefetching t+1 into nxt; then tile t+1, prefetching t+2
    __syncthreads();
    if (!L.chunk_staged) {
      if (tid == 0) plan_staging(c, L, c.tinfo[t], c.tinfo[t]);
      __syncthreads();
      do_staging(c, L);
      __syncthreads();
    }
    if (t + 1 < t_end) load_tile<G, VEC>(c, (t + 1) * kTile, nxt);
    process_tile<G>(c, L, t * kTile, cur, out_base);
    if (t + 1 >= t_end) break;
    __syncthreads();
    if (!L.chunk_staged) {
      if (tid == 0) plan_staging(c, L, c.tinfo[t + 1], c.tinfo[t + 1]);
      __syncthreads();
      do_staging(c, L);
      __syncthreads();
    }
    if (t + 2 < t_end) load_tile<G, VEC>(c, (t + 2) * kTile, cur);
    process_tile<G>(c, L, (t + 1) * kTile, nxt, out_base);
  }
  __syncthreads();
  if (tid == 0) c.fcount[blockIdx.x] = L.run;
  for (uint32_t e = tid; e < nbins; e += kBlock) c.cnt[(int64_t)e * gridDim.x + blockIdx.x] = L.hist[0][e];
}

template <int G>
hipError_t launch_g(const Config& c, hipStream_t st) {
  if (c.vec)
    hipLaunchKernelGGL((filter_kernel<G, true>), dim3(c.filter_grid), dim3(kBlock), 0, st, c);
  else
    hipLaunchKernelGGL((filter_kernel<G, false>), dim3(c.filter_grid), dim3(kBlock), 0, st, c);
  return hipGetLastError();
}

}  // namespace

hipError_t filter_occupancy(int groups, int vec, int* per_cu) {
  const void* k = nullptr;
  switch (groups) {
    case 1: k = vec ? (const void*)filter_kernel<1, true> : (const void*)filter_kernel<1, false>; break;
    case 2: k = vec ? (const void*)filter_kernel<2, true> : (const void*)filter_kernel<2, false>; break;
    default: k = vec ? (const void*)filter_kernel<4, true> : (const void*)filter_kernel<4, false>; break;
  }
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(per_cu, k, kBlock, 0);
}

hipError_t launch_filter(const Config& c, hipStream_t st) {
  switch (c.filter_groups) {
    case 1: return launch_g<1>(c, st);
    case 2: return launch_g<2>(c, st);
    default: return launch_g<4>(c, st);
  }
}

}  // namespace mmbev

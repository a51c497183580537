// Fused point filter: one streaming pass over all points.
//
// Per point (Alg. 1 keep loop with out-of-ROI rate zero): load x, y, z and
// the sweep id, move the point into the current frame (Eq. 6), find the
// candidate ROIs of its coarse BEV cell that admit its sweep, run the exact
// oriented-box test on those candidates only, quantise (Alg. 1 Voxelize:
// range check and voxel indices) and emit (voxel key, point index).
//
// Two phases keep the pass bandwidth-bound:
//   A. for every point of the thread: p' (exact), an approximate cell index
//      (multiplication by the reciprocal voxel size; the cell rectangles of
//      the ROIs are padded by cell_pad voxels, more than the approximation
//      can be off), and all cell-mask loads issued back to back;
//   B. only for points whose cell has a candidate ROI that admits their
//      sweep (a few percent): queued in LDS in point order, then handled
//      densely, all lanes busy: exact quantisation (the correctly rounded
//      quotient's floor, decided by a reciprocal product unless that lies
//      too close to an integer), the exact box test and the key.  The keep
//      decision is therefore exactly the definition's.
// The chunk's poses, budget masks, ROI records and frame offsets are staged
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
// Per tile the order is: phase A (its cell-mask loads issued last), the
// next tile's point loads, phase B; waiting for the cell masks then leaves
// the next tile's loads in flight while phase B runs.  Loads complete in
// order, so phase B reads nothing from global memory on the common path.
//
// Layout: each thread owns G groups of 4 consecutive points; group g of
// thread t starts at point tile*T + 4*(t + 256 g), so each float4 load of a
// column is coalesced across the wave.
#include "launch.hpp"

namespace mmbev {

namespace {

struct alignas(16) FilterLds {
  float pose[kMaxPoseLds][12];  // 48-byte rows: three aligned 16-byte reads each
  uint32_t hist[kSortBins];     // first radix pass digit counts of this chunk
  float roi[6][kMaxLdsRois];  // cx, cy, cos, sin, ext_x, ext_y
  uint32_t bm[kMaxLdsBudgetWords];
  uint32_t off[kMaxLdsFrames + 1];  // point frame offsets clamped to [0, N]
  int32_t roff[kMaxLdsFrames + 1];
  uint32_t wave_tot[kFilterGroups][kWaves];
  uint32_t round_cnt[2][kWaves];  // kept pairs per wave of a phase-B round
  int32_t f0, f1, roi_lo, roi_n;
  int32_t off_lds, pose_lds, bm_lds, chunk_staged;
};

// ST: everything the chunk needs (frame and ROI offsets, poses, budget
// masks, ROI records) is staged in LDS, so every lookup below is a plain LDS
// read.  Without ST each lookup checks whether its table is staged for the
// current tile and reads global memory otherwise.
template <bool ST>
__device__ __forceinline__ int32_t tile_frame(const Config& c, const FilterLds& L, uint32_t i) {
  if (L.f0 == L.f1) return L.f0;
  int32_t lo = L.f0, hi = L.f1;
  if (ST || L.off_lds) {
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
      if (c.frame_off[mid] <= (int64_t)i)
        lo = mid;
      else
        hi = mid - 1;
    }
  }
  return lo;
}

template <bool ST>
__device__ __forceinline__ void load_pose(const Config& c, const FilterLds& L, int32_t b, uint32_t s, float* P) {
  if (ST || L.pose_lds) {
    const float* src = L.pose[(b - L.f0) * c.S + s];
#pragma unroll
    for (int k = 0; k < 12; ++k) P[k] = src[k];
  } else {
    const float* src = c.poses + ((int64_t)b * c.S + s) * 12;
#pragma unroll
    for (int k = 0; k < 12; ++k) P[k] = src[k];
  }
}

template <bool ST>
__device__ __forceinline__ uint32_t budget_word(const Config& c, const FilterLds& L, int32_t b, uint32_t s, int w) {
  if (ST || L.bm_lds) return L.bm[((b - L.f0) * c.S + s) * c.W + w];
  return c.budgetmask[((int64_t)b * c.S + s) * c.W + w];
}

template <bool ST>
__device__ __forceinline__ bool roi_hit(const Config& c, const FilterLds& L, int32_t gj, float px, float py) {
  int32_t lj = gj - L.roi_lo;
  mmbev_roi_t r;
  if (ST || (L.roi_n >= 0 && lj >= 0 && lj < L.roi_n)) {
    if (ST) lj = min(max(lj, 0), L.roi_n - 1);  // in range unless the ROI offsets are invalid
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

// Voxel index of one axis, identical to quantize_axis (correctly rounded
// (p - min) / v, then the range check and truncation): the product with the
// reciprocal voxel size is within 3 ulps of the rounded quotient, so when no
// integer lies within 16 ulps of it (or 2^-60 of zero) its floor is the
// quotient's floor and decides both the range check and the index; otherwise
// the division is done.  Non-finite products always take the division.
__device__ __forceinline__ bool quantize_axis_fast(float p, float mn, float vs, float inv_vs, float Df, int32_t& i) {
  const float t = p - mn;
  const float q = t * inv_vs;
  const float m = fma_rn(fabsf(q), 0x1p-20f, 0x1p-60f);
  const float lo = floorf(q - m), hi = floorf(q + m);
  if (lo == hi) {
    const bool ok = lo >= 0.0f && lo < Df;
    i = ok ? (int32_t)lo : 0;
    return ok;
  }
  return quantize_axis(p, mn, vs, Df, i);
}

// Phase B: exact decision for a point with candidate ROIs, given p'.
template <bool ST>
__device__ __forceinline__ bool exact_keep(const Config& c, const FilterLds& L, int32_t b, uint32_t s, float px,
                                           float py, float pz, uint32_t cand, uint32_t& key) {
  int32_t ix, iy, iz;
  bool in = quantize_axis_fast(px, c.mn[0], c.vs[0], c.inv_vs[0], c.Df[0], ix);
  in &= quantize_axis_fast(py, c.mn[1], c.vs[1], c.inv_vs[1], c.Df[1], iy);
  in &= quantize_axis_fast(pz, c.mn[2], c.vs[2], c.inv_vs[2], c.Df[2], iz);
  if (!in) return false;
  const int32_t r0 = (ST || L.off_lds) ? L.roff[b - L.f0] : min(max(c.roi_off[b], 0), c.R);
  bool hit = false;
  if (c.W == 1) {
    uint32_t m = cand;
    while (m && !hit) {
      const int k = __builtin_ctz(m);
      m &= m - 1;
      hit = roi_hit<ST>(c, L, r0 + k, px, py);
    }
  } else {
    const int32_t cell = (iy >> c.cell_shift) * c.ncx + (ix >> c.cell_shift);
    const uint32_t* cm = c.cellmask + ((int64_t)b * c.ncells + cell) * c.W;
    for (int w = 0; w < c.W && !hit; ++w) {
      uint32_t m = cm[w] & budget_word<ST>(c, L, b, s, w);
      while (m && !hit) {
        const int k = __builtin_ctz(m);
        m &= m - 1;
        hit = roi_hit<ST>(c, L, r0 + w * 32 + k, px, py);
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

// A full tile with 16-byte loads: exactly four loads per group, so the
// compiler's wait counts stay exact across the loop.
template <int G>
__device__ __forceinline__ void load_tile_vec(const Config& c, int64_t base, TileData<G>& d) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int64_t i0 = base + 4 * (int64_t)(tid + kBlock * g);
    const float4 x4 = *reinterpret_cast<const float4*>(c.feat + i0);
    const float4 y4 = *reinterpret_cast<const float4*>(c.feat + c.stride + i0);
    const float4 z4 = *reinterpret_cast<const float4*>(c.feat + 2 * c.stride + i0);
    d.s[g] = *reinterpret_cast<const uint32_t*>(c.sweep + i0);
    d.x[g][0] = x4.x; d.x[g][1] = x4.y; d.x[g][2] = x4.z; d.x[g][3] = x4.w;
    d.y[g][0] = y4.x; d.y[g][1] = y4.y; d.y[g][2] = y4.z; d.y[g][3] = y4.w;
    d.z[g][0] = z4.x; d.z[g][1] = z4.y; d.z[g][2] = z4.z; d.z[g][3] = z4.w;
  }
}

// Any tile, point by point (points past N get sweep 0xff: no point).
template <int G>
__device__ __forceinline__ void load_tile_scalar(const Config& c, int64_t base, TileData<G>& d) {
  const int tid = threadIdx.x;
  const int64_t N = c.N;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int64_t i0 = base + 4 * (int64_t)(tid + kBlock * g);
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
      L.off[e] = (uint32_t)min(max(c.frame_off[L.f0 + e], (int64_t)0), (int64_t)c.N);
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

// Approximate grid cell of (x', y') for the candidate lookup, or -1 when the
// point is clearly outside the grid.  fx = x' * (1/v) - min/v is within a
// small fraction of a voxel of the exact (x' - min) / v; the cell rectangles
// of the ROIs are padded by cell_pad voxels, so a point the exact test keeps
// always finds its ROI here.
__device__ __forceinline__ int32_t approx_cell(const Config& c, int32_t b, float px, float py) {
  const int32_t ix = (int32_t)fma_rn(px, c.inv_vs[0], c.nmin_v[0]);
  const int32_t iy = (int32_t)fma_rn(py, c.inv_vs[1], c.nmin_v[1]);
  const bool ok = (uint32_t)(ix + c.cell_pad) < (uint32_t)c.Dx + 2u * (uint32_t)c.cell_pad &&
                  (uint32_t)(iy + c.cell_pad) < (uint32_t)c.Dy + 2u * (uint32_t)c.cell_pad;
  const int32_t ax = min(max(ix, 0), (int32_t)c.Dx - 1) >> c.cell_shift;
  const int32_t ay = min(max(iy, 0), (int32_t)c.Dy - 1) >> c.cell_shift;
  return ok ? b * c.ncells + ay * c.ncx + ax : -1;
}

// Candidate queue of one tile segment, in point order.
struct FilterQueue {
  uint32_t idx[kFilterQueue];
  uint32_t cand[kFilterQueue];  // candidate-ROI word (W == 1) or 1
  uint32_t fs[kFilterQueue];    // frame << 8 | sweep
  float px[kFilterQueue];       // compensated point (Eq. 6), exact
  float py[kFilterQueue];
  float pz[kFilterQueue];
};

// Per-point state of a tile between its two phases.
template <int G>
struct TileState {
  float px[G][4], py[G][4], pz[G][4];  // p' (Eq. 6), exact
  uint32_t fs[G][4];                   // frame << 8 | sweep
  uint32_t cand[G][4];                 // candidate-ROI word after phase A (0: none)
};

// Phase A of a tile already in registers: p' of every point and the
// issue of its cell-mask load.  The loads are left in flight; the caller
// issues the next tile's loads behind them and phase B waits for them.
template <int G, bool ST>
__device__ __forceinline__ void phase_a(const Config& c, const FilterLds& L, uint32_t base, const TileData<G>& d,
                                        TileState<G>& st) {
  const int tid = threadIdx.x;
  const uint32_t N = (uint32_t)c.N;
  const uint32_t S = (uint32_t)c.S;
  int32_t cidx[G][4];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint32_t i0 = base + 4u * (uint32_t)(tid + kBlock * g);
    uint32_t sq[4];
    int32_t fr[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      fr[q] = tile_frame<ST>(c, L, i0 + q);
      sq[q] = (d.s[g] >> (8 * q)) & 0xffu;
      st.fs[g][q] = ((uint32_t)fr[q] << 8) | sq[q];
    }
    const uint32_t pk = (uint32_t)fr[0] * S + sq[0];
    const bool lane_uniform = i0 + 3 < N && sq[0] < S && sq[1] == sq[0] && sq[2] == sq[0] && sq[3] == sq[0] &&
                              fr[3] == fr[0] && (ST || L.pose_lds);
    const uint32_t pk0 = __builtin_amdgcn_readfirstlane(pk);
    if (__ballot(!lane_uniform || pk != pk0) == 0) {
      // one pose for the whole wave, read as three 16-byte rows
      const int32_t row = (int32_t)pk0 - L.f0 * (int32_t)S;
      const float4 r0 = *reinterpret_cast<const float4*>(&L.pose[row][0]);
      const float4 r1 = *reinterpret_cast<const float4*>(&L.pose[row][4]);
      const float4 r2 = *reinterpret_cast<const float4*>(&L.pose[row][8]);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        st.px[g][q] = fma_rn(r0.x, d.x[g][q], fma_rn(r0.y, d.y[g][q], fma_rn(r0.z, d.z[g][q], r0.w)));
        st.py[g][q] = fma_rn(r1.x, d.x[g][q], fma_rn(r1.y, d.y[g][q], fma_rn(r1.z, d.z[g][q], r1.w)));
        st.pz[g][q] = fma_rn(r2.x, d.x[g][q], fma_rn(r2.y, d.y[g][q], fma_rn(r2.z, d.z[g][q], r2.w)));
        cidx[g][q] = approx_cell(c, fr[q], st.px[g][q], st.py[g][q]);
      }
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        cidx[g][q] = -1;
        st.px[g][q] = st.py[g][q] = st.pz[g][q] = 0.0f;
        if (sq[q] < S && i0 + q < N) {
          float P[12];
          load_pose<ST>(c, L, fr[q], sq[q], P);
          compensate(P, d.x[g][q], d.y[g][q], d.z[g][q], st.px[g][q], st.py[g][q], st.pz[g][q]);
          cidx[g][q] = approx_cell(c, fr[q], st.px[g][q], st.py[g][q]);
        }
      }
    }
  }
  // all cell-mask loads of the thread in flight together (always in bounds)
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t w = c.cellany[max(cidx[g][q], 0)];
      st.cand[g][q] = cidx[g][q] >= 0 ? w : 0u;
    }
}

// Phase B of a tile: budget masks, queue of the candidates in point order
// and, segment by segment of the queue with all lanes busy, the exact
// quantisation and box test and the key; kept pairs are appended in queue
// (= point) order to this workgroup's region at out_base + run.  `round`
// counts the compaction rounds of the workgroup (their LDS counts are
// double-buffered, so one barrier per round suffices).
template <int G, bool ST>
__device__ __forceinline__ void phase_b(const Config& c, FilterLds& L, FilterQueue& Q, uint32_t base,
                                        TileState<G>& st, uint32_t out_base, uint32_t& run, uint32_t& round) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  if (c.W == 1) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (st.cand[g][q])
          st.cand[g][q] &= budget_word<ST>(c, L, (int32_t)(st.fs[g][q] >> 8), st.fs[g][q] & 0xffu, 0);
  }

  // queue positions of the candidates: (group, wave, lane, q) order
  const uint64_t lt = lanemask_lt();
  uint32_t excl[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint32_t n = (st.cand[g][0] != 0) + (st.cand[g][1] != 0) + (st.cand[g][2] != 0) + (st.cand[g][3] != 0);
    const uint64_t b0 = __ballot(n & 1u), b1 = __ballot(n & 2u), b2 = __ballot(n & 4u);
    excl[g] = __popcll(b0 & lt) + 2u * __popcll(b1 & lt) + 4u * __popcll(b2 & lt);
    if (lane == 0) L.wave_tot[g][wave] = __popcll(b0) + 2u * __popcll(b1) + 4u * __popcll(b2);
  }
  __syncthreads();
  uint32_t nq = 0;
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t t = L.wave_tot[g][w];
      if (w == wave) excl[g] += nq;
      nq += t;
    }

  const uint32_t dmask = (1u << c.dbits) - 1u;
  for (uint32_t seg = 0; seg < nq; seg += kFilterQueue) {
    if (seg > 0) __syncthreads();  // previous segment consumed
#pragma unroll
    for (int g = 0; g < G; ++g) {
      uint32_t pos = excl[g];
      const uint32_t i0 = base + 4u * (uint32_t)(tid + kBlock * g);
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (st.cand[g][q]) {
          if (pos - seg < (uint32_t)kFilterQueue) {
            const uint32_t e = pos - seg;
            Q.idx[e] = i0 + q;
            Q.cand[e] = st.cand[g][q];
            Q.fs[e] = st.fs[g][q];
            Q.px[e] = st.px[g][q];
            Q.py[e] = st.py[g][q];
            Q.pz[e] = st.pz[g][q];
          }
          ++pos;
        }
    }
    __syncthreads();
    const uint32_t n = min((uint32_t)kFilterQueue, nq - seg);
    for (uint32_t r0 = 0; r0 < n; r0 += kBlock) {
      const uint32_t e = r0 + tid;
      bool keep = false;
      uint32_t key = 0, i = 0;
      int32_t b = 0;
      if (e < n) {
        i = Q.idx[e];
        const uint32_t fs = Q.fs[e];
        b = (int32_t)(fs >> 8);
        keep = exact_keep<ST>(c, L, b, fs & 0xffu, Q.px[e], Q.py[e], Q.pz[e], Q.cand[e], key);
      }
      const uint64_t kbits = __ballot(keep);
      uint32_t* cnt = L.round_cnt[round & 1u];
      if (lane == 0) cnt[wave] = __popcll(kbits);
      __syncthreads();
      uint32_t before = run, total = 0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const uint32_t t = cnt[w];
        if (w < wave) before += t;
        total += t;
      }
      run += total;
      ++round;
      if (keep) {
        const uint32_t pos = out_base + before + __popcll(kbits & lt);
        c.keys[0][pos] = key;
        c.vals[0][pos] = i;
        uint64_t comp = key;
        if (!c.key_has_frame) comp |= (uint64_t)b << c.kb;
        atomicAdd(&L.hist[comp & dmask], 1u);  // first radix pass: this chunk's digit counts
      }
    }
  }
}

// Stage the tables of tile t alone (chunks that do not fit LDS as a whole).
__device__ __forceinline__ void stage_tile(const Config& c, FilterLds& L, int64_t t) {
  if (threadIdx.x == 0) plan_staging(c, L, c.tinfo[t], c.tinfo[t]);
  __syncthreads();
  do_staging(c, L);
  __syncthreads();
}

// The tiles [t_begin, t_end) of one workgroup.  Full tiles go through a
// two-deep register pipeline with 16-byte loads; the last tile of the input,
// when partial (or every tile, when the rows do not allow 16-byte loads),
// is loaded point by point without prefetch.
template <int G, bool VEC, bool ST>
__device__ __forceinline__ void run_chunk(const Config& c, FilterLds& L, FilterQueue& Q, int64_t t_begin,
                                          int64_t t_end, uint32_t out_base, uint32_t& run, uint32_t& round) {
  constexpr int kTile = kBlock * 4 * G;
  TileData<G> cur, nxt;
  TileState<G> st;
  const int64_t t_full = VEC ? max(t_begin, min(t_end, (int64_t)c.N / kTile)) : t_begin;
  if (t_begin < t_full) load_tile_vec<G>(c, t_begin * kTile, cur);
  for (int64_t t = t_begin; t < t_full; t += 2) {
    // tile t (in cur) with tile t+1 loading into nxt behind its cell-mask
    // loads; then tile t+1 with tile t+2 loading into cur.  Past the last
    // full tile the load repeats that tile (cache hits, values unused), which
    // keeps the number of loads in flight the same on every path.
    __syncthreads();
    if (!ST) stage_tile(c, L, t);
    phase_a<G, ST>(c, L, (uint32_t)(t * kTile), cur, st);
    load_tile_vec<G>(c, min(t + 1, t_full - 1) * kTile, nxt);
    phase_b<G, ST>(c, L, Q, (uint32_t)(t * kTile), st, out_base, run, round);
    if (t + 1 >= t_full) break;
    __syncthreads();
    if (!ST) stage_tile(c, L, t + 1);
    phase_a<G, ST>(c, L, (uint32_t)((t + 1) * kTile), nxt, st);
    load_tile_vec<G>(c, min(t + 2, t_full - 1) * kTile, cur);
    phase_b<G, ST>(c, L, Q, (uint32_t)((t + 1) * kTile), st, out_base, run, round);
  }
  for (int64_t t = t_full; t < t_end; ++t) {
    __syncthreads();
    if (!ST) stage_tile(c, L, t);
    load_tile_scalar<G>(c, t * kTile, cur);
    phase_a<G, ST>(c, L, (uint32_t)(t * kTile), cur, st);
    phase_b<G, ST>(c, L, Q, (uint32_t)(t * kTile), st, out_base, run, round);
  }
}

// Persistent: workgroup w owns the contiguous tiles
// [w*chunk_tiles, (w+1)*chunk_tiles) and appends its kept pairs to its own
// region starting at point index w*chunk_tiles*T, so no workgroup ever waits
// on another.  Per workgroup it leaves the number of kept pairs and their
// digit counts for the first radix pass.
template <int G, bool VEC>
__global__ __launch_bounds__(kBlock) void filter_kernel(Config c) {
  __shared__ FilterLds L;
  __shared__ FilterQueue Q;
  const int tid = threadIdx.x;
  const int64_t t_begin = (int64_t)blockIdx.x * c.filter_chunk_tiles;
  const int64_t t_end = min(t_begin + (int64_t)c.filter_chunk_tiles, (int64_t)c.filter_tiles);
  const uint32_t out_base = blockIdx.x * (uint32_t)c.filter_chunk_points;
  const uint32_t nbins = 1u << c.dbits;

  for (int e = tid; e < kSortBins; e += kBlock) L.hist[e] = 0;
  if (tid == 0) {
    L.chunk_staged = 0;
    if (t_begin < t_end) {
      const TileInfo a = c.tinfo[t_begin], b = c.tinfo[t_end - 1];
      plan_staging(c, L, a, b);
      L.chunk_staged = L.off_lds && L.pose_lds && L.bm_lds && L.roi_n >= 0;
    }
  }
  __syncthreads();
  uint32_t run = 0, round = 0;
  if (__builtin_amdgcn_readfirstlane(L.chunk_staged)) {
    do_staging(c, L);
    run_chunk<G, VEC, true>(c, L, Q, t_begin, t_end, out_base, run, round);
  } else {
    run_chunk<G, VEC, false>(c, L, Q, t_begin, t_end, out_base, run, round);
  }
  __syncthreads();
  if (tid == 0) c.fcount[blockIdx.x] = run;
  for (uint32_t e = tid; e < nbins; e += kBlock) c.cnt[(int64_t)e * gridDim.x + blockIdx.x] = L.hist[e];
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
    default: k = vec ? (const void*)filter_kernel<2, true> : (const void*)filter_kernel<2, false>; break;
  }
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(per_cu, k, kBlock, 0);
}

hipError_t launch_filter(const Config& c, hipStream_t st) {
  switch (c.filter_groups) {
    case 1: return launch_g<1>(c, st);
    default: return launch_g<2>(c, st);
  }
}

}  // namespace mmbev

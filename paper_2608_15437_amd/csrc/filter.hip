// Fused point filter: one streaming pass over all points.
//
// Per point (Alg. 1 keep loop with out-of-ROI rate zero): load x, y, z and
// the sweep id, move the point into the current frame (Eq. 6), find the
// candidate ROIs of its coarse BEV cell that admit its sweep, run the exact
// oriented-box test on those candidates only, quantise (Alg. 1 Voxelize:
// range check) and mark the point kept in its chunk's bitmap.
//
// Two phases keep the pass bandwidth-bound:
//   A. for every point of a lane: p' (exact), an approximate cell index
//      (multiplication by the reciprocal voxel size; the cell rectangles of
//      the ROIs are padded by cell_pad voxels, more than the approximation
//      can be off) and the cell's candidate-ROI word, read from the LDS copy
//      of the frame's cell map;
//   B. only for points whose cell has a candidate ROI that admits their
//      sweep (a few percent): appended with their p' to the wave's queue in
//      LDS and, 64 at a time with every lane busy, decided exactly: exact
//      quantisation (the correctly rounded quotient's floor, decided by a
//      reciprocal product unless that lies too close to an integer), the
//      exact box test and the key.  The keep decision is therefore exactly
//      the definition's.
//
// Wave k of the grid owns filter chunk k: a contiguous run of at most
// fchunk_points points inside one frame (the chunk table and the frame of
// every workgroup are laid out by the staging kernel, or, when the call's
// frames and tables are small enough, by every workgroup for itself before
// it stages its frame's tables into LDS from the poses, ROIs and budgets
// directly, so that no staging kernel runs).  The waves of a
// workgroup share the LDS copy of their frame's poses, budget masks, ROI
// records, ROI offsets and cell map (staged once, behind the only workgroup
// barrier) and are otherwise independent: a wave marks its kept points in
// its own LDS bitmap and writes it, with the kept count, once at the end of
// its chunk.  Nothing waits on another wave: a chained scan across
// workgroups costs one memory round trip per predecessor when many publish
// together, and workgroup barriers leave the waves without candidates idle.
// The compaction lists each chunk's kept points from its bitmap.
//
// Per wave tile (256 points, four consecutive points per lane, one 16-byte
// load per column and lane) the only global loads are the tile's own: vector
// memory loads complete in order, so a wait for a dependent global load (a
// cell word, say) would also wait for every tile loaded before it.  Phases A
// and B read only LDS and registers on the common path, and the next tile's
// loads stay in flight while a tile is handled.  The point loads are
// non-temporal: the points are read once.
#include "launch.hpp"

namespace mmbev {

namespace {

// Tables of the workgroup's frames f0..f1 (one frame unless the point
// offsets are invalid: a frame's chunks fill whole workgroups), staged once
// and shared by its waves.  The poses, ROI records, budget masks and cell
// words go to the dynamic LDS, sized for the call (one frame's sweeps, ROIs
// and cells), so that a workgroup takes no more LDS than its frame needs.
struct alignas(16) FilterLds {
  int32_t roff[kMaxLdsFrames + 1];  // ROI offsets clamped to [0, R]
  int32_t f0, f1, roi_lo, roi_n;
  int32_t chunk_staged;
};

// Dynamic LDS: pose rows [c.lds_pose_cap][12] (48-byte rows: three aligned
// 16-byte reads each), then the ROI records as six rows of c.lds_roi_cap
// (cx, cy, cos, sin, ext_x, ext_y), then c.lds_bm_cap budget-mask words, then
// rows of c.ncells + 1 words per frame: a zero word, read for points outside
// the grid, then the candidate-ROI word of every coarse cell.
extern __shared__ float4 filter_dyn[];

__device__ __forceinline__ const float* lds_pose(int32_t row) {
  return reinterpret_cast<const float*>(filter_dyn) + row * 12;
}
__device__ __forceinline__ float* lds_roi(const Config& c, int k) {
  return reinterpret_cast<float*>(filter_dyn) + c.lds_roi + k * c.lds_roi_cap;
}
__device__ __forceinline__ uint32_t* lds_bm(const Config& c) {
  return reinterpret_cast<uint32_t*>(filter_dyn) + c.lds_bm;
}

// Per-wave state in LDS: the candidate queue (a ring) and the kept bitmap
// of the wave's chunk.
struct WaveLds {
  uint32_t pk[kWaveQueue];    // point offset in the chunk | sweep << 16 | drawn out-of-ROI << 24
  uint32_t cand[kWaveQueue];  // candidate-ROI word (W == 1) or the cell's any-word
  float px[kWaveQueue];       // p' (Eq. 6), exact
  float py[kWaveQueue];
  float pz[kWaveQueue];
  uint32_t bits[kChunkWords];  // bit j: point lo + j of the chunk is kept
};

// Orders the LDS accesses of one wave (its lanes' writes before the other
// lanes' reads, and reads before later writes to the same slots).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ST: everything the workgroup needs (ROI offsets, poses, budget masks, ROI
// records) is staged in LDS, so every lookup below is a plain LDS read
// (ST == 2: the cells' ROI words too, when a frame has several).  Without ST
// (0) every lookup reads global memory.
template <int ST>
__device__ __forceinline__ void load_pose(const Config& c, const FilterLds& L, int32_t b, uint32_t s, float* P) {
  if (ST) {
    const float* src = lds_pose((b - L.f0) * c.S + s);
#pragma unroll
    for (int k = 0; k < 12; ++k) P[k] = src[k];
  } else {
    const float* src = c.poses + ((int64_t)b * c.S + s) * 12;
#pragma unroll
    for (int k = 0; k < 12; ++k) P[k] = src[k];
  }
}

template <int ST>
__device__ __forceinline__ uint32_t budget_word(const Config& c, const FilterLds& L, int32_t b, uint32_t s, int w) {
  if (ST) return lds_bm(c)[((b - L.f0) * c.S + s) * c.W + w];
  return c.budgetmask[((int64_t)b * c.S + s) * c.W + w];
}

template <int ST>
__device__ __forceinline__ int32_t frame_roi_base(const Config& c, const FilterLds& L, int32_t b) {
  if (ST) return L.roff[b - L.f0];
  return min(max(c.roi_off[b], 0), c.R);
}

template <int ST>
__device__ __forceinline__ bool roi_hit(const Config& c, const FilterLds& L, int32_t gj, float px, float py) {
  mmbev_roi_t r;
  if (ST) {
    const int32_t lj = min(max(gj - L.roi_lo, 0), max(L.roi_n - 1, 0));  // in range unless the ROI offsets are invalid
    r.cx = lds_roi(c, 0)[lj];
    r.cy = lds_roi(c, 1)[lj];
    r.cos_yaw = lds_roi(c, 2)[lj];
    r.sin_yaw = lds_roi(c, 3)[lj];
    r.ext_x = lds_roi(c, 4)[lj];
    r.ext_y = lds_roi(c, 5)[lj];
  } else {
    r = c.rois[gj];
  }
  return inside_roi(r, px, py);
}

// Voxel indices of p', identical to quantize_axis on each axis (correctly
// rounded (p - min) / v, then the range check and truncation).  The product
// with the reciprocal voxel size is within 3 ulps of the rounded quotient,
// so when no integer lies within 16 ulps of it (or 2^-60 of zero) its floor
// is the quotient's floor and decides both the range check and the index.
// Only the axes where an integer is that close (and non-finite products)
// take the division, behind a branch the whole wave skips when no lane
// needs it (inside it, a select: no per-lane branch).
__device__ __forceinline__ bool quantize_fast(const Config& c, float px, float py, float pz, int32_t& ix,
                                              int32_t& iy, int32_t& iz) {
  const float p[3] = {px, py, pz};
  float f[3];
  bool amb[3];
#pragma unroll
  for (int d = 0; d < 3; ++d) {
    const float q = (p[d] - c.mn[d]) * c.inv_vs[d];
    const float m = fma_rn(fabsf(q), 0x1p-20f, 0x1p-60f);
    const float lo = floorf(q - m);
    amb[d] = !(lo == floorf(q + m));
    f[d] = lo;
  }
  if (__ballot(amb[0] || amb[1] || amb[2])) {
#pragma unroll
    for (int d = 0; d < 3; ++d) {
      const float exact = (p[d] - c.mn[d]) / c.vs[d];
      f[d] = amb[d] ? exact : f[d];
    }
  }
  const bool ok = f[0] >= 0.0f && f[0] < c.Df[0] && f[1] >= 0.0f && f[1] < c.Df[1] && f[2] >= 0.0f &&
                  f[2] < c.Df[2];
  ix = ok ? (int32_t)f[0] : 0;
  iy = ok ? (int32_t)f[1] : 0;
  iz = ok ? (int32_t)f[2] : 0;
  return ok;
}

// Phase B, at most 32 ROIs per frame: whether a point with candidate-ROI
// word cand (0 for a lane without a point) lies in one of them, each lane
// walking its own bits and stopping at its first hit.  (A loop shared by the
// wave, one broadcast read per distinct ROI, measured slower: most lanes hit
// their first ROI.)
template <int ST>
__device__ __forceinline__ bool roi_test_one_word(const Config& c, const FilterLds& L, int32_t r0, uint32_t cand,
                                                  float px, float py) {
  bool hit = false;
  uint32_t m = cand;
  while (m && !hit) {
    const int k = __builtin_ctz(m);
    m &= m - 1;
    hit = roi_hit<ST>(c, L, r0 + k, px, py);
  }
  return hit;
}

// Phase B, more than 32 ROIs per frame: the ROIs of the point's cell that
// admit its sweep, word by word, tested lane by lane.
template <int ST>
__device__ __forceinline__ bool roi_test_words(const Config& c, const FilterLds& L, int32_t b, uint32_t s,
                                               int32_t r0, int32_t ix, int32_t iy, float px, float py) {
  const int32_t cell = (iy >> c.cell_shift) * c.ncx + (ix >> c.cell_shift);
  bool hit = false;
  if (ST == 2) {  // the word masks the filter built in LDS
    const uint32_t* cm = reinterpret_cast<const uint32_t*>(filter_dyn) + c.lds_wmask + cell * c.W;
    for (int w = 0; w < c.W && !hit; ++w) {
      uint32_t m = cm[w] & budget_word<ST>(c, L, b, s, w);
      while (m && !hit) {
        const int k = __builtin_ctz(m);
        m &= m - 1;
        hit = roi_hit<ST>(c, L, r0 + w * 32 + k, px, py);
      }
    }
    return hit;
  }
  const uint32_t* cm = c.cellmask + ((int64_t)b * c.ncells + cell) * c.W;
  for (int w = 0; w < c.W && !hit; ++w) {
    uint32_t m = cm[w] & budget_word<ST>(c, L, b, s, w);
    while (m && !hit) {
      const int k = __builtin_ctz(m);
      m &= m - 1;
      hit = roi_hit<ST>(c, L, r0 + w * 32 + k, px, py);
    }
  }
  return hit;
}

// Four consecutive points of one lane held in registers.
struct Quad {
  float x[4], y[4], z[4];
  uint32_t s;  // four sweep ids, one byte each (0xff: no point)
};

// The x, y, z and sweep rows from the first point of a wave's full tiles:
// wave-uniform bases, so that a tile's loads take a 32-bit lane offset.
struct TileRows {
  const float* x;
  const float* y;
  const float* z;
  const uint8_t* s;
};

__device__ __forceinline__ TileRows tile_rows(const Config& c, uint32_t a0) {
  return TileRows{c.feat + a0, c.feat + c.stride + a0, c.feat + 2 * c.stride + a0, c.sweep + a0};
}

// Four points with 16-byte loads (point offset off from the rows' first
// point, below kMaxChunkPoints): exactly four loads per lane, so the
// compiler's wait counts stay exact across the loop.  The loads are
// non-temporal: the points are read once, and streaming them through the
// caches would evict (and force the write-back of) the working set of the
// kernels around the filter.
typedef float StreamF4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void load_quad_vec(const TileRows& r, uint32_t off, Quad& d) {
  const uint32_t byte = off * 4u;
  const StreamF4 x4 =
      __builtin_nontemporal_load(reinterpret_cast<const StreamF4*>(reinterpret_cast<const char*>(r.x) + byte));
  const StreamF4 y4 =
      __builtin_nontemporal_load(reinterpret_cast<const StreamF4*>(reinterpret_cast<const char*>(r.y) + byte));
  const StreamF4 z4 =
      __builtin_nontemporal_load(reinterpret_cast<const StreamF4*>(reinterpret_cast<const char*>(r.z) + byte));
  d.s = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(r.s + off));
  d.x[0] = x4.x; d.x[1] = x4.y; d.x[2] = x4.z; d.x[3] = x4.w;
  d.y[0] = y4.x; d.y[1] = y4.y; d.y[2] = y4.z; d.y[3] = y4.w;
  d.z[0] = z4.x; d.z[1] = z4.y; d.z[2] = z4.z; d.z[3] = z4.w;
}

// Any four points, one by one; those at or past `end` get sweep 0xff.
__device__ __forceinline__ void load_quad_scalar(const Config& c, uint32_t i0, uint32_t end, Quad& d) {
  // every load unconditional, at a clamped index (end > 0 at every call):
  // a load behind a condition would be waited for before the next one
  float x[4], y[4], z[4];
  uint32_t sw[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t i = min(i0 + q, end - 1u);
    x[q] = c.feat[i];
    y[q] = c.feat[c.stride + i];
    z[q] = c.feat[2 * c.stride + i];
    sw[q] = c.sweep[i];
  }
  d.s = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const bool ok = i0 + q < end;
    d.x[q] = ok ? x[q] : 0.0f;
    d.y[q] = ok ? y[q] : 0.0f;
    d.z[q] = ok ? z[q] : 0.0f;
    d.s |= (ok ? sw[q] : 0xffu) << (8 * q);
  }
}

// The staging plan of a workgroup: frames f0..f1 of its chunks, their ROI
// range, and whether every table fits LDS (from the ROI offsets of f0 and
// f1 + 1).  Every thread computes it from the same loads.
struct StagePlan {
  int32_t f0, f1, roi_lo, roi_n;
  bool staged;
};

__device__ __forceinline__ StagePlan make_plan(const Config& c, int32_t f0, int32_t f1, int32_t ro0, int32_t ro1) {
  StagePlan p;
  const int32_t nf = f1 - f0 + 1;
  p.f0 = f0;
  p.f1 = f1;
  p.roi_lo = min(max(ro0, 0), c.R);
  p.roi_n = min(max(ro1, p.roi_lo), c.R) - p.roi_lo;
  p.staged = nf <= kMaxLdsFrames && nf * c.S <= c.lds_pose_cap && nf * c.S * c.W <= c.lds_bm_cap &&
             p.roi_n <= c.lds_roi_cap && nf * (c.ncells + 1) <= c.lds_cell_cap;
  return p;
}

// The tables of the workgroup's frame f0 (the caps make a staged plan one
// frame: f1 == f0): ROI offsets, poses, budget masks, ROI records and cell
// words, every load of a thread issued before the first LDS store, so that
// they take one round trip together.
__device__ __forceinline__ void do_staging(const Config& c, FilterLds& L, const StagePlan& pl) {
  static_assert(kMaxLdsBudgetWords <= kBlock && kMaxLdsRois <= kBlock, "one budget word and ROI record per thread");
  constexpr int kPoseRegs = (kMaxPoseLds * 12 + kBlock - 1) / kBlock;
  constexpr int kCellRegs = (kMaxLdsCells + kBlock - 1) / kBlock;
  const int tid = threadIdx.x;
  const int32_t f = pl.f0;
  const int np = c.S * 12, nbm = c.S * c.W, nroi = pl.roi_n, ncell = c.ncells;
  // loads (4-byte: the caller's arrays need only natural alignment)
  const int32_t roff = c.roi_off[f + min(tid, 1)];  // every lane (in bounds): no branch around the load
  float pv[kPoseRegs];
  const float* poses = c.poses + (int64_t)f * np;
#pragma unroll
  for (int j = 0; j < kPoseRegs; ++j) pv[j] = tid + j * kBlock < np ? poses[tid + j * kBlock] : 0.0f;
  const uint32_t bm = tid < nbm ? c.budgetmask[(int64_t)f * nbm + tid] : 0u;
  float rv[6] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
  if (tid < nroi) {
    const mmbev_roi_t& r = c.rois[pl.roi_lo + tid];
    rv[0] = r.cx;
    rv[1] = r.cy;
    rv[2] = r.cos_yaw;
    rv[3] = r.sin_yaw;
    rv[4] = r.ext_x;
    rv[5] = r.ext_y;
  }
  uint32_t cv[kCellRegs];
  const uint32_t* cells = c.cellany + (int64_t)f * ncell;
#pragma unroll
  for (int j = 0; j < kCellRegs; ++j) cv[j] = tid + j * kBlock < ncell ? cells[tid + j * kBlock] : 0u;
  // stores
  uint32_t* dyn = reinterpret_cast<uint32_t*>(filter_dyn);
  if (tid < 2) L.roff[tid] = min(max(roff, 0), c.R);
  float* dynf = reinterpret_cast<float*>(filter_dyn);
#pragma unroll
  for (int j = 0; j < kPoseRegs; ++j)
    if (tid + j * kBlock < np) dynf[tid + j * kBlock] = pv[j];  // pose rows from word 0
  if (tid < nbm) dyn[c.lds_bm + tid] = bm;
  if (tid < nroi)
#pragma unroll
    for (int k = 0; k < 6; ++k) dynf[c.lds_roi + k * c.lds_roi_cap + tid] = rv[k];
  // the frame's cell row: a zero word (points outside the grid), then the cells
  if (tid == 0) dyn[c.lds_cell] = 0u;
#pragma unroll
  for (int j = 0; j < kCellRegs; ++j)
    if (tid + j * kBlock < ncell) dyn[c.lds_cell + 1 + tid + j * kBlock] = cv[j];
}

// Approximate coarse cell of (x', y') inside its frame for the candidate
// lookup, or -1 when the point is clearly outside the grid.  fx = x' * (1/v) - min/v is within a
// small fraction of a voxel of the exact (x' - min) / v; the cell rectangles
// of the ROIs are padded by cell_pad voxels, so a point the exact test keeps
// always finds its ROI here.
// The constants of approx_cell, held in vector registers for the whole tile
// loop: the loop's scalar registers run out (the compiler then spills them
// to vector lanes and reads them back on every use), and an instruction
// reads at most one scalar operand, so a scalar addend costs a move anyway.
// With them, the wave's frame row in the staged tables (fr = b - f0) and
// the LDS word index of its cell words, so that the tile loop does not read
// the workgroup's first frame back from LDS.
struct CellConsts {
  float inv_x, inv_y, nmin_x, nmin_y;
  int32_t pad, span_x, span_y, max_x, max_y, shift, ncx;
  int32_t cell_row;  // staged: word index of frame fr's first cell word in the dynamic LDS
  int32_t fr;        // staged: b - f0
};

template <int ST>
__device__ __forceinline__ CellConsts cell_consts(const Config& c, const FilterLds& L, int32_t b) {
  const int32_t fr = ST ? b - L.f0 : 0;
  CellConsts k{c.inv_vs[0], c.inv_vs[1], c.nmin_v[0], c.nmin_v[1], c.cell_pad,
               (int32_t)c.Dx + 2 * c.cell_pad, (int32_t)c.Dy + 2 * c.cell_pad, (int32_t)c.Dx - 1,
               (int32_t)c.Dy - 1, c.cell_shift, c.ncx, c.lds_cell + fr * (c.ncells + 1) + 1, fr};
  asm volatile("" : "+v"(k.inv_x), "+v"(k.inv_y), "+v"(k.nmin_x), "+v"(k.nmin_y), "+v"(k.pad), "+v"(k.span_x),
               "+v"(k.span_y), "+v"(k.max_x), "+v"(k.max_y), "+v"(k.shift), "+v"(k.ncx), "+v"(k.cell_row));
  return k;
}

// v into [0, hi] in one instruction (the compiler forms the median only for
// constant bounds).
__device__ __forceinline__ uint32_t clamp0(int32_t v, int32_t hi) {
  int32_t r;
  asm("v_med3_i32 %0, %1, 0, %2" : "=v"(r) : "v"(v), "v"(hi));
  return (uint32_t)r;
}

static_assert(kMaxCellSide < (1 << 24), "cell coordinates fit the 24-bit multiply");

__device__ __forceinline__ int32_t approx_cell(const CellConsts& k, float px, float py) {
  const int32_t ix = (int32_t)fma_rn(px, k.inv_x, k.nmin_x);
  const int32_t iy = (int32_t)fma_rn(py, k.inv_y, k.nmin_y);
  const bool ok = (uint32_t)(ix + k.pad) < (uint32_t)k.span_x && (uint32_t)(iy + k.pad) < (uint32_t)k.span_y;
  const uint32_t ax = clamp0(ix, k.max_x) >> k.shift;
  const uint32_t ay = clamp0(iy, k.max_y) >> k.shift;
  uint32_t cell = __umul24(ay, (uint32_t)k.ncx) + ax;
  asm volatile("" : "+v"(cell));  // a select, not a branch around three instructions
  return ok ? (int32_t)cell : -1;
}

// Per-lane state of four points between their two phases.
struct QuadState {
  float px[4], py[4], pz[4];  // p' (Eq. 6), exact
  uint32_t s;                 // the four sweep ids, one byte each
  uint32_t cand[4];           // candidate-ROI word after phase A (0: none); with one ROI word, budget applied
  uint32_t bg;                // bit q: point q is drawn for the out-of-ROI keep
};

// Phase A of four points of a lane (first index i0, frame b for the whole
// wave): p' and the candidate-ROI word of each point's cell (from LDS when
// staged, so that the only global loads in flight are the point tiles),
// ANDed with the sweep's budget word when the frame's ROIs fit one word (a
// single wave-wide read when the wave holds one sweep).
// BG: the out-of-ROI keep rate is nonzero (without it no draw is made and
// the code below is the ROI-only path).
template <int ST, bool BG>
__device__ __forceinline__ void phase_a(const Config& c, const CellConsts& kc, const FilterLds& L, int32_t b,
                                        uint32_t i0, const Quad& d, QuadState& st) {
  const uint32_t S = (uint32_t)c.S;
  int32_t cidx[4];
  uint32_t bw[4];
  st.s = d.s;
  // one sweep for the whole wave: every lane's four sweep bytes equal the
  // first lane's first one
  const uint32_t s0 = __builtin_amdgcn_readfirstlane(d.s) & 0xffu;
  if (ST && s0 < S && __ballot(d.s != s0 * 0x01010101u) == 0) {
    // one pose for the whole wave, read as three 16-byte rows
    const int32_t row = kc.fr * (int32_t)S + (int32_t)s0;
    const float4 r0 = *reinterpret_cast<const float4*>(lds_pose(row));
    const float4 r1 = *reinterpret_cast<const float4*>(lds_pose(row) + 4);
    const float4 r2 = *reinterpret_cast<const float4*>(lds_pose(row) + 8);
    const uint32_t w0 = c.W == 1 ? lds_bm(c)[kc.fr * c.S + s0] : ~0u;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      bw[q] = w0;
      st.px[q] = fma_rn(r0.x, d.x[q], fma_rn(r0.y, d.y[q], fma_rn(r0.z, d.z[q], r0.w)));
      st.py[q] = fma_rn(r1.x, d.x[q], fma_rn(r1.y, d.y[q], fma_rn(r1.z, d.z[q], r1.w)));
      st.pz[q] = fma_rn(r2.x, d.x[q], fma_rn(r2.y, d.y[q], fma_rn(r2.z, d.z[q], r2.w)));
      cidx[q] = approx_cell(kc, st.px[q], st.py[q]);
    }
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t sq = (d.s >> (8 * q)) & 0xffu;
      cidx[q] = -1;
      bw[q] = 0u;
      st.px[q] = st.py[q] = st.pz[q] = 0.0f;
      if (sq < S) {
        bw[q] = c.W == 1 ? budget_word<ST>(c, L, b, sq, 0) : ~0u;
        float P[12];
        load_pose<ST>(c, L, b, sq, P);
        compensate(P, d.x[q], d.y[q], d.z[q], st.px[q], st.py[q], st.pz[q]);
        cidx[q] = approx_cell(kc, st.px[q], st.py[q]);
      }
    }
  }
  // the four cell words (always in bounds); staged, cell -1 reads the zero
  // word in front of the frame's row, so no select is needed
  if (ST) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      st.cand[q] = reinterpret_cast<const uint32_t*>(filter_dyn)[kc.cell_row + cidx[q]] & bw[q];
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t w = c.cellany[(int64_t)b * c.ncells + max(cidx[q], 0)];
      st.cand[q] = cidx[q] >= 0 ? w & bw[q] : 0u;
    }
  }
  // the out-of-ROI keep draw
  st.bg = 0;
  if (BG)
#pragma unroll
    for (int q = 0; q < 4; ++q)
      st.bg |= (cidx[q] >= 0 && ((d.s >> (8 * q)) & 0xffu) < S && background_draw(c, i0 + q)) ? 1u << q : 0u;
}

// Queue and kept-point state of one wave (wave-uniform values).
struct WaveRun {
  uint32_t head;    // ring index of the oldest queued candidate
  uint32_t queued;  // candidates in the ring (< 64 between tiles)
  uint32_t kept;    // points kept so far
  uint32_t lo;      // first point of the wave's chunk
  int32_t b;        // frame of the wave's chunk
  uint32_t k;       // the chunk
};

// Decide the n (<= 64) oldest queued candidates and set the bits of the kept
// ones in the wave's bitmap.  Nothing is written to global memory here: a
// store inside the tile loop would make the compiler wait for it (and, since
// vector memory operations complete in order, for every tile load before it)
// once its source registers are reused.
template <int ST, bool BG>
__device__ __forceinline__ void decide_round(const Config& c, const FilterLds& L, WaveLds& Q, WaveRun& wr,
                                             uint32_t n) {
  const uint32_t lane = (uint32_t)(threadIdx.x & 63);
  // every lane reads a slot of the ring; lanes past n hold no candidate
  const uint32_t e = (wr.head + lane) & (kWaveQueue - 1);
  const bool live = lane < n;
  const uint32_t pk = Q.pk[e];
  const float px = live ? Q.px[e] : 0.0f, py = live ? Q.py[e] : 0.0f, pz = live ? Q.pz[e] : 0.0f;
  int32_t ix, iy, iz;
  const bool in_grid = quantize_fast(c, px, py, pz, ix, iy, iz);
  const uint32_t cand = live && in_grid ? Q.cand[e] : 0u;
  const int32_t r0 = frame_roi_base<ST>(c, L, wr.b);
  bool keep;
  if (c.W == 1) {
    keep = roi_test_one_word<ST>(c, L, r0, cand, px, py);
  } else {
    keep = false;
    if (cand != 0u) keep = roi_test_words<ST>(c, L, wr.b, (pk >> 16) & 0xffu, r0, ix, iy, px, py);
  }
  if (BG) keep = keep || (live && in_grid && ((pk >> 24) & 1u));  // drawn out-of-ROI points in the grid
  if (keep) atomicOr(&Q.bits[(pk & 0xffffu) >> 5], 1u << (pk & 31u));
  wr.kept += (uint32_t)__popcll(__ballot(keep));
  wr.head = (wr.head + n) & (kWaveQueue - 1);
  wr.queued -= n;
  wave_lds_sync();  // slots read before they are written again
}

// Phase B of four points of a lane: the candidates (a candidate ROI that
// admits the sweep, or drawn for the out-of-ROI keep)
// appended in point order (lane, then q) to the wave's ring, deciding full
// rounds of 64 as they become available.
template <int ST, bool BG>
__device__ __forceinline__ void phase_b(const Config& c, const FilterLds& L, WaveLds& Q, uint32_t i0,
                                        QuadState& st, WaveRun& wr) {
  bool has[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) has[q] = st.cand[q] != 0u || (BG && ((st.bg >> q) & 1u));
  const uint64_t lt = lanemask_lt();
  const uint32_t n = (uint32_t)has[0] + (uint32_t)has[1] + (uint32_t)has[2] + (uint32_t)has[3];
  const uint64_t b0 = __ballot(n & 1u), b1 = __ballot(n & 2u), b2 = __ballot(n & 4u);
  const uint32_t rank0 = __popcll(b0 & lt) + 2u * __popcll(b1 & lt) + 4u * __popcll(b2 & lt);
  const uint32_t total = __popcll(b0) + 2u * __popcll(b1) + 4u * __popcll(b2);
  for (uint32_t done = 0; done < total;) {
    // room >= 64 here: fewer than 64 candidates stay queued between rounds
    const uint32_t take = min((uint32_t)kWaveQueue - wr.queued, total - done);
    uint32_t rank = rank0;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (has[q]) {
        if (rank - done < take) {
          const uint32_t e = (wr.head + wr.queued + (rank - done)) & (kWaveQueue - 1);
          Q.pk[e] = (i0 + q - wr.lo) | (((st.s >> (8 * q)) & 0xffu) << 16) | (BG ? ((st.bg >> q) & 1u) << 24 : 0u);
          Q.cand[e] = st.cand[q];
          Q.px[e] = st.px[q];
          Q.py[e] = st.py[q];
          Q.pz[e] = st.pz[q];
        }
        ++rank;
      }
    wr.queued += take;
    done += take;
    wave_lds_sync();
    while (wr.queued >= 64) decide_round<ST, BG>(c, L, Q, wr, 64);
  }
}

// Step k of the register pipeline over the ntiles full tiles from a0: the
// loads of tile k go into buffer k mod kFilterDepth (past the end, loads of
// a small spare region of the workspace that stays in cache: values
// unused), then tile k - (kFilterDepth - 1), loaded that many steps
// earlier, is handled if it exists.  Every step
// issues the same loads in the same order, and the loop over the steps has a
// fixed trip count and no early exit, so the compiler's wait before a tile's
// data counts exactly the loads of the tiles after it.
template <int ST, bool BG, int J>
__device__ __forceinline__ void pipeline_step(const Config& c, const CellConsts& kc, const FilterLds& L, WaveLds& Q,
                                              int32_t b, const TileRows& rows, const TileRows& spare,
                                              uint32_t a0, uint32_t ntiles, uint32_t k0, uint32_t lane4,
                                              Quad (&buf)[kFilterDepth], QuadState& st, WaveRun& wr) {
  const uint32_t k = k0 + (uint32_t)J;
  if (k < ntiles)
    load_quad_vec(rows, k * kWaveTile + lane4, buf[J]);
  else
    load_quad_vec(spare, lane4, buf[J]);
  const uint32_t tile = k - (uint32_t)(kFilterDepth - 1);  // wraps for the first steps
  if (tile < ntiles) {
    const uint32_t t = a0 + tile * kWaveTile;
    phase_a<ST, BG>(c, kc, L, b, t + lane4, buf[(J + 1) % kFilterDepth], st);
    phase_b<ST, BG>(c, L, Q, t + lane4, st, wr);
  }
}

// The points [lo, hi) of one wave (frame b), wave tile by wave tile: the
// points before the first multiple of 4 and a partial last tile are loaded
// point by point; the full tiles between them go through a register
// pipeline of kFilterDepth buffers with 16-byte loads (when the rows allow
// them; otherwise every tile is loaded point by point): the loads of the
// next kFilterDepth - 1 tiles are in flight while a tile is handled.
template <bool VEC, int ST, bool BG>
__device__ __forceinline__ void run_wave(const Config& c, const FilterLds& L, WaveLds& Q, int32_t b, uint32_t lo,
                                         uint32_t hi, WaveRun& wr) {
  const uint32_t lane = (uint32_t)(threadIdx.x & 63), lane4 = 4u * lane;
  Quad buf[kFilterDepth];
  QuadState st;
  const CellConsts kc = cell_consts<ST>(c, L, b);
  static_assert(kChunkWords == 128, "two bitmap words per lane");
  Q.bits[lane] = 0;
  Q.bits[lane + 64] = 0;
  wave_lds_sync();
  const uint32_t a0 = VEC ? min((lo + 3u) & ~3u, hi) : lo;
  if (a0 > lo) {  // head: fewer than 4 points
    load_quad_scalar(c, lo + lane4, a0, buf[0]);
    phase_a<ST, BG>(c, kc, L, b, lo + lane4, buf[0], st);
    phase_b<ST, BG>(c, L, Q, lo + lane4, st, wr);
  }
  const uint32_t ntiles = VEC ? (hi - a0) / kWaveTile : 0u;
  static_assert(kFilterDepth >= 2 && kFilterDepth <= 6, "pipeline steps written out below");
  if (ntiles > 0) {
    const TileRows rows = tile_rows(c, a0);
    const TileRows spare{c.spare_tile, c.spare_tile, c.spare_tile, reinterpret_cast<const uint8_t*>(c.spare_tile)};
    const uint32_t steps = ntiles + (uint32_t)(kFilterDepth - 1);
    for (uint32_t k0 = 0; k0 < steps; k0 += kFilterDepth) {
      pipeline_step<ST, BG, 0>(c, kc, L, Q, b, rows, spare, a0, ntiles, k0, lane4, buf, st, wr);
      pipeline_step<ST, BG, 1>(c, kc, L, Q, b, rows, spare, a0, ntiles, k0, lane4, buf, st, wr);
      if constexpr (kFilterDepth > 2) pipeline_step<ST, BG, 2 % kFilterDepth>(c, kc, L, Q, b, rows, spare, a0, ntiles, k0, lane4, buf, st, wr);
      if constexpr (kFilterDepth > 3) pipeline_step<ST, BG, 3 % kFilterDepth>(c, kc, L, Q, b, rows, spare, a0, ntiles, k0, lane4, buf, st, wr);
      if constexpr (kFilterDepth > 4) pipeline_step<ST, BG, 4 % kFilterDepth>(c, kc, L, Q, b, rows, spare, a0, ntiles, k0, lane4, buf, st, wr);
      if constexpr (kFilterDepth > 5) pipeline_step<ST, BG, 5 % kFilterDepth>(c, kc, L, Q, b, rows, spare, a0, ntiles, k0, lane4, buf, st, wr);
    }
  }
  for (uint32_t t = a0 + ntiles * kWaveTile; t < hi; t += kWaveTile) {
    load_quad_scalar(c, t + lane4, hi, buf[0]);
    phase_a<ST, BG>(c, kc, L, b, t + lane4, buf[0], st);
    phase_b<ST, BG>(c, L, Q, t + lane4, st, wr);
  }
  while (wr.queued > 0) decide_round<ST, BG>(c, L, Q, wr, min(wr.queued, 64u));
  wave_lds_sync();
  // the chunk's bitmap, every word (bits past hi are zero)
  uint32_t* out = c.fbits + (int64_t)wr.k * c.fchunk_words;
  if (lane < (uint32_t)c.fchunk_words) out[lane] = Q.bits[lane];
  if (lane + 64 < (uint32_t)c.fchunk_words) out[lane + 64] = Q.bits[lane + 64];
}

// Scratch of a workgroup that lays out the call itself (the waves' queues
// are not in use before the first tile, so it lives there).
struct FuseLds {
  uint32_t first[kFuseFrames + 1];  // first filter chunk of frame b
  int32_t roff[kFuseFrames + 1];    // ROI offsets as given
  int16_t rect[kMaxLdsRois][4];     // cell rectangles of the frame's ROIs
  uint32_t area[kMaxLdsRois + 1];   // their cells before ROI j (exclusive prefix), then the total
  uint32_t bud[kMaxLdsRois];        // their sweep budgets
  uint32_t tmp[2 * kWaves];
};
static_assert(sizeof(FuseLds) <= kWaves * sizeof(WaveLds), "fits the waves' queues");

// What a workgroup of the fused instance needs to know about the call.
struct FuseLayout {
  uint32_t nchunks;     // filter chunks of the call
  int32_t wf;           // frame of the workgroup's first chunk
  uint32_t ff0, ff1;    // that frame's first chunk and the next frame's
  int64_t fo0, fo1;     // its point offsets
  int32_t ro0, ro1;     // its ROI offsets
};

// Every workgroup of the fused instance (frames B <= kFuseFrames, one per
// thread): the offset checks and the chunk layout the staging kernel makes
// otherwise (the same numbering: each frame's chunks rounded up to whole
// workgroups, none at all when the point offsets are invalid), and the
// frame of its first chunk.  Workgroup 0 also opens the call: the header's
// counters and fault word, the call count and the frames' first chunks,
// which the later kernels read.
__device__ __forceinline__ FuseLayout fuse_layout(const Config& c, FuseLds& F) {
  const int tid = threadIdx.x;
  const int f = min(tid, c.B), fn = min(f + 1, c.B);
  const int64_t o = c.frame_off[f], on = c.frame_off[fn];
  const int32_t ro = c.roi_off[f], rn = c.roi_off[fn];
  const int32_t bad = tid <= c.B ? offset_faults(c, f, o, on, ro, rn) : 0;
  const uint32_t p0 = (uint32_t)min(max(o, (int64_t)0), (int64_t)c.N);
  const uint32_t p1 = max((uint32_t)min(max(on, (int64_t)0), (int64_t)c.N), p0);
  const uint32_t mine = tid < c.B ? frame_chunks(p1 - p0, (uint32_t)c.fchunk_points) : 0u;
  // the chunk counts scanned, and the frames with bad point and bad ROI
  // offsets counted (at most 256 each) in the same pass
  const uint32_t badc = (bad & MMBEV_FAULT_POINT_OFFSETS ? 1u : 0u) | (bad & MMBEV_FAULT_ROI_OFFSETS ? 1u << 16 : 0u);
  uint2 tot;
  const uint32_t run = block_exclusive_scan2<kWaves>(mine, badc, F.tmp, tot).x;
  const int32_t allbad = ((tot.y & 0xffffu) ? MMBEV_FAULT_POINT_OFFSETS : 0) | ((tot.y >> 16) ? MMBEV_FAULT_ROI_OFFSETS : 0);
  // invalid point offsets lay out no chunk at all (frames could overlap)
  const bool no_points = (allbad & MMBEV_FAULT_POINT_OFFSETS) != 0;
  const uint32_t cap = (uint32_t)c.fchunk_max;  // reached only with invalid offsets
  const uint32_t nch = no_points ? 0u : min(tot.x, cap);
  if (tid < c.B) F.first[tid] = no_points ? 0u : min(run, cap);
  if (tid == c.B) F.first[tid] = nch;
  if (tid <= c.B) F.roff[tid] = ro;
  __syncthreads();
  if (blockIdx.x == 0) {
    WsHeader* h = c.hdr;
    if (tid == 0) {
      h->fault = allbad;
      h->epoch = h->epoch + 1;
      h->kept = 0;
      h->voxels = 0;
      h->capped_voxels = 0;
      h->any_capped = 0;
      h->fchunks = nch;
    }
    if (tid <= c.B) c.fchunk_first[tid] = F.first[tid];
  }
  FuseLayout g;
  g.nchunks = nch;
  const uint32_t k0 = (uint32_t)blockIdx.x * kWaves;
  int32_t lo = 0, hi = c.B - 1;  // the last frame whose first chunk is at most k0
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) >> 1;
    if (F.first[mid] <= k0) lo = mid; else hi = mid - 1;
  }
  g.wf = lo;
  g.ff0 = F.first[lo];
  g.ff1 = F.first[lo + 1];
  g.ro0 = F.roff[lo];
  g.ro1 = F.roff[lo + 1];
  g.fo0 = c.frame_off[lo];
  g.fo1 = c.frame_off[lo + 1];
  return g;
}

// The fused instance's tables of frame f (roi_n ROIs from roi_lo): poses,
// ROI records and budgets loaded together; the budget words of every
// (sweep, ROI word) and the frame's cell row (a zero word, then per coarse
// cell the ROIs whose conservative rectangle covers it: with several ROI
// words, their OR, and every word in the word masks at word lds_wmask of
// the dynamic LDS) built in LDS from the records, as the staging kernel
// builds them.
template <bool WIDE>
__device__ __forceinline__ void fuse_staging(const Config& c, FilterLds& L, FuseLds& F, int32_t f, int32_t roi_lo,
                                             int32_t roi_n, int32_t ro0, int32_t ro1) {
  constexpr int kPoseRegs = (kMaxPoseLds * 12 + kBlock - 1) / kBlock;
  const int tid = threadIdx.x;
  const int np = c.S * 12;
  const int W = WIDE ? c.W : 1;
  float pv[kPoseRegs];
  const float* poses = c.poses + (int64_t)f * np;
#pragma unroll
  for (int j = 0; j < kPoseRegs; ++j) pv[j] = tid + j * kBlock < np ? poses[tid + j * kBlock] : 0.0f;
  mmbev_roi_t r{};
  uint32_t bud = 0;
  if (tid < roi_n) {
    r = c.rois[roi_lo + tid];
    bud = c.budget[roi_lo + tid];
  }
  uint32_t* dyn = reinterpret_cast<uint32_t*>(filter_dyn);
  float* dynf = reinterpret_cast<float*>(filter_dyn);
  if (tid == 0) L.roff[0] = min(max(ro0, 0), c.R);
  if (tid == 1) L.roff[1] = min(max(ro1, 0), c.R);
#pragma unroll
  for (int j = 0; j < kPoseRegs; ++j)
    if (tid + j * kBlock < np) dynf[tid + j * kBlock] = pv[j];  // pose rows from word 0
  for (int e = tid; e <= c.ncells; e += kBlock) dyn[c.lds_cell + e] = 0u;
  if (WIDE)
    for (int e = tid; e < c.ncells * W; e += kBlock) dyn[c.lds_wmask + e] = 0u;
  uint32_t area = 0;
  if (tid < roi_n) {
    dynf[c.lds_roi + 0 * c.lds_roi_cap + tid] = r.cx;
    dynf[c.lds_roi + 1 * c.lds_roi_cap + tid] = r.cy;
    dynf[c.lds_roi + 2 * c.lds_roi_cap + tid] = r.cos_yaw;
    dynf[c.lds_roi + 3 * c.lds_roi_cap + tid] = r.sin_yaw;
    dynf[c.lds_roi + 4 * c.lds_roi_cap + tid] = r.ext_x;
    dynf[c.lds_roi + 5 * c.lds_roi_cap + tid] = r.ext_y;
    int16_t* rc = F.rect[tid];
    roi_cell_rect(c, r, rc);
    area = rc[1] >= rc[0] && rc[3] >= rc[2] ? (uint32_t)(rc[1] - rc[0] + 1) * (uint32_t)(rc[3] - rc[2] + 1) : 0u;
    F.bud[tid] = bud;
  }
  // the rectangles' cell counts scanned: one wave for at most 64 ROIs
  // (always so with one ROI word), the workgroup otherwise
  if (!WIDE || roi_n <= 64) {  // uniform
    if (tid < 64) {
      const uint32_t x = wave_inclusive_sum(area);
      F.area[tid] = x - area;
      if (tid == 63) F.area[kMaxLdsRois] = x;
    }
  } else {
    uint32_t total;
    const uint32_t ex = block_exclusive_scan(area, F.tmp, total);
    F.area[tid] = ex;
    if (tid == 0) F.area[kMaxLdsRois] = total;
  }
  __syncthreads();
  if (tid < c.S * W) {  // (sweep s, ROI word w): the word's ROIs whose budget admits s
    const int s = tid / W, w = tid % W;
    uint32_t m = 0;
    for (int j = 32 * w; j < min(32 * w + 32, roi_n); ++j) m |= F.bud[j] > (uint32_t)s ? 1u << (j & 31) : 0u;
    dyn[c.lds_bm + tid] = m;
  }
  // every (ROI, covered cell) pair: the ROI's bit ORed into the cell's word
  // (and, with several ROI words, into the cell's word of that ROI)
  const uint32_t cells = F.area[kMaxLdsRois];
  for (uint32_t i = tid; i < cells; i += kBlock) {
    int32_t lo = 0, hi = roi_n - 1;  // the ROI: the last one whose first pair is at most i
    while (lo < hi) {
      const int32_t mid = (lo + hi + 1) >> 1;
      if (F.area[mid] <= i) lo = mid; else hi = mid - 1;
    }
    const int16_t* rc = F.rect[lo];
    const uint32_t q = i - F.area[lo], wx = (uint32_t)(rc[1] - rc[0] + 1);
    const uint32_t cell = ((uint32_t)rc[2] + q / wx) * (uint32_t)c.ncx + (uint32_t)rc[0] + q % wx;
    atomicOr(&dyn[c.lds_cell + 1 + cell], 1u << (lo & 31));
    if (WIDE) atomicOr(&dyn[c.lds_wmask + cell * (uint32_t)W + (uint32_t)(lo >> 5)], 1u << (lo & 31));
  }
}

// Workgroup w: its waves over filter chunks kWaves*w .. kWaves*w + 3.  Per
// chunk it leaves the bitmap of its kept points, their number, its first
// point and its frame.  BG: the out-of-ROI keep rate is nonzero.
template <bool VEC, bool BG, int FS>
__global__ __launch_bounds__(kBlock, 5) void filter_kernel(Config c) {
  __shared__ FilterLds L;
  __shared__ WaveLds Qs[kWaves];
  const int tid = threadIdx.x;
  // the wave index is the same in all its lanes: uniform, so that the rest
  // of the kernel is uniform control flow for the compiler too
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  WaveLds& Q = Qs[wave];
  FuseLds& F = *reinterpret_cast<FuseLds*>(&Qs[0]);
  uint32_t nchunks, ff0, ff1;
  int32_t wf, ro0, ro1;
  int64_t fo0, fo1;
  if constexpr (FS) {  // the workgroup lays out the call itself
    const FuseLayout g = fuse_layout(c, F);
    nchunks = g.nchunks;
    wf = g.wf;
    ff0 = g.ff0;
    ff1 = g.ff1;
    fo0 = g.fo0;
    fo1 = g.fo1;
    ro0 = g.ro0;
    ro1 = g.ro1;
  } else {
    nchunks = c.hdr->fchunks;
    // frame wf of chunk k0 (loaded with nchunks), then everything that
    // depends only on wf, loaded together: every chunk of the workgroup lies
    // in wf unless the point offsets are invalid (then searches find the
    // frames)
    wf = (int32_t)min(c.wg_frame[blockIdx.x], (uint32_t)c.B - 1u);
    fo0 = c.frame_off[wf];
    fo1 = c.frame_off[wf + 1];
    ff0 = c.fchunk_first[wf];
    ff1 = c.fchunk_first[wf + 1];
    ro0 = c.roi_off[wf];
    ro1 = c.roi_off[wf + 1];
    asm volatile("" ::"s"(fo0), "s"(fo1), "s"(ff0), "s"(ff1), "s"(ro0), "s"(ro1));  // one round trip for all
  }
  const uint32_t k0 = (uint32_t)blockIdx.x * kWaves;

  // this wave's chunk and its points; the staging plan
  const uint32_t k = k0 + (uint32_t)wave;
  const bool any = k0 < nchunks;
  const uint32_t last = any ? min(k0 + kWaves - 1, nchunks - 1) : k0;
  int32_t b = 0;
  uint32_t lo = 0, hi = 0;
  StagePlan pl{0, 0, 0, 0, false};
  if (any && last < ff1) {
    pl = make_plan(c, wf, wf, ro0, ro1);
    if (FS) {  // always staged (the host checked the sizes); ROIs past the cap only with invalid ROI offsets
      pl.roi_n = min(pl.roi_n, c.lds_roi_cap);
      pl.staged = true;
    }
    if (k < nchunks) {
      b = wf;
      const uint32_t P = (uint32_t)c.fchunk_points;
      const uint32_t p0 = (uint32_t)min(max(fo0, (int64_t)0), (int64_t)c.N);
      const uint32_t p1 = max((uint32_t)min(max(fo1, (int64_t)0), (int64_t)c.N), p0);
      const uint64_t l = (uint64_t)p0 + (uint64_t)(k - ff0) * P;
      lo = (uint32_t)min(l, (uint64_t)p1);
      hi = (uint32_t)min(l + P, (uint64_t)p1);
    }
  } else if (any && !FS) {  // (with the fused layout every workgroup's chunks lie in one frame)
    const int32_t f0 = frame_of_chunk(c.fchunk_first, c.B, k0), f1 = frame_of_chunk(c.fchunk_first, c.B, last);
    pl = make_plan(c, f0, f1, c.roi_off[f0], c.roi_off[f1 + 1]);
    if (k < nchunks) {
      b = frame_of_chunk(c.fchunk_first, c.B, k);
      filter_chunk_points(c, b, k, lo, hi);
    }
  }
  // the same in every lane; uniform bounds keep the tile loop a scalar loop
  b = __builtin_amdgcn_readfirstlane(b);
  lo = __builtin_amdgcn_readfirstlane(lo);
  hi = __builtin_amdgcn_readfirstlane(hi);
  if (tid == 0) {
    L.f0 = pl.f0;
    L.f1 = pl.f1;
    L.roi_lo = pl.roi_lo;
    L.roi_n = pl.roi_n;
    L.chunk_staged = pl.staged;
  }
  const bool staged = pl.staged;
  if (FS) {
    if (pl.staged) fuse_staging<FS == 2>(c, L, F, pl.f0, pl.roi_lo, pl.roi_n, ro0, ro1);
  } else if (staged) {
    do_staging(c, L, pl);
  }
  __syncthreads();

  if (k >= nchunks || (FS && !pl.staged)) return;
  WaveRun wr{0u, 0u, 0u, lo, b, k};
  if (staged)
    run_wave<VEC, FS == 2 ? 2 : 1, BG>(c, L, Q, b, lo, hi, wr);
  else
    run_wave<VEC, 0, BG>(c, L, Q, b, lo, hi, wr);
  if (lane == 0) {
    c.fcount[k] = wr.kept;
    c.fchunk_lo[k] = lo;
    c.fchunk_frame[k] = (uint32_t)b;
  }
}

}  // namespace

hipError_t launch_filter(const Config& c, hipStream_t st) {
  // one instance per load form and per rate (none, or a nonzero one)
  const dim3 grid(c.filter_grid), block(kBlock);
  const size_t dyn = (size_t)c.lds_dyn_bytes;
  // FS: 0 the staging kernel's tables, 1 the filter's own (one ROI word
  // per cell), 2 the filter's own with the cells' ROI words in LDS
  const int fs = c.fuse_stage ? (c.lds_wmask >= 0 ? 2 : 1) : 0;
  if (fs == 1) {
    if (c.vec && c.bg_thr == 0u)
      hipLaunchKernelGGL((filter_kernel<true, false, 1>), grid, block, dyn, st, c);
    else if (c.vec)
      hipLaunchKernelGGL((filter_kernel<true, true, 1>), grid, block, dyn, st, c);
    else if (c.bg_thr == 0u)
      hipLaunchKernelGGL((filter_kernel<false, false, 1>), grid, block, dyn, st, c);
    else
      hipLaunchKernelGGL((filter_kernel<false, true, 1>), grid, block, dyn, st, c);
  } else if (fs == 2) {
    if (c.vec && c.bg_thr == 0u)
      hipLaunchKernelGGL((filter_kernel<true, false, 2>), grid, block, dyn, st, c);
    else if (c.vec)
      hipLaunchKernelGGL((filter_kernel<true, true, 2>), grid, block, dyn, st, c);
    else if (c.bg_thr == 0u)
      hipLaunchKernelGGL((filter_kernel<false, false, 2>), grid, block, dyn, st, c);
    else
      hipLaunchKernelGGL((filter_kernel<false, true, 2>), grid, block, dyn, st, c);
  } else if (c.vec && c.bg_thr == 0u) {
    hipLaunchKernelGGL((filter_kernel<true, false, 0>), grid, block, dyn, st, c);
  } else if (c.vec) {
    hipLaunchKernelGGL((filter_kernel<true, true, 0>), grid, block, dyn, st, c);
  } else if (c.bg_thr == 0u) {
    hipLaunchKernelGGL((filter_kernel<false, false, 0>), grid, block, dyn, st, c);
  } else {
    hipLaunchKernelGGL((filter_kernel<false, true, 0>), grid, block, dyn, st, c);
  }
  return hipGetLastError();
}

}  // namespace mmbev

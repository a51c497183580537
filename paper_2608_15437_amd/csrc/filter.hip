// Fused point filter: one streaming pass over all points.
//
// Per point (Alg. 1 keep loop with out-of-ROI rate zero): load x, y, z and
// the sweep id, move the point into the current frame (Eq. 6), quantise it
// (Alg. 1 Voxelize: range check and voxel indices), look up the candidate
// ROIs of its coarse cell that admit its sweep, and run the exact oriented
// box test on those candidates only.  Kept points are written as
// (voxel key, point index) pairs in point-index order: wave ballots give the
// rank inside a wave, LDS gives the rank inside the workgroup, and a chained
// scan with decoupled look-back over dynamically numbered tiles gives the
// global offset.  The digit histograms of every radix pass of the following
// sort are accumulated here, so the sort never re-reads its input to count.
//
// Memory layout: each thread owns kFilterGroups groups of 4 consecutive
// points; group g of thread t starts at point tile*4096 + 4*(t + 256 g), so
// one float4 load per column per group is fully coalesced across a wave.
#include "launch.hpp"

namespace mmbev {

namespace {

struct FilterLds {
  uint32_t hist[kMaxPasses][kSortBins];
  float pose[kMaxPoseLds][12];
  uint32_t wave_tot[kFilterGroups][kWaves];
  uint32_t tile, prefix;
  int32_t f0, f1;
};

// Keep test for one point.  Returns true and the sort key on keep.
__device__ __forceinline__ bool keep_point(const Config& c, const FilterLds& L, bool pose_lds, int64_t i,
                                           float x, float y, float z, uint32_t s, uint32_t& key,
                                           int32_t& frame) {
  if (s >= (uint32_t)c.S) return false;
  int32_t b = L.f0;
  if (L.f1 != L.f0) {
    int32_t lo = L.f0, hi = L.f1;
    while (lo < hi) {
      int32_t mid = (lo + hi + 1) >> 1;
      if (c.frame_off[mid] <= i)
        lo = mid;
      else
        hi = mid - 1;
    }
    b = lo;
  }
  float P[12];
  if (pose_lds) {
    const float* src = L.pose[(b - L.f0) * c.S + s];
#pragma unroll
    for (int k = 0; k < 12; ++k) P[k] = src[k];
  } else {
    const float* src = c.poses + ((int64_t)b * c.S + s) * 12;
#pragma unroll
    for (int k = 0; k < 12; ++k) P[k] = src[k];
  }
  float px, py, pz;
  compensate(P, x, y, z, px, py, pz);
  int32_t ix, iy, iz;
  bool in = quantize_axis(px, c.mn[0], c.vs[0], c.Df[0], ix);
  in &= quantize_axis(py, c.mn[1], c.vs[1], c.Df[1], iy);
  in &= quantize_axis(pz, c.mn[2], c.vs[2], c.Df[2], iz);
  if (!in) return false;
  int32_t cell = (iy >> c.cell_shift) * c.ncx + (ix >> c.cell_shift);
  const uint32_t* cm = c.cellmask + ((int64_t)b * c.ncells + cell) * c.W;
  const uint32_t* bm = c.budgetmask + ((int64_t)b * c.S + s) * c.W;
  int32_t r0 = min(max(c.roi_off[b], 0), c.R);
  bool hit = false;
  for (int w = 0; w < c.W && !hit; ++w) {
    uint32_t m = cm[w] & bm[w];
    while (m) {
      int k = __builtin_ctz(m);
      m &= m - 1;
      if (inside_roi(c.rois[r0 + w * 32 + k], px, py)) {
        hit = true;
        break;
      }
    }
  }
  if (!hit) return false;
  uint32_t kl = ((uint32_t)iz * c.Dy + (uint32_t)iy) * c.Dx + (uint32_t)ix;
  key = (c.key_has_frame && c.fb > 0) ? (((uint32_t)b << c.kb) | kl) : kl;
  frame = b;
  return true;
}

template <bool VEC>
__global__ __launch_bounds__(kBlock) void filter_kernel(Config c) {
  __shared__ FilterLds L;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  WsHeader* h = c.hdr;
  const uint32_t nbins = 1u << c.dbits;

  if (tid == 0) L.tile = atomicAdd(&h->tickets[kSlotFilter], 1u);
  for (int e = tid; e < kMaxPasses * kSortBins; e += kBlock) (&L.hist[0][0])[e] = 0;
  __syncthreads();
  const int64_t tile = L.tile;
  const int64_t base = tile * kFilterTile;
  const int64_t N = c.N;
  if (tid == 0) {
    int64_t last = min(base + kFilterTile, N) - 1;
    L.f0 = c.B == 1 ? 0 : frame_of_point(c.frame_off, c.B, base);
    L.f1 = c.B == 1 ? 0 : max(frame_of_point(c.frame_off, c.B, last), L.f0);
  }
  __syncthreads();
  const int32_t nposes = (L.f1 - L.f0 + 1) * c.S;
  const bool pose_lds = nposes <= kMaxPoseLds;
  if (pose_lds)
    for (int e = tid; e < nposes * 12; e += kBlock) (&L.pose[0][0])[e] = c.poses[(int64_t)L.f0 * c.S * 12 + e];
  __syncthreads();

  uint32_t keys[kFilterGroups][4];
  int32_t frames[kFilterGroups][4];
  uint32_t keepm[kFilterGroups];  // bit q: point q of group g kept

#pragma unroll
  for (int g = 0; g < kFilterGroups; ++g) {
    const int64_t i0 = base + 4 * (int64_t)(tid + kBlock * g);
    float xs[4], ys[4], zs[4];
    uint32_t ss[4];
    if (VEC && i0 + 3 < N) {
      float4 x4 = *reinterpret_cast<const float4*>(c.feat + i0);
      float4 y4 = *reinterpret_cast<const float4*>(c.feat + c.stride + i0);
      float4 z4 = *reinterpret_cast<const float4*>(c.feat + 2 * c.stride + i0);
      uint32_t s4 = *reinterpret_cast<const uint32_t*>(c.sweep + i0);
      xs[0] = x4.x; xs[1] = x4.y; xs[2] = x4.z; xs[3] = x4.w;
      ys[0] = y4.x; ys[1] = y4.y; ys[2] = y4.z; ys[3] = y4.w;
      zs[0] = z4.x; zs[1] = z4.y; zs[2] = z4.z; zs[3] = z4.w;
#pragma unroll
      for (int q = 0; q < 4; ++q) ss[q] = (s4 >> (8 * q)) & 0xffu;
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int64_t i = i0 + q;
        bool ok = i < N;
        xs[q] = ok ? c.feat[i] : 0.0f;
        ys[q] = ok ? c.feat[c.stride + i] : 0.0f;
        zs[q] = ok ? c.feat[2 * c.stride + i] : 0.0f;
        ss[q] = ok ? (uint32_t)c.sweep[i] : 0xffffffffu;
      }
    }
    keepm[g] = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      keys[g][q] = 0;
      frames[g][q] = 0;
      if (keep_point(c, L, pose_lds, i0 + q, xs[q], ys[q], zs[q], ss[q], keys[g][q], frames[g][q]))
        keepm[g] |= 1u << q;
    }
  }

  // rank of each thread's kept points inside the tile: order (group, wave, lane, q)
  uint32_t excl[kFilterGroups];
  const uint64_t lt = lanemask_lt();
#pragma unroll
  for (int g = 0; g < kFilterGroups; ++g) {
    uint32_t cnt = __popc(keepm[g]);
    uint64_t b0 = __ballot(cnt & 1u), b1 = __ballot(cnt & 2u), b2 = __ballot(cnt & 4u);
    excl[g] = __popcll(b0 & lt) + 2u * __popcll(b1 & lt) + 4u * __popcll(b2 & lt);
    if (lane == 0) L.wave_tot[g][wave] = __popcll(b0) + 2u * __popcll(b1) + 4u * __popcll(b2);
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t run = 0;
    for (int g = 0; g < kFilterGroups; ++g)
      for (int w = 0; w < kWaves; ++w) {
        uint32_t t = L.wave_tot[g][w];
        L.wave_tot[g][w] = run;
        run += t;
      }
    const uint32_t tag = tag_of(h->epoch, kSlotFilter);
    uint64_t* st = c.filter_status;
    uint32_t prefix = 0;
    if (tile == 0) {
      status_store(st, status_word(tag, kFlagIncl, run));
    } else {
      status_store(st + tile, status_word(tag, kFlagAgg, run));
      prefix = look_back(st, tile, 1, tag, h);
      status_store(st + tile, status_word(tag, kFlagIncl, prefix + run));
    }
    L.prefix = prefix;
    if (tile == c.filter_tiles - 1) h->kept = prefix + run;
  }
  __syncthreads();

  uint32_t* kout = c.keys[0];
  uint32_t* vout = c.vals[0];
  const uint32_t dmask = nbins - 1u;
#pragma unroll
  for (int g = 0; g < kFilterGroups; ++g) {
    uint32_t pos = L.prefix + L.wave_tot[g][wave] + excl[g];
    const int64_t i0 = base + 4 * (int64_t)(tid + kBlock * g);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (keepm[g] & (1u << q)) {
        kout[pos] = keys[g][q];
        vout[pos] = (uint32_t)(i0 + q);
        ++pos;
        uint64_t comp = c.key_has_frame ? (uint64_t)keys[g][q]
                                        : (((uint64_t)frames[g][q] << c.kb) | (uint64_t)keys[g][q]);
        for (int p = 0; p < c.passes; ++p) atomicAdd(&L.hist[p][(comp >> (p * c.dbits)) & dmask], 1u);
      }
    }
  }
  __syncthreads();
  for (int e = tid; e < c.passes * (int)nbins; e += kBlock) {
    uint32_t v = L.hist[e / nbins][e % nbins];
    if (v) atomicAdd(&h->hist[0][e / nbins][e % nbins], v);
  }
}

}  // namespace

hipError_t launch_filter(const Config& c, hipStream_t st) {
  if (c.filter_tiles == 0) return hipSuccess;
  if (c.vec)
    hipLaunchKernelGGL(filter_kernel<true>, dim3(c.filter_tiles), dim3(kBlock), 0, st, c);
  else
    hipLaunchKernelGGL(filter_kernel<false>, dim3(c.filter_tiles), dim3(kBlock), 0, st, c);
  return hipGetLastError();
}

}  // namespace mmbev

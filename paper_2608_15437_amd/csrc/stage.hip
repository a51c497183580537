// ROI staging (first kernel of a call).
//
// For every frame b it builds, on a coarse bird's-eye-view cell grid laid
// over the voxel grid (cells of 2^cell_shift x 2^cell_shift voxels), one bit
// per ROI of the frame telling whether the ROI can contain a point whose
// voxel lies in that cell, plus one bit per (sweep, ROI) telling whether the
// ROI's sweep budget admits the sweep.  The filter then tests a point only
// against the ROIs whose bits survive the AND of its cell word and its sweep
// word.  Cell ranges are conservative (padded by more than the fp32 error of
// the exact test), so the exact test alone decides membership.
//
// Block (0, 0) also opens the call: it bumps the epoch that tags look-back
// words, clears the per-call counters and digit histograms, and checks the
// frame offsets of points and ROIs.  The blocks of frame 0 also record, for
// every tile of the point filter, its frame range and ROI range, so a filter
// workgroup starts with one load instead of two binary searches.
#include "launch.hpp"

namespace mmbev {

namespace {

constexpr int kMaxRois = 1024;

// Conservative cell rectangle [x0, x1] x [y0, y1] of one ROI; empty when x0 > x1.
__device__ void roi_cell_rect(const Config& c, const mmbev_roi_t& r, int16_t* out) {
  const double u = 1.0 / 16777216.0;  // fp32 unit roundoff
  double cx = r.cx, cy = r.cy, co = r.cos_yaw, si = r.sin_yaw, ex = r.ext_x, ey = r.ext_y;
  int32_t x0 = 0, x1 = c.ncx - 1, y0 = 0, y1 = c.ncy - 1;
  bool finite = isfinite(cx) && isfinite(cy) && isfinite(co) && isfinite(si) && isfinite(ex) && isfinite(ey);
  if (finite && (ex < 0.0 || ey < 0.0)) {
    x0 = 1;  // |l| <= negative extent never holds
    x1 = 0;
  } else if (finite) {
    double n2 = co * co + si * si;
    double hx = (fabs(co) * ex + fabs(si) * ey) / n2;
    double hy = (fabs(si) * ex + fabs(co) * ey) / n2;
    double mag = fabs(cx) + fabs(cy) + hx + hy;
    for (int d = 0; d < 2; ++d) mag += fabs((double)c.mn[d]) + (double)c.vs[d] * (double)c.Df[d];
    double pad = 1e-3 + 16.0 * u * mag;
    if (isfinite(hx) && isfinite(hy) && isfinite(pad)) {
      int32_t lim[2][2];
      double ctr[2] = {cx, cy}, half[2] = {hx, hy};
      for (int d = 0; d < 2; ++d) {
        double lo = (ctr[d] - half[d] - pad - (double)c.mn[d]) / (double)c.vs[d];
        double hi = (ctr[d] + half[d] + pad - (double)c.mn[d]) / (double)c.vs[d];
        double D = (double)c.Df[d];
        lo = fmin(fmax(floor(lo) - (double)c.cell_pad, -1.0), D);
        hi = fmin(fmax(floor(hi) + (double)c.cell_pad, -1.0), D);
        int32_t ilo = (int32_t)lo, ihi = (int32_t)hi;
        if (ihi < 0 || ilo >= (int32_t)D) {
          lim[d][0] = 1;
          lim[d][1] = 0;
        } else {
          ilo = max(ilo, 0);
          ihi = min(ihi, (int32_t)D - 1);
          lim[d][0] = ilo >> c.cell_shift;
          lim[d][1] = ihi >> c.cell_shift;
        }
      }
      x0 = lim[0][0];
      x1 = lim[0][1];
      y0 = lim[1][0];
      y1 = lim[1][1];
    }
  }
  out[0] = (int16_t)x0;
  out[1] = (int16_t)x1;
  out[2] = (int16_t)y0;
  out[3] = (int16_t)y1;
}

__global__ __launch_bounds__(kBlock) void stage_kernel(Config c) {
  __shared__ int16_t s_rect[kMaxRois][4];
  const int tid = threadIdx.x;
  const int b = blockIdx.y;
  WsHeader* h = c.hdr;

  if (blockIdx.x == 0 && b == 0) {
    if (tid == 0) {
      h->fault = 0;
      h->epoch = h->epoch + 1;
      h->kept = 0;
      h->voxels = 0;
      h->capped_voxels = 0;
      h->any_capped = 0;
    }
    uint32_t* hist = &h->hist[0][0];
    for (int e = tid; e < kMaxPasses * kSortBins; e += kBlock) hist[e] = 0;
    __syncthreads();
    int32_t bad = 0;
    for (int f = tid; f <= c.B; f += kBlock) {
      int64_t o = c.frame_off[f];
      if (f == 0 && o != 0) bad |= MMBEV_FAULT_POINT_OFFSETS;
      if (f == c.B && o != (int64_t)c.N) bad |= MMBEV_FAULT_POINT_OFFSETS;
      if (f < c.B && c.frame_off[f + 1] < o) bad |= MMBEV_FAULT_POINT_OFFSETS;
      int32_t ro = c.roi_off[f];
      if (f == 0 && ro != 0) bad |= MMBEV_FAULT_ROI_OFFSETS;
      if (f == c.B && ro != c.R) bad |= MMBEV_FAULT_ROI_OFFSETS;
      if (f < c.B) {
        int32_t rn = c.roi_off[f + 1];
        if (rn < ro || rn - ro > c.max_rois) bad |= MMBEV_FAULT_ROI_OFFSETS;
      }
    }
    if (bad) raise_fault(h, bad);
  }

  // frame and ROI range of every filter tile (rows of frame 0 only)
  if (b == 0)
    for (int64_t t = (int64_t)blockIdx.x * kBlock + tid; t < c.filter_tiles; t += (int64_t)gridDim.x * kBlock) {
      const int64_t first = t * kFilterTile;
      const int64_t last = min(first + kFilterTile, (int64_t)c.N) - 1;
      TileInfo ti;
      ti.f0 = c.B == 1 ? 0 : frame_of_point(c.frame_off, c.B, first);
      ti.f1 = c.B == 1 ? 0 : max(frame_of_point(c.frame_off, c.B, last), ti.f0);
      ti.r_lo = min(max(c.roi_off[ti.f0], 0), c.R);
      ti.r_hi = min(max(c.roi_off[ti.f1 + 1], ti.r_lo), c.R);
      c.tinfo[t] = ti;
    }

  // ROIs of frame b (offsets clamped into [0, R], count into [0, max_rois])
  int32_t r0 = min(max(c.roi_off[b], 0), c.R);
  int32_t r1 = min(max(c.roi_off[b + 1], r0), c.R);
  int32_t n = min(r1 - r0, c.max_rois);
  for (int j = tid; j < n; j += kBlock) roi_cell_rect(c, c.rois[r0 + j], s_rect[j]);
  __syncthreads();

  // one thread per cell (all W words of it) or per (sweep, word) of the budget masks
  const int64_t cell_words = (int64_t)c.ncells * c.W;
  const int64_t total = (int64_t)c.ncells + (int64_t)c.S * c.W;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + tid; e < total; e += (int64_t)gridDim.x * kBlock) {
    if (e < c.ncells) {
      const int32_t cell = (int32_t)e;
      const int32_t cx = cell % c.ncx, cy = cell / c.ncx;
      uint32_t any = 0;
      for (int w = 0; w < c.W; ++w) {
        uint32_t word = 0;
        for (int k = 0; k < 32; ++k) {
          int j = w * 32 + k;
          if (j < n && cx >= s_rect[j][0] && cx <= s_rect[j][1] && cy >= s_rect[j][2] && cy <= s_rect[j][3])
            word |= 1u << k;
        }
        c.cellmask[(int64_t)b * cell_words + (int64_t)cell * c.W + w] = word;
        any |= word;
      }
      if (c.W > 1) c.cellany[(int64_t)b * c.ncells + cell] = any;
    } else {
      int64_t e2 = e - c.ncells;
      int32_t s = (int32_t)(e2 / c.W), w = (int32_t)(e2 % c.W);
      uint32_t word = 0;
      for (int k = 0; k < 32; ++k) {
        int j = w * 32 + k;
        if (j < n && (int32_t)c.budget[r0 + j] > s) word |= 1u << k;
      }
      c.budgetmask[((int64_t)b * c.S + s) * c.W + w] = word;
    }
  }
}

__global__ __launch_bounds__(kBlock) void fill_zero_kernel(uint4* p, size_t n16, uint8_t* tail, size_t ntail) {
  size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x;
  for (; i < n16; i += (size_t)gridDim.x * kBlock) p[i] = make_uint4(0, 0, 0, 0);
  if (blockIdx.x == 0)
    for (size_t t = threadIdx.x; t < ntail; t += kBlock) tail[t] = 0;
}

}  // namespace

hipError_t launch_stage(const Config& c, hipStream_t st) {
  int64_t total = std::max<int64_t>((int64_t)c.ncells + (int64_t)c.S * c.W, c.filter_tiles);
  int gx = (int)std::min<int64_t>((total + kBlock - 1) / kBlock, 128);
  hipLaunchKernelGGL(stage_kernel, dim3(gx, c.B), dim3(kBlock), 0, st, c);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t st) {
  size_t n16 = bytes / 16;
  size_t ntail = bytes - n16 * 16;
  int g = (int)std::min<size_t>((n16 + kBlock - 1) / kBlock + 1, 4096);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(g), dim3(kBlock), 0, st, (uint4*)p, n16,
                     (uint8_t*)p + n16 * 16, ntail);
  return hipGetLastError();
}

}  // namespace mmbev

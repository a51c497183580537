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
// One more workgroup (the last column of frame 0's row; the rest of that
// column exits) opens the call in parallel with the frames' work: it bumps
// the call counter, clears the per-call counters, checks the frame offsets
// of points and ROIs, and lays out the filter's work: every frame is cut
// into chunks of fchunk_points points (the last one shorter), numbered frame
// after frame, so no chunk straddles two frames, and every filter workgroup
// (kWaves consecutive chunks) gets the frame of its first chunk, so that it
// starts with one table load instead of a search.
#include "launch.hpp"

namespace mmbev {

namespace {

constexpr int kMaxRois = 1024;
constexpr int kLdsFirst = kMaxRois * 2;  // chunk starts of up to kLdsFirst - 1 frames in the rectangles' LDS
constexpr int kStageCellsPerThread = 2;  // cells per thread when the ROIs fit one word

// The opening workgroup: counters, offset checks, filter chunk table and
// the frame of every filter workgroup.  s_first: LDS for kLdsFirst words;
// s_bad: one LDS word.  Point offsets that break the contract lay out no
// chunk at all: decreasing offsets would make frames overlap, and the kept
// points of overlapping frames could outnumber the arrays sized for N.
__device__ void open_call(const Config& c, uint32_t* s_tmp, uint32_t* s_first, int32_t* s_bad) {
  const int tid = threadIdx.x;
  WsHeader* h = c.hdr;
  // the offsets checked (every load of an iteration unconditional, at
  // clamped indices, so that they take one round trip together; frame tid's
  // point offsets kept for the chunk count when every thread owns one frame)...
  int32_t bad = 0;
  int64_t own0 = 0, own1 = 0;
  for (int f = tid; f <= c.B; f += kBlock) {
    const int fn = min(f + 1, c.B);
    const int64_t o = c.frame_off[f], on = c.frame_off[fn];
    const int32_t ro = c.roi_off[f], rn = c.roi_off[fn];
    if (f == tid) {
      own0 = o;
      own1 = on;
    }
    bad |= offset_faults(c, f, o, on, ro, rn);
  }
  if (tid == 0) {
    h->fault = 0;
    h->epoch = h->epoch + 1;
    h->kept = 0;
    h->voxels = 0;
    h->capped_voxels = 0;
    h->any_capped = 0;
    *s_bad = 0;
  }
  // ...and ORed in once the cleared fault word is visible to every wave
  __syncthreads();
  if (bad) {
    raise_fault(h, bad);
    atomicOr(s_bad, bad);
  }
  __syncthreads();
  const bool no_points = (*s_bad & MMBEV_FAULT_POINT_OFFSETS) != 0;
  // chunks of frame b: ceil(points / fchunk_points) rounded up to a whole
  // filter workgroup (kWaves chunks), so that a workgroup's chunks never span
  // two frames; thread t owns frames [t*per, (t+1)*per); the count is capped
  // at fchunk_max (reached only with invalid offsets)
  const uint32_t P = (uint32_t)c.fchunk_points;
  const int per = (c.B + kBlock - 1) / kBlock;
  const int b0 = tid * per;
  // points of frame b: from the offsets already loaded when per == 1 (b = tid)
  auto frame_points = [&](int b) -> uint32_t {
    int64_t o0 = own0, o1 = own1;
    if (per != 1) {  // uniform
      const int bb = min(b, c.B - 1);  // loads unconditional, at a clamped frame
      o0 = c.frame_off[bb];
      o1 = c.frame_off[bb + 1];
    }
    const uint32_t f0 = (uint32_t)min(max(o0, (int64_t)0), (int64_t)c.N);
    const uint32_t f1 = max((uint32_t)min(max(o1, (int64_t)0), (int64_t)c.N), f0);
    return f1 - f0;
  };
  uint32_t mine = 0;
  for (int j = 0; j < per; ++j) {
    const int b = b0 + j;
    const uint32_t np = frame_points(b);
    if (b < c.B && !no_points) mine += frame_chunks(np, P);
  }
  uint32_t total;
  uint32_t run = block_exclusive_scan(mine, s_tmp, total);
  const uint32_t cap = (uint32_t)c.fchunk_max;
  const uint32_t nch = min(total, cap);
  const bool in_lds = c.B < kLdsFirst;
  const int32_t G = c.filter_grid;
  for (int j = 0; j < per; ++j) {
    const int b = b0 + j;
    const uint32_t np = frame_points(b);
    if (b < c.B) {
      const uint32_t first = min(run, cap);
      c.fchunk_first[b] = first;
      run += no_points ? 0u : frame_chunks(np, P);
      if (in_lds) {
        s_first[b] = first;
      } else {
        // workgroups g whose first chunk kWaves * g lies in [first, end)
        const uint32_t end = min(run, cap);
        for (uint32_t g = (first + kWaves - 1) / kWaves; g < (end + kWaves - 1) / kWaves; ++g) c.wg_frame[g] = b;
      }
    }
  }
  if (tid == 0) {
    c.fchunk_first[c.B] = nch;
    h->fchunks = nch;
  }
  if (in_lds) {
    // thread t: workgroups [t*per_g, (t+1)*per_g), the first one's frame by
    // a search over the chunk starts, then walking forward
    if (tid == 0) s_first[c.B] = nch;
    __syncthreads();
    const int32_t per_g = (G + kBlock - 1) / kBlock;
    const int32_t g0 = tid * per_g, g1 = min(g0 + per_g, G);
    if (g0 < g1) {
      const uint32_t k = (uint32_t)g0 * kWaves;
      int32_t fb = 0, hi = c.B - 1;
      while (fb < hi) {
        const int32_t mid = (fb + hi + 1) >> 1;
        if (s_first[mid] <= k)
          fb = mid;
        else
          hi = mid - 1;
      }
      for (int32_t g = g0; g < g1; ++g) {
        const uint32_t kg = (uint32_t)g * kWaves;
        while (fb + 1 < c.B && s_first[fb + 1] <= kg) ++fb;
        c.wg_frame[g] = kg < nch ? (uint32_t)fb : kNoFrame;
      }
    }
  } else {
    for (int32_t g = (int32_t)((nch + kWaves - 1) / kWaves) + tid; g < G; g += kBlock) c.wg_frame[g] = kNoFrame;
  }
}

__global__ __launch_bounds__(kBlock) void stage_kernel(Config c) {
  __shared__ __align__(16) int16_t s_rect[kMaxRois][4];
  __shared__ uint32_t s_tmp[kWaves];
  __shared__ uint32_t s_word[kBlock];
  __shared__ int32_t s_bad;
  const int tid = threadIdx.x;
  const int b = blockIdx.y;
  if (blockIdx.x == gridDim.x - 1) {  // the extra column opens the call, beside the frames' work
    if (b == 0) open_call(c, s_tmp, reinterpret_cast<uint32_t*>(&s_rect[0][0]), &s_bad);
    return;
  }

  // ROIs of frame b (offsets clamped into [0, R], count into [0, max_rois])
  const int32_t r0 = min(max(c.roi_off[b], 0), c.R);
  const int32_t r1 = min(max(c.roi_off[b + 1], r0), c.R);
  const int32_t n = min(r1 - r0, c.max_rois);
  for (int j = tid; j < n; j += kBlock) roi_cell_rect(c, c.rois[r0 + j], s_rect[j]);
  __syncthreads();

  const int32_t ncol = (int32_t)gridDim.x - 1;  // without the opening column
  if (c.W == 1) {  // uniform
    // one ROI word: each thread owns kStageCellsPerThread cells at a time
    // and walks the frame's ROI rectangles once for all of them
    const int32_t stride = ncol * kBlock;
    for (int32_t g0 = (int32_t)blockIdx.x * kBlock + tid; g0 < c.ncells; g0 += stride * kStageCellsPerThread) {
      int32_t cx[kStageCellsPerThread], cy[kStageCellsPerThread];
      uint32_t word[kStageCellsPerThread];
#pragma unroll
      for (int i = 0; i < kStageCellsPerThread; ++i) {
        const int32_t cell = g0 + i * stride;
        cx[i] = cell % c.ncx;
        cy[i] = cell < c.ncells ? cell / c.ncx : 0x7fff;  // rows past the grid match no rectangle
        word[i] = 0;
      }
      for (int k = 0; k < n; ++k) {
        const int16_t* rc = s_rect[k];  // same address in every lane
        const int32_t x0 = rc[0], x1 = rc[1], y0 = rc[2], y1 = rc[3];
#pragma unroll
        for (int i = 0; i < kStageCellsPerThread; ++i)
          word[i] |= (cx[i] >= x0 && cx[i] <= x1 && cy[i] >= y0 && cy[i] <= y1) ? 1u << k : 0u;
      }
#pragma unroll
      for (int i = 0; i < kStageCellsPerThread; ++i) {
        const int32_t cell = g0 + i * stride;
        if (cell < c.ncells) c.cellmask[(int64_t)b * c.ncells + cell] = word[i];
      }
    }
  } else {
    // several ROI words: one (cell, word) per thread, the workgroup's cells
    // whole (cpw cells of W words), so that a cell's any-word is an OR in LDS
    const int32_t W = c.W;
    const int32_t cpw = max(kBlock / W, 1);
    const int64_t cell_words = (int64_t)c.ncells * W;
    const int32_t wl = tid % W;
    const int32_t knw = min(32, n - wl * 32);
    for (int32_t cell0 = (int32_t)blockIdx.x * cpw; cell0 < c.ncells; cell0 += ncol * cpw) {
      const int32_t cell = cell0 + tid / W;
      const bool active = tid < cpw * W && cell < c.ncells;
      const int32_t cx = cell % c.ncx, cy = active ? cell / c.ncx : 0x7fff;  // rows past the grid match no rectangle
      uint32_t word = 0;
      for (int k = 0; k < knw; ++k) {
        const int16_t* rc = s_rect[wl * 32 + k];
        word |= (cx >= rc[0] && cx <= rc[1] && cy >= rc[2] && cy <= rc[3]) ? 1u << k : 0u;
      }
      if (active) c.cellmask[(int64_t)b * cell_words + (int64_t)cell * W + wl] = word;
      s_word[tid] = active ? word : 0u;
      __syncthreads();
      if (tid < cpw && cell0 + tid < c.ncells) {
        uint32_t any = 0;
        for (int32_t w = 0; w < W; ++w) any |= s_word[tid * W + w];
        c.cellany[(int64_t)b * c.ncells + cell0 + tid] = any;
      }
      __syncthreads();
    }
  }
  // budget masks: one thread per (sweep, word)
  for (int32_t e = (int32_t)blockIdx.x * kBlock + tid; e < c.S * c.W; e += ncol * kBlock) {
    const int32_t s = e / c.W, w = e % c.W;
    uint32_t word = 0;
    const int kn = min(32, n - w * 32);
    if (kn > 0) {
      uint32_t bv[32];
#pragma unroll
      for (int k = 0; k < 32; ++k) bv[k] = c.budget[r0 + w * 32 + min(k, kn - 1)];  // together, then used
#pragma unroll
      for (int k = 0; k < 32; ++k)
        if (k < kn && (int32_t)bv[k] > s) word |= 1u << k;
    }
    c.budgetmask[((int64_t)b * c.S + s) * c.W + w] = word;
  }
}

__global__ __launch_bounds__(kBlock) void fill_zero_kernel(uint4* p, size_t n16, uint8_t* tail, size_t ntail) {
  size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x;
  for (; i < n16; i += (size_t)gridDim.x * kBlock) p[i] = make_uint4(0, 0, 0, 0);
  if (blockIdx.x == 0)
    for (size_t t = threadIdx.x; t < ntail; t += kBlock) tail[t] = 0;
}

// The fault word of a call, copied to the caller's int32 (one thread).
__global__ void copy_fault_kernel(const WsHeader* h, int32_t* out) {
  if (threadIdx.x == 0) *out = __hip_atomic_load(&h->fault, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace

hipError_t launch_stage(const Config& c, hipStream_t st) {
  // per frame, at most 64 workgroups plus the opening column: with one ROI
  // word, kStageCellsPerThread cells per thread; with several, kBlock / W
  // whole cells per workgroup (one word per thread)
  const int64_t cpw = c.W == 1 ? (int64_t)kBlock * kStageCellsPerThread : std::max<int64_t>(kBlock / c.W, 1);
  const int64_t work = std::max<int64_t>(((int64_t)c.ncells + cpw - 1) / cpw, ((int64_t)c.S * c.W + kBlock - 1) / kBlock);
  const int gx = (int)std::min<int64_t>(std::max<int64_t>(1, work), 64);
  hipLaunchKernelGGL(stage_kernel, dim3(gx + 1, c.B), dim3(kBlock), 0, st, c);
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

hipError_t launch_copy_fault(const WsHeader* h, int32_t* out, hipStream_t st) {
  hipLaunchKernelGGL(copy_fault_kernel, dim3(1), dim3(64), 0, st, h, out);
  return hipGetLastError();
}

}  // namespace mmbev

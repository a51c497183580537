// After the sort: voxels, per-frame cap, mean pooling.
//
// unique    -- flag the first pair of every run of equal (frame, key) in the
//              sorted order: heads are counted per chunk, then numbered (each
//              chunk adds the counts of the chunks before it); writes the
//              first sorted position of each voxel and the first voxel of
//              each frame.
// finalize  -- one workgroup: closes the per-frame voxel ranges (the head
//              scan writes the first voxel of every frame up to the last
//              kept pair's), flags the frames over max_voxels, and writes
//              the output offsets of every frame.
// cap       -- one workgroup per frame over max_voxels: radix select of the
//              voxels with the smallest first point index, then their rank
//              in key order (the output row inside the frame).
// mean      -- one thread per voxel: output row, and the mean of the voxel's
//              first max_points points, recomputing x', y', z' with the same
//              fused chain as the filter (Eq. 6) and summing in double in
//              ascending point order (Alg. 1 VoxelFeatureEncoder read as
//              mean pooling).
#include "launch.hpp"

namespace mmbev {

namespace {

__device__ __forceinline__ uint32_t local_key(const Config& c, uint32_t key) {
  return (c.key_has_frame && c.fb > 0) ? (key & ((1u << c.kb) - 1u)) : key;
}

// Frame b of voxel v from the per-frame voxel offsets: largest b, vox_off[b] <= v.
__device__ __forceinline__ int32_t frame_from_offsets(const Config& c, uint32_t v) {
  int32_t lo = 0, hi = c.B - 1;
  while (lo < hi) {
    int32_t mid = (lo + hi + 1) >> 1;
    if (c.vox_off[mid] <= v)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

// Frame of a sorted pair: from the key's top bits, or from the point index
// through frame offsets staged in LDS (off) or read from global memory.
__device__ __forceinline__ int32_t pair_frame(const Config& c, const uint32_t* off, bool lds, uint32_t key,
                                              uint32_t val) {
  if (c.B == 1) return 0;
  if (c.key_has_frame) return (int32_t)(key >> c.kb);
  if (!lds) return frame_of_point(c.frame_off, c.B, (int64_t)val);
  int32_t lo = 0, hi = c.B - 1;
  while (lo < hi) {
    int32_t mid = (lo + hi + 1) >> 1;
    if (off[mid] <= val)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

// Whether sorted pair k starts a voxel (the first pair, or a new frame or key).
__device__ __forceinline__ bool is_head(const Config& c, const uint32_t* keys, const uint32_t* vals, const uint32_t* off,
                                        bool lds, uint32_t k, int32_t& frame) {
  const uint32_t key = keys[k];
  const bool need_frame = !c.key_has_frame && c.B > 1;
  frame = pair_frame(c, off, lds, key, need_frame ? vals[k] : 0u);
  if (k == 0) return true;
  const uint32_t pk = keys[k - 1];
  if (pk != key) return true;
  if (!need_frame) return false;
  return pair_frame(c, off, lds, pk, vals[k - 1]) != frame;
}

// Heads per chunk of the sorted pairs.
__global__ __launch_bounds__(kBlock) void ucount_kernel(Config c, const uint32_t* keys, const uint32_t* vals) {
  __shared__ uint32_t s_tmp[kWaves];
  extern __shared__ uint32_t dyn_off[];
  const int tid = threadIdx.x;
  const uint32_t K = c.hdr->kept;
  const bool lds = !c.key_has_frame && c.B > 1 && c.B <= kMaxSortLdsFrames;
  if (lds)
    for (int e = tid; e <= c.B; e += kBlock)
      dyn_off[e] = (uint32_t)min(max(c.frame_off[e], (int64_t)0), (int64_t)c.N);
  __syncthreads();
  uint32_t lo, hi;
  chunk_range(K, blockIdx.x, gridDim.x, lo, hi);
  uint32_t n = 0;
  for (uint32_t k = lo + tid; k < hi; k += kBlock) {
    int32_t f;
    n += is_head(c, keys, vals, dyn_off, lds, k, f) ? 1u : 0u;
  }
  uint32_t total;
  (void)block_exclusive_scan(n, s_tmp, total);
  if (tid == 0) c.hcount[blockIdx.x] = total;
}

// Numbers the heads (the chunk's offset is the heads of all earlier chunks):
// first sorted position of every voxel, first voxel of every frame.
__global__ __launch_bounds__(kBlock) void uwrite_kernel(Config c, const uint32_t* keys, const uint32_t* vals) {
  __shared__ uint32_t s_tmp[kWaves];
  __shared__ uint32_t s_run;
  extern __shared__ uint32_t dyn_off[];
  const int tid = threadIdx.x;
  WsHeader* h = c.hdr;
  const uint32_t K = h->kept;
  const bool lds = !c.key_has_frame && c.B > 1 && c.B <= kMaxSortLdsFrames;
  if (lds)
    for (int e = tid; e <= c.B; e += kBlock)
      dyn_off[e] = (uint32_t)min(max(c.frame_off[e], (int64_t)0), (int64_t)c.N);
  {
    uint32_t part = 0;
    for (uint32_t w = tid; w < blockIdx.x; w += kBlock) part += c.hcount[w];
    uint32_t before;
    (void)block_exclusive_scan(part, s_tmp, before);
    if (tid == 0) {
      s_run = before;
      if (blockIdx.x == gridDim.x - 1) h->voxels = before + c.hcount[blockIdx.x];
    }
  }
  __syncthreads();
  uint32_t lo, hi;
  chunk_range(K, blockIdx.x, gridDim.x, lo, hi);
  for (uint32_t base = lo; base < hi; base += kScanTile) {
    // kScanItems consecutive pairs per thread
    const uint32_t first = base + tid * kScanItems;
    uint32_t heads = 0;
    int32_t frame[kScanItems];
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
      frame[j] = -1;
      const uint32_t k = first + j;
      if (k < hi) {
        int32_t f;
        if (is_head(c, keys, vals, dyn_off, lds, k, f)) heads |= 1u << j;
        frame[j] = f;
      }
    }
    uint32_t total;
    const uint32_t excl = block_exclusive_scan(__popc(heads), s_tmp, total);
    uint32_t vid = s_run + excl;
    // frame boundaries: a head whose frame is above its predecessor's starts
    // that frame and every empty frame before it
    int32_t pf = -1;
    if (first > 0 && first < hi) {
      const uint32_t pk = keys[first - 1];
      const bool need_frame = !c.key_has_frame && c.B > 1;
      pf = pair_frame(c, dyn_off, lds, pk, need_frame ? vals[first - 1] : 0u);
    }
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
      if (heads & (1u << j)) {
        c.seg_start[vid] = first + j;
        const int32_t f = min(frame[j], c.B - 1);
        for (int32_t b = pf + 1; b <= f; ++b) c.vox_off[b] = vid;
        ++vid;
      }
      if (frame[j] >= 0) pf = frame[j];
    }
    __syncthreads();
    if (tid == 0) s_run += total;
    __syncthreads();
  }
}

__global__ __launch_bounds__(kBlock) void finalize_kernel(Config c, const uint32_t* keys, const uint32_t* vals) {
  __shared__ uint32_t s_tmp[kWaves];
  __shared__ int32_t s_last;
  const int tid = threadIdx.x;
  WsHeader* h = c.hdr;
  const uint32_t V = h->voxels;
  const uint32_t K = h->kept;
  if (tid == 0) {
    c.seg_start[V] = K;
    s_last = K > 0 ? min(pair_frame(c, nullptr, false, keys[K - 1], vals[K - 1]), c.B - 1) : -1;
  }
  __syncthreads();
  // frames after the last kept pair's frame start at V
  for (int b = s_last + 1 + tid; b <= c.B; b += kBlock) c.vox_off[b] = V;
  __syncthreads();
  uint32_t carry_out = 0, carry_cap = 0;
  for (int chunk = 0; chunk < c.B; chunk += kBlock) {
    const int b = chunk + tid;
    const uint32_t vb = b < c.B ? c.vox_off[b + 1] - c.vox_off[b] : 0u;
    const uint32_t capped = vb > (uint32_t)c.cap;
    const uint32_t outc = capped ? (uint32_t)c.cap : vb;
    uint32_t t1, t2;
    const uint32_t e1 = block_exclusive_scan(outc, s_tmp, t1);
    (void)block_exclusive_scan(capped ? vb : 0u, s_tmp, t2);
    if (b < c.B) c.out_voxel_offsets[b] = (int64_t)(carry_out + e1);
    carry_out += t1;
    carry_cap += t2;
  }
  if (tid == 0) {
    c.out_voxel_offsets[c.B] = (int64_t)carry_out;
    h->capped_voxels = carry_cap;
    h->any_capped = carry_cap > 0 ? 1u : 0u;
  }
}

// One workgroup per frame; frames within the cap return at once.  Selects
// the max_voxels voxels with the smallest first point index (radix select of
// the max_voxels-th smallest first index, four 8-bit rounds; first indices
// are distinct), then numbers the kept voxels in key order.
__global__ __launch_bounds__(kBlock) void cap_kernel(Config c, const uint32_t* vals) {
  __shared__ uint32_t s_hist[256];
  __shared__ uint32_t s_tmp[kWaves];
  __shared__ uint32_t s_sel, s_k;
  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  WsHeader* h = c.hdr;
  const uint32_t v0 = c.vox_off[b];
  const uint32_t nv = c.vox_off[b + 1] - v0;
  if (nv <= (uint32_t)c.cap || h->kept == 0) return;
  const uint32_t K = h->kept;
  uint32_t* fk = c.capkey + v0;
  for (uint32_t v = tid; v < nv; v += kBlock) fk[v] = vals[min(c.seg_start[v0 + v], K - 1)];
  __syncthreads();
  uint32_t prefix = 0, pmask = 0, k = (uint32_t)c.cap;
  for (int shift = 24; shift >= 0; shift -= 8) {
    s_hist[tid] = 0;
    __syncthreads();
    for (uint32_t v = tid; v < nv; v += kBlock) {
      const uint32_t key = fk[v];
      if ((key & pmask) == prefix) atomicAdd(&s_hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    uint32_t total;
    const uint32_t cnt = s_hist[tid];
    const uint32_t excl = block_exclusive_scan(cnt, s_tmp, total);
    if (excl < k && excl + cnt >= k) {  // the bin holding the k-th smallest
      s_sel = (uint32_t)tid;
      s_k = k - excl;
    }
    __syncthreads();
    prefix |= s_sel << shift;
    pmask |= 255u << shift;
    k = s_k;
    __syncthreads();
  }
  const uint32_t threshold = prefix;  // the max_voxels-th smallest first index
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nv; base += kBlock) {
    const uint32_t v = base + tid;
    const bool keep = v < nv && fk[v] <= threshold;
    uint32_t total;
    const uint32_t excl = block_exclusive_scan(keep ? 1u : 0u, s_tmp, total);
    if (v < nv) c.out_rank[v0 + v] = keep ? carry + excl : 0xffffffffu;
    carry += total;
  }
}

// One thread per voxel (grid-stride): output row, kept count, point indices
// and the fp64 mean of every feature.
__global__ __launch_bounds__(kBlock) void mean_kernel(Config c, const uint32_t* keys, const uint32_t* vals) {
  WsHeader* h = c.hdr;
  const uint32_t V = h->voxels;
  const uint32_t K = h->kept;
  const int64_t rows = (int64_t)c.B * c.cap;
  const int C = c.C, M = c.M;
  for (uint32_t v = blockIdx.x * kBlock + threadIdx.x; v < V; v += gridDim.x * kBlock) {
    const int32_t b = frame_from_offsets(c, v);
    const uint32_t v0 = c.vox_off[b];
    const bool capped = c.vox_off[b + 1] - v0 > (uint32_t)c.cap;
    const uint32_t rank = capped ? c.out_rank[v] : v - v0;
    if (rank == 0xffffffffu) continue;
    const int64_t row = c.out_voxel_offsets[b] + (int64_t)rank;
    if (row < 0 || row >= rows) {
      raise_fault(h, MMBEV_FAULT_WAIT);
      continue;
    }
    const uint32_t s0 = min(c.seg_start[v], K), s1 = max(min(c.seg_start[v + 1], K), s0);
    const uint32_t cnt = min(s1 - s0, (uint32_t)M);
    const uint32_t kl = local_key(c, keys[s0]);
    const uint32_t ix = kl % c.Dx, rest = kl / c.Dx;
    const uint32_t iy = rest % c.Dy, iz = rest / c.Dy;
    int32_t* co = c.out_coords + row * 4;
    co[0] = b;
    co[1] = (int32_t)iz;
    co[2] = (int32_t)iy;
    co[3] = (int32_t)ix;
    c.out_counts[row] = (int32_t)cnt;
    double sum[8];
#pragma unroll
    for (int f = 0; f < 8; ++f) sum[f] = 0.0;
    int32_t* pidx = c.out_point_idx + row * M;
    for (uint32_t m = 0; m < cnt; ++m) {
      const uint32_t i = min(vals[s0 + m], (uint32_t)c.N - 1u);
      pidx[m] = (int32_t)i;
      const uint32_t s = min((uint32_t)c.sweep[i], (uint32_t)c.S - 1u);
      const float* P = c.poses + ((int64_t)b * c.S + s) * 12;
      float Pl[12];
#pragma unroll
      for (int q = 0; q < 12; ++q) Pl[q] = P[q];
      float px, py, pz;
      compensate(Pl, c.feat[i], c.feat[c.stride + i], c.feat[2 * c.stride + i], px, py, pz);
      sum[0] += (double)px;
      sum[1] += (double)py;
      sum[2] += (double)pz;
#pragma unroll
      for (int f = 3; f < 8; ++f)
        if (f < C) sum[f] += (double)c.feat[(int64_t)f * c.stride + i];
    }
    for (int m = (int)cnt; m < M; ++m) pidx[m] = -1;
    float* fo = c.out_feats + row * C;
#pragma unroll
    for (int f = 0; f < 8; ++f)
      if (f < C) fo[f] = (float)(sum[f] / (double)cnt);
  }
}

}  // namespace

hipError_t launch_unique(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st) {
  const bool lds = !c.key_has_frame && c.B > 1 && c.B <= kMaxSortLdsFrames;
  const size_t dyn = lds ? (size_t)(c.B + 1) * 4 : 0;
  hipLaunchKernelGGL(ucount_kernel, dim3(c.sort_chunks), dim3(kBlock), dyn, st, c, keys, vals);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(uwrite_kernel, dim3(c.sort_chunks), dim3(kBlock), dyn, st, c, keys, vals);
  return hipGetLastError();
}

hipError_t launch_finalize(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st) {
  hipLaunchKernelGGL(finalize_kernel, dim3(1), dim3(kBlock), 0, st, c, keys, vals);
  return hipGetLastError();
}

hipError_t launch_cap(const Config& c, const uint32_t* vals, hipStream_t st) {
  hipLaunchKernelGGL(cap_kernel, dim3(c.B), dim3(kBlock), 0, st, c, vals);
  return hipGetLastError();
}

hipError_t launch_mean(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st) {
  hipLaunchKernelGGL(mean_kernel, dim3(c.mean_grid), dim3(kBlock), 0, st, c, keys, vals);
  return hipGetLastError();
}

}  // namespace mmbev

// After the sort: voxels, per-frame cap, mean pooling.
//
// unique    -- flag the first pair of every run of equal (frame, key) in the
//              sorted order and number them with a chained scan (decoupled
//              look-back); writes the first sorted position of each voxel.
// finalize  -- one workgroup: per-frame voxel ranges (binary search over the
//              frame-ordered voxels), which frames exceed max_voxels, the
//              output offsets of every frame.
// cap_prep  -- for frames over the cap only: (first point index, voxel id)
//              pairs for the first-appearance sort.
// mean      -- one thread per voxel: keep flag, output row (a chained scan of
//              the keep flags when some frame was capped), and the mean of
//              the voxel's first max_points points, recomputing x', y', z'
//              with the same fused chain as the filter (Eq. 6) and summing
//              in double in ascending point order (Alg. 1 VoxelFeatureEncoder
//              read as mean pooling).
#include "launch.hpp"

namespace mmbev {

namespace {

__device__ __forceinline__ uint32_t local_key(const Config& c, uint32_t key) {
  return (c.key_has_frame && c.fb > 0) ? (key & ((1u << c.kb) - 1u)) : key;
}

__device__ __forceinline__ int32_t frame_of_voxel(const Config& c, const uint32_t* keys, const uint32_t* vals,
                                                  uint32_t v) {
  if (c.B == 1) return 0;
  uint32_t p = min(c.seg_start[v], c.hdr->kept - 1u);  // clamp: never trust device data for an address
  if (c.key_has_frame) return (int32_t)(keys[p] >> c.kb);
  return frame_of_point(c.frame_off, c.B, (int64_t)vals[p]);
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

__global__ __launch_bounds__(kBlock) void unique_kernel(Config c, const uint32_t* keys, const uint32_t* vals) {
  __shared__ uint32_t s_ticket, s_prefix, s_tmp[kWaves];
  const int tid = threadIdx.x;
  WsHeader* h = c.hdr;
  const uint32_t K = h->kept;
  const uint32_t ntiles = (K + kScanTile - 1) / kScanTile;
  if (ntiles == 0) return;
  const uint32_t tag = tag_of(h->epoch, kSlotUnique);
  const bool need_frame = !c.key_has_frame && c.B > 1;

  for (;;) {
    if (tid == 0) s_ticket = atomicAdd(&h->tickets[kSlotUnique], 1u);
    __syncthreads();
    const uint32_t t = s_ticket;
    if (t >= ntiles) break;
    const int64_t base = (int64_t)t * kScanTile + (int64_t)tid * kScanItems;
    uint32_t k[kScanItems];
    if (base + kScanItems <= (int64_t)K) {
      const uint4* src = reinterpret_cast<const uint4*>(keys + base);
#pragma unroll
      for (int q = 0; q < kScanItems / 4; ++q) {
        uint4 u = src[q];
        k[4 * q] = u.x;
        k[4 * q + 1] = u.y;
        k[4 * q + 2] = u.z;
        k[4 * q + 3] = u.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < kScanItems; ++j) k[j] = base + j < (int64_t)K ? keys[base + j] : 0u;
    }
    uint32_t heads = 0;
    uint32_t prev_key = (base > 0 && base < (int64_t)K) ? keys[base - 1] : 0u;
    int32_t prev_frame = -1;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
      int64_t idx = base + j;
      if (idx < (int64_t)K) {
        bool head = idx == 0 || k[j] != prev_key;
        if (!head && need_frame) {
          if (prev_frame < 0) prev_frame = frame_of_point(c.frame_off, c.B, (int64_t)vals[idx - 1]);
          int32_t f = frame_of_point(c.frame_off, c.B, (int64_t)vals[idx]);
          head = f != prev_frame;
          prev_frame = f;
        } else {
          prev_frame = -1;
        }
        if (head) heads |= 1u << j;
        prev_key = k[j];
      }
    }
    uint32_t total;
    uint32_t excl = block_exclusive_scan(__popc(heads), s_tmp, total);
    if (tid == 0) {
      uint32_t prefix = 0;
      uint64_t* st = c.scan_status;
      if (t == 0) {
        status_store(st, status_word(tag, kFlagIncl, total));
      } else {
        status_store(st + t, status_word(tag, kFlagAgg, total));
        prefix = look_back(st, t, 1, tag, h);
        status_store(st + t, status_word(tag, kFlagIncl, prefix + total));
      }
      s_prefix = prefix;
      if (t == ntiles - 1) h->voxels = prefix + total;
    }
    __syncthreads();
    uint32_t v = s_prefix + excl;
    while (heads) {
      int j = __builtin_ctz(heads);
      heads &= heads - 1;
      c.seg_start[v++] = (uint32_t)(base + j);
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(kBlock) void finalize_kernel(Config c, const uint32_t* keys, const uint32_t* vals) {
  __shared__ uint32_t s_tmp[kWaves];
  const int tid = threadIdx.x;
  WsHeader* h = c.hdr;
  const uint32_t V = h->voxels;
  if (tid == 0) c.seg_start[V] = h->kept;
  __syncthreads();
  for (int b = tid; b <= c.B; b += kBlock) {
    uint32_t lo = 0, hi = V;  // first voxel whose frame is >= b
    if (b == c.B) {
      lo = V;
    } else {
      while (lo < hi) {
        uint32_t mid = (lo + hi) >> 1;
        if (frame_of_voxel(c, keys, vals, mid) < b)
          lo = mid + 1;
        else
          hi = mid;
      }
    }
    c.vox_off[b] = lo;
  }
  __syncthreads();
  uint32_t carry_out = 0, carry_cap = 0;
  for (int chunk = 0; chunk < c.B; chunk += kBlock) {
    int b = chunk + tid;
    uint32_t vb = b < c.B ? c.vox_off[b + 1] - c.vox_off[b] : 0u;
    uint32_t capped = vb > (uint32_t)c.cap;
    uint32_t outc = capped ? (uint32_t)c.cap : vb;
    uint32_t t1, t2;
    uint32_t e1 = block_exclusive_scan(outc, s_tmp, t1);
    uint32_t e2 = block_exclusive_scan(capped ? vb : 0u, s_tmp, t2);
    if (b < c.B) {
      c.out_voxel_offsets[b] = (int64_t)(carry_out + e1);
      c.cap_off[b] = carry_cap + e2;
    }
    carry_out += t1;
    carry_cap += t2;
  }
  if (tid == 0) {
    c.out_voxel_offsets[c.B] = (int64_t)carry_out;
    c.cap_off[c.B] = carry_cap;
    h->capped_voxels = carry_cap;
    h->any_capped = carry_cap > 0 ? 1u : 0u;
  }
}

__global__ __launch_bounds__(kBlock) void cap_prep_kernel(Config c, const uint32_t* vals, uint32_t* ckeys,
                                                          uint32_t* cvals) {
  __shared__ uint32_t s_hist[kMaxPasses][kSortBins];
  WsHeader* h = c.hdr;
  if (!h->any_capped) return;
  const int tid = threadIdx.x;
  const uint32_t nbins = 1u << c.cap_dbits;
  for (int e = tid; e < kMaxPasses * kSortBins; e += kBlock) (&s_hist[0][0])[e] = 0;
  __syncthreads();
  const uint32_t V = h->voxels;
  for (uint32_t v = blockIdx.x * kBlock + tid; v < V; v += gridDim.x * kBlock) {
    int32_t b = frame_from_offsets(c, v);
    uint32_t v0 = c.vox_off[b], vb = c.vox_off[b + 1] - v0;
    if (vb > (uint32_t)c.cap) {
      uint32_t q = c.cap_off[b] + (v - v0);
      uint32_t first = vals[min(c.seg_start[v], h->kept - 1u)];
      ckeys[q] = first;
      cvals[q] = v;
      for (int p = 0; p < c.cap_passes; ++p) atomicAdd(&s_hist[p][(first >> (p * c.cap_dbits)) & (nbins - 1)], 1u);
    }
  }
  __syncthreads();
  for (int e = tid; e < c.cap_passes * (int)nbins; e += kBlock) {
    uint32_t x = s_hist[e / nbins][e % nbins];
    if (x) atomicAdd(&h->hist[1][e / nbins][e % nbins], x);
  }
}

__global__ __launch_bounds__(kBlock) void mean_kernel(Config c, const uint32_t* keys, const uint32_t* vals) {
  __shared__ uint32_t s_ticket, s_prefix, s_tmp[kWaves];
  const int tid = threadIdx.x;
  WsHeader* h = c.hdr;
  const uint32_t V = h->voxels;
  const uint32_t K = h->kept;
  const int64_t rows = (int64_t)c.B * c.cap;
  const bool any_capped = h->any_capped != 0;
  const uint32_t ntiles = (V + kMeanTile - 1) / kMeanTile;
  if (ntiles == 0) return;
  const uint32_t tag = tag_of(h->epoch, kSlotMean);
  const int C = c.C, M = c.M;

  for (;;) {
    if (tid == 0) s_ticket = atomicAdd(&h->tickets[kSlotMean], 1u);
    __syncthreads();
    const uint32_t t = s_ticket;
    if (t >= ntiles) break;
    const uint32_t v = t * kMeanTile + tid;
    bool keep = v < V;
    int32_t b = 0;
    if (keep) {
      b = frame_from_offsets(c, v);
      if (any_capped) {
        uint32_t v0 = c.vox_off[b];
        if (c.vox_off[b + 1] - v0 > (uint32_t)c.cap) keep = c.keepflag[c.cap_off[b] + (v - v0)] != 0;
      }
    }
    uint32_t row = v;
    if (any_capped) {
      uint32_t total;
      uint32_t excl = block_exclusive_scan(keep ? 1u : 0u, s_tmp, total);
      if (tid == 0) {
        uint32_t prefix = 0;
        uint64_t* st = c.mean_status;
        if (t == 0) {
          status_store(st, status_word(tag, kFlagIncl, total));
        } else {
          status_store(st + t, status_word(tag, kFlagAgg, total));
          prefix = look_back(st, t, 1, tag, h);
          status_store(st + t, status_word(tag, kFlagIncl, prefix + total));
        }
        s_prefix = prefix;
      }
      __syncthreads();
      row = s_prefix + excl;
    }
    if (keep && (int64_t)row >= rows) {
      raise_fault(h, MMBEV_FAULT_WAIT);
      keep = false;
    }
    if (keep) {
      const uint32_t s0 = min(c.seg_start[v], K), s1 = max(min(c.seg_start[v + 1], K), s0);
      const uint32_t cnt = min(s1 - s0, (uint32_t)M);
      const uint32_t kl = local_key(c, keys[s0]);
      const uint32_t ix = kl % c.Dx, rest = kl / c.Dx;
      const uint32_t iy = rest % c.Dy, iz = rest / c.Dy;
      int32_t* co = c.out_coords + (int64_t)row * 4;
      co[0] = b;
      co[1] = (int32_t)iz;
      co[2] = (int32_t)iy;
      co[3] = (int32_t)ix;
      c.out_counts[row] = (int32_t)cnt;
      double sum[8];
#pragma unroll
      for (int f = 0; f < 8; ++f) sum[f] = 0.0;
      int32_t* pidx = c.out_point_idx + (int64_t)row * M;
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
      float* fo = c.out_feats + (int64_t)row * C;
#pragma unroll
      for (int f = 0; f < 8; ++f)
        if (f < C) fo[f] = (float)(sum[f] / (double)cnt);
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_unique(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st) {
  hipLaunchKernelGGL(unique_kernel, dim3(c.scan_grid), dim3(kBlock), 0, st, c, keys, vals);
  return hipGetLastError();
}

hipError_t launch_finalize(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st) {
  hipLaunchKernelGGL(finalize_kernel, dim3(1), dim3(kBlock), 0, st, c, keys, vals);
  return hipGetLastError();
}

hipError_t launch_cap_prep(const Config& c, const uint32_t* vals, uint32_t* ckeys, uint32_t* cvals,
                           hipStream_t st) {
  hipLaunchKernelGGL(cap_prep_kernel, dim3(c.mean_grid), dim3(kBlock), 0, st, c, vals, ckeys, cvals);
  return hipGetLastError();
}

hipError_t launch_mean(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st) {
  hipLaunchKernelGGL(mean_kernel, dim3(c.mean_grid), dim3(kBlock), 0, st, c, keys, vals);
  return hipGetLastError();
}

}  // namespace mmbev

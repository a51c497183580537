// After the sort: voxels, per-frame cap, mean pooling.
//
// The sorted pairs are grouped by frame and ordered by key inside each
// frame; the pair chunks of the radix passes (each inside one frame) are
// reused.  Per-voxel data sits at slot fstart[b] + v for voxel v of frame b
// (a frame has no more voxels than kept pairs).
// ucount   -- heads (first pair of every run of equal keys inside a frame)
//             per pair chunk;
// uwrite   -- numbers the heads inside their frame (the heads of the frame's
//             earlier chunks come first) and writes each voxel's first
//             sorted pair at its slot;
// finalize -- one workgroup: every frame's voxels, the voxels of the frames
//             before it (global voxel numbering), and the output offsets of
//             every frame (at most max_voxels rows each) with the
//             capped-voxel count;
// cap      -- one workgroup per frame: the frame of each tile of the mean
//             that starts in it; for frames over max_voxels, radix select
//             of the voxels with the smallest first point index, then their
//             rank in key order (the output row inside the frame);
// mean     -- one thread per voxel: output row, and the mean of the voxel's
//             first max_points points from their compact records (x', y',
//             z' of Eq. 6 and the raw features), summed in double in
//             ascending point order (Alg. 1 VoxelFeatureEncoder read as mean
//             pooling).
#include "launch.hpp"

namespace mmbev {

namespace {

// Frame b of global voxel g: largest b in [lo, hi] with vox_off[b] <= g
// (the caller knows g's frame lies in that range).
__device__ __forceinline__ int32_t frame_of_voxel(const Config& c, uint32_t g, int32_t lo, int32_t hi) {
  while (lo < hi) {
    int32_t mid = (lo + hi + 1) >> 1;
    if (c.vox_off[mid] <= g)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

// Whether sorted pair i of a frame whose first pair is ff starts a voxel.
__device__ __forceinline__ bool is_head(const uint32_t* keys, uint32_t ff, uint32_t i) {
  return i == ff || keys[i] != keys[i - 1];
}

__global__ __launch_bounds__(kBlock) void ucount_kernel(Config c, const uint32_t* keys) {
  __shared__ uint32_t s_tmp[kWaves];
  const int tid = threadIdx.x;
  const uint32_t k = blockIdx.x;
  const uint32_t nsc = c.hdr->schunks;
  const uint4 ch = c.schunk[k];  // in bounds for any k < schunk_max: loads with the count
  asm volatile("" ::"s"(ch.x), "s"(ch.y), "s"(ch.z), "s"(ch.w));  // keeps the load above the check
  if (k >= nsc) return;
  const uint32_t lo = ch.x, hi = ch.y, ff = ch.w;
  uint32_t n = 0;
  for (uint32_t base = lo; base < hi; base += kBlock * kCountItems) {
    bool hd[kCountItems];
#pragma unroll
    for (int j = 0; j < kCountItems; ++j) {
      const uint32_t i = base + j * kBlock + tid;
      hd[j] = i < hi && is_head(keys, ff, i);
    }
#pragma unroll
    for (int j = 0; j < kCountItems; ++j) n += hd[j] ? 1u : 0u;
  }
  uint32_t total;
  (void)block_exclusive_scan(n, s_tmp, total);
  if (tid == 0) c.hcount[k] = total;
}

__global__ __launch_bounds__(kBlock) void uwrite_kernel(Config c, const uint32_t* keys) {
  __shared__ uint32_t s_tmp[kWaves];
  __shared__ uint32_t s_off[kCountItems][kWaves];  // heads before row j of wave w in the batch
  __shared__ uint32_t s_batch;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const uint32_t k = blockIdx.x;
  const uint32_t nsc = c.hdr->schunks;
  const uint4 ch = c.schunk[k];  // in bounds for any k < schunk_max: loads with the count
  asm volatile("" ::"s"(ch.x), "s"(ch.y), "s"(ch.z), "s"(ch.w));  // keeps the load above the check
  if (k >= nsc) return;
  const uint32_t lo = ch.x, hi = ch.y, ff = ch.w;
  uint32_t v0;
  {
    uint32_t part = 0;
    for (uint32_t w = c.schunk_first[ch.z] + tid; w < k; w += kBlock) part += c.hcount[w];
    uint32_t before;
    (void)block_exclusive_scan(part, s_tmp, before);
    v0 = before;
  }
  // batches of kCountItems rows of kBlock consecutive pairs (coalesced);
  // heads numbered in pair order: row, then wave, then lane
  for (uint32_t base = lo; base < hi; base += kBlock * kCountItems) {
    uint64_t m[kCountItems];
#pragma unroll
    for (int j = 0; j < kCountItems; ++j) {
      const uint32_t i = base + j * kBlock + tid;
      m[j] = __ballot(i < hi && is_head(keys, ff, i));
    }
    if (lane == 0)
#pragma unroll
      for (int j = 0; j < kCountItems; ++j) s_off[j][wave] = (uint32_t)__popcll(m[j]);
    __syncthreads();
    if (tid == 0) {
      uint32_t run = 0;
      for (int j = 0; j < kCountItems; ++j)
        for (int w = 0; w < kWaves; ++w) {
          const uint32_t x = s_off[j][w];
          s_off[j][w] = run;
          run += x;
        }
      s_batch = run;
    }
    __syncthreads();
    const uint64_t lt = lanemask_lt();
#pragma unroll
    for (int j = 0; j < kCountItems; ++j)
      if ((m[j] >> lane) & 1u)
        c.seg_start[ff + v0 + s_off[j][wave] + (uint32_t)__popcll(m[j] & lt)] = base + j * kBlock + tid;
    v0 += s_batch;
    __syncthreads();
  }
}

// Exclusive prefix of n values in[0..n) written to out (may alias, or null);
// returns the total.  One workgroup, kScanItems consecutive values per thread.
__device__ uint32_t scan_array(const uint32_t* in, uint32_t* out, uint32_t n, uint32_t* s_tmp) {
  const int tid = threadIdx.x;
  uint32_t carry = 0;
  for (uint32_t base = 0; base < n; base += kScanTile) {
    const uint32_t first = base + tid * kScanItems;
    uint32_t v[kScanItems], sum = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
      v[j] = first + j < n ? in[first + j] : 0u;
      sum += v[j];
    }
    uint32_t total;
    uint32_t run = carry + block_exclusive_scan(sum, s_tmp, total);
    if (out)
#pragma unroll
      for (int j = 0; j < kScanItems; ++j)
        if (first + j < n) {
          out[first + j] = run;
          run += v[j];
        }
    carry += total;
  }
  return carry;
}

__global__ __launch_bounds__(kBlock) void finalize_kernel(Config c) {
  __shared__ uint32_t s_tmp[kWaves];
  const int tid = threadIdx.x;
  WsHeader* h = c.hdr;
  const uint32_t ns = h->schunks;
  // heads before every pair chunk (in place), then every frame's voxels
  const uint32_t V = scan_array(c.hcount, c.hcount, ns, s_tmp);
  __syncthreads();
  for (int b = tid; b < c.B; b += kBlock) {
    const uint32_t k0 = min(c.schunk_first[b], ns), k1 = min(c.schunk_first[b + 1], ns);
    c.vcount[b] = (k1 < ns ? c.hcount[k1] : V) - (k0 < ns ? c.hcount[k0] : V);
  }
  __syncthreads();
  (void)scan_array(c.vcount, c.vox_off, (uint32_t)c.B, s_tmp);
  if (tid == 0) {
    c.vox_off[c.B] = V;
    h->voxels = V;
  }
  if (tid == 0) c.tile_frame[(V + kMeanTile - 1) / kMeanTile] = (uint32_t)(c.B - 1);
  uint32_t carry_out = 0, carry_cap = 0;
  for (int chunk = 0; chunk < c.B; chunk += kBlock) {
    const int b = chunk + tid;
    const uint32_t vb = b < c.B ? c.vcount[b] : 0u;
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

// One workgroup per frame: the frame's entries of the mean's tile table;
// then frames within the cap return.  Selects the max_voxels voxels with the smallest first point index (radix select of
// the max_voxels-th smallest first index, four 8-bit rounds; first indices
// are distinct), then numbers the kept voxels in key order.
__global__ __launch_bounds__(kBlock) void cap_kernel(Config c, const uint32_t* vals) {
  __shared__ uint32_t s_hist[256];
  __shared__ uint32_t s_tmp[kWaves];
  __shared__ uint32_t s_sel, s_k;
  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  {
    // frame b for the tiles of kMeanTile voxels whose first voxel is in it
    // (the mean's workgroups search only between the frames of their tile
    // and of the next one)
    const uint32_t v0 = c.vox_off[b], v1 = c.vox_off[b + 1];
    for (uint32_t t = (v0 + kMeanTile - 1) / kMeanTile + tid; (uint64_t)t * kMeanTile < v1; t += kBlock)
      c.tile_frame[t] = (uint32_t)b;
  }
  const uint32_t nv = c.vcount[b];
  if (nv <= (uint32_t)c.cap) return;
  const uint32_t fs = c.fstart[b];
  uint32_t* fk = c.capkey + fs;
  for (uint32_t v = tid; v < nv; v += kBlock) fk[v] = vals[c.seg_start[fs + v]];
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
    if (v < nv) c.out_rank[fs + v] = keep ? carry + excl : 0xffffffffu;
    carry += total;
  }
}

// Workgroups of kMeanTile consecutive voxels (grid-stride), one thread per
// voxel: output row, kept count, point indices and the fp64 mean of every
// feature.  The records of a voxel's points are read kMeanBatch at a time,
// all their loads in flight together.  When the block's rows are consecutive (no frame
// over the cap in it) the rows are assembled in LDS and written as
// contiguous runs; otherwise each thread writes its own row.
constexpr int kMeanBatch = 4;  // more records in flight per thread cost occupancy (VGPRs)

__global__ __launch_bounds__(kBlock) void mean_kernel(Config c, const uint32_t* keys, const uint32_t* vals) {
  extern __shared__ uint32_t sm[];
  __shared__ int64_t s_row0;
  __shared__ uint32_t s_contig;
  WsHeader* h = c.hdr;
  const int tid = threadIdx.x;
  const uint32_t V = h->voxels;
  const uint32_t K = h->kept;
  const int64_t rows = (int64_t)c.B * c.cap;
  const int C = c.C, M = c.M;
  int32_t* l_co = (int32_t*)sm;              // [kMeanTile][4]
  float* l_ft = (float*)(sm + kMeanTile * 4);  // [kMeanTile][C]
  int32_t* l_pi = (int32_t*)(sm + kMeanTile * (4 + C));  // [kMeanTile][M]
  for (uint32_t g0 = blockIdx.x * kMeanTile; g0 < V; g0 += gridDim.x * kMeanTile) {
    const uint32_t g = g0 + tid;
    const uint32_t nblk = min((uint32_t)kMeanTile, V - g0);
    // the tile's voxels lie in frames tile_frame[t] .. tile_frame[t + 1]
    const uint32_t tl = g0 / kMeanTile;
    const int32_t fa = min((int32_t)c.tile_frame[tl], c.B - 1);
    const int32_t fb = min(max((int32_t)c.tile_frame[tl + 1], fa), c.B - 1);
    int64_t row = -1;
    int32_t b = 0;
    uint32_t s0 = 0, cnt = 0;
    if (g < V) {
      b = frame_of_voxel(c, g, fa, fb);
      const uint32_t v = g - c.vox_off[b];
      const uint32_t nv = c.vox_off[b + 1] - c.vox_off[b];
      const uint32_t slot = c.fstart[b] + v;
      const uint32_t rank = nv > (uint32_t)c.cap ? c.out_rank[slot] : v;
      if (rank != 0xffffffffu) {
        row = c.out_voxel_offsets[b] + (int64_t)rank;
        if (row < 0 || row >= rows || slot >= K) {
          raise_fault(h, MMBEV_FAULT_INTERNAL);
          row = -1;
        } else {
          s0 = min(c.seg_start[slot], K - 1u);
          const uint32_t s1 = max(min(v + 1 < nv ? c.seg_start[slot + 1] : c.fstart[b + 1], K), s0 + 1u);
          cnt = min(s1 - s0, (uint32_t)M);
        }
      }
    }
    if (tid == 0) {
      s_row0 = row;
      s_contig = 1;
    }
    __syncthreads();
    if ((uint32_t)tid < nblk && (row < 0 || row != s_row0 + tid)) s_contig = 0;  // every row valid and in order
    // the voxel's coordinates and points
    int32_t co[4] = {0, 0, 0, 0};
    double sum[8];
#pragma unroll
    for (int f = 0; f < 8; ++f) sum[f] = 0.0;
    if (row >= 0) {
      const uint32_t kl = keys[s0];
      const uint32_t ix = kl % c.Dx, rest = kl / c.Dx;
      co[0] = b;
      co[1] = (int32_t)(rest / c.Dy);
      co[2] = (int32_t)(rest % c.Dy);
      co[3] = (int32_t)ix;
    }
    __syncthreads();
    const bool contig = s_contig != 0;
    int32_t* pidx = contig ? l_pi + tid * M : c.out_point_idx + row * M;
    const int RW = c.rec_words;
    for (uint32_t m0 = 0; m0 < cnt; m0 += kMeanBatch) {
      uint32_t q[kMeanBatch];
      uint4 r0[kMeanBatch], r1[kMeanBatch];
#pragma unroll
      for (int j = 0; j < kMeanBatch; ++j) q[j] = m0 + j < cnt ? min(vals[s0 + m0 + j], K - 1u) : 0u;
#pragma unroll
      for (int j = 0; j < kMeanBatch; ++j) {  // one or two 16-byte loads per record
        const uint4* r = reinterpret_cast<const uint4*>(c.rec + (int64_t)q[j] * RW);
        if (m0 + j < cnt) {
          r0[j] = r[0];
          r1[j] = RW > 4 ? r[1] : make_uint4(0, 0, 0, 0);
        } else {
          r0[j] = r1[j] = make_uint4(0, 0, 0, 0);
        }
      }
#pragma unroll
      for (int j = 0; j < kMeanBatch; ++j)
        if (m0 + j < cnt) {
          const uint32_t w[8] = {r0[j].y, r0[j].z, r0[j].w, r1[j].x, r1[j].y, r1[j].z, r1[j].w, 0u};
#pragma unroll
          for (int f = 0; f < 7; ++f) sum[f] += (double)__uint_as_float(w[f]);  // ascending point order
          pidx[m0 + j] = (int32_t)r0[j].x;
        }
      if (C == 8)  // the eighth feature sits in a third 16-byte word
#pragma unroll
        for (int j = 0; j < kMeanBatch; ++j)
          if (m0 + j < cnt) sum[7] += (double)__uint_as_float(c.rec[(int64_t)q[j] * RW + 8]);
    }
    if (row >= 0) {
      for (int m = (int)cnt; m < M; ++m) pidx[m] = -1;
      c.out_counts[row] = (int32_t)cnt;
      if (contig) {
#pragma unroll
        for (int q = 0; q < 4; ++q) l_co[tid * 4 + q] = co[q];
#pragma unroll
        for (int f = 0; f < 8; ++f)
          if (f < C) l_ft[tid * C + f] = (float)(sum[f] / (double)cnt);
      } else {
        int32_t* o = c.out_coords + row * 4;
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = co[q];
        float* fo = c.out_feats + row * C;
#pragma unroll
        for (int f = 0; f < 8; ++f)
          if (f < C) fo[f] = (float)(sum[f] / (double)cnt);
      }
    }
    __syncthreads();
    if (contig) {
      // rows s_row0 .. s_row0 + nblk - 1, written as contiguous runs with
      // non-temporal stores: the call does not read them again, and lines
      // left dirty in the caches would be written back while the next
      // call's filter streams its points
      const int64_t r0 = s_row0;
      for (uint32_t e = tid; e < nblk * 4; e += kBlock) __builtin_nontemporal_store(l_co[e], &c.out_coords[r0 * 4 + e]);
      for (uint32_t e = tid; e < nblk * (uint32_t)C; e += kBlock)
        __builtin_nontemporal_store(l_ft[e], &c.out_feats[r0 * C + e]);
      for (uint32_t e = tid; e < nblk * (uint32_t)M; e += kBlock)
        __builtin_nontemporal_store(l_pi[e], &c.out_point_idx[r0 * M + e]);
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_unique(const Config& c, const uint32_t* keys, hipStream_t st) {
  hipLaunchKernelGGL(ucount_kernel, dim3(c.schunk_max), dim3(kBlock), 0, st, c, keys);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(uwrite_kernel, dim3(c.schunk_max), dim3(kBlock), 0, st, c, keys);
  return hipGetLastError();
}

hipError_t launch_finalize(const Config& c, hipStream_t st) {
  hipLaunchKernelGGL(finalize_kernel, dim3(1), dim3(kBlock), 0, st, c);
  return hipGetLastError();
}

hipError_t launch_cap(const Config& c, const uint32_t* vals, hipStream_t st) {
  hipLaunchKernelGGL(cap_kernel, dim3(c.B), dim3(kBlock), 0, st, c, vals);
  return hipGetLastError();
}

hipError_t launch_mean(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st) {
  const size_t lds = (size_t)kMeanTile * (4 + c.C + c.M) * 4;
  hipLaunchKernelGGL(mean_kernel, dim3(c.mean_grid), dim3(kBlock), lds, st, c, keys, vals);
  return hipGetLastError();
}

}  // namespace mmbev

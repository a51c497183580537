// Stable least-significant-digit radix sort of (key, value) pairs as chunked
// reduce-then-scan passes, with no inter-workgroup waiting.
//
// A pass over the pairs is three launches:
//   count   -- workgroup w counts the digits of its chunk of the input
//              (wave multi-split, one LDS add per distinct digit and wave);
//   rowscan -- workgroup d turns row d of the [digit][chunk] count matrix
//              into exclusive offsets and writes the row total;
//   scatter -- workgroup w walks its chunk in order, tile by tile: ranks each
//              pair inside the tile (wave multi-split), reorders the tile by
//              digit in LDS, and writes every digit's run to
//              base(digit) + offset(digit, w) + pairs of that digit already
//              written from earlier tiles of the chunk.
// Chunks are contiguous and visited in order, so the pass is stable.  The
// first pass reads the point filter's output in place: chunk w of that pass
// is filter wave chunk w's region (kept pairs in point order, a gap after
// them), and its digit counts come from the filter.
//
// Keys are voxel keys; the frame index is part of the key, either in its top
// bits or, when key and frame do not fit 32 bits together, looked up from
// the point index (frames are contiguous point ranges) in LDS.
#include "launch.hpp"

namespace mmbev {

namespace {

__device__ __forceinline__ uint32_t frame_lds(const uint32_t* off, int32_t B, uint32_t val) {
  int32_t lo = 0, hi = B - 1;
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) >> 1;
    if (off[mid] <= val)
      lo = mid;
    else
      hi = mid - 1;
  }
  return (uint32_t)lo;
}

struct DigitOf {
  int shift;
  uint32_t mask;
  bool frame;  // the pass's digit reaches into the frame bits
  bool lds;    // frame offsets staged in LDS
  const uint32_t* off;
  __device__ __forceinline__ uint32_t operator()(const Config& c, uint32_t key, uint32_t val) const {
    uint64_t comp = key;
    if (frame)
      comp |= (uint64_t)(lds ? frame_lds(off, c.B, val) : (uint32_t)frame_of_point(c.frame_off, c.B, (int64_t)val))
              << c.kb;
    return (uint32_t)(comp >> shift) & mask;
  }
};

// Digit extractor of a pass; stages the frame offsets in LDS when needed
// (the caller synchronises before use).
__device__ __forceinline__ DigitOf make_digit(const Config& c, int pass, uint32_t* dyn_off) {
  DigitOf d;
  d.shift = pass * c.dbits;
  d.mask = (1u << c.dbits) - 1u;
  d.frame = !c.key_has_frame && c.B > 1 && d.shift + c.dbits > c.kb;
  d.lds = d.frame && c.B <= kMaxSortLdsFrames;
  d.off = dyn_off;
  if (d.lds)
    for (int e = threadIdx.x; e <= c.B; e += kBlock)
      dyn_off[e] = (uint32_t)min(max(c.frame_off[e], (int64_t)0), (int64_t)c.N);
  return d;
}

// Lanes of this wave holding the same digit (valid lanes only).
__device__ __forceinline__ uint64_t match_digit(uint32_t dig, bool valid, int dbits) {
  uint64_t m = __ballot(valid);
  for (int bit = 0; bit < dbits; ++bit) {
    const uint32_t on = (dig >> bit) & 1u;
    const uint64_t bb = __ballot(on);
    m &= on ? bb : ~bb;
  }
  return m;
}

__global__ __launch_bounds__(kBlock) void count_kernel(Config c, int pass, const uint32_t* kin, const uint32_t* vin) {
  __shared__ uint32_t s_hist[kSortBins];
  extern __shared__ uint32_t dyn_off[];
  const int tid = threadIdx.x;
  const uint32_t K = c.hdr->kept;
  const DigitOf digit = make_digit(c, pass, dyn_off);
  s_hist[tid] = 0;
  __syncthreads();
  uint32_t lo, hi;
  chunk_range(K, blockIdx.x, gridDim.x, lo, hi);
  const uint64_t lt = lanemask_lt();
  for (uint32_t base = lo; base < hi; base += kBlock) {
    const uint32_t k = base + tid;
    const bool valid = k < hi;
    const uint32_t d = valid ? digit(c, kin[k], digit.frame ? vin[k] : 0u) : 0u;
    const uint64_t m = match_digit(d, valid, c.dbits);
    if (valid && (m & lt) == 0) atomicAdd(&s_hist[d], (uint32_t)__popcll(m));
  }
  __syncthreads();
  const uint32_t nbins = 1u << c.dbits;
  if ((uint32_t)tid < nbins) c.cnt[(int64_t)tid * gridDim.x + blockIdx.x] = s_hist[tid];
}

// Row d of the count matrix -> exclusive offsets in place, row total.  With
// fcount (first pass), block 0 also stores the number of kept pairs.
__global__ __launch_bounds__(kBlock) void rowscan_kernel(Config c, int chunks, const uint32_t* fcount) {
  __shared__ uint32_t s_tmp[kWaves];
  const int tid = threadIdx.x;
  uint32_t* row = c.cnt + (int64_t)blockIdx.x * chunks;
  const int per = (chunks + kBlock - 1) / kBlock;
  const int first = tid * per;
  uint32_t sum = 0;
  for (int j = 0; j < per; ++j)
    if (first + j < chunks) sum += row[first + j];
  uint32_t total;
  uint32_t run = block_exclusive_scan(sum, s_tmp, total);
  for (int j = 0; j < per; ++j)
    if (first + j < chunks) {
      const uint32_t x = row[first + j];
      row[first + j] = run;
      run += x;
    }
  if (tid == 0) c.tot[blockIdx.x] = total;
  if (fcount && blockIdx.x == 0) {
    uint32_t ks = 0;
    for (int j = 0; j < per; ++j)
      if (first + j < chunks) ks += fcount[first + j];
    uint32_t kt;
    (void)block_exclusive_scan(ks, s_tmp, kt);
    if (tid == 0) c.hdr->kept = kt;
  }
}

struct ScatterLds {
  uint32_t run[kSortBins];  // next output position of every digit
  uint32_t wave_cnt[kWaves][kSortBins];
  uint32_t local_off[kSortBins];
  uint32_t keys[kSortTile];
  uint32_t vals[kSortTile];
  uint8_t digit[kSortTile];
  uint32_t scan_tmp[kWaves];
};

__global__ __launch_bounds__(kBlock) void scatter_kernel(Config c, int pass, const uint32_t* kin, const uint32_t* vin,
                                                         uint32_t* kout, uint32_t* vout, int first_pass) {
  __shared__ ScatterLds L;
  extern __shared__ uint32_t dyn_off[];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  WsHeader* h = c.hdr;
  const uint32_t K = h->kept;
  const DigitOf digit = make_digit(c, pass, dyn_off);
  const uint32_t nbins = 1u << c.dbits;
  uint32_t lo, hi;
  if (first_pass) {
    lo = blockIdx.x * (uint32_t)c.filter_chunk_points;
    hi = lo + min(c.fcount[blockIdx.x], (uint32_t)c.filter_chunk_points);
  } else {
    chunk_range(K, blockIdx.x, gridDim.x, lo, hi);
  }
  {
    // base(digit) = totals of the smaller digits; plus this chunk's offset
    const uint32_t t = (uint32_t)tid < nbins ? c.tot[tid] : 0u;
    uint32_t total;
    const uint32_t ex = block_exclusive_scan(t, L.scan_tmp, total);
    if ((uint32_t)tid < nbins) L.run[tid] = ex + c.cnt[(int64_t)tid * gridDim.x + blockIdx.x];
  }
  const uint64_t lt = lanemask_lt();
  for (uint32_t base = lo; base < hi; base += kSortTile) {
#pragma unroll
    for (int w = 0; w < kWaves; ++w) L.wave_cnt[w][tid] = 0;
    __syncthreads();
    uint32_t key[kSortItems], val[kSortItems], dig[kSortItems], rank[kSortItems];
    bool valid[kSortItems];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
      const uint32_t k = base + wave * (64 * kSortItems) + r * 64 + lane;
      valid[r] = k < hi;
      key[r] = valid[r] ? kin[k] : 0u;
      val[r] = valid[r] ? vin[k] : 0u;
    }
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) dig[r] = valid[r] ? digit(c, key[r], val[r]) : 0u;
    // wave multi-split over the rounds: tile order is (wave, round, lane)
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
      const uint64_t m = match_digit(dig[r], valid[r], c.dbits);
      uint32_t prior = 0;
      if (valid[r]) prior = L.wave_cnt[wave][dig[r]];
      __builtin_amdgcn_wave_barrier();
      if (valid[r]) {
        rank[r] = prior + __popcll(m & lt);
        if ((m & lt) == 0) L.wave_cnt[wave][dig[r]] = prior + __popcll(m);
      }
      __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    uint32_t tile_cnt = 0;
    if ((uint32_t)tid < nbins) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const uint32_t x = L.wave_cnt[w][tid];
        L.wave_cnt[w][tid] = tile_cnt;
        tile_cnt += x;
      }
    }
    uint32_t tile_total;
    L.local_off[tid] = block_exclusive_scan(tile_cnt, L.scan_tmp, tile_total);
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
      if (valid[r]) {
        const uint32_t lp = L.local_off[dig[r]] + L.wave_cnt[wave][dig[r]] + rank[r];
        L.keys[lp] = key[r];
        L.vals[lp] = val[r];
        L.digit[lp] = (uint8_t)dig[r];
      }
    }
    __syncthreads();
    const uint32_t n_in = min((uint32_t)kSortTile, hi - base);
    for (uint32_t k = tid; k < n_in; k += kBlock) {
      const uint32_t d = L.digit[k];
      const uint32_t gp = L.run[d] + (k - L.local_off[d]);
      if (gp < K) {  // always true when the counts match the pairs
        kout[gp] = L.keys[k];
        vout[gp] = L.vals[k];
      } else {
        raise_fault(h, MMBEV_FAULT_POINT_OFFSETS);
      }
    }
    __syncthreads();
    if ((uint32_t)tid < nbins) L.run[tid] += tile_cnt;
  }
}

size_t frame_lds_bytes(const Config& c, int pass) {
  const bool frame = !c.key_has_frame && c.B > 1 && pass * c.dbits + c.dbits > c.kb;
  return (frame && c.B <= kMaxSortLdsFrames) ? (size_t)(c.B + 1) * 4 : 0;
}

}  // namespace

hipError_t launch_radix_pass(const Config& c, int pass, const uint32_t* kin, const uint32_t* vin, uint32_t* kout,
                             uint32_t* vout, hipStream_t st) {
  const size_t dyn = frame_lds_bytes(c, pass);
  const int nbins = 1 << c.dbits;
  const bool first = pass == 0;
  const int chunks = first ? c.filter_chunks : c.sort_chunks;
  if (!first) {
    hipLaunchKernelGGL(count_kernel, dim3(chunks), dim3(kBlock), dyn, st, c, pass, kin, vin);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(rowscan_kernel, dim3(nbins), dim3(kBlock), 0, st, c, chunks,
                     first ? (const uint32_t*)c.fcount : (const uint32_t*)nullptr);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(scatter_kernel, dim3(chunks), dim3(kBlock), dyn, st, c, pass, kin, vin, kout, vout,
                     first ? 1 : 0);
  return hipGetLastError();
}

}  // namespace mmbev

// One pass of a stable least-significant-digit radix sort of (key, value)
// pairs, onesweep style: a single kernel per digit.
//
// The digit histograms of all passes were counted by the kernel that wrote
// the pairs, so each workgroup starts from the global bin offsets.  A
// persistent grid takes tiles by atomic ticket; each tile
//   1. loads kSortTile pairs, wave-striped so every round of loads is
//      coalesced and the tile order equals (wave, round, lane);
//   2. ranks every pair inside its wave with ballots over the digit bits
//      (wave multi-split), keeping per-wave digit counters in LDS;
//   3. publishes its per-digit counts and obtains the counts of all earlier
//      tiles by decoupled look-back (one lane per digit);
//   4. reorders the tile by digit in LDS and writes each digit's run to its
//      global slot, so consecutive lanes store consecutive addresses.
//
// which = 0 sorts voxel keys; the frame index is part of the key, either in
// its top bits or, when key and frame do not fit 32 bits together, looked up
// from the point index (frames are contiguous point ranges).  which = 1 sorts
// the voxels of over-cap frames by their first point index; in "mark" mode
// the last pass does not store the sorted pairs but the keep flag of each
// voxel: its rank inside its frame is its sorted position minus the frame's
// first position.
#include "launch.hpp"

namespace mmbev {

namespace {

struct SortLds {
  uint32_t bin_start[kSortBins];
  uint32_t wave_cnt[kWaves][kSortBins];
  uint32_t local_off[kSortBins];
  uint32_t global_base[kSortBins];
  uint32_t keys[kSortTile];
  uint32_t vals[kSortTile];
  uint8_t digit[kSortTile];
  uint32_t scan_tmp[kWaves];
  uint32_t ticket;
};

__device__ __forceinline__ uint32_t frame_bits_of(const Config& c, uint32_t val) {
  return (uint32_t)frame_of_point(c.frame_off, c.B, (int64_t)val);
}

template <bool MARK>
__global__ __launch_bounds__(kBlock) void radix_pass_kernel(Config c, int which, int pass, const uint32_t* kin,
                                                            const uint32_t* vin, uint32_t* kout, uint32_t* vout) {
  __shared__ SortLds L;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  WsHeader* h = c.hdr;
  const uint32_t count = which == 0 ? h->kept : h->capped_voxels;
  const uint32_t ntiles = (count + kSortTile - 1) / kSortTile;
  if (ntiles == 0) return;
  const int dbits = which == 0 ? c.dbits : c.cap_dbits;
  const uint32_t nbins = 1u << dbits;
  const uint32_t dmask = nbins - 1u;
  const int shift = pass * dbits;
  // frames must be looked up from the point index when the key lacks them
  const bool frame_lookup = which == 0 && !c.key_has_frame && c.B > 1 && shift + dbits > c.kb;
  const uint32_t slot = (which == 0 ? kSlotSort0 : kSlotCapSort0) + pass;
  const uint32_t tag = tag_of(h->epoch, slot);

  {
    uint32_t v = tid < (int)nbins ? h->hist[which][pass][tid] : 0u;
    uint32_t total;
    uint32_t ex = block_exclusive_scan(v, L.scan_tmp, total);
    L.bin_start[tid] = ex;
  }

  const uint64_t lt = lanemask_lt();
  for (;;) {
    if (tid == 0) L.ticket = atomicAdd(&h->tickets[slot], 1u);
#pragma unroll
    for (int w = 0; w < kWaves; ++w) L.wave_cnt[w][tid] = 0;
    __syncthreads();
    const uint32_t t = L.ticket;
    if (t >= ntiles) break;

    uint32_t key[kSortItems], val[kSortItems], dig[kSortItems], rank[kSortItems];
    bool valid[kSortItems];
    const int64_t tile_base = (int64_t)t * kSortTile;
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
      int64_t k = tile_base + wave * (64 * kSortItems) + r * 64 + lane;
      valid[r] = k < (int64_t)count;
      key[r] = valid[r] ? kin[k] : 0u;
      val[r] = valid[r] ? vin[k] : 0u;
      uint64_t comp = key[r];
      if (frame_lookup) comp |= (uint64_t)frame_bits_of(c, val[r]) << c.kb;
      dig[r] = (uint32_t)(comp >> shift) & dmask;
    }
    // wave multi-split: lanes of this round with the same digit
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
      uint64_t m = __ballot(valid[r]);
      for (int bit = 0; bit < dbits; ++bit) {
        uint32_t on = (dig[r] >> bit) & 1u;
        uint64_t bb = __ballot(on);
        m &= on ? bb : ~bb;
      }
      uint32_t prior = 0;
      if (valid[r]) prior = L.wave_cnt[wave][dig[r]];
      __builtin_amdgcn_wave_barrier();
      if (valid[r]) {
        rank[r] = prior + __popcll(m & lt);
        if (lane == __builtin_ctzll(m)) L.wave_cnt[wave][dig[r]] = prior + __popcll(m);
      }
      __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();

    // per-digit tile counts, wave offsets, local digit offsets
    uint32_t tile_cnt = 0;
    if (tid < (int)nbins) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        uint32_t x = L.wave_cnt[w][tid];
        L.wave_cnt[w][tid] = tile_cnt;
        tile_cnt += x;
      }
    }
    uint32_t tile_total;
    uint32_t loc = block_exclusive_scan(tile_cnt, L.scan_tmp, tile_total);
    L.local_off[tid] = loc;
    if (tid < (int)nbins) {
      uint64_t* st = c.sort_status + (int64_t)t * kSortBins + tid;
      uint32_t prefix = 0;
      if (t == 0) {
        status_store(st, status_word(tag, kFlagIncl, tile_cnt));
      } else {
        status_store(st, status_word(tag, kFlagAgg, tile_cnt));
        prefix = look_back(c.sort_status + tid, t, kSortBins, tag, h);
        status_store(st, status_word(tag, kFlagIncl, prefix + tile_cnt));
      }
      L.global_base[tid] = L.bin_start[tid] + prefix;
    }
    __syncthreads();

    // reorder the tile by digit in LDS
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
      if (valid[r]) {
        uint32_t lp = L.local_off[dig[r]] + L.wave_cnt[wave][dig[r]] + rank[r];
        L.keys[lp] = key[r];
        L.vals[lp] = val[r];
        L.digit[lp] = (uint8_t)dig[r];
      }
    }
    __syncthreads();

    const uint32_t n_in = min((uint32_t)kSortTile, count - t * (uint32_t)kSortTile);
    for (uint32_t k = tid; k < n_in; k += kBlock) {
      uint32_t d = L.digit[k];
      uint32_t gp = L.global_base[d] + (k - L.local_off[d]);
      if (!MARK) {
        if (gp < count) {  // always true when the histograms match the pairs
          kout[gp] = L.keys[k];
          vout[gp] = L.vals[k];
        } else {
          raise_fault(h, MMBEV_FAULT_POINT_OFFSETS);
        }
      } else {
        // gp: rank of this voxel by first point index among all capped voxels
        uint32_t v = L.vals[k];
        int32_t lo = 0, hi = c.B - 1;
        while (lo < hi) {
          int32_t mid = (lo + hi + 1) >> 1;
          if (c.vox_off[mid] <= v)
            lo = mid;
          else
            hi = mid - 1;
        }
        uint32_t first = c.cap_off[lo];
        uint32_t q = first + (v - c.vox_off[lo]);
        if (q < count) c.keepflag[q] = (gp - first) < (uint32_t)c.cap ? 1 : 0;
      }
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_radix_pass(const Config& c, int which, int pass, const uint32_t* kin, const uint32_t* vin,
                             uint32_t* kout, uint32_t* vout, bool mark, hipStream_t st) {
  if (mark)
    hipLaunchKernelGGL(radix_pass_kernel<true>, dim3(c.sort_grid), dim3(kBlock), 0, st, c, which, pass, kin, vin,
                       kout, vout);
  else
    hipLaunchKernelGGL(radix_pass_kernel<false>, dim3(c.sort_grid), dim3(kBlock), 0, st, c, which, pass, kin,
                       vin, kout, vout);
  return hipGetLastError();
}

}  // namespace mmbev

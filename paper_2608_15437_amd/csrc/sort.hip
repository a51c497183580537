// Stable least-significant-digit radix sort of (voxel key, point index)
// pairs, segmented by frame, as chunked reduce-then-scan passes with no
// inter-workgroup waiting.
//
// Frames are never mixed: the pairs are grouped by frame in frame order (the
// filter emits them in point order), every chunk of a pass holds pairs of
// one frame, and a pass moves each pair only inside its frame's range, to
//   fstart(b) + (pairs of frame b with a smaller digit)
//             + (pairs of frame b with this digit in earlier chunks)
//             + (pairs with this digit earlier in this chunk).
// So the keys need no frame bits: ceil(kb / 9) passes of at most 9 bits sort
// every frame.
//
// segments -- one workgroup: the kept-pair prefix of the filter chunks, the
//             first pair of every frame (the prefix at its first filter
//             chunk), and the pair chunks (at most kMaxFrameChunks per frame,
//             whole scatter tiles, or half tiles for frames of at most
//             kHalfTileFramePairs pairs when the call allows; the last of a
//             frame shorter) and the voxel tiles of the later kernels
//             (kVoxTile pairs, the last of a frame shorter).  For calls of
//             at most kSmallChunks filter chunks this work is done by one
//             more workgroup of the compaction launch instead.
// compact  -- one workgroup per filter chunk: its kept pairs (at the start of the
//             chunk's point range) copied to their compact place, and the
//             kept points' records (index, x', y', z', features) written
//             there, so the mean reads compact records instead of points.
// Then per pass:
// count    -- workgroup k counts the digits of pair chunk k (row k of the
//             [chunk][digit] count matrix; per-wave LDS histograms, four
//             copies each for chunks of more than one tile);
// scatter  -- the workgroup of chunk k (chunks dealt to the XCDs in
//             contiguous blocks) sums the count rows of its frame's chunks (the
//             frame's digit totals, and its digits in the earlier chunks:
//             where each of its digits starts), then walks its chunk tile by
//             tile (the next tile's
//             pairs loading while the current one is handled): ranks each
//             pair inside the tile (wave multi-split; half the rounds for a
//             chunk of at most half a tile), reorders the tile by digit in
//             LDS, and writes every digit's run to its place.
#include "launch.hpp"

namespace mmbev {

namespace {

// Lanes of this wave holding the same digit (valid lanes only).  A lane
// differs from this one where some bit's ballot differs from this lane's
// bit: per bit one ballot and (ballot XOR this lane's bit, sign-extended)
// ORed into the difference mask.  Unrolled over the widest digit so that the
// ballots do not wait for each other (narrower digits have zero high bits).
__device__ __forceinline__ uint64_t match_digit(uint32_t dig, bool valid) {
  uint32_t dlo = 0, dhi = 0;
#pragma unroll
  for (int bit = 0; bit < kMaxDigitBits; ++bit) {
    const int32_t sb = __builtin_amdgcn_sbfe((int32_t)dig, bit, 1);  // -1 where the bit is set, else 0
    const uint32_t s = (uint32_t)sb;
    const uint64_t b = __builtin_amdgcn_ballot_w64(sb < 0);
    dlo |= (uint32_t)b ^ s;
    dhi |= (uint32_t)(b >> 32) ^ s;
  }
  return __ballot(valid) & ~(((uint64_t)dhi << 32) | dlo);
}

constexpr int kSegBlock = 1024;  // threads of the segments kernel
constexpr int kSegWaves = kSegBlock / 64;
constexpr int kSegLdsFrames = 4096;  // frame starts kept in LDS up to this many frames
constexpr int kSegPreLds = 16384;  // kept-pair prefixes of up to this many filter chunks kept in LDS (kLds instance)

// The segments kernel's work for a workgroup of BLOCK threads.  kLds: the
// frame starts are built in LDS (B <= kSegLdsFrames, the s_ arrays hold
// kSegLdsFrames + 1 words and s_pre kSegPreLds + 1) and copied out at the
// end; otherwise in the workspace directly (the s_ arrays unused).  (One
// address space per instance: a pointer that may be either compiles to
// generic instructions, whose waits cover both kinds of access.)  s_tmp
// holds 2 * BLOCK / 64 words.
template <bool kLds, int BLOCK>
__device__ __forceinline__ void segments_body(const Config& c, uint32_t* s_tmp, uint32_t* s_fstart, uint32_t* s_sfirst,
                                              uint32_t* s_tfirst, uint32_t* s_pre, unsigned long long* s_most) {
  WsHeader* h = c.hdr;
  const int tid = threadIdx.x;
  const uint32_t nf = h->fchunks;
  // the first filter chunk of this thread's frame (the staging kernel laid
  // the chunks out frame by frame), loaded with the chunk count
  const uint32_t ffirst = c.fchunk_first[min(tid, c.B)];
  // used here, so that its wait is not placed after the prefix stores below
  // (one in-order counter covers loads and stores: a wait for an early load
  // issued after many stores would wait for the stores too)
  asm volatile("" ::"v"(ffirst));
  constexpr bool lds = kLds;
  const bool pre_lds = kLds && nf < (uint32_t)kSegPreLds;  // uniform
  uint32_t* fstart = kLds ? s_fstart : c.fstart;
  if (tid == 0) *s_most = 0ull;
  // kept-point prefix of the filter chunks.  Thread t holds kScanItems
  // consecutive chunks, read with 16-byte loads.
  static_assert(kScanItems % 4 == 0, "16-byte loads");
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nf; base += BLOCK * kScanItems) {
    const uint32_t first = base + tid * kScanItems;
    uint32_t v[kScanItems], sum = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; j += 4) {
      uint4 a = make_uint4(0u, 0u, 0u, 0u);
      if (first + j + 3 < nf) {
        a = *reinterpret_cast<const uint4*>(c.fcount + first + j);
      } else if (first + j < nf) {
        a.x = c.fcount[first + j];
        if (first + j + 1 < nf) a.y = c.fcount[first + j + 1];
        if (first + j + 2 < nf) a.z = c.fcount[first + j + 2];
      }
      v[j] = a.x; v[j + 1] = a.y; v[j + 2] = a.z; v[j + 3] = a.w;
    }
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) sum += v[j];
    uint32_t total;
    uint32_t run = carry + block_exclusive_scan<BLOCK / 64>(sum, s_tmp, total);
    uint32_t pre[kScanItems];
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
      pre[j] = run;
      run += v[j];
    }
    // the thread's prefixes as 16-byte stores (one per four chunks)
#pragma unroll
    for (int j = 0; j < kScanItems; j += 4) {
      if (first + j + 3 < nf)
        *reinterpret_cast<uint4*>(c.fprefix + first + j) = make_uint4(pre[j], pre[j + 1], pre[j + 2], pre[j + 3]);
      else
        for (int u = 0; u < 4; ++u)
          if (first + j + u < nf) c.fprefix[first + j + u] = pre[j + u];
    }
    if (pre_lds)
#pragma unroll
      for (int j = 0; j < kScanItems; ++j)
        if (first + j < nf) s_pre[first + j] = pre[j];
    carry += total;
  }
  const uint32_t K = carry;
  if (tid == 0) c.fprefix[nf] = K;
  __syncthreads();  // the prefixes are in place (LDS, or the workspace)
  // frame b starts at the prefix of its first chunk; frames after the last
  // chunk (and frame B) at K
  if (pre_lds) {  // uniform: the prefixes from LDS
    for (int g = tid; g <= c.B; g += BLOCK) {
      const uint32_t k = min(g == tid ? ffirst : c.fchunk_first[g], nf);
      fstart[g] = k >= nf ? K : s_pre[k];
    }
  } else {
    for (int g = tid; g <= c.B; g += BLOCK) {
      const uint32_t k = min(g == tid ? ffirst : c.fchunk_first[g], nf);
      fstart[g] = k >= nf ? K : c.fprefix[k];
    }
  }
  __syncthreads();
  if (lds)
    for (int g = tid; g <= c.B; g += BLOCK) c.fstart[g] = s_fstart[g];
  // pair chunks (at most kMaxFrameChunks per frame, of frame_chunk_pairs
  // pairs: whole kSortTile multiples, the last one of a frame shorter) and
  // voxel tiles (kVoxTile sorted pairs, the last one of a frame shorter):
  // the frames' counts scanned into their first indices, then every chunk
  // and tile written by its own thread (its frame found by a search over
  // the first indices: the last frame whose first index is at most its own)
  const uint32_t mt = chunk_min_tiles(K, c.B);
  const bool half = half_tile_chunks(K, c.B);
  const int per = (c.B + BLOCK - 1) / BLOCK;
  const int b0 = tid * per;
  unsigned long long most = 0ull;
  uint32_t mine = 0, mine_vt = 0;
  for (int j = 0; j < per; ++j) {
    const int b = b0 + j;
    if (b < c.B) {
      const uint32_t n = fstart[b + 1] - fstart[b];
      mine += (n + frame_chunk_pairs(n, mt, half) - 1) / frame_chunk_pairs(n, mt, half);
      most = max(most, (unsigned long long)n << 32 | (uint32_t)~(uint32_t)b);
      mine_vt += (n + kVoxTile - 1) / kVoxTile;
    }
  }
  {  // the wave's largest (pairs, ~frame): pairs first, then the frame among those
    const uint32_t hi = wave_max((uint32_t)(most >> 32));
    const uint32_t lo = wave_max((uint32_t)(most >> 32) == hi ? (uint32_t)most : 0u);
    if ((tid & 63) == 0 && hi > 0u) atomicMax(s_most, (unsigned long long)hi << 32 | lo);  // read after the scans' barriers
  }
  uint2 tot;
  const uint2 ex = block_exclusive_scan2<BLOCK / 64>(mine, mine_vt, s_tmp, tot);
  uint32_t run = ex.x, run_vt = ex.y;
  const uint32_t total = tot.x, total_vt = tot.y;
  const uint32_t cap = (uint32_t)c.schunk_max;  // never reached: the bound holds for any K <= N
  const uint32_t cap_vt = (uint32_t)c.vtile_max;
  const uint32_t nsc = min(total, cap), nvt = min(total_vt, cap_vt);
  uint32_t* sfirst = kLds ? s_sfirst : c.schunk_first;
  uint32_t* tfirst = kLds ? s_tfirst : c.vt_first;
  for (int j = 0; j < per; ++j) {
    const int b = b0 + j;
    if (b < c.B) {
      const uint32_t n = fstart[b + 1] - fstart[b];
      sfirst[b] = min(run, cap);
      tfirst[b] = min(run_vt, cap_vt);
      run += (n + frame_chunk_pairs(n, mt, half) - 1) / frame_chunk_pairs(n, mt, half);
      run_vt += (n + kVoxTile - 1) / kVoxTile;
    }
  }
  if (tid == 0) {
    sfirst[c.B] = nsc;
    tfirst[c.B] = nvt;
  }
  __syncthreads();
  auto frame_of = [&](const uint32_t* first, uint32_t k) -> int32_t {
    int32_t lo = 0, hi = c.B - 1;
    while (lo < hi) {
      const int32_t mid = (lo + hi + 1) >> 1;
      if (first[mid] <= k) lo = mid; else hi = mid - 1;
    }
    return lo;
  };
  for (uint32_t k = tid; k < nsc; k += BLOCK) {
    const int32_t b = frame_of(sfirst, k);
    const uint32_t f0 = fstart[b], f1 = fstart[b + 1];
    const uint32_t CH = frame_chunk_pairs(f1 - f0, mt, half);
    const uint32_t k0 = sfirst[b], k1 = sfirst[b + 1];
    const uint32_t lo = f0 + (k - k0) * CH;
    c.schunk[k] = make_uint4(lo, min(lo + CH, f1), (uint32_t)b, f0);
    c.schunk_frame[k] = make_uint2(k0, k1);
  }
  for (uint32_t t = tid; t < nvt; t += BLOCK) {
    const int32_t b = frame_of(tfirst, t);
    const uint32_t f0 = fstart[b], f1 = fstart[b + 1];
    const uint32_t lo = f0 + (t - tfirst[b]) * kVoxTile;
    c.vtile[t] = make_uint4(lo, min(lo + kVoxTile, f1), (uint32_t)b, f0);
  }
  if (kLds)
    for (int g = tid; g <= c.B; g += BLOCK) {
      c.schunk_first[g] = s_sfirst[g];
      c.vt_first[g] = s_tfirst[g];
    }
  if (tid == 0) {
    h->schunks = nsc;
    h->vtiles = nvt;
    h->kept = K;
    h->most_frame = ~(uint32_t)(*s_most & 0xffffffffull);
    h->most_pairs = (uint32_t)(*s_most >> 32);
  }
}

template <bool kLds>
__global__ __launch_bounds__(kSegBlock) void segments_kernel(Config c) {
  __shared__ uint32_t s_tmp[2 * kSegWaves];
  __shared__ uint32_t s_fstart[kLds ? kSegLdsFrames + 1 : 1];  // frame starts
  __shared__ uint32_t s_sfirst[kLds ? kSegLdsFrames + 1 : 1];  // first pair chunk of every frame
  __shared__ uint32_t s_tfirst[kLds ? kSegLdsFrames + 1 : 1];  // first voxel tile of every frame
  __shared__ uint32_t s_pre[kLds ? kSegPreLds + 1 : 1];        // kept pairs of the filter chunks before k
  __shared__ unsigned long long s_most;  // (pairs, ~frame) of the frame with the most pairs
  segments_body<kLds, kSegBlock>(c, s_tmp, s_fstart, s_sfirst, s_tfirst, s_pre, &s_most);
}

// Sums of three values over the workgroup (s_tmp: 3 * WAVES words).
template <int WAVES>
__device__ __forceinline__ uint3 block_sum3(uint32_t a, uint32_t b, uint32_t d, uint32_t* s_tmp) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t xa = wave_inclusive_sum(a), xb = wave_inclusive_sum(b), xd = wave_inclusive_sum(d);
  if (lane == 63) {
    s_tmp[wave] = xa;
    s_tmp[WAVES + wave] = xb;
    s_tmp[2 * WAVES + wave] = xd;
  }
  __syncthreads();
  uint3 t = make_uint3(0u, 0u, 0u);
#pragma unroll
  for (int w = 0; w < WAVES; ++w) {
    t.x += s_tmp[w];
    t.y += s_tmp[WAVES + w];
    t.z += s_tmp[2 * WAVES + w];
  }
  __syncthreads();
  return t;
}

// One workgroup per filter chunk: its kept points, listed from the chunk's
// bitmap in increasing index order, get the compact places [fprefix[k],
// fprefix[k+1]).  For each: its record there (point index, p' of Eq. 6 from
// the frame's poses staged in LDS, raw features; 16-byte stores) and its
// voxel key, which the first radix pass pairs with the compact place.  The key is
// the definition's: correctly rounded (p' - min) / v per axis, truncated.
// The reads of a chunk's kept points stay close together (kept points come
// in runs).
constexpr int kCompactItems = 4;
constexpr int kCompactSmallChunk = 1024;  // chunks of at most this many points: two-wave workgroups

// kCompactBlock threads (a chunk's bitmap is at most 128 words, one per
// thread): two waves for small chunks (measured: an 8-frame batch of
// 256-point chunks 24 -> 18.7 us), four for large ones (a 128-frame batch of
// 2,816-point chunks 55 -> 64 us with two).
//
// kSmall (calls of at most kSmallChunks filter chunks): no segments launch.
// Each workgroup sums its own compact place and its frame's bounds from the
// filter's chunk counts (all of them, loaded with its table entries), and
// one more workgroup, the last, does the segments kernel's work (in the
// workspace, for the radix passes and later kernels) beside the others: the
// compaction needs none of it.
template <int kCompactBlock, bool kSmall>
__global__ __launch_bounds__(kCompactBlock) void compact_kernel(Config c, uint32_t* kout) {
  constexpr int kCompactWaves = kCompactBlock / 64;
  constexpr int kSmallItems = kSmall ? kSmallChunks / kCompactBlock : 1;  // chunk counts per thread
  static_assert(kChunkWords <= kCompactBlock, "one bitmap word per thread");
  extern __shared__ float s_pose[];  // [S][12]
  __shared__ uint16_t s_list[kMaxChunkPoints];  // kept point offsets in the chunk, ascending
  __shared__ uint32_t s_tmp[3 * kCompactWaves];
  __shared__ unsigned long long s_most;
  const int tid = threadIdx.x;
  if (kSmall && blockIdx.x == gridDim.x - 1) {  // uniform: the segments kernel's work
    segments_body<false, kCompactBlock>(c, s_tmp, nullptr, nullptr, nullptr, nullptr, &s_most);
    return;
  }
  const uint32_t k = blockIdx.x;
  // the chunk's table entries and bitmap (one word per thread) load together
  // with the chunk count: every address is in bounds for any k < fchunk_max
  // (kSmall: every chunk's count too, at clamped indices)
  const uint32_t nch = c.hdr->fchunks;
  const uint32_t lo = c.fchunk_lo[k], cnt = c.fcount[k];
  uint32_t dst = kSmall ? 0u : c.fprefix[k];
  const uint32_t fr = c.fchunk_frame[k];
  uint32_t word = tid < c.fchunk_words ? c.fbits[(int64_t)k * c.fchunk_words + tid] : 0u;
  uint32_t fcv[kSmallItems];
#pragma unroll
  for (int j = 0; j < kSmallItems; ++j)
    fcv[j] = kSmall ? c.fcount[min((uint32_t)(tid + j * kCompactBlock), (uint32_t)c.fchunk_max - 1u)] : 0u;
  asm volatile("" ::"s"(lo), "s"(dst), "s"(cnt), "s"(fr));  // keeps the loads above the check
  if (k >= nch || cnt == 0u) return;  // uniform: past the chunks, or a chunk that kept no point
  const int32_t b = (int32_t)min(fr, (uint32_t)c.B - 1u);
  const int C = c.C, RW = c.rec_words;
  // the frame's poses: loaded now, stored to LDS once the list is built, so
  // that their loads overlap the listing
  constexpr int kPoseRegs = 4;  // the first 4 * kCompactBlock pose floats in registers; the rest after the listing
  const int np = c.S * 12;
  float pv[kPoseRegs];
#pragma unroll
  for (int u = 0; u < kPoseRegs; ++u) {
    const int e = tid + u * kCompactBlock;
    pv[u] = e < np ? c.poses[(int64_t)b * np + e] : 0.0f;
  }
  uint32_t fs = 0, fe = 0, ff0 = 0, ff1 = 0;
  if (kSmall) {  // the frame's first chunk and the next frame's, loaded with the poses
    ff0 = c.fchunk_first[b];
    ff1 = c.fchunk_first[b + 1];
  } else {
    fs = c.fstart[b];
    fe = c.fstart[b + 1];
  }
  // the bitmap's set bits listed at each word's rank
  uint32_t total;
  uint32_t r = block_exclusive_scan<kCompactWaves>((uint32_t)__popc(word), s_tmp, total);
  while (word) {
    s_list[r++] = (uint16_t)(32 * tid + __builtin_ctz(word));
    word &= word - 1u;
  }
  __syncthreads();  // the list is complete
  const uint32_t n = min(total, cnt);  // equal unless the workspace was corrupted
  uint32_t pi[kCompactItems], sw[kCompactItems];
  float v[kCompactItems][8];
  auto load_batch = [&](uint32_t base) {
#pragma unroll
    for (int u = 0; u < kCompactItems; ++u) {
      const uint32_t t = base + u * kCompactBlock + tid;
      pi[u] = t < n ? min(lo + (uint32_t)s_list[t], (uint32_t)c.N - 1u) : 0u;
    }
#pragma unroll
    for (int u = 0; u < kCompactItems; ++u) {  // all point loads of the batch in flight together
      const bool ok = base + u * kCompactBlock + tid < n;
      const uint32_t i = pi[u];
      sw[u] = ok ? min((uint32_t)c.sweep[i], (uint32_t)c.S - 1u) : 0u;
#pragma unroll
      for (int f = 0; f < 8; ++f) v[u][f] = (ok && f < C) ? c.feat[(int64_t)f * c.stride + i] : 0.0f;
    }
  };
  auto finish_batch = [&](uint32_t base) {
#pragma unroll
    for (int u = 0; u < kCompactItems; ++u) {
      const uint32_t t = base + u * kCompactBlock + tid;
      if (t < n) {
        const uint32_t q = dst + t;
        float px, py, pz;
        compensate(s_pose + sw[u] * 12, v[u][0], v[u][1], v[u][2], px, py, pz);
        int32_t ix, iy, iz;
        const bool in = quantize_axis(px, c.mn[0], c.vs[0], c.Df[0], ix) &&
                        quantize_axis(py, c.mn[1], c.vs[1], c.Df[1], iy) &&
                        quantize_axis(pz, c.mn[2], c.vs[2], c.Df[2], iz);
        if (!in) raise_fault(c.hdr, MMBEV_FAULT_INTERNAL);  // the filter kept it: never
        kout[q] = in ? ((uint32_t)iz * c.Dy + (uint32_t)iy) * c.Dx + (uint32_t)ix : 0u;
        // the record: 16-byte stores when RW is a multiple of four, else
        // 8-byte stores (records are 8-byte aligned)
        const uint32_t w[10] = {pi[u], __float_as_uint(px), __float_as_uint(py), __float_as_uint(pz),
                                __float_as_uint(v[u][3]), __float_as_uint(v[u][4]), __float_as_uint(v[u][5]),
                                __float_as_uint(v[u][6]), __float_as_uint(v[u][7]), 0u};
        uint32_t* rp = c.rec + (int64_t)q * RW;
        if ((RW & 3) == 0) {  // uniform
#pragma unroll
          for (int k = 0; k < 2; ++k)
            if (4 * k < RW)
              reinterpret_cast<uint4*>(rp)[k] = make_uint4(w[4 * k], w[4 * k + 1], w[4 * k + 2], w[4 * k + 3]);
        } else {
#pragma unroll
          for (int k = 0; k < 5; ++k)
            if (2 * k < RW) reinterpret_cast<uint2*>(rp)[k] = make_uint2(w[2 * k], w[2 * k + 1]);
        }
      }
    }
  };
  // the first batch's point loads go out before the poses are stored (the
  // poses' loads were issued before the listing), so the two round trips overlap
  load_batch(0u);
  if (kSmall) {  // kept points of the chunks before k, before the frame's first chunk and before the next frame's
    uint32_t a0 = 0, a1 = 0, a2 = 0;
#pragma unroll
    for (int j = 0; j < kSmallItems; ++j) {
      const uint32_t i = (uint32_t)(tid + j * kCompactBlock);
      const uint32_t v = i < nch ? fcv[j] : 0u;
      a0 += i < k ? v : 0u;
      a1 += i < ff0 ? v : 0u;
      a2 += i < ff1 ? v : 0u;
    }
    const uint3 t = block_sum3<kCompactWaves>(a0, a1, a2, s_tmp);
    dst = t.x;
    fs = t.y;
    fe = t.z;
  }
#pragma unroll
  for (int u = 0; u < kPoseRegs; ++u)
    if (tid + u * kCompactBlock < np) s_pose[tid + u * kCompactBlock] = pv[u];
  for (int e = tid + kPoseRegs * kCompactBlock; e < np; e += kCompactBlock) s_pose[e] = c.poses[(int64_t)b * np + e];
  if (fe - fs > (uint32_t)c.cap) {  // uniform: the frame may exceed the cap: its first-place bits over this chunk's places cleared
    uint32_t* bits = c.capbits + fs / 32 + (uint32_t)b;  // the heads kernel sets them
    for (uint32_t w = (dst - fs) / 32 + tid; w < (dst - fs + cnt + 31) / 32; w += kCompactBlock) bits[w] = 0u;
  }
  __syncthreads();  // the poses are in LDS
  finish_batch(0u);
  for (uint32_t base = kCompactBlock * kCompactItems; base < n; base += kCompactBlock * kCompactItems) {
    load_batch(base);
    finish_batch(base);
  }
}

// The digit counts of pair chunk k ([lo, hi)) into row k.  Q histogram
// copies per wave (lane % Q; rows padded by a word, so that one digit's
// copies lie in different LDS banks): for chunks of more than one tile,
// where the atomics of lanes on one digit are the cost, four; else one (the
// copies' clearing and summing cost more than they save).
template <int Q>
__device__ __forceinline__ void count_chunk(const Config& c, uint32_t* s_hist, uint32_t k, uint32_t lo, uint32_t hi,
                                            const uint32_t* kin, int shift, uint32_t mask, uint32_t nbins) {
  constexpr int kRow = kSortBins + 1;
  const int tid = threadIdx.x, wave = tid >> 6;
  uint32_t* hw = s_hist + (wave * Q + tid % Q) * kRow;
  for (uint32_t e = tid; e < (uint32_t)(kWaves * Q * kRow); e += kBlock) s_hist[e] = 0;
  __syncthreads();
  for (uint32_t base = lo; base < hi; base += kBlock * kCountItems) {
    uint32_t key[kCountItems];
#pragma unroll
    for (int j = 0; j < kCountItems; ++j) {  // all loads of the batch in flight together
      const uint32_t i = base + j * kBlock + tid;
      key[j] = i < hi ? kin[i] : 0u;
    }
#pragma unroll
    for (int j = 0; j < kCountItems; ++j)
      if (base + j * kBlock + tid < hi) atomicAdd(&hw[(key[j] >> shift) & mask], 1u);
  }
  __syncthreads();
  for (uint32_t e = tid; e < nbins; e += kBlock) {
    uint32_t t = 0;
#pragma unroll
    for (int w = 0; w < kWaves * Q; ++w) t += s_hist[w * kRow + e];
    c.cnt[(int64_t)k * kSortBins + e] = t;
  }
  __syncthreads();  // the next chunk clears the histograms
}

__global__ __launch_bounds__(kBlock) void count_kernel(Config c, int pass, const uint32_t* kin) {
  __shared__ uint32_t s_hist[kWaves * 4 * (kSortBins + 1)];  // per wave up to four histogram copies
  // the first chunk's entry loads with the chunk count (in bounds: the grid is at most schunk_max)
  const uint32_t nsc = c.hdr->schunks;
  uint4 ch = c.schunk[blockIdx.x];
  asm volatile("" ::"s"(ch.x), "s"(ch.y));  // keeps the load above the check
  const int shift = pass * c.dbits;
  const uint32_t nbins = 1u << c.dbits;
  const uint32_t mask = nbins - 1u;
  for (uint32_t k = blockIdx.x; k < nsc; k += gridDim.x) {  // a grid of resident size walks the chunks
    if (k != blockIdx.x) ch = c.schunk[k];
    if (ch.y - ch.x > (uint32_t)kSortTile)  // uniform
      count_chunk<4>(c, s_hist, k, ch.x, ch.y, kin, shift, mask, nbins);
    else
      count_chunk<1>(c, s_hist, k, ch.x, ch.y, kin, shift, mask, nbins);
  }
}

struct ScatterLds {
  uint32_t pos[kSortBins];             // per digit: output position of the tile's pair i of that digit, less i
  uint2 kv[kSortTile];                 // the tile reordered by digit: (key, value)
  uint32_t wave_cnt[kWaves][kSortBins];  // a wave's digit counts, then its first place in the reordered tile
  uint32_t scan_tmp[2][kWaves];
};

// A tile's pairs in the order (wave, round, lane): wave w holds pairs
// [base + w * 64 * NR, base + (w + 1) * 64 * NR), NR rounds of 64 (NR =
// kSortItems, or half of it for a chunk of at most half a tile).
template <int NR>
__device__ __forceinline__ void load_sort_tile(const uint32_t* kin, const uint32_t* vin, uint32_t base, uint32_t hi,
                                               uint32_t* key, uint32_t* val) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const uint32_t i = base + wave * (64 * NR) + r * 64 + lane;
    const bool in = r < NR && i < hi;
    key[r] = in ? kin[i] : 0u;
    val[r] = in ? (vin != nullptr ? vin[i] : i) : 0u;  // no values: each key's own position
  }
}

// One pair chunk k of the scatter (entries ch, fc), its tiles in the order
// (wave, round, lane) with NR rounds of 64 per wave: kSortItems, or half of
// it for a chunk of at most half a tile (every wave busy, half the rounds).
template <int NR>
__device__ __forceinline__ void scatter_chunk(const Config& c, ScatterLds& L, int pass, uint32_t k, const uint4 ch,
                                              const uint2 fc, uint32_t K, const uint32_t* kin, const uint32_t* vin,
                                              uint32_t* kout, uint32_t* vout) {
  constexpr int kRows = 8;  // count rows in flight together
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  WsHeader* h = c.hdr;
  const int shift = pass * c.dbits;
  const uint32_t nbins = 1u << c.dbits;
  const uint32_t mask = nbins - 1u;
  const uint32_t e0 = 2u * (uint32_t)tid;  // this thread's digits e0 and e0 + 1
  const bool d0 = e0 < nbins, d1 = e0 + 1u < nbins;
  const uint32_t lo = ch.x, hi = ch.y;
  uint32_t key[kSortItems], val[kSortItems], nkey[kSortItems], nval[kSortItems];
  if (lo < hi) load_sort_tile<NR>(kin, vin, lo, hi, key, val);
  // the first kRows count rows of the frame's chunks (at most
  // kMaxFrameChunks rows) go out now and are summed after the first
  // tile is ranked: digit bases = frame start + the frame's smaller
  // digits + this digit in the frame's earlier chunks
  const uint32_t k0 = fc.x, k1 = max(fc.y, k0);
  uint2 x[kRows];
#pragma unroll
  for (int u = 0; u < kRows; ++u)
    x[u] = k0 + u < k1 ? *reinterpret_cast<const uint2*>(c.cnt + (int64_t)(k0 + u) * kSortBins + e0) : make_uint2(0u, 0u);
  uint32_t run0 = 0, run1 = 0;  // output position of the next pair of digit e0, e0 + 1
  for (uint32_t base = lo; base < hi; base += kSortTile) {
    const bool first = base == lo;
    const bool more = base + kSortTile < hi;
    if (more) load_sort_tile<NR>(kin, vin, base + kSortTile, hi, nkey, nval);
    for (uint32_t e = tid; e < kWaves * kSortBins; e += kBlock) (&L.wave_cnt[0][0])[e] = 0u;
    __syncthreads();  // also: the previous tile's reads of pos and kv are done
    uint32_t rank[kSortItems];
    bool valid[kSortItems];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) valid[r] = r < NR && base + wave * (64 * NR) + r * 64 + lane < hi;
    auto dig = [&](int r) -> uint32_t { return (key[r] >> shift) & mask; };  // recomputed: fewer live registers
    // wave multi-split over the rounds (tile order: wave, round, lane): the
    // first lane of each digit's group adds the group's size to the wave's
    // count of that digit with an LDS atomic that returns the count before
    // it.  A wave's LDS operations complete in issue order, so the rounds'
    // atomics go out back to back; each lane then takes its group's count
    // from the group's first lane (bpermute) and adds its place in the group.
    {
      uint32_t old[kSortItems];
#pragma unroll
      for (int r = NR; r < kSortItems; ++r) rank[r] = 0u;  // rounds a half-tile chunk does not use
#pragma unroll
      for (int r = 0; r < NR; ++r) {
        const uint64_t mm = match_digit(dig(r), valid[r]);
        const uint32_t below = count_below(mm);
        rank[r] = (uint32_t)(mm != 0ull ? __builtin_ctzll(mm) : 0) << 8 | below;  // the group's first lane, the lane's place
        old[r] = 0u;
        if (valid[r] && below == 0) old[r] = atomicAdd(&L.wave_cnt[wave][dig(r)], (uint32_t)__popcll(mm));
      }
#pragma unroll
      for (int r = 0; r < NR; ++r) {
        const uint32_t prior = (uint32_t)__builtin_amdgcn_ds_bpermute((int)(rank[r] >> 8) << 2, (int)old[r]);
        rank[r] = prior + (rank[r] & 0xffu);
      }
    }
    uint32_t ft0 = 0, ft1 = 0, pre0 = 0, pre1 = 0;  // the frame's totals of e0, e1 and their count in earlier chunks
    if (first) {  // uniform
      for (uint32_t kk = k0;; kk += kRows) {
#pragma unroll
        for (int u = 0; u < kRows; ++u) {
          const uint32_t a = d0 ? x[u].x : 0u, b = d1 ? x[u].y : 0u;
          if (kk + u < k) {
            pre0 += a;
            pre1 += b;
          }
          ft0 += a;
          ft1 += b;
        }
        if (kk + kRows >= k1) break;
#pragma unroll
        for (int u = 0; u < kRows; ++u) {  // the next rows' loads in flight together
          const uint32_t kr = kk + kRows + u;
          x[u] = kr < k1 ? *reinterpret_cast<const uint2*>(c.cnt + (int64_t)kr * kSortBins + e0) : make_uint2(0u, 0u);
        }
      }
    }
    __syncthreads();  // the wave counts are complete
    // per digit: the tile's count, each wave's first place inside the
    // tile's run of that digit; one scan over the digits for the tile
    // and, on a chunk's first tile, one for the frame's totals
    const uint2* wc = reinterpret_cast<const uint2*>(&L.wave_cnt[0][0]);
    uint2 cw[kWaves];
#pragma unroll
    for (int w = 0; w < kWaves; ++w) cw[w] = wc[w * (kSortBins / 2) + tid];
    uint32_t t0 = 0, t1 = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      t0 += cw[w].x;
      t1 += cw[w].y;
    }
    const uint32_t xt = wave_inclusive_sum(t0 + t1);
    const uint32_t xf = first ? wave_inclusive_sum(ft0 + ft1) : 0u;
    if (lane == 63) {
      L.scan_tmp[0][wave] = xt;
      L.scan_tmp[1][wave] = xf;
    }
    __syncthreads();
    uint32_t wt = 0, wf = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w)
      if (w < wave) {
        wt += L.scan_tmp[0][w];
        wf += L.scan_tmp[1][w];
      }
    const uint32_t lo0 = wt + xt - (t0 + t1), lo1 = lo0 + t0;  // the digits' first places in the reordered tile
    if (first) {
      const uint32_t fb0 = ch.w + wf + xf - (ft0 + ft1);  // frame start + the frame's smaller digits
      run0 = fb0 + pre0;
      run1 = fb0 + ft0 + pre1;
    }
    uint2* wo = reinterpret_cast<uint2*>(&L.wave_cnt[0][0]);
    uint32_t a0 = lo0, a1 = lo1;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      wo[w * (kSortBins / 2) + tid] = make_uint2(a0, a1);
      a0 += cw[w].x;
      a1 += cw[w].y;
    }
    *reinterpret_cast<uint2*>(&L.pos[e0]) = make_uint2(run0 - lo0, run1 - lo1);  // position of tile place i: pos + i
    run0 += t0;
    run1 += t1;
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSortItems; ++r)
      if (valid[r]) L.kv[L.wave_cnt[wave][dig(r)] + rank[r]] = make_uint2(key[r], val[r]);
    __syncthreads();
    const uint32_t n_in = min((uint32_t)kSortTile, hi - base);
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {  // unrolled: the LDS reads of all rounds in flight together
      const uint32_t i = (uint32_t)(r * kBlock + tid);
      if (i < n_in) {
        const uint2 kv = L.kv[i];
        const uint32_t gp = L.pos[(kv.x >> shift) & mask] + i;
        if (gp < K) {  // always true when the counts match the pairs
          kout[gp] = kv.x;
          vout[gp] = kv.y;
        } else {
          raise_fault(h, MMBEV_FAULT_INTERNAL);
        }
      }
    }
    if (more)
#pragma unroll
      for (int r = 0; r < kSortItems; ++r) {
        key[r] = nkey[r];
        val[r] = nval[r];
      }
  }
}

// Thread t owns digits 2t and 2t + 1 (kSortBins == 2 * kBlock) in every
// per-digit step: the count rows (8-byte loads), the tile's digit totals,
// the scans and the output positions, which it keeps in registers from
// tile to tile.
__global__ __launch_bounds__(kBlock, kScatterPerCu) void scatter_kernel(Config c, int pass, const uint32_t* kin, const uint32_t* vin,
                                                         uint32_t* kout, uint32_t* vout) {
  __shared__ ScatterLds L;
  static_assert(sizeof(ScatterLds) <= 160 * 1024 / kScatterPerCu, "workgroups per CU");
  static_assert(kSortBins == 2 * kBlock, "two digits per thread");
  WsHeader* h = c.hdr;
  const uint32_t nsc = h->schunks, K = h->kept;
  // chunks dealt to the XCDs in contiguous blocks: a frame's chunks share
  // one L2, where their neighbouring digit runs merge into whole lines and
  // their count rows are read once; a grid of resident size walks them
  for (uint32_t wb = blockIdx.x;; wb += gridDim.x) {
    const uint32_t k = xcd_block_unit(wb, nsc);
    if (k >= nsc) break;  // uniform
    const uint4 ch = c.schunk[k];
    const uint2 fc = c.schunk_frame[k];
    // a chunk of at most half a tile: half the rounds per wave
    if (ch.y - ch.x <= (uint32_t)kSortTile / 2u)  // uniform
      scatter_chunk<kSortItems / 2>(c, L, pass, k, ch, fc, K, kin, vin, kout, vout);
    else
      scatter_chunk<kSortItems>(c, L, pass, k, ch, fc, K, kin, vin, kout, vout);
  }
}

}  // namespace

hipError_t launch_segments(const Config& c, hipStream_t st) {
  if (c.B <= kSegLdsFrames)
    hipLaunchKernelGGL(segments_kernel<true>, dim3(1), dim3(kSegBlock), 0, st, c);
  else
    hipLaunchKernelGGL(segments_kernel<false>, dim3(1), dim3(kSegBlock), 0, st, c);
  return hipGetLastError();
}

hipError_t launch_compact(const Config& c, uint32_t* kout, hipStream_t st) {
  const size_t lds = (size_t)c.S * 12 * sizeof(float);
  const dim3 grid(c.fchunk_max + (c.small_call ? 1 : 0));  // small calls: one more workgroup for the segments' work
  if (c.fchunk_points <= kCompactSmallChunk) {
    if (c.small_call)
      hipLaunchKernelGGL((compact_kernel<128, true>), grid, dim3(128), lds, st, c, kout);
    else
      hipLaunchKernelGGL((compact_kernel<128, false>), grid, dim3(128), lds, st, c, kout);
  } else if (c.small_call) {
    hipLaunchKernelGGL((compact_kernel<kBlock, true>), grid, dim3(kBlock), lds, st, c, kout);
  } else {
    hipLaunchKernelGGL((compact_kernel<kBlock, false>), grid, dim3(kBlock), lds, st, c, kout);
  }
  return hipGetLastError();
}

hipError_t launch_radix_pass(const Config& c, int pass, const uint32_t* kin, const uint32_t* vin, uint32_t* kout,
                             uint32_t* vout, hipStream_t st) {
  // grids of resident size (idle workgroups still cost dispatch time)
  const uint32_t cgrid = min((uint32_t)c.schunk_max, (uint32_t)kCountGrid);
  hipLaunchKernelGGL(count_kernel, dim3(cgrid), dim3(kBlock), 0, st, c, pass, kin);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const uint32_t sgrid = min((c.schunk_max + 7u) / 8u * 8u, (uint32_t)(kScatterPerCu * kCus));  // whole rounds of the XCDs
  hipLaunchKernelGGL(scatter_kernel, dim3(sgrid), dim3(kBlock), 0, st, c, pass, kin, vin, kout, vout);
  return hipGetLastError();
}

}  // namespace mmbev

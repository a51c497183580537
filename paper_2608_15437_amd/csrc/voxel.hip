// After the sort: voxels, per-frame cap, mean pooling.
//
// The sorted pairs are grouped by frame and ordered by (key, place) inside
// each frame.  The pairs of every frame are cut into voxel tiles of
// kVoxTile pairs (segments); voxel j of tile t is the tile's j-th head (the
// first pair of a run of equal keys), and its per-voxel data sits at the
// tile-local slot vtile[t].lo + j (a tile has no more heads than pairs), so
// no kernel needs the voxel numbering of other tiles to place its voxels.
// heads  -- one workgroup per tile (grid-stride): the heads numbered in pair order, each
//           one's position (hpos) and place (hplace: its first point, since
//           places follow point order) at its slot; the tile's head count;
// fincap -- workgroup 0: the voxels before every tile (all frames), every
//           frame's voxels and its output offsets (at most max_voxels rows
//           per frame); workgroup 1 + b: frame b, if it has more than
//           max_voxels voxels, keeps the max_voxels voxels whose first
//           point comes first and flags them in key order, with the flag
//           words' prefix (from which the mean numbers them);
// mean   -- blocks of kMeanTile consecutive voxels (grid-stride), one
//           thread per voxel: its tile, its output row, and the mean of its first max_points points from
//           their compact records (x', y', z' of Eq. 6 and the raw
//           features), summed in double in ascending point order (Alg. 1
//           VoxelFeatureEncoder read as mean pooling).
#include "launch.hpp"

namespace mmbev {

namespace {

// One voxel tile (kVoxTile sorted pairs, kHeadItems per thread) per step of
// a grid-stride loop: every pair's key, its predecessor's key and its value
// load together; a pair starts a voxel when it is the frame's first or its
// key differs from its predecessor's.  The heads are numbered in pair order
// (row j of kBlock pairs, then wave, then lane: a ballot per row, the rows'
// and waves' counts scanned by one wave).
constexpr int kHeadItems = kVoxTile / kBlock;
static_assert(kHeadItems * kWaves <= 64, "one wave scans the counts");

__global__ __launch_bounds__(kBlock) void heads_kernel(Config c, const uint32_t* keys, const uint32_t* vals) {
  __shared__ uint32_t s_off[kHeadItems * kWaves];  // heads before (row j, wave w), at j * kWaves + w
  __shared__ uint32_t s_total;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const uint32_t nvt = c.hdr->vtiles;
  for (uint32_t t = blockIdx.x; t < nvt; t += gridDim.x) {
    const uint4 vt = c.vtile[t];
    const uint32_t lo = vt.x, hi = vt.y, ff = vt.w;
    const uint32_t fb = min(vt.z, (uint32_t)c.B - 1u);
    const uint32_t fe = c.fstart[fb + 1];  // the frame's end: a frame with more pairs than max_voxels may be capped
    uint32_t key[kHeadItems], prv[kHeadItems], val[kHeadItems];
#pragma unroll
    for (int j = 0; j < kHeadItems; ++j) {  // all loads in flight together: unconditional, at clamped indices
      const uint32_t i = min(lo + j * kBlock + tid, hi - 1u);  // hi > lo: a tile is never empty
      const uint32_t ip = i > ff ? i - 1u : i;
      key[j] = keys[i];
      prv[j] = keys[ip];
      val[j] = vals[i];
    }
    uint64_t m[kHeadItems];
#pragma unroll
    for (int j = 0; j < kHeadItems; ++j) {  // the frame's first pair is always a head
      const uint32_t i = lo + j * kBlock + tid;
      m[j] = __ballot(i < hi && (i == ff || key[j] != prv[j]));
    }
    if (lane == 0)
#pragma unroll
      for (int j = 0; j < kHeadItems; ++j) s_off[j * kWaves + wave] = (uint32_t)__popcll(m[j]);
    __syncthreads();
    if (wave == 0) {  // exclusive scan of the kHeadItems * kWaves counts
      const uint32_t x = lane < kHeadItems * kWaves ? s_off[lane] : 0u;
      const uint32_t y = wave_inclusive_sum(x);
      if (lane < kHeadItems * kWaves) s_off[lane] = y - x;
      if (lane == 63) s_total = y;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kHeadItems; ++j)
      if ((m[j] >> lane) & 1u) {
        const uint32_t slot = lo + s_off[j * kWaves + wave] + count_below(m[j]);
        c.hpos[slot] = lo + j * kBlock + tid;
        c.hplace[slot] = val[j];
      }
    if (fe - ff > (uint32_t)c.cap) {  // uniform: the heads' places marked for the cap (bits cleared by the compaction)
      uint32_t* bits = c.capbits + ff / 32 + fb;
#pragma unroll
      for (int j = 0; j < kHeadItems; ++j)
        if ((m[j] >> lane) & 1u) {
          const uint32_t q = val[j] - ff;
          atomicOr(&bits[q >> 5], 1u << (q & 31));
        }
    }
    if (tid == 0) c.hcount[t] = s_total;
    __syncthreads();  // the next tile rewrites the counts
  }
}

constexpr int kFinBlock = 1024;
constexpr int kFinWaves = kFinBlock / 64;
constexpr int kCapLdsWords = 16384;  // bitmaps of a capped frame in LDS up to this many words
constexpr int kCapLdsTiles = 8192;   // voxel counts of a capped frame's tiles in LDS up to this many tiles

// Exclusive prefix of n values in[0..n) written to out by one workgroup of
// kFinBlock threads; returns the total.
__device__ uint32_t scan_fin(const uint32_t* in, uint32_t* out, uint32_t n, uint32_t* s_tmp) {
  const int tid = threadIdx.x;
  constexpr int kItems = 8;
  uint32_t carry = 0;
  for (uint32_t base = 0; base < n; base += kFinBlock * kItems) {
    const uint32_t first = base + tid * kItems;
    uint32_t v[kItems], sum = 0;
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
      v[j] = first + j < n ? in[first + j] : 0u;
      sum += v[j];
    }
    uint32_t total;
    uint32_t run = carry + block_exclusive_scan<kFinWaves>(sum, s_tmp, total);
#pragma unroll
    for (int j = 0; j < kItems; ++j)
      if (first + j < n) {
        out[first + j] = run;
        run += v[j];
      }
    carry += total;
  }
  return carry;
}

// Workgroup 0 of fincap.
__device__ void finalize_offsets(const Config& c, uint32_t* s_tmp) {
  const int tid = threadIdx.x;
  WsHeader* h = c.hdr;
  const uint32_t nvt = h->vtiles;
  const uint32_t V = scan_fin(c.hcount, c.hpre, nvt, s_tmp);
  if (tid == 0) c.hpre[nvt] = V;
  __syncthreads();
  // every frame's voxels and its output rows (at most max_voxels)
  uint32_t carry_out = 0, carry_cap = 0;
  for (int32_t chunk = 0; chunk < c.B; chunk += kFinBlock) {
    const int32_t b = chunk + tid;
    uint32_t vb = 0;
    if (b < c.B) {
      const uint32_t t0 = min(c.vt_first[b], nvt), t1 = max(min(c.vt_first[b + 1], nvt), t0);
      const uint32_t v0 = c.hpre[t0];
      vb = c.hpre[t1] - v0;
      c.vox_off[b] = v0;
    }
    const uint32_t capped = vb > (uint32_t)c.cap;
    const uint32_t outc = capped ? (uint32_t)c.cap : vb;
    uint32_t t1, t2;
    const uint32_t e1 = block_exclusive_scan<kFinWaves>(outc, s_tmp, t1);
    (void)block_exclusive_scan<kFinWaves>(capped ? vb : 0u, s_tmp, t2);
    if (b < c.B) c.out_voxel_offsets[b] = (int64_t)(carry_out + e1);
    carry_out += t1;
    carry_cap += t2;
  }
  if (tid == 0) {
    c.vox_off[c.B] = V;
    c.out_voxel_offsets[c.B] = (int64_t)carry_out;
    h->voxels = V;
    h->capped_voxels = carry_cap;
    h->any_capped = carry_cap > 0 ? 1u : 0u;
  }
  __syncthreads();  // the frames' tables in place
  // per tile: the output row of its first voxel (-1 in a frame over the
  // cap, whose rows come from the cap's ranks), and the mean's block i
  // (voxels i * kMeanTile ...) starts in tile mtile[i]
  for (uint32_t t = tid; t < nvt; t += kFinBlock) {
    const uint32_t v0 = c.hpre[t], v1 = c.hpre[t + 1];
    const int32_t b = (int32_t)min(c.vtile[t].z, (uint32_t)c.B - 1u);
    const uint32_t fv0 = c.vox_off[b], fv1 = c.vox_off[b + 1];
    c.trow[t] = fv1 - fv0 > (uint32_t)c.cap ? (int64_t)-1 : c.out_voxel_offsets[b] + (int64_t)(v0 - fv0);
    for (uint32_t i = (v0 + kMeanTile - 1) / kMeanTile; (uint64_t)i * kMeanTile < v1; ++i) c.mtile[i] = t;
  }
  if (tid == 0) c.mtile[(V + kMeanTile - 1) / kMeanTile] = nvt > 0 ? nvt - 1 : 0u;
}

struct CapLds {
  uint32_t hc[kCapLdsTiles];    // voxels of the frame's tiles
  uint32_t area[kCapLdsWords];  // the first-place bits (copied from the workspace), then kept flags and their word prefix
  uint32_t tmp[kFinWaves];
  uint32_t sel;
};

// The frame with the most pairs (found by the segments kernel) gets
// kCapHelpers more workgroups for its cap when it has more than max_voxels
// voxels: its slots are flagged in steps of kCapStepSlots dealt out among
// the workgroups (the flag pass costs one workgroup about a microsecond of
// vector instructions per 8,000 slots); each step's flag words are
// numbered inside the step, and the step's kept count goes to the header,
// whose prefix the mean adds.  No workgroup reads another's results.
constexpr int kCapHelpers = 15;
constexpr int kWordBatch = 8;  // a thread's bitmap or flag words loaded together
static_assert(kCapStepSlots == kFinBlock * 32, "one step of the flag pass: 32 ballots per wave");

// Workgroups sharing the cap of a frame with nk pairs (one unless it takes
// more than one step and at most kMaxCapSteps).
__device__ __forceinline__ uint32_t cap_share(uint32_t nk) {
  const uint32_t steps = (nk + kCapStepSlots - 1) / kCapStepSlots;
  return steps > (uint32_t)kMaxCapSteps ? 1u : min((uint32_t)(1 + kCapHelpers), max(steps, 1u));
}

// Workgroup 1 + b of fincap (and, for the frame with the most pairs, up to
// kCapHelpers more): frame b's voxel cap.  The frame keeps the
// max_voxels voxels whose first place (hplace, distinct, in [fstart[b],
// fstart[b+1])) is smallest.  Every pass runs over the frame's slots
// [fstart[b], fstart[b+1]) in order (tile after tile; slot lo + j of a tile
// holds its voxel j when j < its voxel count): slot order restricted to the
// voxels is key order.  The first places are marked in a bitmap over the
// frame's places (by the heads kernel, every tile's heads at once; the
// compaction clears the frame's words), the max_voxels-th marked place is found from a prefix of
// the words' popcounts, the kept voxels are flagged in slot order (one
// ballot per 64 slots) and numbered by a prefix of those flag words.  The
// tables sit in LDS when they fit, otherwise in the frame's regions of the
// workspace.
// The tables of a capped frame: in LDS (kLds) or in the frame's regions of
// the workspace, each pointer of one address space only, so that the
// compiler emits LDS or global instructions rather than generic ones (whose
// waits would also wait for the other kind).
// kShared: workgroup g of G sharing the flag pass (steps g, g + G, ...):
// the flag words go to the workspace, numbered inside their step, and each
// step's kept count to the header.
template <bool kLds, bool kShared>
__device__ void cap_frame(const Config& c, int32_t b, CapLds& S, uint32_t t0, uint32_t nt, uint32_t g, uint32_t G) {
  const int tid = threadIdx.x, lane = tid & 63;
  const uint32_t fs = c.fstart[b], nk = max(c.fstart[b + 1], fs) - fs;
  const size_t words = (size_t)c.N / 32 + (size_t)c.B + 1;  // one region of the workspace's capbits
  const uint32_t wbase = fs / 32 + (uint32_t)b;
  uint32_t* hc = kLds ? S.hc : c.capbits + 3 * words + t0;
  if (kLds)
    for (uint32_t i = tid; i < nt; i += kFinBlock) hc[i] = c.hcount[t0 + i];
  // slot fs + i holds a voxel when its offset in its tile is below the
  // tile's count (every pass loads at clamped slots, unconditionally, and
  // tests that afterwards, so that its loads are in flight together)
  const uint32_t nw = (nk + 31) / 32;
  // 1. the first places, marked in the workspace by the heads kernel (the
  // compaction cleared them); copied to LDS when the tables fit there
  const uint32_t* gbits = c.capbits + wbase;
  if (kLds)
    for (uint32_t base = 0; base < nw; base += kFinBlock * 8) {
      uint32_t v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = gbits[min(base + u * kFinBlock + (uint32_t)tid, nw - 1u)];  // in flight together
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (base + u * kFinBlock + tid < nw) S.area[base + u * kFinBlock + tid] = v[u];
    }
  const uint32_t* bits = kLds ? S.area : gbits;
  constexpr int kUnroll = 32;  // loads in flight per thread: one workgroup walks the whole frame
  __syncthreads();  // the tiles' counts and the bits are in place
  // 2. the max_voxels-th smallest first place: thread t counts a contiguous run of words
  {
    const uint32_t per = (nw + kFinBlock - 1) / kFinBlock;
    const uint32_t w0 = min(tid * per, nw), w1 = min(w0 + per, nw);
    uint32_t mine = 0;
    for (uint32_t w = w0; w < w1; w += kWordBatch) {
      uint32_t x[kWordBatch];
#pragma unroll
      for (int u = 0; u < kWordBatch; ++u) x[u] = bits[min(w + u, nw - 1u)];  // in flight together
#pragma unroll
      for (int u = 0; u < kWordBatch; ++u)
        if (w + u < w1) mine += (uint32_t)__popc(x[u]);
    }
    uint32_t all;
    const uint32_t before = block_exclusive_scan<kFinWaves>(mine, S.tmp, all);
    const uint32_t want = (uint32_t)c.cap;
    if (before < want && before + mine >= want) {
      uint32_t seen = before;
      for (uint32_t w = w0; w < w1; ++w) {
        uint32_t x = bits[w];
        const uint32_t pc = (uint32_t)__popc(x);
        if (seen + pc >= want) {
          for (uint32_t k = want - seen; k > 1; --k) x &= x - 1u;  // drop the lower set bits
          S.sel = fs + w * 32 + (uint32_t)__builtin_ctz(x);
          break;
        }
        seen += pc;
      }
    }
  }
  __syncthreads();
  const uint32_t thr = S.sel;
  // 3. kept voxels flagged in slot order (after the marks: the area is reused)
  uint32_t* kb = kLds && !kShared ? S.area : c.capbits + words + wbase;
  static_assert(kCapStepSlots == (uint32_t)kFinBlock * kUnroll, "one step of the flag pass");
  for (uint32_t step = g; step * kCapStepSlots < nk; step += G) {  // uniform: every wave takes every step
    const uint32_t base = step * kCapStepSlots + (uint32_t)(tid & ~63);
    uint32_t p[kUnroll], n[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {  // clamped, unconditional loads
      const uint32_t i = min(base + u * kFinBlock + (uint32_t)lane, nk - 1u);
      p[u] = c.hplace[fs + i];
      n[u] = hc[i / kVoxTile];
    }
    // the wave's flag words of this step: ballot u's low half goes to lane
    // u, its high half to lane 32 + u, and every lane stores one word
    static_assert(kUnroll == 32, "one flag word per lane and step");
    uint32_t wv = 0;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t i = base + u * kFinBlock + (uint32_t)lane;
      const uint64_t m = __ballot(i < nk && (i % kVoxTile) < n[u] && p[u] <= thr);
      if ((lane & 31) == u) wv = lane < 32 ? (uint32_t)m : (uint32_t)(m >> 32);
    }
    const uint32_t i0 = base + (uint32_t)(lane & 31) * kFinBlock;  // the slots of this lane's word
    const bool has = i0 < nk && (lane < 32 || i0 + 32 < nk);
    if (has) kb[(i0 >> 5) + (uint32_t)(lane >> 5)] = wv;
    if (kShared) {
      // the step's flag words numbered inside the step: word 2 * wave +
      // 32 * (lane % 32) + lane / 32 of the step's 1,024 (in LDS, then one
      // per thread in word order)
      S.area[2u * (uint32_t)(tid >> 6) + 32u * (uint32_t)(lane & 31) + (uint32_t)(lane >> 5)] = has ? (uint32_t)__popc(wv) : 0u;
      __syncthreads();
      const uint32_t x = S.area[tid];
      uint32_t kept;
      const uint32_t before = block_exclusive_scan<kFinWaves>(x, S.tmp, kept);  // its barriers also free S.area
      const uint32_t w = step * (kCapStepSlots / 32) + (uint32_t)tid;
      if (w < nw) c.capbits[2 * words + wbase + w] = before;
      if (tid == 0) c.hdr->cap_steps[step] = kept;
    }
  }
  if (kShared) return;  // the steps' words are numbered
  __syncthreads();
  // 4. kept voxels before each flag word, both tables written to the
  // frame's regions of the workspace: the mean numbers a kept voxel from its
  // flag word and that word's prefix
  {
    uint32_t* gkb = c.capbits + words + wbase;
    uint32_t* gwp = c.capbits + 2 * words + wbase;
    const uint32_t per = (nw + kFinBlock - 1) / kFinBlock;
    const uint32_t w0 = min(tid * per, nw), w1 = min(w0 + per, nw);
    uint32_t mine = 0;
    for (uint32_t w = w0; w < w1; w += kWordBatch) {
      uint32_t x[kWordBatch];
#pragma unroll
      for (int u = 0; u < kWordBatch; ++u) x[u] = kb[min(w + u, nw - 1u)];  // in flight together
#pragma unroll
      for (int u = 0; u < kWordBatch; ++u)
        if (w + u < w1) mine += (uint32_t)__popc(x[u]);
    }
    uint32_t all;
    uint32_t run = block_exclusive_scan<kFinWaves>(mine, S.tmp, all);
    for (uint32_t w = w0; w < w1; w += kWordBatch) {
      uint32_t x[kWordBatch];
#pragma unroll
      for (int u = 0; u < kWordBatch; ++u) x[u] = kb[min(w + u, nw - 1u)];
#pragma unroll
      for (int u = 0; u < kWordBatch; ++u)
        if (w + u < w1) {
          gwp[w + u] = run;
          if (kLds) gkb[w + u] = x[u];
          run += (uint32_t)__popc(x[u]);
        }
    }
  }
}

__global__ __launch_bounds__(kFinBlock) void fincap_kernel(Config c) {
  __shared__ CapLds S;
  const int tid = threadIdx.x;
  if (blockIdx.x == 0) {
    finalize_offsets(c, S.tmp);
    return;
  }
  // workgroups 1 + B ...: helpers of the frame with the most pairs, which
  // leave at once unless that frame has more than one step of slots and
  // more than max_voxels pairs (a frame has no more voxels than pairs)
  const bool helper = (int32_t)blockIdx.x > c.B;
  const uint32_t most = c.hdr->most_pairs;
  const int32_t most_frame = (int32_t)min(c.hdr->most_frame, (uint32_t)c.B - 1u);
  if (helper && (most <= (uint32_t)c.cap || (uint32_t)blockIdx.x - (uint32_t)c.B >= cap_share(most))) return;
  const int32_t b = helper ? most_frame : (int32_t)blockIdx.x - 1;
  const uint32_t nvt = c.hdr->vtiles;
  const uint32_t t0 = min(c.vt_first[b], nvt), t1 = max(min(c.vt_first[b + 1], nvt), t0);
  const uint32_t nt = t1 - t0;
  // the frame's voxels (and, for tables in the workspace, its tiles' counts)
  const size_t words = (size_t)c.N / 32 + (size_t)c.B + 1;
  const uint32_t fs = c.fstart[b], nk = max(c.fstart[b + 1], fs) - fs;
  const bool lds = nt <= (uint32_t)kCapLdsTiles && 2 * ((nk + 31) / 32) <= (uint32_t)kCapLdsWords;
  const uint32_t g = helper ? (uint32_t)blockIdx.x - (uint32_t)c.B : 0u;
  if (g >= cap_share(nk) || (helper && nk <= (uint32_t)c.cap)) return;  // uniform: a helper with no work
  uint32_t mine = 0;
  for (uint32_t i = tid; i < nt; i += kFinBlock) {
    const uint32_t v = c.hcount[t0 + i];
    if (!lds) c.capbits[3 * words + t0 + i] = v;
    mine += v;
  }
  uint32_t total;
  (void)block_exclusive_scan<kFinWaves>(mine, S.tmp, total);
  if (total <= (uint32_t)c.cap) return;  // uniform
  // shared with helpers when this is the frame with the most pairs and it
  // has more than one step of slots (the helpers decide the same way)
  const uint32_t G = b == most_frame ? cap_share(nk) : 1u;
  if (G > 1) {
    if (lds)
      cap_frame<true, true>(c, b, S, t0, nt, g, G);
    else
      cap_frame<false, true>(c, b, S, t0, nt, g, G);
  } else if (lds) {
    cap_frame<true, false>(c, b, S, t0, nt, 0u, 1u);
  } else {
    cap_frame<false, false>(c, b, S, t0, nt, 0u, 1u);
  }
}

// Blocks of kMeanTile consecutive voxels (grid-stride), one thread per
// voxel: its tile (between the tiles of its block and of the next block),
// output row, kept count, point indices and the fp64 mean of every feature.
// Every lane loads at clamped, in-bounds indices, unconditionally, and the
// masks (a voxel past V, a voxel the cap drops, a point past the count) are
// applied to the values afterwards: the loads of each level are in flight
// together.  The records of a voxel's points (RW words each) are read
// kMeanBatch at a time.  When the block's rows are consecutive (no frame
// over the cap in it) they are assembled in LDS and written as contiguous
// runs; otherwise each thread writes its own row.
constexpr int kMeanBatch = 2;  // records in flight per thread: more cost occupancy (VGPRs), fewer add round trips

template <int RW>
__global__ __launch_bounds__(kBlock, 6) void mean_kernel(Config c, const uint32_t* keys, const uint32_t* vals) {
  extern __shared__ uint32_t sm[];
  __shared__ int64_t s_row0;
  __shared__ uint32_t s_step[kMaxCapSteps];  // a shared cap's kept voxels before each step
  WsHeader* h = c.hdr;
  const int tid = threadIdx.x;
  const uint32_t nvt = h->vtiles;
  const uint32_t K = h->kept;
  const uint32_t V = h->voxels;
  const int64_t rows = (int64_t)c.B * c.cap;
  const int C = c.C, M = c.M;
  int32_t* l_co = (int32_t*)sm;              // [kMeanTile][4]
  float* l_ft = (float*)(sm + kMeanTile * 4);  // [kMeanTile][C]
  int32_t* l_pi = (int32_t*)(sm + kMeanTile * (4 + C));  // [kMeanTile][M]
  if (K == 0u || nvt == 0u) return;  // uniform: no voxel (V is 0 too)
  // the frame whose cap was shared numbers its kept voxels inside steps of
  // kCapStepSlots slots: the steps' counts, scanned once per workgroup
  const uint32_t most = h->most_pairs;
  const int32_t shared_frame = most > (uint32_t)c.cap && cap_share(most) > 1u ? (int32_t)min(h->most_frame, (uint32_t)c.B - 1u) : -1;
  if (shared_frame >= 0) {  // uniform
    if (tid < 64) {
      const uint32_t steps = (most + kCapStepSlots - 1) / kCapStepSlots;
      const uint32_t x = (uint32_t)tid < steps ? h->cap_steps[min(tid, kMaxCapSteps - 1)] : 0u;
      const uint32_t incl = wave_inclusive_sum(x);
      if (tid < kMaxCapSteps) s_step[tid] = incl - x;
    }
    __syncthreads();
  }
  for (uint32_t g0 = blockIdx.x * kMeanTile; g0 < V; g0 += gridDim.x * kMeanTile) {
    const uint32_t v = g0 + tid;
    const bool live = v < V;
    const uint32_t vv = min(v, V - 1u);
    const uint32_t nblk = min((uint32_t)kMeanTile, V - g0);
    // the block's voxels lie in tiles mtile[i] .. mtile[i + 1]; the voxel's
    // tile is the largest t there with hpre[t] <= v
    const uint32_t bi = g0 / kMeanTile;
    const uint32_t ta = min(c.mtile[bi], nvt - 1u);
    const uint32_t tb = min(max(c.mtile[bi + 1], ta), nvt - 1u);
    uint32_t t = ta, z = tb;
    while (t < z) {
      const uint32_t mid = (t + z + 1) >> 1;
      if (c.hpre[mid] <= vv) t = mid; else z = mid - 1;
    }
    // the tile and the next one
    const uint32_t tn = min(t + 1u, nvt - 1u);
    const uint4 vt = c.vtile[t], vn = c.vtile[tn];
    const uint32_t j = vv - c.hpre[t], nh = c.hcount[t], nhn = c.hcount[tn];
    const int64_t tr = c.trow[t];
    const int32_t b = (int32_t)min(vt.z, (uint32_t)c.B - 1u);
    const uint32_t slot = vt.x + j, sl = min(slot, K - 1u);
    // the voxel's heads (and, for a frame over the cap, its rank)
    // a voxel of a frame over the cap: kept when its slot's flag is set, its
    // row inside the frame the kept voxels before it (the flag word's prefix
    // and the word's lower bits); the words of other frames are not read
    // for anything (clamped loads)
    const size_t cwords = (size_t)c.N / 32 + (size_t)c.B + 1;
    const uint32_t rel = slot - min(vt.w, slot);
    const size_t cw = min((size_t)(vt.w / 32 + (uint32_t)b + (rel >> 5)), cwords - 1);
    const uint32_t kw = c.capbits[cwords + cw], pw = c.capbits[2 * cwords + cw];
    const uint32_t soff = b == shared_frame ? s_step[min(rel / kCapStepSlots, (uint32_t)kMaxCapSteps - 1u)] : 0u;
    const uint32_t rank = (kw >> (rel & 31)) & 1u ? soff + pw + (uint32_t)__popc(kw & ((1u << (rel & 31)) - 1u)) : 0xffffffffu;
    const int64_t ob = c.out_voxel_offsets[b];
    const uint32_t s0 = min(c.hpos[sl], K - 1u);
    const uint32_t q0 = c.hplace[sl];  // the first point's place (the head's value)
    const uint32_t e_in = c.hpos[min(sl + 1u, K - 1u)];
    const uint32_t e_nx = c.hpos[min(vn.x, K - 1u)];
    int64_t row = tr >= 0 ? tr + (int64_t)j : (rank != 0xffffffffu ? ob + (int64_t)rank : (int64_t)-1);
    if (!live) row = -1;
    if (row >= 0 && (row >= rows || slot >= K)) {
      raise_fault(h, MMBEV_FAULT_INTERNAL);
      row = -1;
    }
    // the voxel's pairs end at the next head: in this tile, at the next
    // tile's first head (same frame), or at the frame's end
    const bool last = j + 1u >= nh;
    const bool next_same = t + 1u < nvt && vn.z == vt.z;
    uint32_t cnt = 0;
    if (row >= 0) {
      if (!last || !next_same || nhn > 0) {
        const uint32_t e = !last ? e_in : (!next_same ? vt.y : e_nx);
        cnt = min(max(e, s0 + 1u) - s0, (uint32_t)M);
      } else {
        // a voxel that runs through the whole next tile: its first
        // max_points pairs decide the count (read eight at a time)
        const uint32_t fend = min(c.fstart[b + 1], K);
        const uint32_t k0 = keys[s0];
        cnt = 1;
        bool more = true;
        for (uint32_t m0 = 1; m0 < (uint32_t)M && more; m0 += 8) {
          uint32_t kk[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const uint32_t i = s0 + m0 + (uint32_t)u;
            kk[u] = m0 + u < (uint32_t)M && i < fend ? keys[i] : ~k0;
          }
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            more = more && kk[u] == k0;
            cnt += more ? 1u : 0u;
          }
        }
      }
    }
    if (tid == 0) s_row0 = row;
    __syncthreads();
    // every row of the block valid and consecutive
    const bool contig = __syncthreads_and((uint32_t)tid >= nblk || (row >= 0 && row == s_row0 + tid)) != 0;
    // the points' records, kMeanBatch at a time (the first place came with
    // the head); the voxel's key loads with the first batch
    const uint32_t kl = keys[s0];
    double sum[8];
#pragma unroll
    for (int f = 0; f < 8; ++f) sum[f] = 0.0;
    for (uint32_t m0 = 0; m0 < cnt; m0 += kMeanBatch) {
      uint32_t q[kMeanBatch];
#pragma unroll
      for (int u = 0; u < kMeanBatch; ++u)
        q[u] = min(m0 + u == 0 ? q0 : vals[min(s0 + m0 + u, K - 1u)], K - 1u);
      uint32_t w[kMeanBatch][RW];
#pragma unroll
      for (int u = 0; u < kMeanBatch; ++u) {  // 16-byte loads when RW is a multiple of four, else 8-byte loads
        const uint32_t* rp = c.rec + (int64_t)q[u] * RW;
        if constexpr ((RW & 3) == 0) {
#pragma unroll
          for (int k = 0; k < RW / 4; ++k) {
            const uint4 x = reinterpret_cast<const uint4*>(rp)[k];
            w[u][4 * k] = x.x;
            w[u][4 * k + 1] = x.y;
            w[u][4 * k + 2] = x.z;
            w[u][4 * k + 3] = x.w;
          }
        } else {
#pragma unroll
          for (int k = 0; k < RW / 2; ++k) {
            const uint2 x = reinterpret_cast<const uint2*>(rp)[k];
            w[u][2 * k] = x.x;
            w[u][2 * k + 1] = x.y;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < kMeanBatch; ++u)
        if (m0 + u < cnt) {
#pragma unroll
          for (int f = 0; f < 8; ++f)
            if (f < C && f + 1 < RW) sum[f] += (double)__uint_as_float(w[u][f + 1]);  // ascending point order
          if (contig)  // uniform: LDS staging or the row itself
            l_pi[tid * M + m0 + u] = (int32_t)w[u][0];
          else
            c.out_point_idx[row * M + m0 + u] = (int32_t)w[u][0];
        }
    }
    if (row >= 0) {
      const uint32_t ix = kl % c.Dx, rest = kl / c.Dx;
      const int32_t co[4] = {b, (int32_t)(rest / c.Dy), (int32_t)(rest % c.Dy), (int32_t)ix};
      c.out_counts[row] = (int32_t)cnt;
      if (contig) {
        for (int m = (int)cnt; m < M; ++m) l_pi[tid * M + m] = -1;
#pragma unroll
        for (int e = 0; e < 4; ++e) l_co[tid * 4 + e] = co[e];
#pragma unroll
        for (int f = 0; f < 8; ++f)
          if (f < C) l_ft[tid * C + f] = (float)(sum[f] / (double)cnt);
      } else {
        for (int m = (int)cnt; m < M; ++m) c.out_point_idx[row * M + m] = -1;
        int32_t* o = c.out_coords + row * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = co[e];
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

hipError_t launch_heads(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st) {
  // a grid of resident size (six per CU by registers) walks the tiles
  hipLaunchKernelGGL(heads_kernel, dim3(std::min(c.vtile_max, 6 * kCus)), dim3(kBlock), 0, st, c, keys, vals);
  return hipGetLastError();
}

hipError_t launch_fincap(const Config& c, hipStream_t st) {
  hipLaunchKernelGGL(fincap_kernel, dim3(1 + c.B + kCapHelpers), dim3(kFinBlock), 0, st, c);
  return hipGetLastError();
}

hipError_t launch_mean(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st) {
  const size_t lds = (size_t)kMeanTile * (4 + c.C + c.M) * 4;
  // one instance per record width (point index, x', y', z', raw features 3..)
  if (c.rec_words == 4)
    hipLaunchKernelGGL(mean_kernel<4>, dim3(c.mean_grid), dim3(kBlock), lds, st, c, keys, vals);
  else if (c.rec_words == 6)
    hipLaunchKernelGGL(mean_kernel<6>, dim3(c.mean_grid), dim3(kBlock), lds, st, c, keys, vals);
  else if (c.rec_words == 8)
    hipLaunchKernelGGL(mean_kernel<8>, dim3(c.mean_grid), dim3(kBlock), lds, st, c, keys, vals);
  else
    hipLaunchKernelGGL(mean_kernel<10>, dim3(c.mean_grid), dim3(kBlock), lds, st, c, keys, vals);
  return hipGetLastError();
}

}  // namespace mmbev

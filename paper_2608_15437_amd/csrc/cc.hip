// Voxel-grid connected-component proposer (robot deployment, Sec. VI):
// connected components of the occupied bird's-eye-view cells of each frame,
// from the voxel rows of the path.
//
// Cells live on a dense per-frame lattice, but only occupied cells are ever
// touched: occupancy is a bitmap (cleared each call), and the union-find
// parents and cell counts are dense arrays read and written only at
// occupied cells (a cell's first voxel initialises them).  Union-find links
// the larger root under the smaller with a compare-and-swap, so whatever the
// order of the unions every tree's root is the smallest cell of its
// component: the result is unique.  Kept roots are flagged in a second
// bitmap whose per-word prefix turns a root into its cluster index, which
// orders the clusters by frame and smallest cell.
#include "launch.hpp"

namespace mmbev {

namespace {

constexpr int32_t kCcNone = -1;               // row outside the band or invalid
constexpr uint32_t kCcFollower = 0x80000000u;  // row whose cell another row owns
constexpr int kCcWords = kBlock * 16;          // bitmap words per scan block

__device__ __forceinline__ int32_t cc_load(const int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Root of x, halving the path on the way: x's parent becomes its
// grandparent.  That is safe without a compare-and-swap: a node that is not
// a root never becomes one again, only roots are swapped, and an ancestor
// stays an ancestor as trees merge, so every store writes an ancestor.
// Parents only ever point at smaller cells, so the walk ends.
__device__ __forceinline__ int32_t cc_find(int32_t* parent, int32_t x) {
  while (true) {
    const int32_t p = cc_load(parent + x);
    if (p == x) return x;
    const int32_t gp = cc_load(parent + p);
    if (gp == p) return p;
    __hip_atomic_store(parent + x, gp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    x = gp;
  }
}

// Root of x without writing (the passes after the unions).
__device__ __forceinline__ int32_t cc_root(const int32_t* parent, int32_t x) {
  int32_t p = cc_load(parent + x);
  while (p != x) {
    x = p;
    p = cc_load(parent + x);
  }
  return x;
}

// Roots of a and b, the two walks in step (their loads in flight together),
// each halving its path.
__device__ __forceinline__ void cc_find2(int32_t* parent, int32_t& a, int32_t& b) {
  while (true) {
    const int32_t pa = cc_load(parent + a), pb = cc_load(parent + b);
    if (pa == a && pb == b) return;
    const int32_t ga = cc_load(parent + pa), gb = cc_load(parent + pb);
    if (ga != pa) __hip_atomic_store(parent + a, ga, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (gb != pb) __hip_atomic_store(parent + b, gb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    a = ga;
    b = gb;
  }
}

// Joins the trees of a and b: the larger root goes under the smaller.
__device__ __forceinline__ void cc_union(int32_t* parent, int32_t a, int32_t b) {
  while (true) {
    cc_find2(parent, a, b);
    if (a == b) return;
    const int32_t hi = max(a, b), lo = min(a, b);
    int32_t expected = hi;
    if (__hip_atomic_compare_exchange_strong(parent + hi, &expected, lo, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT))
      return;
    a = hi;  // hi was joined meanwhile: start again from the two old roots
    b = lo;
  }
}

__device__ __forceinline__ bool cc_bit(const uint32_t* bits, int32_t cell) {
  return (bits[cell >> 5] >> (cell & 31)) & 1u;
}

// Kept roots before `cell` (cell <= total cells).
__device__ __forceinline__ int64_t cc_rank(const CcConfig& c, int64_t cell) {
  if (cell >= c.cells) return (int64_t)c.hdr->clusters;
  const uint32_t w = (uint32_t)(cell >> 5);
  return (int64_t)c.wpre[w] + __popc(c.rootbits[w] & ((1u << (cell & 31)) - 1u));
}

__device__ __forceinline__ int64_t cc_rows(const CcConfig& c) {
  return min(max(c.voff[c.B], (int64_t)0), c.rows);
}

// Runs of consecutive lanes of a wave (a run starts at a lane whose `head`
// is set; lane 0 always starts one).  Rows arrive sorted by key, so rows
// that hit the same bitmap word or the same cluster sit in such runs, and one
// atomic per run replaces one per row: many rows of one big cluster would
// otherwise serialise on its cache line.
struct WaveRun {
  uint32_t lane, start, end;  // this lane's run is lanes [start, end]
};

__device__ __forceinline__ WaveRun wave_run(bool head) {
  WaveRun w;
  w.lane = __lane_id();
  const uint64_t H = __ballot(head || w.lane == 0);
  const uint64_t above = w.lane == 63 ? 0ull : H & (~0ull << (w.lane + 1));
  w.end = above ? (uint32_t)__builtin_ctzll(above) - 1u : 63u;
  const uint64_t upto = H & ((2ull << w.lane) - 1ull);  // wraps to all ones for lane 63
  w.start = 63u - (uint32_t)__builtin_clzll(upto);
  return w;
}

// op over the lanes [lane, end] of the run: the run's first lane gets the
// whole run.  Every lane of the wave must call it.
template <typename T, typename Op>
__device__ __forceinline__ T run_suffix(T v, const WaveRun& w, Op op) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const T o = __shfl_down(v, d, 64);
    if (w.lane + d <= w.end) v = op(v, o);
  }
  return v;
}

__global__ __launch_bounds__(kBlock) void cc_clear_kernel(CcConfig c) {
  const uint64_t g = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
  if (g < 2 * (uint64_t)c.nwords) c.occ[g] = 0u;  // occ and rootbits are adjacent
  if (g == 0) {
    c.hdr->fault = 0;
    c.hdr->clusters = 0;
  }
}

// Cells of the rows: the first row of a cell initialises its parent and
// count.  Also the contract checks (offsets by thread b, each row inside its
// own frame's rows and on the grid).
__global__ __launch_bounds__(kBlock) void cc_mark_kernel(CcConfig c) {
  const int64_t V = cc_rows(c);
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  const int64_t g0 = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  bool bad = false;
  for (int64_t b = g0; b < c.B; b += stride) {
    const int64_t o0 = c.voff[b], o1 = c.voff[b + 1];
    bad |= (b == 0 && o0 != 0) || o1 < o0 || o1 > c.rows || o1 - o0 > (int64_t)c.max_voxels;
  }
  // whole waves step together (the runs below need every lane)
  for (int64_t base = g0 - (int64_t)__lane_id(); base < V; base += stride) {
    const int64_t r = base + (int64_t)__lane_id();
    bool inb = false;
    int32_t cell = 0;
    if (r < V) {
      const int4 q = c.coords[r];
      const bool on_grid = q.x >= 0 && q.x < c.B && q.y >= 0 && (uint32_t)q.y < c.Dz && q.z >= 0 &&
                           (uint32_t)q.z < c.Dy && q.w >= 0 && (uint32_t)q.w < c.Dx;
      const bool own = on_grid && r >= c.voff[q.x] && r < c.voff[q.x + 1];
      bad |= !own;
      inb = own && q.y >= c.z_min && q.y < c.z_max;
      if (inb) cell = (int32_t)((int64_t)q.x * c.ncell + (int64_t)(q.z >> c.shift) * c.Wx + (q.w >> c.shift));
    }
    // runs of lanes on the same bitmap word: one atomicOr per run; a cell's
    // owner is its first row in the run, if no earlier call set its bit
    const int32_t word = inb ? cell >> 5 : -1;
    const uint32_t bit = inb ? 1u << (cell & 31) : 0u;
    const int32_t prev_word = __shfl_up(word, 1, 64);
    const WaveRun w = wave_run(!inb || prev_word != word);
    const uint32_t run_bits = run_suffix(bit, w, [](uint32_t a, uint32_t b) { return a | b; });
    uint32_t old = 0;
    if (inb && w.lane == w.start) old = atomicOr(c.occ + word, run_bits);
    old = __shfl(old, (int)w.start, 64);
    uint32_t before = bit;  // bits of the lanes [start, lane] of the run
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t o = __shfl_up(before, d, 64);
      if (w.lane >= w.start + d) before |= o;
    }
    const uint32_t earlier = __shfl_up(before, 1, 64);
    const bool first = !(old & bit) && !(w.lane > w.start && (earlier & bit));
    int32_t rc = kCcNone;
    if (inb) {
      if (first) {
        c.parent[cell] = cell;
        c.cnt[cell] = 0;
        rc = cell;
      } else {
        rc = (int32_t)((uint32_t)cell | kCcFollower);
      }
    }
    if (r < V) c.rcell[r] = rc;
  }
  if (bad) atomicOr(&c.hdr->fault, MMBEV_FAULT_VOXELS);
}

// Each occupied cell joins its occupied neighbours that come before it
// (left d, and the row above: a b c left to right), so every edge is taken
// once.  With 8 neighbours some joins are implied by the others' own joins:
// b touches a, c and d, so b alone suffices; without b, d touches a, so d
// and c; without b and d, a and c.  At most two joins per cell.
__global__ __launch_bounds__(kBlock) void cc_hook_kernel(CcConfig c) {
  const int64_t V = cc_rows(c);
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t r = (int64_t)blockIdx.x * kBlock + threadIdx.x; r < V; r += stride) {
    const int32_t u = c.rcell[r];
    if (u < 0) continue;  // none, or a follower (top bit set)
    const int32_t local = (int32_t)(u % c.ncell);
    const int32_t x = local % c.Wx, y = local / c.Wx;
    const int32_t up = u - c.Wx;
    const bool d = x > 0 && cc_bit(c.occ, u - 1);
    const bool b = y > 0 && cc_bit(c.occ, up);
    if (c.conn == 4) {
      if (d) cc_union(c.parent, u, u - 1);
      if (b) cc_union(c.parent, u, up);
      continue;
    }
    const bool a = y > 0 && x > 0 && cc_bit(c.occ, up - 1);
    const bool cc = y > 0 && x + 1 < c.Wx && cc_bit(c.occ, up + 1);
    if (b) {
      cc_union(c.parent, u, up);
    } else {
      if (d)
        cc_union(c.parent, u, u - 1);
      else if (a)
        cc_union(c.parent, u, up - 1);
      if (cc) cc_union(c.parent, u, up + 1);
    }
  }
}

// Roots count their cells; the walks halve the paths, so the later passes,
// which walk from a cell to its root without writing, take a step or two.
// (A cell's parent cannot simply be set to its root here: another thread's
// halving may overwrite it with a grandparent.)
__global__ __launch_bounds__(kBlock) void cc_compress_kernel(CcConfig c) {
  const int64_t V = cc_rows(c);
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  const int64_t g0 = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  for (int64_t base = g0 - (int64_t)__lane_id(); base < V; base += stride) {
    const int64_t r = base + (int64_t)__lane_id();
    const int32_t u = r < V ? c.rcell[r] : -1;
    const int32_t root = u >= 0 ? cc_find(c.parent, u) : -1;
    // runs of lanes with one root add their cells at once
    const WaveRun w = wave_run(__shfl_up(root, 1, 64) != root);
    if (root >= 0 && w.lane == w.start) atomicAdd(c.cnt + root, (int32_t)(w.end - w.start + 1));
  }
}

__global__ __launch_bounds__(kBlock) void cc_roots_kernel(CcConfig c) {
  const int64_t V = cc_rows(c);
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t r = (int64_t)blockIdx.x * kBlock + threadIdx.x; r < V; r += stride) {
    const int32_t u = c.rcell[r];
    if (u < 0) continue;
    if (c.parent[u] == u && c.cnt[u] >= c.min_cells) atomicOr(c.rootbits + (u >> 5), 1u << (u & 31));
  }
}

// Kept roots per block of kCcWords bitmap words.
__global__ __launch_bounds__(kBlock) void cc_blocksum_kernel(CcConfig c) {
  __shared__ uint32_t s_tmp[kWaves];
  const uint32_t w0 = blockIdx.x * kCcWords + threadIdx.x * 16;
  uint32_t sum = 0;
#pragma unroll
  for (int k = 0; k < 16; k += 4) {
    if (w0 + k + 3 < c.nwords) {
      const uint4 v = *reinterpret_cast<const uint4*>(c.rootbits + w0 + k);
      sum += __popc(v.x) + __popc(v.y) + __popc(v.z) + __popc(v.w);
    } else {
      for (int j = 0; j < 4; ++j)
        if (w0 + k + j < c.nwords) sum += __popc(c.rootbits[w0 + k + j]);
    }
  }
  uint32_t total;
  block_exclusive_scan(sum, s_tmp, total);
  if (threadIdx.x == 0) c.bsum[blockIdx.x] = total;
}

// One workgroup: exclusive prefix of the block sums (at most kCcWords blocks)
// and the number of clusters.
__global__ __launch_bounds__(kBlock) void cc_blockscan_kernel(CcConfig c) {
  __shared__ uint32_t s_tmp[kWaves];
  const uint32_t i0 = threadIdx.x * 16;
  uint32_t v[16], sum = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    v[k] = i0 + k < c.nblocks ? c.bsum[i0 + k] : 0u;
    sum += v[k];
  }
  uint32_t total;
  uint32_t ex = block_exclusive_scan(sum, s_tmp, total);
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    if (i0 + k < c.nblocks) c.bsum[i0 + k] = ex;
    ex += v[k];
  }
  if (threadIdx.x == 0) c.hdr->clusters = total;
}

// Per-word exclusive prefix of kept roots.
__global__ __launch_bounds__(kBlock) void cc_wordpre_kernel(CcConfig c) {
  __shared__ uint32_t s_tmp[kWaves];
  const uint32_t w0 = blockIdx.x * kCcWords + threadIdx.x * 16;
  uint32_t pc[16], sum = 0;
#pragma unroll
  for (int k = 0; k < 16; k += 4) {
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (w0 + k + 3 < c.nwords) {
      v = *reinterpret_cast<const uint4*>(c.rootbits + w0 + k);
    } else {
      if (w0 + k < c.nwords) v.x = c.rootbits[w0 + k];
      if (w0 + k + 1 < c.nwords) v.y = c.rootbits[w0 + k + 1];
      if (w0 + k + 2 < c.nwords) v.z = c.rootbits[w0 + k + 2];
    }
    pc[k] = __popc(v.x);
    pc[k + 1] = __popc(v.y);
    pc[k + 2] = __popc(v.z);
    pc[k + 3] = __popc(v.w);
    sum += pc[k] + pc[k + 1] + pc[k + 2] + pc[k + 3];
  }
  uint32_t total;
  uint32_t ex = block_exclusive_scan(sum, s_tmp, total) + c.bsum[blockIdx.x];
#pragma unroll
  for (int k = 0; k < 16; k += 4) {
    uint4 o;
    o.x = ex;
    o.y = ex + pc[k];
    o.z = o.y + pc[k + 1];
    o.w = o.z + pc[k + 2];
    ex = o.w + pc[k + 3];
    if (w0 + k + 3 < c.nwords) {
      *reinterpret_cast<uint4*>(c.wpre + w0 + k) = o;
    } else {
      if (w0 + k < c.nwords) c.wpre[w0 + k] = o.x;
      if (w0 + k + 1 < c.nwords) c.wpre[w0 + k + 1] = o.y;
      if (w0 + k + 2 < c.nwords) c.wpre[w0 + k + 2] = o.z;
    }
  }
}

// Cluster rows of the kept roots (their fixed fields, and the identities of
// the box, sums and counts accumulated next), and the frame offsets.
__global__ __launch_bounds__(kBlock) void cc_init_kernel(CcConfig c) {
  const int64_t V = cc_rows(c);
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  const int64_t g0 = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  for (int64_t b = g0; b <= c.B; b += stride) c.out_off[b] = cc_rank(c, b * (int64_t)c.ncell);
  for (int64_t r = g0; r < V; r += stride) {
    const int32_t u = c.rcell[r];
    if (u < 0 || c.parent[u] != u || !cc_bit(c.rootbits, u)) continue;
    mmbev_cluster_t o;
    o.frame = u / c.ncell;
    o.root = u % c.ncell;
    o.cells = c.cnt[u];
    o.voxels = 0;
    o.points = 0;
    o.x0 = o.y0 = INT32_MAX;
    o.x1 = o.y1 = -1;
    o.reserved = 0;
    o.sum_x = o.sum_y = 0;
    c.out[cc_rank(c, u)] = o;
  }
}

// Labels of the rows, voxel and point counts; each cell (its owning row)
// adds itself to its cluster's box and sums.
__global__ __launch_bounds__(kBlock) void cc_accum_kernel(CcConfig c) {
  const int64_t V = cc_rows(c);
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  const int64_t g0 = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  for (int64_t base = g0 - (int64_t)__lane_id(); base < V; base += stride) {
    const int64_t r = base + (int64_t)__lane_id();
    const int32_t rc = r < V ? c.rcell[r] : kCcNone;
    int32_t id = -1, x = 0, y = 0, pts = 0;
    bool cell_owner = false;
    if (rc != kCcNone) {
      const int32_t u = (int32_t)((uint32_t)rc & ~kCcFollower);
      const int32_t root = cc_root(c.parent, u);
      if (cc_bit(c.rootbits, root)) {
        id = (int32_t)cc_rank(c, root);
        pts = c.counts[r];
        cell_owner = rc >= 0;
        const int32_t local = u % c.ncell;
        x = local % c.Wx;
        y = local / c.Wx;
      }
    }
    if (r < V) c.labels[r] = id;
    // runs of lanes of one cluster: one set of atomics per run; the box and
    // sums take each cell once (its owning row)
    const WaveRun w = wave_run(__shfl_up(id, 1, 64) != id);
    const int32_t points = run_suffix(pts, w, [](int32_t a, int32_t b) { return a + b; });
    const int32_t x0 = run_suffix(cell_owner ? x : INT32_MAX, w, [](int32_t a, int32_t b) { return min(a, b); });
    const int32_t y0 = run_suffix(cell_owner ? y : INT32_MAX, w, [](int32_t a, int32_t b) { return min(a, b); });
    const int32_t x1 = run_suffix(cell_owner ? x : -1, w, [](int32_t a, int32_t b) { return max(a, b); });
    const int32_t y1 = run_suffix(cell_owner ? y : -1, w, [](int32_t a, int32_t b) { return max(a, b); });
    const int64_t sx = run_suffix((int64_t)(cell_owner ? x : 0), w, [](int64_t a, int64_t b) { return a + b; });
    const int64_t sy = run_suffix((int64_t)(cell_owner ? y : 0), w, [](int64_t a, int64_t b) { return a + b; });
    if (id >= 0 && w.lane == w.start) {
      mmbev_cluster_t* o = c.out + id;
      atomicAdd(&o->voxels, (int32_t)(w.end - w.start + 1));
      atomicAdd(&o->points, points);
      if (x1 >= 0) {  // some row of the run owns its cell
        atomicMin(&o->x0, x0);
        atomicMin(&o->y0, y0);
        atomicMax(&o->x1, x1);
        atomicMax(&o->y1, y1);
        atomicAdd(reinterpret_cast<unsigned long long*>(&o->sum_x), (unsigned long long)sx);
        atomicAdd(reinterpret_cast<unsigned long long*>(&o->sum_y), (unsigned long long)sy);
      }
    }
  }
}

}  // namespace

hipError_t launch_clusters(const CcConfig& c, hipStream_t st) {
  const uint32_t clear_grid = (uint32_t)((2 * (uint64_t)c.nwords + kBlock - 1) / kBlock);
  const uint64_t need = (uint64_t)std::max<int64_t>(c.rows, (int64_t)c.B + 1);
  const dim3 rows_grid((uint32_t)std::min<uint64_t>((need + kBlock - 1) / kBlock, kCcRowGrid)), block(kBlock);
  hipLaunchKernelGGL(cc_clear_kernel, dim3(std::max(clear_grid, 1u)), block, 0, st, c);
  hipLaunchKernelGGL(cc_mark_kernel, rows_grid, block, 0, st, c);
  hipLaunchKernelGGL(cc_hook_kernel, rows_grid, block, 0, st, c);
  hipLaunchKernelGGL(cc_compress_kernel, rows_grid, block, 0, st, c);
  hipLaunchKernelGGL(cc_roots_kernel, rows_grid, block, 0, st, c);
  hipLaunchKernelGGL(cc_blocksum_kernel, dim3(c.nblocks), block, 0, st, c);
  hipLaunchKernelGGL(cc_blockscan_kernel, dim3(1), block, 0, st, c);
  hipLaunchKernelGGL(cc_wordpre_kernel, dim3(c.nblocks), block, 0, st, c);
  hipLaunchKernelGGL(cc_init_kernel, rows_grid, block, 0, st, c);
  hipLaunchKernelGGL(cc_accum_kernel, rows_grid, block, 0, st, c);
  return hipGetLastError();
}

}  // namespace mmbev

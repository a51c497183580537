// ScatterToBEV (Alg. 1's return value; Sec. IV-F): the voxel features of
// the path written into a dense bird's-eye-view map with the height folded
// into channels, map[b][c*Dz + iz][iy][ix] = feature c of voxel
// (b, iz, iy, ix), zero where no voxel lies.
//
// Two launches: the whole map is cleared, then every voxel writes its C
// values.  The clear is the whole cost (the map is ~10^4 times larger than
// the voxel rows), so it is shaped for the store rate alone: one 16-byte
// store per thread and one short-lived workgroup per 4 KB, issued in memory
// order.  (Workgroups that loop over larger tiles, or a persistent grid,
// measured 20-30% slower on MI355X for the same bytes.)  The values then
// land in lines the clear has just written; V*C*4 bytes next to the map's
// B*C*Dz*Dy*Dx*4.
#include "launch.hpp"

namespace mmbev {

namespace {

typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr uint64_t kBevFillMax = (uint64_t)1 << 31;  // float4s (or floats) per clear launch
constexpr int kBevScatterGrid = 2048;                // workgroups of the value launch (they loop)

__global__ __launch_bounds__(kBlock) void bev_clear4_kernel(float4_t* p, uint64_t n4) {
  const uint64_t g = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
  if (g < n4) p[g] = float4_t{0.0f, 0.0f, 0.0f, 0.0f};
}

__global__ __launch_bounds__(kBlock) void bev_clear1_kernel(float* p, uint64_t n) {
  const uint64_t g = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
  if (g < n) p[g] = 0.0f;
}

// (iz*Dy + iy)*Dx + ix for in-grid coordinates.
__device__ __forceinline__ uint64_t bev_key(const BevConfig& c, const int4& q) {
  return ((uint64_t)q.y * c.Dy + (uint64_t)q.z) * c.Dx + (uint64_t)q.w;
}

__device__ __forceinline__ bool bev_in_grid(const BevConfig& c, const int4& q) {
  return q.x >= 0 && q.x < c.B && q.y >= 0 && (uint32_t)q.y < c.Dz && q.z >= 0 && (uint32_t)q.z < c.Dy &&
         q.w >= 0 && (uint32_t)q.w < c.Dx;
}

// Rows [0, V) with V = voxel_offsets[B] (clamped to the arrays): each row
// with in-grid coordinates writes its C values.  With a fault word, the
// contract is checked too: offsets (thread b checks frame b), each row's
// frame owning the row, and keys strictly ascending inside a frame.
__global__ __launch_bounds__(kBlock) void bev_values_kernel(BevConfig c) {
  const int64_t V = min(max(c.voff[c.B], (int64_t)0), c.rows);
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  const int64_t g0 = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  bool bad = false;
  if (c.fault) {
    for (int64_t b = g0; b < c.B; b += stride) {
      const int64_t o0 = c.voff[b], o1 = c.voff[b + 1];
      bad |= (b == 0 && o0 != 0) || o1 < o0 || o1 > c.rows || o1 - o0 > (int64_t)c.max_voxels;
    }
  }
  for (int64_t r = g0; r < V; r += stride) {
    const int4 q = c.coords[r];
    if (!bev_in_grid(c, q)) {
      bad = true;
      continue;
    }
    if (c.fault) {
      const int64_t lo = c.voff[q.x], hi = c.voff[q.x + 1];
      bad |= r < lo || r >= hi;
      if (r > lo && r < hi) {
        const int4 p = c.coords[r - 1];
        bad |= !bev_in_grid(c, p) || bev_key(c, p) >= bev_key(c, q);
      }
    }
    float* dst = c.map + ((uint64_t)q.x * c.C * c.Dz + (uint64_t)q.y) * c.plane + (uint64_t)q.z * c.Dx + q.w;
    const float* src = c.feats + r * c.C;
    for (int32_t ch = 0; ch < c.C; ++ch) dst[(uint64_t)ch * c.Dz * c.plane] = src[ch];
  }
  if (bad && c.fault) atomicOr(c.fault, MMBEV_FAULT_VOXELS);
}

}  // namespace

hipError_t launch_bev(const BevConfig& c, hipStream_t st) {
  const uint64_t total = (uint64_t)c.B * (uint64_t)c.C * c.Dz * c.plane;
  if (c.vec) {
    float4_t* p = reinterpret_cast<float4_t*>(c.map);
    for (uint64_t done = 0; done < total / 4;) {
      const uint64_t n = std::min(total / 4 - done, kBevFillMax);
      hipLaunchKernelGGL(bev_clear4_kernel, dim3((uint32_t)((n + kBlock - 1) / kBlock)), dim3(kBlock), 0, st,
                         p + done, n);
      done += n;
    }
    if (total % 4)
      hipLaunchKernelGGL(bev_clear1_kernel, dim3(1), dim3(kBlock), 0, st, c.map + total / 4 * 4, total % 4);
  } else {
    for (uint64_t done = 0; done < total;) {
      const uint64_t n = std::min(total - done, kBevFillMax);
      hipLaunchKernelGGL(bev_clear1_kernel, dim3((uint32_t)((n + kBlock - 1) / kBlock)), dim3(kBlock), 0, st,
                         c.map + done, n);
      done += n;
    }
  }
  const uint64_t need = (uint64_t)std::max<int64_t>(c.rows, c.B);
  const uint32_t grid = (uint32_t)std::min<uint64_t>((need + kBlock - 1) / kBlock, kBevScatterGrid);
  hipLaunchKernelGGL(bev_values_kernel, dim3(std::max(grid, 1u)), dim3(kBlock), 0, st, c);
  return hipGetLastError();
}

}  // namespace mmbev

// Cross-window interaction (Sec. 3.3, Eq. (4)-(7)) on the voxel set: the 4c
// channels of every voxel go through four branches, concatenated:
//   [0, c)    depthwise convolution along x with a long 1D kernel (K_x taps),
//   [c, 2c)   the same along y (K_y taps),
//   [2c, 3c)  depthwise 3 x 3 x 3 convolution,
//   [3c, 4c)  identity.
// Submanifold: outputs at the voxels only, and a tap whose cell holds no voxel
// contributes zero; each tap is a centred cross-correlation tap.
//
// Neighbours are found through a dense cell -> row table of the grid (for the
// 468 x 468 pillar grid 0.9 MB), built per scene by k_cwi_clear + k_cwi_map.
// The work is a gather, bound by memory latency and bandwidth, not a contraction:
// no matrix cores.  A wave takes one branch of a group of rows (so no wave runs
// two branches' loops); lane (row, piece) owns 16 bytes of the row's channels of
// that branch.  Taps go in groups of eight: the table entries of the group are
// requested together, then the neighbour pieces and weights, then the fp32
// multiply-adds (groups of 12 or 16 need 118-150 VGPRs and ran 20% slower on
// the pillar frame: fewer waves hide less latency).  The 3 x 3 x 3 taps are
// visited in-plane first (dz = 0, then +1, -1), and a grid one cell deep
// (pillars) stops after the nine in-plane ones.
// Rows are visited in a caller-given order (for example the window-sorted order
// of the SLA plan, where the neighbours along x and y are mostly in the same or
// the adjacent windows), in contiguous ranges per XCD so that each XCD's L2 holds
// the neighbourhood of its rows.
#include <algorithm>

#include "sla_common.h"

namespace sla {

#ifndef SLA_CWI_GROUP
#define SLA_CWI_GROUP 8
#endif
constexpr int kCwiGroup = SLA_CWI_GROUP;  // taps whose loads are in flight together

__global__ __launch_bounds__(256) void k_cwi_clear(int32_t* __restrict__ map, int64_t cells,
                                                   int32_t* __restrict__ conflicts) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if (i == 0 && conflicts) *conflicts = 0;
  for (int64_t j = i; j < cells; j += stride) map[j] = -1;
}

// Each voxel's row into its cell.  The largest row wins a cell claimed twice (so
// the table is the same whatever the order), and every row that finds its cell
// taken or lies outside the grid is counted.
__global__ __launch_bounds__(256) void k_cwi_map(const int32_t* __restrict__ coords, int32_t n,
                                                 int32_t gx, int32_t gy, int32_t gz,
                                                 int32_t* __restrict__ map,
                                                 int32_t* __restrict__ conflicts) {
  const int32_t r = (int32_t)(blockIdx.x * blockDim.x + threadIdx.x);
  if (r >= n) return;
  const int32_t x = coords[3 * r], y = coords[3 * r + 1], z = coords[3 * r + 2];
  if ((uint32_t)x >= (uint32_t)gx || (uint32_t)y >= (uint32_t)gy || (uint32_t)z >= (uint32_t)gz) {
    if (conflicts) atomicAdd(conflicts, 1);
    return;
  }
  const int32_t prev = atomicMax(&map[((int64_t)z * gy + y) * gx + x], r);
  if (prev != -1 && conflicts) atomicAdd(conflicts, 1);
}

template <typename T>
struct CwiPiece;  // 16 bytes of channels
template <>
struct CwiPiece<float> {
  static constexpr int kElems = 4;
  __device__ static void add(float (&acc)[4], uint4 xv, uint4 wv) {
    const float* xs = reinterpret_cast<const float*>(&xv);
    const float* ws = reinterpret_cast<const float*>(&wv);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = fmaf(ws[e], xs[e], acc[e]);
  }
  __device__ static uint4 pack(const float (&acc)[4]) {
    return make_uint4(__float_as_uint(acc[0]), __float_as_uint(acc[1]), __float_as_uint(acc[2]),
                      __float_as_uint(acc[3]));
  }
};
template <>
struct CwiPiece<_Float16> {
  static constexpr int kElems = 8;
  __device__ static void add(float (&acc)[8], uint4 xv, uint4 wv) {
    const _Float16* xs = reinterpret_cast<const _Float16*>(&xv);
    const _Float16* ws = reinterpret_cast<const _Float16*>(&wv);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = fmaf((float)ws[e], (float)xs[e], acc[e]);
  }
  __device__ static uint4 pack(const float (&acc)[8]) {
    uint4 out;
    uint16_t* o = reinterpret_cast<uint16_t*>(&out);
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = f32_to_u16<_Float16>(acc[e]);
    return out;
  }
};
template <>
struct CwiPiece<bf16_t> {
  static constexpr int kElems = 8;
  __device__ static void add(float (&acc)[8], uint4 xv, uint4 wv) {
    const uint16_t* xs = reinterpret_cast<const uint16_t*>(&xv);
    const uint16_t* ws = reinterpret_cast<const uint16_t*>(&wv);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = fmaf(u16_to_f32<bf16_t>(ws[e]), u16_to_f32<bf16_t>(xs[e]), acc[e]);
  }
  __device__ static uint4 pack(const float (&acc)[8]) {
    uint4 out;
    uint16_t* o = reinterpret_cast<uint16_t*>(&out);
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = f32_to_u16<bf16_t>(acc[e]);
    return out;
  }
};

struct CwiArgs {
  const int32_t* map;
  const int32_t* coords;
  const int32_t* order;  // visiting order (null: 0 .. n-1)
  int32_t n, gx, gy, gz;
  int32_t c;             // channels per branch
  int32_t pq;            // 16-byte pieces per branch row (divides 64)
  int32_t kx, ky;
  int32_t groups;        // row groups of 64 / pq rows
};

// Workgroup b: the four branches (one wave each) of row group g(b); groups are
// dealt in contiguous ranges per XCD (workgroups go to the 8 XCDs round-robin).
template <typename T>
__global__ __launch_bounds__(256) void k_cwi_fwd(CwiArgs a, const T* __restrict__ x,
                                                 const T* __restrict__ w_x,
                                                 const T* __restrict__ w_y,
                                                 const T* __restrict__ w_3, T* __restrict__ y) {
  using P = CwiPiece<T>;
  constexpr int E = P::kElems;
  const int lane = lane_id();
  const int branch = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int32_t per_xcd = (a.groups + 7) / 8;
  const int32_t grp = (int32_t)(blockIdx.x & 7) * per_xcd + (int32_t)(blockIdx.x >> 3);
  if (grp >= a.groups) return;
  const int rows_per = 64 / a.pq;
  const int ri = lane / a.pq, pc = lane - ri * a.pq;
  const int32_t p = grp * rows_per + ri;
  const bool live = ri < rows_per && p < a.n;
  const int32_t row = live ? (a.order ? a.order[p] : p) : 0;
  const bool ok = live && (uint32_t)row < (uint32_t)a.n;
  const int C = 4 * a.c;
  const int col = branch * a.c + pc * E;  // first channel of this lane's piece
  const T* xrow = x + (size_t)(ok ? row : 0) * C;
  T* yrow = y + (size_t)(ok ? row : 0) * C;
  if (branch == 3) {  // identity
    if (ok) *reinterpret_cast<uint4*>(yrow + col) = *reinterpret_cast<const uint4*>(xrow + col);
    return;
  }
  const int32_t cx = ok ? a.coords[3 * row] : 0, cy = ok ? a.coords[3 * row + 1] : 0,
                cz = ok ? a.coords[3 * row + 2] : 0;
  const T* w = branch == 0 ? w_x : (branch == 1 ? w_y : w_3);
  const int taps = branch == 0 ? a.kx : (branch == 1 ? a.ky : (a.gz == 1 ? 9 : 27));
  const int half = branch == 0 ? (a.kx - 1) / 2 : (branch == 1 ? (a.ky - 1) / 2 : 0);
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  for (int t0 = 0; t0 < taps; t0 += kCwiGroup) {
    int32_t nb[kCwiGroup];
#pragma unroll
    for (int u = 0; u < kCwiGroup; ++u) {
      const int t = t0 + u;
      int dx = 0, dy = 0, dz = 0;
      if (branch == 0) dx = t - half;
      else if (branch == 1) dy = t - half;
      else {  // in-plane taps first: visit index t is kernel tap (t + 9) mod 27
        const int k = (t + 9) % 27;
        dx = k % 3 - 1;
        dy = (k / 3) % 3 - 1;
        dz = k / 9 - 1;
      }
      const int32_t nx = cx + dx, ny = cy + dy, nz = cz + dz;
      const bool in = ok && t < taps && (uint32_t)nx < (uint32_t)a.gx &&
                      (uint32_t)ny < (uint32_t)a.gy && (uint32_t)nz < (uint32_t)a.gz;
      nb[u] = in ? a.map[((int64_t)nz * a.gy + ny) * a.gx + nx] : -1;
    }
    uint4 xv[kCwiGroup], wv[kCwiGroup];
#pragma unroll
    for (int u = 0; u < kCwiGroup; ++u) {
      const bool hit = (uint32_t)nb[u] < (uint32_t)a.n;
      xv[u] = hit ? *reinterpret_cast<const uint4*>(x + (size_t)nb[u] * C + col) : make_uint4(0, 0, 0, 0);
      const int tap = branch == 2 ? (t0 + u + 9) % 27 : t0 + u;
      wv[u] = (hit && t0 + u < taps) ? *reinterpret_cast<const uint4*>(w + (size_t)tap * a.c + pc * E)
                                     : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < kCwiGroup; ++u) P::add(acc, xv[u], wv[u]);
  }
  if (ok) *reinterpret_cast<uint4*>(yrow + col) = P::pack(acc);
}

hipError_t launch_cwi_build_map(const int32_t* coords, int32_t n, int32_t gx, int32_t gy,
                                int32_t gz, int32_t* map, int32_t* conflicts, hipStream_t stream) {
  const int64_t cells = (int64_t)gx * gy * gz;
  const int64_t blocks = std::min<int64_t>((cells + 255) / 256, 4096);
  hipLaunchKernelGGL(k_cwi_clear, dim3((unsigned)std::max<int64_t>(blocks, 1)), dim3(256), 0, stream,
                     map, cells, conflicts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || n == 0) return e;
  hipLaunchKernelGGL(k_cwi_map, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, coords, n,
                     gx, gy, gz, map, conflicts);
  return hipGetLastError();
}

// dtype: 0 f32, 1 f16, 2 bf16
hipError_t launch_cwi_forward(const int32_t* map, int32_t gx, int32_t gy, int32_t gz,
                              const int32_t* coords, int32_t n, const int32_t* order, int dtype,
                              int32_t channels, int32_t kx, int32_t ky, const void* x,
                              const void* w_x, const void* w_y, const void* w_3, void* y,
                              hipStream_t stream) {
  CwiArgs a;
  a.map = map;
  a.coords = coords;
  a.order = order;
  a.n = n;
  a.gx = gx;
  a.gy = gy;
  a.gz = gz;
  a.c = channels / 4;
  const int esize = dtype == 0 ? 4 : 2;
  a.pq = a.c * esize / 16;
  a.kx = kx;
  a.ky = ky;
  const int rows_per = 64 / a.pq;
  a.groups = (n + rows_per - 1) / rows_per;
  const unsigned grid = (unsigned)(((int64_t)a.groups + 7) / 8 * 8);
  if (dtype == 0)
    hipLaunchKernelGGL((k_cwi_fwd<float>), dim3(grid), dim3(256), 0, stream, a,
                       static_cast<const float*>(x), static_cast<const float*>(w_x),
                       static_cast<const float*>(w_y), static_cast<const float*>(w_3),
                       static_cast<float*>(y));
  else if (dtype == 1)
    hipLaunchKernelGGL((k_cwi_fwd<_Float16>), dim3(grid), dim3(256), 0, stream, a,
                       static_cast<const _Float16*>(x), static_cast<const _Float16*>(w_x),
                       static_cast<const _Float16*>(w_y), static_cast<const _Float16*>(w_3),
                       static_cast<_Float16*>(y));
  else
    hipLaunchKernelGGL((k_cwi_fwd<bf16_t>), dim3(grid), dim3(256), 0, stream, a,
                       static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w_x),
                       static_cast<const bf16_t*>(w_y), static_cast<const bf16_t*>(w_3),
                       static_cast<bf16_t*>(y));
  return hipGetLastError();
}

}  // namespace sla

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
#ifndef SLA_CWI_TILED
#define SLA_CWI_TILED 1
#endif
constexpr bool kCwiTiled = SLA_CWI_TILED != 0;  // pillar grids: the LDS-tiled kernel

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
  int32_t flip;          // 1: every kernel reversed (the input gradient)
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
      int tap = branch == 2 ? (t0 + u + 9) % 27 : t0 + u;
      if (a.flip) tap = (branch == 2 ? 26 : taps - 1) - tap;  // the mirrored offset's weight
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

// ------------------------------------------------------ tiled (pillar grids)
// On a grid one cell deep every tap stays in the plane, and a tile of cells
// with its halo holds all the neighbours its voxels read.  k_cwi_tiled gives
// each convolution branch tiles of its own shape: kTileLen x kTileWid cells
// along the branch's axis (the halo lies along the axis only), kCubeTile^2 for
// the 3 x 3 taps.  A workgroup reads the table entries of its tile and halo
// once, then the 16-byte pieces of those voxels (a slab of at most 64 bytes of
// the branch's channels) into LDS, with the slab's weights, and computes every
// voxel of the tile from LDS: each neighbour piece crosses L2 about once
// instead of once per tap.  Taps are added in the same order as in k_cwi_fwd.
// Row workgroups copy the identity quarter of every row and write zero branch
// outputs for rows the table does not hold (conflicts).
#ifndef SLA_CWI_TILE_LEN
#define SLA_CWI_TILE_LEN 64
#endif
#ifndef SLA_CWI_TILE_WID
#define SLA_CWI_TILE_WID 4
#endif
#ifndef SLA_CWI_CUBE_TILE
#define SLA_CWI_CUBE_TILE 16
#endif
constexpr int kTileLen = SLA_CWI_TILE_LEN;
constexpr int kTileWid = SLA_CWI_TILE_WID;
constexpr int kCubeTile = SLA_CWI_CUBE_TILE;
constexpr int kSlabPieces = 4;
// cells of the largest band (63 taps) and (cell, piece) loads per thread
constexpr int kMaxBand = (kTileLen + 62) * kTileWid > (kCubeTile + 2) * (kCubeTile + 2)
                             ? (kTileLen + 62) * kTileWid
                             : (kCubeTile + 2) * (kCubeTile + 2);
constexpr int kMapLoads = (kMaxBand + 255) / 256;
constexpr int kBandLoads = (kMaxBand * kSlabPieces + 255) / 256;

struct TileGrid {
  int32_t ax, ay;       // x-axis branch tiles along x and across
  int32_t bx, by;       // y-axis branch tiles across x and along y
  int32_t cx, cy;       // 3 x 3 tiles
  int32_t sp, slabs;    // pieces per slab, slabs per branch row
  int32_t n_x, n_y, n_c, n_r;  // workgroups per role
  int32_t max_cells, max_taps; // LDS sizing
};

// Workgroups of the tiled launch, in 64 bits: a grid whose tiles do not fit one
// launch (a degenerate shape such as 1 x 2^31 cells) takes the gather kernel.
inline int64_t cwi_tile_workgroups(int32_t n, int32_t gx, int32_t gy, int32_t pq) {
  const int64_t slabs = pq / (pq < kSlabPieces ? pq : kSlabPieces);
  const int64_t ax = (gx + kTileLen - 1) / kTileLen, ay = (gy + kTileWid - 1) / kTileWid;
  const int64_t bx = (gx + kTileWid - 1) / kTileWid, by = (gy + kTileLen - 1) / kTileLen;
  const int64_t cx = (gx + kCubeTile - 1) / kCubeTile, cy = (gy + kCubeTile - 1) / kCubeTile;
  return (ax * ay + bx * by + cx * cy) * slabs + (n + 256 / pq - 1) / (256 / pq);
}

inline TileGrid cwi_tile_grid(int32_t n, int32_t gx, int32_t gy, int32_t pq, int32_t kx, int32_t ky) {
  TileGrid t;
  t.ax = (gx + kTileLen - 1) / kTileLen;
  t.ay = (gy + kTileWid - 1) / kTileWid;
  t.bx = (gx + kTileWid - 1) / kTileWid;
  t.by = (gy + kTileLen - 1) / kTileLen;
  t.cx = (gx + kCubeTile - 1) / kCubeTile;
  t.cy = (gy + kCubeTile - 1) / kCubeTile;
  t.sp = pq < kSlabPieces ? pq : kSlabPieces;
  t.slabs = pq / t.sp;
  t.n_x = t.ax * t.ay * t.slabs;
  t.n_y = t.bx * t.by * t.slabs;
  t.n_c = t.cx * t.cy * t.slabs;
  t.n_r = (n + 256 / pq - 1) / (256 / pq);   // 256 / pq rows per workgroup, one identity piece per thread
  t.max_cells = std::max(std::max((kTileLen + kx - 1) * kTileWid, kTileWid * (kTileLen + ky - 1)),
                         (kCubeTile + 2) * (kCubeTile + 2));
  t.max_taps = std::max(std::max(kx, ky), 9);
  return t;
}

inline size_t cwi_tile_lds(const TileGrid& t) {
  const size_t rows = ((size_t)t.max_cells * 4 + 15) / 16 * 16;
  return rows + ((size_t)t.max_cells + t.max_taps) * t.sp * 16;
}

template <typename T>
__global__ __launch_bounds__(256) void k_cwi_tiled(CwiArgs a, TileGrid tg, const T* __restrict__ x,
                                                   const T* __restrict__ w_x,
                                                   const T* __restrict__ w_y,
                                                   const T* __restrict__ w_3, T* __restrict__ y) {
  using P = CwiPiece<T>;
  constexpr int E = P::kElems;
  const int tid = (int)threadIdx.x;
  const int C = 4 * a.c;
  const int pq = a.pq;
  int32_t b = (int32_t)blockIdx.x;
  const int32_t n_tiles = tg.n_x + tg.n_y + tg.n_c;
  if (b >= n_tiles) {
    // row workgroup, one (row, identity piece) per thread: the identity quarter,
    // and zero branch outputs for a row the table does not hold
    const int32_t p = (b - n_tiles) * (256 / pq) + tid / pq;
    const int j = tid % pq;
    if (p >= a.n) return;
    const uint4 v = reinterpret_cast<const uint4*>(x + (size_t)p * C)[3 * pq + j];
    const int32_t cx = a.coords[3 * p], cy = a.coords[3 * p + 1], cz = a.coords[3 * p + 2];
    const bool inside = (uint32_t)cx < (uint32_t)a.gx && (uint32_t)cy < (uint32_t)a.gy && cz == 0;
    const int32_t owner = inside ? a.map[(int64_t)cy * a.gx + cx] : -1;
    uint4* dst = reinterpret_cast<uint4*>(y + (size_t)p * C);
    dst[3 * pq + j] = v;
    if (owner != p) {
      dst[j] = make_uint4(0, 0, 0, 0);
      dst[pq + j] = make_uint4(0, 0, 0, 0);
      dst[2 * pq + j] = make_uint4(0, 0, 0, 0);
    }
    return;
  }
  int role = 0;
  if (b >= tg.n_x + tg.n_y) {
    role = 2;
    b -= tg.n_x + tg.n_y;
  } else if (b >= tg.n_x) {
    role = 1;
    b -= tg.n_x;
  }
  const int32_t slab = b % tg.slabs, tile = b / tg.slabs;
  int TX, TY, hx, hy, tpr;
  if (role == 0) { TX = kTileLen; TY = kTileWid; hx = (a.kx - 1) / 2; hy = 0; tpr = tg.ax; }
  else if (role == 1) { TX = kTileWid; TY = kTileLen; hx = 0; hy = (a.ky - 1) / 2; tpr = tg.bx; }
  else { TX = kCubeTile; TY = kCubeTile; hx = 1; hy = 1; tpr = tg.cx; }
  const int32_t X0 = (tile % tpr) * TX, Y0 = (tile / tpr) * TY;
  const int BW = TX + 2 * hx, BH = TY + 2 * hy, cells = BW * BH;
  const int sp = tg.sp;
  extern __shared__ uint4 s_dyn[];
  int32_t* s_row = reinterpret_cast<int32_t*>(s_dyn);
  uint4* s_x = s_dyn + (tg.max_cells * 4 + 15) / 16;
  uint4* s_w = s_x + (size_t)tg.max_cells * sp;
  // 1. table entries of the tile and its halo (at most kMapLoads x 256 cells).  Every
  // load is issued unconditionally from a clamped cell and the result is
  // discarded afterwards: a load under a divergent branch would be waited for
  // before the other branch may write its register.
  bool any = false;
  {
    int32_t rw[kMapLoads];
    bool ok[kMapLoads];
#pragma unroll
    for (int k = 0; k < kMapLoads; ++k) {
      const int i = tid + 256 * k;
      const int bxx = i % BW, byy = i / BW;
      const int32_t gxx = X0 - hx + bxx, gyy = Y0 - hy + byy;
      ok[k] = i < cells && (uint32_t)gxx < (uint32_t)a.gx && (uint32_t)gyy < (uint32_t)a.gy;
      const int32_t sx = min(max(gxx, 0), a.gx - 1), sy = min(max(gyy, 0), a.gy - 1);
      rw[k] = a.map[(int64_t)sy * a.gx + sx];
    }
#pragma unroll
    for (int k = 0; k < kMapLoads; ++k) {
      const int i = tid + 256 * k;
      const int bxx = i % BW, byy = i / BW;
      const int32_t row = ok[k] && (uint32_t)rw[k] < (uint32_t)a.n ? rw[k] : -1;
      if (i < cells) s_row[i] = row;
      any |= row >= 0 && bxx >= hx && bxx < hx + TX && byy >= hy && byy < hy + TY;
    }
  }
  // the slab's weights in visiting order (the mirrored taps for flip)
  const int taps = role == 0 ? a.kx : (role == 1 ? a.ky : 9);
  const T* w = role == 0 ? w_x : (role == 1 ? w_y : w_3);
  for (int i = tid; i < taps * sp; i += 256) {
    const int t = i / sp, j = i - t * sp;
    int k = role == 2 ? 9 + t : t;
    if (a.flip) k = (role == 2 ? 26 : taps - 1) - k;
    s_w[i] = *reinterpret_cast<const uint4*>(w + (size_t)k * a.c + (slab * sp + j) * E);
  }
  if (!__syncthreads_or(any)) return;
  // 2. the slab's pieces of every voxel of the tile and its halo: a thread's
  // pieces are all requested, then stored
  const int col0 = role * a.c + slab * sp * E;
  {
    // as in step 1: loads of absent cells read row 0 (n > 0) and are dropped
    const int nk = (cells * sp + 255) / 256;   // the same for the whole workgroup
    int32_t rr[kBandLoads];
#pragma unroll
    for (int k = 0; k < kBandLoads; ++k) {
      const int i = tid + 256 * k;
      rr[k] = k < nk && i < cells * sp ? s_row[i / sp] : -1;
    }
    uint4 v[kBandLoads];
#pragma unroll
    for (int k = 0; k < kBandLoads; ++k) {
      if (k >= nk) break;
      const int i = tid + 256 * k;
      const int j = i % sp;
      v[k] = *reinterpret_cast<const uint4*>(x + (size_t)max(rr[k], 0) * C + col0 + j * E);
    }
#pragma unroll
    for (int k = 0; k < kBandLoads; ++k) {
      if (k >= nk) break;
      const int i = tid + 256 * k;
      if (i < cells * sp) s_x[i] = rr[k] >= 0 ? v[k] : make_uint4(0, 0, 0, 0);
    }
  }
  __syncthreads();
  // 3. the tile's voxels
  for (int i = tid; i < TX * TY * sp; i += 256) {
    const int u = i / sp, j = i - u * sp;
    const int ux = u % TX, uy = u / TX;
    const int cell = (uy + hy) * BW + ux + hx;
    const int32_t row = s_row[cell];
    if (row < 0) continue;
    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.f;
    if (role == 2) {
#pragma unroll
      for (int t = 0; t < 9; ++t)  // kernel taps 9 .. 17: dx = t % 3 - 1, dy = t / 3 - 1
        P::add(acc, s_x[(cell + (t / 3 - 1) * BW + t % 3 - 1) * sp + j], s_w[t * sp + j]);
    } else {
      const int step = role == 0 ? 1 : BW;
      const int half = role == 0 ? hx : hy;
      const int c0 = cell - half * step;
      for (int t = 0; t < taps; ++t) P::add(acc, s_x[(c0 + t * step) * sp + j], s_w[t * sp + j]);
    }
    *reinterpret_cast<uint4*>(y + (size_t)row * C + col0 + j * E) = P::pack(acc);
  }
}

// dtype: 0 f32, 1 f16, 2 bf16; flip: every kernel reversed
static hipError_t cwi_forward_launch(const int32_t* map, int32_t gx, int32_t gy, int32_t gz,
                                     const int32_t* coords, int32_t n, const int32_t* order,
                                     int dtype, int32_t channels, int32_t kx, int32_t ky,
                                     const void* x, const void* w_x, const void* w_y,
                                     const void* w_3, void* y, hipStream_t stream, int flip) {
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
  a.flip = flip;
  const int rows_per = 64 / a.pq;
  a.groups = (n + rows_per - 1) / rows_per;
  if (gz == 1 && kCwiTiled && cwi_tile_workgroups(n, gx, gy, a.pq) <= INT32_MAX) {
    const TileGrid tg = cwi_tile_grid(n, gx, gy, a.pq, kx, ky);
    const unsigned tgrid = (unsigned)(tg.n_x + tg.n_y + tg.n_c + tg.n_r);
    const size_t lds = cwi_tile_lds(tg);
    if (dtype == 0)
      hipLaunchKernelGGL((k_cwi_tiled<float>), dim3(tgrid), dim3(256), lds, stream, a, tg,
                         static_cast<const float*>(x), static_cast<const float*>(w_x),
                         static_cast<const float*>(w_y), static_cast<const float*>(w_3),
                         static_cast<float*>(y));
    else if (dtype == 1)
      hipLaunchKernelGGL((k_cwi_tiled<_Float16>), dim3(tgrid), dim3(256), lds, stream, a, tg,
                         static_cast<const _Float16*>(x), static_cast<const _Float16*>(w_x),
                         static_cast<const _Float16*>(w_y), static_cast<const _Float16*>(w_3),
                         static_cast<_Float16*>(y));
    else
      hipLaunchKernelGGL((k_cwi_tiled<bf16_t>), dim3(tgrid), dim3(256), lds, stream, a, tg,
                         static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w_x),
                         static_cast<const bf16_t*>(w_y), static_cast<const bf16_t*>(w_3),
                         static_cast<bf16_t*>(y));
    return hipGetLastError();
  }
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

hipError_t launch_cwi_forward(const int32_t* map, int32_t gx, int32_t gy, int32_t gz,
                              const int32_t* coords, int32_t n, const int32_t* order, int dtype,
                              int32_t channels, int32_t kx, int32_t ky, const void* x,
                              const void* w_x, const void* w_y, const void* w_3, void* y,
                              hipStream_t stream) {
  return cwi_forward_launch(map, gx, gy, gz, coords, n, order, dtype, channels, kx, ky, x, w_x, w_y,
                            w_3, y, stream, 0);
}

// ------------------------------------------------------------------ backward
// The chain rule of the module, per tap: dx[q] += w[t] dy[p] and
// dw[t] += dy[p] x[q] for the voxel q at p's cell + offset_t.
//  * dx: with unique voxels, q is p's neighbour at +o exactly when p is q's at -o,
//    so dx is the forward applied to dy with every kernel reversed (flip); the
//    identity quarter passes dy through.
//  * dw: k_cwi_dw.  A lane owns one (tap, 16-byte piece) pair of a branch, so
//    its fp32 sums are one piece (8 fp16 or 4 fp32 channels) and no sums are
//    exchanged between lanes: a wave covers 64 pairs (the 13 taps x 4 pieces
//    of a 32-channel fp16 branch fit one wave) and walks a contiguous range of
//    rows, kDwBatch rows at a time with all their loads in flight (a row's
//    index and cell are the same for the whole wave: fetched once per 64 rows,
//    one per lane, and broadcast with readlane).  The four waves of a
//    workgroup take adjacent row ranges; their sums are added in wave order
//    and written as the workgroup's partial, and k_cwi_dw_reduce adds the
//    partials in workgroup order.  Every order is fixed, so the result is
//    deterministic.  XCD placement: the row blocks of a (branch, slice) are a
//    multiple of 8 and workgroup j of it takes row block (j mod 8) B / 8 + j / 8
//    (B blocks), so each XCD walks one contiguous eighth of the rows for every
//    branch and slice, and its L2 serves the lines they share.
constexpr int kDwWaves = 4;          // waves per workgroup: adjacent row ranges
constexpr int kDwBatch = 8;          // rows whose loads are in flight together
#ifndef SLA_CWI_DW_ROWS
#define SLA_CWI_DW_ROWS 64
#endif
constexpr int kDwRows = SLA_CWI_DW_ROWS;  // rows per wave, until kDwMaxBlocks is reached
constexpr int kDwMaxBlocks = 512;    // workgroups per (branch, pair slice), at most (a multiple of 8)

struct DwGrid {
  int32_t blocks;        // workgroups per (branch, pair slice)
  int32_t rows;          // rows per wave
  int32_t slices[3];     // pair slices (of 64) per branch
};

inline DwGrid cwi_dw_grid(int32_t n, int32_t c, int esize, int32_t kx, int32_t ky, int32_t gz) {
  DwGrid g;
  const int64_t waves = ((int64_t)n + kDwRows - 1) / kDwRows;
  const int64_t want = std::min<int64_t>(kDwMaxBlocks, std::max<int64_t>(1, (waves + kDwWaves - 1) / kDwWaves));
  g.blocks = (int32_t)((want + 7) / 8 * 8);   // a multiple of 8: one eighth per XCD
  const int64_t per_block = (int64_t)g.blocks * kDwWaves;
  g.rows = (int32_t)(((int64_t)n + per_block - 1) / per_block);
  const int pq = c * esize / 16;
  const int taps[3] = {kx, ky, gz == 1 ? 9 : 27};
  for (int b = 0; b < 3; ++b) g.slices[b] = (taps[b] * pq + 63) / 64;
  return g;
}

template <typename T>
__global__ __launch_bounds__(256) void k_cwi_dw(CwiArgs a, DwGrid g, const T* __restrict__ x,
                                                const T* __restrict__ dy,
                                                float* __restrict__ partial) {
  using P = CwiPiece<T>;
  constexpr int E = P::kElems;
  __shared__ float s_red[kDwWaves][64 * E];
  // workgroups in [branch][pair slice][row block] order
  int32_t b = (int32_t)blockIdx.x;
  int branch = 0;
  const int32_t n0 = g.slices[0] * g.blocks, n1 = n0 + g.slices[1] * g.blocks;
  if (b >= n1) {
    branch = 2;
    b -= n1;
  } else if (b >= n0) {
    branch = 1;
    b -= n0;
  }
  const int32_t slice = b / g.blocks, j = b - slice * g.blocks;
  const int32_t kb = (j & 7) * (g.blocks >> 3) + (j >> 3);
  const int wave = (int)(threadIdx.x >> 6), lane = lane_id();
  const int taps = branch == 0 ? a.kx : (branch == 1 ? a.ky : (a.gz == 1 ? 9 : 27));
  const int half = branch == 0 ? (a.kx - 1) / 2 : (branch == 1 ? (a.ky - 1) / 2 : 0);
  const int base = branch == 0 ? 0 : (branch == 1 ? a.kx : a.kx + a.ky);
  const int pair = slice * 64 + lane;
  const bool valid = pair < taps * a.pq;
  const int t = valid ? pair / a.pq : 0;
  const int pc = valid ? pair - t * a.pq : 0;
  const int C = 4 * a.c;
  const int col = branch * a.c + pc * E;
  const int k = branch == 2 ? (t + 9) % 27 : t;  // kernel tap; 3 x 3 x 3 visited in-plane first
  const int ox = branch == 0 ? t - half : (branch == 2 ? k % 3 - 1 : 0);
  const int oy = branch == 1 ? t - half : (branch == 2 ? (k / 3) % 3 - 1 : 0);
  const int oz = branch == 2 ? k / 9 - 1 : 0;
  const int32_t r0 = min(a.n, (kb * kDwWaves + wave) * g.rows), r1 = min(a.n, r0 + g.rows);
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  // 64 rows at a time: lane l fetches row l's index and cell once, and each
  // batch reads them back with readlane (no memory round trip)
  for (int32_t c0 = r0; c0 < r1; c0 += 64) {
    const int32_t pl = c0 + lane;
    const int32_t lrow = pl < r1 ? (a.order ? a.order[pl] : pl) : -1;
    const bool lok = (uint32_t)lrow < (uint32_t)a.n;
    const int32_t lcx = lok ? a.coords[3 * lrow] : 0, lcy = lok ? a.coords[3 * lrow + 1] : 0,
                  lcz = lok ? a.coords[3 * lrow + 2] : 0;
    const int cnt = min(64, r1 - c0);
    // table entries of the neighbours of rows q0 .. q0 + kDwBatch - 1 (-1: none)
    auto entries = [&](int q0, int32_t (&nb)[kDwBatch]) {
#pragma unroll
      for (int u = 0; u < kDwBatch; ++u) {
        const int32_t row = __builtin_amdgcn_readlane(lrow, q0 + u);  // -1 past the range
        const int32_t cx = __builtin_amdgcn_readlane(lcx, q0 + u), cy = __builtin_amdgcn_readlane(lcy, q0 + u),
                      cz = __builtin_amdgcn_readlane(lcz, q0 + u);
        const int32_t nx = cx + ox, ny = cy + oy, nz = cz + oz;
        const bool in = valid && (uint32_t)row < (uint32_t)a.n && (uint32_t)nx < (uint32_t)a.gx &&
                        (uint32_t)ny < (uint32_t)a.gy && (uint32_t)nz < (uint32_t)a.gz;
        nb[u] = in ? a.map[((int64_t)nz * a.gy + ny) * a.gx + nx] : -1;
      }
    };
    // software pipeline: a batch's neighbour and dy pieces are requested with
    // the next batch's table entries, so each batch waits one round trip
    int32_t nb[kDwBatch];
    entries(0, nb);
    for (int q0 = 0; q0 < cnt; q0 += kDwBatch) {
      uint4 xv[kDwBatch], dv[kDwBatch];
#pragma unroll
      for (int u = 0; u < kDwBatch; ++u) {
        const bool hit = (uint32_t)nb[u] < (uint32_t)a.n;
        const int32_t row = __builtin_amdgcn_readlane(lrow, q0 + u);
        xv[u] = hit ? *reinterpret_cast<const uint4*>(x + (size_t)nb[u] * C + col) : make_uint4(0, 0, 0, 0);
        dv[u] = hit ? *reinterpret_cast<const uint4*>(dy + (size_t)row * C + col) : make_uint4(0, 0, 0, 0);
      }
      int32_t nn[kDwBatch];
      if (q0 + kDwBatch < cnt) {
        entries(q0 + kDwBatch, nn);
      } else {
#pragma unroll
        for (int u = 0; u < kDwBatch; ++u) nn[u] = -1;
      }
#pragma unroll
      for (int u = 0; u < kDwBatch; ++u) P::add(acc, xv[u], dv[u]);  // += dy[row] * x[neighbour]
#pragma unroll
      for (int u = 0; u < kDwBatch; ++u) nb[u] = nn[u];
    }
  }
#pragma unroll
  for (int e = 0; e < E; ++e) s_red[wave][lane * E + e] = acc[e];
  __syncthreads();
  if (wave != 0 || !valid) return;
  const int32_t total = (a.kx + a.ky + 27) * a.c;
  float* dst = partial + (size_t)kb * total + (size_t)(base + k) * a.c + pc * E;
#pragma unroll
  for (int e = 0; e < E; ++e)
    dst[e] = ((s_red[0][lane * E + e] + s_red[1][lane * E + e]) + s_red[2][lane * E + e]) +
             s_red[3][lane * E + e];
}

// dw[i] = sum of the workgroups' partials, in workgroup order (16 interleaved
// slices, then the slices in order).  The 3 x 3 x 3 taps off the plane of a
// one-cell-deep grid are never visited: their gradients are zero.
template <typename T>
__global__ __launch_bounds__(1024) void k_cwi_dw_reduce(const float* __restrict__ partial,
                                                        int32_t blocks, int32_t kx, int32_t ky,
                                                        int32_t c, int32_t gz,
                                                        T* __restrict__ dw_x, T* __restrict__ dw_y,
                                                        T* __restrict__ dw_3) {
  __shared__ float s[16][64];
  const int32_t total = (kx + ky + 27) * c;
  const int e = (int)(threadIdx.x & 63), sl = (int)(threadIdx.x >> 6);
  const int32_t i = (int32_t)blockIdx.x * 64 + e;
  const int32_t i3 = i - (kx + ky) * c;
  const bool unvisited = i3 >= 0 && gz == 1 && (i3 / c) / 9 != 1;
  float acc = 0.f;
  if (i < total && !unvisited) {
#pragma unroll 4
    for (int32_t b = sl; b < blocks; b += 16) acc += partial[(size_t)b * total + i];
  }
  s[sl][e] = acc;
  __syncthreads();
  if (sl != 0 || i >= total) return;
  float r = 0.f;
#pragma unroll
  for (int k = 0; k < 16; ++k) r += s[k][e];
  T* out = i < kx * c ? dw_x + i : (i < (kx + ky) * c ? dw_y + (i - kx * c) : dw_3 + i3);
  if constexpr (std::is_same<T, float>::value) *out = r;
  else *reinterpret_cast<unsigned short*>(out) = f32_to_u16<T>(r);
}

size_t cwi_backward_workspace_bytes(int32_t n, int32_t channels, int32_t kx, int32_t ky, int esize) {
  const int c = channels / 4;
  const DwGrid g = cwi_dw_grid(n, c, esize, kx, ky, 1);
  return (size_t)g.blocks * (size_t)((kx + ky + 27) * c) * sizeof(float);
}

template <typename T>
static hipError_t launch_dw(const CwiArgs& a, const DwGrid& g, const void* x, const void* dy,
                            float* partial, void* dw_x, void* dw_y, void* dw_3, hipStream_t stream) {
  const unsigned grid = (unsigned)((g.slices[0] + g.slices[1] + g.slices[2]) * g.blocks);
  hipLaunchKernelGGL((k_cwi_dw<T>), dim3(grid), dim3(256), 0, stream, a, g, static_cast<const T*>(x),
                     static_cast<const T*>(dy), partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int32_t total = (a.kx + a.ky + 27) * a.c;
  hipLaunchKernelGGL((k_cwi_dw_reduce<T>), dim3((unsigned)((total + 63) / 64)), dim3(1024), 0, stream,
                     partial, g.blocks, a.kx, a.ky, a.c, a.gz, static_cast<T*>(dw_x),
                     static_cast<T*>(dw_y), static_cast<T*>(dw_3));
  return hipGetLastError();
}

hipError_t launch_cwi_backward(const int32_t* map, int32_t gx, int32_t gy, int32_t gz,
                               const int32_t* coords, int32_t n, const int32_t* order, int dtype,
                               int32_t channels, int32_t kx, int32_t ky, const void* x,
                               const void* w_x, const void* w_y, const void* w_3, const void* dy,
                               void* dx, void* dw_x, void* dw_y, void* dw_3, void* workspace,
                               hipStream_t stream) {
  hipError_t e = hipSuccess;
  if (n > 0)
    e = cwi_forward_launch(map, gx, gy, gz, coords, n, order, dtype, channels, kx, ky, dy, w_x, w_y,
                           w_3, dx, stream, 1);
  if (e != hipSuccess) return e;
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
  a.flip = 0;
  const DwGrid g = cwi_dw_grid(n, a.c, esize, kx, ky, gz);
  float* partial = static_cast<float*>(workspace);
  if (dtype == 0) return launch_dw<float>(a, g, x, dy, partial, dw_x, dw_y, dw_3, stream);
  if (dtype == 1) return launch_dw<_Float16>(a, g, x, dy, partial, dw_x, dw_y, dw_3, stream);
  return launch_dw<bf16_t>(a, g, x, dy, partial, dw_x, dw_y, dw_3, stream);
}

}  // namespace sla

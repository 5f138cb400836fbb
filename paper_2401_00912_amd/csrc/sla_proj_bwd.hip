// Backward of the projection layer, SLA and output projection.
//
// Sec. 3.2 trains the shared projection layer that maps every voxel to Q, K and V,
// and the block's output projection; the gradients follow from the forward
//     [q | k | v] = x W_qkv^T + b_qkv,  o = SLA(q, k, v),  y = o W_o^T + b_o
// by the chain rule, for dy = dL/dy over the rows that lie in a window:
//     do = dy W_o,                      dW_o = dy^T o,       db_o = sum_rows dy,
//     dq, dk, dv = SLA backward of do,
//     dx = [dq | dk | dv] W_qkv,        dW_qkv = [dq | dk | dv]^T x,
//     db_qkv = sum_rows [dq | dk | dv].
// q, k, v are recomputed from x (they never reach HBM in the forward), o is the
// forward's output.  The launches:
//   k_prep          W_qkv^T and W_o^T into the workspace, so that every product
//                   below reads its weights as rows, and which rows lie in a
//                   window (from the plan's permutation), in one launch;
//   k_rows_gemm     q | k | v = x W_qkv^T + b_qkv, and do = dy W_o: a row of the
//                   output is a row of the input times a weight matrix held in LDS;
//   (SLA backward)  dq, dk, dv;
//   k_rows_gemm     dx = [dq | dk | dv] W_qkv (zero for rows in no window);
//   k_wgrad         per group of rows, partial dW_qkv, dW_o and the bias
//                   gradients: sums over rows on the matrix cores, the staged rows
//                   read as contraction operands by LDS transpose loads;
//   k_wgrad_reduce  the groups' partials summed in group order.
// Rows are visited in their own order, rows in no window masked out; every sum
// over rows has a fixed order, so the results do not depend on scheduling.
#include <algorithm>

#include "sla_attn_core.h"

namespace sla {

// ------------------------------------------------------------ preparation
// One launch before the products: the weights as rows (W_qkv^T and W_o^T, in
// 32 x 32 tiles, one a workgroup) and the row mask (the other workgroups).
//
// Tile (bx, by) of dst[j][k] = src[k][j] for src [K, N] (row-major), dst [N, K].
template <typename T>
__device__ __forceinline__ void transpose_tile(const T* __restrict__ src, T* __restrict__ dst, int32_t K,
                                               int32_t N, int32_t bx, int32_t by,
                                               unsigned short (&tile)[32][33]) {
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;   // 32 x 8
  const int32_t k0 = by * 32, j0 = bx * 32;
  const unsigned short* s = reinterpret_cast<const unsigned short*>(src);
  unsigned short* d = reinterpret_cast<unsigned short*>(dst);
  for (int r = ty; r < 32; r += 8)
    if (k0 + r < K && j0 + tx < N) tile[r][tx] = s[(size_t)(k0 + r) * N + j0 + tx];
  __syncthreads();
  for (int r = ty; r < 32; r += 8)
    if (j0 + r < N && k0 + tx < K) d[(size_t)(j0 + r) * K + k0 + tx] = tile[tx][r];
}

// mask[row] = 1 for the rows in a window, 0 for the others: the plan's sorted
// positions [0, offsets[W]) hold the rows in windows and, for a plan built from
// window ids, positions [offsets[W], n) the others, so every row is written once.
struct PrepArgs {
  const void* wqkv;          // [3C, C]
  void* wt_qkv;              // [C, 3C]
  const void* wo;            // [C, C]
  void* wt_o;                // [C, C]
  const PlanHeader* hdr;
  const int32_t* perm;
  const int32_t* nvalid;     // offsets[W]
  uint8_t* mask;
  int32_t C, n, W, mask_blocks;
};

template <typename T>
__global__ __launch_bounds__(256) void k_prep(PrepArgs pa) {
  __shared__ unsigned short tile[32][33];
  const int32_t cb = pa.C / 32, tq = cb * 3 * cb, to = cb * cb;
  const int32_t b = (int32_t)blockIdx.x;
  if (b < tq) {
    transpose_tile(static_cast<const T*>(pa.wqkv), static_cast<T*>(pa.wt_qkv), 3 * pa.C, pa.C, b % cb, b / cb,
                   tile);
    return;
  }
  if (b < tq + to) {
    transpose_tile(static_cast<const T*>(pa.wo), static_cast<T*>(pa.wt_o), pa.C, pa.C, (b - tq) % cb,
                   (b - tq) / cb, tile);
    return;
  }
  // the header, the count of rows in windows and the thread's first
  // permutation entry are requested together (every plan holds n permutation
  // entries; a CSR plan's are not used), so the mask waits one round trip
  const PlanHeader* hdr = pa.hdr;
  const int32_t n = pa.n, stride = pa.mask_blocks * 256;
  int32_t p = (b - tq - to) * 256 + (int32_t)threadIdx.x;
  int32_t pr = p < n ? pa.perm[p] : 0;
  const int32_t nv = *pa.nvalid;
  if (hdr->magic != kPlanMagic || hdr->n != pa.n || hdr->num_windows != pa.W) return;
  const bool csr = hdr->csr != 0;
  const int32_t nvalid = max(0, min(nv, n));
  for (; p < n; p += stride) {
    const int32_t row = csr ? p : pr;
    if (p + stride < n) pr = pa.perm[p + stride];
    if ((uint32_t)row < (uint32_t)n) pa.mask[row] = p < nvalid ? 1 : 0;
  }
}

// ------------------------------------------------------------ row products
// out[row][j] = sum_k A(row, k) Wr[j][k] + bias[j] for every row.  A(row, k) =
// a[k / C][row][k % C] over nseg segments [n, C] (K = nseg C); Wr is [N, K]
// row-major (a weight in the [out, in] layout); output column j goes to
// out[j / C][row][j % C].  Rows in no window (mask 0) get zero input, so their
// outputs are the bias (zero when there is none).
//
// A workgroup of 16 waves keeps the weight rows of NB output columns (all N when
// they fit) in LDS, padded rows of K + 8 elements, and walks 16-row tiles, one
// per wave.  With KBH > 0 (K <= 32 KBH) a wave reads its tile's input once into
// registers and forms every 16 NBT-column sub-block from them; with KBH = 0 (K
// = 3C for C = 256) it reads the input again per sub-block, a 256-channel
// segment at a time, the next segment's pieces (or the next tile's first
// segment) in flight while one is formed.
// With the weight rows as the first matrix-core operand and the input rows
// (16-byte pieces of 8 channels) as the second, lane (i, g) receives 4 columns
// of the tile's row i from each tile; the weight rows are staged in an order
// that makes a tile pair's 8 columns of a lane consecutive (one 16-byte piece),
// and lanes i and i ^ 8 trade pieces so that each store writes 8 rows x 128
// bytes.
// When N takes several column blocks, the workgroups of one row range sit 8 ids
// apart: workgroups are dealt to the 8 XCDs in turn, so the column blocks of a
// row range share one XCD, and its L2 serves their common input rows (the
// grid's row ranges are then a multiple of 8).
constexpr int kRowGemmThreads = 1024;

struct RowGemmArgs {
  const void* a[3];
  void* out[3];
  const void* w;             // Wr [N, K]
  const void* bias;          // [N] or null
  const PlanHeader* hdr;
  const uint8_t* mask;       // rows in windows
  int32_t C, K, N, n, W;
  int32_t NB;                // columns a workgroup holds (a multiple of 16 NBT dividing N)
};

template <typename T, int NBT, int KBH>
__global__ __launch_bounds__(kRowGemmThreads) void k_rows_gemm(RowGemmArgs ga) {
  constexpr int SB = 16 * NBT;
  if (ga.hdr->magic != kPlanMagic || ga.hdr->n != ga.n || ga.hdr->num_windows != ga.W) return;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];
  const int K = ga.K, LDW = K + 8, C = ga.C, NB = ga.NB;
  T* s_w = reinterpret_cast<T*>(lds_raw);
  float* s_b = reinterpret_cast<float*>(s_w + NB * LDW);
  const int32_t cols = ga.N / NB;
  const int32_t hi = (int32_t)blockIdx.x >> 3;
  const int32_t rb = (hi / cols) * 8 + ((int32_t)blockIdx.x & 7);   // row range
  const int32_t ranges = (int32_t)gridDim.x / cols;
  const int32_t n0 = (hi % cols) * NB;
  {
    // output column jj of the block is matrix-core row pi(jj): within each 32
    // columns, column 8 g + 4 v + j is row 16 v + 4 g + j (tile v of the pair),
    // so that lane (i, g) receives columns 8 g .. 8 g + 7 of a tile pair and
    // stores them as one 16-byte piece
    auto pi = [](int jj) { return (jj & ~31) | ((jj & 4) << 2) | ((jj & 24) >> 1) | (jj & 3); };
    const int pieces = K / 8;
    const T* w = static_cast<const T*>(ga.w);
    for (int idx = threadIdx.x; idx < NB * pieces; idx += blockDim.x) {
      const int jj = idx / pieces, pc = idx - jj * pieces;
      *reinterpret_cast<uint4*>(s_w + pi(jj) * LDW + 8 * pc) =
          *reinterpret_cast<const uint4*>(w + (size_t)(n0 + jj) * K + 8 * pc);
    }
    const unsigned short* b = static_cast<const unsigned short*>(ga.bias);
    for (int jj = threadIdx.x; jj < NB; jj += blockDim.x) s_b[pi(jj)] = b ? u16_to_f32<T>(b[n0 + jj]) : 0.f;
  }
  __syncthreads();
  using F8 = Frag<T, 8>;
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  const int lane = lane_id(), wv = threadIdx.x >> 6;
  const int i = lane & 15, g = lane >> 4;
  constexpr bool held = KBH > 0;   // the host picks KBH > 0 only when K <= 32 KBH
  constexpr int NW = kRowGemmThreads / 64;
  // the bias-added, rounded outputs of tile `tile`, columns n0 + sb .. + SB - 1
  auto store_block = [&](int32_t tile, int sb, const floatx4 (&acc)[NBT]) {
    const int32_t j0 = n0 + sb;   // a sub-block lies in one output segment (C % SB == 0)
    T* outp = static_cast<T*>(ga.out[j0 / C]);
    // tile pairs 2w and 2w + 1 (64 columns): lanes i and i ^ 8 swap one
    // piece (row rotation by 8 lanes), so that each store writes 8 rows x 128
    // bytes: rows 0-7 of the tile first, then rows 8-15
    const int32_t pa = tile * 16 + (i & 7), pb = pa + 8;
    const uint32_t ccol = (uint32_t)(j0 % C) + (i < 8 ? 8 * g : 32 + 8 * g);
#pragma unroll
    for (int w = 0; w < NBT / 4; ++w) {
      Raw<T, 8> pk[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        float f[8];
#pragma unroll
        for (int v = 0; v < 2; ++v) {
          const int t = 4 * w + 2 * u + v;
          const float4 bias = *reinterpret_cast<const float4*>(s_b + sb + 16 * t + 4 * g);
          f[4 * v + 0] = acc[t][0] + bias.x;
          f[4 * v + 1] = acc[t][1] + bias.y;
          f[4 * v + 2] = acc[t][2] + bias.z;
          f[4 * v + 3] = acc[t][3] + bias.w;
        }
        pk[u] = F8::from_f32(f);
      }
      const uint4 snd = __builtin_bit_cast(uint4, i < 8 ? pk[1] : pk[0]);
      uint4 rcv;
      rcv.x = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)snd.x, 0x128, 0xf, 0xf, false);   // row_ror:8
      rcv.y = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)snd.y, 0x128, 0xf, 0xf, false);
      rcv.z = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)snd.z, 0x128, 0xf, 0xf, false);
      rcv.w = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)snd.w, 0x128, 0xf, 0xf, false);
      const uint4 da = i < 8 ? __builtin_bit_cast(uint4, pk[0]) : rcv;
      const uint4 db = i < 8 ? rcv : __builtin_bit_cast(uint4, pk[1]);
      if (pa < ga.n) *reinterpret_cast<uint4*>(elem_at(outp, (uint32_t)pa * (uint32_t)C + ccol + 64 * w)) = da;
      if (pb < ga.n) *reinterpret_cast<uint4*>(elem_at(outp, (uint32_t)pb * (uint32_t)C + ccol + 64 * w)) = db;
    }
  };
  const int32_t step = ranges * NW;
  if constexpr (held) {
    for (int32_t tile = rb * NW + wv; tile * 16 < ga.n; tile += step) {
      const int32_t p = tile * 16 + i;
      const bool inside = p < ga.n;
      const int32_t row = inside ? p : 0;
      const bool valid = inside && ga.mask[row] != 0;
      // the tile's input: k block kb is channels 32 kb .. + 31 of A, in
      // segment 32 kb / C
      Raw<T, 8> xh[KBH];
#pragma unroll
      for (int kb = 0; kb < KBH; ++kb) {
        xh[kb] = F8::zero();
        if (32 * kb < K) {
          const int s = (32 * kb) / C, c0 = (32 * kb) % C;
          const T* src = static_cast<const T*>(ga.a[s]);
          const Raw<T, 8> xo = __builtin_bit_cast(
              Raw<T, 8>, *reinterpret_cast<const uint4*>(elem_at(src, (uint32_t)row * (uint32_t)C + c0 + 8 * g)));
          if (valid) xh[kb] = xo;
        }
      }
      for (int sb = 0; sb < NB; sb += SB) {
        floatx4 acc[NBT];
#pragma unroll
        for (int t = 0; t < NBT; ++t) acc[t] = zero;
        const T* wsb = s_w + (sb + i) * LDW + 8 * g;
#pragma unroll
        for (int kb = 0; kb < KBH; ++kb) {
          if (32 * kb >= K) break;
#pragma unroll
          for (int t = 0; t < NBT; ++t) {
            const Raw<T, 8> wo = *reinterpret_cast<const Raw<T, 8>*>(wsb + 16 * t * LDW + 32 * kb);
            acc[t] = F8::mma(wo, xh[kb], acc[t]);
          }
        }
        store_block(tile, sb, acc);
      }
    }
  } else {
    // The input 128 channels at a time (a step), all of a step's pieces
    // requested together and the next step's in flight while one is formed;
    // the next tile's first step and mask byte are requested during this
    // tile's last step, so that no tile waits a round trip at its start.  The rows are read unconditionally (rows past n read row 0), and
    // the sums of rows in no window or past n are replaced by those of zero
    // input.
    constexpr int KS = 4, HS = 32 * KS;   // pieces and channels per step (C % HS == 0)
    const int steps = K / HS;
    auto row_of = [&](int32_t t) -> int32_t {
      const int32_t p = t * 16 + i;
      return p < ga.n ? p : 0;
    };
    auto fetch_seg = [&](Raw<T, 8>(&x)[KS], int s, int32_t row) {
      const T* src = static_cast<const T*>(ga.a[(HS * s) / C]);
      const int c0 = (HS * s) % C;
#pragma unroll
      for (int kb = 0; kb < KS; ++kb)
        x[kb] = __builtin_bit_cast(
            Raw<T, 8>, *reinterpret_cast<const uint4*>(elem_at(src, (uint32_t)row * (uint32_t)C + c0 + 32 * kb + 8 * g)));
    };
    Raw<T, 8> xs[KS], xn[KS];
    int32_t tile = rb * NW + wv;
    int32_t row = row_of(tile);
    uint8_t mk = 0;
    if (tile * 16 < ga.n) {
      fetch_seg(xs, 0, row);
      mk = ga.mask[row];
    }
    for (; tile * 16 < ga.n; tile += step) {
      const bool valid = tile * 16 + i < ga.n && mk != 0;
      const int32_t nt = tile + step;
      const bool more = nt * 16 < ga.n;
      const int32_t nrow = row_of(nt);
      uint8_t nmk = 0;
      for (int sb = 0; sb < NB; sb += SB) {
        floatx4 acc[NBT];
#pragma unroll
        for (int t = 0; t < NBT; ++t) acc[t] = zero;
        const T* wsb = s_w + (sb + i) * LDW + 8 * g;
        for (int s = 0; s < steps; ++s) {
          if (s + 1 < steps) {
            fetch_seg(xn, s + 1, row);
          } else if (sb + SB < NB) {
            fetch_seg(xn, 0, row);
          } else if (more) {
            fetch_seg(xn, 0, nrow);
            nmk = ga.mask[nrow];
          }
#pragma unroll
          for (int kb = 0; kb < KS; ++kb)
#pragma unroll
            for (int t = 0; t < NBT; ++t) {
              const Raw<T, 8> wo = *reinterpret_cast<const Raw<T, 8>*>(wsb + 16 * t * LDW + HS * s + 32 * kb);
              acc[t] = F8::mma(wo, xs[kb], acc[t]);
            }
          if (s + 1 < steps) {
#pragma unroll
            for (int kb = 0; kb < KS; ++kb) xs[kb] = xn[kb];
          }
        }
        // lane (i, g) holds row i's sums only: a row in no window or past n
        // gets the sums of zero input, +0
#pragma unroll
        for (int t = 0; t < NBT; ++t) acc[t] = valid ? acc[t] : zero;
        store_block(tile, sb, acc);
#pragma unroll
        for (int kb = 0; kb < KS; ++kb) xs[kb] = xn[kb];
      }
      row = nrow;
      mk = nmk;
    }
  }
}

// ------------------------------------------------------------ weight gradients
// For one row group, four kinds of workgroup: A = dq, dk, dv (with B = x: rows
// 0..C-1, C..2C-1, 2C..3C-1 of dW_qkv and of db_qkv) and A = dy (with B = o:
// dW_o, db_o).  A unit is a 32-row slab m0 of A's gradient rows and a 64-column
// chunk n0 of B's: partial[group][m0 + e][n0 + c] = sum over the group's rows in
// windows of A(row, m0 + e) B(row, n0 + c), and, for n0 = 0, the bias partial
// sum_rows A(row, m0 + e).  The rows 0..n-1 are split into `groups` contiguous
// ranges.
//
// A workgroup of NT / 64 waves (8, or 16 for C = 256) takes as many units of
// one kind (C / 32 x C / 64 of them per kind) and walks its rows 32 at a time:
// the rows of A and B are staged in LDS once (rows in no window stored as
// zeros), the next two jobs' rows loaded into registers while this one is
// summed; each wave reads its columns as operands of a contraction over the
// job's rows with LDS transpose loads and accumulates its 2 x 4 result tiles.
// Every workgroup stages all of B's columns, so fewer, wider workgroups per
// kind stage less: 16 waves for C = 256 (128 A columns and 256 B columns a row,
// twice per kind, against 64 and 256 four times with 8 waves).
struct WgradArgs {
  const void* mats[6];   // dq, dk, dv, x, dy, o [n, C]
  const PlanHeader* hdr;
  const uint8_t* mask;   // rows in windows
  float* part;           // [groups][total]: dW_qkv [3C][C], dW_o [C][C], db_qkv [3C], db_o [C]
  int32_t C, n, W, groups, wgs_per_kind;
};

constexpr int kWgradChunk = 64;    // gradient columns per unit

// threads of a k_wgrad workgroup for a given C
__host__ __device__ constexpr int wgrad_threads(int C) { return C == 256 ? 1024 : 512; }

// A columns a workgroup stages: its NT / 64 units (one a wave) cover
// (NT / 64) / (C / 64) slabs of 32 A columns, each with all C / 64 chunks of
// B's; at most C.
__host__ __device__ constexpr int wgrad_a_cols(int C, int NT) {
  return (NT / 64) / (C / kWgradChunk) * 32 < C ? (NT / 64) / (C / kWgradChunk) * 32 : C;
}

// SP: 16-byte pieces a thread stages per job, at most 32 (na + C) / 8 / NT:
// 1, 2, 2 for C = 64, 128 (512 threads), 256 (1,024 threads)
template <typename T, int SP, int NT>
__global__ __launch_bounds__(NT) void k_wgrad(WgradArgs wa) {
  using F = Frag<T, 8>;
  constexpr int NCB = kWgradChunk / 32;
  constexpr int NWV = NT / 64;
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  if (wa.hdr->magic != kPlanMagic || wa.hdr->n != wa.n || wa.hdr->num_windows != wa.W) return;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];
  const int C = wa.C;
  const int tid = threadIdx.x, lane = lane_id(), wv = tid >> 6;
  const int i = lane & 15, g = lane >> 4;
  const int32_t per_group = 4 * wa.wgs_per_kind;
  // the workgroups of one group are 8 ids apart: workgroups are dealt to the 8
  // XCDs in turn, so they share one XCD and its L2, which serves x to the three
  // kinds that read it (the grid is padded to whole blocks of 8 groups)
  const int32_t hi = (int32_t)blockIdx.x >> 3;
  const int32_t grp = (hi / per_group) * 8 + ((int32_t)blockIdx.x & 7);
  if (grp >= wa.groups) return;
  const int kind = (hi % per_group) / wa.wgs_per_kind;
  const int part_of_kind = (hi % per_group) % wa.wgs_per_kind;
  const int chunks = C / kWgradChunk;
  const int units = (C / 32) * chunks;
  const int unit = part_of_kind * NWV + wv;
  const bool active = unit < units;
  const int slab = active ? unit / chunks : 0, chunk = active ? unit % chunks : 0;
  const int m0 = 32 * slab, n0 = kWgradChunk * chunk;
  // the workgroup's units cover A's columns a0 .. a0 + na - 1 (all of them for
  // C <= 128, half for C = 256) and all of B's: only those are staged
  const int na = wgrad_a_cols(C, NT);
  const int a0 = (part_of_kind * NWV / chunks) * 32;
  const int LDR = na + C + 8;                // staged row: A's columns then B's, padded
  T* stage = reinterpret_cast<T*>(lds_raw);   // [2][32][LDR]
  const T* A = static_cast<const T*>(wa.mats[kind == 3 ? 4 : kind]);
  const T* B = static_cast<const T*>(wa.mats[kind == 3 ? 5 : 3]);
  const int32_t p0 = (int32_t)((int64_t)wa.n * grp / wa.groups);
  const int32_t p1 = (int32_t)((int64_t)wa.n * (grp + 1) / wa.groups);
  float one8[8] = {1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f};
  const Raw<T, 8> ones = F::from_f32(one8);
  floatx4 acc[2][2 * NCB], bacc[2];
#pragma unroll
  for (int et = 0; et < 2; ++et) {
    bacc[et] = zero;
#pragma unroll
    for (int ct = 0; ct < 2 * NCB; ++ct) acc[et][ct] = zero;
  }
  // staging: 32 rows x (na + C) / 8 pieces of 16 bytes, at most SP a thread
  const int per_mat = na / 8, pieces_per_row = per_mat + C / 8;
  const int npieces = 32 * pieces_per_row;
  // the data and the row's mask byte are loaded together; rows in no window
  // are zeroed when stored.  With SP <= 2 two jobs are in flight in registers
  // (sets a and b) while a third is summed from LDS; otherwise one.
  struct Held {
    uint4 v[SP];
    int keep[SP];
  };
  auto load_job = [&](Held& h, int32_t base) {
#pragma unroll
    for (int k = 0; k < SP; ++k) {
      const int idx = tid + k * NT;
      h.v[k] = make_uint4(0, 0, 0, 0);
      h.keep[k] = 0;
      if (idx < npieces) {
        const int r = idx / pieces_per_row, pc = idx - r * pieces_per_row;
        const int32_t row = base + r;
        const T* src = pc < per_mat ? A + a0 + 8 * pc : B + 8 * (pc - per_mat);
        if (row < p1) {
          h.keep[k] = wa.mask[row];
          h.v[k] = *reinterpret_cast<const uint4*>(src + (size_t)row * C);
        }
      }
    }
  };
  auto store_job = [&](const Held& h, T* buf) {
#pragma unroll
    for (int k = 0; k < SP; ++k) {
      const int idx = tid + k * NT;
      if (idx < npieces) {
        const int r = idx / pieces_per_row, pc = idx - r * pieces_per_row;
        *reinterpret_cast<uint4*>(buf + r * LDR + 8 * pc) = h.keep[k] != 0 ? h.v[k] : make_uint4(0, 0, 0, 0);
      }
    }
  };
  // one job's contraction over its 32 rows, its columns read straight from the
  // staged rows (LDS transpose loads)
  auto sum_job = [&](const T* cur) {
    if (!active) return;
    const unsigned short* cu = reinterpret_cast<const unsigned short*>(cur);
    Raw<T, 8> pa[2];
#pragma unroll
    for (int et = 0; et < 2; ++et) {
      pa[et] = lds_cols<T>(cu, LDR, m0 - a0 + 16 * et, i, g);
      bacc[et] = F::mma(pa[et], ones, bacc[et]);
    }
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) {
        const Raw<T, 8> pb = lds_cols<T>(cu, LDR, na + n0 + 32 * cb + 16 * ct, i, g);
#pragma unroll
        for (int et = 0; et < 2; ++et) acc[et][2 * cb + ct] = F::mma(pa[et], pb, acc[et][2 * cb + ct]);
      }
  };
  T* const st0 = stage;
  T* const st1 = stage + 32 * LDR;
  if constexpr (SP <= 2) {
    Held ha, hb;
    if (p0 < p1) {
      load_job(ha, p0);
      store_job(ha, st0);
    }
    // a job past the group's rows loads nothing
    load_job(ha, p0 + 32);
    load_job(hb, p0 + 64);
    __syncthreads();
    // jobs base (in st0), base + 32 (set a), base + 64 (set b)
    for (int32_t base = p0; base < p1; base += 64) {
      sum_job(st0);
      if (base + 32 < p1) store_job(ha, st1);
      load_job(ha, base + 96);
      __syncthreads();
      if (base + 32 >= p1) break;
      sum_job(st1);
      if (base + 64 < p1) store_job(hb, st0);
      load_job(hb, base + 128);
      __syncthreads();
    }
  } else {
    // one job in flight
    Held ha;
    int buf = 0;
    if (p0 < p1) {
      load_job(ha, p0);
      store_job(ha, st0);
    }
    __syncthreads();
    for (int32_t base = p0; base < p1; base += 32) {
      const bool more = base + 32 < p1;
      if (more) load_job(ha, base + 32);
      sum_job(buf ? st1 : st0);
      if (more) store_job(ha, buf ? st0 : st1);
      buf ^= 1;
      __syncthreads();
    }
  }
  if (!active) return;
  // tile (et, ct): lane (c, g) component j is gradient entry
  // [m0 + 16 et + 4 g + j][n0 + 16 ct + c] of this kind's block; the bias tile
  // holds the row sums
  const size_t total = (size_t)4 * C * C + 4 * (size_t)C;
  float* part = wa.part + (size_t)grp * total;
  float* dw = kind == 3 ? part + (size_t)3 * C * C : part + (size_t)kind * C * C;
  float* db = kind == 3 ? part + (size_t)4 * C * C + 3 * C : part + (size_t)4 * C * C + (size_t)kind * C;
#pragma unroll
  for (int et = 0; et < 2; ++et) {
#pragma unroll
    for (int ct = 0; ct < 2 * NCB; ++ct)
#pragma unroll
      for (int j = 0; j < 4; ++j) dw[(size_t)(m0 + 16 * et + 4 * g + j) * C + n0 + 16 * ct + i] = acc[et][ct][j];
    if (chunk == 0 && i == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) db[m0 + 16 * et + 4 * g + j] = bacc[et][j];
    }
  }
}

// Sum of the groups' partials in group order: dW_qkv, dW_o, db_qkv, db_o (fp32).
__global__ __launch_bounds__(256) void k_wgrad_reduce(const float* __restrict__ part, int32_t groups,
                                                      int32_t C, float* __restrict__ dw_qkv,
                                                      float* __restrict__ dw_o,
                                                      float* __restrict__ db_qkv,
                                                      float* __restrict__ db_o) {
  const size_t total = (size_t)4 * C * C + 4 * (size_t)C;
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (size_t)gridDim.x * blockDim.x) {
    // 32 loads in flight, added in group order (groups past the last are
    // neither loaded nor added)
    constexpr int kBatch = 32;
    float s = 0.f;
    for (int32_t gi = 0; gi < groups; gi += kBatch) {
      float v[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) v[u] = gi + u < groups ? part[(size_t)(gi + u) * total + e] : 0.f;
#pragma unroll
      for (int u = 0; u < kBatch; ++u)
        if (gi + u < groups) s += v[u];
    }
    const size_t cc = (size_t)C * C;
    if (e < 3 * cc) dw_qkv[e] = s;
    else if (e < 4 * cc) dw_o[e - 3 * cc] = s;
    else if (e < 4 * cc + 3 * (size_t)C) { if (db_qkv) db_qkv[e - 4 * cc] = s; }
    else if (db_o) db_o[e - 4 * cc - 3 * (size_t)C] = s;
  }
}

// ------------------------------------------------------------ host side
// Workspace: W_qkv^T [C][3C], W_o^T [C][C] (dtype); q, k, v, do, dq, dk, dv
// [n][C] (dtype); the weight-gradient partials [groups][4 C^2 + 4 C] (fp32), with
// one group per 256 rows, the partials held within 32 MiB.
static int32_t wgrad_groups(int64_t n, int32_t C) {
  const int64_t per = ((int64_t)4 * C * C + 4 * (int64_t)C) * 4;
  int64_t g = (n + 255) / 256;
  const int64_t cap = ((int64_t)32 << 20) / per;
  if (g > cap) g = cap;
  if (g < 1) g = 1;
  return (int32_t)g;
}

struct ProjBwdLayout {
  size_t wt_qkv, wt_o, mask, act, act_stride, part, total;
  int32_t groups;
};

static ProjBwdLayout proj_bwd_layout(int64_t n, int32_t C) {
  ProjBwdLayout L;
  size_t off = 0;
  L.wt_qkv = off;
  off = align_up(off + (size_t)3 * C * C * 2, 256);
  L.wt_o = off;
  off = align_up(off + (size_t)C * C * 2, 256);
  L.mask = off;
  off = align_up(off + (size_t)n, 256);
  L.act = off;
  L.act_stride = align_up((size_t)n * C * 2, 256);
  off += 7 * L.act_stride;
  L.groups = wgrad_groups(n, C);
  L.part = off;
  off = align_up(off + (size_t)L.groups * ((size_t)4 * C * C + 4 * (size_t)C) * 4, 256);
  L.total = off;
  return L;
}

size_t projected_backward_workspace_bytes(int64_t n, int32_t C) { return proj_bwd_layout(n, C).total; }

hipError_t launch_backward(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                           int phi, float eps, const void* q, const void* k, const void* v,
                           const void* dout, void* dq, void* dk, void* dv, hipStream_t stream);

template <typename T>
static hipError_t rows_gemm(RowGemmArgs ga, hipStream_t stream) {
  // sub-blocks of 128 output columns when they stay inside one output segment and
  // 128 weight rows fit in LDS, else 64; a workgroup holds the most columns that
  // fit in 150 KB of LDS and divide N
  constexpr size_t kLdsCap = 150 * 1024;
  const auto lds_of = [&](int nb) { return (size_t)nb * (ga.K + 8) * 2 + (size_t)nb * 4; };
  const bool wide = ga.C % 128 == 0 && lds_of(128) <= kLdsCap;
  const int sb = wide ? 128 : 64;
  int nb = sb;
  for (int m = ga.N / sb; m >= 1; --m)
    if (ga.N % (m * sb) == 0 && lds_of(m * sb) <= kLdsCap) {
      nb = m * sb;
      break;
    }
  if (lds_of(nb) > kLdsCap) return hipErrorInvalidValue;
  ga.NB = nb;
  const size_t lds = lds_of(nb);
  const int cols = ga.N / nb;
  const bool small_k = ga.K <= 32 * 4;
  // at most one workgroup per CU, each walking many tiles with its staged
  // weights: row ranges a multiple of 8 (see the kernel), and no more
  // workgroups than CUs, since a workgroup that waits for a free CU would start
  // its fixed share of the tiles a whole launch late
  const int64_t tiles = ((int64_t)ga.n + 16 * (kRowGemmThreads / 64) - 1) / (16 * (kRowGemmThreads / 64));
  int64_t gx;
  if (cols == 1) {
    gx = tiles < 256 ? tiles : 256;   // one column block: any number of row ranges
    if (gx < 1) gx = 1;
  } else {
    gx = 256 / cols / 8 * 8;
    if (gx > tiles) gx = (tiles + 7) / 8 * 8;
    if (gx < 8) gx = 8;
  }
  // the input held in registers for K <= 128 or K <= 384, else streamed 128
  // channels a step (K = 3C with C = 256; 128 weight rows of such K exceed the
  // LDS cap, so a streamed product is never wide)
  const bool streamed = ga.K > 32 * 12;
  if (streamed && (wide || ga.C > 256 || ga.C % 128 != 0)) return hipErrorInvalidValue;
  void (*kern)(RowGemmArgs) =
      streamed ? &k_rows_gemm<T, 4, 0>
      : wide ? (small_k ? &k_rows_gemm<T, 8, 4> : &k_rows_gemm<T, 8, 12>)
             : (small_k ? &k_rows_gemm<T, 4, 4> : &k_rows_gemm<T, 4, 12>);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024 - 1024);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)(gx * cols)), dim3(kRowGemmThreads), lds, stream, ga);
  return hipGetLastError();
}

template <typename T>
static hipError_t projected_backward_t(const void* plan, int32_t n, int32_t W, int dtype, int32_t H,
                                       int32_t d, int phi, float eps, const void* x,
                                       const void* wqkv, const void* bqkv, const void* wo,
                                       const void* o, const void* dy, void* dx, float* dw_qkv,
                                       float* db_qkv, float* dw_o, float* db_o, const void* qkv,
                                       void* workspace, hipStream_t stream) {
  const int32_t C = H * d;
  const PlanLayout lay = plan_layout(n, W);
  const char* pb = static_cast<const char*>(plan);
  const PlanHeader* hdr = reinterpret_cast<const PlanHeader*>(pb + lay.header);
  const int32_t* offs = reinterpret_cast<const int32_t*>(pb + lay.offsets);
  const int32_t* perm = reinterpret_cast<const int32_t*>(pb + lay.perm);
  const ProjBwdLayout L = proj_bwd_layout(n, C);
  char* ws = static_cast<char*>(workspace);
  T* wt_qkv = reinterpret_cast<T*>(ws + L.wt_qkv);
  T* wt_o = reinterpret_cast<T*>(ws + L.wt_o);
  T* act[7];
  for (int m = 0; m < 7; ++m) act[m] = reinterpret_cast<T*>(ws + L.act + m * L.act_stride);
  T *dov = act[3], *dq = act[4], *dk = act[5], *dv = act[6];
  // q, k, v: as the forward saved them ([3][n][C]), else recomputed into the
  // workspace below
  const T* saved = static_cast<const T*>(qkv);
  const size_t nC = (size_t)n * C;
  const T* q = saved ? saved : act[0];
  const T* k = saved ? saved + nC : act[1];
  const T* v = saved ? saved + 2 * nC : act[2];
  float* part = reinterpret_cast<float*>(ws + L.part);
  uint8_t* mask = reinterpret_cast<uint8_t*>(ws + L.mask);
  hipError_t e;
  // the weights as rows of the products below (W_qkv^T for dx, W_o^T for do),
  // and which rows lie in a window
  PrepArgs pa{};
  pa.wqkv = wqkv;
  pa.wt_qkv = wt_qkv;
  pa.wo = wo;
  pa.wt_o = wt_o;
  pa.hdr = hdr;
  pa.perm = perm;
  pa.nvalid = offs + W;
  pa.mask = mask;
  pa.C = C;
  pa.n = n;
  pa.W = W;
  pa.mask_blocks = (int32_t)std::min<int64_t>(1024, std::max<int64_t>(1, ((int64_t)n + 255) / 256));
  const int32_t tiles = (C / 32) * (3 * C / 32) + (C / 32) * (C / 32);
  hipLaunchKernelGGL((k_prep<T>), dim3((unsigned)(tiles + pa.mask_blocks)), dim3(256), 0, stream, pa);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // q | k | v = x W_qkv^T + b_qkv
  RowGemmArgs ga{};
  ga.hdr = hdr;
  ga.mask = mask;
  ga.C = C;
  ga.n = n;
  ga.W = W;
  ga.a[0] = x;
  ga.out[0] = act[0];
  ga.out[1] = act[1];
  ga.out[2] = act[2];
  ga.w = wqkv;
  ga.bias = bqkv;
  ga.K = C;
  ga.N = 3 * C;
  if (!saved && (e = rows_gemm<T>(ga, stream)) != hipSuccess) return e;
  // do = dy W_o
  ga.a[0] = dy;
  ga.out[0] = dov;
  ga.w = wt_o;
  ga.bias = nullptr;
  ga.N = C;
  if ((e = rows_gemm<T>(ga, stream)) != hipSuccess) return e;
  // dq, dk, dv
  if ((e = launch_backward(plan, n, W, dtype, H, d, phi, eps, q, k, v, dov, dq, dk, dv, stream)) != hipSuccess)
    return e;
  // dx = [dq | dk | dv] W_qkv, zero for rows in no window
  ga.a[0] = dq;
  ga.a[1] = dk;
  ga.a[2] = dv;
  ga.out[0] = dx;
  ga.w = wt_qkv;
  ga.K = 3 * C;
  ga.N = C;
  if ((e = rows_gemm<T>(ga, stream)) != hipSuccess) return e;
  // weight and bias gradients: partials per row group, then their ordered sum
  WgradArgs wa{};
  wa.mats[0] = dq;
  wa.mats[1] = dk;
  wa.mats[2] = dv;
  wa.mats[3] = x;
  wa.mats[4] = dy;
  wa.mats[5] = o;
  wa.hdr = hdr;
  wa.mask = mask;
  wa.part = part;
  wa.C = C;
  wa.n = n;
  wa.W = W;
  wa.groups = L.groups;
  const int units = (C / 32) * (C / kWgradChunk);
  const int wnt = wgrad_threads(C);
  wa.wgs_per_kind = (units + wnt / 64 - 1) / (wnt / 64);
  const size_t wlds = (size_t)2 * 32 * (wgrad_a_cols(C, wnt) + C + 8) * 2;
  const void* wk = C == 256 ? reinterpret_cast<const void*>(&k_wgrad<T, 2, 1024>)
                  : C == 128 ? reinterpret_cast<const void*>(&k_wgrad<T, 2, 512>)
                             : reinterpret_cast<const void*>(&k_wgrad<T, 1, 512>);
  if ((e = hipFuncSetAttribute(wk, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024 - 1024)) != hipSuccess)
    return e;
  const dim3 wg((unsigned)(((int64_t)L.groups + 7) / 8 * 8 * 4 * wa.wgs_per_kind));
  if (C == 256) hipLaunchKernelGGL((k_wgrad<T, 2, 1024>), wg, dim3(1024), wlds, stream, wa);
  else if (C == 128) hipLaunchKernelGGL((k_wgrad<T, 2, 512>), wg, dim3(512), wlds, stream, wa);
  else hipLaunchKernelGGL((k_wgrad<T, 1, 512>), wg, dim3(512), wlds, stream, wa);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int64_t total = (int64_t)4 * C * C + 4 * (int64_t)C;
  hipLaunchKernelGGL(k_wgrad_reduce, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream,
                     static_cast<const float*>(part), L.groups, C, dw_qkv, dw_o, db_qkv, db_o);
  return hipGetLastError();
}

// dtype: 1 f16, 2 bf16; C = H d in {64, 128, 256}; phi: 0 elu + 1, 1 ReLU
hipError_t launch_backward_projected(const void* plan, int32_t n, int32_t W, int dtype, int32_t H,
                                     int32_t d, int phi, float eps, const void* x, const void* wqkv,
                                     const void* bqkv, const void* wo, const void* o, const void* dy,
                                     void* dx, float* dw_qkv, float* db_qkv, float* dw_o,
                                     float* db_o, const void* qkv, void* workspace, hipStream_t stream) {
  if (dtype == 1)
    return projected_backward_t<_Float16>(plan, n, W, dtype, H, d, phi, eps, x, wqkv, bqkv, wo, o, dy, dx,
                                          dw_qkv, db_qkv, dw_o, db_o, qkv, workspace, stream);
  return projected_backward_t<bf16_t>(plan, n, W, dtype, H, d, phi, eps, x, wqkv, bqkv, wo, o, dy, dx,
                                      dw_qkv, db_qkv, dw_o, db_o, qkv, workspace, stream);
}

}  // namespace sla

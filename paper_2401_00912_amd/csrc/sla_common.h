// Shared definitions of the SLA library: plan layout, storage-type traits and
// the CDNA4 (gfx950) matrix-core helpers.  Device code in this library is written
// for 64-lane wavefronts only.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <type_traits>

namespace sla {

// ----------------------------------------------------------------------------
// Plan: one caller-owned device buffer holding everything the attention kernels
// need (the window-sorted view of the rows and the chunk table) plus the
// builder's scratch.  Section offsets are a pure function of (n, num_windows).
// ----------------------------------------------------------------------------
constexpr int32_t kPlanMagic = 0x534c4132;   // "SLA2"
constexpr int32_t kMaxWindows = 16384;       // LDS-resident window tables
constexpr int32_t kMinChunkRows = 32;
constexpr int32_t kMaxChunkRows = 64;        // rows one wavefront holds in registers
constexpr int32_t kDefaultChunkRows = 64;

struct PlanHeader {
  int32_t magic;
  int32_t n;            // rows
  int32_t num_windows;  // window slots W
  int32_t chunk_rows;   // L
  int32_t n_chunks;     // chunks of whole windows (written by the builder)
  int32_t csr;          // 1: rows already window-sorted (identity permutation)
  int32_t invalid;      // out-of-range ids / CSR violations seen by the builder
  int32_t n_long;       // windows of more than L rows (written by the builder)
  int32_t n_long4;      // of which more than 2L rows (split four ways; listed first)
  int32_t pad[7];
};
static_assert(sizeof(PlanHeader) == 64, "header is 64 bytes");

// One chunk: rows [row_begin, row_end) of the window-sorted sequence, made of
// windows [win_begin, win_end) (whole windows of at most L rows; empty windows
// may be included).
struct Chunk {
  int32_t row_begin, row_end, win_begin, win_end;
};

// One window of more than L rows: its rows are split among the waves of a
// workgroup (four ways above 2L rows, else two ways), which add their partial
// states.
struct LongWin {
  int32_t window, row_begin, row_end, pad;
};

struct PlanLayout {
  size_t header, totals, perm, offsets, chunks, longs, counts, sorted, total;
  int32_t max_chunks;   // capacity of the chunk table
  int32_t max_long;     // capacity of the long-window table
  int32_t n_blocks;     // builder blocks
  int32_t block_elems;  // rows per builder block
  int32_t counts_ld;    // row stride (ints) of the builder's prefix matrix
};

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Rows per builder block: 1024 x 2^k, k <= 3, the smallest that keeps the
// builder's prefix matrix (one row of num_windows + 1 ints per block) within 2^21
// entries and the block count within kBuilderMaxBlocks, where possible.
constexpr int32_t kBuilderMinBlockElems = 1024;
constexpr int32_t kBuilderMaxBlockElems = 8192;
constexpr int32_t kBuilderMaxBlocks = 8192;
constexpr int64_t kBuilderMaxRows = (int64_t)kBuilderMaxBlockElems * kBuilderMaxBlocks;
__host__ __device__ inline int32_t builder_block_elems(int64_t n, int32_t num_windows) {
  int64_t e = kBuilderMinBlockElems;
  while (e < kBuilderMaxBlockElems &&
         (((n + e - 1) / e) * ((int64_t)num_windows + 1) > (int64_t)1 << 21 ||
          (n + e - 1) / e > kBuilderMaxBlocks))
    e *= 2;
  return (int32_t)e;
}

__host__ __device__ inline PlanLayout plan_layout(int64_t n, int32_t num_windows) {
  PlanLayout L;
  const int64_t W = num_windows;
  L.block_elems = builder_block_elems(n, num_windows);
  L.n_blocks = (int32_t)((n + L.block_elems - 1) / L.block_elems);
  L.counts_ld = (int32_t)align_up((size_t)W + 1, 4);
  // Every chunk holds at least one non-empty window, so min(W, n) bounds the
  // count; a long window has more than kMinChunkRows rows.
  L.max_chunks = (int32_t)(W < n ? W : n);
  const int64_t nl = n / (kMinChunkRows + 1);
  L.max_long = (int32_t)(W < nl ? W : nl);
  size_t off = 0;
  L.header = off;
  off += 256;
  // window totals of the build in progress: at a fixed place for every (n, W), and
  // all zero between builds (the builder clears what it added)
  L.totals = off;
  off = align_up(off + ((size_t)kMaxWindows + 1) * 4, 256);
  L.perm = off;
  off = align_up(off + (size_t)n * 4, 256);
  L.offsets = off;
  off = align_up(off + (size_t)(W + 1) * 4, 256);
  L.chunks = off;
  off = align_up(off + (size_t)(L.max_chunks > 0 ? L.max_chunks : 1) * sizeof(Chunk), 256);
  L.longs = off;
  off = align_up(off + (size_t)(L.max_long > 0 ? L.max_long : 1) * sizeof(LongWin), 256);
  // builder scratch: per block, the exclusive prefix of its window counts; the
  // rows of every block sorted by window
  L.counts = off;
  off = align_up(off + (size_t)L.n_blocks * (size_t)L.counts_ld * 4, 256);
  L.sorted = off;
  off = align_up(off + (size_t)n * 4, 256);
  L.total = off;
  return L;
}

// ----------------------------------------------------------------------------
// Storage types.  Values are widened to fp32 in registers; matrix-core operands
// are narrowed back to the storage type (fp32 stays fp32).
// ----------------------------------------------------------------------------
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

struct bf16_t {
  uint16_t bits;
};

template <typename T>
struct Ty;
template <> struct Ty<float> { static constexpr bool kNarrow = false; };
template <> struct Ty<_Float16> { static constexpr bool kNarrow = true; };
template <> struct Ty<bf16_t> { static constexpr bool kNarrow = true; };

// ----------------------------------------------------------------------------
// Raw fragments: KS consecutive elements of one row kept in their storage format
// (16-bit types as packed u16 vectors, fp32 as floats), loaded and stored with
// one vector access, fed to the matrix cores without conversion.
// ----------------------------------------------------------------------------
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

template <typename T, int KS>
struct RawOf;
template <> struct RawOf<_Float16, 8> { using type = u16x8; };
template <> struct RawOf<_Float16, 4> { using type = u16x4; };
template <> struct RawOf<bf16_t, 8> { using type = u16x8; };
template <> struct RawOf<bf16_t, 4> { using type = u16x4; };
template <> struct RawOf<float, 8> { using type = f32x8; };
template <> struct RawOf<float, 4> { using type = floatx4; };
template <typename T, int KS>
using Raw = typename RawOf<T, KS>::type;

template <typename T>
__device__ __forceinline__ float u16_to_f32(unsigned short u);
template <>
__device__ __forceinline__ float u16_to_f32<_Float16>(unsigned short u) {
  return (float)__builtin_bit_cast(_Float16, u);
}
template <>
__device__ __forceinline__ float u16_to_f32<bf16_t>(unsigned short u) {
  return __uint_as_float((uint32_t)u << 16);
}
template <typename T>
__device__ __forceinline__ unsigned short f32_to_u16(float x);
template <>
__device__ __forceinline__ unsigned short f32_to_u16<_Float16>(float x) {
  return __builtin_bit_cast(unsigned short, (_Float16)x);
}
template <>
__device__ __forceinline__ unsigned short f32_to_u16<bf16_t>(float x) {
  return __builtin_bit_cast(unsigned short, (__bf16)x);
}

template <typename T, int KS>
struct Frag {
  using R = Raw<T, KS>;
  __device__ static R zero() {
    R r;
#pragma unroll
    for (int k = 0; k < KS; ++k) r[k] = 0;
    return r;
  }
  __device__ static void to_f32(R r, float (&x)[KS]) {
#pragma unroll
    for (int k = 0; k < KS; ++k) {
      if constexpr (Ty<T>::kNarrow) x[k] = u16_to_f32<T>(r[k]);
      else x[k] = r[k];
    }
  }
  // round to nearest even into the storage type
  __device__ static R from_f32(const float (&x)[KS]) {
    R r;
#pragma unroll
    for (int k = 0; k < KS; ++k) {
      if constexpr (Ty<T>::kNarrow) r[k] = f32_to_u16<T>(x[k]);
      else r[k] = x[k];
    }
    return r;
  }
  // One 16x16 result tile contracted over the 4 lane groups x KS register slots:
  // lane l = 16 g + i supplies A[i][slot(g, r)] and B[slot(g, r)][i] for r < KS and
  // lane 16 g + n receives D[4 g + j][n] in component j.  Which contraction index
  // a slot stands for is the caller's choice: the hardware pairs the slots of A
  // and B identically.  KS = 8: one 16x16x32 f16/bf16 MFMA (eight 16x16x4 f32);
  // KS = 4: one 16x16x16 f16/bf16 MFMA (four 16x16x4 f32).
  __device__ static floatx4 mma(R a, R b, floatx4 c) {
    if constexpr (std::is_same<T, float>::value) {
#pragma unroll
      for (int k = 0; k < KS; ++k) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[k], b[k], c, 0, 0, 0);
      return c;
    } else if constexpr (std::is_same<T, _Float16>::value) {
      if constexpr (KS == 8)
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, a),
                                                      __builtin_bit_cast(half8_t, b), c, 0, 0, 0);
      else
        return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(half4_t, a),
                                                     __builtin_bit_cast(half4_t, b), c, 0, 0, 0);
    } else {
      if constexpr (KS == 8)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                       __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
      else
        return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(short4_t, a),
                                                         __builtin_bit_cast(short4_t, b), c, 0, 0, 0);
    }
  }
};

// Columns c0 .. c0 + 15 of 32 consecutive 16-bit rows in LDS (`rows` points at
// the first, row stride `ld` elements, 8-byte aligned rows) as the operand of a
// contraction over the rows: slot r of lane (i, g) holds row 8g + r, column
// c0 + i.  Two LDS transpose loads (ds_read_b64_tr_b16): in each group of 16
// lanes, lane i addresses row 8g + 4h + i / 4 at columns c0 + 4 (i % 4) .. + 3
// and receives column c0 + i of rows 8g + 4h .. 8g + 4h + 3 (the lane layout
// measured by an in-bounds probe of the instruction).
template <typename T>
__device__ __forceinline__ Raw<T, 8> lds_cols(const unsigned short* rows, int ld, int c0, int i, int g) {
  typedef short v4s __attribute__((ext_vector_type(4)));
  const unsigned short* p = rows + (8 * g + (i >> 2)) * ld + c0 + 4 * (i & 3);
  const v4s a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)(p));
  const v4s b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)(p + 4 * ld));
  Raw<T, 8> r;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    r[j] = (unsigned short)a[j];
    r[4 + j] = (unsigned short)b[j];
  }
  return r;
}

// 8-slot operand from two 4-row result tiles (rows 4g..4g+3 of two sub-tiles).
template <typename T>
__device__ __forceinline__ Raw<T, 8> pack_rows(floatx4 lo, floatx4 hi) {
  float x[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return Frag<T, 8>::from_f32(x);
}

// ----------------------------------------------------------------------------
// Wave helpers
// ----------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }

}  // namespace sla

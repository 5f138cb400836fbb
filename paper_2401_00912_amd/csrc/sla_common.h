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
constexpr int32_t kPlanMagic = 0x534c4131;   // "SLA1"
constexpr int32_t kMaxWindows = 16384;       // LDS-resident window tables
constexpr int32_t kMinChunkRows = 32;
constexpr int32_t kMaxChunkRows = 4096;
constexpr int32_t kDefaultChunkRows = 128;

struct PlanHeader {
  int32_t magic;
  int32_t n;            // rows
  int32_t num_windows;  // window slots W
  int32_t chunk_rows;   // L
  int32_t n_chunks;     // written by the builder
  int32_t csr;          // 1: rows already window-sorted (identity permutation)
  int32_t invalid;      // out-of-range ids / CSR violations seen by the builder
  // Work counters of the attention kernels (zeroed by the builder; every launch
  // hands out work items from claim[k] and the last workgroup to finish puts both
  // counters of its kernel back to zero): k = 0 forward, 1 backward.
  int32_t claim[2];
  int32_t done[2];
  int32_t pad[5];
};
static_assert(sizeof(PlanHeader) == 64, "header is 64 bytes");

// One chunk: rows [row_begin, row_end) of the window-sorted sequence, made of
// windows [win_begin, win_end) (whole windows; empty windows may be included).
struct Chunk {
  int32_t row_begin, row_end, win_begin, win_end;
};

struct PlanLayout {
  size_t header, perm, offsets, chunks, counts, total;
  int32_t max_chunks;   // capacity of the chunk table
  int32_t n_blocks;     // builder blocks
  int32_t block_elems;  // rows per builder block
};

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Rows per builder block: a power of two >= 1024 chosen so that there are at most
// 64 blocks (the count matrix then has at most 64 * (W + 1) entries).
__host__ __device__ inline int32_t builder_block_elems(int64_t n) {
  int64_t e = 1024;
  while (e * 64 < n) e *= 2;
  return (int32_t)e;
}

__host__ __device__ inline PlanLayout plan_layout(int64_t n, int32_t num_windows) {
  PlanLayout L;
  const int64_t W = num_windows;
  L.block_elems = builder_block_elems(n);
  L.n_blocks = (int32_t)((n + L.block_elems - 1) / L.block_elems);
  // Every chunk holds at least one non-empty window, so W bounds the count.
  L.max_chunks = (int32_t)(W < n ? W : n);
  size_t off = 0;
  L.header = off;
  off += 256;
  L.perm = off;
  off = align_up(off + (size_t)n * 4, 256);
  L.offsets = off;
  off = align_up(off + (size_t)(W + 1) * 4, 256);
  L.chunks = off;
  off = align_up(off + (size_t)(L.max_chunks > 0 ? L.max_chunks : 1) * sizeof(Chunk), 256);
  L.counts = off;
  off = align_up(off + (size_t)L.n_blocks * (size_t)(W + 1) * 4, 256);
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

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round-to-nearest-even fp32 -> bf16 (finite inputs; NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T>
struct Ty;

template <>
struct Ty<float> {
  static constexpr bool kNarrow = false;
  __device__ static float to_f32(float x) { return x; }
  __device__ static float round(float x) { return x; }  // value as the MFMA sees it
};

template <>
struct Ty<_Float16> {
  static constexpr bool kNarrow = true;
  __device__ static float to_f32(_Float16 x) { return (float)x; }
  __device__ static float round(float x) { return (float)(_Float16)x; }
};

template <>
struct Ty<bf16_t> {
  static constexpr bool kNarrow = true;
  __device__ static float to_f32(bf16_t x) { return bf16_to_f32(x.bits); }
  __device__ static float round(float x) { return bf16_to_f32(f32_to_bf16(x)); }
};

// ----------------------------------------------------------------------------
// Fragment I/O: KS consecutive elements of one row (KS = 4 or 8).
// ----------------------------------------------------------------------------
template <typename T, int KS>
__device__ __forceinline__ void load_frag(const T* p, float (&x)[KS]);

template <typename T, int KS>
__device__ __forceinline__ void store_frag(T* p, const float (&x)[KS]);

template <>
__device__ __forceinline__ void load_frag<float, 8>(const float* p, float (&x)[8]) {
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
template <>
__device__ __forceinline__ void load_frag<float, 4>(const float* p, float (&x)[4]) {
  float4 a = *reinterpret_cast<const float4*>(p);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
}
template <>
__device__ __forceinline__ void store_frag<float, 8>(float* p, const float (&x)[8]) {
  *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(x[4], x[5], x[6], x[7]);
}
template <>
__device__ __forceinline__ void store_frag<float, 4>(float* p, const float (&x)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
}

template <>
__device__ __forceinline__ void load_frag<_Float16, 8>(const _Float16* p, float (&x)[8]) {
  half8_t h = *reinterpret_cast<const half8_t*>(p);
#pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = (float)h[i];
}
template <>
__device__ __forceinline__ void load_frag<_Float16, 4>(const _Float16* p, float (&x)[4]) {
  half4_t h = *reinterpret_cast<const half4_t*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) x[i] = (float)h[i];
}
template <>
__device__ __forceinline__ void store_frag<_Float16, 8>(_Float16* p, const float (&x)[8]) {
  half8_t h;
#pragma unroll
  for (int i = 0; i < 8; ++i) h[i] = (_Float16)x[i];
  *reinterpret_cast<half8_t*>(p) = h;
}
template <>
__device__ __forceinline__ void store_frag<_Float16, 4>(_Float16* p, const float (&x)[4]) {
  half4_t h;
#pragma unroll
  for (int i = 0; i < 4; ++i) h[i] = (_Float16)x[i];
  *reinterpret_cast<half4_t*>(p) = h;
}

template <>
__device__ __forceinline__ void load_frag<bf16_t, 8>(const bf16_t* p, float (&x)[8]) {
  uint4 u = *reinterpret_cast<const uint4*>(p);
  uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
template <>
__device__ __forceinline__ void load_frag<bf16_t, 4>(const bf16_t* p, float (&x)[4]) {
  uint2 u = *reinterpret_cast<const uint2*>(p);
  x[0] = __uint_as_float(u.x << 16);
  x[1] = __uint_as_float(u.x & 0xffff0000u);
  x[2] = __uint_as_float(u.y << 16);
  x[3] = __uint_as_float(u.y & 0xffff0000u);
}
template <>
__device__ __forceinline__ void store_frag<bf16_t, 8>(bf16_t* p, const float (&x)[8]) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = (uint32_t)f32_to_bf16(x[2 * i]) | ((uint32_t)f32_to_bf16(x[2 * i + 1]) << 16);
  *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
}
template <>
__device__ __forceinline__ void store_frag<bf16_t, 4>(bf16_t* p, const float (&x)[4]) {
  uint32_t w0 = (uint32_t)f32_to_bf16(x[0]) | ((uint32_t)f32_to_bf16(x[1]) << 16);
  uint32_t w1 = (uint32_t)f32_to_bf16(x[2]) | ((uint32_t)f32_to_bf16(x[3]) << 16);
  *reinterpret_cast<uint2*>(p) = make_uint2(w0, w1);
}

// ----------------------------------------------------------------------------
// Matrix-core contraction over the 4 lane groups x KS register slots of a wave.
//
// For a 16x16 output tile, lane l = 16 g + i supplies A[i][slot(g, r)] and
// B[slot(g, r)][i] for r < KS; the result tile is returned in the standard
// layout: lane 16 g + n holds D[4 g + j][n] in component j.  Which contraction
// index a slot (g, r) stands for is the caller's choice: A and B only have to
// agree, because the hardware pairs A's and B's slots identically.
//   KS = 8: one v_mfma_f32_16x16x32_{f16,bf16}, or eight v_mfma_f32_16x16x4_f32;
//   KS = 4: one v_mfma_f32_16x16x16{f16,bf16_1k}, or four v_mfma_f32_16x16x4_f32.
// ----------------------------------------------------------------------------
template <typename T, int KS>
struct Mma;

template <>
struct Mma<float, 8> {
  __device__ static floatx4 run(const float (&a)[8], const float (&b)[8], floatx4 c) {
#pragma unroll
    for (int r = 0; r < 8; ++r) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[r], b[r], c, 0, 0, 0);
    return c;
  }
};
template <>
struct Mma<float, 4> {
  __device__ static floatx4 run(const float (&a)[4], const float (&b)[4], floatx4 c) {
#pragma unroll
    for (int r = 0; r < 4; ++r) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[r], b[r], c, 0, 0, 0);
    return c;
  }
};
template <>
struct Mma<_Float16, 8> {
  __device__ static floatx4 run(const float (&a)[8], const float (&b)[8], floatx4 c) {
    half8_t ha, hb;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      ha[r] = (_Float16)a[r];
      hb[r] = (_Float16)b[r];
    }
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(ha, hb, c, 0, 0, 0);
  }
};
template <>
struct Mma<_Float16, 4> {
  __device__ static floatx4 run(const float (&a)[4], const float (&b)[4], floatx4 c) {
    half4_t ha, hb;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      ha[r] = (_Float16)a[r];
      hb[r] = (_Float16)b[r];
    }
    return __builtin_amdgcn_mfma_f32_16x16x16f16(ha, hb, c, 0, 0, 0);
  }
};
template <>
struct Mma<bf16_t, 8> {
  __device__ static floatx4 run(const float (&a)[8], const float (&b)[8], floatx4 c) {
    bf16x8_t ha, hb;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      ha[r] = __builtin_bit_cast(__bf16, f32_to_bf16(a[r]));
      hb[r] = __builtin_bit_cast(__bf16, f32_to_bf16(b[r]));
    }
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(ha, hb, c, 0, 0, 0);
  }
};
template <>
struct Mma<bf16_t, 4> {
  __device__ static floatx4 run(const float (&a)[4], const float (&b)[4], floatx4 c) {
    short4_t ha, hb;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      ha[r] = (short)f32_to_bf16(a[r]);
      hb[r] = (short)f32_to_bf16(b[r]);
    }
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ha, hb, c, 0, 0, 0);
  }
};

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
  __device__ static R load(const T* p) {
    if constexpr (Ty<T>::kNarrow) {
      return *reinterpret_cast<const R*>(p);
    } else if constexpr (KS == 8) {
      const float4 a = reinterpret_cast<const float4*>(p)[0];
      const float4 b = reinterpret_cast<const float4*>(p)[1];
      R r;
      r[0] = a.x; r[1] = a.y; r[2] = a.z; r[3] = a.w;
      r[4] = b.x; r[5] = b.y; r[6] = b.z; r[7] = b.w;
      return r;
    } else {
      return *reinterpret_cast<const R*>(p);
    }
  }
  __device__ static void store(T* p, R r) {
    if constexpr (Ty<T>::kNarrow) {
      *reinterpret_cast<R*>(p) = r;
    } else if constexpr (KS == 8) {
      reinterpret_cast<float4*>(p)[0] = make_float4(r[0], r[1], r[2], r[3]);
      reinterpret_cast<float4*>(p)[1] = make_float4(r[4], r[5], r[6], r[7]);
    } else {
      *reinterpret_cast<R*>(p) = r;
    }
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
  // one 16x16 tile contraction over the 4 x KS slots (see Mma above)
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

__device__ __forceinline__ float shfl_xor_f(float x, int m) { return __shfl_xor(x, m, 64); }
__device__ __forceinline__ float shfl_f(float x, int src) { return __shfl(x, src, 64); }

// Make LDS writes of this wave visible to the wave's other lanes.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x = fmaxf(x, shfl_xor_f(x, m));
  return x;
}

}  // namespace sla

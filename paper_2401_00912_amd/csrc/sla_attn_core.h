// Building blocks shared by the SLA attention kernels (sla_attn.hip) and the
// projection fused into them (sla_proj.hip): register layouts and fragments,
// the feature maps, the state contractions, work items and row gathers, and the
// host helpers that size and describe a launch.  The design notes are at the
// top of sla_attn.hip.
#pragma once
#include "sla_common.h"


namespace sla {

constexpr int kWaves = 4;       // waves (heads) per workgroup
constexpr int kSliceRows = 32;  // rows per job

constexpr float kLog2e = 1.4426950408889634f;

constexpr int kPhiElu1 = 0;  // phi(x) = elu(x) + 1
constexpr int kPhiRelu = 1;  // phi(x) = max(x, 0), phi'(0) = 0

// phi(x) = x + 1 for x > 0, exp(x) otherwise, and its derivative.  With 16-bit
// storage the result is rounded to 16 bits for the matrix cores, so the
// hardware exp2 (about 1 ulp of fp32) is ample; fp32 storage keeps expf.
template <typename T>
__device__ __forceinline__ float phi_f(float x) {
  if constexpr (Ty<T>::kNarrow) {
    return x > 0.f ? x + 1.f : __builtin_amdgcn_exp2f(x * kLog2e);
  } else {
    return x > 0.f ? x + 1.f : expf(x);
  }
}

template <typename T>
__device__ __forceinline__ float dphi_f(float x) {
  if constexpr (Ty<T>::kNarrow) {
    return x > 0.f ? 1.f : __builtin_amdgcn_exp2f(x * kLog2e);
  } else {
    return x > 0.f ? 1.f : expf(x);
  }
}

// 1 / x: the hardware reciprocal (1 ulp) for 16-bit storage, a correctly
// rounded division for fp32.
template <typename T>
__device__ __forceinline__ float recip(float x) {
  if constexpr (Ty<T>::kNarrow) {
    return __builtin_amdgcn_rcpf(x);
  } else {
    return 1.f / x;
  }
}

// Power of two p with x * p in [1, 2) (1 for x = 0 or non-finite x; at most
// 2^126, so that p and 1 / p stay finite, for x below the normal range).
// Exponent of x > 0 from its bits; -127 for a subnormal x, which both callers
// clamp to the same power of two as its true exponent.
__device__ __forceinline__ int exponent_of(float x) {
  return (int)((__float_as_uint(x) >> 23) & 0xffu) - 127;
}

__device__ __forceinline__ float pow2_scale_to_one(float x) {
  if (!(x > 0.f) || !(x < 3.0e38f)) return 1.f;
  return ldexpf(1.f, min(-exponent_of(x), 126));
}

// Power of two <= x (1 for x = 0 or non-finite x; at least 2^-126).
__device__ __forceinline__ float pow2_floor(float x) {
  if (!(x > 0.f) || !(x < 3.0e38f)) return 1.f;
  return ldexpf(1.f, max(exponent_of(x), -126));
}

// ---------------------------------------------------------- lane exchanges
// Sum over the 4 lane groups: x + x[l ^ 16], then + [l ^ 32] (VALU lane swaps).
__device__ __forceinline__ float sum_groups(float x) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Make this wave's LDS writes visible to its other lanes.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Max (MAX) or min over the wave, returned wave-uniform: DPP within each row of
// 16 lanes, then the four row results.
template <bool MAX>
__device__ __forceinline__ float wave_reduce(float x) {
  auto step = [&](int y) {
    x = MAX ? fmaxf(x, __int_as_float(y)) : fminf(x, __int_as_float(y));
  };
  step(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xf, 0xf, false));   // quad [1,0,3,2]
  step(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xf, 0xf, false));   // quad [2,3,0,1]
  step(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x141, 0xf, 0xf, false));  // row_half_mirror
  step(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x140, 0xf, 0xf, false));  // row_mirror
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return MAX ? fmaxf(fmaxf(r0, r1), fmaxf(r2, r3)) : fminf(fminf(r0, r1), fminf(r2, r3));
}

template <int D>
struct Geo {
  static constexpr int KS = D / 4;   // slots per lane group along the head dim
  static constexpr int NT = D / 16;  // 16-wide tiles along the head dim
  __device__ static int E(int g, int r) { return 16 * (r >> 2) + 4 * g + (r & 3); }
};

// ----------------------------------------------------------- row fragments
// Element `e` of a tensor: byte offsets fit in 32 bits (the host checks that
// every tensor is smaller than 4 GiB), so the address is a uniform base plus one
// 32-bit lane offset, which the memory instructions take as such.
template <typename T>
__device__ __forceinline__ T* elem_at(T* base, uint32_t e) {
  return reinterpret_cast<T*>(reinterpret_cast<char*>(base) + (uint64_t)(e * (uint32_t)sizeof(T)));
}
template <typename T>
__device__ __forceinline__ const T* elem_at(const T* base, uint32_t e) {
  return reinterpret_cast<const T*>(reinterpret_cast<const char*>(base) + (uint64_t)(e * (uint32_t)sizeof(T)));
}
// Element offset of head `col` of row o of a [n, H, d] tensor (row stride rs).
__device__ __forceinline__ uint32_t row_off(int32_t o, size_t rs, int col) {
  return (uint32_t)o * (uint32_t)rs + (uint32_t)col;
}


// A row fragment (KS elements of one head of one row, in slot order E) moves
// between registers and memory.  16-bit types with head_dim 32: each lane group
// g reads / writes the 8 contiguous elements 8g..8g+7 as one 16-byte access,
// and two lane swaps turn those into slot order: with P_g = elements 8g..8g+3
// and Q_g = 8g+4..8g+7, swapping lane rows 1<->0 and 3<->2 between P and Q, then
// lanes 32..63 of P with lanes 0..31 of Q, leaves elements 4g..4g+3 (slots
// 0..3) in P and 16+4g..16+4g+3 (slots 4..7) in Q.  Stores apply the inverse
// (the swaps in reverse order).  Other types and sizes read and write the NT
// pieces of 4 elements at 16t + 4g directly.  The swaps are cross-lane, so
// fetch/put run them unmasked and guard only the memory access.
template <typename T, int D>
struct RowIO {
  static constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  static constexpr bool kSwizzle = Ty<T>::kNarrow && D == 32;
  using R = Raw<T, KS>;
  __device__ static void swap16(uint32_t& x, uint32_t& y) {
    const auto r = __builtin_amdgcn_permlane16_swap(x, y, false, false);
    x = r[0];
    y = r[1];
  }
  __device__ static void swap32(uint32_t& x, uint32_t& y) {
    const auto r = __builtin_amdgcn_permlane32_swap(x, y, false, false);
    x = r[0];
    y = r[1];
  }
  // `off` is the element offset of the head's first element from `base` (see
  // elem_at: the lane's part is added in 32 bits, so the access is a uniform
  // base plus one 32-bit lane offset).  The load is unconditional (the caller
  // passes a valid row for rows past a job and masks them in the math):
  // merging a guarded load with a default would wait for the load right here.
  // The result is in memory order until arrange() puts it into slot order (kept
  // apart so that a prefetched fragment is not waited for at load time).
  __device__ static R fetch(const T* base, uint32_t off, int g) {
    if constexpr (kSwizzle) {
      return __builtin_bit_cast(R, *reinterpret_cast<const uint4*>(elem_at(base, off + 8 * g)));
    } else if constexpr (Ty<T>::kNarrow) {
      R r;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const u16x4 p = *reinterpret_cast<const u16x4*>(elem_at(base, off + 16 * t + 4 * g));
#pragma unroll
        for (int j = 0; j < 4; ++j) r[4 * t + j] = p[j];
      }
      return r;
    } else {
      R r;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const float4 p = *reinterpret_cast<const float4*>(elem_at(base, off + 16 * t + 4 * g));
        r[4 * t + 0] = p.x;
        r[4 * t + 1] = p.y;
        r[4 * t + 2] = p.z;
        r[4 * t + 3] = p.w;
      }
      return r;
    }
  }
  __device__ static void arrange(R& r) {
    if constexpr (kSwizzle) {
      uint4 w = __builtin_bit_cast(uint4, r);
      swap16(w.x, w.z);
      swap16(w.y, w.w);
      swap32(w.x, w.z);
      swap32(w.y, w.w);
      r = __builtin_bit_cast(R, w);
    }
  }
  __device__ static void put(T* base, uint32_t off, int g, R r, bool ok) {
    if constexpr (kSwizzle) {
      uint4 w = __builtin_bit_cast(uint4, r);
      swap32(w.x, w.z);
      swap32(w.y, w.w);
      swap16(w.x, w.z);
      swap16(w.y, w.w);
      if (ok) *reinterpret_cast<uint4*>(elem_at(base, off + 8 * g)) = w;
    } else if constexpr (Ty<T>::kNarrow) {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        u16x4 p;
#pragma unroll
        for (int j = 0; j < 4; ++j) p[j] = r[4 * t + j];
        if (ok) *reinterpret_cast<u16x4*>(elem_at(base, off + 16 * t + 4 * g)) = p;
      }
    } else {
#pragma unroll
      for (int t = 0; t < NT; ++t)
        if (ok)
          *reinterpret_cast<float4*>(elem_at(base, off + 16 * t + 4 * g)) =
              make_float4(r[4 * t], r[4 * t + 1], r[4 * t + 2], r[4 * t + 3]);
    }
  }
};

// Row head `col` of row o of a [n, H, d] tensor: byte offsets fit in 32 bits (the
// host checks that every tensor is smaller than 4 GiB), so the address is a
// uniform base plus one 32-bit lane offset.
template <typename T>
__device__ __forceinline__ const T* row_at(const T* base, int32_t o, size_t rs, int col) {
  const uint32_t off = ((uint32_t)o * (uint32_t)rs + (uint32_t)col) * (uint32_t)sizeof(T);
  return reinterpret_cast<const T*>(reinterpret_cast<const char*>(base) + off);
}
template <typename T>
__device__ __forceinline__ T* row_at(T* base, int32_t o, size_t rs, int col) {
  const uint32_t off = ((uint32_t)o * (uint32_t)rs + (uint32_t)col) * (uint32_t)sizeof(T);
  return reinterpret_cast<T*>(reinterpret_cast<char*>(base) + off);
}

struct KernelArgs {
  const PlanHeader* hdr;
  const int32_t* perm;
  const int32_t* offs;
  const Chunk* chunks;
  const LongWin* longs;
  int32_t max_chunks, max_long, n, W, H;
  float eps;  // added to the normaliser phi(q) . z
};

// ------------------------------------------------------------------ jobs
// The rows of one 32-row job: sub-tile s covers sorted rows r0 + 16 s + (l & 15);
// NM matrices (K,V / Q / Q,dout) as row fragments.
template <typename T, int KS, int NM>
struct Slice {
  Raw<T, KS> x[NM][2];
  int32_t o[2];  // original row of this lane's row in sub-tile s
  bool ok[2];    // row exists (inside the job and the plan)
};

// ------------------------------------------------------------ states
// A window state (or state gradient) as result tiles:
//   M[et][ct]  lane (c', g) component j = M[16 et + 4 g + j][16 ct + c']
//   V[et]      lane (*, g) component j  = v[16 et + 4 g + j]  (the extra column)
template <int D>
struct State {
  static constexpr int NT = Geo<D>::NT;
  floatx4 M[NT][NT];
  floatx4 V[NT];
  __device__ void clear() {
    const floatx4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int a = 0; a < NT; ++a) {
      V[a] = z;
#pragma unroll
      for (int b = 0; b < NT; ++b) M[a][b] = z;
    }
  }
  // largest |entry| of M and V over the wave
  __device__ float absmax() const {
    float mx = 0.f;
#pragma unroll
    for (int a = 0; a < NT; ++a)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        mx = fmaxf(mx, fabsf(V[a][j]));
#pragma unroll
        for (int b = 0; b < NT; ++b) mx = fmaxf(mx, fabsf(M[a][b][j]));
      }
    return wave_reduce<true>(mx);
  }
};

// Selection matrices of the transposes: slot (g, r) stands for head index E(g, r).
template <typename T, int D>
struct Sel {
  Raw<T, Geo<D>::KS> m[Geo<D>::NT];
  __device__ Sel(int i, int g) {
    constexpr int KS = Geo<D>::KS;
#pragma unroll
    for (int t = 0; t < Geo<D>::NT; ++t) {
      float x[KS];
#pragma unroll
      for (int r = 0; r < KS; ++r) x[r] = (Geo<D>::E(g, r) == 16 * t + i) ? 1.f : 0.f;
      m[t] = Frag<T, KS>::from_f32(x);
    }
  }
};

// phi of a fragment, rounded to the storage type; zero where !ok.  fp16 works on
// packed halves, elu + 1 as phi(x) = 2^(min(x, 0) log2 e) + max(x, 0), which
// equals the definition on both branches.
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

template <typename T, int KS, int PHI>
__device__ __forceinline__ Raw<T, KS> phi_frag(Raw<T, KS> x, bool ok) {
  if constexpr (PHI == kPhiRelu && std::is_same<T, _Float16>::value) {
    constexpr int NW = KS / 2;
    using W = uint32_t __attribute__((ext_vector_type(NW)));
    const W w = __builtin_bit_cast(W, x);
    W out;
    const half2_t zero = {0, 0};
#pragma unroll
    for (int k = 0; k < NW; ++k) {
      const half2_t p = __builtin_bit_cast(half2_t, (uint32_t)w[k]);
      out[k] = ok ? __builtin_bit_cast(uint32_t, __builtin_elementwise_max(p, zero)) : 0u;
    }
    return __builtin_bit_cast(Raw<T, KS>, out);
  } else if constexpr (PHI == kPhiRelu) {
    float f[KS];
    Frag<T, KS>::to_f32(x, f);
#pragma unroll
    for (int r = 0; r < KS; ++r) f[r] = ok ? fmaxf(f[r], 0.f) : 0.f;
    return Frag<T, KS>::from_f32(f);
  } else if constexpr (std::is_same<T, _Float16>::value) {
    constexpr int NW = KS / 2;
    using W = uint32_t __attribute__((ext_vector_type(NW)));
    const W w = __builtin_bit_cast(W, x);
    W out;
    const half2_t zero = {0, 0};
    const half2_t l2e = {(_Float16)kLog2e, (_Float16)kLog2e};
#pragma unroll
    for (int k = 0; k < NW; ++k) {
      const half2_t p = __builtin_bit_cast(half2_t, (uint32_t)w[k]);
      const half2_t mn = __builtin_elementwise_min(p, zero) * l2e;
      const half2_t mx = __builtin_elementwise_max(p, zero);
      half2_t e;
      e.x = __builtin_exp2f16(mn.x);
      e.y = __builtin_exp2f16(mn.y);
      const uint32_t r = __builtin_bit_cast(uint32_t, mx + e);
      out[k] = ok ? r : 0u;
    }
    return __builtin_bit_cast(Raw<T, KS>, out);
  } else {
    float f[KS];
    Frag<T, KS>::to_f32(x, f);
#pragma unroll
    for (int r = 0; r < KS; ++r) f[r] = ok ? phi_f<T>(f[r]) : 0.f;
    return Frag<T, KS>::from_f32(f);
  }
}

// phi of a fragment (as phi_frag) and phi' at the same slots in fp32.  elu + 1
// shares the exponential: with e = exp(min(x, 0)), phi(x) = e + max(x, 0),
// phi'(x) = e.
template <typename T, int KS, int PHI>
__device__ __forceinline__ void phi_dphi(Raw<T, KS> x, bool ok, Raw<T, KS>& phi,
                                         float (&dphi)[KS]) {
  if constexpr (PHI == kPhiRelu) {
    float f[KS];
    Frag<T, KS>::to_f32(x, f);
#pragma unroll
    for (int r = 0; r < KS; ++r) dphi[r] = f[r] > 0.f ? 1.f : 0.f;
    phi = phi_frag<T, KS, PHI>(x, ok);
  } else if constexpr (std::is_same<T, _Float16>::value) {
    constexpr int NW = KS / 2;
    using W = uint32_t __attribute__((ext_vector_type(NW)));
    const W w = __builtin_bit_cast(W, x);
    W out;
    const half2_t zero = {0, 0};
    const half2_t l2e = {(_Float16)kLog2e, (_Float16)kLog2e};
#pragma unroll
    for (int k = 0; k < NW; ++k) {
      const half2_t p = __builtin_bit_cast(half2_t, (uint32_t)w[k]);
      const half2_t mn = __builtin_elementwise_min(p, zero) * l2e;
      const half2_t mx = __builtin_elementwise_max(p, zero);
      half2_t e;
      e.x = __builtin_exp2f16(mn.x);
      e.y = __builtin_exp2f16(mn.y);
      out[k] = ok ? __builtin_bit_cast(uint32_t, mx + e) : 0u;
      dphi[2 * k] = (float)e.x;
      dphi[2 * k + 1] = (float)e.y;
    }
    phi = __builtin_bit_cast(Raw<T, KS>, out);
  } else {
    float f[KS];
    Frag<T, KS>::to_f32(x, f);
#pragma unroll
    for (int r = 0; r < KS; ++r) {
      const float m = fminf(f[r], 0.f);
      const float e = Ty<T>::kNarrow ? __builtin_amdgcn_exp2f(m * kLog2e) : expf(m);
      dphi[r] = e;
      f[r] = ok ? e + fmaxf(f[r], 0.f) : 0.f;
    }
    phi = Frag<T, KS>::from_f32(f);
  }
}

// 8-slot row operand of a row contraction: slot r <-> row r0 + E(g, r) of the
// slice (rows 4g..4g+3 of the two sub-tiles); `val` where the row is in [a, b).
template <typename T>
__device__ __forceinline__ Raw<T, 8> row_mask(int32_t r0, int g, int32_t a, int32_t b, float val) {
  float x[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int32_t row = r0 + Geo<32>::E(g, r);
    x[r] = (row >= a && row < b) ? val : 0.f;
  }
  return Frag<T, 8>::from_f32(x);
}

__device__ __forceinline__ bool sub_overlaps(int32_t r0, int s, int32_t a, int32_t b) {
  return r0 + 16 * s < b && r0 + 16 * s + 16 > a;
}

// Rows [a, b) of one slice into the state: M += phi(K)^T V, V += phi(K)^T 1.
// K is matrix 0, V matrix 1.
template <typename T, int D, int NM, int PHI>
__device__ __forceinline__ void state_seg(const Slice<T, Geo<D>::KS, NM>& sb, int32_t r0,
                                          int32_t a, int32_t b, int i, int g,
                                          const Sel<T, D>& sel, State<D>& st) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  using F = Frag<T, KS>;
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  Raw<T, KS> fk[2], vv[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int32_t row = r0 + 16 * s + i;
    const bool in = sb.ok[s] && row >= a && row < b;
    fk[s] = phi_frag<T, KS, PHI>(sb.x[0][s], in);
    vv[s] = in ? sb.x[1][s] : F::zero();
  }
  // the row transposes, each packed into an operand as soon as it is formed
  auto rows_of = [&](const Raw<T, KS>(&x)[2], int t) -> Raw<T, 8> {
    return pack_rows<T>(F::mma(x[0], sel.m[t], zero), F::mma(x[1], sel.m[t], zero));
  };
  Raw<T, 8> pv[NT];
#pragma unroll
  for (int ct = 0; ct < NT; ++ct) pv[ct] = rows_of(vv, ct);
  // phi(K) is already zero outside [a, b), so z needs no row mask
  float one8[8] = {1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f};
  const Raw<T, 8> ones = Frag<T, 8>::from_f32(one8);
#pragma unroll
  for (int et = 0; et < NT; ++et) {
    const Raw<T, 8> pk = rows_of(fk, et);
    st.V[et] = Frag<T, 8>::mma(pk, ones, st.V[et]);
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) st.M[et][ct] = Frag<T, 8>::mma(pk, pv[ct], st.M[et][ct]);
  }
}

// Operand of a head-dim contraction from result tiles: slot r of lane (i, g) is
// tile[r / 4] component r % 4, times `mul`.
template <typename T, int D>
__device__ __forceinline__ Raw<T, Geo<D>::KS> tiles_operand(const floatx4 (&tl)[Geo<D>::NT],
                                                             float mul) {
  constexpr int KS = Geo<D>::KS;
  float x[KS];
#pragma unroll
  for (int r = 0; r < KS; ++r) x[r] = tl[r >> 2][r & 3] * mul;
  return Frag<T, KS>::from_f32(x);
}

// ------------------------------------------------------------ forward math
template <typename T, int D>
struct FwdOp {
  Raw<T, Geo<D>::KS> A[Geo<D>::NT];  // sig S as operand of result tile ct (contract e)
  Raw<T, Geo<D>::KS> Az;             // sig z in rows 0, 4, 8, 12: the normaliser of every
                                     // row lands in component 0 of every lane group
  float seps;                        // sig eps
};

template <typename T, int D>
__device__ __forceinline__ void make_fwd_op(const State<D>& st, FwdOp<T, D>& op, int i,
                                            float eps) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  const float sig = Ty<T>::kNarrow ? pow2_scale_to_one(st.absmax()) : 1.f;
#pragma unroll
  for (int ct = 0; ct < NT; ++ct) {
    floatx4 col[NT];
#pragma unroll
    for (int et = 0; et < NT; ++et) col[et] = st.M[et][ct];
    op.A[ct] = tiles_operand<T, D>(col, sig);
  }
  const float zmul = (i & 3) == 0 ? sig : 0.f;
  float zx[KS];
#pragma unroll
  for (int r = 0; r < KS; ++r) zx[r] = st.V[r >> 2][r & 3] * zmul;
  op.Az = Frag<T, KS>::from_f32(zx);
  op.seps = sig * eps;
}

// o = phi(q) S / (phi(q) . z + eps) for rows [a, b) of one slice (Q is matrix
// QM): numerator and normaliser both come from the matrix cores with the same
// rounded phi(q) and the same scale sig, which cancels (eps is scaled by sig).
template <typename T, int D, int NM, int QM, int PHI>
__device__ __forceinline__ void apply_seg(const Slice<T, Geo<D>::KS, NM>& sb, int32_t r0,
                                          int32_t a, int32_t b, int i, int g,
                                          const FwdOp<T, D>& op, T* o, size_t rs, int col) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  using F = Frag<T, KS>;
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    if (!sub_overlaps(r0, s, a, b)) continue;
    const int32_t row = r0 + 16 * s + i;
    const bool in = sb.ok[s] && row >= a && row < b;
    const Raw<T, KS> bq = phi_frag<T, KS, PHI>(sb.x[QM][s], in);
    const floatx4 den = F::mma(op.Az, bq, zero);
    const float scale = recip<T>(den[0] + op.seps);
    float ox[KS];
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const floatx4 d4 = F::mma(op.A[ct], bq, zero);
#pragma unroll
      for (int j = 0; j < 4; ++j) ox[4 * ct + j] = d4[j] * scale;
    }
    RowIO<T, D>::put(o, row_off(sb.o[s], rs, col), g, F::from_f32(ox), in);
  }
}

// Target occupancy (waves per SIMD) handed to the register allocator.
#ifndef SLA_FWD_WPE
#define SLA_FWD_WPE 3
#endif
#ifndef SLA_BWD_WPE
#define SLA_BWD_WPE 2
#endif
// fp32 storage doubles the resident rows: ask for half the occupancy
template <typename T, int W16>
constexpr int kWpe = sizeof(T) == 4 ? (W16 > 2 ? W16 / 2 : 1) : W16;

// ----------------------------------------------------------- backward math
// bf16 keeps 8 significant bits, so the backward carries the operands of its
// cancelling differences as a sum of two bf16 values (high part and rounding
// residual, 16 bits together): S^T in dq = (dout S^T - (dout . o) z) / den phi'(q)
// (o = phi(q) S / den, so dout . o = phi(q) . (dout S^T) / den), -dout.o in the dz
// accumulation, and dS^T in dk = (v dS^T + dz) phi'(k).  fp16 (11 bits) and fp32
// need no split.
template <typename T>
constexpr bool kSplitGrad = std::is_same<T, bf16_t>::value;

// Operands of the backward's head-dim contractions for one window.  B first holds
// the state operand (for the Q,dout rows) and is then overwritten with a
// state-gradient operand (for the K,V gradient rows).
template <typename T, int D>
struct BwdOp {
  Raw<T, Geo<D>::KS> A[Geo<D>::NT];  // unused                           | rho dS^T (dfk = v dS^T, tile et)
  Raw<T, Geo<D>::KS> B[Geo<D>::NT];  // sig S^T (dfq = dout S^T, tile et) | rho dS  (dv = phi(k) dS, tile ct)
  Raw<T, Geo<D>::KS> Az;             // sig z in rows 0, 4, 8, 12 (normaliser) | unused
  float z[Geo<D>::KS];               // sig z (as rounded in Az + Azl)    | dz
  float inv_scale;                   // unused                            | 1 / rho
  float bsig;                        // beta sig: phi(q) / den in the state gradients is
                                     // scaled by beta (<= min z, so beta phi(q) / den <= 1)
  float inv_beta;                    // 1 / beta
  float seps;                        // sig eps
  Raw<T, Geo<D>::KS> Al[kSplitGrad<T> ? Geo<D>::NT : 1];  // unused | residual of A (bf16)
  Raw<T, Geo<D>::KS> Bl[kSplitGrad<T> ? Geo<D>::NT : 1];  // residual of B (bf16) | unused
  Raw<T, Geo<D>::KS> Azl;            // residual of Az (bf16)              | unused
};

// The transpose of a state as operands of a head-dim contraction: slot r of lane
// (e', g) of tile et is M[16 et + e'][E(g, r)] * mul.  Goes through the wave's
// own LDS tile (row e, column c, rows padded to keep 16-byte reads aligned).
template <int D>
constexpr int kTrLd = D + 4;

template <typename T, int D, bool LO = false>
__device__ __forceinline__ void transposed_operand(const State<D>& st, float mul, float* tile,
                                                   int i, int g,
                                                   Raw<T, Geo<D>::KS> (&out)[Geo<D>::NT],
                                                   Raw<T, Geo<D>::KS>* out_lo = nullptr) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT, LD = kTrLd<D>;
#pragma unroll
  for (int et = 0; et < NT; ++et)
#pragma unroll
    for (int ct = 0; ct < NT; ++ct)
#pragma unroll
      for (int j = 0; j < 4; ++j) tile[(16 * et + 4 * g + j) * LD + 16 * ct + i] = st.M[et][ct][j];
  wave_lds_sync();
#pragma unroll
  for (int et = 0; et < NT; ++et) {
    float x[KS];
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const float4 p = *reinterpret_cast<const float4*>(tile + (16 * et + i) * LD + 16 * ct + 4 * g);
      x[4 * ct + 0] = p.x * mul;
      x[4 * ct + 1] = p.y * mul;
      x[4 * ct + 2] = p.z * mul;
      x[4 * ct + 3] = p.w * mul;
    }
    out[et] = Frag<T, KS>::from_f32(x);
    if constexpr (LO) {
      float hi[KS];
      Frag<T, KS>::to_f32(out[et], hi);
#pragma unroll
      for (int r = 0; r < KS; ++r) x[r] -= hi[r];
      out_lo[et] = Frag<T, KS>::from_f32(x);
    }
  }
  wave_lds_sync();   // the tile may be written again by the next call
}

// beta bounds phi(q)_e / den through 1 / z_e, for every e with z_e > 0.  Under
// ReLU a feature with z_e = 0 has phi(k_j)_e = 0 for every row of the window, so
// row e of dS and dz_e reach neither dk (phi'(k_j)_e = 0) nor dv (phi(k_j)_e =
// 0): qgrad_seg leaves those features out of the state gradients.
template <typename T, int D, int PHI>
__device__ __forceinline__ void make_state_op(const State<D>& st, BwdOp<T, D>& op, float* tile,
                                              int i, int g, float eps) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  const float sig = Ty<T>::kNarrow ? pow2_scale_to_one(st.absmax()) : 1.f;
  transposed_operand<T, D, kSplitGrad<T>>(st, sig, tile, i, g, op.B, op.Bl);
  // op.z holds sig z rounded exactly as in the normaliser operands: dq subtracts
  // (dout.o) z from dout S^T, and for a row whose normaliser is mostly eps the two
  // terms cancel to eps / den; the same z on both sides keeps that residual exact.
  // bf16 carries z as a pair (Az + Azl), as S^T is carried in B + Bl: a z rounded
  // to 8 bits against an S kept to 16 leaves the cancellation a 2^-9 remainder
  float zmin = 3.0e38f;
  float zx[KS], zl[KS];
#pragma unroll
  for (int r = 0; r < KS; ++r) {
    const float z = st.V[r >> 2][r & 3];
    if (PHI != kPhiRelu || z > 0.f) zmin = fminf(zmin, z);
    const float zh = Ty<T>::kNarrow ? u16_to_f32<T>(f32_to_u16<T>(z * sig)) : z * sig;
    float zs = zh;
    if constexpr (kSplitGrad<T>) {
      const float lo = u16_to_f32<T>(f32_to_u16<T>(z * sig - zh));
      zs = zh + lo;
      zl[r] = (i & 3) == 0 ? lo : 0.f;
    }
    op.z[r] = zs;
    zx[r] = (i & 3) == 0 ? zh : 0.f;
  }
  op.Az = Frag<T, KS>::from_f32(zx);
  if constexpr (kSplitGrad<T>) op.Azl = Frag<T, KS>::from_f32(zl);
  // phi(q)_e / den <= 1 / z_e <= 1 / min z, so beta phi(q) / den <= 1
  const float beta = Ty<T>::kNarrow ? pow2_floor(wave_reduce<false>(zmin)) : 1.f;
  op.bsig = beta * sig;
  op.inv_beta = 1.f / beta;
  op.seps = sig * eps;
}

// From state-gradient tiles that carry a factor `1 / inv_beta`.
template <typename T, int D>
__device__ __forceinline__ void make_grad_op(const State<D>& st, float inv_beta, BwdOp<T, D>& op,
                                             float* tile, int i, int g) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  const float mx = st.absmax() * inv_beta;
  const float rho = Ty<T>::kNarrow ? pow2_scale_to_one(mx) : 1.f;
  op.inv_scale = 1.f / rho;
  const float mul = rho * inv_beta;
  transposed_operand<T, D, kSplitGrad<T>>(st, mul, tile, i, g, op.A, op.Al);
#pragma unroll
  for (int ct = 0; ct < NT; ++ct) {
    floatx4 col[NT];
#pragma unroll
    for (int et = 0; et < NT; ++et) col[et] = st.M[et][ct];
    op.B[ct] = tiles_operand<T, D>(col, mul);
  }
#pragma unroll
  for (int r = 0; r < KS; ++r) op.z[r] = st.V[r >> 2][r & 3] * inv_beta;
}

// Rows [a, b) of one slice: dq, and into gs: M += beta (phi(q)/den)^T dout,
// V += beta (phi(q)/den)^T (-dout.o).  q is matrix QI, dout matrix DI.  The
// normaliser comes from the matrix cores (den' = sig den, plus sig eps); with sig
// folded into z, dphi(q) = (sig dfq - dot sig z) / den'.
template <typename T, int D, int NM, int QI, int DI, int PHI>
__device__ __forceinline__ void qgrad_seg(const Slice<T, Geo<D>::KS, NM>& sb, int32_t r0,
                                          int32_t a, int32_t b, int i, int g,
                                          const Sel<T, D>& sel, const BwdOp<T, D>& op, T* dq,
                                          size_t rs, int col, State<D>& gs) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  using F = Frag<T, KS>;
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  constexpr bool SP = kSplitGrad<T>;
  Raw<T, KS> xr[2], dr[2], nd[2], nl[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int32_t row = r0 + 16 * s + i;
    const bool in = sb.ok[s] && row >= a && row < b;
    dr[s] = in ? sb.x[DI][s] : F::zero();
    xr[s] = F::zero();
    nd[s] = F::zero();
    if constexpr (SP) nl[s] = F::zero();
    if (!sub_overlaps(r0, s, a, b)) continue;
    Raw<T, KS> bq;
    float dphq[KS], fq[KS];
    phi_dphi<T, KS, PHI>(sb.x[QI][s], in, bq, dphq);
    F::to_f32(bq, fq);
    floatx4 den4 = F::mma(op.Az, bq, zero);
    if constexpr (SP) den4 = F::mma(op.Azl, bq, den4);
    const float rden = recip<T>(in ? den4[0] + op.seps : 1.f);
    // dfq = sig dout S^T; dout.o = phi(q) S dout^T / den = phi(q).dfq / den'
    floatx4 dfq[NT];
    float dot = 0.f;
#pragma unroll
    for (int et = 0; et < NT; ++et) {
      dfq[et] = F::mma(op.B[et], dr[s], zero);
      if constexpr (SP) dfq[et] = F::mma(op.Bl[et], dr[s], dfq[et]);
#pragma unroll
      for (int j = 0; j < 4; ++j) dot += fq[4 * et + j] * dfq[et][j];
    }
    dot = sum_groups(dot) * rden;  // lane exchange: every lane takes part
    if (!in) dot = 0.f;
    float dqx[KS];
#pragma unroll
    for (int et = 0; et < NT; ++et)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = 4 * et + j;
        dqx[r] = (dfq[et][j] - dot * op.z[r]) * rden * dphq[r];
      }
    RowIO<T, D>::put(dq, row_off(sb.o[s], rs, col), g, F::from_f32(dqx), in);
    float xs[KS], ns[KS];
    const float w = op.bsig * rden;
#pragma unroll
    for (int r = 0; r < KS; ++r) {
      xs[r] = (PHI != kPhiRelu || op.z[r] > 0.f) ? fq[r] * w : 0.f;
      ns[r] = -dot;
    }
    xr[s] = F::from_f32(xs);
    nd[s] = F::from_f32(ns);
    if constexpr (SP) {
      const float res = -dot - u16_to_f32<T>(f32_to_u16<T>(-dot));
#pragma unroll
      for (int r = 0; r < KS; ++r) ns[r] = res;
      nl[s] = F::from_f32(ns);
    }
  }
  // the row transposes, each packed into an operand as soon as it is formed (the
  // packed operand takes half the registers of its two result tiles)
  auto rows_of = [&](const Raw<T, KS>(&x)[2], int t) -> Raw<T, 8> {
    return pack_rows<T>(F::mma(x[0], sel.m[t], zero), F::mma(x[1], sel.m[t], zero));
  };
  Raw<T, 8> pd[NT];
#pragma unroll
  for (int ct = 0; ct < NT; ++ct) pd[ct] = rows_of(dr, ct);
  const Raw<T, 8> pn = rows_of(nd, 0);
  Raw<T, 8> pl;
  if constexpr (SP) pl = rows_of(nl, 0);
#pragma unroll
  for (int et = 0; et < NT; ++et) {
    const Raw<T, 8> px = rows_of(xr, et);
    gs.V[et] = Frag<T, 8>::mma(px, pn, gs.V[et]);
    if constexpr (SP) gs.V[et] = Frag<T, 8>::mma(px, pl, gs.V[et]);
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) gs.M[et][ct] = Frag<T, 8>::mma(px, pd[ct], gs.M[et][ct]);
  }
}

// Rows [a, b) of one slice: dk = (v dS^T + dz) phi'(k), dv = phi(k) dS.
template <typename T, int D, int NM, int PHI>
__device__ __forceinline__ void kgrad_seg(const Slice<T, Geo<D>::KS, NM>& sb, int32_t r0,
                                          int32_t a, int32_t b, int i, int g,
                                          const BwdOp<T, D>& op, T* dk, T* dv, size_t rs,
                                          int col) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  using F = Frag<T, KS>;
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    if (!sub_overlaps(r0, s, a, b)) continue;
    const int32_t row = r0 + 16 * s + i;
    const bool in = sb.ok[s] && row >= a && row < b;
    Raw<T, KS> fk;
    float dphk[KS];
    phi_dphi<T, KS, PHI>(sb.x[0][s], in, fk, dphk);
    float dkx[KS], dvx[KS];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      floatx4 a4 = F::mma(op.A[t], sb.x[1][s], zero);
      if constexpr (kSplitGrad<T>) a4 = F::mma(op.Al[t], sb.x[1][s], a4);
      const floatx4 b4 = F::mma(op.B[t], fk, zero);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = 4 * t + j;
        dkx[r] = (a4[j] * op.inv_scale + op.z[r]) * dphk[r];
        dvx[r] = b4[j] * op.inv_scale;
      }
    }
    RowIO<T, D>::put(dk, row_off(sb.o[s], rs, col), g, F::from_f32(dkx), in);
    RowIO<T, D>::put(dv, row_off(sb.o[s], rs, col), g, F::from_f32(dvx), in);
  }
}


// ------------------------------------------------------------- work items
// A launch walks a list of work items; workgroup b takes items b, b + G, ...
// (G = grid size, a multiple of 8, about the number of resident workgroups).
// In order:
//   long items   one per (long window, head): the four waves of the workgroup
//                take a quarter of the window's rows each, add their partial
//                states in LDS (in wave order, so every wave holds the same sum)
//                and then form their rows' outputs.  Item numbers are laid out so
//                that the heads of one window share an item residue mod 8, i.e.
//                run on one XCD (workgroups are dealt to the 8 XCDs round-robin),
//                where the L2 serves the other heads' halves of each row.
//   chunk items  one per chunk and group of up to 4 heads (one wave per head;
//                with fewer than 4 heads, several chunks share a workgroup).
// Long items come first: they are the longest-running ones.
//
// Each wave software-pipelines its items: while item k computes, the plan entry
// of item k + 2 and the permutation entries and window offsets of item k + 1 are
// in flight, so an item's row gathers start as soon as the previous item's rows
// have been requested and its data path is one memory round trip long.
struct Items {
  int32_t nL4, nL2, nC, H, hp, hw, cpw, hg;
  int32_t itemsL4, itemsL, total;
};

__device__ __forceinline__ Items work_items(const KernelArgs& a, const PlanHeader* hdr) {
  Items it;
  const int32_t nL = max(0, min(hdr->n_long, a.max_long));
  it.nL4 = max(0, min(hdr->n_long4, nL));
  it.nL2 = nL - it.nL4;
  it.nC = max(0, min(hdr->n_chunks, a.max_chunks));
  it.H = a.H;
  it.hp = (a.H + 1) / 2;
  it.hw = min(a.H, 4);
  it.cpw = 4 / it.hw;
  it.hg = (a.H + 3) / 4;
  it.itemsL4 = ((it.nL4 + 7) & ~7) * a.H;
  it.itemsL = it.itemsL4 + ((it.nL2 + 7) & ~7) * it.hp;
  it.total = it.itemsL + (it.nC + it.cpw - 1) / it.cpw * it.hg;
  return it;
}

struct WaveWork {
  int kind;        // 0: nothing, 1: a chunk, 2: a share of a long window
  int h;           // head
  int32_t ra, rb;  // rows (sorted positions)
  int32_t wb, we;  // windows
  int pair;        // long window: 0 = the four waves share it, 1 = waves 2m, 2m + 1 do
};

// Where item `item` puts wave wv (wave-uniform): table entry index (-1: none),
// the table (0: long windows, 1: chunks), the head, and for a long window how
// many waves share it and which share is this wave's (-1: none, the wave only
// takes part in the workgroup's partial-state exchange).
//   four-way long items: one per (window, head), the four waves take quarters;
//   two-way long items: one per (window, pair of heads), waves 2m and 2m + 1
//     take the halves of head 2 x (item's pair) + m.
struct Slot {
  int32_t idx;
  int table, h, parts, piece;
};

__device__ __forceinline__ Slot item_slot(const Items& it, int32_t item, int wv) {
  Slot sl;
  sl.idx = -1;
  sl.table = 0;
  sl.h = 0;
  sl.parts = 4;
  sl.piece = wv;
  if (item >= it.total) return sl;
  if (item < it.itemsL4) {
    const int32_t r = item >> 3;
    const int32_t j = (r / it.H) * 8 + (item & 7);
    sl.h = r % it.H;
    if (j < it.nL4) sl.idx = j;
  } else if (item < it.itemsL) {
    const int32_t r = (item - it.itemsL4) >> 3;   // itemsL4 is a multiple of 8
    const int32_t j = (r / it.hp) * 8 + (item & 7);
    const int h = (r % it.hp) * 2 + (wv >> 1);
    sl.parts = 2;
    sl.piece = h < it.H ? (wv & 1) : -1;
    sl.h = h < it.H ? h : 0;
    if (j < it.nL2) sl.idx = it.nL4 + j;
  } else {
    const int32_t b = item - it.itemsL;
    const int32_t grp = b / it.hg;
    const int sub = wv / it.hw;
    const int32_t c = grp * it.cpw + sub;
    sl.table = 1;
    sl.h = (b - grp * it.hg) * 4 + wv % it.hw;
    if (sub < it.cpw && c < it.nC && sl.h < it.H) sl.idx = c;
  }
  return sl;
}

// The plan entry of a slot (4 ints; Chunk and LongWin have the same size).
__device__ __forceinline__ int4 slot_entry(const KernelArgs& a, const Slot& sl) {
  if (sl.idx < 0) return make_int4(0, 0, 0, 0);
  if (sl.table == 0) return reinterpret_cast<const int4*>(a.longs)[sl.idx];
  return reinterpret_cast<const int4*>(a.chunks)[sl.idx];
}

__device__ __forceinline__ WaveWork decode_work(const KernelArgs& a, const Slot& sl, int4 e,
                                                int wv) {
  WaveWork ww;
  ww.kind = 0;
  ww.h = sl.h;
  ww.ra = ww.rb = ww.wb = ww.we = 0;
  ww.pair = 0;
  if (sl.idx < 0) return ww;
  if (sl.table == 0) {  // LongWin: window, row_begin, row_end
    const int32_t rs = max(0, min(e.y, a.n));
    const int32_t re = max(rs, min(e.z, a.n));
    const int64_t len = re - rs;
    const int p = sl.piece < 0 ? 0 : sl.piece;
    ww.ra = rs + (int32_t)(len * p / sl.parts);
    ww.rb = sl.piece < 0 ? ww.ra : rs + (int32_t)(len * (p + 1) / sl.parts);
    ww.wb = e.x;
    ww.we = e.x + 1;
    ww.kind = 2;
    ww.pair = sl.parts == 2;
  } else {  // Chunk: row_begin, row_end, win_begin, win_end
    ww.ra = max(0, min(e.x, a.n));
    ww.rb = max(ww.ra, min(min(e.y, a.n), ww.ra + kMaxChunkRows));
    ww.we = max(0, min(e.w, a.W));
    ww.wb = max(0, min(e.z, ww.we));
    ww.kind = 1;
  }
  return ww;
}

// ---------------------------------------------------------- windows of a chunk
// The windows of a chunk, 64 at a time in registers: lane l holds the rows of
// window wp + l clipped to the chunk, and a ballot marks the non-empty ones, so
// that moving to the next window is a few scalar instructions (chunks of small
// windows may also hold many empty ones).  request() issues the loads of a page,
// settle() takes the ballot (so a page can be requested ahead of its use).
struct WinCursor {
  int32_t w;       // current window (-1: finished)
  int32_t ws, we;  // its rows, clipped to the chunk
};

struct Stream {
  const int32_t* offs;
  int32_t rb, re, wend;
  int32_t wp;      // first window of the loaded page
  int32_t a, b;    // rows of window wp + lane, clipped to [rb, re)
  uint64_t live;   // lanes whose window is non-empty
  int lane;
  __device__ __forceinline__ void request(int32_t w0) {
    wp = w0;
    const int32_t w = wp + lane;
    a = b = 0;
    if (w < wend) {
      a = max(offs[w], rb);
      b = min(offs[w + 1], re);
    }
  }
  __device__ __forceinline__ void settle() { live = __ballot(a < b); }
  __device__ __forceinline__ bool next_window(WinCursor& j) {
    for (;;) {
      const int sh = j.w + 1 - wp;   // first lane after the current window
      const uint64_t m = sh <= 0 ? live : (sh >= 64 ? 0ull : live & (~0ull << sh));
      if (m) {
        const int l = __builtin_ctzll(m);
        j.w = wp + l;
        j.ws = __builtin_amdgcn_readlane(a, l);
        j.we = __builtin_amdgcn_readlane(b, l);
        return true;
      }
      if (wp + 64 >= wend) break;
      request(wp + 64);
      settle();
    }
    j.w = -1;
    return false;
  }
};

// ------------------------------------------------------------- row blocks
// Up to kBlockJobs 32-row jobs of one head held in registers: NM matrices as row
// fragments (forward: K, V, Q; backward: K, V, Q, dout).
constexpr int kBlockJobs = kMaxChunkRows / kSliceRows;
constexpr int kBlockRows = kBlockJobs * kSliceRows;

template <typename T, int D, int NM>
struct Block {
  Slice<T, Geo<D>::KS, NM> j[kBlockJobs];
};

// Original rows of sorted rows [base, min(end, base + kBlockRows)): lane (i, g)
// of sub-tile s of job jj takes row base + 32 jj + 16 s + i (-1: none).
struct BlockRows {
  int32_t o[kBlockJobs][2];
};

__device__ __forceinline__ void block_rows(BlockRows& br, int32_t base, int32_t end,
                                           const int32_t* perm, int lane) {
  const int i = lane & 15;
#pragma unroll
  for (int jj = 0; jj < kBlockJobs; ++jj)
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int32_t row = base + kSliceRows * jj + 16 * s + i;
      br.o[jj][s] = row < end ? (perm ? perm[row] : row) : -1;
    }
}

// The matrices selected by `which` (bit m: mats[m]) of the block's rows into slot
// order.  Sub-tiles past `end` are not read (and are zero); rows past `end`
// inside a read sub-tile read row 0, which the math masks.
template <typename T, int D, int NM>
__device__ __forceinline__ void block_fetch(Block<T, D, NM>& bk, const BlockRows& br, int32_t base,
                                            int32_t end, int32_t n, const T* const (&mats)[NM],
                                            unsigned which, size_t rs, int col, int g) {
  using F = Frag<T, Geo<D>::KS>;
#pragma unroll
  for (int jj = 0; jj < kBlockJobs; ++jj)
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const bool ok = (uint32_t)br.o[jj][s] < (uint32_t)n;
      bk.j[jj].ok[s] = ok;
      bk.j[jj].o[s] = ok ? br.o[jj][s] : 0;
      const bool live = base + kSliceRows * jj + 16 * s < end;
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        if (!(which & (1u << m))) continue;
        if (live) bk.j[jj].x[m][s] = RowIO<T, D>::fetch(mats[m], row_off(bk.j[jj].o[s], rs, col), g);
        else bk.j[jj].x[m][s] = F::zero();
      }
    }
}

template <typename T, int D, int NM>
__device__ __forceinline__ void block_arrange(Block<T, D, NM>& bk, unsigned which) {
#pragma unroll
  for (int jj = 0; jj < kBlockJobs; ++jj)
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int m = 0; m < NM; ++m)
        if (which & (1u << m)) RowIO<T, D>::arrange(bk.j[jj].x[m][s]);
}

__device__ __forceinline__ bool job_overlaps(int32_t r0, int32_t a, int32_t b) {
  return r0 < b && r0 + kSliceRows > a;
}

// An item of this wave whose row permutation and windows have been requested.
struct Pending {
  WaveWork ww;
  BlockRows br;
  Stream str;
};

__device__ __forceinline__ void pending_request(Pending& p, const KernelArgs& a, const Slot& sl,
                                                int4 e, int wv, const int32_t* perm, int lane) {
  p.ww = decode_work(a, sl, e, wv);
  p.str.lane = lane;
  p.str.offs = a.offs;
  p.str.rb = p.ww.ra;
  p.str.re = p.ww.rb;
  p.str.wend = p.ww.we;
  p.str.wp = p.ww.wb;
  p.str.a = p.str.b = 0;
  p.str.live = 0;
  if (p.ww.kind != 0) block_rows(p.br, p.ww.ra, min(p.ww.rb, p.ww.ra + kBlockRows), perm, lane);
  if (p.ww.kind == 1) p.str.request(p.ww.wb);
}

// ------------------------------------------------ the item stream, through LDS
// A wave's view of the items ahead of it: the permutation slice of an item's
// first block, the window offsets of a chunk and the plan entry of an item are
// gathered into LDS by the memory system (global_load_lds: lane l's value lands
// at the slot + 4 l) one or two items ahead, and read from LDS at the top of
// the item that needs them.  Values prefetched into registers would have to be
// carried from one item's registers to the next one's, and the copy, or a load
// merged with a default value, waits for the load; through LDS the only wait of
// an item is the one at its top.
struct WaveMeta {
  int32_t perm[2][kMaxChunkRows];   // permutation slices (ring by item parity)
  int32_t offs[2][128];             // offs[wb + l] of a chunk's first 128 window slots
  int4 ent[2];                      // plan entries
};

__device__ __forceinline__ int32_t first_block_rows(const WaveWork& w) {
  return w.kind != 0 ? min(w.rb - w.ra, kMaxChunkRows) : 0;
}

// The permutation slice of an item's first block into `slot` (none in CSR mode).
__device__ __forceinline__ void request_perm(const WaveWork& w, const int32_t* perm, int32_t* slot, int lane) {
  if (perm != nullptr && lane < first_block_rows(w))
    __builtin_amdgcn_global_load_lds(perm + w.ra + lane, (__attribute__((address_space(3))) void*)slot, 4, 0, 0);
}

// The offsets of a chunk's first 128 window slots into `slot` (indices clamped to
// the table; windows past the chunk are ignored when the stream is built).
__device__ __forceinline__ void request_offs(const WaveWork& w, const KernelArgs& a, int32_t* slot, int lane) {
  if (w.kind != 1) return;
  __builtin_amdgcn_global_load_lds(a.offs + min(w.wb + lane, a.W), (__attribute__((address_space(3))) void*)slot,
                                   4, 0, 0);
  __builtin_amdgcn_global_load_lds(a.offs + min(w.wb + 64 + lane, a.W),
                                   (__attribute__((address_space(3))) void*)(slot + 64), 4, 0, 0);
}

// The plan entry of a slot into LDS (4 lanes of 4 bytes).
__device__ __forceinline__ void request_entry(const KernelArgs& a, const Slot& sl, int4* slot, int lane) {
  if (sl.idx < 0 || lane >= 4) return;
  const int32_t* t = sl.table == 0 ? reinterpret_cast<const int32_t*>(a.longs) : reinterpret_cast<const int32_t*>(a.chunks);
  __builtin_amdgcn_global_load_lds(t + 4 * sl.idx + lane, (__attribute__((address_space(3))) void*)slot, 4, 0, 0);
}

__device__ __forceinline__ int4 lds_entry(const int4* slot) {
  typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));
  const u32x4v e = *(const __attribute__((address_space(3))) u32x4v*)slot;
  return make_int4((int)__builtin_amdgcn_readfirstlane(e[0]), (int)__builtin_amdgcn_readfirstlane(e[1]),
                   (int)__builtin_amdgcn_readfirstlane(e[2]), (int)__builtin_amdgcn_readfirstlane(e[3]));
}

// Original rows of an item's first block (the layout of block_rows) from its slice.
__device__ __forceinline__ void block_rows_lds(BlockRows& br, const WaveWork& w, const int32_t* slot, bool csr,
                                               int lane) {
  const int i = lane & 15;
  const int32_t nr = first_block_rows(w);
#pragma unroll
  for (int jj = 0; jj < kBlockJobs; ++jj)
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int lr = kSliceRows * jj + 16 * s + i;
      br.o[jj][s] = lr >= nr ? -1 : (csr ? w.ra + lr : *(const __attribute__((address_space(3))) int32_t*)(slot + lr));
    }
}

// The window stream of a chunk from its offsets slot (page 0; later pages are
// read from the plan as they are reached).
__device__ __forceinline__ void stream_lds(Stream& str, const WaveWork& w, const KernelArgs& a, const int32_t* slot,
                                           int lane) {
  str.lane = lane;
  str.offs = a.offs;
  str.rb = w.ra;
  str.re = w.rb;
  str.wend = w.we;
  str.wp = w.wb;
  str.a = str.b = 0;
  str.live = 0;
  if (w.kind != 1) return;
  const int32_t x0 = *(const __attribute__((address_space(3))) int32_t*)(slot + lane);
  const int32_t x1 = *(const __attribute__((address_space(3))) int32_t*)(slot + lane + 1);
  const bool has = w.wb + lane < w.we;
  str.a = has ? max(x0, w.ra) : 0;
  str.b = has ? min(x1, w.rb) : 0;
}

__device__ __forceinline__ void wait_vm() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void wait_lgkm() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Block until every wave of the workgroup gets here, with this wave's LDS writes
// done (LDS only: loads in flight stay in flight).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// ------------------------------------------------------ partial-state exchange
// A state as result tiles in LDS, one floatx4 per (tile, lane), so that waves of
// a workgroup can add their partial states.
template <int D>
constexpr int kStateTiles = Geo<D>::NT * Geo<D>::NT + Geo<D>::NT;

template <int D>
__device__ __forceinline__ void publish(const State<D>& st, floatx4* slot, int lane) {
  constexpr int NT = Geo<D>::NT;
  int t = 0;
#pragma unroll
  for (int a = 0; a < NT; ++a)
#pragma unroll
    for (int b = 0; b < NT; ++b) slot[(t++) * 64 + lane] = st.M[a][b];
#pragma unroll
  for (int a = 0; a < NT; ++a) slot[(t++) * 64 + lane] = st.V[a];
}

// st = sum of the published states of the waves that share this wave's long
// window (all four, or the pair 2m, 2m + 1), in wave order.
template <int D>
__device__ __forceinline__ void combine(State<D>& st, const floatx4* slots, int lane, int wv,
                                        bool pair) {
  constexpr int NT = Geo<D>::NT, KT = kStateTiles<D>;
  st.clear();
  const int w0 = pair ? (wv & ~1) : 0, nw = pair ? 2 : kWaves;
  for (int w = w0; w < w0 + nw; ++w) {
    const floatx4* sl = slots + w * KT * 64;
    int t = 0;
#pragma unroll
    for (int a = 0; a < NT; ++a)
#pragma unroll
      for (int b = 0; b < NT; ++b) st.M[a][b] += sl[(t++) * 64 + lane];
#pragma unroll
    for (int a = 0; a < NT; ++a) st.V[a] += sl[(t++) * 64 + lane];
  }
}

// The windows an item gives a wave: the windows of a chunk (each one whole), or
// one quarter of a long window (shared: its partial state is added to the other
// three quarters' before use).
struct WinIter {
  WinCursor wc;
  bool shared;
  __device__ __forceinline__ bool first(const WaveWork& ww, Stream& str) {
    shared = ww.kind == 2;
    wc.w = ww.wb - 1;
    if (ww.kind == 1) {
      str.settle();
      return str.next_window(wc);
    }
    wc.ws = ww.ra;
    wc.we = ww.rb;
    return ww.kind == 2;
  }
  __device__ __forceinline__ bool next(const WaveWork& ww, Stream& str) {
    return ww.kind == 1 && str.next_window(wc);
  }
};

// ------------------------------------------------------------ host launchers
// Workgroups of a launch: the resident capacity of the device for the kernel
// (workgroups per CU x CUs, queried once per device and kernel), at most enough
// for every item the plan can hold (long windows have more than kMinChunkRows
// rows), a multiple of 8.
inline int resident_workgroups(const void* kernel) {
  struct Entry {
    const void* kernel;
    int dev, cap;
  };
  static Entry cache[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = 0;
  for (const Entry& e : cache)
    if (e.kernel == kernel && e.dev == dev) return e.cap;
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, 64 * kWaves, 0) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      per_cu < 1 || cus < 1) {
    per_cu = 2;
    cus = 256;
  }
  for (Entry& e : cache)
    if (e.kernel == nullptr) {
      e = Entry{kernel, dev, per_cu * cus};
      break;
    }
  return per_cu * cus;
}

// Workgroups of a launch: a whole number k of the device's resident capacity for
// the kernel (a partial last round of workgroups would start late and set the
// end), with k ~ (row-heads) / (300 x resident).  Small scenes (one Waymo-like
// frame) get one persistent round whose waves prefetch item to item; large ones
// (200k+ rows, several heads) get several rounds, so that the hardware
// dispatcher balances items of very different cost.  At most enough workgroups
// for every item the plan can hold; a multiple of 8.
constexpr int64_t kRowHeadsPerWorkgroup = 300;

inline int grid_size(const void* kernel, const PlanLayout& lay, int32_t n, int32_t H) {
  const int64_t c = resident_workgroups(kernel);
  const int hw = H < 4 ? H : 4, cpw = 4 / hw, hg = (H + 3) / 4;
  const int64_t itemsL = (int64_t)(((lay.max_long + 7) & ~7) + 8) * H;
  const int64_t itemsC = (int64_t)(lay.max_chunks + cpw - 1) / cpw * hg;
  int64_t k = ((int64_t)n * H + c * kRowHeadsPerWorkgroup / 2) / (c * kRowHeadsPerWorkgroup);
  if (k < 1) k = 1;
  int64_t g = k * c;
  if (g > itemsL + itemsC) g = itemsL + itemsC;
  g = (g + 7) & ~7;
  return (int)(g < 8 ? 8 : g);
}

inline KernelArgs kernel_args(const void* plan, const PlanLayout& lay, int32_t n, int32_t W,
                              int32_t H, float eps) {
  const char* base = static_cast<const char*>(plan);
  KernelArgs a;
  a.hdr = reinterpret_cast<const PlanHeader*>(base + lay.header);
  a.perm = reinterpret_cast<const int32_t*>(base + lay.perm);
  a.offs = reinterpret_cast<const int32_t*>(base + lay.offsets);
  a.chunks = reinterpret_cast<const Chunk*>(base + lay.chunks);
  a.longs = reinterpret_cast<const LongWin*>(base + lay.longs);
  a.max_chunks = lay.max_chunks;
  a.max_long = lay.max_long;
  a.n = n;
  a.W = W;
  a.H = H;
  a.eps = eps;
  return a;
}

}  // namespace sla

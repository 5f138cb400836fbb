// SLA forward and backward on the gfx950 matrix cores.
//
// Work decomposition.  One wavefront per (chunk, head); a workgroup holds the
// waves of up to four heads of one chunk, and the grid has one workgroup column
// per chunk-table entry, so that every (chunk, head) of a scene is resident at
// once (about 6 k waves for 1.5 k chunks and 4 heads) and the hardware
// dispatcher balances them.  A chunk is a run of whole windows of the
// window-sorted sequence (see the builder); its rows are read through the plan's
// permutation, so q, k, v stay in the caller's order.
//
// A wave walks its chunk window by window as a stream of 32-row jobs (forward:
// K,V rows into the state, then Q rows through it; backward: K,V, then Q,dout,
// then K,V again) and keeps two jobs' rows in flight ahead of the one it
// computes, so each wave has about three gathers outstanding at any time.
//
// Per window (Eq. (3); the chunk-wise state accumulation of Sec. 3.2 / Fig. 3(b)):
//   state    S = phi(K)^T V and z = phi(K)^T 1 on the matrix cores over the
//            window's rows (z is one more column of the same contraction);
//   forward  o = phi(q) S / (phi(q) . z);
//   backward dq from S, z; dS, dz (one more column again) from q, dout; then
//            dk, dv from dS, dz.
// Window states live in registers only: the HBM traffic is q, k, v (, dout) in,
// o (dq, dk, dv) out, and the plan's permutation and offsets.
//
// Register layouts (lane l = 16 g + i, g = lane group 0..3, KS = head_dim / 4,
// NT = head_dim / 16; slot r of lane group g stands for head-dim index
// E(g, r) = 16 (r / 4) + 4 g + r % 4):
//   row fragment   lane (i, g) holds the KS elements E(g, .) of row i of a 16-row
//                  sub-tile (NT loads of 4 consecutive elements);
//   result tile    a 16x16 matrix-core result: lane (n, g) holds rows 4g..4g+3
//                  of column n.
// The slot order E is chosen so that a state accumulated as result tiles is
// already the matrix operand of the next contraction and so that every
// contraction's result is again a row fragment: states move between steps
// without leaving registers.  A contraction over ROWS needs each lane to hold 8
// rows of one column; multiplying a row fragment by a 0/1 selection matrix on
// the matrix core (exact) gives lane (i, g) rows 4g..4g+3 of column i, and two
// sub-tiles give the 8 rows.
//
// 16-bit storage: matrix-core operands are the stored values or values rounded to
// the storage type.  Derived operands are scaled by a power of two into [1, 2)
// (S, dS) or to at most 1 (phi(q)/den) before rounding and the scale is divided
// out in fp32, so no operand overflows or flushes; phi, the denominators and all
// divisions are fp32.
#include "sla_common.h"

namespace sla {

constexpr int kWaves = 4;       // waves (heads) per workgroup
constexpr int kSliceRows = 32;  // rows per job

constexpr float kLog2e = 1.4426950408889634f;

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

// Power of two p with x * p in [1, 2) (1 for x = 0 or non-finite x).
__device__ __forceinline__ float pow2_scale_to_one(float x) {
  if (!(x > 0.f) || !(x < 3.0e38f)) return 1.f;
  return ldexpf(1.f, -ilogbf(x));
}

// Power of two <= x (1 for x = 0 or non-finite x).
__device__ __forceinline__ float pow2_floor(float x) {
  if (!(x > 0.f) || !(x < 3.0e38f)) return 1.f;
  return ldexpf(1.f, ilogbf(x));
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
  // `row` points at the head's first element.  The load is unconditional (the
  // caller passes a valid row for rows past a job and masks them in the math):
  // merging a guarded load with a default would wait for the load right here.
  // The result is in memory order until arrange() puts it into slot order (kept
  // apart so that a prefetched fragment is not waited for at load time).
  __device__ static R fetch(const T* row, int g) {
    if constexpr (kSwizzle) {
      return __builtin_bit_cast(R, *reinterpret_cast<const uint4*>(row + 8 * g));
    } else if constexpr (Ty<T>::kNarrow) {
      R r;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const u16x4 p = *reinterpret_cast<const u16x4*>(row + 16 * t + 4 * g);
#pragma unroll
        for (int j = 0; j < 4; ++j) r[4 * t + j] = p[j];
      }
      return r;
    } else {
      R r;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const float4 p = *reinterpret_cast<const float4*>(row + 16 * t + 4 * g);
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
  __device__ static void put(T* row, int g, R r, bool ok) {
    if constexpr (kSwizzle) {
      uint4 w = __builtin_bit_cast(uint4, r);
      swap32(w.x, w.z);
      swap32(w.y, w.w);
      swap16(w.x, w.z);
      swap16(w.y, w.w);
      if (ok) *reinterpret_cast<uint4*>(row + 8 * g) = w;
    } else if constexpr (Ty<T>::kNarrow) {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        u16x4 p;
#pragma unroll
        for (int j = 0; j < 4; ++j) p[j] = r[4 * t + j];
        if (ok) *reinterpret_cast<u16x4*>(row + 16 * t + 4 * g) = p;
      }
    } else {
#pragma unroll
      for (int t = 0; t < NT; ++t)
        if (ok)
          *reinterpret_cast<float4*>(row + 16 * t + 4 * g) =
              make_float4(r[4 * t], r[4 * t + 1], r[4 * t + 2], r[4 * t + 3]);
    }
  }
};

struct KernelArgs {
  const PlanHeader* hdr;
  const int32_t* perm;
  const int32_t* offs;
  const Chunk* chunks;
  int32_t max_chunks, n, W, H;
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
// packed halves, phi(x) = 2^(min(x, 0) log2 e) + max(x, 0), which equals the
// definition on both branches.
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

template <typename T, int KS>
__device__ __forceinline__ Raw<T, KS> phi_frag(Raw<T, KS> x, bool ok) {
  if constexpr (std::is_same<T, _Float16>::value) {
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

// phi of a fragment (as phi_frag) and phi' at the same slots in fp32, sharing
// the exponential: with e = exp(min(x, 0)), phi(x) = e + max(x, 0), phi'(x) = e.
template <typename T, int KS>
__device__ __forceinline__ void phi_dphi(Raw<T, KS> x, bool ok, Raw<T, KS>& phi,
                                         float (&dphi)[KS]) {
  if constexpr (std::is_same<T, _Float16>::value) {
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
template <typename T, int D, int NM>
__device__ __forceinline__ void state_seg(const Slice<T, Geo<D>::KS, NM>& sb, int32_t r0,
                                          int32_t a, int32_t b, int i, int g,
                                          const Sel<T, D>& sel, State<D>& st) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  using F = Frag<T, KS>;
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  floatx4 tk[2][NT], tv[2][NT];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int32_t row = r0 + 16 * s + i;
    const bool in = sb.ok[s] && row >= a && row < b;
    const Raw<T, KS> fk = phi_frag<T, KS>(sb.x[0][s], in);
    const Raw<T, KS> vv = in ? sb.x[1][s] : F::zero();
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      tk[s][t] = F::mma(fk, sel.m[t], zero);
      tv[s][t] = F::mma(vv, sel.m[t], zero);
    }
  }
  // phi(K) is already zero outside [a, b), so z needs no row mask
  float one8[8] = {1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f};
  const Raw<T, 8> ones = Frag<T, 8>::from_f32(one8);
#pragma unroll
  for (int et = 0; et < NT; ++et) {
    const Raw<T, 8> pk = pack_rows<T>(tk[0][et], tk[1][et]);
    st.V[et] = Frag<T, 8>::mma(pk, ones, st.V[et]);
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const Raw<T, 8> pv = pack_rows<T>(tv[0][ct], tv[1][ct]);
      st.M[et][ct] = Frag<T, 8>::mma(pk, pv, st.M[et][ct]);
    }
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
};

template <typename T, int D>
__device__ __forceinline__ void make_fwd_op(const State<D>& st, FwdOp<T, D>& op, int i) {
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
}

// o = phi(q) S / (phi(q) . z) for rows [a, b) of one slice (Q is matrix QM):
// numerator and normaliser both come from the matrix cores with the same
// rounded phi(q) and the same scale sig, which cancels.
template <typename T, int D, int NM, int QM>
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
    const Raw<T, KS> bq = phi_frag<T, KS>(sb.x[QM][s], in);
    const floatx4 den = F::mma(op.Az, bq, zero);
    const float scale = recip<T>(den[0]);
    float ox[KS];
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const floatx4 d4 = F::mma(op.A[ct], bq, zero);
#pragma unroll
      for (int j = 0; j < 4; ++j) ox[4 * ct + j] = d4[j] * scale;
    }
    RowIO<T, D>::put(o + (size_t)sb.o[s] * rs + col, g, F::from_f32(ox), in);
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
// Operands of the backward's head-dim contractions for one window.  The same
// registers first hold the state operands (for the Q,dout rows) and are then
// overwritten with the state-gradient operands (for the K,V gradient rows).
template <typename T, int D>
struct BwdOp {
  Raw<T, Geo<D>::KS> A[Geo<D>::NT];  // sig S   (o = phi(q) S, tile ct)  | rho dS^T (dfk = v dS^T, tile et)
  Raw<T, Geo<D>::KS> B[Geo<D>::NT];  // sig S^T (dfq = dout S^T, tile et) | rho dS  (dv = phi(k) dS, tile ct)
  Raw<T, Geo<D>::KS> Az;             // sig z in rows 0, 4, 8, 12 (normaliser) | unused
  float z[Geo<D>::KS];               // sig z                             | dz
  float inv_scale;                   // unused                            | 1 / rho
  float bsig;                        // beta sig: phi(q) / den in the state gradients is
                                     // scaled by beta (<= min z, so beta phi(q) / den <= 1)
  float inv_beta;                    // 1 / beta
};

// The transpose of a state as operands of a head-dim contraction: slot r of lane
// (e', g) of tile et is M[16 et + e'][E(g, r)] * mul.  Goes through the wave's
// own LDS tile (row e, column c, rows padded to keep 16-byte reads aligned).
template <int D>
constexpr int kTrLd = D + 4;

template <typename T, int D>
__device__ __forceinline__ void transposed_operand(const State<D>& st, float mul, float* tile,
                                                   int i, int g,
                                                   Raw<T, Geo<D>::KS> (&out)[Geo<D>::NT]) {
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
  }
  wave_lds_sync();   // the tile may be written again by the next call
}

template <typename T, int D>
__device__ __forceinline__ void make_state_op(const State<D>& st, BwdOp<T, D>& op, float* tile,
                                              int i, int g) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  const float sig = Ty<T>::kNarrow ? pow2_scale_to_one(st.absmax()) : 1.f;
#pragma unroll
  for (int ct = 0; ct < NT; ++ct) {
    floatx4 col[NT];
#pragma unroll
    for (int et = 0; et < NT; ++et) col[et] = st.M[et][ct];
    op.A[ct] = tiles_operand<T, D>(col, sig);
  }
  transposed_operand<T, D>(st, sig, tile, i, g, op.B);
  float zmin = 3.0e38f;
  const float zmul = (i & 3) == 0 ? sig : 0.f;
  float zx[KS];
#pragma unroll
  for (int r = 0; r < KS; ++r) {
    const float z = st.V[r >> 2][r & 3];
    zmin = fminf(zmin, z);
    op.z[r] = z * sig;
    zx[r] = z * zmul;
  }
  op.Az = Frag<T, KS>::from_f32(zx);
  // phi(q)_e / den <= 1 / z_e <= 1 / min z, so beta phi(q) / den <= 1
  const float beta = Ty<T>::kNarrow ? pow2_floor(wave_reduce<false>(zmin)) : 1.f;
  op.bsig = beta * sig;
  op.inv_beta = 1.f / beta;
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
  transposed_operand<T, D>(st, mul, tile, i, g, op.A);
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
// normaliser comes from the matrix cores (den' = sig den); with sig folded into
// z, dphi(q) = (sig dfq - dot sig z) / den'.
template <typename T, int D, int NM, int QI, int DI>
__device__ __forceinline__ void qgrad_seg(const Slice<T, Geo<D>::KS, NM>& sb, int32_t r0,
                                          int32_t a, int32_t b, int i, int g,
                                          const Sel<T, D>& sel, const BwdOp<T, D>& op, T* dq,
                                          size_t rs, int col, State<D>& gs) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  using F = Frag<T, KS>;
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  Raw<T, KS> xr[2], dr[2], nd[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int32_t row = r0 + 16 * s + i;
    const bool in = sb.ok[s] && row >= a && row < b;
    dr[s] = in ? sb.x[DI][s] : F::zero();
    xr[s] = F::zero();
    nd[s] = F::zero();
    if (!sub_overlaps(r0, s, a, b)) continue;
    Raw<T, KS> bq;
    float dphq[KS], fq[KS], dox[KS];
    phi_dphi<T, KS>(sb.x[QI][s], in, bq, dphq);
    F::to_f32(bq, fq);
    F::to_f32(dr[s], dox);
    const floatx4 den4 = F::mma(op.Az, bq, zero);
    const float rden = recip<T>(in ? den4[0] : 1.f);
    float dot = 0.f;
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const floatx4 d4 = F::mma(op.A[ct], bq, zero);
#pragma unroll
      for (int j = 0; j < 4; ++j) dot += dox[4 * ct + j] * d4[j];
    }
    dot = sum_groups(dot) * rden;  // lane exchange: every lane takes part
    if (!in) dot = 0.f;
    float dqx[KS];
#pragma unroll
    for (int et = 0; et < NT; ++et) {
      const floatx4 d4 = F::mma(op.B[et], dr[s], zero);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = 4 * et + j;
        dqx[r] = (d4[j] - dot * op.z[r]) * rden * dphq[r];
      }
    }
    RowIO<T, D>::put(dq + (size_t)sb.o[s] * rs + col, g, F::from_f32(dqx), in);
    float xs[KS], ns[KS];
    const float w = op.bsig * rden;
#pragma unroll
    for (int r = 0; r < KS; ++r) {
      xs[r] = fq[r] * w;
      ns[r] = -dot;
    }
    xr[s] = F::from_f32(xs);
    nd[s] = F::from_f32(ns);
  }
  floatx4 tx[2][NT], td[2][NT], tn[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      tx[s][t] = F::mma(xr[s], sel.m[t], zero);
      td[s][t] = F::mma(dr[s], sel.m[t], zero);
    }
    tn[s] = F::mma(nd[s], sel.m[0], zero);
  }
  const Raw<T, 8> pn = pack_rows<T>(tn[0], tn[1]);
#pragma unroll
  for (int et = 0; et < NT; ++et) {
    const Raw<T, 8> px = pack_rows<T>(tx[0][et], tx[1][et]);
    gs.V[et] = Frag<T, 8>::mma(px, pn, gs.V[et]);
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const Raw<T, 8> pd = pack_rows<T>(td[0][ct], td[1][ct]);
      gs.M[et][ct] = Frag<T, 8>::mma(px, pd, gs.M[et][ct]);
    }
  }
}

// Rows [a, b) of one slice: dk = (v dS^T + dz) phi'(k), dv = phi(k) dS.
template <typename T, int D, int NM>
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
    phi_dphi<T, KS>(sb.x[0][s], in, fk, dphk);
    float dkx[KS], dvx[KS];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const floatx4 a4 = F::mma(op.A[t], sb.x[1][s], zero);
      const floatx4 b4 = F::mma(op.B[t], fk, zero);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = 4 * t + j;
        dkx[r] = (a4[j] * op.inv_scale + op.z[r]) * dphk[r];
        dvx[r] = b4[j] * op.inv_scale;
      }
    }
    RowIO<T, D>::put(dk + (size_t)sb.o[s] * rs + col, g, F::from_f32(dkx), in);
    RowIO<T, D>::put(dv + (size_t)sb.o[s] * rs + col, g, F::from_f32(dvx), in);
  }
}


// ------------------------------------------------------------ job streams
// A wave walks the windows of its chunk; each window is a run of 32-row jobs per
// phase (forward: 0 = K,V state, 1 = Q apply; backward: 0 = K,V state,
// 1 = Q,dout, 2 = K,V gradients).  Jobs are software-pipelined: while job t
// computes, the rows of job t+1 and t+2 are in flight and the permutation
// entries of job t+3 are being fetched.
struct Job {
  int32_t w;       // window (-1: stream finished)
  int32_t ws, we;  // the window's rows, clipped to the chunk
  int32_t r0;      // first row of this job
  int32_t phase;
};

// The windows of a chunk, 64 at a time in registers: lane l holds the rows of
// window wp + l clipped to the chunk, and a ballot marks the non-empty ones, so
// that moving to the next window is a few scalar instructions, not a chain of
// dependent loads of the offsets (chunks of small windows also hold many empty
// ones).
struct Stream {
  const int32_t* offs;
  int32_t rb, re, wend;
  int32_t wp;      // first window of the loaded page
  int32_t a, b;    // rows of window wp + lane, clipped to [rb, re)
  uint64_t live;   // lanes whose window is non-empty
  int lane;
  __device__ __forceinline__ void load_page(int32_t w0) {
    wp = w0;
    const int32_t w = wp + lane;
    a = b = 0;
    if (w < wend) {
      a = max(offs[w], rb);
      b = min(offs[w + 1], re);
    }
    live = __ballot(a < b);
  }
  __device__ __forceinline__ bool next_window(Job& j) {
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
      load_page(wp + 64);
    }
    j.w = -1;
    return false;
  }
  __device__ __forceinline__ Job first(int32_t wb) {
    load_page(wb);
    Job j;
    j.w = wb - 1;
    j.phase = 0;
    j.ws = j.we = j.r0 = 0;
    if (next_window(j)) j.r0 = j.ws;
    return j;
  }
  template <int NPH>
  __device__ __forceinline__ Job next(Job j) {
    if (j.w < 0) return j;
    j.r0 += kSliceRows;
    if (j.r0 < j.we) return j;
    if (++j.phase < NPH) {
      j.r0 = j.ws;
      return j;
    }
    j.phase = 0;
    if (next_window(j)) j.r0 = j.ws;
    return j;
  }
};

template <typename T, int D>
using JobBuf = Slice<T, Geo<D>::KS, 2>;

// A page of the chunk's permutation, held by the wave: register m of lane l is
// the original row of sorted row pb + 64 m + l.  Jobs take their rows from the
// page with lane permutes; a job outside the page (windows longer than it)
// first reloads the page at its own first row.  The reload waits for its loads
// inside its own branch, so the common path never waits on the permutation and
// the prefetched rows stay in flight.
#ifndef SLA_PERM_REGS
#define SLA_PERM_REGS 4
#endif
constexpr int kPermRegs = SLA_PERM_REGS;

struct PermRegs {
  const int32_t* perm;  // null: identity (rows already window-sorted)
  int32_t re;           // end of the chunk's rows
  int32_t pb;           // first sorted row of the page
  int32_t r[kPermRegs];
  __device__ __forceinline__ void load(int32_t pb_, int lane) {
    pb = pb_;
    int32_t x[kPermRegs];
#pragma unroll
    for (int m = 0; m < kPermRegs; ++m) {
      const int32_t row = pb + 64 * m + lane;
      x[m] = perm ? perm[row < re ? row : pb] : row;
    }
#pragma unroll
    for (int m = 0; m < kPermRegs; ++m) {
      asm volatile("" : "+v"(x[m]));  // consumed here: the wait stays in this branch
      r[m] = x[m];
    }
  }
};

// Original rows of a job's two sub-tiles (o = 0 and ok = false past the job).
__device__ __forceinline__ void job_rows(const Job& j, PermRegs& pr, int lane, int32_t (&o)[2],
                                         bool (&ok)[2]) {
  if (j.w >= 0 && (j.r0 < pr.pb || j.r0 + kSliceRows > pr.pb + 64 * kPermRegs)) pr.load(j.r0, lane);
  const int i = lane & 15;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int32_t row = j.r0 + 16 * s + i;
    const int32_t rel = row - pr.pb;
    int32_t x = 0;
#pragma unroll
    for (int m = 0; m < kPermRegs; ++m) {
      const int32_t t = __builtin_amdgcn_ds_bpermute((rel & 63) << 2, pr.r[m]);
      if ((rel >> 6) == m) x = t;
    }
    ok[s] = j.w >= 0 && row < j.we;
    o[s] = ok[s] ? x : 0;
  }
}

// Rows of a job -> the job's two matrices (a, b; b null: the second fragment is
// left as it is, the job's math does not read it).  Rows past the job read row
// 0 (the math masks them; n >= 1 whenever a kernel runs).
template <typename T, int D>
__device__ __forceinline__ void job_load(JobBuf<T, D>& jb, const int32_t (&o)[2],
                                         const bool (&ok)[2], const T* a, const T* b, int32_t n,
                                         size_t rs, int col, int g) {
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    jb.ok[s] = ok[s] && (uint32_t)o[s] < (uint32_t)n;
    jb.o[s] = jb.ok[s] ? o[s] : 0;
    jb.x[0][s] = RowIO<T, D>::fetch(a + (size_t)jb.o[s] * rs + col, g);
    if (b) jb.x[1][s] = RowIO<T, D>::fetch(b + (size_t)jb.o[s] * rs + col, g);
  }
}

// Slot order for the rows of the job about to be computed.
template <typename T, int D>
__device__ __forceinline__ void job_arrange(JobBuf<T, D>& jb) {
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    RowIO<T, D>::arrange(jb.x[0][s]);
    RowIO<T, D>::arrange(jb.x[1][s]);
  }
}

template <typename T, int D>
__device__ __forceinline__ Stream chunk_stream(const KernelArgs& a, int32_t c, int32_t& wb,
                                               int lane) {
  const Chunk ch = a.chunks[c];
  Stream st;
  st.lane = lane;
  st.offs = a.offs;
  st.rb = max(0, min(ch.row_begin, a.n));
  st.re = max(st.rb, min(ch.row_end, a.n));
  st.wend = max(0, min(ch.win_end, a.W));
  wb = max(0, min(ch.win_begin, st.wend));
  return st;
}

// ------------------------------------------------------------------ forward
template <typename T, int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kWpe<T, SLA_FWD_WPE>)))
void k_sla_fwd(KernelArgs a, const T* __restrict__ q, const T* __restrict__ k,
               const T* __restrict__ v, T* __restrict__ o) {
  const int lane = lane_id(), wv = threadIdx.x >> 6;
  const int h = blockIdx.y * kWaves + wv;
  if (h >= a.H) return;
  const PlanHeader* hdr = a.hdr;
  if (hdr->magic != kPlanMagic || hdr->n != a.n || hdr->num_windows != a.W) return;
  const int32_t c = blockIdx.x;
  if (c >= min(hdr->n_chunks, a.max_chunks)) return;
  const int32_t* perm = hdr->csr ? nullptr : a.perm;
  const int i = lane & 15, g = lane >> 4;
  const size_t rs = (size_t)a.H * D;
  const int col = h * D;
  const int32_t n = a.n;
  const Sel<T, D> sel(i, g);
  int32_t wb;
  Stream str = chunk_stream<T, D>(a, c, wb, lane);
  PermRegs pr;
  pr.perm = perm;
  pr.re = str.re;
  pr.load(str.rb, lane);
  auto load_job = [&](JobBuf<T, D>& jb, const Job& j) {
    int32_t o[2];
    bool ok[2];
    job_rows(j, pr, lane, o, ok);
    job_load<T, D>(jb, o, ok, j.phase == 0 ? k : q, j.phase == 0 ? v : (const T*)nullptr, n, rs,
                   col, g);
  };

  // Three buffers used in turn (the loop is unrolled by three so that rows in
  // flight are never copied between registers, which would wait for them).
  Job j0 = str.first(wb);
  Job j1 = str.next<2>(j0);
  Job j2 = str.next<2>(j1);
  JobBuf<T, D> b0, b1, b2;
  load_job(b0, j0);
  load_job(b1, j1);
  State<D> st;
  FwdOp<T, D> op;
  auto step = [&](JobBuf<T, D>& cur, JobBuf<T, D>& nxt) {
    load_job(nxt, j2);
    job_arrange<T, D>(cur);
    if (j0.phase == 0) {
      if (j0.r0 == j0.ws) st.clear();
      state_seg<T, D, 2>(cur, j0.r0, j0.ws, j0.we, i, g, sel, st);
      if (j0.r0 + kSliceRows >= j0.we) make_fwd_op<T, D>(st, op, i);
    } else {
      apply_seg<T, D, 2, 0>(cur, j0.r0, j0.ws, j0.we, i, g, op, o, rs, col);
    }
    j0 = j1;
    j1 = j2;
    j2 = str.next<2>(j2);
  };
  for (;;) {
    if (j0.w < 0) break;
    step(b0, b2);
    if (j0.w < 0) break;
    step(b1, b0);
    if (j0.w < 0) break;
    step(b2, b1);
  }
}

// ----------------------------------------------------------------- backward
template <typename T, int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kWpe<T, SLA_BWD_WPE>)))
void k_sla_bwd(KernelArgs a, const T* __restrict__ q, const T* __restrict__ k,
               const T* __restrict__ v, const T* __restrict__ dout, T* __restrict__ dq,
               T* __restrict__ dk, T* __restrict__ dv) {
  const int lane = lane_id(), wv = threadIdx.x >> 6;
  const int h = blockIdx.y * kWaves + wv;
  if (h >= a.H) return;
  const PlanHeader* hdr = a.hdr;
  if (hdr->magic != kPlanMagic || hdr->n != a.n || hdr->num_windows != a.W) return;
  const int32_t c = blockIdx.x;
  if (c >= min(hdr->n_chunks, a.max_chunks)) return;
  const int32_t* perm = hdr->csr ? nullptr : a.perm;
  const int i = lane & 15, g = lane >> 4;
  const size_t rs = (size_t)a.H * D;
  const int col = h * D;
  const int32_t n = a.n;
  const Sel<T, D> sel(i, g);
  int32_t wb;
  Stream str = chunk_stream<T, D>(a, c, wb, lane);
  PermRegs pr;
  pr.perm = perm;
  pr.re = str.re;
  pr.load(str.rb, lane);
  auto load_job = [&](JobBuf<T, D>& jb, const Job& j) {
    int32_t o[2];
    bool ok[2];
    job_rows(j, pr, lane, o, ok);
    job_load<T, D>(jb, o, ok, j.phase == 1 ? q : k, j.phase == 1 ? dout : v, n, rs, col, g);
  };

  Job j0 = str.first(wb);
  Job j1 = str.next<3>(j0);
  Job j2 = str.next<3>(j1);
  JobBuf<T, D> b0, b1, b2;
  load_job(b0, j0);
  load_job(b1, j1);
  State<D> st;  // phase 0: S, z ; phase 1: beta dS, beta dz
  __shared__ float s_tr[kWaves][D * kTrLd<D>];  // transposes, one tile per wave
  float* tile = s_tr[wv];
  BwdOp<T, D> op;
  auto step = [&](JobBuf<T, D>& cur, JobBuf<T, D>& nxt) {
    load_job(nxt, j2);
    job_arrange<T, D>(cur);
    const bool first = j0.r0 == j0.ws, last = j0.r0 + kSliceRows >= j0.we;
    if (j0.phase == 0) {
      if (first) st.clear();
      state_seg<T, D, 2>(cur, j0.r0, j0.ws, j0.we, i, g, sel, st);
      if (last) make_state_op<T, D>(st, op, tile, i, g);
    } else if (j0.phase == 1) {
      if (first) st.clear();
      qgrad_seg<T, D, 2, 0, 1>(cur, j0.r0, j0.ws, j0.we, i, g, sel, op, dq, rs, col, st);
      if (last) make_grad_op<T, D>(st, op.inv_beta, op, tile, i, g);
    } else {
      kgrad_seg<T, D, 2>(cur, j0.r0, j0.ws, j0.we, i, g, op, dk, dv, rs, col);
    }
    j0 = j1;
    j1 = j2;
    j2 = str.next<3>(j2);
  };
  for (;;) {
    if (j0.w < 0) break;
    step(b0, b2);
    if (j0.w < 0) break;
    step(b1, b0);
    if (j0.w < 0) break;
    step(b2, b1);
  }
}

// ------------------------------------------------------------ host launchers
static inline int grid_x(int32_t max_chunks) {
  return max_chunks < 1 ? 1 : max_chunks;
}

static KernelArgs kernel_args(const void* plan, int32_t n, int32_t W, int32_t H) {
  const PlanLayout lay = plan_layout(n, W);
  const char* base = static_cast<const char*>(plan);
  KernelArgs a;
  a.hdr = reinterpret_cast<const PlanHeader*>(base + lay.header);
  a.perm = reinterpret_cast<const int32_t*>(base + lay.perm);
  a.offs = reinterpret_cast<const int32_t*>(base + lay.offsets);
  a.chunks = reinterpret_cast<const Chunk*>(base + lay.chunks);
  a.max_chunks = lay.max_chunks;
  a.n = n;
  a.W = W;
  a.H = H;
  return a;
}

template <typename T, int D>
static hipError_t fwd_impl(const void* plan, int32_t n, int32_t W, int32_t H, const void* q,
                           const void* k, const void* v, void* o, hipStream_t stream) {
  const KernelArgs a = kernel_args(plan, n, W, H);
  const int waves = H < kWaves ? H : kWaves;
  hipLaunchKernelGGL((k_sla_fwd<T, D>), dim3(grid_x(a.max_chunks), (H + kWaves - 1) / kWaves),
                     dim3(64 * waves), 0, stream, a, static_cast<const T*>(q),
                     static_cast<const T*>(k), static_cast<const T*>(v), static_cast<T*>(o));
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t bwd_impl(const void* plan, int32_t n, int32_t W, int32_t H, const void* q,
                           const void* k, const void* v, const void* dout, void* dq, void* dk,
                           void* dv, hipStream_t stream) {
  const KernelArgs a = kernel_args(plan, n, W, H);
  const int waves = H < kWaves ? H : kWaves;
  hipLaunchKernelGGL((k_sla_bwd<T, D>), dim3(grid_x(a.max_chunks), (H + kWaves - 1) / kWaves),
                     dim3(64 * waves), 0, stream, a, static_cast<const T*>(q),
                     static_cast<const T*>(k), static_cast<const T*>(v),
                     static_cast<const T*>(dout), static_cast<T*>(dq), static_cast<T*>(dk),
                     static_cast<T*>(dv));
  return hipGetLastError();
}

// dtype: 0 f32, 1 f16, 2 bf16
hipError_t launch_forward(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                          const void* q, const void* k, const void* v, void* o,
                          hipStream_t stream) {
  if (d == 32) {
    if (dtype == 0) return fwd_impl<float, 32>(plan, n, W, H, q, k, v, o, stream);
    if (dtype == 1) return fwd_impl<_Float16, 32>(plan, n, W, H, q, k, v, o, stream);
    return fwd_impl<bf16_t, 32>(plan, n, W, H, q, k, v, o, stream);
  }
  if (dtype == 0) return fwd_impl<float, 16>(plan, n, W, H, q, k, v, o, stream);
  if (dtype == 1) return fwd_impl<_Float16, 16>(plan, n, W, H, q, k, v, o, stream);
  return fwd_impl<bf16_t, 16>(plan, n, W, H, q, k, v, o, stream);
}

hipError_t launch_backward(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                           const void* q, const void* k, const void* v, const void* dout,
                           void* dq, void* dk, void* dv, hipStream_t stream) {
  if (d == 32) {
    if (dtype == 0) return bwd_impl<float, 32>(plan, n, W, H, q, k, v, dout, dq, dk, dv, stream);
    if (dtype == 1) return bwd_impl<_Float16, 32>(plan, n, W, H, q, k, v, dout, dq, dk, dv, stream);
    return bwd_impl<bf16_t, 32>(plan, n, W, H, q, k, v, dout, dq, dk, dv, stream);
  }
  if (dtype == 0) return bwd_impl<float, 16>(plan, n, W, H, q, k, v, dout, dq, dk, dv, stream);
  if (dtype == 1) return bwd_impl<_Float16, 16>(plan, n, W, H, q, k, v, dout, dq, dk, dv, stream);
  return bwd_impl<bf16_t, 16>(plan, n, W, H, q, k, v, dout, dq, dk, dv, stream);
}

}  // namespace sla

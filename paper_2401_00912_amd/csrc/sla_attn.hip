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
// Feature maps (template parameter PHI): elu(x) + 1 (Eq. (3) as read from the
// linear-transformer paper that Sec. 3.2 cites), or ReLU with phi'(0) = 0 (the
// "Efficient Attn" variant of Sec. 4.5 / Tab. 7).  Either may add eps >= 0 to the
// normaliser: o = phi(q) S / (phi(q) . z + eps).
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
__device__ __forceinline__ float pow2_scale_to_one(float x) {
  if (!(x > 0.f) || !(x < 3.0e38f)) return 1.f;
  return ldexpf(1.f, min(-ilogbf(x), 126));
}

// Power of two <= x (1 for x = 0 or non-finite x; at least 2^-126).
__device__ __forceinline__ float pow2_floor(float x) {
  if (!(x > 0.f) || !(x < 3.0e38f)) return 1.f;
  return ldexpf(1.f, max(ilogbf(x), -126));
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
  floatx4 tk[2][NT], tv[2][NT];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int32_t row = r0 + 16 * s + i;
    const bool in = sb.ok[s] && row >= a && row < b;
    const Raw<T, KS> fk = phi_frag<T, KS, PHI>(sb.x[0][s], in);
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
    RowIO<T, D>::put(row_at(o, sb.o[s], rs, col), g, F::from_f32(ox), in);
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
// bf16 keeps 8 significant bits, so the backward carries two operands as a
// sum of two bf16 values (high part and rounding residual, 16 bits together):
// -dout.o in the dz accumulation and dS^T in dk = (v dS^T + dz) phi'(k), the
// two terms that cancel there.  fp16 (11 bits) and fp32 need no split.
template <typename T>
constexpr bool kSplitGrad = std::is_same<T, bf16_t>::value;

// Operands of the backward's head-dim contractions for one window.  The same
// registers first hold the state operands (for the Q,dout rows) and are then
// overwritten with the state-gradient operands (for the K,V gradient rows).
template <typename T, int D>
struct BwdOp {
  Raw<T, Geo<D>::KS> A[Geo<D>::NT];  // sig S   (o = phi(q) S, tile ct)  | rho dS^T (dfk = v dS^T, tile et)
  Raw<T, Geo<D>::KS> B[Geo<D>::NT];  // sig S^T (dfq = dout S^T, tile et) | rho dS  (dv = phi(k) dS, tile ct)
  Raw<T, Geo<D>::KS> Az;             // sig z in rows 0, 4, 8, 12 (normaliser) | unused
  float z[Geo<D>::KS];               // sig z (as rounded in Az)          | dz
  float inv_scale;                   // unused                            | 1 / rho
  float bsig;                        // beta sig: phi(q) / den in the state gradients is
                                     // scaled by beta (<= min z, so beta phi(q) / den <= 1)
  float inv_beta;                    // 1 / beta
  float seps;                        // sig eps
  Raw<T, Geo<D>::KS> Al[kSplitGrad<T> ? Geo<D>::NT : 1];  // unused | residual of A (bf16)
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
#pragma unroll
  for (int ct = 0; ct < NT; ++ct) {
    floatx4 col[NT];
#pragma unroll
    for (int et = 0; et < NT; ++et) col[et] = st.M[et][ct];
    op.A[ct] = tiles_operand<T, D>(col, sig);
  }
  transposed_operand<T, D>(st, sig, tile, i, g, op.B);
  // op.z holds sig z rounded exactly as in the normaliser operand Az: dq subtracts
  // (dout.o) z from dout S^T, and for a row whose normaliser is mostly eps the two
  // terms cancel to eps / den; the same z on both sides keeps that residual exact
  float zmin = 3.0e38f;
  float zx[KS];
#pragma unroll
  for (int r = 0; r < KS; ++r) {
    const float z = st.V[r >> 2][r & 3];
    if (PHI != kPhiRelu || z > 0.f) zmin = fminf(zmin, z);
    const float zs = Ty<T>::kNarrow ? u16_to_f32<T>(f32_to_u16<T>(z * sig)) : z * sig;
    op.z[r] = zs;
    zx[r] = (i & 3) == 0 ? zs : 0.f;
  }
  op.Az = Frag<T, KS>::from_f32(zx);
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
    float dphq[KS], fq[KS], dox[KS];
    phi_dphi<T, KS, PHI>(sb.x[QI][s], in, bq, dphq);
    F::to_f32(bq, fq);
    F::to_f32(dr[s], dox);
    const floatx4 den4 = F::mma(op.Az, bq, zero);
    const float rden = recip<T>(in ? den4[0] + op.seps : 1.f);
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
    RowIO<T, D>::put(row_at(dq, sb.o[s], rs, col), g, F::from_f32(dqx), in);
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
  floatx4 tx[2][NT], td[2][NT], tn[2], tl[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      tx[s][t] = F::mma(xr[s], sel.m[t], zero);
      td[s][t] = F::mma(dr[s], sel.m[t], zero);
    }
    tn[s] = F::mma(nd[s], sel.m[0], zero);
    if constexpr (SP) tl[s] = F::mma(nl[s], sel.m[0], zero);
  }
  const Raw<T, 8> pn = pack_rows<T>(tn[0], tn[1]);
  Raw<T, 8> pl;
  if constexpr (SP) pl = pack_rows<T>(tl[0], tl[1]);
#pragma unroll
  for (int et = 0; et < NT; ++et) {
    const Raw<T, 8> px = pack_rows<T>(tx[0][et], tx[1][et]);
    gs.V[et] = Frag<T, 8>::mma(px, pn, gs.V[et]);
    if constexpr (SP) gs.V[et] = Frag<T, 8>::mma(px, pl, gs.V[et]);
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const Raw<T, 8> pd = pack_rows<T>(td[0][ct], td[1][ct]);
      gs.M[et][ct] = Frag<T, 8>::mma(px, pd, gs.M[et][ct]);
    }
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
    RowIO<T, D>::put(row_at(dk, sb.o[s], rs, col), g, F::from_f32(dkx), in);
    RowIO<T, D>::put(row_at(dv, sb.o[s], rs, col), g, F::from_f32(dvx), in);
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
        if (live) bk.j[jj].x[m][s] = RowIO<T, D>::fetch(row_at(mats[m], bk.j[jj].o[s], rs, col), g);
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

// ------------------------------------------------------------------ forward
template <typename T, int D, int PHI>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kWpe<T, SLA_FWD_WPE>)))
void k_sla_fwd(KernelArgs a, const T* __restrict__ q, const T* __restrict__ k,
               const T* __restrict__ v, T* __restrict__ o) {
  constexpr int KT = kStateTiles<D>;
  __shared__ floatx4 s_part[kWaves * KT * 64];  // partial states of a long window
  const int lane = lane_id();
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const PlanHeader* hdr = a.hdr;
  if (hdr->magic != kPlanMagic || hdr->n != a.n || hdr->num_windows != a.W) return;
  const Items it = work_items(a, hdr);
  const int32_t* perm = hdr->csr ? nullptr : a.perm;
  const int i = lane & 15, g = lane >> 4;
  const size_t rs = (size_t)a.H * D;
  const int32_t n = a.n, G = gridDim.x;
  const Sel<T, D> sel(i, g);
  const T* const mats[3] = {k, v, q};
  constexpr unsigned kKV = 3u, kQ = 4u, kAll = 7u;

  int32_t item = blockIdx.x;
  Pending cur;
  {
    const Slot sl = item_slot(it, item, wv);
    pending_request(cur, a, sl, slot_entry(a, sl), wv, perm, lane);
  }
  Slot nsl = item_slot(it, item + G, wv);
  int4 ne = slot_entry(a, nsl);
  while (item < it.total) {
    const WaveWork ww = cur.ww;
    const int col = ww.h * D;
    // a range of more than kBlockRows rows (a quarter of a very long window) is
    // streamed through the block: K, V for the state, then Q for the outputs
    const bool resident = ww.rb - ww.ra <= kBlockRows;
    const unsigned first = resident ? kAll : kKV;
    Block<T, D, 3> bk;
    if (ww.kind != 0) block_fetch<T, D, 3>(bk, cur.br, ww.ra, ww.rb, n, mats, first, rs, col, g);
    // the next item: its rows and windows are requested now, its successor's entry too
    Pending nxt;
    pending_request(nxt, a, nsl, ne, wv, perm, lane);
    nsl = item_slot(it, item + 2 * G, wv);
    ne = slot_entry(a, nsl);

    block_arrange<T, D, 3>(bk, first);
    WinIter wi;
    for (bool more = wi.first(ww, cur.str); more; more = wi.next(ww, cur.str)) {
      const int32_t wa = wi.wc.ws, wb = wi.wc.we;
      State<D> st;
      st.clear();
      for (int32_t base = ww.ra; base < ww.rb; base += kBlockRows) {
        if (base != ww.ra) {
          BlockRows br;
          block_rows(br, base, ww.rb, perm, lane);
          block_fetch<T, D, 3>(bk, br, base, ww.rb, n, mats, kKV, rs, col, g);
          block_arrange<T, D, 3>(bk, kKV);
        }
#pragma unroll
        for (int jj = 0; jj < kBlockJobs; ++jj) {
          const int32_t r0 = base + kSliceRows * jj;
          if (job_overlaps(r0, wa, wb)) state_seg<T, D, 3, PHI>(bk.j[jj], r0, wa, wb, i, g, sel, st);
        }
      }
      if (wi.shared) {
        publish<D>(st, s_part + wv * KT * 64, lane);
        lds_barrier();
        combine<D>(st, s_part, lane, wv, ww.pair);
        lds_barrier();  // the slots may be written by the next long item
      }
      FwdOp<T, D> op;
      make_fwd_op<T, D>(st, op, i, a.eps);
      for (int32_t base = ww.ra; base < ww.rb; base += kBlockRows) {
        if (!resident) {
          BlockRows br;
          block_rows(br, base, ww.rb, perm, lane);
          block_fetch<T, D, 3>(bk, br, base, ww.rb, n, mats, kQ, rs, col, g);
          block_arrange<T, D, 3>(bk, kQ);
        }
#pragma unroll
        for (int jj = 0; jj < kBlockJobs; ++jj) {
          const int32_t r0 = base + kSliceRows * jj;
          if (job_overlaps(r0, wa, wb)) apply_seg<T, D, 3, 2, PHI>(bk.j[jj], r0, wa, wb, i, g, op, o, rs, col);
        }
      }
    }
    item += G;
    cur = nxt;
  }
}

// ----------------------------------------------------------------- backward
// Per window: state S, z from K, V; then dq and the state gradients from Q, dout;
// then dk, dv from K, V (held in registers since the first phase).
template <typename T, int D, int PHI>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kWpe<T, SLA_BWD_WPE>)))
void k_sla_bwd(KernelArgs a, const T* __restrict__ q, const T* __restrict__ k,
               const T* __restrict__ v, const T* __restrict__ dout, T* __restrict__ dq,
               T* __restrict__ dk, T* __restrict__ dv) {
  constexpr int KT = kStateTiles<D>;
  __shared__ floatx4 s_part[2][kWaves * KT * 64];  // partial S, z / dS, dz of a long window
  __shared__ float s_tr[kWaves][D * kTrLd<D>];     // transposes, one tile per wave
  const int lane = lane_id();
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const PlanHeader* hdr = a.hdr;
  if (hdr->magic != kPlanMagic || hdr->n != a.n || hdr->num_windows != a.W) return;
  const Items it = work_items(a, hdr);
  const int32_t* perm = hdr->csr ? nullptr : a.perm;
  const int i = lane & 15, g = lane >> 4;
  const size_t rs = (size_t)a.H * D;
  const int32_t n = a.n, G = gridDim.x;
  const Sel<T, D> sel(i, g);
  float* tile = s_tr[wv];
  const T* const mats[4] = {k, v, q, dout};
  constexpr unsigned kKV = 3u, kQD = 12u, kAll = 15u;

  int32_t item = blockIdx.x;
  Pending cur;
  {
    const Slot sl = item_slot(it, item, wv);
    pending_request(cur, a, sl, slot_entry(a, sl), wv, perm, lane);
  }
  Slot nsl = item_slot(it, item + G, wv);
  int4 ne = slot_entry(a, nsl);
  while (item < it.total) {
    const WaveWork ww = cur.ww;
    const int col = ww.h * D;
    const bool resident = ww.rb - ww.ra <= kBlockRows;
    const unsigned first = resident ? kAll : kKV;
    Block<T, D, 4> bk;
    if (ww.kind != 0) block_fetch<T, D, 4>(bk, cur.br, ww.ra, ww.rb, n, mats, first, rs, col, g);
    Pending nxt;
    pending_request(nxt, a, nsl, ne, wv, perm, lane);
    nsl = item_slot(it, item + 2 * G, wv);
    ne = slot_entry(a, nsl);

    block_arrange<T, D, 4>(bk, first);
    WinIter wi;
    for (bool more = wi.first(ww, cur.str); more; more = wi.next(ww, cur.str)) {
      const int32_t wa = wi.wc.ws, wb = wi.wc.we;
      State<D> st;  // S, z ; then beta dS, beta dz
      BwdOp<T, D> op;
      // phase 0: S, z
      st.clear();
      for (int32_t base = ww.ra; base < ww.rb; base += kBlockRows) {
        if (base != ww.ra) {
          BlockRows br;
          block_rows(br, base, ww.rb, perm, lane);
          block_fetch<T, D, 4>(bk, br, base, ww.rb, n, mats, kKV, rs, col, g);
          block_arrange<T, D, 4>(bk, kKV);
        }
#pragma unroll
        for (int jj = 0; jj < kBlockJobs; ++jj) {
          const int32_t r0 = base + kSliceRows * jj;
          if (job_overlaps(r0, wa, wb)) state_seg<T, D, 4, PHI>(bk.j[jj], r0, wa, wb, i, g, sel, st);
        }
      }
      if (wi.shared) {
        publish<D>(st, s_part[0] + wv * KT * 64, lane);
        lds_barrier();
        combine<D>(st, s_part[0], lane, wv, ww.pair);
      }
      make_state_op<T, D, PHI>(st, op, tile, i, g, a.eps);
      // phase 1: dq and beta dS, beta dz
      st.clear();
      for (int32_t base = ww.ra; base < ww.rb; base += kBlockRows) {
        if (!resident) {
          BlockRows br;
          block_rows(br, base, ww.rb, perm, lane);
          block_fetch<T, D, 4>(bk, br, base, ww.rb, n, mats, kQD, rs, col, g);
          block_arrange<T, D, 4>(bk, kQD);
        }
#pragma unroll
        for (int jj = 0; jj < kBlockJobs; ++jj) {
          const int32_t r0 = base + kSliceRows * jj;
          if (job_overlaps(r0, wa, wb))
            qgrad_seg<T, D, 4, 2, 3, PHI>(bk.j[jj], r0, wa, wb, i, g, sel, op, dq, rs, col, st);
        }
      }
      if (wi.shared) {
        // slot set 1 is free: its last readers passed the barrier above before
        // this item's set-0 reads ended (sets alternate within every long item)
        publish<D>(st, s_part[1] + wv * KT * 64, lane);
        lds_barrier();
        combine<D>(st, s_part[1], lane, wv, ww.pair);
      }
      make_grad_op<T, D>(st, op.inv_beta, op, tile, i, g);
      // phase 2: dk, dv
      for (int32_t base = ww.ra; base < ww.rb; base += kBlockRows) {
        if (!resident) {
          BlockRows br;
          block_rows(br, base, ww.rb, perm, lane);
          block_fetch<T, D, 4>(bk, br, base, ww.rb, n, mats, kKV, rs, col, g);
          block_arrange<T, D, 4>(bk, kKV);
        }
#pragma unroll
        for (int jj = 0; jj < kBlockJobs; ++jj) {
          const int32_t r0 = base + kSliceRows * jj;
          if (job_overlaps(r0, wa, wb)) kgrad_seg<T, D, 4, PHI>(bk.j[jj], r0, wa, wb, i, g, op, dk, dv, rs, col);
        }
      }
    }
    item += G;
    cur = nxt;
  }
}

// ------------------------------------------- projection fused into the forward
// Sec. 3.2: one shared projection layer maps every voxel to Q, K and V before the
// attention, and the block projects the attention output back.  The fused
// forward gathers the voxel features X (whole rows of C channels) and computes
// its head's q, k, v on the matrix cores, so q, k, v never reach HBM:
//   q_e = sum_c X[c] W_qkv[q row e of head h][c] + b   (likewise k, v)
// A contraction over the C channels in 32-wide blocks: with the weight rows as
// the first operand and the feature rows as the second, lane (i, g) receives
// element 16 t + 4 g + j of its row i, which is already the row-fragment slot
// order E(g, r) of the attention math.  The head's weight rows live in LDS for
// the whole launch: a workgroup keeps one head (items are numbered so that
// workgroup b always gets head (b / 8) mod H, with a grid that is a multiple of
// 8 H), and the heads of one chunk share an item residue mod 8, so they run on
// one XCD, whose L2 then serves the other heads' reads of the same X rows.
//   long items   (long window, head): four waves take quarters of a window of
//                more than 2L rows; or (two long windows, head): waves 2m and
//                2m + 1 take the halves of window m (L + 1 .. 2L rows);
//   chunk items  (four chunks, head): one chunk per wave.
// The output o ([n, C], original row order) then goes through the output
// projection, k_out_proj.
constexpr int kProjMaxC = 128;

struct ProjArgs {
  const void* x;  // [n, C] features
  const void* w;  // [3C, C]: the rows of W_q, W_k, W_v
  const void* b;  // [3C] or null
};

struct ProjItems {
  int32_t nL, nL4, nL2p, nC, nCG, H;
  int32_t itemsL4, itemsL, total;
};

__device__ __forceinline__ ProjItems proj_items(const KernelArgs& a, const PlanHeader* hdr) {
  ProjItems it;
  it.nL = max(0, min(hdr->n_long, a.max_long));
  it.nL4 = max(0, min(hdr->n_long4, it.nL));
  it.nL2p = (it.nL - it.nL4 + 1) / 2;
  it.nC = max(0, min(hdr->n_chunks, a.max_chunks));
  it.nCG = (it.nC + 3) / 4;
  it.H = a.H;
  it.itemsL4 = ((it.nL4 + 7) & ~7) * a.H;
  it.itemsL = it.itemsL4 + ((it.nL2p + 7) & ~7) * a.H;
  it.total = it.itemsL + ((it.nCG + 7) & ~7) * a.H;
  return it;
}

// Every section is a multiple of 8 H items, so the head of an item is
// (item / 8) mod H and its unit (window, pair of windows or group of chunks) is
// (item / 8 / H) * 8 + item mod 8.
__device__ __forceinline__ Slot proj_slot(const ProjItems& it, int32_t item, int wv) {
  Slot sl;
  sl.idx = -1;
  sl.table = 0;
  sl.h = 0;
  sl.parts = 4;
  sl.piece = wv;
  if (item >= it.total) return sl;
  const int32_t base = item < it.itemsL4 ? 0 : (item < it.itemsL ? it.itemsL4 : it.itemsL);
  const int32_t r = (item - base) >> 3;
  const int32_t j = (r / it.H) * 8 + (item & 7);
  sl.h = r % it.H;
  if (item < it.itemsL4) {
    if (j < it.nL4) sl.idx = j;
  } else if (item < it.itemsL) {
    // waves 2m, 2m + 1: window 2 j + m of the two-way ones; a missing second
    // window leaves its waves an empty share of the first (they still take part
    // in the exchange)
    const int32_t nL2 = it.nL - it.nL4;
    const int32_t wdx = 2 * j + (wv >> 1);
    sl.parts = 2;
    if (2 * j < nL2) {
      sl.idx = it.nL4 + (wdx < nL2 ? wdx : 2 * j);
      sl.piece = wdx < nL2 ? (wv & 1) : -1;
    }
  } else {
    const int32_t c = 4 * j + wv;
    sl.table = 1;
    if (c < it.nC) sl.idx = c;
  }
  return sl;
}

// Feature rows of a block: lane (i, g) of sub-tile s of job jj holds channels
// 32 kb + 8 g .. + 7 of its row for every 32-channel block kb.
template <typename T, int CB>
struct XBlock {
  Raw<T, 8> x[kBlockJobs][2][CB];
  int32_t o[kBlockJobs][2];
  bool ok[kBlockJobs][2];
};

template <typename T, int CB>
__device__ __forceinline__ void xblock_fetch(XBlock<T, CB>& xb, const BlockRows& br, int32_t base,
                                             int32_t end, int32_t n, const T* x, int g) {
  constexpr int C = 32 * CB;
#pragma unroll
  for (int jj = 0; jj < kBlockJobs; ++jj)
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const bool ok = (uint32_t)br.o[jj][s] < (uint32_t)n;
      xb.ok[jj][s] = ok;
      xb.o[jj][s] = ok ? br.o[jj][s] : 0;
      const bool live = base + kSliceRows * jj + 16 * s < end;
      const T* row = row_at(x, xb.o[jj][s], (size_t)C, 8 * g);
#pragma unroll
      for (int kb = 0; kb < CB; ++kb) {
        if (live) xb.x[jj][s][kb] = __builtin_bit_cast(Raw<T, 8>, *reinterpret_cast<const uint4*>(row + 32 * kb));
        else xb.x[jj][s][kb] = Frag<T, 8>::zero();
      }
    }
}

// The matrices selected by `which` (bit 0: K, 1: V, 2: Q) of one job's rows,
// projected from its features: weight rows in LDS, W_q rows 0..D-1, W_k
// D..2D-1, W_v 2D..3D-1 of the head, LDW elements apart; biases in fp32.
template <typename T, int D, int CB>
__device__ __forceinline__ void project_job(Slice<T, Geo<D>::KS, 3>& sj, const Raw<T, 8> (&xj)[2][CB],
                                            unsigned which, const T* s_w, const float* s_b, int i,
                                            int g) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT, LDW = 32 * CB + 8;
  using F8 = Frag<T, 8>;
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int m = 0; m < 3; ++m) {
    if (!(which & (1u << m))) continue;
    const int wm = m == 0 ? 1 : (m == 1 ? 2 : 0);
    Raw<T, KS> fr[2];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      floatx4 acc[2] = {zero, zero};
#pragma unroll
      for (int kb = 0; kb < CB; ++kb) {
        const Raw<T, 8> w =
            *reinterpret_cast<const Raw<T, 8>*>(s_w + (wm * D + 16 * t + i) * LDW + 32 * kb + 8 * g);
#pragma unroll
        for (int s = 0; s < 2; ++s) acc[s] = F8::mma(w, xj[s][kb], acc[s]);
      }
      const float4 bias = *reinterpret_cast<const float4*>(s_b + wm * D + 16 * t + 4 * g);
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        fr[s][4 * t + 0] = f32_to_u16<T>(acc[s][0] + bias.x);
        fr[s][4 * t + 1] = f32_to_u16<T>(acc[s][1] + bias.y);
        fr[s][4 * t + 2] = f32_to_u16<T>(acc[s][2] + bias.z);
        fr[s][4 * t + 3] = f32_to_u16<T>(acc[s][3] + bias.w);
      }
      // keep the weight reads of later tiles from being hoisted here (each would
      // hold 4 more VGPRs across the MFMAs)
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) sj.x[m][s] = fr[s];
  }
}

// All jobs of a block, job by job (a job's features are dead once its fragments
// exist).
template <typename T, int D, int CB>
__device__ __forceinline__ void project(Block<T, D, 3>& bk, const XBlock<T, CB>& xb, unsigned which,
                                        const T* s_w, const float* s_b, int i, int g) {
#pragma unroll
  for (int jj = 0; jj < kBlockJobs; ++jj) {
    project_job<T, D, CB>(bk.j[jj], xb.x[jj], which, s_w, s_b, i, g);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      bk.j[jj].ok[s] = xb.ok[jj][s];
      bk.j[jj].o[s] = xb.o[jj][s];
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// One 32-row job of a share longer than a block (streamed): rows through the
// permutation, features, and the selected matrices.
template <typename T, int D, int CB>
__device__ __forceinline__ void stream_job(Slice<T, Geo<D>::KS, 3>& sj, int32_t r0, int32_t end,
                                           const int32_t* perm, int32_t n, const T* x,
                                           unsigned which, const T* s_w, const float* s_b, int i,
                                           int g) {
  constexpr int C = 32 * CB;
  Raw<T, 8> xj[2][CB];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int32_t p = r0 + 16 * s + i;
    const int32_t row = p < end ? (perm ? perm[p] : p) : -1;
    const bool ok = (uint32_t)row < (uint32_t)n;
    sj.ok[s] = ok;
    sj.o[s] = ok ? row : 0;
    const bool live = r0 + 16 * s < end;
    const T* src = row_at(x, sj.o[s], (size_t)C, 8 * g);
#pragma unroll
    for (int kb = 0; kb < CB; ++kb) {
      if (live) xj[s][kb] = __builtin_bit_cast(Raw<T, 8>, *reinterpret_cast<const uint4*>(src + 32 * kb));
      else xj[s][kb] = Frag<T, 8>::zero();
    }
  }
  project_job<T, D, CB>(sj, xj, which, s_w, s_b, i, g);
}

// One workgroup's copy of rows [r0, r0 + nr) of a [*, C] weight matrix into LDS
// rows LDW elements apart (16-byte pieces), and of the matching biases (zero
// when there are none).
template <typename T, int C, int LDW>
__device__ __forceinline__ void stage_rows(T* s_w, float* s_b, const T* w, const T* b,
                                           const int32_t (&src)[3], int rows_per, int nblk) {
  const int pieces = C / 8;
  for (int idx = threadIdx.x; idx < nblk * rows_per * pieces; idx += blockDim.x) {
    const int rr = idx / pieces, pc = idx - rr * pieces;
    const int m = rr / rows_per, e = rr - m * rows_per;
    const uint4 val = *reinterpret_cast<const uint4*>(w + (size_t)(src[m] + e) * C + 8 * pc);
    *reinterpret_cast<uint4*>(s_w + rr * LDW + 8 * pc) = val;
  }
  for (int idx = threadIdx.x; idx < nblk * rows_per; idx += blockDim.x) {
    const int m = idx / rows_per, e = idx - m * rows_per;
    s_b[idx] = b ? u16_to_f32<T>(reinterpret_cast<const unsigned short*>(b)[src[m] + e]) : 0.f;
  }
}

#ifndef SLA_PROJ_WPE
#define SLA_PROJ_WPE 2
#endif

template <typename T, int D, int PHI, int CB>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(SLA_PROJ_WPE)))
void k_sla_fwd_proj(KernelArgs a, ProjArgs pa, T* __restrict__ o) {
  constexpr int KT = kStateTiles<D>, C = 32 * CB, LDW = C + 8;
  __shared__ floatx4 s_part[kWaves * KT * 64];             // partial states of a long window
  __shared__ __attribute__((aligned(16))) T s_w[3 * D * LDW];  // W_q, W_k, W_v rows of the head
  __shared__ __attribute__((aligned(16))) float s_b[3 * D];
  const int lane = lane_id();
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const PlanHeader* hdr = a.hdr;
  if (hdr->magic != kPlanMagic || hdr->n != a.n || hdr->num_windows != a.W) return;
  const ProjItems it = proj_items(a, hdr);
  const int head = ((int)blockIdx.x >> 3) % a.H;
  {
    const int32_t src[3] = {head * D, C + head * D, 2 * C + head * D};
    stage_rows<T, C, LDW>(s_w, s_b, static_cast<const T*>(pa.w), static_cast<const T*>(pa.b), src, D, 3);
    __syncthreads();
  }
  const int32_t* perm = hdr->csr ? nullptr : a.perm;
  const T* x = static_cast<const T*>(pa.x);
  const int i = lane & 15, g = lane >> 4;
  const size_t rs = (size_t)a.H * D;
  const int32_t n = a.n, G = gridDim.x;
  const Sel<T, D> sel(i, g);
  constexpr unsigned kKV = 3u, kQ = 4u, kAll = 7u;

  int32_t item = blockIdx.x;
  Pending cur;
  {
    const Slot sl = proj_slot(it, item, wv);
    pending_request(cur, a, sl, slot_entry(a, sl), wv, perm, lane);
  }
  Slot nsl = proj_slot(it, item + G, wv);
  int4 ne = slot_entry(a, nsl);
  while (item < it.total) {
    const WaveWork ww = cur.ww;
    const int col = ww.h * D;
    const bool resident = ww.rb - ww.ra <= kBlockRows;
    const unsigned first = resident ? kAll : kKV;
    // a share of more than kBlockRows rows (a quarter of a very long window) is
    // streamed job by job: K, V for the state, then Q for the outputs.  The two
    // cases are separate branches, each with its own window loop, so that the
    // resident rows are not live in the streamed one.
    XBlock<T, CB> xb;
    if (ww.kind != 0 && resident) xblock_fetch<T, CB>(xb, cur.br, ww.ra, ww.rb, n, x, g);
    // the next item: its rows and windows are requested now, its successor's entry too
    Pending nxt;
    pending_request(nxt, a, nsl, ne, wv, perm, lane);
    nsl = proj_slot(it, item + 2 * G, wv);
    ne = slot_entry(a, nsl);
    WinIter wi;
    if (resident) {
      Block<T, D, 3> bk;
      if (ww.kind != 0) project<T, D, CB>(bk, xb, kAll, s_w, s_b, i, g);
      for (bool more = wi.first(ww, cur.str); more; more = wi.next(ww, cur.str)) {
        const int32_t wa = wi.wc.ws, wb = wi.wc.we;
        State<D> st;
        st.clear();
#pragma unroll
        for (int jj = 0; jj < kBlockJobs; ++jj) {
          const int32_t r0 = ww.ra + kSliceRows * jj;
          if (job_overlaps(r0, wa, wb)) state_seg<T, D, 3, PHI>(bk.j[jj], r0, wa, wb, i, g, sel, st);
        }
        if (wi.shared) {
          publish<D>(st, s_part + wv * KT * 64, lane);
          lds_barrier();
          combine<D>(st, s_part, lane, wv, ww.pair);
          lds_barrier();  // the slots may be written by the next long item
        }
        FwdOp<T, D> op;
        make_fwd_op<T, D>(st, op, i, a.eps);
#pragma unroll
        for (int jj = 0; jj < kBlockJobs; ++jj) {
          const int32_t r0 = ww.ra + kSliceRows * jj;
          if (job_overlaps(r0, wa, wb)) apply_seg<T, D, 3, 2, PHI>(bk.j[jj], r0, wa, wb, i, g, op, o, rs, col);
        }
      }
    } else {
      for (bool more = wi.first(ww, cur.str); more; more = wi.next(ww, cur.str)) {
        const int32_t wa = wi.wc.ws, wb = wi.wc.we;
        State<D> st;
        st.clear();
        for (int32_t r0 = ww.ra; r0 < ww.rb; r0 += kSliceRows) {
          Slice<T, Geo<D>::KS, 3> sj;
          stream_job<T, D, CB>(sj, r0, ww.rb, perm, n, x, kKV, s_w, s_b, i, g);
          state_seg<T, D, 3, PHI>(sj, r0, wa, wb, i, g, sel, st);
        }
        if (wi.shared) {
          publish<D>(st, s_part + wv * KT * 64, lane);
          lds_barrier();
          combine<D>(st, s_part, lane, wv, ww.pair);
          lds_barrier();
        }
        FwdOp<T, D> op;
        make_fwd_op<T, D>(st, op, i, a.eps);
        for (int32_t r0 = ww.ra; r0 < ww.rb; r0 += kSliceRows) {
          Slice<T, Geo<D>::KS, 3> sj;
          stream_job<T, D, CB>(sj, r0, ww.rb, perm, n, x, kQ, s_w, s_b, i, g);
          apply_seg<T, D, 3, 2, PHI>(sj, r0, wa, wb, i, g, op, o, rs, col);
        }
      }
    }
    item += G;
    cur = nxt;
  }
}

// Output projection y = o W_o^T + b_o over the rows that belong to a window
// (sorted positions [0, offsets[W]), read through the permutation): every wave
// takes 16-row tiles; W_o (C x C) lives in LDS for the launch.  Lane (i, g)
// holds channels 32 kb + 8 g .. + 7 of row i as the second operand; output tile
// t gives it y[i][16 t + 4 g + j], and two tiles are one 32-column block in the
// slot order of the row stores.
template <typename T, int CB>
__global__ __launch_bounds__(256) void k_out_proj(KernelArgs a, const T* __restrict__ o,
                                                  const T* __restrict__ w, const T* __restrict__ b,
                                                  T* __restrict__ y) {
  constexpr int C = 32 * CB, LDW = C + 8;
  __shared__ __attribute__((aligned(16))) T s_w[C * LDW];
  __shared__ __attribute__((aligned(16))) float s_b[C];
  const PlanHeader* hdr = a.hdr;
  if (hdr->magic != kPlanMagic || hdr->n != a.n || hdr->num_windows != a.W) return;
  {
    const int32_t src[3] = {0, 0, 0};
    stage_rows<T, C, LDW>(s_w, s_b, w, b, src, C, 1);
    __syncthreads();
  }
  using F8 = Frag<T, 8>;
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  const int32_t* perm = hdr->csr ? nullptr : a.perm;
  const int32_t n = a.n;
  const int32_t nrows = max(0, min(a.offs[a.W], n));
  const int lane = lane_id(), wv = threadIdx.x >> 6;
  const int i = lane & 15, g = lane >> 4;
  for (int32_t tile = (int32_t)blockIdx.x * kWaves + wv; tile * 16 < nrows;
       tile += (int32_t)gridDim.x * kWaves) {
    const int32_t p = tile * 16 + i;
    const int32_t row = p < nrows ? (perm ? perm[p] : p) : -1;
    const bool ok = (uint32_t)row < (uint32_t)n;
    const T* src = row_at(o, ok ? row : 0, (size_t)C, 8 * g);
    Raw<T, 8> xo[CB];
#pragma unroll
    for (int kb = 0; kb < CB; ++kb)
      xo[kb] = __builtin_bit_cast(Raw<T, 8>, *reinterpret_cast<const uint4*>(src + 32 * kb));
#pragma unroll
    for (int hb = 0; hb < CB; ++hb) {
      float f[8];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        const int t = 2 * hb + tt;
        floatx4 acc = zero;
#pragma unroll
        for (int kb = 0; kb < CB; ++kb) {
          const Raw<T, 8> wo =
              *reinterpret_cast<const Raw<T, 8>*>(s_w + (16 * t + i) * LDW + 32 * kb + 8 * g);
          acc = F8::mma(wo, xo[kb], acc);
        }
        const float4 bias = *reinterpret_cast<const float4*>(s_b + 16 * t + 4 * g);
        f[4 * tt + 0] = acc[0] + bias.x;
        f[4 * tt + 1] = acc[1] + bias.y;
        f[4 * tt + 2] = acc[2] + bias.z;
        f[4 * tt + 3] = acc[3] + bias.w;
      }
      RowIO<T, 32>::put(row_at(y, ok ? row : 0, (size_t)C, 32 * hb), g, F8::from_f32(f), ok);
    }
  }
}

// ------------------------------------------------------------ host launchers
// Workgroups of a launch: the resident capacity of the device for the kernel
// (workgroups per CU x CUs, queried once per device and kernel), at most enough
// for every item the plan can hold (long windows have more than kMinChunkRows
// rows), a multiple of 8.
static int resident_workgroups(const void* kernel) {
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

static int grid_size(const void* kernel, const PlanLayout& lay, int32_t n, int32_t H) {
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

static KernelArgs kernel_args(const void* plan, const PlanLayout& lay, int32_t n, int32_t W,
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

template <typename T, int D, int PHI>
static hipError_t fwd_impl(const void* plan, int32_t n, int32_t W, int32_t H, float eps,
                           const void* q, const void* k, const void* v, void* o,
                           hipStream_t stream) {
  const PlanLayout lay = plan_layout(n, W);
  const KernelArgs a = kernel_args(plan, lay, n, W, H, eps);
  const void* kern = reinterpret_cast<const void*>(&k_sla_fwd<T, D, PHI>);
  hipLaunchKernelGGL((k_sla_fwd<T, D, PHI>), dim3(grid_size(kern, lay, n, H)), dim3(64 * kWaves), 0,
                     stream, a, static_cast<const T*>(q), static_cast<const T*>(k),
                     static_cast<const T*>(v), static_cast<T*>(o));
  return hipGetLastError();
}

template <typename T, int D, int PHI>
static hipError_t bwd_impl(const void* plan, int32_t n, int32_t W, int32_t H, float eps,
                           const void* q, const void* k, const void* v, const void* dout, void* dq,
                           void* dk, void* dv, hipStream_t stream) {
  const PlanLayout lay = plan_layout(n, W);
  const KernelArgs a = kernel_args(plan, lay, n, W, H, eps);
  const void* kern = reinterpret_cast<const void*>(&k_sla_bwd<T, D, PHI>);
  hipLaunchKernelGGL((k_sla_bwd<T, D, PHI>), dim3(grid_size(kern, lay, n, H)), dim3(64 * kWaves), 0,
                     stream, a, static_cast<const T*>(q), static_cast<const T*>(k),
                     static_cast<const T*>(v), static_cast<const T*>(dout), static_cast<T*>(dq),
                     static_cast<T*>(dk), static_cast<T*>(dv));
  return hipGetLastError();
}

template <int PHI>
static hipError_t forward_phi(const void* plan, int32_t n, int32_t W, int dtype, int32_t H,
                              int32_t d, float eps, const void* q, const void* k, const void* v,
                              void* o, hipStream_t stream) {
  if (d == 32) {
    if (dtype == 0) return fwd_impl<float, 32, PHI>(plan, n, W, H, eps, q, k, v, o, stream);
    if (dtype == 1) return fwd_impl<_Float16, 32, PHI>(plan, n, W, H, eps, q, k, v, o, stream);
    return fwd_impl<bf16_t, 32, PHI>(plan, n, W, H, eps, q, k, v, o, stream);
  }
  if (dtype == 0) return fwd_impl<float, 16, PHI>(plan, n, W, H, eps, q, k, v, o, stream);
  if (dtype == 1) return fwd_impl<_Float16, 16, PHI>(plan, n, W, H, eps, q, k, v, o, stream);
  return fwd_impl<bf16_t, 16, PHI>(plan, n, W, H, eps, q, k, v, o, stream);
}

template <int PHI>
static hipError_t backward_phi(const void* plan, int32_t n, int32_t W, int dtype, int32_t H,
                               int32_t d, float eps, const void* q, const void* k, const void* v,
                               const void* dout, void* dq, void* dk, void* dv,
                               hipStream_t stream) {
  if (d == 32) {
    if (dtype == 0) return bwd_impl<float, 32, PHI>(plan, n, W, H, eps, q, k, v, dout, dq, dk, dv, stream);
    if (dtype == 1) return bwd_impl<_Float16, 32, PHI>(plan, n, W, H, eps, q, k, v, dout, dq, dk, dv, stream);
    return bwd_impl<bf16_t, 32, PHI>(plan, n, W, H, eps, q, k, v, dout, dq, dk, dv, stream);
  }
  if (dtype == 0) return bwd_impl<float, 16, PHI>(plan, n, W, H, eps, q, k, v, dout, dq, dk, dv, stream);
  if (dtype == 1) return bwd_impl<_Float16, 16, PHI>(plan, n, W, H, eps, q, k, v, dout, dq, dk, dv, stream);
  return bwd_impl<bf16_t, 16, PHI>(plan, n, W, H, eps, q, k, v, dout, dq, dk, dv, stream);
}

// dtype: 0 f32, 1 f16, 2 bf16; phi: 0 elu + 1, 1 ReLU
hipError_t launch_forward(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                          int phi, float eps, const void* q, const void* k, const void* v, void* o,
                          hipStream_t stream) {
  if (phi == kPhiRelu) return forward_phi<kPhiRelu>(plan, n, W, dtype, H, d, eps, q, k, v, o, stream);
  return forward_phi<kPhiElu1>(plan, n, W, dtype, H, d, eps, q, k, v, o, stream);
}

hipError_t launch_backward(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                           int phi, float eps, const void* q, const void* k, const void* v,
                           const void* dout, void* dq, void* dk, void* dv, hipStream_t stream) {
  if (phi == kPhiRelu)
    return backward_phi<kPhiRelu>(plan, n, W, dtype, H, d, eps, q, k, v, dout, dq, dk, dv, stream);
  return backward_phi<kPhiElu1>(plan, n, W, dtype, H, d, eps, q, k, v, dout, dq, dk, dv, stream);
}

// Projected forward: the fused projection + SLA kernel, then the output
// projection.  Workgroups of the fused kernel: as grid_size, rounded up to a
// multiple of 8 H (every workgroup keeps one head), at most enough for every item
// the plan can hold.
template <typename T, int D, int PHI, int CB>
static hipError_t proj_impl(const void* plan, int32_t n, int32_t W, int32_t H, float eps,
                            const void* x, const void* wqkv, const void* bqkv, const void* wo,
                            const void* bo, void* o, void* y, hipStream_t stream) {
  const PlanLayout lay = plan_layout(n, W);
  const KernelArgs a = kernel_args(plan, lay, n, W, H, eps);
  const void* kern = reinterpret_cast<const void*>(&k_sla_fwd_proj<T, D, PHI, CB>);
  const int64_t c = resident_workgroups(kern);
  const int64_t unit = 8 * (int64_t)H;
  const int64_t ml = lay.max_long, mc = lay.max_chunks;
  const int64_t items = (((ml + 7) & ~7) + (((ml + 1) / 2 + 7) & ~7) + (((mc + 3) / 4 + 7) & ~7)) * H;
  int64_t k = ((int64_t)n * H + c * kRowHeadsPerWorkgroup / 2) / (c * kRowHeadsPerWorkgroup);
  if (k < 1) k = 1;
  int64_t g = k * c;
  if (g > items) g = items;
  g = (g + unit - 1) / unit * unit;
  if (g < unit) g = unit;
  const ProjArgs pa{x, wqkv, bqkv};
  hipLaunchKernelGGL((k_sla_fwd_proj<T, D, PHI, CB>), dim3((unsigned)g), dim3(64 * kWaves), 0, stream,
                     a, pa, static_cast<T*>(o));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const void* kout = reinterpret_cast<const void*>(&k_out_proj<T, CB>);
  int64_t go = resident_workgroups(kout);
  const int64_t passes = ((int64_t)n + 16 * kWaves - 1) / (16 * kWaves);
  if (go > passes) go = passes;
  if (go < 1) go = 1;
  hipLaunchKernelGGL((k_out_proj<T, CB>), dim3((unsigned)go), dim3(64 * kWaves), 0, stream, a,
                     static_cast<const T*>(o), static_cast<const T*>(wo), static_cast<const T*>(bo),
                     static_cast<T*>(y));
  return hipGetLastError();
}

template <typename T, int PHI>
static hipError_t projected_t(const void* plan, int32_t n, int32_t W, int32_t H, int32_t d,
                              float eps, const void* x, const void* wqkv, const void* bqkv,
                              const void* wo, const void* bo, void* o, void* y,
                              hipStream_t stream) {
  const int C = H * d;
  if (d == 32) {
    if (C == 128) return proj_impl<T, 32, PHI, 4>(plan, n, W, H, eps, x, wqkv, bqkv, wo, bo, o, y, stream);
    return proj_impl<T, 32, PHI, 2>(plan, n, W, H, eps, x, wqkv, bqkv, wo, bo, o, y, stream);
  }
  if (C == 128) return proj_impl<T, 16, PHI, 4>(plan, n, W, H, eps, x, wqkv, bqkv, wo, bo, o, y, stream);
  return proj_impl<T, 16, PHI, 2>(plan, n, W, H, eps, x, wqkv, bqkv, wo, bo, o, y, stream);
}

// dtype: 1 f16, 2 bf16; C = H d in {64, 128}; phi: 0 elu + 1, 1 ReLU
hipError_t launch_forward_projected(const void* plan, int32_t n, int32_t W, int dtype, int32_t H,
                                    int32_t d, int phi, float eps, const void* x, const void* wqkv,
                                    const void* bqkv, const void* wo, const void* bo, void* o,
                                    void* y, hipStream_t stream) {
  if (dtype == 1) {
    if (phi == kPhiRelu)
      return projected_t<_Float16, kPhiRelu>(plan, n, W, H, d, eps, x, wqkv, bqkv, wo, bo, o, y, stream);
    return projected_t<_Float16, kPhiElu1>(plan, n, W, H, d, eps, x, wqkv, bqkv, wo, bo, o, y, stream);
  }
  if (phi == kPhiRelu)
    return projected_t<bf16_t, kPhiRelu>(plan, n, W, H, d, eps, x, wqkv, bqkv, wo, bo, o, y, stream);
  return projected_t<bf16_t, kPhiElu1>(plan, n, W, H, d, eps, x, wqkv, bqkv, wo, bo, o, y, stream);
}

}  // namespace sla

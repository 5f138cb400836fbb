// Cross-covariance attention inside every window: the XCA design of the
// linear-attention ablation (Sec. 4.5, Tab. 7), which cites XCiT, run on the
// same window-sorted plan as SLA.  For window w and head h, with the window's q
// and k columns L2-normalised over the window's rows (norms floored at 1e-12):
//     A[e][c] = softmax over c of  tau_h qhat[:, e] . khat[:, c]     (d x d),
//     o_i[e]  = sum_c A[e][c] v_i[c]                                 for i in w.
// Like Eq. (3) it needs one d x d reduction over the window's rows per head,
// here q^T k together with the column norms, and then one d x d product per row.
//
// k_xca_fwd: one workgroup per (window, head), the heads of a window on one XCD.
//   1. 64 rows at a time, the window's q and k rows (this head's d columns)
//      are gathered through the plan's permutation into LDS in fp32; thread
//      (e, c-block) accumulates G[e][c] = sum_r q_re k_rc for its EPT columns,
//      and the first wave the squared column norms.
//   2. The logits tau G[e][c] / (|q_e| |k_c|) are bounded by |tau|, so the
//      softmax needs no overflow guard beyond the usual max shift; the row max
//      and sum are reduced over the CPR threads of a row with lane xors.
//   3. Each thread keeps one row e of A in registers and, 64 rows at a time
//      with the v rows in LDS, writes o_i[e] for its rows.  A window of at most
//      64 rows gathers its v rows in step 1 already, into registers, so that
//      their round trip overlaps the sums; longer windows gather v again here.
// fp32 throughout; inputs widened from the storage type, outputs rounded to it.
#include "sla.h"
#include "sla_common.h"

#include <mutex>

namespace sla {

// The dtau partials of the backward without a workspace (sla_backward_xca_noalloc):
// one fp32 per (window, head), held in static device memory on every GPU the
// library runs on.  In host code `scratch` only names the symbol; its address on
// a device comes from hipGetSymbolAddress, looked up once per device.
constexpr size_t kXcaScratchFloats = 262144;   // SLA_XCA_SCRATCH_FLOATS
static_assert(kXcaScratchFloats == SLA_XCA_SCRATCH_FLOATS, "the header states the scratch size");
static __device__ __align__(256) float scratch[kXcaScratchFloats];

namespace {

constexpr int kXcaThreads = 256;
constexpr int kXcaRows = 64;   // rows staged in LDS at a time

template <typename T>
struct XcaIo;
template <>
struct XcaIo<float> {
  static constexpr int kPiece = 4;   // elements per 16-byte piece
  __device__ static void unpack(uint4 u, float (&x)[4]) {
    x[0] = __uint_as_float(u.x); x[1] = __uint_as_float(u.y);
    x[2] = __uint_as_float(u.z); x[3] = __uint_as_float(u.w);
  }
  __device__ static void store(float* p, float x) { *p = x; }
};
template <>
struct XcaIo<_Float16> {
  static constexpr int kPiece = 8;
  __device__ static void unpack(uint4 u, float (&x)[8]) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[2 * j] = (float)__builtin_bit_cast(_Float16, (unsigned short)(w[j] & 0xffffu));
      x[2 * j + 1] = (float)__builtin_bit_cast(_Float16, (unsigned short)(w[j] >> 16));
    }
  }
  __device__ static void store(_Float16* p, float x) { *p = (_Float16)x; }
};
template <>
struct XcaIo<bf16_t> {
  static constexpr int kPiece = 8;
  __device__ static void unpack(uint4 u, float (&x)[8]) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[2 * j] = __uint_as_float(w[j] << 16);
      x[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
    }
  }
  __device__ static void store(bf16_t* p, float x) {
    p->bits = __builtin_bit_cast(unsigned short, (__bf16)x);
  }
};

// Workgroup b -> (window, head) such that the heads of a window share b mod 8:
// workgroups are dealt to the 8 XCDs round-robin, so the heads of a window run
// on one XCD, whose L2 then serves the other heads' quarters of each row's
// 128-byte lines.  The grid is 8 ceil(W / 8) H; workgroups past the last window
// have nothing to do.
__device__ __forceinline__ void xca_item(uint32_t b, int32_t H, int32_t& w, int32_t& h) {
  const uint32_t per = 8u * (uint32_t)H;
  const uint32_t g = b / per, r = b - g * per;
  h = (int32_t)(r >> 3);
  w = (int32_t)(g * 8u + (r & 7u));
}

inline unsigned xca_grid(int32_t W, int32_t H) { return (unsigned)(((int64_t)W + 7) / 8 * 8 * H); }

// LDS row stride of the staged rows: 16-byte aligned rows for float4 reads
template <int D>
constexpr int kXcaLd = D + 4;

// 16-byte pieces of a staged block: piece j = (row r, piece pc); a thread takes
// pieces tid, tid + 256 (at most two: 64 rows of 32 fp32 columns)
template <typename T, int D>
constexpr int kXcaPieces = kXcaRows * D / XcaIo<T>::kPiece;
template <typename T, int D>
constexpr int kXcaPerThread = (kXcaPieces<T, D> + kXcaThreads - 1) / kXcaThreads;

// Gathers the raw pieces of rows [p0, p0 + nr) (sorted positions) of `x` into
// registers (zero past nr or for an out-of-range row) and, when s_row is given,
// records each row's original index there (-1 for none).
template <typename T, int D>
__device__ __forceinline__ void xca_fetch(const int32_t* pm, int32_t p0, int nr, int32_t n,
                                          size_t rs, int col, const T* x,
                                          uint4 (&raw)[kXcaPerThread<T, D>], int32_t* s_row) {
  constexpr int PB = XcaIo<T>::kPiece, PR = D / PB;
#pragma unroll
  for (int u = 0; u < kXcaPerThread<T, D>; ++u) {
    const int j = (int)threadIdx.x + u * kXcaThreads;
    const int r = j / PR, pc = j - r * PR;
    int32_t row = -1;
    if (j < kXcaPieces<T, D> && r < nr) {
      row = pm ? pm[p0 + r] : p0 + r;
      if ((uint32_t)row >= (uint32_t)n) row = -1;
    }
    raw[u] = row >= 0 ? *reinterpret_cast<const uint4*>(x + (size_t)row * rs + col + pc * PB)
                      : make_uint4(0, 0, 0, 0);
    if (s_row && j < kXcaPieces<T, D> && pc == 0) s_row[r] = row;
  }
}

// Raw pieces into an LDS block of fp32 rows.
template <typename T, int D>
__device__ __forceinline__ void xca_put(const uint4 (&raw)[kXcaPerThread<T, D>],
                                        float (*a)[kXcaLd<D>]) {
  constexpr int PB = XcaIo<T>::kPiece, PR = D / PB;
#pragma unroll
  for (int u = 0; u < kXcaPerThread<T, D>; ++u) {
    const int j = (int)threadIdx.x + u * kXcaThreads;
    if (j < kXcaPieces<T, D>) {
      const int r = j / PR, pc = j - r * PR;
      float x[PB];
      XcaIo<T>::unpack(raw[u], x);
#pragma unroll
      for (int e = 0; e < PB; ++e) a[r][pc * PB + e] = x[e];
    }
  }
}

template <typename T, int D>
__global__ __launch_bounds__(kXcaThreads) void k_xca_fwd(
    const PlanHeader* __restrict__ hdr, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ offs, const float* __restrict__ tau, const T* __restrict__ q,
    const T* __restrict__ k, const T* __restrict__ v, T* __restrict__ o, int32_t n, int32_t W,
    int32_t H) {
  constexpr int EPT = D * D / kXcaThreads;   // entries (e, c) per thread: 4 (d = 32) or 1 (d = 16)
  constexpr int CPR = D / EPT;               // threads per row e of G
  constexpr int RPP = kXcaThreads / D;       // output rows per pass of phase 3
  static_assert(D * D % kXcaThreads == 0 && CPR <= 64 && (CPR & (CPR - 1)) == 0, "row groups");
  constexpr int LD = kXcaLd<D>;
  constexpr int NP = kXcaPerThread<T, D>;
  __shared__ __align__(16) float s_a[kXcaRows][LD];   // q rows, then v rows
  __shared__ __align__(16) float s_b[kXcaRows][LD];   // k rows
  __shared__ float s_g[D][D + 1];          // softmax weights A
  __shared__ float s_nrm[2 * D];           // |q_e|, then |k_c|
  __shared__ int32_t s_row[kXcaRows];
  int32_t w, h;
  xca_item(blockIdx.x, H, w, h);
  if (w >= W) return;
  if (hdr->magic != kPlanMagic || hdr->n != n || hdr->num_windows != W) return;
  const int32_t* pm = hdr->csr ? nullptr : perm;
  const int32_t rb = max(0, min(offs[w], n)), re = max(rb, min(offs[w + 1], n));
  if (rb == re) return;
  const int tid = (int)threadIdx.x;
  const size_t rs = (size_t)H * D;
  const int col = h * D;

  // 1. G = q^T k over the window's rows, and the squared column norms
  const int e = tid / CPR, c0 = (tid - e * CPR) * EPT;
  float acc[EPT];
#pragma unroll
  for (int u = 0; u < EPT; ++u) acc[u] = 0.f;
  float nrm = 0.f;
  // a window of at most one block also gathers its v rows now, into registers,
  // so that their round trip overlaps the q^T k sums
  const bool one = re - rb <= kXcaRows;
  uint4 vr[NP];
  for (int32_t p0 = rb; p0 < re; p0 += kXcaRows) {
    const int nr = min(kXcaRows, re - p0);
    if (p0 != rb) __syncthreads();   // the previous block's readers are done
    {
      uint4 qr[NP], kr[NP];
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, q, qr, s_row);
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, k, kr, nullptr);
      if (one) xca_fetch<T, D>(pm, p0, nr, n, rs, col, v, vr, nullptr);
      xca_put<T, D>(qr, s_a);
      xca_put<T, D>(kr, s_b);
    }
    __syncthreads();
    for (int r = 0; r < nr; ++r) {
      const float a = s_a[r][e];
#pragma unroll
      for (int u = 0; u < EPT; ++u) acc[u] += a * s_b[r][c0 + u];
    }
    // the first wave sums the squared columns (q in lanes 0..D-1, k after)
    if (tid < D) {
      for (int r = 0; r < nr; ++r) nrm += s_a[r][tid] * s_a[r][tid];
    } else if (tid < 2 * D) {
      for (int r = 0; r < nr; ++r) nrm += s_b[r][tid - D] * s_b[r][tid - D];
    }
  }
  if (tid < 2 * D) s_nrm[tid] = fmaxf(sqrtf(nrm), 1e-12f);
  __syncthreads();

  // 2. softmax of each row e over c
  const float t = tau[h];
  float g[EPT];
  float mx = -3.0e38f;
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    g[u] = t * acc[u] / (s_nrm[e] * s_nrm[D + c0 + u]);
    mx = fmaxf(mx, g[u]);
  }
#pragma unroll
  for (int m = 1; m < CPR; m <<= 1) mx = fmaxf(mx, __shfl_xor(mx, m, 64));
  float sum = 0.f;
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    g[u] = expf(g[u] - mx);
    sum += g[u];
  }
#pragma unroll
  for (int m = 1; m < CPR; m <<= 1) sum += __shfl_xor(sum, m, 64);
  const float inv = 1.f / sum;
#pragma unroll
  for (int u = 0; u < EPT; ++u) s_g[e][c0 + u] = g[u] * inv;
  // s_a's last readers (the q^T k sums) passed the barrier above
  if (one) xca_put<T, D>(vr, s_a);
  __syncthreads();

  // 3. o_i[e3] = sum_c A[e3][c] v_i[c]
  const int e3 = tid % D, r3 = tid / D;
  float arow[D];
#pragma unroll
  for (int c = 0; c < D; ++c) arow[c] = s_g[e3][c];
  for (int32_t p0 = rb; p0 < re; p0 += kXcaRows) {
    const int nr = min(kXcaRows, re - p0);
    if (!one) {
      __syncthreads();   // s_a and s_row are free
      uint4 raw[NP];
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, v, raw, s_row);
      xca_put<T, D>(raw, s_a);
      __syncthreads();
    }
    for (int r = r3; r < nr; r += RPP) {
      const int32_t row = s_row[r];
      float s = 0.f;
#pragma unroll
      for (int c = 0; c < D; c += 4) {
        const float4 x = *reinterpret_cast<const float4*>(&s_a[r][c]);
        s += arow[c] * x.x + arow[c + 1] * x.y + arow[c + 2] * x.z + arow[c + 3] * x.w;
      }
      if (row >= 0) XcaIo<T>::store(o + (size_t)row * rs + col + e3, s);
    }
  }
}

// ----------------------------------------------- forward on the matrix cores
// 16-bit storage, d = 32: the same three steps with both d x d contractions on
// the matrix cores and the rows staged in LDS in their storage format.
//   1. Wave w forms tile (w / 2, w % 2) of G = sum_r q_r^T k_r.  The contraction
//      runs over rows, so both operands are columns of the staged rows, read
//      with the LDS transpose load: in a group of 16 lanes, lane i of group g
//      addresses row 8g + 4h + i / 4, columns 16t + 4 (i % 4) .. + 3, and
//      receives (the probed lane layout of ds_read_b64_tr_b16) the four
//      elements of column 16t + i in rows 8g + 4h .. + 3: operand slot 4h + j
//      holds row 8g + 4h + j, for A (q) and B (k) alike.  The column norms are
//      summed from the staged rows as in the fp32 path.
//   2. The softmax as before, in fp32 from G in LDS; A is rounded to the storage
//      type (bf16: as a pair of high part and residual, 16 bits together).
//   3. o = v A^T: slot j of lane (i, g) is channel c = 8g + j, so A's row e and
//      v's row r are read as they lie (16 bytes a lane); wave w forms the 16-row
//      tile w of a 64-row block for both halves of d, and lane (i, g) receives
//      o[row 16w + i][16t + 4g .. + 3].
// Columns 16t .. 16t + 15 of rows base .. base + 31 of a staged block as an
// operand of a contraction over the rows (slot r of lane (i, g): row base + 8g + r,
// column 16t + i), by LDS transpose loads.
template <typename T, int LDH>
__device__ __forceinline__ Raw<T, 8> xca_cols(const unsigned short (*s)[LDH], int base, int t, int i,
                                              int g) {
  return lds_cols<T>(&s[base][0], LDH, 16 * t, i, g);
}

template <typename T>
__global__ __launch_bounds__(kXcaThreads) void k_xca_fwd_mma(
    const PlanHeader* __restrict__ hdr, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ offs, const float* __restrict__ tau, const T* __restrict__ q,
    const T* __restrict__ k, const T* __restrict__ v, T* __restrict__ o, int32_t n, int32_t W,
    int32_t H) {
  constexpr int D = 32;
  constexpr int LDH = D + 8;                 // staged 16-bit rows: 80 bytes, 16-byte aligned
  constexpr int EPT = D * D / kXcaThreads;   // softmax: entries (e, c) per thread
  constexpr int CPR = D / EPT;
  constexpr int NP = kXcaPerThread<T, D>;    // one 16-byte piece a thread
  constexpr bool kPair = std::is_same<T, bf16_t>::value;
  using F = Frag<T, 8>;
  static_assert(NP == 1 && kXcaPieces<T, D> == kXcaThreads, "one piece a thread");
  __shared__ __align__(16) unsigned short s_q[kXcaRows][LDH];
  __shared__ __align__(16) unsigned short s_k[kXcaRows][LDH];
  __shared__ __align__(16) unsigned short s_v[kXcaRows][LDH];
  __shared__ __align__(16) unsigned short s_p[kPair ? 2 : 1][D][LDH];   // A (and its residual)
  __shared__ float s_g[D][D + 1];
  __shared__ float s_nrm[2 * D];
  __shared__ int32_t s_row[kXcaRows];
  int32_t w, h;
  xca_item(blockIdx.x, H, w, h);
  if (w >= W) return;
  if (hdr->magic != kPlanMagic || hdr->n != n || hdr->num_windows != W) return;
  const int32_t* pm = hdr->csr ? nullptr : perm;
  const int32_t rb = max(0, min(offs[w], n)), re = max(rb, min(offs[w + 1], n));
  if (rb == re) return;
  const int tid = (int)threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int i = lane & 15, g = lane >> 4;
  const size_t rs = (size_t)H * D;
  const int col = h * D;
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  // piece tid of a block: row tid / 4, channels 8 (tid % 4) .. + 7
  const int pr = tid >> 2, pc = tid & 3;
  auto put = [&](unsigned short (*s)[LDH], uint4 x) { *reinterpret_cast<uint4*>(&s[pr][8 * pc]) = x; };

  // 1. G tile (et, ct) of this wave, and the squared column norms
  const int et = wv >> 1, ct = wv & 1;
  floatx4 acc = zero;
  float nrm = 0.f;
  const bool one = re - rb <= kXcaRows;
  uint4 vr[NP];
  for (int32_t p0 = rb; p0 < re; p0 += kXcaRows) {
    const int nr = min(kXcaRows, re - p0);
    if (p0 != rb) __syncthreads();   // the previous block's readers are done
    {
      uint4 qr[NP], kr[NP];
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, q, qr, s_row);
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, k, kr, nullptr);
      if (one) xca_fetch<T, D>(pm, p0, nr, n, rs, col, v, vr, nullptr);
      put(s_q, qr[0]);
      put(s_k, kr[0]);
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      if (32 * ks >= nr) break;   // rows past nr are zero
      acc = F::mma(xca_cols<T, LDH>(s_q, 32 * ks, et, i, g), xca_cols<T, LDH>(s_k, 32 * ks, ct, i, g), acc);
    }
    if (tid < D) {
      for (int r = 0; r < nr; ++r) {
        const float x = u16_to_f32<T>(s_q[r][tid]);
        nrm += x * x;
      }
    } else if (tid < 2 * D) {
      for (int r = 0; r < nr; ++r) {
        const float x = u16_to_f32<T>(s_k[r][tid - D]);
        nrm += x * x;
      }
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) s_g[16 * et + 4 * g + j][16 * ct + i] = acc[j];
  if (tid < 2 * D) s_nrm[tid] = fmaxf(sqrtf(nrm), 1e-12f);
  __syncthreads();

  // 2. softmax of each row e over c, A to the storage type
  {
    const int e = tid / CPR, c0 = (tid - e * CPR) * EPT;
    const float t = tau[h];
    float gv[EPT];
    float mx = -3.0e38f;
#pragma unroll
    for (int u = 0; u < EPT; ++u) {
      gv[u] = t * s_g[e][c0 + u] / (s_nrm[e] * s_nrm[D + c0 + u]);
      mx = fmaxf(mx, gv[u]);
    }
#pragma unroll
    for (int m = 1; m < CPR; m <<= 1) mx = fmaxf(mx, __shfl_xor(mx, m, 64));
    float sum = 0.f;
#pragma unroll
    for (int u = 0; u < EPT; ++u) {
      gv[u] = expf(gv[u] - mx);
      sum += gv[u];
    }
#pragma unroll
    for (int m = 1; m < CPR; m <<= 1) sum += __shfl_xor(sum, m, 64);
    const float inv = 1.f / sum;
#pragma unroll
    for (int u = 0; u < EPT; ++u) {
      const float a = gv[u] * inv;
      const unsigned short hi = f32_to_u16<T>(a);
      s_p[0][e][c0 + u] = hi;
      if constexpr (kPair) s_p[kPair ? 1 : 0][e][c0 + u] = f32_to_u16<T>(a - u16_to_f32<T>(hi));
    }
  }
  // s_q's last readers (the norms) passed the barrier above; s_v is unused so far
  if (one) put(s_v, vr[0]);
  __syncthreads();

  // 3. o = v A^T, tile wv of each 64-row block
  // tile t2's operand row i is A's row 8 (i / 4) + 4 t2 + i % 4, so that lane
  // (i, g) receives columns 8 g .. 8 g + 7 of o over the two tiles and stores
  // them as one 16-byte piece
  Raw<T, 8> pa[2], pl[2];
#pragma unroll
  for (int t2 = 0; t2 < 2; ++t2) {
    const int e = 8 * (i >> 2) + 4 * t2 + (i & 3);
    pa[t2] = *reinterpret_cast<const Raw<T, 8>*>(&s_p[0][e][8 * g]);
    if constexpr (kPair) pl[t2] = *reinterpret_cast<const Raw<T, 8>*>(&s_p[kPair ? 1 : 0][e][8 * g]);
  }
  for (int32_t p0 = rb; p0 < re; p0 += kXcaRows) {
    const int nr = min(kXcaRows, re - p0);
    if (!one) {
      __syncthreads();   // s_v and s_row are free
      uint4 raw[NP];
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, v, raw, s_row);
      put(s_v, raw[0]);
      __syncthreads();
    }
    const int r = 16 * wv + i;
    if (16 * wv >= nr) continue;   // the whole tile is past the block's rows
    const Raw<T, 8> vb = *reinterpret_cast<const Raw<T, 8>*>(&s_v[r][8 * g]);
    const int32_t row = r < nr ? s_row[r] : -1;
    float f[8];
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      floatx4 d4 = F::mma(pa[t2], vb, zero);
      if constexpr (kPair) d4 = F::mma(pl[t2], vb, d4);
#pragma unroll
      for (int j = 0; j < 4; ++j) f[4 * t2 + j] = d4[j];
    }
    if (row >= 0) *reinterpret_cast<Raw<T, 8>*>(o + (size_t)row * rs + col + 8 * g) = F::from_f32(f);
  }
}

// ---------------------------------------------------------------- backward
// Chain rule of the forward, per (window, head) workgroup, with
// N = qhat^T khat, G = tau N and A = softmax_c(G):
//   dv_i = A^T do_i,  dA = sum_i do_i v_i^T,  dG = A * (dA - rowsum(A * dA)),
//   dtau partial = sum dG * N,
//   dqh[:, e] = sum_c B_q[e][c] k[:, c] with B_q[e][c] = tau dG[e][c] / nk_c,
//   s_e = sum_r qhat_re dqh_re  (the projection of dqh onto qhat, summed over the
//        window's rows; zero where the norm took the floor),
//   dq[:, e] = (dqh[:, e] - qhat[:, e] s_e) / nq_e,
// and likewise dk with B_k[e][c] = tau dG[e][c] / nq_e and t_c = sum_r khat_rc
// dkh_rc.  s_e comes from the rows themselves, as qhat and dqh round, so that
// the difference keeps the cancellation exact where it is exact in real
// arithmetic: in a one-row window qhat = q / |q| is +-1 exactly (the square
// root of a rounded square is the magnitude again in binary floating point), so
// qhat s_e = dqh and dq = 0, as the chain rule gives.
// Passes over the window's rows: q, k (N, as in the forward); dout, v (dA and
// dv); q, k again (dqh, dkh and their projections; then dq, dk, from registers
// for a window of one block, from a further pass over q, k otherwise).  The
// temperature gradient of every (window, head) goes to `part`; k_xca_dtau adds
// the windows in order.
template <typename T, int D>
__global__ __launch_bounds__(kXcaThreads) __attribute__((amdgpu_waves_per_eu(sizeof(T) == 4 ? 4 : 5))) void k_xca_bwd(
    const PlanHeader* __restrict__ hdr, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ offs, const float* __restrict__ tau, const T* __restrict__ q,
    const T* __restrict__ k, const T* __restrict__ v, const T* __restrict__ dout,
    T* __restrict__ dq, T* __restrict__ dk, T* __restrict__ dv, float* __restrict__ part,
    int32_t n, int32_t W, int32_t H) {
  constexpr int EPT = D * D / kXcaThreads;
  constexpr int CPR = D / EPT;
  constexpr int RPP = kXcaThreads / D;
  constexpr int LD = kXcaLd<D>;
  constexpr int NP = kXcaPerThread<T, D>;
  constexpr int NW = kXcaThreads / 64;
  __shared__ __align__(16) float s_a[kXcaRows][LD];
  __shared__ __align__(16) float s_b[kXcaRows][LD];
  // A (rows of D + 1) until pass 2 ends, then B_q[e][c] = tau dG[e][c] / nk_c
  // (rows of LD) in the same place
  __shared__ __align__(16) float s_ab[D * LD];
  float (*const s_g)[D + 1] = reinterpret_cast<float (*)[D + 1]>(s_ab);
  float (*const s_bq)[LD] = reinterpret_cast<float (*)[LD]>(s_ab);
  __shared__ __align__(16) float s_bk[D][LD];   // B_k[c][e] = tau dG[e][c] / nq_e
  __shared__ float s_sp[2 * RPP][D]; // shares of s_e and t_c
  __shared__ float s_nrm[2 * D];     // nq, nk
  __shared__ float s_st[2 * D];      // s_e, t_c
  __shared__ float s_red[NW];
  __shared__ int32_t s_row[kXcaRows];
  const int tid = (int)threadIdx.x;
  int32_t w, h;
  xca_item(blockIdx.x, H, w, h);
  if (w >= W) return;
  const size_t b = (size_t)w * H + h;   // this (window, head)'s temperature partial
  if (hdr->magic != kPlanMagic || hdr->n != n || hdr->num_windows != W) {
    if (tid == 0) part[b] = 0.f;
    return;
  }
  const int32_t* pm = hdr->csr ? nullptr : perm;
  const int32_t rb = max(0, min(offs[w], n)), re = max(rb, min(offs[w + 1], n));
  if (rb == re) {
    if (tid == 0) part[b] = 0.f;
    return;
  }
  const size_t rs = (size_t)H * D;
  const int col = h * D;
  const float t = tau[h];

  // 1. N = qhat^T khat (raw sums and column norms), A
  const int e = tid / CPR, c0 = (tid - e * CPR) * EPT;
  float acc[EPT];
#pragma unroll
  for (int u = 0; u < EPT; ++u) acc[u] = 0.f;
  float nrm = 0.f;
  for (int32_t p0 = rb; p0 < re; p0 += kXcaRows) {
    const int nr = min(kXcaRows, re - p0);
    if (p0 != rb) __syncthreads();
    {
      uint4 qr[NP], kr[NP];
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, q, qr, s_row);
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, k, kr, nullptr);
      xca_put<T, D>(qr, s_a);
      xca_put<T, D>(kr, s_b);
    }
    __syncthreads();
    for (int r = 0; r < nr; ++r) {
      const float x = s_a[r][e];
#pragma unroll
      for (int u = 0; u < EPT; ++u) acc[u] += x * s_b[r][c0 + u];
    }
    if (tid < D) {
      for (int r = 0; r < nr; ++r) nrm += s_a[r][tid] * s_a[r][tid];
    } else if (tid < 2 * D) {
      for (int r = 0; r < nr; ++r) nrm += s_b[r][tid - D] * s_b[r][tid - D];
    }
  }
  if (tid < 2 * D) s_nrm[tid] = fmaxf(sqrtf(nrm), 1e-12f);
  __syncthreads();
  float nn[EPT], a[EPT];
  float mx = -3.0e38f;
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    nn[u] = acc[u] / (s_nrm[e] * s_nrm[D + c0 + u]);
    a[u] = t * nn[u];
    mx = fmaxf(mx, a[u]);
  }
#pragma unroll
  for (int m = 1; m < CPR; m <<= 1) mx = fmaxf(mx, __shfl_xor(mx, m, 64));
  float sum = 0.f;
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    a[u] = expf(a[u] - mx);
    sum += a[u];
  }
#pragma unroll
  for (int m = 1; m < CPR; m <<= 1) sum += __shfl_xor(sum, m, 64);
  const float inv = 1.f / sum;
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    a[u] *= inv;
    s_g[e][c0 + u] = a[u];
  }
  __syncthreads();

  // 2. dA = sum_i do_i v_i^T, and dv_i[x3] = sum_e A[e][x3] do_i[e]
  const int x3 = tid % D, r3 = tid / D;
  float acl[D];
#pragma unroll
  for (int j = 0; j < D; ++j) acl[j] = s_g[j][x3];
  float da[EPT];
#pragma unroll
  for (int u = 0; u < EPT; ++u) da[u] = 0.f;
  for (int32_t p0 = rb; p0 < re; p0 += kXcaRows) {
    const int nr = min(kXcaRows, re - p0);
    __syncthreads();   // s_a, s_b, s_row (and s_g's column reads) are done with
    {
      uint4 dr[NP], vr[NP];
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, dout, dr, s_row);
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, v, vr, nullptr);
      xca_put<T, D>(dr, s_a);
      xca_put<T, D>(vr, s_b);
    }
    __syncthreads();
    for (int r = 0; r < nr; ++r) {
      const float x = s_a[r][e];
#pragma unroll
      for (int u = 0; u < EPT; ++u) da[u] += x * s_b[r][c0 + u];
    }
    for (int r = r3; r < nr; r += RPP) {
      const int32_t row = s_row[r];
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < D; j += 4) {
        const float4 x = *reinterpret_cast<const float4*>(&s_a[r][j]);
        s += acl[j] * x.x + acl[j + 1] * x.y + acl[j + 2] * x.z + acl[j + 3] * x.w;
      }
      if (row >= 0) XcaIo<T>::store(dv + (size_t)row * rs + col + x3, s);
    }
  }

  // 3. dG and the temperature partial
  float rsum = 0.f;
#pragma unroll
  for (int u = 0; u < EPT; ++u) rsum += a[u] * da[u];
#pragma unroll
  for (int m = 1; m < CPR; m <<= 1) rsum += __shfl_xor(rsum, m, 64);
  float dg[EPT], pt = 0.f, srow = 0.f;
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    dg[u] = a[u] * (da[u] - rsum);
    pt += dg[u] * nn[u];
  }
  srow = pt;
#pragma unroll
  for (int m = 1; m < CPR; m <<= 1) srow += __shfl_xor(srow, m, 64);   // sum_c dG N over row e
  // the workgroup's sum of dG * N: the rows' sums, wave by wave, in order
  float wsum = (tid - e * CPR) == 0 ? srow : 0.f;
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) wsum += __shfl_xor(wsum, m, 64);
  __syncthreads();   // the last block's readers of s_a, s_b and every reader of s_g (A,
                     // whose place B_q takes) are done
  if ((tid & 63) == 0) s_red[tid >> 6] = wsum;
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    s_bq[e][c0 + u] = t * dg[u] / s_nrm[D + c0 + u];
    s_bk[c0 + u][e] = t * dg[u] / s_nrm[e];
  }
  __syncthreads();
  if (tid == 0) {
    float tot = 0.f;
#pragma unroll
    for (int j = 0; j < NW; ++j) tot += s_red[j];
    part[b] = tot;
  }

  // 4. dqh[:, x3], dkh[:, x3] for rows r3, r3 + RPP, ... of each block, and their
  //    projections on qhat[:, x3], khat[:, x3]
  const float nq = s_nrm[x3], nk = s_nrm[D + x3];
  constexpr int RPT = kXcaRows / RPP;   // rows of a block per thread
  float gqr[RPT], gkr[RPT];
  // dqh and dkh of this thread's rows of the block in LDS: rows B_q[x3] and
  // B_k[x3] are read 4 columns at a time, outside the loop over the rows, so
  // that only one slice of them is held in registers
  auto grads = [&](int nr) {
#pragma unroll
    for (int m = 0; m < RPT; ++m) {
      gqr[m] = 0.f;
      gkr[m] = 0.f;
    }
#pragma unroll
    for (int j = 0; j < D; j += 4) {
      const float4 bq = *reinterpret_cast<const float4*>(&s_bq[x3][j]);
      const float4 bk = *reinterpret_cast<const float4*>(&s_bk[x3][j]);
#pragma unroll
      for (int m = 0; m < RPT; ++m) {
        const int r = r3 + RPP * m;
        if (r < nr) {
          const float4 kx = *reinterpret_cast<const float4*>(&s_b[r][j]);
          const float4 qx = *reinterpret_cast<const float4*>(&s_a[r][j]);
          gqr[m] += bq.x * kx.x + bq.y * kx.y + bq.z * kx.z + bq.w * kx.w;
          gkr[m] += bk.x * qx.x + bk.y * qx.y + bk.z * qx.z + bk.w * qx.w;
        }
      }
    }
  };
  auto fetch_qk = [&](int32_t p0, int nr) {
    uint4 qr[NP], kr[NP];
    xca_fetch<T, D>(pm, p0, nr, n, rs, col, q, qr, s_row);
    xca_fetch<T, D>(pm, p0, nr, n, rs, col, k, kr, nullptr);
    xca_put<T, D>(qr, s_a);
    xca_put<T, D>(kr, s_b);
  };
  float ps = 0.f, pk = 0.f;   // this thread's share of s_x3 and t_x3, in row order
  for (int32_t p0 = rb; p0 < re; p0 += kXcaRows) {
    const int nr = min(kXcaRows, re - p0);
    __syncthreads();
    fetch_qk(p0, nr);
    __syncthreads();
    grads(nr);
#pragma unroll
    for (int m = 0; m < RPT; ++m) {
      const int r = r3 + RPP * m;
      if (r < nr) {
        ps += (s_a[r][x3] / nq) * gqr[m];
        pk += (s_b[r][x3] / nk) * gkr[m];
      }
    }
  }
  // s_x3 = the RPP shares in order (the floor makes the norm a constant: no projection)
  s_sp[r3][x3] = ps;
  s_sp[RPP + r3][x3] = pk;
  __syncthreads();
  if (tid < 2 * D) {
    const int c = tid & (D - 1), which = tid / D;
    float x = 0.f;
#pragma unroll
    for (int j = 0; j < RPP; ++j) x += s_sp[which * RPP + j][c];
    s_st[tid] = s_nrm[tid] > 1e-12f ? x : 0.f;
  }
  __syncthreads();
  const float sq = s_st[x3], tk = s_st[D + x3];

  // 5. dq[:, x3] and dk[:, x3]; a window of one block still has its q, k rows in
  //    LDS and its dqh, dkh in registers
  const bool one_block = re - rb <= kXcaRows;
  for (int32_t p0 = rb; p0 < re; p0 += kXcaRows) {
    const int nr = min(kXcaRows, re - p0);
    if (!one_block) {
      __syncthreads();
      fetch_qk(p0, nr);
      __syncthreads();
      grads(nr);
    }
#pragma unroll
    for (int m = 0; m < RPT; ++m) {
      const int r = r3 + RPP * m;
      if (r >= nr) continue;
      const int32_t row = s_row[r];
      if (row >= 0) {
        XcaIo<T>::store(dq + (size_t)row * rs + col + x3, (gqr[m] - (s_a[r][x3] / nq) * sq) / nq);
        XcaIo<T>::store(dk + (size_t)row * rs + col + x3, (gkr[m] - (s_b[r][x3] / nk) * tk) / nk);
      }
    }
  }
}

// ---------------------------------------------- backward on the matrix cores
// 16-bit storage, d = 32: the chain rule of k_xca_bwd with its contractions on
// the matrix cores, the rows staged in LDS in their storage format, and the same
// three passes (a window of one block stages all four matrices in the first).
//   1. G tile (w / 2, w % 2) of wave w from transpose reads, as the forward;
//      the norms and the softmax in fp32; A rounded to the storage type (bf16:
//      high part and residual).
//   2. dA = sum_r dout_r^T v_r, tile (w / 2, w % 2), from transpose reads; dv =
//      dout A (dv[r][c] = sum_e A[e][c] dout[r][e]): A's columns by transpose
//      reads, dout's rows as they lie; wave w forms rows 16w .. 16w + 15.
//   3. dG and the temperature share in fp32 as before.  B_q[e][c] = tau dG[e][c]
//      / nk_c spans the range of 1 / nk, which a floored norm (a zero column)
//      makes 10^12 times wider than the rest, so the column factor is split:
//      B_q[e][c] k[r][c] = (tau dG[e][c] s_c / nk_c) (k[r][c] / s_c) with s_c =
//      2^floor(log2 nk_c).  The first factor (within [1/2, 1] of tau dG) is
//      scaled by one power of two into [1, 2) and stored as high part and
//      residual (16 bits in bf16, 22 in fp16, no overflow); the second is the
//      staged row rescaled by a power of two (exact, |k / s_c| < 2).  B_k^T
//      (B_k[c][e] = tau dG[e][c] / nq_e) alike with nq_e.
//   4. dqh = k B_q^T and dkh = q B_k^T for rows 16w + i from row reads; the
//      projections s_e and t_c summed from the same fp32 values over the rows
//      (lanes, then waves, in a fixed order), so the one-row window's exact
//      cancellation holds as in k_xca_bwd; then dq, dk.
__device__ __forceinline__ float xca_pow2_scale(float x) {
  if (!(x > 0.f) || !(x < 3.0e38f)) return 1.f;
  const int ex = (int)((__float_as_uint(x) >> 23) & 0xffu) - 127;
  return ldexpf(1.f, min(-ex, 126));
}

// 2^floor(log2 x) for a normal x > 0 (the norms: at least 1e-12)
__device__ __forceinline__ float xca_pow2_floor(float x) {
  return __uint_as_float(__float_as_uint(x) & 0x7f800000u);
}

// A staged row's 8 channels 8g .. 8g + 7, each times a power of two (exact)
template <typename T>
__device__ __forceinline__ Raw<T, 8> xca_rescale(Raw<T, 8> x, const float (&m)[8]) {
  Raw<T, 8> r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = f32_to_u16<T>(u16_to_f32<T>(x[j]) * m[j]);
  return r;
}

template <typename T>
__global__ __launch_bounds__(kXcaThreads) __attribute__((amdgpu_waves_per_eu(5))) void k_xca_bwd_mma(
    const PlanHeader* __restrict__ hdr, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ offs, const float* __restrict__ tau, const T* __restrict__ q,
    const T* __restrict__ k, const T* __restrict__ v, const T* __restrict__ dout,
    T* __restrict__ dq, T* __restrict__ dk, T* __restrict__ dv, float* __restrict__ part,
    int32_t n, int32_t W, int32_t H) {
  constexpr int D = 32;
  constexpr int LDH = D + 8;
  constexpr int EPT = D * D / kXcaThreads;
  constexpr int CPR = D / EPT;
  constexpr int NP = kXcaPerThread<T, D>;
  constexpr int NW = kXcaThreads / 64;
  constexpr bool kPair = std::is_same<T, bf16_t>::value;
  using F = Frag<T, 8>;
  static_assert(NP == 1 && kXcaPieces<T, D> == kXcaThreads, "one piece a thread");
  __shared__ __align__(16) unsigned short s_q[kXcaRows][LDH];
  __shared__ __align__(16) unsigned short s_k[kXcaRows][LDH];
  __shared__ __align__(16) unsigned short s_d[kXcaRows][LDH];   // dout
  __shared__ __align__(16) unsigned short s_v[kXcaRows][LDH];
  // pass 2: [0] A, [1] its residual; from step 3: B_q and its residual
  __shared__ __align__(16) unsigned short s_m[2][D][LDH];
  // from step 3, in the place of the v rows (read last in pass 2): B_k^T and its
  // residual
  unsigned short (*const s_bk)[D][LDH] = reinterpret_cast<unsigned short (*)[D][LDH]>(&s_v[0][0]);
  __shared__ float s_g[D][D + 1];     // G, then dA
  __shared__ float s_nrm[2 * D];
  __shared__ float s_sp[NW][2 * D];   // the waves' shares of s_e and t_c
  __shared__ float s_st[2 * D];       // s_e, t_c
  __shared__ float s_red[3][NW];      // temperature shares; maxima of |B_q|, |B_k|
  __shared__ int32_t s_row[kXcaRows];
  const int tid = (int)threadIdx.x;
  int32_t w, h;
  xca_item(blockIdx.x, H, w, h);
  if (w >= W) return;
  const size_t b = (size_t)w * H + h;   // this (window, head)'s temperature partial
  if (hdr->magic != kPlanMagic || hdr->n != n || hdr->num_windows != W) {
    if (tid == 0) part[b] = 0.f;
    return;
  }
  const int32_t* pm = hdr->csr ? nullptr : perm;
  const int32_t rb = max(0, min(offs[w], n)), re = max(rb, min(offs[w + 1], n));
  if (rb == re) {
    if (tid == 0) part[b] = 0.f;
    return;
  }
  const int lane = tid & 63, wv = tid >> 6;
  const int i = lane & 15, g = lane >> 4;
  const size_t rs = (size_t)H * D;
  const int col = h * D;
  const float t = tau[h];
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  const int pr = tid >> 2, pc = tid & 3;   // piece tid of a block: row tid / 4, channels 8 (tid % 4) ..
  auto put = [&](unsigned short (*s)[LDH], uint4 x) { *reinterpret_cast<uint4*>(&s[pr][8 * pc]) = x; };
  auto row_op = [&](const unsigned short (*s)[LDH], int r) {
    return *reinterpret_cast<const Raw<T, 8>*>(&s[r][8 * g]);
  };
  const bool one = re - rb <= kXcaRows;
  const int et = wv >> 1, ct = wv & 1;

  // 1. G (raw sums) and the column norms
  floatx4 gacc = zero;
  float nrm = 0.f;
  for (int32_t p0 = rb; p0 < re; p0 += kXcaRows) {
    const int nr = min(kXcaRows, re - p0);
    if (p0 != rb) __syncthreads();
    {
      uint4 qr[NP], kr[NP];
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, q, qr, s_row);
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, k, kr, nullptr);
      if (one) {
        uint4 dr[NP], vr[NP];
        xca_fetch<T, D>(pm, p0, nr, n, rs, col, dout, dr, nullptr);
        xca_fetch<T, D>(pm, p0, nr, n, rs, col, v, vr, nullptr);
        put(s_d, dr[0]);
        put(s_v, vr[0]);
      }
      put(s_q, qr[0]);
      put(s_k, kr[0]);
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      if (32 * ks >= nr) break;
      gacc = F::mma(xca_cols<T, LDH>(s_q, 32 * ks, et, i, g), xca_cols<T, LDH>(s_k, 32 * ks, ct, i, g), gacc);
    }
    if (tid < D) {
      for (int r = 0; r < nr; ++r) {
        const float x = u16_to_f32<T>(s_q[r][tid]);
        nrm += x * x;
      }
    } else if (tid < 2 * D) {
      for (int r = 0; r < nr; ++r) {
        const float x = u16_to_f32<T>(s_k[r][tid - D]);
        nrm += x * x;
      }
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) s_g[16 * et + 4 * g + j][16 * ct + i] = gacc[j];
  if (tid < 2 * D) s_nrm[tid] = fmaxf(sqrtf(nrm), 1e-12f);
  __syncthreads();
  // N = G / (nq nk), A = softmax of tau N over c, thread (e, c0 .. c0 + EPT - 1)
  const int e = tid / CPR, c0 = (tid - e * CPR) * EPT;
  float nn[EPT], a[EPT];
  {
    float mx = -3.0e38f;
#pragma unroll
    for (int u = 0; u < EPT; ++u) {
      nn[u] = s_g[e][c0 + u] / (s_nrm[e] * s_nrm[D + c0 + u]);
      a[u] = t * nn[u];
      mx = fmaxf(mx, a[u]);
    }
#pragma unroll
    for (int m = 1; m < CPR; m <<= 1) mx = fmaxf(mx, __shfl_xor(mx, m, 64));
    float sum = 0.f;
#pragma unroll
    for (int u = 0; u < EPT; ++u) {
      a[u] = expf(a[u] - mx);
      sum += a[u];
    }
#pragma unroll
    for (int m = 1; m < CPR; m <<= 1) sum += __shfl_xor(sum, m, 64);
    const float inv = 1.f / sum;
#pragma unroll
    for (int u = 0; u < EPT; ++u) {
      a[u] *= inv;
      const unsigned short hi = f32_to_u16<T>(a[u]);
      s_m[0][e][c0 + u] = hi;
      if constexpr (kPair) s_m[1][e][c0 + u] = f32_to_u16<T>(a[u] - u16_to_f32<T>(hi));
    }
  }
  __syncthreads();

  // 2. dA, and dv = dout A for rows 16 wv + i of each block
  Raw<T, 8> at[2], atl[2];
#pragma unroll
  for (int t2 = 0; t2 < 2; ++t2) {
    at[t2] = xca_cols<T, LDH>(s_m[0], 0, t2, i, g);
    if constexpr (kPair) atl[t2] = xca_cols<T, LDH>(s_m[1], 0, t2, i, g);
  }
  floatx4 dacc = zero;
  for (int32_t p0 = rb; p0 < re; p0 += kXcaRows) {
    const int nr = min(kXcaRows, re - p0);
    if (!one) {
      __syncthreads();   // the previous block's readers of s_d, s_v, s_row are done
      uint4 dr[NP], vr[NP];
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, dout, dr, s_row);
      xca_fetch<T, D>(pm, p0, nr, n, rs, col, v, vr, nullptr);
      put(s_d, dr[0]);
      put(s_v, vr[0]);
      __syncthreads();
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      if (32 * ks >= nr) break;
      dacc = F::mma(xca_cols<T, LDH>(s_d, 32 * ks, et, i, g), xca_cols<T, LDH>(s_v, 32 * ks, ct, i, g), dacc);
    }
    if (16 * wv < nr) {
      const int r = 16 * wv + i;
      const Raw<T, 8> db = row_op(s_d, r);
      const int32_t row = r < nr ? s_row[r] : -1;
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2) {
        floatx4 d4 = F::mma(at[t2], db, zero);
        if constexpr (kPair) d4 = F::mma(atl[t2], db, d4);
        if (row >= 0) {
          u16x4 pk;
#pragma unroll
          for (int j = 0; j < 4; ++j) pk[j] = f32_to_u16<T>(d4[j]);
          *reinterpret_cast<u16x4*>(dv + (size_t)row * rs + col + 16 * t2 + 4 * g) = pk;
        }
      }
    }
  }
  // s_g's readers (the softmax) passed the barrier after it
#pragma unroll
  for (int j = 0; j < 4; ++j) s_g[16 * et + 4 * g + j][16 * ct + i] = dacc[j];
  __syncthreads();   // also: every reader of A in s_m and of the v rows is done

  // 3. dG, the temperature share, B_q and B_k^T
  float bq[EPT], bk[EPT];
  {
    float da[EPT], rsum = 0.f;
#pragma unroll
    for (int u = 0; u < EPT; ++u) {
      da[u] = s_g[e][c0 + u];
      rsum += a[u] * da[u];
    }
#pragma unroll
    for (int m = 1; m < CPR; m <<= 1) rsum += __shfl_xor(rsum, m, 64);
    float pt = 0.f, mq = 0.f, mk = 0.f;
    const float nqe = s_nrm[e];
#pragma unroll
    for (int u = 0; u < EPT; ++u) {
      const float dg = a[u] * (da[u] - rsum);
      const float nkc = s_nrm[D + c0 + u];
      pt += dg * nn[u];
      bq[u] = t * dg * (xca_pow2_floor(nkc) / nkc);
      bk[u] = t * dg * (xca_pow2_floor(nqe) / nqe);
      mq = fmaxf(mq, fabsf(bq[u]));
      mk = fmaxf(mk, fabsf(bk[u]));
    }
    float srow = pt;
#pragma unroll
    for (int m = 1; m < CPR; m <<= 1) srow += __shfl_xor(srow, m, 64);   // sum_c dG N over row e
    float wsum = (tid - e * CPR) == 0 ? srow : 0.f;
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) {
      wsum += __shfl_xor(wsum, m, 64);
      mq = fmaxf(mq, __shfl_xor(mq, m, 64));
      mk = fmaxf(mk, __shfl_xor(mk, m, 64));
    }
    if (lane == 0) {
      s_red[0][wv] = wsum;
      s_red[1][wv] = mq;
      s_red[2][wv] = mk;
    }
  }
  __syncthreads();
  float mq = 0.f, mk = 0.f;
#pragma unroll
  for (int j = 0; j < NW; ++j) {
    mq = fmaxf(mq, s_red[1][j]);
    mk = fmaxf(mk, s_red[2][j]);
  }
  const float sq_ = xca_pow2_scale(mq), sk_ = xca_pow2_scale(mk);
  if (tid == 0) {
    float tot = 0.f;
#pragma unroll
    for (int j = 0; j < NW; ++j) tot += s_red[0][j];
    part[b] = tot;
  }
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    const float xq = bq[u] * sq_, xk = bk[u] * sk_;
    const unsigned short hq = f32_to_u16<T>(xq), hk = f32_to_u16<T>(xk);
    s_m[0][e][c0 + u] = hq;
    s_m[1][e][c0 + u] = f32_to_u16<T>(xq - u16_to_f32<T>(hq));
    s_bk[0][c0 + u][e] = hk;
    s_bk[1][c0 + u][e] = f32_to_u16<T>(xk - u16_to_f32<T>(hk));
  }
  __syncthreads();

  // 4. dqh, dkh of rows 16 wv + i, their projections, then dq, dk
  const float iq = 1.f / sq_, ik = 1.f / sk_;
  float gq[2][4], gk[2][4];   // dqh[r][16 t2 + 4 g + j], dkh[r][16 t2 + 4 g + j]
  // (the B operands, the norms and the column scales are read from LDS where they
  // are used: held in registers they cost a fourth workgroup per CU)
  auto grads = [&](int r) {
    float ik8[8], iq8[8];   // 1 / s_c for this lane's channels 8g .. 8g + 7
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      ik8[j] = 1.f / xca_pow2_floor(s_nrm[D + 8 * g + j]);
      iq8[j] = 1.f / xca_pow2_floor(s_nrm[8 * g + j]);
    }
    const Raw<T, 8> kb = xca_rescale<T>(row_op(s_k, r), ik8), qb = xca_rescale<T>(row_op(s_q, r), iq8);
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      const floatx4 x = F::mma(row_op(s_m[1], 16 * t2 + i), kb, F::mma(row_op(s_m[0], 16 * t2 + i), kb, zero));
      const floatx4 y = F::mma(row_op(s_bk[1], 16 * t2 + i), qb, F::mma(row_op(s_bk[0], 16 * t2 + i), qb, zero));
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        gq[t2][j] = x[j] * iq;
        gk[t2][j] = y[j] * ik;
      }
    }
  };
  auto fetch_qk = [&](int32_t p0, int nr) {
    uint4 qr[NP], kr[NP];
    xca_fetch<T, D>(pm, p0, nr, n, rs, col, q, qr, s_row);
    xca_fetch<T, D>(pm, p0, nr, n, rs, col, k, kr, nullptr);
    put(s_q, qr[0]);
    put(s_k, kr[0]);
  };
  float ps[2][4] = {}, pk[2][4] = {};
  for (int32_t p0 = rb; p0 < re; p0 += kXcaRows) {
    const int nr = min(kXcaRows, re - p0);
    if (!one) {
      __syncthreads();
      fetch_qk(p0, nr);
      __syncthreads();
    }
    const int r = 16 * wv + i;
    if (16 * wv < nr) {
      grads(r);
      if (r < nr) {
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2) {
          const u16x4 qx = *reinterpret_cast<const u16x4*>(&s_q[r][16 * t2 + 4 * g]);
          const u16x4 kx = *reinterpret_cast<const u16x4*>(&s_k[r][16 * t2 + 4 * g]);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            ps[t2][j] += (u16_to_f32<T>(qx[j]) / s_nrm[16 * t2 + 4 * g + j]) * gq[t2][j];
            pk[t2][j] += (u16_to_f32<T>(kx[j]) / s_nrm[D + 16 * t2 + 4 * g + j]) * gk[t2][j];
          }
        }
      }
    }
  }
  // the rows' shares: over the 16 lanes of a group (rows 16 wv + i), then the waves
#pragma unroll
  for (int m = 1; m < 16; m <<= 1)
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        ps[t2][j] += __shfl_xor(ps[t2][j], m, 64);
        pk[t2][j] += __shfl_xor(pk[t2][j], m, 64);
      }
  if (i == 0) {
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        s_sp[wv][16 * t2 + 4 * g + j] = ps[t2][j];
        s_sp[wv][D + 16 * t2 + 4 * g + j] = pk[t2][j];
      }
  }
  __syncthreads();
  if (tid < 2 * D) {
    float x = 0.f;
#pragma unroll
    for (int j = 0; j < NW; ++j) x += s_sp[j][tid];
    s_st[tid] = s_nrm[tid] > 1e-12f ? x : 0.f;   // a floored norm is a constant: no projection
  }
  __syncthreads();
  float sv[2][4], tv[2][4];
#pragma unroll
  for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      sv[t2][j] = s_st[16 * t2 + 4 * g + j];
      tv[t2][j] = s_st[D + 16 * t2 + 4 * g + j];
    }
  for (int32_t p0 = rb; p0 < re; p0 += kXcaRows) {
    const int nr = min(kXcaRows, re - p0);
    if (!one) {
      __syncthreads();
      fetch_qk(p0, nr);
      __syncthreads();
    }
    const int r = 16 * wv + i;
    if (16 * wv >= nr) continue;
    if (!one) grads(r);
    const int32_t row = r < nr ? s_row[r] : -1;
    if (row < 0) continue;
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      const u16x4 qx = *reinterpret_cast<const u16x4*>(&s_q[r][16 * t2 + 4 * g]);
      const u16x4 kx = *reinterpret_cast<const u16x4*>(&s_k[r][16 * t2 + 4 * g]);
      u16x4 oq, ok;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float nq = s_nrm[16 * t2 + 4 * g + j], nk = s_nrm[D + 16 * t2 + 4 * g + j];
        oq[j] = f32_to_u16<T>((gq[t2][j] - (u16_to_f32<T>(qx[j]) / nq) * sv[t2][j]) / nq);
        ok[j] = f32_to_u16<T>((gk[t2][j] - (u16_to_f32<T>(kx[j]) / nk) * tv[t2][j]) / nk);
      }
      *reinterpret_cast<u16x4*>(dq + (size_t)row * rs + col + 16 * t2 + 4 * g) = oq;
      *reinterpret_cast<u16x4*>(dk + (size_t)row * rs + col + 16 * t2 + 4 * g) = ok;
    }
  }
}

// dtau[h] = sum over windows, in window order, of the (window, head) partials:
// 256 strided sums, then a fixed tree.
__global__ __launch_bounds__(kXcaThreads) void k_xca_dtau(const float* __restrict__ part, int32_t W,
                                                         int32_t H, float* __restrict__ dtau) {
  __shared__ float s[kXcaThreads];
  const int h = (int)blockIdx.x, tid = (int)threadIdx.x;
  float x = 0.f;
  for (int32_t w = tid; w < W; w += kXcaThreads) x += part[(size_t)w * H + h];
  s[tid] = x;
  __syncthreads();
  for (int m = kXcaThreads / 2; m > 0; m >>= 1) {
    if (tid < m) s[tid] += s[tid + m];
    __syncthreads();
  }
  if (tid == 0) dtau[h] = s[0];
}

template <typename T, int D>
hipError_t xca_bwd_impl(const void* plan, int32_t n, int32_t W, int32_t H, const float* tau,
                        const void* q, const void* k, const void* v, const void* dout, void* dq,
                        void* dk, void* dv, float* dtau, float* part, hipStream_t stream) {
  const PlanLayout lay = plan_layout(n, W);
  const char* base = static_cast<const char*>(plan);
  if constexpr (Ty<T>::kNarrow && D == 32)
    hipLaunchKernelGGL((k_xca_bwd_mma<T>), dim3(xca_grid(W, H)), dim3(kXcaThreads), 0, stream,
                       reinterpret_cast<const PlanHeader*>(base + lay.header),
                       reinterpret_cast<const int32_t*>(base + lay.perm),
                       reinterpret_cast<const int32_t*>(base + lay.offsets), tau,
                       static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v),
                       static_cast<const T*>(dout), static_cast<T*>(dq), static_cast<T*>(dk),
                       static_cast<T*>(dv), part, n, W, H);
  else
  hipLaunchKernelGGL((k_xca_bwd<T, D>), dim3(xca_grid(W, H)), dim3(kXcaThreads), 0, stream,
                     reinterpret_cast<const PlanHeader*>(base + lay.header),
                     reinterpret_cast<const int32_t*>(base + lay.perm),
                     reinterpret_cast<const int32_t*>(base + lay.offsets), tau,
                     static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v),
                     static_cast<const T*>(dout), static_cast<T*>(dq), static_cast<T*>(dk),
                     static_cast<T*>(dv), part, n, W, H);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_xca_dtau, dim3((unsigned)H), dim3(kXcaThreads), 0, stream, part, W, H, dtau);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t xca_impl(const void* plan, int32_t n, int32_t W, int32_t H, const float* tau,
                    const void* q, const void* k, const void* v, void* o, hipStream_t stream) {
  const PlanLayout lay = plan_layout(n, W);
  const char* base = static_cast<const char*>(plan);
  if constexpr (Ty<T>::kNarrow && D == 32) {
    hipLaunchKernelGGL((k_xca_fwd_mma<T>), dim3(xca_grid(W, H)), dim3(kXcaThreads), 0, stream,
                       reinterpret_cast<const PlanHeader*>(base + lay.header),
                       reinterpret_cast<const int32_t*>(base + lay.perm),
                       reinterpret_cast<const int32_t*>(base + lay.offsets), tau,
                       static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v),
                       static_cast<T*>(o), n, W, H);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((k_xca_fwd<T, D>), dim3(xca_grid(W, H)), dim3(kXcaThreads), 0, stream,
                     reinterpret_cast<const PlanHeader*>(base + lay.header),
                     reinterpret_cast<const int32_t*>(base + lay.perm),
                     reinterpret_cast<const int32_t*>(base + lay.offsets), tau,
                     static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v),
                     static_cast<T*>(o), n, W, H);
  return hipGetLastError();
}

}  // namespace

// dtype: 0 f32, 1 f16, 2 bf16; d: 16 or 32
hipError_t launch_forward_xca(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                              const float* tau, const void* q, const void* k, const void* v, void* o,
                              hipStream_t stream) {
  if (d == 32) {
    if (dtype == 0) return xca_impl<float, 32>(plan, n, W, H, tau, q, k, v, o, stream);
    if (dtype == 1) return xca_impl<_Float16, 32>(plan, n, W, H, tau, q, k, v, o, stream);
    return xca_impl<bf16_t, 32>(plan, n, W, H, tau, q, k, v, o, stream);
  }
  if (dtype == 0) return xca_impl<float, 16>(plan, n, W, H, tau, q, k, v, o, stream);
  if (dtype == 1) return xca_impl<_Float16, 16>(plan, n, W, H, tau, q, k, v, o, stream);
  return xca_impl<bf16_t, 16>(plan, n, W, H, tau, q, k, v, o, stream);
}

hipError_t launch_backward_xca(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                               const float* tau, const void* q, const void* k, const void* v,
                               const void* dout, void* dq, void* dk, void* dv, float* dtau, float* part,
                               hipStream_t stream) {
  if (d == 32) {
    if (dtype == 0) return xca_bwd_impl<float, 32>(plan, n, W, H, tau, q, k, v, dout, dq, dk, dv, dtau, part, stream);
    if (dtype == 1) return xca_bwd_impl<_Float16, 32>(plan, n, W, H, tau, q, k, v, dout, dq, dk, dv, dtau, part, stream);
    return xca_bwd_impl<bf16_t, 32>(plan, n, W, H, tau, q, k, v, dout, dq, dk, dv, dtau, part, stream);
  }
  if (dtype == 0) return xca_bwd_impl<float, 16>(plan, n, W, H, tau, q, k, v, dout, dq, dk, dv, dtau, part, stream);
  if (dtype == 1) return xca_bwd_impl<_Float16, 16>(plan, n, W, H, tau, q, k, v, dout, dq, dk, dv, dtau, part, stream);
  return xca_bwd_impl<bf16_t, 16>(plan, n, W, H, tau, q, k, v, dout, dq, dk, dv, dtau, part, stream);
}

// Device address of `scratch` on the current device (nullptr and the HIP error
// if it cannot be looked up).  Looked up once per device, with that device current.
static float* scratch_address(hipError_t& err) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static float* addr[kMaxDevices] = {};
  int dev = 0;
  err = hipGetDevice(&dev);
  if (err != hipSuccess) return nullptr;
  if (dev < 0 || dev >= kMaxDevices) {
    err = hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess) return nullptr;
    addr[dev] = static_cast<float*>(p);
  }
  err = hipSuccess;
  return addr[dev];
}

// sla_backward_xca with the dtau partials in `scratch` (num_windows * heads <=
// kXcaScratchFloats, checked by the caller).  Every partial is written by every
// call, so nothing is cleared.
hipError_t launch_backward_xca_noalloc(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                                       const float* tau, const void* q, const void* k, const void* v,
                                       const void* dout, void* dq, void* dk, void* dv, float* dtau,
                                       hipStream_t stream) {
  hipError_t err;
  float* part = scratch_address(err);
  if (part == nullptr) return err;
  return launch_backward_xca(plan, n, W, dtype, H, d, tau, q, k, v, dout, dq, dk, dv, dtau, part, stream);
}

}  // namespace sla

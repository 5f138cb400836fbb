// SLA forward and backward on the gfx950 matrix cores.
//
// Work decomposition: one wavefront per (chunk, head); a workgroup holds the
// waves of consecutive heads of one chunk, so the rows a workgroup gathers are
// shared by its waves through the cache.  A chunk is a run of whole windows of
// the window-sorted sequence (see the builder); the wave walks its windows, and
// for each window
//   1. streams the window's K and V rows (gathered through the plan's
//      permutation) in 32-row tiles and accumulates the state
//      S = phi(K)^T V on the matrix cores and z = sum phi(K) in fp32
//      (Eq. (3) numerator and normaliser; the chunk-wise state accumulation of
//      Sec. 3.2 / Fig. 3(b));
//   2. streams the window's Q rows in 16-row tiles and writes
//      o = phi(q) S / (phi(q) . z) (Eq. (3)).
// The state never leaves the wave (registers + a per-wave LDS tile), so the only
// HBM traffic is reading q, k, v and writing o.
//
// Register layouts (lane l = 16 g + i, g = lane group 0..3, KS = head_dim / 4):
//   natural fragment   lane (i, g) holds elements KS*g .. KS*g + KS - 1 of row i
//                      of a 16-row tile -- one contiguous 16 B (d = 32, 16-bit)
//                      or 8 B (d = 16, 16-bit) load per lane;
//   transposed tile    the contraction over ROWS needs each lane to hold 8 rows
//                      of one column; a natural fragment times a 0/1 selection
//                      matrix on the matrix core (exact) yields lane (i, g)
//                      holding rows 4g .. 4g+3 of column i, the standard 16x16
//                      result layout.  Two 16-row sub-tiles give the 8 rows.
// Contractions over the head dimension (phi(q) S, dS v^T, ...) take natural
// fragments directly; their per-window matrix operand is read from the wave's
// LDS copy of S (or dS), with the output-row order chosen so that each lane's
// results are again KS consecutive elements of one row (one vector store).
//
// 16-bit storage: matrix-core operands are rounded to the storage type.  Derived
// operands are scaled by a power of two into [1, 2) (S, dS) or below 1
// (phi(q)/den) before rounding, and the scale is divided out in fp32, so no
// operand overflows or flushes; the normaliser, divisions and phi are fp32.
#include "sla_common.h"

namespace sla {

template <typename T>
__device__ __forceinline__ float phi_f(float x) {
  if constexpr (Ty<T>::kNarrow) {
    return x > 0.f ? x + 1.f : __expf(x);
  } else {
    return x > 0.f ? x + 1.f : expf(x);
  }
}

template <typename T>
__device__ __forceinline__ float dphi_f(float x) {
  if constexpr (Ty<T>::kNarrow) {
    return x > 0.f ? 1.f : __expf(x);
  } else {
    return x > 0.f ? 1.f : expf(x);
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

template <int D>
struct Geo {
  static constexpr int KS = D / 4;   // slots per lane group along the head dim
  static constexpr int NT = D / 16;  // 16-wide tiles along the head dim
  static constexpr int kScratch = D * D + 2 * D;  // per-wave LDS floats
  // Row of the result tile -> head-dim index, so that lane group g receives the
  // KS consecutive indices KS*g .. KS*g + KS - 1 across the NT tiles.
  __device__ static int out_index(int tile, int m) { return KS * (m >> 2) + 4 * tile + (m & 3); }
};

struct RowSrc {
  const int32_t* perm;  // nullptr: identity
  int32_t n;
  __device__ __forceinline__ int32_t orig(int32_t r, bool& ok) const {
    int32_t o = ok ? (perm ? perm[r] : r) : 0;
    ok = ok && (uint32_t)o < (uint32_t)n;
    return ok ? o : 0;
  }
};

template <typename T, int D>
__device__ __forceinline__ void load_row(const T* base, int32_t orig, bool ok, size_t rowstride,
                                         int col, float (&x)[Geo<D>::KS]) {
  if (ok) {
    load_frag<T, Geo<D>::KS>(base + (size_t)orig * rowstride + col, x);
  } else {
#pragma unroll
    for (int r = 0; r < Geo<D>::KS; ++r) x[r] = 0.f;
  }
}

// Selection matrix for the transpose of tile t: slot (g, r) -> head index KS*g+r.
template <int D>
__device__ __forceinline__ void make_sel(float (&sel)[Geo<D>::NT][Geo<D>::KS], int i, int g) {
#pragma unroll
  for (int t = 0; t < Geo<D>::NT; ++t)
#pragma unroll
    for (int r = 0; r < Geo<D>::KS; ++r) sel[t][r] = (Geo<D>::KS * g + r == 16 * t + i) ? 1.f : 0.f;
}

// Accumulate the state of rows [r0, r0 + 32) n [.., rend) of one window:
// acc[et][ct] += phi(K)^T V (tile et of e, tile ct of c), zp[t] += column sums of
// phi(K) over this lane's rows.
template <typename T, int D>
__device__ __forceinline__ void state_tile(const T* k, const T* v, const RowSrc& src,
                                           int32_t r0, int32_t rend, size_t rowstride, int col,
                                           const float (&sel)[Geo<D>::NT][Geo<D>::KS], int i,
                                           floatx4 (&acc)[Geo<D>::NT][Geo<D>::NT],
                                           float (&zp)[Geo<D>::NT]) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  float kx[2][KS], vx[2][KS];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    bool ok = r0 + 16 * s + i < rend;
    const int32_t o = src.orig(r0 + 16 * s + i, ok);
    load_row<T, D>(k, o, ok, rowstride, col, kx[s]);
    load_row<T, D>(v, o, ok, rowstride, col, vx[s]);
#pragma unroll
    for (int r = 0; r < KS; ++r) kx[s][r] = ok ? Ty<T>::round(phi_f<T>(kx[s][r])) : 0.f;
  }
  floatx4 tk[2][NT], tv[2][NT];
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      tk[s][t] = Mma<T, KS>::run(kx[s], sel[t], zero);
      tv[s][t] = Mma<T, KS>::run(vx[s], sel[t], zero);
    }
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int j = 0; j < 4; ++j) zp[t] += tk[0][t][j] + tk[1][t][j];
#pragma unroll
  for (int et = 0; et < NT; ++et)
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      float a[8], b[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        a[j] = tk[0][et][j];
        a[4 + j] = tk[1][et][j];
        b[j] = tv[0][ct][j];
        b[4 + j] = tv[1][ct][j];
      }
      acc[et][ct] = Mma<T, 8>::run(a, b, acc[et][ct]);
    }
}

// Full state of one window: S into sS[e * D + c] (fp32), z into sZ[e].
// Returns max |S| over the window.
template <typename T, int D>
__device__ __forceinline__ float window_state(const T* k, const T* v, const RowSrc& src,
                                              int32_t ws, int32_t we, size_t rowstride, int col,
                                              const float (&sel)[Geo<D>::NT][Geo<D>::KS], int i,
                                              int g, float* sS, float* sZ) {
  constexpr int NT = Geo<D>::NT;
  floatx4 acc[NT][NT];
  float zp[NT];
#pragma unroll
  for (int a = 0; a < NT; ++a) {
    zp[a] = 0.f;
#pragma unroll
    for (int b = 0; b < NT; ++b) acc[a][b] = {0.f, 0.f, 0.f, 0.f};
  }
  for (int32_t r0 = ws; r0 < we; r0 += 32)
    state_tile<T, D>(k, v, src, r0, we, rowstride, col, sel, i, acc, zp);
  float mx = 0.f;
  wave_lds_sync();
#pragma unroll
  for (int et = 0; et < NT; ++et)
#pragma unroll
    for (int ct = 0; ct < NT; ++ct)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        sS[(16 * et + 4 * g + j) * D + 16 * ct + i] = acc[et][ct][j];
        mx = fmaxf(mx, fabsf(acc[et][ct][j]));
      }
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    float z = zp[t] + shfl_xor_f(zp[t], 16);
    z += shfl_xor_f(z, 32);
    if (g == 0) sZ[16 * t + i] = z;
  }
  wave_lds_sync();
  return wave_max(mx);
}

// ------------------------------------------------------------------ forward
template <typename T, int D>
__global__ __launch_bounds__(512) void k_sla_fwd(const PlanHeader* __restrict__ hdr,
                                                  const int32_t* __restrict__ perm_plan,
                                                  const int32_t* __restrict__ offs,
                                                  const Chunk* __restrict__ chunks,
                                                  int32_t max_chunks, int32_t n, int32_t W,
                                                  int32_t H, int32_t hpw, const T* __restrict__ q,
                                                  const T* __restrict__ k, const T* __restrict__ v,
                                                  T* __restrict__ o) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  extern __shared__ float smem[];
  const int lane = lane_id(), wv = threadIdx.x >> 6;
  const int h = blockIdx.y * hpw + wv;
  if (h >= H) return;
  if (hdr->magic != kPlanMagic || hdr->n != n || hdr->num_windows != W) return;
  const int32_t nchunks = min(hdr->n_chunks, max_chunks);
  RowSrc src{hdr->csr ? nullptr : perm_plan, n};
  float* sS = smem + wv * Geo<D>::kScratch;
  float* sZ = sS + D * D;
  const int i = lane & 15, g = lane >> 4;
  const size_t rowstride = (size_t)H * D;
  const int col = h * D + KS * g;
  float sel[NT][KS];
  make_sel<D>(sel, i, g);

  for (int32_t c = blockIdx.x; c < nchunks; c += gridDim.x) {
    const Chunk ch = chunks[c];
    const int32_t rb = max(0, min(ch.row_begin, n)), re = max(rb, min(ch.row_end, n));
    const int32_t wb = max(0, min(ch.win_begin, W)), wend = max(wb, min(ch.win_end, W));
    for (int32_t w = wb; w < wend; ++w) {
      const int32_t ws = max(offs[w], rb), we = min(offs[w + 1], re);
      if (ws >= we) continue;
      const float mx = window_state<T, D>(k, v, src, ws, we, rowstride, col, sel, i, g, sS, sZ);
      const float sig = Ty<T>::kNarrow ? pow2_scale_to_one(mx) : 1.f;
      float A[NT][KS], zr[KS];
#pragma unroll
      for (int ct = 0; ct < NT; ++ct)
#pragma unroll
        for (int r = 0; r < KS; ++r) A[ct][r] = sig * sS[(KS * g + r) * D + Geo<D>::out_index(ct, i)];
#pragma unroll
      for (int r = 0; r < KS; ++r) zr[r] = sZ[KS * g + r];
      const float inv_sig = 1.f / sig;
      for (int32_t r0 = ws; r0 < we; r0 += 16) {
        bool ok = r0 + i < we;
        const int32_t orow = src.orig(r0 + i, ok);
        float qx[KS];
        load_row<T, D>(q, orow, ok, rowstride, col, qx);
        float den = 0.f;
#pragma unroll
        for (int r = 0; r < KS; ++r) {
          qx[r] = ok ? Ty<T>::round(phi_f<T>(qx[r])) : 0.f;
          den += qx[r] * zr[r];
        }
        den += shfl_xor_f(den, 16);
        den += shfl_xor_f(den, 32);
        const float scale = ok ? inv_sig / den : 0.f;
        float ox[KS];
#pragma unroll
        for (int ct = 0; ct < NT; ++ct) {
          const floatx4 d4 = Mma<T, KS>::run(A[ct], qx, floatx4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
          for (int j = 0; j < 4; ++j) ox[4 * ct + j] = d4[j] * scale;
        }
        if (ok) store_frag<T, KS>(o + (size_t)orow * rowstride + col, ox);
      }
    }
  }
}

// ----------------------------------------------------------------- backward
template <typename T, int D>
__global__ __launch_bounds__(256) void k_sla_bwd(const PlanHeader* __restrict__ hdr,
                                                  const int32_t* __restrict__ perm_plan,
                                                  const int32_t* __restrict__ offs,
                                                  const Chunk* __restrict__ chunks,
                                                  int32_t max_chunks, int32_t n, int32_t W,
                                                  int32_t H, int32_t hpw, const T* __restrict__ q,
                                                  const T* __restrict__ k, const T* __restrict__ v,
                                                  const T* __restrict__ dout, T* __restrict__ dq,
                                                  T* __restrict__ dk, T* __restrict__ dv) {
  constexpr int KS = Geo<D>::KS, NT = Geo<D>::NT;
  extern __shared__ float smem[];
  const int lane = lane_id(), wv = threadIdx.x >> 6;
  const int h = blockIdx.y * hpw + wv;
  if (h >= H) return;
  if (hdr->magic != kPlanMagic || hdr->n != n || hdr->num_windows != W) return;
  const int32_t nchunks = min(hdr->n_chunks, max_chunks);
  RowSrc src{hdr->csr ? nullptr : perm_plan, n};
  float* sS = smem + wv * Geo<D>::kScratch;
  float* sZ = sS + D * D;
  const int i = lane & 15, g = lane >> 4;
  const size_t rowstride = (size_t)H * D;
  const int col = h * D + KS * g;
  float sel[NT][KS];
  make_sel<D>(sel, i, g);
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};

  for (int32_t c = blockIdx.x; c < nchunks; c += gridDim.x) {
    const Chunk ch = chunks[c];
    const int32_t rb = max(0, min(ch.row_begin, n)), re = max(rb, min(ch.row_end, n));
    const int32_t wb = max(0, min(ch.win_begin, W)), wend = max(wb, min(ch.win_end, W));
    for (int32_t w = wb; w < wend; ++w) {
      const int32_t ws = max(offs[w], rb), we = min(offs[w + 1], re);
      if (ws >= we) continue;
      // ---- pass 1: window state
      const float mx = window_state<T, D>(k, v, src, ws, we, rowstride, col, sel, i, g, sS, sZ);
      const float sig = Ty<T>::kNarrow ? pow2_scale_to_one(mx) : 1.f;
      const float inv_sig = 1.f / sig;
      float Anum[NT][KS], Adq[NT][KS], zr[KS];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < KS; ++r) {
          Anum[t][r] = sig * sS[(KS * g + r) * D + Geo<D>::out_index(t, i)];
          Adq[t][r] = sig * sS[Geo<D>::out_index(t, i) * D + KS * g + r];
        }
      float zmin = 3.0e38f;
#pragma unroll
      for (int r = 0; r < KS; ++r) {
        zr[r] = sZ[KS * g + r];
        zmin = fminf(zmin, zr[r]);
      }
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) zmin = fminf(zmin, shfl_xor_f(zmin, m));
      // phi(q)/den <= 1/min(z), so beta = 2^floor(log2 min z) keeps X = beta phi(q)/den <= 1
      const float beta = Ty<T>::kNarrow ? pow2_floor(zmin) : 1.f;
      const float inv_beta = 1.f / beta;

      // ---- pass 2: dq, and dS = sum phi(q)^T dout / den, dz = -sum (dout.o) phi(q) / den
      floatx4 accd[NT][NT];
      float dzp[NT];
#pragma unroll
      for (int a = 0; a < NT; ++a) {
        dzp[a] = 0.f;
#pragma unroll
        for (int b = 0; b < NT; ++b) accd[a][b] = zero;
      }
      for (int32_t r0 = ws; r0 < we; r0 += 32) {
        float xs[2][KS], ds[2][KS], dots[2];
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          bool ok = r0 + 16 * s + i < we;
          const int32_t orow = src.orig(r0 + 16 * s + i, ok);
          float qx[KS], fq[KS];
          load_row<T, D>(q, orow, ok, rowstride, col, qx);
          load_row<T, D>(dout, orow, ok, rowstride, col, ds[s]);
          float den = 0.f;
#pragma unroll
          for (int r = 0; r < KS; ++r) {
            fq[r] = ok ? Ty<T>::round(phi_f<T>(qx[r])) : 0.f;
            den += fq[r] * zr[r];
          }
          den += shfl_xor_f(den, 16);
          den += shfl_xor_f(den, 32);
          if (!ok) den = 1.f;
          const float inv_den = 1.f / den;
          // o and dout . o
          float dot = 0.f;
#pragma unroll
          for (int t = 0; t < NT; ++t) {
            const floatx4 d4 = Mma<T, KS>::run(Anum[t], fq, zero);
#pragma unroll
            for (int j = 0; j < 4; ++j) dot += ds[s][4 * t + j] * (d4[j] * inv_sig * inv_den);
          }
          dot += shfl_xor_f(dot, 16);
          dot += shfl_xor_f(dot, 32);
          dots[s] = ok ? dot : 0.f;
          // dphi(q) = (dout S^T - (dout . o) z) / den ;  dq = dphi(q) * phi'(q)
          float dqx[KS];
#pragma unroll
          for (int t = 0; t < NT; ++t) {
            const floatx4 d4 = Mma<T, KS>::run(Adq[t], ds[s], zero);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int r = 4 * t + j;
              dqx[r] = (d4[j] * inv_sig - dot * zr[r]) * inv_den * dphi_f<T>(qx[r]);
            }
          }
          if (ok) store_frag<T, KS>(dq + (size_t)orow * rowstride + col, dqx);
#pragma unroll
          for (int r = 0; r < KS; ++r) xs[s][r] = ok ? Ty<T>::round(fq[r] * beta * inv_den) : 0.f;
        }
        floatx4 tx[2][NT], td[2][NT];
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
          for (int t = 0; t < NT; ++t) {
            tx[s][t] = Mma<T, KS>::run(xs[s], sel[t], zero);
            td[s][t] = Mma<T, KS>::run(ds[s], sel[t], zero);
          }
        // dz (times beta): lane (i, g) holds rows 4g+j of each sub-tile, column 16t+i
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float dr = shfl_f(dots[s], 4 * g + j);
#pragma unroll
            for (int t = 0; t < NT; ++t) dzp[t] -= tx[s][t][j] * dr;
          }
#pragma unroll
        for (int et = 0; et < NT; ++et)
#pragma unroll
          for (int ct = 0; ct < NT; ++ct) {
            float a[8], b[8];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              a[j] = tx[0][et][j];
              a[4 + j] = tx[1][et][j];
              b[j] = td[0][ct][j];
              b[4 + j] = td[1][ct][j];
            }
            accd[et][ct] = Mma<T, 8>::run(a, b, accd[et][ct]);
          }
      }
      // dS, dz -> LDS (unscaled)
      wave_lds_sync();
      float mxd = 0.f;
#pragma unroll
      for (int et = 0; et < NT; ++et)
#pragma unroll
        for (int ct = 0; ct < NT; ++ct)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float val = accd[et][ct][j] * inv_beta;
            sS[(16 * et + 4 * g + j) * D + 16 * ct + i] = val;
            mxd = fmaxf(mxd, fabsf(val));
          }
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        float z = dzp[t] + shfl_xor_f(dzp[t], 16);
        z += shfl_xor_f(z, 32);
        if (g == 0) sZ[16 * t + i] = z * inv_beta;
      }
      wave_lds_sync();
      mxd = wave_max(mxd);
      const float rho = Ty<T>::kNarrow ? pow2_scale_to_one(mxd) : 1.f;
      const float inv_rho = 1.f / rho;
      float AdK[NT][KS], AdV[NT][KS], dzr[KS];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < KS; ++r) {
          AdK[t][r] = rho * sS[Geo<D>::out_index(t, i) * D + KS * g + r];
          AdV[t][r] = rho * sS[(KS * g + r) * D + Geo<D>::out_index(t, i)];
        }
#pragma unroll
      for (int r = 0; r < KS; ++r) dzr[r] = sZ[KS * g + r];

      // ---- pass 3: dk = (v dS^T + dz) * phi'(k), dv = phi(k) dS
      for (int32_t r0 = ws; r0 < we; r0 += 16) {
        bool ok = r0 + i < we;
        const int32_t orow = src.orig(r0 + i, ok);
        float kx[KS], vx[KS], fk[KS];
        load_row<T, D>(k, orow, ok, rowstride, col, kx);
        load_row<T, D>(v, orow, ok, rowstride, col, vx);
#pragma unroll
        for (int r = 0; r < KS; ++r) fk[r] = ok ? Ty<T>::round(phi_f<T>(kx[r])) : 0.f;
        float dkx[KS], dvx[KS];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const floatx4 a4 = Mma<T, KS>::run(AdK[t], vx, zero);
          const floatx4 b4 = Mma<T, KS>::run(AdV[t], fk, zero);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int r = 4 * t + j;
            dkx[r] = (a4[j] * inv_rho + dzr[r]) * dphi_f<T>(kx[r]);
            dvx[r] = b4[j] * inv_rho;
          }
        }
        if (ok) {
          store_frag<T, KS>(dk + (size_t)orow * rowstride + col, dkx);
          store_frag<T, KS>(dv + (size_t)orow * rowstride + col, dvx);
        }
      }
      wave_lds_sync();
    }
  }
}

// ------------------------------------------------------------ host launchers
struct AttnArgs {
  const PlanHeader* hdr;
  const int32_t* perm;
  const int32_t* offs;
  const Chunk* chunks;
  int32_t max_chunks, n, W, H;
};

static inline int grid_x(int32_t max_chunks) {
  return max_chunks < 1 ? 1 : (max_chunks > 65535 ? 65535 : max_chunks);
}

template <typename T, int D>
static hipError_t fwd_impl(const AttnArgs& a, const void* q, const void* k, const void* v, void* o,
                           hipStream_t stream) {
  const int hpw = a.H < 8 ? a.H : 8;
  dim3 grid(grid_x(a.max_chunks), (a.H + hpw - 1) / hpw);
  const size_t lds = (size_t)hpw * Geo<D>::kScratch * sizeof(float);
  hipLaunchKernelGGL((k_sla_fwd<T, D>), grid, dim3(64 * hpw), lds, stream, a.hdr, a.perm, a.offs,
                     a.chunks, a.max_chunks, a.n, a.W, a.H, hpw, static_cast<const T*>(q),
                     static_cast<const T*>(k), static_cast<const T*>(v), static_cast<T*>(o));
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t bwd_impl(const AttnArgs& a, const void* q, const void* k, const void* v,
                           const void* dout, void* dq, void* dk, void* dv, hipStream_t stream) {
  const int hpw = a.H < 4 ? a.H : 4;
  dim3 grid(grid_x(a.max_chunks), (a.H + hpw - 1) / hpw);
  const size_t lds = (size_t)hpw * Geo<D>::kScratch * sizeof(float);
  hipLaunchKernelGGL((k_sla_bwd<T, D>), grid, dim3(64 * hpw), lds, stream, a.hdr, a.perm, a.offs,
                     a.chunks, a.max_chunks, a.n, a.W, a.H, hpw, static_cast<const T*>(q),
                     static_cast<const T*>(k), static_cast<const T*>(v),
                     static_cast<const T*>(dout), static_cast<T*>(dq), static_cast<T*>(dk),
                     static_cast<T*>(dv));
  return hipGetLastError();
}

static AttnArgs attn_args(const void* plan, int32_t n, int32_t W, int32_t H) {
  const PlanLayout lay = plan_layout(n, W);
  const char* base = static_cast<const char*>(plan);
  AttnArgs a;
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

// dtype: 0 f32, 1 f16, 2 bf16
hipError_t launch_forward(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                          const void* q, const void* k, const void* v, void* o,
                          hipStream_t stream) {
  const AttnArgs a = attn_args(plan, n, W, H);
  if (d == 32) {
    if (dtype == 0) return fwd_impl<float, 32>(a, q, k, v, o, stream);
    if (dtype == 1) return fwd_impl<_Float16, 32>(a, q, k, v, o, stream);
    return fwd_impl<bf16_t, 32>(a, q, k, v, o, stream);
  }
  if (dtype == 0) return fwd_impl<float, 16>(a, q, k, v, o, stream);
  if (dtype == 1) return fwd_impl<_Float16, 16>(a, q, k, v, o, stream);
  return fwd_impl<bf16_t, 16>(a, q, k, v, o, stream);
}

hipError_t launch_backward(const void* plan, int32_t n, int32_t W, int dtype, int32_t H,
                           int32_t d, const void* q, const void* k, const void* v,
                           const void* dout, void* dq, void* dk, void* dv, hipStream_t stream) {
  const AttnArgs a = attn_args(plan, n, W, H);
  if (d == 32) {
    if (dtype == 0) return bwd_impl<float, 32>(a, q, k, v, dout, dq, dk, dv, stream);
    if (dtype == 1) return bwd_impl<_Float16, 32>(a, q, k, v, dout, dq, dk, dv, stream);
    return bwd_impl<bf16_t, 32>(a, q, k, v, dout, dq, dk, dv, stream);
  }
  if (dtype == 0) return bwd_impl<float, 16>(a, q, k, v, dout, dq, dk, dv, stream);
  if (dtype == 1) return bwd_impl<_Float16, 16>(a, q, k, v, dout, dq, dk, dv, stream);
  return bwd_impl<bf16_t, 16>(a, q, k, v, dout, dq, dk, dv, stream);
}

}  // namespace sla

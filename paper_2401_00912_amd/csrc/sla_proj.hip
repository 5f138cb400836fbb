// The projection layer fused into the SLA forward, and the output projection
// (see the section comment below).
#include "sla_attn_core.h"

namespace sla {

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
constexpr int kProjMaxC = 256;
// Above this many 32-channel blocks (C > 128) a block's features are fetched and
// projected one 32-row job at a time, so that at most one job's features are
// live (64 VGPRs for C = 256, as both jobs' for C = 128).
constexpr int kProjBlockFetchMaxCB = 4;

struct ProjArgs {
  const void* x;  // [n, C] features
  const void* w;  // [3C, C]: the rows of W_q, W_k, W_v
  const void* b;  // [3C] or null
  void* qkv;      // [3][n][C]: q, k, v as projected, when they are saved
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

// The matrices selected by `which` (bit 0: K, 1: V, 2: Q) of one job, as
// projected, to the saved q, k, v ([3][n][C], q first) at their rows' head
// columns; lanes past the job's rows store nothing.
template <typename T, int D>
__device__ __forceinline__ void save_job(const Slice<T, Geo<D>::KS, 3>& sj, unsigned which, T* qkv,
                                         size_t nC, size_t rs, int col, int g) {
#pragma unroll
  for (int m = 0; m < 3; ++m) {
    if (!(which & (1u << m))) continue;
    T* base = qkv + (m == 2 ? 0 : (m == 0 ? nC : 2 * nC));
#pragma unroll
    for (int s = 0; s < 2; ++s) RowIO<T, D>::put(base, row_off(sj.o[s], rs, col), g, sj.x[m][s], sj.ok[s]);
  }
}

// One job's features (rows from the block's permutation entries).
template <typename T, int CB>
__device__ __forceinline__ void xjob_fetch(Raw<T, 8> (&xj)[2][CB], int32_t (&o)[2], bool (&ok)[2],
                                           const BlockRows& br, int jj, int32_t base, int32_t end,
                                           int32_t n, const T* x, int g) {
  constexpr int C = 32 * CB;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    ok[s] = (uint32_t)br.o[jj][s] < (uint32_t)n;
    o[s] = ok[s] ? br.o[jj][s] : 0;
    const bool live = base + kSliceRows * jj + 16 * s < end;
    const T* row = row_at(x, o[s], (size_t)C, 8 * g);
#pragma unroll
    for (int kb = 0; kb < CB; ++kb) {
      if (live) xj[s][kb] = __builtin_bit_cast(Raw<T, 8>, *reinterpret_cast<const uint4*>(row + 32 * kb));
      else xj[s][kb] = Frag<T, 8>::zero();
    }
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

// SAVE: q, k, v also go to pa.qkv as they are projected (for a backward that
// does not recompute them).
template <typename T, int D, int PHI, int CB, bool SAVE>
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
  T* const qkv = static_cast<T*>(pa.qkv);
  const size_t nC = (size_t)n * rs;

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
    constexpr bool kByJob = CB > kProjBlockFetchMaxCB;
    XBlock<T, kByJob ? 1 : CB> xb;
    if constexpr (!kByJob) {
      if (ww.kind != 0 && resident) xblock_fetch<T, CB>(xb, cur.br, ww.ra, ww.rb, n, x, g);
    }
    // the next item: its rows and windows are requested now, its successor's entry too
    Pending nxt;
    pending_request(nxt, a, nsl, ne, wv, perm, lane);
    nsl = proj_slot(it, item + 2 * G, wv);
    ne = slot_entry(a, nsl);
    WinIter wi;
    if (resident) {
      Block<T, D, 3> bk;
      if constexpr (kByJob) {
        if (ww.kind != 0) {
#pragma unroll
          for (int jj = 0; jj < kBlockJobs; ++jj) {
            Raw<T, 8> xj[2][CB];
            xjob_fetch<T, CB>(xj, bk.j[jj].o, bk.j[jj].ok, cur.br, jj, ww.ra, ww.rb, n, x, g);
            project_job<T, D, CB>(bk.j[jj], xj, kAll, s_w, s_b, i, g);
            if constexpr (SAVE) save_job<T, D>(bk.j[jj], kAll, qkv, nC, rs, col, g);
            __builtin_amdgcn_sched_barrier(0);
          }
        }
      } else {
        if (ww.kind != 0) {
          project<T, D, CB>(bk, xb, kAll, s_w, s_b, i, g);
          if constexpr (SAVE) {
#pragma unroll
            for (int jj = 0; jj < kBlockJobs; ++jj) save_job<T, D>(bk.j[jj], kAll, qkv, nC, rs, col, g);
          }
        }
      }
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
          if constexpr (SAVE) save_job<T, D>(sj, kKV, qkv, nC, rs, col, g);
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
          if constexpr (SAVE) save_job<T, D>(sj, kQ, qkv, nC, rs, col, g);
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
// C = 256: W_o takes 135 KB of LDS, one workgroup per CU, so that workgroup
// has 16 waves (128 VGPRs per lane: the tiles below fit with the scheduling
// fences between them).
template <int CB>
constexpr int kOutWaves = CB > 4 ? 16 : kWaves;

template <typename T, int CB>
__global__ __launch_bounds__(64 * kOutWaves<CB>) void k_out_proj(KernelArgs a, const T* __restrict__ o,
                                                                 const T* __restrict__ w,
                                                                 const T* __restrict__ b,
                                                                 T* __restrict__ y) {
  constexpr int C = 32 * CB, LDW = C + 8, NW = kOutWaves<CB>;
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
  for (int32_t tile = (int32_t)blockIdx.x * NW + wv; tile * 16 < nrows;
       tile += (int32_t)gridDim.x * NW) {
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
        // C = 256: keep later tiles' weight reads from being hoisted here (all of
        // them at once would not fit in the registers)
        if constexpr (CB > 4) __builtin_amdgcn_sched_barrier(0);
      }
      RowIO<T, 32>::put(y, row_off(ok ? row : 0, (size_t)C, 32 * hb), g, F8::from_f32(f), ok);
    }
  }
}

// ------------------------------------------------------------ host launchers
// Resident workgroups of a launch of `threads`-thread workgroups (workgroups per
// CU x CUs; queried per call, for the launches that are not 256 threads wide).
inline int64_t resident_for(const void* kernel, int threads) {
  int per_cu = 0, cus = 0, dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      per_cu < 1 || cus < 1) {
    per_cu = 1;
    cus = 256;
  }
  return (int64_t)per_cu * cus;
}

// Projected forward: the fused projection + SLA kernel, then the output
// projection.  Workgroups of the fused kernel: as grid_size, rounded up to a
// multiple of 8 H (every workgroup keeps one head), at most enough for every item
// the plan can hold.
template <typename T, int D, int PHI, int CB>
static hipError_t proj_impl(const void* plan, int32_t n, int32_t W, int32_t H, float eps,
                            const void* x, const void* wqkv, const void* bqkv, const void* wo,
                            const void* bo, void* o, void* y, void* qkv, hipStream_t stream) {
  const PlanLayout lay = plan_layout(n, W);
  const KernelArgs a = kernel_args(plan, lay, n, W, H, eps);
  void (*fk)(KernelArgs, ProjArgs, T*) =
      qkv ? &k_sla_fwd_proj<T, D, PHI, CB, true> : &k_sla_fwd_proj<T, D, PHI, CB, false>;
  const void* kern = reinterpret_cast<const void*>(fk);
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
  const ProjArgs pa{x, wqkv, bqkv, qkv};
  hipLaunchKernelGGL(fk, dim3((unsigned)g), dim3(64 * kWaves), 0, stream, a, pa, static_cast<T*>(o));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const void* kout = reinterpret_cast<const void*>(&k_out_proj<T, CB>);
  int64_t go = kOutWaves<CB> == kWaves ? resident_workgroups(kout) : resident_for(kout, 64 * kOutWaves<CB>);
  const int64_t passes = ((int64_t)n + 16 * kOutWaves<CB> - 1) / (16 * kOutWaves<CB>);
  if (go > passes) go = passes;
  if (go < 1) go = 1;
  hipLaunchKernelGGL((k_out_proj<T, CB>), dim3((unsigned)go), dim3(64 * kOutWaves<CB>), 0, stream, a,
                     static_cast<const T*>(o), static_cast<const T*>(wo), static_cast<const T*>(bo),
                     static_cast<T*>(y));
  return hipGetLastError();
}

template <typename T, int PHI>
static hipError_t projected_t(const void* plan, int32_t n, int32_t W, int32_t H, int32_t d,
                              float eps, const void* x, const void* wqkv, const void* bqkv,
                              const void* wo, const void* bo, void* o, void* y, void* qkv,
                              hipStream_t stream) {
  const int C = H * d;
  if (d == 32) {
    if (C == 256) return proj_impl<T, 32, PHI, 8>(plan, n, W, H, eps, x, wqkv, bqkv, wo, bo, o, y, qkv, stream);
    if (C == 128) return proj_impl<T, 32, PHI, 4>(plan, n, W, H, eps, x, wqkv, bqkv, wo, bo, o, y, qkv, stream);
    return proj_impl<T, 32, PHI, 2>(plan, n, W, H, eps, x, wqkv, bqkv, wo, bo, o, y, qkv, stream);
  }
  if (C == 256) return proj_impl<T, 16, PHI, 8>(plan, n, W, H, eps, x, wqkv, bqkv, wo, bo, o, y, qkv, stream);
  if (C == 128) return proj_impl<T, 16, PHI, 4>(plan, n, W, H, eps, x, wqkv, bqkv, wo, bo, o, y, qkv, stream);
  return proj_impl<T, 16, PHI, 2>(plan, n, W, H, eps, x, wqkv, bqkv, wo, bo, o, y, qkv, stream);
}

// dtype: 1 f16, 2 bf16; C = H d in {64, 128, 256}; phi: 0 elu + 1, 1 ReLU
hipError_t launch_forward_projected(const void* plan, int32_t n, int32_t W, int dtype, int32_t H,
                                    int32_t d, int phi, float eps, const void* x, const void* wqkv,
                                    const void* bqkv, const void* wo, const void* bo, void* o,
                                    void* y, void* qkv, hipStream_t stream) {
  if (dtype == 1) {
    if (phi == kPhiRelu)
      return projected_t<_Float16, kPhiRelu>(plan, n, W, H, d, eps, x, wqkv, bqkv, wo, bo, o, y, qkv, stream);
    return projected_t<_Float16, kPhiElu1>(plan, n, W, H, d, eps, x, wqkv, bqkv, wo, bo, o, y, qkv, stream);
  }
  if (phi == kPhiRelu)
    return projected_t<bf16_t, kPhiRelu>(plan, n, W, H, d, eps, x, wqkv, bqkv, wo, bo, o, y, qkv, stream);
  return projected_t<bf16_t, kPhiElu1>(plan, n, W, H, d, eps, x, wqkv, bqkv, wo, bo, o, y, qkv, stream);
}

}  // namespace sla

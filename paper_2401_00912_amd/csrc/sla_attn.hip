// SLA forward and backward on the gfx950 matrix cores.
//
// Work decomposition.  A persistent grid (about one workgroup per resident
// slot, a multiple of 8) of four-wave workgroups walks a list of work items (see
// item_slot in the core header): first one item per long window and head, whose
// rows the four waves (or two, for windows of medium length) split between them
// and whose partial states they add in LDS, then one item per chunk and group of
// up to four heads, one wave per head.  A chunk is a run of whole short windows
// of the window-sorted sequence (see the builder); its rows are read through the
// plan's permutation, so q, k, v stay in the caller's order.
//
// A wave holds its item's rows (up to kMaxChunkRows of q, k, v, and dout in the
// backward) in registers for the whole item and walks its windows from there; a
// share of a very long window that exceeds that is streamed through in blocks.
// Items are software-pipelined per wave through an LDS ring: while item k
// computes, the permutation slice and window offsets of item k + 1 and the plan
// entry of item k + 2 are already in flight.
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
#include "sla_attn_core.h"

namespace sla {

// ------------------------------------------------------------------ forward
template <typename T, int D, int PHI>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kWpe<T, SLA_FWD_WPE>)))
void k_sla_fwd(KernelArgs a, const T* __restrict__ q, const T* __restrict__ k,
               const T* __restrict__ v, T* __restrict__ o) {
  constexpr int KT = kStateTiles<D>;
  __shared__ floatx4 s_part[kWaves * KT * 64];  // partial states of a long window
  __shared__ WaveMeta s_meta[kWaves];            // the items ahead (perm slices, offsets, entries)
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

  WaveMeta& meta = s_meta[wv];
  const bool csr = perm == nullptr;
  int32_t item = blockIdx.x;
  WaveWork wc, wn;
  {
    const Slot s0 = item_slot(it, item, wv), s1 = item_slot(it, item + G, wv);
    wc = decode_work(a, s0, slot_entry(a, s0), wv);
    wn = decode_work(a, s1, slot_entry(a, s1), wv);
  }
  request_perm(wc, perm, meta.perm[0], lane);
  request_perm(wn, perm, meta.perm[1], lane);
  request_offs(wc, a, meta.offs[0], lane);
  request_entry(a, item_slot(it, item + 2 * G, wv), &meta.ent[0], lane);
  int par = 0;   // ring slot of the current item
  while (item < it.total) {
    const WaveWork ww = wc;
    const int col = ww.h * D;
    // a range of more than kBlockRows rows (a quarter of a very long window) is
    // streamed through the block: K, V for the state, then Q for the outputs
    const bool resident = ww.rb - ww.ra <= kBlockRows;
    const unsigned first = resident ? kAll : kKV;
    // the item's rows and windows, and the entry of the item after next, from LDS
    wait_vm();
    BlockRows br;
    block_rows_lds(br, ww, meta.perm[par], csr, lane);
    Stream str;
    stream_lds(str, ww, a, meta.offs[par], lane);
    const WaveWork wnn = decode_work(a, item_slot(it, item + 2 * G, wv), lds_entry(&meta.ent[par]), wv);
    wait_lgkm();
    // requests ahead: the slice of the item after next, the next item's windows,
    // the entry after that; then this item's rows (whose wait covers these)
    request_perm(wnn, perm, meta.perm[par], lane);
    request_offs(wn, a, meta.offs[par ^ 1], lane);
    request_entry(a, item_slot(it, item + 3 * G, wv), &meta.ent[par ^ 1], lane);
    Block<T, D, 3> bk;
    if (ww.kind != 0) block_fetch<T, D, 3>(bk, br, ww.ra, ww.rb, n, mats, first, rs, col, g);

    block_arrange<T, D, 3>(bk, first);
    WinIter wi;
    for (bool more = wi.first(ww, str); more; more = wi.next(ww, str)) {
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
    wc = wn;
    wn = wnn;
    par ^= 1;
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
  __shared__ WaveMeta s_meta[kWaves];              // the items ahead (perm slices, offsets, entries)
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

  WaveMeta& meta = s_meta[wv];
  const bool csr = perm == nullptr;
  int32_t item = blockIdx.x;
  WaveWork wc, wn;
  {
    const Slot s0 = item_slot(it, item, wv), s1 = item_slot(it, item + G, wv);
    wc = decode_work(a, s0, slot_entry(a, s0), wv);
    wn = decode_work(a, s1, slot_entry(a, s1), wv);
  }
  request_perm(wc, perm, meta.perm[0], lane);
  request_perm(wn, perm, meta.perm[1], lane);
  request_offs(wc, a, meta.offs[0], lane);
  request_entry(a, item_slot(it, item + 2 * G, wv), &meta.ent[0], lane);
  int par = 0;   // ring slot of the current item
  while (item < it.total) {
    const WaveWork ww = wc;
    const int col = ww.h * D;
    const bool resident = ww.rb - ww.ra <= kBlockRows;
    const unsigned first = resident ? kAll : kKV;
    // the item's rows and windows, and the entry of the item after next, from LDS
    wait_vm();
    BlockRows br;
    block_rows_lds(br, ww, meta.perm[par], csr, lane);
    Stream str;
    stream_lds(str, ww, a, meta.offs[par], lane);
    const WaveWork wnn = decode_work(a, item_slot(it, item + 2 * G, wv), lds_entry(&meta.ent[par]), wv);
    wait_lgkm();
    // requests ahead (see the forward); then this item's rows
    request_perm(wnn, perm, meta.perm[par], lane);
    request_offs(wn, a, meta.offs[par ^ 1], lane);
    request_entry(a, item_slot(it, item + 3 * G, wv), &meta.ent[par ^ 1], lane);
    Block<T, D, 4> bk;
    if (ww.kind != 0) block_fetch<T, D, 4>(bk, br, ww.ra, ww.rb, n, mats, first, rs, col, g);

    block_arrange<T, D, 4>(bk, first);
    WinIter wi;
    for (bool more = wi.first(ww, str); more; more = wi.next(ww, str)) {
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
    wc = wn;
    wn = wnn;
    par ^= 1;
  }
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

}  // namespace sla

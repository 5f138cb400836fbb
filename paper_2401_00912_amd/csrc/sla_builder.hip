// Segment builder: stable counting sort of rows by window id, CSR window offsets
// and the chunk table (Sec. 3.2 / Fig. 3(a): voxels ordered by window into one
// flattened matrix that is partitioned into chunks; the offset generation timed
// in Fig. 5 computes the start of every chunk).
//
// Mode A (ids given), two launches over builder blocks of E rows:
//   k_count    per block, a histogram of its rows' window ids (LDS atomics; the
//              counts are order-free, hence deterministic) -> count matrix;
//   k_scatter  per block: the column prefix of the count matrix over the blocks
//              before it and the column totals (read straight from the matrix),
//              the exclusive scan of the totals (= offsets) in LDS, then the
//              stable rank of every row among the rows of its window in this
//              block (wave ballots on the id bits give the lanes sharing an id;
//              waves take their bases in order) and perm[offsets[id] + block
//              prefix + rank] = row.  One more workgroup (the last) computes the
//              same totals and publishes the offsets, the chunk table and the
//              header.
// Mode B (CSR offsets given) and n = 0: one workgroup, k_plan, validates the
// offsets and writes the chunk table and header.
#include <atomic>

#include "sla_common.h"

namespace sla {

#ifndef SLA_BUILD_THREADS
#define SLA_BUILD_THREADS 1024
#endif
constexpr int kBuildThreads = SLA_BUILD_THREADS;  // threads of every builder workgroup

// Workgroup barrier for LDS traffic only: this wave's LDS operations complete,
// then every wave arrives.  Threads of a builder workgroup exchange data through
// LDS alone, so global loads in flight (the next phase's inputs) stay in flight.
__device__ __forceinline__ void lds_sync() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// ------------------------------------------------------------------ k_count
__global__ __launch_bounds__(kBuildThreads) void k_count(const int32_t* __restrict__ ids, int32_t n,
                                                         int32_t W, int32_t E, int32_t ld,
                                                         int32_t* __restrict__ counts) {
  __shared__ int32_t hist[kMaxWindows + 1];
  for (int i = threadIdx.x; i <= W; i += blockDim.x) hist[i] = 0;
  lds_sync();
  const int64_t base = (int64_t)blockIdx.x * E;
  const int64_t end = base + E < n ? base + E : n;
  for (int64_t i = base + threadIdx.x; i < end; i += blockDim.x) {
    const int32_t id = ids[i];
    atomicAdd(&hist[(uint32_t)id < (uint32_t)W ? id : W], 1);
  }
  lds_sync();
  int32_t* row = counts + (size_t)blockIdx.x * ld;
  for (int i = threadIdx.x; i < ld; i += blockDim.x) row[i] = i <= W ? hist[i] : 0;
}

// -------------------------------------------------------- block-wide scans
struct OpSum {
  __device__ int32_t operator()(int32_t a, int32_t b) const { return a + b; }
};
struct OpSum64 {
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const { return a + b; }
};
struct OpMax {
  __device__ int32_t operator()(int32_t a, int32_t b) const { return a > b ? a : b; }
};
// Max of each 32-bit half of a packed pair.
struct OpMax2 {
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const {
    const uint32_t hi = max((uint32_t)(a >> 32), (uint32_t)(b >> 32));
    const uint32_t lo = max((uint32_t)a, (uint32_t)b);
    return ((uint64_t)hi << 32) | lo;
  }
};


// One step of a wave scan: v op (v moved by the DPP control CTRL into the rows
// of ROWS); lanes the move does not reach take the identity.
template <int CTRL, int ROWS, class Op, typename V>
__device__ __forceinline__ V dpp_scan_step(V v, V identity, Op op) {
  if constexpr (sizeof(V) == 4) {
    return op(v, (V)__builtin_amdgcn_update_dpp((int)identity, (int)v, CTRL, ROWS, 0xf, false));
  } else {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)identity, (int)(uint32_t)v,
                                                              CTRL, ROWS, 0xf, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)(identity >> 32),
                                                              (int)(uint32_t)(v >> 32), CTRL, ROWS, 0xf,
                                                              false);
    return op(v, ((V)hi << 32) | lo);
  }
}

// Inclusive scan over the 64 lanes in lane order: shifts by 1, 2, 4 and 8
// lanes inside each row of 16, then lane 15 of rows 0 and 2 into rows 1 and 3,
// then lane 31 into rows 2 and 3 (DPP moves, no LDS round trips).
template <class Op, typename V>
__device__ __forceinline__ V wave_inclusive_scan(V v, V identity, Op op) {
  v = dpp_scan_step<0x111, 0xf>(v, identity, op);  // row_shr:1
  v = dpp_scan_step<0x112, 0xf>(v, identity, op);  // row_shr:2
  v = dpp_scan_step<0x114, 0xf>(v, identity, op);  // row_shr:4
  v = dpp_scan_step<0x118, 0xf>(v, identity, op);  // row_shr:8
  v = dpp_scan_step<0x142, 0xa>(v, identity, op);  // row_bcast:15
  v = dpp_scan_step<0x143, 0xc>(v, identity, op);  // row_bcast:31
  return v;
}

template <typename V>
__device__ __forceinline__ V read_lane(V v, int lane) {
  if constexpr (sizeof(V) == 4) {
    return (V)__builtin_amdgcn_readlane((int)v, lane);
  } else {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
    return ((V)hi << 32) | lo;
  }
}

// Exclusive scan of one value per thread in thread order; *total gets the
// reduction of all values.  Each wave scans its lanes, publishes its total in
// s[0..15], and after one barrier every wave scans the wave totals itself.
// Ends with a barrier so s can be reused.
template <class Op, typename V = int32_t>
__device__ V block_exscan(V x, V identity, Op op, V* s, V* total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nwv = blockDim.x >> 6;
  const V inc = wave_inclusive_scan(x, identity, op);
  if (lane == 63) s[wv] = inc;
  lds_sync();
  const V tinc = wave_inclusive_scan(lane < nwv ? s[lane] : identity, identity, op);
  const V before = wv > 0 ? read_lane(tinc, wv - 1) : identity;
  *total = read_lane(tinc, nwv - 1);
  V ex = __shfl_up(inc, 1, 64);
  if (lane == 0) ex = identity;
  const V r = op(before, ex);
  lds_sync();
  return r;
}

// ------------------------------------------------------ chunk / long tables
// Work tables from the offsets in LDS, in sequence order (pages of P = L/2 rows):
// a window of more than L rows is "long" and goes to the long-window table
// (four-way ones, of more than 2L rows, first, then two-way ones); a window of
// P+1..L rows is a chunk of its own; a window of 1..P rows opens a chunk unless
// the previous non-empty window is short and starts in the same page.  A chunk
// runs to the next event (chunk start or long window).  s_aux: LDS scratch of at
// least W ints.  Every thread of the block calls it; returns the number of
// chunks and sets *n_long and *n_long4.
__device__ int32_t build_tables(const int32_t* s_off, int32_t* s_aux, int32_t W, int32_t L,
                                Chunk* __restrict__ chunks, LongWin* __restrict__ longs,
                                int32_t* s_scan, uint64_t* s_scan2, int32_t* n_long,
                                int32_t* n_long4) {
  const int tid = threadIdx.x, T = blockDim.x;
  const int32_t page = L >> 1;
  const int P = (W + T - 1) / T;
  const int w0 = min(tid * P, W), w1 = min(w0 + P, W);
  // the start of the last non-empty window and the end of the last window of
  // more than P rows before my range decide the kind of my first window
  int32_t aggStart = -1, aggWide = -1;
  for (int w = w0; w < w1; ++w) {
    const int32_t len = s_off[w + 1] - s_off[w];
    if (len > 0) aggStart = s_off[w];
    if (len > page) aggWide = s_off[w + 1];
  }
  // both maxima in one scan of (value + 1) pairs
  uint64_t tmp;
  const uint64_t both = block_exscan<OpMax2, uint64_t>(
      ((uint64_t)(uint32_t)(aggStart + 1) << 32) | (uint32_t)(aggWide + 1), 0ull, OpMax2(), s_scan2,
      &tmp);
  const int32_t lastStart = (int32_t)(both >> 32) - 1;
  const int32_t lastWideEnd = (int32_t)(uint32_t)both - 1;
  // 0: no event, 1: opens a chunk, 2: two-way long window, 3: four-way long
  // window.  ls / ll: start of the previous non-empty window / end of the
  // previous window of more than P rows (ll == a exactly when the previous
  // non-empty window is not short).
  auto kind = [&](int32_t& ls, int32_t& ll, int w) -> int {
    const int32_t a = s_off[w], len = s_off[w + 1] - a;
    if (len <= 0) return 0;
    int k = 0;
    if (len > L) k = len > 2 * L ? 3 : 2;
    else if (len > page || ls < 0 || ll == a || (ls / page) != (a / page)) k = 1;
    ls = a;
    if (len > page) ll = a + len;
    return k;
  };
  uint64_t cnt = 0;   // chunks, two-way, four-way: 21 bits each (W <= 16384)
  {
    int32_t ls = lastStart, ll = lastWideEnd;
    for (int w = w0; w < w1; ++w) {
      const int k = kind(ls, ll, w);
      if (k) cnt += 1ull << (21 * (k - 1));
    }
  }
  uint64_t tot = 0;
  const uint64_t ex = block_exscan<OpSum64, uint64_t>(cnt, 0ull, OpSum64(), s_scan2, &tot);
  constexpr uint64_t kMask = (1ull << 21) - 1;
  const int32_t s0 = (int32_t)(ex & kMask), t0 = (int32_t)((ex >> 21) & kMask),
                f0 = (int32_t)(ex >> 42);
  const int32_t nC = (int32_t)(tot & kMask), n2 = (int32_t)((tot >> 21) & kMask),
                n4 = (int32_t)(tot >> 42);
  {
    // the event list in sequence order: s_aux[event index] = window
    int32_t ls = lastStart, ll = lastWideEnd, e = s0 + t0 + f0;
    for (int w = w0; w < w1; ++w)
      if (kind(ls, ll, w)) s_aux[e++] = w;
  }
  lds_sync();
  {
    int32_t ls = lastStart, ll = lastWideEnd, sc = s0, s2 = t0, s4 = f0;
    const int32_t nE = nC + n2 + n4;
    for (int w = w0; w < w1; ++w) {
      const int k = kind(ls, ll, w);
      if (k == 1) {
        const int32_t e = sc + s2 + s4;
        Chunk ch;
        ch.win_begin = w;
        ch.win_end = e + 1 < nE ? s_aux[e + 1] : W;
        ch.row_begin = s_off[w];
        ch.row_end = s_off[ch.win_end];
        chunks[sc++] = ch;
      } else if (k >= 2) {
        LongWin lw;
        lw.window = w;
        lw.row_begin = s_off[w];
        lw.row_end = s_off[w + 1];
        lw.pad = 0;
        longs[k == 3 ? s4++ : n4 + s2++] = lw;
      }
    }
  }
  *n_long = n2 + n4;
  *n_long4 = n4;
  return nC;
}

__device__ void write_header(PlanHeader* hdr, int32_t n, int32_t W, int32_t L, int32_t n_chunks,
                             int32_t n_long, int32_t n_long4, int32_t csr, int32_t invalid,
                             int32_t* invalid_out) {
  hdr->magic = kPlanMagic;
  hdr->n = n;
  hdr->num_windows = W;
  hdr->chunk_rows = L;
  hdr->n_chunks = n_chunks;
  hdr->n_long = n_long;
  hdr->n_long4 = n_long4;
  hdr->csr = csr;
  hdr->invalid = invalid;
  if (invalid_out) *invalid_out = invalid;
}

// ------------------------------------------------------------------ k_plan
// One workgroup.  csr == 1: offsets_io is the caller's CSR input; it is validated
// and clamped.  csr == 0 (n = 0 in mode A): every window is empty.
__global__ __launch_bounds__(kBuildThreads) void k_plan(int32_t csr, int32_t W, int32_t n,
                                                        int32_t L, int32_t* __restrict__ offsets_io,
                                                        int32_t* __restrict__ invalid_out,
                                                        PlanHeader* __restrict__ hdr,
                                                        int32_t* __restrict__ plan_offsets,
                                                        Chunk* __restrict__ chunks,
                                                        LongWin* __restrict__ longs) {
  __shared__ int32_t s_off[kMaxWindows + 1];
  __shared__ int32_t s_aux[kMaxWindows + 1];
  __shared__ int32_t s_scan[33];
  __shared__ uint64_t s_scan2[33];
  const int tid = threadIdx.x, T = blockDim.x;
  int32_t invalid = 0, total = 0;
  if (csr) {
    // s_off = running max of clamp(x, 0, n)
    const int P = (W + 1 + T - 1) / T;
    const int w0 = min(tid * P, W + 1), w1 = min(w0 + P, W + 1);
    int32_t bad = 0, mx = 0;
    for (int w = w0; w < w1; ++w) {
      const int32_t x = offsets_io[w];
      bad += (x < 0 || x > n);
      if (w > 0) bad += x < offsets_io[w - 1];
      const int32_t cx = x < 0 ? 0 : (x > n ? n : x);
      mx = cx > mx ? cx : mx;
    }
    const int32_t ex_max = block_exscan(mx, 0, OpMax(), s_scan, &total);
    int32_t bad_total = 0;
    block_exscan(bad, 0, OpSum(), s_scan, &bad_total);
    int32_t run = ex_max;
    for (int w = w0; w < w1; ++w) {
      const int32_t x = offsets_io[w];
      const int32_t cx = x < 0 ? 0 : (x > n ? n : x);
      run = cx > run ? cx : run;
      s_off[w] = run;
    }
    invalid = bad_total;
    if (tid == 0) invalid += (offsets_io[0] != 0) + (offsets_io[W] != n);
  } else {
    for (int w = tid; w <= W; w += T) s_off[w] = 0;
  }
  lds_sync();
  for (int w = tid; w <= W; w += T) {
    plan_offsets[w] = s_off[w];
    if (!csr && offsets_io) offsets_io[w] = s_off[w];
  }
  int32_t n_long = 0, n_long4 = 0;
  const int32_t n_chunks =
      build_tables(s_off, s_aux, W, L, chunks, longs, s_scan, s_scan2, &n_long, &n_long4);
  if (tid == 0) write_header(hdr, n, W, L, n_chunks, n_long, n_long4, csr, invalid, invalid_out);
}

// --------------------------------------------------------------- k_scatter
// Lanes whose (valid) key equals this lane's key; 0 for invalid lanes.  One
// ballot per key bit: a lane matches iff it agrees with this lane on every bit.
__device__ __forceinline__ uint64_t match_key(int32_t key, bool valid, int nbits) {
  uint64_t m = __ballot(valid);
  for (int b = 0; b < nbits; ++b) {
    const bool bit = (key >> b) & 1;
    const uint64_t bal = __ballot(valid && bit);
    m &= bit ? bal : ~bal;
  }
  return valid ? m : 0ull;
}

__device__ __forceinline__ uint64_t lanemask_lt(int lane) {
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Dynamic LDS: base[W + 1], tot[W + 1], hist[max(nws W, W + 1)] (overlap) or
// base[W + 1], hist[max(nws W, W + 1)] with tot = hist (no overlap, large W);
// nws = waves that rank rows.  Blocks 0..nb-1 rank and scatter the rows of
// builder block blockIdx.x; block nb publishes the offsets and builds the chunk
// and long-window tables and the header, in parallel with the others.
//
// A ranking block requests its rows' window ids and its share of the count
// matrix first; with `overlap` it counts its rows per wave (which needs only the
// ids) while the matrix is in flight; then the column prefix and totals, the
// offsets, the per-wave prefix and the scatter.
constexpr int kMatBatch = 16;   // count-matrix rows a thread has in flight at once

__global__ __launch_bounds__(kBuildThreads) void k_scatter(
    const int32_t* __restrict__ ids, int32_t n, int32_t W, int32_t L, int32_t E, int32_t nb,
    int32_t ld, int32_t nws, int32_t overlap, const int32_t* __restrict__ counts,
    int32_t* __restrict__ perm, int32_t* __restrict__ perm_out, int32_t* __restrict__ plan_offsets,
    int32_t* __restrict__ offsets_out, Chunk* __restrict__ chunks, LongWin* __restrict__ longs,
    PlanHeader* __restrict__ hdr, int32_t* __restrict__ invalid_out) {
  extern __shared__ int32_t lds[];
  __shared__ int32_t s_scan[33];
  __shared__ uint64_t s_scan2[33];
  int32_t* base = lds;                              // offsets[w] + rows of window w in earlier blocks
  int32_t* tot = lds + (W + 1);                     // column totals
  int32_t* hist = overlap ? tot + (W + 1) : tot;    // per-wave row counts (table block: scratch)
  const int tid = threadIdx.x, T = blockDim.x;
  const int lane = tid & 63, wv = tid >> 6;
  const int32_t blk = blockIdx.x;
  const bool tables = blk == nb;

  // this wave's rows [rbeg, rend): ids of the first two 64-row groups
  const int64_t span = E / nws;
  const int64_t rbeg = (int64_t)blk * E + wv * span;
  const int64_t rend = rbeg + span < n ? rbeg + span : n;
  const bool ranks = !tables && wv < nws;
  int32_t id0 = -1, id1 = -1;
  if (ranks) {
    if (rbeg + lane < rend) id0 = ids[rbeg + lane];
    if (rbeg + 64 + lane < rend) id1 = ids[rbeg + 64 + lane];
  }

  // count-matrix shares: unit (part, g) sums rows [part RP, part RP + RP) of
  // column group g (4 columns, one 16-B load per row); a thread takes units tid,
  // tid + T, ...; the first kMatBatch rows of its first unit are requested now
  const int G = ld >> 2;
  const int R = max(1, min(T / G, nb));
  const int RP = (nb + R - 1) / R;
  const int NU = R * G;
  int4 x[kMatBatch];
  {
    const int part = tid / G, cg = tid - part * G;
    const int b0 = part * RP, b1 = min(b0 + RP, nb);
#pragma unroll
    for (int u = 0; u < kMatBatch; ++u)
      x[u] = tid < NU && b0 + u < b1 ? reinterpret_cast<const int4*>(counts + (size_t)(b0 + u) * ld)[cg]
                                     : make_int4(0, 0, 0, 0);
  }

  for (int w = tid; w <= W; w += T) {
    base[w] = 0;
    tot[w] = 0;
  }
  if (!tables && overlap)   // every thread of the block: the loop is strided over all of them
    for (int i = tid; i < nws * W; i += T) hist[i] = 0;
  lds_sync();

  // (a) ranking blocks: per-wave window counts of the wave's rows
  const int nbits = W > 1 ? 32 - __clz(W - 1) : 0;
  int32_t* h = hist + wv * W;
  const uint64_t lt = lanemask_lt(lane);
  // returns the row's rank among this wave's rows of its window (-1: invalid id)
  auto count_group = [&](int32_t id) -> int32_t {
    const bool valid = (uint32_t)id < (uint32_t)W;
    const uint64_t m = match_key(id, valid, nbits);
    if (!valid) return -1;
    const int32_t hb = h[id];
    if ((m & lt) == 0) h[id] = hb + __popcll(m);
    return hb + __popcll(m & lt);
  };
  auto id_at = [&](int64_t r) -> int32_t { return r + lane < rend ? ids[r + lane] : -1; };
  int32_t rk0 = -1, rk1 = -1;   // ranks of the first two groups' rows
  auto count_rows = [&]() {
    if (ranks) {
      rk0 = count_group(id0);
      if (rbeg + 64 < rend) rk1 = count_group(id1);
      for (int64_t r = rbeg + 128; r < rend; r += 64) count_group(id_at(r));
    }
  };
  if (overlap) count_rows();

  // (b) column prefix over the earlier blocks and column totals
  for (int unit = tid; unit < NU; unit += T) {
    const int part = unit / G, cg = unit - part * G;
    const int b0 = part * RP, b1 = min(b0 + RP, nb);
    int4 pre = make_int4(0, 0, 0, 0), sum = make_int4(0, 0, 0, 0);
    for (int b = b0; b < b1; b += kMatBatch) {
      if (unit != tid || b != b0) {
#pragma unroll
        for (int u = 0; u < kMatBatch; ++u)
          x[u] = b + u < b1 ? reinterpret_cast<const int4*>(counts + (size_t)(b + u) * ld)[cg]
                            : make_int4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < kMatBatch; ++u) {
        sum.x += x[u].x; sum.y += x[u].y; sum.z += x[u].z; sum.w += x[u].w;
        if (b + u < blk) { pre.x += x[u].x; pre.y += x[u].y; pre.z += x[u].z; pre.w += x[u].w; }
      }
    }
    const int w = 4 * cg;
    const int32_t p4[4] = {pre.x, pre.y, pre.z, pre.w}, t4[4] = {sum.x, sum.y, sum.z, sum.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (w + k <= W) {
        if (R > 1) {
          atomicAdd(&base[w + k], p4[k]);
          atomicAdd(&tot[w + k], t4[k]);
        } else {
          base[w + k] = p4[k];
          tot[w + k] = t4[k];
        }
      }
    }
  }
  lds_sync();
  const int32_t invalid = tot[W];   // column W counts the out-of-range ids

  // (c) offsets = exclusive scan of the column totals; base += offsets
  {
    const int P = (W + T - 1) / T;
    const int w0 = min(tid * P, W), w1 = min(w0 + P, W);
    int32_t local = 0;
    for (int w = w0; w < w1; ++w) local += tot[w];
    int32_t total = 0;
    int32_t ex = block_exscan(local, 0, OpSum(), s_scan, &total);
    if (tables) {
      // the table block: base[0..W] become the offsets
      for (int w = w0; w < w1; ++w) {
        const int32_t t = tot[w];
        base[w] = ex;
        plan_offsets[w] = ex;
        if (offsets_out) offsets_out[w] = ex;
        ex += t;
      }
      if (tid == 0) {
        base[W] = total;
        plan_offsets[W] = total;
        if (offsets_out) offsets_out[W] = total;
      }
      lds_sync();
      int32_t n_long = 0, n_long4 = 0;
      const int32_t n_chunks =
          build_tables(base, hist, W, L, chunks, longs, s_scan, s_scan2, &n_long, &n_long4);
      if (tid == 0) write_header(hdr, n, W, L, n_chunks, n_long, n_long4, 0, invalid, invalid_out);
      return;
    }
    for (int w = w0; w < w1; ++w) {
      const int32_t t = tot[w];
      base[w] += ex;
      ex += t;
    }
  }
  if (!overlap) {
    // hist takes the place of the totals now
    lds_sync();
    for (int i = tid; i < nws * W; i += T) hist[i] = 0;
    lds_sync();
    count_rows();
    lds_sync();
  }
  // (d) exclusive prefix of the per-wave counts over the waves (all of a
  // window's counts are read before any is written back)
  for (int w = tid; w < W; w += T) {
    int32_t t[kBuildThreads / 64];
#pragma unroll
    for (int v = 0; v < kBuildThreads / 64; ++v) t[v] = v < nws ? hist[v * W + w] : 0;
    int32_t run = 0;
#pragma unroll
    for (int v = 0; v < kBuildThreads / 64; ++v) {
      if (v < nws) hist[v * W + w] = run;
      run += t[v];
    }
  }
  lds_sync();

  // (e) scatter, each wave with its running counters
  auto scatter_group = [&](int64_t r, int32_t id) {
    const int64_t i = r + lane;
    const bool valid = (uint32_t)id < (uint32_t)W;
    const uint64_t m = match_key(id, valid, nbits);
    if (valid) {
      const int32_t hb = h[id];
      const int32_t pos = base[id] + hb + __popcll(m & lt);
      if ((uint32_t)pos < (uint32_t)n) {
        perm[pos] = (int32_t)i;
        if (perm_out) perm_out[pos] = (int32_t)i;
      }
      if ((m & lt) == 0) h[id] = hb + __popcll(m);
    }
  };
  auto place = [&](int64_t r, int32_t id, int32_t rk) {
    if (rk < 0) return;
    const int32_t pos = base[id] + h[id] + rk;
    if ((uint32_t)pos < (uint32_t)n) {
      perm[pos] = (int32_t)(r + lane);
      if (perm_out) perm_out[pos] = (int32_t)(r + lane);
    }
  };
  if (ranks) {
    if (span <= 128) {
      // every row of the wave was ranked by the counting pass
      place(rbeg, id0, rk0);
      if (rbeg + 64 < rend) place(rbeg + 64, id1, rk1);
    } else {
      scatter_group(rbeg, id0);
      if (rbeg + 64 < rend) scatter_group(rbeg + 64, id1);
      for (int64_t r = rbeg + 128; r < rend; r += 64) scatter_group(r, id_at(r));
    }
  }
}

// Waves of k_scatter that rank rows: as many as the LDS holds (<= 16), and at
// most one per 64 rows of a block.
// Prefers the overlapped layout; large W falls back to the sequential one.
static int scatter_waves(int32_t W, int32_t E, size_t* lds_bytes, int* overlap) {
  constexpr size_t kLds = 160 * 1024 - 1024;   // leave room for the static arrays
  auto bytes = [&](int v, int ov) {
    const size_t h = (size_t)v * W > (size_t)W + 1 ? (size_t)v * W : (size_t)W + 1;
    return ((ov ? 2 : 1) * ((size_t)W + 1) + h) * 4;
  };
  for (int ov = 1; ov >= 0; --ov) {
    int nws = kBuildThreads / 64;
    while (nws > 1 && (bytes(nws, ov) > kLds || (int64_t)nws * 64 > E)) nws >>= 1;
    if (bytes(nws, ov) <= kLds || ov == 0) {
      *lds_bytes = bytes(nws, ov);
      *overlap = ov;
      return nws;
    }
  }
  return 1;
}

// ------------------------------------------------------------ host launchers
hipError_t launch_build(const int32_t* ids, int32_t n, int32_t W, int32_t L, int32_t* perm_out,
                        int32_t* offsets_io, int32_t* invalid_out, void* plan, hipStream_t stream) {
  const PlanLayout lay = plan_layout(n, W);
  char* base = static_cast<char*>(plan);
  PlanHeader* hdr = reinterpret_cast<PlanHeader*>(base + lay.header);
  int32_t* perm = reinterpret_cast<int32_t*>(base + lay.perm);
  int32_t* offs = reinterpret_cast<int32_t*>(base + lay.offsets);
  Chunk* chunks = reinterpret_cast<Chunk*>(base + lay.chunks);
  LongWin* longs = reinterpret_cast<LongWin*>(base + lay.longs);
  int32_t* counts = reinterpret_cast<int32_t*>(base + lay.counts);
  const int csr = ids == nullptr;
  if (csr || lay.n_blocks == 0) {
    hipLaunchKernelGGL(k_plan, dim3(1), dim3(kBuildThreads), 0, stream, csr, W, n, L, offsets_io,
                       invalid_out, hdr, offs, chunks, longs);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_count, dim3(lay.n_blocks), dim3(kBuildThreads), 0, stream, ids, n, W,
                     lay.block_elems, lay.counts_ld, counts);
  size_t lds = 0;
  int overlap = 0;
  const int nws = scatter_waves(W, lay.block_elems, &lds, &overlap);
  // the dynamic LDS of k_scatter exceeds the default limit: raise it once per device
  // (atomic: host threads may build plans concurrently; setting it twice is harmless)
  static std::atomic<bool> lds_attr[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64 || !lds_attr[dev].load(std::memory_order_acquire)) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_scatter),
                            hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024 - 1024);
    if (e != hipSuccess) return e;
    if (dev >= 0 && dev < 64) lds_attr[dev].store(true, std::memory_order_release);
  }
  hipLaunchKernelGGL(k_scatter, dim3(lay.n_blocks + 1), dim3(kBuildThreads), lds, stream, ids, n, W, L,
                     lay.block_elems, lay.n_blocks, lay.counts_ld, nws, overlap, counts, perm, perm_out,
                     offs, offsets_io, chunks, longs, hdr, invalid_out);
  return hipGetLastError();
}

}  // namespace sla

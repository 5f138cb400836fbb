// Segment builder: stable counting sort of rows by window id, CSR window offsets
// and the chunk table (Sec. 3.2 / Fig. 3(a): voxels ordered by window into one
// flattened matrix that is partitioned into chunks; the offset generation timed
// in Fig. 5 computes the start of every chunk).
//
// Mode A (ids given), two launches:
//   k_sort   per builder block of E rows: a stable LSD radix sort of the block's
//            rows by window id in LDS, and the exclusive prefix of the block's
//            window counts (the start of every window's run in the block);
//            it also adds the block's window counts to the plan's window totals;
//   k_merge  one workgroup turns the totals into the offsets, the chunk and
//            long-window tables and the header (and clears the totals); the
//            others take a range of windows each: offsets from the blocks' prefix
//            rows, and every sorted position of the range filled from the run of
//            the block it falls in.
// No workgroup waits on another, and every sum is an integer sum, so the result
// is deterministic.  The totals must be zero when a build starts: a new plan
// buffer is zero-filled once, and every build leaves them zero.
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

// -------------------------------------------------------- block-wide scans
struct OpSum {
  __device__ int32_t operator()(int32_t a, int32_t b) const { return a + b; }
};
struct OpSum64 {
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const { return a + b; }
};
template <typename V>
struct OpSumT {
  __device__ V operator()(V a, V b) const { return a + b; }
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

// Exclusive scan of one value per thread in thread order with one barrier; *total
// gets the reduction of all values.  The wave totals in s[0..15] must stay
// untouched until the caller's next barrier.
template <class Op, typename V>
__device__ __forceinline__ V block_exscan1(V x, V identity, Op op, V* s, V* total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nwv = blockDim.x >> 6;
  const V inc = wave_inclusive_scan(x, identity, op);
  if (lane == 63) s[wv] = inc;
  // exclusive inside the wave: the inclusive value of the lane before (wave_shr:1)
  V ex;
  if constexpr (sizeof(V) == 4) {
    ex = (V)__builtin_amdgcn_update_dpp((int)identity, (int)inc, 0x138, 0xf, 0xf, false);
  } else {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)identity, (int)(uint32_t)inc,
                                                              0x138, 0xf, 0xf, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)(identity >> 32),
                                                              (int)(uint32_t)(inc >> 32), 0x138, 0xf, 0xf,
                                                              false);
    ex = ((V)hi << 32) | lo;
  }
  lds_sync();
  V before = identity, all = identity;
  for (int u = 0; u < nwv; ++u) {
    const V t = s[u];
    if (u < wv) before = op(before, t);
    all = op(all, t);
  }
  *total = all;
  return op(before, ex);
}

// ------------------------------------------------------ chunk / long tables
// Work tables from the offsets in LDS, in sequence order (pages of P = L/2 rows):
// a window of more than L rows is "long" and goes to the long-window table
// (four-way ones, of more than 2L rows, first, then two-way ones); a window of
// P+1..L rows is a chunk of its own; a window of 1..P rows opens a chunk unless
// the previous non-empty window is short and starts in the same page.  A chunk
// runs to the next event (chunk start or long window).  s_aux: LDS scratch of at
// least W ints.  Every thread of the block calls it (at most 32 windows a thread:
// W <= 32 blockDim.x); returns the number of chunks and sets *n_long and
// *n_long4.
__device__ int32_t build_tables(const int32_t* s_off, int32_t* s_aux, int32_t W, int32_t L,
                                Chunk* __restrict__ chunks, LongWin* __restrict__ longs,
                                int32_t* s_scan, uint64_t* s_scan2, int32_t* n_long,
                                int32_t* n_long4) {
  const int tid = threadIdx.x, T = blockDim.x;
  const int32_t page = L >> 1;
  // x / page = (x m) >> 37 with m = ceil(2^37 / page), exact for 0 <= x < 2^31 and
  // page <= 32 (the rounding error stays below 1/64, the distance of x / page to
  // the next integer at least 1/32)
  const uint64_t pm = ((1ull << 37) + (uint64_t)page - 1) / (uint64_t)page;
  auto page_of = [&](int32_t x) -> uint32_t { return (uint32_t)(((uint64_t)(uint32_t)x * pm) >> 37); };
  const int P = (W + T - 1) / T;
  const int w0 = min(tid * P, W), w1 = min(w0 + P, W);
  // the start of the last non-empty window and the end of the last window of
  // more than P rows before my range decide the kind of my first window
  int32_t aggStart = -1, aggWide = -1;
  for (int w = w0; w < w1; ++w) {
    const int32_t a = s_off[w], len = s_off[w + 1] - a;
    if (len > 0) aggStart = a;
    if (len > page) aggWide = a + len;
  }
  // both maxima in one scan of (value + 1) pairs
  uint64_t tmp;
  const uint64_t both = block_exscan1<OpMax2, uint64_t>(
      ((uint64_t)(uint32_t)(aggStart + 1) << 32) | (uint32_t)(aggWide + 1), 0ull, OpMax2(), s_scan2,
      &tmp);
  // 0: no event, 1: opens a chunk, 2: two-way long window, 3: four-way long
  // window; 2 bits a window in `codes`
  uint64_t codes = 0;
  uint64_t cnt = 0;   // chunks, two-way, four-way: 21 bits each (W <= 16384)
  {
    int32_t ls = (int32_t)(both >> 32) - 1;          // start of the previous non-empty window
    int32_t ll = (int32_t)(uint32_t)both - 1;        // end of the previous window of > P rows
    for (int w = w0; w < w1; ++w) {
      const int32_t a = s_off[w], len = s_off[w + 1] - a;
      int k = 0;
      if (len > 0) {
        if (len > L) k = len > 2 * L ? 3 : 2;
        else if (len > page || ls < 0 || ll == a || page_of(ls) != page_of(a)) k = 1;
        ls = a;
        if (len > page) ll = a + len;
      }
      codes |= (uint64_t)k << (2 * (w - w0));
      if (k) cnt += 1ull << (21 * (k - 1));
    }
  }
  lds_sync();   // s_scan2 is reused
  uint64_t tot = 0;
  const uint64_t ex = block_exscan1<OpSum64, uint64_t>(cnt, 0ull, OpSum64(), s_scan2, &tot);
  constexpr uint64_t kMask = (1ull << 21) - 1;
  const int32_t s0 = (int32_t)(ex & kMask), t0 = (int32_t)((ex >> 21) & kMask),
                f0 = (int32_t)(ex >> 42);
  const int32_t nC = (int32_t)(tot & kMask), n2 = (int32_t)((tot >> 21) & kMask),
                n4 = (int32_t)(tot >> 42);
  {
    // the event list in sequence order: s_aux[event index] = window
    int32_t e = s0 + t0 + f0;
    for (int w = w0; w < w1; ++w)
      if ((codes >> (2 * (w - w0))) & 3u) s_aux[e++] = w;
  }
  lds_sync();
  {
    int32_t sc = s0, s2 = t0, s4 = f0;
    const int32_t nE = nC + n2 + n4;
    for (int w = w0; w < w1; ++w) {
      const int k = (int)((codes >> (2 * (w - w0))) & 3u);
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

// -------------------------------------------- tables straight from the totals
// The same tables as build_tables, from window lengths (the totals) rather than
// offsets, with one scan fewer: a segment of windows is summarised by the rows
// it holds, the start of its last non-empty window and the end of its last
// window of more than P rows (both relative to the segment's first row, -1 for
// none).  Joining two segments adds rows and shifts the second one's positions
// by the first one's rows, so one scan over the threads' segments gives each
// thread its first offset and the two positions the chunk rule needs.
struct WinSeg {
  int32_t rows, last_start, wide_end;
};

__device__ __forceinline__ WinSeg seg_join(WinSeg a, WinSeg b) {
  WinSeg r;
  r.rows = a.rows + b.rows;
  r.last_start = b.last_start >= 0 ? a.rows + b.last_start : a.last_start;
  r.wide_end = b.wide_end >= 0 ? a.rows + b.wide_end : a.wide_end;
  return r;
}

// v joined after the value CTRL moves in (the identity where nothing moves in)
template <int CTRL, int ROWS>
__device__ __forceinline__ WinSeg seg_step(WinSeg v) {
  WinSeg m;
  m.rows = __builtin_amdgcn_update_dpp(0, v.rows, CTRL, ROWS, 0xf, false);
  m.last_start = __builtin_amdgcn_update_dpp(-1, v.last_start, CTRL, ROWS, 0xf, false);
  m.wide_end = __builtin_amdgcn_update_dpp(-1, v.wide_end, CTRL, ROWS, 0xf, false);
  return seg_join(m, v);
}

// Exclusive join over the threads of the block, in thread order (one barrier;
// s[0..15] must stay untouched until the caller's next barrier).
__device__ __forceinline__ WinSeg seg_exscan(WinSeg v, WinSeg* s) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  WinSeg inc = v;
  inc = seg_step<0x111, 0xf>(inc);  // row_shr:1
  inc = seg_step<0x112, 0xf>(inc);  // row_shr:2
  inc = seg_step<0x114, 0xf>(inc);  // row_shr:4
  inc = seg_step<0x118, 0xf>(inc);  // row_shr:8
  inc = seg_step<0x142, 0xa>(inc);  // row_bcast:15
  inc = seg_step<0x143, 0xc>(inc);  // row_bcast:31
  if (lane == 63) s[wv] = inc;
  WinSeg ex;   // the inclusive value of the lane before (wave_shr:1)
  ex.rows = __builtin_amdgcn_update_dpp(0, inc.rows, 0x138, 0xf, 0xf, false);
  ex.last_start = __builtin_amdgcn_update_dpp(-1, inc.last_start, 0x138, 0xf, 0xf, false);
  ex.wide_end = __builtin_amdgcn_update_dpp(-1, inc.wide_end, 0x138, 0xf, 0xf, false);
  lds_sync();
  WinSeg before = {0, -1, -1};
  for (int u = 0; u < wv; ++u) before = seg_join(before, s[u]);
  return seg_join(before, ex);
}

// Reads (and clears) the window totals totals[0..W], writes the offsets (to the
// plan, to offsets_out when given, and to s_off[0..W]), the chunk and
// long-window tables; returns the chunk count, sets *n_long, *n_long4 and
// *invalid (rows with an out-of-range id).  LDS: s_off[W + 1], s_aux[W].  At
// most 32 windows a thread.
__device__ int32_t tables_from_totals(int32_t* __restrict__ totals, int32_t W, int32_t L,
                                      int32_t* __restrict__ plan_offsets,
                                      int32_t* __restrict__ offsets_out, int32_t* s_off,
                                      int32_t* s_aux, Chunk* __restrict__ chunks,
                                      LongWin* __restrict__ longs, WinSeg* s_seg, uint64_t* s_scan2,
                                      int32_t* n_long, int32_t* n_long4, int32_t* invalid) {
  const int tid = threadIdx.x, T = blockDim.x;
  const int32_t page = L >> 1;
  // x / page = (x m) >> 37 with m = ceil(2^37 / page) (as in build_tables)
  const uint64_t pm = ((1ull << 37) + (uint64_t)page - 1) / (uint64_t)page;
  auto page_of = [&](int32_t x) -> uint32_t { return (uint32_t)(((uint64_t)(uint32_t)x * pm) >> 37); };
  const int P = (W + T - 1) / T;
  const int w0 = min(tid * P, W), w1 = min(w0 + P, W);
  // this thread's windows as a segment; their lengths stay in LDS
  WinSeg own = {0, -1, -1};
  for (int w = w0; w < w1; ++w) {
    const int32_t len = totals[w];
    totals[w] = 0;
    s_aux[w] = len;
    if (len > 0) own.last_start = own.rows;
    if (len > page) own.wide_end = own.rows + len;
    own.rows += len;
  }
  if (tid == 0) {
    *invalid = totals[W];
    totals[W] = 0;
  }
  const WinSeg ex = seg_exscan(own, s_seg);
  // 0: no event, 1: opens a chunk, 2: two-way long window, 3: four-way long
  // window; 2 bits a window in `codes`
  uint64_t codes = 0;
  uint64_t cnt = 0;   // chunks, two-way, four-way: 21 bits each (W <= 16384)
  {
    int32_t a = ex.rows, ls = ex.last_start, ll = ex.wide_end;
    for (int w = w0; w < w1; ++w) {
      const int32_t len = s_aux[w];
      int k = 0;
      if (len > 0) {
        if (len > L) k = len > 2 * L ? 3 : 2;
        else if (len > page || ls < 0 || ll == a || page_of(ls) != page_of(a)) k = 1;
        ls = a;
        if (len > page) ll = a + len;
      }
      codes |= (uint64_t)k << (2 * (w - w0));
      if (k) cnt += 1ull << (21 * (k - 1));
      s_off[w] = a;
      plan_offsets[w] = a;
      if (offsets_out) offsets_out[w] = a;
      a += len;
    }
    if (w1 == W && w0 < w1) {
      s_off[W] = a;
      plan_offsets[W] = a;
      if (offsets_out) offsets_out[W] = a;
    }
  }
  uint64_t tot = 0;
  const uint64_t exc = block_exscan1<OpSum64, uint64_t>(cnt, 0ull, OpSum64(), s_scan2, &tot);
  constexpr uint64_t kMask = (1ull << 21) - 1;
  const int32_t s0 = (int32_t)(exc & kMask), t0 = (int32_t)((exc >> 21) & kMask),
                f0 = (int32_t)(exc >> 42);
  const int32_t nC = (int32_t)(tot & kMask), n2 = (int32_t)((tot >> 21) & kMask),
                n4 = (int32_t)(tot >> 42);
  lds_sync();   // every window's length has been read from s_aux
  {
    int32_t e = s0 + t0 + f0;
    for (int w = w0; w < w1; ++w)
      if ((codes >> (2 * (w - w0))) & 3u) s_aux[e++] = w;
  }
  lds_sync();   // the event list and s_off
  {
    int32_t sc = s0, s2 = t0, s4 = f0;
    const int32_t nE = nC + n2 + n4;
    for (int w = w0; w < w1; ++w) {
      const int k = (int)((codes >> (2 * (w - w0))) & 3u);
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

// ------------------------------------------------------------ row ranking
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

// ------------------------------------------------------------------ k_sort
// One workgroup per builder block of E = 1024 R rows.  Sorts the block's rows by
// key (window id; W for an id outside [0, W); W + 1 for the padding after the
// last row) with a stable LSD radix sort in LDS, 8 key bits per pass (at most two
// passes, W <= 16384): a wave ranks its rows 64 at a time in row order (ballots
// find the lanes with the same digit), a scan over (digit, wave) gives every row
// its place.  Writes
//   sorted[block E + p]   row at position p of the block's sorted order;
//   counts[block][x]      rows of the block with key < x, x = 0..W (the start of
//                         window x's run in the block's sorted order);
// and adds its window counts (x = 0..W; x = W counts the ids outside [0, W)) to
// the window totals, integer atomics, so the sums do not depend on their order.
// Both go out as soon as the histogram is complete, under the radix passes.
// LDS: hist[ld] | buf[2][E] | wcnt[2][256][17] (one count table when R = 8).
constexpr int kSortThreads = 1024;
constexpr int kSortWaves = kSortThreads / 64;
constexpr int kDigits = 256;
// (digit, wave) counters kCountLd ints apart per digit: with 16 the 64 lanes of a
// wave, each on its own digit, would all fall in two LDS banks
constexpr int kCountLd = kSortWaves + 1;
constexpr int kPosBits = 13;   // position of a row in its block (E <= 8192)

// Exclusive sum over the threads of the block in thread order, one barrier; the
// wave totals in s[0..15] must stay untouched until the caller's next barrier.
template <typename V>
__device__ __forceinline__ V block_exsum(V x, V* s) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const V inc = wave_inclusive_scan(x, (V)0, OpSumT<V>());
  if (lane == 63) s[wv] = inc;
  lds_sync();
  V before = 0;
  for (int u = 0; u < wv; ++u) before += s[u];
  return before + inc - x;
}

template <int R>
__global__ __launch_bounds__(kSortThreads) void k_sort(const int32_t* __restrict__ ids, int32_t n,
                                                      int32_t W, int32_t ld,
                                                      int32_t* __restrict__ counts,
                                                      int32_t* __restrict__ sorted,
                                                      int32_t* __restrict__ totals) {
  constexpr int E = kSortThreads * R;
  constexpr bool kTwoTables = R <= 4;   // LDS budget at W = 16384
  constexpr int kTable = kDigits * kCountLd;
  static_assert(E <= (1 << kPosBits), "row positions fit their field");
  extern __shared__ int32_t lds[];
  __shared__ uint64_t s_scan[kSortWaves];
  int32_t* hist = lds;
  uint32_t* buf = reinterpret_cast<uint32_t*>(lds + ld);   // buf[0..E) and buf[E..2E)
  int32_t* wcnt = lds + ld + 2 * E;                         // table t at wcnt + t kTable
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t base = (int64_t)blockIdx.x * E;
  const int32_t rows = (int32_t)(n - base < E ? n - base : E);
  // sub-group r of wave wv holds positions wv 64 R + 64 r + lane (row order)
  uint32_t el[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int pos = wv * 64 * R + 64 * r + lane;
    uint32_t key = (uint32_t)W + 1u;
    if (pos < rows) {
      const int32_t id = ids[base + pos];
      key = (uint32_t)id < (uint32_t)W ? (uint32_t)id : (uint32_t)W;
    }
    el[r] = (key << kPosBits) | (uint32_t)pos;
  }
  for (int i = tid; i < ld; i += kSortThreads) hist[i] = 0;
  for (int i = tid; i < (kTwoTables ? 2 : 1) * kTable; i += kSortThreads) wcnt[i] = 0;
  lds_sync();
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const uint32_t key = el[r] >> kPosBits;
    if (key <= (uint32_t)W) atomicAdd(&hist[key], 1);
  }

  const int kbits = 32 - __clz(W + 1);   // bits of the largest key, W + 1
  const int X = (W + 1 + kSortThreads - 1) / kSortThreads;
  const int x0 = min(tid * X, W + 1), x1 = min(x0 + X, W + 1);
  const uint64_t lt = lanemask_lt(lane);
  for (int pass = 0, shift = 0; shift < kbits; ++pass, shift += 8) {
    const int dbits = kbits - shift < 8 ? kbits - shift : 8;
    int32_t* tab = wcnt + (kTwoTables ? pass * kTable : 0);
    // (1) ranks inside the wave, sub-groups in row order
    int32_t rk[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int32_t d = (int32_t)((el[r] >> (kPosBits + shift)) & 0xffu);
      const uint64_t m = match_key(d, true, dbits);
      int32_t* slot = &tab[d * kCountLd + wv];
      const int32_t before = *slot;   // a wave's LDS accesses complete in order
      if ((m & lt) == 0) *slot = before + __popcll(m);
      rk[r] = before + __popcll(m & lt);
    }
    lds_sync();
    // (2) exclusive scan of the table in (digit, wave) order, four entries a
    // thread; the first pass also scans the histogram (high half of the sum)
    int32_t v[4], hsum = 0;
    uint64_t sum = 0;
    // entries 4 tid .. 4 tid + 3 of the (digit, wave) order: digit tid / 4, waves
    // 4 (tid % 4) .. + 3
    int32_t* ent = tab + (tid >> 2) * kCountLd + 4 * (tid & 3);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      v[k] = ent[k];
      sum += (uint32_t)v[k];
    }
    if (pass == 0) {
      for (int x = x0; x < x1; ++x) hsum += hist[x];
      sum |= (uint64_t)(uint32_t)hsum << 32;
    }
    const uint64_t ex = block_exsum<uint64_t>(sum, s_scan);
    int32_t e = (int32_t)(uint32_t)ex;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      ent[k] = e;
      e += v[k];
    }
    if (pass == 0) {
      // the block's prefix row and its share of the totals leave now
      int32_t h = (int32_t)(ex >> 32);
      int32_t* row = counts + (size_t)blockIdx.x * ld;
      for (int x = x0; x < x1; ++x) {
        const int32_t c = hist[x];
        row[x] = h;
        h += c;
        if (c) __hip_atomic_fetch_add(totals + x, c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    lds_sync();
    // (3) every row to its place
    uint32_t* dst = buf + (pass & 1) * E;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int32_t d = (int32_t)((el[r] >> (kPosBits + shift)) & 0xffu);
      dst[tab[d * kCountLd + wv] + rk[r]] = el[r];
    }
    lds_sync();
#pragma unroll
    for (int r = 0; r < R; ++r) el[r] = dst[wv * 64 * R + 64 * r + lane];
    if (!kTwoTables && shift + 8 < kbits) {
      for (int i = tid; i < kTable; i += kSortThreads) tab[i] = 0;
      lds_sync();
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int pos = wv * 64 * R + 64 * r + lane;
    if (pos < rows) sorted[base + pos] = (int32_t)(base + (el[r] & ((1u << kPosBits) - 1u)));
  }
}

// ------------------------------------------------------------------ k_merge
// Workgroup 0 writes the offsets (the exclusive scan of the window totals), the
// chunk and long-window tables and the header, and clears the totals for the next
// build.  Workgroup 1 + r takes the range of ww windows [w0, w0 + nx): from the
// blocks' prefix rows (counts[b][x], x = w0..w0 + nx) it forms, per column x, the
// exclusive sum over blocks ex[x][b] = sum_{b' < b} counts[b'][x]; ex[x][nb] is
// offsets[x] (rows with a window id below x, over all blocks), and the rows of
// window w in block b follow those of blocks b' < b:
//   sorted position offsets[w] + pre(b) + j, pre(b) = ex[w + 1][b] - ex[w][b],
//   is row sorted[b E + counts[b][w] + j].
// Every sorted position of the range finds its block by binary search over pre.
// No workgroup waits for another.
constexpr int kMergeThreads = 1024;

__global__ __launch_bounds__(kMergeThreads) void k_merge(
    int32_t n, int32_t W, int32_t L, int32_t E, int32_t nb, int32_t ld, int32_t ww,
    const int32_t* __restrict__ counts, const int32_t* __restrict__ sorted,
    int32_t* __restrict__ totals, int32_t* __restrict__ perm, int32_t* __restrict__ perm_out,
    int32_t* __restrict__ plan_offsets, int32_t* __restrict__ offsets_out,
    Chunk* __restrict__ chunks, LongWin* __restrict__ longs, PlanHeader* __restrict__ hdr,
    int32_t* __restrict__ invalid_out) {
  extern __shared__ int32_t lds[];
  __shared__ int32_t s_scan[33];
  __shared__ uint64_t s_scan2[33];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (blockIdx.x == 0) {
    __shared__ WinSeg s_seg[kMergeThreads / 64];
    __shared__ int32_t s_invalid;
    int32_t* s_off = lds;
    int32_t* s_aux = lds + (W + 1);
    int32_t n_long = 0, n_long4 = 0;
    const int32_t n_chunks = tables_from_totals(totals, W, L, plan_offsets, offsets_out, s_off, s_aux, chunks,
                                                longs, s_seg, s_scan2, &n_long, &n_long4, &s_invalid);
    lds_sync();
    if (tid == 0) write_header(hdr, n, W, L, n_chunks, n_long, n_long4, 0, s_invalid, invalid_out);
    return;
  }
  const int32_t w0 = ((int32_t)blockIdx.x - 1) * ww;
  const int nx = min(ww, W - w0);
  const int S = nb + 1;
  int32_t* ex = lds;   // ex[xi S + b], xi = 0..nx, b = 0..nb
  // (1) the tile, row by row of the matrix (nx + 1 consecutive ints per block)
  for (int f = tid; f < nb * (nx + 1); f += kMergeThreads) {
    const int b = f / (nx + 1), xi = f - b * (nx + 1);
    ex[xi * S + b + 1] = counts[(size_t)b * ld + w0 + xi];
  }
  if (tid <= nx) ex[tid * S] = 0;
  lds_sync();
  // (2) inclusive scan of every column over the blocks, one wave a column
  for (int xi = wv; xi <= nx; xi += kMergeThreads / 64) {
    int32_t carry = 0;
    for (int b0 = 1; b0 <= nb; b0 += 64) {
      const int b = b0 + lane;
      const int32_t v = b <= nb ? ex[xi * S + b] : 0;
      const int32_t inc = wave_inclusive_scan(v, 0, OpSum()) + carry;
      if (b <= nb) ex[xi * S + b] = inc;
      carry = __builtin_amdgcn_readlane(inc, 63);
    }
  }
  lds_sync();
  // (3) the range's sorted positions
  const int32_t p0 = ex[nb], p1 = ex[nx * S + nb];
  for (int32_t p = p0 + tid; p < p1; p += kMergeThreads) {
    int lo = 0, hi = nx - 1;   // last window of the range starting at or before p
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (ex[mid * S + nb] <= p) lo = mid; else hi = mid - 1;
    }
    const int wi = lo;
    const int32_t q = p - ex[wi * S + nb];
    const int32_t* e0 = ex + wi * S;
    const int32_t* e1 = e0 + S;
    int bl = 0, bh = nb - 1;   // last block whose rows of window wi start at or before q
    while (bl < bh) {
      const int mid = (bl + bh + 1) >> 1;
      if (e1[mid] - e0[mid] <= q) bl = mid; else bh = mid - 1;
    }
    const int32_t j = q - (e1[bl] - e0[bl]);
    const int32_t start = e0[bl + 1] - e0[bl];
    const int64_t at = (int64_t)bl * E + start + j;
    const int32_t row = at < n ? sorted[at] : 0;
    if (p < n) {
      perm[p] = row;
      if (perm_out) perm_out[p] = row;
    }
  }
  // (4) the last range also lists the rows whose ids are out of range, after every
  // window (sorted positions offsets[W] .. n - 1), in row order: in block b they
  // follow its rows in windows, and blocks before b hold pre(b) = b E - ex[W][b]
  if (w0 + nx == W) {
    const int32_t* eW = ex + nx * S;
    const int32_t q0 = eW[nb];
    for (int32_t p = q0 + tid; p < n; p += kMergeThreads) {
      const int32_t q = p - q0;
      int bl = 0, bh = nb - 1;
      while (bl < bh) {
        const int mid = (bl + bh + 1) >> 1;
        if ((int64_t)mid * E - eW[mid] <= q) bl = mid; else bh = mid - 1;
      }
      const int64_t j = q - ((int64_t)bl * E - eW[bl]);
      const int64_t at = (int64_t)bl * E + (eW[bl + 1] - eW[bl]) + j;
      const int32_t row = at < n ? sorted[at] : 0;
      perm[p] = row;
      if (perm_out) perm_out[p] = row;
    }
  }
}

// ------------------------------------------------------------ host launchers
// Windows per merge workgroup: about 256 range workgroups, the tile within 96 KB.
static int merge_windows(int32_t W, int32_t nb) {
  const int by_lds = (24 * 1024) / (nb + 1) - 1;
  int ww = (W + 255) / 256;
  if (ww > by_lds) ww = by_lds;
  return ww < 1 ? 1 : ww;
}

template <typename K>
static hipError_t raise_lds_limit(K* kernel, std::atomic<bool>* done, int dev) {
  if (dev >= 0 && dev < 64 && done[dev].load(std::memory_order_acquire)) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024 - 1024);
  if (e == hipSuccess && dev >= 0 && dev < 64) done[dev].store(true, std::memory_order_release);
  return e;
}

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
  int32_t* sorted = reinterpret_cast<int32_t*>(base + lay.sorted);
  int32_t* totals = reinterpret_cast<int32_t*>(base + lay.totals);
  const int csr = ids == nullptr;
  if (csr || lay.n_blocks == 0) {
    hipLaunchKernelGGL(k_plan, dim3(1), dim3(kBuildThreads), 0, stream, csr, W, n, L, offsets_io,
                       invalid_out, hdr, offs, chunks, longs);
    return hipGetLastError();
  }
  if (lay.n_blocks > kBuilderMaxBlocks) return hipErrorInvalidValue;
  // the dynamic LDS of both kernels may exceed the default limit: raise it once per
  // device (atomic: host threads may build plans concurrently; setting it twice is harmless)
  static std::atomic<bool> attr_sort[4][64] = {}, attr_merge[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const int R = lay.block_elems / kSortThreads;
  const size_t sort_lds =
      ((size_t)lay.counts_ld + 2 * (size_t)lay.block_elems + (R <= 4 ? 2 : 1) * kDigits * kCountLd) * 4;
  const dim3 sg(lay.n_blocks), st(kSortThreads);
  switch (R) {
    case 1:
      if ((e = raise_lds_limit(&k_sort<1>, attr_sort[0], dev)) != hipSuccess) return e;
      hipLaunchKernelGGL(k_sort<1>, sg, st, sort_lds, stream, ids, n, W, lay.counts_ld, counts, sorted, totals);
      break;
    case 2:
      if ((e = raise_lds_limit(&k_sort<2>, attr_sort[1], dev)) != hipSuccess) return e;
      hipLaunchKernelGGL(k_sort<2>, sg, st, sort_lds, stream, ids, n, W, lay.counts_ld, counts, sorted, totals);
      break;
    case 4:
      if ((e = raise_lds_limit(&k_sort<4>, attr_sort[2], dev)) != hipSuccess) return e;
      hipLaunchKernelGGL(k_sort<4>, sg, st, sort_lds, stream, ids, n, W, lay.counts_ld, counts, sorted, totals);
      break;
    case 8:
      if ((e = raise_lds_limit(&k_sort<8>, attr_sort[3], dev)) != hipSuccess) return e;
      hipLaunchKernelGGL(k_sort<8>, sg, st, sort_lds, stream, ids, n, W, lay.counts_ld, counts, sorted, totals);
      break;
    default:
      return hipErrorInvalidValue;
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int ww = merge_windows(W, lay.n_blocks);
  const int groups = (W + ww - 1) / ww;
  const size_t tile = (size_t)(ww + 1) * (lay.n_blocks + 1), tables = 2 * ((size_t)W + 1);
  const size_t merge_lds = (tile > tables ? tile : tables) * 4;
  if ((e = raise_lds_limit(&k_merge, attr_merge, dev)) != hipSuccess) return e;
  hipLaunchKernelGGL(k_merge, dim3(groups + 1), dim3(kMergeThreads), merge_lds, stream, n, W, L,
                     lay.block_elems, lay.n_blocks, lay.counts_ld, ww, counts, sorted, totals, perm,
                     perm_out, offs, offsets_io, chunks, longs, hdr, invalid_out);
  return hipGetLastError();
}

}  // namespace sla

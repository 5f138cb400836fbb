// Segment builder: stable counting sort of rows by window id, CSR window offsets
// and the chunk table (Sec. 3.2 / Fig. 3(a): voxels ordered by window into one
// flattened matrix that is partitioned into chunks; Fig. 5 caption: "offsets
// generation" computes the start of every chunk).
//
// Three launches in mode A (ids given), one in mode B (CSR given):
//   k_count    per builder block, a histogram of its rows' window ids (LDS atomics;
//              the counts are order-free, hence deterministic);
//   k_plan     one workgroup: per-window column prefix over the blocks, exclusive
//              scan -> offsets, then the chunk table from the offsets;
//   k_scatter  per builder block, the stable rank of every row among the rows of
//              the same window in this block (wave ballots on the id bits give the
//              set of lanes sharing an id; waves then take their base in order),
//              and perm[offsets[id] + block prefix + rank] = row.
#include "sla_common.h"

namespace sla {

constexpr int kPlanThreads = 1024;

// ------------------------------------------------------------------ k_count
__global__ __launch_bounds__(256) void k_count(const int32_t* __restrict__ ids, int32_t n,
                                                int32_t W, int32_t E, int32_t* __restrict__ counts) {
  __shared__ int32_t hist[kMaxWindows + 1];
  for (int i = threadIdx.x; i <= W; i += blockDim.x) hist[i] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * E;
  const int64_t end = base + E < n ? base + E : n;
  for (int64_t i = base + threadIdx.x; i < end; i += blockDim.x) {
    const int32_t id = ids[i];
    atomicAdd(&hist[(uint32_t)id < (uint32_t)W ? id : W], 1);
  }
  __syncthreads();
  int32_t* row = counts + (size_t)blockIdx.x * (W + 1);
  for (int i = threadIdx.x; i <= W; i += blockDim.x) row[i] = hist[i];
}

// -------------------------------------------------------- block-wide scans
struct OpSum {
  __device__ int32_t operator()(int32_t a, int32_t b) const { return a + b; }
};
struct OpMax {
  __device__ int32_t operator()(int32_t a, int32_t b) const { return a > b ? a : b; }
};

// Exclusive scan of one value per thread in thread order; *total gets the
// reduction of all values.  Uses s[0..32]; ends with a barrier so s can be reused.
template <class Op>
__device__ int32_t block_exscan(int32_t x, int32_t identity, Op op, int32_t* s, int32_t* total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nwv = blockDim.x >> 6;
  int32_t inc = x;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int32_t y = __shfl_up(inc, d, 64);
    if (lane >= d) inc = op(inc, y);
  }
  if (lane == 63) s[wv] = inc;
  __syncthreads();
  if (wv == 0) {
    const int32_t v = lane < nwv ? s[lane] : identity;
    int32_t inc2 = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int32_t y = __shfl_up(inc2, d, 64);
      if (lane >= d) inc2 = op(inc2, y);
    }
    int32_t ex2 = __shfl_up(inc2, 1, 64);
    if (lane == 0) ex2 = identity;
    if (lane < nwv) s[lane] = ex2;
    if (lane == nwv - 1) s[32] = inc2;
  }
  __syncthreads();
  int32_t ex = __shfl_up(inc, 1, 64);
  if (lane == 0) ex = identity;
  const int32_t r = op(s[wv], ex);
  *total = s[32];
  __syncthreads();
  return r;
}

// ------------------------------------------------------------------ k_plan
// csr == 0: counts holds the [n_blocks][W + 1] block histograms (column W =
// out-of-range ids).  Each column is replaced by its exclusive prefix over the
// blocks (k_scatter reads it) and the column totals are scanned into offsets.
// csr == 1: offsets_io is the caller's CSR input; it is validated and clamped.
__global__ __launch_bounds__(kPlanThreads) void k_plan(int32_t csr, int32_t* __restrict__ counts,
                                                       int32_t nb, int32_t W, int32_t n, int32_t L,
                                                       int32_t* __restrict__ offsets_io,
                                                       int32_t* __restrict__ invalid_out,
                                                       PlanHeader* __restrict__ hdr,
                                                       int32_t* __restrict__ plan_offsets,
                                                       Chunk* __restrict__ chunks) {
  __shared__ int32_t s_off[kMaxWindows + 1];
  __shared__ int32_t s_aux[kMaxWindows + 1];
  __shared__ int32_t s_scan[33];
  const int tid = threadIdx.x, T = blockDim.x;
  int32_t invalid = 0, total = 0;

  if (!csr) {
    // column prefix over blocks, window totals into s_aux (s_aux[W] = invalid rows)
    for (int w = tid; w <= W; w += T) {
      int32_t run = 0;
      int b = 0;
      for (; b + 8 <= nb; b += 8) {
        int32_t c[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) c[u] = counts[(size_t)(b + u) * (W + 1) + w];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          counts[(size_t)(b + u) * (W + 1) + w] = run;
          run += c[u];
        }
      }
      for (; b < nb; ++b) {
        const int32_t c = counts[(size_t)b * (W + 1) + w];
        counts[(size_t)b * (W + 1) + w] = run;
        run += c;
      }
      s_aux[w] = run;
    }
    __syncthreads();
    invalid = s_aux[W];
    // exclusive scan of the totals: thread t owns windows [t P, t P + P)
    const int P = (W + T - 1) / T;
    const int w0 = tid * P, w1 = min(w0 + P, W);
    int32_t local = 0;
    for (int w = w0; w < w1; ++w) local += s_aux[w];
    int32_t ex = block_exscan(local, 0, OpSum(), s_scan, &total);
    for (int w = w0; w < w1; ++w) {
      s_off[w] = ex;
      ex += s_aux[w];
    }
    if (tid == 0) s_off[W] = total;
  } else {
    // validate and clamp the caller's offsets: s_off = running max of clamp(x, 0, n)
    const int P = (W + 1 + T - 1) / T;
    const int w0 = tid * P, w1 = min(w0 + P, W + 1);
    int32_t bad = 0, mx = 0;
    for (int w = w0; w < w1; ++w) {
      const int32_t x = offsets_io[w];
      bad += (x < 0 || x > n);
      if (w > 0) bad += x < offsets_io[w - 1];
      const int32_t cx = x < 0 ? 0 : (x > n ? n : x);
      mx = cx > mx ? cx : mx;
    }
    int32_t ex_max = block_exscan(mx, 0, OpMax(), s_scan, &total);
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
    if (tid == 0) {
      invalid += (offsets_io[0] != 0) + (offsets_io[W] != n);
    }
  }
  __syncthreads();

  // publish offsets
  for (int w = tid; w <= W; w += T) {
    plan_offsets[w] = s_off[w];
    if (!csr && offsets_io) offsets_io[w] = s_off[w];
  }

  // ---- chunk table (page rule) ----
  const int32_t page = L >> 1;
  const int P = (W + T - 1) / T;
  const int w0 = tid * P, w1 = min(w0 + P, W);
  int32_t aggStart = -1, aggLong = -1;
  for (int w = w0; w < w1; ++w) {
    const int32_t len = s_off[w + 1] - s_off[w];
    if (len > 0) aggStart = s_off[w];
    if (len > page) aggLong = s_off[w + 1];
  }
  int32_t tmp;
  int32_t lastStart = block_exscan(aggStart, -1, OpMax(), s_scan, &tmp);
  int32_t lastLongEnd = block_exscan(aggLong, -1, OpMax(), s_scan, &tmp);
  // count chunk starts among my windows
  int32_t cnt = 0;
  {
    int32_t ls = lastStart, ll = lastLongEnd;
    for (int w = w0; w < w1; ++w) {
      const int32_t a = s_off[w], len = s_off[w + 1] - a;
      if (len <= 0) continue;
      const bool is_long = len > page;
      const bool start = is_long || ls < 0 || ll == a || (ls / page) != (a / page);
      cnt += start;
      ls = a;
      if (is_long) ll = a + len;
    }
  }
  int32_t n_chunks = 0;
  int32_t c = block_exscan(cnt, 0, OpSum(), s_scan, &n_chunks);
  // s_aux is free again: record each chunk's first window
  {
    int32_t ls = lastStart, ll = lastLongEnd;
    for (int w = w0; w < w1; ++w) {
      const int32_t a = s_off[w], len = s_off[w + 1] - a;
      if (len <= 0) continue;
      const bool is_long = len > page;
      const bool start = is_long || ls < 0 || ll == a || (ls / page) != (a / page);
      if (start) s_aux[c++] = w;
      ls = a;
      if (is_long) ll = a + len;
    }
  }
  __syncthreads();
  for (int i = tid; i < n_chunks; i += T) {
    const int32_t wb = s_aux[i];
    const int32_t we = i + 1 < n_chunks ? s_aux[i + 1] : W;
    Chunk ch;
    ch.row_begin = s_off[wb];
    ch.row_end = s_off[we];
    ch.win_begin = wb;
    ch.win_end = we;
    chunks[i] = ch;
  }
  if (tid == 0) {
    hdr->magic = kPlanMagic;
    hdr->n = n;
    hdr->num_windows = W;
    hdr->chunk_rows = L;
    hdr->n_chunks = n_chunks;
    hdr->csr = csr;
    hdr->invalid = invalid;
    hdr->claim[0] = hdr->claim[1] = 0;
    hdr->done[0] = hdr->done[1] = 0;
    if (invalid_out) *invalid_out = invalid;
  }
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

__global__ __launch_bounds__(256) void k_scatter(const int32_t* __restrict__ ids, int32_t n,
                                                  int32_t W, int32_t E,
                                                  const int32_t* __restrict__ colpref,
                                                  const int32_t* __restrict__ offs,
                                                  int32_t* __restrict__ perm,
                                                  int32_t* __restrict__ perm_out) {
  __shared__ int32_t hist[2 * kMaxWindows];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int nbits = W > 1 ? 32 - __clz(W - 1) : 0;
  for (int i = threadIdx.x; i < nw * W; i += blockDim.x) hist[i] = 0;
  __syncthreads();
  const int64_t span = E / nw;
  const int64_t wbeg = (int64_t)blockIdx.x * E + wv * span;
  const int64_t wend = wbeg + span < n ? wbeg + span : n;
  int32_t* h = hist + wv * W;
  const uint64_t lt = lanemask_lt(lane);

  // per-wave histogram, rows in order
  for (int64_t g = wbeg; g < wend; g += 64) {
    const int64_t i = g + lane;
    const bool in = i < wend;
    const int32_t id = in ? ids[i] : -1;
    const bool valid = in && (uint32_t)id < (uint32_t)W;
    const uint64_t m = match_key(id, valid, nbits);
    if (valid && (m & lt) == 0) h[id] += __popcll(m);
  }
  __syncthreads();
  // base of every wave inside the block, per window
  for (int w = threadIdx.x; w < W; w += blockDim.x) {
    int32_t run = 0;
    for (int v = 0; v < nw; ++v) {
      const int32_t t = hist[v * W + w];
      hist[v * W + w] = run;
      run += t;
    }
  }
  __syncthreads();
  const int32_t* cp = colpref + (size_t)blockIdx.x * (W + 1);
  for (int64_t g = wbeg; g < wend; g += 64) {
    const int64_t i = g + lane;
    const bool in = i < wend;
    const int32_t id = in ? ids[i] : -1;
    const bool valid = in && (uint32_t)id < (uint32_t)W;
    const uint64_t m = match_key(id, valid, nbits);
    if (valid) {
      const int32_t base = h[id];
      const int32_t pos = offs[id] + cp[id] + base + __popcll(m & lt);
      if ((uint32_t)pos < (uint32_t)n) {
        perm[pos] = (int32_t)i;
        if (perm_out) perm_out[pos] = (int32_t)i;
      }
      if ((m & lt) == 0) h[id] = base + __popcll(m);
    }
  }
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
  int32_t* counts = reinterpret_cast<int32_t*>(base + lay.counts);
  const int csr = ids == nullptr;
  if (!csr && lay.n_blocks > 0) {
    hipLaunchKernelGGL(k_count, dim3(lay.n_blocks), dim3(256), 0, stream, ids, n, W,
                       lay.block_elems, counts);
  }
  hipLaunchKernelGGL(k_plan, dim3(1), dim3(kPlanThreads), 0, stream, csr, counts,
                     csr ? 0 : lay.n_blocks, W, n, L, offsets_io, invalid_out, hdr, offs, chunks);
  if (!csr && lay.n_blocks > 0) {
    const int nw = W <= kMaxWindows / 2 ? 4 : 2;
    hipLaunchKernelGGL(k_scatter, dim3(lay.n_blocks), dim3(64 * nw), 0, stream, ids, n, W,
                       lay.block_elems, counts, offs, perm, perm_out);
  }
  return hipGetLastError();
}

}  // namespace sla

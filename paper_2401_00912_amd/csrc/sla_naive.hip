// The naive scatter-based SLA forward that Sec. 3.2 ("Hardware Efficient
// Implementation") sets against the chunk-wise kernel, kept as a GPU comparator
// (its time and memory against the chunk-wise path reproduce the shape of
// Fig. 4): every voxel's kv matrix phi(k)^T v (d x d, plus phi(k) as column d
// for the normaliser) is cached in HBM, the cached matrices are summed within
// each window, and each voxel's output is read off its window's sum.
//
//   k_naive_kv      one workgroup per 4 voxels: kv[row][h][e][c] = phi(k_e) v_c
//                   for c < d, phi(k_e) for c = d (fp32; N x H x d x (d + 1)
//                   floats, written as float4);
//   k_naive_window  one workgroup per (window, head): the segmented sum of the
//                   window's cached matrices (each wave a strided subset of the
//                   rows, four in flight per lane, the partial sums then added in
//                   wave order), then o = phi(q) S / (phi(q) . z) for the window's
//                   rows.
//
// The arithmetic is plain fp32 on the vector units: this is the baseline the
// chunk-wise path is measured against, not a second production path.
#include "sla_common.h"

namespace sla {

constexpr int kNaiveThreads = 256;

template <typename T>
__device__ __forceinline__ float load_f32(const T* p);
template <>
__device__ __forceinline__ float load_f32<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load_f32<_Float16>(const _Float16* p) { return (float)*p; }
template <>
__device__ __forceinline__ float load_f32<bf16_t>(const bf16_t* p) {
  return __uint_as_float((uint32_t)p->bits << 16);
}

template <typename T>
__device__ __forceinline__ void store_f32(T* p, float x);
template <>
__device__ __forceinline__ void store_f32<float>(float* p, float x) { *p = x; }
template <>
__device__ __forceinline__ void store_f32<_Float16>(_Float16* p, float x) { *p = (_Float16)x; }
template <>
__device__ __forceinline__ void store_f32<bf16_t>(bf16_t* p, float x) {
  p->bits = __builtin_bit_cast(unsigned short, (__bf16)x);
}

__device__ __forceinline__ float naive_phi(float x) { return x > 0.f ? x + 1.f : expf(x); }

// kv of kNaiveRows voxels (rows blockIdx.x * kNaiveRows ...), all heads: phi(k)
// and v of the rows in LDS, then the cached matrices written as float4.
constexpr int kNaiveRows = 4;

template <typename T, int D>
__global__ __launch_bounds__(kNaiveThreads) void k_naive_kv(const T* __restrict__ k,
                                                           const T* __restrict__ v, int32_t n,
                                                           int32_t H, float* __restrict__ kv) {
  constexpr int DC = D + 1;
  extern __shared__ float s_kv[];   // [kNaiveRows][H][D] phi(k), then v
  const int32_t r0 = blockIdx.x * kNaiveRows;
  const int32_t nr = min(kNaiveRows, n - r0);
  if (nr <= 0) return;
  const size_t rs = (size_t)H * D;
  float* s_fk = s_kv;
  float* s_v = s_kv + kNaiveRows * rs;
  for (int j = threadIdx.x; j < nr * (int)rs; j += kNaiveThreads) {
    s_fk[j] = naive_phi(load_f32<T>(k + (size_t)r0 * rs + j));
    s_v[j] = load_f32<T>(v + (size_t)r0 * rs + j);
  }
  __syncthreads();
  // rows r0 .. r0 + nr - 1 are contiguous in kv: nr * H * D * DC floats
  const int64_t total4 = (int64_t)nr * (int64_t)rs * DC / 4;
  float4* out = reinterpret_cast<float4*>(kv + (size_t)r0 * rs * DC);
  for (int64_t j4 = threadIdx.x; j4 < total4; j4 += kNaiveThreads) {
    float x[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t j = 4 * j4 + u;
      const int64_t he = j / DC;            // (row, head, e) flattened
      const int c = (int)(j - he * DC);
      const float fk = s_fk[he];
      x[u] = c < D ? fk * s_v[he / D * D + c] : fk;
    }
    out[j4] = make_float4(x[0], x[1], x[2], x[3]);
  }
}

// Window sum and outputs for (window blockIdx.x, head blockIdx.y).
template <typename T, int D>
__global__ __launch_bounds__(kNaiveThreads) void k_naive_window(
    const PlanHeader* __restrict__ hdr, const int32_t* __restrict__ perm,
    const int32_t* __restrict__ offs, const T* __restrict__ q, const float* __restrict__ kv,
    T* __restrict__ o, int32_t n, int32_t W, int32_t H) {
  constexpr int DC = D + 1;
  constexpr int NV = D * DC / 4;          // float4 per cached matrix (D * DC is a multiple of 4)
  constexpr int RG = kNaiveThreads / 64;  // row groups: a wave per group of rows
  __shared__ float4 s_part[RG][NV];
  __shared__ float s_state[D * DC];
  __shared__ float s_phi[kNaiveThreads / D][D];
  if (hdr->magic != kPlanMagic || hdr->n != n || hdr->num_windows != W) return;
  const int32_t w = blockIdx.x, h = blockIdx.y;
  const int32_t* pm = hdr->csr ? nullptr : perm;
  const int32_t rb = max(0, min(offs[w], n)), re = max(rb, min(offs[w + 1], n));
  if (rb == re) return;
  // segmented sum of the cached matrices: wave g sums rows rb + g, rb + g + RG, ...
  // (four rows in flight per lane), then the RG partial sums are added in order
  const int lane = threadIdx.x & 63, g = threadIdx.x >> 6;
  for (int v4 = lane; v4 < NV; v4 += 64) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    int32_t p = rb + g;
    for (; p + 3 * RG < re; p += 4 * RG) {
      float4 x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int32_t row = pm ? pm[p + u * RG] : p + u * RG;
        x[u] = (uint32_t)row < (uint32_t)n
                   ? reinterpret_cast<const float4*>(kv + ((size_t)row * H + h) * D * DC)[v4]
                   : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        acc.x += x[u].x; acc.y += x[u].y; acc.z += x[u].z; acc.w += x[u].w;
      }
    }
    for (; p < re; p += RG) {
      const int32_t row = pm ? pm[p] : p;
      if ((uint32_t)row < (uint32_t)n) {
        const float4 x = reinterpret_cast<const float4*>(kv + ((size_t)row * H + h) * D * DC)[v4];
        acc.x += x.x; acc.y += x.y; acc.z += x.z; acc.w += x.w;
      }
    }
    s_part[g][v4] = acc;
  }
  __syncthreads();
  for (int j = threadIdx.x; j < D * DC; j += kNaiveThreads) {
    float acc = 0.f;
#pragma unroll
    for (int gg = 0; gg < RG; ++gg) acc += reinterpret_cast<const float*>(s_part[gg])[j];
    s_state[j] = acc;
  }
  __syncthreads();
  // outputs: kNaiveThreads / D rows at a time, one thread per (row, column c)
  const size_t rs = (size_t)H * D;
  const int c = threadIdx.x % D, slot = threadIdx.x / D;
  for (int32_t p0 = rb; p0 < re; p0 += kNaiveThreads / D) {
    const int32_t p = p0 + slot;
    const int32_t row = p < re ? (pm ? pm[p] : p) : -1;
    const bool ok = (uint32_t)row < (uint32_t)n;
    s_phi[slot][c] = ok ? naive_phi(load_f32<T>(q + (size_t)row * rs + h * D + c)) : 0.f;
    __syncthreads();
    float num = 0.f, den = 0.f;
#pragma unroll 8
    for (int e = 0; e < D; ++e) {
      const float fq = s_phi[slot][e];
      num += fq * s_state[e * DC + c];
      den += fq * s_state[e * DC + D];
    }
    if (ok) store_f32<T>(o + (size_t)row * rs + h * D + c, num / den);
    __syncthreads();
  }
}

template <typename T, int D>
static hipError_t naive_impl(const void* plan, int32_t n, int32_t W, int32_t H, const void* q,
                             const void* k, const void* v, void* o, void* workspace,
                             hipStream_t stream) {
  const PlanLayout lay = plan_layout(n, W);
  const char* base = static_cast<const char*>(plan);
  float* kv = static_cast<float*>(workspace);
  const size_t lds = 2 * (size_t)kNaiveRows * H * D * sizeof(float);
  if (lds > 64 * 1024) return hipErrorInvalidValue;   // heads * head_dim <= 2048
  hipLaunchKernelGGL((k_naive_kv<T, D>), dim3((n + kNaiveRows - 1) / kNaiveRows),
                     dim3(kNaiveThreads), lds, stream, static_cast<const T*>(k),
                     static_cast<const T*>(v), n, H, kv);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_naive_window<T, D>), dim3(W, H), dim3(kNaiveThreads), 0, stream,
                     reinterpret_cast<const PlanHeader*>(base + lay.header),
                     reinterpret_cast<const int32_t*>(base + lay.perm),
                     reinterpret_cast<const int32_t*>(base + lay.offsets),
                     static_cast<const T*>(q), kv, static_cast<T*>(o), n, W, H);
  return hipGetLastError();
}

size_t naive_workspace_bytes(int64_t n, int32_t H, int32_t d) {
  return (size_t)n * (size_t)H * (size_t)d * (size_t)(d + 1) * sizeof(float);
}

// dtype: 0 f32, 1 f16, 2 bf16
hipError_t launch_forward_scatter(const void* plan, int32_t n, int32_t W, int dtype, int32_t H,
                                  int32_t d, const void* q, const void* k, const void* v,
                                  void* o, void* workspace, hipStream_t stream) {
  if (d == 32) {
    if (dtype == 0) return naive_impl<float, 32>(plan, n, W, H, q, k, v, o, workspace, stream);
    if (dtype == 1) return naive_impl<_Float16, 32>(plan, n, W, H, q, k, v, o, workspace, stream);
    return naive_impl<bf16_t, 32>(plan, n, W, H, q, k, v, o, workspace, stream);
  }
  if (dtype == 0) return naive_impl<float, 16>(plan, n, W, H, q, k, v, o, workspace, stream);
  if (dtype == 1) return naive_impl<_Float16, 16>(plan, n, W, H, q, k, v, o, workspace, stream);
  return naive_impl<bf16_t, 16>(plan, n, W, H, q, k, v, o, workspace, stream);
}

}  // namespace sla

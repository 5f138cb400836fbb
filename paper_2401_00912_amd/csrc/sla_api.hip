// C ABI of libsla: argument validation (synchronous, before any launch) and
// dispatch to the kernels.  No allocation, no synchronisation.
#include "sla.h"
#include "sla_common.h"

#define SLA_EXPORT extern "C" __attribute__((visibility("default")))

namespace sla {
hipError_t launch_build(const int32_t* ids, int32_t n, int32_t W, int32_t L, int32_t* perm_out,
                        int32_t* offsets_io, int32_t* invalid_out, void* plan, hipStream_t stream);
hipError_t launch_forward(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                          int phi, float eps, const void* q, const void* k, const void* v, void* o,
                          hipStream_t stream);
hipError_t launch_backward(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                           int phi, float eps, const void* q, const void* k, const void* v,
                           const void* dout, void* dq, void* dk, void* dv, hipStream_t stream);
hipError_t launch_forward_projected(const void* plan, int32_t n, int32_t W, int dtype, int32_t H,
                                    int32_t d, int phi, float eps, const void* x, const void* wqkv,
                                    const void* bqkv, const void* wo, const void* bo, void* o,
                                    void* y, void* qkv, hipStream_t stream);
hipError_t launch_backward_projected(const void* plan, int32_t n, int32_t W, int dtype, int32_t H,
                                     int32_t d, int phi, float eps, const void* x, const void* wqkv,
                                     const void* bqkv, const void* wo, const void* o, const void* dy,
                                     void* dx, float* dw_qkv, float* db_qkv, float* dw_o,
                                     float* db_o, const void* qkv, void* workspace,
                                     hipStream_t stream);
size_t projected_backward_workspace_bytes(int64_t n, int32_t C);
size_t naive_workspace_bytes(int64_t n, int32_t H, int32_t d);
hipError_t launch_cwi_build_map(const int32_t* coords, int32_t n, int32_t gx, int32_t gy,
                                int32_t gz, int32_t* map, int32_t* conflicts, hipStream_t stream);
hipError_t launch_cwi_forward(const int32_t* map, int32_t gx, int32_t gy, int32_t gz,
                              const int32_t* coords, int32_t n, const int32_t* order, int dtype,
                              int32_t channels, int32_t kx, int32_t ky, const void* x,
                              const void* w_x, const void* w_y, const void* w_3, void* y,
                              hipStream_t stream);
size_t cwi_backward_workspace_bytes(int32_t n, int32_t channels, int32_t kx, int32_t ky, int esize);
hipError_t launch_cwi_backward(const int32_t* map, int32_t gx, int32_t gy, int32_t gz,
                               const int32_t* coords, int32_t n, const int32_t* order, int dtype,
                               int32_t channels, int32_t kx, int32_t ky, const void* x,
                               const void* w_x, const void* w_y, const void* w_3, const void* dy,
                               void* dx, void* dw_x, void* dw_y, void* dw_3, void* workspace,
                               hipStream_t stream);
hipError_t launch_forward_scatter(const void* plan, int32_t n, int32_t W, int dtype, int32_t H,
                                  int32_t d, const void* q, const void* k, const void* v,
                                  void* o, void* workspace, hipStream_t stream);
hipError_t launch_forward_xca(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                              const float* tau, const void* q, const void* k, const void* v, void* o,
                              hipStream_t stream);
hipError_t launch_backward_xca(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                               const float* tau, const void* q, const void* k, const void* v,
                               const void* dout, void* dq, void* dk, void* dv, float* dtau, float* part,
                               hipStream_t stream);
hipError_t launch_backward_xca_noalloc(const void* plan, int32_t n, int32_t W, int dtype, int32_t H, int32_t d,
                                       const float* tau, const void* q, const void* k, const void* v,
                                       const void* dout, void* dq, void* dk, void* dv, float* dtau,
                                       hipStream_t stream);
}  // namespace sla

namespace {

constexpr int32_t kAbiVersion = 8;

// cells of a CWI grid, or -1 when a side is not positive or the grid has more
// than INT32_MAX cells
int64_t cwi_cells(int32_t gx, int32_t gy, int32_t gz) {
  if (gx < 1 || gy < 1 || gz < 1) return -1;
  const int64_t cells = (int64_t)gx * gy * gz;
  return cells > INT32_MAX ? -1 : cells;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

bool sizes_ok(int64_t n, int32_t W) { return n >= 0 && n < INT32_MAX && W >= 1; }

sla_status_t check_tensor_args(int64_t n, int32_t W, int dtype, int32_t heads, int32_t head_dim,
                               const void* plan, size_t plan_bytes) {
  if (!sizes_ok(n, W) || heads < 1) return SLA_E_ARG;
  if (heads > 65535) return SLA_E_UNSUPPORTED;
  if (dtype < 0 || dtype > 2) return SLA_E_ARG;
  if (head_dim != 16 && head_dim != 32) return SLA_E_UNSUPPORTED;
  if (W > sla::kMaxWindows) return SLA_E_UNSUPPORTED;
  if ((int64_t)heads * head_dim > (1 << 20)) return SLA_E_UNSUPPORTED;
  // the kernels address rows with 32-bit byte offsets: every tensor < 4 GiB
  const int64_t esize = dtype == 0 ? 4 : 2;
  if (n > 0 && (int64_t)n * heads * head_dim * esize > (int64_t)UINT32_MAX) return SLA_E_UNSUPPORTED;
  if (plan == nullptr || !aligned(plan, 256)) return SLA_E_ARG;
  if (plan_bytes < sla::plan_layout(n, W).total) return SLA_E_WORKSPACE;
  return SLA_OK;
}

sla_status_t hip_status(hipError_t e) { return e == hipSuccess ? SLA_OK : SLA_E_HIP; }

// feature map known, eps finite and >= 0 (NaN fails both comparisons)
bool variant_ok(int phi, float eps) {
  return (phi == SLA_PHI_ELU1 || phi == SLA_PHI_RELU) && eps >= 0.f && eps <= 3.0e38f;
}

sla_status_t forward_impl(const void* plan, size_t plan_bytes, int64_t n, int32_t num_windows,
                          sla_dtype_t dtype, int32_t heads, int32_t head_dim, int phi, float eps,
                          const void* q, const void* k, const void* v, void* o,
                          sla_stream_t stream) {
  const sla_status_t st = check_tensor_args(n, num_windows, (int)dtype, heads, head_dim, plan, plan_bytes);
  if (st != SLA_OK) return st;
  if (!variant_ok(phi, eps)) return SLA_E_ARG;
  if (n == 0) return SLA_OK;
  if (!q || !k || !v || !o) return SLA_E_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16)) return SLA_E_ARG;
  return hip_status(sla::launch_forward(plan, (int32_t)n, num_windows, (int)dtype, heads, head_dim,
                                        phi, eps, q, k, v, o, static_cast<hipStream_t>(stream)));
}

sla_status_t backward_impl(const void* plan, size_t plan_bytes, int64_t n, int32_t num_windows,
                           sla_dtype_t dtype, int32_t heads, int32_t head_dim, int phi, float eps,
                           const void* q, const void* k, const void* v, const void* dout,
                           void* dq, void* dk, void* dv, sla_stream_t stream) {
  const sla_status_t st = check_tensor_args(n, num_windows, (int)dtype, heads, head_dim, plan, plan_bytes);
  if (st != SLA_OK) return st;
  if (!variant_ok(phi, eps)) return SLA_E_ARG;
  if (n == 0) return SLA_OK;
  if (!q || !k || !v || !dout || !dq || !dk || !dv) return SLA_E_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(dout, 16) ||
      !aligned(dq, 16) || !aligned(dk, 16) || !aligned(dv, 16))
    return SLA_E_ARG;
  return hip_status(sla::launch_backward(plan, (int32_t)n, num_windows, (int)dtype, heads,
                                         head_dim, phi, eps, q, k, v, dout, dq, dk, dv,
                                         static_cast<hipStream_t>(stream)));
}

}  // namespace

SLA_EXPORT int32_t sla_abi_version(void) { return kAbiVersion; }

SLA_EXPORT const char* sla_status_string(sla_status_t s) {
  switch (s) {
    case SLA_OK: return "SLA_OK";
    case SLA_E_ARG: return "SLA_E_ARG: invalid argument (null/misaligned pointer, bad size or enum)";
    case SLA_E_UNSUPPORTED: return "SLA_E_UNSUPPORTED: head_dim must be 16 or 32; too many windows";
    case SLA_E_WORKSPACE: return "SLA_E_WORKSPACE: plan buffer smaller than sla_plan_bytes()";
    case SLA_E_HIP: return "SLA_E_HIP: HIP runtime or launch failure";
  }
  return "SLA: unknown status";
}

SLA_EXPORT int32_t sla_max_windows(void) { return sla::kMaxWindows; }

SLA_EXPORT int32_t sla_default_chunk_rows(void) { return sla::kDefaultChunkRows; }

SLA_EXPORT size_t sla_plan_bytes(int64_t n, int32_t num_windows) {
  if (!sizes_ok(n, num_windows) || num_windows > sla::kMaxWindows) return 0;
  return sla::plan_layout(n, num_windows).total;
}

SLA_EXPORT sla_status_t sla_plan_layout(int64_t n, int32_t num_windows, sla_plan_layout_t* out) {
  if (out == nullptr || !sizes_ok(n, num_windows)) return SLA_E_ARG;
  if (num_windows > sla::kMaxWindows) return SLA_E_UNSUPPORTED;
  const sla::PlanLayout L = sla::plan_layout(n, num_windows);
  out->header = L.header;
  out->perm = L.perm;
  out->offsets = L.offsets;
  out->chunks = L.chunks;
  out->longs = L.longs;
  out->total = L.total;
  out->max_chunks = L.max_chunks;
  out->max_long = L.max_long;
  return SLA_OK;
}

SLA_EXPORT sla_status_t sla_build_segments(const int32_t* window_ids, int64_t n,
                                           int32_t num_windows, int32_t chunk_rows,
                                           int32_t* perm_out, int32_t* offsets,
                                           int32_t* invalid_count, void* plan, size_t plan_bytes,
                                           sla_stream_t stream) {
  if (!sizes_ok(n, num_windows)) return SLA_E_ARG;
  if (num_windows > sla::kMaxWindows) return SLA_E_UNSUPPORTED;
  if (chunk_rows == 0) chunk_rows = sla::kDefaultChunkRows;
  if (chunk_rows < sla::kMinChunkRows || chunk_rows > sla::kMaxChunkRows || (chunk_rows & 1))
    return SLA_E_ARG;
  if (plan == nullptr || !aligned(plan, 256)) return SLA_E_ARG;
  if (plan_bytes < sla::plan_layout(n, num_windows).total) return SLA_E_WORKSPACE;
  if (window_ids == nullptr) {
    if (offsets == nullptr || perm_out != nullptr) return SLA_E_ARG;  // CSR input mode
  } else if (n > 0 && !aligned(window_ids, 4)) {
    return SLA_E_ARG;
  } else if (n > sla::kBuilderMaxRows) {
    return SLA_E_UNSUPPORTED;
  }
  return hip_status(sla::launch_build(window_ids,
                                      (int32_t)n, num_windows, chunk_rows, perm_out, offsets,
                                      invalid_count, plan, static_cast<hipStream_t>(stream)));
}

SLA_EXPORT sla_status_t sla_forward(const void* plan, size_t plan_bytes, int64_t n,
                                    int32_t num_windows, sla_dtype_t dtype, int32_t heads,
                                    int32_t head_dim, const void* q, const void* k, const void* v,
                                    void* o, sla_stream_t stream) {
  return forward_impl(plan, plan_bytes, n, num_windows, dtype, heads, head_dim, SLA_PHI_ELU1, 0.f,
                      q, k, v, o, stream);
}

SLA_EXPORT sla_status_t sla_backward(const void* plan, size_t plan_bytes, int64_t n,
                                     int32_t num_windows, sla_dtype_t dtype, int32_t heads,
                                     int32_t head_dim, const void* q, const void* k,
                                     const void* v, const void* dout, void* dq, void* dk, void* dv,
                                     sla_stream_t stream) {
  return backward_impl(plan, plan_bytes, n, num_windows, dtype, heads, head_dim, SLA_PHI_ELU1,
                       0.f, q, k, v, dout, dq, dk, dv, stream);
}

SLA_EXPORT sla_status_t sla_forward_ex(const void* plan, size_t plan_bytes, int64_t n,
                                       int32_t num_windows, sla_dtype_t dtype, int32_t heads,
                                       int32_t head_dim, sla_feature_map_t feature_map, float eps,
                                       const void* q, const void* k, const void* v, void* o,
                                       sla_stream_t stream) {
  return forward_impl(plan, plan_bytes, n, num_windows, dtype, heads, head_dim, (int)feature_map,
                      eps, q, k, v, o, stream);
}

SLA_EXPORT sla_status_t sla_backward_ex(const void* plan, size_t plan_bytes, int64_t n,
                                        int32_t num_windows, sla_dtype_t dtype, int32_t heads,
                                        int32_t head_dim, sla_feature_map_t feature_map,
                                        float eps, const void* q, const void* k, const void* v,
                                        const void* dout, void* dq, void* dk, void* dv,
                                        sla_stream_t stream) {
  return backward_impl(plan, plan_bytes, n, num_windows, dtype, heads, head_dim, (int)feature_map,
                       eps, q, k, v, dout, dq, dk, dv, stream);
}

SLA_EXPORT sla_status_t sla_forward_projected(const void* plan, size_t plan_bytes, int64_t n,
                                              int32_t num_windows, sla_dtype_t dtype,
                                              int32_t heads, int32_t head_dim,
                                              sla_feature_map_t feature_map, float eps,
                                              const void* x, const void* w_qkv, const void* b_qkv,
                                              const void* w_o, const void* b_o, void* o, void* y,
                                              void* qkv_out, sla_stream_t stream) {
  const sla_status_t st = check_tensor_args(n, num_windows, (int)dtype, heads, head_dim, plan, plan_bytes);
  if (st != SLA_OK) return st;
  if (!variant_ok((int)feature_map, eps)) return SLA_E_ARG;
  if (dtype != SLA_F16 && dtype != SLA_BF16) return SLA_E_UNSUPPORTED;
  const int64_t C = (int64_t)heads * head_dim;
  if (C != 64 && C != 128 && C != 256) return SLA_E_UNSUPPORTED;
  if (n == 0) return SLA_OK;
  if (!x || !w_qkv || !w_o || !o || !y) return SLA_E_ARG;
  if (!aligned(x, 16) || !aligned(w_qkv, 16) || !aligned(w_o, 16) || !aligned(o, 16) ||
      !aligned(y, 16) || !aligned(b_qkv, 2) || !aligned(b_o, 2) || !aligned(qkv_out, 16))
    return SLA_E_ARG;
  return hip_status(sla::launch_forward_projected(plan, (int32_t)n, num_windows, (int)dtype, heads,
                                                  head_dim, (int)feature_map, eps, x, w_qkv, b_qkv,
                                                  w_o, b_o, o, y, qkv_out,
                                                  static_cast<hipStream_t>(stream)));
}

SLA_EXPORT size_t sla_backward_projected_workspace_bytes(int64_t n, int32_t heads, int32_t head_dim) {
  if (n < 0 || n >= INT32_MAX || heads < 1 || (head_dim != 16 && head_dim != 32)) return 0;
  const int64_t C = (int64_t)heads * head_dim;
  if (C != 64 && C != 128 && C != 256) return 0;
  return sla::projected_backward_workspace_bytes(n, (int32_t)C);
}

SLA_EXPORT sla_status_t sla_backward_projected(const void* plan, size_t plan_bytes, int64_t n,
                                               int32_t num_windows, sla_dtype_t dtype,
                                               int32_t heads, int32_t head_dim,
                                               sla_feature_map_t feature_map, float eps,
                                               const void* x, const void* w_qkv, const void* b_qkv,
                                               const void* w_o, const void* o, const void* dy,
                                               void* dx, float* dw_qkv, float* db_qkv, float* dw_o,
                                               float* db_o, const void* qkv, void* workspace,
                                               size_t workspace_bytes, sla_stream_t stream) {
  const sla_status_t st = check_tensor_args(n, num_windows, (int)dtype, heads, head_dim, plan, plan_bytes);
  if (st != SLA_OK) return st;
  if (!variant_ok((int)feature_map, eps)) return SLA_E_ARG;
  if (dtype != SLA_F16 && dtype != SLA_BF16) return SLA_E_UNSUPPORTED;
  const int64_t C = (int64_t)heads * head_dim;
  if (C != 64 && C != 128 && C != 256) return SLA_E_UNSUPPORTED;
  if (!x || !w_qkv || !w_o || !o || !dy || !dx || !dw_qkv || !dw_o) return SLA_E_ARG;
  if (!aligned(x, 16) || !aligned(w_qkv, 16) || !aligned(w_o, 16) || !aligned(o, 16) ||
      !aligned(dy, 16) || !aligned(dx, 16) || !aligned(b_qkv, 2) || !aligned(dw_qkv, 4) ||
      !aligned(dw_o, 4) || !aligned(db_qkv, 4) || !aligned(db_o, 4) || !aligned(qkv, 16))
    return SLA_E_ARG;
  if (workspace == nullptr || !aligned(workspace, 256)) return SLA_E_ARG;
  if (workspace_bytes < sla::projected_backward_workspace_bytes(n, (int32_t)C)) return SLA_E_WORKSPACE;
  return hip_status(sla::launch_backward_projected(plan, (int32_t)n, num_windows, (int)dtype, heads,
                                                   head_dim, (int)feature_map, eps, x, w_qkv, b_qkv,
                                                   w_o, o, dy, dx, dw_qkv, db_qkv, dw_o, db_o, qkv,
                                                   workspace, static_cast<hipStream_t>(stream)));
}

SLA_EXPORT size_t sla_scatter_workspace_bytes(int64_t n, int32_t heads, int32_t head_dim) {
  if (n < 0 || heads < 1 || (head_dim != 16 && head_dim != 32)) return 0;
  return sla::naive_workspace_bytes(n, heads, head_dim);
}

SLA_EXPORT sla_status_t sla_forward_scatter(const void* plan, size_t plan_bytes, int64_t n,
                                            int32_t num_windows, sla_dtype_t dtype, int32_t heads,
                                            int32_t head_dim, const void* q, const void* k,
                                            const void* v, void* o, void* workspace,
                                            size_t workspace_bytes, sla_stream_t stream) {
  const sla_status_t st = check_tensor_args(n, num_windows, (int)dtype, heads, head_dim, plan, plan_bytes);
  if (st != SLA_OK) return st;
  if ((int64_t)heads * head_dim > 2048) return SLA_E_UNSUPPORTED;   // the kv kernel's LDS rows
  if (n == 0) return SLA_OK;
  if (!q || !k || !v || !o || !workspace) return SLA_E_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16) ||
      !aligned(workspace, 16))
    return SLA_E_ARG;
  if (workspace_bytes < sla::naive_workspace_bytes(n, heads, head_dim)) return SLA_E_WORKSPACE;
  return hip_status(sla::launch_forward_scatter(plan, (int32_t)n, num_windows, (int)dtype, heads,
                                                head_dim, q, k, v, o, workspace,
                                                static_cast<hipStream_t>(stream)));
}

SLA_EXPORT sla_status_t sla_forward_xca(const void* plan, size_t plan_bytes, int64_t n,
                                        int32_t num_windows, sla_dtype_t dtype, int32_t heads,
                                        int32_t head_dim, const float* tau, const void* q,
                                        const void* k, const void* v, void* o, sla_stream_t stream) {
  const sla_status_t st = check_tensor_args(n, num_windows, (int)dtype, heads, head_dim, plan, plan_bytes);
  if (st != SLA_OK) return st;
  // one 256-thread workgroup per (window, head), windows padded to a multiple of
  // 8: the launch's work-items must fit 32 bits
  if (((int64_t)num_windows + 7) / 8 * 8 * heads * 256 > (int64_t)UINT32_MAX) return SLA_E_UNSUPPORTED;
  if (n == 0) return SLA_OK;
  if (!tau || !q || !k || !v || !o) return SLA_E_ARG;
  if (!aligned(tau, 4) || !aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16))
    return SLA_E_ARG;
  return hip_status(sla::launch_forward_xca(plan, (int32_t)n, num_windows, (int)dtype, heads, head_dim,
                                            tau, q, k, v, o, static_cast<hipStream_t>(stream)));
}

SLA_EXPORT size_t sla_xca_backward_workspace_bytes(int32_t num_windows, int32_t heads) {
  if (num_windows < 1 || heads < 1) return 0;
  return (size_t)num_windows * (size_t)heads * sizeof(float);
}

SLA_EXPORT sla_status_t sla_backward_xca(const void* plan, size_t plan_bytes, int64_t n,
                                         int32_t num_windows, sla_dtype_t dtype, int32_t heads,
                                         int32_t head_dim, const float* tau, const void* q,
                                         const void* k, const void* v, const void* dout, void* dq,
                                         void* dk, void* dv, float* dtau, void* workspace,
                                         size_t workspace_bytes, sla_stream_t stream) {
  const sla_status_t st = check_tensor_args(n, num_windows, (int)dtype, heads, head_dim, plan, plan_bytes);
  if (st != SLA_OK) return st;
  if (((int64_t)num_windows + 7) / 8 * 8 * heads * 256 > (int64_t)UINT32_MAX) return SLA_E_UNSUPPORTED;
  if (!tau || !dtau || !workspace || !aligned(tau, 4) || !aligned(dtau, 4) || !aligned(workspace, 4))
    return SLA_E_ARG;
  if (workspace_bytes < sla_xca_backward_workspace_bytes(num_windows, heads)) return SLA_E_WORKSPACE;
  if (n > 0) {
    if (!q || !k || !v || !dout || !dq || !dk || !dv) return SLA_E_ARG;
    for (const void* p : {q, k, v, dout, static_cast<const void*>(dq), static_cast<const void*>(dk),
                          static_cast<const void*>(dv)})
      if (!aligned(p, 16)) return SLA_E_ARG;
  }
  return hip_status(sla::launch_backward_xca(plan, (int32_t)n, num_windows, (int)dtype, heads, head_dim,
                                             tau, q, k, v, dout, dq, dk, dv, dtau,
                                             static_cast<float*>(workspace),
                                             static_cast<hipStream_t>(stream)));
}

SLA_EXPORT sla_status_t sla_backward_xca_noalloc(const void* plan, size_t plan_bytes, int64_t n,
                                                 int32_t num_windows, sla_dtype_t dtype, int32_t heads,
                                                 int32_t head_dim, const float* tau, const void* q,
                                                 const void* k, const void* v, const void* dout, void* dq,
                                                 void* dk, void* dv, float* dtau, sla_stream_t stream) {
  const sla_status_t st = check_tensor_args(n, num_windows, (int)dtype, heads, head_dim, plan, plan_bytes);
  if (st != SLA_OK) return st;
  if (((int64_t)num_windows + 7) / 8 * 8 * heads * 256 > (int64_t)UINT32_MAX) return SLA_E_UNSUPPORTED;
  if ((int64_t)num_windows * heads > (int64_t)SLA_XCA_SCRATCH_FLOATS) return SLA_E_UNSUPPORTED;
  if (!tau || !dtau || !aligned(tau, 4) || !aligned(dtau, 4)) return SLA_E_ARG;
  if (n > 0) {
    if (!q || !k || !v || !dout || !dq || !dk || !dv) return SLA_E_ARG;
    for (const void* p : {q, k, v, dout, static_cast<const void*>(dq), static_cast<const void*>(dk),
                          static_cast<const void*>(dv)})
      if (!aligned(p, 16)) return SLA_E_ARG;
  }
  return hip_status(sla::launch_backward_xca_noalloc(plan, (int32_t)n, num_windows, (int)dtype, heads,
                                                     head_dim, tau, q, k, v, dout, dq, dk, dv, dtau,
                                                     static_cast<hipStream_t>(stream)));
}

SLA_EXPORT size_t sla_cwi_map_bytes(int32_t gx, int32_t gy, int32_t gz) {
  const int64_t cells = cwi_cells(gx, gy, gz);
  return cells < 0 ? 0 : (size_t)cells * sizeof(int32_t);
}

SLA_EXPORT sla_status_t sla_cwi_build_map(const int32_t* coords, int64_t n, int32_t gx,
                                          int32_t gy, int32_t gz, int32_t* map,
                                          size_t map_bytes, int32_t* conflicts,
                                          sla_stream_t stream) {
  const int64_t cells = cwi_cells(gx, gy, gz);
  if (cells < 0 || n < 0 || n >= INT32_MAX) return SLA_E_ARG;
  if (map == nullptr || !aligned(map, 4)) return SLA_E_ARG;
  if (map_bytes < (size_t)cells * sizeof(int32_t)) return SLA_E_WORKSPACE;
  if (n > 0 && (coords == nullptr || !aligned(coords, 4))) return SLA_E_ARG;
  if (conflicts && !aligned(conflicts, 4)) return SLA_E_ARG;
  return hip_status(sla::launch_cwi_build_map(coords, (int32_t)n, gx, gy, gz, map, conflicts,
                                              static_cast<hipStream_t>(stream)));
}

// shapes of sla_cwi_forward / sla_cwi_backward (see sla.h)
static sla_status_t cwi_shape_ok(int64_t n, int dtype, int32_t channels, int32_t kx, int32_t ky) {
  if (n < 0 || n >= INT32_MAX) return SLA_E_ARG;
  if (dtype < 0 || dtype > 2) return SLA_E_ARG;
  const int64_t esize = dtype == 0 ? 4 : 2;
  if (channels < 4 || channels % 4) return SLA_E_UNSUPPORTED;
  const int64_t piece_bytes = (int64_t)(channels / 4) * esize;
  if (piece_bytes % 16) return SLA_E_UNSUPPORTED;
  const int64_t pq = piece_bytes / 16;
  if (pq > 64 || (64 % pq)) return SLA_E_UNSUPPORTED;
  if (kx < 1 || ky < 1 || kx > 63 || ky > 63 || !(kx & 1) || !(ky & 1)) return SLA_E_UNSUPPORTED;
  if (n > 0 && (int64_t)n * channels * esize > (int64_t)UINT32_MAX * 4) return SLA_E_UNSUPPORTED;
  return SLA_OK;
}

SLA_EXPORT sla_status_t sla_cwi_forward(const int32_t* map, int32_t gx, int32_t gy, int32_t gz,
                                        const int32_t* coords, int64_t n, const int32_t* order,
                                        sla_dtype_t dtype, int32_t channels, int32_t taps_x,
                                        int32_t taps_y, const void* x, const void* w_x,
                                        const void* w_y, const void* w_3, void* y,
                                        sla_stream_t stream) {
  if (cwi_cells(gx, gy, gz) < 0) return SLA_E_ARG;
  // four branches of c channels; a branch row is a whole number of 16-byte
  // pieces, and that number divides 64 (one wave holds whole rows)
  const sla_status_t st = cwi_shape_ok(n, (int)dtype, channels, taps_x, taps_y);
  if (st != SLA_OK) return st;
  if (n == 0) return SLA_OK;
  if (!map || !coords || !x || !w_x || !w_y || !w_3 || !y) return SLA_E_ARG;
  if (!aligned(map, 4) || !aligned(coords, 4) || (order && !aligned(order, 4)) || !aligned(x, 16) ||
      !aligned(w_x, 16) || !aligned(w_y, 16) || !aligned(w_3, 16) || !aligned(y, 16))
    return SLA_E_ARG;
  return hip_status(sla::launch_cwi_forward(map, gx, gy, gz, coords, (int32_t)n, order, (int)dtype,
                                            channels, taps_x, taps_y, x, w_x, w_y, w_3, y,
                                            static_cast<hipStream_t>(stream)));
}

SLA_EXPORT size_t sla_cwi_backward_workspace_bytes(int64_t n, sla_dtype_t dtype, int32_t channels,
                                                   int32_t taps_x, int32_t taps_y) {
  if (cwi_shape_ok(n, (int)dtype, channels, taps_x, taps_y) != SLA_OK) return 0;
  return sla::cwi_backward_workspace_bytes((int32_t)n, channels, taps_x, taps_y,
                                           dtype == SLA_F32 ? 4 : 2);
}

SLA_EXPORT sla_status_t sla_cwi_backward(const int32_t* map, int32_t gx, int32_t gy, int32_t gz,
                                         const int32_t* coords, int64_t n, const int32_t* order,
                                         sla_dtype_t dtype, int32_t channels, int32_t taps_x,
                                         int32_t taps_y, const void* x, const void* w_x,
                                         const void* w_y, const void* w_3, const void* dy, void* dx,
                                         void* dw_x, void* dw_y, void* dw_3, void* workspace,
                                         size_t workspace_bytes, sla_stream_t stream) {
  if (cwi_cells(gx, gy, gz) < 0) return SLA_E_ARG;
  const sla_status_t st = cwi_shape_ok(n, (int)dtype, channels, taps_x, taps_y);
  if (st != SLA_OK) return st;
  if (!dw_x || !dw_y || !dw_3 || !w_x || !w_y || !w_3) return SLA_E_ARG;
  if (!aligned(w_x, 16) || !aligned(w_y, 16) || !aligned(w_3, 16) || !aligned(dw_x, 4) ||
      !aligned(dw_y, 4) || !aligned(dw_3, 4))
    return SLA_E_ARG;
  if (!workspace || !aligned(workspace, 16)) return SLA_E_ARG;
  if (workspace_bytes < sla::cwi_backward_workspace_bytes((int32_t)n, channels, taps_x, taps_y,
                                                          dtype == SLA_F32 ? 4 : 2))
    return SLA_E_WORKSPACE;
  if (n > 0) {
    if (!map || !coords || !x || !dy || !dx) return SLA_E_ARG;
    if (!aligned(map, 4) || !aligned(coords, 4) || (order && !aligned(order, 4)) || !aligned(x, 16) ||
        !aligned(dy, 16) || !aligned(dx, 16))
      return SLA_E_ARG;
  }
  // n = 0 still writes zero kernel gradients
  return hip_status(sla::launch_cwi_backward(map, gx, gy, gz, coords, (int32_t)n, order, (int)dtype,
                                             channels, taps_x, taps_y, x, w_x, w_y, w_3, dy, dx, dw_x,
                                             dw_y, dw_3, workspace, static_cast<hipStream_t>(stream)));
}

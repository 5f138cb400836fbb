/*
 * sla.h -- C ABI of libsla, Scattered Linear Attention (SLA) on AMD Instinct
 * MI355X (gfx950).
 *
 * SLA ("ScatterFormer", He et al., arXiv 2401.00912, Sec. 3.2) applies linear
 * attention separately inside every window of a voxel scene, with all voxels of
 * the scene held in ONE flattened matrix ordered by window (Sec. 3.2, Fig. 3(a)):
 *
 *   Eq. (2)  SLA(Q, K, V) = Concat_j LA(Q^j, K^j, V^j) over the non-empty windows;
 *   Eq. (3)  for window w and each head, with phi the kernel feature map,
 *              S_w = sum_{i in w} phi(k_i)^T v_i ,   z_w = sum_{i in w} phi(k_i),
 *              o_i = phi(q_i) S_w / (phi(q_i) . z_w)     for every i in w.
 *
 * Readings of the paper fixed by this library:
 *   phi(x) = elu(x) + 1 (x + 1 for x > 0, exp(x) otherwise): the feature map of
 *     the linear-attention paper Sec. 3.2 cites for LA;
 *   attention is non-causal inside a window (Eq. (3) sums over the whole window);
 *   no 1/sqrt(d) scale and no epsilon in the denominator (Eq. (3) has neither;
 *     sla_forward_ex / sla_backward_ex add an epsilon and a ReLU feature map);
 *   heads are independent; channel c of a row is head c / head_dim.
 *
 * Conventions shared by every entry point:
 *   - Every pointer argument except `plan_bytes`-style sizes is a DEVICE pointer
 *     on the current HIP device.  The caller owns all memory; the library never
 *     allocates, frees or synchronises.
 *   - `stream` is a hipStream_t (NULL = the null stream).  All device work is
 *     enqueued on it, in order; calls return before the work finishes.
 *   - Argument errors that the host can see are reported synchronously, before
 *     anything is enqueued, by the returned status.  A failed launch gives
 *     SLA_E_HIP.
 *   - Rows: q, k, v, o, dout, dq, dk, dv are row-major contiguous
 *     [n, heads, head_dim] arrays of `dtype`, in the caller's ORIGINAL row order
 *     (the library gathers and scatters through the plan's permutation), with
 *     16-byte aligned base pointers.  head_dim must be 16 or 32.
 *   - Re-entrant: sla_forward / sla_backward only read the plan, so calls on
 *     different streams may share one plan; they must not share outputs, and a
 *     plan must not be rebuilt while a call that reads it is in flight.
 */
#ifndef SLA_H
#define SLA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SLA_OK = 0,
  SLA_E_ARG = 1,          /* null / misaligned pointer, negative size, bad enum  */
  SLA_E_UNSUPPORTED = 2,  /* head_dim not 16/32, too many windows                */
  SLA_E_WORKSPACE = 3,    /* plan buffer smaller than sla_plan_bytes()           */
  SLA_E_HIP = 4           /* a HIP launch or runtime call failed                 */
} sla_status_t;

typedef enum { SLA_F32 = 0, SLA_F16 = 1, SLA_BF16 = 2 } sla_dtype_t;

/* Kernel feature map phi of Eq. (3) (sla_forward_ex / sla_backward_ex). */
typedef enum {
  SLA_PHI_ELU1 = 0,  /* elu(x) + 1: x + 1 for x > 0, exp(x) otherwise (the default)     */
  SLA_PHI_RELU = 1   /* max(x, 0), derivative 1 for x > 0 and 0 otherwise (phi'(0) = 0) */
} sla_feature_map_t;

typedef void* sla_stream_t; /* hipStream_t */

/* Version of this interface (bumped on any incompatible change). */
int32_t sla_abi_version(void);

/* Static description of a status code; never NULL. */
const char* sla_status_string(sla_status_t status);

/* Largest window-slot count supported (window tables live in on-chip memory). */
int32_t sla_max_windows(void);

/* Chunk length L used when sla_build_segments() is given chunk_rows = 0. */
int32_t sla_default_chunk_rows(void);

/*
 * Bytes of the plan buffer for n rows and num_windows window slots.
 * The plan holds the window-sorted view of the rows (Sec. 3.2: the flattened,
 * window-ordered matrix), its CSR window offsets, the chunk table (Fig. 3(a); the
 * Fig. 5 caption's "offsets generation" = start row of each chunk), the table of
 * long windows and the builder's scratch.  Returns 0 for invalid sizes.
 */
size_t sla_plan_bytes(int64_t n, int32_t num_windows);

/* Byte offsets of the plan's sections (for inspection by tests and tools). */
typedef struct {
  size_t header;     /* 64-byte header, see below                          */
  size_t perm;       /* int32[n]: sorted position -> original row           */
  size_t offsets;    /* int32[num_windows + 1]: CSR over sorted positions   */
  size_t chunks;     /* int32[max_chunks][4]: row_begin, row_end,
                        win_begin, win_end                                  */
  size_t longs;      /* int32[max_long][4]: window, row_begin, row_end, 0   */
  size_t total;      /* == sla_plan_bytes(n, num_windows)                   */
  int32_t max_chunks;
  int32_t max_long;
} sla_plan_layout_t;
/* Plan header (int32 fields in order): magic, n, num_windows, chunk_rows,
 * n_chunks, csr (1 = rows were already window-sorted), invalid, n_long, n_long4
 * (long windows of more than 2 chunk_rows rows, listed first in the long table),
 * then padding. */

sla_status_t sla_plan_layout(int64_t n, int32_t num_windows, sla_plan_layout_t* out /* host */);

/*
 * Segment builder: the "sort by window, flatten, partition into chunks" steps of
 * Sec. 3.2 / Fig. 3(a) and the chunk offsets of the Fig. 5 caption.
 *
 * Mode A, window_ids != NULL (int32[n], one window slot per row, rows in any
 * order): stable sort of the rows by window id.  Writes into the plan
 *   perm[p]     original row at sorted position p; rows of one window keep their
 *               original relative order, so the result is unique;
 *   offsets[w]  first sorted position of window w (empty windows allowed);
 * and the chunk table.  If perm_out / offsets are not NULL they receive copies
 * (int32[n] / int32[num_windows + 1]).  Rows whose id is outside
 * [0, num_windows) are counted and left out of every window (their output rows
 * are then never written); perm lists them after every window, at sorted
 * positions offsets[num_windows] .. n - 1 in row order, so perm is a permutation
 * of all n rows.
 *
 * Mode B, window_ids == NULL: rows are already window-sorted and `offsets`
 * (int32[num_windows + 1], device) is an INPUT: offsets[0] = 0, non-decreasing,
 * offsets[num_windows] = n.  perm_out must be NULL (the permutation is the
 * identity).  Violations are counted; the plan is then clamped into range so no
 * kernel reads out of bounds, but outputs are undefined.
 *
 * Work tables (both modes), with L = chunk_rows (0 = default 64; else even,
 * 32..64) and pages of L/2 rows: a window of more than L rows is "long" and is
 * listed in the long-window table (the forward and backward split its rows among
 * four wavefronts of one workgroup if it has more than 2L rows, else among two,
 * which add their partial window states; four-way windows are listed first,
 * then two-way ones, each group in sequence order); a window of L/2 + 1 .. L
 * rows is a chunk of its own; shorter windows are packed into one chunk while
 * they start in the same page, so a packed chunk never splits a window and never
 * exceeds L - 1 rows.  Empty windows get nothing.  The chunk table is in
 * sequence order.
 *
 * invalid_count (device int32, may be NULL) receives the number of out-of-range
 * ids (mode A) or offset violations (mode B).  The plan must be at least
 * sla_plan_bytes(n, num_windows) bytes, 256-byte aligned.  Valid for num_windows
 * in [1, sla_max_windows()]; mode A also needs n <= 2^26 (SLA_E_UNSUPPORTED
 * beyond).
 *
 * Plan scratch: mode A accumulates window totals in a region of the plan that
 * must read zero when the build starts, and every build leaves it zero again.
 * So zero-fill a plan buffer once after allocating it (hipMemset), before its
 * first build; after that it can be rebuilt any number of times, for any n and
 * num_windows it is large enough for.  Builds into one plan buffer must not
 * overlap in time.
 */
sla_status_t sla_build_segments(const int32_t* window_ids, int64_t n, int32_t num_windows,
                                int32_t chunk_rows, int32_t* perm_out, int32_t* offsets,
                                int32_t* invalid_count, void* plan, size_t plan_bytes,
                                sla_stream_t stream);

/*
 * Forward, Eq. (2)-(3): o = SLA(q, k, v).  `plan` must have been built by
 * sla_build_segments() with the same n and num_windows (the kernels check the
 * plan header and write nothing otherwise); it is only read.  Every row that
 * belongs to a window is written; a window of one row returns its own value (to rounding).
 * Arithmetic: phi and the normaliser in fp32; the two contractions phi(K)^T V and
 * phi(Q) S on the matrix cores with fp32 accumulation, their operands rounded to
 * `dtype` (fp32 stays fp32).
 */
sla_status_t sla_forward(const void* plan, size_t plan_bytes, int64_t n, int32_t num_windows,
                         sla_dtype_t dtype, int32_t heads, int32_t head_dim, const void* q,
                         const void* k, const void* v, void* o, sla_stream_t stream);

/*
 * Backward of Eq. (3) (the paper trains the model but does not write the
 * gradients; they follow from Eq. (3) by the chain rule): given dout = dL/do,
 * writes dq, dk, dv for every row that belongs to a window.  Window states are
 * recomputed from k and v; the state gradients are accumulated in fp32.
 */
sla_status_t sla_backward(const void* plan, size_t plan_bytes, int64_t n, int32_t num_windows,
                          sla_dtype_t dtype, int32_t heads, int32_t head_dim, const void* q,
                          const void* k, const void* v, const void* dout, void* dq, void* dk,
                          void* dv, sla_stream_t stream);

/*
 * Linear-attention variants (Sec. 4.5 / Tab. 7 trains the model with other
 * linear-attention designs; its "Efficient Attn" row is ReLU-kernel linear
 * attention, whose normaliser carries a small epsilon): forward and backward as
 * above with the feature map chosen by `feature_map` and eps added to the
 * normaliser,
 *     o_i = phi(q_i) S / (phi(q_i) . z + eps).
 * sla_forward / sla_backward are these calls with SLA_PHI_ELU1 and eps = 0.
 * eps must be finite and >= 0 and feature_map one of the enum values, else
 * SLA_E_ARG.  With eps = 0 a zero normaliser (under ReLU: a query row with no
 * positive entry, or one whose positive features are all absent from the
 * window's keys) gives 0/0 = NaN in that row's output, and in the backward NaN
 * in the gradients of that row and of its window's keys and values; with
 * eps > 0 such a row's output is 0.  phi and eps are applied in fp32; the
 * operands of the matrix cores are as in sla_forward.
 */
sla_status_t sla_forward_ex(const void* plan, size_t plan_bytes, int64_t n, int32_t num_windows,
                            sla_dtype_t dtype, int32_t heads, int32_t head_dim,
                            sla_feature_map_t feature_map, float eps, const void* q,
                            const void* k, const void* v, void* o, sla_stream_t stream);

sla_status_t sla_backward_ex(const void* plan, size_t plan_bytes, int64_t n, int32_t num_windows,
                             sla_dtype_t dtype, int32_t heads, int32_t head_dim,
                             sla_feature_map_t feature_map, float eps, const void* q,
                             const void* k, const void* v, const void* dout, void* dq, void* dk,
                             void* dv, sla_stream_t stream);

/*
 * Projection layer, SLA and output projection in two launches, q, k, v kept in
 * registers.  Sec. 3.2 maps every voxel of the scene to Q, K and V with one
 * shared projection layer before the attention; the attention block projects
 * its output back.  Read as linear layers with bias in the [out, in] weight
 * layout:
 *     [q | k | v] = x W_qkv^T + b_qkv,   o = SLA(q, k, v)  (as sla_forward_ex),
 *     y = o W_o^T + b_o.
 *   x      [n, C] features in original row order, C = heads * head_dim;
 *   w_qkv  [3C, C]: rows 0..C-1 give q, C..2C-1 k, 2C..3C-1 v (channel c of q,
 *          k, v is head c / head_dim as everywhere);
 *   b_qkv  [3C] or NULL (no bias);  w_o [C, C];  b_o [C] or NULL;
 *   o      [n, C] output: SLA's output before the output projection;
 *   y      [n, C] output;
 *   qkv_out [3][n][C] output or NULL: q, k, v (three consecutive [n, C]
 *          tensors, q first) as projected, for sla_backward_projected to use
 *          instead of recomputing them; rows in no window are not written.
 *          It costs the forward the stores of 3 n C values.
 * All in `dtype`, which must be SLA_F16 or SLA_BF16; C must be 64, 128 or 256
 * (else SLA_E_UNSUPPORTED).  x, w_qkv, w_o, o, y, qkv_out 16-byte aligned.  Rows
 * in no window get neither o nor y.  The projections run on the matrix cores
 * with fp32 accumulation; q, k, v are rounded to `dtype` (as if stored) before
 * the attention, o is rounded before the output projection.
 */
sla_status_t sla_forward_projected(const void* plan, size_t plan_bytes, int64_t n,
                                   int32_t num_windows, sla_dtype_t dtype, int32_t heads,
                                   int32_t head_dim, sla_feature_map_t feature_map, float eps,
                                   const void* x, const void* w_qkv, const void* b_qkv,
                                   const void* w_o, const void* b_o, void* o, void* y,
                                   void* qkv_out, sla_stream_t stream);

/*
 * Backward of sla_forward_projected: the projection layer and output projection
 * of Sec. 3.2 are trained with the attention; their gradients follow from the
 * forward by the chain rule.  For dy = dL/dy [n, C] over the rows in windows:
 *     do = dy W_o,   dW_o = dy^T o,   db_o = sum over rows of dy,
 *     dq, dk, dv = SLA backward of do (as sla_backward_ex, same feature map, eps),
 *     dx = [dq | dk | dv] W_qkv,   dW_qkv = [dq | dk | dv]^T x,
 *     db_qkv = sum over rows of [dq | dk | dv].
 *   x, w_qkv, b_qkv, w_o: the forward's inputs (layouts as there; b_o takes no
 *          part); o [n, C]: the forward's o output; dy [n, C]; all in `dtype`.
 *   dx     [n, C] in `dtype`: every row is written, zero for rows in no window.
 *   dw_qkv [3C, C], dw_o [C, C] (fp32, required); db_qkv [3C], db_o [C] (fp32,
 *          may be NULL).  Rows in no window take no part in these sums.
 *   qkv    [3][n][C] or NULL: the forward's qkv_out, for the same x, weights and
 *          plan; given, q, k, v are read from it instead of being recomputed.
 *   workspace: device, 256-byte aligned, at least
 *          sla_backward_projected_workspace_bytes(n, heads, head_dim) bytes
 *          (else SLA_E_WORKSPACE): the recomputed q, k, v, do, dq, dk, dv, the
 *          weights as rows and the weight-gradient partials.
 * Without qkv, q, k, v are recomputed from x (rounded to `dtype`, as in the
 * forward; the same products in the same order, so the same values); do, dq,
 * dk, dv are rounded to `dtype` as stored; all products accumulate in fp32 on the
 * matrix cores.  The sums over rows run over the plan's sorted rows in groups
 * whose partials are added in group order: the results are deterministic.
 * Same dtype, C and alignment rules as sla_forward_projected; dy, dx and qkv
 * 16-byte aligned, the fp32 outputs 4-byte aligned.
 */
size_t sla_backward_projected_workspace_bytes(int64_t n, int32_t heads, int32_t head_dim);

sla_status_t sla_backward_projected(const void* plan, size_t plan_bytes, int64_t n,
                                    int32_t num_windows, sla_dtype_t dtype, int32_t heads,
                                    int32_t head_dim, sla_feature_map_t feature_map, float eps,
                                    const void* x, const void* w_qkv, const void* b_qkv,
                                    const void* w_o, const void* o, const void* dy, void* dx,
                                    float* dw_qkv, float* db_qkv, float* dw_o, float* db_o,
                                    const void* qkv, void* workspace, size_t workspace_bytes,
                                    sla_stream_t stream);

/*
 * Cross-window interaction (Sec. 3.3, Eq. (4)-(7)), the module that follows SLA
 * in every block: the channels of each voxel, 4c of them, go through four
 * branches whose outputs are concatenated,
 *   [0, c)    depthwise convolution along x with taps_x taps (w_x [taps_x, c]),
 *   [c, 2c)   depthwise convolution along y with taps_y taps (w_y [taps_y, c]),
 *   [2c, 3c)  depthwise 3 x 3 x 3 convolution (w_3 [27, c], tap
 *             (dx + 1) + 3 (dy + 1) + 9 (dz + 1)),
 *   [3c, 4c)  identity;
 * the paper's axis kernels have window size + 1 taps (13 for 12 x 12 windows).
 * Read as submanifold convolutions on the voxel set: outputs only at the voxels,
 * a tap whose cell holds no voxel contributes zero, each tap a centred
 * cross-correlation tap (y[p] = sum_t w[t] x[p + t - (taps - 1) / 2]), no bias.
 *
 * Voxels are cells (x, y, z) of a gx x gy x gz grid (pillars: gz = 1), given as
 * int32 coords [n, 3].  Neighbours are found through a dense cell -> row table
 * (`map`, int32 [gx gy gz], caller-owned, sla_cwi_map_bytes() bytes), built per
 * scene by sla_cwi_build_map: -1 in empty cells.  Coordinates must be unique and
 * inside the grid; rows that are not are counted in *conflicts (device int32,
 * may be NULL; a cell claimed twice keeps the larger row) and their outputs, and
 * those of their neighbours, are undefined.
 *
 * sla_cwi_forward: x, y [n, channels] in original row order, `dtype` throughout
 * (fp32 accumulation), channels = 4c with c * (element size) a multiple of 16
 * bytes and 64 divisible by c * (element size) / 16 (fp16/bf16: channels 32 x 2^k
 * up to 2048; fp32: 16 x 2^k up to 1024); taps odd, 1..63; else
 * SLA_E_UNSUPPORTED.  `order` (int32
 * [n], may be NULL = 0..n-1) is the order in which rows are visited on grids
 * more than one cell deep, e.g. the SLA plan's permutation: rows of one window
 * together keep the neighbours in cache.  Pillar grids (gz = 1) are processed
 * in tiles of cells and ignore it; there a row the table does not hold gets
 * zero branch outputs.  Results do not depend on `order`.  x, y and the
 * weights 16-byte aligned.
 */
size_t sla_cwi_map_bytes(int32_t gx, int32_t gy, int32_t gz);

sla_status_t sla_cwi_build_map(const int32_t* coords, int64_t n, int32_t gx, int32_t gy,
                               int32_t gz, int32_t* map, size_t map_bytes, int32_t* conflicts,
                               sla_stream_t stream);

sla_status_t sla_cwi_forward(const int32_t* map, int32_t gx, int32_t gy, int32_t gz,
                             const int32_t* coords, int64_t n, const int32_t* order,
                             sla_dtype_t dtype, int32_t channels, int32_t taps_x, int32_t taps_y,
                             const void* x, const void* w_x, const void* w_y, const void* w_3,
                             void* y, sla_stream_t stream);

/*
 * Backward of sla_cwi_forward (the chain rule; the paper does not write it out):
 * given dy = dL/dy [n, channels], writes dx [n, channels] and the kernel
 * gradients dw_x [taps_x, c], dw_y [taps_y, c], dw_3 [27, c], all in `dtype`
 * (rounded from fp32 sums).  Same table, coordinates, order and shapes as the
 * forward (the table must hold every voxel: no conflicts).  `workspace`
 * (caller-owned, 16-byte aligned, at least sla_cwi_backward_workspace_bytes(),
 * which returns 0 for an unsupported shape) receives fp32 partial sums of the
 * kernel gradients, one set per block of rows (at most 512 sets); they are
 * added in a fixed order, so the result is deterministic.  With n = 0 the
 * kernel gradients are zero.
 */
size_t sla_cwi_backward_workspace_bytes(int64_t n, sla_dtype_t dtype, int32_t channels,
                                        int32_t taps_x, int32_t taps_y);

sla_status_t sla_cwi_backward(const int32_t* map, int32_t gx, int32_t gy, int32_t gz,
                              const int32_t* coords, int64_t n, const int32_t* order,
                              sla_dtype_t dtype, int32_t channels, int32_t taps_x, int32_t taps_y,
                              const void* x, const void* w_x, const void* w_y, const void* w_3,
                              const void* dy, void* dx, void* dw_x, void* dw_y, void* dw_3,
                              void* workspace, size_t workspace_bytes, sla_stream_t stream);

/*
 * The naive scatter-based forward that Sec. 3.2 ("Hardware Efficient
 * Implementation") contrasts with the chunk-wise kernel, kept as a comparator
 * for Fig. 4's time-and-memory comparison: the kv matrix phi(k)^T v of every
 * voxel (with phi(k) as one more column) is cached in `workspace` (fp32,
 * N x heads x head_dim x (head_dim + 1) floats, caller-owned, 16-byte aligned,
 * at least sla_scatter_workspace_bytes() bytes), the cached matrices are summed
 * per window in sorted-row order, and o = phi(q) S / (phi(q) . z) as in
 * sla_forward.  Same plan, layouts, dtypes and errors as sla_forward, plus
 * SLA_E_WORKSPACE for a short workspace and SLA_E_UNSUPPORTED for heads x
 * head_dim above 2048.  All arithmetic is fp32 on the vector
 * units.  It exists to be measured against sla_forward, not as a fast path.
 */
size_t sla_scatter_workspace_bytes(int64_t n, int32_t heads, int32_t head_dim);

sla_status_t sla_forward_scatter(const void* plan, size_t plan_bytes, int64_t n,
                                 int32_t num_windows, sla_dtype_t dtype, int32_t heads,
                                 int32_t head_dim, const void* q, const void* k, const void* v,
                                 void* o, void* workspace, size_t workspace_bytes,
                                 sla_stream_t stream);

/*
 * The XCA design of the linear-attention ablation (Sec. 4.5, Tab. 7), which
 * cites cross-covariance attention (XCiT), applied inside every window of the
 * plan.  For window w and head h, with the window's q and k columns normalised
 * over the window's rows (qhat[:, e] = q[:, e] / max(|q[:, e]|_2, 1e-12), k
 * likewise):
 *     A[e][c] = softmax over c of  tau[h] qhat[:, e] . khat[:, c]   (d x d),
 *     o_i[e]  = sum_c A[e][c] v_i[c]                               for i in w.
 * tau: device float [heads], the per-head temperatures (4-byte aligned).  Same
 * plan, row layouts, dtypes and errors as sla_forward (rows in no window are
 * not written), plus SLA_E_UNSUPPORTED when num_windows x heads x 256 exceeds
 * 2^32 - 1 (one 256-thread workgroup per window and head, windows padded
 * to a multiple of 8).  fp32 arithmetic on
 * the vector units; outputs rounded to `dtype`.  Its backward is sla_backward_xca.
 */
sla_status_t sla_forward_xca(const void* plan, size_t plan_bytes, int64_t n, int32_t num_windows,
                             sla_dtype_t dtype, int32_t heads, int32_t head_dim, const float* tau,
                             const void* q, const void* k, const void* v, void* o,
                             sla_stream_t stream);

/*
 * Backward of sla_forward_xca (the chain rule; the paper does not write it):
 * given dout, writes dq, dk, dv for every row in a window and dtau[heads] (fp32,
 * device, 4-byte aligned), the gradient of the temperatures summed over the
 * windows.  With N = qhat^T khat and A the softmax of tau N, per window and head:
 *     dv_i = A^T dout_i,   dA = sum_i dout_i v_i^T,
 *     dG = A * (dA - rowsum(A * dA)),   dtau += sum dG * N,
 *     dqhat = tau khat dG^T, dkhat = tau qhat dG, and through the
 *     normalisation dq[:, e] = (dqhat[:, e] - qhat[:, e] (qhat[:, e] . dqhat[:, e])) / |q[:, e]|
 *     (a column whose norm took the 1e-12 floor gets dqhat[:, e] / 1e-12), dk alike.
 * `workspace` (caller-owned, 4-byte aligned, at least
 * sla_xca_backward_workspace_bytes(num_windows, heads) bytes) receives one fp32
 * partial of dtau per (window, head); the partials are then added in window
 * order, so dtau is deterministic.  Errors as sla_forward_xca, plus
 * SLA_E_WORKSPACE for a short workspace.  With n = 0, dtau is zero.
 */
size_t sla_xca_backward_workspace_bytes(int32_t num_windows, int32_t heads);

sla_status_t sla_backward_xca(const void* plan, size_t plan_bytes, int64_t n, int32_t num_windows,
                              sla_dtype_t dtype, int32_t heads, int32_t head_dim, const float* tau,
                              const void* q, const void* k, const void* v, const void* dout,
                              void* dq, void* dk, void* dv, float* dtau, void* workspace,
                              size_t workspace_bytes, sla_stream_t stream);

/*
 * sla_backward_xca without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  The per-(window, head) partials of dtau go to
 * a buffer of SLA_XCA_SCRATCH_FLOATS floats (1 MiB) that the library keeps in
 * static device memory, one copy on every GPU it runs on, for the life of the
 * process; the first call on a device looks its address up (no allocation, no
 * hipMalloc / hipFree, no allocating library call).  Every partial is rewritten by
 * every call, so the buffer needs no clearing and keeps the last call's values.
 * num_windows * heads must not exceed SLA_XCA_SCRATCH_FLOATS (SLA_E_UNSUPPORTED
 * otherwise, returned before anything is enqueued).  All calls on one GPU share
 * the buffer: calls that may overlap on one GPU (different streams with no order
 * between them) race and must not be issued.  Outputs equal those of
 * sla_backward_xca bit for bit; other arguments and errors as sla_backward_xca.
 */
#define SLA_XCA_SCRATCH_FLOATS 262144

sla_status_t sla_backward_xca_noalloc(const void* plan, size_t plan_bytes, int64_t n, int32_t num_windows,
                                      sla_dtype_t dtype, int32_t heads, int32_t head_dim, const float* tau,
                                      const void* q, const void* k, const void* v, const void* dout,
                                      void* dq, void* dk, void* dv, float* dtau, sla_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SLA_H */

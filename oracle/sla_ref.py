"""CPU oracle for Scattered Linear Attention (SLA) -- TEST INFRASTRUCTURE ONLY.

This module is the slow, obviously-correct reference that the HIP path is checked
against.  Only the test suite, the smoke check and the benchmark's CPU-baseline leg
may import it; the product path never calls it and has no CPU fallback.

Everything is plain numpy in float64.  Inputs stored in 16-bit formats are widened
exactly (float16 through numpy, bfloat16 bit patterns by a 16-bit shift), so the
oracle sees exactly the values the GPU sees.  There is no chunking, blocking or
reordering beyond what the definitions below state.

Paper: "ScatterFormer: Efficient Voxel Transformer with Scattered Linear Attention"
(He, Li, Zhang, Zhang; arXiv 2401.00912).

What is computed, and the passage it follows
--------------------------------------------
* ``phi`` / ``dphi``: the kernel feature map.  Sec. 3.2 (after Eq. (3)) speaks
  only of a kernel function and attributes LA to the linear-transformer paper it cites,
  whose feature map is elu(x)+1.  Reading taken: phi(x) = x + 1 for x > 0 and
  exp(x) otherwise.  This is ``feature_map="elu1"``, the default.
* ``phi_relu`` / ``dphi_relu``: the variant of Sec. 4.5 / Tab. 7, which trains
  the model with other linear-attention designs; its "Efficient Attn" row cites a
  ReLU-kernel linear attention, whose normaliser carries a small epsilon so that
  rows with phi(q) . z = 0 stay finite.  Reading taken: phi(x) = max(x, 0),
  phi'(x) = 1 for x > 0 and 0 otherwise (phi'(0) = 0).  This is
  ``feature_map="relu"``.
* ``eps``: Eq. (3) has no epsilon, so the default is 0.  For either map an
  ``eps >= 0`` may be added to the normaliser, o_i = phi(q_i) S / (phi(q_i) . z +
  eps); with eps = 0 a zero normaliser gives 0/0 = NaN, which is not masked.
* ``segments_ref``: Sec. 3.2 orders all voxels of the scene by window so that each
  window is one contiguous sub-matrix of a single flattened matrix.  Read as a
  stable sort of rows by window id plus CSR offsets over the window slots; this
  result is unique.
* ``chunk_plan_ref``: Sec. 3.2 / Fig. 3(a) partition the flattened matrix into
  chunks, and the offset-generation step timed in Fig. 5 computes each chunk's
  start row.  The packing rule written here (chunks of whole short
  windows, a table of long windows that are split among workers) is this
  library's own plan rule (the paper does not give one); it is pinned by its
  invariants.
* ``sla_forward_ref``: Eq. (2) (concatenation over the M non-empty windows of
  per-window linear attention) and Eq. (3) (per-window normalised linear
  attention), evaluated in the phi(Q)(phi(K)^T V) order of Sec. 3.1.  Non-causal:
  every row of a window sees the whole window (Eq. (3) sums over all m^j rows).
  No 1/sqrt(d) scale (Eq. (3) has none); epsilon as above.
* ``sla_backward_ref``: the paper trains the model but does not write the
  backward pass; the gradients here are derived from Eq. (3) by the chain rule
  (derivation in the docstring).
* ``sla_projected_forward_ref``: Sec. 3.2 maps every voxel of the scene to Q, K
  and V with one shared projection layer before the attention, and the attention
  block projects its output back.  Reading taken: linear layers with bias in the
  usual [out, in] weight layout, Q = X W_q^T + b_q (likewise K, V) with
  W_qkv = [W_q; W_k; W_v] stacked by rows, and Y = SLA(Q, K, V) W_o^T + b_o, heads
  split from the C channels as in the plain path.
* ``sla_projected_backward_ref``: the gradients of that chain (input, both
  weights, both biases) by the chain rule, for the loss sum(y . dy) over the rows
  that lie in a window (the paper trains the projections but does not write the
  gradients out).
* ``cwi_forward_ref``: the cross-window interaction of Sec. 3.3, Eq. (4)-(7): the
  4c channels split into four quarters, two depthwise convolutions with long 1D
  kernels along the two grid axes (window size + 1 taps), a depthwise 3 x 3 x 3
  convolution and an identity, concatenated.  Read as submanifold (sparse)
  convolutions, as on voxel sets: outputs only at the voxels, a tap whose cell
  holds no voxel contributes zero; each tap a centred cross-correlation tap (the
  deep-learning "convolution"); the first axis branch along x, the second along
  y; no bias (the block's normalisation follows).
* ``xca_forward_ref``: the XCA row of the same ablation (Sec. 4.5, Tab. 7), which
  cites cross-covariance attention (XCiT).  Reading taken: XCiT's operation
  applied inside every window of the flattened matrix, per head: the window's
  q and k columns are L2-normalised over the window's rows (a norm below 1e-12
  counts as 1e-12), A = softmax over c of tau_h qhat[:, e] . khat[:, c] (a d x d
  matrix per window and head; tau_h is the head's learned temperature, an
  input here), and o_i[e] = sum_c A[e, c] v_i[c] for every row i of the window.
  It needs the same per-window d x d reduction over the window's rows as Eq. (3).
* ``xca_backward_ref``: its gradients with respect to q, k, v and the
  temperatures, by the chain rule (the paper trains the model with XCA but does
  not write them out).
* ``cwi_backward_ref``: the gradients of that module with respect to its input
  and its three kernels, by the chain rule (the paper trains the model but does
  not write them out).
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "widen",
    "phi",
    "dphi",
    "phi_relu",
    "dphi_relu",
    "feature_map",
    "FEATURE_MAPS",
    "segments_ref",
    "chunk_plan_ref",
    "sla_forward_ref",
    "sla_backward_ref",
    "sla_projected_forward_ref",
    "cwi_forward_ref",
    "cwi_backward_ref",
    "xca_forward_ref",
    "xca_backward_ref",
]


# --------------------------------------------------------------------------- inputs
def widen(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of a stored input array to float64.

    dtype: "f32" (numpy float32), "f16" (numpy float16) or "bf16" (numpy uint16
    holding bfloat16 bit patterns: the float32 with those 16 high bits).
    """
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    if dtype == "f16":
        return np.asarray(x, dtype=np.float16).astype(np.float64)
    if dtype == "bf16":
        bits = np.asarray(x, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


# --------------------------------------------------------------------- feature map
def phi(x: np.ndarray) -> np.ndarray:
    """elu(x) + 1: x + 1 for x > 0, exp(x) for x <= 0 (Sec. 3.2, reading above)."""
    x = np.asarray(x, dtype=np.float64)
    return np.where(x > 0.0, x + 1.0, np.exp(np.minimum(x, 0.0)))


def dphi(x: np.ndarray) -> np.ndarray:
    """Derivative of phi: 1 for x > 0, exp(x) for x <= 0 (continuous at 0)."""
    x = np.asarray(x, dtype=np.float64)
    return np.where(x > 0.0, 1.0, np.exp(np.minimum(x, 0.0)))


def phi_relu(x: np.ndarray) -> np.ndarray:
    """ReLU feature map of the Tab. 7 variant: max(x, 0)."""
    x = np.asarray(x, dtype=np.float64)
    return np.where(x > 0.0, x, 0.0)


def dphi_relu(x: np.ndarray) -> np.ndarray:
    """Derivative of phi_relu: 1 for x > 0, 0 for x <= 0 (phi'(0) = 0)."""
    x = np.asarray(x, dtype=np.float64)
    return np.where(x > 0.0, 1.0, 0.0)


FEATURE_MAPS = ("elu1", "relu")


def feature_map(name: str):
    """(phi, phi') of a feature map by name: "elu1" (Sec. 3.2) or "relu" (Tab. 7)."""
    if name == "elu1":
        return phi, dphi
    if name == "relu":
        return phi_relu, dphi_relu
    raise ValueError(f"unknown feature map {name!r}")


def _check_eps(eps) -> float:
    eps = float(eps)
    if not (np.isfinite(eps) and eps >= 0.0):
        raise ValueError(f"eps must be finite and >= 0, not {eps!r}")
    return eps


# ------------------------------------------------------------------ segment builder
def segments_ref(ids: np.ndarray, num_windows: int):
    """Stable sort of rows by window id (Sec. 3.2, flattened window-sorted matrix).

    Returns (perm, offsets, invalid_count):
      perm[p]    original row of sorted position p, ties in original row order;
                 rows whose id is outside [0, num_windows) are left out.
      offsets    int64 [num_windows + 1], offsets[w] = first sorted position of
                 window w; empty windows have offsets[w] == offsets[w + 1].
      invalid_count  number of rows with an out-of-range id.
    """
    ids = np.asarray(ids, dtype=np.int64)
    valid = (ids >= 0) & (ids < num_windows)
    rows = np.nonzero(valid)[0]
    order = np.argsort(ids[rows], kind="stable")
    perm = rows[order]
    counts = np.bincount(ids[rows], minlength=num_windows)
    offsets = np.zeros(num_windows + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    return perm.astype(np.int64), offsets, int((~valid).sum())


def chunk_plan_ref(offsets: np.ndarray, chunk_rows: int):
    """This library's work plan over window-sorted rows (plain sequential rule).

    Sec. 3.2 / Fig. 3(a) cut the flattened matrix into pieces that are processed
    independently; the paper fixes no packing rule, so this is the library's own,
    pinned by its invariants.  With L = chunk_rows (even) and pages of P = L // 2
    rows, every non-empty window is exactly one of:
      * long  (more than L rows): listed in the long-window table and nowhere
        else (its rows are split among several workers, whose partial states are
        added before the output is formed): four ways if it has more than 2L
        rows, two ways otherwise;
      * mid   (P < rows <= L): a chunk of its own;
      * short (1..P rows): opens a new chunk unless the previous non-empty window
        is short and starts in the same page (page = start_row // P); otherwise it
        joins that chunk.  A chunk of short windows therefore never splits a
        window and never exceeds 2P - 1 = L - 1 rows.
    A chunk runs from its first window to the next "event" (the next chunk's first
    window or the next long window, whichever comes first; the last one to
    num_windows), so empty windows between are included; its rows are
    [offsets[win_begin], offsets[win_end]).

    Returns (chunks, longs, n_four): chunks int64 [n_chunks, 4] of (row_begin,
    row_end, win_begin, win_end) in sequence order; longs int64 [n_long] window
    ids, the four-way windows first, then the two-way ones, each group in
    sequence order; n_four the number of four-way windows.
    """
    off = [int(x) for x in offsets]
    nw = len(off) - 1
    page = chunk_rows // 2
    events = []  # (window, is_chunk_start) in sequence order
    prev = None  # (start_row, is_short) of the previous non-empty window
    for w in range(nw):
        n = off[w + 1] - off[w]
        if n <= 0:
            continue
        short = n <= page
        if n > chunk_rows:
            events.append((w, False))
        elif not short or prev is None or not prev[1] or (prev[0] // page) != (off[w] // page):
            events.append((w, True))
        prev = (off[w], short)
    chunks, four, two = [], [], []
    for e, (w, is_chunk) in enumerate(events):
        if not is_chunk:
            (four if off[w + 1] - off[w] > 2 * chunk_rows else two).append(w)
            continue
        we = events[e + 1][0] if e + 1 < len(events) else nw
        chunks.append((off[w], off[we], w, we))
    return (np.asarray(chunks, dtype=np.int64).reshape(-1, 4),
            np.asarray(four + two, dtype=np.int64), len(four))


def _window_rows(offsets, perm, w):
    lo, hi = int(offsets[w]), int(offsets[w + 1])
    if perm is None:
        return np.arange(lo, hi)
    return np.asarray(perm[lo:hi], dtype=np.int64)


# -------------------------------------------------------------------------- forward
def sla_forward_ref(q, k, v, offsets, perm=None, feature_map_name="elu1", eps=0.0):
    """SLA forward, Eq. (2)-(3), per window and per head.

    q, k, v: float64 [n, H, d] in original row order.  offsets: [W + 1] CSR over
    sorted positions; perm: sorted position -> original row (None = identity,
    i.e. rows already window-sorted).  For window w with rows R and each head:
        S = sum_{j in R} phi(k_j)^T v_j            (d x d)
        z = sum_{j in R} phi(k_j)                  (d)
        o_i = (phi(q_i) S) / (phi(q_i) . z + eps)  for every i in R.
    phi is chosen by ``feature_map_name`` ("elu1" or "relu"); eps >= 0 (0 in
    Eq. (3)).  Rows that belong to no window are NaN.
    """
    fphi, _ = feature_map(feature_map_name)
    eps = _check_eps(eps)
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    out = np.full(q.shape, np.nan)
    for w in range(len(offsets) - 1):
        rows = _window_rows(offsets, perm, w)
        if rows.size == 0:
            continue
        fq = fphi(q[rows])  # [m, H, d]
        fk = fphi(k[rows])
        vv = v[rows]
        S = np.einsum("mhe,mhc->hec", fk, vv)
        z = fk.sum(axis=0)  # [H, d]
        num = np.einsum("mhe,hec->mhc", fq, S)
        den = np.einsum("mhe,he->mh", fq, z) + eps
        out[rows] = num / den[:, :, None]
    return out


# ------------------------------------------------------------------------- backward
def sla_backward_ref(q, k, v, dout, offsets, perm=None, feature_map_name="elu1", eps=0.0):
    """Gradients of sum(dout * SLA(q, k, v)) with respect to q, k, v.

    Derived from Eq. (3) by the chain rule (the paper does not write them out).
    Per window and head, with fq_i = phi(q_i), fk_j = phi(k_j), S, z as in the
    forward, den_i = fq_i . z + eps and o_i = fq_i S / den_i:
        g_i   = dout_i / den_i                      d loss / d num_i
        s_i   = -(dout_i . o_i) / den_i             d loss / d den_i
        dfq_i = g_i S^T + s_i z                     d loss / d phi(q_i)
        dS    = sum_i fq_i^T g_i ,  dz = sum_i s_i fq_i
        dfk_j = v_j dS^T + dz ,     dv_j = fk_j dS
        dq = dfq * phi'(q) ,        dk = dfk * phi'(k)
    (eps is a constant, so it only enters through den.)  Rows that belong to no
    window are NaN.
    """
    fphi, fdphi = feature_map(feature_map_name)
    eps = _check_eps(eps)
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    dout = np.asarray(dout, dtype=np.float64)
    dq = np.full(q.shape, np.nan)
    dk = np.full(q.shape, np.nan)
    dv = np.full(q.shape, np.nan)
    for w in range(len(offsets) - 1):
        rows = _window_rows(offsets, perm, w)
        if rows.size == 0:
            continue
        qq, kk, vv, do = q[rows], k[rows], v[rows], dout[rows]
        fq, fk = fphi(qq), fphi(kk)
        S = np.einsum("mhe,mhc->hec", fk, vv)
        z = fk.sum(axis=0)
        den = np.einsum("mhe,he->mh", fq, z) + eps
        o = np.einsum("mhe,hec->mhc", fq, S) / den[:, :, None]
        g = do / den[:, :, None]
        s = -np.einsum("mhc,mhc->mh", do, o) / den
        dfq = np.einsum("mhc,hec->mhe", g, S) + s[:, :, None] * z[None, :, :]
        dS = np.einsum("mhe,mhc->hec", fq, g)
        dz = np.einsum("mh,mhe->he", s, fq)
        dfk = np.einsum("mhc,hec->mhe", vv, dS) + dz[None, :, :]
        dv[rows] = np.einsum("mhe,hec->mhc", fk, dS)
        dq[rows] = dfq * fdphi(qq)
        dk[rows] = dfk * fdphi(kk)
    return dq, dk, dv


# ------------------------------------------------------------ projected forward
def sla_projected_forward_ref(x, w_qkv, b_qkv, w_o, b_o, heads, offsets, perm=None,
                              feature_map_name="elu1", eps=0.0):
    """Projection layer, SLA and output projection (Sec. 3.2, reading above).

    x: float64 [n, C] voxel features in original row order, C = heads * d.
    w_qkv: [3C, C] (rows 0..C-1 give Q, C..2C-1 K, 2C..3C-1 V); b_qkv: [3C] or None.
    w_o: [C, C]; b_o: [C] or None.  Returns (o, y): o [n, heads, d] the SLA output
    (NaN for rows in no window) and y [n, C] = o W_o^T + b_o.
    """
    x = np.asarray(x, dtype=np.float64)
    w_qkv = np.asarray(w_qkv, dtype=np.float64)
    w_o = np.asarray(w_o, dtype=np.float64)
    n, C = x.shape
    if C % heads or w_qkv.shape != (3 * C, C) or w_o.shape != (C, C):
        raise ValueError("shapes: x [n, C], w_qkv [3C, C], w_o [C, C], C a multiple of heads")
    d = C // heads
    qkv = x @ w_qkv.T
    if b_qkv is not None:
        qkv = qkv + np.asarray(b_qkv, dtype=np.float64)
    q, k, v = (qkv[:, i * C:(i + 1) * C].reshape(n, heads, d) for i in range(3))
    o = sla_forward_ref(q, k, v, offsets, perm, feature_map_name, eps)
    y = o.reshape(n, C) @ w_o.T
    if b_o is not None:
        y = y + np.asarray(b_o, dtype=np.float64)
    return o, y


def _rows_in_windows(offsets, perm, n):
    """Boolean [n]: rows that belong to a window (the first offsets[-1] sorted
    positions)."""
    offsets = np.asarray(offsets, dtype=np.int64)
    pos = np.arange(int(offsets[-1]))
    rows = pos if perm is None else np.asarray(perm, dtype=np.int64)[pos]
    mask = np.zeros(n, dtype=bool)
    mask[rows] = True
    return mask


def sla_projected_backward_ref(x, w_qkv, b_qkv, w_o, b_o, dy, heads, offsets, perm=None,
                               feature_map_name="elu1", eps=0.0):
    """Gradients of the projected forward (``sla_projected_forward_ref``) by the
    chain rule, for the loss L = sum over rows in windows of y . dy.

    dy: [n, C] gradient of y.  Rows in no window produce no y, so they take no
    part: their dy is ignored and their dx is 0.  Returns float64
    (dx [n, C], dw_qkv [3C, C], db_qkv [3C], dw_o [C, C], db_o [C]):
        do = dy W_o                                  (y = o W_o^T + b_o)
        dW_o = dy^T o,  db_o = sum_rows dy
        dq, dk, dv = SLA backward of do              (``sla_backward_ref``)
        dqkv = [dq | dk | dv]                        ([q | k | v] = x W_qkv^T + b_qkv)
        dx = dqkv W_qkv,  dW_qkv = dqkv^T x,  db_qkv = sum_rows dqkv
    """
    x = np.asarray(x, dtype=np.float64)
    w_qkv = np.asarray(w_qkv, dtype=np.float64)
    w_o = np.asarray(w_o, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    n, C = x.shape
    if C % heads or w_qkv.shape != (3 * C, C) or w_o.shape != (C, C) or dy.shape != (n, C):
        raise ValueError("shapes: x, dy [n, C], w_qkv [3C, C], w_o [C, C], C a multiple of heads")
    d = C // heads
    qkv = x @ w_qkv.T
    if b_qkv is not None:
        qkv = qkv + np.asarray(b_qkv, dtype=np.float64)
    q, k, v = (qkv[:, i * C:(i + 1) * C].reshape(n, heads, d) for i in range(3))
    inside = _rows_in_windows(offsets, perm, n)
    o = sla_forward_ref(q, k, v, offsets, perm, feature_map_name, eps).reshape(n, C)
    o = np.where(inside[:, None], o, 0.0)
    g = np.where(inside[:, None], dy, 0.0)
    dw_o = g.T @ o
    db_o = g.sum(axis=0)
    do = (g @ w_o).reshape(n, heads, d)
    dq, dk, dv = sla_backward_ref(q, k, v, do, offsets, perm, feature_map_name, eps)
    dqkv = np.concatenate([t.reshape(n, C) for t in (dq, dk, dv)], axis=1)
    dqkv = np.where(inside[:, None], dqkv, 0.0)
    dx = dqkv @ w_qkv
    dw_qkv = dqkv.T @ x
    db_qkv = dqkv.sum(axis=0)
    return dx, dw_qkv, db_qkv, dw_o, db_o


# ---------------------------------------------------------- cross-window interaction
def cwi_forward_ref(coords, x, w_x, w_y, w_3, grid):
    """Cross-window interaction, Eq. (4)-(7) of Sec. 3.3, on sparse voxels.

    coords: int [n, 3] cell (x, y, z) of every voxel, unique, inside grid
    (gx, gy, gz).  x: float64 [n, 4c] features.  w_x [K_x, c] and w_y [K_y, c] (K
    odd) the depthwise kernels of the two axis branches, w_3 [27, c] the 3 x 3 x 3
    one, tap (dx + 1) + 3 (dy + 1) + 9 (dz + 1).  Returns [n, 4c]:
        channels [0, c)    sum_t w_x[t] x[cell + (t - (K_x - 1) / 2) e_x]
        channels [c, 2c)   sum_t w_y[t] x[cell + (t - (K_y - 1) / 2) e_y]
        channels [2c, 3c)  sum over the 27 offsets of w_3[tap] x[cell + offset]
        channels [3c, 4c)  x (identity)
    where a cell holding no voxel (or outside the grid) contributes zero.
    """
    coords = np.asarray(coords, dtype=np.int64)
    x = np.asarray(x, dtype=np.float64)
    w_x, w_y, w_3 = (np.asarray(w, dtype=np.float64) for w in (w_x, w_y, w_3))
    n, C = x.shape
    c = C // 4
    gx, gy, gz = (int(g) for g in grid)
    if C % 4 or w_x.shape[1] != c or w_y.shape[1] != c or w_3.shape != (27, c):
        raise ValueError("x [n, 4c], w_x [K_x, c], w_y [K_y, c], w_3 [27, c]")
    if w_x.shape[0] % 2 == 0 or w_y.shape[0] % 2 == 0:
        raise ValueError("axis kernels need an odd number of taps")
    table = np.full(gx * gy * gz, -1, dtype=np.int64)  # cell -> voxel row
    cell = (coords[:, 2] * gy + coords[:, 1]) * gx + coords[:, 0]
    table[cell] = np.arange(n)

    def neighbour(dx, dy, dz):
        """Row of the voxel at cell + (dx, dy, dz), or -1."""
        nx, ny, nz = coords[:, 0] + dx, coords[:, 1] + dy, coords[:, 2] + dz
        inside = (nx >= 0) & (nx < gx) & (ny >= 0) & (ny < gy) & (nz >= 0) & (nz < gz)
        rows = np.full(n, -1, dtype=np.int64)
        rows[inside] = table[(nz[inside] * gy + ny[inside]) * gx + nx[inside]]
        return rows

    out = np.zeros((n, C))
    out[:, 3 * c:] = x[:, 3 * c:]
    for branch, w, axis in ((0, w_x, 0), (1, w_y, 1)):
        half = (w.shape[0] - 1) // 2
        for t in range(w.shape[0]):
            off = [0, 0, 0]
            off[axis] = t - half
            rows = neighbour(*off)
            ok = rows >= 0
            lo = branch * c
            out[ok, lo:lo + c] += w[t] * x[rows[ok], lo:lo + c]
    for dz in (-1, 0, 1):
        for dy in (-1, 0, 1):
            for dx in (-1, 0, 1):
                rows = neighbour(dx, dy, dz)
                ok = rows >= 0
                out[ok, 2 * c:3 * c] += w_3[(dx + 1) + 3 * (dy + 1) + 9 * (dz + 1)] * x[rows[ok], 2 * c:3 * c]
    return out


def _cwi_neighbours(coords, grid):
    """neighbour(dx, dy, dz) -> row of the voxel at cell + offset for every voxel,
    or -1 (a dense cell table, as in cwi_forward_ref)."""
    coords = np.asarray(coords, dtype=np.int64)
    n = coords.shape[0]
    gx, gy, gz = (int(g) for g in grid)
    table = np.full(gx * gy * gz, -1, dtype=np.int64)
    table[(coords[:, 2] * gy + coords[:, 1]) * gx + coords[:, 0]] = np.arange(n)

    def neighbour(dx, dy, dz):
        nx, ny, nz = coords[:, 0] + dx, coords[:, 1] + dy, coords[:, 2] + dz
        inside = (nx >= 0) & (nx < gx) & (ny >= 0) & (ny < gy) & (nz >= 0) & (nz < gz)
        rows = np.full(n, -1, dtype=np.int64)
        rows[inside] = table[(nz[inside] * gy + ny[inside]) * gx + nx[inside]]
        return rows

    return neighbour


def cwi_backward_ref(coords, x, w_x, w_y, w_3, dy, grid):
    """Gradients of sum(dy * cwi_forward_ref(coords, x, w_x, w_y, w_3, grid)).

    Every tap of the forward adds w[t] * x[q] to out[p] for the voxel q at p's
    cell + offset_t.  So, per tap:  dx[q] += w[t] * dy[p]  and
    dw[t] += dy[p] * x[q]  (elementwise over the branch's channels); the identity
    quarter passes dy through.  Returns (dx [n, 4c], dw_x, dw_y, dw_3).
    """
    x = np.asarray(x, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    w_x, w_y, w_3 = (np.asarray(w, dtype=np.float64) for w in (w_x, w_y, w_3))
    n, C = x.shape
    c = C // 4
    neighbour = _cwi_neighbours(coords, grid)
    dx = np.zeros((n, C))
    dx[:, 3 * c:] = dy[:, 3 * c:]
    dws = [np.zeros_like(w_x), np.zeros_like(w_y), np.zeros_like(w_3)]

    def tap(branch, t, w, off):
        rows = neighbour(*off)
        ok = np.nonzero(rows >= 0)[0]
        lo = branch * c
        q = rows[ok]
        np.add.at(dx, (q, slice(lo, lo + c)), w[t] * dy[ok, lo:lo + c])
        dws[branch][t] = (dy[ok, lo:lo + c] * x[q, lo:lo + c]).sum(axis=0)

    for branch, w, axis in ((0, w_x, 0), (1, w_y, 1)):
        half = (w.shape[0] - 1) // 2
        for t in range(w.shape[0]):
            off = [0, 0, 0]
            off[axis] = t - half
            tap(branch, t, w, off)
    for dz in (-1, 0, 1):
        for dy_ in (-1, 0, 1):
            for dx_ in (-1, 0, 1):
                tap(2, (dx_ + 1) + 3 * (dy_ + 1) + 9 * (dz + 1), w_3, (dx_, dy_, dz))
    return dx, dws[0], dws[1], dws[2]


# ---------------------------------------------------------------------- XCA variant
XCA_NORM_FLOOR = 1e-12


def xca_forward_ref(q, k, v, tau, offsets, perm=None):
    """Cross-covariance attention inside every window (Sec. 4.5, Tab. 7, XCA row).

    q, k, v: float64 [n, H, d] in original row order; tau: [H] temperatures;
    offsets / perm as in ``sla_forward_ref``.  For window w with rows R and head h:
        qhat[:, e] = q[R, h, e] / max(||q[R, h, e]||_2, 1e-12)      (likewise khat)
        G[e, c]    = tau[h] * qhat[:, e] . khat[:, c]                (d x d)
        A[e, :]    = softmax(G[e, :])                                 (over c)
        o_i[e]     = sum_c A[e, c] v[i, h, c]                         for i in R.
    Rows that belong to no window are NaN.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    tau = np.asarray(tau, dtype=np.float64)
    n, H, d = q.shape
    if tau.shape != (H,):
        raise ValueError("tau must hold one temperature per head")
    out = np.full(q.shape, np.nan)
    for w in range(len(offsets) - 1):
        rows = _window_rows(offsets, perm, w)
        if rows.size == 0:
            continue
        for h in range(H):
            qw = q[rows, h, :]          # [m, d]
            kw = k[rows, h, :]
            qn = np.maximum(np.sqrt((qw * qw).sum(axis=0)), XCA_NORM_FLOOR)   # [d]
            kn = np.maximum(np.sqrt((kw * kw).sum(axis=0)), XCA_NORM_FLOOR)
            qhat = qw / qn
            khat = kw / kn
            G = tau[h] * (qhat.T @ khat)                 # [d, d]: row e, column c
            G = G - G.max(axis=1, keepdims=True)
            A = np.exp(G)
            A = A / A.sum(axis=1, keepdims=True)
            out[rows, h, :] = v[rows, h, :] @ A.T        # o_i[e] = sum_c A[e, c] v_i[c]
    return out


def xca_backward_ref(q, k, v, tau, dout, offsets, perm=None):
    """Gradients of ``xca_forward_ref``: (dq, dk, dv [n, H, d], dtau [H]).

    Per window and head, with m rows, Qh = q / nq and Kh = k / nk column-wise
    (nq_e = max(|q[:, e]|, 1e-12)), N = Qh^T Kh, G = tau N, A = softmax_c(G),
    o_i = A v_i:
        dv_i   = A^T do_i                     dA = sum_i do_i v_i^T
        dG     = A * (dA - rowsum(A * dA))    (softmax backward, rows e)
        dtau  += sum_{e,c} dG[e, c] N[e, c]   (over every window)
        dQh    = tau Kh dG^T                  dKh = tau Qh dG
        dq[:, e] = (dQh[:, e] - Qh[:, e] (Qh[:, e] . dQh[:, e])) / nq_e   when |q[:, e]| > 1e-12,
                 = dQh[:, e] / 1e-12                                        otherwise (the floor
                                                                            is a constant there);
        likewise dk from dKh.
    Rows that belong to no window are NaN in dq, dk, dv.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(dout, dtype=np.float64)
    tau = np.asarray(tau, dtype=np.float64)
    n, H, d = q.shape
    dq = np.full(q.shape, np.nan)
    dk = np.full(q.shape, np.nan)
    dv = np.full(q.shape, np.nan)
    dtau = np.zeros(H)

    def unnormalise(x, xh, nx, dxh):
        raw = np.sqrt((x * x).sum(axis=0))
        proj = dxh - xh * (xh * dxh).sum(axis=0)
        return np.where(raw > XCA_NORM_FLOOR, proj, dxh) / nx

    for w in range(len(offsets) - 1):
        rows = _window_rows(offsets, perm, w)
        if rows.size == 0:
            continue
        for h in range(H):
            qw, kw, vw, dow = q[rows, h, :], k[rows, h, :], v[rows, h, :], do[rows, h, :]
            nq = np.maximum(np.sqrt((qw * qw).sum(axis=0)), XCA_NORM_FLOOR)
            nk = np.maximum(np.sqrt((kw * kw).sum(axis=0)), XCA_NORM_FLOOR)
            qh, kh = qw / nq, kw / nk
            N = qh.T @ kh
            G = tau[h] * N
            A = np.exp(G - G.max(axis=1, keepdims=True))
            A = A / A.sum(axis=1, keepdims=True)
            dv[rows, h, :] = dow @ A                   # dv_i[c] = sum_e A[e, c] do_i[e]
            dA = dow.T @ vw                            # dA[e, c] = sum_i do_i[e] v_i[c]
            dG = A * (dA - (A * dA).sum(axis=1, keepdims=True))
            dtau[h] += (dG * N).sum()
            dqh = tau[h] * (kh @ dG.T)                 # [m, d]: dqh[r, e] = tau sum_c dG[e, c] kh[r, c]
            dkh = tau[h] * (qh @ dG)                   # dkh[r, c] = tau sum_e dG[e, c] qh[r, e]
            dq[rows, h, :] = unnormalise(qw, qh, nq, dqh)
            dk[rows, h, :] = unnormalise(kw, kh, nk, dkh)
    return dq, dk, dv, dtau

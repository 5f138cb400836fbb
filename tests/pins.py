"""Independent checks ("pins") of the CPU oracle against what the paper and the
mathematics fix.  Each check takes the function under test as an argument so the
mutation tests can run the same checks against oracle copies with planted
mistakes and confirm that some check fails.

None of these re-types the oracle's formulas: they use a different association
order (the quadratic form of Sec. 3.1), exact rational arithmetic, closed forms
of special cases, invariants of Eq. (3) and finite differences.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np


# ------------------------------------------------------------------ tiny inputs
def tiny_case(seed: int, windows: int = 5, max_len: int = 7, heads: int = 2, d: int = 4,
              shuffle: bool = True, scale: float = 1.0):
    rng = np.random.default_rng([99, seed])
    lengths = rng.integers(0, max_len + 1, size=windows)
    lengths[rng.integers(0, windows)] = max(1, lengths.max())
    n = int(lengths.sum())
    ids = np.repeat(np.arange(windows), lengths)
    if shuffle:
        ids = ids[rng.permutation(n)]
    q = rng.standard_normal((n, heads, d)) * scale
    k = rng.standard_normal((n, heads, d)) * scale
    v = rng.standard_normal((n, heads, d))
    do = rng.standard_normal((n, heads, d))
    return ids, q, k, v, do


def segments_plain(ids, num_windows):
    """Window lists by direct enumeration (no sort): rows of window w in row order."""
    groups = [[] for _ in range(num_windows)]
    for r, w in enumerate(ids):
        if 0 <= w < num_windows:
            groups[w].append(r)
    perm = [r for g in groups for r in g]
    offsets = [0]
    for g in groups:
        offsets.append(offsets[-1] + len(g))
    return np.asarray(perm, dtype=np.int64), np.asarray(offsets, dtype=np.int64)


# --------------------------------------------------------------- forward checks
def _phi_scalar(x: float) -> float:
    return x + 1.0 if x > 0 else math.exp(x)


def brute_forward(q, k, v, ids, num_windows):
    """Quadratic form of Sec. 3.1: o_i = sum_j (phi(q_i).phi(k_j)) v_j / sum_j phi(q_i).phi(k_j),
    j over the rows with the same window id as i; plain Python loops."""
    n, H, d = q.shape
    out = np.full((n, H, d), np.nan)
    for i in range(n):
        wi = ids[i]
        if not (0 <= wi < num_windows):
            continue
        for h in range(H):
            num = [0.0] * d
            den = 0.0
            for j in range(n):
                if ids[j] != wi:
                    continue
                a = 0.0
                for e in range(d):
                    a += _phi_scalar(q[i, h, e]) * _phi_scalar(k[j, h, e])
                den += a
                for c in range(d):
                    num[c] += a * v[j, h, c]
            for c in range(d):
                out[i, h, c] = num[c] / den
    return out


def exact_forward(qf, kf, vf, ids):
    """Exact rational evaluation for inputs with q, k > 0 (phi(x) = x + 1 exactly)."""
    n, H, d = len(qf), len(qf[0]), len(qf[0][0])
    out = np.zeros((n, H, d))
    for i in range(n):
        for h in range(H):
            num = [Fraction(0)] * d
            den = Fraction(0)
            for j in range(n):
                if ids[j] != ids[i]:
                    continue
                a = sum((qf[i][h][e] + 1) * (kf[j][h][e] + 1) for e in range(d))
                den += a
                for c in range(d):
                    num[c] += a * vf[j][h][c]
            for c in range(d):
                out[i, h, c] = float(num[c] / den)
    return out


def rel_err(x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    scale = max(np.nanmax(np.abs(ref)), 1e-300)
    return float(np.nanmax(np.abs(x - ref)) / scale)


def forward_pin_failures(fwd, seg):
    """Run every forward pin against ``fwd(q, k, v, offsets, perm)`` (float64) and
    ``seg(ids, W) -> (perm, offsets, invalid)``; return the names that fail."""
    fails = []

    def run(ids, q, k, v, W):
        perm, off, _ = seg(ids, W)
        return fwd(q, k, v, off, perm)

    # 1. quadratic form (brute force), shuffled rows, several seeds
    for seed in range(4):
        ids, q, k, v, _ = tiny_case(seed)
        W = int(ids.max()) + 2
        if rel_err(run(ids, q, k, v, W), brute_forward(q, k, v, ids, W)) > 1e-12:
            fails.append(f"bruteforce[{seed}]")
    # 2. exact rationals with positive q, k
    rng = np.random.default_rng(7)
    n, H, d = 9, 2, 3
    ids = rng.integers(0, 3, size=n)
    qi = rng.integers(1, 17, size=(n, H, d))
    ki = rng.integers(1, 17, size=(n, H, d))
    vi = rng.integers(-16, 17, size=(n, H, d))
    qf = [[[Fraction(int(x), 8) for x in row] for row in r] for r in qi]
    kf = [[[Fraction(int(x), 8) for x in row] for row in r] for r in ki]
    vf = [[[Fraction(int(x), 8) for x in row] for row in r] for r in vi]
    if rel_err(run(ids, qi / 8.0, ki / 8.0, vi / 8.0, 3), exact_forward(qf, kf, vf, ids)) > 1e-14:
        fails.append("exact_rational")
    # 3. a window of one row returns its own value
    ids, q, k, v, _ = tiny_case(11)
    W = int(ids.max()) + 1
    ids1 = np.concatenate([ids, [W]])
    q1 = np.concatenate([q, np.full((1,) + q.shape[1:], -3.0)])
    k1 = np.concatenate([k, np.full((1,) + q.shape[1:], 2.5)])
    v1 = np.concatenate([v, np.arange(np.prod(q.shape[1:]), dtype=float).reshape((1,) + q.shape[1:])])
    o1 = run(ids1, q1, k1, v1, W + 1)
    if rel_err(o1[-1], v1[-1]) > 1e-15:
        fails.append("singleton")
    # 4. identical keys in a window -> every output is the window mean of v
    ids, q, k, v, _ = tiny_case(12, windows=3)
    k2 = k.copy()
    for w in range(3):
        rows = np.nonzero(ids == w)[0]
        if rows.size:
            k2[rows] = k[rows[0]]
    o2 = run(ids, q, k2, v, 3)
    for w in range(3):
        rows = np.nonzero(ids == w)[0]
        if rows.size and rel_err(o2[rows], np.broadcast_to(v[rows].mean(axis=0), o2[rows].shape)) > 1e-13:
            fails.append("identical_keys")
            break
    # 5. phi(q) concentrated on one feature e0 -> weights phi(k[:, e0])
    ids, q, k, v, _ = tiny_case(13, d=5)
    e0 = 2
    q3 = np.full_like(q, -80.0)
    q3[:, :, e0] = 0.7
    o3 = run(ids, q3, k, v, int(ids.max()) + 1)
    exp3 = np.full_like(v, np.nan)
    for w in np.unique(ids):
        rows = np.nonzero(ids == w)[0]
        wt = np.array([[_phi_scalar(k[r, h, e0]) for h in range(q.shape[1])] for r in rows])
        exp3[rows] = (wt[:, :, None] * v[rows]).sum(0) / wt.sum(0)[:, None]
    if rel_err(o3, exp3) > 1e-12:
        fails.append("one_feature_query")
    # 6. window independence (Eq. (2) concatenation): changing other windows' values
    ids, q, k, v, _ = tiny_case(14, windows=4)
    W = 4
    base = run(ids, q, k, v, W)
    other = ids != ids[0]
    qx, kx, vx = q.copy(), k.copy(), v.copy()
    qx[other] += 3.0
    kx[other] -= 2.0
    vx[other] *= -5.0
    mine = ids == ids[0]
    if not np.array_equal(run(ids, qx, kx, vx, W)[mine], base[mine]):
        fails.append("window_independence")
    # 7. relabelling windows and permuting rows permutes the output
    p = np.random.default_rng(3).permutation(len(ids))
    relabel = np.array([2, 0, 3, 1])
    if rel_err(run(relabel[ids][p], q[p], k[p], v[p], W), base[p]) > 1e-14:
        fails.append("permutation")
    # 8. affine equivariance, linearity in v, convex hull
    c = np.linspace(-2, 2, v.shape[1] * v.shape[2]).reshape(v.shape[1:])
    if rel_err(run(ids, q, k, v + c, W), base + c) > 1e-13:
        fails.append("affine")
    v2 = np.random.default_rng(4).standard_normal(v.shape)
    if rel_err(run(ids, q, k, 2 * v - 3 * v2, W), 2 * base - 3 * run(ids, q, k, v2, W)) > 1e-13:
        fails.append("linearity")
    for w in np.unique(ids):
        rows = ids == w
        lo = v[rows].min(axis=0) - 1e-12
        hi = v[rows].max(axis=0) + 1e-12
        if np.any(base[rows] < lo) or np.any(base[rows] > hi):
            fails.append("convex_hull")
            break
    return fails


# -------------------------------------------------------------- backward checks
def _loss(fwd, seg, ids, W, q, k, v, do):
    perm, off, _ = seg(ids, W)
    return float(np.nansum(fwd(q, k, v, off, perm) * do))


def backward_pin_failures(bwd, fwd, seg):
    """Pins for ``bwd(q, k, v, dout, offsets, perm) -> (dq, dk, dv)``."""
    fails = []
    # 1. central finite differences
    for seed in range(2):
        ids, q, k, v, do = tiny_case(20 + seed, windows=3, max_len=5, d=3)
        W = 3
        perm, off, _ = seg(ids, W)
        dq, dk, dv = bwd(q, k, v, do, off, perm)
        eps = 1e-6
        for name, x, g in (("dq", q, dq), ("dk", k, dk), ("dv", v, dv)):
            num = np.zeros_like(x)
            for idx in np.ndindex(x.shape):
                xp = x.copy()
                xm = x.copy()
                xp[idx] += eps
                xm[idx] -= eps
                args_p = [q, k, v]
                args_m = [q, k, v]
                pos = {"dq": 0, "dk": 1, "dv": 2}[name]
                args_p[pos] = xp
                args_m[pos] = xm
                num[idx] = (_loss(fwd, seg, ids, W, *args_p, do) - _loss(fwd, seg, ids, W, *args_m, do)) / (2 * eps)
            if rel_err(g, num) > 1e-6:
                fails.append(f"finite_difference_{name}[{seed}]")
    # invariants on a bigger tiny case
    ids, q, k, v, do = tiny_case(30, windows=6, max_len=9, d=4)
    W = 6
    perm, off, _ = seg(ids, W)
    dq, dk, dv = bwd(q, k, v, do, off, perm)
    fq = np.where(q > 0, q + 1, np.exp(np.minimum(q, 0)))
    fk = np.where(k > 0, k + 1, np.exp(np.minimum(k, 0)))
    dfq = dq / np.where(q > 0, 1.0, np.exp(np.minimum(q, 0)))
    dfk = dk / np.where(k > 0, 1.0, np.exp(np.minimum(k, 0)))
    for w in range(W):
        rows = ids == w
        if not rows.any():
            continue
        # 2. sum of dv over a window = sum of dout (affine equivariance in v)
        if rel_err(dv[rows].sum(0), do[rows].sum(0)) > 1e-12:
            fails.append("sum_dv")
            break
        # 4. scaling all phi(k) of a window leaves the output unchanged
        if np.max(np.abs((dfk[rows] * fk[rows]).sum(axis=(0, 2)))) > 1e-12 * max(1.0, np.abs(dfk).max()):
            fails.append("phik_scale")
            break
    # 3. scaling one phi(q_i) leaves o_i unchanged
    if np.max(np.abs((dfq * fq).sum(axis=2))) > 1e-12 * max(1.0, np.abs(dfq).max()):
        fails.append("phiq_scale")
    # 5. one-row windows: dv = dout, dq = dk = 0
    ids1 = np.arange(4)
    rng = np.random.default_rng(5)
    q1, k1, v1, do1 = (rng.standard_normal((4, 2, 3)) for _ in range(4))
    perm1, off1, _ = seg(ids1, 4)
    a, b, c = bwd(q1, k1, v1, do1, off1, perm1)
    if rel_err(c, do1) > 1e-15 or np.abs(a).max() > 1e-13 or np.abs(b).max() > 1e-13:
        fails.append("singleton_grad")
    return fails

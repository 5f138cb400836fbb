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


def _relu_scalar(x: float) -> float:
    return x if x > 0 else 0.0


def brute_forward(q, k, v, ids, num_windows, fmap="elu1", eps=0.0):
    """Quadratic form of Sec. 3.1: o_i = sum_j (phi(q_i).phi(k_j)) v_j / (sum_j phi(q_i).phi(k_j) + eps),
    j over the rows with the same window id as i; plain Python loops."""
    f = _phi_scalar if fmap == "elu1" else _relu_scalar
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
                    a += f(q[i, h, e]) * f(k[j, h, e])
                den += a
                for c in range(d):
                    num[c] += a * v[j, h, c]
            den += eps
            for c in range(d):
                out[i, h, c] = num[c] / den if den != 0.0 else math.nan
    return out


def exact_forward(qf, kf, vf, ids, shift=1, eps=Fraction(0)):
    """Exact rational evaluation for inputs with q, k > 0, where phi(x) = x + shift
    exactly (shift 1: elu + 1; shift 0: ReLU), with eps added to the normaliser."""
    n, H, d = len(qf), len(qf[0]), len(qf[0][0])
    out = np.zeros((n, H, d))
    for i in range(n):
        for h in range(H):
            num = [Fraction(0)] * d
            den = Fraction(0)
            for j in range(n):
                if ids[j] != ids[i]:
                    continue
                a = sum((qf[i][h][e] + shift) * (kf[j][h][e] + shift) for e in range(d))
                den += a
                for c in range(d):
                    num[c] += a * vf[j][h][c]
            den += eps
            for c in range(d):
                out[i, h, c] = float(num[c] / den)
    return out


def rel_err(x, ref):
    """max |x - ref| / max |ref| over the entries where ref is a number; inf if
    x and ref are NaN in different places."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if not np.array_equal(np.isnan(x), np.isnan(ref)):
        return math.inf
    if np.isnan(ref).all():
        return 0.0
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


# ------------------------------------------- feature-map variants and epsilon
# The ReLU feature map of the Tab. 7 variant (phi(x) = max(x, 0), phi'(0) = 0)
# and an eps >= 0 added to the normaliser, for either map.  ``fwd`` and ``bwd``
# take (..., offsets, perm, feature_map_name, eps).
def _away_from_zero(x, gap=1e-3):
    """Inputs kept at least `gap` from the ReLU kink (finite differences)."""
    return np.where(np.abs(x) < gap, np.where(x < 0, -gap, gap), x)


def variant_forward_pin_failures(fwd, seg):
    fails = []

    def run(ids, q, k, v, W, fmap, eps):
        perm, off, _ = seg(ids, W)
        return fwd(q, k, v, off, perm, fmap, eps)

    # 1. quadratic form (brute force), both maps, with and without eps; with
    #    eps = 0 some ReLU rows have a zero normaliser and are NaN on both sides
    for fmap in ("relu", "elu1"):
        for eps in (0.0, 0.3):
            for seed in range(3):
                ids, q, k, v, _ = tiny_case(40 + seed)
                W = int(ids.max()) + 2
                with np.errstate(invalid="ignore", divide="ignore"):
                    got = run(ids, q, k, v, W, fmap, eps)
                if rel_err(got, brute_forward(q, k, v, ids, W, fmap, eps)) > 1e-12:
                    fails.append(f"bruteforce_{fmap}_eps{eps}[{seed}]")
    # 2. exact rationals with positive q, k and eps = 1/4, both maps
    rng = np.random.default_rng(8)
    n, H, d = 9, 2, 3
    ids = rng.integers(0, 3, size=n)
    qi = rng.integers(1, 17, size=(n, H, d))
    ki = rng.integers(1, 17, size=(n, H, d))
    vi = rng.integers(-16, 17, size=(n, H, d))
    qf = [[[Fraction(int(x), 8) for x in row] for row in r] for r in qi]
    kf = [[[Fraction(int(x), 8) for x in row] for row in r] for r in ki]
    vf = [[[Fraction(int(x), 8) for x in row] for row in r] for r in vi]
    for fmap, shift in (("relu", 0), ("elu1", 1)):
        exact = exact_forward(qf, kf, vf, ids, shift=shift, eps=Fraction(1, 4))
        if rel_err(run(ids, qi / 8.0, ki / 8.0, vi / 8.0, 3, fmap, 0.25), exact) > 1e-14:
            fails.append(f"exact_rational_{fmap}")
    # 3. for x > 0, relu(x + 1) = elu(x) + 1: the ReLU path on q + 1, k + 1 is the
    #    elu path on q, k (a cross-check against the pinned default map)
    ids, q, k, v, _ = tiny_case(45)
    qp, kp = np.abs(q) + 0.01, np.abs(k) + 0.01
    W = int(ids.max()) + 1
    for eps in (0.0, 0.5):
        if rel_err(run(ids, qp + 1, kp + 1, v, W, "relu", eps), run(ids, qp, kp, v, W, "elu1", eps)) > 1e-14:
            fails.append(f"relu_shift_is_elu_eps{eps}")
    # 4. ReLU is positively homogeneous: scaling q (or every k) by t > 0 is the
    #    same as dividing eps by t
    ids, q, k, v, _ = tiny_case(46)
    W = int(ids.max()) + 1
    t = 2.5
    base = run(ids, q, k, v, W, "relu", 0.8)
    if rel_err(run(ids, t * q, k, v, W, "relu", 0.8 * t), base) > 1e-13:
        fails.append("relu_q_homogeneous")
    if rel_err(run(ids, q, t * k, v, W, "relu", 0.8 * t), base) > 1e-13:
        fails.append("relu_k_homogeneous")
    with np.errstate(invalid="ignore", divide="ignore"):
        b0 = run(ids, q, k, v, W, "relu", 0.0)
        if rel_err(run(ids, t * q, k / t, v, W, "relu", 0.0), b0) > 1e-13:
            fails.append("relu_scale_invariant")
    # 5. with eps the weights sum to s_i = o_i(v = 1) < 1: o(v + c) = o(v) + s c
    for fmap in ("relu", "elu1"):
        b = run(ids, q, k, v, W, fmap, 0.7)
        s1 = run(ids, q, k, np.ones_like(v), W, fmap, 0.7)
        c = np.linspace(-2, 2, v.shape[1] * v.shape[2]).reshape(v.shape[1:])
        if rel_err(run(ids, q, k, v + c, W, fmap, 0.7), b + s1 * c) > 1e-13:
            fails.append(f"affine_eps_{fmap}")
        if not (np.all(s1 < 1.0) and np.all(s1 >= 0.0) and np.ptp(s1, axis=2).max() < 1e-14):
            fails.append(f"weight_sum_eps_{fmap}")
    # 6. ReLU zero cases with eps > 0: a query with no positive entry, and a
    #    window whose keys have none, give o = 0 exactly (NaN when eps = 0)
    ids = np.array([0, 0, 0, 1, 1])
    rng = np.random.default_rng(9)
    q, k, v = (rng.standard_normal((5, 1, 3)) for _ in range(3))
    q[1] = -np.abs(q[1])
    k[3:] = -np.abs(k[3:]) - 0.1
    q[[0, 2, 3, 4]] = np.abs(q[[0, 2, 3, 4]]) + 0.1
    k[:3] = np.abs(k[:3]) + 0.1
    o = run(ids, q, k, v, 2, "relu", 0.25)
    if not (np.all(o[1] == 0.0) and np.all(o[3:] == 0.0) and np.all(o[[0, 2]] != 0.0)):
        fails.append("relu_zero_rows")
    with np.errstate(invalid="ignore", divide="ignore"):
        o0 = run(ids, q, k, v, 2, "relu", 0.0)
    if not (np.isnan(o0[[1, 3, 4]]).all() and np.isfinite(o0[[0, 2]]).all()):
        fails.append("relu_zero_rows_eps0_nan")
    return fails


def _loss_v(fwd, seg, ids, W, q, k, v, do, fmap, eps):
    perm, off, _ = seg(ids, W)
    return float(np.nansum(fwd(q, k, v, off, perm, fmap, eps) * do))


def variant_backward_pin_failures(bwd, fwd, seg):
    fails = []
    # 1. central finite differences, both maps, eps = 0.3, inputs away from the kink
    for fmap in ("relu", "elu1"):
        ids, q, k, v, do = tiny_case(50, windows=3, max_len=5, d=3)
        q, k = _away_from_zero(q), _away_from_zero(k)
        W = 3
        perm, off, _ = seg(ids, W)
        grads = bwd(q, k, v, do, off, perm, fmap, 0.3)
        h = 1e-6
        for pos, name in enumerate(("dq", "dk", "dv")):
            x = (q, k, v)[pos]
            num = np.zeros_like(x)
            for idx in np.ndindex(x.shape):
                args_p, args_m = [q, k, v], [q, k, v]
                xp, xm = x.copy(), x.copy()
                xp[idx] += h
                xm[idx] -= h
                args_p[pos], args_m[pos] = xp, xm
                num[idx] = (_loss_v(fwd, seg, ids, W, *args_p, do, fmap, 0.3)
                            - _loss_v(fwd, seg, ids, W, *args_m, do, fmap, 0.3)) / (2 * h)
            if rel_err(grads[pos], num) > 1e-6:
                fails.append(f"finite_difference_{fmap}_{name}")
    # 2. sum of dv over a window = sum_i s_i dout_i, s_i = o_i(v = 1)
    ids, q, k, v, do = tiny_case(51, windows=4, max_len=8, d=4)
    W = 4
    perm, off, _ = seg(ids, W)
    for fmap in ("relu", "elu1"):
        _, _, dv = bwd(q, k, v, do, off, perm, fmap, 0.6)
        s1 = fwd(q, k, np.ones_like(v), off, perm, fmap, 0.6)[:, :, :1]
        for w in range(W):
            rows = ids == w
            if rows.any() and rel_err(dv[rows].sum(0), (s1[rows] * do[rows]).sum(0)) > 1e-12:
                fails.append(f"sum_dv_eps_{fmap}")
                break
    # 3. ReLU, eps = 0, every normaliser positive: o is invariant to scaling one
    #    query row, and to scaling every key of a window, so q . dq = 0 per row
    #    and head, and sum_window k . dk = 0 per head (Euler)
    ids, q, k, v, do = tiny_case(52, windows=4, max_len=8, d=4)
    q[:, :, 0] = np.abs(q[:, :, 0]) + 0.1
    k[:, :, 0] = np.abs(k[:, :, 0]) + 0.1
    perm, off, _ = seg(ids, W)
    dq, dk, _ = bwd(q, k, v, do, off, perm, "relu", 0.0)
    scale = max(1.0, np.abs(dq).max(), np.abs(dk).max())
    if np.abs((q * dq).sum(axis=2)).max() > 1e-12 * scale:
        fails.append("relu_euler_q")
    for w in range(W):
        rows = ids == w
        if rows.any() and np.abs((k[rows] * dk[rows]).sum(axis=(0, 2))).max() > 1e-12 * scale:
            fails.append("relu_euler_k")
            break
    # 4. with eps > 0 the same scalings act as eps -> eps / t, so
    #    sum q . dq = sum k . dk = -eps dL/deps (dL/deps by finite differences)
    eps, h = 0.4, 1e-6
    dq, dk, _ = bwd(q, k, v, do, off, perm, "relu", eps)
    dl = (_loss_v(fwd, seg, ids, W, q, k, v, do, "relu", eps + h)
          - _loss_v(fwd, seg, ids, W, q, k, v, do, "relu", eps - h)) / (2 * h)
    if abs((q * dq).sum() + eps * dl) > 1e-7 * max(1.0, abs(eps * dl)):
        fails.append("relu_euler_q_eps")
    if abs((k * dk).sum() + eps * dl) > 1e-7 * max(1.0, abs(eps * dl)):
        fails.append("relu_euler_k_eps")
    # 5. phi'(0) = 0: entries at or below zero get no gradient under ReLU
    ids, q, k, v, do = tiny_case(53, windows=3, max_len=6, d=4)
    q[::2, :, 1] = 0.0
    k[1::3, :, 2] = 0.0
    W = 3
    perm, off, _ = seg(ids, W)
    dq, dk, _ = bwd(q, k, v, do, off, perm, "relu", 0.3)
    if np.any(dq[q <= 0] != 0.0) or np.any(dk[k <= 0] != 0.0):
        fails.append("relu_dphi_at_zero")
    # (not vacuous: most positive entries do get a gradient; a feature e with
    # z_e = 0 in its window legitimately gets none, as then S[e, :] = 0 too)
    if (np.count_nonzero(dq[q > 0]) < 0.6 * np.count_nonzero(q > 0)
            or np.count_nonzero(dk[k > 0]) < 0.6 * np.count_nonzero(k > 0)):
        fails.append("relu_gradient_vanishes")
    # 6. relu(x + 1) = elu(x) + 1 for x > 0: gradients agree as well
    ids, q, k, v, do = tiny_case(54, windows=3, max_len=6, d=4)
    qp, kp = np.abs(q) + 0.01, np.abs(k) + 0.01
    perm, off, _ = seg(ids, W)
    for eps in (0.0, 0.5):
        a = bwd(qp + 1, kp + 1, v, do, off, perm, "relu", eps)
        b = bwd(qp, kp, v, do, off, perm, "elu1", eps)
        if max(rel_err(x, y) for x, y in zip(a, b)) > 1e-13:
            fails.append(f"relu_shift_is_elu_grad_eps{eps}")
    return fails


# ----------------------------------------------------------- projected forward
# ``fwd_proj(x, w_qkv, b_qkv, w_o, b_o, heads, offsets, perm, fmap, eps) -> (o, y)``:
# the projection layer of Sec. 3.2, SLA, and the output projection.
def brute_projected(x, w_qkv, b_qkv, w_o, b_o, heads, ids, W, fmap="elu1", eps=0.0):
    """Plain loops: every projection as a sum over input channels, the attention
    as the quadratic form, then the output projection."""
    n, C = x.shape
    d = C // heads
    qkv = np.zeros((n, 3 * C))
    for r in range(n):
        for j in range(3 * C):
            acc = 0.0 if b_qkv is None else float(b_qkv[j])
            for c in range(C):
                acc += x[r, c] * w_qkv[j, c]
            qkv[r, j] = acc
    q = qkv[:, :C].reshape(n, heads, d)
    k = qkv[:, C:2 * C].reshape(n, heads, d)
    v = qkv[:, 2 * C:].reshape(n, heads, d)
    o = brute_forward(q, k, v, ids, W, fmap, eps)
    of = o.reshape(n, C)
    y = np.full((n, C), np.nan)
    for r in range(n):
        if np.isnan(of[r]).any():
            continue
        for j in range(C):
            acc = 0.0 if b_o is None else float(b_o[j])
            for c in range(C):
                acc += of[r, c] * w_o[j, c]
            y[r, j] = acc
    return o, y


def projected_pin_failures(fwd_proj, seg, fwd):
    fails = []
    rng = np.random.default_rng(70)
    # 1. brute force, heads in {1, 2, 3}, with and without biases, both maps
    for seed, heads, d, bias, fmap, eps in ((0, 2, 2, True, "elu1", 0.0), (1, 1, 3, False, "elu1", 0.0),
                                            (2, 3, 2, True, "relu", 0.2), (3, 2, 3, True, "elu1", 0.5)):
        ids, _, _, _, _ = tiny_case(80 + seed, windows=4, max_len=5)
        n, C = len(ids), heads * d
        x = rng.standard_normal((n, C))
        wq = rng.standard_normal((3 * C, C)) / np.sqrt(C)
        wo = rng.standard_normal((C, C)) / np.sqrt(C)
        bq = rng.standard_normal(3 * C) if bias else None
        bo = rng.standard_normal(C) if bias else None
        W = int(ids.max()) + 1
        perm, off, _ = seg(ids, W)
        with np.errstate(invalid="ignore", divide="ignore"):
            o, y = fwd_proj(x, wq, bq, wo, bo, heads, off, perm, fmap, eps)
            ob, yb = brute_projected(x, wq, bq, wo, bo, heads, ids, W, fmap, eps)
        if rel_err(o, ob) > 1e-12 or rel_err(y, yb) > 1e-12:
            fails.append(f"projected_bruteforce[{seed}]")
    # 2. block structure: W_q = I, W_k = 2 I, W_v = a permutation, W_o = I, no bias
    #    gives the plain SLA of (x, 2 x, x P^T)
    ids, _, _, _, _ = tiny_case(90, windows=5, max_len=6)
    heads, d = 2, 3
    n, C = len(ids), heads * d
    x = rng.standard_normal((n, C))
    P = np.eye(C)[rng.permutation(C)]
    wq = np.concatenate([np.eye(C), 2 * np.eye(C), P])
    W = int(ids.max()) + 1
    perm, off, _ = seg(ids, W)
    o, y = fwd_proj(x, wq, None, np.eye(C), None, heads, off, perm, "elu1", 0.0)
    ref = fwd(x.reshape(n, heads, d), 2 * x.reshape(n, heads, d), (x @ P.T).reshape(n, heads, d), off, perm)
    if rel_err(o, ref) > 1e-14 or rel_err(y, ref.reshape(n, C)) > 1e-14:
        fails.append("projected_blocks")
    # 3. biases: b_v = c shifts every o by c (weights sum to 1), so y by W_o c;
    #    b_o shifts y
    wq = rng.standard_normal((3 * C, C)) / np.sqrt(C)
    wo = rng.standard_normal((C, C)) / np.sqrt(C)
    o0, y0 = fwd_proj(x, wq, None, wo, None, heads, off, perm, "elu1", 0.0)
    c = rng.standard_normal(C)
    bq = np.concatenate([np.zeros(2 * C), c])
    o1, y1 = fwd_proj(x, wq, bq, wo, None, heads, off, perm, "elu1", 0.0)
    if rel_err(o1, o0 + c.reshape(heads, d)) > 1e-13 or rel_err(y1, y0 + wo @ c) > 1e-13:
        fails.append("projected_value_bias")
    bo = rng.standard_normal(C)
    _, y2 = fwd_proj(x, wq, None, wo, bo, heads, off, perm, "elu1", 0.0)
    if rel_err(y2, y0 + bo) > 1e-13:
        fails.append("projected_output_bias")
    return fails


# ---------------------------------------------------------- projected backward
# ``bwd_proj(x, w_qkv, b_qkv, w_o, b_o, dy, heads, offsets, perm, fmap, eps)
#   -> (dx, dw_qkv, db_qkv, dw_o, db_o)``: gradients of sum(y . dy) over the rows
# in windows.  Pinned against central differences of the plain-loop forward
# (``brute_projected``), which shares nothing with the backward.
def _proj_loss(x, wq, bq, wo, bo, dy, heads, ids, W, fmap, eps):
    _, y = brute_projected(x, wq, bq, wo, bo, heads, ids, W, fmap, eps)
    inside = ~np.isnan(y).any(axis=1)
    return float((y[inside] * dy[inside]).sum())


def projected_backward_pin_failures(bwd_proj, seg, bwd):
    fails = []
    rng = np.random.default_rng(71)
    h = 1e-5
    # 1. every entry of every gradient against a central difference of the loss
    #    (both maps, with and without biases, a row in no window)
    for seed, heads, d, bias, fmap, eps in ((0, 2, 2, True, "elu1", 0.0), (1, 1, 3, False, "relu", 0.3),
                                            (2, 2, 2, True, "relu", 0.5)):
        ids, _, _, _, _ = tiny_case(180 + seed, windows=3, max_len=4)
        W = int(ids.max()) + 1
        ids = np.concatenate([ids, [W + 2]])      # one row outside every window
        n, C = len(ids), heads * d
        x = rng.standard_normal((n, C))
        wq = rng.standard_normal((3 * C, C)) / np.sqrt(C)
        wo = rng.standard_normal((C, C)) / np.sqrt(C)
        bq = rng.standard_normal(3 * C) if bias else None
        bo = rng.standard_normal(C) if bias else None
        dy = rng.standard_normal((n, C))
        perm, off, _ = seg(ids, W)
        got = bwd_proj(x, wq, bq, wo, bo, dy, heads, off, perm, fmap, eps)
        # without a bias its gradient is still defined: the derivative at a zero bias
        params = [x, wq, np.zeros(3 * C) if bq is None else bq, wo, np.zeros(C) if bo is None else bo]
        for which, g in zip(range(5), got):
            fd = np.zeros_like(params[which])
            for idx in np.ndindex(params[which].shape):
                args = [None if t is None else t.copy() for t in params]
                args[which][idx] += h
                lp = _proj_loss(*args, dy, heads, ids, W, fmap, eps)
                args[which][idx] -= 2 * h
                lm = _proj_loss(*args, dy, heads, ids, W, fmap, eps)
                fd[idx] = (lp - lm) / (2 * h)
            if g.shape != fd.shape or rel_err(g, fd) > 1e-6:
                fails.append(f"projected_bwd_fd[{seed}][{which}]")
        # the row in no window gets no input gradient
        if np.any(got[0][-1] != 0.0):
            fails.append(f"projected_bwd_outside_row[{seed}]")
        # bias gradients are the row sums of dy and of [dq | dk | dv]
        if rel_err(got[4], dy[:-1].sum(axis=0)) > 1e-13:
            fails.append(f"projected_bwd_db_o[{seed}]")
    # 2. W_qkv = [I; I; I], W_o = I, no biases: the plain SLA backward of (x, x, x),
    #    dx = dq + dk + dv and dW_qkv = [dq | dk | dv]^T x
    ids, _, _, _, _ = tiny_case(190, windows=5, max_len=6)
    heads, d = 2, 3
    n, C = len(ids), heads * d
    W = int(ids.max()) + 1
    perm, off, _ = seg(ids, W)
    x = rng.standard_normal((n, C))
    dy = rng.standard_normal((n, C))
    wq = np.concatenate([np.eye(C)] * 3)
    dx, dwq, dbq, dwo, dbo = bwd_proj(x, wq, None, np.eye(C), None, dy, heads, off, perm, "elu1", 0.0)
    x3, dy3 = x.reshape(n, heads, d), dy.reshape(n, heads, d)
    dq, dk, dv = bwd(x3, x3, x3, dy3, off, perm)
    ref = (dq + dk + dv).reshape(n, C)
    dqkv = np.concatenate([t.reshape(n, C) for t in (dq, dk, dv)], axis=1)
    if rel_err(dx, ref) > 1e-13 or rel_err(dwq, dqkv.T @ x) > 1e-13 or rel_err(dbq, dqkv.sum(axis=0)) > 1e-13:
        fails.append("projected_bwd_identity")
    # 3. directional derivatives on a larger case (adjoint identities): for a random
    #    direction t of each argument, <grad, t> = d/ds L(arg + s t) at s = 0
    ids, _, _, _, _ = tiny_case(191, windows=6, max_len=8)
    heads, d = 2, 3
    n, C = len(ids), heads * d
    W = int(ids.max()) + 1
    perm, off, _ = seg(ids, W)
    x = rng.standard_normal((n, C))
    wq = rng.standard_normal((3 * C, C)) / np.sqrt(C)
    wo = rng.standard_normal((C, C)) / np.sqrt(C)
    bq, bo = rng.standard_normal(3 * C), rng.standard_normal(C)
    dy = rng.standard_normal((n, C))
    got = bwd_proj(x, wq, bq, wo, bo, dy, heads, off, perm, "elu1", 0.0)
    params = [x, wq, bq, wo, bo]
    for which in range(5):
        t = rng.standard_normal(params[which].shape)
        args_p = [a.copy() for a in params]
        args_m = [a.copy() for a in params]
        args_p[which] += h * t
        args_m[which] -= h * t
        dd = (_proj_loss(*args_p, dy, heads, ids, W, "elu1", 0.0)
              - _proj_loss(*args_m, dy, heads, ids, W, "elu1", 0.0)) / (2 * h)
        if abs(float((got[which] * t).sum()) - dd) > 1e-6 * max(1.0, abs(dd)):
            fails.append(f"projected_bwd_direction[{which}]")
    return fails


# ------------------------------------------------------ cross-window interaction
def cwi_pin_failures(cwi):
    """Pins for ``cwi(coords, x, w_x, w_y, w_3, grid) -> [n, 4c]`` (Eq. (4)-(7))."""
    from scipy import ndimage

    fails = []
    rng = np.random.default_rng(90)
    c = 3
    # 1. a sparse set is the dense grid with zeros in the empty cells, sampled at
    #    the voxels: compare with scipy's zero-padded correlations on the grid
    for seed, grid, fill, kx, ky in ((0, (9, 7, 3), 1.0, 5, 3), (1, (11, 10, 4), 0.35, 7, 9),
                                     (2, (13, 6, 1), 0.6, 13, 5)):
        r2 = np.random.default_rng([91, seed])
        gx, gy, gz = grid
        occ = r2.random((gz, gy, gx)) < fill
        occ.flat[r2.integers(occ.size)] = True
        zz, yy, xx = np.nonzero(occ)
        order = r2.permutation(zz.size)
        coords = np.stack([xx, yy, zz], axis=1)[order]
        n = coords.shape[0]
        x = r2.standard_normal((n, 4 * c))
        w_x, w_y, w_3 = r2.standard_normal((kx, c)), r2.standard_normal((ky, c)), r2.standard_normal((27, c))
        got = cwi(coords, x, w_x, w_y, w_3, grid)
        dense = np.zeros((gz, gy, gx, 4 * c))
        dense[coords[:, 2], coords[:, 1], coords[:, 0]] = x
        exp = np.zeros((gz, gy, gx, 4 * c))
        for ch in range(c):
            exp[..., ch] = ndimage.correlate1d(dense[..., ch], w_x[:, ch], axis=2, mode="constant")
            exp[..., c + ch] = ndimage.correlate1d(dense[..., c + ch], w_y[:, ch], axis=1, mode="constant")
            k3 = w_3[:, ch].reshape(3, 3, 3)  # [dz][dy][dx]
            exp[..., 2 * c + ch] = ndimage.correlate(dense[..., 2 * c + ch], k3, mode="constant")
        exp[..., 3 * c:] = dense[..., 3 * c:]
        ref = exp[coords[:, 2], coords[:, 1], coords[:, 0]]
        if rel_err(got, ref) > 1e-12:
            fails.append(f"cwi_dense_correlate[{seed}]")
    # 2. a lone voxel: every branch is its centre tap times the input
    x1 = rng.standard_normal((1, 4 * c))
    w_x, w_y, w_3 = rng.standard_normal((5, c)), rng.standard_normal((3, c)), rng.standard_normal((27, c))
    out1 = cwi(np.array([[2, 3, 1]]), x1, w_x, w_y, w_3, (6, 6, 3))
    exp1 = np.concatenate([w_x[2] * x1[0, :c], w_y[1] * x1[0, c:2 * c], w_3[13] * x1[0, 2 * c:3 * c],
                           x1[0, 3 * c:]])
    if rel_err(out1[0], exp1) > 1e-15:
        fails.append("cwi_single_voxel")
    # 3. translating every voxel (inside the grid) leaves the outputs unchanged,
    #    and permuting the rows permutes them
    coords = np.array([[1, 1, 0], [2, 1, 0], [1, 2, 0], [4, 2, 0], [2, 2, 0], [3, 3, 0]])
    x = rng.standard_normal((6, 4 * c))
    base = cwi(coords, x, w_x, w_y, w_3, (8, 8, 2))
    if rel_err(cwi(coords + np.array([3, 2, 1]), x, w_x, w_y, w_3, (8, 8, 2)), base) > 1e-15:
        fails.append("cwi_translation")
    p = rng.permutation(6)
    if rel_err(cwi(coords[p], x[p], w_x, w_y, w_3, (8, 8, 2)), base[p]) > 1e-15:
        fails.append("cwi_permutation")
    return fails


def cwi_backward_pin_failures(cwi_bwd, cwi_fwd):
    """Pins for ``cwi_bwd(coords, x, w_x, w_y, w_3, dy, grid) -> (dx, dw_x, dw_y, dw_3)``."""
    fails = []
    rng = np.random.default_rng(95)
    c = 2
    grid = (7, 6, 3)
    occ = rng.random(grid[::-1]) < 0.45
    zz, yy, xx = np.nonzero(occ)
    coords = np.stack([xx, yy, zz], axis=1)[rng.permutation(zz.size)]
    n = coords.shape[0]
    x = rng.standard_normal((n, 4 * c))
    dy = rng.standard_normal((n, 4 * c))
    w_x, w_y, w_3 = rng.standard_normal((5, c)), rng.standard_normal((3, c)), rng.standard_normal((27, c))
    dx, dwx, dwy, dw3 = cwi_bwd(coords, x, w_x, w_y, w_3, dy, grid)
    out = cwi_fwd(coords, x, w_x, w_y, w_3, grid)
    # 1. the module is linear in x: <dy, F(x)> = <dx, x> (adjoint / dot-product test)
    if abs((dy * out).sum() - (dx * x).sum()) > 1e-12 * max(1.0, abs((dy * out).sum())):
        fails.append("cwi_adjoint_x")
    # 2. the convolution branches are linear in their kernels: <dw, w> recovers
    #    each branch's share of <dy, F>
    for b, (dw, w) in enumerate(((dwx, w_x), (dwy, w_y), (dw3, w_3))):
        share = (dy[:, b * c:(b + 1) * c] * out[:, b * c:(b + 1) * c]).sum()
        if abs((dw * w).sum() - share) > 1e-12 * max(1.0, abs(share)):
            fails.append(f"cwi_adjoint_w{b}")
    # 3. central finite differences on a few entries of x and of each kernel
    h = 1e-6

    def loss(x_, wx_, wy_, w3_):
        return float((dy * cwi_fwd(coords, x_, wx_, wy_, w3_, grid)).sum())

    for idx in ((0, 0), (n // 2, c + 1), (n - 1, 2 * c), (3, 3 * c)):
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        fd = (loss(xp, w_x, w_y, w_3) - loss(xm, w_x, w_y, w_3)) / (2 * h)
        if abs(fd - dx[idx]) > 1e-6 * max(1.0, abs(fd)):
            fails.append(f"cwi_fd_dx{idx}")
    for b, (w, dw) in enumerate(((w_x, dwx), (w_y, dwy), (w_3, dw3))):
        idx = (w.shape[0] // 2 + 1, c - 1)
        args_p = [w_x.copy(), w_y.copy(), w_3.copy()]
        args_m = [w_x.copy(), w_y.copy(), w_3.copy()]
        args_p[b][idx] += h
        args_m[b][idx] -= h
        fd = (loss(x, *args_p) - loss(x, *args_m)) / (2 * h)
        if abs(fd - dw[idx]) > 1e-6 * max(1.0, abs(fd)):
            fails.append(f"cwi_fd_dw{b}")
    return fails


# ----------------------------------------------------------------- XCA variant
def brute_xca(q, k, v, tau, ids, num_windows):
    """XCA per window with plain Python loops, normalising after the dot product,
    G[e][c] = tau (sum_j q_je k_jc) / (|q_e| |k_c|), and each softmax weight as
    1 / sum_c' exp(G[e][c'] - G[e][c])."""
    n, H, d = q.shape
    out = np.full((n, H, d), np.nan)
    for w in range(num_windows):
        rows = [r for r in range(n) if ids[r] == w]
        if not rows:
            continue
        for h in range(H):
            nq = [max(math.sqrt(sum(q[r, h, e] ** 2 for r in rows)), 1e-12) for e in range(d)]
            nk = [max(math.sqrt(sum(k[r, h, c] ** 2 for r in rows)), 1e-12) for c in range(d)]
            G = [[tau[h] * sum(q[r, h, e] * k[r, h, c] for r in rows) / (nq[e] * nk[c]) for c in range(d)]
                 for e in range(d)]
            A = [[1.0 / sum(math.exp(G[e][c2] - G[e][c]) for c2 in range(d)) for c in range(d)]
                 for e in range(d)]
            for r in rows:
                for e in range(d):
                    out[r, h, e] = sum(A[e][c] * v[r, h, c] for c in range(d))
    return out


def xca_pin_failures(xca, seg):
    """Pins for ``xca(q, k, v, tau, offsets, perm) -> [n, H, d]`` (Tab. 7, XCA row)."""
    fails = []

    def run(ids, q, k, v, tau, W):
        perm, offs, _ = seg(ids, W)
        return xca(q, k, v, tau, offs, perm)

    # 1. brute force on tiny shuffled scenes
    for seed in range(3):
        ids, q, k, v, _ = tiny_case(seed, windows=4, max_len=6, heads=2, d=3)
        tau = np.array([0.7, 2.5])
        if rel_err(run(ids, q, k, v, tau, 4), brute_xca(q, k, v, tau, ids, 4)) > 1e-12:
            fails.append(f"xca_brute[{seed}]")
    # 2. tau = 0: every softmax row is uniform, o_i[e] = mean_c v_ic
    ids, q, k, v, _ = tiny_case(7, windows=3, max_len=5, heads=2, d=4)
    got = run(ids, q, k, v, np.zeros(2), 3)
    ok = (ids >= 0) & (ids < 3)
    exp = np.repeat(v.mean(axis=2, keepdims=True), 4, axis=2)
    if rel_err(got[ok], exp[ok]) > 1e-14:
        fails.append("xca_tau_zero")
    # 3. v constant across channels: o_i[e] = v_i (each softmax row sums to 1 over c)
    vc = np.repeat(v[:, :, :1], 4, axis=2)
    if rel_err(run(ids, q, k, vc, np.array([1.5, -3.0]), 3)[ok], vc[ok]) > 1e-13:
        fails.append("xca_rows_sum_to_one")
    # 4. orthonormal structure: q columns s_e U_e and k columns with khat_{pi(e)} = U_e
    #    (pi a 3-cycle on the first three channels), so G[e][c] = tau [c = pi(e)] and
    #    o_i[e] = (e^tau v_i,pi(e) + sum_{c != pi(e)} v_ic) / (e^tau + d - 1)
    rng = np.random.default_rng(5)
    m, d, H = 6, 4, 2
    pi = [1, 2, 0, 3]
    qs = np.zeros((m, H, d))
    ks = np.zeros((m, H, d))
    tau = np.array([2.0, -1.25])
    for h in range(H):
        U, _ = np.linalg.qr(rng.standard_normal((m, d)))
        s = rng.uniform(0.5, 3.0, size=d)
        t = rng.uniform(0.5, 3.0, size=d)
        for e in range(d):
            qs[:, h, e] = s[e] * U[:, e]
            ks[:, h, pi[e]] = t[pi[e]] * U[:, e]
    vs = rng.standard_normal((m, H, d))
    got = run(np.zeros(m, dtype=np.int64), qs, ks, vs, tau, 1)
    exp = np.empty((m, H, d))
    for h in range(H):
        big = math.exp(tau[h])
        for e in range(d):
            rest = vs[:, h, :].sum(axis=1) - vs[:, h, pi[e]]
            exp[:, h, e] = (big * vs[:, h, pi[e]] + rest) / (big + d - 1)
    if rel_err(got, exp) > 1e-12:
        fails.append("xca_orthonormal_closed_form")
    # 5. a zero q column: its normalised column is zero, so its softmax row is uniform
    q0 = q.copy()
    q0[:, :, 2] = 0.0
    got = run(ids, q0, k, v, np.array([1.5, -3.0]), 3)
    if rel_err(got[ok][:, :, 2], v[ok].mean(axis=2)) > 1e-14:
        fails.append("xca_zero_column")
    # 6. windows are independent and rows may come in any order
    p = np.random.default_rng(6).permutation(len(ids))
    base = run(ids, q, k, v, np.array([1.5, -3.0]), 3)
    if not np.array_equal(np.isnan(run(ids[p], q[p], k[p], v[p], np.array([1.5, -3.0]), 3)),
                          np.isnan(base[p])) or \
            rel_err(run(ids[p], q[p], k[p], v[p], np.array([1.5, -3.0]), 3)[ok[p]], base[p][ok[p]]) > 1e-13:
        fails.append("xca_row_permutation")
    return fails


def xca_backward_pin_failures(xca_bwd, xca_fwd, seg):
    """Pins for ``xca_bwd(q, k, v, tau, dout, offsets, perm) -> (dq, dk, dv, dtau)``
    against the pinned forward: central differences of L = <dout, o>, the adjoint
    identity in v, and the invariance of o to a positive scale of any q or k
    column within a window."""
    fails = []
    ids, q, k, v, do = tiny_case(11, windows=4, max_len=6, heads=2, d=3)
    W = 4
    tau = np.array([1.3, -2.1])
    perm, offs, _ = seg(ids, W)
    dq, dk, dv, dtau = xca_bwd(q, k, v, tau, do, offs, perm)

    def loss(q_, k_, v_, t_):
        o = xca_fwd(q_, k_, v_, t_, offs, perm)
        ok = ~np.isnan(o[:, 0, 0])
        return float((do[ok] * o[ok]).sum())

    # 1. central differences on every entry of q, k, v (of rows in a window) and of tau
    rows = np.nonzero((ids >= 0) & (ids < W))[0]
    step = 1e-6
    for name, arr, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(arr)
        for r in rows:
            for h in range(arr.shape[1]):
                for e in range(arr.shape[2]):
                    a1, a2 = arr.copy(), arr.copy()
                    a1[r, h, e] += step
                    a2[r, h, e] -= step
                    args1 = {"q": q, "k": k, "v": v}
                    args2 = dict(args1)
                    args1[name], args2[name] = a1, a2
                    num[r, h, e] = (loss(args1["q"], args1["k"], args1["v"], tau)
                                    - loss(args2["q"], args2["k"], args2["v"], tau)) / (2 * step)
        if rel_err(grad[rows], num[rows]) > 1e-6:
            fails.append(f"xca_bwd_fd_{name}")
    num_tau = np.array([(loss(q, k, v, tau + step * np.eye(2)[h]) - loss(q, k, v, tau - step * np.eye(2)[h]))
                        / (2 * step) for h in range(2)])
    if rel_err(dtau, num_tau) > 1e-6:
        fails.append("xca_bwd_fd_tau")
    # 2. o is linear in v: <dout, o> = <dv, v>
    if abs(loss(q, k, v, tau) - float((dv[rows] * v[rows]).sum())) > 1e-12 * max(1.0, abs(loss(q, k, v, tau))):
        fails.append("xca_bwd_adjoint_v")
    # 3. scaling a q (or k) column of one window leaves o unchanged, so the
    #    gradient along that column vanishes: sum_r dq[r, e] q[r, e] = 0 per window
    worst = 0.0
    for w in range(W):
        rw = np.nonzero(ids == w)[0]
        if rw.size == 0:
            continue
        for x, g in ((q, dq), (k, dk)):
            dots = (g[rw] * x[rw]).sum(axis=0)
            worst = max(worst, float(np.abs(dots).max()) / max(float(np.abs(g[rw]).max()), 1e-300))
    if worst > 1e-12:
        fails.append("xca_bwd_scale_invariance")
    # 4. rows in no window get no gradient (NaN)
    bad = np.nonzero((ids < 0) | (ids >= W))[0]
    if bad.size and not all(np.isnan(g[bad]).all() for g in (dq, dk, dv)):
        fails.append("xca_bwd_rows_outside")
    return fails

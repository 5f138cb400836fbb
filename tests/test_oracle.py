"""CPU tests: the oracle against its pins, and mutation tests showing that a
plausible mistake planted in a copy of the oracle fails at least one pin."""
import importlib.util
import os
import types

import numpy as np
import pytest

import oracle
from oracle import sla_ref
from tests import pins

import workloads


# ------------------------------------------------------------------ widening
def test_widen_exact():
    assert oracle.widen(np.array([0x3F80, 0xC000, 0x0000, 0x3E80], dtype=np.uint16), "bf16").tolist() == [
        1.0, -2.0, 0.0, 0.25]
    x = np.array([1.0, -2.5, 65504.0, 6.103515625e-05], dtype=np.float16)
    assert oracle.widen(x, "f16").tolist() == [1.0, -2.5, 65504.0, 6.103515625e-05]
    # bf16 rounding of the generator is round-to-nearest-even
    f = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -9)], dtype=np.float32)
    assert oracle.widen(workloads.to_bf16_bits(f), "bf16").tolist() == [1.0, 1.0 + 2 ** -6, -1.0]


def test_phi_values():
    x = np.array([-1000.0, -1.0, 0.0, 0.5, 3.0])
    assert np.allclose(oracle.phi(x), [0.0, np.exp(-1.0), 1.0, 1.5, 4.0], rtol=0, atol=1e-300)
    assert np.allclose(oracle.dphi(x), [0.0, np.exp(-1.0), 1.0, 1.0, 1.0], rtol=0, atol=1e-300)


# ------------------------------------------------------------ segment builder
@pytest.mark.parametrize("seed", range(6))
def test_segments_vs_enumeration(seed):
    rng = np.random.default_rng(seed)
    W = int(rng.integers(1, 40))
    n = int(rng.integers(0, 300))
    ids = rng.integers(-2, W + 2, size=n)
    perm, off, inv = oracle.segments_ref(ids, W)
    p2, o2 = pins.segments_plain(ids, W)
    assert np.array_equal(perm, p2)
    assert np.array_equal(off, o2)
    assert inv == int(((ids < 0) | (ids >= W)).sum())
    # invariants: ids[perm] non-decreasing, ties ascending, offsets[W] = #valid
    s = ids[perm]
    assert np.all(np.diff(s) >= 0)
    same = np.diff(s) == 0
    assert np.all(np.diff(perm)[same] > 0)
    assert off[-1] == n - inv


# ---------------------------------------------------------------- chunk plan
def _check_plan_invariants(off, L, chunks, longs, n_four):
    off = np.asarray(off)
    nw = len(off) - 1
    page = L // 2
    lengths = np.diff(off)
    nonempty = np.nonzero(lengths > 0)[0]
    # every non-empty window is in exactly one chunk or in the long table
    owner = np.zeros(nw, dtype=np.int64)
    for rb, re, wb, we in chunks:
        owner[wb:we][lengths[wb:we] > 0] += 1
    owner[np.asarray(longs, dtype=np.int64)] += 1
    assert np.array_equal(owner[nonempty], np.ones(nonempty.size, dtype=np.int64))
    assert np.all(owner[lengths == 0] == 0)
    # long windows: more than L rows; four-way ones (more than 2L rows) first,
    # then two-way ones, each group in sequence order
    assert all(lengths[w] > L for w in longs)
    four, two = list(longs[:n_four]), list(longs[n_four:])
    assert all(lengths[w] > 2 * L for w in four) and all(lengths[w] <= 2 * L for w in two)
    assert four == sorted(four) and two == sorted(two)
    # chunks: whole windows, in order, disjoint, rows tiled by the long windows
    covered = np.zeros(int(off[-1]), dtype=np.int64)
    for w in longs:
        covered[off[w]:off[w + 1]] += 1
    for a, b in zip(chunks[:-1], chunks[1:]):
        assert a[3] <= b[2]
    for rb, re, wb, we in chunks:
        assert rb < re and wb < we
        assert off[wb] == rb and off[we] == re          # whole windows only
        covered[rb:re] += 1
        inside = lengths[wb:we]
        assert inside[0] > 0                           # a chunk opens on a non-empty window
        assert np.all(inside <= L)
        if (inside > page).any():                      # a mid window is alone
            assert (inside > 0).sum() == 1
        else:
            assert re - rb <= L - 1                     # packs stay under L rows
            starts = off[wb:we][inside > 0]
            assert np.all(starts // page == starts[0] // page)
    if nonempty.size:
        assert np.all(covered[off[nonempty[0]]:] == 1)


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("L", [8, 32, 48, 64])
def test_chunk_plan_invariants(seed, L):
    rng = np.random.default_rng([seed, L])
    W = int(rng.integers(1, 200))
    lengths = rng.integers(0, 3 * L, size=W) * (rng.random(W) < 0.8)
    if seed % 3 == 0:
        lengths = rng.integers(0, 8, size=W)
    off = workloads.offsets_from_lengths(lengths).astype(np.int64)
    chunks, longs, n_four = oracle.chunk_plan_ref(off, L)
    _check_plan_invariants(off, L, chunks.tolist(), longs.tolist(), n_four)


def test_chunk_plan_hand_example():
    # L = 8, pages of 4 rows.  Windows: 3, 0, 2, 5, 1, 1, 0, 2, 9, 4, 0, 17 rows.
    # rows:  w0 [0,3)  w1 empty  w2 [3,5)  w3 [5,10) mid  w4 [10,11)  w5 [11,12)
    #        w6 empty  w7 [12,14)  w8 [14,23) long  w9 [23,27)  w10 empty
    #        w11 [27,44) long
    # w0 opens; w2 starts at row 3 (page 0, same as w0) -> joins; w3 has 5 > 4
    # rows -> alone; w4 follows a mid window -> opens; w5 starts at 11 (page 2,
    # same as w4's 10) -> joins; w7 starts at 12 (page 3) -> opens and ends where
    # the long window w8 begins; w8 (9 rows: more than 8, at most 16) is a two-way
    # long window; w9 follows a long window -> opens and ends where w11 begins;
    # w11 (17 > 16 rows) is a four-way long window, listed first.
    off = workloads.offsets_from_lengths(np.array([3, 0, 2, 5, 1, 1, 0, 2, 9, 4, 0, 17]))
    chunks, longs, n_four = oracle.chunk_plan_ref(off, 8)
    assert chunks.tolist() == [[0, 5, 0, 3], [5, 10, 3, 4], [10, 12, 4, 7], [12, 14, 7, 8],
                               [23, 27, 9, 11]]
    assert longs.tolist() == [11, 8] and n_four == 1


def test_chunk_plan_empty():
    chunks, longs, n_four = oracle.chunk_plan_ref(np.zeros(5, dtype=np.int64), 64)
    assert chunks.shape == (0, 4) and longs.shape == (0,) and n_four == 0


# ------------------------------------------------------------------ forward pins
def test_forward_pins():
    assert pins.forward_pin_failures(oracle.sla_forward_ref, oracle.segments_ref) == []


def test_forward_single_window_is_plain_linear_attention():
    # Sec. 3.1: with one window SLA is kernelised linear attention on the whole
    # sequence, phi(Q)(phi(K)^T V) / phi(Q)(phi(K)^T 1).
    rng = np.random.default_rng(1)
    q, k, v = (rng.standard_normal((20, 3, 6)) for _ in range(3))
    fq = np.where(q > 0, q + 1, np.exp(np.minimum(q, 0)))
    fk = np.where(k > 0, k + 1, np.exp(np.minimum(k, 0)))
    ref = np.stack([fq[:, h] @ (fk[:, h].T @ v[:, h]) / (fq[:, h] @ fk[:, h].sum(0))[:, None]
                    for h in range(3)], axis=1)
    out = oracle.sla_forward_ref(q, k, v, np.array([0, 20]), None)
    assert pins.rel_err(out, ref) < 1e-13


def test_forward_empty_and_invalid_rows():
    ids = np.array([3, -1, 3, 7, 0])
    rng = np.random.default_rng(2)
    q, k, v = (rng.standard_normal((5, 1, 2)) for _ in range(3))
    perm, off, inv = oracle.segments_ref(ids, 5)
    assert inv == 2
    o = oracle.sla_forward_ref(q, k, v, off, perm)
    assert np.isnan(o[1]).all() and np.isnan(o[3]).all()
    assert np.isfinite(o[[0, 2, 4]]).all()
    assert np.allclose(o[4], v[4], rtol=1e-15)


# ----------------------------------------------------------------- backward pins
def test_backward_pins():
    assert pins.backward_pin_failures(oracle.sla_backward_ref, oracle.sla_forward_ref,
                                      oracle.segments_ref) == []


# -------------------------------------------------------------- mutation tests
class _NumpyProxy:
    """numpy with einsum rewritten for chosen subscripts (mutation tests only)."""

    def __init__(self, rewrite):
        self._rewrite = rewrite

    def __getattr__(self, name):
        return getattr(np, name)

    def einsum(self, sub, *ops):
        if sub in self._rewrite:
            return self._rewrite[sub](*ops)
        return np.einsum(sub, *ops)


def _fresh_oracle():
    path = os.path.join(os.path.dirname(sla_ref.__file__), "sla_ref.py")
    spec = importlib.util.spec_from_file_location("sla_ref_mutant", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


FWD_MUTANTS = {
    "state_transposed": {"einsum": {"mhe,mhc->hec": lambda a, b: np.einsum("mhe,mhc->hce", a, b)}},
    "no_normaliser": {"einsum": {"mhe,he->mh": lambda a, b: np.ones(a.shape[:2])}},
    "normaliser_from_first_feature": {"einsum": {"mhe,he->mh": lambda a, b: a[:, :, 0] * b[None, :, 0]}},
    "phi_relu_plus_one": {"phi": lambda x: np.maximum(np.asarray(x, float), 0) + 1},
    "phi_exp_everywhere": {"phi": lambda x: np.exp(np.asarray(x, float))},
    "phi_shifted_branch": {"phi": lambda x: np.where(np.asarray(x) > 0, np.asarray(x) + 1, np.exp(np.asarray(x)) + 1e-3)},
}

BWD_MUTANTS = {
    "dS_transposed": {"einsum": {"mhc,hec->mhe": lambda a, b: np.einsum("mhc,hce->mhe", a, b)}},
    "no_dz": {"einsum": {"mh,mhe->he": lambda a, b: np.zeros(b.shape[1:])}},
    "wrong_sign_s": {"einsum": {"mhc,mhc->mh": lambda a, b: -np.einsum("mhc,mhc->mh", a, b)}},
    "no_dphi": {"dphi": lambda x: np.ones_like(np.asarray(x, float))},
    "dv_uses_transposed_dS": {"einsum": {"mhe,hec->mhc": lambda a, b: np.einsum("mhe,hce->mhc", a, b)}},
}


def _apply(mod, spec):
    if "einsum" in spec:
        mod.np = _NumpyProxy(spec["einsum"])
    for name in ("phi", "dphi"):
        if name in spec:
            setattr(mod, name, spec[name])
    return mod


@pytest.mark.parametrize("name", sorted(FWD_MUTANTS))
def test_forward_mutant_is_caught(name):
    mod = _apply(_fresh_oracle(), FWD_MUTANTS[name])
    with np.errstate(all="ignore"):
        fails = pins.forward_pin_failures(mod.sla_forward_ref, oracle.segments_ref)
    assert fails, f"planted mistake {name} passed every forward pin"


@pytest.mark.parametrize("name", sorted(BWD_MUTANTS))
def test_backward_mutant_is_caught(name):
    mod = _apply(_fresh_oracle(), BWD_MUTANTS[name])
    with np.errstate(all="ignore"):
        fails = pins.backward_pin_failures(mod.sla_backward_ref, oracle.sla_forward_ref,
                                           oracle.segments_ref)
    assert fails, f"planted mistake {name} passed every backward pin"


def test_segments_mutant_is_caught():
    # an unstable sort is a plausible mistake: ties must keep row order
    def unstable(ids, W):
        ids = np.asarray(ids)
        valid = (ids >= 0) & (ids < W)
        rows = np.nonzero(valid)[0]
        perm = rows[np.argsort(-ids[rows], kind="stable")[::-1]]
        off = np.concatenate([[0], np.cumsum(np.bincount(ids[rows], minlength=W))])
        return perm, off, int((~valid).sum())

    rng = np.random.default_rng(0)
    ids = rng.integers(0, 5, size=50)
    p1, _, _ = unstable(ids, 5)
    p2, _ = pins.segments_plain(ids, 5)
    assert not np.array_equal(p1, p2)


# ------------------------------------------- feature-map variants and epsilon
def test_phi_relu_values():
    x = np.array([-2.0, -0.0, 0.0, 1e-300, 3.5])
    assert oracle.phi_relu(x).tolist() == [0.0, 0.0, 0.0, 1e-300, 3.5]
    assert oracle.dphi_relu(x).tolist() == [0.0, 0.0, 0.0, 1.0, 1.0]
    with pytest.raises(ValueError):
        oracle.feature_map("gelu")
    with pytest.raises(ValueError):
        oracle.sla_forward_ref(np.ones((1, 1, 1)), np.ones((1, 1, 1)), np.ones((1, 1, 1)),
                               np.array([0, 1]), None, "relu", -1e-9)


def test_variant_forward_pins():
    assert pins.variant_forward_pin_failures(oracle.sla_forward_ref, oracle.segments_ref) == []


def test_variant_backward_pins():
    assert pins.variant_backward_pin_failures(oracle.sla_backward_ref, oracle.sla_forward_ref,
                                              oracle.segments_ref) == []


def test_default_map_and_eps_unchanged():
    # the default call is Eq. (3) as before: elu + 1 and no epsilon
    ids, q, k, v, do = pins.tiny_case(60)
    perm, off, _ = oracle.segments_ref(ids, int(ids.max()) + 1)
    assert np.array_equal(oracle.sla_forward_ref(q, k, v, off, perm),
                          oracle.sla_forward_ref(q, k, v, off, perm, "elu1", 0.0))
    a = oracle.sla_backward_ref(q, k, v, do, off, perm)
    b = oracle.sla_backward_ref(q, k, v, do, off, perm, "elu1", 0.0)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))


def _oracle_from_source(replacements):
    """A copy of the oracle module with source edits: (old, new, occurrence), the
    occurrence index counting from 0, or None for every occurrence."""
    path = os.path.join(os.path.dirname(sla_ref.__file__), "sla_ref.py")
    src = open(path).read()
    for old, new, which in replacements:
        count = src.count(old)
        assert count > 0 and (which is None or which < count), f"mutation site {old!r} not found"
        if which is None:
            src = src.replace(old, new)
        else:
            at = -1
            for _ in range(which + 1):
                at = src.index(old, at + 1)
            src = src[:at] + new + src[at + len(old):]
    mod = types.ModuleType("sla_ref_mutant")
    exec(compile(src, path, "exec"), mod.__dict__)
    return mod


_DEN = 'den = np.einsum("mhe,he->mh", fq, z) + eps'
VARIANT_FWD_MUTANTS = {
    "eps_dropped": [(_DEN, 'den = np.einsum("mhe,he->mh", fq, z)', 0)],
    "eps_in_numerator": [('num = np.einsum("mhe,hec->mhc", fq, S)',
                          'num = np.einsum("mhe,hec->mhc", fq, S) + eps', 0)],
    "eps_scales_normaliser": [(_DEN, 'den = np.einsum("mhe,he->mh", fq, z) * (1.0 + eps)', 0)],
    "eps_squared": [(_DEN, 'den = np.einsum("mhe,he->mh", fq, z) + eps * eps', 0)],
    "relu_leaky": [("return np.where(x > 0.0, x, 0.0)", "return np.where(x > 0.0, x, 0.01 * x)", 0)],
    "relu_offset": [("return np.where(x > 0.0, x, 0.0)", "return np.where(x > 0.0, x + 1e-9, 0.0)", 0)],
    "relu_is_elu": [("return phi_relu, dphi_relu", "return phi, dphi", 0)],
}

VARIANT_BWD_MUTANTS = {
    "bwd_eps_dropped": [(_DEN, 'den = np.einsum("mhe,he->mh", fq, z)', 1)],
    "relu_dphi_one_at_zero": [("return np.where(x > 0.0, 1.0, 0.0)", "return np.where(x >= 0.0, 1.0, 0.0)", 0)],
    "relu_dphi_ones": [("return np.where(x > 0.0, 1.0, 0.0)", "return np.where(x > 0.0, 1.0, 1.0)", 0)],
    "relu_dq_elu_derivative": [("dq[rows] = dfq * fdphi(qq)", "dq[rows] = dfq * dphi(qq)", 0)],
    "relu_dk_elu_derivative": [("dk[rows] = dfk * fdphi(kk)", "dk[rows] = dfk * dphi(kk)", 0)],
    "bwd_eps_in_s_only": [('s = -np.einsum("mhc,mhc->mh", do, o) / den',
                           's = -np.einsum("mhc,mhc->mh", do, o) / (den - eps)', 0)],
}


@pytest.mark.parametrize("name", sorted(VARIANT_FWD_MUTANTS))
def test_variant_forward_mutant_is_caught(name):
    mod = _oracle_from_source(VARIANT_FWD_MUTANTS[name])
    with np.errstate(all="ignore"):
        fails = pins.variant_forward_pin_failures(mod.sla_forward_ref, oracle.segments_ref)
    assert fails, f"planted mistake {name} passed every variant forward pin"


@pytest.mark.parametrize("name", sorted(VARIANT_BWD_MUTANTS))
def test_variant_backward_mutant_is_caught(name):
    mod = _oracle_from_source(VARIANT_BWD_MUTANTS[name])
    with np.errstate(all="ignore"):
        fails = pins.variant_backward_pin_failures(mod.sla_backward_ref, oracle.sla_forward_ref,
                                                   oracle.segments_ref)
    assert fails, f"planted mistake {name} passed every variant backward pin"


# ------------------------------------------------------------ projected forward
def test_projected_pins():
    assert pins.projected_pin_failures(oracle.sla_projected_forward_ref, oracle.segments_ref,
                                       oracle.sla_forward_ref) == []


PROJECTED_MUTANTS = {
    "q_k_blocks_swapped": [("q, k, v = (qkv[:, i * C:(i + 1) * C]", "k, q, v = (qkv[:, i * C:(i + 1) * C]", 0)],
    "output_weight_not_transposed": [("y = o.reshape(n, C) @ w_o.T", "y = o.reshape(n, C) @ w_o", 0)],
    "input_weight_not_transposed": [("qkv = x @ w_qkv.T", "qkv = x @ w_qkv.reshape(C, 3 * C)", 0)],
    "heads_interleaved": [(".reshape(n, heads, d) for i in range(3))",
                          ".reshape(n, d, heads).transpose(0, 2, 1) for i in range(3))", 0)],
    "bias_dropped": [("qkv = qkv + np.asarray(b_qkv, dtype=np.float64)", "qkv = qkv", 0)],
}


@pytest.mark.parametrize("name", sorted(PROJECTED_MUTANTS))
def test_projected_mutant_is_caught(name):
    mod = _oracle_from_source(PROJECTED_MUTANTS[name])
    with np.errstate(all="ignore"):
        fails = pins.projected_pin_failures(mod.sla_projected_forward_ref, oracle.segments_ref,
                                            oracle.sla_forward_ref)
    assert fails, f"planted mistake {name} passed every projected pin"


# ----------------------------------------------------------- projected backward
def test_projected_backward_pins():
    assert pins.projected_backward_pin_failures(oracle.sla_projected_backward_ref, oracle.segments_ref,
                                                oracle.sla_backward_ref) == []


PROJECTED_BWD_MUTANTS = {
    "dw_o_transposed": [("dw_o = g.T @ o", "dw_o = o.T @ g", 0)],
    "do_weight_transposed": [("do = (g @ w_o).reshape(n, heads, d)", "do = (g @ w_o.T).reshape(n, heads, d)", 0)],
    "dx_weight_transposed_blocks": [("dx = dqkv @ w_qkv", "dx = dqkv @ w_qkv[np.r_[C:2 * C, 0:C, 2 * C:3 * C]]", 0)],
    "dw_qkv_from_projected_rows": [("dw_qkv = dqkv.T @ x", "dw_qkv = dqkv.T @ qkv[:, :C]", 0)],
    "outside_dy_counted": [("g = np.where(inside[:, None], dy, 0.0)", "g = dy", 0)],
    "outside_dqkv_zeroed_late": [("dqkv = np.where(inside[:, None], dqkv, 0.0)",
                                  "dqkv = np.where(np.isnan(dqkv), 1.0, dqkv)", 0)],
    "db_qkv_dropped_v": [("db_qkv = dqkv.sum(axis=0)", "db_qkv = np.concatenate([dqkv[:, :2 * C].sum(axis=0), np.zeros(C)])", 0)],
}


@pytest.mark.parametrize("name", sorted(PROJECTED_BWD_MUTANTS))
def test_projected_backward_mutant_is_caught(name):
    mod = _oracle_from_source(PROJECTED_BWD_MUTANTS[name])
    with np.errstate(all="ignore"):
        fails = pins.projected_backward_pin_failures(mod.sla_projected_backward_ref, oracle.segments_ref,
                                                     oracle.sla_backward_ref)
    assert fails, f"planted mistake {name} passed every projected backward pin"


# ------------------------------------------------------ cross-window interaction
def test_cwi_pins():
    assert pins.cwi_pin_failures(oracle.cwi_forward_ref) == []


CWI_MUTANTS = {
    "kernel_flipped": [("off[axis] = t - half", "off[axis] = half - t", 0)],
    "axes_swapped": [("for branch, w, axis in ((0, w_x, 0), (1, w_y, 1)):",
                      "for branch, w, axis in ((0, w_x, 1), (1, w_y, 0)):", 0)],
    "cube_taps_transposed": [("w_3[(dx + 1) + 3 * (dy + 1) + 9 * (dz + 1)]", "w_3[(dz + 1) + 3 * (dy + 1) + 9 * (dx + 1)]", 0)],
    "identity_dropped": [("out[:, 3 * c:] = x[:, 3 * c:]", "out[:, 3 * c:] = 0.0", 0)],
    "off_centre": [("half = (w.shape[0] - 1) // 2", "half = w.shape[0] // 2 - 1", 0)],
    "branch_channels_shifted": [("lo = branch * c", "lo = (branch + 1) % 3 * c", 0)],
}


@pytest.mark.parametrize("name", sorted(CWI_MUTANTS))
def test_cwi_mutant_is_caught(name):
    mod = _oracle_from_source(CWI_MUTANTS[name])
    with np.errstate(all="ignore"):
        fails = pins.cwi_pin_failures(mod.cwi_forward_ref)
    assert fails, f"planted mistake {name} passed every CWI pin"


def test_cwi_backward_pins():
    assert pins.cwi_backward_pin_failures(oracle.cwi_backward_ref, oracle.cwi_forward_ref) == []


CWI_BWD_MUTANTS = {
    "dx_gathered_not_scattered": [("np.add.at(dx, (q, slice(lo, lo + c)), w[t] * dy[ok, lo:lo + c])",
                                   "dx[ok, lo:lo + c] += w[t] * dy[q, lo:lo + c]", 0)],
    "identity_grad_dropped": [("dx[:, 3 * c:] = dy[:, 3 * c:]", "dx[:, 3 * c:] = 0.0", 0)],
    "dw_from_own_row": [("dws[branch][t] = (dy[ok, lo:lo + c] * x[q, lo:lo + c]).sum(axis=0)",
                         "dws[branch][t] = (dy[ok, lo:lo + c] * x[ok, lo:lo + c]).sum(axis=0)", 0)],
    "cube_grad_taps_flipped": [("tap(2, (dx_ + 1) + 3 * (dy_ + 1) + 9 * (dz + 1), w_3, (dx_, dy_, dz))",
                                "tap(2, (1 - dx_) + 3 * (1 - dy_) + 9 * (1 - dz), w_3, (dx_, dy_, dz))", 0)],
}


@pytest.mark.parametrize("name", sorted(CWI_BWD_MUTANTS))
def test_cwi_backward_mutant_is_caught(name):
    mod = _oracle_from_source(CWI_BWD_MUTANTS[name])
    with np.errstate(all="ignore"):
        fails = pins.cwi_backward_pin_failures(mod.cwi_backward_ref, oracle.cwi_forward_ref)
    assert fails, f"planted mistake {name} passed every CWI backward pin"


# ------------------------------------------------------------------ XCA variant
def test_xca_pins():
    assert pins.xca_pin_failures(oracle.xca_forward_ref, oracle.segments_ref) == []


XCA_MUTANTS = {
    "softmax_over_rows": [("G = G - G.max(axis=1, keepdims=True)", "G = G - G.max(axis=0, keepdims=True)", 0),
                          ("A = A / A.sum(axis=1, keepdims=True)", "A = A / A.sum(axis=0, keepdims=True)", 0)],
    "attention_transposed": [("out[rows, h, :] = v[rows, h, :] @ A.T", "out[rows, h, :] = v[rows, h, :] @ A", 0)],
    "q_not_normalised": [("qhat = qw / qn", "qhat = qw", 0)],
    "norm_over_channels": [("kn = np.maximum(np.sqrt((kw * kw).sum(axis=0)), XCA_NORM_FLOOR)",
                            "kn = np.maximum(np.sqrt((kw * kw).sum(axis=1, keepdims=True)), XCA_NORM_FLOOR)", 0)],
    "first_head_temperature": [("G = tau[h] * (qhat.T @ khat)", "G = tau[0] * (qhat.T @ khat)", 0)],
    "no_norm_floor": [("qn = np.maximum(np.sqrt((qw * qw).sum(axis=0)), XCA_NORM_FLOOR)",
                       "qn = np.sqrt((qw * qw).sum(axis=0))", 0)],
}


@pytest.mark.parametrize("name", sorted(XCA_MUTANTS))
def test_xca_mutant_is_caught(name):
    mod = _oracle_from_source(XCA_MUTANTS[name])
    with np.errstate(all="ignore"):
        fails = pins.xca_pin_failures(mod.xca_forward_ref, oracle.segments_ref)
    assert fails, f"planted mistake {name} passed every XCA pin"


def test_xca_backward_pins():
    assert pins.xca_backward_pin_failures(oracle.xca_backward_ref, oracle.xca_forward_ref,
                                          oracle.segments_ref) == []


XCA_BWD_MUTANTS = {
    "dv_transposed": [("dv[rows, h, :] = dow @ A", "dv[rows, h, :] = dow @ A.T", 0)],
    "softmax_backward_without_row_term": [("dG = A * (dA - (A * dA).sum(axis=1, keepdims=True))",
                                           "dG = A * dA", 0)],
    "normalisation_backward_without_projection": [("proj = dxh - xh * (xh * dxh).sum(axis=0)",
                                                   "proj = dxh", 0)],
    "dtau_from_logits": [("dtau[h] += (dG * N).sum()", "dtau[h] += (dG * G).sum()", 0)],
    "dkh_transposed": [("dkh = tau[h] * (qh @ dG)", "dkh = tau[h] * (qh @ dG.T)", 0)],
}


@pytest.mark.parametrize("name", sorted(XCA_BWD_MUTANTS))
def test_xca_backward_mutant_is_caught(name):
    mod = _oracle_from_source(XCA_BWD_MUTANTS[name])
    with np.errstate(all="ignore"):
        fails = pins.xca_backward_pin_failures(mod.xca_backward_ref, oracle.xca_forward_ref, oracle.segments_ref)
    assert fails, f"planted mistake {name} passed every XCA backward pin"

"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Builder outputs (perm, offsets, chunk and long-window tables) must match bit
for bit; outputs and
gradients must match within 1e-5 (fp32) or 2e-2 (fp16/bf16) per head, measured
as max|x - ref| / max(max|ref|, floor) with floor = 1e-3 max|v| (o),
1e-3 max|dout| (dv) and 1e-3 max|dout| max|v| (dq, dk).
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import workloads
from tests.gpu_util import TOL, p999, rel_err_per_head, to_dev, to_host64, torch_dtype

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def sla():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2401_00912_amd import sla as S

    S.lib()
    return S


# ------------------------------------------------------------------- helpers
def build(S, ids=None, W=None, chunk_rows=0, offsets=None, n=None):
    import torch

    if ids is not None:
        plan = S.build_segments(to_dev(ids.astype(np.int32)), num_windows=W, chunk_rows=chunk_rows)
    else:
        plan = S.build_segments(None, num_windows=W, chunk_rows=chunk_rows,
                                offsets=to_dev(offsets.astype(np.int32)), n=n)
    torch.cuda.synchronize()
    return plan


def check_plan(S, plan, ids, W, chunk_rows, offsets_in=None):
    header, perm, offs, chunks, longs = S.read_plan(plan)
    L = chunk_rows or 64
    if ids is not None:
        p_ref, o_ref, inv = oracle.segments_ref(ids, W)
        nvalid = len(p_ref)
        assert header["invalid"] == inv
        assert int(plan.invalid.cpu()[0]) == inv
        assert np.array_equal(offs.astype(np.int64), o_ref), "offsets differ"
        assert np.array_equal(perm[:nvalid].astype(np.int64), p_ref), "perm differs"
        # rows outside every window follow, in row order
        outside = np.flatnonzero((ids < 0) | (ids >= W))
        assert np.array_equal(perm[nvalid:].astype(np.int64), outside), "perm tail differs"
        assert np.array_equal(plan.perm.cpu().numpy()[:nvalid].astype(np.int64), p_ref)
        assert np.array_equal(plan.offsets.cpu().numpy().astype(np.int64), o_ref)
        assert header["csr"] == 0
    else:
        o_ref = offsets_in.astype(np.int64)
        assert np.array_equal(offs.astype(np.int64), o_ref)
        assert header["csr"] == 1
    ch_ref, lw_ref, n_four = oracle.chunk_plan_ref(o_ref, L)
    assert header["n_chunks"] == len(ch_ref) and header["n_long"] == len(lw_ref)
    assert header["n_long4"] == n_four
    assert np.array_equal(chunks.astype(np.int64), ch_ref), "chunk table differs"
    assert np.array_equal(longs[:, 0].astype(np.int64), lw_ref), "long-window table differs"
    assert np.array_equal(longs[:, 1].astype(np.int64), o_ref[lw_ref])
    assert np.array_equal(longs[:, 2].astype(np.int64), o_ref[lw_ref + 1])
    assert header["magic"] == 0x534C4132 and header["chunk_rows"] == L
    return o_ref, (p_ref if ids is not None else None)


def run_forward(S, plan, wl_q, wl_k, wl_v, dtype, fmap=None, eps=None):
    import torch

    q, k, v = to_dev(wl_q, dtype), to_dev(wl_k, dtype), to_dev(wl_v, dtype)
    o = torch.full_like(q, float("nan"))
    S.forward(plan, q, k, v, out=o, feature_map=fmap, eps=eps)
    torch.cuda.synchronize()
    return to_host64(o, dtype)


def _oracle_variant(fmap, eps):
    return ("elu1" if fmap is None else fmap), (0.0 if eps is None else eps)


def _match_nan(got, ref, rows, label):
    """Rows of a window: NaN exactly where the oracle has NaN (a zero normaliser
    with eps = 0); those entries are then left out of the error."""
    bad = np.isnan(ref) & rows[:, None, None]
    assert np.array_equal(np.isnan(got) & rows[:, None, None], bad), f"{label}: NaN positions differ"
    if bad.any():
        got, ref = np.where(bad, 0.0, got), np.where(bad, 0.0, ref)
    return got, ref


def forward_parity(S, ids, offsets, n, W, q, k, v, dtype, chunk_rows=0, label="", fmap=None, eps=None):
    plan = build(S, ids=ids, W=W, chunk_rows=chunk_rows, offsets=offsets, n=n)
    off, perm = check_plan(S, plan, ids, W, chunk_rows, offsets)
    got = run_forward(S, plan, q, k, v, dtype, fmap, eps)
    w = lambda a: oracle.widen(a, dtype)  # noqa: E731
    with np.errstate(invalid="ignore", divide="ignore"):
        ref = oracle.sla_forward_ref(w(q), w(k), w(v), off, perm, *_oracle_variant(fmap, eps))
    rows = np.zeros(n, dtype=bool)
    rows[perm if perm is not None else np.arange(off[-1])] = True
    assert np.isnan(ref[~rows]).all()
    g0, r0 = _match_nan(got, ref, rows, label)
    floor = 1e-3 * max(float(np.abs(w(v)).max()) if v.size else 1.0, 1e-30)
    err = rel_err_per_head(g0, r0, floor, rows)
    _say(f"[fwd {label}] n={n} W={W} dtype={dtype} rel_err={err:.3e} p99.9={p999(g0[rows], r0[rows]):.3e}")
    assert err <= TOL[dtype], f"{label}: forward relative error {err:.3e}"
    return got, ref


# Gradients are held to half the 2e-2 bar in fp16 and bf16: the cancelling terms
# of dq and dk (dout S^T against (dout.o) z, v dS^T against dz) run as hi/lo bf16
# pairs, so what is left is the rounding of the stored inputs' images
GRAD_TOL = {"f32": 1e-5, "f16": 1e-2, "bf16": 1e-2}


def backward_parity(S, ids, offsets, n, W, q, k, v, do, dtype, chunk_rows=0, label="", fmap=None,
                    eps=None):
    import torch

    plan = build(S, ids=ids, W=W, chunk_rows=chunk_rows, offsets=offsets, n=n)
    off, perm = check_plan(S, plan, ids, W, chunk_rows, offsets)
    tq, tk, tv, tdo = (to_dev(a, dtype) for a in (q, k, v, do))
    outs = [torch.full_like(tq, float("nan")) for _ in range(3)]
    S.backward(plan, tq, tk, tv, tdo, *outs, feature_map=fmap, eps=eps)
    torch.cuda.synchronize()
    got = [to_host64(t, dtype) for t in outs]
    w = lambda a: oracle.widen(a, dtype)  # noqa: E731
    ref = oracle.sla_backward_ref(w(q), w(k), w(v), w(do), off, perm, *_oracle_variant(fmap, eps))
    rows = ~np.isnan(ref[0][:, 0, 0])
    mv, mdo = float(np.abs(w(v)).max()), float(np.abs(w(do)).max())
    floors = (1e-3 * mdo * mv, 1e-3 * mdo * mv, 1e-3 * mdo)
    for name, x, r, fl in zip(("dq", "dk", "dv"), got, ref, floors):
        err = rel_err_per_head(x, r, fl, rows)
        _say(f"[bwd {label}] {name} n={n} dtype={dtype} rel_err={err:.3e}")
        assert err <= GRAD_TOL[dtype], f"{label}: {name} relative error {err:.3e}"
    return got, ref


# ------------------------------------------------------------------- builder
@pytest.mark.parametrize("cfg", [2, 3, 4, 5])
def test_builder_configs(sla, cfg):
    wl = workloads.make_config(cfg, with_grad=False)
    _say(f"[builder cfg{cfg}] n={wl['n']} W={wl['num_windows']}")
    for L in (0, 32, 48):
        plan = build(sla, ids=wl["ids"], W=wl["num_windows"], chunk_rows=L)
        check_plan(sla, plan, wl["ids"], wl["num_windows"], L)


@pytest.mark.parametrize("seed", range(10))
def test_builder_random(sla, seed):
    rng = np.random.default_rng([7, seed])
    W = int(rng.choice([1, 2, 3, 63, 64, 1000, 4096, 8192, 8193, 16384]))
    n = int(rng.choice([0, 1, 5, 777, 4096, 65537, 130000]))
    ids = rng.integers(0, W, size=n).astype(np.int32)
    if seed % 3 == 1 and n:
        bad = rng.random(n) < 0.01
        ids[bad] = rng.choice([-1, W, W + 5, -(2 ** 31)], size=int(bad.sum()))
    if seed % 4 == 2:
        ids = np.sort(ids)
    L = int(rng.choice([32, 34, 48, 62, 64]))
    _say(f"[builder random {seed}] n={n} W={W} L={L}")
    plan = build(sla, ids=ids, W=W, chunk_rows=L)
    check_plan(sla, plan, ids, W, L)


# sort blocks of 1024, 2048 and 8192 rows, one to ~1000 blocks, already sorted ids
@pytest.mark.parametrize("W,n,L,srt", [(16384, 1_000_000, 64, False), (8193, 100_000, 64, False),
                                       (6000, 65_536, 48, False), (1, 200_000, 32, False),
                                       (2, 65_537, 64, True), (1521, 2_000_000, 64, False),
                                       (300, 4097, 32, True)])
def test_builder_shapes(sla, W, n, L, srt):
    rng = np.random.default_rng([8, W, n])
    ids = rng.integers(0, W, size=n).astype(np.int32)
    if srt:
        ids = np.sort(ids)
    _say(f"[builder shapes] n={n} W={W} L={L} sorted={srt}")
    plan = build(sla, ids=ids, W=W, chunk_rows=L)
    check_plan(sla, plan, ids, W, L)


# the most rows mode A takes (2^26: 8,192 sort blocks of 8,192 rows), with the most
# windows and out-of-range ids, and all rows in one window
@pytest.mark.parametrize("W,bad", [(16384, 0.001), (1, 0.0)])
def test_builder_max_rows(sla, W, bad):
    n = 1 << 26
    rng = np.random.default_rng([10, W])
    ids = rng.integers(0, W, size=n, dtype=np.int32)
    if bad:
        ids[rng.random(n) < bad] = W
    _say(f"[builder max rows] n={n} W={W}")
    plan = build(sla, ids=ids, W=W)
    check_plan(sla, plan, ids, W, 0)


def test_builder_reuses_plan_buffer(sla):
    # one zero-filled buffer rebuilt for other sizes: the builder's window totals sit
    # at a fixed place and every build leaves them zero (block sizes 4096 and 1024)
    import torch

    rng = np.random.default_rng(9)
    cases = [(500_000, 16384), (60_000, 1521), (5, 3), (200_000, 4096), (500_000, 16384), (777, 1)]
    buf = sla.new_plan_buffer(max(n for n, _ in cases), 16384, "cuda")
    for n, W in cases:
        ids = rng.integers(0, W, size=n).astype(np.int32)
        ids[rng.random(n) < 0.002] = W + 3
        _say(f"[builder reuse] n={n} W={W}")
        plan = sla.build_segments(to_dev(ids), num_windows=W, plan_buf=buf)
        torch.cuda.synchronize()
        check_plan(sla, plan, ids, W, 0)


def test_builder_degenerate(sla):
    for ids, W in ((np.zeros(5000, np.int32), 1), (np.full(5000, 7, np.int32), 64),
                   (np.arange(3000, dtype=np.int32)[::-1].copy(), 3000),
                   (np.full(10, -3, np.int32), 4)):
        plan = build(sla, ids=ids, W=W)
        check_plan(sla, plan, ids, W, 0)


def test_builder_csr(sla):
    wl = workloads.make_config(1)
    plan = build(sla, W=wl["num_windows"], offsets=wl["offsets"], n=wl["n"])
    check_plan(sla, plan, None, wl["num_windows"], 0, wl["offsets"])
    # violations are counted and the plan stays in range
    bad = wl["offsets"].copy()
    bad[10], bad[11] = bad[11] + 5, bad[10]
    plan = build(sla, W=wl["num_windows"], offsets=bad, n=wl["n"])
    header, _, offs, chunks, longs = sla.read_plan(plan)
    assert header["invalid"] > 0
    assert np.all(np.diff(offs) >= 0) and offs.min() >= 0 and offs.max() <= wl["n"]
    assert np.all(chunks[:, 0] <= chunks[:, 1]) and chunks[:, 1].max() <= wl["n"]
    assert np.all(longs[:, 1] <= longs[:, 2]) and (longs.size == 0 or longs[:, 2].max() <= wl["n"])


# ------------------------------------------------------------------- forward
@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_forward_config(sla, cfg):
    wl = workloads.make_config(cfg)
    _say(f"[fwd cfg{cfg}] {wl['name']}")
    forward_parity(sla, wl["ids"], wl["offsets"], wl["n"], wl["num_windows"], wl["q"], wl["k"], wl["v"],
                   wl["dtype"], label=f"cfg{cfg}")


SHAPES = [(2, 32), (4, 32), (8, 16), (8, 32), (1, 16), (3, 32)]


def _adversarial_lengths(rng, L):
    return np.array([0, 1, 1, L - 1, L, L + 1, 1024, 2, 0, 0, L // 2, L // 2 + 1, 3, 17, 33, 31, 32,
                     64, 65, 1, 100, 5], dtype=np.int64)[rng.permutation(22)]


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", SHAPES)
def test_forward_shapes(sla, dtype, shape):
    H, d = shape
    rng = np.random.default_rng([11, H, d, len(dtype)])
    lengths = _adversarial_lengths(rng, 128)
    ids = workloads.ids_from_lengths(lengths, rng)
    n, W = ids.size, lengths.size
    q, k, v = (workloads.normal_values(rng, n, H, d, dtype) for _ in range(3))
    forward_parity(sla, ids, None, n, W, q, k, v, dtype, label=f"shape{shape}")


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_forward_special_layouts(sla, dtype):
    rng = np.random.default_rng([12, len(dtype)])
    H, d = 4, 32
    cases = {
        "one_window": np.array([3000]),
        "all_singletons": np.ones(2000, dtype=np.int64),
        "empty_slots": np.array([0, 0, 5, 0, 0, 0, 40, 0]),
        "long_window": np.array([2500, 3, 1]),
    }
    for name, lengths in cases.items():
        ids = workloads.ids_from_lengths(lengths, rng)
        n, W = ids.size, lengths.size
        q, k, v = (workloads.normal_values(rng, n, H, d, dtype) for _ in range(3))
        got, ref = forward_parity(sla, ids, None, n, W, q, k, v, dtype, label=name)
        if name == "all_singletons":
            vv = oracle.widen(v, dtype)
            assert rel_err_per_head(got, vv, 1e-3) <= TOL[dtype]


@pytest.mark.parametrize("L", [32, 48, 64])
def test_forward_chunk_rows(sla, L):
    wl = workloads.make_config(2)
    forward_parity(sla, wl["ids"], None, wl["n"], wl["num_windows"], wl["q"], wl["k"], wl["v"], wl["dtype"],
                   chunk_rows=L, label=f"L{L}")


def test_forward_large_values(sla):
    # operands are scaled before rounding to 16 bits: big windows of big values must not overflow
    rng = np.random.default_rng(13)
    lengths = np.array([1024, 500, 7, 1])
    ids = workloads.ids_from_lengths(lengths, rng)
    n = ids.size
    q = workloads.cast_values(rng.standard_normal((n, 2, 32)).astype(np.float32) * 4, "f16")
    k = workloads.cast_values(rng.standard_normal((n, 2, 32)).astype(np.float32) * 4, "f16")
    v = workloads.cast_values(rng.standard_normal((n, 2, 32)).astype(np.float32) * 3000, "f16")
    forward_parity(sla, ids, None, n, 4, q, k, v, "f16", label="large")


def test_forward_window_independence_and_determinism(sla):
    import torch

    wl = workloads.make_config(2)
    dtype = wl["dtype"]
    plan = build(sla, ids=wl["ids"], W=wl["num_windows"])
    a = run_forward(sla, plan, wl["q"], wl["k"], wl["v"], dtype)
    b = run_forward(sla, plan, wl["q"], wl["k"], wl["v"], dtype)
    assert np.array_equal(a, b), "repeat runs differ"
    # change every value outside window 0 of the rows' windows: window 0's rows are unchanged
    target = int(np.bincount(wl["ids"]).argmax())
    other = wl["ids"] != target
    q2, k2, v2 = wl["q"].copy(), wl["k"].copy(), wl["v"].copy()
    q2[other] = -q2[other]
    k2[other] = k2[other] * 2
    v2[other] = v2[other] + 1
    c = run_forward(sla, plan, q2, k2, v2, dtype)
    mine = ~other
    assert np.array_equal(a[mine], c[mine])
    torch.cuda.synchronize()


def test_n_zero(sla):
    import torch

    plan = build(sla, ids=np.zeros(0, np.int32), W=5)
    header, _, offs, chunks, longs = sla.read_plan(plan)
    assert header["n_chunks"] == 0 and header["n_long"] == 0 and np.all(offs == 0)
    q = torch.empty((0, 2, 32), dtype=torch.float16, device="cuda")
    sla.forward(plan, q, q, q)
    sla.backward(plan, q, q, q, q)
    torch.cuda.synchronize()


# ------------------------------------------------------------------ backward
def test_backward_config5(sla):
    wl = workloads.make_config(5)
    _say(f"[bwd cfg5] {wl['name']}")
    backward_parity(sla, wl["ids"], None, wl["n"], wl["num_windows"], wl["q"], wl["k"], wl["v"], wl["dout"],
                    wl["dtype"], label="cfg5")
    # cfg 5 re-shuffles rows every iteration: a re-shuffled frame must also match
    sh = workloads.shuffled(wl, [5, 2, 0])
    backward_parity(sla, sh["ids"], None, sh["n"], sh["num_windows"], sh["q"], sh["k"], sh["v"], sh["dout"],
                    sh["dtype"], label="cfg5-shuffled")
    forward_parity(sla, sh["ids"], None, sh["n"], sh["num_windows"], sh["q"], sh["k"], sh["v"], sh["dtype"],
                   label="cfg5-shuffled")


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", SHAPES)
def test_backward_shapes(sla, dtype, shape):
    H, d = shape
    rng = np.random.default_rng([21, H, d, len(dtype)])
    lengths = _adversarial_lengths(rng, 128)
    ids = workloads.ids_from_lengths(lengths, rng)
    n, W = ids.size, lengths.size
    q, k, v, do = (workloads.normal_values(rng, n, H, d, dtype) for _ in range(4))
    backward_parity(sla, ids, None, n, W, q, k, v, do, dtype, label=f"shape{shape}")


def test_backward_csr_fp32(sla):
    wl = workloads.make_config(1, with_grad=True)
    backward_parity(sla, None, wl["offsets"], wl["n"], wl["num_windows"], wl["q"], wl["k"], wl["v"],
                    wl["dout"], wl["dtype"], label="cfg1-bwd")


def test_backward_determinism(sla):
    import torch

    wl = workloads.make_config(5)
    plan = build(sla, ids=wl["ids"], W=wl["num_windows"])
    tq, tk, tv, tdo = (to_dev(wl[x], "f16") for x in ("q", "k", "v", "dout"))
    r1 = [t.clone() for t in sla.backward(plan, tq, tk, tv, tdo)]
    r2 = sla.backward(plan, tq, tk, tv, tdo)
    torch.cuda.synchronize()
    for a, b in zip(r1, r2):
        assert torch.equal(a, b)


def test_streams_share_a_plan(sla):
    # the interface allows forward and backward calls on different streams to
    # read one plan at the same time: two streams (default priority) run their
    # own inputs through it, interleaved, and every result must equal the
    # sequential one bit for bit
    import torch

    wl = workloads.make_config(5)
    plan = build(sla, ids=wl["ids"], W=wl["num_windows"])
    rng = np.random.default_rng(68)
    sets = []
    for _ in range(2):
        q, k, v, do = (to_dev(workloads.cast_values(rng.standard_normal(wl["q"].shape).astype(np.float32), "f16"),
                              "f16") for _ in range(4))
        sets.append((q, k, v, do))
    ref = []
    for q, k, v, do in sets:
        o = sla.forward(plan, q, k, v)
        ref.append([o.clone()] + [t.clone() for t in sla.backward(plan, q, k, v, do)])
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [[torch.empty_like(sets[i][0]) for _ in range(4)] for i in range(2)]
    for s_ in streams:
        s_.wait_stream(torch.cuda.current_stream())
    for _ in range(3):
        for i, s_ in enumerate(streams):
            with torch.cuda.stream(s_):
                q, k, v, do = sets[i]
                sla.forward(plan, q, k, v, out=outs[i][0])
                sla.backward(plan, q, k, v, do, outs[i][1], outs[i][2], outs[i][3])
    torch.cuda.synchronize()
    for i in range(2):
        for a, b in zip(ref[i], outs[i]):
            assert torch.equal(a, b)


def test_graph_replays(sla):
    # the whole path captured in one HIP graph (segment build, forward, backward,
    # their ReLU / eps variants, the XCA forward and backward, the fused projection, cell
    # table, cross-window interaction forward and backward), replayed three
    # times; before each replay the outputs, the plan buffer and the cell table
    # are scribbled over by eager work, and every replay must reproduce the eager
    # results bit for bit
    import torch

    wl = workloads.make_config(5)
    W = wl["num_windows"]
    ids = to_dev(wl["ids"].astype(np.int32))
    q, k, v, do = (to_dev(wl[x], "f16") for x in ("q", "k", "v", "dout"))
    f = workloads.make_cwi_frame()
    grid = f["grid"]
    cc = torch.from_numpy(f["coords"]).cuda()
    x = to_dev(f["x"], "f16")
    w = [to_dev(f[key], "f16") for key in ("w_x", "w_y", "w_3")]
    dy = to_dev(workloads.cast_values(np.random.default_rng(69).standard_normal(f["x"].shape).astype(np.float32),
                                      "f16"), "f16")

    n, H, d = q.shape
    C = H * d
    rng = np.random.default_rng(70)
    xp = to_dev(workloads.cast_values(rng.standard_normal((n, C)).astype(np.float32), "f16"), "f16")
    wq = to_dev(workloads.cast_values((rng.standard_normal((3 * C, C)) / np.sqrt(C)).astype(np.float32), "f16"),
                "f16")
    wo = to_dev(workloads.cast_values((rng.standard_normal((C, C)) / np.sqrt(C)).astype(np.float32), "f16"), "f16")
    tau = torch.tensor(np.linspace(0.5, 3.0, H), dtype=torch.float32, device="cuda")

    def path():
        plan = sla.build_segments(ids, num_windows=W)
        o = sla.forward(plan, q, k, v)
        grads = sla.backward(plan, q, k, v, do)
        o_relu = sla.forward(plan, q, k, v, feature_map="relu", eps=1e-3)
        grads_relu = sla.backward(plan, q, k, v, do, feature_map="relu", eps=1e-3)
        o_xca = sla.forward_xca(plan, q, k, v, tau)
        g_xca = sla.backward_xca(plan, q, k, v, tau, do)
        po = torch.empty((n, H, d), dtype=torch.float16, device="cuda")
        py = torch.empty((n, C), dtype=torch.float16, device="cuda")
        sla.forward_projected(plan, xp, wq, wo, H, None, None, po, py)
        m, _ = sla.cwi_build_map(cc, grid)
        y = sla.cwi_forward(m, grid, cc, x, *w)
        back = sla.cwi_backward(m, grid, cc, x, *w, dy)
        return plan, m, [o, *grads, o_relu, *grads_relu, o_xca, *g_xca, po, py, y, *back]

    _, _, eager = path()
    eager = [t.clone() for t in eager]
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            plan_g, map_g, outs = path()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in outs:
            t.fill_(float("nan"))
        plan_g.buf.fill_(0xA5)
        map_g.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(eager, outs)):
            assert torch.equal(a, b), f"replay {rep}: output {i} differs from the eager result"


# ------------------------------------------------------- naive comparator
def scatter_parity(S, ids, offsets, n, W, q, k, v, dtype, label=""):
    import torch

    plan = build(S, ids=ids, W=W, offsets=offsets, n=n)
    off, perm = check_plan(S, plan, ids, W, 0, offsets)
    tq, tk, tv = to_dev(q, dtype), to_dev(k, dtype), to_dev(v, dtype)
    o = torch.full_like(tq, float("nan"))
    S.forward_scatter(plan, tq, tk, tv, out=o)
    torch.cuda.synchronize()
    got = to_host64(o, dtype)
    w = lambda a: oracle.widen(a, dtype)  # noqa: E731
    ref = oracle.sla_forward_ref(w(q), w(k), w(v), off, perm)
    rows = ~np.isnan(ref[:, 0, 0])
    floor = 1e-3 * max(float(np.abs(w(v)).max()) if v.size else 1.0, 1e-30)
    err = rel_err_per_head(got, ref, floor, rows)
    _say(f"[scatter {label}] n={n} W={W} dtype={dtype} rel_err={err:.3e}")
    assert err <= TOL[dtype], f"{label}: scatter forward relative error {err:.3e}"
    assert np.isnan(got[~rows]).all(), "rows outside every window were written"


@pytest.mark.parametrize("cfg", [1, 2])
def test_forward_scatter_config(sla, cfg):
    wl = workloads.make_config(cfg)
    scatter_parity(sla, wl["ids"], wl["offsets"], wl["n"], wl["num_windows"], wl["q"], wl["k"], wl["v"],
                   wl["dtype"], label=f"cfg{cfg}")


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", [(2, 32), (8, 16), (3, 32)])
def test_forward_scatter_shapes(sla, dtype, shape):
    H, d = shape
    rng = np.random.default_rng([31, H, d, len(dtype)])
    lengths = _adversarial_lengths(rng, 128)
    ids = workloads.ids_from_lengths(lengths, rng)
    ids[rng.random(ids.size) < 0.01] = -1          # rows outside every window stay unwritten
    n, W = ids.size, lengths.size
    q, k, v = (workloads.normal_values(rng, n, H, d, dtype) for _ in range(3))
    scatter_parity(sla, ids, None, n, W, q, k, v, dtype, label=f"shape{shape}")


# ------------------------------------------- feature-map variants and epsilon
VARIANTS = [("relu", 0.0), ("relu", 1e-3), ("elu1", 0.5)]


@pytest.mark.parametrize("fmap,eps", VARIANTS)
@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_variant_forward_config(sla, cfg, fmap, eps):
    # with eps = 0 some ReLU rows of config 3 (d = 16, singleton windows) have a
    # zero normaliser: NaN on both sides, checked position by position
    wl = workloads.make_config(cfg)
    forward_parity(sla, wl["ids"], wl["offsets"], wl["n"], wl["num_windows"], wl["q"], wl["k"], wl["v"],
                   wl["dtype"], label=f"cfg{cfg}-{fmap}-{eps}", fmap=fmap, eps=eps)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", [(2, 32), (8, 16), (3, 32)])
def test_variant_forward_shapes(sla, dtype, shape):
    H, d = shape
    rng = np.random.default_rng([41, H, d, len(dtype)])
    lengths = _adversarial_lengths(rng, 128)
    ids = workloads.ids_from_lengths(lengths, rng)
    n, W = ids.size, lengths.size
    q, k, v = (workloads.normal_values(rng, n, H, d, dtype) for _ in range(3))
    for fmap, eps in (("relu", 1e-4), ("elu1", 0.25)):
        forward_parity(sla, ids, None, n, W, q, k, v, dtype, label=f"shape{shape}-{fmap}", fmap=fmap, eps=eps)


@pytest.mark.parametrize("fmap,eps", [("relu", 1e-6), ("relu", 0.05), ("elu1", 1e-3)])
def test_variant_backward_config5(sla, fmap, eps):
    wl = workloads.make_config(5)
    backward_parity(sla, wl["ids"], None, wl["n"], wl["num_windows"], wl["q"], wl["k"], wl["v"], wl["dout"],
                    wl["dtype"], label=f"cfg5-{fmap}-{eps}", fmap=fmap, eps=eps)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", [(2, 32), (8, 16), (3, 32)])
def test_variant_backward_shapes(sla, dtype, shape):
    H, d = shape
    rng = np.random.default_rng([42, H, d, len(dtype)])
    lengths = _adversarial_lengths(rng, 128)
    ids = workloads.ids_from_lengths(lengths, rng)
    n, W = ids.size, lengths.size
    q, k, v, do = (workloads.normal_values(rng, n, H, d, dtype) for _ in range(4))
    for fmap, eps in (("relu", 1e-4), ("elu1", 0.25)):
        backward_parity(sla, ids, None, n, W, q, k, v, do, dtype, label=f"shape{shape}-{fmap}", fmap=fmap,
                        eps=eps)


def test_variant_default_is_plain(sla):
    # the _ex calls with elu + 1 and eps = 0 are the plain calls, bit for bit
    import torch

    wl = workloads.make_config(5)
    plan = build(sla, ids=wl["ids"], W=wl["num_windows"])
    tq, tk, tv, tdo = (to_dev(wl[x], "f16") for x in ("q", "k", "v", "dout"))
    assert torch.equal(sla.forward(plan, tq, tk, tv), sla.forward(plan, tq, tk, tv, feature_map="elu1", eps=0.0))
    a = sla.backward(plan, tq, tk, tv, tdo)
    b = sla.backward(plan, tq, tk, tv, tdo, feature_map="elu1", eps=0.0)
    torch.cuda.synchronize()
    assert all(torch.equal(x, y) for x, y in zip(a, b))


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_variant_relu_zero_rows(sla, dtype):
    # a query with no positive entry, and a window whose keys have none: o = 0
    # exactly with eps > 0, NaN with eps = 0 (the oracle agrees position by position)
    rng = np.random.default_rng([43, len(dtype)])
    lengths = np.array([40, 1, 70, 5, 200, 1])
    ids = workloads.ids_from_lengths(lengths, rng)
    n, H, d = ids.size, 2, 32
    q, k, v = (rng.standard_normal((n, H, d)).astype(np.float32) for _ in range(3))
    zq = rng.random(n) < 0.1                                  # queries with no positive entry
    q[zq] = -np.abs(q[zq])
    zk = (ids == 1) | (ids == 3)                              # windows whose keys have none
    k[zk] = -np.abs(k[zk])
    q, k, v = (workloads.cast_values(x, dtype) for x in (q, k, v))
    got, _ = forward_parity(sla, ids, None, n, lengths.size, q, k, v, dtype, label="relu-zero", fmap="relu",
                            eps=1e-3)
    assert np.all(got[zq] == 0.0) and np.all(got[zk] == 0.0)
    got0, ref0 = forward_parity(sla, ids, None, n, lengths.size, q, k, v, dtype, label="relu-zero-eps0",
                                fmap="relu", eps=0.0)
    assert np.isnan(got0[zq | zk]).all() and np.isnan(ref0[zq | zk]).all()


def test_variant_relu_absent_features(sla):
    # features that no key of a window has (z_e = 0) while the queries are large
    # on them and small elsewhere: the state-gradient operands must stay finite in
    # fp16 (those features reach neither dk nor dv) and match the oracle
    rng = np.random.default_rng(44)
    lengths = np.array([300, 40, 3, 1, 65])
    ids = workloads.ids_from_lengths(lengths, rng)
    n, H, d = ids.size, 2, 32
    q, k, v, do = (rng.standard_normal((n, H, d)).astype(np.float32) for _ in range(4))
    k[:, :, :8] = -np.abs(k[:, :, :8]) - 0.01                 # features 0..7 absent from every key
    q[:, :, :8] = np.abs(q[:, :, :8]) * 60 + 100
    few = rng.random(n) < 0.3                                 # rows active on one tiny feature only
    q[few, :, 8:] = -1.0
    q[few, :, 8] = 1e-3
    q, k, v, do = (workloads.cast_values(x, "f16") for x in (q, k, v, do))
    W = lengths.size
    for eps in (1e-6, 0.1):
        forward_parity(sla, ids, None, n, W, q, k, v, "f16", label=f"absent-{eps}", fmap="relu", eps=eps)
        backward_parity(sla, ids, None, n, W, q, k, v, do, "f16", label=f"absent-{eps}", fmap="relu", eps=eps)


# ------------------------------------------------- projection fused into SLA
def projected_parity(S, ids, offsets, n, W, H, d, dtype, fmap="elu1", eps=0.0, bias=True, seed=0,
                     label="", chunk_rows=0):
    import torch

    rng = np.random.default_rng([51, seed, H, d])
    C = H * d
    cast = lambda a: workloads.cast_values(np.asarray(a, dtype=np.float32), dtype)  # noqa: E731
    x = cast(rng.standard_normal((n, C)))
    wq = cast(rng.standard_normal((3 * C, C)) / np.sqrt(C))
    wo = cast(rng.standard_normal((C, C)) / np.sqrt(C))
    bq = cast(0.2 * rng.standard_normal(3 * C)) if bias else None
    bo = cast(0.2 * rng.standard_normal(C)) if bias else None
    plan = build(S, ids=ids, W=W, chunk_rows=chunk_rows, offsets=offsets, n=n)
    off, perm = check_plan(S, plan, ids, W, chunk_rows, offsets)
    dev = lambda a: None if a is None else to_dev(a, dtype)  # noqa: E731
    o = torch.full((n, H, d), float("nan"), dtype=torch_dtype(dtype), device="cuda")
    y = torch.full((n, C), float("nan"), dtype=torch_dtype(dtype), device="cuda")
    S.forward_projected(plan, dev(x), dev(wq), dev(wo), H, dev(bq), dev(bo), o, y, fmap, eps)
    torch.cuda.synchronize()
    go, gy = to_host64(o, dtype), to_host64(y, dtype)
    w = lambda a: None if a is None else oracle.widen(a, dtype)  # noqa: E731
    with np.errstate(invalid="ignore", divide="ignore"):
        ro, ry = oracle.sla_projected_forward_ref(w(x), w(wq), w(bq), w(wo), w(bo), H, off, perm, fmap, eps)
    rows = np.zeros(n, dtype=bool)
    rows[perm if perm is not None else np.arange(off[-1])] = True
    assert np.isnan(go[~rows]).all() and np.isnan(gy[~rows]).all(), "rows in no window were written"
    g0, r0 = _match_nan(go, ro, rows, label)
    gy3, ry3 = _match_nan(gy.reshape(n, H, d), ry.reshape(n, H, d), rows, label)
    eo = rel_err_per_head(g0, r0, 1e-3 * float(np.nanmax(np.abs(r0))) if rows.any() else 1.0, rows)
    ey = rel_err_per_head(gy3, ry3, 1e-3 * float(np.nanmax(np.abs(ry3))) if rows.any() else 1.0, rows)
    _say(f"[proj {label}] n={n} H={H} d={d} {dtype} {fmap} eps={eps} o rel_err={eo:.3e} y rel_err={ey:.3e}")
    assert eo <= TOL[dtype], f"{label}: o relative error {eo:.3e}"
    assert ey <= TOL[dtype], f"{label}: y relative error {ey:.3e}"


@pytest.mark.parametrize("cfg", [2, 3, 4, 5])
def test_projected_config(sla, cfg):
    # config 3 (bf16, H = 8, d = 16) has windows of up to 1,024 rows: quarters of
    # more than 64 rows take the streamed path; config 4 (bf16, H = 8, d = 32) has
    # C = 256, whose features are fetched and projected one 32-row job at a time
    wl = workloads.make_config(cfg, with_grad=False)
    projected_parity(sla, wl["ids"], wl["offsets"], wl["n"], wl["num_windows"], wl["heads"], wl["head_dim"],
                     wl["dtype"], label=f"cfg{cfg}")


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("shape", [(4, 32), (8, 16), (2, 32), (4, 16), (8, 32), (16, 16)])
def test_projected_shapes(sla, dtype, shape):
    H, d = shape
    rng = np.random.default_rng([52, H, d, len(dtype)])
    lengths = _adversarial_lengths(rng, 128)
    ids = workloads.ids_from_lengths(lengths, rng)
    ids[rng.random(ids.size) < 0.01] = -1          # rows outside every window stay unwritten
    n, W = ids.size, lengths.size
    projected_parity(sla, ids, None, n, W, H, d, dtype, seed=1, label=f"shape{shape}")
    projected_parity(sla, ids, None, n, W, H, d, dtype, fmap="relu", eps=1e-3, bias=False, seed=2,
                     label=f"shape{shape}-relu")


def test_projected_csr_and_chunk_rows(sla):
    wl = workloads.make_config(2, with_grad=False)
    perm, off, _ = oracle.segments_ref(wl["ids"], wl["num_windows"])
    # rows already window-sorted: CSR mode, no permutation
    projected_parity(sla, None, off, wl["n"], wl["num_windows"], 4, 32, "f16", seed=3, label="csr")
    projected_parity(sla, wl["ids"], None, wl["n"], wl["num_windows"], 4, 32, "f16", seed=4, label="L32",
                     chunk_rows=32)


def test_projected_long_windows(sla):
    # four-way windows above 256 rows (streamed), two-way windows with an odd
    # count (a pair whose second window is missing), and a one-window scene
    rng = np.random.default_rng(53)
    for lengths in (np.array([700, 300, 257, 256, 100, 90, 70, 3, 1]), np.array([2000]), np.array([65])):
        ids = workloads.ids_from_lengths(lengths, rng)
        for dtype in ("f16", "bf16"):
            projected_parity(sla, ids, None, ids.size, lengths.size, 4, 32, dtype, seed=5,
                             label=f"long{lengths.size}")


# ---------------------------------------------------------- projected backward
def projected_backward_parity(S, ids, offsets, n, W, H, d, dtype, fmap="elu1", eps=0.0, bias=True, seed=0,
                              label=""):
    import torch

    rng = np.random.default_rng([57, seed, H, d])
    C = H * d
    cast = lambda a: workloads.cast_values(np.asarray(a, dtype=np.float32), dtype)  # noqa: E731
    x = cast(rng.standard_normal((n, C)))
    wq = cast(rng.standard_normal((3 * C, C)) / np.sqrt(C))
    wo = cast(rng.standard_normal((C, C)) / np.sqrt(C))
    bq = cast(0.2 * rng.standard_normal(3 * C)) if bias else None
    bo = cast(0.2 * rng.standard_normal(C)) if bias else None
    dy = cast(rng.standard_normal((n, C)))
    plan = build(S, ids=ids, W=W, offsets=offsets, n=n)
    off, perm = check_plan(S, plan, ids, W, 0, offsets)
    dev = lambda a: None if a is None else to_dev(a, dtype)  # noqa: E731
    tx, twq, two, tbq, tdy = dev(x), dev(wq), dev(wo), dev(bq), dev(dy)
    o, _ = S.forward_projected(plan, tx, twq, two, H, tbq, dev(bo), None, None, fmap, eps)
    dx = torch.full((n, C), float("nan"), dtype=torch_dtype(dtype), device="cuda")
    got = S.backward_projected(plan, tx, twq, two, o, tdy, H, tbq, fmap, eps, dx=dx)
    torch.cuda.synchronize()
    gdx = to_host64(got[0], dtype)
    gw = [t.cpu().numpy().astype(np.float64) for t in got[1:]]
    w = lambda a: None if a is None else oracle.widen(a, dtype)  # noqa: E731
    ref = oracle.sla_projected_backward_ref(w(x), w(wq), w(bq), w(wo), w(bo), w(dy), H, off, perm, fmap, eps)
    rows = np.zeros(n, dtype=bool)
    rows[perm if perm is not None else np.arange(off[-1])] = True
    assert np.all(gdx[~rows] == 0.0), f"{label}: dx of rows in no window is not zero"
    edx = rel_err_per_head(gdx.reshape(n, H, d), ref[0].reshape(n, H, d), 1e-3 * float(np.abs(ref[0]).max()),
                           rows)
    names = ("dw_qkv", "db_qkv", "dw_o", "db_o")
    errs = []
    for name, g, r in zip(names, gw, ref[1:]):
        assert np.all(np.isfinite(g)), f"{label}: {name} not finite"
        errs.append(float(np.abs(g - r).max()) / max(float(np.abs(r).max()), 1e-30))
    _say(f"[proj-bwd {label}] n={n} H={H} d={d} {dtype} {fmap} eps={eps} dx {edx:.3e} "
         + " ".join(f"{nm} {e:.3e}" for nm, e in zip(names, errs)))
    assert edx <= TOL[dtype], f"{label}: dx relative error {edx:.3e}"
    for nm, e in zip(names, errs):
        assert e <= TOL[dtype], f"{label}: {nm} relative error {e:.3e}"
    return got


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_projected_backward_config(sla, cfg):
    wl = workloads.make_config(cfg, with_grad=False)
    projected_backward_parity(sla, wl["ids"], None, wl["n"], wl["num_windows"], wl["heads"], wl["head_dim"],
                              wl["dtype"], label=f"cfg{cfg}")


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("shape", [(2, 32), (8, 16), (4, 16), (16, 16)])
def test_projected_backward_shapes(sla, dtype, shape):
    # adversarial window lengths, 1% of the rows in no window, both maps
    H, d = shape
    rng = np.random.default_rng([58, H, d, len(dtype)])
    lengths = _adversarial_lengths(rng, 128)
    ids = workloads.ids_from_lengths(lengths, rng)
    ids[rng.random(ids.size) < 0.01] = -1
    n, W = ids.size, lengths.size
    projected_backward_parity(sla, ids, None, n, W, H, d, dtype, seed=1, label=f"shape{shape}")
    projected_backward_parity(sla, ids, None, n, W, H, d, dtype, fmap="relu", eps=1e-3, bias=False, seed=2,
                              label=f"shape{shape}-relu")


@pytest.mark.parametrize("dtype,shape,long", [("f16", (4, 32), False), ("bf16", (8, 32), False),
                                              ("f16", (2, 32), True), ("bf16", (8, 16), True)])
def test_projected_saved_qkv(sla, dtype, shape, long):
    # the forward's saved q, k, v: the projection of x (checked against float64
    # from the same rounded inputs), o and y unchanged by saving, and the
    # backward that reads them equal, bit for bit, to the one that recomputes
    # them (the same products in the same order).  `long` adds a window of 1,024
    # rows, whose shares are projected job by job (streamed).  d = 16 stores its
    # fragments as four 8-byte pieces, d = 32 (16-bit) as one 16-byte piece.
    import torch

    H, d = shape
    C = H * d
    rng = np.random.default_rng([59, H, d, int(long)])
    lengths = _adversarial_lengths(rng, 64) if long else rng.integers(1, 90, size=48)
    ids = workloads.ids_from_lengths(np.asarray(lengths, dtype=np.int64), rng)
    ids[rng.random(ids.size) < 0.01] = -1
    n, W = ids.size, len(lengths)
    cast = lambda a: workloads.cast_values(np.asarray(a, dtype=np.float32), dtype)  # noqa: E731
    x = cast(rng.standard_normal((n, C)))
    wq = cast(rng.standard_normal((3 * C, C)) / np.sqrt(C))
    wo = cast(rng.standard_normal((C, C)) / np.sqrt(C))
    bq = cast(0.2 * rng.standard_normal(3 * C))
    dy = cast(rng.standard_normal((n, C)))
    plan = build(sla, ids=ids, W=W)
    off, perm = check_plan(sla, plan, ids, W, 0)
    tx, twq, two, tbq, tdy = (to_dev(a, dtype) for a in (x, wq, wo, bq, dy))
    zeros = lambda *shape: torch.zeros(shape, dtype=torch_dtype(dtype), device="cuda")  # noqa: E731
    o0, y0 = sla.forward_projected(plan, tx, twq, two, H, tbq, None, zeros(n, H, d), zeros(n, C))
    qkv = torch.full((3, n, C), float("nan"), dtype=torch_dtype(dtype), device="cuda")
    o1, y1 = sla.forward_projected(plan, tx, twq, two, H, tbq, None, zeros(n, H, d), zeros(n, C), qkv_out=qkv)
    torch.cuda.synchronize()
    assert torch.equal(o0, o1) and torch.equal(y0, y1), "saving q, k, v changed o or y"
    rows = np.zeros(n, dtype=bool)
    rows[perm[: off[-1]] if perm is not None else np.arange(off[-1])] = True
    w = lambda a: oracle.widen(a, dtype)  # noqa: E731
    ref = w(x) @ w(wq).T + w(bq)
    got = to_host64(qkv, dtype)
    for m, name in enumerate("qkv"):
        e = rel_err_per_head(got[m].reshape(n, H, d), ref[:, m * C:(m + 1) * C].reshape(n, H, d),
                             1e-3 * float(np.abs(ref).max()), rows)
        assert e <= (2e-3 if dtype == "f16" else 1e-2), f"saved {name}: {e:.2e}"
    a = sla.backward_projected(plan, tx, twq, two, o1, tdy, H, tbq)
    b = sla.backward_projected(plan, tx, twq, two, o1, tdy, H, tbq, qkv=qkv)
    torch.cuda.synchronize()
    for name, ta, tb in zip(("dx", "dw_qkv", "db_qkv", "dw_o", "db_o"), a, b):
        assert torch.equal(ta, tb), f"{name} differs between recomputed and saved q, k, v"


@pytest.mark.parametrize("dtype,shape", [("f16", (2, 32)), ("bf16", (8, 32))])
def test_projected_backward_tiny(sla, dtype, shape):
    # fewer rows than one 16-row tile: the row products' and the weight
    # gradients' grids are mostly idle (padded to whole blocks of 8 row ranges
    # or groups), one row lies in no window
    H, d = shape
    ids = np.array([1, 0, -1, 1, 1], dtype=np.int32)
    projected_backward_parity(sla, ids, None, ids.size, 3, H, d, dtype, seed=3, label=f"tiny{shape}")


def test_projected_backward_csr_and_determinism(sla):
    import torch

    wl = workloads.make_config(2, with_grad=False)
    perm, off, _ = oracle.segments_ref(wl["ids"], wl["num_windows"])
    a = projected_backward_parity(sla, None, off, wl["n"], wl["num_windows"], 4, 32, "f16", seed=3, label="csr")
    b = projected_backward_parity(sla, None, off, wl["n"], wl["num_windows"], 4, 32, "f16", seed=3, label="csr")
    for x, y in zip(a, b):
        assert torch.equal(x, y), "two runs differ"


# ---------------------------------------------------- cross-window interaction
def cwi_parity(S, coords, grid, x, w_x, w_y, w_3, dtype, order=None, label=""):
    import torch

    cc = torch.from_numpy(np.ascontiguousarray(coords.astype(np.int32))).cuda()
    m, conflicts = S.cwi_build_map(cc, grid)
    tord = None if order is None else torch.from_numpy(np.ascontiguousarray(order.astype(np.int32))).cuda()
    dev = lambda a: to_dev(a, dtype)  # noqa: E731
    y = torch.full(x.shape, float("nan"), dtype=torch_dtype(dtype), device="cuda")
    S.cwi_forward(m, grid, cc, dev(x), dev(w_x), dev(w_y), dev(w_3), order=tord, y=y)
    torch.cuda.synchronize()
    assert int(conflicts.cpu()[0]) == 0
    got = to_host64(y, dtype)
    w = lambda a: oracle.widen(a, dtype)  # noqa: E731
    ref = oracle.cwi_forward_ref(coords, w(x), w(w_x), w(w_y), w(w_3), grid)
    n, C = x.shape
    err = rel_err_per_head(got.reshape(n, 4, C // 4), ref.reshape(n, 4, C // 4),
                           1e-3 * float(np.abs(ref).max()) if n else 1.0)
    _say(f"[cwi {label}] n={n} C={C} grid={grid} {dtype} rel_err={err:.3e}")
    assert err <= TOL[dtype], f"{label}: CWI relative error {err:.3e}"
    # the identity branch is a copy, bit for bit
    assert np.array_equal(got[:, 3 * C // 4:], w(x)[:, 3 * C // 4:])
    return m


def test_cwi_frame(sla):
    # a Waymo-like pillar frame, visited in the SLA plan's window order and in row order
    f = workloads.make_cwi_frame()
    perm, _, _ = oracle.segments_ref(f["ids"], f["num_windows"])
    for order in (perm, None):
        cwi_parity(sla, f["coords"], f["grid"], f["x"], f["w_x"], f["w_y"], f["w_3"], f["dtype"], order=order,
                   label="frame" + ("-window-order" if order is not None else ""))


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("C,kx,ky", [(32, 13, 13), (64, 5, 31), (128, 1, 63), (256, 13, 3)])
def test_cwi_voxels(sla, dtype, C, kx, ky):
    # 3D voxel grids (the 3 x 3 x 3 branch sees all its z taps), random occupancy
    # including runs along both axes, rows shuffled
    if dtype == "f32" and C == 32:
        C = 16
    rng = np.random.default_rng([61, C, kx, len(dtype)])
    grid = (37, 29, 5)
    occ = rng.random(grid[::-1]) < 0.3
    zz, yy, xx = np.nonzero(occ)
    coords = np.stack([xx, yy, zz], axis=1)[rng.permutation(zz.size)]
    n, c = coords.shape[0], C // 4
    cast = lambda a: workloads.cast_values(a.astype(np.float32), dtype)  # noqa: E731
    x = cast(rng.standard_normal((n, C)))
    w_x, w_y, w_3 = (cast(rng.standard_normal((k, c)) / np.sqrt(k)) for k in (kx, ky, 27))
    cwi_parity(sla, coords, grid, x, w_x, w_y, w_3, dtype, order=rng.permutation(n), label=f"vox{C}")


def test_cwi_conflicts_and_empty(sla):
    import torch

    coords = np.array([[1, 1, 0], [2, 1, 0], [1, 1, 0], [9, 0, 0], [0, 7, 0]], dtype=np.int32)
    m, conflicts = sla.cwi_build_map(torch.from_numpy(coords).cuda(), (8, 8, 1))
    torch.cuda.synchronize()
    assert int(conflicts.cpu()[0]) == 2                      # a taken cell, a cell outside the grid
    table = m.cpu().numpy().reshape(8, 8)
    assert table[1, 1] == 2 and table[1, 2] == 1 and table[7, 0] == 4 and (table >= 0).sum() == 3
    m0, c0 = sla.cwi_build_map(torch.zeros((0, 3), dtype=torch.int32, device="cuda"), (4, 4, 2))
    torch.cuda.synchronize()
    assert int(c0.cpu()[0]) == 0 and bool((m0 == -1).all())


CWI_DW_TOL = {"f32": 1e-5, "f16": 2e-3, "bf16": 1e-2}   # fp32 sums rounded once to the storage type


def cwi_backward_parity(S, coords, grid, x, w_x, w_y, w_3, dy, dtype, order=None, label="", repeat=False):
    import torch

    cc = torch.from_numpy(np.ascontiguousarray(coords.astype(np.int32))).cuda()
    m, conflicts = S.cwi_build_map(cc, grid)
    tord = None if order is None else torch.from_numpy(np.ascontiguousarray(order.astype(np.int32))).cuda()
    dev = lambda a: to_dev(a, dtype)  # noqa: E731
    args = (m, grid, cc, dev(x), dev(w_x), dev(w_y), dev(w_3), dev(dy))
    got = S.cwi_backward(*args, order=tord)
    torch.cuda.synchronize()
    assert int(conflicts.cpu()[0]) == 0
    got = [to_host64(t, dtype) for t in got]
    w = lambda a: oracle.widen(a, dtype)  # noqa: E731
    ref = oracle.cwi_backward_ref(coords, w(x), w(w_x), w(w_y), w(w_3), w(dy), grid)
    n, C = x.shape
    errs = []
    if n:
        errs.append(rel_err_per_head(got[0].reshape(n, 4, C // 4), ref[0].reshape(n, 4, C // 4),
                                     1e-3 * float(np.abs(ref[0]).max())))
        # the identity quarter passes dy through, bit for bit
        assert np.array_equal(got[0][:, 3 * C // 4:], w(dy)[:, 3 * C // 4:])
    else:
        errs.append(0.0)
    for g, r in zip(got[1:], ref[1:]):
        scale = max(float(np.abs(r).max()), 1e-30)
        errs.append(float(np.abs(g - r).max()) / scale if r.size else 0.0)
        if n == 0:
            assert not np.any(g), "kernel gradients of an empty set must be zero"
    _say(f"[cwi-bwd {label}] n={n} C={C} grid={grid} {dtype} dx={errs[0]:.3e} "
         f"dw_x={errs[1]:.3e} dw_y={errs[2]:.3e} dw_3={errs[3]:.3e}")
    assert errs[0] <= TOL[dtype], f"{label}: dx relative error {errs[0]:.3e}"
    assert max(errs[1:]) <= CWI_DW_TOL[dtype], f"{label}: kernel-gradient relative error {max(errs[1:]):.3e}"
    if repeat:   # fixed reduction order: a second call (into given buffers) gives the same bits
        out = tuple(torch.full_like(t, float("nan")) for t in (args[3], *args[4:7]))
        ws = torch.empty(S.cwi_backward_workspace_bytes(n, args[3].dtype, C, w_x.shape[0], w_y.shape[0]),
                         dtype=torch.uint8, device="cuda")
        again = [to_host64(t, dtype) for t in S.cwi_backward(*args, order=tord, workspace=ws, out=out)]
        torch.cuda.synchronize()
        assert all(np.array_equal(a, b) for a, b in zip(got, again))


def test_cwi_backward_frame(sla):
    # the Waymo-like pillar frame, in the SLA plan's window order and in row order
    f = workloads.make_cwi_frame()
    perm, _, _ = oracle.segments_ref(f["ids"], f["num_windows"])
    rng = np.random.default_rng(63)
    dy = workloads.cast_values(rng.standard_normal(f["x"].shape).astype(np.float32), f["dtype"])
    for order in (perm, None):
        cwi_backward_parity(sla, f["coords"], f["grid"], f["x"], f["w_x"], f["w_y"], f["w_3"], dy, f["dtype"],
                            order=order, label="frame" + ("-window-order" if order is not None else ""),
                            repeat=order is not None)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("C,kx,ky", [(32, 13, 13), (64, 5, 31), (128, 1, 63), (256, 13, 3)])
def test_cwi_backward_voxels(sla, dtype, C, kx, ky):
    # 3D voxel grids (all 27 cube taps), random occupancy, rows shuffled
    if dtype == "f32" and C == 32:
        C = 16
    rng = np.random.default_rng([64, C, kx, len(dtype)])
    grid = (37, 29, 5)
    occ = rng.random(grid[::-1]) < 0.3
    zz, yy, xx = np.nonzero(occ)
    coords = np.stack([xx, yy, zz], axis=1)[rng.permutation(zz.size)]
    n, c = coords.shape[0], C // 4
    cast = lambda a: workloads.cast_values(a.astype(np.float32), dtype)  # noqa: E731
    x, dy = cast(rng.standard_normal((n, C))), cast(rng.standard_normal((n, C)))
    w_x, w_y, w_3 = (cast(rng.standard_normal((k, c)) / np.sqrt(k)) for k in (kx, ky, 27))
    cwi_backward_parity(sla, coords, grid, x, w_x, w_y, w_3, dy, dtype, order=rng.permutation(n),
                        label=f"vox{C}")


def test_cwi_backward_small_and_empty(sla):
    # a handful of voxels (one row group, most lanes idle), a lone voxel, and none
    rng = np.random.default_rng(65)
    for n in (5, 1, 0):
        cells = rng.choice(6 * 5 * 2, size=n, replace=False)
        coords = np.stack([cells % 6, (cells // 6) % 5, cells // 30], axis=1)
        x, dy = (workloads.cast_values(rng.standard_normal((n, 64)).astype(np.float32), "f16") for _ in range(2))
        w_x, w_y, w_3 = (workloads.cast_values(rng.standard_normal((k, 16)).astype(np.float32), "f16")
                         for k in (7, 3, 27))
        cwi_backward_parity(sla, coords.reshape(n, 3), (6, 5, 2), x, w_x, w_y, w_3, dy, "f16", label=f"n{n}")


@pytest.mark.parametrize("dtype,C,kx,ky", [("f16", 128, 13, 13), ("bf16", 64, 5, 31), ("f32", 64, 1, 63),
                                           ("f16", 512, 13, 3), ("f16", 32, 13, 13), ("f32", 16, 3, 3)])
def test_cwi_tiled_matches_gather(sla, dtype, C, kx, ky):
    # A pillar scene (one cell deep) takes the LDS-tiled kernel; the same scene in
    # a grid two cells deep takes the gather kernel, whose extra 3 x 3 x 3 taps all
    # land on empty cells.  Both add the same taps in the same order, so forward,
    # dx and the kernel gradients agree bit for bit.  Occupancy: a dense block,
    # random cells elsewhere, the grid's border rows and columns.
    import torch

    rng = np.random.default_rng([66, C, kx, ky, len(dtype)])
    gx, gy = 150, 97
    occ = rng.random((gy, gx)) < 0.35
    occ[20:60, 30:90] = True
    occ[0, :] |= rng.random(gx) < 0.7
    occ[:, gx - 1] |= rng.random(gy) < 0.7
    yy, xx = np.nonzero(occ)
    perm = rng.permutation(yy.size)
    coords = np.stack([xx, yy, np.zeros_like(xx)], axis=1)[perm].astype(np.int32)
    n, c = coords.shape[0], C // 4
    cast = lambda a: workloads.cast_values(a.astype(np.float32), dtype)  # noqa: E731
    x, dy = cast(rng.standard_normal((n, C))), cast(rng.standard_normal((n, C)))
    w_x, w_y, w_3 = (cast(rng.standard_normal((k, c)) / np.sqrt(k)) for k in (kx, ky, 27))
    dev = lambda a: to_dev(a, dtype)  # noqa: E731
    cc = torch.from_numpy(coords).cuda()
    outs = []
    for grid in ((gx, gy, 1), (gx, gy, 2)):
        m, conflicts = sla.cwi_build_map(cc, grid)
        y = sla.cwi_forward(m, grid, cc, dev(x), dev(w_x), dev(w_y), dev(w_3))
        back = sla.cwi_backward(m, grid, cc, dev(x), dev(w_x), dev(w_y), dev(w_3), dev(dy))
        torch.cuda.synchronize()
        assert int(conflicts.cpu()[0]) == 0
        outs.append([to_host64(t, dtype) for t in (y, *back)])
    names = ("y", "dx", "dw_x", "dw_y", "dw_3")
    for name, a, b in zip(names, *outs):
        assert np.array_equal(a, b), f"{name}: tiled and gather paths differ"
    # and the pair against the oracle, forward and dx
    w = lambda a: oracle.widen(a, dtype)  # noqa: E731
    ref = oracle.cwi_forward_ref(coords, w(x), w(w_x), w(w_y), w(w_3), (gx, gy, 1))
    err = rel_err_per_head(outs[0][0].reshape(n, 4, c), ref.reshape(n, 4, c), 1e-3 * float(np.abs(ref).max()))
    _say(f"[cwi-tiled] n={n} C={C} taps=({kx},{ky}) {dtype} rel_err={err:.3e}")
    assert err <= TOL[dtype]


@pytest.mark.parametrize("grid,density", [((1, 1, 1), 1.0), ((3, 70, 1), 0.5), ((70, 3, 1), 0.5),
                                          ((65, 5, 1), 1.0), ((17, 17, 1), 0.2)])
def test_cwi_tiled_edges(sla, grid, density):
    # pillar grids smaller than a tile or its halo along one axis, partial tiles,
    # a full grid and a lone voxel: forward and backward against the oracle
    rng = np.random.default_rng([67, grid[0], grid[1]])
    gx, gy, _ = grid
    occ = rng.random((gy, gx)) < density
    occ.flat[rng.integers(occ.size)] = True          # at least one voxel
    yy, xx = np.nonzero(occ)
    coords = np.stack([xx, yy, np.zeros_like(xx)], axis=1)[rng.permutation(yy.size)].astype(np.int32)
    n, C = coords.shape[0], 64
    c = C // 4
    cast = lambda a: workloads.cast_values(a.astype(np.float32), "f16")  # noqa: E731
    x, dy = cast(rng.standard_normal((n, C))), cast(rng.standard_normal((n, C)))
    w_x, w_y, w_3 = (cast(rng.standard_normal((k, c)) / np.sqrt(k)) for k in (13, 13, 27))
    cwi_parity(sla, coords, grid, x, w_x, w_y, w_3, "f16", label=f"edge{grid}")
    cwi_backward_parity(sla, coords, grid, x, w_x, w_y, w_3, dy, "f16", label=f"edge{grid}")


# ------------------------------------------------------------------ XCA variant
def xca_parity(S, ids, offsets, n, W, q, k, v, tau, dtype, label=""):
    import torch

    plan = build(S, ids=ids, W=W, offsets=offsets, n=n)
    off, perm = check_plan(S, plan, ids, W, 0, offsets)
    tq, tk, tv = (to_dev(a, dtype) for a in (q, k, v))
    tau32 = np.asarray(tau, dtype=np.float32)
    o = torch.full_like(tq, float("nan"))
    S.forward_xca(plan, tq, tk, tv, torch.from_numpy(tau32).to(tq.device), out=o)
    torch.cuda.synchronize()
    got = to_host64(o, dtype)
    w = lambda a: oracle.widen(a, dtype)  # noqa: E731
    ref = oracle.xca_forward_ref(w(q), w(k), w(v), tau32.astype(np.float64), off, perm)
    rows = np.zeros(n, dtype=bool)
    rows[perm if perm is not None else np.arange(off[-1])] = True
    assert np.isnan(got[~rows]).all(), f"{label}: a row in no window was written"
    floor = 1e-3 * max(float(np.abs(w(v)).max()) if v.size else 1.0, 1e-30)
    err = rel_err_per_head(got, ref, floor, rows)
    _say(f"[xca {label}] n={n} W={W} dtype={dtype} rel_err={err:.3e}")
    assert err <= TOL[dtype], f"{label}: XCA relative error {err:.3e}"
    return got, ref


def _xca_tau(H):
    return np.linspace(-1.5, 4.0, H) if H > 1 else np.array([2.0])


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_xca_config(sla, cfg):
    wl = workloads.make_config(cfg)
    H = wl["q"].shape[1]
    xca_parity(sla, wl["ids"], wl["offsets"], wl["n"], wl["num_windows"], wl["q"], wl["k"], wl["v"],
               _xca_tau(H), wl["dtype"], label=f"cfg{cfg}")


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", [(2, 32), (8, 16), (3, 32), (1, 16)])
def test_xca_shapes(sla, dtype, shape):
    # empty windows, singletons, windows of 63/64/65 rows (one and two LDS
    # blocks) and one of 1024 rows (16 blocks)
    H, d = shape
    rng = np.random.default_rng([43, H, d, len(dtype)])
    lengths = _adversarial_lengths(rng, 64)
    ids = workloads.ids_from_lengths(lengths, rng)
    n, W = ids.size, lengths.size
    q, k, v = (workloads.normal_values(rng, n, H, d, dtype) for _ in range(3))
    xca_parity(sla, ids, None, n, W, q, k, v, _xca_tau(H), dtype, label=f"shape{shape}")


@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_xca_degenerate(sla, dtype):
    # a zero q column (its norm takes the floor: a uniform softmax row), a zero k
    # column, tau = 0 in one head and a sharp softmax (tau = 40) in another, and
    # rows with invalid window ids (in no window: left unwritten)
    rng = np.random.default_rng([44, len(dtype)])
    H, d = 4, 32
    lengths = np.array([5, 1, 70, 0, 33, 2], dtype=np.int64)
    ids = workloads.ids_from_lengths(lengths, rng)
    ids = np.concatenate([ids, np.array([-1, 6, 99], dtype=ids.dtype)])
    n, W = ids.size, lengths.size
    q, k, v = (workloads.normal_values(rng, n, H, d, dtype) for _ in range(3))
    q[:, 1, 7] = 0
    k[:, 2, 30] = 0
    xca_parity(sla, ids, None, n, W, q, k, v, np.array([0.0, 40.0, 1.0, -3.0]), dtype, label="degenerate")


def test_xca_rows_in_order_and_csr(sla):
    # CSR plan (rows already window-sorted, no permutation) against the same
    # scene through ids: the same outputs, bit for bit
    import torch

    wl = workloads.make_config(1)
    offs = wl["offsets"]
    n, W = wl["n"], wl["num_windows"]
    got_csr, _ = xca_parity(sla, None, offs, n, W, wl["q"], wl["k"], wl["v"], _xca_tau(wl["q"].shape[1]),
                            wl["dtype"], label="csr")
    ids = np.repeat(np.arange(W), np.diff(offs)).astype(np.int32)
    got_ids, _ = xca_parity(sla, ids, None, n, W, wl["q"], wl["k"], wl["v"], _xca_tau(wl["q"].shape[1]),
                            wl["dtype"], label="ids")
    assert np.array_equal(got_csr, got_ids)
    torch.cuda.synchronize()


# ------------------------------------------------------------ XCA backward
# dq, dk and dv are held to the same bars as every other gradient (1e-5 in fp32,
# 2e-2 in fp16 / bf16).  dtau is an fp32 result computed from the exactly widened
# inputs in every storage type, so it is held to 1e-5 of the largest head's value.
XCA_DTAU_TOL = 1e-5
# the largest finite value of each storage type: a gradient beyond it rounds to
# +-inf (round to nearest; a column whose norm takes the 1e-12 floor has
# gradients near 1e12, beyond fp16's range)
_DTYPE_MAX = {"f32": float(np.finfo(np.float32).max), "f16": 65504.0, "bf16": 3.3895313892515355e38}


def _split_overflow(name, x, r, dtype, label):
    """Entries whose reference rounds past the storage type's range must be inf
    of the reference's sign; they are then left out of the relative error."""
    big = np.abs(r) > _DTYPE_MAX[dtype] * (1 + 2.0 ** -12)
    if big.any():
        assert np.array_equal(x[big], np.sign(r[big]) * np.inf), f"{label}: {name} overflow not rounded to inf"
        x, r = x.copy(), r.copy()
        x[big] = 0.0
        r[big] = 0.0
    return x, r


def xca_backward_parity(S, ids, offsets, n, W, q, k, v, do, tau, dtype, label=""):
    import torch

    plan = build(S, ids=ids, W=W, offsets=offsets, n=n)
    off, perm = check_plan(S, plan, ids, W, 0, offsets)
    tq, tk, tv, tdo = (to_dev(a, dtype) for a in (q, k, v, do))
    tau32 = np.asarray(tau, dtype=np.float32)
    outs = [torch.full_like(tq, float("nan")) for _ in range(3)]
    dq, dk, dv, dtau = S.backward_xca(plan, tq, tk, tv, torch.from_numpy(tau32).to(tq.device), tdo, *outs)
    torch.cuda.synchronize()
    got = [to_host64(t, dtype) for t in (dq, dk, dv)]
    w = lambda a: oracle.widen(a, dtype)  # noqa: E731
    ref = oracle.xca_backward_ref(w(q), w(k), w(v), tau32.astype(np.float64), w(do), off, perm)
    rows = np.zeros(n, dtype=bool)
    rows[perm if perm is not None else np.arange(off[-1])] = True
    for name, x, r in zip(("dq", "dk", "dv"), got, ref[:3]):
        assert np.isnan(x[~rows]).all(), f"{label}: {name} written outside every window"
        xs, rr = _split_overflow(name, x[rows], r[rows], dtype, label)
        err = rel_err_per_head(xs, rr, 1e-30)
        _say(f"[xca-bwd {label}] {name} n={n} dtype={dtype} rel_err={err:.3e}")
        assert err <= GRAD_TOL[dtype], f"{label}: {name} relative error {err:.3e}"
    dt = dtau.cpu().numpy().astype(np.float64)
    derr = float(np.abs(dt - ref[3]).max()) / max(float(np.abs(ref[3]).max()), 1e-30)
    _say(f"[xca-bwd {label}] dtau rel_err={derr:.3e}")
    assert derr <= XCA_DTAU_TOL, f"{label}: dtau relative error {derr:.3e}"
    return got, dt


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_xca_backward_config(sla, cfg):
    wl = workloads.make_config(cfg)
    H = wl["q"].shape[1]
    do = workloads.normal_values(np.random.default_rng([cfg, 9]), wl["n"], H, wl["q"].shape[2], wl["dtype"])
    xca_backward_parity(sla, wl["ids"], wl["offsets"], wl["n"], wl["num_windows"], wl["q"], wl["k"], wl["v"],
                        do, np.linspace(0.5, 3.0, H), wl["dtype"], label=f"cfg{cfg}")


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", [(2, 32), (8, 16), (3, 32)])
def test_xca_backward_shapes(sla, dtype, shape):
    H, d = shape
    rng = np.random.default_rng([45, H, d, len(dtype)])
    lengths = _adversarial_lengths(rng, 64)
    ids = workloads.ids_from_lengths(lengths, rng)
    n, W = ids.size, lengths.size
    q, k, v, do = (workloads.normal_values(rng, n, H, d, dtype) for _ in range(4))
    tau = np.linspace(-1.5, 4.0, H) + 0.25
    xca_backward_parity(sla, ids, None, n, W, q, k, v, do, tau, dtype, label=f"shape{shape}")


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_xca_backward_degenerate(sla, dtype):
    # the norm floor in the backward: a zero q column (head 1) and a zero k column
    # (head 2), whose gradients are dqh / 1e-12 (beyond fp16's range: +-inf there);
    # tau = 0 (head 0: dq = dk = 0, dtau from the uniform softmax); and in head 3
    # one- and two-row windows whose q and k columns are small (1e-3), where the
    # exact dq and dk of a one-row window are 0
    rng = np.random.default_rng([47, len(dtype)])
    H, d = 4, 32
    lengths = np.array([5, 1, 70, 0, 33, 2, 1, 2, 1], dtype=np.int64)
    ids = workloads.ids_from_lengths(lengths, rng)
    n, W = ids.size, lengths.size
    q, k, v, do = (workloads.normal_values(rng, n, H, d, dtype) for _ in range(4))
    q[:, 1, 7] = 0
    k[:, 2, 30] = 0
    small = np.isin(ids, np.flatnonzero(lengths <= 2))
    for x in (q, k):
        x32 = oracle.widen(x, dtype)
        x32[small, 3, :] *= 1e-3
        x[...] = workloads.cast_values(x32.astype(np.float32), dtype)
    xca_backward_parity(sla, ids, None, n, W, q, k, v, do, np.array([0.0, 2.0, 1.0, -3.0]), dtype,
                        label=f"degenerate-{dtype}")


def test_xca_backward_deterministic_and_empty(sla):
    import torch

    rng = np.random.default_rng(46)
    lengths = np.array([40, 0, 130, 1, 64], dtype=np.int64)
    ids = workloads.ids_from_lengths(lengths, rng)
    n, W, H, d = ids.size, lengths.size, 4, 32
    q, k, v, do = (workloads.normal_values(rng, n, H, d, "f16") for _ in range(4))
    tau = np.array([1.0, 2.0, -0.5, 3.0])
    a = xca_backward_parity(sla, ids, None, n, W, q, k, v, do, tau, "f16", label="determinism")
    b = xca_backward_parity(sla, ids, None, n, W, q, k, v, do, tau, "f16", label="determinism")
    for x, y in zip(a[0], b[0]):
        assert np.array_equal(x, y, equal_nan=True)
    assert np.array_equal(a[1], b[1])
    # n = 0: nothing to write, dtau is zero
    plan = build(sla, ids=np.zeros(0, dtype=np.int32), W=3)
    e = torch.zeros((0, 2, 16), dtype=torch.float16, device="cuda")
    dtau = torch.full((2,), float("nan"), device="cuda")
    sla.backward_xca(plan, e, e, e, torch.ones(2, device="cuda"), e, dtau=dtau)
    torch.cuda.synchronize()
    assert torch.equal(dtau.cpu(), torch.zeros(2))

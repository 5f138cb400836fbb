"""CPU tests of the C ABI: the built library loads, exports every function that
include/sla.h declares, and rejects bad arguments synchronously (host-side checks
run before anything is launched, so no GPU is needed)."""
import ctypes
import os
import re

import pytest

from paper_2401_00912_amd import sla

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sla.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sla_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(sla.LIB_PATH):
        from paper_2401_00912_amd import build

        build.build()
    return sla.lib()


def test_header_declares_the_abi():
    assert declared_functions() == sorted(sla.EXPORTED)


def test_every_declared_symbol_is_exported(L):
    for name in declared_functions():
        assert hasattr(L, name), name


def test_only_the_abi_is_exported():
    import subprocess

    out = subprocess.run(["nm", "-D", "--defined-only", sla.LIB_PATH], capture_output=True, text=True).stdout
    ours = sorted({l.split()[-1] for l in out.splitlines() if " T sla_" in l})
    assert ours == sorted(sla.EXPORTED)


def test_queries(L):
    assert L.sla_abi_version() == 8
    assert L.sla_max_windows() == 16384
    assert L.sla_default_chunk_rows() == 64
    for s in range(5):
        assert sla.status_string(s).startswith("SLA_")
    assert sla.plan_bytes(0, 1) > 0
    assert sla.plan_bytes(-1, 4) == 0
    assert sla.plan_bytes(10, 0) == 0
    assert sla.plan_bytes(10, 16385) == 0
    lay = sla.plan_layout(60000, 1521)
    assert lay.total == sla.plan_bytes(60000, 1521)
    assert lay.header == 0 and lay.perm % 256 == 0 and lay.offsets % 256 == 0 and lay.chunks % 256 == 0
    assert lay.offsets >= lay.perm + 4 * 60000
    assert lay.chunks >= lay.offsets + 4 * 1522
    assert lay.max_chunks == 1521
    assert lay.longs % 256 == 0 and lay.longs >= lay.chunks + 16 * 1521
    assert lay.max_long == min(1521, 60000 // 33) and lay.total >= lay.longs + 16 * lay.max_long
    assert sla.plan_layout(100, 8).max_long == 3 and sla.plan_layout(100, 2).max_long == 2


FAKE = 1 << 20  # a 256-aligned fake device address: never dereferenced, every call below fails validation


def fwd(L, **kw):
    a = dict(plan=FAKE, plan_bytes=sla.plan_bytes(100, 8), n=100, W=8, dtype=1, H=4, d=32,
             q=FAKE, k=FAKE, v=FAKE, o=FAKE)
    a.update(kw)
    return L.sla_forward(a["plan"], a["plan_bytes"], a["n"], a["W"], a["dtype"], a["H"], a["d"],
                         a["q"], a["k"], a["v"], a["o"], None)


def test_forward_argument_errors(L):
    assert fwd(L, d=24) == sla.SLA_E_UNSUPPORTED
    assert fwd(L, d=64) == sla.SLA_E_UNSUPPORTED
    assert fwd(L, H=0) == sla.SLA_E_ARG
    assert fwd(L, n=-1) == sla.SLA_E_ARG
    assert fwd(L, W=0) == sla.SLA_E_ARG
    assert fwd(L, W=20000, plan_bytes=1 << 30) == sla.SLA_E_UNSUPPORTED
    assert fwd(L, dtype=7) == sla.SLA_E_ARG
    assert fwd(L, plan=None) == sla.SLA_E_ARG
    assert fwd(L, plan=FAKE + 16) == sla.SLA_E_ARG
    assert fwd(L, plan_bytes=100) == sla.SLA_E_WORKSPACE
    assert fwd(L, q=None) == sla.SLA_E_ARG
    assert fwd(L, o=FAKE + 2) == sla.SLA_E_ARG
    assert fwd(L, n=0) == sla.SLA_OK  # nothing to do, nothing launched


def test_backward_argument_errors(L):
    nb = sla.plan_bytes(100, 8)
    args = [FAKE, nb, 100, 8, 1, 4, 32] + [FAKE] * 7 + [None]
    bad = list(args)
    bad[6] = 8
    assert L.sla_backward(*bad) == sla.SLA_E_UNSUPPORTED
    bad = list(args)
    bad[10] = None  # dout
    assert L.sla_backward(*bad) == sla.SLA_E_ARG
    bad = list(args)
    bad[1] = 10
    assert L.sla_backward(*bad) == sla.SLA_E_WORKSPACE


def test_build_argument_errors(L):
    nb = sla.plan_bytes(100, 8)
    b = lambda ids, n, W, L_, perm, off, plan, pb: L.sla_build_segments(  # noqa: E731
        ids, n, W, L_, perm, off, None, plan, pb, None)
    assert b(FAKE, 100, 8, 33, None, None, FAKE, nb) == sla.SLA_E_ARG       # odd chunk rows
    assert b(FAKE, 100, 8, 16, None, None, FAKE, nb) == sla.SLA_E_ARG       # too small
    assert b(FAKE, 100, 8, 66, None, None, FAKE, nb) == sla.SLA_E_ARG       # too large
    assert b(FAKE, 100, 8, 0, None, None, FAKE, 64) == sla.SLA_E_WORKSPACE
    assert b(FAKE, 100, 8, 0, None, None, None, nb) == sla.SLA_E_ARG
    assert b(None, 100, 8, 0, None, None, FAKE, nb) == sla.SLA_E_ARG        # CSR mode needs offsets
    assert b(None, 100, 8, 0, FAKE, FAKE, FAKE, nb) == sla.SLA_E_ARG        # CSR mode has no perm
    assert b(FAKE + 1, 100, 8, 0, None, None, FAKE, nb) == sla.SLA_E_ARG    # misaligned ids
    assert b(FAKE, 100, 16385, 0, None, None, FAKE, 1 << 30) == sla.SLA_E_UNSUPPORTED
    # window ids (mode A) for at most 2^26 rows: 8,192 sort blocks of 8,192
    assert b(FAKE, (1 << 26) + 1, 8, 0, None, None, FAKE, 1 << 40) == sla.SLA_E_UNSUPPORTED
    assert b(FAKE, -5, 8, 0, None, None, FAKE, nb) == sla.SLA_E_ARG


def test_scatter_argument_errors(L):
    nb = sla.plan_bytes(100, 8)
    need = sla.scatter_workspace_bytes(100, 4, 32)
    assert need == 100 * 4 * 32 * 33 * 4
    assert sla.scatter_workspace_bytes(100, 4, 24) == 0
    assert sla.scatter_workspace_bytes(-1, 4, 32) == 0
    call = lambda **kw: L.sla_forward_scatter(  # noqa: E731
        kw.get("plan", FAKE), kw.get("pb", nb), kw.get("n", 100), 8, 1, 4, kw.get("d", 32), FAKE,
        FAKE, FAKE, FAKE, kw.get("ws", FAKE), kw.get("wsb", need), None)
    assert call(wsb=need - 1) == sla.SLA_E_WORKSPACE
    assert call(ws=None) == sla.SLA_E_ARG
    assert call(ws=FAKE + 4) == sla.SLA_E_ARG
    assert call(d=24) == sla.SLA_E_UNSUPPORTED
    assert call(pb=10) == sla.SLA_E_WORKSPACE
    assert call(n=0) == sla.SLA_OK
    big = L.sla_forward_scatter(FAKE, sla.plan_bytes(100, 8), 100, 8, 1, 128, 32, FAKE, FAKE, FAKE,
                                FAKE, FAKE, sla.scatter_workspace_bytes(100, 128, 32), None)
    assert big == sla.SLA_E_UNSUPPORTED


def test_xca_argument_errors(L):
    nb = sla.plan_bytes(100, 8)
    call = lambda **kw: L.sla_forward_xca(  # noqa: E731
        kw.get("plan", FAKE), kw.get("pb", nb), kw.get("n", 100), kw.get("W", 8), kw.get("dt", 1),
        kw.get("H", 4), kw.get("d", 32), kw.get("tau", FAKE), FAKE, FAKE, FAKE, kw.get("o", FAKE), None)
    assert call(tau=None) == sla.SLA_E_ARG
    assert call(tau=FAKE + 2) == sla.SLA_E_ARG      # tau is float32: 4-byte aligned
    assert call(o=FAKE + 8) == sla.SLA_E_ARG
    assert call(o=None) == sla.SLA_E_ARG
    assert call(d=24) == sla.SLA_E_UNSUPPORTED
    assert call(dt=3) == sla.SLA_E_ARG
    assert call(pb=10) == sla.SLA_E_WORKSPACE
    assert call(plan=FAKE + 64) == sla.SLA_E_ARG
    assert call(n=0) == sla.SLA_OK
    assert call(n=0, tau=None) == sla.SLA_OK          # nothing to do, nothing read
    # one 256-thread workgroup per (window, head): 16384 windows x 1024 heads is too many
    assert call(W=16384, H=1024, d=16, pb=sla.plan_bytes(100, 16384)) == sla.SLA_E_UNSUPPORTED


def test_xca_backward_argument_errors(L):
    nb = sla.plan_bytes(100, 8)
    assert L.sla_xca_backward_workspace_bytes(8, 4) == 8 * 4 * 4
    assert L.sla_xca_backward_workspace_bytes(0, 4) == 0
    need = 8 * 4 * 4
    call = lambda **kw: L.sla_backward_xca(  # noqa: E731
        FAKE, kw.get("pb", nb), kw.get("n", 100), 8, 1, 4, kw.get("d", 32), kw.get("tau", FAKE), FAKE, FAKE,
        FAKE, FAKE, FAKE, FAKE, kw.get("dv", FAKE), kw.get("dtau", FAKE), kw.get("ws", FAKE),
        kw.get("wsb", need), None)
    assert call(wsb=need - 1) == sla.SLA_E_WORKSPACE
    assert call(ws=None) == sla.SLA_E_ARG
    assert call(dtau=None) == sla.SLA_E_ARG
    assert call(dtau=FAKE + 2) == sla.SLA_E_ARG
    assert call(tau=None) == sla.SLA_E_ARG
    assert call(dv=FAKE + 8) == sla.SLA_E_ARG
    assert call(dv=None) == sla.SLA_E_ARG
    assert call(d=24) == sla.SLA_E_UNSUPPORTED
    assert call(pb=10) == sla.SLA_E_WORKSPACE


def test_variant_argument_errors(L):
    nb = sla.plan_bytes(100, 8)
    f = lambda fm, eps, **kw: L.sla_forward_ex(  # noqa: E731
        FAKE, nb, kw.get("n", 100), 8, 1, 4, kw.get("d", 32), fm, eps, FAKE, FAKE, FAKE,
        kw.get("o", FAKE), None)
    b = lambda fm, eps: L.sla_backward_ex(FAKE, nb, 100, 8, 1, 4, 32, fm, eps,  # noqa: E731
                                          *([FAKE] * 7), None)
    for call in (f, b):
        assert call(2, 0.0) == sla.SLA_E_ARG             # unknown feature map
        assert call(-1, 0.0) == sla.SLA_E_ARG
        assert call(1, -1e-6) == sla.SLA_E_ARG           # eps < 0
        assert call(1, float("nan")) == sla.SLA_E_ARG
        assert call(0, float("inf")) == sla.SLA_E_ARG
    assert f(1, 1e-6, d=24) == sla.SLA_E_UNSUPPORTED     # the shared checks still apply
    assert f(1, 1e-6, o=FAKE + 2) == sla.SLA_E_ARG
    assert f(1, 1e-6, n=0) == sla.SLA_OK
    assert f(0, 0.0, n=0) == sla.SLA_OK
    with pytest.raises(ValueError):
        sla._variant("gelu", 0.0)
    assert sla._variant(None, None) is None
    assert sla._variant("relu", None) == (1, 0.0) and sla._variant(None, 1e-3) == (0, 1e-3)


def test_projected_argument_errors(L):
    nb = sla.plan_bytes(100, 8)
    def call(dtype=1, H=4, d=32, fm=0, eps=0.0, n=100, x=FAKE, y=FAKE, bq=None, qkv=None):
        return L.sla_forward_projected(FAKE, nb, n, 8, dtype, H, d, fm, eps, x, FAKE, bq, FAKE, None,
                                       FAKE, y, qkv, None)
    assert call(dtype=0) == sla.SLA_E_UNSUPPORTED        # fp32 is not supported
    assert call(H=3) == sla.SLA_E_UNSUPPORTED            # C = 96
    assert call(H=16) == sla.SLA_E_UNSUPPORTED           # C = 512
    assert call(d=24) == sla.SLA_E_UNSUPPORTED
    assert call(fm=3) == sla.SLA_E_ARG
    assert call(eps=-1.0) == sla.SLA_E_ARG
    assert call(x=FAKE + 8) == sla.SLA_E_ARG
    assert call(y=None) == sla.SLA_E_ARG
    assert call(bq=FAKE + 1) == sla.SLA_E_ARG
    assert call(qkv=FAKE + 8) == sla.SLA_E_ARG          # q, k, v saved at a 16-byte boundary
    assert call(n=0) == sla.SLA_OK


def test_projected_backward_argument_errors(L):
    nb = sla.plan_bytes(100, 8)
    need = sla.backward_projected_workspace_bytes(100, 4, 32)
    assert need > 0
    assert sla.backward_projected_workspace_bytes(100, 3, 32) == 0            # C = 96
    assert sla.backward_projected_workspace_bytes(-1, 4, 32) == 0
    # the workspace grows with n
    assert sla.backward_projected_workspace_bytes(1000, 4, 32) > need

    def call(dtype=1, H=4, d=32, fm=0, eps=0.0, x=FAKE, dy=FAKE, dx=FAKE, dwq=FAKE, dwo=FAKE, dbq=None,
             ws=FAKE, wsb=None, qkv=None):
        return L.sla_backward_projected(FAKE, nb, 100, 8, dtype, H, d, fm, eps, x, FAKE, None, FAKE, FAKE,
                                        dy, dx, dwq, dbq, dwo, None, qkv, ws, need if wsb is None else wsb,
                                        None)
    assert call(dtype=0) == sla.SLA_E_UNSUPPORTED        # fp32 is not supported
    assert call(H=3) == sla.SLA_E_UNSUPPORTED            # C = 96
    assert call(d=24) == sla.SLA_E_UNSUPPORTED
    assert call(fm=3) == sla.SLA_E_ARG
    assert call(eps=-1.0) == sla.SLA_E_ARG
    assert call(x=FAKE + 8) == sla.SLA_E_ARG
    assert call(dy=None) == sla.SLA_E_ARG
    assert call(dx=FAKE + 4) == sla.SLA_E_ARG
    assert call(dwq=None) == sla.SLA_E_ARG
    assert call(dwo=FAKE + 2) == sla.SLA_E_ARG
    assert call(dbq=FAKE + 1) == sla.SLA_E_ARG
    assert call(qkv=FAKE + 4) == sla.SLA_E_ARG
    assert call(ws=None) == sla.SLA_E_ARG
    assert call(ws=FAKE + 16) == sla.SLA_E_ARG
    assert call(wsb=need - 1) == sla.SLA_E_WORKSPACE


def test_cwi_argument_errors(L):
    assert sla.cwi_map_bytes(468, 468, 1) == 4 * 468 * 468
    assert sla.cwi_map_bytes(0, 4, 1) == 0 and sla.cwi_map_bytes(1 << 16, 1 << 16, 1) == 0
    mb = sla.cwi_map_bytes(8, 8, 1)
    bm = lambda **k: L.sla_cwi_build_map(k.get("coords", FAKE), k.get("n", 10), 8, 8, k.get("gz", 1),  # noqa: E731
                                         k.get("map", FAKE), k.get("mb", mb), None, None)
    assert bm(mb=mb - 4) == sla.SLA_E_WORKSPACE
    assert bm(map=None) == sla.SLA_E_ARG
    assert bm(coords=None) == sla.SLA_E_ARG
    assert bm(gz=0) == sla.SLA_E_ARG
    assert bm(n=-1) == sla.SLA_E_ARG

    def fw(dtype=1, C=128, kx=13, ky=13, n=10, x=FAKE, order=None):
        return L.sla_cwi_forward(FAKE, 8, 8, 1, FAKE, n, order, dtype, C, kx, ky, x, FAKE, FAKE, FAKE, FAKE,
                                 None)
    assert fw(kx=12) == sla.SLA_E_UNSUPPORTED        # even taps
    assert fw(ky=65) == sla.SLA_E_UNSUPPORTED
    assert fw(C=96) == sla.SLA_E_UNSUPPORTED         # 3 pieces of 16 bytes per branch row: 64 % 3 != 0
    assert fw(C=48) == sla.SLA_E_UNSUPPORTED         # 24 bytes per branch row: not whole pieces
    assert fw(C=4096) == sla.SLA_E_UNSUPPORTED       # 128 pieces per branch row: more than a wave
    assert fw(dtype=0, C=48) == sla.SLA_E_UNSUPPORTED  # fp32: 48 bytes per branch row: 3 pieces
    assert fw(dtype=5) == sla.SLA_E_ARG
    assert fw(x=FAKE + 4) == sla.SLA_E_ARG
    assert fw(order=FAKE + 2) == sla.SLA_E_ARG
    assert fw(n=0) == sla.SLA_OK


def test_cwi_backward_argument_errors(L):
    wb = L.sla_cwi_backward_workspace_bytes
    # a workgroup per 256 rows (four waves of 64), rounded up to a multiple of 8, at most 512
    assert wb(60000, 1, 128, 13, 13) == 240 * 53 * 32 * 4
    assert wb(100, 1, 128, 13, 13) == 8 * 53 * 32 * 4
    assert wb(10 ** 6, 1, 128, 13, 13) == 512 * 53 * 32 * 4
    assert wb(0, 1, 128, 13, 13) == 8 * 53 * 32 * 4              # the zero gradients still go through it
    assert wb(100, 1, 2048, 63, 63) == 8 * 153 * 512 * 4
    assert wb(100, 1, 96, 13, 13) == 0
    need = wb(100, 1, 128, 13, 13)

    def bw(ws=FAKE, wsb=need, n=100, dx=FAKE, C=128):
        return L.sla_cwi_backward(FAKE, 8, 8, 1, FAKE, n, None, 1, C, 13, 13, FAKE, FAKE, FAKE, FAKE, FAKE, dx,
                                  FAKE, FAKE, FAKE, ws, wsb, None)
    assert bw(wsb=need - 4) == sla.SLA_E_WORKSPACE
    assert bw(ws=None) == sla.SLA_E_ARG
    assert bw(dx=None) == sla.SLA_E_ARG
    assert bw(C=96) == sla.SLA_E_UNSUPPORTED


def test_cwi_binding_rejects_bad_tensors(L):
    # the binding's checks run before the C call (CPU tensors never reach it)
    import torch

    n, c = 10, 8
    grid = (8, 8, 1)
    coords = torch.zeros((n, 3), dtype=torch.int32)
    x = torch.zeros((n, 4 * c), dtype=torch.float16)
    w = [torch.zeros((k, c), dtype=torch.float16) for k in (5, 3, 27)]
    good_map = torch.zeros(64, dtype=torch.int32)
    with pytest.raises(ValueError, match="map"):
        sla.cwi_forward(torch.zeros(63, dtype=torch.int32), grid, coords, x, *w)   # one cell short
    with pytest.raises(ValueError, match="map"):
        sla.cwi_forward(good_map.float(), grid, coords, x, *w)
    with pytest.raises(ValueError, match="y must"):
        sla.cwi_forward(good_map, grid, coords, x, *w, y=torch.zeros((n, 4 * c + 8), dtype=torch.float16))
    with pytest.raises(ValueError, match="order"):
        sla.cwi_forward(good_map, grid, coords, x, *w, order=torch.zeros(n - 1, dtype=torch.int32))
    with pytest.raises(ValueError, match="coords"):
        sla.cwi_forward(good_map, grid, coords.t(), x, *w)
    with pytest.raises(ValueError, match="w_3"):
        sla.cwi_forward(good_map, grid, coords, x, w[0], w[1], torch.zeros((9, c), dtype=torch.float16))
    with pytest.raises(ValueError, match="dy must"):
        sla.cwi_backward(good_map, grid, coords, x, *w, x.float())
    with pytest.raises(ValueError, match="map"):
        sla.cwi_backward(torch.zeros(10, dtype=torch.int32), grid, coords, x, *w, x)


def test_xca_backward_binding_rejects_bad_dtau_and_workspace(L):
    # dtau and the workspace are checked before the C call: a short or 16-bit dtau
    # would let the temperature kernel write past its end, and a workspace on
    # another device would be handed over as a foreign pointer
    import torch

    n, H, d = 6, 4, 16
    plan = sla.Plan(buf=torch.zeros(sla.plan_bytes(n, 2), dtype=torch.uint8), n=n, num_windows=2,
                    chunk_rows=64, perm=None, offsets=None, invalid=None)
    q = torch.zeros((n, H, d), dtype=torch.float16)
    tau = torch.ones(H, dtype=torch.float32)
    args = (plan, q, q, q, tau, q)
    for bad in (torch.zeros(H, dtype=torch.float16), torch.zeros(H - 1), torch.zeros(2 * H)[::2],
                torch.zeros((H, 1)), torch.zeros(H, device="meta")):
        with pytest.raises(ValueError, match="dtau"):
            sla.backward_xca(*args, dtau=bad)
    with pytest.raises(ValueError, match="workspace"):
        sla.backward_xca(*args, dtau=torch.zeros(H), workspace=torch.zeros(64, dtype=torch.uint8, device="meta"))
    with pytest.raises(ValueError, match="workspace"):
        sla.backward_xca(*args, dtau=torch.zeros(H), workspace=torch.zeros(64, dtype=torch.uint8)[::2])


def test_projected_saved_qkv_argument_errors(L):
    # the saved q, k, v buffer is checked before the C call: a short, strided,
    # wrongly typed or foreign buffer would be written past its end by the
    # forward, or read past it by the backward
    import torch

    n, H, d = 6, 4, 32
    C = H * d
    plan = sla.Plan(buf=torch.zeros(sla.plan_bytes(n, 2), dtype=torch.uint8), n=n, num_windows=2,
                    chunk_rows=64, perm=None, offsets=None, invalid=None)
    x = torch.zeros((n, C), dtype=torch.float16)
    w_qkv = torch.zeros((3 * C, C), dtype=torch.float16)
    w_o = torch.zeros((C, C), dtype=torch.float16)
    for bad in (torch.zeros((3, n - 1, C), dtype=torch.float16), torch.zeros((3, n, C), dtype=torch.bfloat16),
                torch.zeros((3, n, 2 * C), dtype=torch.float16)[:, :, ::2], torch.zeros((n, C), dtype=torch.float16),
                torch.zeros((3, n, C), dtype=torch.float16, device="meta")):
        with pytest.raises(ValueError, match="qkv_out must"):
            sla.forward_projected(plan, x, w_qkv, w_o, H, qkv_out=bad)
        with pytest.raises(ValueError, match="qkv must"):
            sla.backward_projected(plan, x, w_qkv, w_o, x, x, H, qkv=bad)


def test_xca_backward_noalloc_argument_errors(L):
    # the size limit of the static buffer and the pointer checks are host-side:
    # nothing is enqueued (and no device is touched) when they fail
    assert L.sla_backward_xca_noalloc is not None
    W = 16384
    nb = sla.plan_bytes(100, W)
    call = lambda **kw: L.sla_backward_xca_noalloc(  # noqa: E731
        FAKE, kw.get("pb", nb), kw.get("n", 100), kw.get("W", W), 1, kw.get("H", 16), 32, kw.get("tau", FAKE),
        FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, kw.get("dv", FAKE), kw.get("dtau", FAKE), None)
    assert call(H=17) == sla.SLA_E_UNSUPPORTED          # 16384 x 17 partials > 262144
    assert call(dtau=None) == sla.SLA_E_ARG
    assert call(dtau=FAKE + 2) == sla.SLA_E_ARG
    assert call(tau=None) == sla.SLA_E_ARG
    assert call(dv=None) == sla.SLA_E_ARG
    assert call(dv=FAKE + 8) == sla.SLA_E_ARG
    assert call(pb=10) == sla.SLA_E_WORKSPACE

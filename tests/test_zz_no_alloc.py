"""The XCA backward without a workspace (sla_backward_xca_noalloc, through the C
ABI) against the same backward with a caller workspace (sla_backward_xca): equal
bit for bit, on two calls in a row, the second with a smaller input, so that the
static buffer's contents from the first call cannot leak into the second."""
from __future__ import annotations

import numpy as np
import pytest

import workloads
from tests.gpu_util import to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sla():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2401_00912_amd import sla as S

    S.lib()
    return S


def _case(S, seed, lengths, H, d, dtype):
    import torch

    rng = np.random.default_rng(seed)
    ids = workloads.ids_from_lengths(np.asarray(lengths, dtype=np.int64), rng)
    n, W = ids.size, len(lengths)
    q, k, v, do = (to_dev(workloads.normal_values(rng, n, H, d, dtype), dtype) for _ in range(4))
    tau = torch.from_numpy(np.linspace(-1.0, 3.0, H).astype(np.float32)).cuda()
    plan = S.build_segments(to_dev(ids.astype(np.int32)), num_windows=W)
    return plan, q, k, v, tau, do


def _both(S, args, noalloc_first):
    import torch

    def run(fn):
        outs = [torch.full_like(args[1], float("nan")) for _ in range(3)]
        dtau = torch.full_like(args[4], float("nan"))
        return fn(*args, *outs, dtau=dtau)

    if noalloc_first:
        a = run(S.backward_xca_noalloc)
        b = run(S.backward_xca)
    else:
        b = run(S.backward_xca)
        a = run(S.backward_xca_noalloc)
    torch.cuda.synchronize()
    return a, b


def test_noalloc_equals_workspace_call_twice(sla):
    import torch

    # first call: 40 windows x 4 heads (160 partials), second: 9 windows x 2 heads
    big = _case(sla, 71, [5, 0, 70, 1, 33, 2, 64, 65, 130, 12] * 4, 4, 32, "f16")
    small = _case(sla, 72, [3, 1, 0, 40, 9, 17, 2, 66, 5], 2, 16, "bf16")
    for args, first in ((big, True), (small, False), (big, False), (small, True)):
        a, b = _both(sla, args, first)
        for x, y, name in zip(a, b, ("dq", "dk", "dv", "dtau")):
            assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x,
                               y.view(torch.int16) if y.dtype == torch.bfloat16 else y) or \
                torch.equal(torch.isnan(x), torch.isnan(y)) and torch.equal(torch.nan_to_num(x), torch.nan_to_num(y)), name
        assert torch.isfinite(a[3]).all()

"""lpp_kernel_snapshot_noalloc (the snapshot with its work table in the
library's fixed device array) against lpp_kernel_snapshot (the same kernel
with a plan the library allocates): bit-identical v and weight layouts, on
two calls in a row (the second with a smaller conv list and parameter
vector, so it runs over the first call's table), in fp32 and bf16; lists
beyond the array's 128 convs are rejected before anything runs."""
import sys

import numpy as np
import pytest

from paper_2203_06638_amd import lpp
from paper_2203_06638_amd import models as PM
from tests.test_gpu_snapshot import model_convs, random_convs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _device():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    torch.cuda.init()


def _both(convs, d, wf, dtype, x):
    tdt = torch.float32 if dtype == lpp.FP32 else torch.bfloat16
    xd = torch.from_numpy(x).cuda()
    outs = []
    for noalloc in (False, True):
        v = torch.full((d,), 7.0, device="cuda")
        wb = torch.zeros(max(wf, 1), device="cuda", dtype=tdt)
        if noalloc:
            lpp.kernel_snapshot_noalloc(convs, d, dtype, max(wf, 1), xd, v, wb)
        else:
            plan = lpp.SnapshotPlan(convs, d, dtype, max(wf, 1))
            plan.run(xd, v, wb)
            torch.cuda.synchronize()
            plan.close()
        outs.append((v.cpu().numpy(), wb.view(torch.int16 if dtype == lpp.BF16 else torch.int32).cpu().numpy()))
    return outs


@pytest.mark.parametrize("dtype", [lpp.FP32, lpp.BF16])
def test_noalloc_matches_plan_two_calls(dtype):
    big = PM.wrn16_8(100) if dtype == lpp.BF16 else PM.resnet20(10)
    calls = [model_convs(big, dtype)]
    small, d2, wf2 = random_convs(np.random.default_rng(5 + dtype), dtype)
    calls.append((small, d2, wf2))
    assert calls[1][1] < calls[0][1] and len(calls[1][0]) < len(calls[0][0])
    for i, (convs, d, wf) in enumerate(calls):
        x = np.random.default_rng(i).standard_normal(d).astype(np.float32)
        say("no-alloc call", i, "dtype", dtype, "convs", len(convs), "d", d)
        (v0, w0), (v1, w1) = _both(convs, d, wf, dtype, x)
        assert np.array_equal(v0, v1)
        assert np.array_equal(w0, w1)


def test_noalloc_rejects_more_than_128_convs():
    convs = [(i * 16, 4, 4, 4, 1, 1, i * 64, i * 64 + 32) for i in range(129)]
    e = torch.zeros(129 * 64, device="cuda")
    with pytest.raises(lpp.LppError) as ei:
        lpp.kernel_snapshot_noalloc(convs, 129 * 16, lpp.FP32, 129 * 64, e, e, e)
    assert ei.value.code == lpp.EINVAL

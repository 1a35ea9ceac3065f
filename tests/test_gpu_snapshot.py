"""The snapshot kernel (Alg. 1, updater: collect a snapshot of the shared
model) through its stand-alone entry point, against its definition: every
conv weight W[cout][cin][kh][kw] transposed into W_f[cout][kh][kw][cin_p]
(padding channels untouched) and W_d[cin][kh][kw][cout], exactly (fp32) or
rounded to the nearest bf16 (ties to even), and every other entry copied
into v.  Conv lists: random shapes with ragged channel tiles, 1x1, 3x3, 5x5
and 7x7 filters, 3-channel (stem) inputs and unaligned tensor starts; and
the conv lists of the workloads' models (ResNet-20, WRN-16-8, ResNet-18,
ResNet-50) at their full sizes."""
import sys

import numpy as np
import pytest

import synth
from paper_2203_06638_amd import lpp
from paper_2203_06638_amd import models as PM

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _device():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    torch.cuda.init()


def random_convs(rng, dtype):
    """A sorted list of conv descriptors with gaps (other parameters) between
    the weight tensors, and d."""
    vw = 8 if dtype == lpp.BF16 else 4
    convs, pos, wf = [], int(rng.integers(0, 7)), 0
    for _ in range(int(rng.integers(1, 5))):
        k = int(rng.choice([1, 3, 5, 7]))
        cin = int(rng.choice([3, vw, 2 * vw, 3 * vw, 40, 96, 200]))
        cin_p = (cin + vw - 1) // vw * vw
        cout = vw * int(rng.integers(1, 20))
        nf, nd = cout * k * k * cin_p, cin * k * k * cout
        dst_f = wf
        dst_d = wf + (nf + 63) // 64 * 64
        wf = dst_d + (nd + 63) // 64 * 64
        convs.append((pos, cout, cin, cin_p, k, k, dst_f, dst_d))
        pos += cout * cin * k * k + int(rng.integers(0, 9))
    return convs, pos + int(rng.integers(0, 5000)), wf


def model_convs(model, dtype):
    """The conv list of a model's parameter vector, every conv given both
    layouts (the image's channels padded to 4, or 8 for bf16)."""
    vw = 8 if dtype == lpp.BF16 else 4
    convs, poff, wf = [], 0, 0
    for rec in model.layers:
        op, in0, _, cin, cout, k, _, _, bias = rec[:9]
        if op == lpp.CONV:
            cin_p = (cin + vw - 1) // vw * vw if in0 < 0 else cin
            nf, nd = cout * k * k * cin_p, cin * k * k * cout
            dst_f = wf
            dst_d = wf + (nf + 63) // 64 * 64
            wf = dst_d + (nd + 63) // 64 * 64
            convs.append((poff, cout, cin, cin_p, k, k, dst_f, dst_d))
            poff += cout * cin * k * k + (cout if bias else 0)
        elif op == lpp.BN:
            poff += 2 * cout
        elif op == lpp.LINEAR:
            poff += cout * cin + cout
    assert poff == model.d
    return convs, poff, wf


def expected(x, convs, d, wf, dtype):
    """v (nan where not written) and wbuf from the definition."""
    cast = synth.round_to_bf16 if dtype == lpp.BF16 else (lambda a: a)
    v = x.copy()
    wb = np.zeros(max(wf, 1), np.float32)
    for (src, cout, cin, cin_p, kh, kw, dst_f, dst_d) in convs:
        n = cout * cin * kh * kw
        W = x[src:src + n].reshape(cout, cin, kh, kw)
        v[src:src + n] = np.nan
        Wf = np.zeros((cout, kh, kw, cin_p), np.float32)
        Wf[..., :cin] = W.transpose(0, 2, 3, 1)
        wb[dst_f:dst_f + Wf.size] = cast(Wf).ravel()
        wb[dst_d:dst_d + n] = cast(np.ascontiguousarray(W.transpose(1, 2, 3, 0))).ravel()
    return v, wb


def run_snapshot(convs, d, wf, dtype, x):
    plan = lpp.SnapshotPlan(convs, d, dtype, max(wf, 1))
    xd = torch.from_numpy(x).cuda()
    vd = torch.full((d,), float("nan"), device="cuda")
    wd = torch.zeros(max(wf, 1), device="cuda", dtype=torch.float32 if dtype == lpp.FP32 else torch.bfloat16)
    plan.run(xd, vd, wd)
    torch.cuda.synchronize()
    plan.close()
    wb = wd.float().cpu().numpy()
    return vd.cpu().numpy(), wb


def check(x, convs, d, wf, dtype):
    got_v, got_w = run_snapshot(convs, d, wf, dtype, x)
    want_v, want_w = expected(x, convs, d, wf, dtype)
    conv_mask = np.isnan(want_v)
    assert np.array_equal(got_v[~conv_mask], want_v[~conv_mask])
    assert np.all(np.isnan(got_v[conv_mask]))          # conv weights are not copied into v
    assert np.array_equal(got_w, want_w)


@pytest.mark.parametrize("dtype", [lpp.FP32, lpp.BF16])
@pytest.mark.parametrize("seed", range(6))
def test_random_conv_lists(dtype, seed):
    rng = np.random.default_rng(100 * seed + dtype)
    convs, d, wf = random_convs(rng, dtype)
    say("snapshot random", seed, "dtype", dtype, "convs", [c[1:6] for c in convs], "d", d)
    x = rng.standard_normal(d).astype(np.float32)
    check(x, convs, d, wf, dtype)


@pytest.mark.parametrize("name,dtype", [("resnet20", lpp.FP32), ("wrn16_8", lpp.BF16), ("resnet18", lpp.BF16),
                                        ("resnet50", lpp.BF16), ("squeezenet", lpp.FP32)])
def test_workload_models(name, dtype):
    model = {"resnet20": lambda: PM.resnet20(10), "wrn16_8": lambda: PM.wrn16_8(100),
             "resnet18": lambda: PM.resnet18(1000), "resnet50": lambda: PM.resnet50(1000),
             "squeezenet": lambda: PM.squeezenet_p4(10)}[name]()
    convs, d, wf = model_convs(model, dtype)
    if name == "squeezenet":     # its 10-output classifier runs as a per-pixel linear layer, not a conv
        convs = [c for c in convs if c[1] % 4 == 0]
    say("snapshot", name, "d", d, "convs", len(convs))
    x = synth.init_params(model.specs, 3)
    check(x, convs, d, wf, dtype)


def test_empty_and_conv_free_vectors():
    """No convs: v is a copy; d = 0 launches nothing."""
    x = np.random.default_rng(1).standard_normal(4099).astype(np.float32)
    check(x, [], 4099, 0, lpp.FP32)
    plan = lpp.SnapshotPlan([], 0, lpp.FP32, 1)
    e = torch.zeros(4, device="cuda")
    plan.run(e, e, e)
    torch.cuda.synchronize()
    plan.close()


def test_invalid_lists_are_rejected_before_launch():
    bad = [
        ([(0, 6, 4, 4, 3, 3, 0, 256)], 1000, lpp.FP32, 1000),        # cout not a multiple of 4
        ([(0, 8, 4, 4, 3, 3, 0, 512)], 100, lpp.FP32, 1000),         # weights beyond d
        ([(0, 8, 4, 4, 3, 3, 0, 512)], 1000, lpp.FP32, 600),         # W_d beyond wbuf
        ([(0, 8, 4, 4, 3, 3, 2, 512)], 1000, lpp.FP32, 1000),        # unaligned W_f
        ([(300, 8, 4, 4, 1, 1, 0, 64), (0, 8, 4, 4, 1, 1, 128, 192)], 1000, lpp.FP32, 1000),   # unsorted
        ([(0, 8, 12, 8, 1, 1, 0, 128)], 1000, lpp.FP32, 1000),       # cin > cin_p
        ([(0, 8, 4, 4, 1, 1, 0, 64)], 1000, lpp.BF16, 1000),         # bf16 needs multiples of 8
    ]
    for convs, d, dt, wf in bad:
        with pytest.raises(lpp.LppError) as ei:
            lpp.SnapshotPlan(convs, d, dt, wf)
        assert ei.value.code == lpp.EINVAL

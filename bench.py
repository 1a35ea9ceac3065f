"""Throughput of the LPP-SGD per-node step on one MI355X.

Workload (the headline configuration): ResNet-20 (CIFAR shapes, 10 classes),
fp32, batch 128 of synthetic N(0, 1) 3x32x32 images with uniform labels;
P = 4 layer-block partitions, one worker per block on its own HIP stream,
K = 1 replica, momentum 0.9, lr 0.1, asynchronous (Hogwild) mode.  A step is
one worker iteration of Alg. 1: counter read&inc, snapshot, full forward,
backward truncated at the worker's block, lock-free block update.  Workers
are issued round-robin.  samples/s = 128 * steps / wall time of the timed
region (inputs resident in HBM before it starts).

Also reported, on the same JSON line:
  roofline      the dominant kernel family's algorithmic flops per launch
                over its average launch time (HIP events recorded in the
                kernels' own dispatch packets, worker 0 alone right after the
                timed region), against the fp32 matrix peak;
  cpu_baseline  the fp64 oracle's step timed on the host cores on a bounded
                sample (a baseline, not a target);
  hbm_kernels   the block-update, replica-averaging and snapshot kernels
                on 1 GiB-scale buffers (and the snapshot at the bf16
                workloads' sizes), as achieved HBM GB/s;
  workloads     the other configurations, each on a short run: ResNet-20
                with 100 classes and K = 4 replicas of P = 4 workers
                (averaging every 8 steps per replica), WRN-16-8 (bf16
                activations, fp32 master weights, K = 2, averaging every 4)
                and ResNet-18 at 224x224 (bf16, K = 2, averaging every 8),
                with samples/s and their dominant kernel family's fraction
                of the matrix peak of their dtype.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import threading
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "train samples/sec (fwd+partial bwd+update), ResNet-20 b128; MFMA util, HBM GB/s"

# Hardware queues per process (HIP reads GPU_MAX_HW_QUEUES once, at start-up).
# The headline's four worker streams run fastest with more queues than streams
# (measured: 259K samples/s with HIP's default of 4, 295K with 5, 6, 8 or 16);
# the multi-replica workloads (8 and 16 worker streams) run fastest with 4, so
# they run in child processes with that setting (--hw-queues and
# --workload-hw-queues change them).
PEAK_FP32_TFLOPS = 157.3
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
FAMILIES = ["conv_fwd", "conv_dgrad", "conv_wgrad", "wgrad_reduce", "bn_stats", "bn_act", "bn_bwd", "head",
            "relu", "add", "concat", "maxpool", "gap", "linear", "softmax_ce", "bias_grad", "snapshot", "image",
            "sgd_update"]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--batch", type=int, default=128)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--hw-queues", type=int, default=8, help="GPU_MAX_HW_QUEUES for the headline run (1..32)")
    ap.add_argument("--workload-hw-queues", type=int, default=4, help="GPU_MAX_HW_QUEUES for the other workloads")
    ap.add_argument("--no-hbm", action="store_true")
    ap.add_argument("--cpu-steps", type=int, default=8)
    ap.add_argument("--replicas", type=int, default=1, help="K (the headline workload has K = 1)")
    ap.add_argument("--workers-used", type=int, default=0,
                    help="issue steps to only the first n workers (0 = all); for latency studies")
    ap.add_argument("--issue-threads", type=int, default=1,
                    help="host threads issuing steps; each owns a fixed set of workers")
    ap.add_argument("--no-workloads", action="store_true", help="skip the other configurations")
    ap.add_argument("--workloads", default="resnet20_100_k4,wrn16_8_bf16,resnet18_bf16,resnet50_bf16,squeezenet_k2",
                    help="comma-separated subset of the other configurations")
    ap.add_argument("--workload-steps", type=int, default=64)
    ap.add_argument("--only-workload", default=None, help="run just one of the other configurations (for profiling)")
    ap.add_argument("--extras", action="store_true",
                    help="only the partial- vs full-backward throughput and the worker-stream sweep (ResNet-20)")
    ap.add_argument("--delays", action="store_true",
                    help="only the delay statistics of traced async runs (ResNet-20, K=2 x P=4) against H")
    # HBM traffic of the roofline kernel (run each under rocprofv3 --pmc):
    ap.add_argument("--roofline-only", metavar="FAMILY", default=None,
                    help="only the roofline pass: worker 0 alone, kernels of FAMILY launched one by one")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only a plain device copy of 256 MiB, ten times (counter calibration)")
    ap.add_argument("--summarize-traffic", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "CAL_FETCH_DIR", "CAL_WRITE_DIR"),
                    help="turn the four counter runs into the traffic summary under profiles/")
    ap.add_argument("--traffic-family", default="conv_fwd", choices=("conv_fwd", "sgd_update", "average"),
                    help="kernel family --summarize-traffic reads")
    ap.add_argument("--hbm-only", action="store_true",
                    help="only the update and averaging kernels on 1 GiB arrays (for their counters)")
    return ap.parse_args()


def _time_launches(torch, fn, reps, warm=3):
    """Average GPU time (s) of fn() over reps launches, HIP events on the
    current stream around the whole run (the launches queue back to back)."""
    for _ in range(warm):
        fn(0)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(reps):
        fn(i)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps / 1e3


def _hbm_entry(nbytes, t, **kw):
    gbs = nbytes / t / 1e9
    out = {"GB/s": round(gbs, 1), "frac": round(gbs / PEAK_HBM_GBS, 3), "us_per_launch": round(t * 1e6, 2)}
    out.update(kw)
    return out


def _model_snap_convs(model, dtype, lpp):
    """Conv descriptors of a model's parameter vector for the stand-alone
    snapshot (the same layouts lpp_init gives the worker buffers) and the
    algorithmic bytes of one snapshot."""
    vw = 8 if dtype == lpp.BF16 else 4
    eb = 2 if dtype == lpp.BF16 else 4
    convs, poff, wf, nconv = [], 0, 0, 0
    for rec in model.layers:
        op, in0, _, cin, cout, k, _, _, bias = rec[:9]
        if op == lpp.CONV:
            cin_p = (cin + vw - 1) // vw * vw if in0 < 0 else cin
            nf, nd = cout * k * k * cin_p, cin * k * k * cout
            convs.append((poff, cout, cin, cin_p, k, k, wf, wf + (nf + 63) // 64 * 64))
            wf += (nf + 63) // 64 * 64 + (nd + 63) // 64 * 64
            nconv += cout * cin * k * k
            poff += cout * cin * k * k + (cout if bias else 0)
        elif op == lpp.BN:
            poff += 2 * cout
        elif op == lpp.LINEAR:
            poff += cout * cin + cout
    return convs, poff, wf, (4 + 2 * eb) * nconv + 8 * (poff - nconv)


def hbm_kernels(torch, lpp):
    """The streaming kernels as achieved HBM GB/s (algorithmic bytes over
    the average launch time):
      sgd_update   block update with momentum, 20 B/param, on 256M-float
                   (1 GiB) arrays, each four times the 256 MB last-level cache;
      average_k2/4 averaging rounds over 2 and 4 replicas of 1 GiB
                   (8 B per parameter per replica);
      snapshot_*   the snapshot on a 236M-parameter vector of 3x3 convs
                   512 -> 512 separated by 1024 other parameters (fp32:
                   12 B per conv weight, bf16 cast: 8 B), and at the WRN-16-8
                   and ResNet-18 parameter vectors (bf16), rotating over
                   buffer sets whose footprint exceeds the last-level cache."""
    from paper_2203_06638_amd import models as PM
    n = 256 << 20
    out = {}
    x, m, g = (torch.randn(n, device="cuda") for _ in range(3))
    t = _time_launches(torch, lambda i: lpp.kernel_sgd_update(x, m, g, 1e-3, 0.9, 0.0), 20)
    out["sgd_update"] = _hbm_entry(20.0 * n, t, bytes_per_param=20, params=n)
    del m, g
    reps = [x] + [torch.randn(n, device="cuda") for _ in range(3)]
    for k in (2, 4):
        t = _time_launches(torch, lambda i: lpp.kernel_average(reps[:k]), 20)
        out["average_k%d" % k] = _hbm_entry(8.0 * k * n, t, bytes_per_param=8 * k, params=n)
    del reps, x
    torch.cuda.empty_cache()
    # snapshot on a 1 GiB-scale parameter vector
    nconv, co, ci, gap = 100, 512, 512, 1024
    per = co * ci * 9
    for dtype, name in ((lpp.FP32, "snapshot_f32"), (lpp.BF16, "snapshot_bf16")):
        vw = 8 if dtype == lpp.BF16 else 4
        convs, pos, wf = [], 0, 0
        for _ in range(nconv):
            convs.append((pos, co, ci, ci, 3, 3, wf, wf + per))
            wf += 2 * per
            pos += per + gap
        d = pos
        plan = lpp.SnapshotPlan(convs, d, dtype, wf)
        xs = torch.randn(d, device="cuda")
        vs = torch.empty(d, device="cuda")
        wb = torch.zeros(wf, device="cuda", dtype=torch.float32 if dtype == lpp.FP32 else torch.bfloat16)
        t = _time_launches(torch, lambda i: plan.run(xs, vs, wb), 10)
        eb = 4 if dtype == lpp.FP32 else 2
        by = (4 + 2 * eb) * nconv * per + 8 * (d - nconv * per)
        out[name] = _hbm_entry(by, t, bytes_per_launch=by, params=d,
                               what="%d 3x3 convs 512->512, %d other parameters between them" % (nconv, gap))
        plan.close()
        del xs, vs, wb
        torch.cuda.empty_cache()
    # snapshot at the bf16 workloads' sizes, rotating over buffer sets
    for mname, build in (("wrn16_8", lambda: PM.wrn16_8(100)), ("resnet18", lambda: PM.resnet18(1000))):
        model = build()
        convs, d, wf, by = _model_snap_convs(model, lpp.BF16, lpp)
        plan = lpp.SnapshotPlan(convs, d, lpp.BF16, wf)
        sets = 8
        bufs = [(torch.randn(d, device="cuda"), torch.empty(d, device="cuda"),
                 torch.zeros(wf, device="cuda", dtype=torch.bfloat16)) for _ in range(sets)]
        t = _time_launches(torch, lambda i: plan.run(*bufs[i % sets]), 64)
        out["snapshot_" + mname] = _hbm_entry(by, t, bytes_per_launch=by, params=d,
                                              what="bf16 cast, %d buffer sets in rotation (%.0f MB touched)"
                                                   % (sets, sets * (by / 1e6)))
        plan.close()
        del bufs
        torch.cuda.empty_cache()
    return out


# the other configurations: (model builder, input shape, classes, dtype, K, H)
def _workloads():
    from paper_2203_06638_amd import models as PM
    from paper_2203_06638_amd import lpp
    return {
        "resnet20_100_k4": (lambda: PM.resnet20(100), (3, 32, 32), 100, lpp.FP32, 4, 8,
                            "ResNet-20 (100 classes), batch 128, fp32, K=4 replicas x P=4 workers on 16 HIP "
                            "streams, averaging every 8 steps per replica, momentum 0.9, async"),
        "wrn16_8_bf16": (lambda: PM.wrn16_8(100), (3, 32, 32), 100, lpp.BF16, 2, 4,
                         "WRN-16-8 (100 classes), batch 128, bf16 activations / fp32 master weights, K=2 x P=4 "
                         "workers on 8 HIP streams, averaging every 4 steps per replica, momentum 0.9, async"),
        "resnet18_bf16": (lambda: PM.resnet18(1000), (3, 224, 224), 1000, lpp.BF16, 2, 8,
                          "ResNet-18 (1000 classes), batch 128 of 3x224x224, bf16 activations / fp32 master "
                          "weights, K=2 x P=4 workers on 8 HIP streams, averaging every 8 steps per replica, "
                          "momentum 0.9, async"),
        "resnet50_bf16": (lambda: PM.resnet50(1000), (3, 224, 224), 1000, lpp.BF16, 2, 8,
                          "ResNet-50 (1000 classes), batch 32 of 3x224x224, bf16 activations / fp32 master "
                          "weights, K=2 x P=4 workers on 8 HIP streams, averaging every 8 steps per replica, "
                          "momentum 0.9, async", 32),
        "squeezenet_k2": (lambda: PM.squeezenet_p4(10), (3, 32, 32), 10, lpp.FP32, 2, 8,
                          "SqueezeNet v1.0 (10 classes, 32x32), batch 128, fp32, K=2 replicas x P=4 workers on 8 "
                          "HIP streams, averaging every 8 steps per replica, momentum 0.9, async"),
    }


def run_workload_child(name, steps, hw_queues):
    """run_workload in a child process (its own hardware-queue setting)."""
    import subprocess
    env = dict(os.environ)
    env["GPU_MAX_HW_QUEUES"] = str(hw_queues)
    r = subprocess.run([sys.executable, os.path.abspath(__file__), "--only-workload", name, "--workload-steps",
                        str(steps)], env=env, capture_output=True, text=True, timeout=900)
    if r.returncode != 0:
        raise RuntimeError("workload %s failed (exit %d):\n%s" % (name, r.returncode, r.stderr[-3000:]))
    out = json.loads(r.stdout.strip().splitlines()[-1])
    out["hw_queues"] = int(env.get("GPU_MAX_HW_QUEUES", "4"))
    return out


def run_workload(torch, lpp, name, steps, B=128, P=4):
    """Short async run of one configuration: warm-up (graphs captured),
    then `steps` worker steps issued round-robin over the K*P workers with
    an averaging round whenever every replica has advanced H steps; then
    the kernel families on worker 0 alone."""
    import synth
    build, shape, ncls, dtype, K, H, desc = _workloads()[name][:7]
    B = (_workloads()[name][7:] or (B,))[0]
    model = build()
    info = lpp.describe(model, B, dtype=dtype)
    pool = []
    for b in range(4):
        img = synth.images(200 + b, B, *shape)
        if dtype == lpp.BF16:
            img = synth.round_to_bf16(img)
        pool.append((torch.from_numpy(img).cuda(), torch.from_numpy(synth.labels(200 + b, B, ncls)).cuda()))
    streams = [torch.cuda.Stream() for _ in range(K * P)]
    ctx = lpp.Context(model, K=K, batch=B, mode=lpp.ASYNC, dtype=dtype, momentum=0.9, streams=streams,
                      avg_stream=torch.cuda.Stream())
    ctx.set_params(synth.init_params(model.specs, 2))
    nw = K * P

    def issue(n, start):
        for s in range(start, start + n):
            w = s % nw
            img, lab = pool[(s // nw) % len(pool)]
            ctx.step(w, img, lab, w % P + 1, 0.05)
            if (s + 1) % (H * K) == 0:
                ctx.average()

    issue(2 * nw, 0)
    ctx.sync()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    issue(steps, 2 * nw)
    ctx.sync()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    fams = {}
    for f in FAMILIES:
        ctx.timer_enable(f)
        for s in range(P):
            img, lab = pool[s % len(pool)]
            ctx.step(0, img, lab, s + 1, 0.0)
        ms, n, work = ctx.timer_read()
        fams[f] = (ms, n, work)
    ctx.timer_enable(None)
    loss = ctx.get_loss(0)
    ctx.close()
    dom = max(fams, key=lambda f: fams[f][0])
    ms, n, work = fams[dom]
    mfma = dom.startswith("conv_")
    peak = (PEAK_BF16_TFLOPS if dtype == lpp.BF16 else PEAK_FP32_TFLOPS) if mfma else PEAK_HBM_GBS
    ach = work / (ms / 1e3) / (1e12 if mfma else 1e9) if ms > 0 else 0.0
    mean_flops = info.fwd_flops + sum(info.bwd_flops[i] for i in range(1, P + 1)) / P
    conv = {f: round(fams[f][2] / (fams[f][0] / 1e3) / 1e12, 1) for f in ("conv_fwd", "conv_dgrad", "conv_wgrad")
            if fams[f][0] > 0}
    hbm = {f: round(fams[f][2] / (fams[f][0] / 1e3) / 1e9, 1)
           for f in ("snapshot", "sgd_update", "bn_act", "bn_bwd", "maxpool", "relu", "add", "concat", "image")
           if f in fams and fams[f][0] > 0 and fams[f][2] > 0}
    return {"workload": desc, "dtype": "bf16" if dtype == lpp.BF16 else "f32", "value": round(B * steps / dt, 1),
            "unit": "samples/s", "steps": steps, "ms_per_step": round(dt / steps * 1e3, 4),
            "mean_step_gflop": round(mean_flops / 1e9, 2), "model_tflops": round(mean_flops * steps / dt / 1e12, 2),
            "roofline": {"kernel": dom, "bound": "mfma" if mfma else "hbm", "achieved": round(ach, 2),
                         "peak": peak, "unit": "TFLOP/s" if mfma else "GB/s", "frac": round(ach / peak, 4),
                         "timed": "HIP events in the dispatch packets of each launch, worker 0 alone, "
                                   "partitions 1..4"},
            "conv_tflops_by_family": conv,
            "hbm_gbs_by_family": hbm,
            "family_ms_per_4_steps": {f: round(v[0], 3) for f, v in sorted(fams.items(), key=lambda t: -t[1][0])},
            "final_loss_worker0": round(loss, 4)}


# ---------------------------------------------------------------------------
# HBM traffic of the roofline kernel: FETCH_SIZE and WRITE_SIZE per dispatch
# from two rocprofv3 --pmc runs of --roofline-only, each scaled by what the
# same counter reads for a plain copy of known size (--copy-calibration).
# The summary records a hash of the kernel sources; a later change to them
# makes the figure stale and bench.py then reports traffic as null.

TRAFFIC_FILE = os.path.join(ROOT, "profiles", "conv_fwd_resnet20_b128_fp32_traffic.md")
TRAFFIC_SOURCES = ["paper_2203_06638_amd/csrc/conv_f32.hip", "paper_2203_06638_amd/csrc/launch.h",
                   "paper_2203_06638_amd/csrc/bnacc.h"]
COPY_BYTES = 256 << 20
# kernel-name prefixes of each timed family (the library's launchers)
FAMILY_KERNELS = {"conv_fwd": ("void lpp::conv_tile_f32<0,", "void lpp::conv_igemm_f32<0,", "void lpp::conv_lds_f32<0,",
                               "void lpp::conv_bf16_k<"),
                  "sgd_update": ("lpp::sgd_update_k(",),
                  "average": ("void lpp::average_k<",)}


def _sources_hash():
    import hashlib
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _counter_rows(d, counter):
    """(kernel name, value) per dispatch from a rocprofv3 counter-collection
    CSV under directory d."""
    import csv
    import glob
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] == counter:
                    rows.append((r["Kernel_Name"], float(r["Counter_Value"])))
    return rows


def summarize_traffic(fetch_dir, write_dir, cfetch_dir, cwrite_dir, family="conv_fwd"):
    pref = FAMILY_KERNELS[family]
    out = {}
    for key, d, cd, counter in (("fetch", fetch_dir, cfetch_dir, "FETCH_SIZE"),
                                ("write", write_dir, cwrite_dir, "WRITE_SIZE")):
        fam = [v for k, v in _counter_rows(d, counter) if k.startswith(pref)]
        cal = _counter_rows(cd, counter)
        # the copy kernel: the dispatches with the largest reading
        top = max(v for _, v in cal)
        cal_vals = [v for _, v in cal if v >= 0.9 * top]
        kib = sum(cal_vals) / len(cal_vals)
        factor = COPY_BYTES / (kib * 1024.0)
        out[key] = {"launches": len(fam), "kib_per_launch": round(sum(fam) / len(fam), 1),
                    "copy_kib": round(kib, 1), "copy_bytes": COPY_BYTES, "factor": round(factor, 4),
                    "bytes_per_launch": round(sum(fam) / len(fam) * 1024.0 * factor)}
    out["traffic_bytes_per_launch"] = out["fetch"]["bytes_per_launch"] + out["write"]["bytes_per_launch"]
    out["family"] = family
    out["sources_sha256"] = _sources_hash()
    return out


def read_traffic():
    """Bytes per launch of the roofline family from the committed summary,
    or None if there is none or the kernel sources changed since."""
    try:
        with open(TRAFFIC_FILE) as fh:
            for line in fh:
                if line.startswith("TRAFFIC_JSON "):
                    t = json.loads(line[len("TRAFFIC_JSON "):])
                    return t["traffic_bytes_per_launch"] if t["sources_sha256"] == _sources_hash() else None
    except OSError:
        return None
    return None


def mode_and_stream_extras(torch, steps=400, warmup=40, B=128):
    """Two extras on the headline workload (ResNet-20, batch 128, async,
    momentum 0.9, one worker per stream): the partial backward's throughput
    against the full one (every worker on its own block = LPP, every worker on
    the whole model = LAP, and the policy's steady state of alternating the
    two), and the throughput against the number of blocks and worker streams
    P (units split into P runs of consecutive units; P = 4 is the balanced
    split of the headline)."""
    import synth
    from paper_2203_06638_amd import lpp
    from paper_2203_06638_amd import models as PM
    pool = []
    for b in range(8):
        pool.append((torch.from_numpy(synth.images(300 + b, B, 3, 32, 32)).cuda(),
                     torch.from_numpy(synth.labels(300 + b, B, 10)).cuda()))

    def rate(model, part_of):
        P = model.P
        streams = [torch.cuda.Stream() for _ in range(P)]
        ctx = lpp.Context(model, K=1, batch=B, mode=lpp.ASYNC, momentum=0.9, streams=streams)
        ctx.set_params(synth.init_params(model.specs, 1))

        def issue(n, start):
            for s in range(start, start + n):
                w = s % P
                img, lab = pool[(s // P) % len(pool)]
                ctx.step(w, img, lab, part_of(w, s // P), 0.1)

        issue(warmup + 2 * P, 0)      # every (worker, partition) graph captured
        ctx.sync()
        t0 = time.perf_counter()
        issue(steps, warmup + 2 * P)
        ctx.sync()
        dt = time.perf_counter() - t0
        ctx.close()
        return round(B * steps / dt, 1)

    m4 = PM.resnet20(10)
    modes = {"lpp": rate(m4, lambda w, it: w + 1),
             "lap": rate(m4, lambda w, it: 0),
             "alternating": rate(m4, lambda w, it: 0 if it % 2 == 0 else w + 1)}
    modes["lpp_over_lap"] = round(modes["lpp"] / modes["lap"], 3)
    sweep = {}
    for P in (1, 2, 4, 6, 8):
        n_units = 11
        blocks = [1, 1, 1, 2, 2, 3, 3, 3, 4, 4, 4] if P == 4 else [u * P // n_units + 1 for u in range(n_units)]
        sweep[str(P)] = rate(PM.resnet_cifar(20, (16, 32, 64), 10, blocks=blocks), lambda w, it: w + 1)
    return {"workload": "ResNet-20 (10 classes), batch 128, fp32, async, momentum 0.9, one worker per stream",
            "steps": steps, "modes_samples_per_s": modes, "streams_samples_per_s": sweep}


def delay_statistics(torch, Hs=(1, 2, 4, 8, 16), T=256, B=128):
    """Traced async runs of the LPP-SGD policy (ResNet-20, K = 2 replicas x
    P = 4 workers, T updates per replica, T_st = T/10) for several
    synchronization periods H: the estimated probability of Assumption 1's
    good iterates and the staleness of the snapshots."""
    import synth
    from paper_2203_06638_amd import delays as D
    from paper_2203_06638_amd import lpp
    from paper_2203_06638_amd import models as PM
    from paper_2203_06638_amd import policy as PL
    model = PM.resnet20(10)
    pool = [(torch.from_numpy(synth.images(300 + b, B, 3, 32, 32)).cuda(),
             torch.from_numpy(synth.labels(300 + b, B, 10)).cuda()) for b in range(4)]
    out = {"workload": "ResNet-20 (10 classes), batch %d, fp32, K=2 replicas x P=4 workers, async, T=%d updates "
                       "per replica, T_st=T/10, warm-up + cosine LR" % (B, T), "runs": {}}
    for H in Hs:
        ctx = lpp.Context(model, K=2, batch=B, mode=lpp.ASYNC, momentum=0.9,
                          streams=[torch.cuda.Stream() for _ in range(8)], avg_stream=torch.cuda.Stream())
        ctx.set_params(synth.init_params(model.specs, 3))
        ctx.trace_enable(4 * T)
        PL.run(ctx, pool, PL.Schedule(T=T, T_st=T // 10, H=H, base_lr=0.05, warm_lr=0.125, warmup=T // 10))
        steps, rounds, khz = ctx.trace_read()
        ctx.close()
        _, summ = D.analyze(steps, rounds)
        summ.pop("staleness_hist")
        out["runs"]["H=%d" % H] = summ
    return out


def _oracle_rate(o, shape, ncls, batch, steps, bf16, seed):
    """Samples/s of the oracle's updater iteration (snapshot, forward, full
    backward restricted to the block, update) over `steps` steps, partitions
    cycling over the blocks."""
    import synth
    from oracle import lppref as R
    x = synth.init_params(o.specs, seed).astype(np.float64)
    m = np.zeros(o.d)
    img = synth.images(seed + 6, batch, *shape)
    if bf16:
        img = synth.round_to_bf16(img)
    lab = synth.labels(seed + 6, batch, ncls)
    R.step(o, x, m, img[:1], lab[:1], o.P, 0.0, 0.9)   # load and warm the library
    t0 = time.perf_counter()
    for s in range(steps):
        R.step(o, x, m, img, lab, s % o.P + 1, 0.1, 0.9)
    dt = time.perf_counter() - t0
    return batch * steps / dt, dt


def cpu_baseline(steps, batch):
    """The oracle (fp64 C, OpenMP), compiled for this host (-O3
    -march=native), timed on bounded samples: `steps` ResNet-20 worker steps
    at the headline's batch, and 2 steps each of WRN-16-8 (batch 4) and
    ResNet-18 at 224x224 (batch 2) -- the oracle's time is linear in the
    batch, so samples/s of a small batch stands for the workload's."""
    import tempfile
    from oracle import build as OB
    from oracle import lppref as R
    from oracle import models as OM
    R.use_library(OB.build_native(tempfile.mkdtemp(prefix="lppref_native_")))
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    build = "gcc -O3 -march=native -fopenmp"
    v, dt = _oracle_rate(OM.resnet20_p4(), (3, 32, 32), 10, batch, steps, False, 1)
    head = {"value": round(v, 2), "unit": "samples/s", "cores": threads, "kind": "oracle", "build": build,
            "sample": "%d ResNet-20 worker steps (fwd + full bwd restricted to the block + update), batch %d, "
                      "fp64, %.1f s" % (steps, batch, dt)}
    others = {}
    for name, o, shape, ncls, b in (("wrn16_8_bf16", OM.wrn16_8_p4(), (3, 32, 32), 100, 4),
                                    ("resnet18_bf16", OM.resnet18_p4(), (3, 224, 224), 1000, 2)):
        v, dt = _oracle_rate(o, shape, ncls, b, 2, True, 2)
        others[name] = {"value": round(v, 3), "unit": "samples/s", "cores": threads, "kind": "oracle",
                        "build": build, "sample": "2 worker steps at batch %d (fp64 on the bf16-rounded images), "
                                                  "%.1f s" % (b, dt)}
    return head, others


def main():
    a = parse()
    if a.summarize_traffic:
        t = summarize_traffic(*a.summarize_traffic, family=a.traffic_family)
        print("TRAFFIC_JSON " + json.dumps(t))
        return
    if a.gpus != 1:
        print("bench.py measures one GPU only: the library runs the per-node step on a single MI355X "
              "(--gpus %d is not supported)" % a.gpus, file=sys.stderr)
        sys.exit(2)
    if not (1 <= a.hw_queues <= 32 and 1 <= a.workload_hw_queues <= 32):
        print("hardware queues must be in 1..32", file=sys.stderr)
        sys.exit(2)
    if not a.only_workload:
        os.environ["GPU_MAX_HW_QUEUES"] = str(a.hw_queues)
    import torch
    import synth
    from paper_2203_06638_amd import lpp
    from paper_2203_06638_amd import models as PM

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.init()
    if a.copy_calibration:
        x = torch.empty(COPY_BYTES // 4, device="cuda")
        y = torch.empty_like(x)
        x.fill_(1.0)
        for _ in range(10):
            y.copy_(x)
        torch.cuda.synchronize()
        print("copied %d bytes ten times" % COPY_BYTES)
        return
    if a.delays:
        print(json.dumps(delay_statistics(torch)), flush=True)
        return
    if a.extras:
        print(json.dumps(mode_and_stream_extras(torch)), flush=True)
        return
    if a.hbm_only:
        print(json.dumps(hbm_kernels(torch, lpp)), flush=True)
        return
    if a.only_workload:
        from paper_2203_06638_amd import lpp as _lpp
        print(json.dumps(run_workload(torch, _lpp, a.only_workload, a.workload_steps)), flush=True)
        return
    B, P, K = a.batch, 4, a.replicas
    model = PM.resnet20(10)
    info = lpp.describe(model, B)
    x0 = synth.init_params(model.specs, 1)
    pool = []
    for b in range(8):
        img = torch.from_numpy(synth.images(100 + b, B, 3, 32, 32)).cuda()
        lab = torch.from_numpy(synth.labels(100 + b, B, 10)).cuda()
        pool.append((img, lab))
    streams = [torch.cuda.Stream() for _ in range(K * P)]
    ctx = lpp.Context(model, K=K, batch=B, mode=lpp.ASYNC, momentum=0.9, streams=streams)
    ctx.set_params(x0)

    issue = [0.0]
    nw = a.workers_used or K * P
    nthr = max(1, min(a.issue_threads, nw))

    def run_range(start, n, thr):
        for s in range(start, start + n):
            w = s % nw
            if w % nthr != thr:
                continue
            img, lab = pool[(s // nw) % len(pool)]
            ctx.step(w, img, lab, w % P + 1, 0.1)

    def run(n, start):
        # step s goes to worker s mod (K*P); worker w is always issued by
        # host thread w mod nthr, so one worker is never entered twice at once
        t = time.perf_counter()
        if nthr == 1:
            run_range(start, n, 0)
        else:
            ths = [threading.Thread(target=run_range, args=(start, n, i)) for i in range(nthr)]
            for th in ths:
                th.start()
            for th in ths:
                th.join()
        issue[0] += time.perf_counter() - t

    run(a.warmup, 0)
    ctx.sync()
    if a.roofline_only:
        ctx.timer_enable(a.roofline_only)
        for s in range(a.steps):
            img, lab = pool[s % len(pool)]
            ctx.step(0, img, lab, s % P + 1, 0.1)
        ms, launches, work = ctx.timer_read()
        ctx.timer_enable(None)
        ctx.close()
        print(json.dumps({"family": a.roofline_only, "launches": launches, "avg_launch_us": ms / launches * 1e3,
                          "work_per_launch": work / launches}))
        return
    # find the dominant kernel family on a short untimed pass (a kernel timer
    # makes the library launch kernels one by one so each can be bracketed)
    fam_time = {}
    probe = 4 * P
    pos = a.warmup
    for f in FAMILIES:
        ctx.timer_enable(f)
        run(probe, pos)
        pos += probe
        ms, n, work = ctx.timer_read()
        fam_time[f] = ms
    ctx.timer_enable(None)
    dom = max(fam_time, key=fam_time.get)
    run(4 * P, pos)                      # graphs of every (worker, partition) exist before timing
    pos += 4 * P
    # timed region: graph replays, nothing else
    ctx.sync()
    torch.cuda.synchronize()
    issue[0] = 0.0
    t0 = time.perf_counter()
    run(a.steps, pos)
    ctx.sync()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    issue_ms = issue[0] / a.steps * 1e3
    pos += a.steps
    # roofline pass: worker 0 alone on its stream, partitions cycling, every
    # launch of the dominant family bracketed by HIP events on that stream
    # (with the other streams idle the events time the kernel itself)
    rsteps = min(a.steps, 400)
    ctx.sync()
    ctx.timer_enable(dom)
    for s in range(rsteps):
        img, lab = pool[s % len(pool)]
        ctx.step(0, img, lab, s % P + 1, 0.1)
    ms, launches, work = ctx.timer_read()
    ctx.timer_enable(None)
    losses = [ctx.get_loss(w) for w in range(K * P)]
    ctx.close()

    value = B * a.steps / dt
    mfma = dom.startswith("conv_") or dom == "linear"
    scale = 1e12 if mfma else 1e9
    achieved = (work / launches) / (ms / launches / 1e3) / scale if launches else 0.0
    peak = PEAK_FP32_TFLOPS if mfma else PEAK_HBM_GBS
    mean_flops = info.fwd_flops + sum(info.bwd_flops[i] for i in range(1, P + 1)) / P
    res = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(dt / a.steps * 1e3, 4),
        "host_issue_ms_per_step": round(issue_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "ResNet-20 (10 classes), batch %d, fp32, P=4 partial-backprop workers on 4 HIP "
                               "streams, K=1, momentum 0.9, async" % B, "issue_threads": nthr,
                   "global_batch": B, "partitions": P, "replicas": K,
                   "hw_queues": int(os.environ.get("GPU_MAX_HW_QUEUES", "4")),
                   "mean_step_gflop": round(mean_flops / 1e9, 3),
                   "model_tflops": round(mean_flops * a.steps / dt / 1e12, 2)},
        "roofline": {"kernel": dom, "bound": "mfma" if mfma else "hbm", "achieved": round(achieved, 2),
                     "peak": peak, "unit": "TFLOP/s" if mfma else "GB/s", "frac": round(achieved / peak, 4),
                     "traffic": read_traffic() if dom == "conv_fwd" else None, "launches": launches, "avg_launch_us": round(ms / launches * 1e3, 2),
                     "timed": "HIP events recorded in the dispatch packets of each launch of the family "
                              "(start with its first kernel, stop with its last) on worker 0's stream, %d steps "
                              "of worker 0 alone (partitions 1..4 in turn) right after the timed region" % rsteps,
                     "family_ms_probe": {k: round(v, 3) for k, v in sorted(fam_time.items(), key=lambda t: -t[1])}},
        "final_losses": [round(l, 4) for l in losses],
    }
    if not a.no_hbm:
        res["hbm_kernels"] = hbm_kernels(torch, lpp)
    if not a.no_workloads:
        res["workloads"] = {}
        torch.cuda.empty_cache()
        for name in [w for w in a.workloads.split(",") if w]:
            res["workloads"][name] = run_workload_child(name, a.workload_steps, a.workload_hw_queues)
            print("workload %s: %s samples/s" % (name, res["workloads"][name].get("value")), file=sys.stderr,
                  flush=True)
    if not a.no_cpu_baseline:
        res["cpu_baseline"], others = cpu_baseline(a.cpu_steps, B)
        for name, cb in others.items():
            if name in res.get("workloads", {}):
                res["workloads"][name]["cpu_baseline"] = cb
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

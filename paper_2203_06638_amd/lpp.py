"""Python binding of liblpp.so (argument marshalling only).

Every step of the LPP-SGD hot path runs in the HIP library; this module only
converts Python/torch arguments to the C ABI of include/lpp.h and raises
LppError on a non-zero status.  torch provides device memory and streams.
The library must have been built (paper_2203_06638_amd/build.py); there is
no fallback of any kind.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblpp.so")
_LIB = None

CONV, BN, RELU, ADD, MAXPOOL, GAP, LINEAR, CONCAT = range(8)
FP32, BF16 = 0, 1
SEQUENTIAL, ASYNC = 0, 1
OK, EINVAL, ENOMEM, EHIP, ESTATE, EUNSUPPORTED = 0, -1, -2, -3, -4, -5
STATUS = {0: "LPP_OK", -1: "LPP_EINVAL", -2: "LPP_ENOMEM", -3: "LPP_EHIP", -4: "LPP_ESTATE", -5: "LPP_EUNSUPPORTED"}


class LppError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("%s: %s" % (STATUS.get(code, code), msg))
        self.code = code


class Layer(C.Structure):
    _fields_ = [("op", C.c_int), ("in0", C.c_int), ("in1", C.c_int), ("cin", C.c_int), ("cout", C.c_int),
                ("k", C.c_int), ("stride", C.c_int), ("pad", C.c_int), ("bias", C.c_int), ("block", C.c_int)]


class ModelDesc(C.Structure):
    _fields_ = [("n_layers", C.c_int), ("layers", C.POINTER(Layer)), ("in_c", C.c_int), ("in_h", C.c_int),
                ("in_w", C.c_int), ("n_classes", C.c_int), ("batch", C.c_int), ("dtype", C.c_int),
                ("momentum", C.c_float), ("weight_decay", C.c_float), ("bn_eps", C.c_float)]


class Options(C.Structure):
    _fields_ = [("mode", C.c_int), ("worker_streams", C.POINTER(C.c_void_p)), ("avg_stream", C.c_void_p),
                ("unfused", C.c_int), ("no_graphs", C.c_int)]


class Batch(C.Structure):
    _fields_ = [("images", C.c_void_p), ("labels", C.c_void_p), ("n", C.c_int)]


class TraceStep(C.Structure):
    _fields_ = [("worker", C.c_int), ("replica", C.c_int), ("partition", C.c_int), ("counter", C.c_long),
                ("t", C.c_ulonglong * 4)]


class TraceAvg(C.Structure):
    _fields_ = [("index", C.c_long), ("n_replicas", C.c_int), ("counter_min", C.c_long), ("t", C.c_ulonglong * 2)]


class SnapConv(C.Structure):
    _fields_ = [("src", C.c_long), ("cout", C.c_int), ("cin", C.c_int), ("cin_p", C.c_int), ("kh", C.c_int),
                ("kw", C.c_int), ("dst_f", C.c_long), ("dst_d", C.c_long)]


class ModelInfo(C.Structure):
    _fields_ = [("d", C.c_long), ("P", C.c_int), ("block_lo", C.c_long * 65), ("block_hi", C.c_long * 65),
                ("fwd_flops", C.c_double), ("bwd_flops", C.c_double * 65)]


def lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("liblpp.so is not built (run paper_2203_06638_amd/build.py); there is no fallback")
        L = C.CDLL(LIB_PATH)
        ctx = C.c_void_p
        fp = C.POINTER(C.c_float)
        sig = {
            "lpp_describe": ([C.POINTER(ModelDesc), C.c_int, C.POINTER(ModelInfo)], C.c_int),
            "lpp_init": ([C.POINTER(ModelDesc), C.c_int, C.c_int, C.POINTER(Options), C.POINTER(ctx)], C.c_int),
            "lpp_step": ([ctx, C.c_int, C.POINTER(Batch), C.c_int, C.c_float], C.c_int),
            "lpp_average": ([ctx, C.POINTER(C.c_int), C.c_int], C.c_int),
            "lpp_set_params": ([ctx, C.c_int, fp, C.c_long], C.c_int),
            "lpp_get_params": ([ctx, C.c_int, fp, C.c_long], C.c_int),
            "lpp_get_grad": ([ctx, C.c_int, fp, C.c_long], C.c_int),
            "lpp_get_momentum": ([ctx, C.c_int, fp, C.c_long], C.c_int),
            "lpp_set_momentum": ([ctx, C.c_int, fp, C.c_long], C.c_int),
            "lpp_get_loss": ([ctx, C.c_int, fp], C.c_int),
            "lpp_get_logits": ([ctx, C.c_int, fp, C.c_long], C.c_int),
            "lpp_get_activation": ([ctx, C.c_int, C.c_int, fp, C.c_long], C.c_int),
            "lpp_get_activation_grad": ([ctx, C.c_int, C.c_int, fp, C.c_long], C.c_int),
            "lpp_num_params": ([ctx], C.c_long),
            "lpp_block_range": ([ctx, C.c_int, C.POINTER(C.c_long), C.POINTER(C.c_long)], C.c_int),
            "lpp_counter": ([ctx, C.c_int], C.c_long),
            "lpp_sync": ([ctx], C.c_int),
            "lpp_destroy": ([ctx], C.c_int),
            "lpp_last_error": ([], C.c_char_p),
            "lpp_timer_enable": ([ctx, C.c_char_p], C.c_int),
            "lpp_timer_read": ([ctx, C.POINTER(C.c_double), C.POINTER(C.c_long), C.POINTER(C.c_double)], C.c_int),
            "lpp_trace_enable": ([ctx, C.c_long], C.c_int),
            "lpp_trace_read": ([ctx, C.POINTER(TraceStep), C.c_long, C.POINTER(C.c_long), C.POINTER(TraceAvg), C.c_long,
                                C.POINTER(C.c_long)], C.c_int),
            "lpp_trace_clock_khz": ([ctx], C.c_long),
            "lpp_kernel_sgd_update": ([C.c_void_p, C.c_void_p, C.c_void_p, C.c_long, C.c_float, C.c_float,
                                       C.c_float, C.c_void_p], C.c_int),
            "lpp_kernel_average": ([C.POINTER(C.c_void_p), C.c_int, C.c_long, C.c_void_p], C.c_int),
            "lpp_snapshot_plan_create": ([C.POINTER(SnapConv), C.c_int, C.c_long, C.c_int, C.c_long,
                                          C.POINTER(C.c_void_p)], C.c_int),
            "lpp_kernel_snapshot": ([C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p], C.c_int),
            "lpp_snapshot_plan_destroy": ([C.c_void_p], C.c_int),
            "lpp_kernel_snapshot_noalloc": ([C.POINTER(SnapConv), C.c_int, C.c_long, C.c_int, C.c_long, C.c_void_p,
                                             C.c_void_p, C.c_void_p, C.c_void_p], C.c_int),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _LIB = L
    return _LIB


def _check(rc):
    if rc != 0:
        raise LppError(rc, lib().lpp_last_error().decode())


def _fptr(a):
    return a.ctypes.data_as(C.POINTER(C.c_float))


def make_desc(model, batch, dtype=FP32, momentum=0.0, weight_decay=0.0, bn_eps=1e-5):
    """ModelDesc for a models.Model; the returned object keeps its layer
    array alive."""
    arr = (Layer * len(model.layers))(*[Layer(*rec) for rec in model.layers])
    c, h, w = model.in_shape
    desc = ModelDesc(len(model.layers), arr, c, h, w, model.n_classes, batch, dtype, momentum, weight_decay, bn_eps)
    desc._keep = arr
    return desc


def describe(model, batch=1, **kw):
    info = ModelInfo()
    desc = make_desc(model, batch, **kw)
    _check(lib().lpp_describe(C.byref(desc), model.P, C.byref(info)))
    return info


def _stream_handle(s):
    if s is None:
        return None
    return C.c_void_p(s.cuda_stream if hasattr(s, "cuda_stream") else int(s))


class Context:
    """One lpp_ctx: K replicas x P workers of `model` on the current device."""

    def __init__(self, model, K, batch, mode=SEQUENTIAL, dtype=FP32, momentum=0.0, weight_decay=0.0,
                 bn_eps=1e-5, streams=None, avg_stream=None, unfused=False, graphs=True):
        self.model = model
        self.K, self.P, self.batch = K, model.P, batch
        self._desc = make_desc(model, batch, dtype, momentum, weight_decay, bn_eps)
        opt = Options(mode, None, None, int(unfused), int(not graphs))
        if streams is not None:
            assert len(streams) == K * model.P
            self._streams = (C.c_void_p * len(streams))(*[_stream_handle(s).value for s in streams])
            opt.worker_streams = C.cast(self._streams, C.POINTER(C.c_void_p))
        if avg_stream is not None:
            opt.avg_stream = _stream_handle(avg_stream)
        self._ctx = C.c_void_p()
        _check(lib().lpp_init(C.byref(self._desc), K, model.P, C.byref(opt), C.byref(self._ctx)))
        self.d = int(lib().lpp_num_params(self._ctx))

    # -- the three calls of the method --
    def step(self, worker, images, labels, partition, lr):
        """images: device float32 NCHW tensor; labels: device int32 tensor."""
        b = Batch(images.data_ptr(), labels.data_ptr(), images.shape[0])
        _check(lib().lpp_step(self._ctx, worker, C.byref(b), partition, lr))

    def average(self, replicas=None):
        if replicas is None:
            _check(lib().lpp_average(self._ctx, None, 0))
        else:
            arr = (C.c_int * len(replicas))(*replicas)
            _check(lib().lpp_average(self._ctx, arr, len(replicas)))

    # -- accessors --
    def set_params(self, x, replica=-1):
        x = np.ascontiguousarray(x, np.float32)
        assert x.shape == (self.d,)
        _check(lib().lpp_set_params(self._ctx, replica, _fptr(x), self.d))

    def get_params(self, replica=0):
        out = np.empty(self.d, np.float32)
        _check(lib().lpp_get_params(self._ctx, replica, _fptr(out), self.d))
        return out

    def get_grad(self, worker):
        out = np.empty(self.d, np.float32)
        _check(lib().lpp_get_grad(self._ctx, worker, _fptr(out), self.d))
        return out

    def get_momentum(self, worker):
        out = np.empty(self.d, np.float32)
        _check(lib().lpp_get_momentum(self._ctx, worker, _fptr(out), self.d))
        return out

    def set_momentum(self, worker, m):
        m = np.ascontiguousarray(m, np.float32)
        _check(lib().lpp_set_momentum(self._ctx, worker, _fptr(m), self.d))

    def get_loss(self, worker):
        out = np.zeros(1, np.float32)
        _check(lib().lpp_get_loss(self._ctx, worker, _fptr(out)))
        return float(out[0])

    def get_logits(self, worker):
        out = np.empty((self.batch, self.model.n_classes), np.float32)
        _check(lib().lpp_get_logits(self._ctx, worker, _fptr(out), out.size))
        return out

    def get_activation(self, worker, layer, shape):
        out = np.empty((self.batch,) + tuple(shape), np.float32)
        _check(lib().lpp_get_activation(self._ctx, worker, layer, _fptr(out), out.size))
        return out

    def get_activation_grad(self, worker, layer, shape):
        out = np.empty((self.batch,) + tuple(shape), np.float32)
        _check(lib().lpp_get_activation_grad(self._ctx, worker, layer, _fptr(out), out.size))
        return out

    def block_range(self, i):
        lo, hi = C.c_long(), C.c_long()
        _check(lib().lpp_block_range(self._ctx, i, C.byref(lo), C.byref(hi)))
        return lo.value, hi.value

    def counter(self, replica):
        return int(lib().lpp_counter(self._ctx, replica))

    def sync(self):
        _check(lib().lpp_sync(self._ctx))

    def timer_enable(self, family):
        _check(lib().lpp_timer_enable(self._ctx, family.encode() if family else None))

    def timer_read(self):
        ms, n, work = C.c_double(), C.c_long(), C.c_double()
        _check(lib().lpp_timer_read(self._ctx, C.byref(ms), C.byref(n), C.byref(work)))
        return ms.value, n.value, work.value

    def trace_enable(self, capacity):
        _check(lib().lpp_trace_enable(self._ctx, capacity))

    def trace_read(self):
        """(steps, rounds, clock_khz): lists of dicts in issue order."""
        ns, na = C.c_long(), C.c_long()
        _check(lib().lpp_trace_read(self._ctx, None, 0, C.byref(ns), None, 0, C.byref(na)))
        st = (TraceStep * max(1, ns.value))()
        av = (TraceAvg * max(1, na.value))()
        _check(lib().lpp_trace_read(self._ctx, st, ns.value, C.byref(ns), av, na.value, C.byref(na)))
        steps = [dict(worker=r.worker, replica=r.replica, partition=r.partition, counter=r.counter, t=list(r.t))
                 for r in st[:ns.value]]
        rounds = [dict(index=r.index, n_replicas=r.n_replicas, counter_min=r.counter_min, t=list(r.t))
                  for r in av[:na.value]]
        return steps, rounds, int(lib().lpp_trace_clock_khz(self._ctx))

    def close(self):
        if self._ctx:
            _check(lib().lpp_destroy(self._ctx))
            self._ctx = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()


def kernel_sgd_update(x, m, g, lr, mu=0.0, wd=0.0, stream=None):
    """In-place block update on whole device tensors x, m (or None), g."""
    _check(lib().lpp_kernel_sgd_update(x.data_ptr(), m.data_ptr() if m is not None else None, g.data_ptr(),
                                       x.numel(), lr, mu, wd, _stream_handle(stream)))


def kernel_average(reps, stream=None):
    """In-place averaging round over a list of equally sized device tensors."""
    arr = (C.c_void_p * len(reps))(*[r.data_ptr() for r in reps])
    _check(lib().lpp_kernel_average(arr, len(reps), reps[0].numel(), _stream_handle(stream)))


def _snap_convs(convs):
    """host array of lpp_snap_conv from (src, cout, cin, cin_p, kh, kw, dst_f, dst_d) tuples"""
    return (SnapConv * max(1, len(convs)))(*[SnapConv(*c) for c in convs])


class SnapshotPlan:
    """lpp_snapshot_plan_create / lpp_kernel_snapshot / lpp_snapshot_plan_destroy.
    convs: (src, cout, cin, cin_p, kh, kw, dst_f, dst_d) tuples sorted by src."""

    def __init__(self, convs, d, dtype, wbuf_elems):
        arr = _snap_convs(convs)
        self._p = C.c_void_p()
        _check(lib().lpp_snapshot_plan_create(arr, len(convs), d, dtype, wbuf_elems, C.byref(self._p)))

    def run(self, x, v, wbuf, stream=None):
        """x, v: device float32 tensors of d floats; wbuf: device tensor of
        wbuf_elems float32 (FP32) or 16-bit (BF16) elements."""
        _check(lib().lpp_kernel_snapshot(self._p, x.data_ptr(), v.data_ptr(), wbuf.data_ptr(),
                                         _stream_handle(stream)))

    def close(self):
        if self._p:
            _check(lib().lpp_snapshot_plan_destroy(self._p))
            self._p = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def kernel_snapshot_noalloc(convs, d, dtype, wbuf_elems, x, v, wbuf, stream=None):
    """lpp_kernel_snapshot_noalloc on device tensors (see SnapshotPlan.run)."""
    arr = _snap_convs(convs)
    _check(lib().lpp_kernel_snapshot_noalloc(arr, len(convs), d, dtype, wbuf_elems, x.data_ptr(), v.data_ptr(),
                                             wbuf.data_ptr(), _stream_handle(stream)))

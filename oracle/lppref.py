"""ctypes front end of the fp64 CPU oracle (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this module.  It loads oracle/liblppref.so (built by oracle/build.py) and
never touches the HIP library.

Functions follow the paper's Algorithm 1 (arXiv 2203.06638, Sec. 3):
  forward_backward : loss, logits and the full minibatch gradient at x
  block_update     : x_i -= lr * direction over block i only (Sec. 5, -|_i)
  step             : one updater iteration with a zero-delay snapshot
  average          : one averaging round over replicas
  run_sequential   : the deterministic sequential schedule of updaters and
                     averaging rounds (zero-delay case of eqs. (minoriter),
                     (majoriter), (update) of Sec. 5)
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from . import models as M

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

BN_EPS = 1e-5


class RefLayer(C.Structure):
    _fields_ = [("op", C.c_int), ("in0", C.c_int), ("in1", C.c_int), ("cin", C.c_int), ("cout", C.c_int),
                ("k", C.c_int), ("stride", C.c_int), ("pad", C.c_int), ("bias", C.c_int), ("poff", C.c_long)]


def use_library(path):
    """Load the oracle from another build of lppref.c (e.g. build_native)."""
    global _LIB
    _LIB = _load(path)


def lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "liblppref.so")
        if not os.path.exists(path):
            from . import build as _b
            _b.build()
        _LIB = _load(path)
    return _LIB


def _load(path):
    L = C.CDLL(path)
    dp = C.POINTER(C.c_double)
    L.ref_forward_backward.argtypes = [C.POINTER(RefLayer), C.c_int, C.c_int, C.c_int, C.c_int, C.c_int,
                                       dp, dp, C.POINTER(C.c_int), C.c_double, dp, dp, dp]
    L.ref_num_params.argtypes = [C.POINTER(RefLayer), C.c_int]
    L.ref_num_params.restype = C.c_long
    L.ref_shapes.argtypes = [C.POINTER(RefLayer), C.c_int, C.c_int, C.c_int, C.c_int, C.POINTER(C.c_int)]
    L.ref_block_update.argtypes = [dp, dp, dp, C.c_long, C.c_long, C.c_double, C.c_double, C.c_double]
    L.ref_average.argtypes = [C.POINTER(dp), C.c_int, C.c_long]
    L.ref_step.argtypes = [C.POINTER(RefLayer), C.c_int, C.c_int, C.c_int, C.c_int, C.c_int,
                           dp, dp, dp, C.POINTER(C.c_int), C.c_long, C.c_long, C.c_double, C.c_double,
                           C.c_double, C.c_double, dp, dp, dp]
    L.ref_activation_grad.argtypes = [C.POINTER(RefLayer), C.c_int, C.c_int, C.c_int, C.c_int, C.c_int,
                                      dp, dp, C.POINTER(C.c_int), C.c_double, C.c_int, dp]
    L.ref_grad_scale.argtypes = [C.POINTER(RefLayer), C.c_int, C.c_int, C.c_int, C.c_int, C.c_int,
                                 dp, dp, C.POINTER(C.c_int), C.c_double, dp, dp]
    L.ref_kink_margin.argtypes = [C.POINTER(RefLayer), C.c_int, C.c_int, C.c_int, C.c_int, C.c_int,
                                  dp, dp, C.c_double, dp]
    L.ref_activation.argtypes = [C.POINTER(RefLayer), C.c_int, C.c_int, C.c_int, C.c_int, C.c_int,
                                 dp, dp, C.c_double, C.c_int, dp]
    return L


def _dp(a):
    return a.ctypes.data_as(C.POINTER(C.c_double))


def _layers(net):
    arr = (RefLayer * len(net.layers))()
    for i, r in enumerate(net.layers):
        arr[i] = RefLayer(r["op"], r["in0"], r["in1"], r["cin"], r["cout"], r["k"], r["stride"], r["pad"],
                          r["bias"], r["poff"])
    return arr


def num_params(net):
    return int(lib().ref_num_params(_layers(net), len(net.layers)))


def shapes(net):
    out = np.zeros(3 * len(net.layers), np.int32)
    rc = lib().ref_shapes(_layers(net), len(net.layers), *net.in_shape, out.ctypes.data_as(C.POINTER(C.c_int)))
    if rc:
        raise ValueError("inconsistent model")
    return out.reshape(-1, 3)


def forward_backward(net, x, images, labels, grad=True):
    """Returns (loss, logits[N, classes], grad[d] or None), all fp64."""
    x = np.ascontiguousarray(x, np.float64)
    img = np.ascontiguousarray(images, np.float64)
    lab = np.ascontiguousarray(labels, np.int32)
    n = img.shape[0]
    assert img.shape[1:] == net.in_shape and x.shape == (net.d,)
    logits = np.zeros((n, net.n_classes), np.float64)
    loss = np.zeros(1, np.float64)
    g = np.zeros(net.d, np.float64) if grad else None
    rc = lib().ref_forward_backward(_layers(net), len(net.layers), n, *net.in_shape, _dp(x), _dp(img),
                                    lab.ctypes.data_as(C.POINTER(C.c_int)), BN_EPS, _dp(logits), _dp(loss),
                                    _dp(g) if grad else None)
    if rc:
        raise ValueError("inconsistent model")
    return float(loss[0]), logits, g


def activation(net, x, images, layer):
    """Forward only; the output of layer `layer` as an fp64 NCHW array."""
    x = np.ascontiguousarray(x, np.float64)
    img = np.ascontiguousarray(images, np.float64)
    n = img.shape[0]
    c, h, w = shapes(net)[layer]
    out = np.zeros((n, c, h, w), np.float64)
    rc = lib().ref_activation(_layers(net), len(net.layers), n, *net.in_shape, _dp(x), _dp(img), BN_EPS,
                              layer, _dp(out))
    if rc:
        raise ValueError("inconsistent model")
    return out


def activation_grad(net, x, images, labels, layer):
    """Gradient of the loss w.r.t. the output of layer `layer` (fp64 NCHW)."""
    x = np.ascontiguousarray(x, np.float64)
    img = np.ascontiguousarray(images, np.float64)
    lab = np.ascontiguousarray(labels, np.int32)
    n = img.shape[0]
    c, h, w = shapes(net)[layer]
    out = np.zeros((n, c, h, w), np.float64)
    rc = lib().ref_activation_grad(_layers(net), len(net.layers), n, *net.in_shape, _dp(x), _dp(img),
                                   lab.ctypes.data_as(C.POINTER(C.c_int)), BN_EPS, layer, _dp(out))
    if rc:
        raise ValueError("inconsistent model")
    return out


def grad_scale(net, x, images, labels):
    """(gradient, condition scale): for every parameter, the full gradient
    and the sum of the magnitudes of the products it sums (fp64)."""
    x = np.ascontiguousarray(x, np.float64)
    img = np.ascontiguousarray(images, np.float64)
    lab = np.ascontiguousarray(labels, np.int32)
    g = np.zeros(net.d, np.float64)
    sc = np.zeros(net.d, np.float64)
    rc = lib().ref_grad_scale(_layers(net), len(net.layers), img.shape[0], *net.in_shape, _dp(x), _dp(img),
                              lab.ctypes.data_as(C.POINTER(C.c_int)), BN_EPS, _dp(g), _dp(sc))
    if rc:
        raise ValueError("inconsistent model")
    return g, sc


def kink_margin(net, x, images):
    """Smallest distance (relative to the layer's largest input) of any ReLU
    input from 0, or of any max-pool window's runner-up from its maximum.
    Gradients of two evaluations in different precisions agree only when
    this exceeds their disagreement on those inputs."""
    x = np.ascontiguousarray(x, np.float64)
    img = np.ascontiguousarray(images, np.float64)
    out = np.zeros(1, np.float64)
    rc = lib().ref_kink_margin(_layers(net), len(net.layers), img.shape[0], *net.in_shape, _dp(x), _dp(img),
                               BN_EPS, _dp(out))
    if rc:
        raise ValueError("inconsistent model")
    return float(out[0])


def block_update(x, m, g, lo, hi, lr, mu=0.0, wd=0.0):
    """In place on x (and m if given); see ref_block_update."""
    assert x.dtype == np.float64 and g.dtype == np.float64
    lib().ref_block_update(_dp(x), _dp(m) if m is not None else None, _dp(g), lo, hi, lr, mu, wd)


def step(net, x, m, images, labels, partition, lr, mu=0.0, wd=0.0):
    """One zero-delay updater iteration on replica x (in place, fp64).
    Returns (grad restricted to the block, loss, logits)."""
    lo, hi = net.block_range(partition)
    img = np.ascontiguousarray(images, np.float64)
    lab = np.ascontiguousarray(labels, np.int32)
    n = img.shape[0]
    g = np.zeros(net.d, np.float64)
    loss = np.zeros(1, np.float64)
    logits = np.zeros((n, net.n_classes), np.float64)
    rc = lib().ref_step(_layers(net), len(net.layers), n, *net.in_shape, _dp(x),
                        _dp(m) if m is not None else None, _dp(img), lab.ctypes.data_as(C.POINTER(C.c_int)),
                        lo, hi, lr, mu, wd, BN_EPS, _dp(g), _dp(loss), _dp(logits))
    if rc:
        raise ValueError("inconsistent model")
    return g, float(loss[0]), logits


def average(reps):
    """One averaging round over the given fp64 replica arrays (in place)."""
    n = len(reps)
    d = reps[0].shape[0]
    ptrs = (C.POINTER(C.c_double) * n)(*[_dp(r) for r in reps])
    lib().ref_average(ptrs, n, d)


def run_sequential(net, x0, schedule, batches, K, P, H, lr, mu=0.0, wd=0.0):
    """Deterministic sequential schedule.

    schedule : list of (worker, partition, batch_key) in issue order; worker w
               belongs to replica q = w // P and keeps its own momentum.
    batches  : dict batch_key -> (images, labels)
    H        : averaging period.  Replica q's counter C_q counts its updates
               (Alg. 1, read&inc); an averaging round over all K replicas runs
               as soon as every counter has advanced by at least H since the
               previous round (Alg. 1, averaging loop, s_cur - s_pre >= K_j
               with K_j = H).  H <= 0 disables averaging.
    Returns (replicas, momenta, losses).
    """
    reps = [np.array(x0, np.float64) for _ in range(K)]
    moms = [np.zeros(net.d, np.float64) for _ in range(K * P)] if mu != 0.0 else [None] * (K * P)
    counters = [0] * K
    s_pre = 0
    losses = []
    for (w, part, key) in schedule:
        q = w // P
        counters[q] += 1
        img, lab = batches[key]
        _, loss, _ = step(net, reps[q], moms[w], img, lab, part, lr, mu, wd)
        losses.append(loss)
        if H > 0 and min(counters) - s_pre >= H:
            s_pre = min(counters)
            average(reps)
    return reps, moms, losses

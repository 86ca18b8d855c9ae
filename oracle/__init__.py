"""CPU oracle for spiking-layer training: forward scan and BPTT backward.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  It shares no
code with the GPU library (``paper_2211_10725_amd``) and imports nothing from
it: both sides receive the same seeded input arrays from the caller.

The arithmetic lives in ``snn_oracle.c`` (plain C, OpenMP over independent
outputs, fixed reduction order).  This module only marshals numpy arrays and
chains layers in the paper's order (synapse -> neuron forward, loss, then the
reverse).  Every function names the passage of the paper it follows:

* eq. (3)  Heaviside spike, strict ``u > thr``;
* eq. (4)  Leaky neuron with reset by subtraction;
* eqs. (5)-(6) current-based ("Synaptic") neuron;
* eq. (7)  recurrent leaky neuron ("RLeaky", one recurrent weight per neuron);
* eqs. (8)-(9) fast-sigmoid surrogate for the spike's derivative;
* Sec. III-C / Table I  dense 784-1000-10 and conv 5C12-MP2-5C64-MP2-10 nets;
* Sec. V  rate-coded readout (class = output neuron with the most spikes);
* Sec. IV  the AdamW weight update the paper trains with.

Parity status: the dense and convolutional synapses, the scans, the losses
and the backward recursion are pinned by the tests in ``tests/test_oracle_*``
(closed forms, hand-worked tables, finite differences, library special
cases).  The placement of the surrogate slope k and the choice of a detached
reset are conventions the paper does not fix; with k = 1 the surrogate reduces
to eq. (9) exactly, which is pinned.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "snn_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

LEAKY, SYNAPTIC, RLEAKY = 0, 1, 2
NEURONS = {"leaky": LEAKY, "synaptic": SYNAPTIC, "rleaky": RLEAKY}


def build(verbose: bool = False) -> str:
    """Compile ``snn_oracle.c`` into ``liboracle.so`` with gcc (always)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
           "-ffp-contract=off", "-o", _LIB + ".tmp", _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        i64, dbl, flt, i32 = ctypes.c_int64, ctypes.c_double, ctypes.c_float, ctypes.c_int
        P = ctypes.c_void_p
        L.orc_dense_fwd.argtypes = [i64, i64, i64, P, P, P, P]
        L.orc_dense_bwd.argtypes = [i64, i64, i64, P, P, P, P, P, P]
        L.orc_conv_fwd.argtypes = [i64, i64, i64, i64, i64, i64, P, P, P, P]
        L.orc_conv_bwd.argtypes = [i64, i64, i64, i64, i64, i64, P, P, P, P, P, P]
        L.orc_maxpool2_fwd.argtypes = [i64, i64, i64, P, P, P]
        L.orc_maxpool2_bwd.argtypes = [i64, i64, i64, P, P, P]
        L.orc_scan_fwd.argtypes = [i32, i64, i64, flt, flt, flt, P, P, P, P]
        L.orc_scan_fwd_smooth.argtypes = [i32, i64, i64, dbl, dbl, dbl, dbl, i32, P, P, P, P]
        L.orc_scan_bwd.argtypes = [i32, i64, i64, dbl, dbl, dbl, dbl, dbl, i32, P, P, i32, P]
        L.orc_scan_fwd_rleaky.argtypes = [i64, i64, i64, flt, flt, P, P, P, P, P]
        L.orc_scan_fwd_smooth_rleaky.argtypes = [i64, i64, i64, dbl, dbl, dbl, i32, P, P, P, P, P]
        L.orc_scan_bwd_rleaky.argtypes = [i64, i64, i64, dbl, dbl, dbl, dbl, i32, i32, P, P, P,
                                          i32, P, P]
        L.orc_loss_ce.argtypes = [i64, i64, P, P, P]
        L.orc_loss_ce.restype = dbl
        L.orc_loss_mse.argtypes = [i64, i64, P, P, P]
        L.orc_loss_mse.restype = dbl
        L.orc_adamw.argtypes = [i64, P, P, P, P, i64, dbl, dbl, dbl, dbl, dbl]
        L.orc_num_threads.restype = i32
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def num_threads() -> int:
    return int(lib().orc_num_threads())


# --------------------------------------------------------------------------
# Primitives
# --------------------------------------------------------------------------
def dense_fwd(x, W, b=None):
    """I = x W^T + b in double (the "w x_t" term of eqs. 4/5).  x [M,n_in]."""
    x, W = _f64(x), _f64(W)
    M, n_in = x.shape
    n_out = W.shape[0]
    assert W.shape == (n_out, n_in)
    b = None if b is None else _f64(b)
    I = np.empty((M, n_out), np.float64)
    lib().orc_dense_fwd(M, n_in, n_out, _p(x), _p(W), _p(b), _p(I))
    return I


def dense_bwd(dI, x, W, want_dw=True, want_db=True, want_dx=True):
    """(dW, db, dx) of I = x W^T + b, in double."""
    dI, x, W = _f64(dI), _f64(x), _f64(W)
    M, n_out = dI.shape
    n_in = x.shape[1]
    dW = np.empty((n_out, n_in)) if want_dw else None
    db = np.empty(n_out) if want_db else None
    dx = np.empty((M, n_in)) if want_dx else None
    lib().orc_dense_bwd(M, n_in, n_out, _p(dI), _p(x), _p(W), _p(dW), _p(db), _p(dx))
    return dW, db, dx


def conv_fwd(x, w, b=None):
    """Valid KxK cross-correlation, stride 1, + bias.  x [N,C,H,W]."""
    x, w = _f64(x), _f64(w)
    N, C, H, W_ = x.shape
    Co, C2, K, K2 = w.shape
    assert C2 == C and K == K2
    b = None if b is None else _f64(b)
    y = np.empty((N, Co, H - K + 1, W_ - K + 1))
    lib().orc_conv_fwd(N, C, H, W_, Co, K, _p(x), _p(w), _p(b), _p(y))
    return y


def conv_bwd(dy, x, w, want_dw=True, want_db=True, want_dx=True):
    dy, x, w = _f64(dy), _f64(x), _f64(w)
    N, C, H, W_ = x.shape
    Co, _, K, _ = w.shape
    dw = np.empty(w.shape) if want_dw else None
    db = np.empty(Co) if want_db else None
    dx = np.empty(x.shape) if want_dx else None
    lib().orc_conv_bwd(N, C, H, W_, Co, K, _p(dy), _p(x), _p(w), _p(dw), _p(db), _p(dx))
    return dw, db, dx


def maxpool2_fwd(x):
    """2x2/2 max-pool over the last two axes; ties go to the first maximum in
    row-major window order.  Returns (pooled, argmax in 0..3 as int8)."""
    x = _f64(x)
    lead = x.shape[:-2]
    H, W_ = x.shape[-2:]
    P = int(np.prod(lead)) if lead else 1
    y = np.empty(lead + (H // 2, W_ // 2))
    arg = np.empty(lead + (H // 2, W_ // 2), np.int8)
    lib().orc_maxpool2_fwd(P, H, W_, _p(x), _p(y), _p(arg))
    return y, arg


def maxpool2_bwd(dy, arg, H, W_):
    dy = _f64(dy)
    arg = np.ascontiguousarray(arg, np.int8)
    lead = dy.shape[:-2]
    P = int(np.prod(lead)) if lead else 1
    dx = np.empty(lead + (H, W_))
    lib().orc_maxpool2_bwd(P, H, W_, _p(dy), _p(arg), _p(dx))
    return dx


def _rec_weights(v, C, dtype):
    """Recurrent weights of eq. (7), one per neuron; column c is neuron c % N."""
    v = np.ascontiguousarray(np.ravel(v), dtype=dtype)
    assert v.size >= 1 and C % v.size == 0, (v.size, C)
    return v


def scan_fwd(I, neuron, beta, thr=1.0, alpha=0.0, v=None):
    """fp32 neuron scan (eqs. 3-7).  I [T, ...] fp32 currents, time-major; v
    the recurrent weights [N] of the 'rleaky' neuron (N = last dim of I).
    Returns (z uint8, u fp32, counts fp32 [...])."""
    I = np.ascontiguousarray(I, dtype=np.float32)
    T = I.shape[0]
    C = int(np.prod(I.shape[1:]))
    z = np.empty(I.shape, np.uint8)
    u = np.empty(I.shape, np.float32)
    cnt = np.empty(I.shape[1:], np.float32)
    nt = NEURONS.get(neuron, neuron)
    if nt == RLEAKY:
        v = _rec_weights(v, C, np.float32)
        lib().orc_scan_fwd_rleaky(T, C, v.size, float(beta), float(thr), _p(v), _p(I), _p(z),
                                  _p(u), _p(cnt))
    else:
        lib().orc_scan_fwd(nt, T, C, float(alpha), float(beta), float(thr), _p(I), _p(z), _p(u),
                           _p(cnt))
    return z, u, cnt


def scan_fwd_smooth(I, neuron, beta, thr, slope, alpha=0.0, reset_surrogate=False, v=None):
    """Double-precision smooth scan for finite differences (not the method)."""
    I = _f64(I)
    T = I.shape[0]
    C = int(np.prod(I.shape[1:]))
    z = np.empty(I.shape)
    u = np.empty(I.shape)
    cnt = np.empty(I.shape[1:])
    nt = NEURONS.get(neuron, neuron)
    if nt == RLEAKY:
        v = _rec_weights(v, C, np.float64)
        lib().orc_scan_fwd_smooth_rleaky(T, C, v.size, beta, thr, slope,
                                         int(bool(reset_surrogate)), _p(v), _p(I), _p(z),
                                         _p(u), _p(cnt))
    else:
        lib().orc_scan_fwd_smooth(nt, T, C, alpha, beta, thr, slope, int(bool(reset_surrogate)),
                                  _p(I), _p(z), _p(u), _p(cnt))
    return z, u, cnt


def scan_bwd(u, g, neuron, beta, thr=1.0, slope=25.0, alpha=0.0,
             reset_surrogate=False, s_scale=1.0):
    """BPTT through the neuron scan with the fast-sigmoid surrogate (eq. 9,
    slope k).  u [T, ...] saved membrane; g = dL/dz, [T, ...] or [...] (the
    same for every t).  Returns dL/dI [T, ...] in double."""
    u = _f64(u)
    T = u.shape[0]
    C = int(np.prod(u.shape[1:]))
    g = _f64(g)
    bcast = 1 if g.shape == u.shape[1:] else 0
    if not bcast:
        assert g.shape == u.shape
    dI = np.empty(u.shape)
    lib().orc_scan_bwd(NEURONS.get(neuron, neuron), T, C, alpha, beta, thr, slope, s_scale,
                       int(bool(reset_surrogate)), _p(u), _p(g), bcast, _p(dI))
    return dI


def scan_bwd_rleaky(u, g, beta, thr, slope, v, reset_surrogate=False, s_scale=1.0,
                    smooth_z=False):
    """BPTT through the recurrent neuron of eq. (7).  Returns (dL/dI [T, ...],
    dL/dv [N]) in double; dL/dv sums the columns of each neuron."""
    u = _f64(u)
    T = u.shape[0]
    C = int(np.prod(u.shape[1:]))
    g = _f64(g)
    bcast = 1 if g.shape == u.shape[1:] else 0
    if not bcast:
        assert g.shape == u.shape
    v = _rec_weights(v, C, np.float64)
    dI = np.empty(u.shape)
    dv_col = np.empty(C)
    lib().orc_scan_bwd_rleaky(T, C, v.size, beta, thr, slope, s_scale, int(bool(reset_surrogate)),
                              int(bool(smooth_z)), _p(v), _p(u), _p(g), bcast, _p(dI),
                              _p(dv_col))
    return dI, dv_col.reshape(-1, v.size).sum(axis=0)


def adamw(theta, g, m, v, t, lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=1e-2):
    """One AdamW step t >= 1 (Sec. IV: every network is trained with AdamW),
    in double.  Returns new (theta, m, v); the inputs are not modified."""
    th, m2, v2 = _f64(theta).copy(), _f64(m).copy(), _f64(v).copy()
    gg = _f64(g)
    assert th.shape == gg.shape == m2.shape == v2.shape and t >= 1
    lib().orc_adamw(th.size, _p(th), _p(gg), _p(m2), _p(v2), int(t), float(lr),
                    float(betas[0]), float(betas[1]), float(eps), float(weight_decay))
    return th, m2, v2


def population_counts(counts, P):
    """Population code (Sec. V): P output neurons per class, class k pooling
    the spike counts of neurons k*P .. k*P + P - 1 of each sample.
    counts [B, K*P] -> [B, K]."""
    c = _f64(counts)
    B = c.shape[0]
    return c.reshape(B, -1, P).sum(axis=2)


def loss_ce(counts, labels, P=1):
    """Spike-count cross-entropy, mean over the batch, on the class counts
    (pooled over populations of P neurons when P > 1).  Returns (L, dL/dc)
    with dL/dc per output neuron: every neuron of a population receives its
    class's gradient."""
    c = population_counts(counts, P) if P > 1 else _f64(counts)
    B, K = c.shape
    y = np.ascontiguousarray(labels, np.int32)
    g = np.empty((B, K))
    L = lib().orc_loss_ce(B, K, _p(c), _p(y), _p(g))
    return L, (np.repeat(g, P, axis=1) if P > 1 else g)


def loss_mse(counts, targets, P=1):
    """Spike-count mean-squared error, mean over all class entries (pooled
    over populations of P neurons when P > 1; targets [B, K])."""
    c = population_counts(counts, P) if P > 1 else _f64(counts)
    y = _f64(targets)
    assert c.shape == y.shape
    g = np.empty(c.shape)
    B = c.shape[0]
    K = int(np.prod(c.shape[1:]))
    L = lib().orc_loss_mse(B, K, _p(c), _p(y), _p(g))
    return L, (np.repeat(g, P, axis=1) if P > 1 else g)


# --------------------------------------------------------------------------
# Network driver: layers in order forward, loss, layers in reverse backward
# --------------------------------------------------------------------------
def _layer_out_shape(spec):
    if spec["kind"] == "dense":
        return (spec["n_out"],)
    if spec["kind"] == "conv":
        k = spec.get("k", 5)
        return (spec["c_out"], (spec["h"] - k + 1) // 2, (spec["w"] - k + 1) // 2)
    if spec["kind"] == "none":
        return (spec["n"],)
    raise ValueError(spec["kind"])


def layer_fwd(spec, x, W=None, b=None, smooth=False, slope=25.0, reset_surrogate=False,
              v=None):
    """One spiking layer forward.  ``spec`` is a plain dict:
    kind ('dense' | 'conv' | 'none'), sizes, neuron ('leaky'|'synaptic'|'rleaky'),
    beta, alpha, thr; v the recurrent weights of an 'rleaky' layer.  x is
    [T, B, ...] (spikes as 0/1 or currents).
    Method mode: currents are rounded to fp32 and the scan runs in fp32.
    Smooth mode: everything in double with the smooth spike."""
    T, B = x.shape[:2]
    out = {"x": x}
    if spec["kind"] == "dense":
        I = dense_fwd(np.reshape(x, (T * B, -1)), W, b).reshape(T, B, -1)
    elif spec["kind"] == "conv":
        y = conv_fwd(np.reshape(x, (T * B, spec["c_in"], spec["h"], spec["w"])), W, b)
        if not smooth:
            # the pool's selection is taken on the fp32 currents
            y = y.astype(np.float32).astype(np.float64)
        p, arg = maxpool2_fwd(y)
        out["conv_shape"] = y.shape
        out["arg"] = arg
        I = p.reshape((T, B) + p.shape[1:])
    elif spec["kind"] == "none":
        I = np.asarray(x)
    else:
        raise ValueError(spec["kind"])
    nt = spec["neuron"]
    if smooth:
        z, u, cnt = scan_fwd_smooth(I, nt, spec["beta"], spec["thr"], slope,
                                    spec.get("alpha", 0.0), reset_surrogate, v=v)
        out.update(I=I, z=z, u=u, counts=cnt)
    else:
        I32 = np.asarray(I, np.float32)
        z, u, cnt = scan_fwd(I32, nt, spec["beta"], spec["thr"], spec.get("alpha", 0.0), v=v)
        out.update(I=I32, z=z, u=u, counts=cnt)
    return out


def layer_bwd(spec, fwd, g, W=None, slope=25.0, reset_surrogate=False, s_scale=1.0,
              want_dx=True, v=None, smooth=False):
    """One spiking layer backward.  g = dL/dz of this layer's output spikes,
    [T, B, ...] or [B, ...] (broadcast over t).  Returns dict with dI and the
    parameter / input gradients (double); 'dv' for an 'rleaky' layer.  smooth:
    the forward was the smooth one, so z_{t-1} in dL/dv is the smooth spike."""
    u = fwd["u"]
    T, B = u.shape[:2]
    res = {}
    if spec["neuron"] == "rleaky":
        dI, dv = scan_bwd_rleaky(u, g, spec["beta"], spec["thr"], slope, v, reset_surrogate,
                                 s_scale, smooth_z=smooth)
        res["dv"] = dv
    else:
        dI = scan_bwd(u, g, spec["neuron"], spec["beta"], spec["thr"], slope,
                      spec.get("alpha", 0.0), reset_surrogate, s_scale)
    res["dI"] = dI
    x = fwd["x"]
    if spec["kind"] == "dense":
        dW, db, dx = dense_bwd(dI.reshape(T * B, -1), np.reshape(x, (T * B, -1)), W,
                               want_dx=want_dx)
        res.update(dW=dW, db=db, dx=None if dx is None else dx.reshape(np.shape(x)))
    elif spec["kind"] == "conv":
        Ho, Wo = fwd["conv_shape"][2:]
        dY = maxpool2_bwd(dI.reshape((T * B,) + dI.shape[2:]), fwd["arg"], Ho, Wo)
        xx = np.reshape(x, (T * B, spec["c_in"], spec["h"], spec["w"]))
        dW, db, dx = conv_bwd(dY, xx, W, want_dx=want_dx)
        res.update(dW=dW, db=db, dx=None if dx is None else dx.reshape(np.shape(x)))
    elif spec["kind"] == "none":
        res.update(dx=dI)
    return res


def net_step(layers, params, x, loss="ce", labels=None, targets=None, smooth=False,
             slope=25.0, reset_surrogate=False, pop=1):
    """One forward + BPTT step of a feed-forward spiking network.

    layers: list of layer spec dicts; params: list of (W, b) (None for 'none'),
    or (W, b, v) for an 'rleaky' layer; x: [T, B, ...] input.  The loss is
    taken on the last layer's spike counts summed over T (and pooled over
    populations of ``pop`` neurons per class, Sec. V).  Returns (loss, per-layer forward dicts, per-layer backward
    dicts)."""
    fwds = []
    h = x
    for spec, prm in zip(layers, params):
        W, b = prm[0], prm[1]
        v = prm[2] if len(prm) > 2 else None
        f = layer_fwd(spec, h, W, b, smooth=smooth, slope=slope,
                      reset_surrogate=reset_surrogate, v=v)
        fwds.append(f)
        h = f["z"]
    counts = fwds[-1]["counts"]
    B = counts.shape[0]
    if loss == "ce":
        L, gc = loss_ce(counts.reshape(B, -1), labels, pop)
    else:
        L, gc = loss_mse(counts.reshape(B, -1), targets, pop)
    g = gc.reshape(counts.shape)
    s_scale = slope / 2.0 if smooth else 1.0
    bwds = [None] * len(layers)
    for li in range(len(layers) - 1, -1, -1):
        spec = layers[li]
        W = params[li][0]
        v = params[li][2] if len(params[li]) > 2 else None
        r = layer_bwd(spec, fwds[li], g, W, slope, reset_surrogate, s_scale,
                      want_dx=(li > 0) or spec["kind"] == "none", v=v, smooth=smooth)
        bwds[li] = r
        g = r["dx"]
    return L, fwds, bwds

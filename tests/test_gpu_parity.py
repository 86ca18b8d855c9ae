"""GPU path vs CPU oracle, through the C ABI, on identical seeded inputs.

Stage tests feed the oracle the GPU's own inputs to that stage (teacher
forcing), so that a legal spike flip in one stage cannot cascade into the
next.  Scans given identical fp32 currents must be bit-identical.
"""
import numpy as np
import pytest

import oracle
import paper_2211_10725_amd as snn
from paper_2211_10725_amd import workloads as wls
from tests.parity import assert_close, assert_spikes, spike_flips

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"


def _t(a, dtype=None):
    t = torch.as_tensor(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(DEV)


def _np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def _none_desc(T, B, N, neuron="leaky", beta=0.9, alpha=0.0, thr=1.0, slope=25.0,
               reset=snn.RESET_DETACHED):
    spec = dict(kind="none", n=N, neuron=neuron, beta=beta, alpha=alpha, thr=thr)
    return snn.layer_desc(spec, T, B, slope=slope, reset_grad=reset), spec


def _assert_fp32_sum(a, terms_abs, K, what):
    """A priori bound of an fp32 sum of K products, any order:
    |fl(sum) - sum| <= (K + 1) u sum|terms|, u = 2^-24 (plus one rounding)."""
    bound = (K + 2) * 2.0 ** -24 * terms_abs
    err = np.abs(np.asarray(a, np.float64))
    assert (err <= bound).all(), f"{what}: error above the fp32 summation bound"


def _ws(nbytes):
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=DEV)


# ---------------------------------------------------------------------------
# neuron scans
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("neuron,alpha,beta", [("leaky", 0.0, 0.95), ("synaptic", 0.9, 0.8)])
@pytest.mark.parametrize("T,B,N", [(1, 2, 8), (7, 3, 101), (33, 4, 256), (50, 5, 1001),
                                   (6, 8, 65536), (3, 9, 65537)])
def test_scan_fwd_bit_exact(neuron, alpha, beta, T, B, N):
    rng = np.random.default_rng(T * 1000 + N)
    I = rng.normal(0.3, 0.8, (T, B, N)).astype(np.float32)
    d, spec = _none_desc(T, B, N, neuron, beta, alpha)
    x = _t(I)
    spk = torch.empty((T, B, N), dtype=torch.uint8, device=DEV)
    saved = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
    counts = torch.empty((B, N), dtype=torch.float32, device=DEV)
    snn.snn_neuron_fwd(d, x, spk, saved, counts)
    z, u, c = oracle.scan_fwd(I, neuron, beta, 1.0, alpha)
    np.testing.assert_array_equal(_np(spk), z)
    np.testing.assert_array_equal(_np(saved), u)
    np.testing.assert_array_equal(_np(counts), c)


def test_scan_fwd_in_place_and_f16_spikes():
    T, B, N = 20, 3, 64
    rng = np.random.default_rng(11)
    I = rng.normal(0.3, 0.8, (T, B, N)).astype(np.float32)
    d, _ = _none_desc(T, B, N, "synaptic", 0.8, 0.6)
    d.out_dtype = snn.F16
    buf = _t(I)
    spk = torch.empty((T, B, N), dtype=torch.float16, device=DEV)
    snn.snn_neuron_fwd(d, buf, spk, buf, None)        # currents overwritten by u
    z, u, _ = oracle.scan_fwd(I, "synaptic", 0.8, 1.0, 0.6)
    np.testing.assert_array_equal(_np(buf), u)
    np.testing.assert_array_equal(_np(spk).astype(np.uint8), z)


@pytest.mark.parametrize("neuron,alpha,beta", [("leaky", 0.0, 0.95), ("synaptic", 0.9, 0.8)])
@pytest.mark.parametrize("reset", [snn.RESET_DETACHED, snn.RESET_SURROGATE])
@pytest.mark.parametrize("bcast", [True, False])
@pytest.mark.parametrize("T,B,N", [(1, 2, 8), (9, 3, 37), (40, 4, 512), (5, 8, 65536)])
def test_scan_bwd(neuron, alpha, beta, reset, bcast, T, B, N):
    rng = np.random.default_rng(7 * T + N)
    I = rng.normal(0.3, 0.8, (T, B, N)).astype(np.float32)
    d, spec = _none_desc(T, B, N, neuron, beta, alpha, reset=reset)
    x = _t(I)
    spk = torch.empty((T, B, N), dtype=torch.uint8, device=DEV)
    saved = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
    snn.snn_neuron_fwd(d, x, spk, saved, None)
    g = rng.normal(0, 1, (B, N) if bcast else (T, B, N)).astype(np.float32)
    dI = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
    snn.snn_neuron_bwd(d, snn.GRAD_BCAST if bcast else snn.GRAD_FULL, _t(g), saved, dI, None, None)
    ref = oracle.scan_bwd(_np(saved), g, neuron, beta, 1.0, 25.0, alpha, reset == snn.RESET_SURROGATE)
    assert_close(_np(dI), ref, 1e-3, what="dL/dI")


@pytest.mark.parametrize("gdt,tdt", [(snn.F16, torch.float16), (snn.BF16, torch.bfloat16)])
def test_scan_bwd_half_gradient_operand(gdt, tdt):
    T, B, N = 30, 4, 96
    rng = np.random.default_rng(5)
    I = rng.normal(0.3, 0.8, (T, B, N)).astype(np.float32)
    spec = dict(kind="dense", n_in=8, n_out=N, neuron="leaky", beta=0.9)
    d = snn.layer_desc(spec, T, B, grad_dtype=gdt)
    dn, _ = _none_desc(T, B, N, "leaky", 0.9)
    saved = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
    spk = torch.empty((T, B, N), dtype=torch.uint8, device=DEV)
    snn.snn_neuron_fwd(dn, _t(I), spk, saved, None)
    g = rng.normal(0, 0.01, (B, N)).astype(np.float32)
    dI = torch.empty((T, B, N), dtype=tdt, device=DEV)
    snn.snn_neuron_bwd(d, snn.GRAD_BCAST, _t(g), saved, dI, None, None)
    ref = oracle.scan_bwd(_np(saved), g, "leaky", 0.9, 1.0, 25.0)
    assert_close(_np(dI.float()), ref, 2e-2, what="half dL/dI")


# ---------------------------------------------------------------------------
# synaptic contractions
# ---------------------------------------------------------------------------
GEMM_SHAPES = [(37, 29, 53), (800, 1000, 784), (128, 10, 1000), (300, 7, 33), (64, 130, 1),
               (5, 300, 17)]


PATHS = {"split": 0, "fp32mfma": snn.FLAG_FP32_MFMA}


# (1040, 1100, 1000): large enough for the 256 x 256 asynchronous kernel with
# fp16 weights, ragged in M and N, and a last k-tile of 8 values
@pytest.mark.parametrize("M,N,K", GEMM_SHAPES + [(12800, 1000, 784), (1040, 1100, 1000)])
@pytest.mark.parametrize("wdt", ["f32", "f16"])
@pytest.mark.parametrize("path", list(PATHS))
def test_synapse_fwd(M, N, K, wdt, path):
    rng = np.random.default_rng(M + N + K)
    x = (rng.random((M, K)) < 0.5).astype(np.uint8)
    W = rng.uniform(-1, 1, (N, K)).astype(np.float32)
    if wdt == "f16":
        W = W.astype(np.float16).astype(np.float32)
    b = rng.uniform(-1, 1, N).astype(np.float32)
    spec = dict(kind="dense", n_in=K, n_out=N, neuron="leaky", beta=0.9)
    d = snn.layer_desc(spec, 1, M, w_dtype=snn.F16 if wdt == "f16" else snn.F32,
                       flags=PATHS[path])
    cur = torch.empty((M, N), dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_layer_workspace_bytes(d))
    Wt = _t(W, torch.float16 if wdt == "f16" else torch.float32)
    snn.snn_synapse_fwd(d, _t(x), Wt, _t(b), cur, None, ws)
    ref = oracle.dense_fwd(x, W, b)
    got = _np(cur)
    assert_close(got, ref, 1e-3, what="currents")
    _assert_fp32_sum(got - ref, x.astype(np.float64) @ np.abs(W).T.astype(np.float64) + np.abs(b),
                     K, "currents")


# (12800, 10, 1000) and (5000, 7, 1003): layers with few outputs, large enough
# for the skinny kernels (short contraction for dx, few rows for dW); 1003
# inputs give unaligned rows and a partial last group of 4 columns
@pytest.mark.parametrize("M,N,K", GEMM_SHAPES + [(12800, 1000, 784), (12800, 10, 1000),
                                                 (5000, 7, 1003)])
@pytest.mark.parametrize("path", list(PATHS))
def test_synapse_bwd(M, N, K, path):
    """dW = dI^T x (split over K = T*B) and dx = dI W."""
    rng = np.random.default_rng(3 * M + N)
    x = (rng.random((M, K)) < 0.5).astype(np.uint8)
    W = rng.uniform(-1, 1, (N, K)).astype(np.float32)
    dI = rng.normal(0, 1, (M, N)).astype(np.float32)
    spec = dict(kind="dense", n_in=K, n_out=N, neuron="leaky", beta=0.9)
    d = snn.layer_desc(spec, 1, M, flags=PATHS[path])
    gW = torch.empty((N, K), dtype=torch.float32, device=DEV)
    gx = torch.empty((M, K), dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_layer_workspace_bytes(d))
    snn.snn_synapse_bwd(d, _t(dI), None, _t(x), _t(W), gW, gx, ws)
    rW, _, rx = oracle.dense_bwd(dI, x, W)
    gotW, gotx = _np(gW), _np(gx)
    assert_close(gotW, rW, 1e-3, what="dW")
    assert_close(gotx, rx, 1e-3, what="dx")
    aI = np.abs(dI).astype(np.float64)
    _assert_fp32_sum(gotW - rW, aI.T @ x.astype(np.float64), M, "dW")
    _assert_fp32_sum(gotx - rx, aI @ np.abs(W).astype(np.float64), N, "dx")


GRAD_TYPES = {"f32": (snn.F32, torch.float32), "bf16": (snn.BF16, torch.bfloat16),
              "f16": (snn.F16, torch.float16)}


@pytest.mark.parametrize("M,N,K", [(300, 130, 77), (12800, 1000, 784), (2048, 512, 1024),
                                   (1040, 1100, 1000), (12800, 10, 1000), (5000, 7, 1003)])
@pytest.mark.parametrize("gdt", list(GRAD_TYPES))
@pytest.mark.parametrize("wdt", ["f32", "f16"])
def test_synapse_bwd_operand_types(M, N, K, gdt, wdt):
    """dW and dx with 16-bit gradient operands and/or fp16 weights: products
    of the given (rounded) values are exact, so the result is their fp32 sum."""
    rng = np.random.default_rng(M + 7 * N)
    x = (rng.random((M, K)) < 0.5).astype(np.uint8)
    W = rng.uniform(-1, 1, (N, K)).astype(np.float32)
    if wdt == "f16":
        W = W.astype(np.float16).astype(np.float32)
    dI = rng.normal(0, 1e-3, (M, N)).astype(np.float32)
    gcode, tdt = GRAD_TYPES[gdt]
    dI_t = _t(dI, tdt)
    dI_used = _np(dI_t.float()).astype(np.float64)      # the values the GPU sees
    spec = dict(kind="dense", n_in=K, n_out=N, neuron="leaky", beta=0.9)
    d = snn.layer_desc(spec, 1, M, grad_dtype=gcode, w_dtype=snn.F16 if wdt == "f16" else snn.F32)
    gW = torch.empty((N, K), dtype=torch.float32, device=DEV)
    gx = torch.empty((M, K), dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_layer_workspace_bytes(d))
    Wt = _t(W, torch.float16 if wdt == "f16" else torch.float32)
    snn.snn_synapse_bwd(d, dI_t, None, _t(x), Wt, gW, gx, ws)
    rW, _, rx = oracle.dense_bwd(dI_used, x, W)
    gotW, gotx = _np(gW), _np(gx)
    assert_close(gotW, rW, 1e-3, what="dW")
    assert_close(gotx, rx, 1e-3, what="dx")
    aI = np.abs(dI_used)
    _assert_fp32_sum(gotW - rW, aI.T @ x.astype(np.float64), M, "dW")
    _assert_fp32_sum(gotx - rx, aI @ np.abs(W).astype(np.float64), N, "dx")


# ---------------------------------------------------------------------------
# convolutional synapse: 5x5 valid conv + 2x2 max-pool of the currents
# ---------------------------------------------------------------------------
def _conv_case(NB, Ci, H, W, Co, seed, dens=0.5):
    rng = np.random.default_rng(seed)
    x = (rng.random((NB, Ci, H, W)) < dens).astype(np.uint8)
    w = rng.uniform(-0.3, 0.3, (Co, Ci, 5, 5)).astype(np.float32)
    b = rng.uniform(-0.2, 0.2, Co).astype(np.float32)
    spec = dict(kind="conv", c_in=Ci, h=H, w=W, c_out=Co, neuron="leaky", beta=0.5)
    d = snn.layer_desc(spec, 1, NB)
    return x, w, b, d


def _conv_fwd_gpu(d, x, w, b):
    cur = torch.empty((d.B, d.n_out), dtype=torch.float32, device=DEV)
    arg = torch.empty(d.B * d.n_out, dtype=torch.uint8, device=DEV)
    snn.snn_synapse_fwd(d, _t(x), _t(w), _t(b), cur, arg, _ws(snn.snn_layer_workspace_bytes(d)))
    return _np(cur), _np(arg)


@pytest.mark.parametrize("NB,Ci,H,W,Co", [(3, 1, 28, 28, 12), (5, 12, 12, 12, 64), (2, 3, 9, 11, 5),
                                          (1, 2, 6, 6, 2)])
def test_conv_pool_fwd(NB, Ci, H, W, Co):
    x, w, b, d = _conv_case(NB, Ci, H, W, Co, seed=NB * 100 + Co)
    cur, arg = _conv_fwd_gpu(d, x, w, b)
    y = oracle.conv_fwd(x, w, b)                          # double
    y32 = y.astype(np.float32).astype(np.float64)          # the pool decides on fp32 currents
    p, a = oracle.maxpool2_fwd(y32)
    cur = cur.reshape(p.shape)
    arg = arg.reshape(a.shape)
    assert_close(cur, p, 1e-3, what="pooled currents")
    # fp32 accumulation of Ci*25 terms, any order
    terms = oracle.conv_fwd(x, np.abs(w), np.abs(b))
    bound = (Ci * 25 + 2) * 2.0 ** -24 * oracle.maxpool2_fwd(terms)[0]
    assert (np.abs(cur - p) <= bound + 1e-30).all()
    # the selection must agree wherever the window's top two differ by more
    # than the fp32 error; elsewhere the chosen element must be a maximum
    Hp, Wp = a.shape[2], a.shape[3]
    win = y32[:, :, :2 * Hp, :2 * Wp].reshape(NB, Co, Hp, 2, Wp, 2)
    win = win.transpose(0, 1, 2, 4, 3, 5).reshape(a.shape + (4,))
    srt = np.sort(win, axis=-1)
    clear = (srt[..., -1] - srt[..., -2]) > 2 * bound.reshape(a.shape) + 1e-6
    assert (arg[clear] == a[clear]).all()
    chosen = np.take_along_axis(win, arg[..., None].astype(np.int64), -1)[..., 0]
    assert (np.abs(chosen - srt[..., -1]) <= 2 * bound.reshape(a.shape) + 1e-6).all()


def test_conv_pool_ties_first_maximum():
    """All-zero receptive fields give conv output = bias exactly in every
    window position: the first element must be chosen."""
    x = np.zeros((2, 1, 8, 8), np.uint8)
    x[1, 0, 3, 3] = 1
    w = np.full((3, 1, 5, 5), 0.25, np.float32)
    b = np.array([0.5, -0.5, 0.0], np.float32)
    spec = dict(kind="conv", c_in=1, h=8, w=8, c_out=3, neuron="leaky", beta=0.5)
    d = snn.layer_desc(spec, 1, 2)
    cur, arg = _conv_fwd_gpu(d, x, w, b)
    p, a = oracle.maxpool2_fwd(oracle.conv_fwd(x, w, b).astype(np.float32).astype(np.float64))
    np.testing.assert_array_equal(cur.reshape(p.shape), p)
    np.testing.assert_array_equal(arg.reshape(a.shape), a)
    assert (a[0] == 0).all()


@pytest.mark.parametrize("NB,Ci,H,W,Co", [(3, 1, 28, 28, 12), (4, 12, 12, 12, 64), (2, 3, 9, 11, 5)])
def test_conv_pool_bwd(NB, Ci, H, W, Co):
    """Backward teacher-forced on the GPU's own pool selection."""
    x, w, b, d = _conv_case(NB, Ci, H, W, Co, seed=7 * NB + Co)
    cur, arg = _conv_fwd_gpu(d, x, w, b)
    rng = np.random.default_rng(1)
    dI = rng.normal(0, 1, cur.shape).astype(np.float32)
    gW = torch.empty(w.shape, dtype=torch.float32, device=DEV)
    gx = torch.empty(x.shape, dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_layer_workspace_bytes(d))
    arg_t = _t(arg)
    snn.snn_synapse_bwd(d, _t(dI), arg_t, _t(x), _t(w), gW, gx, ws)
    Ho, Wo = H - 4, W - 4
    dY = oracle.maxpool2_bwd(dI.reshape(NB, Co, Ho // 2, Wo // 2), arg.reshape(NB, Co, Ho // 2, Wo // 2),
                             Ho, Wo)
    if Ho % 2 or Wo % 2:
        pass  # the dropped row/column of the conv output gets no gradient (zeros from the pool)
    rW, _, rx = oracle.conv_bwd(dY, x, w)
    assert_close(_np(gW), rW, 1e-3, what="conv dW")
    assert_close(_np(gx), rx, 1e-3, what="conv dx")


# ---------------------------------------------------------------------------
# losses
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("B,K", [(1, 10), (32, 10), (513, 10), (7, 3)])
def test_loss_ce(B, K):
    rng = np.random.default_rng(B)
    c = rng.integers(0, 26, (B, K)).astype(np.float32)
    y = rng.integers(0, K, B).astype(np.int32)
    loss = torch.empty(4, dtype=torch.float32, device=DEV)
    g = torch.empty((B, K), dtype=torch.float32, device=DEV)
    snn.snn_loss(snn.LOSS_CE_COUNT, B, K, _t(c), _t(y), None, loss, g, None)
    L, rg = oracle.loss_ce(c, y)
    assert abs(_np(loss)[0] - L) <= 1e-6 * max(1.0, abs(L))
    assert_close(_np(g), rg, 1e-5, what="CE grad")


@pytest.mark.parametrize("B,K", [(1, 1), (64, 1000), (64, 65536), (3, 7)])
def test_loss_mse(B, K):
    rng = np.random.default_rng(K)
    c = rng.integers(0, 200, (B, K)).astype(np.float32)
    y = rng.uniform(0, 50, (B, K)).astype(np.float32)
    loss = torch.empty(4, dtype=torch.float32, device=DEV)
    g = torch.empty((B, K), dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_loss_workspace_bytes(snn.LOSS_MSE_COUNT, B, K))
    snn.snn_loss(snn.LOSS_MSE_COUNT, B, K, _t(c), None, _t(y), loss, g, ws)
    L, rg = oracle.loss_mse(c, y)
    assert abs(_np(loss)[0] - L) <= 1e-6 * abs(L)
    assert_close(_np(g), rg, 1e-6, what="MSE grad")


# ---------------------------------------------------------------------------
# whole training steps
# ---------------------------------------------------------------------------
def _saved_u(net, li):
    d = net.descs[li]
    n = d.T * d.B * d.n_out
    return _np(net.saved[li][: n * 4].view(torch.float32)).reshape(d.T, d.B, d.n_out)


def spec_n_out(spec):
    if spec["kind"] == "conv":
        return spec["c_out"] * ((spec["h"] - 4) // 2) * ((spec["w"] - 4) // 2)
    return spec["n_out"] if spec["kind"] == "dense" else spec["n"]


def _gpu_currents(net, li, xin):
    """Currents of layer li recomputed by the stage call on the GPU's input
    (conv layers: into a scratch selection buffer, the saved one untouched)."""
    d = net.descs[li]
    cur = torch.empty((d.T, d.B, d.n_out), dtype=torch.float32, device=DEV)
    arg = torch.empty(d.T * d.B * d.n_out, dtype=torch.uint8, device=DEV) \
        if d.synapse == snn.SYN_CONV5_POOL2 else None
    snn.snn_synapse_fwd(d, xin, net.W[li], net.b[li], cur, arg, net.ws)
    return _np(cur)


def _check_step_teacher_forced(wl, inp, net, x_dev, tol=1e-3):
    """Every stage of the GPU step against the oracle fed the GPU's inputs:
    contraction vs oracle contraction on the same spikes; oracle scan on the
    GPU's own currents must reproduce spikes, membrane and counts exactly."""
    T, B = wl.T, wl.B
    n = len(wl.layers)
    h = inp["x"]
    xs = []
    for li, spec in enumerate(wl.layers):
        W, b = inp["params"][li]
        xs.append(h)
        z_gpu = _np(net.spk[li])
        u_gpu = _saved_u(net, li)
        if spec["kind"] == "dense":
            xin = np.asarray(h, np.float64).reshape(T * B, -1)
            I_orc = oracle.dense_fwd(xin, W, b).reshape(T, B, -1)
            I = _gpu_currents(net, li, x_dev if li == 0 else net.spk[li - 1])
            assert_close(I, I_orc, tol, what=f"L{li} currents")
        elif spec["kind"] == "conv":
            xin = np.asarray(h, np.float64).reshape(T * B, spec["c_in"], spec["h"], spec["w"])
            y32 = oracle.conv_fwd(xin, W, b).astype(np.float32).astype(np.float64)
            I_orc = oracle.maxpool2_fwd(y32)[0].reshape(T, B, -1)
            I = _gpu_currents(net, li, x_dev if li == 0 else net.spk[li - 1])
            assert_close(I, I_orc, tol, what=f"L{li} conv currents")
        else:
            I = np.asarray(h, np.float32)
        z, u, c = oracle.scan_fwd(I, spec["neuron"], spec["beta"], spec["thr"],
                                  spec.get("alpha", 0.0))
        np.testing.assert_array_equal(z_gpu, z, err_msg=f"L{li} spikes")
        np.testing.assert_array_equal(u_gpu, u, err_msg=f"L{li} membrane")
        if li == n - 1:
            np.testing.assert_array_equal(_np(net.counts).reshape(c.shape), c)
        h = z_gpu  # teacher-force the next layer on the GPU's spikes
    L, gc = (oracle.loss_ce(_np(net.counts), inp["labels"]) if wl.loss == "ce"
             else oracle.loss_mse(_np(net.counts), inp["targets"]))
    assert abs(_np(net.loss)[0] - L) <= 1e-5 * max(1.0, abs(L))
    assert_close(_np(net.gcounts), gc, 1e-5, what="dL/dcounts")
    g = _np(net.gcounts)
    for li in range(n - 1, -1, -1):
        spec = wl.layers[li]
        W = inp["params"][li][0]
        u_gpu = _saved_u(net, li)
        dI = oracle.scan_bwd(u_gpu, g, spec["neuron"], spec["beta"], spec["thr"], wl.slope,
                             spec.get("alpha", 0.0))
        if spec["kind"] == "none":
            assert_close(_np(net.gx[li]), dI, tol, what="dL/dI")
            break
        if spec["kind"] == "conv":
            Ho, Wo = spec["h"] - 4, spec["w"] - 4
            pa = net.pool_arg(li)[: T * B * spec_n_out(spec)]
            arg = _np(pa).reshape(T * B, spec["c_out"], Ho // 2, Wo // 2)
            dY = oracle.maxpool2_bwd(dI.reshape(arg.shape), arg, Ho, Wo)
            xin = np.asarray(xs[li], np.float64).reshape(T * B, spec["c_in"], spec["h"], spec["w"])
            dW, db, dx = oracle.conv_bwd(dY, xin, W, want_dx=li > 0)
            assert_close(_np(net.gW[li]), dW, tol, what=f"L{li} conv dW")
            assert_close(_np(net.gb[li]), db, tol, what=f"L{li} conv db")
            if li > 0:
                gx = _np(net.gx[li])
                assert_close(gx.reshape(dx.shape), dx, tol, what=f"L{li} conv dx")
                g = gx
            continue
        xin = np.asarray(xs[li], np.float64).reshape(T * B, -1)
        dW, db, dx = oracle.dense_bwd(dI.reshape(T * B, -1), xin, W, want_dx=li > 0)
        bW = bx = None
        if net.descs[li].grad_dtype == snn.BF16:
            # dL/dI handed to the contractions in bf16: a-priori rounding bound
            aI = np.abs(dI.reshape(T * B, -1))
            bW = 2.0 ** -8 * (aI.T @ np.abs(xin))
            bx = 2.0 ** -8 * (aI @ np.abs(W).astype(np.float64)) if li > 0 else None
        assert_close(_np(net.gW[li]), dW, tol, what=f"L{li} dW", abs_bound=bW)
        assert_close(_np(net.gb[li]), db, tol, what=f"L{li} db")
        if li > 0:
            gx = _np(net.gx[li])
            assert_close(gx.reshape(T * B, -1), dx, tol, what=f"L{li} dx", abs_bound=bx)
            g = gx  # teacher-force the layer below on the GPU's gradient


@pytest.mark.parametrize("name", ["dsnn_leaky_t25_b32", "dsnn_synaptic_t50_b256", "csnn_t25_b128"])
@pytest.mark.parametrize("path", list(PATHS))
def test_step_full_size_teacher_forced(name, path):
    wl = wls.get(name)
    inp = wls.make_inputs(wl, seed=0)
    net = snn.Network(wl, inp["params"], device=DEV, flags=PATHS[path])
    x = _t(inp["x"])
    net.step(x, labels=_t(inp["labels"]))
    _check_step_teacher_forced(wl, inp, net, x)


@pytest.mark.parametrize("name,T,B,width", [("dsnn_synaptic_t50_b256", 20, 16, 200),
                                            ("dsnn_leaky_t25_b32", 25, 8, 300),
                                            ("scan_wide_t1000_b64", 60, 4, 1000),
                                            ("csnn_t25_b128", 6, 4, None),
                                            ("dsnn_half_t100_b512", 12, 8, 320)])
@pytest.mark.parametrize("reset", [snn.RESET_DETACHED, snn.RESET_SURROGATE])
@pytest.mark.parametrize("path", list(PATHS))
def test_step_scaled_teacher_forced(name, T, B, width, reset, path):
    wl = wls.scaled(wls.get(name), T=T, B=B, width=width)
    inp = wls.make_inputs(wl, seed=1)
    net = snn.Network(wl, inp["params"], device=DEV, reset_grad=reset, flags=PATHS[path])
    lab = _t(inp["labels"]) if wl.loss == "ce" else None
    tgt = _t(inp["targets"]) if wl.loss == "mse" else None
    x = _t(inp["x"])
    net.step(x, labels=lab, targets=tgt)
    if reset == snn.RESET_DETACHED:
        _check_step_teacher_forced(wl, inp, net, x, tol=2e-2 if wl.dtype == "f16" else 1e-3)
    # the stage calls give the same bytes as the layer calls
    snap = [_np(t).copy() for t in net.gW if t is not None] + [_np(net.loss).copy()]
    net.step_stages(x, labels=lab, targets=tgt)
    snap2 = [_np(t) for t in net.gW if t is not None] + [_np(net.loss)]
    for a, b in zip(snap, snap2):
        np.testing.assert_array_equal(a, b)


def test_step_end_to_end_unforced():
    """The whole step, oracle run on its own; flips are counted, gradient
    columns downstream of a flip are excluded."""
    wl = wls.get("dsnn_leaky_t25_b32")
    inp = wls.make_inputs(wl, seed=2)
    net = snn.Network(wl, inp["params"], device=DEV)
    net.step(_t(inp["x"]), labels=_t(inp["labels"]))
    L, fwds, bwds = oracle.net_step(wl.layers, inp["params"], inp["x"].astype(np.float64), "ce",
                                    labels=inp["labels"], slope=wl.slope)
    roots = 0
    for li, f in enumerate(fwds):
        agree, r, illegal = spike_flips(_np(net.spk[li]), f["z"], f["u"], 1.0)
        assert illegal == 0 and agree >= 0.9999
        roots += r
    if roots == 0:
        assert abs(_np(net.loss)[0] - L) <= 1e-5 * abs(L)
        for li in range(len(wl.layers)):
            assert_close(_np(net.gW[li]), bwds[li]["dW"], 1e-3, what=f"L{li} dW")
            assert_close(_np(net.gb[li]), bwds[li]["db"], 1e-3, what=f"L{li} db")


def test_deterministic():
    wl = wls.get("dsnn_synaptic_t50_b256")
    wl = wls.scaled(wl, T=10, B=32)
    inp = wls.make_inputs(wl, seed=3)
    net = snn.Network(wl, inp["params"], device=DEV)
    x, y = _t(inp["x"]), _t(inp["labels"])
    net.step(x, labels=y)
    a = [_np(t).copy() for t in net.gW + net.gb] + [_np(net.loss).copy()]
    net.step(x, labels=y)
    b = [_np(t) for t in net.gW + net.gb] + [_np(net.loss)]
    for p, q in zip(a, b):
        np.testing.assert_array_equal(p, q)


def test_empty_time_and_batch():
    for T, B in [(0, 4), (4, 0)]:
        spec = dict(kind="dense", n_in=16, n_out=8, neuron="leaky", beta=0.9)
        d = snn.layer_desc(spec, T, B)
        x = torch.empty((max(T * B, 1), 16), dtype=torch.uint8, device=DEV)
        W = torch.ones((8, 16), dtype=torch.float32, device=DEV)
        spk = torch.empty(256, dtype=torch.uint8, device=DEV)
        saved = torch.empty(256, dtype=torch.uint8, device=DEV)
        counts = torch.full((max(B, 1), 8), 7.0, device=DEV)
        snn.snn_layer_fwd(d, x, W, None, spk, saved, counts, _ws(256))
        if B > 0:
            assert (_np(counts) == 0).all()
        gW = torch.full((8, 16), 3.0, device=DEV)
        gb = torch.full((8,), 3.0, device=DEV)
        g = torch.zeros(256, dtype=torch.float32, device=DEV)
        snn.snn_layer_bwd(d, snn.GRAD_BCAST, g, x, W, saved, gW, gb, None,
                          _ws(snn.snn_layer_workspace_bytes(d)))
        assert (_np(gW) == 0).all() and (_np(gb) == 0).all()

"""Parity at the full benchmark sizes, on sampled outputs.

The wide scan (65536 neurons x 64 samples x 1000 steps) and the deep
half-precision net (784-4096-4096-10, T=100, B=512) are run through the same
layer calls the benchmark times; the oracle then recomputes sampled columns
and rows one by one, fed the GPU's own inputs to each stage.
"""
import numpy as np
import pytest

import oracle
import paper_2211_10725_amd as snn
from paper_2211_10725_amd import workloads as wls
from tests.parity import assert_close

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda"


def _np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def _u(net, li):
    d = net.descs[li]
    return net.saved[li][: d.T * d.B * d.n_out * 4].view(torch.float32).view(d.T, d.B, d.n_out)


def test_scan_wide_full_size_sampled():
    wl = wls.get("scan_wide_t1000_b64")
    T, B, N = wl.T, wl.B, wl.layers[0]["n"]
    spec = wl.layers[0]
    net = snn.Network(wl, wls.init_params(wl, 0), device=DEV)
    x = wls.device_currents(wl, 0)
    tgt_h = wls.targets(wl, 0)
    net.step(x, targets=torch.as_tensor(tgt_h).to(DEV))
    # loss and dL/dcounts over all 64 x 65536 counts
    counts = _np(net.counts)
    L, gc = oracle.loss_mse(counts, tgt_h)
    assert abs(_np(net.loss)[0] - L) <= 1e-6 * abs(L)
    assert_close(_np(net.gcounts), gc, 1e-5, what="dL/dcounts")
    rng = np.random.default_rng(0)
    cols = [(0, 0), (B - 1, N - 1), (B - 1, 0), (0, N - 1)] + \
        [(int(b), int(n)) for b, n in zip(rng.integers(0, B, 252), rng.integers(0, N, 252))]
    bi = torch.tensor([c[0] for c in cols], device=DEV)
    ni = torch.tensor([c[1] for c in cols], device=DEV)
    I = _np(x[:, bi, ni])                       # [T, S] currents of the sampled columns
    z_g = _np(net.spk[0][:, bi, ni])
    u_g = _np(_u(net, 0)[:, bi, ni])
    z, u, c = oracle.scan_fwd(I, spec["neuron"], spec["beta"], spec["thr"])
    np.testing.assert_array_equal(z_g, z)
    np.testing.assert_array_equal(u_g, u)
    np.testing.assert_array_equal(counts[bi.cpu().numpy(), ni.cpu().numpy()], c)
    g = gc[bi.cpu().numpy(), ni.cpu().numpy()]
    dI = oracle.scan_bwd(u_g, g, spec["neuron"], spec["beta"], spec["thr"], wl.slope)
    assert_close(_np(net.gx[0][:, bi, ni]), dI, 1e-3, what="dL/dI")


def test_half_net_full_size_sampled():
    wl = wls.get("dsnn_half_t100_b512")
    T, B = wl.T, wl.B
    inp = wls.make_inputs(wl, 0)
    net = snn.Network(wl, inp["params"], device=DEV)
    x = torch.as_tensor(inp["x"]).to(DEV)
    net.step(x, labels=torch.as_tensor(inp["labels"]).to(DEV))
    rng = np.random.default_rng(1)
    tol = 2e-2
    xs_dev = [x] + net.spk[:-1]
    # ---- forward, layer by layer, teacher-forced on the GPU's spikes
    for li, spec in enumerate(wl.layers):
        W, b = inp["params"][li]
        d = net.descs[li]
        cur = torch.empty((T, B, d.n_out), dtype=torch.float32, device=DEV)
        snn.snn_synapse_fwd(d, xs_dev[li], net.W[li], net.b[li], cur, None, net.ws)
        xin = _np(xs_dev[li]).reshape(T * B, -1)
        rows = rng.integers(0, T * B, 64)
        I_rows = oracle.dense_fwd(xin[rows].astype(np.float64), W, b)
        assert_close(_np(cur).reshape(T * B, -1)[rows], I_rows, 1e-3, what=f"L{li} currents")
        bs = rng.integers(0, B, 2)
        ns = rng.integers(0, d.n_out, 128) if d.n_out > 128 else np.arange(d.n_out)
        Ic = _np(cur[:, bs][:, :, ns])            # [T, 2, S]
        z, u, c = oracle.scan_fwd(Ic, spec["neuron"], spec["beta"], spec["thr"])
        np.testing.assert_array_equal(_np(net.spk[li][:, bs][:, :, ns]), z)
        np.testing.assert_array_equal(_np(_u(net, li)[:, bs][:, :, ns]), u)
        del cur
    counts = _np(net.counts)
    L, gc = oracle.loss_ce(counts, inp["labels"])
    assert abs(_np(net.loss)[0] - L) <= 1e-5 * max(1.0, abs(L))
    # ---- backward, teacher-forced on the GPU's membrane and upstream gradient
    g_full = _np(net.gcounts)                      # [B, 10], the same for every t
    for li in range(len(wl.layers) - 1, -1, -1):
        spec = wl.layers[li]
        W = inp["params"][li][0]
        d = net.descs[li]
        u_dev = _u(net, li)
        xin = _np(xs_dev[li]).reshape(T, B, -1)
        gx_dev = net.gx[li] if li > 0 else None
        if li == len(wl.layers) - 1:
            cols_o = np.arange(d.n_out)
        else:
            cols_o = rng.integers(0, d.n_out, 8)
        # dW rows and db entries for sampled output neurons o (all t, b)
        u_o = _np(u_dev[:, :, cols_o])
        g_o = g_full[:, cols_o] if g_full.ndim == 2 else g_full[:, :, cols_o]
        dI_o = oracle.scan_bwd(u_o, g_o, spec["neuron"], spec["beta"], spec["thr"], wl.slope)
        dW_o = dI_o.reshape(T * B, -1).T @ xin.reshape(T * B, -1).astype(np.float64)
        aI = np.abs(dI_o.reshape(T * B, -1))
        bW = 2.0 ** -8 * (aI.T @ np.abs(xin.reshape(T * B, -1)).astype(np.float64))
        assert_close(_np(net.gW[li])[cols_o], dW_o, tol, what=f"L{li} dW rows", abs_bound=bW)
        assert_close(_np(net.gb[li])[cols_o], dI_o.sum(axis=(0, 1)), tol, what=f"L{li} db")
        if gx_dev is None:
            break
        # dx for two sampled samples b: needs dL/dI of every output neuron of b
        bs = rng.integers(0, B, 2)
        u_b = _np(u_dev[:, bs])
        g_b = g_full[bs] if g_full.ndim == 2 else g_full[:, bs]
        dI_b = oracle.scan_bwd(u_b, g_b, spec["neuron"], spec["beta"], spec["thr"], wl.slope)
        dx_b = dI_b.reshape(-1, d.n_out) @ W.astype(np.float64)
        bx = 2.0 ** -8 * (np.abs(dI_b.reshape(-1, d.n_out)) @ np.abs(W).astype(np.float64))
        got = _np(gx_dev[:, bs]).reshape(-1, d.n_in)
        assert_close(got, dx_b, tol, what=f"L{li} dx", abs_bound=bx)
        g_full = _np(gx_dev)                        # teacher-force the layer below

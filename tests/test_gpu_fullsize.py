"""Parity at the full benchmark sizes, on sampled outputs.

The wide scan (65536 neurons x 64 samples x 1000 steps) and the deep
half-precision net (784-4096-4096-10, T=100, B=512) run through the same
calls, descriptors and shapes the benchmark times.  Every stage is fed seeded
synthetic inputs of its full-size shape; the oracle recomputes sampled
columns and rows from the same seeded inputs (it never reads a value the GPU
computed).  The whole step is then checked for agreement with the stage calls
on the GPU itself.
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


def _gen(seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return g


def _seeded_normal(shape, mean, std, seed, dtype=torch.float32):
    x = torch.empty(shape, dtype=torch.float32, device=DEV)
    x.normal_(mean, std, generator=_gen(seed))
    return x.to(dtype)


def _seeded_spikes(shape, p, seed):
    return (torch.rand(shape, generator=_gen(seed), device=DEV) < p).to(torch.uint8)


def test_scan_wide_full_size_sampled():
    wl = wls.get("scan_wide_t1000_b64")
    T, B, N = wl.T, wl.B, wl.layers[0]["n"]
    spec = wl.layers[0]
    net = snn.Network(wl, wls.init_params(wl, 0), device=DEV)
    d = net.descs[0]
    x = wls.device_currents(wl, 0)                 # seeded currents [T, B, N]
    spk = torch.empty((T, B, N), dtype=torch.uint8, device=DEV)
    u = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
    counts = torch.empty((B, N), dtype=torch.float32, device=DEV)
    ck = snn.ckpt_buffer(d)
    snn.snn_neuron_fwd(d, x, None, spk, ck, counts, u_out=u)
    rng = np.random.default_rng(0)
    cols = [(0, 0), (B - 1, N - 1), (B - 1, 0), (0, N - 1)] + \
        [(int(b), int(n)) for b, n in zip(rng.integers(0, B, 252), rng.integers(0, N, 252))]
    bi = torch.tensor([c[0] for c in cols], device=DEV)
    ni = torch.tensor([c[1] for c in cols], device=DEV)
    bh, nh = bi.cpu().numpy(), ni.cpu().numpy()
    I = _np(x[:, bi, ni])                       # seeded currents of the sampled columns
    z_o, u_o, c_o = oracle.scan_fwd(I, spec["neuron"], spec["beta"], spec["thr"])
    np.testing.assert_array_equal(_np(spk[:, bi, ni]), z_o)
    np.testing.assert_array_equal(_np(u[:, bi, ni]), u_o)
    np.testing.assert_array_equal(_np(counts)[bh, nh], c_o)
    # loss over all 64 x 65536 counts, on seeded spike counts and targets
    c_s = rng.integers(0, 120, (B, N)).astype(np.float32)
    tgt_h = wls.targets(wl, 0)
    loss = torch.empty(4, dtype=torch.float32, device=DEV)
    gc = torch.empty((B, N), dtype=torch.float32, device=DEV)
    snn.snn_loss(snn.LOSS_MSE_COUNT, B, N, 1, torch.as_tensor(c_s).to(DEV),
                 None, torch.as_tensor(tgt_h).to(DEV), loss, gc, net.ws)
    L, gc_o = oracle.loss_mse(c_s, tgt_h)
    assert abs(_np(loss)[0] - L) <= 1e-6 * abs(L)
    assert_close(_np(gc), gc_o, 1e-5, what="dL/dcounts")
    # reverse scan with a seeded gradient broadcast over t, recomputing the
    # membrane from the currents and the forward's checkpoints
    g = _seeded_normal((B, N), 0.0, 1e-6, seed=5)
    dI = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
    del u
    snn.snn_neuron_bwd(d, snn.GRAD_BCAST, g, None, x, ck, dI, None, None, None)
    dI_o = oracle.scan_bwd(u_o, _np(g)[bh, nh], spec["neuron"], spec["beta"], spec["thr"],
                           wl.slope)
    assert_close(_np(dI[:, bi, ni]), dI_o, 1e-3, what="dL/dI")
    del dI
    # the whole step is the same calls: same spikes, counts and checkpoints
    net.step(x, targets=torch.as_tensor(tgt_h).to(DEV))
    assert torch.equal(net.spk[0], spk) and torch.equal(net.parts[0][1][: ck.numel()], ck)
    assert torch.equal(net.counts, counts)


def test_half_net_full_size_sampled():
    wl = wls.get("dsnn_half_t100_b512")
    T, B = wl.T, wl.B
    inp = wls.make_inputs(wl, 0)
    net = snn.Network(wl, inp["params"], device=DEV)
    rng = np.random.default_rng(1)
    tol = 2e-2
    n = len(wl.layers)
    for li, spec in enumerate(wl.layers):
        W, b = inp["params"][li]
        d = net.descs[li]
        # ---- synapse forward on seeded spikes (the input's rates for layer 0)
        xin_dev = torch.as_tensor(inp["x"]).to(DEV) if li == 0 else \
            _seeded_spikes((T, B, d.n_in), 0.15, seed=100 + li)
        if d.in_dtype == snn.F16:
            xin_dev = xin_dev.to(torch.float16)  # spikes as the layer reads them
        cur = torch.empty((T, B, d.n_out), dtype=torch.float32, device=DEV)
        snn.snn_synapse_fwd(d, xin_dev, net.W[li], net.b[li], cur, None, net.ws)
        rows = rng.integers(0, T * B, 64)
        rows_t = torch.as_tensor(rows, device=DEV)
        xr = _np(xin_dev.reshape(T * B, -1)[rows_t]).astype(np.float64)
        I_rows = oracle.dense_fwd(xr, W, b)
        assert_close(_np(cur.reshape(T * B, -1)[rows_t]), I_rows, 1e-3, what=f"L{li} currents")
        del cur
        # ---- neuron scan on seeded currents
        Is = _seeded_normal((T, B, d.n_out), 0.1, 0.6, seed=200 + li)
        spk = torch.empty((T, B, d.n_out), device=DEV,
                          dtype=torch.float16 if d.out_dtype == snn.F16 else torch.uint8)
        u = torch.empty((T, B, d.n_out), dtype=torch.float32, device=DEV)
        ck = snn.ckpt_buffer(d)
        snn.snn_neuron_fwd(d, Is, None, spk, ck, None, u_out=u)
        bs = torch.as_tensor(rng.integers(0, B, 2), device=DEV)
        ns = torch.as_tensor(rng.integers(0, d.n_out, 128) if d.n_out > 128
                             else np.arange(d.n_out), device=DEV)
        I_c = _np(Is[:, bs][:, :, ns])                          # [T, 2, S]
        z_o, u_o, _ = oracle.scan_fwd(I_c, spec["neuron"], spec["beta"], spec["thr"])
        np.testing.assert_array_equal(_np(spk[:, bs][:, :, ns]), z_o)
        np.testing.assert_array_equal(_np(u[:, bs][:, :, ns]), u_o)
        # ---- reverse scan with a seeded upstream gradient (bf16 dL/dI out)
        last = li == n - 1
        g = _seeded_normal((B, d.n_out) if last else (T, B, d.n_out), 0.0, 1e-4, seed=300 + li)
        # (the layer's 16-bit dL/dI operand: bf16, or fp16 scaled by a power of two)
        scaled = d.grad_dtype == snn.F16
        gdt = torch.float16 if scaled else torch.bfloat16
        sc = torch.empty(4, dtype=torch.float32, device=DEV) if scaled else None
        dcur = torch.empty((T, B, d.n_out), dtype=gdt, device=DEV)
        snn.snn_neuron_bwd(d, snn.GRAD_BCAST if last else snn.GRAD_FULL, g, None, Is, ck, dcur,
                           None, None, net.ws, dcur_scale=sc)
        S = float(_np(sc)[0]) if scaled else 1.0
        g_c = _np(g[bs][:, ns]) if last else _np(g[:, bs][:, :, ns])
        dI_o = oracle.scan_bwd(u_o, g_c, spec["neuron"], spec["beta"], spec["thr"], wl.slope)
        assert_close(_np(dcur[:, bs][:, :, ns].float()) / S, dI_o, tol, what=f"L{li} dL/dI")
        del Is, spk, u, dcur, ck
        # ---- synapse backward on seeded 16-bit dL/dI: sampled dW rows, dx rows
        S = 2.0 ** 20 if scaled else 1.0
        dI = _seeded_normal((T * B, d.n_out), 0.0, 1e-4 * S, seed=400 + li, dtype=gdt)
        sc = torch.full((4,), S, dtype=torch.float32, device=DEV) if scaled else None
        gW = torch.empty((d.n_out, d.n_in), dtype=torch.float32, device=DEV)
        gx = torch.empty((T * B, d.n_in), dtype=torch.float32, device=DEV) if li > 0 else None
        snn.snn_synapse_bwd(d, dI, None, xin_dev, net.W[li], gW, gx, net.ws, dcur_scale=sc)
        xall = _np(xin_dev.reshape(T * B, -1)).astype(np.float64)
        cols_o = np.arange(d.n_out) if last else rng.integers(0, d.n_out, 8)
        dI_h = _np(dI.float()).astype(np.float64) / S           # the seeded 16-bit values
        dW_o, _, _ = oracle.dense_bwd(dI_h[:, cols_o], xall, W[cols_o], want_db=False,
                                      want_dx=False)
        # fp32 sums of exact products: within 1e-3, or the a-priori bound of an
        # fp32 sum of K terms in any order, (K + 2) 2^-24 sum|terms|
        bW = (T * B + 2) * 2.0 ** -24 * (np.abs(dI_h[:, cols_o]).T @ xall)
        assert_close(_np(gW)[cols_o], dW_o, 1e-3, what=f"L{li} dW rows", abs_bound=bW)
        if gx is not None:
            _, _, dx_o = oracle.dense_bwd(dI_h[rows], xall[rows], W, want_dw=False,
                                          want_db=False)
            bx = (d.n_out + 2) * 2.0 ** -24 * (np.abs(dI_h[rows]) @ np.abs(W).astype(np.float64))
            assert_close(_np(gx)[rows], dx_o, 1e-3, what=f"L{li} dx rows", abs_bound=bx)
        del dI, gW, gx, xin_dev
    # ---- the whole step: layer calls and stage calls give the same bytes
    x = torch.as_tensor(inp["x"]).to(DEV)
    y = torch.as_tensor(inp["labels"]).to(DEV)
    net.step(x, labels=y)
    snap = [_np(t).copy() for t in net.gW + net.gb] + [_np(net.loss).copy()]
    net.step_stages(x, labels=y)
    for a, b2 in zip(snap, [_np(t) for t in net.gW + net.gb] + [_np(net.loss)]):
        np.testing.assert_array_equal(a, b2)

"""GPU path vs CPU oracle, through the C ABI, on identical seeded inputs.

The oracle only ever sees seeded inputs and its own results.  Whole-step
checks run the oracle's chain on its own and feed each GPU stage the oracle's
inputs to that stage, so that a legal spike flip in one stage cannot cascade
into the next.  Scans given identical fp32 currents must be bit-identical.
"""
import copy

import numpy as np
import pytest

import oracle
import paper_2211_10725_amd as snn
from paper_2211_10725_amd import workloads as wls
from tests.parity import assert_close, assert_spikes, pow2_scale, spike_flips

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


def _assert_checkpoints(d, ck, u):
    """The forward's checkpoints are the oracle's membrane after every
    ckpt_interval-th step (the current-based neuron's second plane, i, is
    checked through the recomputed backward)."""
    lay = snn.snn_layer_saved_layout(d)
    C = d.B * d.n_out
    got = _np(ck)[: lay.ckpt_count * C].reshape(lay.ckpt_count, C)
    for c in range(lay.ckpt_count):
        t = (c + 1) * lay.ckpt_interval - 1
        np.testing.assert_array_equal(got[c], np.asarray(u).reshape(d.T, C)[t],
                                      err_msg=f"checkpoint {c}")


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
    ck = snn.ckpt_buffer(d)
    snn.snn_neuron_fwd(d, x, None, spk, ck, counts, u_out=saved)
    z, u, c = oracle.scan_fwd(I, neuron, beta, 1.0, alpha)
    np.testing.assert_array_equal(_np(spk), z)
    np.testing.assert_array_equal(_np(saved), u)
    np.testing.assert_array_equal(_np(counts), c)
    _assert_checkpoints(d, ck, u)
    # without the membrane output: the same spikes, counts and checkpoints
    spk2, ck2 = torch.empty_like(spk), snn.ckpt_buffer(d)
    snn.snn_neuron_fwd(d, x, None, spk2, ck2, counts)
    np.testing.assert_array_equal(_np(spk2), z)
    np.testing.assert_array_equal(_np(counts), c)
    lay = snn.snn_layer_saved_layout(d)
    used = lay.ckpt_planes * lay.ckpt_count * B * N
    np.testing.assert_array_equal(_np(ck2)[:used], _np(ck)[:used])


def test_scan_fwd_in_place_and_f16_spikes():
    T, B, N = 20, 3, 64
    rng = np.random.default_rng(11)
    I = rng.normal(0.3, 0.8, (T, B, N)).astype(np.float32)
    d, _ = _none_desc(T, B, N, "synaptic", 0.8, 0.6)
    d.out_dtype = snn.F16
    buf = _t(I)
    spk = torch.empty((T, B, N), dtype=torch.float16, device=DEV)
    snn.snn_neuron_fwd(d, buf, None, spk, snn.ckpt_buffer(d), None,
                       u_out=buf)                           # currents overwritten by u
    z, u, _ = oracle.scan_fwd(I, "synaptic", 0.8, 1.0, 0.6)
    np.testing.assert_array_equal(_np(buf), u)
    np.testing.assert_array_equal(_np(spk).astype(np.uint8), z)


# SNN_SPK_BITS: (5, 8, 65536) takes two-column lanes (the even and odd
# columns' ballots interleaved), (3, 9, 65600) one-column lanes on a wide
# layer (4.3M columns, not a multiple of 128), the others one-column lanes.
@pytest.mark.parametrize("neuron,alpha,beta", [("leaky", 0.0, 0.95), ("synaptic", 0.9, 0.8)])
@pytest.mark.parametrize("T,B,N", [(1, 1, 64), (7, 3, 128), (5, 8, 65536), (3, 9, 65600)])
def test_scan_fwd_packed_bits(neuron, alpha, beta, T, B, N):
    """Spikes packed 64 to a word: neuron n of row (t, b) is bit n % 8 of
    byte n / 8 of the row, the oracle's spikes packed; counts and checkpoints
    as with byte spikes."""
    rng = np.random.default_rng(T * 1000 + N + 7)
    I = rng.normal(0.3, 0.8, (T, B, N)).astype(np.float32)
    d, _ = _none_desc(T, B, N, neuron, beta, alpha)
    d.out_dtype = snn.SPK_BITS
    bits = torch.full((T, B, N // 8), 0xA5, dtype=torch.uint8, device=DEV)
    counts = torch.empty((B, N), dtype=torch.float32, device=DEV)
    ck = snn.ckpt_buffer(d)
    snn.snn_neuron_fwd(d, _t(I), None, bits, ck, counts)
    z, u, c = oracle.scan_fwd(I, neuron, beta, 1.0, alpha)
    want = np.packbits(np.asarray(z, np.uint8).reshape(T, B, N), axis=-1, bitorder="little")
    np.testing.assert_array_equal(_np(bits), want)
    np.testing.assert_array_equal(_np(counts), c)
    _assert_checkpoints(d, ck, u)


def test_network_bf16_input_spikes():
    """An fp32 net given its input spikes as bf16 0/1 (the operand type of
    the three-plane contractions: no widening of the spikes per call)
    computes what it computes from byte spikes, bit for bit, through the
    layer calls and through the stage calls: the 784-1000-10 synaptic net at
    full size, whose first layer's forward and weight gradient run on the
    asynchronous kernel."""
    wl = wls.get("dsnn_synaptic_t50_b256")
    inp = wls.make_inputs(wl, seed=5)
    x, lab = _t(inp["x"]), _t(inp["labels"])
    xb = x.to(torch.bfloat16)
    nets = [snn.Network(wl, inp["params"], device=DEV, input_bf16=f) for f in (False, True)]
    assert nets[1].descs[0].in_dtype == snn.BF16
    nets[0].step(x, labels=lab)
    want = [_np(t).copy() for t in nets[0].gW + nets[0].gb + nets[0].spk +
            [nets[0].counts, nets[0].loss[:1]]]
    for stages in (False, True):
        if stages:
            nets[1].step_stages(xb, labels=lab)
        else:
            nets[1].step(xb, labels=lab)
        got = [_np(t) for t in nets[1].gW + nets[1].gb + nets[1].spk +
               [nets[1].counts, nets[1].loss[:1]]]
        for a, b in zip(want, got):
            np.testing.assert_array_equal(a, b)


def test_network_packed_output_spikes():
    """A scan-only network with its spikes packed gives the unpacked
    network's spikes, counts, loss and gradients bit for bit."""
    wl = wls.scaled(wls.get("scan_wide_t1000_b64"), T=40, B=16, width=65536)
    inp = wls.make_inputs(wl, seed=3)
    x, tgt = _t(inp["x"]), _t(inp["targets"])
    nets = [snn.Network(wl, inp["params"], device=DEV, spike_bits=sb) for sb in (False, True)]
    for net in nets:
        net.step(x, targets=tgt)
    assert nets[1].descs[0].out_dtype == snn.SPK_BITS
    z = _np(nets[0].spk[0])
    np.testing.assert_array_equal(_np(nets[1].spk[0]),
                                  np.packbits(z, axis=-1, bitorder="little"))
    for a, b in ((nets[0].counts, nets[1].counts), (nets[0].loss[:1], nets[1].loss[:1]),
                 (nets[0].gx[0], nets[1].gx[0])):
        np.testing.assert_array_equal(_np(a), _np(b))


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
    ck = snn.ckpt_buffer(d)
    snn.snn_neuron_fwd(d, x, None, spk, ck, None, u_out=saved)
    _, u, _ = oracle.scan_fwd(I, neuron, beta, 1.0, alpha)
    np.testing.assert_array_equal(_np(saved), u)
    g = rng.normal(0, 1, (B, N) if bcast else (T, B, N)).astype(np.float32)
    dI = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
    snn.snn_neuron_bwd(d, snn.GRAD_BCAST if bcast else snn.GRAD_FULL, _t(g), None, x, ck, dI,
                       None, None, None)
    ref = oracle.scan_bwd(u, g, neuron, beta, 1.0, 25.0, alpha, reset == snn.RESET_SURROGATE)
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
    x, ck = _t(I), snn.ckpt_buffer(dn)
    snn.snn_neuron_fwd(dn, x, None, spk, ck, None, u_out=saved)
    _, u, _ = oracle.scan_fwd(I, "leaky", 0.9, 1.0)
    np.testing.assert_array_equal(_np(saved), u)
    g = rng.normal(0, 0.01, (B, N)).astype(np.float32)
    dI = torch.empty((T, B, N), dtype=tdt, device=DEV)
    sc = torch.full((4,), float("nan"), dtype=torch.float32, device=DEV)
    snn.snn_neuron_bwd(d, snn.GRAD_BCAST, _t(g), None, x, ck, dI, None, None,
                       _ws(snn.snn_layer_workspace_bytes(d)), dcur_scale=sc)
    ref = oracle.scan_bwd(u, g, "leaky", 0.9, 1.0, 25.0)
    S = 1.0
    if gdt == snn.F16:
        # S = 2^e, the largest with max|g| F S <= 2^15, F = sum_{k<T} 0.9^k
        S = float(_np(sc)[0])
        F = (1.0 - 0.9 ** T) / (1.0 - 0.9)
        assert S == pow2_scale([np.abs(g).max() * F])
        assert np.abs(_np(dI.float())).max() <= 2.0 ** 15
    assert_close(_np(dI.float()) / S, ref, 2e-2, what="half dL/dI")


# The input gradient of a readout (dense, <= 16 outputs) folded into the
# reverse scan of the layer below (SNN_GRAD_FOLD): the scan computes
# g[t,b,n] = sum_j dI_up[t,b,j] W_up[j,n] itself.  N = 64: a workgroup's 256
# columns span 5 batch rows; ragged column counts; n_up 1 and 16; N = 4096
# (over 512k columns) the 2-column lanes; N = 1018 over 512k columns, also
# 2-column lanes with ragged workgroups.
FOLD_SHAPES = [(7, 5, 64, 10), (9, 3, 1000, 10), (5, 4, 100, 1), (6, 2, 130, 16),
               (40, 3, 257, 7), (3, 128, 4096, 10), (2, 516, 1018, 10)]


@pytest.mark.parametrize("neuron,alpha,beta", [("leaky", 0.0, 0.95), ("synaptic", 0.9, 0.8),
                                               ("rleaky", 0.0, 0.9)])
@pytest.mark.parametrize("T,B,N,nup", FOLD_SHAPES)
def test_scan_bwd_fold(neuron, alpha, beta, T, B, N, nup):
    rng = np.random.default_rng(T * 31 + N + nup)
    I = rng.normal(0.3, 0.8, (T, B, N)).astype(np.float32)
    v = rng.uniform(-1.0, 1.5, N).astype(np.float32) if neuron == "rleaky" else None
    d, _ = _none_desc(T, B, N, neuron, beta, alpha)
    spk = torch.empty((T, B, N), dtype=torch.uint8, device=DEV)
    saved = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
    v_t = None if v is None else _t(v)
    x, ck = _t(I), snn.ckpt_buffer(d)
    snn.snn_neuron_fwd(d, x, v_t, spk, ck, None, u_out=saved)
    _, u, _ = oracle.scan_fwd(I, neuron, beta, 1.0, alpha, v=v)
    np.testing.assert_array_equal(_np(saved), u)
    dup = rng.normal(0, 0.1, (T, B, nup)).astype(np.float32)
    wup = rng.uniform(-1, 1, (nup, N)).astype(np.float32)
    g = dup.astype(np.float64) @ wup.astype(np.float64)   # the readout's dx
    dI = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
    gv = None if v is None else torch.empty(N, dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_layer_workspace_bytes(d))
    snn.snn_neuron_bwd(d, snn.GRAD_FOLD, (_t(dup), _t(wup)), v_t, x, ck, dI, None, gv, ws)
    if neuron == "rleaky":
        ref, dv = oracle.scan_bwd_rleaky(u, g, beta, 1.0, 25.0, v)
        assert_close(_np(gv), dv, 1e-3, what="dL/dv")
    else:
        ref = oracle.scan_bwd(u, g, neuron, beta, 1.0, 25.0, alpha)
    assert_close(_np(dI), ref, 1e-3, what="dL/dI (folded)")


def test_scan_bwd_fold_half_operands():
    """bf16 dL/dI and fp16 weights above (the fp16 network's readout), a bf16
    gradient written below; products of the given values are exact."""
    T, B, N, nup = 12, 6, 320, 10
    rng = np.random.default_rng(21)
    I = rng.normal(0.3, 0.8, (T, B, N)).astype(np.float32)
    spec = dict(kind="dense", n_in=8, n_out=N, neuron="leaky", beta=0.9)
    d = snn.layer_desc(spec, T, B, grad_dtype=snn.BF16)
    dn, _ = _none_desc(T, B, N, "leaky", 0.9)
    spk = torch.empty((T, B, N), dtype=torch.uint8, device=DEV)
    x, ck = _t(I), snn.ckpt_buffer(dn)
    snn.snn_neuron_fwd(dn, x, None, spk, ck, None)
    _, u, _ = oracle.scan_fwd(I, "leaky", 0.9, 1.0)
    dup = torch.as_tensor(rng.normal(0, 0.01, (T, B, nup)).astype(np.float32)).to(torch.bfloat16)
    wup = torch.as_tensor(rng.uniform(-1, 1, (nup, N)).astype(np.float32)).to(torch.float16)
    g = dup.float().numpy().astype(np.float64) @ wup.float().numpy().astype(np.float64)
    dI = torch.empty((T, B, N), dtype=torch.bfloat16, device=DEV)
    gb = torch.empty(N, dtype=torch.float32, device=DEV)
    snn.snn_neuron_bwd(d, snn.GRAD_FOLD, (dup.to(DEV), wup.to(DEV)), None, x, ck, dI, gb, None,
                       _ws(snn.snn_layer_workspace_bytes(d)))
    ref = oracle.scan_bwd(u, g, "leaky", 0.9, 1.0, 25.0)
    assert_close(_np(dI.float()), ref, 2e-2, what="half dL/dI (folded)")
    assert_close(_np(gb), ref.sum(axis=(0, 1)), 1e-3, what="db (folded)")


def _bf16_parts(x):
    """The three exact bf16 parts of fp32 values, hi = bf16(x), mid =
    bf16(x - hi), lo = bf16(x - hi - mid) (round to nearest even; every
    subtraction exact), as uint16 bit patterns."""
    x = torch.as_tensor(np.ascontiguousarray(x, np.float32))
    hi = x.to(torch.bfloat16)
    r = x - hi.float()
    mid = r.to(torch.bfloat16)
    lo = (r - mid.float()).to(torch.bfloat16)
    return [t.view(torch.int16).numpy().view(np.uint16) for t in (hi, mid, lo)]


@pytest.mark.parametrize("gkind", ["fold", "full", "bcast"])
@pytest.mark.parametrize("gdt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("T,B,N", [(37, 5, 300), (20, 3, 64), (16, 1100, 512), (7, 130, 4096)])
def test_scan_bwd_transposed_operand(gkind, gdt, T, B, N):
    """The reverse scan's transposed dL/dI (the weight gradient's operand,
    [P][N][B*T] with K index b*T + t) holds exactly the row-major dL/dI's
    16-bit parts: bf16 parts of fp32, or the bf16 / scaled fp16 value; one
    and two column lanes, ragged chunks (T not a multiple of 16 or 4)."""
    rng = np.random.default_rng(T * 7 + N + B)
    I = rng.normal(0.3, 0.8, (T, B, N)).astype(np.float32)
    gcode, tdt = GRAD_TYPES[gdt]
    spec = dict(kind="dense", n_in=8, n_out=N, neuron="synaptic" if N == 300 else "leaky",
                beta=0.8, alpha=0.5)
    d = snn.layer_desc(spec, T, B, grad_dtype=gcode)
    dn, _ = _none_desc(T, B, N, spec["neuron"], 0.8, 0.5)
    x, ck = _t(I), snn.ckpt_buffer(dn)
    spk = torch.empty((T, B, N), dtype=torch.uint8, device=DEV)
    snn.snn_neuron_fwd(dn, x, None, spk, ck, None)
    if gkind == "fold":
        nup = 10
        g = (_t(rng.normal(0, 0.1, (T, B, nup)).astype(np.float32)),
             _t(rng.uniform(-1, 1, (nup, N)).astype(np.float32)))
        kind = snn.GRAD_FOLD
    elif gkind == "full":
        g, kind = _t(rng.normal(0, 0.1, (T, B, N)).astype(np.float32)), snn.GRAD_FULL
    else:
        g, kind = _t(rng.normal(0, 0.1, (B, N)).astype(np.float32)), snn.GRAD_BCAST
    P = 3 if gcode == snn.F32 else 1
    ws = _ws(snn.snn_layer_workspace_bytes(d))
    sc = torch.empty(4, dtype=torch.float32, device=DEV)
    dI = torch.empty((T, B, N), dtype=tdt, device=DEV)
    snn.snn_neuron_bwd(d, kind, g, None, x, ck, dI, None, None, ws, dcur_scale=sc)
    dt = torch.full((P, N, B * T), 0x7fff, dtype=torch.int16, device=DEV)
    snn.snn_neuron_bwd(d, kind, g, None, x, ck, None, None, None, ws, dcur_scale=sc, dcur_t=dt)
    got = _np(dt).view(np.uint16)
    if gcode == snn.F32:
        parts = _bf16_parts(_np(dI))
    else:
        parts = [_np(dI.view(torch.int16)).view(np.uint16)]
    for p in range(P):
        want = parts[p].reshape(T, B, N).transpose(2, 1, 0).reshape(N, B * T)
        np.testing.assert_array_equal(got[p], want, err_msg=f"plane {p}")


def test_synapse_bwd_transposed_operand_same_bytes():
    """The weight gradient from the scan's transposed operand equals the one
    from the row-major dL/dI (transposed inside the call): the same operand
    bytes in the same contraction."""
    # 9600 rows and 602 neurons (not a multiple of 8, which the M/N-contiguous
    # asynchronous kernel needs): the transposed path for fp32 dL/dI
    T, B, N, K = 40, 240, 602, 784
    rng = np.random.default_rng(3)
    spec = dict(kind="dense", n_in=K, n_out=N, neuron="leaky", beta=0.9)
    # with 600 neurons a 16-bit or fp32 dL/dI is contracted in its own layout:
    # no transposed operand (an fp32 one as the three planes of its values)
    spec600 = dict(spec, n_out=600)
    for gdt in ("bf16", "f16"):
        assert snn.snn_layer_dcur_t_bytes(snn.layer_desc(spec600, T, B,
                                                         grad_dtype=GRAD_TYPES[gdt][0])) == 0
    assert snn.snn_layer_dcur_t_layout(snn.layer_desc(spec600, T, B)) == snn.DCUR_T_PLANES
    assert snn.snn_layer_dcur_t_layout(snn.layer_desc(spec, T, B)) == snn.DCUR_T_TRANSPOSED
    for gdt in ("f32",):
        gcode, tdt = GRAD_TYPES[gdt]
        d = snn.layer_desc(spec, T, B, grad_dtype=gcode)
        assert snn.snn_layer_dcur_t_bytes(d) > 0
        I = rng.normal(0.3, 0.8, (T, B, N)).astype(np.float32)
        dn, _ = _none_desc(T, B, N, "leaky", 0.9)
        xc, ck = _t(I), snn.ckpt_buffer(dn)
        snn.snn_neuron_fwd(dn, xc, None, torch.empty((T, B, N), dtype=torch.uint8, device=DEV),
                           ck, None)
        g = _t(rng.normal(0, 0.1, (B, N)).astype(np.float32))
        ws = _ws(snn.snn_layer_workspace_bytes(d))
        dI = torch.empty((T, B, N), dtype=tdt, device=DEV)
        dt = torch.empty(snn.snn_layer_dcur_t_bytes(d), dtype=torch.uint8, device=DEV)
        snn.snn_neuron_bwd(d, snn.GRAD_BCAST, g, None, xc, ck, dI, None, None, ws, dcur_t=dt)
        x = _t((rng.random((T, B, K)) < 0.3).astype(np.uint8))
        W = _t(rng.uniform(-0.05, 0.05, (N, K)).astype(np.float32))
        gW1 = torch.empty((N, K), dtype=torch.float32, device=DEV)
        gW2 = torch.empty_like(gW1)
        snn.snn_synapse_bwd(d, dI, None, x, W, gW1, None, ws)
        snn.snn_synapse_bwd(d, None, None, x, W, gW2, None, ws, dcur_t=dt)
        np.testing.assert_array_equal(_np(gW1), _np(gW2))
        rW, _, _ = oracle.dense_bwd(_np(dI.float()).astype(np.float64).reshape(T * B, N),
                                    _np(x).reshape(T * B, K), _np(W), want_db=False,
                                    want_dx=False)
        assert_close(_np(gW2), rW, 1e-3, what=f"dW from the transposed {gdt} operand")


def _bf16_rne(x):
    """bf16 bits of fp32 values, round to nearest even (finite values)."""
    b = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    return ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)


def _bf16_val(h):
    return (h.astype(np.uint32) << 16).view(np.float32)


def _three_parts(x):
    """hi = bf16(x), mid = bf16(x - hi), lo = bf16(x - hi - mid), each
    difference exact in fp32."""
    x = np.asarray(x, np.float32)
    hi = _bf16_rne(x)
    r = x - _bf16_val(hi)
    mid = _bf16_rne(r)
    lo = _bf16_rne(r - _bf16_val(mid))
    return np.stack([hi, mid, lo])


def test_synapse_bwd_planes_operand_same_bytes():
    """An fp32 dL/dI that the weight gradient reads in its own layout: the
    reverse scan writes its three exact bf16 parts as [3][T*B][n_out] (the
    split of the fp32 values it writes beside them, bit for bit; the parts
    add up to the value exactly), and the weight gradient from them equals
    the one from the fp32 dL/dI (split inside the call)."""
    T, B, N, K = 40, 240, 600, 784
    rng = np.random.default_rng(5)
    spec = dict(kind="dense", n_in=K, n_out=N, neuron="leaky", beta=0.9)
    d = snn.layer_desc(spec, T, B)
    assert snn.snn_layer_dcur_t_layout(d) == snn.DCUR_T_PLANES
    nb = snn.snn_layer_dcur_t_bytes(d)
    assert nb >= 3 * T * B * N * 2
    I = rng.normal(0.3, 0.8, (T, B, N)).astype(np.float32)
    dn, _ = _none_desc(T, B, N, "leaky", 0.9)
    xc, ck = _t(I), snn.ckpt_buffer(dn)
    snn.snn_neuron_fwd(dn, xc, None, torch.empty((T, B, N), dtype=torch.uint8, device=DEV), ck,
                       None)
    g = _t(rng.normal(0, 0.1, (B, N)).astype(np.float32))
    ws = _ws(snn.snn_layer_workspace_bytes(d))
    dI = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
    dt = torch.zeros(nb, dtype=torch.uint8, device=DEV)
    snn.snn_neuron_bwd(d, snn.GRAD_BCAST, g, None, xc, ck, dI, None, None, ws, dcur_t=dt)
    dI_h = _np(dI)
    planes = _np(dt[:3 * T * B * N * 2].view(torch.int16)).view(np.uint16).reshape(3, T * B, N)
    want = _three_parts(dI_h.reshape(T * B, N))
    np.testing.assert_array_equal(planes, want)
    total = sum(_bf16_val(planes[p]).astype(np.float64) for p in range(3))
    np.testing.assert_array_equal(total, dI_h.reshape(T * B, N).astype(np.float64))
    x = _t((rng.random((T, B, K)) < 0.3).astype(np.uint8))
    W = _t(rng.uniform(-0.05, 0.05, (N, K)).astype(np.float32))
    gW1 = torch.empty((N, K), dtype=torch.float32, device=DEV)
    gW2 = torch.empty_like(gW1)
    snn.snn_synapse_bwd(d, dI, None, x, W, gW1, None, ws)
    snn.snn_synapse_bwd(d, None, None, x, W, gW2, None, ws, dcur_t=dt)
    np.testing.assert_array_equal(_np(gW1), _np(gW2))
    rW, _, _ = oracle.dense_bwd(dI_h.astype(np.float64).reshape(T * B, N),
                                _np(x).reshape(T * B, K), _np(W), want_db=False, want_dx=False)
    assert_close(_np(gW2), rW, 1e-3, what="dW from the scan's planes")
    _assert_fp32_sum(_np(gW2) - rW, np.abs(dI_h.reshape(T * B, N)).astype(np.float64).T @
                     _np(x).reshape(T * B, K).astype(np.float64), T * B, "dW")


@pytest.mark.parametrize("reset", [snn.RESET_DETACHED, snn.RESET_SURROGATE])
def test_step_fp32_planes_operand(reset):
    """784-704-704-10 in fp32 over 9600 rows: both hidden layers' weight
    gradients read dL/dI as the three bf16 planes the reverse scan writes,
    the upper one beside the fp32 dL/dI its input gradient needs.  Stage by
    stage against the oracle, and the layer calls give the stage calls'
    bytes."""
    wl = copy.deepcopy(wls.get("dsnn_half_t100_b512"))
    wl.dtype = "f32"
    wl = wls.scaled(wl, T=40, B=240, width=704)
    inp = wls.make_inputs(wl, seed=6)
    net = snn.Network(wl, inp["params"], device=DEV, reset_grad=reset)
    assert [snn.snn_layer_dcur_t_layout(d) for d in net.descs[:2]] == [snn.DCUR_T_PLANES] * 2
    _check_step_stagewise(wl, inp, reset)
    x, lab = _t(inp["x"]), _t(inp["labels"])
    net.step(x, labels=lab)
    ref = [_np(t).copy() for t in net.gW + net.gb]
    net.step_stages(x, labels=lab)
    for a, b in zip(ref, [_np(t) for t in net.gW + net.gb]):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("name,T,B,width", [("dsnn_synaptic_t50_b256", 40, 240, 602)])
def test_step_with_scan_transposed_operand(name, T, B, width):
    """A whole step whose reverse scans write the weight gradients' operands
    transposed gives the layer calls' gradients bit for bit (the same operand
    bytes in the same contractions)."""
    wl = wls.scaled(wls.get(name), T=T, B=B, width=width)
    inp = wls.make_inputs(wl, seed=2)
    net = snn.Network(wl, inp["params"], device=DEV)
    assert any(b > 0 for b in net.dcur_t_bytes)
    x, lab = _t(inp["x"]), _t(inp["labels"])
    net.step(x, labels=lab)
    ref = [_np(t).copy() for t in net.gW + net.gb]
    net.transposed_operand = True
    net.step_stages(x, labels=lab)
    for a, b in zip(ref, [_np(t) for t in net.gW + net.gb]):
        np.testing.assert_array_equal(a, b)


# recurrent neuron (eq. 7): one recurrent weight per neuron, column c of the
# [T, B*N] layout is neuron c % N.  (8, 65537) takes the 2-column lanes with
# pairs that straddle two samples; (9, 65537) the 1-column lanes (odd count).
RLEAKY_SHAPES = [(1, 2, 8), (7, 3, 101), (33, 4, 256), (50, 5, 1001), (6, 8, 65537),
                 (3, 9, 65537)]


def _rleaky_case(T, B, N, seed):
    rng = np.random.default_rng(seed)
    I = rng.normal(0.3, 0.8, (T, B, N)).astype(np.float32)
    v = rng.uniform(-1.0, 1.5, N).astype(np.float32)
    return I, v, rng


@pytest.mark.parametrize("T,B,N", RLEAKY_SHAPES)
def test_rleaky_scan_fwd_bit_exact(T, B, N):
    I, v, _ = _rleaky_case(T, B, N, seed=T * 100 + N)
    d, _ = _none_desc(T, B, N, "rleaky", 0.9)
    spk = torch.empty((T, B, N), dtype=torch.uint8, device=DEV)
    saved = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
    counts = torch.empty((B, N), dtype=torch.float32, device=DEV)
    ck = snn.ckpt_buffer(d)
    snn.snn_neuron_fwd(d, _t(I), _t(v), spk, ck, counts, u_out=saved)
    z, u, c = oracle.scan_fwd(I, "rleaky", 0.9, 1.0, v=v)
    _assert_checkpoints(d, ck, u)
    np.testing.assert_array_equal(_np(spk), z)
    np.testing.assert_array_equal(_np(saved), u)
    np.testing.assert_array_equal(_np(counts), c)


@pytest.mark.parametrize("reset", [snn.RESET_DETACHED, snn.RESET_SURROGATE])
@pytest.mark.parametrize("bcast", [True, False])
@pytest.mark.parametrize("T,B,N", [(1, 2, 8), (9, 3, 37), (40, 4, 512), (5, 8, 65538)])
def test_rleaky_scan_bwd(reset, bcast, T, B, N):
    """dL/dI and the recurrent weights' gradient dL/dv (summed over the batch)."""
    I, v, rng = _rleaky_case(T, B, N, seed=7 * T + N)
    d, _ = _none_desc(T, B, N, "rleaky", 0.9, reset=reset)
    spk = torch.empty((T, B, N), dtype=torch.uint8, device=DEV)
    saved = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
    v_t = _t(v)
    x, ck = _t(I), snn.ckpt_buffer(d)
    snn.snn_neuron_fwd(d, x, v_t, spk, ck, None, u_out=saved)
    _, u, _ = oracle.scan_fwd(I, "rleaky", 0.9, 1.0, v=v)
    np.testing.assert_array_equal(_np(saved), u)
    g = rng.normal(0, 1, (B, N) if bcast else (T, B, N)).astype(np.float32)
    dI = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
    gv = torch.empty(N, dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_layer_workspace_bytes(d))
    snn.snn_neuron_bwd(d, snn.GRAD_BCAST if bcast else snn.GRAD_FULL, _t(g), v_t, x, ck, dI,
                       None, gv, ws)
    ref, dv = oracle.scan_bwd_rleaky(u, g, 0.9, 1.0, 25.0, v, reset == snn.RESET_SURROGATE)
    assert_close(_np(dI), ref, 1e-3, what="dL/dI")
    assert_close(_np(gv), dv, 1e-3, what="dL/dv")


def test_rleaky_zero_weight_matches_leaky_kernel():
    """v = 0 is eq. (4): the recurrent kernel gives the Leaky kernel's bytes."""
    T, B, N = 20, 4, 300
    I, _, rng = _rleaky_case(T, B, N, seed=3)
    out = []
    for neuron, v in (("rleaky", _t(np.zeros(N, np.float32))), ("leaky", None)):
        d, _ = _none_desc(T, B, N, neuron, 0.9, reset=snn.RESET_SURROGATE)
        spk = torch.empty((T, B, N), dtype=torch.uint8, device=DEV)
        saved = torch.empty((T, B, N), dtype=torch.float32, device=DEV)
        snn.snn_neuron_fwd(d, _t(I), v, spk, snn.ckpt_buffer(d), None, u_out=saved)
        out += [_np(spk), _np(saved)]
    np.testing.assert_array_equal(out[0], out[2])
    np.testing.assert_array_equal(out[1], out[3])


def test_rleaky_empty_batch_zero_gradient():
    d, _ = _none_desc(0, 4, 16, "rleaky", 0.9)
    gv = torch.full((16,), 5.0, device=DEV)
    g = torch.zeros(256, dtype=torch.float32, device=DEV)
    buf = torch.empty(256, dtype=torch.float32, device=DEV)
    v = torch.ones(16, dtype=torch.float32, device=DEV)
    snn.snn_neuron_bwd(d, snn.GRAD_BCAST, g, v, buf, buf, buf, None, gv, _ws(256))
    assert (_np(gv) == 0).all()


# ---------------------------------------------------------------------------
# synaptic contractions
# ---------------------------------------------------------------------------
GEMM_SHAPES = [(37, 29, 53), (800, 1000, 784), (128, 10, 1000), (300, 7, 33), (64, 130, 1),
               (5, 300, 17)]


PATHS = {"split": 0, "fp32mfma": snn.FLAG_FP32_MFMA}


# (1040, 1100, 1000): large enough for the 256 x 256 asynchronous kernel with
# fp16 weights, ragged in M and N, and a last k-tile of 8 values; with fp32
# weights (12800, 1000, 784) and (12850, 1000, 1000) run its three-plane
# mode, the latter ragged in M, N and K.  Layers with at most 16 outputs:
# (12800, 10, 1000) the readout, (5000, 7, 1003) rows not 4-aligned,
# (777, 16, 1500) and (2000, 10, 4096) long contractions; (600, 8192, 256)
# the widest layer whose bias the asynchronous kernel stages in LDS, and
# (520, 8200, 256) one that goes to another kernel for that reason.
@pytest.mark.parametrize("M,N,K", GEMM_SHAPES + [(12800, 1000, 784), (12850, 1000, 1000),
                                                 (1040, 1100, 1000), (600, 8192, 256),
                                                 (520, 8200, 256),
                                                 (12800, 10, 1000), (5000, 7, 1003),
                                                 (777, 16, 1500), (2000, 10, 4096)])
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
# inputs give unaligned rows and a partial last group of 4 columns.
# (8197, 130, 1003): the weight gradient's operands are transposed first, with
# ragged rows and columns on both sides of every transpose.  (9640, 600, 784):
# the weight gradient on the asynchronous kernel's three-plane mode in the
# operands' own layouts, ragged in both tile dimensions, a partial last
# k-tile and 19 splits over K.
@pytest.mark.parametrize("M,N,K", GEMM_SHAPES + [(12800, 1000, 784), (12800, 10, 1000),
                                                 (5000, 7, 1003), (8197, 130, 1003),
                                                 (9640, 600, 784)])
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
                                   (1040, 1100, 1000), (12800, 10, 1000), (5000, 7, 1003),
                                   (1037, 1101, 1003)])
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
    # rounded on the host (fp16 scaled by a power of two, as the scans write it)
    S = pow2_scale(dI) if gcode == snn.F16 else 1.0
    dI_h = torch.as_tensor(dI * np.float32(S)).to(tdt)
    dI_used = dI_h.float().numpy().astype(np.float64) / S   # the values the GPU sees
    dI_t = dI_h.to(DEV)
    sc = _t(np.full(4, S, np.float32)) if gcode == snn.F16 else None
    spec = dict(kind="dense", n_in=K, n_out=N, neuron="leaky", beta=0.9)
    d = snn.layer_desc(spec, 1, M, grad_dtype=gcode, w_dtype=snn.F16 if wdt == "f16" else snn.F32)
    gW = torch.empty((N, K), dtype=torch.float32, device=DEV)
    gx = torch.empty((M, K), dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_layer_workspace_bytes(d))
    Wt = _t(W, torch.float16 if wdt == "f16" else torch.float32)
    snn.snn_synapse_bwd(d, dI_t, None, _t(x), Wt, gW, gx, ws, dcur_scale=sc)
    rW, _, rx = oracle.dense_bwd(dI_used, x, W)
    gotW, gotx = _np(gW), _np(gx)
    assert_close(gotW, rW, 1e-3, what="dW")
    assert_close(gotx, rx, 1e-3, what="dx")
    aI = np.abs(dI_used)
    _assert_fp32_sum(gotW - rW, aI.T @ x.astype(np.float64), M, "dW")
    _assert_fp32_sum(gotx - rx, aI @ np.abs(W).astype(np.float64), N, "dx")


# (rows T*B, n_out, n_in, x dtype): weight gradients of a 16-bit dL/dI large
# enough for the asynchronous pipeline, which stages dL/dI [T*B][n_out] and x
# [T*B][n_in] tiles as they are stored; ragged 256-tiles on both sides, a
# partial last k-tile (rows not a multiple of 64) and splits over K.
MN_DW_SHAPES = [(9640, 600, 784, "u8"), (8200, 264, 520, "f16"), (12800, 1000, 784, "f16")]


@pytest.mark.parametrize("M,N,K,xdt", MN_DW_SHAPES)
@pytest.mark.parametrize("gdt", ["bf16", "f16"])
def test_synapse_bwd_dw_own_layout(M, N, K, xdt, gdt):
    """dW = dI^T x from the M/N-contiguous operands (no transpose in memory):
    products of the 16-bit values are exact, so the result is their fp32 sum."""
    if gdt == "bf16" and xdt == "f16":
        pytest.skip("bf16 dL/dI against fp16 x has no common MFMA type")
    rng = np.random.default_rng(M + N + K)
    gcode, tdt = GRAD_TYPES[gdt]
    if xdt == "u8":
        x = (rng.random((M, K)) < 0.3).astype(np.uint8)
        x_dev, in_dt = _t(x), snn.U8
    else:
        x = (rng.random((M, K)) < 0.3).astype(np.float16)
        x_dev, in_dt = _t(x, torch.float16), snn.F16
    dI = rng.normal(0, 1e-3, (M, N)).astype(np.float32)
    S = pow2_scale(dI) if gcode == snn.F16 else 1.0
    dI_h = torch.as_tensor(dI * np.float32(S)).to(tdt)
    dI_used = dI_h.float().numpy().astype(np.float64) / S
    sc = _t(np.full(4, S, np.float32)) if gcode == snn.F16 else None
    spec = dict(kind="dense", n_in=K, n_out=N, neuron="leaky", beta=0.9)
    d = snn.layer_desc(spec, 1, M, grad_dtype=gcode, in_dtype=in_dt, w_dtype=snn.F16)
    assert snn.snn_layer_dcur_t_bytes(d) == 0
    gW = torch.empty((N, K), dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_layer_workspace_bytes(d))
    W = _t(np.zeros((N, K), np.float16), torch.float16)
    snn.snn_synapse_bwd(d, dI_h.to(DEV), None, x_dev, W, gW, None, ws, dcur_scale=sc)
    xf = x.astype(np.float64)
    rW = dI_used.T @ xf
    got = _np(gW)
    assert_close(got, rW, 1e-3, what="dW")
    _assert_fp32_sum(got - rW, np.abs(dI_used).T @ xf, M, "dW")


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


# Up to 4 input channels of at most 4096 pixels in all, and at most 128
# output channels, take the direct convolution-and-pool kernel ((3, 1, 28,
# 28, 12); (1, 2, 6, 6, 2) one cell; (2, 4, 9, 11, 5), (2, 3, 9, 11, 5) and
# (300, 3, 15, 13, 70) several channels).  Spike input with Ci * 25 <= 320,
# Co <= 64, at most 32 pooled cells per channel and images of a whole number
# of 4-byte words runs the one-pass kernel: (5, 12, 12, 12, 64) and (800,
# ...) two row tiles per wave at 16 cells, (2, 8, 9, 11, 5) ragged, (1, 8, 6,
# 6, 2) one cell, (5, 7, 12, 12, 33) part of a channel tile, (2, 8, 7, 37,
# 40) a 259-pixel image, (3, 12, 14, 14, 64) 25 cells and (2, 6, 20, 12, 8)
# 32 (four row tiles per wave); past them the gather and the contraction,
# which pools its own output when it makes one pass over K ((300, 5, 15, 13,
# 70), 70 channels; (2, 5, 9, 11, 5), 495-byte images) or pools after it
# ((4, 13, 9, 9, 8), 325 columns split over K).
@pytest.mark.parametrize("NB,Ci,H,W,Co", [(3, 1, 28, 28, 12), (1, 2, 6, 6, 2), (2, 4, 9, 11, 5),
                                          (2, 3, 9, 11, 5), (300, 3, 15, 13, 70),
                                          (5, 12, 12, 12, 64), (2, 8, 9, 11, 5), (1, 8, 6, 6, 2),
                                          (800, 12, 12, 12, 64), (5, 7, 12, 12, 33),
                                          (2, 8, 7, 37, 40), (3, 12, 14, 14, 64), (2, 6, 20, 12, 8),
                                          (300, 5, 15, 13, 70), (2, 5, 9, 11, 5), (4, 13, 9, 9, 8)])
def test_conv_pool_fwd(NB, Ci, H, W, Co):
    x, w, b, d = _conv_case(NB, Ci, H, W, Co, seed=NB * 100 + Co)
    _check_conv_fwd(x, w, b, d)


# One input channel takes the direct convolution-and-pool kernel while the
# image fits its LDS buffer (4096 pixels): odd sizes, more output channels
# than threads per image, the largest staged image, one past it (contraction
# path), and real-valued input currents.
@pytest.mark.parametrize("NB,H,W,Co,real", [(4, 9, 11, 5, False), (2, 64, 64, 70, False),
                                           (3, 65, 64, 3, False), (3, 28, 28, 12, True)])
def test_conv_pool_fwd_one_channel(NB, H, W, Co, real):
    x, w, b, d = _conv_case(NB, 1, H, W, Co, seed=NB + H + Co)
    if real:
        x = np.random.default_rng(H).uniform(-1, 1, x.shape).astype(np.float32)
        spec = dict(kind="conv", c_in=1, h=H, w=W, c_out=Co, neuron="leaky", beta=0.5)
        d = snn.layer_desc(spec, 1, NB, in_dtype=snn.F32)
    _check_conv_fwd(x, w, b, d)


@pytest.mark.parametrize("NB,Ci,H,W,Co", [(3, 3, 16, 16, 20), (2, 4, 32, 32, 12)])
def test_conv_pool_fwd_direct_channels_real(NB, Ci, H, W, Co):
    """Real-valued input to the direct kernel with several input channels
    (the largest image it stages: 4 x 32 x 32)."""
    x, w, b, _ = _conv_case(NB, Ci, H, W, Co, seed=NB + Ci + H)
    x = np.random.default_rng(W).uniform(-1, 1, x.shape).astype(np.float32)
    spec = dict(kind="conv", c_in=Ci, h=H, w=W, c_out=Co, neuron="leaky", beta=0.5)
    d = snn.layer_desc(spec, 1, NB, in_dtype=snn.F32)
    _check_conv_fwd(x, w, b, d)


def _check_conv_fwd(x, w, b, d):
    NB, Ci = x.shape[0], x.shape[1]
    Co = w.shape[0]
    cur, arg = _conv_fwd_gpu(d, x, w, b)
    y = oracle.conv_fwd(x, w, b)                          # double
    y32 = y.astype(np.float32).astype(np.float64)          # the pool decides on fp32 currents
    p, a = oracle.maxpool2_fwd(y32)
    cur = cur.reshape(p.shape)
    arg = arg.reshape(a.shape)
    assert_close(cur, p, 1e-3, what="pooled currents")
    # fp32 accumulation of Ci*25 terms, any order
    terms = oracle.conv_fwd(np.abs(x), np.abs(w), np.abs(b))
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


# (3, 8, 11, 12, 16): an odd conv row outside every window.  Both gradients
# run in one pass each when Ci * 25 <= 320, Co <= 64 and at most 16 pooled
# cells per channel (the weight gradient up to 32 cells, on images of a
# whole number of 4-byte words): (4, 12, 12, 12, 64) and (300, ...) at the
# 16-cell limit (more images than compute units: a workgroup takes
# several), (2, 4, 9, 11, 5) and (3, 8, 11, 12, 16) ragged (6 and 12 cells),
# (5, 7, 12, 12, 33) half of the second k-step, (3, 5, 9, 21, 24) and (2, 4,
# 7, 37, 40) images of 189 and 259 pixels (two and one channel groups in the
# gather); (3, 12, 14, 14, 64) 25 cells and (2, 3, 20, 12, 8) 32: the weight
# gradient in one pass, the input gradient on the contraction; past each
# limit the gather-and-contraction path for both: 144 cells (one input
# channel), 36 cells (2, 4, 16, 16, 8), 70 output channels, 13 * 25 = 325
# inputs per channel and 297-byte images (2, 3, 9, 11, 5).  (1100, 12, 12,
# 12, 64): four or five images per workgroup, through every register set and
# buffer the kernels alternate.
@pytest.mark.parametrize("NB,Ci,H,W,Co", [(3, 1, 28, 28, 12), (4, 12, 12, 12, 64), (2, 4, 9, 11, 5),
                                          (3, 8, 11, 12, 16), (300, 12, 12, 12, 64),
                                          (5, 7, 12, 12, 33), (3, 5, 9, 21, 24), (2, 4, 7, 37, 40),
                                          (3, 12, 14, 14, 64), (2, 3, 20, 12, 8),
                                          (2, 4, 16, 16, 8), (2, 2, 8, 8, 70), (2, 13, 9, 9, 8),
                                          (2, 3, 9, 11, 5), (1100, 12, 12, 12, 64)])
def test_conv_pool_bwd(NB, Ci, H, W, Co):
    """Backward given the oracle's pool selection (one byte per pooled current)."""
    x, w, b, d = _conv_case(NB, Ci, H, W, Co, seed=7 * NB + Co)
    y32 = oracle.conv_fwd(x, w, b).astype(np.float32).astype(np.float64)
    _, arg = oracle.maxpool2_fwd(y32)
    rng = np.random.default_rng(1)
    dI = rng.normal(0, 1, arg.shape).astype(np.float32)
    gW = torch.empty(w.shape, dtype=torch.float32, device=DEV)
    gx = torch.empty(x.shape, dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_layer_workspace_bytes(d))
    snn.snn_synapse_bwd(d, _t(dI), _t(arg.astype(np.uint8)), _t(x), _t(w), gW, gx, ws)
    Ho, Wo = H - 4, W - 4
    # an odd conv output's last row / column is outside every window: zero gradient
    dY = oracle.maxpool2_bwd(dI, arg, Ho, Wo)
    rW, _, rx = oracle.conv_bwd(dY, x, w)
    assert_close(_np(gW), rW, 1e-3, what="conv dW")
    assert_close(_np(gx), rx, 1e-3, what="conv dx")
    # fp32 accuracy: dx^T sums at most six part products per output channel
    # (each within 2^-26 of the exact product), col2im at most 25 of those;
    # dW sums three exact part products per window row
    tW, _, tx = oracle.conv_bwd(np.abs(dY), x, np.abs(w))
    bound = ((6 * Co + 27) * 2.0 ** -24 + 2.0 ** -26) * tx
    assert (np.abs(_np(gx) - rx) <= bound + 1e-30).all()
    Mw = 4 * NB * (Ho // 2) * (Wo // 2)
    assert (np.abs(_np(gW) - rW) <= (3 * Mw + 2) * 2.0 ** -24 * tW + 1e-30).all()


@pytest.mark.parametrize("NB,Ci,H,W,Co", [(4, 6, 12, 12, 20), (3, 2, 28, 28, 12)])
def test_conv_pool_bwd_real_input(NB, Ci, H, W, Co):
    """Real-valued input: the weight gradient runs on the contraction path
    (the one-pass kernel takes spikes only), the input gradient in one pass
    where the image fits."""
    x, w, b, _ = _conv_case(NB, Ci, H, W, Co, seed=5 * NB + Ci)
    x = np.random.default_rng(Co).uniform(-1, 1, x.shape).astype(np.float32)
    spec = dict(kind="conv", c_in=Ci, h=H, w=W, c_out=Co, neuron="leaky", beta=0.5)
    d = snn.layer_desc(spec, 1, NB, in_dtype=snn.F32)
    y32 = oracle.conv_fwd(x, w, b).astype(np.float32).astype(np.float64)
    _, arg = oracle.maxpool2_fwd(y32)
    dI = np.random.default_rng(2).normal(0, 1, arg.shape).astype(np.float32)
    gW = torch.empty(w.shape, dtype=torch.float32, device=DEV)
    gx = torch.empty(x.shape, dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_layer_workspace_bytes(d))
    snn.snn_synapse_bwd(d, _t(dI), _t(arg.astype(np.uint8)), _t(x), _t(w), gW, gx, ws)
    dY = oracle.maxpool2_bwd(dI, arg, H - 4, W - 4)
    rW, _, rx = oracle.conv_bwd(dY, x, w)
    assert_close(_np(gW), rW, 1e-3, what="conv dW")
    assert_close(_np(gx), rx, 1e-3, what="conv dx")


# ---------------------------------------------------------------------------
# losses
# ---------------------------------------------------------------------------
# at most 16 classes, 128 rows and 12288 counts take the one-workgroup kernel
# ((1, 10), (32, 10), (7, 3), (128, 16)); (129, 16), (513, 10), (4096, 64),
# (4097, 10), (64, 65) and (5, 1500) (a row past the LDS staging) the
# row-per-wave kernel and its separate sum
@pytest.mark.parametrize("B,K", [(1, 10), (32, 10), (7, 3), (128, 16), (129, 16), (513, 10),
                                 (4096, 64), (4097, 10), (64, 65), (5, 1500)])
def test_loss_ce(B, K):
    rng = np.random.default_rng(B)
    c = rng.integers(0, 26, (B, K)).astype(np.float32)
    y = rng.integers(0, K, B).astype(np.int32)
    loss = torch.empty(4, dtype=torch.float32, device=DEV)
    g = torch.empty((B, K), dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_loss_workspace_bytes(snn.LOSS_CE_COUNT, B, K))
    snn.snn_loss(snn.LOSS_CE_COUNT, B, K, 1, _t(c), _t(y), None, loss, g, ws)
    L, rg = oracle.loss_ce(c, y)
    assert abs(_np(loss)[0] - L) <= 1e-6 * max(1.0, abs(L))
    assert_close(_np(g), rg, 1e-5, what="CE grad")


@pytest.mark.parametrize("K,P", [(10, 1), (16, 1), (7, 3), (16, 6)])
def test_loss_ce_one_and_two_launches_agree(K, P):
    """The one-workgroup cross-entropy (the most rows it takes: 128) and the
    row-per-wave path (the same rows and one more) give the same per-row
    gradients up to the 1/B factor, and the loss matches the oracle.  16
    classes of 6 neurons over 128 rows fill its 12288-count LDS buffer."""
    rng = np.random.default_rng(77 + K)
    B = 128
    c = rng.integers(0, 26, (B, K * P)).astype(np.float32)
    y = rng.integers(0, K, B).astype(np.int32)
    ws = _ws(snn.snn_loss_workspace_bytes(snn.LOSS_CE_COUNT, B + 1, K))
    # B rows: one launch; B + 1 rows (one repeated): the row-per-wave path
    c2, y2 = np.concatenate([c, c[:1]]), np.concatenate([y, y[:1]])
    out = []
    for cc, yy in ((c, y), (c2, y2)):
        loss = torch.empty(4, dtype=torch.float32, device=DEV)
        g = torch.empty(cc.shape, dtype=torch.float32, device=DEV)
        snn.snn_loss(snn.LOSS_CE_COUNT, len(cc), K, P, _t(cc), _t(yy), None, loss, g, ws)
        out.append((_np(loss)[0], _np(g)))
    L, rg = oracle.loss_ce(c, y, P)
    assert abs(out[0][0] - L) <= 1e-6 * max(1.0, abs(L))
    assert_close(out[0][1], rg, 1e-5, what="CE grad")
    L2, _ = oracle.loss_ce(c2, y2, P)
    assert abs(out[1][0] - L2) <= 1e-6 * max(1.0, abs(L2))
    # the gradient is (softmax - onehot) / B: rescale the B + 1 rows' by (B + 1) / B
    g1 = out[0][1].astype(np.float64) * B
    g2 = out[1][1][:B].astype(np.float64) * (B + 1)
    np.testing.assert_allclose(g1, g2, rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("B,K", [(1, 1), (64, 1000), (64, 65536), (3, 7)])
def test_loss_mse(B, K):
    rng = np.random.default_rng(K)
    c = rng.integers(0, 200, (B, K)).astype(np.float32)
    y = rng.uniform(0, 50, (B, K)).astype(np.float32)
    loss = torch.empty(4, dtype=torch.float32, device=DEV)
    g = torch.empty((B, K), dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_loss_workspace_bytes(snn.LOSS_MSE_COUNT, B, K))
    snn.snn_loss(snn.LOSS_MSE_COUNT, B, K, 1, _t(c), None, _t(y), loss, g, ws)
    L, rg = oracle.loss_mse(c, y)
    assert abs(_np(loss)[0] - L) <= 1e-6 * abs(L)
    assert_close(_np(g), rg, 1e-6, what="MSE grad")


@pytest.mark.parametrize("kind", [snn.LOSS_CE_COUNT, snn.LOSS_MSE_COUNT])
@pytest.mark.parametrize("B,K,P", [(128, 10, 50), (3, 7, 2), (300, 10, 1), (2, 1, 9)])
def test_loss_population(kind, B, K, P):
    """Population code (Sec. V): class k pools neurons kP .. kP+P-1."""
    rng = np.random.default_rng(B * K + P)
    c = rng.integers(0, 3, (B, K * P)).astype(np.float32)
    loss = torch.empty(4, dtype=torch.float32, device=DEV)
    g = torch.empty((B, K * P), dtype=torch.float32, device=DEV)
    ws = _ws(snn.snn_loss_workspace_bytes(kind, B, K))
    if kind == snn.LOSS_CE_COUNT:
        y = rng.integers(0, K, B).astype(np.int32)
        snn.snn_loss(kind, B, K, P, _t(c), _t(y), None, loss, g, ws)
        L, rg = oracle.loss_ce(c, y, P)
    else:
        y = rng.uniform(0, 2 * P, (B, K)).astype(np.float32)
        snn.snn_loss(kind, B, K, P, _t(c), None, _t(y), loss, g, ws)
        L, rg = oracle.loss_mse(c, y, P)
    assert abs(_np(loss)[0] - L) <= 1e-6 * max(1.0, abs(L))
    assert_close(_np(g), rg, 1e-5, what="dL/dcounts")


# ---------------------------------------------------------------------------
# whole training steps
# ---------------------------------------------------------------------------
_TORCH_GRAD = {snn.F32: torch.float32, snn.BF16: torch.bfloat16, snn.F16: torch.float16}


def _saved_from_oracle(d, f, v, x_dev):
    """The forward-to-backward state of snn_layer_bwd built from the oracle's
    forward, at the offsets the library reports: the oracle's currents, the
    checkpoints of a forward scan of those currents (bit-identical to the
    oracle's scan, as the neuron-stage checks show), and, for conv layers,
    the oracle's pool selection.  Returns (saved, currents, checkpoints)."""
    saved = torch.zeros(snn.snn_layer_saved_bytes(d), dtype=torch.uint8, device=DEV)
    cur, ck, pool = snn.saved_parts(d, saved)
    I = _t(np.ascontiguousarray(f["I"], np.float32).reshape(d.T, d.B, d.n_out))
    if cur is not None:
        cur.copy_(I)
    else:
        cur = x_dev  # the layer's input holds its currents
    if pool is not None:
        pool.copy_(_t(np.asarray(f["arg"]).astype(np.uint8).reshape(pool.shape)))
    spk = _spk_buf(d)
    snn.snn_neuron_fwd(d, cur, v, spk, ck, None)
    return saved, cur, ck


def _layer_input(spec, f, d):
    """The oracle's input to a layer in the type the layer's descriptor reads
    (currents fp32; spikes as bytes or as fp16 0/1)."""
    x = np.asarray(f["x"])
    if spec["kind"] == "none":
        return _t(x.astype(np.float32))
    return _t(x.astype(np.float16) if d.in_dtype == snn.F16 else x.astype(np.uint8))


def _spk_buf(d):
    return torch.empty((d.T, d.B, d.n_out), dtype=torch.float16 if d.out_dtype == snn.F16
                       else torch.uint8, device=DEV)


def _check_step_stagewise(wl, inp, reset=snn.RESET_DETACHED, flags=0, tol=1e-3):
    """Each layer's GPU calls, fed the oracle's inputs to that layer, against
    the oracle's outputs.  The oracle runs its own chain and sees no GPU value.

    forward:  synapse stage (currents within tol); neuron stage on the
              oracle's fp32 currents (spikes, membrane, counts bit-identical);
              the whole layer call (spikes equal up to legal flips);
    loss:     on the oracle's spike counts;
    backward: neuron stage on the oracle's membrane and upstream gradient;
              synapse stage on the oracle's dL/dI (rounded on the host to the
              gradient operand type) and pool selection; the whole layer call
              on the oracle's saved state."""
    rs = reset == snn.RESET_SURROGATE
    T, B = wl.T, wl.B
    n = len(wl.layers)
    P = wl.pop
    L, fwds, bwds = oracle.net_step(wl.layers, inp["params"], inp["x"], wl.loss,
                                    labels=inp.get("labels"), targets=inp.get("targets"),
                                    slope=wl.slope, reset_surrogate=rs, pop=P)
    net = snn.Network(wl, inp["params"], device=DEV, reset_grad=reset, flags=flags)
    xs = []
    for li, spec in enumerate(wl.layers):
        f, d = fwds[li], net.descs[li]
        x_dev = _layer_input(spec, f, d)
        xs.append(x_dev)
        if spec["kind"] != "none":
            cur = torch.empty((T, B, d.n_out), dtype=torch.float32, device=DEV)
            arg = torch.empty(T * B * d.n_out, dtype=torch.uint8, device=DEV) \
                if spec["kind"] == "conv" else None
            snn.snn_synapse_fwd(d, x_dev, net.W[li], net.b[li], cur, arg, net.ws)
            assert_close(_np(cur), f["I"].reshape(T, B, -1), tol, what=f"L{li} currents")
        spk = _spk_buf(d)
        u = torch.empty((T, B, d.n_out), dtype=torch.float32, device=DEV)
        cnt = torch.empty((B, d.n_out), dtype=torch.float32, device=DEV)
        snn.snn_neuron_fwd(d, _t(f["I"].reshape(T, B, -1)), net.v[li], spk, snn.ckpt_buffer(d),
                           cnt, u_out=u)
        np.testing.assert_array_equal(_np(spk), f["z"].reshape(T, B, -1), err_msg=f"L{li} spikes")
        np.testing.assert_array_equal(_np(u), f["u"].reshape(T, B, -1), err_msg=f"L{li} membrane")
        np.testing.assert_array_equal(_np(cnt), f["counts"].reshape(B, -1))
        saved = torch.empty(snn.snn_layer_saved_bytes(d), dtype=torch.uint8, device=DEV)
        snn.snn_layer_fwd(d, x_dev, net.W[li], net.b[li], net.v[li], spk, saved, cnt, net.ws)
        assert_spikes(_np(spk), f["z"].reshape(T, B, -1), f["u"].reshape(T, B, -1), spec["thr"],
                      what=f"L{li} layer call")
    # loss on the oracle's counts
    c_o = np.asarray(fwds[-1]["counts"], np.float32).reshape(B, -1)
    K = c_o.shape[1] // P
    loss = torch.empty(4, dtype=torch.float32, device=DEV)
    gc = torch.empty(c_o.shape, dtype=torch.float32, device=DEV)
    if wl.loss == "ce":
        snn.snn_loss(snn.LOSS_CE_COUNT, B, K, P, _t(c_o), _t(inp["labels"]), None, loss, gc,
                     net.ws)
        L2, gc_o = oracle.loss_ce(c_o, inp["labels"], P)
    else:
        snn.snn_loss(snn.LOSS_MSE_COUNT, B, K, P, _t(c_o), None, _t(inp["targets"]), loss, gc,
                     net.ws)
        L2, gc_o = oracle.loss_mse(c_o, inp["targets"], P)
    assert abs(_np(loss)[0] - L2) <= 1e-5 * max(1.0, abs(L2))
    assert_close(_np(gc), gc_o, 1e-5, what="dL/dcounts")
    g = gc_o
    for li in range(n - 1, -1, -1):
        spec, f, r, d = wl.layers[li], fwds[li], bwds[li], net.descs[li]
        bcast = li == n - 1
        kind = snn.GRAD_BCAST if bcast else snn.GRAD_FULL
        g_dev = _t(np.asarray(g, np.float32).reshape((B, d.n_out) if bcast else (T, B, d.n_out)))
        dI_o = r["dI"].reshape(T, B, -1)
        saved, cur_s, ck_s = _saved_from_oracle(d, f, net.v[li], xs[li])
        vv = net.v[li]
        gv = None if vv is None else torch.empty_like(vv)
        gv2 = None if vv is None else torch.empty_like(vv)
        if spec["kind"] == "none":
            dcur = torch.empty((T, B, d.n_out), dtype=torch.float32, device=DEV)
            snn.snn_neuron_bwd(d, kind, g_dev, vv, cur_s, ck_s, dcur, None, gv, net.ws)
            assert_close(_np(dcur), dI_o, tol, what="dL/dI")
            snn.snn_layer_bwd(d, kind, g_dev, xs[li], None, vv, saved, None, None, gv2, dcur,
                              net.ws)
            assert_close(_np(dcur), dI_o, tol, what="layer dL/dI")
            if vv is not None:
                assert_close(_np(gv), r["dv"], tol, what="neuron-stage dL/dv")
                assert_close(_np(gv2), r["dv"], tol, what="dL/dv")
            g = r["dx"]
            continue
        half = d.grad_dtype != snn.F32
        gdt = _TORCH_GRAD[d.grad_dtype]
        scaled = d.grad_dtype == snn.F16
        sc = torch.empty(4, dtype=torch.float32, device=DEV) if scaled else None
        dcur = torch.empty((T, B, d.n_out), dtype=gdt, device=DEV)
        gb = torch.empty_like(net.gb[li])
        snn.snn_neuron_bwd(d, kind, g_dev, vv, cur_s, ck_s, dcur, gb, gv, net.ws, dcur_scale=sc)
        S = float(_np(sc)[0]) if scaled else 1.0
        assert_close(_np(dcur.float()) / S, dI_o, 2e-2 if half else tol, what=f"L{li} dL/dI")
        assert_close(_np(gb), r["db"], tol, what=f"L{li} neuron-stage db")
        if vv is not None:
            assert_close(_np(gv), r["dv"], tol, what=f"L{li} neuron-stage dL/dv")
        if net.fold[li]:
            # the readout's dx computed inside this scan, from the oracle's
            # dL/dI of the readout (rounded to its gradient type) and weights
            up = net.descs[li + 1]
            dup = torch.from_numpy(np.ascontiguousarray(bwds[li + 1]["dI"], np.float32)
                                   .reshape(T, B, -1)).to(_TORCH_GRAD[up.grad_dtype]).to(DEV)
            fold_g = (dup, net.W[li + 1])
            dI_r, db_r, dW_r, bW_f = dI_o, r["db"], r["dW"], None
            if half:
                # the oracle's chain from the dL/dI the fold reads (bf16)
                assert spec["kind"] == "dense" and vv is None
                g_r = (dup.float().cpu().numpy().astype(np.float64).reshape(T * B, -1)
                       @ np.asarray(inp["params"][li + 1][0], np.float64)).reshape(T, B, -1)
                dI_r = oracle.scan_bwd(f["u"].reshape(T, B, -1), g_r, spec["neuron"],
                                       spec["beta"], spec["thr"], wl.slope,
                                       spec.get("alpha", 0.0), rs)
                db_r = dI_r.reshape(T * B, -1).sum(axis=0)
                xin_ = np.asarray(f["x"], np.float64).reshape(T * B, -1)
                dW_r, _, _ = oracle.dense_bwd(dI_r.reshape(T * B, -1), xin_, inp["params"][li][0],
                                              want_db=False, want_dx=False)
                # dL/dI handed to the contraction in bf16
                bW_f = 2.0 ** -8 * (np.abs(dI_r.reshape(T * B, -1)).T @ np.abs(xin_))
            dcur_f, gb_f = torch.empty_like(dcur), torch.empty_like(gb)
            gv_f = None if vv is None else torch.empty_like(vv)
            snn.snn_neuron_bwd(d, snn.GRAD_FOLD, fold_g, vv, cur_s, ck_s, dcur_f, gb_f, gv_f,
                               net.ws,
                               dcur_scale=sc)
            S = float(_np(sc)[0]) if scaled else 1.0
            assert_close(_np(dcur_f.float()) / S, dI_r, 2e-2 if half else tol,
                         what=f"L{li} folded dL/dI")
            assert_close(_np(gb_f), db_r, tol, what=f"L{li} folded db")
            if vv is not None:
                assert_close(_np(gv_f), r["dv"], tol, what=f"L{li} folded dL/dv")
            gW_f = torch.empty_like(net.gW[li])
            snn.snn_layer_bwd(d, snn.GRAD_FOLD, fold_g, xs[li], net.W[li], vv, saved, gW_f,
                              gb_f, gv_f, None, net.ws)
            assert_close(_np(gW_f), dW_r, tol, what=f"L{li} folded layer dW", abs_bound=bW_f)
        # synapse stage on the oracle's dL/dI, rounded on the host
        W = inp["params"][li][0]
        xin = np.asarray(f["x"], np.float64)
        gW = torch.empty_like(net.gW[li])
        gx = torch.empty((T, B, d.n_in), dtype=torch.float32, device=DEV) if li > 0 else None
        S = pow2_scale(dI_o) if scaled else 1.0
        dI_h = torch.from_numpy(np.ascontiguousarray(dI_o * S, np.float32)).to(gdt)
        sc_h = _t(np.full(4, S, np.float32)) if scaled else None
        arg_dev = _t(np.asarray(f["arg"]).astype(np.uint8)) if spec["kind"] == "conv" else None
        snn.snn_synapse_bwd(d, dI_h.to(DEV), arg_dev, xs[li], net.W[li], gW, gx, net.ws,
                            dcur_scale=sc_h)
        if half:
            dI_used = dI_h.float().numpy().astype(np.float64).reshape(T * B, -1) / S
            sW, _, sx = oracle.dense_bwd(dI_used, xin.reshape(T * B, -1), W, want_db=False,
                                         want_dx=li > 0)
        else:
            sW, sx = r["dW"], r["dx"]
        assert_close(_np(gW), sW, tol, what=f"L{li} synapse-stage dW")
        if li > 0:
            assert_close(_np(gx).reshape(sx.shape), sx, tol, what=f"L{li} synapse-stage dx")
        # the whole layer call on the oracle's saved state and upstream gradient
        gW2, gb2 = torch.empty_like(gW), torch.empty_like(gb)
        gx2 = torch.empty((T, B, d.n_in), dtype=torch.float32, device=DEV) if li > 0 else None
        snn.snn_layer_bwd(d, kind, g_dev, xs[li], net.W[li], vv, saved, gW2, gb2, gv2, gx2,
                          net.ws)
        if vv is not None:
            assert_close(_np(gv2), r["dv"], tol, what=f"L{li} dL/dv")
        bW = bx = None
        if half:
            # dL/dI handed to the contractions in bf16: a-priori rounding bound
            aI = np.abs(dI_o.reshape(T * B, -1))
            bW = 2.0 ** -8 * (aI.T @ np.abs(xin.reshape(T * B, -1)))
            bx = 2.0 ** -8 * (aI @ np.abs(W).astype(np.float64)) if li > 0 else None
        assert_close(_np(gW2), r["dW"], tol, what=f"L{li} dW", abs_bound=bW)
        assert_close(_np(gb2), r["db"], tol, what=f"L{li} db")
        if li > 0:
            assert_close(_np(gx2).reshape(T * B, -1), r["dx"].reshape(T * B, -1), tol,
                         what=f"L{li} dx", abs_bound=bx)
        g = r["dx"]


@pytest.mark.parametrize("name", ["dsnn_leaky_t25_b32", "dsnn_synaptic_t50_b256", "csnn_t25_b128",
                                  "dsnn_rleaky_t25_b128", "pop_dsnn_t1_b128", "pop_csnn_t1_b128"])
@pytest.mark.parametrize("path", list(PATHS))
def test_step_full_size_stagewise(name, path):
    wl = wls.get(name)
    inp = wls.make_inputs(wl, seed=0)
    _check_step_stagewise(wl, inp, flags=PATHS[path])


@pytest.mark.parametrize("name,T,B,width", [("dsnn_synaptic_t50_b256", 20, 16, 200),
                                            ("dsnn_leaky_t25_b32", 25, 8, 300),
                                            ("scan_wide_t1000_b64", 60, 4, 1000),
                                            ("csnn_t25_b128", 6, 4, None),
                                            ("dsnn_half_t100_b512", 12, 8, 320),
                                            ("dsnn_rleaky_t25_b128", 15, 6, 130),
                                            ("pop_dsnn_t1_b128", 1, 16, 200),
                                            ("pop_csnn_t1_b128", 1, 5, None)])
@pytest.mark.parametrize("reset", [snn.RESET_DETACHED, snn.RESET_SURROGATE])
@pytest.mark.parametrize("path", list(PATHS))
def test_step_scaled_stagewise(name, T, B, width, reset, path):
    wl = wls.scaled(wls.get(name), T=T, B=B, width=width)
    inp = wls.make_inputs(wl, seed=1)
    _check_step_stagewise(wl, inp, reset, PATHS[path], tol=2e-2 if wl.dtype == "f16" else 1e-3)
    # the whole step through the network: stage calls give the same bytes as
    # the layer calls
    net = snn.Network(wl, inp["params"], device=DEV, reset_grad=reset, flags=PATHS[path])
    lab = _t(inp["labels"]) if wl.loss == "ce" else None
    tgt = _t(inp["targets"]) if wl.loss == "mse" else None
    x = _t(inp["x"])
    net.step(x, labels=lab, targets=tgt)
    snap = [_np(t).copy() for t in net.gW if t is not None] + [_np(net.loss).copy()]
    net.step_stages(x, labels=lab, targets=tgt)
    snap2 = [_np(t) for t in net.gW if t is not None] + [_np(net.loss)]
    for a, b in zip(snap, snap2):
        np.testing.assert_array_equal(a, b)
    # the readout's dx folded into the scan below, or contracted and read back
    if any(net.fold):
        plain = snn.Network(wl, inp["params"], device=DEV, reset_grad=reset, flags=PATHS[path],
                            fold=False)
        plain.step(x, labels=lab, targets=tgt)
        bounds = [None] * len(wl.layers)
        if wl.dtype == "f16":
            # The two paths bound the fp16 dL/dI scale differently (the folded
            # upstream gradient by its factors, the read one by its max), so
            # values below fp16's normal range round differently, and a bf16
            # dL/dI further down may round the other way: each path's weight
            # gradient is within the a-priori bf16 bound 2^-8 sum|terms| of the
            # exact one, so the two differ by at most 2^-7 sum|terms| (terms
            # from the oracle's chain on the same inputs).
            _, fw, bw = oracle.net_step(wl.layers, inp["params"], inp["x"], wl.loss,
                                        labels=inp.get("labels"), targets=inp.get("targets"),
                                        slope=wl.slope, reset_surrogate=reset == snn.RESET_SURROGATE)
            for li in range(len(wl.layers)):
                aI = np.abs(bw[li]["dI"].reshape(wl.T * wl.B, -1))
                ax = np.abs(np.asarray(fw[li]["x"], np.float64).reshape(wl.T * wl.B, -1))
                bounds[li] = 2.0 ** -7 * (aI.T @ ax)
        for li, (a, b) in enumerate(zip(net.gW, plain.gW)):
            if a is not None:
                assert_close(_np(a), _np(b), 2e-2 if wl.dtype == "f16" else 1e-3,
                             what=f"L{li} dW folded vs not", abs_bound=bounds[li])


@pytest.mark.parametrize("reset", [snn.RESET_DETACHED, snn.RESET_SURROGATE])
def test_step_recurrent_conv_stagewise(reset):
    """Recurrent neurons (eq. 7) behind the convolutional synapses: one
    recurrent weight per pooled output neuron."""
    wl = wls.scaled(wls.get("csnn_t25_b128"), T=6, B=3)
    for spec in wl.layers:
        spec["neuron"] = "rleaky"
    inp = wls.make_inputs(wl, seed=4)
    assert all(len(p) == 3 for p in inp["params"])
    _check_step_stagewise(wl, inp, reset)


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
        snn.snn_layer_fwd(d, x, W, None, None, spk, saved, counts, _ws(256))
        if B > 0:
            assert (_np(counts) == 0).all()
        gW = torch.full((8, 16), 3.0, device=DEV)
        gb = torch.full((8,), 3.0, device=DEV)
        g = torch.zeros(256, dtype=torch.float32, device=DEV)
        snn.snn_layer_bwd(d, snn.GRAD_BCAST, g, x, W, None, saved, gW, gb, None, None,
                          _ws(snn.snn_layer_workspace_bytes(d)))
        assert (_np(gW) == 0).all() and (_np(gb) == 0).all()

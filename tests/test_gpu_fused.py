"""The whole step of a two-layer dense SNN as one launch (snn_fused_step),
against the oracle's chain on the same inputs.

Its contractions take the same exact products as the layer calls and
accumulate them in fp32 in their own order, so a current may differ from the
oracle's fp64 value rounded to fp32 by a few units in the last place, and a
membrane within that distance of the threshold may spike on one side only (a
legal flip, as for the layer calls).  The hidden spikes must agree up to legal
flips; where none occurs, the readout's counts equal the oracle's bit for bit,
the loss agrees to fp64 rounding and the gradients within the layer calls'
tolerance."""
import numpy as np
import pytest
import torch

import oracle
import paper_2211_10725_amd as snn
from paper_2211_10725_amd import workloads as wls
from tests.parity import assert_close, spike_flips

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _t(a, dtype=None):
    t = torch.as_tensor(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(DEV)


def _np(t):
    return t.detach().cpu().numpy()


def _case(name, T=None, B=None, width=None, neuron=None, pop=None, loss=None, seed=1):
    # scaled() returns a copy, so the changes below stay local
    wl = wls.scaled(wls.get(name), T=T, B=B, width=width)
    if neuron is not None:
        for spec in wl.layers:
            spec["neuron"] = neuron
            spec.setdefault("alpha", 0.9)
    if pop is not None:
        wl.pop = pop
        wl.layers[-1]["n_out"] = 5 * pop
    if loss is not None:
        wl.loss = loss
    return wl, wls.make_inputs(wl, seed=seed)


def _run(wl, inp, reset=snn.RESET_DETACHED):
    net = snn.Network(wl, inp["params"], device=DEV, reset_grad=reset)
    assert net.fdesc is not None
    lab = _t(inp["labels"]) if wl.loss == "ce" else None
    tgt = _t(inp["targets"]) if wl.loss == "mse" else None
    net.step_fused(_t(inp["x"]), labels=lab, targets=tgt)
    torch.cuda.synchronize()
    assert int(_np(net.fstatus)[0]) == 0
    return net


def _check(wl, inp, net, reset=snn.RESET_DETACHED):
    """Returns the number of flipped hidden columns (0: fully compared)."""
    L, fwds, bwds = oracle.net_step(wl.layers, inp["params"], inp["x"].astype(np.float64),
                                    wl.loss, labels=inp.get("labels"),
                                    targets=inp.get("targets"), slope=wl.slope,
                                    reset_surrogate=reset == snn.RESET_SURROGATE,
                                    pop=getattr(wl, "pop", 1))
    agree, roots, illegal = spike_flips(_np(net.spk[0]), fwds[0]["z"], fwds[0]["u"],
                                        wl.layers[0]["thr"])
    assert illegal == 0 and agree >= 0.9999, (agree, roots, illegal)
    if roots:
        return roots
    np.testing.assert_array_equal(_np(net.counts), fwds[-1]["counts"].reshape(wl.B, -1))
    assert abs(float(_np(net.loss)[0]) - L) <= 1e-5 * max(1.0, abs(L))
    for li in range(2):
        assert_close(_np(net.gW[li]), bwds[li]["dW"], 1e-3, what=f"L{li} dW")
        assert_close(_np(net.gb[li]), bwds[li]["db"], 1e-3, what=f"L{li} db")
    return 0


@pytest.mark.parametrize("B", [8, 32])
def test_fused_step_dense_leaky(B):
    """784-1000-10 Leaky, T = 25 (the small-batch sweep's net) at B = 8, 32;
    seeds until one step is compared in full (flips are rare)."""
    compared = 0
    for seed in range(1, 6):
        wl, inp = _case("dsnn_leaky_t25_b32", B=B, seed=seed)
        compared += _check(wl, inp, _run(wl, inp)) == 0
    assert compared >= 1


@pytest.mark.parametrize("reset", [snn.RESET_DETACHED, snn.RESET_SURROGATE])
def test_fused_step_synaptic_ragged(reset):
    """Current-based neurons, both reset readings; 304 hidden neurons (a
    partial last workgroup), 7 steps, 5 samples."""
    wl, inp = _case("dsnn_synaptic_t50_b256", T=7, B=5, width=304, seed=4)
    assert _check(wl, inp, _run(wl, inp, reset), reset) == 0


def test_fused_step_population_mse():
    """Population readout (5 classes of 3 neurons) and the MSE loss."""
    wl, inp = _case("dsnn_leaky_t25_b32", T=9, B=6, pop=3, loss="mse", seed=5)
    assert _check(wl, inp, _run(wl, inp)) == 0


def test_fused_step_repeatable():
    """Two launches give the same bytes (the barrier counters are clear after
    each)."""
    wl, inp = _case("dsnn_leaky_t25_b32", B=8, seed=6)
    net = _run(wl, inp)
    a = [_np(t).copy() for t in net.gW + net.gb + [net.loss, net.counts, net.spk[0]]]
    net.step_fused(_t(inp["x"]), labels=_t(inp["labels"]))
    b = [_np(t) for t in net.gW + net.gb + [net.loss, net.counts, net.spk[0]]]
    for p, q in zip(a, b):
        np.testing.assert_array_equal(p, q)


def test_fused_step_gives_up_and_recovers():
    """A wait limit of one poll: a workgroup that reaches a barrier before the
    others gives up, the step reports status 1 and still ends; the next step
    with the default limit completes and is right."""
    wl, inp = _case("dsnn_leaky_t25_b32", B=8, seed=7)
    net = snn.Network(wl, inp["params"], device=DEV)
    lab = _t(inp["labels"])
    x = _t(inp["x"])
    fd = net.fdesc
    tight = snn.fused_desc(fd.hidden, fd.readout, fd.loss_kind, fd.pop, wait_limit=1)
    seen = []
    for _ in range(3):
        snn.snn_fused_step(tight, x, net.W[0], net.b[0], net.W[1], net.b[1], lab, None, net.loss,
                           net.counts, net.gW[0], net.gb[0], net.gW[1], net.gb[1], net.fstatus,
                           net.fws, spk_hidden=net.spk[0])
        torch.cuda.synchronize()
        seen.append(int(_np(net.fstatus)[0]))
    assert set(seen) <= {0, 1} and 1 in seen, seen
    net.step_fused(x, labels=lab)
    torch.cuda.synchronize()
    assert int(_np(net.fstatus)[0]) == 0
    _check(wl, inp, net)


def test_fused_step_refusals():
    """Networks the fused step does not run are refused before any launch."""
    wl, inp = _case("dsnn_leaky_t25_b32", B=8)
    net = snn.Network(wl, inp["params"], device=DEV)
    fd = net.fdesc
    bad = snn.fused_desc(fd.hidden.copy(), fd.readout.copy(), fd.loss_kind, fd.pop)
    bad.readout.n_out = 17
    assert snn.snn_fused_step_check(bad) != 0
    bad = snn.fused_desc(fd.hidden.copy(), fd.readout.copy(), fd.loss_kind, fd.pop)
    bad.hidden.neuron = snn.RLEAKY
    assert snn.snn_fused_step_check(bad) != 0
    bad = snn.fused_desc(fd.hidden.copy(), fd.readout.copy(), fd.loss_kind, fd.pop)
    bad.readout.n_in = 999
    assert snn.snn_fused_step_check(bad) != 0
    big = snn.fused_desc(fd.hidden.copy(), fd.readout.copy(), fd.loss_kind, fd.pop)
    big.hidden.B = big.readout.B = 4096  # state of T*B rows no longer fits in LDS
    assert snn.snn_fused_step_check(big) != 0
    assert snn.snn_fused_step_workspace_bytes(big) == 0
    long = snn.fused_desc(fd.hidden.copy(), fd.readout.copy(), fd.loss_kind, fd.pop)
    long.hidden.T = long.readout.T = 33  # the readout's rows are two 16-step blocks
    assert snn.snn_fused_step_check(long) != 0
    odd = snn.fused_desc(fd.hidden.copy(), fd.readout.copy(), fd.loss_kind, fd.pop)
    odd.hidden.n_in = 783  # inputs in whole runs of 8
    assert snn.snn_fused_step_check(odd) != 0

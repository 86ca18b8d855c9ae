"""Named workloads and seeded synthetic inputs.

This module holds no arithmetic of the method: it only describes network
shapes and neuron hyper-parameters and draws seeded random tensors.  Both the
GPU path and the CPU oracle receive the arrays it produces, so parity tests
compare the two on identical bytes.

The inputs stand in for the MNIST-shaped workloads the paper measures on
(Sec. III-C: 28x28 images rate-coded into spike trains, T = 25 by default):
per sample and feature a firing rate r ~ U[0, rate_hi] is drawn, then
x[t,b,f] ~ Bernoulli(r[b,f]) independently for every time step.  Weights
and biases follow PyTorch's default layer init, U(-1/sqrt(fan_in),
+1/sqrt(fan_in)); the recurrent weights of recurrent neurons (eq. 7), one
per neuron, are drawn U(-rec_hi, rec_hi).  Labels are uniform over the 10
classes.
"""
from __future__ import annotations

import copy
import math
from dataclasses import dataclass, field

import numpy as np


@dataclass
class Workload:
    name: str
    T: int
    B: int
    layers: list            # list of layer spec dicts (plain data)
    loss: str = "ce"        # 'ce' (labels) or 'mse' (targets)
    rate_hi: float = 1.0    # input firing rate ~ U[0, rate_hi]
    slope: float = 25.0     # fast-sigmoid surrogate slope k
    dtype: str = "f32"      # operand dtype of the synaptic contraction
    input: str = "spikes"   # 'spikes' (Bernoulli) or 'currents' (normal)
    current_mean: float = 0.0
    current_std: float = 1.0
    target_hi: float = 50.0
    rec_hi: float = 0.5     # recurrent weights of 'rleaky' layers ~ U(-rec_hi, rec_hi)
    pop: int = 1            # output neurons per class (population code when > 1)
    description: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def in_shape(self):
        s = self.layers[0]
        if s["kind"] == "dense":
            return (s["n_in"],)
        if s["kind"] == "conv":
            return (s["c_in"], s["h"], s["w"])
        return (s["n"],)

    @property
    def classes(self):
        """Number of classes: output neurons divided by the population size."""
        return self.out_features // self.pop

    @property
    def out_features(self):
        s = self.layers[-1]
        if s["kind"] == "dense":
            return s["n_out"]
        if s["kind"] == "none":
            return s["n"]
        k = s.get("k", 5)
        return s["c_out"] * ((s["h"] - k + 1) // 2) * ((s["w"] - k + 1) // 2)


def _dense(n_in, n_out, neuron, beta, alpha=0.0, thr=1.0):
    return dict(kind="dense", n_in=n_in, n_out=n_out, neuron=neuron, beta=beta,
                alpha=alpha, thr=thr)


def _conv(c_in, h, w, c_out, neuron, beta, alpha=0.0, thr=1.0, k=5):
    return dict(kind="conv", c_in=c_in, h=h, w=w, c_out=c_out, k=k, neuron=neuron,
                beta=beta, alpha=alpha, thr=thr)


WORKLOADS = {
    # Dense 784-1000-10 (Table I), Leaky beta 0.95, T 25, batch 32, fp32.
    "dsnn_leaky_t25_b32": Workload(
        "dsnn_leaky_t25_b32", T=25, B=32,
        layers=[_dense(784, 1000, "leaky", 0.95), _dense(1000, 10, "leaky", 0.95)],
        description="Dense SNN 784-1000-10, Leaky beta=0.95, T=25, B=32, fp32"),
    # Same net with current-based neurons (eqs. 5-6), alpha 0.9 beta 0.8.
    "dsnn_synaptic_t50_b256": Workload(
        "dsnn_synaptic_t50_b256", T=50, B=256,
        layers=[_dense(784, 1000, "synaptic", 0.8, 0.9),
                _dense(1000, 10, "synaptic", 0.8, 0.9)],
        description="Dense SNN 784-1000-10, Synaptic alpha=0.9 beta=0.8, T=50, B=256, fp32"),
    # Conv 5C12-MP2-5C64-MP2-10 (Table I) on 1x28x28, Leaky beta 0.5.
    "csnn_t25_b128": Workload(
        "csnn_t25_b128", T=25, B=128,
        layers=[_conv(1, 28, 28, 12, "leaky", 0.5), _conv(12, 12, 12, 64, "leaky", 0.5),
                _dense(1024, 10, "leaky", 0.5)],
        description="Conv SNN 5C12-MP2-5C64-MP2-10, Leaky beta=0.5, T=25, B=128, fp32"),
    # The dense net with recurrent neurons (eq. 7, one recurrent weight per
    # neuron), Leaky beta 0.95 as the default dense net.
    "dsnn_rleaky_t25_b128": Workload(
        "dsnn_rleaky_t25_b128", T=25, B=128,
        layers=[_dense(784, 1000, "rleaky", 0.95), _dense(1000, 10, "rleaky", 0.95)],
        description="Dense SNN 784-1000-10, recurrent Leaky (eq. 7) beta=0.95, one recurrent "
                    "weight per neuron ~U(-0.5,0.5), T=25, B=128, fp32"),
    # Population codes (Sec. V): one time step, 500 output neurons pooled as
    # 50 per class, on CIFAR-10-shaped 3x32x32 rate-coded inputs; the DSNN
    # with the wider input layer and the CSNN with the wider terminal layer.
    "pop_dsnn_t1_b128": Workload(
        "pop_dsnn_t1_b128", T=1, B=128, pop=50,
        layers=[_dense(3072, 1000, "leaky", 0.95), _dense(1000, 500, "leaky", 0.95)],
        description="Population-coded dense SNN 3072-1000-500 (50 neurons per class), "
                    "Leaky beta=0.95, T=1, B=128, fp32"),
    "pop_csnn_t1_b128": Workload(
        "pop_csnn_t1_b128", T=1, B=128, pop=50,
        layers=[_conv(3, 32, 32, 12, "leaky", 0.5), _conv(12, 14, 14, 64, "leaky", 0.5),
                _dense(1600, 500, "leaky", 0.5)],
        description="Population-coded conv SNN 3x32x32-5C12-MP2-5C64-MP2-500 (50 neurons "
                    "per class), Leaky beta=0.5, T=1, B=128, fp32"),
    # Deeper, wider dense net in half precision operands.
    "dsnn_half_t100_b512": Workload(
        "dsnn_half_t100_b512", T=100, B=512, rate_hi=0.5, dtype="f16",
        layers=[_dense(784, 4096, "leaky", 0.9), _dense(4096, 4096, "leaky", 0.9),
                _dense(4096, 10, "leaky", 0.9)],
        description="Dense SNN 784-4096-4096-10, Leaky beta=0.9, T=100, B=512, "
                    "fp16 operands, fp32 accumulate and state"),
    # One wide Leaky layer driven directly by currents (scan only), MSE loss.
    "scan_wide_t1000_b64": Workload(
        "scan_wide_t1000_b64", T=1000, B=64, loss="mse", input="currents",
        current_mean=0.3, current_std=0.5, target_hi=50.0,
        layers=[dict(kind="none", n=65536, neuron="leaky", beta=0.95, alpha=0.0, thr=1.0)],
        description="Single Leaky layer, 65536 neurons, currents N(0.3,0.5) "
                    "[T=1000,B=64], MSE on spike counts vs U[0,50]"),
}


def get(name: str) -> Workload:
    return copy.deepcopy(WORKLOADS[name])


def scaled(wl: Workload, T=None, B=None, width=None) -> Workload:
    """Same distributions and neuron parameters at a smaller size.  ``width``
    replaces hidden widths of dense nets (and N of a scan-only layer)."""
    w = copy.deepcopy(wl)
    if T is not None:
        w.T = T
    if B is not None:
        w.B = B
    if width is not None:
        for i, s in enumerate(w.layers):
            if s["kind"] == "none":
                s["n"] = width
            elif s["kind"] == "dense":
                if i < len(w.layers) - 1:
                    s["n_out"] = width
                if i > 0 and w.layers[i - 1]["kind"] == "dense":
                    s["n_in"] = w.layers[i - 1]["n_out"]
    w.name = f"{wl.name}@T{w.T}B{w.B}" + (f"W{width}" if width else "")
    return w


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _n_out(s) -> int:
    """Output neurons per sample of a layer spec."""
    if s["kind"] == "dense":
        return s["n_out"]
    if s["kind"] == "none":
        return s["n"]
    k = s.get("k", 5)
    return s["c_out"] * ((s["h"] - k + 1) // 2) * ((s["w"] - k + 1) // 2)


def init_params(wl: Workload, seed: int):
    """Per layer (W, b) as float32 arrays, U(-1/sqrt(fan_in), 1/sqrt(fan_in)),
    and (W, b, v) for recurrent layers, v [n_out] ~ U(-rec_hi, rec_hi).
    For fp16 workloads the weights are rounded once to fp16 (round to
    nearest even) and returned as float32 holding those fp16 values, so both
    sides see identical operands."""
    rng = _rng(10_000 + seed)
    params = []
    for s in wl.layers:
        if s["kind"] == "none":
            W = b = None
        else:
            if s["kind"] == "dense":
                shape, fan_in, n_b = (s["n_out"], s["n_in"]), s["n_in"], s["n_out"]
            else:
                k = s.get("k", 5)
                shape, fan_in, n_b = (s["c_out"], s["c_in"], k, k), s["c_in"] * k * k, s["c_out"]
            bound = 1.0 / math.sqrt(fan_in)
            W = rng.uniform(-bound, bound, size=shape).astype(np.float32)
            b = rng.uniform(-bound, bound, size=n_b).astype(np.float32)
            if wl.dtype == "f16":
                W = W.astype(np.float16).astype(np.float32)
                b = b.astype(np.float16).astype(np.float32)
        if s["neuron"] == "rleaky":
            v = rng.uniform(-wl.rec_hi, wl.rec_hi, size=_n_out(s)).astype(np.float32)
            params.append((W, b, v))
        else:
            params.append((W, b))
    return params


def spike_input(wl: Workload, seed: int) -> np.ndarray:
    """Bernoulli rate-coded spike trains, uint8 [T, B, *in_shape]."""
    rng = _rng(seed)
    feat = int(np.prod(wl.in_shape))
    rate = rng.uniform(0.0, wl.rate_hi, size=(wl.B, feat))
    x = np.empty((wl.T, wl.B, feat), np.uint8)
    for t in range(wl.T):
        x[t] = rng.random((wl.B, feat)) < rate
    return x.reshape((wl.T, wl.B) + tuple(wl.in_shape))


def current_input(wl: Workload, seed: int) -> np.ndarray:
    """Normal input currents, float32 [T, B, N] (host; small sizes only)."""
    rng = _rng(seed)
    n = wl.layers[0]["n"]
    return rng.normal(wl.current_mean, wl.current_std, size=(wl.T, wl.B, n)).astype(np.float32)


def labels(wl: Workload, seed: int) -> np.ndarray:
    return _rng(20_000 + seed).integers(0, wl.classes, size=wl.B).astype(np.int32)


def targets(wl: Workload, seed: int) -> np.ndarray:
    return _rng(30_000 + seed).uniform(0.0, wl.target_hi,
                                       size=(wl.B, wl.classes)).astype(np.float32)


def make_inputs(wl: Workload, seed: int = 0) -> dict:
    """All host inputs of one step: x, params, labels or targets."""
    d = {"params": init_params(wl, seed)}
    d["x"] = spike_input(wl, seed) if wl.input == "spikes" else current_input(wl, seed)
    if wl.loss == "ce":
        d["labels"] = labels(wl, seed)
    else:
        d["targets"] = targets(wl, seed)
    return d


def device_currents(wl: Workload, seed: int, device="cuda"):
    """Normal currents generated directly in device memory with torch's
    seeded generator (for sizes too large to draw on the host)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    n = wl.layers[0]["n"]
    x = torch.empty((wl.T, wl.B, n), dtype=torch.float32, device=device)
    x.normal_(wl.current_mean, wl.current_std, generator=g)
    return x


def device_spikes(wl: Workload, seed: int, device="cuda"):
    """Bernoulli rate-coded spikes generated in device memory (uint8)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    feat = int(np.prod(wl.in_shape))
    rate = torch.rand((wl.B, feat), generator=g, device=device) * wl.rate_hi
    x = torch.empty((wl.T, wl.B, feat), dtype=torch.uint8, device=device)
    for t in range(wl.T):
        x[t] = (torch.rand((wl.B, feat), generator=g, device=device) < rate).to(torch.uint8)
    return x.reshape((wl.T, wl.B) + tuple(wl.in_shape))

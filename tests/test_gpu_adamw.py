"""Fused AdamW update on the GPU (snn_adamw) against the oracle's AdamW step.

Parameters, gradients and moments are seeded; both sides read the same fp32
values (the hyper-parameters too: the ABI takes them as fp32).  The GPU keeps
fp32 state, the oracle computes in double: moments agree to fp32 rounding,
and the parameter's change agrees within 1e-3 of the change or within the
rounding of the stored fp32 parameter.
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

# ragged sizes around the 4-element lanes and 4096-element chunks, an empty one
SIZES = [1, 3, 4, 4095, 4096, 4097, 0, 100003, 1 << 20]


def _np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def _state(n, rng, step):
    p = rng.normal(0, 1, n).astype(np.float32)
    g = rng.normal(0, 0.05, n).astype(np.float32)
    if step == 1:
        m = np.zeros(n, np.float32)
        v = np.zeros(n, np.float32)
    else:
        m = rng.normal(0, 0.01, n).astype(np.float32)
        v = (rng.random(n) * 1e-3).astype(np.float32)
    return p, g, m, v


def _orc(p, g, m, v, step, hp):
    """The oracle's step with the hyper-parameters the library receives: the
    ABI takes them as fp32, so both sides use the fp32 values."""
    f = lambda x: float(np.float32(x))  # noqa: E731
    return oracle.adamw(p, g, m, v, step, f(hp["lr"]), (f(hp["betas"][0]), f(hp["betas"][1])),
                        f(hp["eps"]), f(hp["weight_decay"]))


def _check_param(p_gpu, p_old, p_ref, what, steps=1):
    """The change of the parameter within 1e-3, or within the fp32 rounding
    of the stored parameter: per step the decay factor, the decayed value and
    the result are each rounded once (3 x 2^-24 of |theta| per step)."""
    d_gpu = p_gpu.astype(np.float64) - p_old.astype(np.float64)
    d_ref = p_ref - p_old.astype(np.float64)
    mag = np.maximum(np.abs(p_ref), np.abs(p_old.astype(np.float64)))
    assert_close(d_gpu, d_ref, 1e-3, what=what, abs_bound=3 * steps * 2.0 ** -24 * mag + 1e-30)


def _run(sizes, seed, step, hp, half=False):
    rng = np.random.default_rng(seed)
    host = [_state(n, rng, step) for n in sizes]
    dev = []
    for p, g, m, v in host:
        h = torch.empty(len(p), dtype=torch.float16, device=DEV) if half else None
        dev.append(tuple(torch.as_tensor(a).to(DEV) for a in (p, g, m, v)) + (h,))
    snn.snn_adamw(dev, step, **hp)
    for (p, g, m, v), (pd, gd, md, vd, hd) in zip(host, dev):
        pr, mr, vr = _orc(p, g, m, v, step, hp)
        n = len(p)
        assert_close(_np(md), mr, 1e-5, what=f"m (n={n})")
        assert_close(_np(vd), vr, 1e-5, what=f"v (n={n})")
        _check_param(_np(pd), p, pr, f"param (n={n})")
        np.testing.assert_array_equal(_np(gd), g)       # the gradient is read only
        if hd is not None:
            # the fp16 copy is the updated fp32 param rounded to nearest even
            np.testing.assert_array_equal(_np(hd), _np(pd).astype(np.float16))


HP = dict(lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=1e-2)


@pytest.mark.parametrize("step", [1, 2, 7, 1000])
@pytest.mark.parametrize("wd", [0.0, 1e-2])
def test_adamw_matches_oracle(step, wd):
    _run(SIZES, seed=step, step=step, hp=dict(HP, weight_decay=wd))


def test_adamw_other_hyperparameters_and_half_copy():
    hp = dict(lr=3e-2, betas=(0.8, 0.95), eps=1e-6, weight_decay=0.1)
    _run([5, 4099, 70001], seed=11, step=3, hp=hp, half=True)


def test_adamw_more_tensors_than_one_launch():
    """37 tensors (16 per launch), empty ones in between."""
    sizes = [(i * 977) % 5003 if i % 5 else 0 for i in range(37)]
    _run(sizes, seed=5, step=4, hp=HP)


def test_adamw_repeated_steps_track_the_oracle():
    rng = np.random.default_rng(9)
    n = 50001
    p, _, m, v = _state(n, rng, 1)
    pd, md, vd = (torch.as_tensor(a).to(DEV) for a in (p, m, v))
    pr, mr, vr = p.astype(np.float64), m.astype(np.float64), v.astype(np.float64)
    for t in range(1, 9):
        g = rng.normal(0, 0.05, n).astype(np.float32)
        snn.snn_adamw([(pd, torch.as_tensor(g).to(DEV), md, vd, None)], t, **HP)
        pr, mr, vr = _orc(pr, g, mr, vr, t, HP)
    _check_param(_np(pd), p, pr, "param after 8 steps", steps=8)
    assert_close(_np(md), mr, 1e-4, what="m after 8 steps")
    assert_close(_np(vd), vr, 1e-4, what="v after 8 steps")


def test_adamw_full_size_half_net():
    """Every parameter of the 784-4096-4096-10 fp16 net in one call (20 M
    values): fp32 masters updated, fp16 weights rewritten from them."""
    wl = wls.get("dsnn_half_t100_b512")
    params = wls.init_params(wl, 0)
    net = snn.Network(wl, params, device=DEV)
    net.init_adamw(**HP)
    rng = np.random.default_rng(4)
    grads = []
    for (master, G, m, v, half) in net.opt_tensors:
        g = rng.normal(0, 1e-3, G.shape).astype(np.float32)
        G.copy_(torch.as_tensor(g))
        grads.append(g)
    net.update()
    for li, (W, b) in enumerate(params):
        for k, (P0, ti) in enumerate(((W, 2 * li), (b, 2 * li + 1))):
            master, G, m, v, half = net.opt_tensors[ti]
            pr, mr, vr = _orc(P0, grads[ti], np.zeros(P0.shape), np.zeros(P0.shape), 1, HP)
            _check_param(_np(master), P0, pr, f"L{li} {'W' if k == 0 else 'b'}")
            assert_close(_np(m), mr, 1e-5, what="m")
            if half is not None:
                np.testing.assert_array_equal(_np(half), _np(master).astype(np.float16))
    # the network's fp16 weights are the ones updated
    assert net.W[0].dtype == torch.float16
    np.testing.assert_array_equal(_np(net.W[0]), _np(net.opt_tensors[0][0]).astype(np.float16))

"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: values
worked by hand from the paper's equations (tests/golden/), closed forms of
the linear recurrence, finite differences of a smooth network, library
routines in float64, exact rational arithmetic, and invariants.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from tests.conftest import GOLDEN


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------------------
# P2: hand-worked T=4 traces (eqs. 3-6)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("case", _golden("hand_tables_t4.json")["cases"], ids=lambda c: c["name"])
def test_hand_tables(case):
    I = np.array(case["I"], np.float32).reshape(4, 1)
    z, u, cnt = oracle.scan_fwd(I, case["neuron"], case["beta"], 1.0, case["alpha"])
    assert z.ravel().tolist() == case["z"]
    assert cnt[0] == case["count"]
    if case["exact"]:
        assert u.ravel().tolist() == case["u"]
    else:
        np.testing.assert_allclose(u.ravel(), case["u"], rtol=1e-6)


# ---------------------------------------------------------------------------
# P3: hand-worked BPTT gradients with the fast-sigmoid surrogate (eqs. 8-9)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("case", _golden("hand_gradients_t4.json")["cases"], ids=lambda c: c["name"])
def test_hand_gradients(case):
    traces = {c["name"]: c for c in _golden("hand_tables_t4.json")["cases"]}
    tr = traces[case["trace"]]
    I = np.array(tr["I"], np.float32).reshape(4, 1)
    z, u, _ = oracle.scan_fwd(I, tr["neuron"], tr["beta"], 1.0, tr["alpha"])
    g = np.ones((4, 1))
    dI = oracle.scan_bwd(u, g, tr["neuron"], tr["beta"], 1.0, case["slope"], tr["alpha"],
                         case["reset_surrogate"])
    np.testing.assert_allclose(dI.ravel(), case["dI"], rtol=0, atol=1.5e-7)
    # the surrogate values themselves: with T=1 and g=1, dI equals s exactly
    for t, s in enumerate(case["s"]):
        d1 = oracle.scan_bwd(u[t:t + 1], np.ones((1, 1)), "leaky", tr["beta"], 1.0,
                             case["slope"])
        assert d1[0, 0] == pytest.approx(float(Fraction(s)), rel=1e-15)


def test_slope_one_is_eq9():
    """With slope k = 1 the surrogate is exactly eq. (9): 1/(1+|thr-u|)^2."""
    u = np.array([[0.0], [0.5], [1.0], [1.25], [3.0], [-2.0]], np.float32)
    for t in range(u.shape[0]):
        d = oracle.scan_bwd(u[t:t + 1], np.ones((1, 1)), "leaky", 0.9, 1.0, 1.0)
        expect = [1 / 4.0, 1 / 2.25, 1.0, 1 / 1.5625, 1 / 9.0, 1 / 16.0][t]
        assert d[0, 0] == pytest.approx(expect, rel=1e-15)


# ---------------------------------------------------------------------------
# P1: closed-form LIF response to a constant current
# ---------------------------------------------------------------------------
def _closed_form_train(I, beta, thr, T):
    """Spike steps (1-based) and membrane from the between-spike closed form."""
    spikes, us = [], []
    t_last, u_last = 0, None
    for t in range(1, T + 1):
        if u_last is None:
            u = I * (1 - beta ** t) / (1 - beta)
        else:
            k = t - t_last
            u = beta ** (k - 1) * (beta * u_last + I - thr) + I * (1 - beta ** (k - 1)) / (1 - beta)
        us.append(u)
        if u > thr:
            spikes.append(t)
            t_last, u_last = t, u
    return spikes, np.array(us)


@pytest.mark.parametrize("case", [c for c in _golden("closed_form_lif.json")["cases"]
                                  if c["t1"] is not None], ids=lambda c: f"I{c['I']}b{c['beta']}")
def test_closed_form_first_spike_and_train(case):
    T = 200
    I, beta, thr = case["I"], case["beta"], case["thr"]
    Iv = np.full((T, 1), I, np.float32)
    z, u, cnt = oracle.scan_fwd(Iv, "leaky", beta, thr)
    got = (np.nonzero(z.ravel())[0] + 1).tolist()
    assert got[0] == case["t1"]
    assert u[case["t1"] - 1, 0] == pytest.approx(case["u_t1"], rel=2e-6)
    if "u_t1_minus_1" in case:
        assert u[case["t1"] - 2, 0] == pytest.approx(case["u_t1_minus_1"], rel=2e-6)
    # whole train against the closed form (in double); margins are far above
    # the fp32 rounding of the recurrence, so the spike steps must agree
    spikes, us = _closed_form_train(I, beta, thr, T)
    assert np.min(np.abs(us - thr)) > 1e-4
    assert got == spikes
    np.testing.assert_allclose(u.ravel(), us, rtol=0, atol=2e-5)
    if "period" in case:
        assert all(b - a == case["period"] for a, b in zip(got, got[1:]))
        assert cnt[0] == len(range(case["t1"], T + 1, case["period"]))


def test_silent_boundary():
    """I/(1-beta) == thr: membrane tends to thr, reaches exactly 1.0 in fp32
    and never fires because eq. (3) needs u > thr."""
    T = 60
    z, u, cnt = oracle.scan_fwd(np.full((T, 1), 0.5, np.float32), "leaky", 0.5, 1.0)
    assert cnt[0] == 0 and z.sum() == 0
    assert u[T - 1, 0] == 1.0
    for t in range(1, 25):  # exact dyadic values 1 - 2^-t while representable
        assert u[t - 1, 0] == 1.0 - 2.0 ** -t


def test_no_spike_without_drive_reaching_threshold():
    """Firing condition I/(1-beta) > thr (geometric-series limit)."""
    for I, beta, fires in [(0.049, 0.95, False), (0.051, 0.95, True), (0.29, 0.7, False),
                           (0.31, 0.7, True)]:
        _, _, cnt = oracle.scan_fwd(np.full((2000, 1), I, np.float32), "leaky", beta, 1.0)
        assert (cnt[0] > 0) == fires


# ---------------------------------------------------------------------------
# fp32 recurrence: the decay-plus-input term is one correctly rounded fma
# ---------------------------------------------------------------------------
def _round_f32(q: Fraction) -> float:
    """Round an exact rational to the nearest fp32, ties to even."""
    f = np.float32(float(q))
    cands = {float(f), float(np.nextafter(f, np.float32(np.inf))),
             float(np.nextafter(f, np.float32(-np.inf)))}
    best = min(cands, key=lambda c: (abs(Fraction(c) - q),
                                     int(np.float32(c).view(np.uint32)) & 1))
    return best


def test_fused_multiply_add_rounding():
    rng = np.random.default_rng(7)
    n = 4000
    beta = np.float32(0.95)
    I1 = rng.uniform(-1.0, 1.0, n).astype(np.float32)   # u_1 = I1 <= thr: no spike
    I2 = rng.uniform(-1.0, 1.0, n).astype(np.float32)
    I = np.stack([I1, I2])
    _, u, _ = oracle.scan_fwd(I, "leaky", float(beta), 1.0)
    for j in range(n):
        exact = Fraction(float(beta)) * Fraction(float(I1[j])) + Fraction(float(I2[j]))
        assert float(u[1, j]) == _round_f32(exact)


# ---------------------------------------------------------------------------
# P5: special cases reducing to textbook / library routines
# ---------------------------------------------------------------------------
def test_dense_matches_numpy_float64():
    rng = np.random.default_rng(1)
    M, n_in, n_out = 37, 53, 29
    x = (rng.random((M, n_in)) < 0.4).astype(np.float64)
    W = rng.uniform(-1, 1, (n_out, n_in))
    b = rng.uniform(-1, 1, n_out)
    np.testing.assert_allclose(oracle.dense_fwd(x, W, b), x @ W.T + b, rtol=1e-13, atol=1e-13)
    dI = rng.normal(size=(M, n_out))
    dW, db, dx = oracle.dense_bwd(dI, x, W)
    np.testing.assert_allclose(dW, dI.T @ x, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, dI.sum(0), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dx, dI @ W, rtol=1e-12, atol=1e-12)


def test_conv_pool_match_torch_float64():
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    rng = np.random.default_rng(2)
    x = (rng.random((3, 2, 12, 11)) < 0.5).astype(np.float64)
    w = rng.normal(size=(4, 2, 5, 5))
    b = rng.normal(size=4)
    y = oracle.conv_fwd(x, w, b)
    xt = torch.tensor(x, requires_grad=True)
    wt = torch.tensor(w, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    yt = F.conv2d(xt, wt, bt)
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-12, atol=1e-12)
    # pooling of the oracle's own conv output, forward and backward
    yl = torch.tensor(y, requires_grad=True)
    pt = F.max_pool2d(yl, 2)
    p, arg = oracle.maxpool2_fwd(y)
    np.testing.assert_array_equal(p, pt.detach().numpy())
    dp = rng.normal(size=p.shape)
    pt.backward(torch.tensor(dp))
    dy = oracle.maxpool2_bwd(dp, arg, y.shape[2], y.shape[3])
    np.testing.assert_array_equal(dy, yl.grad.numpy())
    # conv backward for that upstream gradient
    gx, gw, gb = torch.autograd.grad(yt, (xt, wt, bt), torch.tensor(dy))
    dw, db, dx = oracle.conv_bwd(dy, x, w)
    np.testing.assert_allclose(dw, gw.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(db, gb.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dx, gx.numpy(), rtol=1e-11, atol=1e-11)


def test_maxpool_ties_first_maximum():
    x = np.array([[[[1.0, 3.0], [3.0, 0.0]]],
                  [[[2.0, 2.0], [2.0, 2.0]]],
                  [[[0.0, 1.0], [5.0, 5.0]]]])
    p, arg = oracle.maxpool2_fwd(x)
    assert p.ravel().tolist() == [3.0, 2.0, 5.0]
    assert arg.ravel().tolist() == [1, 0, 2]


def test_ce_loss_values_and_library():
    torch = pytest.importorskip("torch")
    L, g = oracle.loss_ce(np.full((4, 10), 7.0), np.array([0, 3, 9, 5]))
    assert L == pytest.approx(math.log(10.0), rel=1e-15)
    c = np.zeros((1, 10))
    c[0, 0] = 3.0
    L, g = oracle.loss_ce(c, np.array([0]))
    assert L == pytest.approx(0.3702410, abs=5e-8)
    assert g[0, 0] + 1.0 == pytest.approx(0.6905679, abs=5e-8)
    rng = np.random.default_rng(3)
    counts = rng.integers(0, 26, (17, 10)).astype(np.float64)
    y = rng.integers(0, 10, 17)
    L, g = oracle.loss_ce(counts, y)
    ct = torch.tensor(counts, requires_grad=True)
    Lt = torch.nn.functional.cross_entropy(ct, torch.tensor(y, dtype=torch.long))
    Lt.backward()
    assert L == pytest.approx(Lt.item(), rel=1e-14)
    np.testing.assert_allclose(g, ct.grad.numpy(), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(g.sum(1), 0.0, atol=1e-15)


def test_mse_loss_library():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(4)
    c = rng.integers(0, 100, (5, 33)).astype(np.float64)
    y = rng.uniform(0, 50, (5, 33))
    L, g = oracle.loss_mse(c, y)
    ct = torch.tensor(c, requires_grad=True)
    Lt = torch.nn.functional.mse_loss(ct, torch.tensor(y))
    Lt.backward()
    assert L == pytest.approx(Lt.item(), rel=1e-14)
    np.testing.assert_allclose(g, ct.grad.numpy(), rtol=1e-13, atol=1e-16)


def test_synaptic_alpha_zero_is_leaky():
    rng = np.random.default_rng(5)
    I = rng.normal(0.3, 0.6, (40, 64)).astype(np.float32)
    a = oracle.scan_fwd(I, "leaky", 0.9, 1.0)
    b = oracle.scan_fwd(I, "synaptic", 0.9, 1.0, alpha=0.0)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    g = rng.normal(size=(40, 64))
    for rs in (False, True):
        da = oracle.scan_bwd(a[1], g, "leaky", 0.9, 1.0, 25.0, reset_surrogate=rs)
        db = oracle.scan_bwd(a[1], g, "synaptic", 0.9, 1.0, 25.0, alpha=0.0, reset_surrogate=rs)
        np.testing.assert_array_equal(da, db)


def test_beta_zero_detached_has_no_carry():
    """beta = 0 with a detached reset: nothing flows back in time, so
    dI_t = g_t * s_t and dW is a single matrix product (g*s)^T x."""
    rng = np.random.default_rng(6)
    T, B, n_in, n_out = 6, 3, 7, 5
    x = (rng.random((T, B, n_in)) < 0.5).astype(np.float64)
    W = rng.normal(0, 1, (n_out, n_in))
    spec = dict(kind="dense", n_in=n_in, n_out=n_out, neuron="leaky", beta=0.0, thr=1.0)
    f = oracle.layer_fwd(spec, x, W, None)
    g = rng.normal(size=(T, B, n_out))
    r = oracle.layer_bwd(spec, f, g, W, slope=25.0)
    # the same quantity evaluated one step at a time (T = 1 scans)
    per_step = np.stack([oracle.scan_bwd(f["u"][t:t + 1], g[t:t + 1], "leaky", 0.0)[0]
                         for t in range(T)])
    np.testing.assert_allclose(r["dI"], per_step, rtol=0, atol=0)
    np.testing.assert_allclose(r["dW"], per_step.reshape(T * B, n_out).T @ x.reshape(T * B, n_in),
                               rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# P6: invariants
# ---------------------------------------------------------------------------
def test_invariants():
    rng = np.random.default_rng(8)
    T, C = 30, 500
    I = rng.normal(0.2, 1.0, (T, C)).astype(np.float32)
    for neuron, alpha, beta in [("leaky", 0.0, 0.9), ("synaptic", 0.6, 0.8)]:
        z, u, cnt = oracle.scan_fwd(I, neuron, beta, 1.0, alpha)
        assert set(np.unique(z).tolist()) <= {0, 1}
        assert np.array_equal(cnt, z.sum(0).astype(np.float32))
        assert cnt.min() >= 0 and cnt.max() <= T
        # z_t is exactly the threshold test on the saved membrane
        assert np.array_equal(z, (u > 1.0).astype(np.uint8))
        if neuron == "leaky":
            bound = (np.abs(I).max() + 1.0) / (1 - beta)
            assert np.abs(u).max() <= bound
        g1, g2 = rng.normal(size=(T, C)), rng.normal(size=(T, C))
        for rs in (False, True):
            d1 = oracle.scan_bwd(u, g1, neuron, beta, 1.0, 25.0, alpha, rs)
            d2 = oracle.scan_bwd(u, g2, neuron, beta, 1.0, 25.0, alpha, rs)
            d12 = oracle.scan_bwd(u, g1 + g2, neuron, beta, 1.0, 25.0, alpha, rs)
            np.testing.assert_allclose(d12, d1 + d2, rtol=1e-12, atol=1e-12)
            d0 = oracle.scan_bwd(u, np.zeros((T, C)), neuron, beta, 1.0, 25.0, alpha, rs)
            assert not d0.any()
    # surrogate in (0, 1]
    s = oracle.scan_bwd(I[:1].copy(), np.ones((1, C)), "leaky", 0.9, 1.0, 25.0)
    assert (s > 0).all() and (s <= 1).all()
    # no weights, no bias: no spikes
    spec = dict(kind="dense", n_in=20, n_out=7, neuron="leaky", beta=0.9, thr=1.0)
    x = (rng.random((10, 4, 20)) < 0.5).astype(np.float64)
    f = oracle.layer_fwd(spec, x, np.zeros((7, 20)), np.zeros(7))
    assert f["z"].sum() == 0


def test_broadcast_gradient_equals_repeated():
    rng = np.random.default_rng(9)
    T, C = 12, 40
    u = rng.normal(1.0, 0.3, (T, C)).astype(np.float32)
    g = rng.normal(size=C)
    for neuron in ("leaky", "synaptic"):
        a = oracle.scan_bwd(u, g, neuron, 0.8, 1.0, 25.0, 0.7)
        b = oracle.scan_bwd(u, np.broadcast_to(g, (T, C)).copy(), neuron, 0.8, 1.0, 25.0, 0.7)
        np.testing.assert_array_equal(a, b)


# ---------------------------------------------------------------------------
# P4: finite differences on tiny smooth networks (same slope both passes)
# ---------------------------------------------------------------------------
def _fd_check(layers, params, x, labels, reset_surrogate, slope=25.0, eps=1e-6):
    L, fwds, bwds = oracle.net_step(layers, params, x, "ce", labels=labels, smooth=True,
                                    slope=slope, reset_surrogate=reset_surrogate)
    if not reset_surrogate:
        margin = min(np.abs(f["u"] - s["thr"]).min() for f, s in zip(fwds, layers))
        if margin < 1e-4:
            return None

    def loss_of(ps):
        h = x
        for spec, prm in zip(layers, ps):
            f = oracle.layer_fwd(spec, h, prm[0], prm[1], smooth=True, slope=slope,
                                 reset_surrogate=reset_surrogate,
                                 v=prm[2] if len(prm) > 2 else None)
            h = f["z"]
        B = x.shape[1]
        return oracle.loss_ce(f["counts"].reshape(B, -1), labels)[0]

    worst = 0.0
    for li in range(len(params)):
        names = ("dW", "db", "dv")[:len(params[li])]
        for pi, grad in enumerate(bwds[li][k] for k in names):
            P = params[li][pi]
            flat = P.reshape(-1)          # a view: edits change params in place
            fd = np.zeros(P.size)
            for j in range(P.size):
                keep = flat[j]
                flat[j] = keep + eps
                lp = loss_of(params)
                flat[j] = keep - eps
                lm = loss_of(params)
                flat[j] = keep
                fd[j] = (lp - lm) / (2 * eps)
            an = np.asarray(grad).ravel()
            err = np.abs(fd - an) / (np.abs(an) + 1e-8)
            worst = max(worst, float(err.max()))
            assert np.all(np.abs(fd - an) <= 1e-5 * np.abs(an) + 1e-8), (li, pi, fd, an)
    return worst


@pytest.mark.parametrize("neuron,alpha", [("leaky", 0.0), ("synaptic", 0.6)])
@pytest.mark.parametrize("reset_surrogate", [False, True])
def test_finite_differences_dense(neuron, alpha, reset_surrogate):
    T, B = 5, 2
    for seed in range(50):
        rng = np.random.default_rng(100 + seed)
        layers = [dict(kind="dense", n_in=3, n_out=4, neuron=neuron, beta=0.8, alpha=alpha, thr=1.0),
                  dict(kind="dense", n_in=4, n_out=2, neuron=neuron, beta=0.8, alpha=alpha, thr=1.0)]
        params = [(rng.uniform(-1, 1.5, (4, 3)), rng.uniform(-0.2, 0.8, 4)),
                  (rng.uniform(-1, 1.5, (2, 4)), rng.uniform(-0.2, 0.8, 2))]
        x = (rng.random((T, B, 3)) < 0.6).astype(np.float64)
        y = rng.integers(0, 2, B)
        if _fd_check(layers, params, x, y, reset_surrogate) is not None:
            return
    pytest.fail("no seed with a reset margin above 1e-4")


@pytest.mark.parametrize("reset_surrogate", [False, True])
def test_finite_differences_conv(reset_surrogate):
    T, B = 5, 2
    for seed in range(50):
        rng = np.random.default_rng(300 + seed)
        layers = [dict(kind="conv", c_in=1, h=6, w=6, c_out=2, k=3, neuron="leaky", beta=0.7,
                       thr=1.0),
                  dict(kind="dense", n_in=8, n_out=2, neuron="leaky", beta=0.7, thr=1.0)]
        params = [(rng.uniform(-0.5, 0.8, (2, 1, 3, 3)), rng.uniform(-0.2, 0.5, 2)),
                  (rng.uniform(-1, 1.5, (2, 8)), rng.uniform(-0.2, 0.8, 2))]
        x = (rng.random((T, B, 1, 6, 6)) < 0.6).astype(np.float64)
        y = rng.integers(0, 2, B)
        # the pool's selection must not switch under +-eps: require a clear winner
        yy = oracle.conv_fwd(x.reshape(T * B, 1, 6, 6), params[0][0], params[0][1])
        win = np.sort(yy.reshape(T * B, 2, 2, 2, 2, 2).transpose(0, 1, 2, 4, 3, 5)
                      .reshape(T * B, 2, 2, 2, 4), axis=-1)
        if (win[..., -1] - win[..., -2]).min() < 1e-3:
            continue
        if _fd_check(layers, params, x, y, reset_surrogate) is not None:
            return
    pytest.fail("no seed with clear pool winners and reset margins")


# ---------------------------------------------------------------------------
# P6: recurrent leaky neuron (eq. 7), one recurrent weight per neuron
# ---------------------------------------------------------------------------
_RL = _golden("hand_rleaky_t4.json")
_RL_TRACES = {t["name"]: t for t in _RL["traces"]}


@pytest.mark.parametrize("tr", _RL["traces"], ids=lambda t: t["name"])
def test_rleaky_hand_traces(tr):
    I = np.array(tr["I"], np.float32).reshape(4, 1)
    z, u, cnt = oracle.scan_fwd(I, "rleaky", tr["beta"], tr["thr"], v=[tr["v"]])
    np.testing.assert_array_equal(u[:, 0], np.array(tr["u"], np.float32))
    np.testing.assert_array_equal(z[:, 0], tr["z"])
    assert cnt[0] == sum(tr["z"])


@pytest.mark.parametrize("case", _RL["gradients"], ids=lambda c: c["name"])
def test_rleaky_hand_gradients(case):
    tr = _RL_TRACES[case["trace"]]
    u = np.array(tr["u"]).reshape(4, 1)
    g = np.array(case["g"], np.float64).reshape(4, 1)
    dI, dv = oracle.scan_bwd_rleaky(u, g, tr["beta"], tr["thr"], case["slope"], [tr["v"]],
                                    case["reset_surrogate"])
    want = np.array([float(Fraction(q)) for q in case["dI"]])
    np.testing.assert_allclose(dI[:, 0], want, rtol=1e-14, atol=1e-15)
    assert abs(dv[0] - float(Fraction(case["dv"]))) <= 1e-14


def _rand_currents(seed, T=40, B=3, N=7):
    rng = np.random.default_rng(seed)
    return rng.normal(0.4, 0.8, (T, B, N)).astype(np.float32), rng


def test_rleaky_zero_weight_is_leaky():
    """v = 0 leaves only the reset of eq. (4): same spikes and membrane bit for bit,
    and the same BPTT gradients for either reading of the reset."""
    I, rng = _rand_currents(11)
    v = np.zeros(I.shape[-1], np.float32)
    zr, ur, cr = oracle.scan_fwd(I, "rleaky", 0.9, 1.0, v=v)
    zl, ul, cl = oracle.scan_fwd(I, "leaky", 0.9, 1.0)
    np.testing.assert_array_equal(zr, zl)
    np.testing.assert_array_equal(ur, ul)
    np.testing.assert_array_equal(cr, cl)
    assert zr.any() and not zr.all()
    g = rng.normal(0, 1, I.shape)
    for rs in (False, True):
        dr, _ = oracle.scan_bwd_rleaky(ur, g, 0.9, 1.0, 25.0, v, rs)
        dl = oracle.scan_bwd(ul, g, "leaky", 0.9, 1.0, 25.0, 0.0, rs)
        np.testing.assert_allclose(dr, dl, rtol=1e-13, atol=1e-300)


def test_rleaky_threshold_weight_is_integrator():
    """v = thr cancels the reset: u_t = sum_j beta^(t-j) I_j, the plain linear
    recurrence (computed here as a triangular matrix product in float64).  With
    beta = 1/2 and currents on a coarse dyadic grid the fp32 scan is exact."""
    T, C = 24, 64
    rng = np.random.default_rng(5)
    I = (rng.integers(-16, 48, (T, C)) / 16.0).astype(np.float32)
    z, u, _ = oracle.scan_fwd(I, "rleaky", 0.5, 1.0, v=np.ones(C, np.float32))
    t = np.arange(T)
    Lmat = np.where(t[:, None] >= t[None, :], 0.5 ** (t[:, None] - t[None, :]).clip(0), 0.0)
    np.testing.assert_allclose(u, Lmat @ I.astype(np.float64), rtol=1e-6, atol=1e-6)
    np.testing.assert_array_equal(z, (Lmat @ I.astype(np.float64)) > 1.0)
    assert z.any()
    # backward: with the reset-through-surrogate reading the carry is exactly beta,
    # the detached Leaky recursion; dL/dv is then sum_{t>=1} lam_t z_{t-1}
    g = rng.normal(0, 1, (T, C))
    dr, dv = oracle.scan_bwd_rleaky(u, g, 0.5, 1.0, 25.0, np.ones(C), True)
    dl = oracle.scan_bwd(u, g, "leaky", 0.5, 1.0, 25.0, 0.0, False)
    np.testing.assert_allclose(dr, dl, rtol=1e-13)
    np.testing.assert_allclose(dv, (dl[1:] * z[:-1]).sum(axis=0), rtol=1e-12)


def test_rleaky_weight_shared_across_batch():
    """Column c is neuron c % N: the batch rows use the same v and dL/dv sums them."""
    I, rng = _rand_currents(12)
    T, B, N = I.shape
    v = rng.uniform(-1, 1.5, N).astype(np.float32)
    z, u, _ = oracle.scan_fwd(I, "rleaky", 0.85, 1.0, v=v)
    g = rng.normal(0, 1, (B, N))
    dI, dv = oracle.scan_bwd_rleaky(u, g, 0.85, 1.0, 25.0, v)
    for b in range(B):
        zb, ub, _ = oracle.scan_fwd(I[:, b], "rleaky", 0.85, 1.0, v=v)
        np.testing.assert_array_equal(zb, z[:, b])
        np.testing.assert_array_equal(ub, u[:, b])
    parts = [oracle.scan_bwd_rleaky(u[:, b], g[b], 0.85, 1.0, 25.0, v)[1] for b in range(B)]
    np.testing.assert_allclose(dv, np.sum(parts, axis=0), rtol=1e-12)


@pytest.mark.parametrize("reset_surrogate", [False, True])
def test_finite_differences_rleaky(reset_surrogate):
    """Smooth dense 3-4-2 net with recurrent hidden and output layers: dW, db and
    the recurrent weights' gradient dv against central differences."""
    T, B = 6, 2
    for seed in range(50):
        rng = np.random.default_rng(500 + seed)
        layers = [dict(kind="dense", n_in=3, n_out=4, neuron="rleaky", beta=0.8, thr=1.0),
                  dict(kind="dense", n_in=4, n_out=2, neuron="rleaky", beta=0.8, thr=1.0)]
        params = [(rng.uniform(-1, 1.5, (4, 3)), rng.uniform(-0.2, 0.8, 4),
                   rng.uniform(-0.8, 1.2, 4)),
                  (rng.uniform(-1, 1.5, (2, 4)), rng.uniform(-0.2, 0.8, 2),
                   rng.uniform(-0.8, 1.2, 2))]
        x = (rng.random((T, B, 3)) < 0.6).astype(np.float64)
        y = rng.integers(0, 2, B)
        if _fd_check(layers, params, x, y, reset_surrogate) is not None:
            return
    pytest.fail("no seed with a reset margin above 1e-4")


# ---------------------------------------------------------------------------
# P7: the AdamW weight update (Sec. IV trains every network with AdamW)
# ---------------------------------------------------------------------------
def test_adamw_first_step_closed_form():
    """From zero moments the bias-corrected estimates are g and g^2, so the
    first step is theta (1 - lr wd) - lr g / (|g| + eps)."""
    rng = np.random.default_rng(1)
    th0 = rng.normal(0, 1, 1000)
    g = rng.normal(0, 0.1, 1000)
    lr, wd, eps = 3e-3, 0.05, 1e-8
    th, m, v = oracle.adamw(th0, g, np.zeros(1000), np.zeros(1000), 1, lr, (0.9, 0.999), eps, wd)
    np.testing.assert_allclose(th, th0 * (1 - lr * wd) - lr * g / (np.abs(g) + eps), rtol=1e-13,
                               atol=1e-16)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-14)
    np.testing.assert_allclose(v, 0.001 * g * g, rtol=1e-12)


def test_adamw_constant_gradient_moves_linearly():
    """A constant gradient keeps mhat = g and vhat = g^2 at every step: without
    weight decay each step moves theta by lr g / (|g| + eps)."""
    th0 = np.array([0.5, -1.0, 2.0, 0.0])
    g = np.array([0.2, -0.05, 1e-3, 3.0])
    th, m, v = th0, np.zeros(4), np.zeros(4)
    lr, eps = 1e-2, 1e-8
    for t in range(1, 31):
        th, m, v = oracle.adamw(th, g, m, v, t, lr, (0.9, 0.999), eps, 0.0)
    np.testing.assert_allclose(th, th0 - 30 * lr * g / (np.abs(g) + eps), rtol=1e-11)


def test_adamw_decay_is_decoupled():
    """With a zero gradient only the decay acts: theta (1 - lr wd), exactly."""
    th0 = np.linspace(-3, 3, 101)
    th, m, v = oracle.adamw(th0, np.zeros(101), np.zeros(101), np.zeros(101), 1, 1e-3,
                            (0.9, 0.999), 1e-8, 0.1)
    np.testing.assert_array_equal(th, th0 - 1e-3 * 0.1 * th0)
    assert not m.any() and not v.any()


def test_adamw_matches_torch_float64():
    """torch.optim.AdamW in float64 over several steps (a library special case)."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(2)
    th0 = rng.normal(0, 1, (37, 11))
    grads = [rng.normal(0, 0.3, th0.shape) for _ in range(6)]
    P = torch.nn.Parameter(torch.tensor(th0, dtype=torch.float64))
    opt = torch.optim.AdamW([P], lr=2e-3, betas=(0.85, 0.995), eps=1e-7, weight_decay=0.02)
    th, m, v = th0, np.zeros_like(th0), np.zeros_like(th0)
    for t, g in enumerate(grads, start=1):
        P.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        th, m, v = oracle.adamw(th, g, m, v, t, 2e-3, (0.85, 0.995), 1e-7, 0.02)
    np.testing.assert_allclose(th, P.detach().numpy(), rtol=1e-12, atol=1e-15)
    st = opt.state[P]
    np.testing.assert_allclose(m, st["exp_avg"].numpy(), rtol=1e-12, atol=1e-18)
    np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-12, atol=1e-20)


def test_adamw_scale_invariance():
    """With eps = 0 the update does not depend on the gradient's scale."""
    rng = np.random.default_rng(3)
    th0 = rng.normal(0, 1, 50)
    gs = [rng.normal(0, 1, 50) for _ in range(4)]
    runs = []
    for c in (1.0, 1e-3, 256.0):
        th, m, v = th0, np.zeros(50), np.zeros(50)
        for t, g in enumerate(gs, start=1):
            th, m, v = oracle.adamw(th, c * g, m, v, t, 1e-2, (0.9, 0.99), 0.0, 0.01)
        runs.append(th)
    np.testing.assert_allclose(runs[1], runs[0], rtol=1e-12)
    np.testing.assert_allclose(runs[2], runs[0], rtol=1e-12)


# ---------------------------------------------------------------------------
# P8: population code (Sec. V): P output neurons per class, counts pooled
# ---------------------------------------------------------------------------
def test_population_of_one_is_the_plain_readout():
    rng = np.random.default_rng(4)
    c = rng.integers(0, 26, (9, 10)).astype(np.float64)
    y = rng.integers(0, 10, 9)
    L1, g1 = oracle.loss_ce(c, y, P=1)
    L0, g0 = oracle.loss_ce(c, y)
    assert L1 == L0 and np.array_equal(g1, g0)


def test_population_uniform_counts_closed_form():
    """Equal pooled counts: L = log K and every neuron of class k gets
    (1/K - [k = y]) / B."""
    B, K, P = 4, 10, 50
    c = np.ones((B, K * P))
    y = np.array([0, 3, 9, 3])
    L, g = oracle.loss_ce(c, y, P)
    assert abs(L - math.log(K)) < 1e-14
    want = np.repeat((np.full((B, K), 1.0 / K) - np.eye(K)[y]) / B, P, axis=1)
    np.testing.assert_allclose(g, want, rtol=1e-14, atol=1e-17)


def test_population_pooling_by_hand():
    """Two classes of three neurons: class counts 1+0+2 = 3 and 4+1+0 = 5;
    MSE against targets (2, 7): L = ((3-2)^2 + (5-7)^2) / 2 = 2.5, and each
    neuron of class k receives 2 (c_k - y_k) / 2."""
    c = np.array([[1.0, 0.0, 2.0, 4.0, 1.0, 0.0]])
    L, g = oracle.loss_mse(c, np.array([[2.0, 7.0]]), P=3)
    assert L == 2.5
    np.testing.assert_array_equal(g, [[1.0, 1.0, 1.0, -2.0, -2.0, -2.0]])


def test_population_invariant_to_order_within_class_and_fd():
    rng = np.random.default_rng(6)
    B, K, P = 5, 4, 7
    c = rng.integers(0, 3, (B, K * P)).astype(np.float64)
    y = rng.integers(0, K, B)
    L, g = oracle.loss_ce(c, y, P)
    perm = np.concatenate([k * P + rng.permutation(P) for k in range(K)])
    L2, _ = oracle.loss_ce(c[:, perm], y, P)
    assert abs(L - L2) < 1e-14
    # central differences of the loss in each neuron's count
    eps = 1e-6
    for j in rng.integers(0, K * P, 6):
        for b in range(B):
            cp, cm = c.copy(), c.copy()
            cp[b, j] += eps
            cm[b, j] -= eps
            fd = (oracle.loss_ce(cp, y, P)[0] - oracle.loss_ce(cm, y, P)[0]) / (2 * eps)
            assert abs(fd - g[b, j]) < 1e-8

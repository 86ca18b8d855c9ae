"""Comparison protocol between the GPU path and the CPU oracle.

* Spikes: agreement >= 99.99 % per tensor; a disagreement is legal only where
  the oracle's membrane sits within 1e-4 of the threshold (a "root" flip),
  or later in the same column (a flip changes that neuron's future through
  the reset).  With identical fp32 currents the two scans are bit-identical,
  which the stage tests require.
* Floating point: elementwise |a - o| <= tol * (|o| + 1e-2 * max|o|) and
  normwise ||a - o|| / ||o|| <= tol, tol = 1e-3 for fp32 paths and 2e-2 for
  half-precision operands.  Where an operand was rounded to bf16 on purpose
  (the gradient operand of the half-precision net), an element may instead
  stay within the a-priori rounding bound 2^-8 * sum|terms| (each rounded
  value is off by at most 2^-9 of itself): near-zero results of cancelling
  sums carry that error whatever their size.
"""
import numpy as np


def assert_close(a, o, tol=1e-3, what="", abs_bound=None):
    a = np.asarray(a, np.float64)
    o = np.asarray(o, np.float64)
    assert a.shape == o.shape, (what, a.shape, o.shape)
    if o.size == 0:
        return
    scale = np.abs(o).max()
    err = np.abs(a - o)
    bound = tol * (np.abs(o) + 1e-2 * scale)
    if abs_bound is not None:
        bound = np.maximum(bound, np.asarray(abs_bound, np.float64).reshape(bound.shape))
    bad = err > bound
    if scale == 0.0:
        assert err.max() == 0.0, what
        return
    assert not bad.any(), (f"{what}: {bad.sum()} of {o.size} beyond tolerance, worst "
                           f"{(err - bound).max():.3e} (err {err.max():.3e}, max|o| {scale:.3e})")
    nrm = np.linalg.norm(o)
    if nrm > 0:
        assert np.linalg.norm(a - o) / nrm <= tol, what


def spike_flips(z_gpu, z_orc, u_orc, thr, margin=1e-4):
    """Return (agreement fraction, number of root flips, illegal root flips).
    Tensors are [T, ...]; columns are the trailing dims."""
    zg = np.asarray(z_gpu).reshape(z_gpu.shape[0], -1)
    zo = np.asarray(z_orc).reshape(zg.shape)
    uo = np.asarray(u_orc, np.float64).reshape(zg.shape)
    diff = zg != zo
    agree = 1.0 - diff.mean() if diff.size else 1.0
    cols = np.nonzero(diff.any(0))[0]
    illegal = 0
    for c in cols:
        t = int(np.argmax(diff[:, c]))  # first disagreement = root
        if abs(uo[t, c] - thr) >= margin:
            illegal += 1
    return agree, len(cols), illegal


def assert_spikes(z_gpu, z_orc, u_orc, thr, what=""):
    agree, roots, illegal = spike_flips(z_gpu, z_orc, u_orc, thr)
    assert illegal == 0, f"{what}: {illegal} spike flips where |u - thr| >= 1e-4"
    assert agree >= 0.9999, f"{what}: spike agreement {agree:.6f}"
    return roots


def pow2_scale(x, top=2.0 ** 15):
    """The largest power of two S with max|x| * S <= top (1 for all zeros):
    the scale under which an fp16 gradient operand is handed to the
    contractions."""
    m = float(np.abs(np.asarray(x, np.float64)).max()) if np.size(x) else 0.0
    if m == 0.0:
        return 1.0
    e = int(np.floor(np.log2(top / m)))
    while m * 2.0 ** e > top:
        e -= 1
    while m * 2.0 ** (e + 1) <= top:
        e += 1
    return 2.0 ** e

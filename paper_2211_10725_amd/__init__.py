"""MI355X-native spiking-layer training: time-stepped forward and BPTT backward.

Thin ctypes binding over ``libsnn.so`` (C ABI declared in ``include/snn.h``).
The functions below have the ABI's names and only marshal arguments: torch
tensors supply device pointers and the HIP stream, every step of the method
runs in the library's HIP kernels.  There is no CPU fallback: if the library
is missing, the first call raises.

``Network`` chains the layer calls of a feed-forward spiking network (layers
ascending in the forward pass, loss on the output spike counts, layers
descending in the backward pass), the training step the paper times
(Sec. IV "Baseline Throughput", without the optimizer update).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import workloads  # noqa: F401  (seeded inputs; no method arithmetic)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsnn.so")

# element types, neuron models, synapses, gradient kinds, losses (snn.h)
F32, F16, BF16, U8 = 0, 1, 2, 3
SPK_BITS = 4  # spikes packed 64 to a word (an output type only)
LEAKY, SYNAPTIC, RLEAKY = 0, 1, 2
SYN_DENSE, SYN_CONV5_POOL2, SYN_NONE = 0, 1, 2
RESET_DETACHED, RESET_SURROGATE = 0, 1
GRAD_FULL, GRAD_BCAST, GRAD_FOLD = 0, 1, 2
LOSS_CE_COUNT, LOSS_MSE_COUNT = 0, 1
FLAG_FP32_MFMA = 1
ABI_VERSION = 11
DCUR_T_TRANSPOSED, DCUR_T_PLANES = 1, 2

STATUS = {0: "SNN_OK", 1: "SNN_ERR_NULL", 2: "SNN_ERR_SHAPE", 3: "SNN_ERR_DTYPE",
          4: "SNN_ERR_ALIGN", 5: "SNN_ERR_UNSUPPORTED", 6: "SNN_ERR_WORKSPACE",
          7: "SNN_ERR_HIP"}

EXPORTS = ["snn_abi_version", "snn_status_str", "snn_layer_saved_bytes",
           "snn_layer_workspace_bytes", "snn_layer_fwd", "snn_layer_bwd",
           "snn_loss_workspace_bytes", "snn_loss", "snn_synapse_fwd", "snn_neuron_fwd",
           "snn_neuron_bwd", "snn_synapse_bwd", "snn_adamw", "snn_loss_noalloc",
           "snn_layer_saved_layout", "snn_layer_dcur_t_bytes", "snn_layer_dcur_t_layout",
           "snn_fused_step_check", "snn_fused_step_workspace_bytes", "snn_fused_step"]


class LayerDesc(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("B", ctypes.c_int32),
                ("synapse", ctypes.c_int32), ("neuron", ctypes.c_int32),
                ("n_in", ctypes.c_int32), ("n_out", ctypes.c_int32),
                ("c_in", ctypes.c_int32), ("h_in", ctypes.c_int32),
                ("w_in", ctypes.c_int32), ("c_out", ctypes.c_int32),
                ("in_dtype", ctypes.c_int32), ("w_dtype", ctypes.c_int32),
                ("out_dtype", ctypes.c_int32), ("grad_dtype", ctypes.c_int32),
                ("reset_grad", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("beta", ctypes.c_float), ("alpha", ctypes.c_float),
                ("threshold", ctypes.c_float), ("slope", ctypes.c_float)]

    def copy(self):
        d = LayerDesc()
        ctypes.pointer(d)[0] = self
        return d


class SavedLayout(ctypes.Structure):
    _fields_ = [("bytes", ctypes.c_size_t), ("cur_offset", ctypes.c_size_t),
                ("cur_bytes", ctypes.c_size_t), ("ckpt_offset", ctypes.c_size_t),
                ("ckpt_bytes", ctypes.c_size_t), ("pool_offset", ctypes.c_size_t),
                ("pool_bytes", ctypes.c_size_t), ("ckpt_interval", ctypes.c_int32),
                ("ckpt_count", ctypes.c_int32), ("ckpt_planes", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class FusedDesc(ctypes.Structure):
    _fields_ = [("hidden", LayerDesc), ("readout", LayerDesc), ("loss_kind", ctypes.c_int32),
                ("pop", ctypes.c_int32), ("wait_limit", ctypes.c_uint32),
                ("reserved", ctypes.c_int32)]


class GradIn(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("n_up", ctypes.c_int32),
                ("g", ctypes.c_void_p), ("dcur_up", ctypes.c_void_p), ("w_up", ctypes.c_void_p),
                ("dcur_up_dtype", ctypes.c_int32), ("w_up_dtype", ctypes.c_int32)]


class AdamwTensor(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("m", ctypes.c_void_p),
                ("v", ctypes.c_void_p), ("param_half", ctypes.c_void_p), ("n", ctypes.c_int64)]


class AdamwHparams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float),
                ("step", ctypes.c_int32)]


class SNNError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn} failed: {STATUS.get(status, status)} "
                         f"({_lib.snn_status_str(status).decode() if _lib else ''})")


_lib = None


def lib():
    """Load libsnn.so (built in-tree by ``build.build()``); raise if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"HIP library {LIB_PATH} is not built; run __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    P, S = ctypes.c_void_p, ctypes.c_size_t
    D = ctypes.POINTER(LayerDesc)
    G = ctypes.POINTER(GradIn)
    i32 = ctypes.c_int32
    sig = {
        "snn_abi_version": ([], ctypes.c_int),
        "snn_status_str": ([ctypes.c_int], ctypes.c_char_p),
        "snn_layer_saved_bytes": ([D], S),
        "snn_layer_saved_layout": ([D, ctypes.POINTER(SavedLayout)], ctypes.c_int),
        "snn_layer_workspace_bytes": ([D], S),
        "snn_layer_fwd": ([D, P, P, P, P, P, P, P, P, S, P], ctypes.c_int),
        "snn_layer_bwd": ([D, G, P, P, P, P, P, P, P, P, P, S, P], ctypes.c_int),
        "snn_loss_workspace_bytes": ([i32, i32, i32], S),
        "snn_loss": ([i32, i32, i32, i32, P, P, P, P, P, P, S, P], ctypes.c_int),
        "snn_loss_noalloc": ([i32, i32, i32, i32, P, P, P, P, P, P], ctypes.c_int),
        "snn_synapse_fwd": ([D, P, P, P, P, P, P, S, P], ctypes.c_int),
        "snn_neuron_fwd": ([D, P, P, P, P, P, P, P], ctypes.c_int),
        "snn_neuron_bwd": ([D, G, P, P, P, P, P, P, P, P, P, S, P], ctypes.c_int),
        "snn_synapse_bwd": ([D, P, P, P, P, P, P, P, P, P, S, P], ctypes.c_int),
        "snn_layer_dcur_t_bytes": ([D], S),
        "snn_layer_dcur_t_layout": ([D], i32),
        "snn_fused_step_check": ([ctypes.POINTER(FusedDesc)], ctypes.c_int),
        "snn_fused_step_workspace_bytes": ([ctypes.POINTER(FusedDesc)], S),
        "snn_fused_step": ([ctypes.POINTER(FusedDesc)] + [P] * 16 + [S, P], ctypes.c_int),
        "snn_adamw": ([ctypes.POINTER(AdamwTensor), i32, ctypes.POINTER(AdamwHparams), P],
                      ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    if L.snn_abi_version() != ABI_VERSION:
        raise RuntimeError("libsnn.so ABI version mismatch")
    _lib = L
    return L


# --------------------------------------------------------------------------
# argument marshalling
# --------------------------------------------------------------------------
def _p(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(fn, st):
    if st != 0:
        raise SNNError(fn, st)


def _dtype_code(t):
    import torch
    return {torch.float32: F32, torch.bfloat16: BF16, torch.float16: F16}[t.dtype]


def _grad_in(kind, g):
    """The upstream gradient argument: g a tensor for GRAD_FULL / GRAD_BCAST,
    or (dcur_up, w_up) for GRAD_FOLD (dL/dI [T,B,n_up] and the weights
    [n_up, n_out] of the dense layer above)."""
    if kind == GRAD_FOLD:
        dup, wup = g
        return GradIn(kind, int(wup.shape[0]), None, _p(dup), _p(wup), _dtype_code(dup),
                      _dtype_code(wup))
    return GradIn(kind, 0, _p(g), None, None, 0, 0)


I32 = 100  # int32 arguments (labels, status): not a layer dtype
_ELEM = {F32: 4, F16: 2, BF16: 2, U8: 1, I32: 4}


def _need(fn, t, dtype_code, count, what):
    """A tensor argument must hold at least `count` elements of the type the
    descriptor names (the library cannot see buffer sizes): raise before the
    call instead of letting a kernel run past the buffer."""
    if t is None or isinstance(t, int):
        return
    es = _ELEM[dtype_code]
    if t.element_size() != es or t.numel() < count:
        raise ValueError(f"{fn}: {what} needs {count} elements of {es} bytes, got "
                         f"{t.numel()} of {t.element_size()}")


def _check_fwd_io(fn, d, x=None, spk=None):
    rows = d.T * d.B
    _need(fn, x, d.in_dtype, rows * d.n_in, "x")
    if d.out_dtype == SPK_BITS:
        _need(fn, spk, U8, rows * d.n_out // 8, "spk_out (packed bits)")
    else:
        _need(fn, spk, d.out_dtype, rows * d.n_out, "spk_out")


def snn_layer_saved_bytes(desc: LayerDesc) -> int:
    return int(lib().snn_layer_saved_bytes(ctypes.byref(desc)))


def snn_layer_saved_layout(desc: LayerDesc) -> SavedLayout:
    out = SavedLayout()
    _check("snn_layer_saved_layout", lib().snn_layer_saved_layout(ctypes.byref(desc),
                                                                  ctypes.byref(out)))
    return out


def saved_parts(desc: LayerDesc, saved):
    """Views of a saved-state buffer (uint8 tensor of snn_layer_saved_bytes):
    (currents fp32 [T,B,n_out] or None, checkpoints fp32, pool selection u8
    [T,B,n_out] or None), at the offsets the library reports."""
    lay = snn_layer_saved_layout(desc)
    T, B, n = desc.T, desc.B, desc.n_out
    cur = None
    if lay.cur_bytes:
        cur = saved[lay.cur_offset: lay.cur_offset + T * B * n * 4].view(
            __import__("torch").float32).view(T, B, n)
    ck = saved[lay.ckpt_offset: lay.ckpt_offset + lay.ckpt_bytes].view(
        __import__("torch").float32)
    pool = None
    if lay.pool_bytes:
        pool = saved[lay.pool_offset: lay.pool_offset + T * B * n].view(T, B, n)
    return cur, ck, pool


def ckpt_buffer(desc: LayerDesc, device="cuda"):
    """A device buffer for the checkpoints of snn_neuron_fwd / snn_neuron_bwd."""
    import torch
    lay = snn_layer_saved_layout(desc)
    return torch.empty(max(64, lay.ckpt_bytes // 4), dtype=torch.float32, device=device)


def snn_layer_dcur_t_bytes(desc: LayerDesc) -> int:
    return int(lib().snn_layer_dcur_t_bytes(ctypes.byref(desc)))


def _dcur_t_written(desc: LayerDesc) -> int:
    """Bytes snn_neuron_bwd writes to a dcur_t argument: the layer's operand
    when its weight gradient takes one, else the transposed layout
    ([P][n_out][T*B] 16-bit, P = 3 for an fp32 dL/dI)."""
    n = snn_layer_dcur_t_bytes(desc)
    if n > 0:
        return n
    return (3 if desc.grad_dtype == F32 else 1) * desc.n_out * desc.T * desc.B * 2


def snn_layer_dcur_t_layout(desc: LayerDesc) -> int:
    """DCUR_T_TRANSPOSED or DCUR_T_PLANES: the layout of the dcur_t operand
    snn_neuron_bwd writes for this layer."""
    return int(lib().snn_layer_dcur_t_layout(ctypes.byref(desc)))


def snn_layer_workspace_bytes(desc: LayerDesc) -> int:
    return int(lib().snn_layer_workspace_bytes(ctypes.byref(desc)))


def snn_loss_workspace_bytes(kind: int, B: int, K: int) -> int:
    return int(lib().snn_loss_workspace_bytes(kind, B, K))


def snn_layer_fwd(desc, x, w, bias, v, spk_out, saved, counts, ws, stream=None):
    _check_fwd_io("snn_layer_fwd", desc, x, spk_out)
    _check("snn_layer_fwd", lib().snn_layer_fwd(
        ctypes.byref(desc), _p(x), _p(w), _p(bias), _p(v), _p(spk_out), _p(saved), _p(counts),
        _p(ws), _nbytes(ws), _stream(stream)))


def snn_layer_bwd(desc, grad_kind, g, x, w, v, saved, grad_w, grad_b, grad_v, grad_x, ws,
                  stream=None):
    _check_fwd_io("snn_layer_bwd", desc, x)
    gi = _grad_in(grad_kind, g)
    _check("snn_layer_bwd", lib().snn_layer_bwd(
        ctypes.byref(desc), ctypes.byref(gi), _p(x), _p(w), _p(v), _p(saved), _p(grad_w),
        _p(grad_b), _p(grad_v), _p(grad_x), _p(ws), _nbytes(ws), _stream(stream)))


def snn_loss(kind, B, K, P, counts, labels, targets, loss, grad_counts, ws, stream=None):
    _check("snn_loss", lib().snn_loss(kind, B, K, P, _p(counts), _p(labels), _p(targets),
                                      _p(loss), _p(grad_counts), _p(ws), _nbytes(ws),
                                      _stream(stream)))


def snn_loss_noalloc(kind, B, K, P, counts, labels, targets, loss, grad_counts, stream=None):
    _check("snn_loss_noalloc", lib().snn_loss_noalloc(kind, B, K, P, _p(counts), _p(labels),
                                                      _p(targets), _p(loss), _p(grad_counts),
                                                      _stream(stream)))


def fused_desc(hidden, readout, loss_kind, pop=1, wait_limit=0) -> FusedDesc:
    f = FusedDesc()
    f.hidden, f.readout = hidden, readout
    f.loss_kind, f.pop, f.wait_limit, f.reserved = loss_kind, pop, wait_limit, 0
    return f


def snn_fused_step_check(fd) -> int:
    return lib().snn_fused_step_check(ctypes.byref(fd))


def snn_fused_step_workspace_bytes(fd) -> int:
    return lib().snn_fused_step_workspace_bytes(ctypes.byref(fd))


def snn_fused_step(fd, x, w0, b0, w1, b1, labels, targets, loss, counts, gw0, gb0, gw1, gb1,
                   status, ws, stream=None, spk_hidden=None):
    h, r = fd.hidden, fd.readout
    _need("snn_fused_step", x, U8, h.T * h.B * h.n_in, "x")
    _need("snn_fused_step", w0, F32, h.n_out * h.n_in, "w0")
    _need("snn_fused_step", w1, F32, r.n_out * r.n_in, "w1")
    _need("snn_fused_step", gw0, F32, h.n_out * h.n_in, "grad_w0")
    _need("snn_fused_step", gw1, F32, r.n_out * r.n_in, "grad_w1")
    _need("snn_fused_step", counts, F32, h.B * r.n_out, "counts")
    _need("snn_fused_step", b0, F32, h.n_out, "b0")
    _need("snn_fused_step", b1, F32, r.n_out, "b1")
    _need("snn_fused_step", gb0, F32, h.n_out, "grad_b0")
    _need("snn_fused_step", gb1, F32, r.n_out, "grad_b1")
    _need("snn_fused_step", loss, F32, 1, "loss")
    _need("snn_fused_step", status, I32, 1, "status")
    _need("snn_fused_step", spk_hidden, U8, h.T * h.B * h.n_out, "spk_hidden")
    if fd.loss_kind == LOSS_CE_COUNT:
        _need("snn_fused_step", labels, I32, h.B, "labels")
    else:
        _need("snn_fused_step", targets, F32, h.B * (r.n_out // max(fd.pop, 1)), "targets")
    _check("snn_fused_step", lib().snn_fused_step(
        ctypes.byref(fd), _p(x), _p(w0), _p(b0), _p(w1), _p(b1), _p(labels), _p(targets),
        _p(loss), _p(counts), _p(spk_hidden), _p(gw0), _p(gb0), _p(gw1), _p(gb1), _p(status),
        _p(ws), _nbytes(ws), _stream(stream)))


def snn_synapse_fwd(desc, x, w, bias, cur, pool_arg, ws, stream=None):
    _check_fwd_io("snn_synapse_fwd", desc, x)
    _check("snn_synapse_fwd", lib().snn_synapse_fwd(
        ctypes.byref(desc), _p(x), _p(w), _p(bias), _p(cur), _p(pool_arg), _p(ws), _nbytes(ws),
        _stream(stream)))


def snn_neuron_fwd(desc, cur, v, spk_out, ckpt, counts, stream=None, u_out=None):
    """ckpt: checkpoints (ckpt_buffer); u_out: the membrane of every step, or None."""
    _check_fwd_io("snn_neuron_fwd", desc, None, spk_out)
    _need("snn_neuron_fwd", u_out, F32, desc.T * desc.B * desc.n_out, "u_out")
    _need("snn_neuron_fwd", ckpt, F32, snn_layer_saved_layout(desc).ckpt_bytes // 4, "ckpt")
    _check("snn_neuron_fwd", lib().snn_neuron_fwd(
        ctypes.byref(desc), _p(cur), _p(v), _p(spk_out), _p(ckpt), _p(u_out), _p(counts),
        _stream(stream)))


def snn_neuron_bwd(desc, grad_kind, g, v, cur, ckpt, dcur, grad_b, grad_v, ws, stream=None,
                   dcur_scale=None, dcur_t=None):
    """cur, ckpt: the forward's currents and checkpoints.  dcur_scale: device
    fp32 scalar receiving the power of two an fp16 dcur is scaled by
    (required for grad_dtype F16).  dcur_t: the weight gradient's operand in
    the layout snn_layer_dcur_t_layout names (transposed, or an fp32 dL/dI's
    three bf16 planes; snn_layer_dcur_t_bytes), or None; dcur may then be
    None."""
    if dcur_t is not None and dcur_t.numel() * dcur_t.element_size() < _dcur_t_written(desc):
        raise ValueError("snn_neuron_bwd: dcur_t smaller than the operand the scan writes")
    _need("snn_neuron_bwd", cur, F32, desc.T * desc.B * desc.n_out, "cur")
    _need("snn_neuron_bwd", ckpt, F32, snn_layer_saved_layout(desc).ckpt_bytes // 4, "ckpt")
    _need("snn_neuron_bwd", dcur, desc.grad_dtype if desc.synapse != SYN_NONE else F32,
          desc.T * desc.B * desc.n_out, "dcur")
    gi = _grad_in(grad_kind, g)
    _check("snn_neuron_bwd", lib().snn_neuron_bwd(
        ctypes.byref(desc), ctypes.byref(gi), _p(v), _p(cur), _p(ckpt), _p(dcur), _p(dcur_t),
        _p(dcur_scale), _p(grad_b), _p(grad_v), _p(ws), _nbytes(ws), _stream(stream)))


def snn_synapse_bwd(desc, dcur, pool_arg, x, w, grad_w, grad_x, ws, stream=None,
                    dcur_scale=None, dcur_t=None):
    _check_fwd_io("snn_synapse_bwd", desc, x)
    _need("snn_synapse_bwd", dcur, desc.grad_dtype, desc.T * desc.B * desc.n_out, "dcur")
    if dcur_t is not None and dcur_t.numel() * dcur_t.element_size() < \
            snn_layer_dcur_t_bytes(desc):
        raise ValueError("snn_synapse_bwd: dcur_t smaller than snn_layer_dcur_t_bytes")
    _check("snn_synapse_bwd", lib().snn_synapse_bwd(
        ctypes.byref(desc), _p(dcur), _p(dcur_t), _p(dcur_scale), _p(pool_arg), _p(x), _p(w),
        _p(grad_w), _p(grad_x), _p(ws), _nbytes(ws), _stream(stream)))


def snn_adamw(tensors, step, lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=1e-2,
              stream=None):
    """tensors: sequence of (param, grad, m, v, param_half or None) device
    tensors (fp32, param_half fp16), all updated in one fused pass."""
    arr = (AdamwTensor * max(1, len(tensors)))()
    for i, (p, g, m, v, h) in enumerate(tensors):
        arr[i] = AdamwTensor(_p(p), _p(g), _p(m), _p(v), _p(h), p.numel())
    hp = AdamwHparams(lr, betas[0], betas[1], eps, weight_decay, step)
    _check("snn_adamw", lib().snn_adamw(arr, len(tensors), ctypes.byref(hp), _stream(stream)))


# --------------------------------------------------------------------------
# descriptors from plain layer specs
# --------------------------------------------------------------------------
_NEURON = {"leaky": LEAKY, "synaptic": SYNAPTIC, "rleaky": RLEAKY}


def layer_desc(spec: dict, T: int, B: int, in_dtype=U8, w_dtype=F32, out_dtype=U8,
               grad_dtype=F32, slope=25.0, reset_grad=RESET_DETACHED, flags=0) -> LayerDesc:
    d = LayerDesc()
    d.flags = flags
    d.T, d.B = T, B
    d.neuron = _NEURON[spec["neuron"]]
    d.beta = spec["beta"]
    d.alpha = spec.get("alpha", 0.0)
    d.threshold = spec.get("thr", 1.0)
    d.slope = slope
    d.reset_grad = reset_grad
    d.in_dtype, d.w_dtype, d.out_dtype, d.grad_dtype = in_dtype, w_dtype, out_dtype, grad_dtype
    if spec["kind"] == "dense":
        d.synapse = SYN_DENSE
        d.n_in, d.n_out = spec["n_in"], spec["n_out"]
    elif spec["kind"] == "conv":
        d.synapse = SYN_CONV5_POOL2
        d.c_in, d.h_in, d.w_in, d.c_out = spec["c_in"], spec["h"], spec["w"], spec["c_out"]
        d.n_in = d.c_in * d.h_in * d.w_in
        d.n_out = d.c_out * ((d.h_in - 4) // 2) * ((d.w_in - 4) // 2)
    else:
        d.synapse = SYN_NONE
        d.n_in = d.n_out = spec["n"]
        d.in_dtype = F32
    return d


class Network:
    """Device buffers and the layer-call sequence of one training step.

    All buffers are allocated once here (torch, device memory only); ``step``
    then only enqueues library calls on the current stream."""

    def __init__(self, wl, params, device="cuda", reset_grad=RESET_DETACHED, flags=0, fold=True,
                 spike_bits=False, input_bf16=False):
        import torch
        self.torch = torch
        self.wl = wl
        self.device = device
        T, B = wl.T, wl.B
        half = wl.dtype == "f16"
        self.descs = []
        self.W, self.b, self.v = [], [], []
        for li, spec in enumerate(wl.layers):
            in_dt = F32 if spec["kind"] == "none" else U8
            # input_bf16: an fp32 net's input spikes given as bf16 0/1, the
            # operand type of its three-plane contractions (no widening pass
            # before the first layer's forward and weight gradient)
            if li == 0 and input_bf16 and not half and spec["kind"] == "dense":
                in_dt = BF16
            # half-precision nets hand dL/dI to the contractions in bf16, which
            # keeps fp32's exponent range for the small BPTT gradients
            d = layer_desc(spec, T, B, in_dtype=in_dt, w_dtype=F16 if half else F32,
                           out_dtype=U8, grad_dtype=BF16 if half else F32, slope=wl.slope,
                           reset_grad=reset_grad, flags=flags)
            self.descs.append(d)
            W, b = params[li][0], params[li][1]
            # recurrent weights of an 'rleaky' layer: (W, b, v)
            v = params[li][2] if len(params[li]) > 2 else None
            self.v.append(None if v is None else torch.as_tensor(np.ascontiguousarray(
                v, np.float32)).to(device))
            if W is None:
                self.W.append(None)
                self.b.append(None)
            else:
                wdt = torch.float16 if half else torch.float32
                self.W.append(torch.as_tensor(np.ascontiguousarray(W)).to(device=device, dtype=wdt))
                self.b.append(torch.as_tensor(np.ascontiguousarray(b)).to(device=device,
                                                                         dtype=torch.float32))
        u8 = torch.uint8
        # Spikes that feed a large fp16 contraction (a dense layer above with
        # at least 256 outputs) are written as fp16 0/1 by the scan, the
        # operand type that contraction stages directly; other spikes as bytes.
        for li in range(len(self.descs) - 1):
            up = self.descs[li + 1]
            if half and up.synapse == SYN_DENSE and up.n_out >= 256 and up.n_in >= 256:
                self.descs[li].out_dtype = F16
                up.in_dtype = F16
        # spike_bits: the last layer's spikes, which no contraction reads,
        # packed 64 to a word (layers of a multiple of 64 neurons)
        if spike_bits and self.descs[-1].n_out % 64 == 0:
            self.descs[-1].out_dtype = SPK_BITS
        self.spk = [torch.empty((T, B, d.n_out // 8 if d.out_dtype == SPK_BITS else d.n_out),
                                dtype=torch.float16 if d.out_dtype == F16 else u8, device=device)
                    for d in self.descs]
        self.in_shape = (T, B) + tuple(wl.in_shape)
        self.saved = [torch.empty(snn_layer_saved_bytes(d), dtype=u8, device=device)
                      for d in self.descs]
        # (currents, checkpoints, pool selection) views of each saved buffer
        self.layouts = [snn_layer_saved_layout(d) for d in self.descs]
        self.parts = [saved_parts(d, sv) for d, sv in zip(self.descs, self.saved)]
        self.gW = [None if w is None else torch.empty(w.shape, dtype=torch.float32, device=device)
                   for w in self.W]
        self.gb = [None if b is None else torch.empty(b.shape, dtype=torch.float32, device=device)
                   for b in self.b]
        self.gv = [None if v is None else torch.empty(v.shape, dtype=torch.float32, device=device)
                   for v in self.v]
        # dL/dx of layer l is the upstream gradient of layer l-1
        self.gx = [None] + [torch.empty((T, B, d.n_in), dtype=torch.float32, device=device)
                            for d in self.descs[1:]]
        if self.descs[0].synapse == SYN_NONE:
            self.gx[0] = torch.empty((T, B, self.descs[0].n_in), dtype=torch.float32, device=device)
        # A dense layer with at most 16 outputs (the readout) above a layer of
        # at least 64 neurons: its input gradient dx = dI W is folded into the
        # reverse scan of the layer below (SNN_GRAD_FOLD), which then reads the
        # readout's dL/dI (kept in dup) instead of a [T,B,n] gradient.
        n = len(self.descs)
        self.fold = [fold and li + 1 < n and self.descs[li + 1].synapse == SYN_DENSE
                     and self.descs[li + 1].n_out <= 16 and self.descs[li].n_out >= 64
                     for li in range(n)]
        gdt = {F32: torch.float32, BF16: torch.bfloat16, F16: torch.float16}
        self.dup = [None] * n
        for li in range(n - 1):
            if self.fold[li]:
                self.gx[li + 1] = None
        # The fp16 net's gradient operand dL/dI: fp16 scaled by a power of two
        # (one MFMA pass against the fp16 weights of the input gradient) for
        # layers whose input gradient is a contraction; bf16 otherwise (the
        # weight gradient against spikes is one pass in either type).  The
        # scale needs a bound of the upstream gradient: cheap for a broadcast
        # or folded one, one extra read of a full [T,B,n] gradient otherwise.
        self.scale = [None] * n
        for li, d in enumerate(self.descs):
            if not half or d.synapse != SYN_DENSE or d.neuron == RLEAKY:
                continue
            if li > 0 and self.gx[li] is not None:
                d.grad_dtype = F16
                self.scale[li] = torch.empty(4, dtype=torch.float32, device=device)
        for li in range(n - 1):
            if self.fold[li]:
                up = self.descs[li + 1]
                self.dup[li + 1] = torch.empty((T, B, up.n_out), dtype=gdt[up.grad_dtype],
                                               device=device)
        # K classes, P output neurons per class (a population code when P > 1)
        self.P = getattr(wl, "pop", 1)
        n_last = self.descs[-1].n_out
        assert n_last % self.P == 0, (n_last, self.P)
        K = n_last // self.P
        self.K = K
        self.counts = torch.empty((B, n_last), dtype=torch.float32, device=device)
        self.loss = torch.empty(4, dtype=torch.float32, device=device)  # [0] is the loss
        self.gcounts = torch.empty((B, n_last), dtype=torch.float32, device=device)
        self.loss_kind = LOSS_CE_COUNT if wl.loss == "ce" else LOSS_MSE_COUNT
        ws = max([snn_layer_workspace_bytes(d) for d in self.descs] +
                 [snn_loss_workspace_bytes(self.loss_kind, B, K), 256])
        self.ws = torch.empty(ws, dtype=u8, device=device)
        # the reverse scan's transposed dL/dI for the weight gradient (stage
        # calls; the layer calls keep it in the workspace)
        self.dcur_t_bytes = [snn_layer_dcur_t_bytes(d) for d in self.descs]
        self.dcur_t_layout = [snn_layer_dcur_t_layout(d) for d in self.descs]
        self.transposed_operand = False
        self.dcur_t = torch.empty(max(self.dcur_t_bytes + [256]), dtype=u8, device=device)
        # The whole step as one cooperative launch (step_fused): two dense
        # layers on spike input with fp32 weights, small enough for one
        # co-resident grid; None where snn_fused_step_check refuses the net.
        self.fdesc = None
        if n == 2 and not half and all(d.synapse == SYN_DENSE for d in self.descs):
            fd = fused_desc(self.descs[0].copy(), self.descs[1].copy(), self.loss_kind, self.P)
            if snn_fused_step_check(fd) == 0:
                self.fdesc = fd
                self.fws = torch.empty(max(256, snn_fused_step_workspace_bytes(fd)), dtype=u8,
                                       device=device)
                self.fstatus = torch.zeros(4, dtype=torch.int32, device=device)

    def forward(self, x, stream=None):
        h = x
        n = len(self.descs)
        for li, d in enumerate(self.descs):
            snn_layer_fwd(d, h, self.W[li], self.b[li], self.v[li], self.spk[li], self.saved[li],
                          self.counts if li == n - 1 else None, self.ws, stream)
            h = self.spk[li]

    def loss_and_grad(self, labels=None, targets=None, stream=None):
        snn_loss(self.loss_kind, self.wl.B, self.K, self.P, self.counts, labels, targets,
                 self.loss, self.gcounts, self.ws, stream)

    def _grad_below(self, li):
        """The upstream gradient argument of layer li - 1."""
        if self.fold[li - 1]:
            return GRAD_FOLD, (self.dup[li], self.W[li])
        return GRAD_FULL, self.gx[li]

    def backward(self, x, stream=None):
        n = len(self.descs)
        kind, g = GRAD_BCAST, self.gcounts
        for li in range(n - 1, -1, -1):
            d = self.descs[li]
            xin = x if li == 0 else self.spk[li - 1]
            if self.dup[li] is not None:
                # dL/dI kept for the layer below; no dx of its own
                cur, ck, _ = self.parts[li]
                snn_neuron_bwd(d, kind, g, self.v[li], xin if cur is None else cur, ck,
                               self.dup[li], self.gb[li], self.gv[li], self.ws, stream,
                               dcur_scale=self.scale[li])
                snn_synapse_bwd(d, self.dup[li], self.pool_arg(li), xin, self.W[li], self.gW[li],
                                None, self.ws, stream, dcur_scale=self.scale[li])
            else:
                snn_layer_bwd(d, kind, g, xin, self.W[li], self.v[li], self.saved[li],
                              self.gW[li], self.gb[li], self.gv[li], self.gx[li], self.ws, stream)
            if li > 0:
                kind, g = self._grad_below(li)

    def step(self, x, labels=None, targets=None, stream=None):
        self.forward(x, stream)
        self.loss_and_grad(labels, targets, stream)
        self.backward(x, stream)

    def step_fused(self, x, labels=None, targets=None, stream=None):
        """The step as one snn_fused_step launch (needs ``fdesc``): the loss,
        the readout's counts, the hidden spikes and the weight and bias
        gradients land in the buffers ``step`` writes; ``fstatus[0]`` is 0
        after a completed step."""
        if self.fdesc is None:
            raise RuntimeError("step_fused: the library's fused step does not run this network")
        snn_fused_step(self.fdesc, x, self.W[0], self.b[0], self.W[1], self.b[1], labels, targets,
                       self.loss, self.counts, self.gW[0], self.gb[0], self.gW[1], self.gb[1],
                       self.fstatus, self.fws, stream, spk_hidden=self.spk[0])

    def capture_step(self, x, labels=None, targets=None, warmup=2):
        """Capture one forward + loss + BPTT step into a HIP graph (torch's
        CUDAGraph on ROCm) and return it; ``graph.replay()`` then reruns the
        step on the same buffers with one launch from the host.  The library
        records no memset, allocates nothing and never synchronises, so every
        call of the step can be captured."""
        torch = self.torch
        side = torch.cuda.Stream()  # default priority
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for _ in range(warmup):
                self.step(x, labels, targets)
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=side):
            self.step(x, labels, targets)
        return graph

    def init_adamw(self, lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=1e-2):
        """Optimizer state for ``update``: zero moments per parameter tensor
        and, for fp16 weights, an fp32 master copy (the fp16 weights the
        contractions read are rewritten from it after every update)."""
        torch = self.torch
        self.opt = dict(lr=lr, betas=betas, eps=eps, weight_decay=weight_decay)
        self.opt_t = 0
        self.opt_tensors = []
        for li in range(len(self.descs)):
            for P, G in ((self.W[li], self.gW[li]), (self.b[li], self.gb[li]),
                         (self.v[li], self.gv[li])):
                if P is None:
                    continue
                half = P.dtype == torch.float16
                master = P.float().contiguous() if half else P
                self.opt_tensors.append((master, G, torch.zeros_like(master),
                                         torch.zeros_like(master), P if half else None))

    def update(self, stream=None):
        """One AdamW step over every parameter with the gradients of the last
        backward (Sec. IV: the paper's training step ends with it)."""
        self.opt_t += 1
        snn_adamw(self.opt_tensors, self.opt_t, stream=stream, **self.opt)

    def pool_arg(self, li):
        """The 2x2 pool selection of conv layer li inside its saved buffer
        (None for other layers), at the offset the library reports."""
        return self.parts[li][2]

    # the same work through the stage calls, with a hook between stages
    # (update: finish with the AdamW step of ``init_adamw``; fused_bwd: each
    # layer's backward as one snn_layer_bwd call, hooked as "layer_bwd", as in
    # ``backward``, except for the layers listed in ``staged``).  A dense
    # layer's synapse backward is two stage calls, the weight gradient
    # ("synapse_bwd_dw") then the input gradient ("synapse_bwd_dx"): the same
    # kernels in the same order as one snn_synapse_bwd call with both outputs.
    def step_stages(self, x, labels=None, targets=None, stream=None, hook=None, update=False,
                    fused_bwd=False, staged=()):
        torch = self.torch
        hook = hook or (lambda name, li: None)
        n = len(self.descs)
        h = x
        for li, d in enumerate(self.descs):
            cur, ck, _ = self.parts[li]
            if d.synapse != SYN_NONE:
                hook("synapse_fwd", li)
                snn_synapse_fwd(d, h, self.W[li], self.b[li], cur, self.pool_arg(li), self.ws,
                                stream)
                hook("synapse_fwd_end", li)
            else:
                cur = h
            hook("neuron_fwd", li)
            snn_neuron_fwd(d, cur, self.v[li], self.spk[li], ck,
                           self.counts if li == n - 1 else None, stream)
            hook("neuron_fwd_end", li)
            h = self.spk[li]
        hook("loss", -1)
        self.loss_and_grad(labels, targets, stream)
        hook("loss_end", -1)
        kind, g = GRAD_BCAST, self.gcounts
        for li in range(n - 1, -1, -1):
            d = self.descs[li]
            xin = x if li == 0 else self.spk[li - 1]
            if d.synapse == SYN_NONE:
                hook("neuron_bwd", li)
                snn_neuron_bwd(d, kind, g, self.v[li], xin, self.parts[li][1], self.gx[li], None,
                               self.gv[li], self.ws, stream)
                hook("neuron_bwd_end", li)
                continue
            if fused_bwd and self.dup[li] is None and li not in staged:
                hook("layer_bwd", li)
                snn_layer_bwd(d, kind, g, xin, self.W[li], self.v[li], self.saved[li],
                              self.gW[li], self.gb[li], self.gv[li], self.gx[li], self.ws, stream)
                hook("layer_bwd_end", li)
                if li > 0:
                    kind, g = self._grad_below(li)
                continue
            dcur_bytes = d.T * d.B * d.n_out * (2 if d.grad_dtype in (F16, BF16) else 4)
            if self.dup[li] is not None:
                dcur, rest = self.dup[li], self.ws
            else:
                dcur = self.ws[:dcur_bytes]
                if d.grad_dtype == BF16:
                    dcur = dcur.view(torch.bfloat16)
                elif d.grad_dtype == F16:
                    dcur = dcur.view(torch.float16)
                else:
                    dcur = dcur.view(torch.float32)
                rest = self.ws[(dcur_bytes + 255) // 256 * 256:]
            sc = self.scale[li]
            # the weight gradient's operand written by the scan: transposed
            # (transposed_operand=True; off by default, it measured slower
            # than one transpose, as in the layer call), or the three bf16
            # planes of an fp32 dL/dI in its own layout (always, as in the
            # layer call); the row-major dL/dI only where the input gradient
            # needs it.
            use_t = self.transposed_operand or self.dcur_t_layout[li] == DCUR_T_PLANES
            dt = self.dcur_t if use_t and self.dcur_t_bytes[li] > 0 and \
                self.dup[li] is None else None
            rm = dcur if dt is None or self.gx[li] is not None or self.dup[li] is not None \
                else None
            hook("neuron_bwd", li)
            cur, ck, _ = self.parts[li]
            snn_neuron_bwd(d, kind, g, self.v[li], cur, ck, rm, self.gb[li],
                           self.gv[li], rest, stream, dcur_scale=sc, dcur_t=dt)
            hook("neuron_bwd_end", li)
            if d.synapse == SYN_DENSE:
                hook("synapse_bwd_dw", li)
                snn_synapse_bwd(d, rm, None, xin, self.W[li], self.gW[li], None, rest, stream,
                                dcur_scale=sc, dcur_t=dt)
                hook("synapse_bwd_dw_end", li)
                if self.gx[li] is not None:
                    hook("synapse_bwd_dx", li)
                    snn_synapse_bwd(d, dcur, None, xin, self.W[li], None, self.gx[li], rest,
                                    stream, dcur_scale=sc)
                    hook("synapse_bwd_dx_end", li)
            else:
                hook("synapse_bwd", li)
                snn_synapse_bwd(d, dcur, self.pool_arg(li), xin, self.W[li], self.gW[li],
                                self.gx[li], rest, stream)
                hook("synapse_bwd_end", li)
            if li > 0:
                kind, g = self._grad_below(li)
        if update:
            hook("update", -1)
            self.update(stream)
            hook("update_end", -1)

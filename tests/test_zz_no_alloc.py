"""snn_loss_noalloc, the loss for callers that cannot allocate: the same
kernels as snn_loss, with their partial sums in a device array the library
holds instead of a caller's workspace.  Its results must equal snn_loss's bit
for bit, on consecutive calls with different sizes (the array keeps the last
call's contents)."""
import ctypes

import numpy as np
import pytest

import paper_2211_10725_amd as snn

torch = pytest.importorskip("torch")


def test_noalloc_rejects_sizes_beyond_its_array():
    # validation only (fake aligned addresses, never dereferenced): cross-entropy
    # over more than 131072 rows needs more than the 1 MiB the library holds
    L = snn.lib()
    st = L.snn_loss_noalloc(snn.LOSS_CE_COUNT, 131073, 10, 1, 16, 32, None, 48, 64, None)
    assert st == 6  # SNN_ERR_WORKSPACE
    assert L.snn_loss_noalloc(snn.LOSS_CE_COUNT, 4, 10, 1, None, 32, None, 48, 64, None) == 1
    assert L.snn_loss_noalloc(snn.LOSS_MSE_COUNT, 4, 10, 1, 16, None, None, 48, 64, None) == 1
    assert L.snn_loss_noalloc(7, 4, 10, 1, 16, 32, None, 48, 64, None) == 5


def _inputs(kind, B, K, P, seed):
    rng = np.random.default_rng(seed)
    counts = torch.as_tensor(rng.integers(0, 30, (B, K * P)).astype(np.float32)).cuda()
    labels = torch.as_tensor(rng.integers(0, K, B).astype(np.int32)).cuda()
    targets = torch.as_tensor(rng.uniform(0, 50, (B, K)).astype(np.float32)).cuda()
    return counts, (labels if kind == snn.LOSS_CE_COUNT else None), \
        (targets if kind == snn.LOSS_MSE_COUNT else None)


def _with_workspace(kind, B, K, P, counts, labels, targets):
    loss = torch.empty(4, dtype=torch.float32, device="cuda")
    grad = torch.empty_like(counts)
    ws = torch.empty(max(256, snn.snn_loss_workspace_bytes(kind, B, K)), dtype=torch.uint8,
                     device="cuda")
    snn.snn_loss(kind, B, K, P, counts, labels, targets, loss, grad, ws)
    torch.cuda.synchronize()
    return loss[0].item(), grad.cpu().numpy()


def _noalloc(kind, B, K, P, counts, labels, targets):
    loss = torch.full((4,), float("nan"), dtype=torch.float32, device="cuda")
    grad = torch.full_like(counts, float("nan"))
    snn.snn_loss_noalloc(kind, B, K, P, counts, labels, targets, loss, grad)
    torch.cuda.synchronize()
    return loss[0].item(), grad.cpu().numpy()


# (kind, [(B, K, P) of the first call, then a smaller second call]): the
# cross-entropy sizes take the two-launch path whose row losses go to the
# scratch (more than 128 rows or more than 16 classes); the MSE sizes use
# several first-pass blocks
CASES = [(snn.LOSS_CE_COUNT, [(300, 10, 1), (200, 10, 1)]),
         (snn.LOSS_CE_COUNT, [(1000, 20, 3), (129, 17, 2)]),
         (snn.LOSS_MSE_COUNT, [(64, 5000, 1), (33, 700, 2)])]


@pytest.mark.gpu
@pytest.mark.parametrize("kind,sizes", CASES)
def test_noalloc_equals_workspace_loss(kind, sizes):
    for i, (B, K, P) in enumerate(sizes):
        counts, labels, targets = _inputs(kind, B, K, P, seed=B * 7 + i)
        l_ws, g_ws = _with_workspace(kind, B, K, P, counts, labels, targets)
        l_na, g_na = _noalloc(kind, B, K, P, counts, labels, targets)
        assert np.isfinite(l_ws)
        assert l_na == l_ws, (i, l_na, l_ws)
        np.testing.assert_array_equal(g_na, g_ws)


@pytest.mark.gpu
def test_noalloc_is_an_exported_c_symbol():
    # called directly through ctypes, without the binding's wrapper
    L = ctypes.CDLL(snn.LIB_PATH)
    B, K = 300, 10
    counts, labels, _ = _inputs(snn.LOSS_CE_COUNT, B, K, 1, seed=3)
    loss = torch.empty(4, dtype=torch.float32, device="cuda")
    f = L.snn_loss_noalloc
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_int32] * 4 + [ctypes.c_void_p] * 6
    st = f(snn.LOSS_CE_COUNT, B, K, 1, counts.data_ptr(), labels.data_ptr(), None,
           loss.data_ptr(), None, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert st == 0
    l_ws, _ = _with_workspace(snn.LOSS_CE_COUNT, B, K, 1, counts, labels, None)
    assert loss[0].item() == l_ws

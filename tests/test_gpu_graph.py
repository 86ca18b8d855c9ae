"""The whole training step captured in a HIP graph and replayed.

Each replay must give exactly the bytes of the same step run eagerly (every
kernel sums in a fixed order).  Replays are interleaved with eager work and
synchronisations, and every replay is checked, not only the first.
"""
import numpy as np
import pytest

import paper_2211_10725_amd as snn
from paper_2211_10725_amd import workloads as wls

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda"


def _np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def _outputs(net):
    out = [net.counts, net.loss[:1], net.gcounts]
    out += [t for t in net.spk]
    out += [t for t in net.gW + net.gb + net.gv + net.gx if t is not None]
    return [_np(t).copy() for t in out]


@pytest.mark.parametrize("name,T,B,width", [("dsnn_leaky_t25_b32", 25, 8, None),
                                            ("dsnn_synaptic_t50_b256", 20, 16, 300),
                                            ("csnn_t25_b128", 5, 4, None),
                                            ("dsnn_rleaky_t25_b128", 10, 8, 200),
                                            ("pop_dsnn_t1_b128", 1, 32, None),
                                            ("scan_wide_t1000_b64", 50, 4, 2000),
                                            # the benchmark's default network at full size
                                            ("dsnn_synaptic_t50_b256", 50, 256, None)])
def test_graph_replay_matches_eager(name, T, B, width):
    wl = wls.scaled(wls.get(name), T=T, B=B, width=width)
    lab = tgt = None
    eager = snn.Network(wl, wls.init_params(wl, 0), device=DEV)
    graphed = snn.Network(wl, wls.init_params(wl, 0), device=DEV)
    seeds = [1, 2, 3]
    inputs = []
    for sd in seeds:
        inp = wls.make_inputs(wl, sd)
        inputs.append((torch.as_tensor(inp["x"]).to(DEV),
                       torch.as_tensor(inp["labels"]).to(DEV) if wl.loss == "ce" else None,
                       torch.as_tensor(inp["targets"]).to(DEV) if wl.loss == "mse" else None))
    # the graph reads its inputs from fixed buffers: copy each batch in first
    x_buf = torch.empty_like(inputs[0][0])
    lab_buf = None if inputs[0][1] is None else torch.empty_like(inputs[0][1])
    tgt_buf = None if inputs[0][2] is None else torch.empty_like(inputs[0][2])
    x_buf.copy_(inputs[0][0])
    if lab_buf is not None:
        lab_buf.copy_(inputs[0][1])
    if tgt_buf is not None:
        tgt_buf.copy_(inputs[0][2])
    g = graphed.capture_step(x_buf, lab_buf, tgt_buf)
    torch.cuda.synchronize()
    for rep in range(2):
        for x, lab, tgt in inputs:
            # eager work on the same device between replays
            eager.step(x, labels=lab, targets=tgt)
            want = _outputs(eager)
            x_buf.copy_(x)
            if lab_buf is not None:
                lab_buf.copy_(lab)
            if tgt_buf is not None:
                tgt_buf.copy_(tgt)
            torch.cuda.synchronize()
            g.replay()
            got = _outputs(graphed)
            for i, (a, b) in enumerate(zip(got, want)):
                np.testing.assert_array_equal(a, b, err_msg=f"{name} replay {rep} output {i}")

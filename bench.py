#!/usr/bin/env python
"""Training-step benchmark on one MI355X.

A step is one forward + BPTT pass of the whole spiking network over one batch
of synthetic rate-coded input (synapse and neuron scan per layer, loss on the
output spike counts, then the reverse scan and weight/input gradients per
layer), the quantity the paper times per minibatch (Sec. IV, "Baseline
Throughput") minus the optimizer update.  Default workload: the largest
network, dense 784-4096-4096-10 with Leaky neurons (beta 0.9), T = 100,
batch 512, fp16 weights and spikes with fp32 accumulation and fp32 membrane
state; after it, in the same run, the scan-bound wide layer (65536 Leaky
neurons driven by given currents, T = 1000, batch 64).

Prints one JSON line: samples/s over the timed steps, the roofline of the
stage that takes the most time per step (any stage of the step, forward or
backward; timed with HIP events on the step's stream inside the timed
region), the per-stage time split, the CPU oracle timed on this host, and the
scan-bound layer's own figures under "scan_wide".
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "SNN training samples/sec (fwd+BPTT) at 1 GPU; scan HBM GB/s, GEMM MFMA %"
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E, GB/s
PEAK_FP32_MFMA_TFLOPS = 157.3  # MI355X dense fp32 matrix
# fp32 fma on the vector ALUs without packed math: 256 CUs x 4 SIMDs x 16
# lanes x 2 flops x 2.4 GHz (the packed-fp32 rate, 157.3, is not used)
PEAK_FP32_VALU_TFLOPS = 78.6
PEAK_FP16_MFMA_TFLOPS = 2500.0
DEFAULT_WORKLOAD = "dsnn_half_t100_b512"
SCAN_WORKLOAD = "scan_wide_t1000_b64"


# kernel sources behind each kind of stage (a stored counter profile of a
# stage stays valid while these files are unchanged)
STAGE_SOURCES = {
    "synapse": ["snn_internal.hpp", "gemm.hip", "gemm_mfma16.hip", "gemm_async.hip", "skinny.hip"],
    "conv": ["snn_internal.hpp", "gemm.hip", "gemm_mfma16.hip", "gemm_async.hip", "skinny.hip",
             "conv.hip"],
    "neuron": ["snn_internal.hpp", "neuron.hpp", "scan.hip"],
}


def csrc_hash(files=None) -> str:
    """Hash of kernel sources (all of them, or the named files)."""
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2211_10725_amd", "csrc")
    for f in sorted(files or os.listdir(d)):
        with open(os.path.join(d, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def stage_sources(stage_key: str, workload: str):
    """Kernel sources a stage of a workload runs: a conv layer's synapse
    stages also depend on conv.hip."""
    if not stage_key.startswith("synapse"):
        return STAGE_SOURCES["neuron"]
    from paper_2211_10725_amd import workloads as wls
    m = re.search(r"\[L(\d+)\]", stage_key)
    layers = wls.get(workload).layers if workload in wls.WORKLOADS else []
    conv = m is not None and int(m.group(1)) < len(layers) and \
        layers[int(m.group(1))].get("kind") == "conv"
    return STAGE_SOURCES["conv" if conv else "synapse"]


def stored_traffic(workload: str, stage_key: str):
    """HBM bytes per launch of a stage of a workload from its committed counter
    summary, if the stage's kernel sources are unchanged since the counters
    were taken."""
    path = os.path.join(ROOT, "profiles", f"{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    m = re.search(rf"^\|\s*{re.escape(stage_key)}\s*\|[^|]*\|[^|]*\|[^|]*\|\s*([0-9.eE+]+)\s*\|"
                  rf"\s*([0-9a-f]+)\s*\|", txt, re.M)
    if not m or m.group(2) != csrc_hash(stage_sources(stage_key, workload)):
        return None
    return float(m.group(1))


def _dtype_bytes(code):
    return {0: 4, 1: 2, 2: 2, 3: 1, 4: 0.125}[code]  # 4: spikes packed to bits


def _macs(d):
    """Multiply-adds of a layer's product over all T*B rows (a 5x5 valid conv
    counts Co x Ci x 25 per conv output, every output)."""
    TB = d.T * d.B
    if d.synapse == 1:
        return TB * (d.h_in - 4) * (d.w_in - 4) * d.c_out * d.c_in * 25
    return TB * d.n_out * d.n_in


def stage_work(net, name, li):
    """Algorithmic work of one stage launch: ('flop', F) for contractions,
    ('byte', Bytes) for scans.  Per-unit figures:
      contraction  2 M N K flops (one multiply and one add per MAC); the
                   synapse backward of a dense layer is two stages, dW
                   (K = T*B) and dx (K = n_out), each 2 M N K; a conv layer's
                   backward is one stage with both
      forward scan 4 B read current + s B write spike per (t, b, n) (s = 1
                   for bytes, 2 for fp16 spikes, 1/8 packed to bits), + 4 P B per (b, n) per
                   checkpoint (P = 1 state plane, 2 for the current-based
                   neuron), + 4 B count per (b, n) of the layer that counts
      reverse scan 4 B read current (the membrane is recomputed from it) +
                   4 B read dL/dz (full upstream gradient only) + w B write
                   dL/dI per (t, b, n) (w = 4 for fp32, 2 for a 16-bit
                   gradient operand), + the checkpoints read, + 4 B colsum
                   per (b, n), + 4 B recurrent-weight column sum per (b, n)
                   for recurrent neurons (eq. 7); with the readout's input
                   gradient folded in, dL/dz is not read but computed from
                   the readout's dL/dI (its operand bytes per (t, b, readout
                   neuron))"""
    d = net.descs[li]
    TB = d.T * d.B
    macs = _macs(d)
    if name == "synapse_fwd":
        return "flop", 2.0 * macs
    if name in ("synapse_bwd_dw", "synapse_bwd_dx"):
        return "flop", 2.0 * macs
    if name == "synapse_bwd":
        # conv: dW, and dx below the input layer unless the layer below folds it in
        dx = li > 0 and net.gx[li] is not None
        return "flop", 2.0 * macs * (2 if dx else 1)
    el = TB * d.n_out
    cols = d.B * d.n_out
    lay = net.layouts[li]
    ckpt = 4.0 * lay.ckpt_planes * lay.ckpt_count * cols
    if name == "neuron_fwd":
        counts = 4.0 * cols if li == len(net.descs) - 1 else 0.0
        return "byte", (4.0 + _dtype_bytes(d.out_dtype)) * el + ckpt + counts
    if name == "neuron_bwd":
        rec = 4.0 * cols if d.neuron == 2 else 0.0
        wr = _dtype_bytes(d.grad_dtype) if d.synapse != 2 else 4.0
        colsum = 4.0 * cols if d.synapse != 2 else 0.0
        if net.fold[li]:
            up = net.descs[li + 1]
            return "byte", (4.0 + wr) * el + _dtype_bytes(up.grad_dtype) * TB * up.n_out + \
                ckpt + colsum + rec
        full = li < len(net.descs) - 1
        return "byte", (4.0 + (4.0 if full else 0.0) + wr) * el + ckpt + colsum + rec
    return None, 0.0


def run_pmc_mode(net, x, y, tgt, steps):
    """Kernels for counter collection: a 1 GiB device copy (calibration of
    FETCH_SIZE / WRITE_SIZE against known bytes) and a few training steps
    through the stage calls.  A one-element fill kernel marks every stage
    boundary, so a dispatch list can be cut into stages; the stage names are
    printed in order."""
    import torch
    a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    for _ in range(3):
        b.copy_(a)
    mark = torch.zeros(1, dtype=torch.int32, device="cuda")
    names = []

    def hook(name, li):
        mark.fill_(len(names))
        names.append(f"{name}[L{li}]" if li >= 0 else name)

    for _ in range(steps):
        net.step_stages(x, labels=y, targets=tgt, hook=hook)
    torch.cuda.synchronize()
    print(json.dumps({"pmc_mode": True, "copy_bytes": 2 * (1 << 30), "steps": steps,
                      "csrc_hash": csrc_hash(), "stage_marks": names}))


def macs_per_sample(wl):
    """Multiply-adds of one sample's fwd+BPTT step (contractions), or the
    neuron-update count for a scan-only layer (for sizing the CPU sample)."""
    tot = 0
    for i, s in enumerate(wl.layers):
        if s["kind"] == "dense":
            m = s["n_in"] * s["n_out"]
        elif s["kind"] == "conv":
            # the oracle's direct conv loops run ~8x slower per MAC than its dense ones
            m = 8 * s["c_in"] * 25 * s["c_out"] * (s["h"] - 4) * (s["w"] - 4)
        else:
            m = 4 * s["n"]
        tot += m * (3 if i > 0 else 2)
    return tot * wl.T


def cpu_baseline(wl, seed, target_macs=3.0e11):
    """The oracle as it stands, on this host's cores, on a bounded sample of
    the same workload: B_s samples of identical shape and distribution (B_s
    chosen for roughly ten seconds of oracle work), scaled to samples/s."""
    import oracle
    from paper_2211_10725_amd import workloads as wls
    bs = int(max(1, min(wl.B, round(target_macs / macs_per_sample(wl)))))
    chunks = 1
    if wl.input == "currents":
        # host memory: each sample is T x N currents plus fp64 adjoints, so
        # the scan-only layer runs as steps of 4 samples (samples are
        # independent), as many as fit in about ten seconds
        bs, chunks = min(bs, 4), max(1, wl.B // 4)
    ws_ = wls.scaled(wl, B=bs)
    done, dt = 0, 0.0
    for c in range(chunks):
        inp = wls.make_inputs(ws_, seed + c)
        t0 = time.perf_counter()
        oracle.net_step(ws_.layers, inp["params"], inp["x"], ws_.loss, labels=inp.get("labels"),
                        targets=inp.get("targets"), slope=ws_.slope, pop=ws_.pop)
        dt += time.perf_counter() - t0
        done += bs
        if dt >= 10.0:
            break
    steps = done // bs
    what = (f"{done} of {wl.B} samples" if steps == 1 else
            f"{steps} steps of {bs} samples ({done} of {wl.B})")
    return {"value": round(done / dt, 3), "unit": "samples/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{what} of {wl.name} (T={wl.T}), fwd+BPTT in {dt:.2f} s; C oracle, "
                      f"OpenMP, fp64 contractions"}


def _inputs(wl, seed):
    import torch
    from paper_2211_10725_amd import workloads as wls
    if wl.input == "currents":
        # 4 bytes x T x B x N: drawn directly in device memory
        x = wls.device_currents(wl, seed)
    else:
        x = torch.as_tensor(wls.spike_input(wl, seed)).to("cuda")
    y = torch.as_tensor(wls.labels(wl, seed)).cuda() if wl.loss == "ce" else None
    tgt = torch.as_tensor(wls.targets(wl, seed)).cuda() if wl.loss == "mse" else None
    return x, y, tgt


def _split(net, x, y, tgt, stream, steps, upd=False):
    """Per-stage time (ms, mean over ``steps`` passes through the stage calls,
    outside the timed region), keyed "name[Lli]" ("loss", "update")."""
    import torch
    evs = []

    def rec(name, li):
        e = torch.cuda.Event(enable_timing=True)
        e.record(stream)
        evs.append((name, li, e))

    for _ in range(steps):
        net.step_stages(x, labels=y, targets=tgt, hook=rec, update=upd)
    torch.cuda.synchronize()
    split = {}
    for (n0, l0, e0), (n1, l1, e1) in zip(evs, evs[1:]):
        if n1 == n0 + "_end" and l1 == l0:
            key = f"{n0}[L{l0}]" if l0 >= 0 else n0
            split[key] = split.get(key, 0.0) + e0.elapsed_time(e1) / steps
    return split


def _parse_key(key):
    if "[L" not in key:
        return key, -1
    return key.split("[L")[0], int(key.split("[L")[1].rstrip("]"))


def fused_bench(args, wl, net, x, y, tgt, stream):
    """The step as one snn_fused_step launch per step: the kernel is the whole
    step, so its roofline is the step's contraction flops (hidden currents,
    readout currents, dW0, as exact three-part bf16 MFMA passes) per launch."""
    import torch
    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            net.step_fused(x, labels=y, targets=tgt)
        torch.cuda.synchronize()
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        marks[0].record(stream)
        for i in range(args.steps):
            net.step_fused(x, labels=y, targets=tgt)
            marks[i + 1].record(stream)
        torch.cuda.synchronize()
    if int(net.fstatus[0].item()) != 0:
        print("snn_fused_step gave up at a grid barrier (status 1)", file=sys.stderr)
        sys.exit(1)
    total_ms = marks[0].elapsed_time(marks[-1])
    per_step = sorted(marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps))
    ms = total_ms / args.steps
    h, r = net.descs
    rows = wl.T * wl.B
    flops = 2.0 * rows * (2 * h.n_in * h.n_out + r.n_in * r.n_out)  # algorithmic
    out = {
        "metric": METRIC, "value": round(wl.B * args.steps / (total_ms / 1000.0), 1),
        "unit": "samples/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": wl.name, "description": wl.description, "T": wl.T,
                   "batch": wl.B, "layers": [_layer_str(s) for s in wl.layers],
                   "precision": "fp32 weights, currents, state and gradients; products "
                                "exact, fp32 accumulation",
                   "includes": "forward + loss + BPTT backward, no optimizer update",
                   "launch": "one snn_fused_step kernel per step"},
        "step_ms": {"median": round(per_step[len(per_step) // 2], 5),
                    "p10": round(per_step[len(per_step) // 10], 5),
                    "p90": round(per_step[(9 * len(per_step)) // 10], 5)},
        "roofline": {"bound": "mfma", "achieved": round(flops / (ms / 1000.0) / 1e12, 3),
                     "peak": 2500.0, "unit": "TFLOP/s", "peak_basis": "bf16/fp16 dense MFMA",
                     "mfma_passes": 3,
                     "frac": round(flops / (ms / 1000.0) / 1e12 / 2500.0, 5),
                     "traffic": None, "kernel": "fused_step_kernel (the whole step)",
                     "avg_launch_ms": round(ms, 5), "share_of_step": 1.0},
    }
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--scan-leg", choices=["auto", "on", "off"], default="auto",
                    help="after the main workload, time the scan-bound wide layer in the "
                         "same run (auto: only with the default workload)")
    ap.add_argument("--mode", choices=["bench", "pmc"], default="bench")
    ap.add_argument("--batch", type=int, default=None,
                    help="run the workload at this batch size (same layers and T)")
    ap.add_argument("--graph", action="store_true",
                    help="capture the forward + BPTT step in a HIP graph and time its replays")
    ap.add_argument("--update", action="store_true",
                    help="end every step with the fused AdamW update (the paper's "
                         "training step); the default step is forward + BPTT")
    ap.add_argument("--fused", action="store_true",
                    help="run each step as one snn_fused_step launch (two dense layers on "
                         "spike input with fp32 weights, small batches)")
    ap.add_argument("--fp32-mfma", action="store_true",
                    help="contract spike x fp32 with fp32 MFMA instead of the exact "
                         "three-pass bf16 split")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2211_10725_amd as snn
    from paper_2211_10725_amd import workloads as wls

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    snn.lib()  # fail loudly before anything else if the HIP library is missing
    torch.cuda.set_device(0)
    wl = wls.get(args.workload)
    if args.batch is not None:
        wl = wls.scaled(wl, B=args.batch)
    if args.graph and args.update:
        print("--graph captures the forward + BPTT step only (the AdamW step count is a "
              "host value)", file=sys.stderr)
        sys.exit(2)
    stream = torch.cuda.Stream()  # default priority
    params = wls.init_params(wl, args.seed)
    # a scan-only layer's spikes (read by nothing in the step) packed to bits;
    # an fp32 net's input spikes stored as bf16 0/1 when its first product
    # runs on the asynchronous kernel's three-plane mode (no widening passes)
    l0 = wl.layers[0]
    bf16_in = (wl.dtype == "f32" and l0["kind"] == "dense" and not args.fp32_mfma and
               _async_ok(3, 0, wl.T * wl.B, l0["n_out"], l0["n_in"]))
    net = snn.Network(wl, params, device="cuda",
                      flags=snn.FLAG_FP32_MFMA if args.fp32_mfma else 0,
                      spike_bits=l0["kind"] == "none", input_bf16=bf16_in)
    if args.update:
        net.init_adamw(lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=1e-2)
    upd = bool(args.update)
    with torch.cuda.stream(stream):
        x, y, tgt = _inputs(wl, args.seed)
        if bf16_in:
            x = x.to(torch.bfloat16)
    torch.cuda.synchronize()

    if args.mode == "pmc":
        with torch.cuda.stream(stream):
            run_pmc_mode(net, x, y, tgt, max(1, args.steps))
        return

    if args.fused:
        if net.fdesc is None or args.graph or upd:
            print("--fused runs two dense layers on spike input with fp32 weights, small "
                  "enough for one co-resident grid, without --graph or --update",
                  file=sys.stderr)
            sys.exit(2)
        fused_bench(args, wl, net, x, y, tgt, stream)
        return

    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            net.step_stages(x, labels=y, targets=tgt, update=upd, fused_bwd=True)
        torch.cuda.synchronize()

        # per-stage split (untimed passes through the stage calls): the
        # roofline stage is the one that takes the most time per step, over
        # every stage of the step
        split = _split(net, x, y, tgt, stream, 5, upd)
        cand = {k: v for k, v in split.items() if k != "update"}
        dom_key = max(cand, key=cand.get)
        dom_name, dom_li = _parse_key(dom_key)
        # the backward of the layer holding the roofline stage runs as stage
        # calls (the same kernels in the same order as its one layer call),
        # so that events can bracket that stage
        staged = (dom_li,) if dom_name.startswith(("neuron_bwd", "synapse_bwd")) else ()

        kev = []

        def rec_dom(name, li):
            if li == dom_li and name in (dom_name, dom_name + "_end"):
                e = torch.cuda.Event(enable_timing=True)
                e.record(stream)
                kev.append(e)

        marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        if args.graph:
            graph = net.capture_step(x, labels=y, targets=tgt)
            for _ in range(args.warmup):
                graph.replay()
            torch.cuda.synchronize()
            marks[0].record(stream)
            for i in range(args.steps):
                graph.replay()
                marks[i + 1].record(stream)
            torch.cuda.synchronize()
            # graph replays cannot host events between their kernels: the
            # roofline stage is timed in eager steps right after them
            for _ in range(min(args.steps, 20)):
                net.step_stages(x, labels=y, targets=tgt, hook=rec_dom)
            torch.cuda.synchronize()
        else:
            torch.cuda.synchronize()
            marks[0].record(stream)
            for i in range(args.steps):
                # stage calls forward, one layer call per layer backward
                net.step_stages(x, labels=y, targets=tgt, hook=rec_dom, update=upd,
                                fused_bwd=True, staged=staged)
                marks[i + 1].record(stream)
            torch.cuda.synchronize()
        total_ms = marks[0].elapsed_time(marks[-1])
        per_step = sorted(marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps))
        kms = [kev[i].elapsed_time(kev[i + 1]) for i in range(0, len(kev), 2)]
        k_avg_ms = sum(kms) / len(kms)

    ms_per_step = total_ms / args.steps
    value = wl.B * args.steps / (total_ms / 1000.0)
    roof = _roofline(net, dom_name, dom_li, k_avg_ms, args.fp32_mfma)
    roof["traffic"] = stored_traffic(wl.name, dom_key)
    roof["kernel"] = dom_key + _stage_kernels(net, dom_name, dom_li, args.fp32_mfma)
    roof["avg_launch_ms"] = round(k_avg_ms, 5)
    roof["share_of_step"] = round(cand[dom_key] / sum(cand.values()), 4)
    if args.graph:
        roof["timed"] = "eager steps right after the graph replays"
    half = wl.dtype == "f16"
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "samples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f16" if half else "f32", "data": "synthetic",
        "config": {"workload": wl.name, "description": wl.description, "T": wl.T,
                   "batch": wl.B, "layers": [_layer_str(s) for s in wl.layers],
                   "precision": ("fp16 weights and spikes, fp32 MFMA accumulation, fp32 "
                                 "currents and membrane state, 16-bit dL/dI operand of the "
                                 "backward contractions, fp32 weight gradients") if half else
                                ("fp32 weights, currents, state and gradients; products "
                                 "exact, fp32 accumulation"),
                   "surrogate_slope": wl.slope,
                   "input": ("Bernoulli rate-coded spikes" +
                             (", stored as bf16 0/1" if bf16_in else ""))
                   if wl.input == "spikes" else "normal currents",
                   "includes": "forward + loss + BPTT backward + fused AdamW update"
                   if upd else "forward + loss + BPTT backward, no optimizer update",
                   "launch": "one HIP graph replay per step" if args.graph
                   else "eager library calls",
                   "output_spikes": "packed bits" if net.descs[-1].out_dtype == snn.SPK_BITS
                   else "bytes"},
        "step_ms": {"median": round(per_step[len(per_step) // 2], 5),
                    "p10": round(per_step[len(per_step) // 10], 5),
                    "p90": round(per_step[(9 * len(per_step)) // 10], 5)},
        "roofline": roof,
        "stage_ms": {k: round(v, 5) for k, v in split.items()},
        "stage_roofline": _stage_rooflines(net, split, args.fp32_mfma),
    }
    if upd and split.get("update") and net.opt_tensors:
        # fused AdamW: read param, grad, m, v and write param, m, v (4 B each)
        # per parameter, plus the 2 B fp16 copy of fp16 weights
        nb = sum(28 * t[0].numel() + (2 * t[0].numel() if t[4] is not None else 0)
                 for t in net.opt_tensors)
        gbs = nb / (split["update"] / 1000.0) / 1e9
        out["stage_roofline"]["update"] = {"GB/s": round(gbs, 1),
                                           "frac": round(gbs / PEAK_HBM_GBS, 4),
                                           "bytes": nb}
    syn = sum(v for k, v in split.items() if k.startswith("synapse"))
    neu = sum(v for k, v in split.items() if k.startswith("neuron"))
    out["spiking_vs_synaptic_ms"] = {"neuron_scans": round(neu, 5), "contractions": round(syn, 5)}
    del net, x
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.seed)
    scan_leg = args.scan_leg == "on" or (args.scan_leg == "auto" and
                                         args.workload == DEFAULT_WORKLOAD and
                                         args.batch is None and not args.graph)
    if scan_leg:
        out["scan_wide"] = scan_wide_leg(args, stream)
    print(json.dumps(out), flush=True)


def scan_wide_leg(args, stream):
    """The scan-bound workload in the same run, after the main workload's
    buffers are freed: one Leaky layer of 65536 neurons on given currents
    [T=1000, B=64], forward scan, MSE loss on the counts, reverse scan.  Its
    kernels are HBM-bound; each scan is reported against its algorithmic
    bytes."""
    import torch

    import paper_2211_10725_amd as snn
    from paper_2211_10725_amd import workloads as wls
    wl = wls.get(SCAN_WORKLOAD)
    net = snn.Network(wl, wls.init_params(wl, args.seed), device="cuda", spike_bits=True)
    steps, warm = max(2, min(args.steps, 10)), 5
    with torch.cuda.stream(stream):
        x, y, tgt = _inputs(wl, args.seed)
        for _ in range(warm):
            net.step_stages(x, labels=y, targets=tgt, fused_bwd=True)
        torch.cuda.synchronize()
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        marks[0].record(stream)
        for i in range(steps):
            net.step_stages(x, labels=y, targets=tgt, fused_bwd=True)
            marks[i + 1].record(stream)
        torch.cuda.synchronize()
        total_ms = marks[0].elapsed_time(marks[-1])
        split = _split(net, x, y, tgt, stream, 3)
    el = wl.T * wl.B * wl.layers[0]["n"]
    scans = {}
    for key in ("neuron_fwd[L0]", "neuron_bwd[L0]"):
        name, li = _parse_key(key)
        _, nbytes = stage_work(net, name, li)
        gbs = nbytes / (split[key] / 1000.0) / 1e9
        scans[key] = {"ms": round(split[key], 4), "GB/s": round(gbs, 1),
                      "frac": round(gbs / PEAK_HBM_GBS, 4),
                      "bytes_per_element": round(nbytes / el, 4),
                      "kernel": _stage_kernels(net, name, li, False).lstrip(": ")}
    out = {"workload": wl.name, "description": wl.description, "steps": steps,
           "warmup": warm, "ms_per_step": round(total_ms / steps, 5),
           "value": round(wl.B * steps / (total_ms / 1000.0), 1), "unit": "samples/s",
           "dtype": "f32", "output_spikes": "packed bits",
           "stage_ms": {k: round(v, 5) for k, v in split.items()},
           "scan_roofline": scans}
    del net, x
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.seed)
    return out


def _roofline(net, name, li, ms, fp32_mfma):
    kind, work = stage_work(net, name, li)
    if kind == "flop":
        achieved = work / (ms / 1000.0) / 1e12
        ckind, passes = _contraction_kind(net, li, fp32_mfma, name)
        if ckind == "valu":
            roof = {"bound": "alu", "achieved": round(achieved, 3), "peak": PEAK_FP32_VALU_TFLOPS,
                    "unit": "TFLOP/s", "peak_basis": "fp32 fma on the vector ALUs, no packed math"}
        else:
            if ckind == "mfma16":
                peak, basis = PEAK_FP16_MFMA_TFLOPS, "bf16/fp16 dense MFMA"
            else:
                peak, basis = PEAK_FP32_MFMA_TFLOPS, "fp32 dense MFMA"
            roof = {"bound": "mfma", "achieved": round(achieved, 3), "peak": peak,
                    "unit": "TFLOP/s", "peak_basis": basis, "mfma_passes": passes,
                    "executed_mfma_frac": round(passes * achieved / peak, 4)}
    else:
        achieved = work / (ms / 1000.0) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s"}
    roof["frac"] = round(achieved / roof["peak"], 4)
    roof["algorithmic_per_launch"] = work
    return roof


def _stage_rooflines(net, split, fp32_mfma):
    """Each stage's algorithmic rate against its own roof (scans: GB/s of
    8 TB/s; contractions: TFLOP/s of the MFMA peak of the type they run on),
    from the untimed split pass."""
    out = {}
    for key, ms in split.items():
        if "[L" not in key or ms <= 0:
            continue
        name, li = _parse_key(key)
        kind, work = stage_work(net, name, li)
        if kind == "flop":
            ck, _ = _contraction_kind(net, li, fp32_mfma, name)
            peak = {"mfma16": PEAK_FP16_MFMA_TFLOPS, "valu": PEAK_FP32_VALU_TFLOPS}.get(
                ck, PEAK_FP32_MFMA_TFLOPS)
            a = work / (ms / 1000.0) / 1e12
            out[key] = {"TFLOP/s": round(a, 2), "frac": round(a / peak, 4)}
        elif kind == "byte":
            a = work / (ms / 1000.0) / 1e9
            out[key] = {"GB/s": round(a, 1), "frac": round(a / PEAK_HBM_GBS, 4)}
    return out


# exact 16-bit parts of an operand type on the matrix cores (mirrors the
# operand classification in gemm_mfma16.hip): spikes, bf16 and fp16 (against
# fp16 or spikes) are one part, fp32 three bf16 parts, fp16 against a bf16
# operand two bf16 parts
def _parts(dt, other):
    if dt == 0:
        return 3
    if dt == 1 and other == 2:
        return 2
    return 1


def _contraction_kind(net, li, fp32_mfma, stage="synapse_fwd"):
    """How the library runs a contraction of layer li: ('mfma16', passes),
    ('mfma32', 1) or ('valu', 1).  Mirrors the routing in gemm.hip, api.hip
    and conv.hip.  A conv layer's product has one row per conv output that a
    pool window reads and one column per output channel."""
    d = net.descs[li]
    if stage == "synapse_fwd":
        if _direct_conv(net, li):
            return "valu", 1
        if _narrow_contraction(net, li, fp32_mfma):
            return "mfma16", 3 if d.w_dtype == 0 else 1
        if d.synapse == 1:
            rows = 4 * d.T * d.B * ((d.h_in - 4) // 2) * ((d.w_in - 4) // 2)
            cols = d.c_out
        else:
            rows, cols = d.T * d.B, d.n_out
        wide = rows >= 64 and cols >= 64
        if fp32_mfma or not wide or d.in_dtype not in (1, 2, 3):
            return "mfma32", 1
        return "mfma16", _parts(d.w_dtype, d.in_dtype)
    if stage == "synapse_bwd_dw":
        # dW = dI^T x: dL/dI (grad_dtype) against the layer's input
        if fp32_mfma:
            return "mfma32", 1
        a, b = d.grad_dtype, d.in_dtype
        p = _parts(a, b) * _parts(b, a)
        return ("mfma16", p) if p <= 6 else ("mfma32", 1)
    if stage == "synapse_bwd_dx":
        if fp32_mfma:
            return "mfma32", 1
        a, b = d.grad_dtype, d.w_dtype
        p = _parts(a, b) * _parts(b, a)
        return ("mfma16", p) if p <= 6 else ("mfma32", 1)
    # conv backward: one-pass kernels on the 16-bit cores (dW 3 exact passes,
    # dx 6 part products) where the image fits, else the fp32 contractions
    dx = li > 0 and net.gx[li] is not None
    if _conv_one_pass_fw(net, li, fp32_mfma) and (not dx or _conv_one_pass(net, li, fp32_mfma)):
        return "mfma16", (4.5 if dx else 3)
    return "mfma32", 1


def _conv_one_pass(net, li, fp32_mfma):
    """Whether layer li's conv input gradient runs as conv_dx_kernel: mirrors
    dx_one_pass in conv.hip (at most 12 input and 64 output channels, 16
    pooled cells per channel, 512 pixels)."""
    d = net.descs[li]
    hp, wp = (d.h_in - 4) // 2, (d.w_in - 4) // 2
    return (d.synapse == 1 and not fp32_mfma and d.c_in * 25 <= 320 and d.c_out <= 64
            and hp * wp <= 16 and d.h_in * d.w_in <= 512)


def _conv_one_pass_fw(net, li, fp32_mfma):
    """Whether layer li's conv forward and weight gradient run as
    conv_fwd_kernel and conv_dw_kernel: mirrors dw_one_pass in conv.hip
    (spike input, up to 32 pooled cells, images of whole 4-byte words)."""
    d = net.descs[li]
    hp, wp = (d.h_in - 4) // 2, (d.w_in - 4) // 2
    return (d.synapse == 1 and not fp32_mfma and d.in_dtype == 3 and d.c_in * 25 <= 320
            and d.c_out <= 64 and hp * wp <= 32 and d.h_in * d.w_in <= 512
            and d.c_in * d.h_in * d.w_in % 4 == 0)


def _direct_conv(net, li):
    """Whether layer li's forward runs as the one-kernel convolution and pool
    on the vector ALUs (mirrors the routing in conv.hip: at most 4 input
    channels of 4096 pixels in all, at most 128 output channels)."""
    d = net.descs[li]
    return (d.synapse == 1 and d.c_in <= 4 and d.c_in * d.h_in * d.w_in <= 4096
            and d.c_out <= 128)


def _narrow_contraction(net, li, fp32_mfma):
    """Whether layer li's forward product runs on the kernel for at most 16
    outputs (mirrors narrow_fwd_applies in skinny.hip)."""
    d = net.descs[li]
    if fp32_mfma or d.synapse != 0 or d.n_out > 16 or d.n_in < 256:
        return False
    return (d.in_dtype == 3 and d.w_dtype in (0, 1)) or (d.in_dtype == 1 and d.w_dtype == 1)


def _async_passes(a, b, M, N, K, mn=False):
    """Mirrors gemm_async_applies in gemm_async.hip: 0 when the asynchronous
    256x256 kernel does not take the product, else its MFMA passes (3 for
    spikes against an fp32 operand held as three bf16 planes).  mn: both
    operands M/N-contiguous."""
    if K % 8 or K < 256 or M < 256 or N < 256 or (mn and (M % 8 or N % 8)):
        return 0
    if (a, b) in ((0, 3), (3, 0), (0, 2), (2, 0)):  # fp32 against spikes or bf16
        tiles = -(-M // 256) * -(-N // 256)
        nk = -(-K // 64)
        S = max(1, min(256 // tiles, 3 * nk // 16, 64)) if tiles < 256 else 1
        k_chunk = -(-nk // S) * 64
        splits = -(-K // k_chunk)
        return 3 if tiles * splits >= 192 and M * N * K >= 2 ** 32 else 0
    ok_type = (a in (3, 1) and b in (3, 1)) or (a in (3, 2) and b in (3, 2))
    return 1 if ok_type and M * N * K >= 2 ** 30 else 0


def _async_ok(a, b, M, N, K, mn=False):
    return _async_passes(a, b, M, N, K, mn) > 0


def _async_contraction(net, li, fp32_mfma):
    """Whether layer li's forward product runs on the asynchronous 256x256
    kernel."""
    d = net.descs[li]
    if fp32_mfma or d.synapse != 0:
        return False
    return _async_ok(d.in_dtype, d.w_dtype, d.T * d.B, d.n_out, d.n_in)


def _stage_kernels(net, name, li, fp32_mfma):
    """Kernels a stage enqueues (matched against the rocprofv3 summary)."""
    d = net.descs[li]
    if name == "neuron_fwd":
        return ": neuron_fwd_kernel"
    scale = (" (+ grad_bound_kernel + grad_scale_kernel: the power of two of the fp16 dL/dI)"
             if d.grad_dtype == 1 else "")
    if name == "neuron_bwd" and net.fold[li]:
        return ": neuron_bwd_kernel (the readout's dx folded in) + bias_reduce_kernel" + scale
    if name == "neuron_bwd":
        return ": neuron_bwd_kernel" + (" + bias_reduce_kernel" if d.synapse != 2 else "")
    if name in ("synapse_bwd_dw", "synapse_bwd_dx"):
        kind, passes = _contraction_kind(net, li, fp32_mfma, name)
        M, K = d.T * d.B, d.n_out
        if name == "synapse_bwd_dw":
            if d.n_out <= 16:
                return ": few_rows_mfma_kernel / few_rows_kernel + splitk_reduce_kernel"
            # mirrors dw_plan in api.hip
            sfx = f" ({passes} pass{'es' if passes > 1 else ''}, + splitk_reduce_kernel when split over K)"
            if (not fp32_mfma and d.synapse == 0 and
                    _async_ok(d.grad_dtype, d.in_dtype, d.n_out, d.n_in, M, mn=True)):
                what = ("dL/dI (the 3 bf16 planes the reverse scan writes)" if d.grad_dtype == 0
                        else "dL/dI")
                widen = "widen_kernel (x to 16 bits) + " if d.in_dtype == 3 else ""
                return (f": {widen}gemm_async_kernel reading {what} and x in their own "
                        f"layouts{sfx}")
            big = 2.0 * M * d.n_in * d.n_out >= 2 ** 30
            trans = big and not (d.grad_dtype == 0 and d.in_dtype == 3 and M <= 8192)
            gemm = ("gemm_async_kernel" if trans and
                    _async_ok(d.grad_dtype, d.in_dtype, d.n_out, d.n_in, M) else
                    "gemm16_kernel" if kind == "mfma16" else "gemm_f32_kernel")
            pre = ("transpose_kernel (dL/dI^T" + (" as 3 bf16 planes" if d.grad_dtype == 0
                                                  else "") + ") + transpose_u8_kernel (x^T) + "
                   if trans else "")
            return f": {pre}{gemm}{sfx}"
        big = 2.0 * M * d.n_in * K >= 2 ** 30
        gemm = ("gemm_async_kernel" if big and passes == 1 and
                _async_ok(d.grad_dtype, d.w_dtype, M, d.n_in, K) else
                "gemm16_kernel" if kind == "mfma16" else "gemm_f32_kernel")
        pre = "transpose_kernel (W^T) + " if big and kind == "mfma16" else ""
        return f": {pre}{gemm} ({passes} pass{'es' if passes > 1 else ''}, " \
               "+ splitk_reduce_kernel when split over K)"
    if name == "synapse_bwd":
        one, one_w = _conv_one_pass(net, li, fp32_mfma), _conv_one_pass_fw(net, li, fp32_mfma)
        if one_w:
            dw = "conv_dw_kernel + splitk_reduce_wide_kernel"
        elif d.c_in * 25 <= 75:
            dw = "conv_dw_small_kernel + splitk_reduce_wide_kernel"
        else:
            dw = "unpool_t_kernel + im2col_t_kernel + contraction"
        if not (li > 0 and net.gx[li] is not None):
            return f": {dw} (conv weight gradient)"
        if one:
            return f": {dw} + conv_dx_kernel (conv weight and input gradients)"
        if one_w:
            return (f": {dw} + unpool_t_kernel + contraction + col2im_kernel "
                    "(conv weight and input gradients)")
        return (": unpool_t_kernel + im2col_t_kernel + contractions + col2im_kernel "
                "(conv weight and input gradients)")
    if name == "synapse_fwd" and _async_contraction(net, li, fp32_mfma):
        if d.w_dtype == 0:
            widen = "widen_kernel (spikes to bf16) + " if d.in_dtype == 3 else ""
            return (f": {widen}split_planes_kernel (weights as 3 bf16 planes) + "
                    "gemm_async_kernel (3 passes)")
        widen = " widen_kernel (spikes to fp16) +" if d.in_dtype == 3 else ""
        return f":{widen} gemm_async_kernel"
    if name == "synapse_fwd" and _narrow_contraction(net, li, fp32_mfma):
        return ": narrow_fwd_kernel (16 outputs per MFMA tile, weights staged in LDS)"
    if name == "synapse_fwd" and _direct_conv(net, li):
        return ": conv1_pool_kernel (convolution and pool in one kernel)"
    if name == "synapse_fwd" and _conv_one_pass_fw(net, li, fp32_mfma):
        return ": conv_fwd_kernel (gather, contraction in 3 exact bf16 passes and pool in one kernel)"
    if name == "loss":
        return ": loss kernels"
    kind, passes = _contraction_kind(net, li, fp32_mfma)
    if d.synapse == 1:
        g = "gemm16_kernel" if kind == "mfma16" else "gemm_f32_kernel"
        pool = (" pooling in its epilogue (+ pool_kernel when split over K)" if kind == "mfma16"
                else " + pool_kernel")
        gather = ("im2col_lds_kernel" if d.c_in * d.h_in * d.w_in <= 16384 and d.c_in * 25 <= 1008
                  else "im2col_kernel")
        return f": {gather} + {g}{pool} (the whole stage is timed)"
    if kind == "mfma16" and passes == 3:
        return (": gemm16_kernel, 3 exact bf16 passes (+ split_planes_kernel when the weights"
                " are split into planes up front, + splitk_reduce_kernel when split over K)")
    if kind == "mfma16":
        return ": gemm16_kernel (+ splitk_reduce_kernel when split over K)"
    return ": gemm_f32_kernel (+ splitk_reduce_kernel when split over K)"


def _layer_str(s):
    if s["kind"] == "dense":
        return f"dense {s['n_in']}->{s['n_out']} {s['neuron']}"
    if s["kind"] == "conv":
        return f"conv5 {s['c_in']}->{s['c_out']} pool2 {s['neuron']}"
    return f"scan-only {s['n']} {s['neuron']}"


if __name__ == "__main__":
    main()

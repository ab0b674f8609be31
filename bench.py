#!/usr/bin/env python3
"""Benchmark of the fused training step of the fixed fan-in sparse layer.

One step = one call of ffsl_train_step on one batch: gathered forward, fused
BCE, dW, dbias, dX and Adam over every [L,k] slot of the layer, inputs and
state resident in HBM.  Default workload: the largest label space,
L = 3 145 728 labels, fan-in k = 32, batch B = 64, d = 768, bf16 values, int32
indices, fp32 Adam moments (seeded synthetic data).

Prints one JSON line: throughput in sample*labels/s, the roofline of the main
sweep kernel (its duration measured with HIP events on its own stream), the
SET update measured separately, and the CPU oracle's rate on a bounded sample
of the same workload.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, published


def sweep_source_hash():
    h = hashlib.sha256()
    for name in ("sweep.hip", "sweep_mx.hip", "sweep_wide.hip", "batch_prep.hip", "sweep_dev.h", "ffsl_internal.h"):
        with open(os.path.join(ROOT, "paper_2411_03171_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


class HipEvents:
    """hipEvent_t pairs through the HIP runtime that torch already loaded."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        ev = ctypes.c_void_p()
        rc = self.hip.hipEventCreate(ctypes.byref(ev))
        if rc != 0:
            raise RuntimeError("hipEventCreate failed: %d" % rc)
        return ev

    def record(self, ev, stream):
        rc = self.hip.hipEventRecord(ev, stream)
        if rc != 0:
            raise RuntimeError("hipEventRecord failed: %d" % rc)

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(ms), a, b)
        if rc != 0:
            raise RuntimeError("hipEventElapsedTime failed: %d" % rc)
        return ms.value

    def destroy(self, ev):
        self.hip.hipEventDestroy(ev)


def fused_step_bytes(w, value_bytes):
    """Algorithmic HBM bytes of one fused step: every [L,k] array once.

    read W, I, m, v and write W, m, v per slot; read and write bias, bias_m,
    bias_v per row; X, targets and dX are O(B*d) and left out.
    """
    per_slot = value_bytes + 4 + 4 + 4 + value_bytes + 4 + 4
    return w.L * w.k * per_slot + w.L * 24


def set_bytes(w, value_bytes, n):
    """Algorithmic bytes of one SET update: read W, I; write I, W, m, v at n slots per row."""
    return w.L * (w.k * (value_bytes + 4) + n * (4 + value_bytes + 8))


def load_traffic(workload, src_hash, key="bytes_per_launch"):
    """HBM traffic measured with rocprofv3 counters (per launch of the main
    sweep kernel, or per step over all batch passes), if the profile was taken
    on the current sweep source; else None."""
    path = os.path.join(ROOT, "profiles", "sweep_fused_%s_traffic.json" % workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_hash") != src_hash:
        return None
    return t.get(key)


def time_dense_parts(torch, ffsl, synth, ev, stream, dev, reps):
    """The dense intermediate layer (fwd + bwd) at the C3 shape and the
    auxiliary head (fwd + bwd) at the C5 shape, each timed alone with HIP
    events around the library calls (median of `reps`)."""
    import numpy as np
    lib = ffsl.load()
    rng = np.random.default_rng(3)

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    def median_us(fn):
        fn()
        torch.cuda.synchronize()
        ms = []
        for _ in range(reps):
            a, b = ev.create(), ev.create()
            ev.record(a, stream)
            fn()
            ev.record(b, stream)
            torch.cuda.synchronize()
            ms.append(ev.elapsed_ms(a, b))
            ev.destroy(a)
            ev.destroy(b)
        return sorted(ms)[len(ms) // 2] * 1e3

    out = {}
    # intermediate layer, C3: X [128,768] -> H [128,2048]
    w3 = synth.WORKLOADS["c3_inter2048_L1M"]
    B, din, dout = w3.B, w3.din, w3.d
    X = bf(synth.gen_x(rng, B, din, "layernorm", "bf16"))
    W1 = bf(synth.make_dense(rng, din, dout))
    c = torch.zeros(dout, device=dev)
    A = torch.empty((B, dout), device=dev)
    H = torch.empty((B, dout), dtype=torch.bfloat16, device=dev)
    dH = torch.randn((B, dout), device=dev) * 1e-2
    dW1 = torch.empty((din, dout), device=dev)
    dc = torch.empty(dout, device=dev)
    dX = torch.empty((B, din), device=dev)
    ws = torch.empty(lib.ffsl_dense_workspace_bytes(B, din, dout), dtype=torch.uint8, device=dev)
    p = lambda t: ctypes.c_void_p(t.data_ptr())

    def dense_step():
        ffsl._check(lib.ffsl_dense_gelu_fwd(p(X), B, din, dout, p(W1), p(c), p(A), p(H), p(ws), ws.numel(),
                                            stream))
        ffsl._check(lib.ffsl_dense_gelu_bwd(p(X), B, din, dout, p(W1), p(A), p(dH), p(dW1), p(dc), p(dX), 0,
                                            p(ws), ws.numel(), stream))
    us = median_us(dense_step)
    flops = 3 * 2.0 * B * din * dout
    # W1 read twice, dW1 written, A written and read, H written, dH read, dA written and read
    byts = 2 * din * dout * 2 + din * dout * 4 + B * dout * (4 + 4 + 2 + 4 + 2 + 2)
    out["dense_gelu"] = {"shape": {"B": B, "din": din, "dout": dout}, "us_median": us,
                         "flops": flops, "tflops": flops / (us * 1e-6) / 1e12, "mfma_peak_tflops": 2500.0,
                         "algorithmic_bytes": byts, "gbs": byts / (us * 1e-6) / 1e9}
    # auxiliary head, C5: X [128,768], C = 8192 clusters over L = 1M labels
    w5 = synth.WORKLOADS["c5_aux8192_L1M"]
    B, d, C = w5.B, w5.d, w5.aux_clusters
    X5 = bf(synth.gen_x(rng, B, d, "layernorm", "bf16"))
    Wa = bf(synth.make_dense(rng, d, C))
    ca = torch.zeros(C, device=dev)
    off, lab = synth.gen_targets(rng, B, w5.L, w5.mean_pos, w5.zipf_s)
    offt = torch.from_numpy(off.astype(np.int32)).to(dev)
    labt = torch.from_numpy(lab.astype(np.int32)).to(dev)
    loss = torch.zeros(1, device=dev)
    dWa = torch.empty((d, C), device=dev)
    dca = torch.empty(C, device=dev)
    dX5 = torch.empty((B, d), device=dev)
    ws5 = torch.empty(lib.ffsl_aux_workspace_bytes(B, d, C), dtype=torch.uint8, device=dev)

    def aux_step():
        ffsl._check(lib.ffsl_aux_bce_fwd_bwd(p(X5), B, d, C, w5.L, p(Wa), p(ca), p(offt), p(labt), len(lab),
                                             1.0 / B, p(loss), p(dWa), p(dca), p(dX5), None, 0, p(ws5),
                                             ws5.numel(), stream))
    us = median_us(aux_step)
    flops = 3 * 2.0 * B * d * C
    # Wa read twice, dWa written, the bf16 dlogits written once and read by both products
    byts = 2 * d * C * 2 + d * C * 4 + B * C * (2 + 2 + 2)
    out["aux_head"] = {"shape": {"B": B, "d": d, "C": C}, "us_median": us,
                       "flops": flops, "tflops": flops / (us * 1e-6) / 1e12, "mfma_peak_tflops": 2500.0,
                       "algorithmic_bytes": byts, "gbs": byts / (us * 1e-6) / 1e9}
    return out


def time_composed(torch, ffsl, synth, ev, stream, dev, reps, seed):
    """One whole training step of each workload with dense parts, through
    paper_2411_03171_amd.model: the intermediate layer + sparse layer at the C3
    sizes, the sparse layer + auxiliary head at the C5 sizes (Adam on every
    parameter, no SET).  Each is timed with HIP events around the step (median
    of `reps`), next to the same sparse layer's step alone on an input of its
    width, so the dense parts' share is visible."""
    import numpy as np
    from paper_2411_03171_amd.model import Model

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    def median_ms(fn):
        for t in range(1, 4):
            fn(t)
        torch.cuda.synchronize()
        ms = []
        for t in range(4, 4 + reps):
            a, b = ev.create(), ev.create()
            ev.record(a, stream)
            fn(t)
            ev.record(b, stream)
            torch.cuda.synchronize()
            ms.append(ev.elapsed_ms(a, b))
            ev.destroy(a)
            ev.destroy(b)
        return sorted(ms)[len(ms) // 2]

    out = {}
    for name in ("c3_inter2048_L1M", "c5_aux8192_L1M"):
        w = synth.WORKLOADS[name]
        print("[bench] composed step %s: generating" % name, file=sys.stderr, flush=True)
        inp = synth.make_layer_inputs(w, seed)
        layer = ffsl.SparseLayer(bf(inp.W), torch.from_numpy(inp.I).to(dev),
                                 bias=torch.from_numpy(inp.bias).to(dev), B_max=w.B, nnz_max=len(inp.lab),
                                 unfused=False).bind(w.d)
        X = bf(inp.X)
        off = torch.from_numpy(inp.off.astype(np.int32)).to(dev)
        lab = torch.from_numpy(inp.lab).to(dev)
        if w.din:
            model = Model(layer, W1=bf(synth.make_intermediate(w, seed)), c=torch.zeros(w.d, device=dev))
            Xs = bf(synth.gen_x(np.random.default_rng(seed + 1), w.B, w.d, "layernorm", "bf16"))
        else:
            model = Model(layer, Wa=bf(synth.make_aux(w, seed)), ca=torch.zeros(w.aux_clusters, device=dev),
                          aux_w0=1.0, aux_cutoff_epoch=None)
            Xs = X
        ms = median_ms(lambda t: model.train_step(X, off, lab, t))
        ms_sparse = median_ms(lambda t: layer.train_step(Xs, off, lab, t))
        # the sparse layer's step against the HBM roofline: every [L,k] array
        # once (as for the main workload); traffic from the counters when a
        # profile of the current source holds it (bytes per step, all passes)
        sb = fused_step_bytes(w, 2 if w.value == "bf16" else 4)
        sgbs = sb / (ms_sparse * 1e-3) / 1e9
        straffic = load_traffic(w.name, sweep_source_hash(), key="bytes_per_step")
        out[name] = {"ms_median": ms, "sparse_ms_median": ms_sparse, "dense_parts_ms": ms - ms_sparse,
                     "value": w.B * w.L / (ms * 1e-3), "unit": "sample*labels/s",
                     "sparse_roofline": {"bound": "hbm", "achieved": sgbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                         "frac": sgbs / HBM_PEAK_GBS, "algorithmic_bytes": sb,
                                         "traffic": straffic,
                                         "note": "whole sparse step (all batch passes, dX reduction) timed"},
                     "shape": {"L": w.L, "k": w.k, "B": w.B, "d": w.d, "din": w.din,
                               "aux_clusters": w.aux_clusters}}
        print("[bench] composed step %s: %.3f ms (sparse layer alone %.3f ms)" % (name, ms, ms_sparse),
              file=sys.stderr, flush=True)
        layer.close()
        del model, layer, X, Xs
        torch.cuda.synchronize()
    return out


def time_c2_run(torch, ffsl, synth, dev, seed):
    """The C2 workload's whole run: 100 fused training steps on fresh seeded
    batches (all uploaded before the timed region), SET fused into the step
    after every 20th (ffsl_train_step_set), timed with torch events around
    the run."""
    import numpy as np
    w = synth.WORKLOADS["c2_bf16_L131072"]

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    inp = synth.make_layer_inputs(w, seed)
    host = synth.make_batches(w, w.steps, seed)
    batches = [(bf(X), torch.from_numpy(off.astype(np.int32)).to(dev), torch.from_numpy(lab).to(dev))
               for X, off, lab in host]
    nnz_max = max(len(b[2]) for b in host)
    layer = ffsl.SparseLayer(bf(inp.W), torch.from_numpy(inp.I).to(dev), bias=torch.from_numpy(inp.bias).to(dev),
                             B_max=w.B, nnz_max=nnz_max, unfused=False).bind(w.d)
    loss = torch.empty(1, device=dev)
    dX = torch.empty((w.B, w.d), device=dev)
    ex = torch.zeros(1, dtype=torch.int32, device=dev)

    def run():
        for t in range(1, w.steps + 1):
            X, off, lab = batches[t - 1]
            if t % w.set_every == 0:
                layer.train_step_set(X, off, lab, t, w.set_frac, seed, t // w.set_every, loss_out=loss, dX_out=dX,
                                     mask=False, exhausted_out=ex)
            else:
                layer.train_step(X, off, lab, t, loss_out=loss, dX_out=dX)

    run()   # a first run warms up; the timed run continues from its state
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    run()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b)
    out = {"steps": w.steps, "set_every": w.set_every, "set_frac": w.set_frac, "ms_total": ms,
           "ms_per_step": ms / w.steps, "value": w.B * w.L * w.steps / (ms * 1e-3), "unit": "sample*labels/s",
           "exhausted_rows": int(ex.cpu()[0]),
           "shape": {"L": w.L, "k": w.k, "B": w.B, "d": w.d}}
    layer.close()
    return out


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def cpu_threads():
    """Threads for the multi-core leg: the CPU share this process may use
    (affinity), at most 16 (one GPU's share of the box)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(n, os.cpu_count() or 1, 16))


def cpu_baseline(w, inp, target_s=5.0, set_target_s=2.0):
    """The oracle (float64, plain loops, unchanged) on bounded samples of the
    same workload, three legs:
      - single thread: one fused step (forward, BCE, dW, dbias, dX, Adam) on a
        block of label rows;
      - multi-core: the same call on T disjoint row blocks at once, one thread
        per block (the oracle's C calls release the GIL; the blocks' dX
        partials would add up to the step's dX);
      - SET: one prune-and-regrow round on a block of rows.
    Each block is calibrated to about target_s seconds of work."""
    import concurrent.futures as cf

    import numpy as np

    import oracle
    from paper_2411_03171_amd import synth
    oracle.build()
    X = synth.bf16_bits_to_f32(inp.X).astype(np.float64) if w.value == "bf16" else \
        inp.X.astype(np.float64)
    W = synth.bf16_bits_to_f32(inp.W).astype(np.float64) if w.value == "bf16" else \
        inp.W.astype(np.float64)

    def targets(r0, Ls):
        off = np.zeros(w.B + 1, dtype=np.int64)
        labs = []
        for b in range(w.B):
            seg = inp.lab[inp.off[b]:inp.off[b + 1]]
            seg = seg[(seg >= r0) & (seg < r0 + Ls)] - r0
            labs.append(seg)
            off[b + 1] = off[b] + len(seg)
        return off, np.concatenate(labs).astype(np.int32)

    def step(r0, Ls):
        off, lab = targets(r0, Ls)
        sl = slice(r0, r0 + Ls)
        t0 = time.perf_counter()
        oracle.train_step(X, W[sl], inp.I[sl], np.zeros(Ls), np.zeros((Ls, w.k)), np.zeros((Ls, w.k)),
                          np.zeros(Ls), np.zeros(Ls), off, lab, 1.0 / w.B, t=1, w_bf16=(w.value == "bf16"))
        return time.perf_counter() - t0

    # single thread, calibrated
    Ls = min(w.L, 16384)
    dt = step(0, Ls)
    Ls = int(min(w.L, max(Ls, Ls * target_s / max(dt, 1e-3))))
    dt = step(0, Ls)
    single = w.B * Ls / dt

    # multi-core: T blocks of Lb rows in T threads
    T = cpu_threads()
    Lb = max(1, min(Ls, w.L // T))
    with cf.ThreadPoolExecutor(max_workers=T) as ex:
        t0 = time.perf_counter()
        list(ex.map(lambda p: step(p * Lb, Lb), range(T)))
        dt_mc = time.perf_counter() - t0
    multi = w.B * T * Lb / dt_mc

    # SET: one round on a block of rows (fraction mode, the workload's fraction)
    Wbits = inp.W if w.value == "bf16" else inp.W.view(np.uint32)
    zeros = None

    def set_round(Lr):
        nonlocal zeros
        if zeros is None or zeros.shape[0] < Lr:
            zeros = np.zeros((Lr, w.k), dtype=np.float32)
        t0 = time.perf_counter()
        oracle.set_update(Wbits[:Lr], inp.I[:Lr], zeros[:Lr], zeros[:Lr], w.d, w.set_frac, 7, 0)
        return time.perf_counter() - t0

    Lr = min(w.L, 65536)
    ds = set_round(Lr)
    Lr = int(min(w.L, max(Lr, Lr * set_target_s / max(ds, 1e-3))))
    ds = set_round(Lr)
    return {
        "value": multi,
        "unit": "sample*labels/s",
        "cores": T,
        "kind": "oracle",
        "sample": "one fused step (forward, BCE, dW, dbias, dX, Adam; float64) of the oracle on %d disjoint "
                  "blocks of %d label rows of the workload (same X, targets restricted to each block), one "
                  "thread per block, %.1f s wall" % (T, Lb, dt_mc),
        "single_thread": {"value": single, "unit": "sample*labels/s", "cores": 1,
                          "sample": "first %d of %d label rows, %.1f s" % (Ls, w.L, dt)},
        "set": {"rows_per_s": Lr / ds, "s_per_full_set": w.L * ds / Lr, "cores": 1,
                "sample": "one SET round (fraction %g) on the first %d of %d rows, %.1f s" % (w.set_frac, Lr,
                                                                                             w.L, ds)},
        "cpu_model": cpu_model(),
        "cpu_count": os.cpu_count(),
    }


def sweep_kernel_name(w):
    """The kernel the library picks for the fused step of this workload."""
    if w.value == "bf16" and w.k == 32 and w.d % 128 == 0 and 128 <= w.d <= 768:
        return "k_sweep_mx (fused bf16 fan-in-32 path, %d pass(es) of 64 samples)" % ((w.B + 63) // 64)
    if w.value == "bf16" and w.k == 64 and w.d % 128 == 0 and 128 <= w.d <= 2048 and w.L < (1 << 24):
        return "k_sweep_wide (fused bf16 fan-in-64 path, %d pass(es) of 16 samples)" % ((w.B + 15) // 16)
    return "k_sweep (fused mode)"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="c4_bf16_L3M")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--set-reps", type=int, default=10)
    ap.add_argument("--dense-reps", type=int, default=20)
    ap.add_argument("--idx16-reps", type=int, default=10,
                    help="timed steps and inference calls of the same layer with 16-bit indices (0 skips)")
    ap.add_argument("--infer-reps", type=int, default=10,
                    help="timed top-k inference calls (0 skips them)")
    ap.add_argument("--hinge-reps", type=int, default=10,
                    help="squared hinge steps per case (0 skips them, e.g. under a kernel trace "
                         "whose per-kernel average should cover the BCE step only)")
    ap.add_argument("--copy-reps", type=int, default=5,
                    help="timed 1 GiB device copies for the achievable streaming rate (0 skips them)")
    ap.add_argument("--c2-run", type=int, default=1,
                    help="time the C2 workload's 100-step run with SET every 20 steps (0 skips it)")
    ap.add_argument("--composed-reps", type=int, default=5,
                    help="whole steps of the workloads with dense parts, each (0 skips them)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sparse-only", action="store_true",
                    help="for a workload with dense parts, time its sparse layer alone (at the "
                         "layer's own input width)")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="run one plain device copy of this size first (counter calibration)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this build runs on one GPU; the label-sharded multi-GPU layout is "
              "designed but not built, so --gpus must be 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2411_03171_amd import ffsl, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    ffsl.load()
    dev = "cuda:0"
    w = synth.WORKLOADS[args.workload]
    if w.din or w.aux_clusters:
        if not args.sparse_only:
            print("bench.py: workload %s has dense parts; the fused-step bench runs the sparse "
                  "workloads (or the sparse layer alone with --sparse-only)" % w.name, file=sys.stderr)
            sys.exit(2)
        w = synth.dataclasses.replace(w, din=0, aux_clusters=0)
    print("[bench] generating %s (L=%d k=%d B=%d d=%d %s)" % (w.name, w.L, w.k, w.B, w.d, w.value),
          file=sys.stderr, flush=True)
    inp = synth.make_layer_inputs(w, args.seed)
    vb = 2 if w.value == "bf16" else 4

    def to_dev(a):
        if w.value == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)

    layer = ffsl.SparseLayer(to_dev(inp.W), torch.from_numpy(inp.I).to(dev),
                             bias=torch.from_numpy(inp.bias).to(dev), B_max=w.B,
                             nnz_max=len(inp.lab), unfused=False).bind(w.d)
    X = to_dev(inp.X)
    off = torch.from_numpy(inp.off.astype(np.int32)).to(dev)
    lab = torch.from_numpy(inp.lab).to(dev)
    loss = torch.empty(1, device=dev)
    dX = torch.empty((w.B, w.d), device=dev)
    torch.cuda.synchronize()
    print("[bench] state resident: %.1f MB" % (torch.cuda.memory_allocated() / 1e6),
          file=sys.stderr, flush=True)

    if args.copy_probe_mb:
        # a plain copy of known size: under rocprofv3 --pmc its FETCH_SIZE and
        # WRITE_SIZE give the counters' scale for the sweep kernel's traffic
        nb = args.copy_probe_mb << 20
        src = torch.empty(nb // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        print("[bench] copy probe: %d MiB read + %d MiB written" % (args.copy_probe_mb,
              args.copy_probe_mb), file=sys.stderr, flush=True)

    ev = HipEvents()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    t = 0
    for _ in range(args.warmup):
        t += 1
        layer.train_step(X, off, lab, t=t, loss_out=loss, dX_out=dX)
    torch.cuda.synchronize()
    print("[bench] warmup done (%d steps)" % args.warmup, file=sys.stderr, flush=True)

    starts = [ev.create() for _ in range(args.steps)]
    stops = [ev.create() for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        t += 1
        layer.set_timing_events(starts[i], stops[i])
        layer.train_step(X, off, lab, t=t, loss_out=loss, dX_out=dX)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    layer.set_timing_events(None, None)
    kern_ms = [ev.elapsed_ms(a, b) for a, b in zip(starts, stops)]
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    kern_avg_ms = sum(kern_ms) / len(kern_ms)
    final_loss = float(loss.cpu()[0])
    print("[bench] timed %d steps: %.3f ms/step, sweep kernel %.3f ms avg, loss %.5f" %
          (args.steps, ms_per_step, kern_avg_ms, final_loss), file=sys.stderr, flush=True)

    # device memory held for the step: the layer state, its workspace and the
    # batch (torch's peak counter; the paper's memory metric)
    peak_mem = int(torch.cuda.max_memory_allocated())
    state_bytes = ffsl.footprint_bytes(w.L, w.k, vb, bias=True)
    step_bytes = fused_step_bytes(w, vb)
    achieved = step_bytes / (kern_avg_ms * 1e-3) / 1e9
    src_hash = sweep_source_hash()
    traffic = load_traffic(w.name, src_hash)

    # SET, measured separately (no mask output; one kernel per call)
    n_set = int(np.floor(w.set_frac * w.k + 1e-9))
    set_ms = []
    exhausted = torch.zeros(1, dtype=torch.int32, device=dev)
    for r in range(args.set_reps):
        a, b = ev.create(), ev.create()
        ev.record(a, stream)
        layer.set_update(w.set_frac, seed=args.seed, set_round=r, mask=False, exhausted_out=exhausted)
        ev.record(b, stream)
        torch.cuda.synchronize()
        set_ms.append(ev.elapsed_ms(a, b))
    sb = set_bytes(w, vb, n_set)
    set_ms_med = sorted(set_ms)[len(set_ms) // 2] if set_ms else None
    set_gbs = sb / (set_ms_med * 1e-3) / 1e9 if set_ms else None
    if set_ms:
        print("[bench] SET: %.3f ms median, %.0f GB/s algorithmic, exhausted rows %d" %
              (set_ms_med, set_gbs, int(exhausted.cpu()[0])), file=sys.stderr, flush=True)

    # SET fused into a training step (one call) against a plain step, both
    # timed alone with events: the marginal cost of a SET step
    def one_step(fn):
        a, b = ev.create(), ev.create()
        ev.record(a, stream)
        fn()
        ev.record(b, stream)
        torch.cuda.synchronize()
        return ev.elapsed_ms(a, b)

    plain_ms, fused_ms = [], []
    for r in range(args.set_reps):
        t += 1
        plain_ms.append(one_step(lambda: layer.train_step(X, off, lab, t=t, loss_out=loss, dX_out=dX)))
        t += 1
        fused_ms.append(one_step(lambda: layer.train_step_set(X, off, lab, t=t, frac=w.set_frac, seed=args.seed,
                                                              set_round=1000 + r, loss_out=loss, dX_out=dX,
                                                              mask=False, exhausted_out=exhausted)))
    plain_med = sorted(plain_ms)[len(plain_ms) // 2] if plain_ms else None
    fused_med = sorted(fused_ms)[len(fused_ms) // 2] if fused_ms else None
    if fused_ms:
        print("[bench] step with SET in one call: %.3f ms median (plain step %.3f ms): SET adds %.3f ms" %
              (fused_med, plain_med, fused_med - plain_med), file=sys.stderr, flush=True)

    # the squared hinge (same step, other loss): scores near zero give a
    # dlogit everywhere; a bias of -4 puts every label without a positive in
    # the batch past the margin, so waves with no positive skip their dW work
    hinge = {"dense_dlogits": None, "past_margin": None}
    bias_saved = layer.bias.clone()
    for case, fill in (("dense_dlogits", None), ("past_margin", -4.0)) if args.hinge_reps > 0 else ():
        if fill is not None:
            layer.bias.fill_(fill)
        hm = []
        for r in range(args.hinge_reps):
            t += 1
            hm.append(one_step(lambda: layer.train_step(X, off, lab, t=t, loss_out=loss, dX_out=dX,
                                                        flags=ffsl.FFSL_LOSS_SQHINGE)))
        hinge[case] = sorted(hm)[len(hm) // 2]
    layer.bias.copy_(bias_saved)
    torch.cuda.synchronize()
    if args.hinge_reps > 0:
        print("[bench] squared hinge step: %.3f ms (dense dlogits), %.3f ms (past the margin); BCE %s ms" %
              (hinge["dense_dlogits"], hinge["past_margin"], "%.3f" % plain_med if plain_med else "-"),
              file=sys.stderr, flush=True)

    # inference over the whole label space: each sample's top 5 labels and
    # P@1..P@5 (the scores never reach memory)
    infer = None
    if args.infer_reps > 0:
        K_INF = 5
        lib = ffsl.load()
        ws_inf = torch.empty(max(int(lib.ffsl_topk_workspace_bytes(layer._handle, w.B, K_INF)), 256),
                             dtype=torch.uint8, device=dev)
        layer.infer_topk(X, K_INF, off, lab, workspace=ws_inf)   # first call sets the kernel up
        torch.cuda.synchronize()
        im = sorted(one_step(lambda: layer.infer_topk(X, K_INF, off, lab, workspace=ws_inf))
                    for _ in range(args.infer_reps))
        single_ms = im[len(im) // 2]

        # back-to-back calls between two events, as a serving loop issues them
        # (the timed training steps run the same way): the host's setup of a
        # call overlaps the previous call's kernels
        def infer_calls():
            for _ in range(args.infer_reps):
                layer.infer_topk(X, K_INF, off, lab, workspace=ws_inf)
        inf_ms = one_step(infer_calls) / args.infer_reps
        inf_bytes = w.L * w.k * (vb + 4) + 4 * w.L + w.B * w.d * vb
        inf_gbs = inf_bytes / (inf_ms * 1e-3) / 1e9
        # every (label row, slot, sample) reads one X value from LDS
        lds_bytes = w.L * w.k * w.B * vb
        infer = {"topk": K_INF, "ms_per_call": inf_ms, "calls": args.infer_reps,
                 "ms_median_single_call": single_ms, "algorithmic_bytes": inf_bytes, "achieved": inf_gbs,
                 "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": inf_gbs / HBM_PEAK_GBS,
                 "lds_gather_bytes": lds_bytes,
                 "sample_labels_per_s": w.B * w.L / (inf_ms * 1e-3)}
        print("[bench] inference top-%d: %.3f ms per call over %d back-to-back calls (%.3f ms median of single "
              "calls), %.0f GB/s algorithmic (%.1f%% of HBM peak)" %
              (K_INF, inf_ms, args.infer_reps, single_ms, inf_gbs, 100 * inf_gbs / HBM_PEAK_GBS),
              file=sys.stderr, flush=True)

    # the same layer with 16-bit indices (2 bytes per slot less): the fused
    # step and the inference call
    idx16 = None
    if args.idx16_reps > 0:
        I16 = torch.from_numpy(inp.I.astype(np.uint16).view(np.int16)).to(dev)
        layer16 = ffsl.SparseLayer(layer.W.clone(), I16, bias=layer.bias.clone(), B_max=w.B,
                                   nnz_max=len(inp.lab), unfused=False).bind(w.d)
        # the two layers' calls interleaved, so both medians come from the same
        # stretch of time
        t16 = 0
        for _ in range(5):
            t16 += 1
            layer16.train_step(X, off, lab, t=t16, loss_out=loss, dX_out=dX)
        st, st32 = [], []
        for _ in range(args.idx16_reps):
            t16 += 1
            st.append(one_step(lambda: layer16.train_step(X, off, lab, t=t16, loss_out=loss, dX_out=dX)))
            t += 1
            st32.append(one_step(lambda: layer.train_step(X, off, lab, t=t, loss_out=loss, dX_out=dX)))
        st16 = sorted(st)[len(st) // 2]
        b16 = step_bytes - w.L * w.k * 2
        idx16 = {"step_ms_median": st16, "step_algorithmic_bytes": b16,
                 "step_achieved": b16 / (st16 * 1e-3) / 1e9,
                 "int32_step_ms_median": sorted(st32)[len(st32) // 2]}
        if infer is not None:
            layer16.infer_topk(X, 5, off, lab, workspace=ws_inf)
            torch.cuda.synchronize()
            im16, im32 = [], []
            for _ in range(args.idx16_reps):
                im16.append(one_step(lambda: layer16.infer_topk(X, 5, off, lab, workspace=ws_inf)))
                im32.append(one_step(lambda: layer.infer_topk(X, 5, off, lab, workspace=ws_inf)))
            idx16["infer_ms_median"] = sorted(im16)[len(im16) // 2]
            idx16["int32_infer_ms_median"] = sorted(im32)[len(im32) // 2]
            idx16["infer_algorithmic_bytes"] = infer["algorithmic_bytes"] - w.L * w.k * 2
        print("[bench] 16-bit indices: step %.3f ms (%.3f GB) vs %.3f ms int32; inference %s ms vs %s ms" %
              (st16, b16 / 1e9, idx16["int32_step_ms_median"],
               "%.3f" % idx16["infer_ms_median"] if "infer_ms_median" in idx16 else "-",
               "%.3f" % idx16["int32_infer_ms_median"] if "infer_ms_median" in idx16 else "-"),
              file=sys.stderr, flush=True)
        del layer16, I16
        torch.cuda.synchronize()

    dense = {"dense_gelu": None, "aux_head": None}
    if args.dense_reps > 0:
        dense = time_dense_parts(torch, ffsl, synth, ev, stream, dev, args.dense_reps)
        print("[bench] dense GELU layer (C3 shape): %.1f us fwd+bwd; aux head (C5 shape): %.1f us" %
              (dense["dense_gelu"]["us_median"], dense["aux_head"]["us_median"]), file=sys.stderr, flush=True)

    # the achievable streaming rate on this device: a plain 1 GiB device copy
    # (read + write), median of a few, event-timed
    copy = None
    if args.copy_reps > 0:
        nb = 1 << 30
        src = torch.empty(nb // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        dst.copy_(src)
        cms = []
        for _ in range(args.copy_reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            dst.copy_(src)
            b.record()
            torch.cuda.synchronize()
            cms.append(a.elapsed_time(b))
        del src, dst
        cmed = sorted(cms)[len(cms) // 2]
        copy = {"bytes": 2 * nb, "ms_median": cmed, "gbs": 2 * nb / (cmed * 1e-3) / 1e9}
        print("[bench] device copy: %.0f GB/s (read + write)" % copy["gbs"], file=sys.stderr, flush=True)

    c2_run = None
    if args.c2_run:
        c2_run = time_c2_run(torch, ffsl, synth, dev, args.seed)
        print("[bench] C2 run: %d steps with SET every %d in %.2f ms (%.3f ms/step)" %
              (c2_run["steps"], c2_run["set_every"], c2_run["ms_total"], c2_run["ms_per_step"]),
              file=sys.stderr, flush=True)

    composed = None
    if args.composed_reps > 0:
        composed = time_composed(torch, ffsl, synth, ev, stream, dev, args.composed_reps, args.seed)

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, inp)
        print("[bench] oracle: %.3e sample*labels/s on %d threads (%s); single thread %.3e; SET %.1f s per "
              "full round" % (cpu["value"], cpu["cores"], cpu["sample"], cpu["single_thread"]["value"],
                              cpu["set"]["s_per_full_set"]), file=sys.stderr, flush=True)

    value = w.B * w.L / (ms_per_step * 1e-3)
    out = {
        "metric": "sample*labels/s of the fused fwd+BCE+bwd+Adam step",
        "value": value,
        "unit": "sample*labels/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.value,
        "data": "synthetic (seeded; Zipf targets, LayerNorm-ed Gaussian X; no dataset)",
        "config": {"workload": w.name, "L": w.L, "k": w.k, "B": w.B, "d": w.d,
                   "values": w.value, "indices": "int32", "moments": "fp32",
                   "positives_mean": w.mean_pos, "zipf_s": w.zipf_s},
        "roofline": {
            "bound": "hbm",
            "kernel": sweep_kernel_name(w),
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": step_bytes,
            "kernel_ms_avg": kern_avg_ms,
            "kernel_ms_median": sorted(kern_ms)[len(kern_ms) // 2],
            "kernel_ms_min": min(kern_ms),
            "source_hash": src_hash,
            "frac_of_copy": achieved / copy["gbs"] if copy else None,
        },
        "copy_peak": copy,
        "memory": {"peak_allocated_bytes": peak_mem, "layer_state_bytes": state_bytes,
                   "note": "torch.cuda.max_memory_allocated after the timed steps (state, workspace, batch)"},
        "set_update": {
            "ms_median": set_ms_med,
            "algorithmic_bytes": sb,
            "achieved": set_gbs,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": set_gbs / HBM_PEAK_GBS,
            "frac_of_copy": set_gbs / copy["gbs"] if copy else None,
            "prune_per_row": n_set,
        } if set_ms else None,
        "set_in_step": {
            "ms_median": fused_med,
            "plain_step_ms_median": plain_med,
            "marginal_ms": fused_med - plain_med,
            "note": "ffsl_train_step_set: SET applied in the sweep that applies Adam",
        } if fused_ms else None,
        "sqhinge_step": {
            "ms_median_dense_dlogits": hinge["dense_dlogits"],
            "ms_median_past_margin": hinge["past_margin"],
            "bce_step_ms_median": plain_med,
            "note": "FFSL_LOSS_SQHINGE; past_margin: bias -4, dW work skipped where a wave has no dlogit",
        },
        "infer_topk": infer,
        "idx16": idx16,
        "dense_gelu": dense["dense_gelu"],
        "aux_head": dense["aux_head"],
        "composed_step": composed,
        "c2_run": c2_run,
        "cpu_baseline": cpu,
        "loss": final_loss,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

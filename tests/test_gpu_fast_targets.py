"""Targets on the fused fast paths, whose positives are sorted once per call
into per-pass key lists: no positives, a sample without positives, repeated
labels, labels outside [0,L) (ignored, as the header states), and positive
counts at and just past the 1024 the sweeps keep on chip (beyond it they scan
the CSR arrays).  Loss, dX and dW (read from the first Adam moment,
m = (1 - beta1) dW when it starts at zero) are checked against the oracle run
on the in-range labels."""
import numpy as np
import pytest

import oracle
from paper_2411_03171_amd import synth
from parity import assert_close, batch_to_gpu, make_gpu_layer, note, rtol_for, values_f64

pytestmark = pytest.mark.gpu

W1 = synth.WORKLOADS

SHAPES = {
    # fan-in 32 at d = 768: two batch passes of 64 samples
    "mx": synth.scaled(W1["c4_bf16_L3M"], L=700, B=100, name="mx_targets"),
    # fan-in 64 on the wide path: three passes of 16 samples, the last ragged
    "wide": synth.dataclasses.replace(synth.scaled(W1["c3_inter2048_L1M"], L=500, d=256, B=40,
                                                   name="wide_targets"), din=0),
}


def target_sets(B, L, rng):
    """(name, off, lab) triples; lab may hold labels outside [0,L)."""
    sets = [("none", np.zeros(B + 1, dtype=np.int64), np.zeros(0, dtype=np.int32))]
    per = [[3, 3, 3], [], [-1, L, L + 7, 0], [L - 1]]
    per += [list(rng.integers(0, L, size=rng.integers(0, 4))) for _ in range(B - len(per))]
    sets.append(("edge",) + csr(per))
    for n in (1024, 1025):
        samples = np.sort(rng.integers(0, B, size=n))
        labels = rng.integers(0, L, size=n)
        per = [list(labels[samples == b]) for b in range(B)]
        sets.append(("n%d" % n,) + csr(per))
    return sets


def csr(per):
    off = np.zeros(len(per) + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(p) for p in per])
    lab = np.array([x for p in per for x in p], dtype=np.int32)
    return off, lab


def in_range(off, lab, L):
    keep = (lab >= 0) & (lab < L)
    per = [lab[off[b]:off[b + 1]][keep[off[b]:off[b + 1]]] for b in range(len(off) - 1)]
    return csr([list(p) for p in per])


@pytest.mark.parametrize("shape", sorted(SHAPES))
def test_fast_path_targets(shape):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    w = SHAPES[shape]
    inp = synth.make_layer_inputs(w, 5)
    rng = np.random.default_rng(11)
    bias = (rng.standard_normal(w.L) * 0.1).astype(np.float32)
    X64 = values_f64(inp.X, w.value)
    W64 = values_f64(inp.W, w.value)
    rtol = rtol_for(w.value)
    s = 1.0 / w.B
    b1 = 0.9
    for name, off, lab in target_sets(w.B, w.L, rng):
        note("fast-path targets %s %s nnz=%d" % (shape, name, len(lab)))
        layer = make_gpu_layer(inp, w, bias_values=bias, unfused=False, nnz_max=max(len(lab), 1))
        X, offt, labt = batch_to_gpu(inp.X, off, lab, w.value)
        loss, dX = layer.train_step(X, offt, labt, t=1, s=s, beta1=b1)
        torch.cuda.synchronize()
        off_r, lab_r = in_range(off, lab, w.L)
        ref = oracle.loss_and_grads(X64, W64, inp.I, bias.astype(np.float64), off_r, lab_r, s)
        assert_close(loss.cpu().numpy()[0], ref["loss"], rtol, "loss " + name)
        assert_close(dX.cpu().numpy(), ref["dX"], rtol, "dX " + name)
        assert_close(layer.m.cpu().numpy() / (1.0 - b1), ref["dW"], rtol, "dW " + name)
        assert_close(layer.bias_m.cpu().numpy() / (1.0 - b1), ref["dbias"], rtol, "dbias " + name)

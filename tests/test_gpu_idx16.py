"""16-bit indices (ffsl_create_layer_ex with FFSL_IDX_U16, Sec. 2.2's
16-bit index storage).  Against the oracle directly: the u16 layer's training
step (fused and unfused), its SET in both prune modes and the fused step with
SET (bit-exact on every row), and its top-k inference.  Against the same
layer with int32 indices: every call must give the same results -- the
storage differs, the arithmetic does not.  Compared bit for bit
(weights, indices, moments, bias, masks, loss, dX): every path forms its sums
in a fixed order.  Shapes: the fan-in 32 fast path in one and several batch
passes with and without fused SET, the wide fan-in 64 path, the general path
(bf16 at width 320, fp32), SET in both prune modes, top-k inference."""
import numpy as np
import pytest

import oracle
from paper_2411_03171_amd import synth
from tests.parity import (RTOL_BF16, RTOL_F32, assert_close, batch_to_gpu, from_torch_bits, note,
                          to_torch_values, values_f64)

pytestmark = pytest.mark.gpu

W1 = synth.WORKLOADS
CASES = {
    "c4s": (synth.scaled(W1["c4_bf16_L3M"], L=3001, name="c4s"), True),
    "mx200": (synth.scaled(W1["c4_bf16_L3M"], L=777, B=200, name="mx200"), True),
    "w1024": (synth.scaled(W1["c3_inter2048_L1M"], L=777, d=1024, B=37, name="w1024"), True),
    "mx320": (synth.scaled(W1["c4_bf16_L3M"], L=1003, d=320, B=37, name="mx320"), True),
    "c1": (W1["c1_fp32_L4096"], True),
    "k7": (synth.scaled(W1["c1_fp32_L4096"], L=500, d=40, k=7, B=9, name="k7"), True),
}


def _layer(inp, w, bias, idx16, m0, v0):
    import torch
    from paper_2411_03171_amd.ffsl import SparseLayer
    dev = "cuda:0"
    I = torch.from_numpy(inp.I.astype(np.uint16).view(np.int16) if idx16 else inp.I).to(dev)
    layer = SparseLayer(to_torch_values(inp.W, w.value, dev), I, bias=torch.from_numpy(bias).to(dev),
                        m=torch.from_numpy(m0), v=torch.from_numpy(v0), B_max=w.B,
                        nnz_max=max(len(inp.lab), 1), unfused=True)
    return layer.bind(w.d)


def _state(name):
    w, exact = CASES[name]
    if w.din:
        w = synth.dataclasses.replace(w, din=0)
    inp = synth.make_layer_inputs(w, 5)
    rng = np.random.default_rng(42)
    bias = (rng.standard_normal(w.L) * 0.1).astype(np.float32)
    m0 = (rng.standard_normal((w.L, w.k)) * 1e-3).astype(np.float32)
    v0 = (rng.random((w.L, w.k)) * 1e-5).astype(np.float32)
    return w, exact, inp, bias, m0, v0


def _snap(layer, w, extra):
    out = {"W": from_torch_bits(layer.W, w.value).copy(),
           "I": layer.I.cpu().numpy().view(np.uint16).astype(np.int32) if layer.I.dtype.itemsize == 2
           else layer.I.cpu().numpy().copy(),
           "m": layer.m.cpu().numpy().view(np.uint32).copy(), "v": layer.v.cpu().numpy().view(np.uint32).copy(),
           "bias": layer.bias.cpu().numpy().view(np.uint32).copy()}
    out.update(extra)
    return out


def _compare(a, b, exact, value):
    rtol = RTOL_F32 if value == "f32" else RTOL_BF16
    for key in a:
        if key in ("dX", "loss") and not exact:
            assert_close(a[key], np.asarray(b[key], dtype=np.float64), rtol, key)
        else:
            x, y = np.asarray(a[key]), np.asarray(b[key])
            if x.dtype.kind == "f":
                x, y = x.view(np.uint32), y.view(np.uint32)
            assert np.array_equal(x, y), key


@pytest.mark.parametrize("name", list(CASES))
def test_idx16_train_step_equals_int32(name):
    import torch
    w, exact, inp, bias, m0, v0 = _state(name)
    runs = []
    for idx16 in (False, True):
        note("idx16 train step %s idx16=%s" % (name, idx16))
        layer = _layer(inp, w, bias, idx16, m0, v0)
        X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
        loss, dX = layer.train_step(X, off, lab, t=2, lr=1e-2)
        torch.cuda.synchronize()
        runs.append(_snap(layer, w, {"dX": dX.cpu().numpy(), "loss": loss.cpu().numpy()}))
    _compare(runs[1], runs[0], exact, w.value)


@pytest.mark.parametrize("name", ["c1", "mx320", "k7"])
def test_idx16_unfused_calls_equal_int32(name):
    """Forward with logits, backward (dW, dbias, dX) and the unfused Adam."""
    import torch
    w, exact, inp, bias, m0, v0 = _state(name)
    runs = []
    for idx16 in (False, True):
        note("idx16 unfused %s idx16=%s" % (name, idx16))
        layer = _layer(inp, w, bias, idx16, m0, v0)
        X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
        loss, z = layer.forward_loss(X, off, lab, logits=True)
        dX = layer.backward(X, off, lab)
        dW = layer.dW.cpu().numpy().copy()
        layer.adam_step(3, lr=1e-2, wd=1e-4)
        torch.cuda.synchronize()
        runs.append(_snap(layer, w, {"z": z.cpu().numpy(), "loss": loss.cpu().numpy(), "dX": dX.cpu().numpy(),
                                     "dW": dW}))
    _compare(runs[1], runs[0], True, w.value)


# the fused step with SET runs on the fan-in 32 path (one batch pass, several)
SET_CASES = [(n, m) for n in ("c4s", "c1", "w1024") for m in ("fraction", "threshold")] + \
    [("c4s", "fused"), ("mx200", "fused")]


@pytest.mark.parametrize("name,mode", SET_CASES)
def test_idx16_set_equals_int32(name, mode):
    import torch
    w, exact, inp, bias, m0, v0 = _state(name)
    runs = []
    for idx16 in (False, True):
        note("idx16 SET %s %s idx16=%s" % (name, mode, idx16))
        layer = _layer(inp, w, bias, idx16, m0, v0)
        extra = {}
        if mode == "fraction":
            mask, ex = layer.set_update(0.25, 99, 3)
        elif mode == "threshold":
            mask, ex = layer.set_update_threshold(0.05, 99, 3)
        else:
            X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
            loss, dX, mask, ex = layer.train_step_set(X, off, lab, t=1, frac=0.1, seed=99, set_round=3)
            extra = {"dX": dX.cpu().numpy(), "loss": loss.cpu().numpy()}
        torch.cuda.synchronize()
        extra.update({"mask": mask.cpu().numpy(), "ex": ex.cpu().numpy()})
        runs.append(_snap(layer, w, extra))
    _compare(runs[1], runs[0], True, w.value)
    assert runs[1]["mask"].sum() > 0


@pytest.mark.parametrize("name", ["c4s", "w1024", "k7"])
def test_idx16_topk_equals_int32(name):
    import torch
    w, exact, inp, bias, m0, v0 = _state(name)
    outs = []
    for idx16 in (False, True):
        note("idx16 topk %s idx16=%s" % (name, idx16))
        layer = _layer(inp, w, bias, idx16, m0, v0)
        X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
        top, sc, p = layer.infer_topk(X, 5, off, lab)
        torch.cuda.synchronize()
        outs.append((top.cpu().numpy(), sc.cpu().numpy().view(np.uint32), p.cpu().numpy().view(np.uint32)))
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)


def test_idx16_validate_indices():
    import torch
    w, exact, inp, bias, m0, v0 = _state("c1")
    I = inp.I.copy()
    I[3, 2] = I[3, 5]          # a repeated index in row 3
    inp.I = I
    layer = _layer(inp, w, bias, True, m0, v0)
    bad = layer.validate_indices()
    torch.cuda.synchronize()
    assert int(bad.cpu().numpy()[0]) == 1


# ---------------------------------------------------------------- against the oracle

def _u16_indices(layer):
    return layer.I.cpu().numpy().view(np.uint16).astype(np.int32)


@pytest.mark.parametrize("name", ["c4s", "mx200", "w1024", "mx320", "c1", "k7"])
@pytest.mark.parametrize("fused", [False, True])
def test_idx16_step_against_oracle(name, fused):
    """The u16 layer's step against the oracle's forward, loss, backward and
    Adam (the checks of the int32 layer's parity test)."""
    import torch
    from tests.test_gpu_layer import adam_reference, check_step_result
    w, exact, inp, bias, m0, v0 = _state(name)
    s, t, lr, wd = 1.0 / w.B, 3, 1e-2, 1e-4
    r, Wn, mn, vn, bn, _, _ = adam_reference(w, inp, bias, s, t=t, lr=lr, wd=wd, m0=m0.astype(np.float64),
                                             v0=v0.astype(np.float64))
    note("idx16 %s step %s vs oracle" % ("fused" if fused else "unfused", name))
    layer = _layer(inp, w, bias, True, m0, v0)
    X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    if fused:
        loss, dX = layer.train_step(X, off, lab, t=t, s=s, lr=lr, wd=wd)
    else:
        loss = torch.empty(1, device="cuda:0")
        dX = layer.backward(X, off, lab, s=s, loss_out=loss)
        layer.adam_step(t, lr=lr, wd=wd)
    torch.cuda.synchronize()
    check_step_result(w, inp, layer, loss, dX, r, Wn, mn, vn, bn, t, lr, fused)
    np.testing.assert_array_equal(_u16_indices(layer), inp.I)


@pytest.mark.parametrize("name,mode", [("c4s", "fraction"), ("c4s", "threshold"), ("w1024", "fraction"),
                                       ("c1", "fraction"), ("c1", "threshold"), ("k7", "fraction")])
def test_idx16_set_against_oracle(name, mode):
    """SET on the u16 layer: indices, masks, W, m, v bit for bit against the
    oracle on the same state."""
    import torch
    w, exact, inp, bias, m0, v0 = _state(name)
    seed, rnd = 0x1616, 2
    note("idx16 SET %s %s vs oracle" % (name, mode))
    layer = _layer(inp, w, bias, True, m0, v0)
    if mode == "fraction":
        mask, ex = layer.set_update(0.25, seed, rnd)
    else:
        mask, ex = layer.set_update_threshold(0.05, seed, rnd)
    torch.cuda.synchronize()
    Wb = inp.W.view(np.uint32) if w.value == "f32" else inp.W
    if mode == "fraction":
        Wr, Ir, mr, vr, maskr, exr = oracle.set_update(Wb, inp.I, m0, v0, w.d, 0.25, seed, rnd)
    else:
        Wr, Ir, mr, vr, maskr, exr = oracle.set_update_threshold(Wb, inp.I, m0, v0, w.d, float(np.float32(0.05)),
                                                                 seed, rnd)
    assert int(ex.cpu().numpy()[0]) == exr
    np.testing.assert_array_equal(_u16_indices(layer), Ir)
    np.testing.assert_array_equal(mask.cpu().numpy(), maskr)
    Wg = from_torch_bits(layer.W, w.value)
    np.testing.assert_array_equal(Wg.view(np.uint32) if w.value == "f32" else Wg, Wr)
    np.testing.assert_array_equal(layer.m.cpu().numpy().view(np.uint32), mr.view(np.uint32))
    np.testing.assert_array_equal(layer.v.cpu().numpy().view(np.uint32), vr.view(np.uint32))
    assert maskr.sum() > 0


@pytest.mark.parametrize("name", ["c4s", "mx200"])
def test_idx16_fused_step_set_against_oracle(name):
    """The one-call step with SET on the u16 layer: the oracle's SET on the
    GPU's exact pre-SET state (the u16 layer's plain step on a copy), bit for
    bit on every row."""
    import torch
    w, exact, inp, bias, m0, v0 = _state(name)
    X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    note("idx16 step+SET %s vs oracle: plain step on a copy" % name)
    twin = _layer(inp, w, bias, True, m0, v0)
    twin.train_step(X, off, lab, t=1, lr=1e-2)
    torch.cuda.synchronize()
    pre = (from_torch_bits(twin.W, w.value).copy(), _u16_indices(twin), twin.m.cpu().numpy().copy(),
           twin.v.cpu().numpy().copy())
    del twin
    note("idx16 step+SET %s vs oracle: one call" % name)
    layer = _layer(inp, w, bias, True, m0, v0)
    loss, dX, mask, ex = layer.train_step_set(X, off, lab, t=1, frac=0.1, seed=99, set_round=3, lr=1e-2)
    torch.cuda.synchronize()
    Wr, Ir, mr, vr, maskr, exr = oracle.set_update(*pre, w.d, 0.1, 99, 3)
    assert int(ex.cpu().numpy()[0]) == exr == 0
    np.testing.assert_array_equal(_u16_indices(layer), Ir)
    np.testing.assert_array_equal(mask.cpu().numpy(), maskr)
    np.testing.assert_array_equal(from_torch_bits(layer.W, w.value), Wr)
    np.testing.assert_array_equal(layer.m.cpu().numpy().view(np.uint32), mr.view(np.uint32))
    np.testing.assert_array_equal(layer.v.cpu().numpy().view(np.uint32), vr.view(np.uint32))


@pytest.mark.parametrize("name", ["c4s", "w1024", "k7"])
def test_idx16_topk_against_oracle(name):
    """Top-k inference on the u16 layer against the oracle's scores (the
    validity checks of the int32 layer's top-k test)."""
    import torch
    from tests.test_gpu_topk import check_topk
    w, exact, inp, bias, m0, v0 = _state(name)
    K = 5
    Xv, Wv = values_f64(inp.X, w.value), values_f64(inp.W, w.value)
    z = oracle.forward(Xv, Wv, inp.I, bias.astype(np.float64))
    tol = 1e-5 * oracle.forward(np.abs(Xv), np.abs(Wv), inp.I, np.abs(bias).astype(np.float64)) + 1e-30
    note("idx16 topk %s vs oracle" % name)
    layer = _layer(inp, w, bias, True, m0, v0)
    X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    top, sc, p = layer.infer_topk(X, K, off, lab)
    torch.cuda.synchronize()
    top = top.cpu().numpy()
    check_topk(top, sc.cpu().numpy().astype(np.float64), z, tol, K)
    np.testing.assert_allclose(p.cpu().numpy(), oracle.precision_at_k(top, inp.off, inp.lab), rtol=1e-6, atol=1e-7)

"""GPU parity of the squared hinge loss (FFSL_LOSS_SQHINGE) against the oracle on
the same seeded inputs: forward and loss, the unfused backward, and the fused
step on every sweep (fan-in 32 fast path in one and four batch passes, the
wide fan-in 64 path, the general path in bf16 and fp32).  One case puts most
labels past the margin, so that whole waves have zero dlogits and the fused
paths skip their dW products."""
import numpy as np
import pytest

import oracle
from paper_2411_03171_amd import synth
from tests.parity import (RTOL_BF16, assert_close, batch_to_gpu, from_torch_bits, make_gpu_layer, note,
                          rtol_for, values_f64)
from tests.test_gpu_layer import fused_update_bound

pytestmark = pytest.mark.gpu

W1 = synth.WORKLOADS
CASES = {
    "c4s": synth.scaled(W1["c4_bf16_L3M"], L=3001, name="c4s"),
    "mx200": synth.scaled(W1["c4_bf16_L3M"], L=777, B=200, name="mx200"),
    "c3s": synth.scaled(W1["c3_inter2048_L1M"], L=700, name="c3s"),
    "w1024": synth.scaled(W1["c3_inter2048_L1M"], L=777, d=1024, B=37, name="w1024"),
    "mx320": synth.scaled(W1["c4_bf16_L3M"], L=1003, d=320, B=37, name="mx320"),
    "c1": W1["c1_fp32_L4096"],
}


def _inputs(name, seed, margin=False):
    w = CASES[name]
    if w.din:
        w = synth.dataclasses.replace(w, din=0)
    inp = synth.make_layer_inputs(w, seed)
    rng = np.random.default_rng(900 + seed)
    L = inp.I.shape[0]
    if margin:
        # scores near -4: every label without a positive is past the margin
        bias = (-4.0 + 0.05 * rng.standard_normal(L)).astype(np.float32)
    else:
        bias = (rng.standard_normal(L) * 0.1).astype(np.float32)
    return w, inp, bias


def _ref(w, inp, bias, s):
    return oracle.loss_and_grads(values_f64(inp.X, w.value), values_f64(inp.W, w.value), inp.I,
                                 bias.astype(np.float64), inp.off, inp.lab, s, loss="sqhinge")


@pytest.fixture(scope="module")
def ffsl_mod():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2411_03171_amd import ffsl
    ffsl.load()
    return ffsl


@pytest.mark.parametrize("name", list(CASES))
def test_sqhinge_forward_and_backward(ffsl_mod, name):
    import torch
    w, inp, bias = _inputs(name, seed=1)
    s = 1.0 / w.B
    rtol = rtol_for(w.value)
    ref = _ref(w, inp, bias, s)
    note("sqhinge forward %s" % name)
    layer = make_gpu_layer(inp, w, bias_values=bias)
    X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    loss, z = layer.forward_loss(X, off, lab, s=s, logits=True, flags=ffsl_mod.FFSL_LOSS_SQHINGE)
    torch.cuda.synchronize()
    assert_close(z.cpu().numpy(), ref["z"], rtol, "logits")
    assert_close(loss.cpu().numpy()[0], ref["loss"], rtol, "loss")
    note("sqhinge backward %s" % name)
    loss2 = torch.empty(1, device="cuda:0")
    dX = layer.backward(X, off, lab, s=s, loss_out=loss2, flags=ffsl_mod.FFSL_LOSS_SQHINGE)
    torch.cuda.synchronize()
    assert_close(layer.dW.cpu().numpy(), ref["dW"], rtol, "dW")
    assert_close(layer.dbias.cpu().numpy(), ref["dbias"], rtol, "dbias")
    assert_close(dX.cpu().numpy(), ref["dX"], rtol, "dX")
    assert_close(loss2.cpu().numpy()[0], ref["loss"], rtol, "loss (backward)")


@pytest.mark.parametrize("margin", [False, True], ids=["active", "margin"])
@pytest.mark.parametrize("name", list(CASES))
def test_sqhinge_fused_step(ffsl_mod, name, margin):
    import torch
    w, inp, bias = _inputs(name, seed=2, margin=margin)
    s = 1.0 / w.B
    t, lr = 3, 1e-2
    rtol = rtol_for(w.value)
    rng = np.random.default_rng(17)
    L, k = inp.I.shape
    m0 = (rng.standard_normal((L, k)) * 1e-3).astype(np.float32)
    v0 = (rng.random((L, k)) * 1e-5).astype(np.float32)
    r = _ref(w, inp, bias, s)
    if margin:
        # most rows have no dlogit at all: the skip is exercised
        assert (np.abs(r["g"]).max(axis=0) == 0).mean() > 0.5
    W = values_f64(inp.W, w.value)
    Wn, mn, vn = oracle.adam(W, m0, v0, r["dW"], t, lr=lr)
    bn, _, _ = oracle.adam(bias.astype(np.float64), np.zeros(L), np.zeros(L), r["dbias"], t, lr=lr)
    note("sqhinge fused step %s %s" % (name, "margin" if margin else "active"))
    layer = make_gpu_layer(inp, w, bias_values=bias, unfused=False)
    layer.m.copy_(torch.from_numpy(m0))
    layer.v.copy_(torch.from_numpy(v0))
    X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    loss, dX = layer.train_step(X, off, lab, t=t, s=s, lr=lr, flags=ffsl_mod.FFSL_LOSS_SQHINGE)
    torch.cuda.synchronize()
    Wg = values_f64(from_torch_bits(layer.W, w.value), w.value)
    if w.value == "bf16":
        # the stored weight is the update rounded to bf16 (one ulp), plus the
        # effect of rounding the dlogits to bf16 in the fused paths
        Wref = values_f64(oracle.round_bf16(Wn), "bf16")
        allow = (2.0 ** -7 * np.maximum(np.abs(Wg), np.abs(Wref)) + 1e-5 * lr
                 + 1.5 * fused_update_bound(r, inp, w, mn, vn, t, lr))
        assert np.all(np.abs(Wg - Wref) <= allow), int((np.abs(Wg - Wref) > allow).sum())
    else:
        # (bf16: the per-slot bound above is the bar; the hinge's dlogits are
        # up to twice BCE's, so their bf16 rounding moves some near-zero
        # gradients' Adam updates further than a blanket tolerance allows)
        assert_close(Wg, Wn, rtol, "W")
    assert_close(layer.m.cpu().numpy(), mn, rtol, "m")
    # v carries the gradient squared, so its relative error is twice the
    # gradient's (the hinge's 1 - yz cancels near the margin)
    assert_close(layer.v.cpu().numpy(), vn, 2 * rtol, "v")
    assert_close(layer.bias.cpu().numpy(), bn, rtol, "bias")
    assert_close(dX.cpu().numpy(), r["dX"], rtol, "dX")
    assert_close(loss.cpu().numpy()[0], r["loss"], rtol, "loss")
    if margin:
        # rows with no dlogit keep m, v decayed exactly as Adam does with g = 0
        quiet = np.abs(r["g"]).max(axis=0) == 0
        assert_close(layer.m.cpu().numpy()[quiet], (0.9 * m0.astype(np.float64))[quiet], rtol, "m quiet")


def test_sqhinge_with_set_in_one_call(ffsl_mod):
    """The squared hinge through ffsl_train_step_set equals ffsl_train_step with
    the same flag followed by ffsl_set_update, bit for bit."""
    import torch
    w, inp, bias = _inputs("c4s", seed=3)
    outs = []
    for fused in (False, True):
        layer = make_gpu_layer(inp, w, bias_values=bias, unfused=False)
        X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
        if fused:
            loss, dX, mask, ex = layer.train_step_set(X, off, lab, t=1, frac=0.1, seed=5, set_round=1,
                                                      flags=ffsl_mod.FFSL_LOSS_SQHINGE)
        else:
            loss, dX = layer.train_step(X, off, lab, t=1, flags=ffsl_mod.FFSL_LOSS_SQHINGE)
            mask, ex = layer.set_update(0.1, 5, 1)
        torch.cuda.synchronize()
        outs.append((from_torch_bits(layer.W, "bf16").copy(), layer.I.cpu().numpy().copy(),
                     layer.m.cpu().numpy().view(np.uint32).copy(), mask.cpu().numpy().copy(),
                     dX.cpu().numpy().view(np.uint32).copy()))
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)

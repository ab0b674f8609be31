"""Multi-step runs: training steps on fresh batches with SET every few steps,
on the GPU and in the oracle.

Between SET rounds each side follows its own trajectory (the oracle's state is
float64, rounded to the stored type after each update as the GPU stores it);
per step the loss and dX must agree within the bar of the value type.  At
every SET round the oracle is re-synced to the GPU's exact pre-SET state (the
bits of W, I, m, v after the GPU's training step), runs its SET on that state,
and the GPU's post-SET W, I, m, v and mask must equal the oracle's bit for bit
on every row.  The oracle then continues from that common state (with the
GPU's bias state), so a later SET round is checked the same way.

Where the library fuses SET into the step (ffsl_train_step_set, the bf16
fan-in-32 fast path), the pre-SET state comes from a twin layer with the same
state that runs the plain ffsl_train_step on the same batch.

Cases: the largest workload's shape (B = 64, one batch pass of the fast path)
and the LF-AmazonTitles-131K stand-in (B = 128, two batch passes), both with
SET fused into the step; the fp32 correctness workload (general path, k = 16)
and a bf16 width off the fast path (d = 320, general path), both with the step
and SET as separate calls."""
import numpy as np
import pytest

import oracle
from paper_2411_03171_amd import synth
from tests.parity import RTOL_BF16, RTOL_F32, assert_close, from_torch_bits, note, to_torch_values, values_f64

pytestmark = pytest.mark.gpu

W1 = synth.WORKLOADS
CASES = {
    # name: (workload, SET fused into the step)
    "c4s": (synth.scaled(W1["c4_bf16_L3M"], L=3000, name="c4s"), True),
    "c2s": (synth.scaled(W1["c2_bf16_L131072"], L=3000, name="c2s"), True),
    "c1": (synth.scaled(W1["c1_fp32_L4096"], L=1500, name="c1m"), False),
    "mx320": (synth.scaled(W1["c4_bf16_L3M"], L=1003, d=320, B=37, name="mx320"), False),
}
STEPS, SET_EVERY, SEED = 8, 4, 99


def _bits(W, value):
    """Stored weights (float32 or bf16 bit patterns) as the oracle's SET takes them."""
    return W.view(np.uint32) if value == "f32" else W


def _layer_from(W, I, bias, m, v, bm, bv, w, nnz_max):
    import torch
    from paper_2411_03171_amd import ffsl
    return ffsl.SparseLayer(W, I, bias=bias, m=m, v=v, bias_m=bm, bias_v=bv, B_max=w.B, nnz_max=nnz_max,
                            unfused=False).bind(w.d)


def _state(layer, value):
    return (from_torch_bits(layer.W, value).copy(), layer.I.cpu().numpy().copy(), layer.m.cpu().numpy().copy(),
            layer.v.cpu().numpy().copy(), layer.bias.cpu().numpy().copy(), layer.bias_m.cpu().numpy().copy(),
            layer.bias_v.cpu().numpy().copy())


@pytest.mark.parametrize("name", list(CASES))
def test_steps_with_set(name):
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    w, fused = CASES[name]
    inp = synth.make_layer_inputs(w, 4)
    batches = synth.make_batches(w, STEPS, seed=4)
    dev = "cuda:0"
    nnz_max = max(len(b[2]) for b in batches)
    rng = np.random.default_rng(44)
    L, k = inp.I.shape
    bias0 = (rng.standard_normal(L) * 0.1).astype(np.float32)
    layer = _layer_from(to_torch_values(inp.W, w.value, dev), torch.from_numpy(inp.I).to(dev),
                        torch.from_numpy(bias0).to(dev), None, None, None, None, w, nnz_max)
    rtol = RTOL_F32 if w.value == "f32" else RTOL_BF16
    W = values_f64(inp.W, w.value)
    I = inp.I.copy()
    m, v = np.zeros((L, k)), np.zeros((L, k))
    bias, bm, bv = bias0.astype(np.float64), np.zeros(L), np.zeros(L)
    s, lr, frac = 1.0 / w.B, 1e-3, 0.1
    set_round = 0
    n = oracle.set_prune_count(k, frac)
    for step in range(1, STEPS + 1):
        X, off, lab = batches[step - 1]
        Xt = to_torch_values(X, w.value, dev)
        offt = torch.from_numpy(off.astype(np.int32)).to(dev)
        labt = torch.from_numpy(lab).to(dev)
        set_now = step % SET_EVERY == 0
        note("%s step %d nnz=%d set=%s" % (name, step, len(lab), set_now))
        if set_now and fused:
            # the twin runs the plain step from the same state: its result is
            # the pre-SET state of the fused call
            twin = _layer_from(layer.W.clone(), layer.I.clone(), layer.bias.clone(), layer.m.clone(),
                               layer.v.clone(), layer.bias_m.clone(), layer.bias_v.clone(), w, nnz_max)
            twin.train_step(Xt, offt, labt, t=step, s=s, lr=lr)
            loss_g, dX_g, mask_g, ex_g = layer.train_step_set(Xt, offt, labt, t=step, frac=frac, seed=SEED,
                                                              set_round=set_round, s=s, lr=lr)
            torch.cuda.synchronize()
            pre = _state(twin, w.value)
            del twin
        else:
            loss_g, dX_g = layer.train_step(Xt, offt, labt, t=step, s=s, lr=lr)
            torch.cuda.synchronize()
            if set_now:
                pre = _state(layer, w.value)
                mask_g, ex_g = layer.set_update(frac, SEED, set_round)
                torch.cuda.synchronize()
        r = oracle.train_step(values_f64(X, w.value), W, I, bias, m, v, bm, bv, off, lab, s, t=step, lr=lr,
                              w_bf16=(w.value == "bf16"))
        W, m, v, bias, bm, bv = r["W"], r["m"], r["v"], r["bias"], r["bias_m"], r["bias_v"]
        assert_close(np.array([float(loss_g.cpu()[0])]), np.array([r["loss"]]), rtol, "loss")
        assert_close(dX_g.cpu().numpy(), r["dX"], rtol, "dX")
        if not set_now:
            continue
        # SET on the GPU's exact pre-SET state: bit-exact on every row
        note("%s SET round %d" % (name, set_round))
        Wp, Ip, mp, vp, bp, bmp, bvp = pre
        Wr, Ir, mr, vr, maskr, exr = oracle.set_update(_bits(Wp, w.value), Ip, mp, vp, w.d, frac, SEED, set_round)
        post = _state(layer, w.value)
        assert int(ex_g.cpu().numpy()[0]) == exr == 0
        np.testing.assert_array_equal(post[1], Ir)
        np.testing.assert_array_equal(mask_g.cpu().numpy(), maskr)
        np.testing.assert_array_equal(_bits(post[0], w.value), Wr)
        np.testing.assert_array_equal(post[2].view(np.uint32), mr.view(np.uint32))
        np.testing.assert_array_equal(post[3].view(np.uint32), vr.view(np.uint32))
        assert (maskr.sum(axis=1) == n).all()
        # the bias is not SET's: the post-SET bias state is the pre-SET one
        np.testing.assert_array_equal(post[4].view(np.uint32), bp.view(np.uint32))
        # the oracle continues from the common state
        W = values_f64(Wr.view(np.float32) if w.value == "f32" else Wr, w.value)
        I, m, v = Ir.copy(), mr.astype(np.float64), vr.astype(np.float64)
        bias, bm, bv = bp.astype(np.float64), bmp.astype(np.float64), bvp.astype(np.float64)
        set_round += 1
    # after the last step (a SET step) both sides hold the same state
    post = _state(layer, w.value)
    assert_close(values_f64(post[0], w.value), W, rtol, "W after %d steps" % STEPS)
    np.testing.assert_array_equal(post[1], I)
    # the contract's invariants on every row
    Ig = post[1]
    assert np.all(np.diff(np.sort(Ig, axis=1), axis=1) > 0)
    assert Ig.min() >= 0 and Ig.max() < w.d

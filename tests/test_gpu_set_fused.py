"""GPU parity of ffsl_train_step_set, the training step with SET prune-and-regrow
fused into the sweep that applies Adam.  Its contract is the result of
ffsl_train_step followed by ffsl_set_update on the same stream, so both are
run on identical copies of the state and must agree bit for bit (weights,
indices, moments, bias, masks, exhausted count, loss and dX).  The oracle
(train step, then SET) checks one case directly.  Shapes: one, two and four
batch passes, the narrowest width (d = 128: a quarter of the draws meet a
held column, so many rows are finished by the row-list SET kernel), a single
sample, the largest number of pruned slots the fused path takes, and shapes
where the library runs the two calls back to back (other widths, other
fan-ins, more pruned slots)."""
import numpy as np
import pytest

import oracle
from paper_2411_03171_amd import synth
from tests.parity import (RTOL_BF16, assert_close, batch_to_gpu, from_torch_bits, make_gpu_layer, note,
                          values_f64)

pytestmark = pytest.mark.gpu

W1 = synth.WORKLOADS
CASES = {
    # fused: passes of 64 samples (1, 2 and 4), widths 768 and 128, B = 1
    "c4s": synth.scaled(W1["c4_bf16_L3M"], L=3001, name="c4s"),
    "c2s": synth.scaled(W1["c2_bf16_L131072"], L=2000, name="c2s"),
    "mx200": synth.scaled(W1["c4_bf16_L3M"], L=777, B=200, name="mx200"),
    "mx128": synth.scaled(W1["c4_bf16_L3M"], L=257, d=128, B=64, name="mx128"),
    "b1": synth.scaled(W1["c4_bf16_L3M"], L=513, B=1, name="b1"),
    # back to back: a width off the fused path, fan-in 64
    "mx320": synth.scaled(W1["c4_bf16_L3M"], L=1003, d=320, B=37, name="mx320"),
    "w1024": synth.scaled(W1["c3_inter2048_L1M"], L=777, d=1024, B=37, name="w1024"),
}
# prune fractions at k = 32: n = 3 (the workloads'), 4 (the most the fused
# path takes: its four draws per row made ahead), 8 and 9 (back to back), 0
# (no SET; only the mask is written)
FRACS = [0.1, 0.125, 0.25, 0.3, 0.0]


def _state(name, seed):
    w = CASES[name]
    if w.din:
        w = synth.dataclasses.replace(w, din=0)
    inp = synth.make_layer_inputs(w, seed)
    rng = np.random.default_rng(500 + seed)
    L, k = inp.I.shape
    bias = (rng.standard_normal(L) * 0.1).astype(np.float32)
    m0 = (rng.standard_normal((L, k)) * 1e-3).astype(np.float32)
    v0 = (rng.random((L, k)) * 1e-5).astype(np.float32)
    return w, inp, bias, m0, v0


def _run(w, inp, bias, m0, v0, fused, frac, wd, t=3, lr=1e-2, seed=77, rnd=5):
    import torch
    layer = make_gpu_layer(inp, w, bias_values=bias, unfused=False)
    layer.m.copy_(torch.from_numpy(m0))
    layer.v.copy_(torch.from_numpy(v0))
    X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    s = 1.0 / w.B
    if fused:
        loss, dX, mask, ex = layer.train_step_set(X, off, lab, t=t, frac=frac, seed=seed, set_round=rnd, s=s,
                                                  lr=lr, wd=wd)
    else:
        loss, dX = layer.train_step(X, off, lab, t=t, s=s, lr=lr, wd=wd)
        mask, ex = layer.set_update(frac, seed, rnd)
    torch.cuda.synchronize()
    return {
        "W": from_torch_bits(layer.W, w.value).copy(),
        "I": layer.I.cpu().numpy().copy(),
        "m": layer.m.cpu().numpy().copy(),
        "v": layer.v.cpu().numpy().copy(),
        "bias": layer.bias.cpu().numpy().copy(),
        "mask": mask.cpu().numpy().copy(),
        "ex": int(ex.cpu().numpy()[0]),
        "loss": float(loss.cpu()[0]),
        "dX": dX.cpu().numpy().copy(),
    }


@pytest.mark.parametrize("frac", FRACS)
@pytest.mark.parametrize("name", list(CASES))
def test_fused_equals_step_then_set(name, frac):
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    w, inp, bias, m0, v0 = _state(name, seed=3)
    wd = 1e-4 if name in ("c4s", "mx200") else 0.0
    note("train+SET %s frac=%g: back to back" % (name, frac))
    ref = _run(w, inp, bias, m0, v0, False, frac, wd)
    note("train+SET %s frac=%g: one call" % (name, frac))
    got = _run(w, inp, bias, m0, v0, True, frac, wd)
    # every path forms its sums in a fixed order: everything bit for bit
    exact = ("W", "I", "m", "v", "bias", "mask", "dX")
    for key in exact:
        a, b = got[key], ref[key]
        if a.dtype.kind == "f":
            a, b = a.view(np.uint32), b.view(np.uint32)
        bad = np.argwhere(a != b)
        assert len(bad) == 0, "%s differs at %d entries, first %s" % (key, len(bad), bad[:4].tolist())
    assert got["ex"] == ref["ex"]
    assert np.float32(got["loss"]).view(np.uint32) == np.float32(ref["loss"]).view(np.uint32)
    # no row runs out of attempts at these widths: every row regrows n slots
    n = int(np.floor(frac * inp.I.shape[1] + 1e-9))
    assert got["ex"] == 0
    assert (got["mask"].sum(axis=1) == n).all()


def _step_only(w, inp, bias, m0, v0, wd, t, lr):
    """The plain training step (no SET) from the same state: the pre-SET state
    of the one-call step."""
    import torch
    layer = make_gpu_layer(inp, w, bias_values=bias, unfused=False)
    layer.m.copy_(torch.from_numpy(m0))
    layer.v.copy_(torch.from_numpy(v0))
    X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    layer.train_step(X, off, lab, t=t, s=1.0 / w.B, lr=lr, wd=wd)
    torch.cuda.synchronize()
    return (from_torch_bits(layer.W, w.value).copy(), layer.I.cpu().numpy().copy(), layer.m.cpu().numpy().copy(),
            layer.v.cpu().numpy().copy())


@pytest.mark.parametrize("name,frac,wd", [("c4s", 0.1, 0.0), ("mx200", 0.25, 1e-4), ("b1", 0.1, 0.0)])
def test_fused_against_oracle(name, frac, wd):
    """The one-call step against the oracle.  The step's loss and dX against the
    oracle's step within the bf16 bar; SET bit for bit on every row: the
    oracle's SET runs on the GPU's exact pre-SET state (W bits, I, m, v of the
    plain step on an identical copy), and the one-call result must equal it in
    W, I, m, v and the mask."""
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    w, inp, bias, m0, v0 = _state(name, seed=4)
    seed, rnd, t, lr = 123, 2, 3, 1e-2
    note("train+SET %s vs oracle: one call" % name)
    got = _run(w, inp, bias, m0, v0, True, frac, wd, t=t, lr=lr, seed=seed, rnd=rnd)
    note("train+SET %s vs oracle: the plain step on a copy" % name)
    Wp, Ip, mp, vp = _step_only(w, inp, bias, m0, v0, wd, t, lr)
    Wr, Ir, mr, vr, maskr, exr = oracle.set_update(Wp, Ip, mp, vp, w.d, frac, seed, rnd)
    assert exr == 0 and got["ex"] == 0
    np.testing.assert_array_equal(got["I"], Ir)
    np.testing.assert_array_equal(got["mask"], maskr)
    np.testing.assert_array_equal(got["W"], Wr)
    np.testing.assert_array_equal(got["m"].view(np.uint32), mr.view(np.uint32))
    np.testing.assert_array_equal(got["v"].view(np.uint32), vr.view(np.uint32))
    n = oracle.set_prune_count(w.k, frac)
    assert (maskr.sum(axis=1) == n).all()
    # the step itself against the oracle's step
    X = values_f64(inp.X, "bf16")
    W = values_f64(inp.W, "bf16")
    r = oracle.train_step(X, W, inp.I, bias.astype(np.float64), m0.astype(np.float64), v0.astype(np.float64),
                          np.zeros(len(bias)), np.zeros(len(bias)), inp.off, inp.lab, 1.0 / w.B, t=t, lr=lr,
                          wd=wd, w_bf16=True)
    assert_close(np.array([got["loss"]]), np.array([r["loss"]]), RTOL_BF16, "loss")
    assert_close(got["dX"], r["dX"], RTOL_BF16, "dX")
    assert_close(got["m"][maskr == 0], r["m"][maskr == 0], RTOL_BF16, "m of the survivors")
    # regrown columns are new to the row
    for l in np.nonzero(maskr.any(axis=1))[0][:200]:
        regrown = Ir[l][maskr[l] == 1]
        assert not (set(regrown.tolist()) & set(inp.I[l].tolist()))

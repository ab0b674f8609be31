"""Checkpoint and resume: a run of 2N training steps (with SET rounds) must equal,
bit for bit, a run of N steps whose whole state is saved to disk, loaded into
a fresh layer and run for N more steps.  The state of the method is W, I, the
Adam moments, the bias and its moments, the step counter t and the SET round;
nothing else (the SET draws are counted by (row, round), not drawn from a
running generator), so a resumed run cannot drift.

CPU: the oracle's float64 trajectory through numpy .npz files.  GPU: the
library's layer state (W bits, I, m, v, bias state) saved to host files and
uploaded into a new layer, on the fused fast path and on the general path;
both paths form every sum in a fixed order, so the runs agree bit for bit."""
import numpy as np
import pytest

import oracle
from paper_2411_03171_amd import synth
from tests.parity import from_torch_bits, note, to_torch_values, values_f64

W1 = synth.WORKLOADS
N_STEPS, SET_EVERY, FRAC, SEED = 3, 2, 0.25, 5


def _oracle_steps(state, batches, t0, w, round0):
    W, I, m, v, bias, bm, bv = state
    rnd = round0
    for i, (X, off, lab) in enumerate(batches):
        t = t0 + i
        r = oracle.train_step(values_f64(X, w.value), W, I, bias, m, v, bm, bv, off, lab, 1.0 / w.B, t=t,
                              lr=1e-2, wd=1e-4, w_bf16=(w.value == "bf16"))
        W, m, v, bias, bm, bv = r["W"], r["m"], r["v"], r["bias"], r["bias_m"], r["bias_v"]
        if t % SET_EVERY == 0:
            Wbits = oracle.round_bf16(W) if w.value == "bf16" else W.astype(np.float32).view(np.uint32)
            Wb, I, mf, vf, _, ex = oracle.set_update(Wbits, I, m.astype(np.float32), v.astype(np.float32), w.d,
                                                     FRAC, SEED, rnd)
            assert ex == 0
            W = oracle.bf16_to_f64(Wb) if w.value == "bf16" else Wb.view(np.float32).astype(np.float64)
            m, v = mf.astype(np.float64), vf.astype(np.float64)
            rnd += 1
    return (W, I, m, v, bias, bm, bv), rnd


@pytest.mark.parametrize("name", ["c1", "c4s"])
def test_oracle_checkpoint_resume_is_bitwise(tmp_path, name):
    w = W1["c1_fp32_L4096"] if name == "c1" else synth.scaled(W1["c4_bf16_L3M"], L=300, name="c4s")
    w = synth.scaled(w, L=min(w.L, 500), name=name)
    inp = synth.make_layer_inputs(w, 11)
    batches = synth.make_batches(w, 2 * N_STEPS, seed=12)
    L, k = inp.I.shape
    s0 = (values_f64(inp.W, w.value), inp.I.copy(), np.zeros((L, k)), np.zeros((L, k)), np.zeros(L), np.zeros(L),
          np.zeros(L))
    straight, rnd_a = _oracle_steps(s0, batches, 1, w, 0)
    half, rnd = _oracle_steps(s0, batches[:N_STEPS], 1, w, 0)
    path = tmp_path / "ckpt.npz"
    names = ("W", "I", "m", "v", "bias", "bias_m", "bias_v")
    np.savez(path, t=N_STEPS, set_round=rnd, **dict(zip(names, half)))
    with np.load(path, allow_pickle=False) as f:
        loaded = tuple(f[n].copy() for n in names)
        t_next, rnd_b = int(f["t"]) + 1, int(f["set_round"])
    resumed, rnd_b = _oracle_steps(loaded, batches[N_STEPS:], t_next, w, rnd_b)
    assert rnd_a == rnd_b
    for n, a, b in zip(names, straight, resumed):
        assert a.dtype == b.dtype and np.array_equal(a, b), n
    # the SET rounds did change the topology
    assert not np.array_equal(straight[1], inp.I)


def _gpu_layer(W, I, bias, m, v, bm, bv, w, nnz_max):
    from paper_2411_03171_amd import ffsl
    return ffsl.SparseLayer(W, I, bias=bias, m=m, v=v, bias_m=bm, bias_v=bv, B_max=w.B, nnz_max=nnz_max,
                            unfused=False).bind(w.d)


def _gpu_steps(layer, batches, t0, w, rnd):
    import torch
    dev = "cuda:0"
    for i, (X, off, lab) in enumerate(batches):
        t = t0 + i
        Xt = to_torch_values(X, w.value, dev)
        offt = torch.from_numpy(off.astype(np.int32)).to(dev)
        labt = torch.from_numpy(lab).to(dev)
        if t % SET_EVERY == 0:
            layer.train_step_set(Xt, offt, labt, t=t, frac=FRAC, seed=SEED, set_round=rnd, lr=1e-2, wd=1e-4)
            rnd += 1
        else:
            layer.train_step(Xt, offt, labt, t=t, lr=1e-2, wd=1e-4)
    torch.cuda.synchronize()
    return rnd


@pytest.mark.gpu
@pytest.mark.parametrize("name", ["c4s", "c2s", "c1", "mx320"])
def test_gpu_checkpoint_resume_is_bitwise(tmp_path, name):
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ws = {"c4s": synth.scaled(W1["c4_bf16_L3M"], L=2000, name="c4s"),
          "c2s": synth.scaled(W1["c2_bf16_L131072"], L=1500, name="c2s"),
          "c1": W1["c1_fp32_L4096"],
          "mx320": synth.scaled(W1["c4_bf16_L3M"], L=1003, d=320, B=37, name="mx320")}
    w = ws[name]
    inp = synth.make_layer_inputs(w, 13)
    batches = synth.make_batches(w, 2 * N_STEPS, seed=14)
    nnz_max = max(len(b[2]) for b in batches)
    dev = "cuda:0"
    L = w.L
    bias0 = torch.from_numpy((np.random.default_rng(15).standard_normal(L) * 0.1).astype(np.float32))

    def fresh():
        return _gpu_layer(to_torch_values(inp.W, w.value, dev), torch.from_numpy(inp.I).to(dev), bias0.to(dev),
                          None, None, None, None, w, nnz_max)

    note("checkpoint %s: straight run of %d steps" % (name, 2 * N_STEPS))
    a = fresh()
    rnd_a = _gpu_steps(a, batches, 1, w, 0)
    note("checkpoint %s: %d steps, save, load, %d steps" % (name, N_STEPS, N_STEPS))
    b = fresh()
    rnd = _gpu_steps(b, batches[:N_STEPS], 1, w, 0)
    path = tmp_path / "layer.npz"
    np.savez(path, W=from_torch_bits(b.W, w.value), I=b.I.cpu().numpy(), m=b.m.cpu().numpy(),
             v=b.v.cpu().numpy(), bias=b.bias.cpu().numpy(), bias_m=b.bias_m.cpu().numpy(),
             bias_v=b.bias_v.cpu().numpy(), t=N_STEPS, set_round=rnd)
    del b
    with np.load(path, allow_pickle=False) as f:
        st = {n: f[n].copy() for n in f.files}
    c = _gpu_layer(to_torch_values(st["W"], w.value, dev), torch.from_numpy(st["I"]).to(dev),
                   torch.from_numpy(st["bias"]).to(dev), torch.from_numpy(st["m"]), torch.from_numpy(st["v"]),
                   torch.from_numpy(st["bias_m"]), torch.from_numpy(st["bias_v"]), w, nnz_max)
    rnd_c = _gpu_steps(c, batches[N_STEPS:], int(st["t"]) + 1, w, int(st["set_round"]))
    assert rnd_a == rnd_c
    for n in ("W", "I", "m", "v", "bias", "bias_m", "bias_v"):
        x, y = getattr(a, n), getattr(c, n)
        assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x.view(torch.int32),
                           y.view(torch.int16) if y.dtype == torch.bfloat16 else y.view(torch.int32)), n
    assert not torch.equal(a.I.cpu(), torch.from_numpy(inp.I))

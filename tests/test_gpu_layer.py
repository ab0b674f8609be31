"""GPU parity of the sparse layer: the HIP path through the C ABI against the
CPU oracle on the same seeded inputs, at sizes the oracle finishes in seconds
that still span several 256-row chunks, several batch tiles and ragged tails.
"""
import numpy as np
import pytest

import oracle
from paper_2411_03171_amd import synth
from tests.parity import (assert_close, batch_to_gpu, from_torch_bits, make_gpu_layer, note,
                          rtol_for, values_f64)

pytestmark = pytest.mark.gpu

W1 = synth.WORKLOADS
CASES = {
    # fp32 correctness workload at full size
    "c1": W1["c1_fp32_L4096"],
    # bf16 workloads scaled down in L (ragged against 256-row chunks), full B, d, k
    "c2s": synth.scaled(W1["c2_bf16_L131072"], L=2000),
    "c3s": synth.scaled(W1["c3_inter2048_L1M"], L=700, name="c3s"),
    "c4s": synth.scaled(W1["c4_bf16_L3M"], L=3001),
    "c5s": synth.scaled(W1["c5_aux8192_L1M"], L=1500),
    # shapes off the common path: odd fan-in, full fan-in, wide fan-in, tiny batch
    "k5": synth.scaled(W1["c1_fp32_L4096"], L=700, k=5, name="k5"),
    "kfull": synth.scaled(W1["c1_fp32_L4096"], L=300, d=16, k=16, B=7, name="kfull"),
    "k100": synth.scaled(W1["c4_bf16_L3M"], L=600, k=100, B=20, name="k100"),
    "b1": synth.scaled(W1["c4_bf16_L3M"], L=513, B=1, name="b1"),
    # the fused bf16 fan-in-32 fast path at other widths (narrowest, odd tile
    # count) with a ragged batch
    "mx128": synth.scaled(W1["c4_bf16_L3M"], L=257, d=128, B=64, name="mx128"),
    "mx320": synth.scaled(W1["c4_bf16_L3M"], L=1003, d=320, B=37, name="mx320"),
    # a batch of 200 on the fused fast path: four passes (first, two middle, last)
    "mx200": synth.scaled(W1["c4_bf16_L3M"], L=777, B=200, name="mx200"),
    # more positives per batch (about 1900) than the fast path keeps on chip
    "mxdense": synth.dataclasses.replace(synth.scaled(W1["c4_bf16_L3M"], L=700, name="mxdense"),
                                         mean_pos=30.0),
    # the fused bf16 fan-in-64 wide path (passes of 16 samples): another width
    # with a ragged last pass and a ragged chunk, a single pass at the
    # narrowest width, and more positives per pass (about 1300) than it keeps
    # on chip
    "w1024": synth.scaled(W1["c3_inter2048_L1M"], L=777, d=1024, B=37, name="w1024"),
    "w128": synth.scaled(W1["c3_inter2048_L1M"], L=301, d=128, B=16, name="w128"),
    "wdense": synth.dataclasses.replace(synth.scaled(W1["c3_inter2048_L1M"], L=900, name="wdense"),
                                        mean_pos=80.0),
}


def case_inputs(name, seed=0):
    w = CASES[name]
    if w.din:   # the sparse layer of the intermediate-layer workload sees width d
        w = synth.dataclasses.replace(w, din=0)
    inp = synth.make_layer_inputs(w, seed)
    rng = np.random.default_rng(1000 + seed)
    bias = (rng.standard_normal(w.L) * 0.1).astype(np.float32)
    return w, inp, bias


def oracle_grads(w, inp, bias, s):
    X = values_f64(inp.X, w.value)
    W = values_f64(inp.W, w.value)
    return oracle.loss_and_grads(X, W, inp.I, bias.astype(np.float64), inp.off, inp.lab, s)


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2411_03171_amd import ffsl
    ffsl.load()
    return torch


@pytest.mark.parametrize("name", list(CASES))
def test_forward_loss_and_logits(torch_cuda, name):
    torch = torch_cuda
    w, inp, bias = case_inputs(name)
    note("forward %s B=%d d=%d L=%d k=%d %s" % (name, w.B, w.d, w.L, w.k, w.value))
    layer = make_gpu_layer(inp, w, bias_values=bias)
    X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    s = 1.0 / w.B
    loss, z = layer.forward_loss(X, off, lab, s=s, logits=True)
    torch.cuda.synchronize()
    ref = oracle_grads(w, inp, bias, s)
    rtol = rtol_for(w.value)
    assert_close(z.cpu().numpy(), ref["z"], rtol, "logits")
    assert_close(loss.cpu().numpy()[0], ref["loss"], rtol, "loss")


@pytest.mark.parametrize("name", list(CASES))
def test_backward(torch_cuda, name):
    torch = torch_cuda
    w, inp, bias = case_inputs(name, seed=1)
    note("backward %s" % name)
    layer = make_gpu_layer(inp, w, bias_values=bias)
    X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    s = 1.0 / w.B
    loss = torch.empty(1, device="cuda:0")
    dX = layer.backward(X, off, lab, s=s, loss_out=loss)
    torch.cuda.synchronize()
    ref = oracle_grads(w, inp, bias, s)
    rtol = rtol_for(w.value)
    assert_close(layer.dW.cpu().numpy(), ref["dW"], rtol, "dW")
    assert_close(layer.dbias.cpu().numpy(), ref["dbias"], rtol, "dbias")
    assert_close(dX.cpu().numpy(), ref["dX"], rtol, "dX")
    assert_close(loss.cpu().numpy()[0], ref["loss"], rtol, "loss")


def adam_reference(w, inp, bias, s, t=1, lr=1e-3, wd=0.0, m0=None, v0=None):
    r = oracle_grads(w, inp, bias, s)
    W = values_f64(inp.W, w.value)
    L, k = W.shape
    m0 = np.zeros((L, k)) if m0 is None else m0
    v0 = np.zeros((L, k)) if v0 is None else v0
    Wn, mn, vn = oracle.adam(W, m0, v0, r["dW"], t, lr=lr, wd=wd)
    bn, bmn, bvn = oracle.adam(bias.astype(np.float64), np.zeros(L), np.zeros(L), r["dbias"], t,
                               lr=lr, wd=wd)
    return r, Wn, mn, vn, bn, bmn, bvn


def fused_update_bound(r, inp, w, mn, vn, t, lr, b1=0.9, b2=0.999, eps=1e-8):
    """How far rounding the dlogits to bf16 (the fused path) can move each
    slot's Adam update.  dW[l,j] moves by at most
    dd = 2^-9 * sum_b |g[b,l]| |X[b,I[l,j]]|; the update lr * mh / (sqrt(vh) + eps)
    (mh = m/(1-b1^t), vh = v/(1-b2^t)) then moves by at most its first-order
    change through m ((1-b1) dd) and v ((1-b2) 2 |dW| dd)."""
    if w.value == "f32":
        return 0.0
    X = values_f64(inp.X, w.value)
    ag = np.abs(r["g"]).T                      # [L, B]
    L, k = inp.I.shape
    dd = np.empty((L, k))
    for j in range(k):
        dd[:, j] = (ag * np.abs(X[:, inp.I[:, j]]).T).sum(axis=1)
    dd *= 2.0 ** -9
    bc1, bc2 = 1.0 - b1 ** t, 1.0 - b2 ** t
    mh, vh = mn / bc1, vn / bc2
    sv = np.sqrt(vh)
    den = sv + eps
    d_m = (1.0 - b1) * dd / bc1 / den
    d_v = np.abs(mh) * (1.0 - b2) * 2.0 * np.abs(r["dW"]) * dd / bc2 / np.maximum(2.0 * sv * den * den, 1e-300)
    return lr * (d_m + d_v)


@pytest.mark.parametrize("name", ["c1", "c2s", "c3s", "c4s", "c5s", "mx200", "w1024", "w128", "wdense", "k5",
                                  "k100", "b1"])
@pytest.mark.parametrize("wd", [0.0, 1e-4])
def test_unfused_step_and_fused_step(torch_cuda, name, wd):
    torch = torch_cuda
    w, inp, bias = case_inputs(name, seed=2)
    s = 1.0 / w.B
    t, lr = 3, 1e-2
    rng = np.random.default_rng(7)
    L, k = inp.I.shape
    m0 = (rng.standard_normal((L, k)) * 1e-3).astype(np.float32)
    v0 = (rng.random((L, k)) * 1e-5).astype(np.float32)
    r, Wn, mn, vn, bn, _, _ = adam_reference(w, inp, bias, s, t=t, lr=lr, wd=wd,
                                             m0=m0.astype(np.float64), v0=v0.astype(np.float64))
    rtol = rtol_for(w.value)
    # m0, v0 start non-zero so that a dW error shows up in m and v
    for fused in (False, True):
        note("%s step %s wd=%g" % ("fused" if fused else "unfused", name, wd))
        layer = make_gpu_layer(inp, w, bias_values=bias)
        layer.m.copy_(torch.from_numpy(m0))
        layer.v.copy_(torch.from_numpy(v0))
        X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
        if fused:
            loss, dX = layer.train_step(X, off, lab, t=t, s=s, lr=lr, wd=wd)
        else:
            loss = torch.empty(1, device="cuda:0")
            dX = layer.backward(X, off, lab, s=s, loss_out=loss)
            layer.adam_step(t, lr=lr, wd=wd)
        torch.cuda.synchronize()
        check_step_result(w, inp, layer, loss, dX, r, Wn, mn, vn, bn, t, lr, fused)


def check_step_result(w, inp, layer, loss, dX, r, Wn, mn, vn, bn, t, lr, fused):
    """A training step's W, m, v, bias, dX and loss against the oracle's step
    (r: loss_and_grads; Wn, mn, vn, bn: the oracle's Adam results)."""
    rtol = rtol_for(w.value)
    Wbits = from_torch_bits(layer.W, w.value)
    Wg = values_f64(Wbits, w.value)
    W0 = values_f64(inp.W, w.value)
    if w.value == "f32":
        assert_close(Wg - W0, Wn - W0, rtol, "W update")
    else:
        # the stored weight is the oracle's update rounded to bf16; fp32 and
        # float64 results may straddle a rounding boundary in rare slots
        Wref = values_f64(oracle.round_bf16(Wn), "bf16")
        diff = np.abs(Wg - Wref)
        # one bf16 ulp of the larger neighbour, plus an absolute floor for
        # weights that an update drives to ~0: there the fp32 update itself
        # (dW summed in fp32, then m/sqrt(v)) differs from float64 by up to
        # ~1e-5 of its size, which is ~lr.
        allow = 2.0 ** -7 * np.maximum(np.abs(Wg), np.abs(Wref)) + 1e-5 * lr
        if fused:
            allow = allow + 1.5 * fused_update_bound(r, inp, w, mn, vn, t, lr)
        bad = diff > allow
        if bad.any():
            rows = ["slot      gpu          ref(bf16)    oracle       start        allow"]
            for (li, ji) in np.argwhere(bad)[:8]:
                rows.append("%5d,%-3d %+.6e %+.6e %+.6e %+.6e %.2e" % (
                    li, ji, Wg[li, ji], Wref[li, ji], Wn[li, ji], W0[li, ji], allow[li, ji]))
            rows.append("count %d of %d" % (bad.sum(), bad.size))
            raise AssertionError("W off by more than 1 ulp\n" + "\n".join(rows))
        if not fused:
            assert (diff > 0).mean() < 1e-3, (diff > 0).mean()
    assert_close(Wg, Wn, rtol, "W")
    assert_close(layer.m.cpu().numpy(), mn, rtol, "m")
    assert_close(layer.v.cpu().numpy(), vn, rtol, "v")
    assert_close(layer.bias.cpu().numpy(), bn, rtol, "bias")
    assert_close(dX.cpu().numpy(), r["dX"], rtol, "dX")
    assert_close(loss.cpu().numpy()[0], r["loss"], rtol, "loss")


def test_edge_targets(torch_cuda):
    """No positives at all, a sample without positives, repeated labels."""
    torch = torch_cuda
    w = synth.scaled(W1["c1_fp32_L4096"], L=300, B=5, name="edge")
    inp = synth.make_layer_inputs(w, 3)
    bias = np.zeros(w.L, dtype=np.float32)
    for off, lab in [
        (np.zeros(6, dtype=np.int64), np.zeros(0, dtype=np.int32)),
        (np.array([0, 2, 2, 5, 5, 6]), np.array([3, 3, 0, 299, 0, 7], dtype=np.int32)),
    ]:
        note("edge targets nnz=%d" % len(lab))
        inp2 = synth.dataclasses.replace(inp, off=off, lab=lab)
        layer = make_gpu_layer(inp2, w, bias_values=bias, nnz_max=8)
        X, offt, labt = batch_to_gpu(inp.X, off, lab, w.value)
        loss, z = layer.forward_loss(X, offt, labt, s=0.2, logits=True)
        dX = layer.backward(X, offt, labt, s=0.2)
        torch.cuda.synchronize()
        ref = oracle_grads(w, inp2, bias, 0.2)
        assert_close(z.cpu().numpy(), ref["z"], 1e-5, "logits")
        assert_close(loss.cpu().numpy()[0], ref["loss"], 1e-5, "loss")
        assert_close(layer.dW.cpu().numpy(), ref["dW"], 1e-5, "dW")
        assert_close(dX.cpu().numpy(), ref["dX"], 1e-5, "dX")


def test_accumulate_flags(torch_cuda):
    torch = torch_cuda
    w, inp, bias = case_inputs("c4s", seed=4)
    note("accumulate flags c4s")
    layer = make_gpu_layer(inp, w, bias_values=bias)
    X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    base = torch.full((w.B, w.d), 0.5, device="cuda:0")
    loss = torch.full((1,), 2.0, device="cuda:0")
    from paper_2411_03171_amd.ffsl import FFSL_ACCUM_DX, FFSL_ACCUM_LOSS
    layer.backward(X, off, lab, dX_out=base, loss_out=loss, flags=FFSL_ACCUM_DX | FFSL_ACCUM_LOSS)
    torch.cuda.synchronize()
    ref = oracle_grads(w, inp, bias, 1.0 / w.B)
    assert_close(base.cpu().numpy(), ref["dX"] + 0.5, 2e-2, "dX accumulated")
    assert_close(loss.cpu().numpy()[0], ref["loss"] + 2.0, 2e-2, "loss accumulated")


@pytest.mark.parametrize("name", ["c2s", "c4s", "w1024", "c1", "mx320", "k100"])
def test_run_to_run_reproducible_loss_and_weights(torch_cuda, name):
    """Every sum is formed in a fixed order on every path (the fast paths'
    matrix-core dX and fixed reduction trees; the general path's dX adds taken
    wave by wave), so two runs give the same bits: the fused step (loss, W, m,
    dX) and the unfused backward (dW, dX)."""
    torch = torch_cuda
    w, inp, bias = case_inputs(name, seed=5)
    outs = []
    for rep in range(2):
        note("reproducibility %s rep %d" % (name, rep))
        layer = make_gpu_layer(inp, w, bias_values=bias)
        X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
        loss, dX = layer.train_step(X, off, lab, t=1)
        torch.cuda.synchronize()
        unf = make_gpu_layer(inp, w, bias_values=bias)
        dXu = unf.backward(X, off, lab)
        torch.cuda.synchronize()
        outs.append([loss.cpu().numpy().copy(), from_torch_bits(layer.W, w.value).copy(),
                     layer.m.cpu().numpy().copy(), dX.cpu().numpy().copy(), unf.dW.cpu().numpy().copy(),
                     dXu.cpu().numpy().copy()])
    for i, what in enumerate(("loss", "W", "m", "dX", "dW (unfused)", "dX (unfused)")):
        a, b = np.asarray(outs[0][i]), np.asarray(outs[1][i])
        if a.dtype.kind == "f":
            a, b = a.view(np.uint32), b.view(np.uint32)
        assert np.array_equal(a, b), what


def test_errors_are_reported_before_launch(torch_cuda):
    torch = torch_cuda
    from paper_2411_03171_amd.ffsl import FfslError
    w, inp, bias = case_inputs("c1")
    layer = make_gpu_layer(inp, w, bias_values=bias)
    X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    # regrowing more weights than there are inactive columns (d = k)
    wf, inpf, biasf = case_inputs("kfull")
    full = make_gpu_layer(inpf, wf, bias_values=biasf)
    with pytest.raises(FfslError):
        full.set_update(0.1, 0, 0)
    # B above B_max
    Xbig = torch.zeros((w.B + 1, w.d), device="cuda:0")
    offbig = torch.zeros(w.B + 2, dtype=torch.int32, device="cuda:0")
    with pytest.raises(FfslError):
        layer.forward_loss(Xbig, offbig, lab[:0])
    with pytest.raises(FfslError):
        layer.adam_step(0)


def test_workspace_carries_only_what_the_path_uses(torch_cuda):
    """The dW carry and the fast paths' batch buffers are reserved only for
    shapes the fused fast paths take (bf16, fan-in 32 up to width 768 or fan-in
    64 up to 2048): an fp32 layer of the same shape, or a bf16 layer at a width
    off the fast path, needs only the partial sums."""
    from paper_2411_03171_amd import ffsl
    lib = ffsl.load()
    L, B, nnz = 3_145_728, 128, 1024
    bf16 = lib.ffsl_workspace_bytes_ex(L, 768, 32, ffsl.FFSL_BF16, B, nnz)
    f32 = lib.ffsl_workspace_bytes_ex(L, 768, 32, ffsl.FFSL_F32, B, nnz)
    off_path = lib.ffsl_workspace_bytes_ex(L, 320, 32, ffsl.FFSL_BF16, B, nnz)
    carry = 4 * (L * 32 + L)
    assert bf16 >= f32 + carry
    assert off_path < f32 and f32 < carry
    # the call without a type is the bf16 layout (an upper bound for both)
    assert lib.ffsl_workspace_bytes(L, 768, 32, B, nnz) == bf16
    assert lib.ffsl_workspace_bytes_ex(L, 768, 32, 9, B, nnz) == 0


@pytest.mark.parametrize("name", ["c4s", "mx200", "w1024", "c1", "mx320"])
def test_nan_in_x_gives_nan_loss_and_a_normal_return(torch_cuda, name):
    """A NaN in one input column of one sample: the call returns normally, the
    loss is NaN (as the oracle's), the rows that gather that column get NaN
    weights, and the clean samples' dX and the other rows' weights still match
    the oracle.  A clean step afterwards runs as usual."""
    torch = torch_cuda
    w, inp, bias = case_inputs(name, seed=6)
    Xbad = inp.X.copy()
    b_nan, col = 1, 5
    if w.value == "f32":
        Xbad[b_nan, col] = np.nan
    else:
        Xbad[b_nan, col] = 0x7FC0
    inp_bad = synth.dataclasses.replace(inp, X=Xbad)
    # lr as in the step parity test: at 1e-3 the fp32 rounding of the stored
    # W (about 1e-8) would be a visible part of an fp32 update
    s, t, lr = 1.0 / w.B, 3, 1e-2
    # non-zero moments, so that the update is not the first step's lr*sign(dW)
    # (which amplifies the rounding of near-zero gradients)
    rng = np.random.default_rng(8)
    m0 = (rng.standard_normal((w.L, w.k)) * 1e-3).astype(np.float32)
    v0 = (rng.random((w.L, w.k)) * 1e-5).astype(np.float32)
    r, Wn, mn, vn, bn, _, _ = adam_reference(w, inp_bad, bias, s, t=t, lr=lr, m0=m0.astype(np.float64),
                                             v0=v0.astype(np.float64))
    assert np.isnan(r["loss"])
    note("NaN in X %s" % name)
    layer = make_gpu_layer(inp_bad, w, bias_values=bias)
    layer.m.copy_(torch.from_numpy(m0))
    layer.v.copy_(torch.from_numpy(v0))
    X, off, lab = batch_to_gpu(Xbad, inp.off, inp.lab, w.value)
    loss, dX = layer.train_step(X, off, lab, t=t, s=s, lr=lr)
    torch.cuda.synchronize()
    assert np.isnan(float(loss.cpu()[0]))
    touched = np.any(inp.I == col, axis=1)
    assert touched.any() and not touched.all()
    Wg = values_f64(from_torch_bits(layer.W, w.value), w.value)
    assert np.isnan(Wg[touched]).all()
    assert np.isfinite(Wg[~touched]).all()
    rtol = rtol_for(w.value)
    W0 = values_f64(inp.W, w.value)
    if w.value == "f32":
        assert_close(Wg[~touched] - W0[~touched], Wn[~touched] - W0[~touched], rtol,
                     "W update of the rows that do not gather the NaN column")
    else:
        assert_close(Wg[~touched], Wn[~touched], rtol, "W of the rows that do not gather the NaN column")
    clean = np.arange(w.B) != b_nan
    dXg = dX.cpu().numpy()
    assert np.isfinite(dXg[clean]).all()
    assert_close(dXg[clean], r["dX"][clean], rtol, "dX of the clean samples")
    # the device and the library carry on
    note("NaN in X %s: a clean step afterwards" % name)
    layer2 = make_gpu_layer(inp, w, bias_values=bias)
    X2, off2, lab2 = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    loss2, _ = layer2.train_step(X2, off2, lab2, t=1, s=s)
    torch.cuda.synchronize()
    assert np.isfinite(float(loss2.cpu()[0]))

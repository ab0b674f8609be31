"""Parity at full size, in the launch configuration the benchmark times: one
fused training step (ffsl_train_step) on a freshly created layer.

- The largest workload (L = 3 145 728 labels, k = 32, B = 64, d = 768, bf16):
  the oracle runs over the whole layer in row blocks (rows are independent;
  the loss and dX sum over blocks), so every row's W, m, v and bias is
  checked, as are the loss and the full dX.
- The C3 and C5 sparse layers (L = 1 048 576, B = 128; fan-in 64 at width
  2048, fan-in 32 at width 768), whose steps run in several batch passes:
  sampled outputs the oracle computes cheaply, three row blocks' state over
  every sample and four samples' dX over every row."""
import numpy as np
import pytest

import oracle
from paper_2411_03171_amd import synth
from tests.parity import RTOL_BF16, assert_close, from_torch_bits, note, values_f64

pytestmark = pytest.mark.gpu

BLOCK = 1 << 19


def _block_targets(off, lab, r0, r1):
    """CSR targets restricted to labels in [r0, r1), relabelled from 0."""
    B = len(off) - 1
    noff = np.zeros(B + 1, dtype=np.int64)
    parts = []
    for b in range(B):
        seg = lab[off[b]:off[b + 1]]
        seg = seg[(seg >= r0) & (seg < r1)] - r0
        parts.append(seg)
        noff[b + 1] = noff[b] + len(seg)
    return noff, (np.concatenate(parts) if parts else np.zeros(0)).astype(np.int32)


def test_fused_step_full_c4():
    import torch
    from paper_2411_03171_amd import ffsl
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    w = synth.WORKLOADS["c4_bf16_L3M"]
    note("full-size fused step %s: generating inputs" % w.name)
    inp = synth.make_layer_inputs(w, 0)
    dev = "cuda:0"

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    layer = ffsl.SparseLayer(bf(inp.W), torch.from_numpy(inp.I).to(dev),
                             bias=torch.from_numpy(inp.bias).to(dev), B_max=w.B,
                             nnz_max=len(inp.lab), unfused=False).bind(w.d)
    X = bf(inp.X)
    off = torch.from_numpy(inp.off.astype(np.int32)).to(dev)
    lab = torch.from_numpy(inp.lab).to(dev)
    s, lr = 1.0 / w.B, 1e-3
    note("full-size fused step %s: GPU step" % w.name)
    loss, dX = layer.train_step(X, off, lab, t=1, s=s, lr=lr)
    torch.cuda.synchronize()
    Wg = values_f64(from_torch_bits(layer.W, "bf16"), "bf16")
    mg = layer.m.cpu().numpy()
    vg = layer.v.cpu().numpy()
    bg = layer.bias.cpu().numpy()
    loss_g = float(loss.cpu()[0])
    dX_g = dX.cpu().numpy()
    del layer
    torch.cuda.empty_cache()

    note("full-size fused step %s: oracle in blocks of %d rows" % (w.name, BLOCK))
    Xd = values_f64(inp.X, "bf16")
    loss_ref = 0.0
    dX_ref = np.zeros((w.B, w.d))
    for r0 in range(0, w.L, BLOCK):
        r1 = min(w.L, r0 + BLOCK)
        boff, blab = _block_targets(inp.off, inp.lab, r0, r1)
        W0 = values_f64(inp.W[r0:r1], "bf16")
        n = r1 - r0
        r = oracle.train_step(Xd, W0, inp.I[r0:r1], inp.bias[r0:r1].astype(np.float64),
                              np.zeros((n, w.k)), np.zeros((n, w.k)), np.zeros(n), np.zeros(n),
                              boff, blab, s, t=1, lr=lr, w_bf16=True)
        loss_ref += r["loss"]
        dX_ref += r["dX"]
        # W to the bf16 bar; beyond that, the stored weight is within one bf16
        # ulp of the oracle's rounded update (plus the bf16-dlogit allowance)
        # except where the first Adam step, which moves every weight by about
        # lr * sign(dW), meets a gradient so close to zero that rounding the
        # dlogits to bf16 can flip its sign.  That rounding moves dW[l,j] by at
        # most 2^-9 * sum_b |g[b,l]| |X[b,I[l,j]]|, so a flipped slot's reference
        # gradient must lie within that bound (with a margin for fp32 sums).
        assert_close(Wg[r0:r1], r["W"], RTOL_BF16, "W rows %d.." % r0)
        diff = np.abs(Wg[r0:r1] - r["W"])
        allow = 2.0 ** -7 * np.maximum(np.abs(Wg[r0:r1]), np.abs(r["W"])) + 1e-5 * lr + 2.0 ** -7 * lr
        off_l, off_j = np.nonzero(diff > allow)
        assert len(off_l) < 1e-3 * diff.size, len(off_l)
        if len(off_l):
            cols = inp.I[r0:r1][off_l, off_j]
            bound = 2.0 ** -9 * (np.abs(r["g"][:, off_l]) * np.abs(Xd[:, cols])).sum(axis=0)
            dW_off = np.abs(r["dW"][off_l, off_j])
            assert np.all(dW_off <= 1.5 * bound + 1e-6 * np.abs(r["dW"]).max()), \
                float(np.max(dW_off / np.maximum(bound, 1e-30)))
        assert_close(mg[r0:r1], r["m"], RTOL_BF16, "m rows %d.." % r0)
        assert_close(vg[r0:r1], r["v"], RTOL_BF16, "v rows %d.." % r0)
        assert_close(bg[r0:r1], r["bias"], RTOL_BF16, "bias rows %d.." % r0)
        del r
    assert_close(np.array([loss_g]), np.array([loss_ref]), RTOL_BF16, "loss")
    assert_close(dX_g, dX_ref, RTOL_BF16, "dX")


SAMPLED = {
    # the C3 sparse layer (fan-in 64, width 2048: eight 16-sample passes) and
    # the C5 sparse layer (fan-in 32, width 768: two 64-sample passes)
    "c3": synth.dataclasses.replace(synth.WORKLOADS["c3_inter2048_L1M"], din=0),
    "c5": synth.dataclasses.replace(synth.WORKLOADS["c5_aux8192_L1M"], aux_clusters=0),
}
SAMPLE_ROWS = 1 << 15
SAMPLES = [0, 37, 90, 127]


@pytest.mark.parametrize("name", list(SAMPLED))
def test_fused_step_full_sampled(name):
    """The full C3 and C5 sparse layers in the launch configuration the
    benchmark times (all batch passes of one fused step): W, m, v and bias of
    three 32768-row blocks against the oracle over those rows and every
    sample, and four samples' dX rows against the oracle over every row."""
    import torch
    from paper_2411_03171_amd import ffsl
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    w = SAMPLED[name]
    note("full-size sampled step %s: generating inputs" % name)
    inp = synth.make_layer_inputs(w, 2)
    dev = "cuda:0"

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    layer = ffsl.SparseLayer(bf(inp.W), torch.from_numpy(inp.I).to(dev),
                             bias=torch.from_numpy(inp.bias).to(dev), B_max=w.B,
                             nnz_max=len(inp.lab), unfused=False).bind(w.d)
    s, lr = 1.0 / w.B, 1e-3
    note("full-size sampled step %s: GPU step (L=%d k=%d d=%d B=%d)" % (name, w.L, w.k, w.d, w.B))
    _, dX = layer.train_step(bf(inp.X), torch.from_numpy(inp.off.astype(np.int32)).to(dev),
                             torch.from_numpy(inp.lab).to(dev), t=1, s=s, lr=lr)
    torch.cuda.synchronize()
    Wg = values_f64(from_torch_bits(layer.W, "bf16"), "bf16")
    mg, vg, bg = layer.m.cpu().numpy(), layer.v.cpu().numpy(), layer.bias.cpu().numpy()
    dX_g = dX.cpu().numpy()
    del layer
    torch.cuda.empty_cache()

    Xd = values_f64(inp.X, "bf16")
    for r0 in (0, w.L // 2, w.L - SAMPLE_ROWS):
        r1 = r0 + SAMPLE_ROWS
        note("full-size sampled step %s: oracle rows %d.." % (name, r0))
        boff, blab = _block_targets(inp.off, inp.lab, r0, r1)
        n = r1 - r0
        r = oracle.train_step(Xd, values_f64(inp.W[r0:r1], "bf16"), inp.I[r0:r1],
                              inp.bias[r0:r1].astype(np.float64), np.zeros((n, w.k)), np.zeros((n, w.k)),
                              np.zeros(n), np.zeros(n), boff, blab, s, t=1, lr=lr, w_bf16=True)
        assert_close(Wg[r0:r1], r["W"], RTOL_BF16, "W rows %d.." % r0)
        # beyond the bar: within one bf16 ulp of the rounded update, except on
        # the few slots where the bf16 dlogits can flip a near-zero gradient's
        # sign on this first Adam step (bounded as in the C4 test)
        diff = np.abs(Wg[r0:r1] - r["W"])
        allow = 2.0 ** -7 * np.maximum(np.abs(Wg[r0:r1]), np.abs(r["W"])) + 1e-5 * lr + 2.0 ** -7 * lr
        off_l, off_j = np.nonzero(diff > allow)
        assert len(off_l) < 1e-3 * diff.size, len(off_l)
        if len(off_l):
            cols = inp.I[r0:r1][off_l, off_j]
            bound = 2.0 ** -9 * (np.abs(r["g"][:, off_l]) * np.abs(Xd[:, cols])).sum(axis=0)
            dW_off = np.abs(r["dW"][off_l, off_j])
            assert np.all(dW_off <= 1.5 * bound + 1e-6 * np.abs(r["dW"]).max())
        assert_close(mg[r0:r1], r["m"], RTOL_BF16, "m rows %d.." % r0)
        assert_close(vg[r0:r1], r["v"], RTOL_BF16, "v rows %d.." % r0)
        assert_close(bg[r0:r1], r["bias"], RTOL_BF16, "bias rows %d.." % r0)
        del r
    # dX rows of a few samples: their dlogits over every label, scattered
    # through every row (the same loss scale 1/B as the full batch)
    note("full-size sampled step %s: oracle dX of samples %s" % (name, SAMPLES))
    soff = [0]
    slab = []
    for b in SAMPLES:
        seg = inp.lab[inp.off[b]:inp.off[b + 1]]
        slab.extend(seg.tolist())
        soff.append(len(slab))
    ref = oracle.loss_and_grads(Xd[SAMPLES], values_f64(inp.W, "bf16"), inp.I, inp.bias.astype(np.float64),
                                np.array(soff, dtype=np.int64), np.array(slab, dtype=np.int32), s)
    assert_close(dX_g[SAMPLES], ref["dX"], RTOL_BF16, "dX rows %s" % SAMPLES)

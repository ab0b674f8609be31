"""SET at full size: the largest workload (L = 3 145 728 labels, k = 32,
d = 768, bf16) and the C3 sparse layer (L = 1 048 576, k = 64, d = 2048).
The Adam moments start non-zero (seeded), so that zeroing them at the regrown
slots, and leaving them bit for bit at the others, is checked at full size.
The largest workload: both prune modes against the oracle on three blocks of rows
(start, middle, end; the draw counter of a row is its index in the layer, so
a block is checked with the oracle's row offset), and the training step with
SET in one call against the step followed by SET, bit for bit over the whole
layer."""
import numpy as np
import pytest

import oracle
from paper_2411_03171_amd import synth
from tests.parity import from_torch_bits, note

pytestmark = pytest.mark.gpu

C4 = synth.WORKLOADS["c4_bf16_L3M"]
ROWS = 20000


def _layer(inp, w, dev="cuda:0", mv=None):
    import torch
    from paper_2411_03171_amd import ffsl
    W = torch.from_numpy(np.ascontiguousarray(inp.W).view(np.int16)).view(torch.bfloat16).to(dev)
    m = v = None
    if mv is not None:
        m, v = (torch.from_numpy(a).to(dev) for a in mv)
    return ffsl.SparseLayer(W, torch.from_numpy(inp.I).to(dev), bias=torch.from_numpy(inp.bias).to(dev),
                            m=m, v=v, B_max=w.B, nnz_max=len(inp.lab), unfused=False).bind(w.d)


def _moments(L, k, seed):
    """Seeded non-zero Adam moments of a layer (m signed, v positive)."""
    rng = np.random.default_rng(seed)
    m = rng.standard_normal((L, k), dtype=np.float32) * np.float32(1e-3)
    v = rng.random((L, k), dtype=np.float32) * np.float32(1e-5) + np.float32(1e-9)
    return m, v


@pytest.fixture(scope="module")
def c4_inputs():
    note("full-size SET: generating inputs")
    return synth.make_layer_inputs(C4, 0)


@pytest.mark.parametrize("mode", ["fraction", "threshold"])
def test_set_full_c4_against_oracle(c4_inputs, mode):
    import torch
    inp, w = c4_inputs, C4
    seed, rnd = 0xC4C4C4C4, 3
    m0, v0 = _moments(w.L, w.k, 41)
    note("full-size SET %s: GPU" % mode)
    layer = _layer(inp, w, mv=(m0, v0))
    if mode == "fraction":
        mask, ex = layer.set_update(w.set_frac, seed, rnd)
    else:
        mask, ex = layer.set_update_threshold(0.02, seed, rnd)
    torch.cuda.synchronize()
    assert int(ex.cpu()[0]) == 0
    starts = [0, w.L // 2 - ROWS // 2, w.L - ROWS]
    got = []
    for r0 in starts:
        sl = slice(r0, r0 + ROWS)
        got.append((from_torch_bits(layer.W[sl], "bf16"), layer.I[sl].cpu().numpy(), layer.m[sl].cpu().numpy(),
                    layer.v[sl].cpu().numpy(), mask[sl].cpu().numpy()))
    del layer
    torch.cuda.empty_cache()
    for r0, (Wg, Ig, mg, vg, maskg) in zip(starts, got):
        note("full-size SET %s: oracle rows %d.." % (mode, r0))
        sl = slice(r0, r0 + ROWS)
        if mode == "fraction":
            Wr, Ir, mr, vr, maskr, exr = oracle.set_update(inp.W[sl], inp.I[sl], m0[sl], v0[sl], w.d, w.set_frac,
                                                           seed, rnd, row0=r0)
        else:
            Wr, Ir, mr, vr, maskr, exr = oracle.set_update_threshold(inp.W[sl], inp.I[sl], m0[sl], v0[sl], w.d,
                                                                     float(np.float32(0.02)), seed, rnd, row0=r0)
        assert exr == 0
        np.testing.assert_array_equal(Ig, Ir)
        np.testing.assert_array_equal(maskg, maskr)
        np.testing.assert_array_equal(Wg, Wr)
        np.testing.assert_array_equal(mg.view(np.uint32), mr.view(np.uint32))
        np.testing.assert_array_equal(vg.view(np.uint32), vr.view(np.uint32))
        # the moments really were non-zero where SET zeroed them
        assert np.all(m0[sl][maskr == 1] != 0) and np.all(mr[maskr == 1] == 0)


def test_fused_step_set_full_c4_equals_step_then_set(c4_inputs):
    import torch
    inp, w = c4_inputs, C4
    dev = "cuda:0"
    X = torch.from_numpy(np.ascontiguousarray(inp.X).view(np.int16)).view(torch.bfloat16).to(dev)
    off = torch.from_numpy(inp.off.astype(np.int32)).to(dev)
    lab = torch.from_numpy(inp.lab).to(dev)
    mv = _moments(w.L, w.k, 43)
    note("full-size step+SET: one call")
    a = _layer(inp, w, mv=mv)
    la, dXa, ma, exa = a.train_step_set(X, off, lab, t=3, frac=w.set_frac, seed=11, set_round=1)
    note("full-size step+SET: step, then SET")
    b = _layer(inp, w, mv=mv)
    lb, dXb = b.train_step(X, off, lab, t=3)
    mb, exb = b.set_update(w.set_frac, 11, 1)
    torch.cuda.synchronize()
    for name, x, y in (("W", a.W.view(torch.int16), b.W.view(torch.int16)), ("I", a.I, b.I),
                       ("m", a.m.view(torch.int32), b.m.view(torch.int32)),
                       ("v", a.v.view(torch.int32), b.v.view(torch.int32)),
                       ("bias", a.bias.view(torch.int32), b.bias.view(torch.int32)), ("mask", ma, mb),
                       ("dX", dXa.view(torch.int32), dXb.view(torch.int32)),
                       ("loss", la.view(torch.int32), lb.view(torch.int32)), ("exhausted", exa, exb)):
        assert torch.equal(x, y), name
    assert int(ma.sum().item()) == w.L * int(np.floor(w.set_frac * w.k + 1e-9))


def test_set_full_c3_against_oracle():
    """SET on the full C3 sparse layer (L = 1 048 576, k = 64, d = 2048: rows too
    wide for the LDS tiles, so the one-lane-per-row kernel), fraction mode, on
    three row blocks against the oracle."""
    import torch
    w = synth.dataclasses.replace(synth.WORKLOADS["c3_inter2048_L1M"], din=0)
    note("full-size SET c3: generating inputs")
    inp = synth.make_layer_inputs(w, 1)
    seed, rnd = 0xC3C3C3C3, 5
    m0, v0 = _moments(w.L, w.k, 47)
    note("full-size SET c3: GPU")
    layer = _layer(inp, w, mv=(m0, v0))
    mask, ex = layer.set_update(w.set_frac, seed, rnd)
    torch.cuda.synchronize()
    assert int(ex.cpu()[0]) == 0
    starts = [0, w.L // 2 - ROWS // 2, w.L - ROWS]
    got = []
    for r0 in starts:
        sl = slice(r0, r0 + ROWS)
        got.append((from_torch_bits(layer.W[sl], "bf16"), layer.I[sl].cpu().numpy(), layer.m[sl].cpu().numpy(),
                    layer.v[sl].cpu().numpy(), mask[sl].cpu().numpy()))
    del layer
    torch.cuda.empty_cache()
    for r0, (Wg, Ig, mg, vg, maskg) in zip(starts, got):
        note("full-size SET c3: oracle rows %d.." % r0)
        sl = slice(r0, r0 + ROWS)
        Wr, Ir, mr, vr, maskr, exr = oracle.set_update(inp.W[sl], inp.I[sl], m0[sl], v0[sl], w.d, w.set_frac,
                                                       seed, rnd, row0=r0)
        assert exr == 0
        np.testing.assert_array_equal(Ig, Ir)
        np.testing.assert_array_equal(maskg, maskr)
        np.testing.assert_array_equal(Wg, Wr)
        np.testing.assert_array_equal(mg.view(np.uint32), mr.view(np.uint32))
        np.testing.assert_array_equal(vg.view(np.uint32), vr.view(np.uint32))
        assert np.all(v0[sl][maskr == 1] != 0) and np.all(vr[maskr == 1] == 0)

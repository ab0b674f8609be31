"""GPU parity of SET prune-and-regrow: indices, masks and the rewritten W, m, v
must equal the oracle bit for bit on identical (generator-produced) state."""
import zlib

import numpy as np
import pytest

import oracle
from paper_2411_03171_amd import synth
from tests.parity import from_torch_bits, note, to_torch_values

pytestmark = pytest.mark.gpu


def set_state(seed, L, k, d, value, ties=False):
    rng = np.random.default_rng(seed)
    W = synth.gen_w(rng, L, k, value)
    if ties:
        W32 = (rng.integers(-3, 4, size=(L, k)) * 0.125).astype(np.float32)
        W32[rng.random((L, k)) < 0.1] = -0.0
        W = W32 if value == "f32" else synth.f32_to_bf16_bits(W32)
    I = synth.gen_indices(rng, L, k, d)
    perm = rng.permuted(np.tile(np.arange(k), (L, 1)), axis=1)
    I = np.take_along_axis(I, perm, axis=1).astype(np.int32)
    m = rng.standard_normal((L, k)).astype(np.float32)
    v = rng.random((L, k)).astype(np.float32)
    return W, I, m, v


def bits(W, value):
    return W.view(np.uint32) if value == "f32" else W


def run_gpu_set(W, I, m, v, d, value, frac, seed, rnd, tau=None):
    import torch
    from paper_2411_03171_amd.ffsl import SparseLayer
    dev = "cuda:0"
    layer = SparseLayer(to_torch_values(W, value, dev), torch.from_numpy(I).to(dev), bias=None,
                        m=torch.from_numpy(m), v=torch.from_numpy(v), B_max=1, nnz_max=1,
                        unfused=False).bind(d)
    if tau is None:
        mask, ex = layer.set_update(frac, seed, rnd)
    else:
        mask, ex = layer.set_update_threshold(tau, seed, rnd)
    torch.cuda.synchronize()
    return (from_torch_bits(layer.W, value), layer.I.cpu().numpy(), layer.m.cpu().numpy(),
            layer.v.cpu().numpy(), mask.cpu().numpy(), int(ex.cpu().numpy()[0]))


CASES = [
    # name, L, k, d, value, frac, ties
    ("c1", 4096, 16, 128, "f32", 0.3, False),
    ("c1ties", 4096, 16, 128, "f32", 0.3, True),
    ("c2", 5000, 32, 768, "bf16", 0.1, False),
    ("c2ties", 3000, 32, 768, "bf16", 0.25, True),
    ("c3", 2000, 64, 2048, "bf16", 0.1, False),
    ("k5", 1000, 5, 40, "bf16", 0.5, False),
    ("k100", 700, 100, 768, "bf16", 0.2, False),
    ("forced", 1000, 8, 10, "bf16", 0.25, False),   # d = k + n: regrown set forced
    ("all", 500, 8, 16, "f32", 1.0, False),         # every weight replaced
    ("none", 300, 16, 64, "bf16", 0.05, False),     # n = 0
    # rows too wide for two LDS-tiled workgroups per CU: one row per lane in registers
    ("f32_k32_ties", 3000, 32, 768, "f32", 0.25, True),   # n = 8: accepted columns past four in LDS
    ("w2048_k32", 2000, 32, 2048, "bf16", 0.1, False),
    ("k64_tight", 500, 64, 70, "bf16", 0.09, False),      # n = 5 of 6 free columns
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_set_bit_exact(case):
    name, L, k, d, value, frac, ties = case
    note("set %s L=%d k=%d d=%d frac=%g" % (name, L, k, d, frac))
    W, I, m, v = set_state(zlib.crc32(name.encode()) & 0xffff, L, k, d, value, ties)
    seed, rnd = 0x1234567890ABCDEF, 7
    Wg, Ig, mg, vg, maskg, exg = run_gpu_set(W, I, m, v, d, value, frac, seed, rnd)
    Wr, Ir, mr, vr, maskr, exr = oracle.set_update(bits(W, value), I, m, v, d, frac, seed, rnd)
    assert exg == exr == 0
    assert np.array_equal(Ig, Ir)
    assert np.array_equal(maskg, maskr)
    assert np.array_equal(bits(Wg, value), Wr)
    assert np.array_equal(mg.view(np.uint32), mr.view(np.uint32))
    assert np.array_equal(vg.view(np.uint32), vr.view(np.uint32))


def test_set_consecutive_rounds(tmp_path):
    """Two rounds in a row on the GPU equal two oracle rounds."""
    import torch
    from paper_2411_03171_amd.ffsl import SparseLayer
    L, k, d, value = 2000, 32, 768, "bf16"
    W, I, m, v = set_state(5, L, k, d, value)
    note("set consecutive rounds")
    dev = "cuda:0"
    layer = SparseLayer(to_torch_values(W, value, dev), torch.from_numpy(I).to(dev), bias=None,
                        m=torch.from_numpy(m), v=torch.from_numpy(v), B_max=1, nnz_max=1,
                        unfused=False).bind(d)
    layer.set_update(0.1, 42, 0)
    layer.set_update(0.1, 42, 1)
    torch.cuda.synchronize()
    s1 = oracle.set_update(W, I, m, v, d, 0.1, 42, 0)
    s2 = oracle.set_update(s1[0], s1[1], s1[2], s1[3], d, 0.1, 42, 1)
    assert np.array_equal(layer.I.cpu().numpy(), s2[1])
    assert np.array_equal(from_torch_bits(layer.W, value), s2[0])


TH_CASES = [
    # name, L, k, d, value, tau, ties
    ("c2_tau05", 5000, 32, 768, "bf16", 0.05, False),
    ("c2_tau01", 3000, 32, 768, "bf16", 0.01, False),
    ("ties_at_tau", 3000, 32, 768, "bf16", 0.125, True),    # |W| = tau is kept
    ("c1_f32", 4096, 16, 128, "f32", 0.1, False),
    ("c3", 2000, 64, 2048, "bf16", 0.02, False),
    ("k100", 700, 100, 768, "bf16", 0.03, False),
    ("none", 300, 16, 64, "bf16", 0.0, False),
    ("all", 400, 8, 64, "f32", float("inf"), False),
    ("exhausts", 600, 8, 12, "bf16", 0.2, False),          # rows with n > d - k stay unchanged
    ("c3_many", 1000, 64, 2048, "bf16", 0.1, False),       # tens of slots per row
    ("k64_exhausts", 300, 64, 67, "bf16", 0.004, False),   # one-lane rows, some run out of draws
]


@pytest.mark.parametrize("case", TH_CASES, ids=[c[0] for c in TH_CASES])
def test_set_threshold_bit_exact(case):
    """Threshold prune mode: the GPU equals the oracle bit for bit, including
    the per-row counts and rows that run out of draws."""
    name, L, k, d, value, tau, ties = case
    tau = float(np.float32(tau))   # the value the library receives
    note("set threshold %s L=%d k=%d d=%d tau=%g" % (name, L, k, d, tau))
    W, I, m, v = set_state(zlib.crc32(name.encode()) & 0xffff, L, k, d, value, ties)
    if value == "f32" and name == "c1_f32":
        W = W.copy()
        W[7, 2] = np.nan
    seed, rnd = 0x0F1E2D3C4B5A6978, 11
    Wg, Ig, mg, vg, maskg, exg = run_gpu_set(W, I, m, v, d, value, 0.0, seed, rnd, tau=tau)
    Wr, Ir, mr, vr, maskr, exr = oracle.set_update_threshold(bits(W, value), I, m, v, d, tau, seed, rnd)
    assert exg == exr
    if name.endswith("exhausts"):
        assert exr > 0
    else:
        assert exr == 0
    assert np.array_equal(Ig, Ir)
    assert np.array_equal(maskg, maskr)
    assert np.array_equal(bits(Wg, value), Wr)
    assert np.array_equal(mg.view(np.uint32), mr.view(np.uint32))
    assert np.array_equal(vg.view(np.uint32), vr.view(np.uint32))
    counts = maskr.sum(axis=1)
    if name not in ("none", "all") and not name.endswith("exhausts"):
        assert counts.min() < counts.max()     # the count varies by row

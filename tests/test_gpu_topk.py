"""GPU parity of top-k inference (ffsl_infer_topk) against the oracle.

The kernel's scores are fp32 sums; the oracle's are float64.  Where two labels'
scores are closer than the rounding of those sums, either order is correct.
So each sample's result is checked as follows:
- the returned scores equal the oracle's scores of the returned labels,
  within a bound derived from the sums;
- the list is sorted by (score desc, label asc) and holds distinct labels;
- no label left out scores above the last returned one by more than that
  bound (nothing is missed);
- every oracle top-k label whose margin over the k-th score exceeds the bound
  is returned (the unique part agrees exactly).
P@k is compared with the oracle's P@k of the returned labels, and with the
oracle's own top-k where the sets agree.  Cases with exact ties (zero weights,
so a score is its bias) must match the oracle label for label, including
-inf and NaN scores.  Shapes: the largest label space's layout (fan-in 32, 64
samples, width 768) in one and two batch tiles, fan-in 64 at width 2048, odd
fan-in, a partial 32-slot round, fp32, ragged tiles, topk from 1 to 16,
topk = L, and label spaces large enough that more than 256 scan workgroups
meet in the merge."""
import numpy as np
import pytest

import oracle
from paper_2411_03171_amd import synth
from tests.parity import batch_to_gpu, make_gpu_layer, note, values_f64

pytestmark = pytest.mark.gpu

W1 = synth.WORKLOADS
C4 = W1["c4_bf16_L3M"]
CASES = {
    "c4s": synth.scaled(C4, L=3001, name="c4s"),
    "c4s_b100": synth.scaled(C4, L=2111, B=100, name="c4s_b100"),
    "c3s": synth.dataclasses.replace(synth.scaled(W1["c3_inter2048_L1M"], L=1500, B=40, name="c3s"), din=0),
    "c1": W1["c1_fp32_L4096"],
    "odd_k7": synth.scaled(C4, L=777, B=5, d=50, k=7, name="odd_k7"),
    "k40_f32": synth.dataclasses.replace(synth.scaled(W1["c1_fp32_L4096"], L=901, B=70, d=256, k=40,
                                                      name="k40_f32")),
    "b1": synth.scaled(C4, L=513, B=1, name="b1"),
    # one sample per lane (16-sample tiles) fits two scan workgroups per CU:
    # with this many rows the merge takes more than 256 workgroup lists per
    # sample
    "c1_bigL": synth.scaled(W1["c1_fp32_L4096"], L=120000, B=16, name="c1_bigL"),
    "b16_bigL": synth.scaled(C4, L=90000, B=16, d=256, name="b16_bigL"),
}
TOPKS = {"c4s": [1, 2, 3, 5, 7, 8, 16], "c4s_b100": [5], "c3s": [3, 16], "c1": [5, 12], "odd_k7": [2, 9],
         "k40_f32": [4], "b1": [1, 16], "c1_bigL": [4], "b16_bigL": [8]}


@pytest.fixture(scope="module")
def ffsl_mod():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2411_03171_amd import ffsl
    ffsl.load()
    return ffsl


def _inputs(name, seed):
    w = CASES[name]
    inp = synth.make_layer_inputs(w, seed)
    rng = np.random.default_rng(700 + seed)
    bias = (rng.standard_normal(w.L) * 0.3).astype(np.float32)
    return w, inp, bias


def _oracle_scores(w, inp, bias):
    X = values_f64(inp.X, w.value)
    W = values_f64(inp.W, w.value)
    z = oracle.forward(X, W, inp.I, bias.astype(np.float64))
    # a bound on the fp32 rounding of each score: the sum of the magnitudes of its terms
    za = oracle.forward(np.abs(X), np.abs(W), inp.I, np.abs(bias).astype(np.float64))
    return z, 1e-5 * za + 1e-30


def _targets_with_hits(z, K, seed):
    """Positives that include some of the oracle's best labels, so P@k is not
    trivially zero (oracle-derived inputs)."""
    rng = np.random.default_rng(seed)
    top, _ = oracle.topk(z, K)
    B, L = z.shape
    off, lab = [0], []
    for b in range(B):
        pos = [int(t) for t in top[b] if t >= 0 and rng.random() < 0.5]
        pos += rng.integers(0, L, size=rng.integers(0, 4)).tolist()
        if pos:
            pos.append(pos[0])   # a repeated positive counts once
        lab += pos
        off.append(len(lab))
    return np.array(off, dtype=np.int64), np.array(lab, dtype=np.int32)


def check_topk(top, sc, z, tol, K):
    B, L = z.shape
    ref_top, _ = oracle.topk(z, K)
    for b in range(B):
        lab, s = top[b], sc[b]
        sel = lab[lab >= 0]
        n = len(sel)
        assert (lab[n:] == -1).all() and np.all(sc[b, n:] == -np.inf), (b, lab)
        assert len(set(sel.tolist())) == n and sel.max(initial=0) < L, (b, lab)
        # returned scores are the labels' scores
        assert np.all(np.abs(s[:n] - z[b, sel]) <= tol[b, sel]), (b, s[:n], z[b, sel])
        # sorted by (score desc, label asc)
        for j in range(n - 1):
            assert s[j] > s[j + 1] or (s[j] == s[j + 1] and sel[j] < sel[j + 1]), (b, j, s, sel)
        selectable = ~np.isnan(z[b])
        assert n == min(K, int(selectable.sum())), (b, n)
        if n == 0:
            continue
        # nothing missed: labels left out score at most the last one plus the bound
        rest = selectable.copy()
        rest[sel] = False
        zk = z[b, sel].min()
        slack = tol[b, sel].max() + tol[b]
        assert np.all(z[b, rest] <= zk + slack[rest]), (b, np.nonzero(z[b, rest] > zk + slack[rest]))
        # the unique part of the oracle's top-k is returned
        rt = ref_top[b][ref_top[b] >= 0]
        zk_ref = z[b, rt].min()
        clear = rt[z[b, rt] > zk_ref + 2 * tol[b, rt].max() + 2 * tol[b, rt]]
        assert set(clear.tolist()) <= set(sel.tolist()), (b, clear, sel)
    return ref_top


@pytest.mark.parametrize("name,K", [(n, k) for n in CASES for k in TOPKS[n]])
def test_topk_against_oracle(ffsl_mod, name, K):
    import torch
    w, inp, bias = _inputs(name, seed=K)
    z, tol = _oracle_scores(w, inp, bias)
    off, lab = _targets_with_hits(z, K, seed=K)
    note("topk %s K=%d (L=%d k=%d d=%d B=%d %s)" % (name, K, w.L, w.k, w.d, w.B, w.value))
    layer = make_gpu_layer(inp, w, bias_values=bias, nnz_max=max(len(lab), 1))
    X, offt, labt = batch_to_gpu(inp.X, off, lab, w.value)
    top, sc, p = layer.infer_topk(X, K, offt, labt)
    torch.cuda.synchronize()
    top, sc, p = top.cpu().numpy(), sc.cpu().numpy().astype(np.float64), p.cpu().numpy()
    ref_top = check_topk(top, sc, z, tol, K)
    np.testing.assert_allclose(p, oracle.precision_at_k(top, off, lab), rtol=1e-6, atol=1e-7)
    same = np.all(top == ref_top, axis=1)
    assert same.mean() > 0.9, same.mean()
    if same.all():
        np.testing.assert_allclose(p, oracle.precision_at_k(ref_top, off, lab), rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("value", ["bf16", "f32"])
def test_topk_exact_ties(ffsl_mod, value):
    """Zero weights: every score is its bias exactly, on both sides.  Biases
    drawn from a few values (many exact ties, both signs of zero), with -inf
    and NaN among them: the result must equal the oracle's label for label."""
    import torch
    w = synth.scaled(C4, L=1999, B=19, d=96, k=32, name="ties")
    if value == "f32":
        w = synth.dataclasses.replace(w, value="f32")
    inp = synth.make_layer_inputs(w, 3)
    inp.W = np.zeros_like(inp.W)
    rng = np.random.default_rng(9)
    bias = rng.choice(np.array([1.5, 0.25, 0.0, -0.0, -1.0, -np.inf, np.nan], dtype=np.float32), size=w.L,
                      p=[0.002, 0.004, 0.3, 0.3, 0.2, 0.1, 0.094])
    K = 16
    z = oracle.forward(values_f64(inp.X, w.value), values_f64(inp.W, w.value), inp.I, bias.astype(np.float64))
    ref_top, ref_sc = oracle.topk(z, K)
    note("topk ties %s" % value)
    layer = make_gpu_layer(inp, w, bias_values=bias)
    X, _, _ = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    top, sc, _ = layer.infer_topk(X, K)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(top.cpu().numpy(), ref_top)
    np.testing.assert_array_equal(sc.cpu().numpy().astype(np.float64), ref_sc)


def test_topk_few_selectable_and_k_equal_l(ffsl_mod):
    """topk = L on a tiny layer (the whole order), and rows where most scores
    are NaN so fewer than topk labels can be returned."""
    import torch
    w = synth.scaled(W1["c1_fp32_L4096"], L=12, B=9, d=40, k=6, name="tiny")
    inp = synth.make_layer_inputs(w, 4)
    bias = np.linspace(-1, 1, w.L).astype(np.float32)
    for K, nan_from in ((12, None), (12, 5), (3, 10)):
        bv = bias.copy()
        if nan_from is not None:
            bv[nan_from:] = np.nan
        z, tol = _oracle_scores(w, inp, bv)
        note("topk tiny K=%d nan_from=%s" % (K, nan_from))
        layer = make_gpu_layer(inp, w, bias_values=bv)
        X, _, _ = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
        top, sc, _ = layer.infer_topk(X, K)
        torch.cuda.synchronize()
        check_topk(top.cpu().numpy(), sc.cpu().numpy().astype(np.float64), z, tol, K)


def test_topk_full_size_sampled(ffsl_mod):
    """The largest label space (L = 3 145 728, fan-in 32, 64 samples, width
    768), as the benchmark runs it; the oracle scores 4 of the samples."""
    import torch
    w = C4
    inp = synth.make_layer_inputs(w, 0)
    rng = np.random.default_rng(1)
    bias = (rng.standard_normal(w.L) * 0.3).astype(np.float32)
    K = 5
    note("topk full size L=%d" % w.L)
    layer = make_gpu_layer(inp, w, bias_values=bias, unfused=False)
    X, _, _ = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    top, sc, _ = layer.infer_topk(X, K)
    torch.cuda.synchronize()
    top, sc = top.cpu().numpy(), sc.cpu().numpy().astype(np.float64)
    rows = np.array([0, 17, 40, 63])
    Xs = values_f64(inp.X, w.value)[rows]
    Wv = values_f64(inp.W, w.value)
    z = oracle.forward(Xs, Wv, inp.I, bias.astype(np.float64))
    za = oracle.forward(np.abs(Xs), np.abs(Wv), inp.I, np.abs(bias).astype(np.float64))
    check_topk(top[rows], sc[rows], z, 1e-5 * za + 1e-30, K)

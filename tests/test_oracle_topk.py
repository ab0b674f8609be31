"""Pins of the oracle's inference functions (CPU): the top-k selection and
Precision@k (appendix on evaluation metrics).

- A hand-computed case with known top lists and P@1..P@3.
- Top-k against numpy's lexsort, an independent library sort, on rows with
  many exact ties, NaN scores and -inf scores.  K ranges from 1 to L.
- Precision@k against a set-based count in plain Python, with repeated
  positives and empty (-1) entries.
- The composed inference pass against a dense masked product.
"""
import numpy as np
import pytest

import oracle




def _lexsort_topk(z, K):
    B, L = z.shape
    lab = np.full((B, K), -1, dtype=np.int32)
    sc = np.full((B, K), -np.inf)
    for b in range(B):
        order = np.lexsort((np.arange(L), -z[b]))   # score descending, then label ascending
        order = [l for l in order if not np.isnan(z[b, l])][:K]
        lab[b, :len(order)] = order
        sc[b, :len(order)] = z[b, order]
    return lab, sc


def test_topk_hand_example():
    z = np.array([[0.9, 0.1, 0.5, 0.7],
                  [1.0, 1.0, np.nan, 1.0]])
    lab, sc = oracle.topk(z, 3)
    assert lab.tolist() == [[0, 3, 2], [0, 1, 3]]
    assert sc.tolist() == [[0.9, 0.7, 0.5], [1.0, 1.0, 1.0]]
    lab4, sc4 = oracle.topk(z, 4)
    assert lab4.tolist() == [[0, 3, 2, 1], [0, 1, 3, -1]]
    assert sc4[1, 3] == -np.inf
    # positives {2, 3} and {1}: P@1 = 0, P@2 = (1/2 + 1/2)/2, P@3 = (2/3 + 1/3)/2
    p = oracle.precision_at_k(lab, np.array([0, 2, 3]), np.array([2, 3, 1]))
    np.testing.assert_allclose(p, [0.0, 0.5, 0.5], rtol=0, atol=1e-15)


@pytest.mark.parametrize("K", [1, 3, 5, 16, 64, 300])
def test_topk_against_lexsort(K):
    rng = np.random.default_rng(K)
    B, L = 7, 300
    z = np.round(rng.standard_normal((B, L)) * 4) / 4   # many exact ties
    z[rng.random((B, L)) < 0.05] = np.nan
    z[rng.random((B, L)) < 0.03] = -np.inf
    z[3, :] = 0.5                                       # a row of equal scores
    z[5, :] = np.nan                                    # nothing selectable
    z[6, :290] = np.nan                                 # fewer than K selectable
    lab, sc = oracle.topk(z, K)
    ref_lab, ref_sc = _lexsort_topk(z, K)
    np.testing.assert_array_equal(lab, ref_lab)
    np.testing.assert_array_equal(sc, ref_sc)


def test_topk_is_the_full_order_at_k_equal_l():
    rng = np.random.default_rng(3)
    z = rng.standard_normal((4, 50))
    lab, sc = oracle.topk(z, 50)
    for b in range(4):
        assert sorted(lab[b].tolist()) == list(range(50))
        assert np.all(np.diff(sc[b]) <= 0)
        np.testing.assert_array_equal(sc[b], z[b, lab[b]])


def _precision_sets(top, off, lab):
    B, K = top.shape
    out = np.zeros(K)
    for b in range(B):
        pos = set(lab[off[b]:off[b + 1]].tolist())
        for k in range(1, K + 1):
            out[k - 1] += sum(1 for t in top[b, :k] if t >= 0 and t in pos) / k
    return out / B


def test_precision_at_k_against_sets():
    rng = np.random.default_rng(11)
    B, L, K = 40, 60, 8
    top = np.stack([rng.permutation(L)[:K] for _ in range(B)]).astype(np.int32)
    top[rng.random((B, K)) < 0.1] = -1
    counts = rng.integers(0, 12, size=B)
    off = np.concatenate([[0], np.cumsum(counts)])
    lab = rng.integers(0, L, size=off[-1]).astype(np.int32)   # repeats possible
    lab[::7] = top.ravel()[: len(lab[::7])].clip(0)           # make hits likely
    np.testing.assert_allclose(oracle.precision_at_k(top, off, lab), _precision_sets(top, off, lab),
                               rtol=0, atol=1e-14)


def test_precision_at_k_extremes():
    top = np.array([[4, 2, 9], [1, 0, 3]], dtype=np.int32)
    # every predicted label relevant: P@k = 1
    off = np.array([0, 3, 6])
    lab = np.array([9, 4, 2, 3, 1, 0], dtype=np.int32)
    np.testing.assert_array_equal(oracle.precision_at_k(top, off, lab), [1.0, 1.0, 1.0])
    # no positives at all: P@k = 0
    np.testing.assert_array_equal(oracle.precision_at_k(top, np.array([0, 0, 0]), np.zeros(0, np.int32)),
                                  [0.0, 0.0, 0.0])


def test_infer_topk_composition_against_dense_product():
    rng = np.random.default_rng(5)
    B, d, L, k, K = 6, 20, 90, 5, 7
    X = rng.standard_normal((B, d))
    I = np.stack([rng.choice(d, size=k, replace=False) for _ in range(L)]).astype(np.int32)
    W = rng.standard_normal((L, k))
    bias = rng.standard_normal(L)
    M = np.zeros((L, d))
    for l in range(L):
        M[l, I[l]] = W[l]
    z = X @ M.T + bias
    off = np.array([0, 2, 2, 5, 6, 9, 12])
    lab = rng.integers(0, L, size=12).astype(np.int32)
    top, sc, p = oracle.infer_topk(X, W, I, bias, K, off, lab)
    ref_lab, ref_sc = _lexsort_topk(z, K)
    np.testing.assert_array_equal(top, ref_lab)
    np.testing.assert_allclose(sc, ref_sc, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(p, _precision_sets(ref_lab, off, lab), rtol=0, atol=1e-14)

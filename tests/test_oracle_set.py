"""Pins of the oracle's SET prune-and-regrow and of its Philox generator.

Philox4x64-10 is pinned to numpy.random.Philox, an independent library
implementation of the SC'11 generator.  The SET draw stream is then re-derived
here in plain Python on top of numpy's Philox (not the oracle's), so a wrong
counter layout, word order, column map or acceptance rule in the oracle fails.
Selection is pinned to a stable argsort of |W| and to brute force; the
invariants the paper fixes (fan-in stays k, as many regrown as pruned, regrown
weights start at zero) are checked on every case.
"""
import itertools

import numpy as np
import pytest

from paper_2411_03171_amd import synth

SET_KEY_HI = 0x5345545F52454752  # "SET_REGR"
MASK64 = (1 << 64) - 1


def numpy_philox_block(ctr, key):
    """Philox4x64-10 block at counter `ctr` via numpy (which pre-increments)."""
    v = sum(int(c) << (64 * i) for i, c in enumerate(ctr))
    v = (v - 1) % (1 << 256)
    c = np.array([(v >> (64 * i)) & MASK64 for i in range(4)], dtype=np.uint64)
    g = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=c)
    return g.random_raw(4)


@pytest.mark.parametrize("trial", range(40))
def test_philox_matches_numpy(oracle, trial):
    rng = np.random.default_rng(trial)
    ctr = rng.integers(0, 2**64, size=4, dtype=np.uint64, endpoint=False)
    if trial % 4 == 0:
        ctr[0] = 0          # borrow through the word boundary in the reference
    if trial % 5 == 0:
        ctr[:] = 0
    key = rng.integers(0, 2**64, size=2, dtype=np.uint64, endpoint=False)
    got = oracle.philox4x64_10(ctr, key)
    ref = numpy_philox_block(ctr, key)
    assert np.array_equal(got, ref)


def absbits(Wbits):
    if Wbits.dtype == np.uint16:
        return (Wbits & 0x7FFF).astype(np.int64)
    return (Wbits & 0x7FFFFFFF).astype(np.int64)


def python_set(Wbits, I, d, frac, seed, set_round, allow=False, row0=0):
    """The SET contract re-derived in plain Python on numpy's Philox."""
    Wb, I = Wbits.copy(), I.copy()
    L, k = I.shape
    n = int(np.floor(frac * k + 1e-9))
    mask = np.zeros((L, k), dtype=np.uint8)
    cap = 64 * k + 4096
    keys = absbits(Wbits)
    for l in range(L):
        order = np.lexsort((np.arange(k), keys[l]))
        pruned = sorted(order[:n].tolist())
        pre = set(I[l].tolist())
        if allow:
            pre -= {int(I[l, p]) for p in pruned}
        acc = []
        block = None
        for a in range(cap):
            if len(acc) == n:
                break
            if a % 4 == 0:
                block = numpy_philox_block((row0 + l, set_round, a // 4, 0), (seed, SET_KEY_HI))
            c = (int(block[a % 4]) * d) >> 64
            if c not in pre and c not in acc:
                acc.append(c)
        assert len(acc) == n
        for p, c in zip(pruned, acc):
            I[l, p] = c
            Wb[l, p] = 0
            mask[l, p] = 1
    return Wb, I, mask


def make_state(seed, L, k, d, value="bf16", ties=False):
    rng = np.random.default_rng(seed)
    W = synth.gen_w(rng, L, k, value)
    if ties:   # many exact ties, signed zeros
        W32 = rng.integers(-3, 4, size=(L, k)).astype(np.float32) * 0.125
        W32[rng.random((L, k)) < 0.1] = -0.0
        W = W32 if value == "f32" else synth.f32_to_bf16_bits(W32)
    if value == "f32":
        W = W.view(np.uint32)
    I = synth.gen_indices(rng, L, k, d)
    perm = rng.permuted(np.tile(np.arange(k), (L, 1)), axis=1)
    I = np.take_along_axis(I, perm, axis=1)
    m = rng.standard_normal((L, k)).astype(np.float32)
    v = rng.random((L, k)).astype(np.float32)
    return W, I, m, v


def check_invariants(W0, I0, m0, v0, W1, I1, m1, v1, mask, d, n):
    L, k = I0.shape
    for l in range(L):
        assert len(set(I1[l].tolist())) == k                       # fan-in stays k, distinct
    assert I1.min() >= 0 and I1.max() < d
    changed = I1 != I0
    assert np.array_equal(changed, mask.astype(bool))
    assert np.all(mask.sum(axis=1) == n)                           # pruned == regrown
    for l in range(L):
        new = set(I1[l][mask[l] == 1].tolist())
        assert not (new & set(I0[l].tolist()))                    # regrown were inactive
    keep = mask == 0
    assert np.array_equal(W1[keep], W0[keep])                      # survivors untouched
    assert np.array_equal(m1[keep], m0[keep]) and np.array_equal(v1[keep], v0[keep])
    assert np.all(W1[~keep] == 0) and np.all(m1[~keep] == 0) and np.all(v1[~keep] == 0)


@pytest.mark.parametrize("value", ["bf16", "f32"])
@pytest.mark.parametrize("ties", [False, True])
def test_set_matches_python_contract(oracle, value, ties):
    L, k, d, frac = 300, 16, 64, 0.3
    W, I, m, v = make_state(17, L, k, d, value, ties)
    W1, I1, m1, v1, mask, ex = oracle.set_update(W, I, m, v, d, frac, seed=1234, set_round=3)
    assert ex == 0
    Wr, Ir, maskr = python_set(W, I, d, frac, 1234, 3)
    assert np.array_equal(I1, Ir) and np.array_equal(mask, maskr) and np.array_equal(W1, Wr)
    check_invariants(W, I, m, v, W1, I1, m1, v1, mask, d, oracle.set_prune_count(k, frac))


def test_set_selection_is_stable_argsort_of_magnitude(oracle):
    L, k, d, frac = 500, 32, 768, 0.1
    W, I, m, v = make_state(3, L, k, d, "bf16", ties=True)
    _, _, _, _, mask, _ = oracle.set_update(W, I, m, v, d, frac, seed=1, set_round=0)
    n = oracle.set_prune_count(k, frac)
    mag = np.abs(synth.bf16_bits_to_f32(W).astype(np.float64))
    order = np.argsort(mag, axis=1, kind="stable")[:, :n]
    ref = np.zeros((L, k), dtype=np.uint8)
    np.put_along_axis(ref, order, 1, axis=1)
    assert np.array_equal(mask, ref)


def test_set_selection_brute_force_small_rows(oracle):
    rng = np.random.default_rng(8)
    k, d = 6, 12
    for trial in range(30):
        W = synth.f32_to_bf16_bits((rng.integers(-2, 3, size=(1, k)) * 0.5).astype(np.float32))
        I = synth.gen_indices(rng, 1, k, d)
        frac = [0.17, 0.34, 0.5, 0.67][trial % 4]
        n = oracle.set_prune_count(k, frac)
        _, _, _, _, mask, _ = oracle.set_update(W, I, None, None, d, frac, seed=trial, set_round=0)
        keys = absbits(W)[0]
        best = min(itertools.combinations(range(k), n),
                   key=lambda S: sorted((keys[j], j) for j in S))
        # the chosen set is the n smallest (key, slot) pairs
        want = sorted(range(k), key=lambda j: (keys[j], j))[:n]
        assert sorted(want) == sorted(best) or n == 0
        assert sorted(np.nonzero(mask[0])[0].tolist()) == sorted(want)


def test_set_nan_is_never_pruned_before_finite(oracle):
    W = synth.f32_to_bf16_bits(np.array([[np.nan, 0.5, -np.inf, 0.25, 1.0, 2.0]], np.float32))
    I = np.array([[0, 1, 2, 3, 4, 5]], dtype=np.int32)
    _, _, _, _, mask, _ = oracle.set_update(W, I, None, None, 20, 0.5, seed=0, set_round=0)
    assert np.nonzero(mask[0])[0].tolist() == [1, 3, 4]


def test_set_edge_cases(oracle):
    # n == 0
    W, I, m, v = make_state(0, 20, 16, 40)
    W1, I1, m1, v1, mask, _ = oracle.set_update(W, I, m, v, 40, 0.05, seed=0, set_round=0)
    assert np.array_equal(I1, I) and mask.sum() == 0
    # exactly n inactive columns: d = k + n -> the regrown set is forced
    k, n = 8, 2
    d = k + n
    W, I, m, v = make_state(1, 50, k, d)
    W1, I1, m1, v1, mask, ex = oracle.set_update(W, I, m, v, d, 0.25, seed=5, set_round=0)
    assert ex == 0
    for l in range(50):
        assert set(I1[l][mask[l] == 1]) == set(range(d)) - set(I[l])
    check_invariants(W, I, m, v, W1, I1, m1, v1, mask, d, n)
    # too few inactive columns is rejected
    with pytest.raises(ValueError):
        oracle.set_update(W, I, m, v, d, 0.5, seed=5, set_round=0)
    # every weight replaced (frac = 1) when d >= 2k
    W, I, m, v = make_state(2, 30, 4, 8)
    W1, I1, m1, v1, mask, ex = oracle.set_update(W, I, m, v, 8, 1.0, seed=2, set_round=9)
    assert mask.all() and ex == 0
    check_invariants(W, I, m, v, W1, I1, m1, v1, mask, 8, 4)


def test_set_allow_regrow_pruned_variant(oracle):
    W, I, m, v = make_state(4, 200, 8, 12)
    W1, I1, _, _, mask, _ = oracle.set_update(W, I, m, v, 12, 0.5, seed=3, set_round=1,
                                              allow_regrow_pruned=True)
    _, Ir, maskr = python_set(W, I, 12, 0.5, 3, 1, allow=True)
    assert np.array_equal(I1, Ir)
    # survivors' columns are never re-drawn, distinctness holds
    for l in range(200):
        assert len(set(I1[l].tolist())) == 8


def test_set_rounds_and_seeds_differ(oracle):
    W, I, m, v = make_state(5, 100, 16, 128)
    a = oracle.set_update(W, I, m, v, 128, 0.25, seed=1, set_round=0)[1]
    b = oracle.set_update(W, I, m, v, 128, 0.25, seed=1, set_round=1)[1]
    c = oracle.set_update(W, I, m, v, 128, 0.25, seed=2, set_round=0)[1]
    assert not np.array_equal(a, b) and not np.array_equal(a, c)


def test_set_regrowth_is_uniform(oracle):
    # chi-square test over the regrown columns of many rows, d = 64
    L, k, d = 20000, 8, 64
    rng = np.random.default_rng(0)
    W = synth.gen_w(rng, L, k, "bf16")
    I = np.tile(np.arange(k, dtype=np.int32), (L, 1))      # columns 0..7 held
    _, I1, _, _, mask, _ = oracle.set_update(W, I, None, None, d, 0.25, seed=99, set_round=0)
    cols = I1[mask == 1]
    counts = np.bincount(cols, minlength=d)[k:]
    exp = cols.size / (d - k)
    chi2 = ((counts - exp) ** 2 / exp).sum()
    # 55 degrees of freedom: the 0.999 quantile is about 93
    assert chi2 < 93, chi2
    assert counts.min() > 0


def test_set_row_block_equals_whole_layer(oracle):
    W, I, m, v = make_state(6, 400, 16, 96)
    whole = oracle.set_update(W, I, m, v, 96, 0.25, seed=11, set_round=2)
    blk = oracle.set_update(W[150:260], I[150:260], m[150:260], v[150:260], 96, 0.25, seed=11,
                            set_round=2, row0=150)
    assert np.array_equal(whole[1][150:260], blk[1])
    assert np.array_equal(whole[4][150:260], blk[4])
    _, Ir, _ = python_set(W[150:260], I[150:260], 96, 0.25, 11, 2, row0=150)
    assert np.array_equal(Ir, blk[1])


# --------------------------------------------------------------------------
# threshold prune mode (the appendix's "rewire threshold")

def values_of(Wbits):
    if Wbits.dtype == np.uint16:
        return synth.bf16_bits_to_f32(Wbits).astype(np.float64)
    return Wbits.view(np.float32).astype(np.float64)


def python_set_threshold(Wbits, I, d, tau, seed, set_round, row0=0):
    """Threshold SET re-derived in plain Python: the slots with |W| < tau
    (decoded to real numbers here) are pruned, regrowth as in python_set."""
    Wb, I = Wbits.copy(), I.copy()
    L, k = I.shape
    mask = np.zeros((L, k), dtype=np.uint8)
    cap = 64 * k + 4096
    mags = np.abs(values_of(Wbits))
    ex = 0
    for l in range(L):
        pruned = [j for j in range(k) if mags[l, j] < tau]
        n = len(pruned)
        pre = set(I[l].tolist())
        acc = []
        block = None
        for a in range(cap):
            if len(acc) == n:
                break
            if a % 4 == 0:
                block = numpy_philox_block((row0 + l, set_round, a // 4, 0), (seed, SET_KEY_HI))
            c = (int(block[a % 4]) * d) >> 64
            if c not in pre and c not in acc:
                acc.append(c)
        if len(acc) < n:
            ex += 1
            continue
        for p, c in zip(pruned, acc):
            I[l, p] = c
            Wb[l, p] = 0
            mask[l, p] = 1
    return Wb, I, mask, ex


@pytest.mark.parametrize("value", ["bf16", "f32"])
@pytest.mark.parametrize("tau", [0.05, 0.01, 0.125])
def test_set_threshold_matches_python_contract(oracle, value, tau):
    L, k, d = 300, 16, 64
    W, I, m, v = make_state(19, L, k, d, value, ties=(tau == 0.125))
    if value == "f32":
        W = W.copy()
        W[5, 3] = np.float32(np.nan).view(np.uint32)      # NaN is never below tau
    W1, I1, m1, v1, mask, ex = oracle.set_update_threshold(W, I, m, v, d, tau, seed=77, set_round=2)
    Wr, Ir, maskr, exr = python_set_threshold(W, I, d, tau, 77, 2)
    assert ex == exr == 0
    assert np.array_equal(I1, Ir) and np.array_equal(mask, maskr) and np.array_equal(W1, Wr)
    # per-row counts equal the number of magnitudes below tau; the rest of the contract
    n_row = (np.abs(values_of(W)) < tau).sum(axis=1)
    assert np.array_equal(mask.sum(axis=1), n_row)
    assert n_row.min() < n_row.max()                        # the count really varies by row
    for l in range(L):
        assert len(set(I1[l].tolist())) == k
        assert not (set(I1[l][mask[l] == 1].tolist()) & set(I[l].tolist()))
    keep = mask == 0
    assert np.array_equal(W1[keep], W[keep]) and np.array_equal(m1[keep], m[keep])
    assert np.all(W1[~keep] == 0) and np.all(m1[~keep] == 0) and np.all(v1[~keep] == 0)


def test_set_threshold_reduces_to_fraction_mode(oracle):
    """When every row holds exactly n magnitudes below tau, threshold mode is
    fraction mode with frac = n/k, bit for bit."""
    rng = np.random.default_rng(3)
    L, k, d, n = 200, 32, 768, 5
    W32 = (rng.uniform(0.2, 0.5, size=(L, k)) * rng.choice([-1, 1], size=(L, k))).astype(np.float32)
    for l in range(L):
        W32[l, rng.choice(k, size=n, replace=False)] = rng.uniform(-0.09, 0.09, size=n).astype(np.float32)
    W = synth.f32_to_bf16_bits(W32)
    I = synth.gen_indices(rng, L, k, d)
    m = rng.standard_normal((L, k)).astype(np.float32)
    v = rng.random((L, k)).astype(np.float32)
    a = oracle.set_update_threshold(W, I, m, v, d, 0.1, seed=5, set_round=9)
    b = oracle.set_update(W, I, m, v, d, n / k, seed=5, set_round=9)
    for x, y in zip(a[:5], b[:5]):
        assert np.array_equal(x, y)


def test_set_threshold_extremes(oracle):
    L, k, d = 50, 8, 40
    W, I, m, v = make_state(23, L, k, d, "bf16")
    W1, I1, _, _, mask, ex = oracle.set_update_threshold(W, I, m, v, d, 0.0, seed=1, set_round=1)
    assert ex == 0 and mask.sum() == 0 and np.array_equal(I1, I) and np.array_equal(W1, W)
    W1, I1, _, _, mask, ex = oracle.set_update_threshold(W, I, m, v, d, np.inf, seed=1, set_round=1)
    assert ex == 0 and np.all(mask == 1) and np.all(W1 == 0)
    for l in range(L):      # the whole row is new
        assert not (set(I1[l].tolist()) & set(I[l].tolist())) and len(set(I1[l].tolist())) == k

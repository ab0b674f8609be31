"""CPU oracle for the fixed fan-in sparse classification layer.

TEST INFRASTRUCTURE ONLY: the test-suite, the smoke check and the CPU-baseline
leg of the benchmark are the only callers.  The product library never imports
this package, and this package imports nothing from the product.

The arithmetic lives in ``ffsl_oracle.c`` (plain loops, float64); this module
only marshals numpy arrays through ctypes and composes the per-step functions
in the order the method applies them (forward, loss, backward, Adam; SET).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ffsl_oracle.c")
_LIB = os.path.join(_HERE, "libffsl_oracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc into oracle/libffsl_oracle.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-D_GNU_SOURCE", "-fPIC", "-shared", "-Wall",
             "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        i64, u64, dbl, vp = ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p
        L.ffslref_forward.argtypes = [i64, i64, i64, i64, vp, vp, vp, vp, vp]
        L.ffslref_forward.restype = None
        L.ffslref_targets_dense.argtypes = [i64, i64, vp, vp, vp]
        L.ffslref_targets_dense.restype = None
        L.ffslref_bce.argtypes = [i64, vp, vp, dbl, vp]
        L.ffslref_bce.restype = dbl
        L.ffslref_sqhinge.argtypes = [i64, vp, vp, dbl, vp]
        L.ffslref_sqhinge.restype = dbl
        L.ffslref_backward.argtypes = [i64, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp]
        L.ffslref_backward.restype = None
        L.ffslref_adam.argtypes = [i64, vp, vp, vp, vp, i64, dbl, dbl, dbl, dbl, dbl]
        L.ffslref_adam.restype = None
        L.ffslref_round_bf16.argtypes = [dbl]
        L.ffslref_round_bf16.restype = ctypes.c_uint16
        L.ffslref_round_bf16_array.argtypes = [i64, vp, vp]
        L.ffslref_round_bf16_array.restype = None
        L.ffslref_philox4x64_10.argtypes = [vp, vp, vp]
        L.ffslref_philox4x64_10.restype = None
        L.ffslref_set_prune_count.argtypes = [i64, dbl]
        L.ffslref_set_prune_count.restype = i64
        L.ffslref_set_update.argtypes = [i64, i64, i64, ctypes.c_int, vp, vp, vp, vp, vp,
                                         dbl, u64, u64, ctypes.c_int, u64]
        L.ffslref_set_update.restype = i64
        L.ffslref_set_update_threshold.argtypes = [i64, i64, i64, ctypes.c_int, vp, vp, vp, vp, vp,
                                                   dbl, u64, u64, ctypes.c_int, u64]
        L.ffslref_set_update_threshold.restype = i64
        L.ffslref_dense_gelu_fwd.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp]
        L.ffslref_dense_gelu_fwd.restype = None
        L.ffslref_dense_gelu_bwd.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp, vp, vp]
        L.ffslref_dense_gelu_bwd.restype = None
        L.ffslref_aux_bce.argtypes = [i64, i64, i64, i64, vp, vp, vp, vp, vp, dbl, vp, vp, vp, vp]
        L.ffslref_aux_bce.restype = dbl
        L.ffslref_topk.argtypes = [i64, i64, vp, i64, vp, vp]
        L.ffslref_topk.restype = None
        L.ffslref_precision_at_k.argtypes = [i64, i64, vp, vp, vp, vp]
        L.ffslref_precision_at_k.restype = None
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _i64(a):
    return np.ascontiguousarray(a, dtype=np.int64)


# --------------------------------------------------------------------------
# bf16 helpers (bit patterns held as uint16)

def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float64."""
    u32 = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u32.view(np.float32).astype(np.float64)


def round_bf16(x) -> np.ndarray:
    """float64 -> nearest bf16 (ties to even), as uint16 bit patterns."""
    x = _f64(x)
    out = np.empty(x.shape, dtype=np.uint16)
    lib().ffslref_round_bf16_array(x.size, _p(x), _p(out))
    return out


# --------------------------------------------------------------------------
# sparse layer

def forward(X, W, I, bias=None):
    """z[b,l] = bias[l] + sum_j W[l,j] X[b,I[l,j]]  (float64 [B,L])."""
    X, W, I = _f64(X), _f64(W), _i32(I)
    B, d = X.shape
    L, k = W.shape
    b = None if bias is None else _f64(bias)
    z = np.empty((B, L), dtype=np.float64)
    lib().ffslref_forward(B, d, L, k, _p(X), _p(W), _p(I), _p(b), _p(z))
    return z


def targets_dense(B, L, off, lab):
    off, lab = _i64(off), _i32(lab)
    y = np.empty((B, L), dtype=np.uint8)
    lib().ffslref_targets_dense(B, L, _p(off), _p(lab), _p(y))
    return y


def bce(z, y, s):
    """Returns (loss, g) for BCE-with-logits summed and scaled by s."""
    z = _f64(z)
    y = np.ascontiguousarray(y, dtype=np.uint8)
    g = np.empty_like(z)
    loss = lib().ffslref_bce(z.size, _p(z), _p(y), float(s), _p(g))
    return loss, g


def sqhinge(z, y, s):
    """Returns (loss, g) for the squared hinge loss summed and scaled by s."""
    z = _f64(z)
    y = np.ascontiguousarray(y, dtype=np.uint8)
    g = np.empty_like(z)
    loss = lib().ffslref_sqhinge(z.size, _p(z), _p(y), float(s), _p(g))
    return loss, g


LOSSES = {"bce": bce, "sqhinge": sqhinge}


def backward(X, W, I, g, want_dbias=True, want_dx=True):
    X, W, I, g = _f64(X), _f64(W), _i32(I), _f64(g)
    B, d = X.shape
    L, k = W.shape
    dW = np.empty((L, k), dtype=np.float64)
    dbias = np.empty(L, dtype=np.float64) if want_dbias else None
    dX = np.empty((B, d), dtype=np.float64) if want_dx else None
    lib().ffslref_backward(B, d, L, k, _p(X), _p(W), _p(I), _p(g), _p(dW), _p(dbias), _p(dX))
    return dW, dbias, dX


def adam(p, m, v, grad, t, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, wd=0.0):
    """In place on float64 copies; returns (p, m, v)."""
    p, m, v, grad = _f64(p).copy(), _f64(m).copy(), _f64(v).copy(), _f64(grad)
    lib().ffslref_adam(p.size, _p(p), _p(m), _p(v), _p(grad), int(t), lr, b1, b2, eps, wd)
    return p, m, v


def loss_and_grads(X, W, I, bias, off, lab, s, loss="bce"):
    """Forward, the loss (BCE or squared hinge) and both backward products for
    one batch."""
    B = X.shape[0]
    L = W.shape[0]
    z = forward(X, W, I, bias)
    y = targets_dense(B, L, off, lab)
    loss, g = LOSSES[loss](z, y, s)
    dW, dbias, dX = backward(X, W, I, g)
    return dict(z=z, y=y, loss=loss, g=g, dW=dW, dbias=dbias, dX=dX)


def train_step(X, W, I, bias, m, v, bm, bv, off, lab, s, t, lr=1e-3, b1=0.9,
               b2=0.999, eps=1e-8, wd=0.0, w_bf16=False, loss="bce"):
    """One step of the method on the sparse layer: forward, loss (BCE or squared
    hinge), backward, Adam.

    W is float64 (the stored values widened).  With ``w_bf16`` the updated
    weights are rounded to bf16 as a bf16-stored weight would be; the result
    ``W`` is then float64 of those bf16 values.  Returns a dict with the new
    state, the loss and dX.
    """
    r = loss_and_grads(X, W, I, bias, off, lab, s, loss=loss)
    Wn, mn, vn = adam(W, m, v, r["dW"], t, lr, b1, b2, eps, wd)
    if w_bf16:
        Wn = bf16_to_f64(round_bf16(Wn))
    bn, bmn, bvn = adam(bias, bm, bv, r["dbias"], t, lr, b1, b2, eps, wd)
    r.update(W=Wn, m=mn, v=vn, bias=bn, bias_m=bmn, bias_v=bvn)
    return r


# --------------------------------------------------------------------------
# SET

def philox4x64_10(ctr, key):
    c = np.ascontiguousarray(ctr, dtype=np.uint64)
    kk = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.empty(4, dtype=np.uint64)
    lib().ffslref_philox4x64_10(_p(c), _p(kk), _p(out))
    return out


def set_prune_count(k, frac):
    return int(lib().ffslref_set_prune_count(int(k), float(frac)))


def set_update(Wbits, I, m, v, d, frac, seed, set_round, allow_regrow_pruned=False, row0=0):
    """SET on copies of the state.  Wbits is uint16 (bf16) or uint32 (fp32).

    The arrays may be a block of rows starting at layer row ``row0``.

    Returns (Wbits, I, m, v, mask, exhausted_rows).
    """
    Wb = np.ascontiguousarray(Wbits).copy()
    if Wb.dtype == np.uint16:
        wbits = 16
    elif Wb.dtype == np.uint32:
        wbits = 32
    else:
        raise TypeError("Wbits must be uint16 or uint32 bit patterns")
    L, k = Wb.shape
    Ic = _i32(I).copy()
    mc = None if m is None else np.ascontiguousarray(m, dtype=np.float32).copy()
    vc = None if v is None else np.ascontiguousarray(v, dtype=np.float32).copy()
    mask = np.empty((L, k), dtype=np.uint8)
    ex = lib().ffslref_set_update(L, int(d), k, wbits, _p(Wb), _p(Ic), _p(mc), _p(vc),
                                  _p(mask), float(frac), int(seed) & (2**64 - 1),
                                  int(set_round) & (2**64 - 1), int(bool(allow_regrow_pruned)),
                                  int(row0))
    if ex < 0:
        raise ValueError("invalid SET arguments")
    return Wb, Ic, mc, vc, mask, int(ex)


# --------------------------------------------------------------------------
# dense parts

def set_update_threshold(Wbits, I, m, v, d, tau, seed, set_round, allow_regrow_pruned=False, row0=0):
    """SET in threshold mode (every slot with |W| < tau is pruned, as many
    columns regrown in its row) on copies of the state; arguments and result
    as set_update."""
    Wb = np.ascontiguousarray(Wbits).copy()
    if Wb.dtype == np.uint16:
        wbits = 16
    elif Wb.dtype == np.uint32:
        wbits = 32
    else:
        raise TypeError("Wbits must be uint16 or uint32 bit patterns")
    L, k = Wb.shape
    Ic = _i32(I).copy()
    mc = None if m is None else np.ascontiguousarray(m, dtype=np.float32).copy()
    vc = None if v is None else np.ascontiguousarray(v, dtype=np.float32).copy()
    mask = np.empty((L, k), dtype=np.uint8)
    ex = lib().ffslref_set_update_threshold(L, int(d), k, wbits, _p(Wb), _p(Ic), _p(mc), _p(vc),
                                            _p(mask), float(tau), int(seed) & (2**64 - 1),
                                            int(set_round) & (2**64 - 1), int(bool(allow_regrow_pruned)),
                                            int(row0))
    if ex < 0:
        raise ValueError("invalid SET arguments")
    return Wb, Ic, mc, vc, mask, int(ex)


def dense_gelu_fwd(X, W1, c=None):
    X, W1 = _f64(X), _f64(W1)
    B, din = X.shape
    dout = W1.shape[1]
    cc = None if c is None else _f64(c)
    A = np.empty((B, dout))
    H = np.empty((B, dout))
    lib().ffslref_dense_gelu_fwd(B, din, dout, _p(X), _p(W1), _p(cc), _p(A), _p(H))
    return A, H


def dense_gelu_bwd(X, W1, A, dH):
    X, W1, A, dH = _f64(X), _f64(W1), _f64(A), _f64(dH)
    B, din = X.shape
    dout = W1.shape[1]
    dW1 = np.empty((din, dout))
    dc = np.empty(dout)
    dX = np.empty((B, din))
    lib().ffslref_dense_gelu_bwd(B, din, dout, _p(X), _p(W1), _p(A), _p(dH), _p(dW1), _p(dc), _p(dX))
    return dW1, dc, dX


def aux_bce(X, Wa, ca, off, lab, s, L):
    """The auxiliary cluster head over the labels [0, L) (labels outside are
    ignored), cluster(l) = l mod C."""
    X, Wa = _f64(X), _f64(Wa)
    B, d = X.shape
    C = Wa.shape[1]
    cc = None if ca is None else _f64(ca)
    off, lab = _i64(off), _i32(lab)
    Za = np.empty((B, C))
    dWa = np.empty((d, C))
    dca = np.empty(C)
    dXa = np.empty((B, d))
    loss = lib().ffslref_aux_bce(B, d, C, int(L), _p(X), _p(Wa), _p(cc), _p(off), _p(lab), float(s),
                                 _p(Za), _p(dWa), _p(dca), _p(dXa))
    return dict(loss=loss, Za=Za, dWa=dWa, dca=dca, dXa=dXa)


# --------------------------------------------------------------------------
# inference

def topk(z, K):
    """Top-K labels of each row of the scores z [B,L]: descending score, equal
    scores by ascending label, NaN never selected, missing entries -1/-inf.
    Returns (labels int32 [B,K], scores float64 [B,K])."""
    z = _f64(z)
    B, L = z.shape
    lab = np.empty((B, K), dtype=np.int32)
    sc = np.empty((B, K), dtype=np.float64)
    lib().ffslref_topk(B, L, _p(z), K, _p(lab), _p(sc))
    return lab, sc


def precision_at_k(top_lab, off, lab):
    """P@1..P@K averaged over the samples (float64 [K])."""
    top_lab = _i32(top_lab)
    B, K = top_lab.shape
    off, lab = _i64(off), _i32(lab)
    out = np.empty(K, dtype=np.float64)
    lib().ffslref_precision_at_k(B, K, _p(top_lab), _p(off), _p(lab), _p(out))
    return out


def infer_topk(X, W, I, bias, K, off=None, lab=None):
    """Scores of every label (forward), each sample's top-K, and P@k when the
    targets are given: the whole inference pass, composed in that order."""
    z = forward(X, W, I, bias)
    top, sc = topk(z, K)
    p = None if off is None else precision_at_k(top, off, lab)
    return top, sc, p

"""Shared helpers of the parity tests: tolerance metric and input plumbing.

Tolerances (written once here, used by every parity test):
  fp32 values          RTOL_F32  = 1e-5
  bf16 values, fp32 accumulation  RTOL_BF16 = 2e-2
A tensor passes when   max|a-b| <= rtol * max|b|   and   ||a-b||_2 <= rtol * ||b||_2
(scale-relative: entries of dX cancel, so an elementwise relative test would
flag rounding noise on near-zero sums).
"""
from __future__ import annotations

import sys

import numpy as np

from paper_2411_03171_amd import synth

RTOL_F32 = 1e-5
RTOL_BF16 = 2e-2


def rtol_for(value):
    return RTOL_F32 if value == "f32" else RTOL_BF16


def assert_close(got, ref, rtol, what=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), what + ": non-finite values"
    scale = np.max(np.abs(ref)) if ref.size else 0.0
    err = np.max(np.abs(got - ref)) if ref.size else 0.0
    assert err <= rtol * scale + 1e-30, "%s: max err %.3e > %.1e * %.3e" % (what, err, rtol, scale)
    n_err = np.linalg.norm((got - ref).ravel())
    n_ref = np.linalg.norm(ref.ravel())
    assert n_err <= rtol * n_ref + 1e-30, "%s: l2 err %.3e > %.1e * %.3e" % (what, n_err, rtol, n_ref)


def note(msg):
    """Name the case on stdout before a GPU step (flushed)."""
    print("[case] " + msg, flush=True)
    sys.stdout.flush()


def values_f64(arr, value):
    """Stored values (float32 array or bf16 bit patterns) widened to float64."""
    if value == "f32":
        return np.asarray(arr, dtype=np.float32).astype(np.float64)
    return synth.bf16_bits_to_f32(arr).astype(np.float64)


def to_torch_values(arr, value, device):
    import torch
    if value == "f32":
        return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(device)
    t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.uint16).view(np.int16))
    return t.view(torch.bfloat16).to(device)


def from_torch_bits(t, value):
    """GPU tensor of stored values -> numpy (float32, or bf16 bit patterns)."""
    import torch
    t = t.detach().cpu()
    if value == "f32":
        return t.numpy().astype(np.float32)
    return t.view(torch.int16).numpy().view(np.uint16)


def make_gpu_layer(inp, w, device="cuda:0", bias=True, unfused=True, B_max=None, nnz_max=None,
                   bias_values=None):
    import torch
    from paper_2411_03171_amd.ffsl import SparseLayer
    W = to_torch_values(inp.W, w.value, device)
    I = torch.from_numpy(inp.I).to(device)
    b = None
    if bias:
        bv = inp.bias if bias_values is None else bias_values
        b = torch.from_numpy(np.ascontiguousarray(bv, dtype=np.float32)).to(device)
    layer = SparseLayer(W, I, bias=b, B_max=B_max or w.B, nnz_max=nnz_max or max(len(inp.lab), 1),
                        unfused=unfused)
    return layer.bind(w.d)


def batch_to_gpu(X, off, lab, value, device="cuda:0"):
    import torch
    Xt = to_torch_values(X, value, device)
    offt = torch.from_numpy(np.asarray(off, dtype=np.int32)).to(device)
    labt = torch.from_numpy(np.asarray(lab, dtype=np.int32)).to(device)
    return Xt, offt, labt

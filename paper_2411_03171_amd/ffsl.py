"""Python binding of libffsl (the C ABI in include/ffsl.h).

Argument marshalling only: every step of the layer runs in the HIP kernels of
libffsl.so.  PyTorch provides device memory and the current stream.  There is
no fallback: if the library is missing or no GPU is present the calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libffsl.so")

FFSL_OK, FFSL_EINVAL, FFSL_EUNSUPPORTED, FFSL_EHIP = 0, -1, -2, -3
FFSL_F32, FFSL_BF16 = 0, 1
FFSL_ACCUM_DX, FFSL_ACCUM_LOSS, FFSL_LOSS_SQHINGE = 1, 2, 4
FFSL_IDX_I32, FFSL_IDX_U16 = 0, 1
FFSL_TOPK_SCRATCH_BYTES = 32 << 20   # static scratch of ffsl_infer_topk_noalloc per GPU

# (name, restype, argtypes) for every entry point of include/ffsl.h
_i32, _i64, _u32, _u64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint64
_f32, _vp, _sz = ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t
_int = ctypes.c_int
SIGNATURES = {
    "ffsl_last_error": (ctypes.c_char_p, []),
    "ffsl_version": (_int, []),
    "ffsl_workspace_bytes": (_sz, [_i64, _i32, _i32, _i32, _i32]),
    "ffsl_workspace_bytes_ex": (_sz, [_i64, _i32, _i32, _i32, _i32, _i32]),
    "ffsl_create_layer": (_int, [ctypes.POINTER(_vp), _i64, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp,
                                 _vp, _vp, _vp, _vp, _vp, _sz, _i32, _i32]),
    "ffsl_create_layer_ex": (_int, [ctypes.POINTER(_vp), _i64, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp,
                                     _vp, _vp, _vp, _vp, _vp, _vp, _sz, _i32, _i32]),
    "ffsl_destroy_layer": (_int, [_vp]),
    "ffsl_forward_loss": (_int, [_vp, _vp, _i32, _vp, _vp, _i32, _f32, _vp, _vp, _u32, _vp]),
    "ffsl_backward": (_int, [_vp, _vp, _i32, _vp, _vp, _i32, _f32, _vp, _vp, _u32, _vp]),
    "ffsl_adam_step": (_int, [_vp, _i64, _f32, _f32, _f32, _f32, _f32, _vp]),
    "ffsl_train_step": (_int, [_vp, _vp, _i32, _vp, _vp, _i32, _f32, _i64, _f32, _f32, _f32, _f32,
                               _f32, _vp, _vp, _u32, _vp]),
    "ffsl_train_step_set": (_int, [_vp, _vp, _i32, _vp, _vp, _i32, _f32, _i64, _f32, _f32, _f32, _f32,
                                   _f32, _vp, _vp, _u32, _f32, _u64, _u64, _vp, _vp, _vp]),
    "ffsl_set_update": (_int, [_vp, _f32, _u64, _u64, _vp, _vp, _vp]),
    "ffsl_set_update_threshold": (_int, [_vp, _f32, _u64, _u64, _vp, _vp, _vp]),
    "ffsl_validate_indices": (_int, [_vp, _vp, _vp]),
    "ffsl_topk_workspace_bytes": (_sz, [_vp, _i32, _i32]),
    "ffsl_infer_topk": (_int, [_vp, _vp, _i32, _i32, _vp, _vp, _vp, _vp, _i32, _vp, _vp, _sz, _vp]),
    "ffsl_infer_topk_noalloc": (_int, [_vp, _vp, _i32, _i32, _vp, _vp, _vp, _vp, _i32, _vp, _vp]),
    "ffsl_set_timing_events": (_int, [_vp, _vp, _vp]),
    "ffsl_dense_workspace_bytes": (_sz, [_i32, _i32, _i32]),
    "ffsl_dense_gelu_fwd": (_int, [_vp, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp]),
    "ffsl_dense_gelu_bwd": (_int, [_vp, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _u32, _vp, _sz,
                                   _vp]),
    "ffsl_aux_workspace_bytes": (_sz, [_i32, _i32, _i32]),
    "ffsl_aux_bce_fwd_bwd": (_int, [_vp, _i32, _i32, _i32, _i64, _vp, _vp, _vp, _vp, _i32, _f32, _vp, _vp, _vp,
                                    _vp, _vp, _u32, _vp, _sz, _vp]),
    "ffsl_adam_dense": (_int, [_vp, _i32, _vp, _vp, _vp, _i64, _i64, _f32, _f32, _f32, _f32, _f32, _vp]),
}

_lib = None


class FfslError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("libffsl error %d: %s" % (code, msg))
        self.code = code


def load(path: str = LIB_PATH):
    """Load libffsl.so and declare its signatures; raises if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise FileNotFoundError(
                "%s is not built; run __graft_entry__.build() (hipcc, gfx950)" % path)
        lib = ctypes.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _lib = lib
    return _lib


def _check(rc):
    if rc != FFSL_OK:
        raise FfslError(rc, load().ffsl_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(torch):
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def footprint_bytes(L: int, k: int, value_bytes: int, bias: bool = True, unfused_grad: bool = False,
                    index_bytes: int = 4) -> int:
    """Resident bytes of the layer's training state: W, I, m, v per slot, bias state per row.

    The paper's accounting (Sec. 2.2) is value + index per slot for inference
    and value + grad + two moments sharing one index for training.
    """
    per_slot = value_bytes + index_bytes + 8 + (4 if unfused_grad else 0)
    per_row = (12 + (4 if unfused_grad else 0)) if bias else 0
    return L * k * per_slot + L * per_row


class SparseLayer:
    """A fixed fan-in layer whose state lives in torch tensors on the GPU.

    State: W [L,k] (float32 or bfloat16), I [L,k] int32 (or 16-bit indices:
    I given as int16 holding the uint16 bit patterns, d <= 65536), bias [L] f32, Adam
    moments m, v [L,k] f32 and bias_m, bias_v [L] f32; optional dW [L,k] and
    dbias [L] for the unfused path; a workspace sized by libffsl.
    """

    def __init__(self, W, I, bias=None, m=None, v=None, bias_m=None, bias_v=None,
                 B_max: int = 128, nnz_max: int = 4096, unfused: bool = True):
        import torch
        self.torch = torch
        lib = load()
        if not W.is_cuda:
            raise ValueError("layer state must live on the GPU")
        dev = W.device
        L, k = W.shape
        self.L, self.k = int(L), int(k)
        self.d = None
        if W.dtype == torch.bfloat16:
            self.vt = FFSL_BF16
        elif W.dtype == torch.float32:
            self.vt = FFSL_F32
        else:
            raise TypeError("W must be float32 or bfloat16")
        f32 = dict(dtype=torch.float32, device=dev)
        self.W = W.contiguous()
        self.idx = FFSL_IDX_U16 if I.dtype == torch.int16 else FFSL_IDX_I32
        self.I = I.to(device=dev, dtype=torch.int16 if self.idx == FFSL_IDX_U16 else torch.int32).contiguous()
        self.bias = bias.to(**f32).contiguous() if bias is not None else None
        self.m = m.to(**f32).contiguous() if m is not None else torch.zeros((L, k), **f32)
        self.v = v.to(**f32).contiguous() if v is not None else torch.zeros((L, k), **f32)
        if self.bias is not None:
            self.bias_m = bias_m.to(**f32).contiguous() if bias_m is not None else torch.zeros(L, **f32)
            self.bias_v = bias_v.to(**f32).contiguous() if bias_v is not None else torch.zeros(L, **f32)
        else:
            self.bias_m = self.bias_v = None
        self.dW = torch.empty((L, k), **f32) if unfused else None
        self.dbias = torch.empty(L, **f32) if (unfused and self.bias is not None) else None
        self.B_max, self.nnz_max = int(B_max), int(nnz_max)
        self._handle = None

    def bind(self, d: int):
        """Create the C handle for input width d (allocates the workspace)."""
        torch = self.torch
        lib = load()
        self.d = int(d)
        nbytes = lib.ffsl_workspace_bytes_ex(self.L, self.d, self.k, self.vt, self.B_max, self.nnz_max)
        if nbytes == 0:
            raise FfslError(FFSL_EINVAL, lib.ffsl_last_error().decode())
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.W.device)
        h = ctypes.c_void_p()
        _check(lib.ffsl_create_layer_ex(
            ctypes.byref(h), self.L, self.d, self.k, self.vt, self.idx, _ptr(self.W), _ptr(self.I),
            _ptr(self.bias), _ptr(self.m), _ptr(self.v), _ptr(self.bias_m), _ptr(self.bias_v),
            _ptr(self.dW), _ptr(self.dbias), _ptr(self.workspace), nbytes, self.B_max,
            self.nnz_max))
        self._handle = h
        return self

    def close(self):
        if self._handle is not None:
            load().ffsl_destroy_layer(self._handle)
            self._handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -------------------------------------------------------------- calls

    def _batch(self, X, off, lab):
        torch = self.torch
        if X.dim() != 2 or X.shape[1] != self.d:
            raise ValueError("X must be [B, %d]" % self.d)
        want = torch.bfloat16 if self.vt == FFSL_BF16 else torch.float32
        if X.dtype != want or not X.is_cuda or not X.is_contiguous():
            raise TypeError("X must be a contiguous %s CUDA tensor" % want)
        off = off.to(device=X.device, dtype=torch.int32).contiguous()
        lab = lab.to(device=X.device, dtype=torch.int32).contiguous()
        if off.numel() != X.shape[0] + 1:
            raise ValueError("tgt_off must have B+1 entries")
        return X, off, lab, int(lab.numel())

    def forward_loss(self, X, off, lab, s=None, logits=False, loss_out=None, flags=0):
        torch = self.torch
        X, off, lab, nnz = self._batch(X, off, lab)
        B = X.shape[0]
        s = 1.0 / B if s is None else float(s)
        loss = loss_out if loss_out is not None else torch.empty(1, dtype=torch.float32, device=X.device)
        z = torch.empty((B, self.L), dtype=torch.float32, device=X.device) if logits else None
        _check(load().ffsl_forward_loss(self._handle, _ptr(X), B, _ptr(off), _ptr(lab), nnz, s,
                                        _ptr(loss), _ptr(z), flags, _stream(torch)))
        return (loss, z) if logits else loss

    def backward(self, X, off, lab, s=None, dX_out=None, flags=0, loss_out=None):
        torch = self.torch
        X, off, lab, nnz = self._batch(X, off, lab)
        B = X.shape[0]
        s = 1.0 / B if s is None else float(s)
        dX = dX_out if dX_out is not None else torch.empty((B, self.d), dtype=torch.float32,
                                                           device=X.device)
        _check(load().ffsl_backward(self._handle, _ptr(X), B, _ptr(off), _ptr(lab), nnz, s,
                                    _ptr(loss_out), _ptr(dX), flags, _stream(torch)))
        return dX

    def adam_step(self, t, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0):
        _check(load().ffsl_adam_step(self._handle, int(t), lr, beta1, beta2, eps, wd,
                                     _stream(self.torch)))

    def train_step(self, X, off, lab, t, s=None, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0,
                   loss_out=None, dX_out=None, want_dx=True, flags=0):
        torch = self.torch
        X, off, lab, nnz = self._batch(X, off, lab)
        B = X.shape[0]
        s = 1.0 / B if s is None else float(s)
        loss = loss_out if loss_out is not None else torch.empty(1, dtype=torch.float32, device=X.device)
        dX = dX_out
        if dX is None and want_dx:
            dX = torch.empty((B, self.d), dtype=torch.float32, device=X.device)
        _check(load().ffsl_train_step(self._handle, _ptr(X), B, _ptr(off), _ptr(lab), nnz, s, int(t),
                                      lr, beta1, beta2, eps, wd, _ptr(loss), _ptr(dX), flags,
                                      _stream(torch)))
        return loss, dX

    def train_step_set(self, X, off, lab, t, frac, seed, set_round, s=None, lr=1e-3, beta1=0.9,
                       beta2=0.999, eps=1e-8, wd=0.0, loss_out=None, dX_out=None, want_dx=True, flags=0,
                       mask=True, exhausted_out=None):
        """train_step followed by set_update, fused where the library can."""
        torch = self.torch
        X, off, lab, nnz = self._batch(X, off, lab)
        B = X.shape[0]
        s = 1.0 / B if s is None else float(s)
        loss = loss_out if loss_out is not None else torch.empty(1, dtype=torch.float32, device=X.device)
        dX = dX_out
        if dX is None and want_dx:
            dX = torch.empty((B, self.d), dtype=torch.float32, device=X.device)
        msk = torch.empty((self.L, self.k), dtype=torch.uint8, device=self.W.device) if mask else None
        ex = exhausted_out
        if ex is None:
            ex = torch.zeros(1, dtype=torch.int32, device=self.W.device)
        _check(load().ffsl_train_step_set(self._handle, _ptr(X), B, _ptr(off), _ptr(lab), nnz, s, int(t),
                                          lr, beta1, beta2, eps, wd, _ptr(loss), _ptr(dX), flags,
                                          float(frac), int(seed) & (2**64 - 1), int(set_round) & (2**64 - 1),
                                          _ptr(msk), _ptr(ex), _stream(torch)))
        return loss, dX, msk, ex

    def set_update(self, frac, seed, set_round, mask=True, exhausted_out=None):
        torch = self.torch
        msk = torch.empty((self.L, self.k), dtype=torch.uint8, device=self.W.device) if mask else None
        ex = exhausted_out
        if ex is None:
            ex = torch.zeros(1, dtype=torch.int32, device=self.W.device)
        _check(load().ffsl_set_update(self._handle, float(frac), int(seed) & (2**64 - 1),
                                      int(set_round) & (2**64 - 1), _ptr(msk), _ptr(ex),
                                      _stream(torch)))
        return msk, ex

    def set_update_threshold(self, tau, seed, set_round, mask=True, exhausted_out=None):
        """SET in threshold mode: prune every |W| < tau, regrow as many per row."""
        torch = self.torch
        msk = torch.empty((self.L, self.k), dtype=torch.uint8, device=self.W.device) if mask else None
        ex = exhausted_out
        if ex is None:
            ex = torch.zeros(1, dtype=torch.int32, device=self.W.device)
        _check(load().ffsl_set_update_threshold(self._handle, float(tau), int(seed) & (2**64 - 1),
                                                int(set_round) & (2**64 - 1), _ptr(msk), _ptr(ex),
                                                _stream(torch)))
        return msk, ex

    def set_timing_events(self, start, stop):
        """Raw hipEvent_t handles (ints) or None; see ffsl_set_timing_events."""
        _check(load().ffsl_set_timing_events(self._handle, start, stop))

    def infer_topk(self, X, topk, off=None, lab=None, scores=True, workspace=None):
        """Each sample's topk labels (int32 [B, topk]), their scores (fp32, or
        None) and, when the relevant labels are given, P@1..P@topk averaged
        over the batch (fp32 [topk], or None)."""
        torch = self.torch
        if X.dim() != 2 or X.shape[1] != self.d:
            raise ValueError("X must be [B, %d]" % self.d)
        want = torch.bfloat16 if self.vt == FFSL_BF16 else torch.float32
        if X.dtype != want or not X.is_cuda or not X.is_contiguous():
            raise TypeError("X must be a contiguous %s CUDA tensor" % want)
        B = X.shape[0]
        lib = load()
        need = lib.ffsl_topk_workspace_bytes(self._handle, B, int(topk))
        if need == 0:
            raise FfslError(FFSL_EUNSUPPORTED, "top-k inference: unsupported shape or topk")
        ws = workspace if workspace is not None else _workspace(torch, need, X.device)
        top = torch.empty((B, topk), dtype=torch.int32, device=X.device)
        sc = torch.empty((B, topk), dtype=torch.float32, device=X.device) if scores else None
        p = None
        nnz = 0
        if off is not None:
            off = off.to(device=X.device, dtype=torch.int32).contiguous()
            lab = lab.to(device=X.device, dtype=torch.int32).contiguous()
            if off.numel() != B + 1:
                raise ValueError("tgt_off must have B+1 entries")
            nnz = int(lab.numel())
            p = torch.empty(topk, dtype=torch.float32, device=X.device)
        _check(lib.ffsl_infer_topk(self._handle, _ptr(X), B, int(topk), _ptr(top), _ptr(sc), _ptr(off),
                                   _ptr(lab), nnz, _ptr(p), _ptr(ws), ws.numel(), _stream(torch)))
        return top, sc, p

    def validate_indices(self):
        torch = self.torch
        bad = torch.zeros(1, dtype=torch.int32, device=self.W.device)
        _check(load().ffsl_validate_indices(self._handle, _ptr(bad), _stream(torch)))
        return bad


# ---------------------------------------------------------------------------
# dense parts: the intermediate GELU layer and the auxiliary cluster head


def _bf16_2d(t, name):
    import torch
    if t.dtype != torch.bfloat16 or not t.is_cuda or t.dim() != 2 or not t.is_contiguous():
        raise TypeError("%s must be a contiguous 2-D bfloat16 CUDA tensor" % name)
    return t


def _workspace(torch, nbytes, dev):
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=dev)


def dense_gelu_fwd(X, W1, c=None, split=True):
    """H = GELU(X W1 + c) (bf16) and the pre-activation A (fp32) for the backward.
    split=False runs the product in one pass (no workspace)."""
    import torch
    lib = load()
    _bf16_2d(X, "X")
    _bf16_2d(W1, "W1")
    B, din = X.shape
    dout = W1.shape[1]
    A = torch.empty((B, dout), dtype=torch.float32, device=X.device)
    H = torch.empty((B, dout), dtype=torch.bfloat16, device=X.device)
    ws = _workspace(torch, lib.ffsl_dense_workspace_bytes(B, din, dout), X.device) if split else None
    _check(lib.ffsl_dense_gelu_fwd(_ptr(X), B, din, dout, _ptr(W1), _ptr(c), _ptr(A), _ptr(H), _ptr(ws),
                                   0 if ws is None else ws.numel(), _stream(torch)))
    return A, H


def dense_gelu_bwd(X, W1, A, dH, want_dc=True, dX_out=None, flags=0):
    """dW1, dc and dX of the intermediate layer for the upstream gradient dH (fp32)."""
    import torch
    lib = load()
    B, din = X.shape
    dout = W1.shape[1]
    dev = X.device
    dW1 = torch.empty((din, dout), dtype=torch.float32, device=dev)
    dc = torch.empty(dout, dtype=torch.float32, device=dev) if want_dc else None
    dX = dX_out if dX_out is not None else torch.empty((B, din), dtype=torch.float32, device=dev)
    ws_bytes = lib.ffsl_dense_workspace_bytes(B, din, dout)
    if ws_bytes == 0:
        raise FfslError(FFSL_EINVAL, lib.ffsl_last_error().decode())
    ws = _workspace(torch, ws_bytes, dev)
    _check(lib.ffsl_dense_gelu_bwd(_ptr(X), B, din, dout, _ptr(W1), _ptr(A), _ptr(dH), _ptr(dW1), _ptr(dc),
                                   _ptr(dX), flags, _ptr(ws), ws.numel(), _stream(torch)))
    return dW1, dc, dX


def aux_bce_fwd_bwd(X, Wa, ca, off, lab, n_labels, s=None, want_logits=False, dX_out=None, loss_out=None,
                    flags=0):
    """Loss, dWa, dca, dX (and optionally the logits) of the auxiliary cluster
    head over the labels [0, n_labels) (the sparse layer's L)."""
    import torch
    lib = load()
    _bf16_2d(X, "X")
    _bf16_2d(Wa, "Wa")
    B, d = X.shape
    C = Wa.shape[1]
    dev = X.device
    s = 1.0 / B if s is None else s
    loss = loss_out if loss_out is not None else torch.zeros(1, dtype=torch.float32, device=dev)
    dWa = torch.empty((d, C), dtype=torch.float32, device=dev)
    dca = torch.empty(C, dtype=torch.float32, device=dev) if ca is not None else None
    dX = dX_out if dX_out is not None else torch.empty((B, d), dtype=torch.float32, device=dev)
    Z = torch.empty((B, C), dtype=torch.float32, device=dev) if want_logits else None
    ws_bytes = lib.ffsl_aux_workspace_bytes(B, d, C)
    if ws_bytes == 0:
        raise FfslError(FFSL_EINVAL, lib.ffsl_last_error().decode())
    ws = _workspace(torch, ws_bytes, dev)
    _check(lib.ffsl_aux_bce_fwd_bwd(_ptr(X), B, d, C, int(n_labels), _ptr(Wa), _ptr(ca), _ptr(off), _ptr(lab), int(lab.numel()),
                                    float(s), _ptr(loss), _ptr(dWa), _ptr(dca), _ptr(dX), _ptr(Z), flags,
                                    _ptr(ws), ws.numel(), _stream(torch)))
    return loss, dWa, dca, dX, Z


def adam_dense(param, grad, m, v, t, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0):
    """Adam / AdamW step in place on a flat (any-shape, contiguous) parameter tensor."""
    import torch
    lib = load()
    if param.dtype == torch.bfloat16:
        vt = FFSL_BF16
    elif param.dtype == torch.float32:
        vt = FFSL_F32
    else:
        raise TypeError("param must be float32 or bfloat16")
    n = param.numel()
    for name, x in (("grad", grad), ("m", m), ("v", v)):
        if x.dtype != torch.float32 or x.numel() != n or not x.is_contiguous():
            raise TypeError("%s must be a contiguous float32 tensor with %d elements" % (name, n))
    _check(lib.ffsl_adam_dense(_ptr(param), vt, _ptr(grad), _ptr(m), _ptr(v), n, int(t), lr, beta1, beta2, eps,
                               wd, _stream(torch)))


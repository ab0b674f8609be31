"""The paper's architectures around the fixed fan-in layer, composed from the
library's calls (Sec. 2.3 and Fig. 1 left):

- an optional wide intermediate layer between the encoder's features and the
  sparse classifier, H = GELU(X W1 + c), trained with it;
- an optional auxiliary meta-classifier over label clusters next to the
  sparse classifier, whose loss (with a weight that decays to zero at a cut-off
  epoch) adds to the sparse layer's and whose gradient adds to the encoder's.

One training step runs, in order: the intermediate layer's forward; the
sparse layer's fused step (forward, loss, dW, dX, Adam), with SET after it
when the schedule says so; the auxiliary head's forward and backward, adding
into the loss and dX; the intermediate layer's backward from the sparse
layer's dX; and Adam on the dense parameters.  Every step is a libffsl call;
this module only sequences them and holds the dense parameters and their
optimiser state.  The learning rates of the intermediate layer and the
auxiliary head default to the fixed values of the paper's DST settings.
"""
from __future__ import annotations

from typing import Optional

from . import ffsl, schedule


class Model:
    """Sparse layer (a bound ffsl.SparseLayer) plus optional dense parts.

    W1 [din, d] bf16 and c [d] fp32 (nullable) make the intermediate layer;
    Wa [d_in, C] bf16 and ca [C] fp32 (nullable) make the auxiliary head,
    where d_in is the sparse layer's input width without an intermediate
    layer (the auxiliary head reads the encoder's features X).
    """

    def __init__(self, sparse, W1=None, c=None, Wa=None, ca=None, *, lr=1e-3, wd=1e-4,
                 lr_inter=2.01e-4, wd_inter=0.0, lr_aux=5.01e-4, wd_aux=0.0,
                 set_frac=0.0, set_interval=0, total_steps=0, set_seed=0,
                 aux_w0=1.0, aux_cutoff_epoch: Optional[float] = None, loss_flags=0):
        import torch
        self.torch = torch
        self.sparse = sparse
        self.W1, self.c, self.Wa, self.ca = W1, c, Wa, ca
        self.lr, self.wd = lr, wd
        self.lr_inter, self.wd_inter = lr_inter, wd_inter
        self.lr_aux, self.wd_aux = lr_aux, wd_aux
        self.set_frac, self.set_interval, self.total_steps, self.set_seed = set_frac, set_interval, total_steps, set_seed
        self.aux_w0, self.aux_cutoff_epoch = aux_w0, aux_cutoff_epoch
        self.loss_flags = loss_flags
        z = lambda t: None if t is None else torch.zeros(t.shape, dtype=torch.float32, device=t.device)
        self.mW1, self.vW1, self.mc, self.vc = z(W1), z(W1), z(c), z(c)
        self.mWa, self.vWa, self.mca, self.vca = z(Wa), z(Wa), z(ca), z(ca)
        if W1 is not None and sparse.d != W1.shape[1]:
            raise ValueError("the intermediate layer's width must be the sparse layer's input width")

    def set_due(self, t: int) -> bool:
        return (self.set_frac > 0 and self.set_interval > 0 and
                schedule.set_due(t, self.set_interval, self.total_steps))

    def train_step(self, X, off, lab, t: int, epoch: float = 0.0):
        """One step at Adam step t (>= 1) and (fractional) epoch; returns the
        loss (sparse + weighted auxiliary, device fp32 [1]), the gradient of
        the encoder's features (fp32 [B, din]) and the SET mask (or None)."""
        sp = self.sparse
        A = None
        Xs = X
        if self.W1 is not None:
            A, Xs = ffsl.dense_gelu_fwd(X, self.W1, self.c)
        mask = None
        if self.set_due(t):
            loss, dXs, mask, _ = sp.train_step_set(Xs, off, lab, t, self.set_frac, self.set_seed,
                                                   schedule.set_round(t, self.set_interval), lr=self.lr,
                                                   wd=self.wd, flags=self.loss_flags)
        else:
            loss, dXs = sp.train_step(Xs, off, lab, t, lr=self.lr, wd=self.wd, flags=self.loss_flags)
        dX = dXs
        if self.W1 is not None:
            dW1, dc, dX = ffsl.dense_gelu_bwd(X, self.W1, A, dXs, want_dc=self.c is not None)
            ffsl.adam_dense(self.W1, dW1, self.mW1, self.vW1, t, lr=self.lr_inter, wd=self.wd_inter)
            if self.c is not None:
                ffsl.adam_dense(self.c, dc, self.mc, self.vc, t, lr=self.lr_inter, wd=self.wd_inter)
        if self.Wa is not None:
            w = schedule.aux_weight(epoch, self.aux_w0, self.aux_cutoff_epoch)
            if w > 0.0:
                _, dWa, dca, dX, _ = ffsl.aux_bce_fwd_bwd(
                    X, self.Wa, self.ca, off, lab, sp.L, s=w / X.shape[0], dX_out=dX, loss_out=loss,
                    flags=ffsl.FFSL_ACCUM_DX | ffsl.FFSL_ACCUM_LOSS)
                ffsl.adam_dense(self.Wa, dWa, self.mWa, self.vWa, t, lr=self.lr_aux, wd=self.wd_aux)
                if self.ca is not None:
                    ffsl.adam_dense(self.ca, dca, self.mca, self.vca, t, lr=self.lr_aux, wd=self.wd_aux)
        return loss, dX, mask

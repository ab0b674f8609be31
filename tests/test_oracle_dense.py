"""Pins of the oracle's dense parts (intermediate layer with GELU, auxiliary
cluster head) against torch autograd in float64 (exact-erf GELU)."""
import numpy as np
import torch


def test_dense_gelu_forward_backward_matches_torch(oracle):
    rng = np.random.default_rng(0)
    B, din, dout = 5, 7, 9
    X = rng.standard_normal((B, din))
    W1 = rng.standard_normal((din, dout)) * 0.5
    c = rng.standard_normal(dout)
    dH = rng.standard_normal((B, dout))
    A, H = oracle.dense_gelu_fwd(X, W1, c)
    Xt = torch.tensor(X, requires_grad=True)
    Wt = torch.tensor(W1, requires_grad=True)
    ct = torch.tensor(c, requires_grad=True)
    Ht = torch.nn.functional.gelu(Xt @ Wt + ct)
    np.testing.assert_allclose(H, Ht.detach().numpy(), rtol=1e-13, atol=1e-15)
    Ht.backward(torch.tensor(dH))
    dW1, dc, dX = oracle.dense_gelu_bwd(X, W1, A, dH)
    np.testing.assert_allclose(dW1, Wt.grad.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(dc, ct.grad.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(dX, Xt.grad.numpy(), rtol=1e-12, atol=1e-14)


def test_gelu_special_values(oracle):
    X = np.array([[0.0], [1.0], [-1.0], [10.0], [-10.0]])
    A, H = oracle.dense_gelu_fwd(X, np.array([[1.0]]))
    from math import erf, sqrt
    ref = [0.0, 0.5 * (1 + erf(1 / sqrt(2))), -0.5 * (1 - erf(1 / sqrt(2))), 10.0, 0.0]
    np.testing.assert_allclose(H[:, 0], ref, atol=1e-15)


def test_aux_head_matches_torch(oracle):
    rng = np.random.default_rng(1)
    B, d, C, L = 4, 6, 5, 23
    X = rng.standard_normal((B, d))
    Wa = rng.standard_normal((d, C)) * 0.3
    ca = rng.standard_normal(C)
    off = np.array([0, 2, 3, 6, 7])
    lab = np.array([3, 8, 22, 0, 5, 10, 4], dtype=np.int32)   # 0,5,10 share cluster 0
    s = 1 / B
    r = oracle.aux_bce(X, Wa, ca, off, lab, s, L)
    ya = np.zeros((B, C))
    for b in range(B):
        for l in lab[off[b]:off[b + 1]]:
            ya[b, l % C] = 1
    assert ya[2].tolist() == [1, 0, 0, 0, 0]
    Xt = torch.tensor(X, requires_grad=True)
    Wt = torch.tensor(Wa, requires_grad=True)
    ct = torch.tensor(ca, requires_grad=True)
    loss = torch.nn.functional.binary_cross_entropy_with_logits(
        Xt @ Wt + ct, torch.tensor(ya), reduction="sum") * s
    loss.backward()
    np.testing.assert_allclose(r["loss"], loss.item(), rtol=1e-13)
    np.testing.assert_allclose(r["dWa"], Wt.grad.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(r["dca"], ct.grad.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(r["dXa"], Xt.grad.numpy(), rtol=1e-12, atol=1e-14)


def test_label_range_is_the_same_for_both_heads(oracle):
    """A label outside [0, L) is not a label of the layer: the sparse head's
    targets and the auxiliary head's cluster targets both ignore it, so a batch
    with such labels gives the results of the batch without them.  Pinned
    against a hand-built cluster multi-hot and torch's BCE, and by the sparse
    targets of both batches."""
    rng = np.random.default_rng(2)
    B, d, C, L = 3, 5, 4, 10
    X = rng.standard_normal((B, d))
    Wa = rng.standard_normal((d, C)) * 0.3
    ca = rng.standard_normal(C)
    # out of range: -1, -7 (negative), 10 = L, 11 and 14 (clusters 2, 3, 2 if
    # they were taken, none of them a cluster the sample already has);
    # in range: 2, 9, 4
    off = np.array([0, 3, 5, 8])
    lab = np.array([2, 11, -1, 9, 14, 4, -7, 10], dtype=np.int32)
    keep = (lab >= 0) & (lab < L)
    off_in = np.concatenate([[0], np.cumsum([keep[off[b]:off[b + 1]].sum() for b in range(B)])])
    lab_in = lab[keep]
    s = 0.5
    r = oracle.aux_bce(X, Wa, ca, off, lab, s, L)
    r_in = oracle.aux_bce(X, Wa, ca, off_in, lab_in, s, L)
    for key in ("loss", "Za", "dWa", "dca", "dXa"):
        np.testing.assert_array_equal(r[key], r_in[key])
    ya = np.zeros((B, C))
    ya[0, 2 % C] = 1
    ya[1, 9 % C] = 1
    ya[2, 4 % C] = 1
    loss = torch.nn.functional.binary_cross_entropy_with_logits(
        torch.tensor(X @ Wa + ca), torch.tensor(ya), reduction="sum") * s
    np.testing.assert_allclose(r["loss"], loss.item(), rtol=1e-13)
    # the sparse head's targets drop the same labels
    y = oracle.targets_dense(B, L, off, lab)
    y_in = oracle.targets_dense(B, L, off_in, lab_in)
    np.testing.assert_array_equal(y, y_in)
    assert y.sum() == 3
    # the other reading (labels >= L mapped to l mod C) gives other targets,
    # so the pin tells the two apart
    ya_other = ya.copy()
    ya_other[0, 11 % C] = ya_other[1, 14 % C] = ya_other[2, 10 % C] = 1
    assert not np.array_equal(ya, ya_other)
    loss_other = torch.nn.functional.binary_cross_entropy_with_logits(
        torch.tensor(X @ Wa + ca), torch.tensor(ya_other), reduction="sum") * s
    assert abs(r["loss"] - loss_other.item()) > 1e-3

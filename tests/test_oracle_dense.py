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
    r = oracle.aux_bce(X, Wa, ca, off, lab, s)
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

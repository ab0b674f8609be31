"""GPU parity of the dense parts (the intermediate GELU layer and the
auxiliary cluster head) and of the flat Adam step, through the C ABI, against
the float64 oracle on identical generator-produced inputs: the full C3 and C5
shapes and small ragged ones."""
import numpy as np
import pytest

import oracle
from paper_2411_03171_amd import synth
from tests.parity import RTOL_BF16, RTOL_F32, assert_close, note, to_torch_values

pytestmark = pytest.mark.gpu

W1_ = synth.WORKLOADS

# (name, B, din, dout): the C3 intermediate layer and smaller ragged shapes
DENSE = [
    ("c3", W1_["c3_inter2048_L1M"].B, W1_["c3_inter2048_L1M"].din, W1_["c3_inter2048_L1M"].d),
    ("ragged", 37, 136, 264),
    ("b1", 1, 64, 72),
]
# (name, B, d, C, L, mean positives): the C5 auxiliary head and ragged ones
AUX = [
    ("c5", W1_["c5_aux8192_L1M"].B, W1_["c5_aux8192_L1M"].d, W1_["c5_aux8192_L1M"].aux_clusters,
     W1_["c5_aux8192_L1M"].L, W1_["c5_aux8192_L1M"].mean_pos),
    ("ragged", 37, 136, 104, 5000, 6.0),
    ("b1", 1, 64, 40, 300, 3.0),
]


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2411_03171_amd import ffsl
    ffsl.load()
    return torch


def _x(rng, B, d):
    return synth.gen_x(rng, B, d, "layernorm", "bf16")


def _f64(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


@pytest.mark.parametrize("case", DENSE, ids=[c[0] for c in DENSE])
def test_dense_gelu_fwd_bwd(torch_cuda, case):
    torch = torch_cuda
    from paper_2411_03171_amd import ffsl
    name, B, din, dout = case
    rng = np.random.default_rng(11)
    X = _x(rng, B, din)
    W1 = synth.make_dense(rng, din, dout)
    c = (rng.standard_normal(dout) * 0.1).astype(np.float32)
    dH = (rng.standard_normal((B, dout)) * 1e-2).astype(np.float32)
    A_ref, H_ref = oracle.dense_gelu_fwd(_f64(X), _f64(W1), c.astype(np.float64))
    dev = "cuda:0"
    Xt, Wt = to_torch_values(X, "bf16", dev), to_torch_values(W1, "bf16", dev)
    ct = torch.from_numpy(c).to(dev)
    note("dense gelu fwd %s B=%d din=%d dout=%d" % (name, B, din, dout))
    # the product split over K (with a workspace) and in one pass
    for split in (True, False):
        A, H = ffsl.dense_gelu_fwd(Xt, Wt, ct, split=split)
        torch.cuda.synchronize()
        assert_close(A.cpu().numpy(), A_ref, RTOL_F32, "A (split=%s)" % split)
        assert_close(H.float().cpu().numpy(), H_ref, RTOL_BF16, "H (split=%s)" % split)
    # backward from the same pre-activation on both sides
    A32 = A_ref.astype(np.float32)
    dW1_ref, dc_ref, dX_ref = oracle.dense_gelu_bwd(_f64(X), _f64(W1), A32.astype(np.float64),
                                                     dH.astype(np.float64))
    note("dense gelu bwd %s" % name)
    dW1, dc, dX = ffsl.dense_gelu_bwd(Xt, Wt, torch.from_numpy(A32).to(dev), torch.from_numpy(dH).to(dev))
    torch.cuda.synchronize()
    assert_close(dc.cpu().numpy(), dc_ref, RTOL_F32, "dc")
    assert_close(dW1.cpu().numpy(), dW1_ref, RTOL_BF16, "dW1")
    assert_close(dX.cpu().numpy(), dX_ref, RTOL_BF16, "dX")
    # FFSL_ACCUM_DX adds into an existing dX
    R = rng.standard_normal((B, din)).astype(np.float32) * float(np.abs(dX_ref).max())
    Rt = torch.from_numpy(R).to(dev)
    note("dense gelu bwd accumulate %s" % name)
    ffsl.dense_gelu_bwd(Xt, Wt, torch.from_numpy(A32).to(dev), torch.from_numpy(dH).to(dev), dX_out=Rt,
                        flags=ffsl.FFSL_ACCUM_DX)
    torch.cuda.synchronize()
    assert_close(Rt.cpu().numpy() - R, dX_ref, RTOL_BF16, "dX accumulated")


@pytest.mark.parametrize("case", AUX, ids=[c[0] for c in AUX])
def test_aux_bce_fwd_bwd(torch_cuda, case):
    torch = torch_cuda
    from paper_2411_03171_amd import ffsl
    name, B, d, C, L, mean_pos = case
    rng = np.random.default_rng(23)
    X = _x(rng, B, d)
    Wa = synth.make_dense(rng, d, C)
    ca = (rng.standard_normal(C) * 0.1).astype(np.float32)
    off, lab = synth.gen_targets(rng, B, L, mean_pos, 1.1)
    s = 1.0 / B
    ref = oracle.aux_bce(_f64(X), _f64(Wa), ca.astype(np.float64), off, lab, s, L)
    dev = "cuda:0"
    Xt, Wt = to_torch_values(X, "bf16", dev), to_torch_values(Wa, "bf16", dev)
    offt = torch.from_numpy(off.astype(np.int32)).to(dev)
    labt = torch.from_numpy(lab.astype(np.int32)).to(dev)
    note("aux bce %s B=%d d=%d C=%d nnz=%d" % (name, B, d, C, len(lab)))
    loss, dWa, dca, dX, Z = ffsl.aux_bce_fwd_bwd(Xt, Wt, torch.from_numpy(ca).to(dev), offt, labt, L, s,
                                                 want_logits=True)
    torch.cuda.synchronize()
    assert_close(Z.cpu().numpy(), ref["Za"], RTOL_F32, "Za")
    assert_close(np.array([float(loss.cpu()[0])]), np.array([ref["loss"]]), RTOL_F32, "loss")
    assert_close(dca.cpu().numpy(), ref["dca"], RTOL_F32, "dca")
    assert_close(dWa.cpu().numpy(), ref["dWa"], RTOL_BF16, "dWa")
    assert_close(dX.cpu().numpy(), ref["dXa"], RTOL_BF16, "dXa")
    # accumulate into an existing loss and dX (the sparse layer's)
    R = rng.standard_normal((B, d)).astype(np.float32) * float(np.abs(ref["dXa"]).max())
    Rt = torch.from_numpy(R).to(dev)
    l0 = torch.full((1,), 3.5, dtype=torch.float32, device=dev)
    note("aux bce accumulate %s" % name)
    ffsl.aux_bce_fwd_bwd(Xt, Wt, torch.from_numpy(ca).to(dev), offt, labt, L, s, dX_out=Rt, loss_out=l0,
                         flags=ffsl.FFSL_ACCUM_DX | ffsl.FFSL_ACCUM_LOSS)
    torch.cuda.synchronize()
    assert_close(Rt.cpu().numpy() - R, ref["dXa"], RTOL_BF16, "dXa accumulated")
    assert abs(float(l0.cpu()[0]) - 3.5 - ref["loss"]) <= RTOL_F32 * max(abs(ref["loss"]), 1.0)


def test_aux_bce_no_positives_and_no_bias(torch_cuda):
    torch = torch_cuda
    from paper_2411_03171_amd import ffsl
    rng = np.random.default_rng(5)
    B, d, C = 3, 32, 16
    X = _x(rng, B, d)
    Wa = synth.make_dense(rng, d, C)
    off = np.zeros(B + 1, dtype=np.int64)
    lab = np.zeros(0, dtype=np.int32)
    ref = oracle.aux_bce(_f64(X), _f64(Wa), None, off, lab, 0.5, 100)
    dev = "cuda:0"
    note("aux bce empty targets")
    loss, dWa, dca, dX, _ = ffsl.aux_bce_fwd_bwd(
        to_torch_values(X, "bf16", dev), to_torch_values(Wa, "bf16", dev), None,
        torch.zeros(B + 1, dtype=torch.int32, device=dev), torch.zeros(0, dtype=torch.int32, device=dev), 100, 0.5)
    torch.cuda.synchronize()
    assert dca is None
    assert_close(np.array([float(loss.cpu()[0])]), np.array([ref["loss"]]), RTOL_F32, "loss")
    assert_close(dWa.cpu().numpy(), ref["dWa"], RTOL_BF16, "dWa")
    assert_close(dX.cpu().numpy(), ref["dXa"], RTOL_BF16, "dXa")


def test_aux_bce_labels_outside_the_layer(torch_cuda):
    """Labels outside [0, n_labels) (negative, n_labels itself, beyond) are
    ignored by the auxiliary head, as by the sparse layer."""
    torch = torch_cuda
    from paper_2411_03171_amd import ffsl
    rng = np.random.default_rng(9)
    B, d, C, L = 6, 64, 24, 50
    X = _x(rng, B, d)
    Wa = synth.make_dense(rng, d, C)
    ca = (rng.standard_normal(C) * 0.1).astype(np.float32)
    off = np.array([0, 3, 4, 4, 7, 9, 12], dtype=np.int64)
    lab = np.array([5, 50, -1, 73, 49, 0, 2**31 - 1, 24, 51, -2**31, 26, 99], dtype=np.int32)
    s = 1.0 / B
    ref = oracle.aux_bce(_f64(X), _f64(Wa), ca.astype(np.float64), off, lab, s, L)
    dev = "cuda:0"
    note("aux bce labels outside [0, L)")
    loss, dWa, dca, dX, Z = ffsl.aux_bce_fwd_bwd(
        to_torch_values(X, "bf16", dev), to_torch_values(Wa, "bf16", dev), torch.from_numpy(ca).to(dev),
        torch.from_numpy(off.astype(np.int32)).to(dev), torch.from_numpy(lab).to(dev), L, s, want_logits=True)
    torch.cuda.synchronize()
    assert_close(np.array([float(loss.cpu()[0])]), np.array([ref["loss"]]), RTOL_F32, "loss")
    assert_close(dca.cpu().numpy(), ref["dca"], RTOL_F32, "dca")
    assert_close(dWa.cpu().numpy(), ref["dWa"], RTOL_BF16, "dWa")
    assert_close(dX.cpu().numpy(), ref["dXa"], RTOL_BF16, "dXa")


@pytest.mark.parametrize("value", ["f32", "bf16"])
def test_adam_dense_matches_oracle(torch_cuda, value):
    torch = torch_cuda
    from paper_2411_03171_amd import ffsl
    rng = np.random.default_rng(7)
    n = 100_003
    p32 = (rng.standard_normal(n) * 0.05).astype(np.float32)
    p = p32 if value == "f32" else synth.f32_to_bf16_bits(p32)
    g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    v = (rng.random(n) * 1e-6).astype(np.float32)
    pf = p32.astype(np.float64) if value == "f32" else _f64(p)
    pr, mr, vr = oracle.adam(pf, m.astype(np.float64), v.astype(np.float64), g.astype(np.float64), t=3,
                             lr=1e-3, wd=1e-4)
    dev = "cuda:0"
    pt = to_torch_values(p, value, dev)
    mt, vt = torch.from_numpy(m).to(dev), torch.from_numpy(v).to(dev)
    note("adam dense %s n=%d" % (value, n))
    ffsl.adam_dense(pt, torch.from_numpy(g).to(dev), mt, vt, t=3, lr=1e-3, wd=1e-4)
    torch.cuda.synchronize()
    assert_close(mt.cpu().numpy(), mr, RTOL_F32, "m")
    assert_close(vt.cpu().numpy(), vr, RTOL_F32, "v")
    got = pt.float().cpu().numpy().astype(np.float64)
    if value == "f32":
        assert_close(got, pr, RTOL_F32, "p")
    else:
        # bf16 write-back: within one bf16 ulp of the exact update
        ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(pr), 1e-30))) - 7)
        assert np.all(np.abs(got - pr) <= ulp + 1e-12)


def test_dense_errors(torch_cuda):
    torch = torch_cuda
    from paper_2411_03171_amd import ffsl
    dev = "cuda:0"
    X = torch.zeros((4, 100), dtype=torch.bfloat16, device=dev)
    W = torch.zeros((100, 64), dtype=torch.bfloat16, device=dev)
    with pytest.raises(ffsl.FfslError):   # width not a multiple of 8
        ffsl.dense_gelu_fwd(X, W)
    flat = torch.zeros(4 * 64 + 1, dtype=torch.bfloat16, device=dev)
    Xm = flat[1:].view(4, 64)             # 2-byte offset: misaligned
    W2 = torch.zeros((64, 64), dtype=torch.bfloat16, device=dev)
    with pytest.raises(ffsl.FfslError):
        ffsl.dense_gelu_fwd(Xm, W2)
    lib = ffsl.load()
    assert lib.ffsl_dense_workspace_bytes(0, 64, 64) == 0
    assert lib.ffsl_aux_workspace_bytes(4, 64, 12) == 0
    p = torch.zeros(8, dtype=torch.float32, device=dev)
    with pytest.raises(ffsl.FfslError):   # t must be >= 1
        ffsl.adam_dense(p, p.clone(), p.clone(), p.clone(), t=0)

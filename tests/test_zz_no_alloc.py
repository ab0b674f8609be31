"""ffsl_infer_topk_noalloc, the inference call for callers that cannot
allocate device memory, against ffsl_infer_topk (the same call with a
workspace), through the C ABI: labels, scores and P@k bit for bit, on two
calls in a row whose second is smaller (fewer samples, smaller topk, so the
shared scratch holds the first call's leftovers); and a call that needs more
scratch than the static array holds is refused before anything runs."""
import ctypes

import numpy as np
import pytest

from paper_2411_03171_amd import synth
from tests.parity import batch_to_gpu, make_gpu_layer, note

pytestmark = pytest.mark.gpu


def _call(lib, layer, X, B, K, off, lab, noalloc):
    import torch
    from paper_2411_03171_amd import ffsl
    dev = X.device
    top = torch.full((B, K), -7, dtype=torch.int32, device=dev)
    sc = torch.full((B, K), 7.0, dtype=torch.float32, device=dev)
    p = torch.full((K,), 7.0, dtype=torch.float32, device=dev)
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    P = ffsl._ptr
    if noalloc:
        rc = lib.ffsl_infer_topk_noalloc(layer._handle, P(X), B, K, P(top), P(sc), P(off), P(lab), int(lab.numel()),
                                         P(p), st)
    else:
        need = lib.ffsl_topk_workspace_bytes(layer._handle, B, K)
        ws = torch.empty(need, dtype=torch.uint8, device=dev)
        rc = lib.ffsl_infer_topk(layer._handle, P(X), B, K, P(top), P(sc), P(off), P(lab), int(lab.numel()), P(p),
                                 P(ws), need, st)
    ffsl._check(rc)
    torch.cuda.synchronize()
    return top.cpu().numpy(), sc.cpu().numpy().view(np.uint32), p.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("name", ["c4", "c1"])
def test_noalloc_topk_equals_workspace_call(name):
    import torch
    from paper_2411_03171_amd import ffsl
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    lib = ffsl.load()
    if name == "c4":
        # the largest label space, as the benchmark's inference call
        w = synth.WORKLOADS["c4_bf16_L3M"]
        calls = [(64, 8), (17, 3)]
    else:
        w = synth.scaled(synth.WORKLOADS["c1_fp32_L4096"], L=3001, B=100, name="c1n")
        calls = [(100, 16), (9, 1)]
    inp = synth.make_layer_inputs(w, 21)
    bias = (np.random.default_rng(22).standard_normal(w.L) * 0.3).astype(np.float32)
    layer = make_gpu_layer(inp, w, bias_values=bias, unfused=False)
    X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    for B, K in calls:
        Xb = X[:B].contiguous()
        offb = off[:B + 1].contiguous()
        note("noalloc topk %s B=%d K=%d" % (name, B, K))
        got = _call(lib, layer, Xb, B, K, offb, lab, True)
        ref = _call(lib, layer, Xb, B, K, offb, lab, False)
        for a, b, what in zip(got, ref, ("labels", "scores", "P@k")):
            np.testing.assert_array_equal(a, b, err_msg=what)
        assert (got[0] >= 0).all()


def test_noalloc_topk_refuses_more_than_its_scratch():
    import torch
    from paper_2411_03171_amd import ffsl
    lib = ffsl.load()
    w = synth.scaled(synth.WORKLOADS["c4_bf16_L3M"], L=5000, B=1024, name="big")
    inp = synth.make_layer_inputs(w, 23)
    layer = make_gpu_layer(inp, w, unfused=False)
    X, off, lab = batch_to_gpu(inp.X, inp.off, inp.lab, w.value)
    assert lib.ffsl_topk_workspace_bytes(layer._handle, 1024, 16) > ffsl.FFSL_TOPK_SCRATCH_BYTES
    top = torch.empty((1024, 16), dtype=torch.int32, device=X.device)
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    note("noalloc topk: a call past the scratch")
    rc = lib.ffsl_infer_topk_noalloc(layer._handle, ffsl._ptr(X), 1024, 16, ffsl._ptr(top), None, None, None, 0,
                                     None, st)
    assert rc == ffsl.FFSL_EINVAL
    assert b"scratch" in lib.ffsl_last_error()

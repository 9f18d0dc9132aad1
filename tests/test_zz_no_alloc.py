"""caffe_conv_forward_noalloc: the forward pass on the library's static
scratch array, called through the C ABI, against caffe_conv_forward on a
caller-provided workspace (the same kernels, so the outputs must agree bit
for bit), and against the CPU oracle at the fp32 / bf16 tolerances.  Two
calls in a row on each case, the second with a smaller batch, so that the
second call runs on what the first left in the shared array."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_1408_5093_amd as cc
from helpers import TOL_BF16, TOL_F32, assert_close

pytestmark = pytest.mark.gpu

# (N1, N2, C, H, W, K, k, s, p, g, relu, bf16): the LeNet conv2 shape runs
# split-K (its partials live in the scratch), the CaffeNet conv5 shape runs
# the channel-blocked GEMM on packed weights, conv1's on its tap table, and
# the inner-product shape the dense split-K GEMM
CASES = [
    (64, 16, 20, 12, 12, 50, 5, 1, 0, 1, False, False),
    (8, 3, 384, 13, 13, 256, 3, 1, 1, 2, True, False),
    (6, 2, 3, 227, 227, 96, 11, 4, 0, 1, True, False),
    (256, 40, 4096, 1, 1, 1000, 1, 1, 0, 1, False, False),
    (8, 3, 96, 27, 27, 256, 5, 1, 2, 2, True, True),
]


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _run(case, N, seed):
    _, _, C, H, W, K, k, s, p, g, relu, bf16 = case
    lib = cc.load()
    rng = np.random.default_rng([1408, 5093, 77, seed])
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    w = (rng.standard_normal((K, C // g, k, k)) * 0.05).astype(np.float32)
    b = rng.standard_normal(K).astype(np.float32)
    op = torch.bfloat16 if bf16 else torch.float32
    xt = torch.from_numpy(x).cuda().to(op)
    wt = torch.from_numpy(w).cuda().to(op)
    bt = torch.from_numpy(b).cuda()
    d = cc.conv_desc(xt.shape, wt.shape, s, p, g, relu, cc.CAFFE_BF16 if bf16 else cc.CAFFE_F32)
    Ho, Wo = cc.conv_out_shape(d)
    need = cc.conv_workspace_size(d, cc.PASS_FORWARD)
    assert need <= cc.NOALLOC_SCRATCH_BYTES
    y_ref = torch.full((N, K, Ho, Wo), float("nan"), device="cuda")
    y = torch.full((N, K, Ho, Wo), float("nan"), device="cuda")
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device="cuda")
    print(f"noalloc case {case} N={N}", flush=True)
    cc.check(lib.caffe_conv_forward(ctypes.byref(d), _ptr(xt), _ptr(wt), _ptr(bt), _ptr(y_ref),
                                    _ptr(ws), need, _stream()))
    cc.check(lib.caffe_conv_forward_noalloc(ctypes.byref(d), _ptr(xt), _ptr(wt), _ptr(bt), _ptr(y),
                                            _stream()))
    torch.cuda.synchronize()
    assert torch.equal(y, y_ref), "static-scratch forward differs from the workspace forward"
    # parity with the oracle on the operands the GPU consumed
    xs = xt.float().cpu().numpy()[: min(N, 2)]
    ws_ = wt.float().cpu().numpy()
    ref = oracle.conv_forward(xs, ws_, b, s, p, g, relu)
    assert_close(y[: min(N, 2)].cpu().numpy(), ref, TOL_BF16 if bf16 else TOL_F32, "noalloc forward")


@pytest.mark.parametrize("case", CASES)
def test_noalloc_forward_matches_workspace_forward(case):
    N1, N2 = case[0], case[1]
    _run(case, N1, 0)
    _run(case, N2, 1)


def test_noalloc_forward_rejects_oversized_workspace():
    """bf16 CaffeNet conv1 at N=256 stages more input than the array holds:
    refused on the host with CAFFE_ERR_WORKSPACE, nothing launched."""
    lib = cc.load()
    d = cc.conv_desc((256, 3, 227, 227), (96, 3, 11, 11), 4, 0, 1, True, cc.CAFFE_BF16)
    assert cc.conv_workspace_size(d, cc.PASS_FORWARD) > cc.NOALLOC_SCRATCH_BYTES
    P = ctypes.c_void_p
    st = lib.caffe_conv_forward_noalloc(ctypes.byref(d), P(0x1000), P(0x2000), None, P(0x3000),
                                        None)
    assert st == cc.CAFFE_ERR_WORKSPACE
    assert b"static scratch" in lib.caffe_last_error()

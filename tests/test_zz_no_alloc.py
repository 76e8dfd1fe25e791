"""The allocation-free packed forward (lcvq_linear_fwd_packed_noalloc), called
through the C ABI, against the workspace entry point (lcvq_linear_fwd_packed) on
the same inputs: the same kernels, so the outputs must match bit for bit.  Two
calls in a row, the second with a smaller input, so the second reads a scratch
array that still holds the first call's contents."""
import ctypes

import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lc():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_10531_amd as lc
    lc._lib.load()
    return lc


def _inputs(m, n, N, d, seed):
    import torch
    g = torch.Generator(device="cuda").manual_seed(seed)
    P = torch.randint(0, 256, (m, n // 4), dtype=torch.uint8, device="cuda", generator=g)
    X = torch.randn((N, n), device="cuda", generator=g).to(torch.bfloat16)
    A, b = (torch.from_numpy(x).cuda() for x in synth.draw_map(d, seed))
    return P, A, b, X


def _noalloc(lc, P, A, b, X, d, Y):
    m, n = P.shape[0], P.shape[1] * 4
    st = ctypes.c_void_p(__import__("torch").cuda.current_stream().cuda_stream)
    return lc._lib.load().lcvq_linear_fwd_packed_noalloc(X.shape[0], m, n, d, P.data_ptr(), A.data_ptr(),
                                                         b.data_ptr(), X.data_ptr(), Y.data_ptr(),
                                                         lc._lib.BF16 if Y.dtype == __import__("torch").bfloat16
                                                         else lc._lib.F32, st)


# first call: the K-split path (tile counters and partials in the scratch array);
# second call: smaller, another path and fewer tokens
CASES = [((8192, 28672, 16, 8), (4096, 4096, 5, 4)),
         ((28672, 8192, 3, 8), (264, 1024, 1, 8)),
         ((4096, 11008, 16, 8), (512, 4096, 9, 8))]


@pytest.mark.parametrize("first,second", CASES)
def test_noalloc_matches_the_workspace_entry_point_on_two_calls(lc, first, second):
    import torch
    for (m, n, N, d), seed, ydt in ((first, 1, torch.bfloat16), (second, 2, torch.float32)):
        P, A, b, X = _inputs(m, n, N, d, seed)
        Y_ws = lc.linear_fwd_packed(P, A, b, X, d, out_dtype=ydt)
        Y_na = torch.full((N, m), float("nan"), dtype=ydt, device="cuda")
        assert _noalloc(lc, P, A, b, X, d, Y_na) == lc._lib.OK, lc._lib.last_error()
        torch.cuda.synchronize()
        assert torch.equal(Y_na.view(torch.int16 if ydt == torch.bfloat16 else torch.int32),
                           Y_ws.view(torch.int16 if ydt == torch.bfloat16 else torch.int32)), (m, n, N, d)


def test_noalloc_binding_and_limits(lc):
    import torch
    assert lc._lib.load().lcvq_packed_scratch_bytes() == 8 << 20
    P, A, b, X = _inputs(1024, 2048, 7, 8, 3)
    Y = torch.empty((7, 1024), dtype=torch.bfloat16, device="cuda")
    lc.linear_fwd_packed_noalloc(P, A, b, X, 8, out=Y)
    torch.cuda.synchronize()
    assert torch.equal(Y, lc.linear_fwd_packed(P, A, b, X, 8))
    # a shape whose workspace exceeds the array is refused before anything is enqueued
    big_n = 1 << 20
    assert lc._lib.load().lcvq_linear_fwd_packed_noalloc(1, 64, big_n, 8, P.data_ptr(), A.data_ptr(), b.data_ptr(),
                                                          X.data_ptr(), Y.data_ptr(), lc._lib.BF16,
                                                          None) == lc._lib.EUNSUPPORTED
    assert "scratch" in lc._lib.last_error()

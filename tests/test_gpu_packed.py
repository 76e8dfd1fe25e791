"""Parity of the layer output from packed 2-bit codes (lcvq_linear_fwd_packed)
with the fp64 oracle, through the C ABI.

Y is compared by relative Frobenius error <= 2e-2 (bf16 activations, X' rounded
to bf16, fp32 accumulation), as for lcvq_linear_fwd."""
import numpy as np
import pytest

import oracle as orc
import synth
from helpers import assert_close, rel_fro, to_dev, to_host

pytestmark = pytest.mark.gpu

TOL = 2e-2


@pytest.fixture(scope="module")
def lc():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_10531_amd as lc
    lc._lib.load()
    return lc


def _inputs(N, m, n, d, seed):
    inp = synth.layer_inputs(N, m, n, d, "bf16", k=seed, z_lo=-1.0, z_hi=4.0)
    codes = orc.quantize(orc.widen(inp["Z"], "bf16"))
    return inp, orc.pack2bit(codes)


def _run(lc, inp, P, d, y_dtype, calls=1):
    import torch
    tdt = torch.bfloat16 if y_dtype == "bf16" else torch.float32
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    Pd, X = torch.from_numpy(P).cuda(), to_dev(inp["X"], "bf16")
    outs = [lc.linear_fwd_packed(Pd, A, b, X, d, out_dtype=tdt) for _ in range(calls)]
    torch.cuda.synchronize()
    return [to_host(Y) for Y in outs]


def _ref(inp, P, d, n):
    return orc.linear_forward_packed(P, inp["A"].astype(np.float64), inp["b"].astype(np.float64),
                                     orc.widen(inp["X"], "bf16"), d, n)


# (N, m, n): one and several 16-token passes, K split over blocks (m = 64 with
# n = 4096) or not, ragged row tiles (m % 64 != 0), K not a multiple of 256
SHAPES = [(1, 64, 64), (5, 72, 320), (16, 256, 1024), (17, 200, 4096), (16, 64, 4096), (33, 1000, 768),
          (3, 8, 8192)]


@pytest.mark.parametrize("y_dtype", ["bf16", "f32"])
@pytest.mark.parametrize("d", [8, 4])
@pytest.mark.parametrize("N,m,n", SHAPES)
def test_packed_forward(lc, N, m, n, d, y_dtype):
    inp, P = _inputs(N, m, n, d, seed=N + m + n + d)
    got = _run(lc, inp, P, d, y_dtype, calls=2)
    ref = _ref(inp, P, d, n)
    for Y in got:   # a second call (counters reset by its prepass) gives the same result
        assert_close(Y, ref, TOL, 'Y')
    assert np.array_equal(got[0], got[1])


def test_packed_forward_matches_latent_forward(lc):
    """From the packed codes of Z, the output agrees with lcvq_linear_fwd on Z itself."""
    import torch
    N, m, n, d = 16, 512, 2048, 8
    inp, P = _inputs(N, m, n, d, seed=3)
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    Z, X = to_dev(inp["Z"], "bf16"), to_dev(inp["X"], "bf16")
    packed = torch.empty((m, n // 4), dtype=torch.uint8, device="cuda")
    Y1 = lc.linear_fwd(Z, A, b, X, d, packed_out=packed)
    Y2 = lc.linear_fwd_packed(packed, A, b, X, d, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert np.array_equal(packed.cpu().numpy(), P)
    assert rel_fro(to_host(Y2), to_host(Y1)) <= 1e-2


def test_packed_forward_extreme_codes(lc):
    """All codes 3 or all 0 (the extreme bytes 0xFF and 0x00)."""
    import torch
    N, m, n, d = 4, 64, 512, 4
    inp, _ = _inputs(N, m, n, d, seed=9)
    for byte in (0xFF, 0x00, 0x1B):
        P = np.full((m, n // 4), byte, np.uint8)
        got = _run(lc, inp, P, d, "f32")[0]
        assert_close(got, _ref(inp, P, d, n), TOL, 'Y')


def test_packed_forward_degenerate(lc):
    import torch
    d = 8
    A, b = torch.eye(d, device="cuda"), torch.zeros(d, device="cuda")
    P = torch.zeros((16, 16), dtype=torch.uint8, device="cuda")            # m = 16, n = 64
    Y = lc.linear_fwd_packed(P, A, b, torch.empty((0, 64), dtype=torch.bfloat16, device="cuda"), d)
    assert Y.shape == (0, 16)
    Y = lc.linear_fwd_packed(torch.zeros((16, 0), dtype=torch.uint8, device="cuda"), A, b,
                             torch.empty((3, 0), dtype=torch.bfloat16, device="cuda"), d,
                             out=torch.full((3, 16), 5.0, dtype=torch.bfloat16, device="cuda"))
    torch.cuda.synchronize()
    assert torch.all(Y == 0)
    with pytest.raises(lc.LcvqError):             # n % 64 != 0
        lc.linear_fwd_packed(torch.zeros((16, 8), dtype=torch.uint8, device="cuda"), A, b,
                             torch.zeros((1, 32), dtype=torch.bfloat16, device="cuda"), d)


@pytest.mark.parametrize("N", [1, 16])
@pytest.mark.parametrize("m,n", [(28672, 8192), (8192, 28672), (4096, 4096)])
def test_packed_forward_full_size_sampled(lc, N, m, n):
    """Full-size matrices in the benchmark's launch configuration: sampled rows."""
    import torch
    d = 8
    r = synth.rng(m + n + N)
    P = r.integers(0, 256, size=(m, n // 4), dtype=np.uint8)    # uniformly random codes
    X = synth.draw_activations(N, n, 7 + N, "bf16")
    A, b = synth.draw_map(d, 1)
    Y = lc.linear_fwd_packed(torch.from_numpy(P).cuda(), torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda(),
                             to_dev(X, "bf16"), d)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(32), r.integers(0, m, 96), [m - 1]]))
    ref = orc.linear_forward_packed(P[rows], A.astype(np.float64), b.astype(np.float64), orc.widen(X, "bf16"), d, n)
    assert_close(to_host(Y)[:, rows], ref, TOL, 'Y')


@pytest.mark.parametrize("d", [8, 4])
@pytest.mark.parametrize("N,m,n", [(3, 12344, 6144), (1, 12352, 6144), (2, 12344, 6208), (17, 12352, 6144)])
def test_packed_forward_few_tokens_long_rows(lc, N, m, n, d):
    """Few tokens with at least 24 product steps per block and one block per
    row tile: each block computes the X'' rows of its steps into LDS itself
    (no prepass); ragged last row tile (m % 64 != 0), K not a multiple of 256;
    17 tokens: a 16-token pass with the prepass, then a 1-token pass without.
    Two calls give the same bits (the offsets are summed in a fixed order)."""
    inp, P = _inputs(N, m, n, d, seed=m + N + d)
    got = _run(lc, inp, P, d, "f32", calls=2)
    assert_close(got[0], _ref(inp, P, d, n), TOL, 'Y')
    assert np.array_equal(got[0], got[1])


@pytest.mark.parametrize("N", [2, 3])
def test_packed_forward_full_size_two_three_tokens(lc, N):
    """28672 x 8192 at 2 tokens (X'' computed into LDS by the product blocks)
    and 3 tokens, sampled rows."""
    import torch
    m, n, d = 28672, 8192, 8
    r = synth.rng(m + n + N)
    P = r.integers(0, 256, size=(m, n // 4), dtype=np.uint8)
    X = synth.draw_activations(N, n, 7 + N, "bf16")
    A, b = synth.draw_map(d, 1)
    Y = lc.linear_fwd_packed(torch.from_numpy(P).cuda(), torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda(),
                             to_dev(X, "bf16"), d)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(32), r.integers(0, m, 96), [m - 1]]))
    ref = orc.linear_forward_packed(P[rows], A.astype(np.float64), b.astype(np.float64), orc.widen(X, "bf16"), d, n)
    assert_close(to_host(Y)[:, rows], ref, TOL, 'Y')

"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Codes and packed words are compared bit for bit.  Floating-point results are
compared by relative Frobenius error: <= 2e-2 for bf16 inputs with fp32
accumulation, <= 1e-5 in fp32 mode."""
import numpy as np
import pytest

import oracle as orc
import synth
from helpers import assert_close, rel_fro, to_dev, to_host, unpack2bit

pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-2, "f32": 1e-5}


@pytest.fixture(scope="module")
def lc():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_10531_amd as lc
    lc._lib.load()
    return lc


def _special_latents(shape, dtype, seed):
    """Latents with exact ties, range edges, signed zeros and out-of-range values mixed in."""
    r = synth.rng(seed)
    z = r.uniform(-2.0, 5.0, size=shape).astype(np.float32)
    special = np.array([-0.5, 0.5, 1.5, 2.5, 3.5, -0.0, 0.0, 3.0, -1e-3, 3.4999, 1e30, -1e30, 0.49, 2.51],
                       np.float32)
    idx = r.integers(0, z.size, size=z.size // 5)
    z.reshape(-1)[idx] = special[r.integers(0, special.size, size=idx.size)]
    return synth.bf16_bits(z) if dtype == "bf16" else z


# ---------------------------------------------------------------- codes -----

def test_quantiser_exhaustive_bf16(lc):
    import torch
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).reshape(256, 256)
    Z = to_dev(bits, "bf16")
    packed = lc.pack2bit(Z)
    torch.cuda.synchronize()
    got = unpack2bit(packed.cpu().numpy(), 256)
    want = orc.quantize(orc.widen(bits, "bf16"))
    assert np.array_equal(got, want)
    # the same codes through the dense decode with A = I, b = 0
    W = lc.dequant(Z, torch.eye(8, device="cuda"), torch.zeros(8, device="cuda"), 8, out_dtype=torch.float32)
    assert np.array_equal(to_host(W), want.astype(np.float64))


def test_quantiser_fp32_boundaries(lc):
    pts = []
    for h in [-1.5, -0.5, 0.5, 1.5, 2.5, 3.5, 4.5]:
        lo = hi = np.float32(h)
        for _ in range(32):
            lo = np.nextafter(lo, np.float32(-np.inf))
            hi = np.nextafter(hi, np.float32(np.inf))
            pts += [lo, hi]
        pts.append(np.float32(h))
    z = np.concatenate([np.array(pts, np.float32),
                        np.array([np.inf, -np.inf, np.nan, -np.nan, 0.0, -0.0], np.float32),
                        synth.rng(3).uniform(-3, 6, 64 * 1024 - len(pts) - 6).astype(np.float32)])
    z = z[: (z.size // 64) * 64].reshape(-1, 64)
    got = unpack2bit(lc.pack2bit(to_dev(z, "f32")).cpu().numpy(), 64)
    assert np.array_equal(got, orc.quantize(z.astype(np.float64)))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("m,n", [(37, 132), (64, 256), (1, 4), (5, 20)])
def test_pack2bit(lc, dtype, m, n):
    Z = _special_latents((m, n), dtype, m * n)
    got = lc.pack2bit(to_dev(Z, dtype)).cpu().numpy()
    want = orc.pack2bit(orc.quantize(orc.widen(Z, dtype)))
    assert np.array_equal(got, want)


def test_pack2bit_from_u8_codes(lc):
    import torch
    codes = synth.rng(8).integers(0, 6, size=(33, 68)).astype(np.uint8)     # 4, 5 are taken as 3
    got = lc.pack2bit(torch.from_numpy(codes).cuda()).cpu().numpy()
    assert np.array_equal(got, orc.pack2bit(np.minimum(codes, 3)))


# --------------------------------------------------------------- decode -----

@pytest.mark.parametrize("d", [4, 8])
@pytest.mark.parametrize("src", ["latent_bf16", "latent_f32", "u8", "packed"])
@pytest.mark.parametrize("out", ["bf16", "f32"])
@pytest.mark.parametrize("m,groups", [(40, 24), (3, 5), (125, 65)])  # whole 16-byte chunks; a tail; two per thread
def test_dequant(lc, d, src, out, m, groups):
    import torch
    n = groups * d
    A, b = synth.draw_map(d, 1)
    A = (A * 50).astype(np.float32)           # O(1) map so rounding is visible
    Zf = _special_latents((m, n), "f32", 11 + m)
    codes = orc.quantize(Zf.astype(np.float64))
    if src == "latent_bf16":
        Zb = synth.bf16_bits(Zf)
        codes = orc.quantize(orc.widen(Zb, "bf16"))
        W = lc.dequant(to_dev(Zb, "bf16"), torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda(), d,
                       out_dtype=getattr(torch, "bfloat16" if out == "bf16" else "float32"))
    elif src == "latent_f32":
        W = lc.dequant(to_dev(Zf, "f32"), torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda(), d,
                       out_dtype=getattr(torch, "bfloat16" if out == "bf16" else "float32"))
    elif src == "u8":
        W = lc.dequant(torch.from_numpy(codes).cuda(), torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda(), d,
                       out_dtype=getattr(torch, "bfloat16" if out == "bf16" else "float32"))
    else:
        P = torch.from_numpy(orc.pack2bit(codes)).cuda()
        W = lc.dequant(P, torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda(), d, n=n,
                       src_kind=lc.SRC_PACKED2, out_dtype=getattr(torch, "bfloat16" if out == "bf16" else "float32"))
    want = orc.decode(codes, A.astype(np.float64), b.astype(np.float64), d)
    got = to_host(W)
    if out == "f32":
        assert np.allclose(got, want, rtol=1e-6, atol=1e-6)
    else:
        assert np.allclose(got, want, rtol=2 ** -8, atol=1e-6)


@pytest.mark.parametrize("d", [8, 4])
@pytest.mark.parametrize("src", ["packed", "u8"])
def test_dequant_many_chunks_sampled(lc, d, src):
    """6144 x 8192 codes: every wave of the decode takes several trips of its
    chunk loop (the next pair of chunks loaded while the current pair is
    decoded and stored) and the grid ends in a partial stride; sampled rows
    against the oracle."""
    import torch
    m, n = 6144, 8192
    A, b = synth.draw_map(d, 2)
    A = (A * 50).astype(np.float32)
    codes = synth.rng(77 + d).integers(0, 4, size=(m, n), dtype=np.uint8)
    At, bt = torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda()
    if src == "packed":
        W = lc.dequant(torch.from_numpy(orc.pack2bit(codes)).cuda(), At, bt, d, n=n, src_kind=lc.SRC_PACKED2,
                       out_dtype=torch.bfloat16)
    else:
        W = lc.dequant(torch.from_numpy(codes).cuda(), At, bt, d, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, 1, m // 2, m - 1], synth.rng(78).integers(0, m, 60)]))
    want = orc.decode(codes[rows], A.astype(np.float64), b.astype(np.float64), d)
    got = to_host(W[torch.from_numpy(rows).cuda()])
    assert np.allclose(got, want, rtol=2 ** -8, atol=1e-6)


# ---------------------------------------------------------- linear layer ----

def _run_layer(lc, N, m, n, d, dtype, mask_mode=0, z_lo=-0.5, z_hi=3.5, k=0, dz_dtype=None):
    import torch
    inp = synth.layer_inputs(N, m, n, d, dtype, k=k, z_lo=z_lo, z_hi=z_hi)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    Z, X, dY = to_dev(inp["Z"], dtype), to_dev(inp["X"], dtype), to_dev(inp["dY"], dtype)
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    packed = torch.empty((m, n // 4), dtype=torch.uint8, device="cuda")
    Y = lc.linear_fwd(Z, A, b, X, d, packed_out=packed)
    dX, dZ, dA, db = lc.linear_bwd(Z, A, b, X, dY, d, mask_mode=mask_mode, dz_dtype=dz_dtype or tdt)
    torch.cuda.synchronize()
    v = {key: orc.widen(inp[key], dtype) for key in ("Z", "X", "dY")}
    A64, b64 = inp["A"].astype(np.float64), inp["b"].astype(np.float64)
    Yref, codes = orc.linear_forward(v["Z"], A64, b64, v["X"], d)
    ref = orc.linear_backward(v["Z"], A64, b64, v["X"], v["dY"], d, mask_mode)
    got = dict(Y=to_host(Y), dX=to_host(dX), dZ=to_host(dZ), dA=to_host(dA), db=to_host(db),
               packed=packed.cpu().numpy())
    return got, dict(Y=Yref, codes=codes, mask=orc.ste_mask(v["Z"], mask_mode), **ref)


SHAPES = [  # (N, m, n): several tiles, ragged token / row / column tails
    (300, 320, 512),
    (1000, 264, 328),
    (256, 256, 256),
    (513, 520, 1096),
    (1, 8, 8),
    (77, 24, 64),
]


@pytest.mark.parametrize("d", [8, 4])
@pytest.mark.parametrize("N,m,n", SHAPES)
def test_layer_bf16(lc, N, m, n, d):
    got, ref = _run_layer(lc, N, m, n, d, "bf16", z_lo=-2.0, z_hi=5.0, k=N + m + n + d)
    assert np.array_equal(got["packed"], orc.pack2bit(ref["codes"]))
    for key in ("Y", "dX", "dZ", "dA", "db"):
        assert_close(got[key], ref[key], TOL["bf16"], key)
    assert np.all(got["dZ"][~ref["mask"]] == 0.0)


@pytest.mark.parametrize("N,m,n,d", [(16, 256, 256, 8), (37, 72, 200, 4), (130, 100, 96, 8), (3, 4, 8, 4)])
def test_layer_fp32(lc, N, m, n, d):
    got, ref = _run_layer(lc, N, m, n, d, "f32", z_lo=-2.0, z_hi=5.0, k=7)
    assert np.array_equal(got["packed"], orc.pack2bit(ref["codes"]))
    for key in ("Y", "dX", "dZ", "dA", "db"):
        assert_close(got[key], ref[key], TOL["f32"], key)
    assert np.all(got["dZ"][~ref["mask"]] == 0.0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_mask_latent_mode_and_fp32_grad(lc, dtype):
    import torch
    got, ref = _run_layer(lc, 200, 136, 264, 8, dtype, mask_mode=1, z_lo=-2.0, z_hi=5.0, k=3,
                          dz_dtype=torch.float32)
    assert np.all(got["dZ"][~ref["mask"]] == 0.0)
    assert_close(got["dZ"], ref["dZ"], TOL[dtype], 'dZ')


@pytest.mark.parametrize("dtype,dzt", [("bf16", "f32"), ("bf16", "bf16"), ("f32", "f32")])
def test_accumulate(lc, dtype, dzt):
    """accumulate=1 adds to dZ, dA, db (gradient accumulation), also into a bf16 dZ:
    two calls give twice the oracle's gradients."""
    import torch
    N, m, n, d = 96, 64, 128, 8
    inp = synth.layer_inputs(N, m, n, d, dtype, k=5, z_lo=-2.0, z_hi=5.0)
    Z, X, dY = to_dev(inp["Z"], dtype), to_dev(inp["X"], dtype), to_dev(inp["dY"], dtype)
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    tdz = torch.float32 if dzt == "f32" else torch.bfloat16
    _, dZ1, dA1, db1 = lc.linear_bwd(Z, A, b, X, dY, d, need_dX=False, dz_dtype=tdz)
    dZ = dZ1.clone()
    dA, db = dA1.clone(), db1.clone()
    lc.linear_bwd(Z, A, b, X, dY, d, accumulate=True, need_dX=False, dZ=dZ, dA=dA, db=db)
    torch.cuda.synchronize()
    # bf16 dZ: the sum is rounded once more (one bf16 rounding of 2 dZ)
    assert rel_fro(to_host(dZ), 2 * to_host(dZ1)) <= (1e-6 if dzt == "f32" else 2.0 ** -8)
    assert rel_fro(to_host(dA), 2 * to_host(dA1)) <= 1e-6
    assert rel_fro(to_host(db), 2 * to_host(db1)) <= 1e-6
    v = {key: orc.widen(inp[key], dtype) for key in ("Z", "X", "dY")}
    ref = orc.linear_backward(v["Z"], inp["A"].astype(np.float64), inp["b"].astype(np.float64), v["X"], v["dY"], d)
    for key, got in (("dZ", dZ), ("dA", dA), ("db", db)):
        assert_close(to_host(got), 2 * ref[key], TOL[dtype], key)


def test_identity_map_reproduces_codes_in_forward(lc):
    # A = I, b = 0 and one-hot X rows: Y row t reads the codes of column t
    import torch
    m, n = 64, 128
    Zb = synth.draw_latent(m, n, 2, "bf16", -1.0, 4.0)
    X = np.zeros((n, n), np.float32)
    X[np.arange(n), np.arange(n)] = 1.0
    Y = lc.linear_fwd(to_dev(Zb, "bf16"), torch.eye(8, device="cuda"), torch.zeros(8, device="cuda"),
                      to_dev(synth.bf16_bits(X), "bf16"), 8)
    codes = orc.quantize(orc.widen(Zb, "bf16"))
    assert np.array_equal(to_host(Y), codes.T.astype(np.float64))


def test_degenerate_sizes(lc):
    import torch
    d = 8
    A, b = torch.eye(d, device="cuda"), torch.zeros(d, device="cuda")
    # N = 0: nothing to compute
    Z = torch.ones(16, 16, dtype=torch.bfloat16, device="cuda")
    Y = lc.linear_fwd(Z, A, b, torch.empty(0, 16, dtype=torch.bfloat16, device="cuda"), d)
    assert Y.shape == (0, 16)
    _, dZ, dA, db = lc.linear_bwd(Z, A, b, torch.empty(0, 16, dtype=torch.bfloat16, device="cuda"),
                                  torch.empty(0, 16, dtype=torch.bfloat16, device="cuda"), d, need_dX=False)
    torch.cuda.synchronize()
    assert torch.all(dZ == 0) and torch.all(dA == 0) and torch.all(db == 0)
    # n = 0: Y is an N x m matrix of zeros
    Y = lc.linear_fwd(torch.empty(16, 0, dtype=torch.bfloat16, device="cuda"), A, b,
                      torch.empty(5, 0, dtype=torch.bfloat16, device="cuda"), d,
                      out=torch.full((5, 16), 7.0, dtype=torch.bfloat16, device="cuda"))
    torch.cuda.synchronize()
    assert torch.all(Y == 0)


# ------------------------------------------------ full-size, sampled -----

@pytest.mark.parametrize("d", [8])
def test_layer_4096_sampled(lc, d):
    """The 4096 x 4096 layer with 4096 tokens, in the launch configuration the
    benchmark times: all codes bit-exact; Y, dX and dZ on sampled rows; dA, db
    in full."""
    import torch
    N = m = n = 4096
    inp = synth.layer_inputs(N, m, n, d, "bf16", k=0)
    Z, X, dY = to_dev(inp["Z"], "bf16"), to_dev(inp["X"], "bf16"), to_dev(inp["dY"], "bf16")
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    packed = torch.empty((m, n // 4), dtype=torch.uint8, device="cuda")
    Y = lc.linear_fwd(Z, A, b, X, d, packed_out=packed)
    dX, dZ, dA, db = lc.linear_bwd(Z, A, b, X, dY, d)
    torch.cuda.synchronize()
    v = {key: orc.widen(inp[key], "bf16") for key in ("Z", "X", "dY")}
    A64, b64 = inp["A"].astype(np.float64), inp["b"].astype(np.float64)
    codes = orc.quantize(v["Z"])
    assert np.array_equal(packed.cpu().numpy(), orc.pack2bit(codes))
    W = orc.decode(codes, A64, b64, d)
    rows = np.unique(np.concatenate([np.arange(64), synth.rng(99).integers(0, 4096, 192), [4095]]))
    assert_close(to_host(Y[rows]), orc.forward(v["X"][rows], W), TOL["bf16"], 'Y')
    assert_close(to_host(dX[rows]), orc.grad_input(v["dY"][rows], W), TOL["bf16"], 'dX')
    dW_rows = orc.grad_weight(v["dY"][:, rows], v["X"])
    mask = orc.ste_mask(v["Z"][rows])
    assert_close(to_host(dZ[rows]), orc.grad_latent(dW_rows, A64, d, mask), TOL["bf16"], 'dZ')
    dA_ref, db_ref = orc.grad_map(orc.grad_weight(v["dY"], v["X"]), codes, d)
    assert_close(to_host(dA), dA_ref, TOL["bf16"], 'dA')
    assert_close(to_host(db), db_ref, TOL["bf16"], 'db')

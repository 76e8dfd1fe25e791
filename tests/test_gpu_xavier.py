"""The quantiser domain of the Xavier reparameterisation (eq. xavier_preprocess,
Sec. 3.4) against the fp64 oracle, through the C ABI: codes of fp32
fma(W_p, 1/s', t) bit-exact, floating-point results to the usual bar, and the
latent gradient scaled by 1/s'."""
import ctypes

import numpy as np
import pytest

import oracle as orc
import synth
from helpers import assert_close, to_dev, to_host, unpack2bit

pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-2, "f32": 1e-5}


@pytest.fixture(scope="module")
def lc():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_10531_amd as lc
    lc._lib.load()
    return lc


def _xavier_latents(m, n, dtype, seed):
    """W_p = s' (Z - t) for code-domain Z ~ U(-2, 5) (codes, boundaries and the
    clip range all exercised), stored in `dtype`."""
    sp, t = orc.xavier_params(m, n)
    z = synth.rng(seed).uniform(-2.0, 5.0, size=(m, n))
    w = (sp * (z - t)).astype(np.float32)
    return synth.bf16_bits(w) if dtype == "bf16" else w


def test_xavier_quantiser_exhaustive_bf16(lc):
    """All 65 536 bf16 latents through the forward's quantise blocks."""
    import torch
    m = n = 256
    qs, qb = lc.xavier_quantizer(m, n)
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).reshape(m, n)
    Z = to_dev(bits, "bf16")
    X = torch.zeros((1, n), dtype=torch.bfloat16, device="cuda")
    packed = torch.empty((m, n // 4), dtype=torch.uint8, device="cuda")
    A, b = torch.eye(8, device="cuda"), torch.zeros(8, device="cuda")
    lc.linear_fwd(Z, A, b, X, 8, packed_out=packed, q_scale=qs, q_shift=qb)
    torch.cuda.synchronize()
    want = orc.quantize(orc.widen(bits, "bf16"), np.float32(qs), np.float32(qb))
    assert np.array_equal(unpack2bit(packed.cpu().numpy(), n), want)
    assert len(np.unique(want)) == 4


def _run(lc, N, m, n, d, dtype, mask_mode, dge, seed):
    import torch
    inp = synth.layer_inputs(N, m, n, d, dtype, k=seed)
    Wh = _xavier_latents(m, n, dtype, seed)
    qs, qb = lc.xavier_quantizer(m, n)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    W, X, dY = to_dev(Wh, dtype), to_dev(inp["X"], dtype), to_dev(inp["dY"], dtype)
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    packed = torch.empty((m, n // 4), dtype=torch.uint8, device="cuda")
    Y = lc.linear_fwd(W, A, b, X, d, packed_out=packed, q_scale=qs, q_shift=qb)
    if dge is None:
        dX, dZ, dA, db = lc.linear_bwd(W, A, b, X, dY, d, mask_mode=mask_mode, dz_dtype=torch.float32, q_scale=qs,
                                       q_shift=qb)
    else:
        dX, dZ, dA, db = lc.linear_bwd_dge(W, A, b, X, dY, d, k=dge[0], cap=dge[1], mask_mode=mask_mode,
                                           dz_dtype=torch.float32, q_scale=qs, q_shift=qb)
    torch.cuda.synchronize()
    v = {"W": orc.widen(Wh, dtype), "X": orc.widen(inp["X"], dtype), "dY": orc.widen(inp["dY"], dtype)}
    A64, b64 = inp["A"].astype(np.float64), inp["b"].astype(np.float64)
    qs32, qb32 = np.float32(qs), np.float32(qb)
    Yref, codes = orc.linear_forward(v["W"], A64, b64, v["X"], d, qs32, qb32)
    ref = orc.linear_backward(v["W"], A64, b64, v["X"], v["dY"], d, mask_mode, dge=dge, scale=qs32, shift=qb32)
    got = dict(Y=to_host(Y), dX=to_host(dX), dZ=to_host(dZ), dA=to_host(dA), db=to_host(db))
    return got, dict(Y=Yref, codes=codes, **ref), packed.cpu().numpy(), \
        orc.ste_mask(v["W"], mask_mode, qs32, qb32)


@pytest.mark.parametrize("dge", [None, (5.0, 3.0)])
@pytest.mark.parametrize("mask_mode", [0, 1])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("N,m,n,d", [(300, 320, 512, 8), (77, 24, 64, 4), (130, 136, 264, 8)])
def test_xavier_layer(lc, N, m, n, d, dtype, mask_mode, dge):
    got, ref, packed, mask = _run(lc, N, m, n, d, dtype, mask_mode, dge, seed=N + m + d)
    assert np.array_equal(packed, orc.pack2bit(ref["codes"]))
    for key in ("Y", "dX", "dZ", "dA", "db"):
        assert_close(got[key], ref[key], TOL[dtype], key)
    assert np.all(got["dZ"][~mask] == 0.0)
    assert mask.any() and (~mask).any()


def test_xavier_quantizer_values(lc):
    """lcvq_xavier_quantizer against eq. xavier_preprocess: (1 / s', t) rounded to fp32."""
    for m, n in ((4096, 4096), (11008, 4096), (3, 5)):
        sp, t = orc.xavier_params(m, n)
        qs, qb = lc.xavier_quantizer(m, n)
        assert qs == float(np.float32(1.0 / sp)) and qb == float(np.float32(t))


@pytest.mark.parametrize("src", ["u8", "packed"])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_xavier_init_round_trip(lc, dtype, src):
    """codes -> W_p = s'(W_z - t) (lcvq_xavier_init) -> forward with the Xavier quantiser
    returns the same codes; W_p equals lcvq_dequant with A = s' I, b = -s' t (bit for
    bit from byte codes, whose decode is the same fma; to fp32 rounding from packed
    codes, whose decode sums two half-group tables)."""
    import torch
    m, n, d = 200, 264, 8
    codes = synth.rng(5).integers(0, 4, size=(m, n), dtype=np.uint8)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    csrc = torch.from_numpy(codes if src == "u8" else orc.pack2bit(codes)).cuda()
    W = lc.xavier_init(csrc, m, n, out_dtype=tdt)
    qs, qb = lc.xavier_quantizer(m, n)
    packed = torch.empty((m, n // 4), dtype=torch.uint8, device="cuda")
    X = torch.zeros((4, n), dtype=tdt, device="cuda")
    lc.linear_fwd(W, torch.eye(d, device="cuda"), torch.zeros(d, device="cuda"), X, d, packed_out=packed,
                  q_scale=qs, q_shift=qb)
    sp, t = orc.xavier_params(m, n)
    Wd = lc.dequant(csrc, torch.eye(d, device="cuda") * sp, torch.full((d,), -sp * t, device="cuda"), d, n=n,
                    src_kind=lc.SRC_CODES_U8 if src == "u8" else lc.SRC_PACKED2, out_dtype=tdt)
    torch.cuda.synchronize()
    assert np.array_equal(packed.cpu().numpy(), orc.pack2bit(codes))
    if src == "u8":
        assert torch.equal(W, Wd)
    else:
        assert_close(to_host(W), to_host(Wd), 4e-3 if dtype == "bf16" else 1e-7, "W_p vs dequant")
    assert_close(to_host(W), sp * (codes.astype(np.float64) - t), 4e-3 if dtype == "bf16" else 1e-7, "W_p")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_ex_entry_points_in_the_code_domain_match_the_plain_ones(lc, dtype):
    """lcvq_linear_fwd_ex / lcvq_linear_bwd_ex with (1, 0) and the STE give the
    plain entry points' results bit for bit."""
    import torch
    N, m, n, d = 64, 72, 136, 8
    inp = synth.layer_inputs(N, m, n, d, dtype, k=2, z_lo=-2.0, z_hi=5.0)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    Z, X, dY = to_dev(inp["Z"], dtype), to_dev(inp["X"], dtype), to_dev(inp["dY"], dtype)
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    lib = lc._lib.load()
    dt = lc._lib.BF16 if dtype == "bf16" else lc._lib.F32
    ws = torch.empty(max(lc.workspace_bytes(lc.OP_FWD, N, m, n, d, tdt),
                         lc.workspace_bytes(lc.OP_BWD, N, m, n, d, tdt)), dtype=torch.uint8, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    Y1 = lc.linear_fwd(Z, A, b, X, d)
    Y2 = torch.empty_like(Y1)
    lc._lib.check(lib.lcvq_linear_fwd_ex(N, m, n, d, dt, Z.data_ptr(), 1.0, 0.0, A.data_ptr(), b.data_ptr(),
                                         X.data_ptr(), Y2.data_ptr(), None, ws.data_ptr(), ws.numel(), stream),
                  "lcvq_linear_fwd_ex")
    dX1, dZ1, _, _ = lc.linear_bwd(Z, A, b, X, dY, d, need_map=False, dz_dtype=torch.float32)
    dX2, dZ2 = torch.empty_like(dX1), torch.empty_like(dZ1)
    lc._lib.check(lib.lcvq_linear_bwd_ex(N, m, n, d, dt, Z.data_ptr(), 1.0, 0.0, A.data_ptr(), b.data_ptr(),
                                         X.data_ptr(), dY.data_ptr(), 0, lc.EST_STE, 0.0, 0.0, 0, dX2.data_ptr(),
                                         dZ2.data_ptr(), lc._lib.F32, None, None, ws.data_ptr(), ws.numel(),
                                         stream), "lcvq_linear_bwd_ex")
    torch.cuda.synchronize()
    assert torch.equal(Y1, Y2) and torch.equal(dX1, dX2) and torch.equal(dZ1, dZ2)

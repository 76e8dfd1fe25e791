"""Parity of the backward with the differentiable gradient estimator (eq. dge,
Sec. 3.3) against the fp64 oracle, through the C ABI.

Same bar as the straight-through backward: relative Frobenius error <= 2e-2
for bf16 inputs and <= 1e-5 in fp32 mode; dZ exactly 0 where the mask is 0."""
import numpy as np
import pytest

import oracle as orc
import synth
from helpers import assert_close, rel_fro, to_dev, to_host

pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-2, "f32": 1e-5}


@pytest.fixture(scope="module")
def lc():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_10531_amd as lc
    lc._lib.load()
    return lc


def _with_special_latents(Z, dtype, seed):
    """Mix in the middles of rounding intervals (slope = cap), integers (slope
    1/k), range edges and non-finite values."""
    r = synth.rng(seed)
    z = orc.widen(Z, dtype).astype(np.float32) if dtype == "bf16" else np.array(Z, np.float32)
    special = np.array([0.5, 1.5, 2.5, -0.5, 3.5, 0.0, -0.0, 1.0, 3.0, 0.25, 2.75, -1e-3, 3.001,
                        np.nan, np.inf, -np.inf], np.float32)
    idx = r.integers(0, z.size, size=z.size // 6)
    z.reshape(-1)[idx] = special[r.integers(0, special.size, size=idx.size)]
    return synth.bf16_bits(z) if dtype == "bf16" else z


def _run(lc, N, m, n, d, dtype, mask_mode, k, cap, seed, special=True, dz_dtype=None, accumulate_twice=False):
    import torch
    inp = synth.layer_inputs(N, m, n, d, dtype, k=seed, z_lo=-2.0, z_hi=5.0)
    Zh = _with_special_latents(inp["Z"], dtype, seed) if special else inp["Z"]
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    Z, X, dY = to_dev(Zh, dtype), to_dev(inp["X"], dtype), to_dev(inp["dY"], dtype)
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    dX, dZ, dA, db = lc.linear_bwd_dge(Z, A, b, X, dY, d, k=k, cap=cap, mask_mode=mask_mode,
                                       dz_dtype=dz_dtype or tdt)
    if accumulate_twice:
        lc.linear_bwd_dge(Z, A, b, X, dY, d, k=k, cap=cap, mask_mode=mask_mode, accumulate=True,
                          need_dX=False, dZ=dZ, dA=dA, db=db)
    torch.cuda.synchronize()
    v = {"Z": orc.widen(Zh, dtype), "X": orc.widen(inp["X"], dtype), "dY": orc.widen(inp["dY"], dtype)}
    ref = orc.linear_backward(v["Z"], inp["A"].astype(np.float64), inp["b"].astype(np.float64), v["X"],
                              v["dY"], d, mask_mode, dge=(k, cap))
    got = dict(dX=to_host(dX), dZ=to_host(dZ), dA=to_host(dA), db=to_host(db))
    return got, ref, orc.ste_mask(v["Z"], mask_mode), v["Z"]


SHAPES = [(300, 320, 512), (513, 520, 1096), (77, 24, 64), (1, 8, 8)]


@pytest.mark.parametrize("mask_mode", [1, 0])
@pytest.mark.parametrize("d", [8, 4])
@pytest.mark.parametrize("N,m,n", SHAPES)
def test_dge_bf16(lc, N, m, n, d, mask_mode):
    got, ref, mask, _ = _run(lc, N, m, n, d, "bf16", mask_mode, 5.0, 3.0, seed=N + m + n + d + mask_mode)
    for key in ("dX", "dZ", "dA", "db"):
        assert_close(got[key], ref[key], TOL["bf16"], key)
    assert np.all(np.isfinite(got["dZ"]))
    assert np.all(got["dZ"][~mask] == 0.0)


@pytest.mark.parametrize("mask_mode", [1, 0])
@pytest.mark.parametrize("N,m,n,d", [(16, 256, 256, 8), (37, 72, 200, 4), (130, 100, 96, 8)])
def test_dge_fp32(lc, N, m, n, d, mask_mode):
    got, ref, mask, _ = _run(lc, N, m, n, d, "f32", mask_mode, 5.0, 3.0, seed=11 + d + mask_mode)
    for key in ("dX", "dZ", "dA", "db"):
        assert_close(got[key], ref[key], TOL["f32"], key)
    assert np.all(got["dZ"][~mask] == 0.0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("k,cap", [(5.0, 10.0), (2.0, 1.5), (9.0, 3.0)])
def test_dge_other_sharpness_and_caps(lc, dtype, k, cap):
    import torch
    got, ref, mask, _ = _run(lc, 96, 64, 256, 8, dtype, 1, k, cap, seed=int(10 * k + cap),
                             dz_dtype=torch.float32)
    assert_close(got["dZ"], ref["dZ"], TOL[dtype], 'dZ')
    assert np.all(got["dZ"][~mask] == 0.0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_dge_slope_elementwise_against_straight_through(lc, dtype):
    """dZ with the estimator equals slope(Z) times the straight-through dZ of the
    same device call sequence, element by element (both use the same product)."""
    import torch
    N, m, n, d = 64, 64, 256, 8
    inp = synth.layer_inputs(N, m, n, d, dtype, k=4, z_lo=-2.0, z_hi=5.0)
    Zh = _with_special_latents(inp["Z"], dtype, 4)
    Z, X, dY = to_dev(Zh, dtype), to_dev(inp["X"], dtype), to_dev(inp["dY"], dtype)
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    _, dZs, _, _ = lc.linear_bwd(Z, A, b, X, dY, d, mask_mode=1, need_dX=False, need_map=False,
                                 dz_dtype=torch.float32)
    _, dZd, _, _ = lc.linear_bwd_dge(Z, A, b, X, dY, d, k=5.0, cap=3.0, mask_mode=1, need_dX=False,
                                     need_map=False, dz_dtype=torch.float32)
    torch.cuda.synchronize()
    slope = orc.dge_slope(orc.widen(Zh, dtype), 5.0, 3.0)
    s, g = to_host(dZs), to_host(dZd)
    live = s != 0
    # the device slope comes from the hardware log2 / exp2 (about 1e-6 relative)
    assert np.allclose(g[live], slope[live] * s[live], rtol=2e-6, atol=0)
    assert np.all(g[~live] == 0.0)
    zf = orc.widen(Zh, dtype)
    with np.errstate(invalid="ignore"):
        mid = live & (np.abs(zf - np.floor(zf) - 0.5) == 0)
    # the cap, exactly: the fp32 product cap * dW rounded once
    assert mid.any() and np.array_equal(g[mid], (3.0 * s[mid]).astype(np.float32).astype(np.float64))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_dge_k_one_is_straight_through(lc, dtype):
    import torch
    N, m, n, d = 100, 72, 136, 8
    inp = synth.layer_inputs(N, m, n, d, dtype, k=8, z_lo=-2.0, z_hi=5.0)
    Zh = _with_special_latents(inp["Z"], dtype, 8)
    Z, X, dY = to_dev(Zh, dtype), to_dev(inp["X"], dtype), to_dev(inp["dY"], dtype)
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    for mode in (0, 1):
        dXs, dZs, dAs, dbs = lc.linear_bwd(Z, A, b, X, dY, d, mask_mode=mode, dz_dtype=torch.float32)
        dXd, dZd, dAd, dbd = lc.linear_bwd_dge(Z, A, b, X, dY, d, k=1.0, cap=3.0, mask_mode=mode,
                                               dz_dtype=torch.float32)
        torch.cuda.synchronize()
        assert torch.equal(dZs, dZd)
        assert torch.equal(dXs, dXd)
        if dtype == "bf16":  # per-block partial sums added in a fixed order: the same bits
            assert torch.equal(dAd, dAs) and torch.equal(dbd, dbs)
        else:  # the fp32 path sums with atomics, in an unspecified order
            assert rel_fro(to_host(dAd), to_host(dAs)) <= 1e-6
            assert rel_fro(to_host(dbd), to_host(dbs)) <= 1e-6


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_dge_accumulate(lc, dtype):
    import torch
    got, ref, _, _ = _run(lc, 96, 64, 128, 8, dtype, 1, 5.0, 3.0, seed=21, dz_dtype=torch.float32,
                          accumulate_twice=True)
    for key in ("dZ", "dA", "db"):
        assert_close(got[key], 2 * ref[key], TOL[dtype], key)


def test_dge_4096_sampled(lc):
    """The 4096 x 4096 layer with 4096 tokens: dZ on sampled rows, dA and db in full."""
    import torch
    N = m = n = 4096
    d = 8
    inp = synth.layer_inputs(N, m, n, d, "bf16", k=0, z_lo=-2.0, z_hi=5.0)
    Z, X, dY = to_dev(inp["Z"], "bf16"), to_dev(inp["X"], "bf16"), to_dev(inp["dY"], "bf16")
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    dX, dZ, dA, db = lc.linear_bwd_dge(Z, A, b, X, dY, d)
    torch.cuda.synchronize()
    v = {key: orc.widen(inp[key], "bf16") for key in ("Z", "X", "dY")}
    A64 = inp["A"].astype(np.float64)
    rows = np.unique(np.concatenate([np.arange(32), synth.rng(98).integers(0, 4096, 96), [4095]]))
    dW_rows = orc.grad_weight(v["dY"][:, rows], v["X"])
    mask = orc.ste_mask(v["Z"][rows], orc.MASK_LATENT)
    want = np.where(mask, orc.grad_codes(dW_rows, A64, d) * orc.dge_slope(v["Z"][rows], 5.0, 3.0), 0.0)
    assert_close(to_host(dZ[rows]), want, TOL["bf16"], 'dZ')
    assert np.all(to_host(dZ[rows])[~mask] == 0.0)
    codes = orc.quantize(v["Z"])
    dA_ref, db_ref = orc.grad_map(orc.grad_weight(v["dY"], v["X"]), codes, d)
    assert_close(to_host(dA), dA_ref, TOL["bf16"], 'dA')
    assert_close(to_host(db), db_ref, TOL["bf16"], 'db')

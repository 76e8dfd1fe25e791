"""The training pair (lcvq_linear_fwd_train / lcvq_linear_bwd_train) through the
C ABI: the forward saves the codes in the input-gradient operand layout, both
straight-through masks and X' in the weight-gradient operand layout, and the
backward reads them instead of rebuilding them from Z and X.  The kernels are
the same and so are the values they see, so Y, the packed codes, dX and dZ
must equal those of the plain calls bit for bit (dA and db too: they are
per-block partial sums added in a fixed order), and everything meets the
oracle's bar."""
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


def _bits(t):
    import torch
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32)


def _pair(lc, Z, A, b, X, dY, d, saved=None, dge=None, mask_mode=0, q=(1.0, 0.0), dz_dtype=None, accumulate=False,
          grads=None):
    import torch
    m, n = Z.shape
    packed = torch.empty((m, n // 4), dtype=torch.uint8, device="cuda")
    Y = lc.linear_fwd(Z, A, b, X, d, packed_out=packed, q_scale=q[0], q_shift=q[1], saved=saved)
    kw = dict(mask_mode=mask_mode, q_scale=q[0], q_shift=q[1], dz_dtype=dz_dtype, saved=saved, accumulate=accumulate)
    if grads is not None:
        kw.update(dX=grads[0], dZ=grads[1], dA=grads[2], db=grads[3])
    if dge is None:
        dX, dZ, dA, db = lc.linear_bwd(Z, A, b, X, dY, d, **kw)
    else:
        dX, dZ, dA, db = lc.linear_bwd_dge(Z, A, b, X, dY, d, k=dge[0], cap=dge[1], **kw)
    torch.cuda.synchronize()
    return dict(Y=Y, packed=packed, dX=dX, dZ=dZ, dA=dA, db=db)


SHAPES = [(300, 320, 512, 8), (1000, 264, 328, 8), (513, 520, 1096, 4), (77, 24, 64, 4), (1, 8, 8, 8), (256, 256, 256, 8)]


@pytest.mark.parametrize("N,m,n,d", SHAPES)
@pytest.mark.parametrize("variant", ["ste_rounded", "ste_latent", "dge", "xavier"])
def test_training_pair_matches_plain_calls_and_oracle(lc, N, m, n, d, variant):
    import torch
    k = N + m + n + d
    inp = synth.layer_inputs(N, m, n, d, "bf16", k=k, z_lo=-2.0, z_hi=5.0)
    q = (1.0, 0.0)
    if variant == "xavier":
        q = lc.xavier_quantizer(m, n)
        sp, t = orc.xavier_params(m, n)
        inp["Z"] = synth.bf16_bits((sp * (synth.rng(k).uniform(-2.0, 5.0, (m, n)) - t)).astype(np.float32))
    Z, X, dY = to_dev(inp["Z"], "bf16"), to_dev(inp["X"], "bf16"), to_dev(inp["dY"], "bf16")
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    mask_mode = 1 if variant in ("ste_latent", "dge") else 0
    dge = (5.0, 3.0) if variant == "dge" else None
    saved = lc.new_saved(N, m, n, d, torch.bfloat16, "cuda")
    saved.fill_(0xA5)                                      # no stale zeros to hide a missing write
    plain = _pair(lc, Z, A, b, X, dY, d, dge=dge, mask_mode=mask_mode, q=q)
    train = _pair(lc, Z, A, b, X, dY, d, saved=saved, dge=dge, mask_mode=mask_mode, q=q)
    for key in ("Y", "packed", "dX", "dZ", "dA", "db"):
        assert torch.equal(_bits(train[key]) if key != "packed" else train[key],
                           _bits(plain[key]) if key != "packed" else plain[key]), key
    v = {key: orc.widen(inp[key], "bf16") for key in ("Z", "X", "dY")}
    A64, b64 = inp["A"].astype(np.float64), inp["b"].astype(np.float64)
    qs, qb = np.float32(q[0]), np.float32(q[1])
    Yref, codes = orc.linear_forward(v["Z"], A64, b64, v["X"], d, qs, qb)
    ref = orc.linear_backward(v["Z"], A64, b64, v["X"], v["dY"], d, mask_mode, dge=dge, scale=qs, shift=qb)
    assert np.array_equal(train["packed"].cpu().numpy(), orc.pack2bit(codes))
    assert_close(to_host(train["Y"]), Yref, TOL["bf16"], "Y")
    for key in ("dX", "dZ", "dA", "db"):
        assert_close(to_host(train[key]), ref[key], TOL["bf16"], key)


def test_training_pair_accumulates(lc):
    """accumulate=1 through the saved state: two backward calls give twice the gradients."""
    import torch
    N, m, n, d = 200, 136, 264, 8
    inp = synth.layer_inputs(N, m, n, d, "bf16", k=9, z_lo=-2.0, z_hi=5.0)
    Z, X, dY = to_dev(inp["Z"], "bf16"), to_dev(inp["X"], "bf16"), to_dev(inp["dY"], "bf16")
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    saved = lc.new_saved(N, m, n, d, torch.bfloat16, "cuda")
    one = _pair(lc, Z, A, b, X, dY, d, saved=saved, dz_dtype=torch.float32)
    grads = (one["dX"].clone(), one["dZ"].clone(), one["dA"].clone(), one["db"].clone())
    lc.linear_bwd(Z, A, b, X, dY, d, accumulate=True, dX=grads[0], dZ=grads[1], dA=grads[2], db=grads[3], saved=saved)
    torch.cuda.synchronize()
    for i, key in ((1, "dZ"), (2, "dA"), (3, "db")):
        assert rel_fro(to_host(grads[i]), 2 * to_host(one[key])) <= 1e-6, key


def test_training_pair_fp32_needs_no_saved_state(lc):
    import torch
    N, m, n, d = 37, 72, 200, 4
    assert lc.saved_bytes(N, m, n, d, torch.float32) == 0
    inp = synth.layer_inputs(N, m, n, d, "f32", k=3, z_lo=-2.0, z_hi=5.0)
    Z, X, dY = to_dev(inp["Z"], "f32"), to_dev(inp["X"], "f32"), to_dev(inp["dY"], "f32")
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    saved = lc.new_saved(N, m, n, d, torch.float32, "cuda")
    plain = _pair(lc, Z, A, b, X, dY, d)
    train = _pair(lc, Z, A, b, X, dY, d, saved=saved)
    for key in ("Y", "packed", "dX", "dZ"):
        assert torch.equal(train[key], plain[key]), key


def test_training_pair_full_size(lc):
    """The 4096 x 4096 layer with 4096 tokens, as the benchmark times it: the pair
    against the plain calls, bit for bit."""
    import torch
    N = m = n = 4096
    d = 8
    g = torch.Generator(device="cuda").manual_seed(11)
    Z = torch.empty((m, n), device="cuda").uniform_(-2.0, 5.0, generator=g).to(torch.bfloat16)
    X = torch.randn((N, n), device="cuda", generator=g).to(torch.bfloat16)
    dY = torch.randn((N, m), device="cuda", generator=g).to(torch.bfloat16)
    A, b = (torch.from_numpy(x).cuda() for x in synth.draw_map(d, 0))
    saved = lc.new_saved(N, m, n, d, torch.bfloat16, "cuda")
    plain = _pair(lc, Z, A, b, X, dY, d)
    train = _pair(lc, Z, A, b, X, dY, d, saved=saved)
    for key in ("Y", "packed", "dX", "dZ", "dA", "db"):
        assert torch.equal(_bits(train[key]) if key != "packed" else train[key],
                           _bits(plain[key]) if key != "packed" else plain[key]), key

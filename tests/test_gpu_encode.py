"""Parity of LC encode (lcvq_encode) with the oracle, through the C ABI: codes
and packed words bit-exact (the oracle takes the codes' fp32 decisions in the
kernel's operation order, and is itself pinned to brute-force nearest-codeword
search)."""
import numpy as np
import pytest

import oracle as orc
import synth
from helpers import to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lc():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_10531_amd as lc
    lc._lib.load()
    return lc


def _maps(d, kind, seed):
    if kind == "init":          # eq. init_ab with a random orthogonal G: nearest codewords
        q, r = np.linalg.qr(synth.rng(seed).standard_normal((d, d)))
        A, b = orc.init_map(q * np.sign(np.diag(r)))
        return A.astype(np.float32), b.astype(np.float32)
    return synth.draw_map(d, seed)  # the training maps: A near 0.02 I


def _weights(m, n, kind, dtype, seed):
    scale = 1.0 if kind == "init" else 0.03
    w = (synth.rng(seed).standard_normal((m, n)) * scale).astype(np.float32)
    return synth.bf16_bits(w) if dtype == "bf16" else w


@pytest.mark.parametrize("kind", ["init", "train"])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("d", [8, 4])
@pytest.mark.parametrize("m,n", [(37, 264), (256, 1024), (1, 8), (130, 96)])
def test_encode(lc, m, n, d, dtype, kind):
    import torch
    A, b = _maps(d, kind, m + d)
    Wh = _weights(m, n, kind, dtype, m + n + d)
    codes, packed = lc.encode(to_dev(Wh, dtype), torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda(), d,
                              codes=True, packed=True)
    torch.cuda.synchronize()
    want = orc.encode(orc.widen(Wh, dtype), A, b, d)
    assert np.array_equal(codes.cpu().numpy(), want)
    assert np.array_equal(packed.cpu().numpy(), orc.pack2bit(want))
    if m * n >= 64:
        assert len(np.unique(want)) == 4


def test_encode_non_finite_weights(lc):
    import torch
    d, m, n = 8, 16, 64
    A, b = _maps(d, "init", 3)
    w = (synth.rng(4).standard_normal((m, n))).astype(np.float32)
    w.reshape(-1)[::7] = np.nan
    w.reshape(-1)[3::11] = np.inf
    w.reshape(-1)[5::13] = -np.inf
    codes, _ = lc.encode(to_dev(w, "f32"), torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda(), d)
    torch.cuda.synchronize()
    assert np.array_equal(codes.cpu().numpy(), orc.encode(w.astype(np.float64), A, b, d))


@pytest.mark.parametrize("d", [8, 4])
def test_encode_of_decoded_codewords_round_trips(lc, d):
    """codes -> codewords (lcvq_dequant, fp32) -> lcvq_encode gives the codes back."""
    import torch
    A, b = _maps(d, "init", 9 + d)
    m, n = 96, 512
    C = synth.rng(10 + d).integers(0, 4, size=(m, n), dtype=np.uint8)
    Ad, bd = torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda()
    W = lc.dequant(torch.from_numpy(C).cuda(), Ad, bd, d, out_dtype=torch.float32)
    codes, packed = lc.encode(W, Ad, bd, d, codes=True, packed=True)
    torch.cuda.synchronize()
    assert np.array_equal(codes.cpu().numpy(), C)
    assert np.array_equal(packed.cpu().numpy(), orc.pack2bit(C))


def test_encode_full_size_sampled(lc):
    """28672 x 8192 bf16 weight in the benchmark's launch configuration: sampled rows."""
    import torch
    d, m, n = 8, 28672, 8192
    A, b = _maps(d, "init", 5)
    Wh = _weights(m, n, "init", "bf16", 6)
    _, packed = lc.encode(to_dev(Wh, "bf16"), torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda(), d,
                          codes=False, packed=True)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(16), synth.rng(7).integers(0, m, 48), [m - 1]]))
    want = orc.encode(orc.widen(Wh[rows], "bf16"), A, b, d)
    assert np.array_equal(packed.cpu().numpy()[rows], orc.pack2bit(want))

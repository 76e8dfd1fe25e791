"""Parity of LC encode (lcvq_encode) with the oracle, through the C ABI.

The oracle is the definition: codes = clip(round(v), 0, 3) with v = A^-1 (w - b)
in fp64 (eq. lc_codebook solved for the code vector; the nearest codeword of
eq. vq_assign when A = s G with G orthogonal).  The kernel evaluates v in fp32,
so the two may differ only where the exact v lies within the kernel's fp32
error bound of a decision boundary (0.5, 1.5 or 2.5).  Every other code must be
bit-exact, and the packed words must equal the packed form of the kernel's own
byte codes.  Scaled orthogonal maps are also checked against brute-force
nearest-codeword search."""
import numpy as np
import pytest

import oracle as orc
import synth
from helpers import to_dev

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24                     # unit roundoff of fp32
BOUNDARIES = np.array([0.5, 1.5, 2.5])  # where clip(round(v), 0, 3) changes value


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


def fp32_band(W, A, b, d):
    """Per element, a bound on |v_fp32 - v| for the kernel's fp32 evaluation of
    v = A^-1 (w - b): one rounding of w - b, an fp32 inverse whose error is
    taken as 4 d kappa u ||A^-1|| (kappa the infinity-norm condition number),
    and a d-term fma chain.  Summed and doubled for safety:
        2 u (4 d kappa + d + 1) ||A^-1||_inf sum_j |w_j - b_j|."""
    A64 = np.asarray(A, np.float64)
    Ainv = np.linalg.inv(A64)
    ninv = np.abs(Ainv).sum(axis=1).max()
    kappa = np.abs(A64).sum(axis=1).max() * ninv
    m, n = W.shape
    with np.errstate(invalid="ignore"):
        T = np.abs(W.reshape(m, n // d, d) - np.asarray(b, np.float64)).sum(axis=-1, keepdims=True)
    # a group with a non-finite weight has an infinite or NaN v: no rounding
    # band, its codes must match exactly
    band = 2.0 * U32 * (4 * d * kappa + d + 1) * ninv * np.where(np.isfinite(T), T, 0.0)
    return np.broadcast_to(band, (m, n // d, d)).reshape(m, n)


def check_codes(got, W, A, b, d):
    """Bit-exact outside the band around the decision boundaries; returns
    (elements in the band, disagreements)."""
    V = orc.encode_values(W, A, b, d)
    want = orc.quantize(V)
    with np.errstate(invalid="ignore"):
        dist = np.abs(V[..., None] - BOUNDARIES).min(axis=-1)
        in_band = dist <= fp32_band(W, A, b, d)
    diff = got != want
    assert not np.any(diff & ~in_band), (
        f"{int((diff & ~in_band).sum())} codes differ outside the fp32 band; first at "
        f"{np.argwhere(diff & ~in_band)[0].tolist()}")
    assert in_band.mean() < 1e-2, f"band too wide to be a test: {in_band.mean():.3%} of the elements"
    return int(in_band.sum()), int(diff.sum())


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
    got = codes.cpu().numpy()
    check_codes(got, orc.widen(Wh, dtype), A, b, d)
    assert np.array_equal(packed.cpu().numpy(), orc.pack2bit(got))
    if m * n >= 64:
        assert len(np.unique(got)) == 4


@pytest.mark.parametrize("d", [4, 8])
def test_encode_is_the_nearest_codeword_for_scaled_orthogonal_maps(lc, d):
    """Brute force over all 4^d codewords (eq. vq_assign) in fp64: wherever the best
    codeword is clearly nearer than the second best, the kernel must return it."""
    import torch
    A, b = _maps(d, "init", 40 + d)
    groups = 2048 if d == 4 else 192
    W = (synth.rng(41 + d).standard_normal((1, groups * d)) * 1.3).astype(np.float32)
    codes, _ = lc.encode(to_dev(W, "f32"), torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda(), d)
    torch.cuda.synchronize()
    got = codes.cpu().numpy().reshape(groups, d)
    Zall = np.array(np.meshgrid(*[np.arange(4)] * d, indexing="ij")).reshape(d, -1).T
    book = Zall @ A.astype(np.float64).T + b.astype(np.float64)       # codewords A z + b
    w = W.astype(np.float64).reshape(groups, d)
    dist = (w ** 2).sum(1)[:, None] - 2 * w @ book.T + (book ** 2).sum(1)[None, :]
    order = np.argsort(dist, axis=1)[:, :2]
    best = Zall[order[:, 0]]
    margin = dist[np.arange(groups), order[:, 1]] - dist[np.arange(groups), order[:, 0]]
    clear = margin > 1e-4
    assert clear.mean() > 0.98
    assert np.array_equal(got[clear], best[clear])


def test_encode_non_finite_weights(lc):
    """Non-finite weights follow the written sum v_k = sum_j Ainv[k, j] (w_j - b_j)
    in IEEE arithmetic (inf -> code 3, -inf and NaN -> 0)."""
    import torch
    d, m, n = 8, 16, 64
    A, b = _maps(d, "init", 3)
    w = (synth.rng(4).standard_normal((m, n))).astype(np.float32)
    w.reshape(-1)[::7] = np.nan
    w.reshape(-1)[3::11] = np.inf
    w.reshape(-1)[5::13] = -np.inf
    codes, _ = lc.encode(to_dev(w, "f32"), torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda(), d)
    torch.cuda.synchronize()
    check_codes(codes.cpu().numpy(), w.astype(np.float64), A, b, d)


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


def test_encode_singular_map_gives_code_zero(lc):
    """A map with a zero pivot has no inverse; the kernel's v is NaN there, i.e. code 0."""
    import torch
    d, m, n = 8, 8, 64
    w = synth.rng(12).standard_normal((m, n)).astype(np.float32)
    for A in (np.zeros((d, d), np.float32), np.diag([1, 1, 1, 0, 1, 1, 1, 1]).astype(np.float32)):
        codes, _ = lc.encode(to_dev(w, "f32"), torch.from_numpy(A).cuda(), torch.zeros(d, device="cuda"), d)
        torch.cuda.synchronize()
        assert not codes.cpu().numpy().any()


def test_encode_full_size_sampled(lc):
    """28672 x 8192 bf16 weight in the benchmark's launch configuration: sampled rows."""
    import torch
    d, m, n = 8, 28672, 8192
    A, b = _maps(d, "init", 5)
    Wh = _weights(m, n, "init", "bf16", 6)
    codes, packed = lc.encode(to_dev(Wh, "bf16"), torch.from_numpy(A).cuda(), torch.from_numpy(b).cuda(), d,
                              codes=True, packed=True)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(16), synth.rng(7).integers(0, m, 48), [m - 1]]))
    got = codes.cpu().numpy()[rows]
    check_codes(got, orc.widen(Wh[rows], "bf16"), A, b, d)
    assert np.array_equal(packed.cpu().numpy()[rows], orc.pack2bit(got))

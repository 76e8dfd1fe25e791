"""Pins of the fp64 oracle against what the paper and mathematics fix (CPU only).

Each oracle function is checked against something other than itself: brute
force, closed forms, finite differences of the forward definition, hand-worked
integer examples, and the initial-codebook levels of eq. init_ab."""
import os

import numpy as np
import pytest

import oracle as orc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _all_bf16_values():
    bits = np.arange(1 << 16, dtype=np.uint32)
    return (bits << 16).view(np.float32).astype(np.float64)


def _nearest_code_bruteforce(z):
    """Nearest of {0,1,2,3}; on an exact tie the even code.  Independent of rint/clip."""
    out = np.empty(z.shape, dtype=np.int64)
    for i, v in enumerate(z):
        if np.isnan(v):
            out[i] = 0
            continue
        best, bestd = None, None
        for c in range(4):
            dist = abs(v - c)
            if bestd is None or dist < bestd or (dist == bestd and c % 2 == 0):
                best, bestd = c, dist
        out[i] = best
    return out


# ------------------------------------------------------------- widening -----

def test_widen_bf16_known_bits():
    bits = np.array([0x0000, 0x3F80, 0x4000, 0x4040, 0xBF00, 0x7F80, 0xFF80, 0x3F00], np.uint16)
    v = orc.widen(bits, "bf16")
    assert list(v) == [0.0, 1.0, 2.0, 3.0, -0.5, np.inf, -np.inf, 0.5]


# ------------------------------------------------------------ quantiser -----

def test_quantize_hand_cases():
    z = np.array([-0.7, 0.5, 1.5, 3.6, 2.5, 3.5, -0.5, 3.2, 0.49, 0.51, 1e30, -1e30,
                  np.inf, -np.inf, np.nan, -0.0, 2.4999, 1.0])
    assert orc.quantize(z).tolist() == [0, 0, 2, 3, 2, 3, 0, 3, 0, 1, 3, 0, 3, 0, 0, 0, 2, 1]


def test_quantize_exhaustive_bf16_is_nearest_code_ties_even():
    z = _all_bf16_values()
    got = orc.quantize(z).astype(np.int64)
    assert got.min() >= 0 and got.max() <= 3
    # brute force only where it matters (|z| <= 8); outside, the answer is 0 or 3
    sel = np.abs(np.nan_to_num(z, nan=0.0)) <= 8.0
    assert np.array_equal(got[sel], _nearest_code_bruteforce(z[sel]))
    far = ~sel & ~np.isnan(z)
    assert np.all(got[far & (z > 0)] == 3) and np.all(got[far & (z < 0)] == 0)
    assert np.all(got[np.isnan(z)] == 0)


def test_quantize_fp32_around_every_half_point():
    pts = []
    for h in [-1.5, -0.5, 0.5, 1.5, 2.5, 3.5, 4.5]:
        x = np.float32(h)
        lo, hi = x, x
        for _ in range(64):
            lo = np.nextafter(lo, np.float32(-np.inf))
            hi = np.nextafter(hi, np.float32(np.inf))
            pts += [lo, hi]
        pts.append(x)
    z = np.array(pts, dtype=np.float32).astype(np.float64)
    z = np.concatenate([z, np.random.default_rng(7).uniform(-2, 5, 20000).astype(np.float32)])
    assert np.array_equal(orc.quantize(z).astype(np.int64), _nearest_code_bruteforce(z))


def test_mask_closed_forms_exhaustive_bf16():
    z = _all_bf16_values()
    fin = ~np.isnan(z)
    rounded = orc.ste_mask(z, orc.MASK_ROUNDED)
    latent = orc.ste_mask(z, orc.MASK_LATENT)
    # round-half-even keeps -0.5 (-> -0) inside and pushes 3.5 (-> 4) outside
    assert np.array_equal(rounded[fin], (z[fin] >= -0.5) & (z[fin] < 3.5))
    assert np.array_equal(latent[fin], (z[fin] >= 0.0) & (z[fin] <= 3.0))
    assert not rounded[~fin].any() and not latent[~fin].any()
    hand = orc.ste_mask(np.array([-0.7, 0.5, 1.5, 3.6, 3.2, -0.5, 3.5]), orc.MASK_ROUNDED)
    assert hand.tolist() == [False, True, True, False, True, True, False]
    assert orc.ste_mask(np.array([3.2]), orc.MASK_LATENT).tolist() == [False]


# --------------------------------------------------------------- decode -----

UT4 = np.triu(np.ones((4, 4)))            # A[j, k] = 1 for k >= j (not symmetric)


def test_decode_hand_example():
    # row codes (0,1,2,3 | 3,2,1,0), A upper-triangular ones, b = (1,2,3,4):
    # component j of group g = sum_{k >= j} z_k + b_j
    codes = np.array([[0, 1, 2, 3, 3, 2, 1, 0]])
    W = orc.decode(codes, UT4, np.array([1.0, 2, 3, 4]), 4)
    assert W.tolist() == [[7, 8, 8, 7, 7, 5, 4, 4]]


@pytest.mark.parametrize("d", [4, 8])
def test_decode_identity_map_reproduces_codes(d):
    codes = np.random.default_rng(d).integers(0, 4, size=(5, 4 * d))
    W = orc.decode(codes, np.eye(d), np.zeros(d), d)
    assert np.array_equal(W, codes.astype(np.float64))


@pytest.mark.parametrize("d", [4, 8])
def test_decode_zero_codes_give_offset(d):
    b = np.arange(1.0, d + 1)
    W = orc.decode(np.zeros((3, 2 * d), np.uint8), np.random.default_rng(1).standard_normal((d, d)), b, d)
    assert np.array_equal(W, np.tile(b, (3, 2)))


def test_init_levels_golden():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "init_ab_levels.txt")) if l.strip() and l[0] != "#"]
    levels = np.array([float(r[1]) for r in rows])
    A, b = orc.init_map(np.eye(4))
    W = orc.decode(np.array([[0, 1, 2, 3], [3, 3, 3, 3]]), A, b, 4)
    assert np.allclose(W[0], levels, rtol=0, atol=1e-15)
    assert np.allclose(W[1], levels[3], rtol=0, atol=1e-15)


@pytest.mark.parametrize("d", [4, 8])
def test_init_codebook_zero_mean_identity_covariance(d):
    # over all 4^d code vectors, z has mean mu*1 and covariance (5/4) I, so
    # A z + B with eq. init_ab has mean 0 and covariance s^2 (5/4) G G^T = I exactly
    G, _ = np.linalg.qr(np.random.default_rng(11 + d).standard_normal((d, d)))
    A, b = orc.init_map(G)
    grid = np.stack(np.meshgrid(*[np.arange(4)] * d, indexing="ij"), -1).reshape(-1, d)
    W = orc.decode(grid.reshape(1, -1), A, b, d).reshape(-1, d)
    assert np.allclose(W.mean(0), 0, atol=1e-12)
    assert np.allclose(np.cov(W.T, bias=True), np.eye(d), atol=1e-12)


# -------------------------------------------------------------- forward -----

def test_forward_hand_example():
    X = np.array([[1.0, 0, 2, -1, 0, 0, 0, 1]])
    codes = np.array([[0, 1, 2, 3, 3, 2, 1, 0]])
    W = orc.decode(codes, UT4, np.array([1.0, 2, 3, 4]), 4)
    # 1*7 + 2*8 - 1*7 + 1*4
    assert orc.forward(X, W).tolist() == [[20.0]]
    assert orc.forward_reformulated(X, codes, UT4, np.array([1.0, 2, 3, 4]), 4).tolist() == [[20.0]]


@pytest.mark.parametrize("d", [4, 8])
def test_forward_equals_reformulated(d):
    r = np.random.default_rng(3 + d)
    N, m, n = 7, 9, 6 * d
    X = r.standard_normal((N, n))
    codes = r.integers(0, 4, size=(m, n))
    A, b = r.standard_normal((d, d)), r.standard_normal(d)
    Y1 = orc.forward(X, orc.decode(codes, A, b, d))
    Y2 = orc.forward_reformulated(X, codes, A, b, d)
    assert np.allclose(Y1, Y2, rtol=1e-12, atol=1e-12)


def test_forward_zero_codes_closed_form():
    r = np.random.default_rng(5)
    d, N, m, n = 8, 4, 3, 32
    X, A, b = r.standard_normal((N, n)), r.standard_normal((d, d)), r.standard_normal(d)
    Y = orc.forward(X, orc.decode(np.zeros((m, n), np.uint8), A, b, d))
    per_token = sum(X[:, c] * b[c % d] for c in range(n))
    assert np.allclose(Y, per_token[:, None] * np.ones((1, m)), rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------- backward -----

def test_backward_hand_example():
    # N = m = 1, dY = 1: dW = X, dX = W_hat row, dA = sum_g outer(X_g, z_g), db = sum_g X_g,
    # dcode[g*d+k] = sum_{j<=k} X[g*d+j] (A upper-triangular ones)
    X = np.array([[1.0, 0, 2, -1, 0, 0, 0, 1]])
    Z = np.array([[0.1, 1.2, 1.9, 3.3, 2.6, 2.2, 0.8, -0.3]])        # codes 0,1,2,3,3,2,1,0
    out = orc.linear_backward(Z, UT4, np.array([1.0, 2, 3, 4]), X, np.array([[1.0]]), 4)
    assert out["dX"].tolist() == [[7, 8, 8, 7, 7, 5, 4, 4]]
    assert out["dA"].tolist() == [[0, 1, 2, 3], [0, 0, 0, 0], [0, 2, 4, 6], [3, 1, -1, -3]]
    assert out["db"].tolist() == [1, 0, 2, 0]
    assert out["dZ"].tolist() == [[1, 1, 3, 2, 0, 0, 0, 1]]


def _fd(f, x, idx, h):
    xp, xm = x.copy(), x.copy()
    xp[idx] += h
    xm[idx] -= h
    return (f(xp) - f(xm)) / (2 * h)


@pytest.mark.parametrize("d", [4, 8])
def test_backward_matches_finite_differences(d):
    # L = <dY, Y> is linear in X, A, b and W_hat (codes fixed), so central
    # differences are exact up to fp64 rounding.
    r = np.random.default_rng(20 + d)
    N, m, n = 3, 4, 2 * d
    X, dY = r.standard_normal((N, n)), r.standard_normal((N, m))
    Z = r.uniform(-1.0, 4.0, size=(m, n))
    A, b = r.standard_normal((d, d)), r.standard_normal(d)
    codes = orc.quantize(Z)
    out = orc.linear_backward(Z, A, b, X, dY, d)

    def loss(X_=X, A_=A, b_=b):
        return float(np.sum(dY * orc.forward(X_, orc.decode(codes, A_, b_, d))))

    for idx in np.ndindex(X.shape):
        assert np.isclose(_fd(lambda v: loss(X_=v), X, idx, 0.5), out["dX"][idx], rtol=1e-9, atol=1e-9)
    for idx in np.ndindex(A.shape):
        assert np.isclose(_fd(lambda v: loss(A_=v), A, idx, 0.5), out["dA"][idx], rtol=1e-9, atol=1e-9)
    for j in range(d):
        assert np.isclose(_fd(lambda v: loss(b_=v), b, (j,), 0.5), out["db"][j], rtol=1e-9, atol=1e-9)
    W = orc.decode(codes, A, b, d)
    for idx in np.ndindex(W.shape):
        g = _fd(lambda v: float(np.sum(dY * orc.forward(X, v))), W, idx, 0.5)
        assert np.isclose(g, out["dW"][idx], rtol=1e-9, atol=1e-9)
    # straight-through: d/dcode with codes relaxed to reals, masked by the clip range
    Cf = codes.astype(np.float64)
    dcode = np.zeros_like(Cf)
    for idx in np.ndindex(Cf.shape):
        dcode[idx] = _fd(lambda v: float(np.sum(dY * orc.forward(X, orc.decode(v, A, b, d)))), Cf, idx, 0.5)
    mask = orc.ste_mask(Z)
    assert np.allclose(out["dZ"][mask], dcode[mask], rtol=1e-9, atol=1e-9)
    assert np.all(out["dZ"][~mask] == 0.0)
    assert (~mask).any() and mask.any()


@pytest.mark.parametrize("d", [4, 8])
def test_grad_latent_identity_map_is_weight_grad(d):
    r = np.random.default_rng(40 + d)
    N, m, n = 5, 6, 3 * d
    X, dY = r.standard_normal((N, n)), r.standard_normal((N, m))
    Z = r.uniform(0.0, 3.0, size=(m, n))        # every latent inside the clip range
    out = orc.linear_backward(Z, np.eye(d), np.zeros(d), X, dY, d)
    assert np.allclose(out["dZ"], dY.T @ X, rtol=1e-12, atol=1e-12)


def test_mask_latent_mode_in_backward():
    r = np.random.default_rng(9)
    d, N, m, n = 4, 2, 3, 8
    Z = np.array([[3.2, 0.2, 1.0, 2.0, -0.3, 1.1, 2.2, 3.0]] * m)
    out_r = orc.linear_backward(Z, np.eye(d), np.zeros(d), r.standard_normal((N, n)),
                                r.standard_normal((N, m)), d, orc.MASK_ROUNDED)
    out_l = orc.linear_backward(Z, np.eye(d), np.zeros(d), r.standard_normal((N, n)),
                                r.standard_normal((N, m)), d, orc.MASK_LATENT)
    assert np.all(out_r["dZ"][:, [0, 4]] != 0)          # 3.2 and -0.3 round inside [0, 3]
    assert np.all(out_l["dZ"][:, [0, 4]] == 0)          # but lie outside it


# ------------------------------------ differentiable gradient estimator -----

def test_dge_surrogate_hand_values():
    # eq. dge with delta = 1, k = 5: f(1/4) = (1 - 2^-1/5) / 2, f(3/4) = (1 + 2^-1/5) / 2
    F = orc.dge_surrogate(np.array([0.0, 0.25, 0.5, 0.75, 1.0, 2.25, -0.75]), 5.0)
    t = 2.0 ** -0.2
    want = [0.0, (1 - t) / 2, 0.5, (1 + t) / 2, 1.0, 2 + (1 - t) / 2, -1 + (1 - t) / 2]
    assert np.allclose(F, want, rtol=0, atol=1e-15)


def test_dge_surrogate_limits():
    z = np.random.default_rng(3).uniform(-2.0, 5.0, 1000)
    assert np.allclose(orc.dge_surrogate(z, 1.0), z, rtol=0, atol=1e-12)        # k = 1: identity
    far = np.abs(z - np.floor(z) - 0.5) > 0.05                                  # k -> inf: round()
    assert np.allclose(orc.dge_surrogate(z[far], 1e6), np.rint(z[far]), rtol=0, atol=1e-4)
    ints = np.arange(-3.0, 6.0)
    assert np.array_equal(orc.dge_surrogate(ints, 5.0), ints)                    # fixed at integers
    assert np.array_equal(orc.dge_surrogate(ints + 0.5, 5.0), ints + 0.5)        # and at the steps


def test_dge_slope_hand_values():
    s = orc.dge_slope(np.array([0.0, 0.25, 0.5, 0.75, 1.0, 3.25, -0.75]), 5.0, 3.0)
    q = 0.2 * 2.0 ** 0.8                    # (1/5) |2/4 - 1|^(1/5 - 1)
    assert np.allclose(s, [0.2, q, 3.0, q, 0.2, q, q], rtol=1e-15, atol=0)
    assert np.array_equal(orc.dge_slope(np.array([0.5, 1.5, -2.5]), 5.0, 7.25), [7.25] * 3)
    # k = 1: slope 1 everywhere, the middle of the interval included
    assert np.array_equal(orc.dge_slope(np.array([0.0, 0.3, 0.5, 2.9]), 1.0, 3.0), [1.0] * 4)


def test_dge_slope_is_derivative_of_surrogate():
    r = np.random.default_rng(11)
    z = r.uniform(-2.0, 5.0, 4000)
    z = z[np.abs(z - np.floor(z) - 0.5) > 0.02]
    for k in (2.0, 5.0, 9.0):
        h = 1e-6
        fd = (orc.dge_surrogate(z + h, k) - orc.dge_surrogate(z - h, k)) / (2 * h)
        assert np.allclose(orc.dge_slope(z, k, 1e30), fd, rtol=1e-6, atol=0)


@pytest.mark.parametrize("k,cap", [(5.0, 3.0), (5.0, 10.0), (3.0, 2.0)])
def test_dge_capped_slope_mean_closed_form(k, cap):
    # With w = |2x - 1| uniform on [0, 1] for x uniform, the slope is (1/k) w^(1/k-1),
    # whose integral is w^(1/k); it exceeds the cap below w_c = (k cap)^(1/(1/k-1)).
    # Mean of the capped slope = cap w_c + 1 - w_c^(1/k).  The uncapped mean is 1.
    wc = (k * cap) ** (1.0 / (1.0 / k - 1.0))
    want = cap * wc + 1.0 - wc ** (1.0 / k)
    n = 2_000_000
    x = (np.arange(n) + 0.5) / n                    # midpoint rule over one interval
    got = orc.dge_slope(x, k, cap).mean()
    assert abs(got - want) < 2e-6
    assert want < 1.0


@pytest.mark.parametrize("d", [4, 8])
def test_dge_backward_matches_finite_differences_of_surrogate(d):
    # Through the surrogate F of eq. dge the loss L(Z) = <dY, X decode(clip(F(Z), 0, 3))^T>
    # is differentiable wherever F is (off the half-integers) and clip is (off 0 and 3):
    # there dL/dZ is the estimator's dZ with the latent mask and an inactive cap.
    r = np.random.default_rng(50 + d)
    N, m, n = 3, 4, 2 * d
    X, dY = r.standard_normal((N, n)), r.standard_normal((N, m))
    A, b = r.standard_normal((d, d)), r.standard_normal(d)
    frac = r.uniform(0.05, 0.45, size=(m, n)) + 0.5 * r.integers(0, 2, size=(m, n))
    Z = r.integers(-2, 5, size=(m, n)) + frac      # latents in (-2, 5), clear of the kinks
    k = 5.0
    out = orc.linear_backward(Z, A, b, X, dY, d, orc.MASK_LATENT, dge=(k, 1e30))

    def loss(Z_):
        c = np.clip(orc.dge_surrogate(Z_, k), 0.0, 3.0)
        return float(np.sum(dY * orc.forward(X, orc.decode(c, A, b, d))))

    g = np.array([_fd(loss, Z, idx, 1e-6) for idx in np.ndindex(Z.shape)]).reshape(Z.shape)
    assert np.allclose(out["dZ"], g, rtol=1e-6, atol=1e-8)
    inside = (Z >= 0) & (Z <= 3)
    assert inside.any() and (~inside).any()
    assert np.all(out["dZ"][~inside] == 0.0)


def test_dge_non_finite_latents_get_no_gradient():
    d = 4
    Z = np.array([[np.nan, np.inf, -np.inf, 1.25]])
    out = orc.linear_backward(Z, np.eye(d), np.zeros(d), np.ones((2, 4)), np.ones((2, 1)), d, orc.MASK_LATENT,
                              dge=(5.0, 3.0))
    assert out["dZ"][0, :3].tolist() == [0.0, 0.0, 0.0]
    assert out["dZ"][0, 3] == 2.0 * 0.2 * 2.0 ** 0.8      # dW = 2, slope at x = 1/4


def test_dge_with_k_one_is_straight_through():
    r = np.random.default_rng(12)
    d, N, m, n = 8, 4, 5, 16
    Z = r.uniform(-2.0, 5.0, (m, n))
    Z[0, :4] = [0.5, 1.5, 2.5, -0.5]                # middles of the rounding intervals
    X, dY = r.standard_normal((N, n)), r.standard_normal((N, m))
    A, b = r.standard_normal((d, d)), r.standard_normal(d)
    for mode in (orc.MASK_ROUNDED, orc.MASK_LATENT):
        ste = orc.linear_backward(Z, A, b, X, dY, d, mode)
        dge = orc.linear_backward(Z, A, b, X, dY, d, mode, dge=(1.0, 3.0))
        assert np.array_equal(ste["dZ"], dge["dZ"])
        for key in ("dX", "dA", "db"):
            assert np.array_equal(ste[key], dge[key])


# ------------------------------------------------- quantiser domain (3.4) ---

def _fma_exact(a, b, c):
    """Correctly rounded binary32 a*b + c by exact rational arithmetic (brute force)."""
    from fractions import Fraction
    v = Fraction(float(a)) * Fraction(float(b)) + Fraction(float(c))
    f = np.float32(float(v))                       # nearest fp64, then fp32: may double-round
    cands = [np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))]
    dist = [abs(Fraction(float(x)) - v) for x in cands]
    best = min(dist)
    ties = [x for x, dd in zip(cands, dist) if dd == best]
    if len(ties) > 1:                              # exact tie: even significand
        ties = [x for x in ties if (np.float32(x).view(np.uint32) & 1) == 0]
    return float(ties[0])


def test_fma_f32_against_exact_rounding():
    r = np.random.default_rng(31)
    a = r.standard_normal(3000).astype(np.float32) * np.float32(0.03)
    b = np.float32(1.0 / 0.018)
    c = np.float32(1.5)
    got = orc.fma_f32(a, b, c)
    want = np.array([_fma_exact(x, b, c) for x in a])
    assert np.array_equal(got, want)
    # Double-rounding cases: with a = +-2^-24 (1 + i 2^-23), b = 1 - i 2^-23 and
    # c = 1 + 2^-23, a b + c = 1 + 3 2^-24 - i^2 2^-70 or 1 + 2^-24 + i^2 2^-70,
    # i.e. i^2 2^-70 off an fp32 midpoint.  Rounding to fp64 first lands on the
    # midpoint, whose tie goes the other way than the correct rounding.
    naive_wrong = 0
    for i in range(1, 40):
        for sgn in (1.0, -1.0):
            for e in (0, -7, 5):                   # same pattern at other exponents
                x = np.float32(sgn * 2.0 ** (-24 + e) * (1.0 + i * 2.0 ** -23))
                y = np.float32(1.0 - i * 2.0 ** -23)
                z = np.float32(2.0 ** e * (1.0 + 2.0 ** -23))
                want = _fma_exact(x, y, z)
                assert orc.fma_f32(x, y, z) == want, (i, sgn, e)
                naive_wrong += float(np.float32(float(x) * float(y) + float(z))) != want
    assert naive_wrong > 0


def test_xavier_params_hand_values():
    sp, t = orc.xavier_params(4096, 4096)
    a = np.sqrt(6.0 / 8192)
    assert t == 1.5 and np.isclose(sp, 2 * a / 3, rtol=1e-15)
    sp2, _ = orc.xavier_params(11008, 4096)
    assert np.isclose(sp2, 2 * np.sqrt(6.0 / 15104) / 3, rtol=1e-15)


@pytest.mark.parametrize("m,n", [(4096, 4096), (11008, 4096), (256, 256), (28672, 8192)])
@pytest.mark.parametrize("store", ["bf16", "f32"])
def test_xavier_init_quantises_back_to_its_codes(m, n, store):
    # eq. xavier_preprocess preserves the codes: quantising W_p / s' + t returns W_z
    codes = np.arange(4, dtype=np.uint8).repeat(64)
    W = orc.xavier_init(codes, m, n).astype(np.float32)
    if store == "bf16":
        import synth
        W = orc.widen(synth.bf16_bits(W), "bf16")
    sp, t = orc.xavier_params(m, n)
    assert np.array_equal(orc.quantize(W, np.float32(1.0 / sp), np.float32(t)), codes)


def test_xavier_init_statistics():
    # over uniform codes: mean exactly 0, range exactly [-a, a] (Xavier's uniform bound)
    m, n = 4096, 11008
    W = orc.xavier_init(np.arange(4), m, n)
    a = np.sqrt(6.0 / (m + n))
    assert abs(W.mean()) < 1e-18
    assert np.isclose(W.max(), a, rtol=1e-15) and np.isclose(W.min(), -a, rtol=1e-15)


def test_quantiser_scale_in_backward_matches_finite_differences():
    # STE through code = W * scale + shift: relaxing round() to the identity, the loss
    # <dY, X decode(W scale + shift)^T> has gradient scale * dL/dcode
    r = np.random.default_rng(41)
    d, N, m, n = 4, 3, 4, 8
    scale, shift = np.float32(8.0), np.float32(1.5)      # exact in fp32
    W = r.uniform(-0.15, 0.15, (m, n))                   # codes inside (0, 3): mask 1
    X, dY = r.standard_normal((N, n)), r.standard_normal((N, m))
    A, b = r.standard_normal((d, d)), r.standard_normal(d)
    out = orc.linear_backward(W, A, b, X, dY, d, orc.MASK_LATENT, scale=scale, shift=shift)

    def loss(W_):
        return float(np.sum(dY * orc.forward(X, orc.decode(W_ * float(scale) + float(shift), A, b, d))))

    g = np.array([_fd(loss, W, idx, 1e-3) for idx in np.ndindex(W.shape)]).reshape(W.shape)
    assert np.allclose(out["dZ"], g, rtol=1e-9, atol=1e-9)
    unit = orc.linear_backward(W * float(scale) + float(shift), A, b, X, dY, d, orc.MASK_LATENT)
    assert np.allclose(out["dZ"], float(scale) * unit["dZ"], rtol=1e-12, atol=0)


# ------------------------------------------------------------ LC encode -----

def _orthogonal(d, seed):
    q, r = np.linalg.qr(np.random.default_rng(seed).standard_normal((d, d)))
    return q * np.sign(np.diag(r))


def test_encode_hand_example_upper_triangular_map():
    # A maps code vector z to A z + b (eq. lc_codebook).  With z = (0.3, 1.7, 2.4, 3.9)
    # the weight w = A z + b is computed by hand below; back substitution gives z
    # again, which rounds and clips to codes (0, 2, 2, 3).  A transposed A, a
    # dropped offset or a flipped one give (1, 1, 3, 2), (1, 1, 2, 3), (2, 0, 2, 3).
    A = np.array([[2, 1, 0, 0], [0, 1, 0, 0], [0, 0, 4, 1], [0, 0, 0, 2]], np.float64)
    b = np.array([0.5, -1.0, 0.0, 0.25])
    w = np.array([[2 * 0.3 + 1.7 + 0.5, 1.7 - 1.0, 4 * 2.4 + 3.9, 2 * 3.9 + 0.25]])
    assert np.allclose(orc.encode_values(w, A, b, 4), [[0.3, 1.7, 2.4, 3.9]], rtol=0, atol=1e-12)
    assert orc.encode(w, A, b, 4).tolist() == [[0, 2, 2, 3]]


@pytest.mark.parametrize("d", [4, 8])
def test_encode_values_invert_the_decode(d):
    # decode(v) = A v + b per group must give the weight back (decode is pinned on its own)
    A, b = (x.astype(np.float64) for x in (0.02 * (np.eye(d) + 0.3 * np.random.default_rng(d).standard_normal((d, d))),
                                           np.random.default_rng(d + 1).standard_normal(d) * 0.01))
    W = np.random.default_rng(d + 2).standard_normal((5, 6 * d)) * 0.05
    assert np.allclose(orc.decode(orc.encode_values(W, A, b, d), A, b, d), W, rtol=0, atol=1e-13)


def test_encode_non_finite_weights_follow_the_written_sum():
    # identity map: the entry itself is 1 * w_k (+inf -> code 3, -inf and NaN -> 0),
    # while the other components of that group meet 0 * inf = NaN -> code 0; a
    # finite group beside it is untouched
    w = np.array([[np.inf, 1.2, 2.0, 0.4, 1.2, -np.inf, 2.6, 0.4, np.nan, 1.2, 2.0, 3.0, 0.7, 1.6, 2.4, 9.0]])
    assert orc.encode(w, np.eye(4), np.zeros(4), 4).tolist() == [[3, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 1, 2, 2, 3]]
    # a dense map spreads one infinite entry over the whole group with the signs of A^-1
    A = np.array([[1.0, 0.5], [-0.25, 1.0]])
    v = orc.encode_values(np.array([[np.inf, 0.0]]), A, np.zeros(2), 2)
    assert np.array_equal(np.sign(v), np.sign(np.linalg.inv(A)[:, 0])[None, :]) and np.isinf(v).all()


@pytest.mark.parametrize("d", [4, 8])
def test_encode_identity_map_is_the_quantiser(d):
    W = np.random.default_rng(60 + d).uniform(-2.0, 5.0, (7, 4 * d)).astype(np.float32)
    assert np.array_equal(orc.encode(W, np.eye(d), np.zeros(d), d), orc.quantize(W))


@pytest.mark.parametrize("d", [4, 8])
def test_encode_returns_the_codes_of_exact_codewords(d):
    # init map of eq. init_ab: A = s G, b = -s G mu 1; every codeword encodes to itself
    A, b = orc.init_map(_orthogonal(d, 70 + d))
    C = np.random.default_rng(71 + d).integers(0, 4, size=(9, 5 * d)).astype(np.uint8)
    W = orc.decode(C, A, b, d).astype(np.float32)
    assert np.array_equal(orc.encode(W, A, b, d), C)


@pytest.mark.parametrize("d", [4, 8])
def test_encode_is_the_nearest_codeword_for_an_orthogonal_map(d):
    # brute force over all 4^d codewords (eq. vq_assign) in fp64
    A, b = orc.init_map(_orthogonal(d, 80 + d))
    A, b = A.astype(np.float32), b.astype(np.float32)
    groups = 400 if d == 4 else 60
    W = (np.random.default_rng(81 + d).standard_normal((groups, d)) * 1.3).astype(np.float32)
    Z = np.array(np.meshgrid(*[np.arange(4)] * d, indexing="ij")).reshape(d, -1).T      # all codewords
    book = Z @ A.astype(np.float64).T + b.astype(np.float64)                            # c = A z + b
    dist = ((W.astype(np.float64)[:, None, :] - book[None]) ** 2).sum(-1)
    order = np.argsort(dist, axis=1)
    best = Z[order[:, 0]]
    margin = dist[np.arange(groups), order[:, 1]] - dist[np.arange(groups), order[:, 0]]
    got = orc.encode(W.reshape(1, -1), A, b, d).reshape(groups, d)
    clear = margin > 1e-9
    assert clear.sum() > 0.99 * groups
    assert np.array_equal(got[clear], best[clear])


# ------------------------------------------------------------- packing ------

def test_pack_hand_values():
    assert orc.pack2bit(np.array([[1, 2, 3, 0]])).tolist() == [[0x39]]
    assert orc.pack2bit(np.array([[3, 3, 3, 3, 0, 0, 0, 0]])).tolist() == [[0xFF, 0x00]]
    for c in range(8):
        row = np.zeros((1, 8), np.uint8)
        row[0, c] = 1
        expect = [0, 0]
        expect[c // 4] = 1 << (2 * (c % 4))
        assert orc.pack2bit(row).tolist() == [expect]


def test_unpack_hand_values():
    assert orc.unpack2bit(np.array([[0x39]], np.uint8), 4).tolist() == [[1, 2, 3, 0]]
    assert orc.unpack2bit(np.array([[0xFF, 0x00, 0x1B]], np.uint8), 12).tolist() == \
        [[3, 3, 3, 3, 0, 0, 0, 0, 3, 2, 1, 0]]


def test_forward_from_packed_codes_is_forward_from_latent():
    r = np.random.default_rng(17)
    for d in (4, 8):
        N, m, n = 5, 7, 64
        Z = r.uniform(-1.0, 4.0, (m, n))
        X, A, b = r.standard_normal((N, n)), r.standard_normal((d, d)), r.standard_normal(d)
        Y, codes = orc.linear_forward(Z, A, b, X, d)
        # brute force: one output at a time from the bytes, no unpack helper
        P = orc.pack2bit(codes)
        Yb = np.zeros((N, m))
        for t in range(N):
            for rr in range(m):
                acc = 0.0
                for c in range(n):
                    code = (int(P[rr, c // 4]) >> (2 * (c % 4))) & 3
                    g, k = divmod(c, d)
                    w = sum(A[k, kk] * ((int(P[rr, (g * d + kk) // 4]) >> (2 * ((g * d + kk) % 4))) & 3)
                            for kk in range(d)) + b[k]
                    acc += X[t, c] * w
                    assert code == codes[rr, c]
                Yb[t, rr] = acc
        assert np.allclose(orc.linear_forward_packed(P, A, b, X, d, n), Yb, rtol=1e-12, atol=1e-12)
        assert np.allclose(Y, Yb, rtol=1e-12, atol=1e-12)


def test_pack_round_trip():
    codes = np.random.default_rng(2).integers(0, 4, size=(7, 64)).astype(np.uint8)
    p = orc.pack2bit(codes)
    assert p.shape == (7, 16)
    unpacked = np.stack([(p >> (2 * i)) & 3 for i in range(4)], axis=-1).reshape(7, 64)
    assert np.array_equal(unpacked, codes)
    assert np.array_equal(orc.unpack2bit(p, 64), codes)


# ------------------------------------------------------------ optimiser -----

def test_adamw_first_step_closed_form():
    theta, g = np.array([1.0, -2.0, 0.5]), np.array([0.3, -4.0, 1e-3])
    t1, m1, m2 = orc.adamw_step(theta, g, 0 * g, 0 * g, 1, lr=1e-2)
    assert np.allclose(t1, theta - 1e-2 * g / (np.abs(g) + 1e-8), rtol=0, atol=1e-15)
    t1w, _, _ = orc.adamw_step(theta, g, 0 * g, 0 * g, 1, lr=1e-2, weight_decay=0.1)
    assert np.allclose(t1w, theta * (1 - 1e-3) - 1e-2 * g / (np.abs(g) + 1e-8), rtol=0, atol=1e-15)


def test_adamw_constant_gradient_steps_are_equal():
    # with a constant gradient the bias-corrected moments equal g and g^2 at every step
    theta, g = np.array([0.0, 0.0]), np.array([2.0, -0.5])
    m1, m2 = 0 * g, 0 * g
    for step in range(1, 6):
        new, m1, m2 = orc.adamw_step(theta, g, m1, m2, step, lr=0.1)
        assert np.allclose(theta - new, 0.1 * g / (np.abs(g) + 1e-8), rtol=1e-12, atol=0)
        theta = new

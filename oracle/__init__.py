"""Plain fp64 CPU oracle of the LC-VQ linear layer (LC-QAT, arXiv 2606.10531).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import it: only the
test suite, the smoke check and the benchmark's CPU-baseline leg use it.  It
shares no code with the HIP library.

Every function computes the plain definition from the paper, in float64, on
inputs widened exactly from their fp32 / bf16 bits.  Library primitives
(numpy's rint, matmul and reshape) serve as single steps; there is no blocking,
fusion or reordering beyond what the definitions state.

Notation (paper -> here): proxy weights W_p -> Z (m x n); integer weights W_z ->
codes (values 0..3, bit-width b = 2); map A (d x d) and offset B -> A, b;
group size d; effective weight W_hat (m x n); activations X (N x n); output
Y (N x m).  Group g of row r covers columns [g*d, (g+1)*d).

Readings of the paper where it is silent or inconsistent:
  * Orientation: Y = X W_hat^T (nn.Linear convention); this is the only one
    that agrees term by term with the reformulated forward of Sec. 3.2.
  * round() is IEEE round-half-to-even; clip bounds are inclusive.
  * Codeword of row r, group g: W_hat[r, g*d + j] = sum_k A[j, k] code[r, g*d + k] + b[j].
  * STE mask: the straight-through estimator (Sec. 3.3) passes the gradient
    through round(); clip() still has its ordinary derivative, so
    mask = [0 <= round(Z) <= 3] ("rounded").  The alternative
    mask = [0 <= Z <= 3] ("latent") is also provided.
  * NaN latents quantise to code 0 with mask 0; +-inf clip to 3 / 0, mask 0.
  * Xavier reparameterisation (eq. xavier_preprocess, Sec. 3.4): with W_p =
    s' (W_z - t), the quantiser acts on W_p / s' + t.  The kernels compute that
    affine value as one fp32 fused multiply-add with fp32 scale 1/s' and shift
    t, and the codes are decided on that fp32 value; the oracle takes the same
    decision (fma_f32 below).  The latent's gradient gains the factor 1/s'.
  * Differentiable gradient estimator (eq. dge, Sec. 3.3): the paper gives f on
    one rounding interval of width delta = 1 (the interval of round() on the
    code-domain latent).  It is extended periodically, F(z) = floor(z) +
    f(z - floor(z)), which is continuous and steps at the half-integers like
    round().  Its slope f' is unbounded at the middle of each interval, so it
    is capped at a caller-given value.  clip() keeps its ordinary derivative;
    through clip(F(Z), 0, 3) that is the "latent" mask [0 <= Z <= 3] (F is
    increasing with F(0) = 0 and F(3) = 3); the "rounded" mask stays available.
"""
from __future__ import annotations

import numpy as np

CODE_MAX = 3            # 2^b - 1 for b = 2 (eq. quant_param, Sec. 3.2)
MASK_ROUNDED = 0
MASK_LATENT = 1


# ---------------------------------------------------------------- inputs ----

def widen(x, dtype: str) -> np.ndarray:
    """Exact fp64 value of a stored tensor: fp32 array, or uint16 bf16 bits."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        bits = np.asarray(x, dtype=np.uint16).astype(np.uint32) << 16
        return bits.view(np.float32).astype(np.float64)
    raise ValueError(dtype)


# -------------------------------------------------- quantiser domain -----

def fma_f32(a, b, c) -> np.ndarray:
    """a * b + c for fp32 values, rounded once to fp32 (binary32 fused multiply-add).

    a * b is exact in fp64 (24 + 24 significant bits).  The sum is split into
    its fp64 rounding s and the exact remainder e (TwoSum), and s is rounded to
    fp32; that is the correctly rounded result unless s lies exactly halfway
    between two fp32 values while e != 0, where e decides the direction."""
    a, b, c = (np.asarray(x, dtype=np.float32).astype(np.float64) for x in (a, b, c))
    p = a * b
    with np.errstate(invalid="ignore", over="ignore"):
        s = p + c
        bv = s - p
        e = (p - (s - bv)) + (c - bv)
        r32 = s.astype(np.float32)
        r = r32.astype(np.float64)
        up = np.nextafter(r32, np.float32(np.inf)).astype(np.float64)
        dn = np.nextafter(r32, np.float32(-np.inf)).astype(np.float64)
        out = np.where((s > r) & (s == (r + up) / 2) & (e > 0), up, r)
        out = np.where((s < r) & (s == (r + dn) / 2) & (e < 0), dn, out)
    return out


def code_domain(W: np.ndarray, scale: float = 1.0, shift: float = 0.0) -> np.ndarray:
    """The value the quantiser rounds: W itself in the code domain (scale 1, shift
    0), else fp32(W * scale + shift) with fp32 scale and shift (Sec. 3.4)."""
    W = np.asarray(W, dtype=np.float64)
    if scale == 1.0 and shift == 0.0:
        return W
    return fma_f32(W, scale, shift)


def xavier_params(m: int, n: int, bits: int = 2):
    """(s', t) of eq. xavier_preprocess: s' = 2a / (2^b - 1), t = (2^b - 1) / 2,
    a = sqrt(6 / (m + n))."""
    a = np.sqrt(6.0 / (m + n))
    return 2.0 * a / (2 ** bits - 1), (2 ** bits - 1) / 2.0


def xavier_init(codes: np.ndarray, m: int, n: int, bits: int = 2) -> np.ndarray:
    """Initial proxy weights W_p = s' (W_z - t) of eq. xavier_preprocess."""
    sp, t = xavier_params(m, n, bits)
    return sp * (np.asarray(codes, dtype=np.float64) - t)


# ------------------------------------------------------------ quantiser -----

def quantize(Z: np.ndarray, scale: float = 1.0, shift: float = 0.0) -> np.ndarray:
    """Integer weights W_z = clip(round(W_p), 0, 2^b - 1)  (eq. quant_param, Sec. 3.2),
    with W_p taken through code_domain (Sec. 3.4) when scale / shift are given.

    Returns uint8 codes in {0, 1, 2, 3}."""
    Z = code_domain(Z, scale, shift)
    u = np.rint(Z)                                  # round half to even
    codes = np.clip(u, 0.0, CODE_MAX)
    codes = np.where(np.isnan(Z), 0.0, codes)
    return codes.astype(np.uint8)


def ste_mask(Z: np.ndarray, mode: int = MASK_ROUNDED, scale: float = 1.0, shift: float = 0.0) -> np.ndarray:
    """Where the straight-through gradient of eq. quant_param is passed (Sec. 3.3).

    rounded: derivative of clip() evaluated at round(Z): 1 iff 0 <= round(Z) <= 3.
    latent : 1 iff 0 <= Z <= 3.
    (Z in the code domain, code_domain(W, scale, shift).)"""
    Z = code_domain(Z, scale, shift)
    if mode == MASK_ROUNDED:
        u = np.rint(Z)
        return (u >= 0.0) & (u <= CODE_MAX)
    if mode == MASK_LATENT:
        return (Z >= 0.0) & (Z <= CODE_MAX)
    raise ValueError(mode)


# ---------------------------------- differentiable gradient estimator ------

def dge_surrogate(Z: np.ndarray, k: float) -> np.ndarray:
    """Smooth stand-in for round() (eq. dge, Sec. 3.3) with delta = 1:
        f(x) = 1/2 (1 + sign(2x - 1) |2x - 1|^(1/k))   on one interval x in [0, 1],
    extended periodically: F(z) = floor(z) + f(z - floor(z))."""
    Z = np.asarray(Z, dtype=np.float64)
    fl = np.floor(Z)
    v = 2.0 * (Z - fl) - 1.0
    return fl + 0.5 * (1.0 + np.sign(v) * np.abs(v) ** (1.0 / k))


def dge_slope(Z: np.ndarray, k: float, cap: float) -> np.ndarray:
    """Slope of the surrogate, f'(x) = (1/k) |2x - 1|^(1/k - 1) at the position x
    of Z within its rounding interval (Sec. 3.3, delta = 1), capped at `cap`
    (f' is unbounded where x = 1/2)."""
    Z = np.asarray(Z, dtype=np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):     # w = 0 at x = 1/2; NaN for non-finite Z
        w = np.abs(2.0 * (Z - np.floor(Z)) - 1.0)
        fp = (1.0 / k) * w ** (1.0 / k - 1.0)
    return np.minimum(fp, cap)


# --------------------------------------------------------------- decode -----

def decode(codes: np.ndarray, A: np.ndarray, b: np.ndarray, d: int) -> np.ndarray:
    """Effective weight W_hat from codes (eq. lc_codebook, Sec. 2.2; def. forward, Sec. 3.2).

    Columns split into G = n/d groups of d consecutive columns; group g of row r
    is the codeword A z + B with z = codes[r, g*d:(g+1)*d]:
        W_hat[r, g*d + j] = sum_k A[j, k] * codes[r, g*d + k] + b[j].
    `codes` may be float (the tests relax it to a continuous variable)."""
    C = np.asarray(codes, dtype=np.float64)
    m, n = C.shape
    assert n % d == 0
    A = np.asarray(A, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    z = C.reshape(m, n // d, d)                     # z[r, g, k]
    w = z @ A.T + b                                 # w[r, g, j] = sum_k z[r,g,k] A[j,k] + b[j]
    return w.reshape(m, n)


# -------------------------------------------------------------- forward -----

def forward(X: np.ndarray, W_hat: np.ndarray) -> np.ndarray:
    """Layer output Y = X W_hat^T  (Sec. 3.2, orientation as read above)."""
    return np.asarray(X, dtype=np.float64) @ np.asarray(W_hat, dtype=np.float64).T


def forward_reformulated(X: np.ndarray, codes: np.ndarray, A: np.ndarray, b: np.ndarray,
                         d: int) -> np.ndarray:
    """Reformulated forward (def. forward_x, Sec. 3.2):
        Y = sum_i (X_i A) W_{z,i}^T + sum_i (X_i B) 1^T,
    X_i = the d columns of group i.  Algebraically identical to forward(X, decode(...))."""
    X = np.asarray(X, dtype=np.float64)
    C = np.asarray(codes, dtype=np.float64)
    N, n = X.shape
    G = n // d
    Xi = X.reshape(N, G, d)                          # X_i for every group
    XA = (Xi @ np.asarray(A, dtype=np.float64)).reshape(N, n)   # [X_1 A, ..., X_G A]
    XB = (Xi @ np.asarray(b, dtype=np.float64)).sum(axis=1)     # sum_i X_i B  (length N)
    return XA @ C.T + XB[:, None]


# ------------------------------------------------------------- backward -----

def grad_input(dY: np.ndarray, W_hat: np.ndarray) -> np.ndarray:
    """dL/dX = dY W_hat (chain rule of Y = X W_hat^T)."""
    return np.asarray(dY, dtype=np.float64) @ np.asarray(W_hat, dtype=np.float64)


def grad_weight(dY: np.ndarray, X: np.ndarray) -> np.ndarray:
    """dL/dW_hat = dY^T X (chain rule of Y = X W_hat^T).  m x n."""
    return np.asarray(dY, dtype=np.float64).T @ np.asarray(X, dtype=np.float64)


def grad_codes(dW: np.ndarray, A: np.ndarray, d: int) -> np.ndarray:
    """dL/dcode[r, g*d + k] = sum_j dW[r, g*d + j] * A[j, k]  (chain rule of decode)."""
    dW = np.asarray(dW, dtype=np.float64)
    m, n = dW.shape
    return (dW.reshape(m, n // d, d) @ np.asarray(A, dtype=np.float64)).reshape(m, n)


def grad_latent(dW: np.ndarray, A: np.ndarray, d: int, mask: np.ndarray) -> np.ndarray:
    """Straight-through gradient of the proxy weights (Sec. 3.3): round() passes the
    gradient unchanged, clip() zeroes it outside its range:  dZ = mask * dL/dcode."""
    return np.where(mask, grad_codes(dW, A, d), 0.0)


def grad_map(dW: np.ndarray, codes: np.ndarray, d: int):
    """Gradients of the shared map (chain rule of decode):
        dA[j, k] = sum_{r,g} dW[r, g*d + j] * code[r, g*d + k]
        db[j]    = sum_{r,g} dW[r, g*d + j]."""
    dW = np.asarray(dW, dtype=np.float64)
    C = np.asarray(codes, dtype=np.float64)
    w = dW.reshape(-1, d)                            # one row per (r, g): dW_g
    z = C.reshape(-1, d)                             # matching code vectors
    return w.T @ z, w.sum(axis=0)


# ----------------------------------------------------------- whole layer ----

def linear_forward(Z, A, b, X, d, scale: float = 1.0, shift: float = 0.0):
    """Y and the codes of one LC-VQ linear call (all inputs fp64 values)."""
    codes = quantize(Z, scale, shift)
    return forward(X, decode(codes, A, b, d)), codes


def linear_backward(Z, A, b, X, dY, d, mask_mode: int = MASK_ROUNDED, dge=None, scale: float = 1.0,
                    shift: float = 0.0):
    """(dX, dZ, dA, db, dW_hat) of one LC-VQ linear call (all inputs fp64 values).

    dge = None: straight-through estimator.  dge = (k, cap): the differentiable
    gradient estimator (Sec. 3.3), dZ = mask * dge_slope(Z) * dL/dcode.  With a
    quantiser scale / shift (Sec. 3.4) mask and slope are taken at the code-domain
    value and the chain rule through it multiplies dZ by the scale."""
    codes = quantize(Z, scale, shift)
    W_hat = decode(codes, A, b, d)
    dW = grad_weight(dY, X)
    dX = grad_input(dY, W_hat)
    u = code_domain(Z, scale, shift)
    mask = ste_mask(u, mask_mode)
    if dge is None:
        dZ = grad_latent(dW, A, d, mask)
    else:
        with np.errstate(invalid="ignore"):
            dZ = np.where(mask, grad_codes(dW, A, d) * dge_slope(u, *dge), 0.0)
    if scale != 1.0:
        dZ = dZ * np.float64(np.float32(scale))
    dA, db = grad_map(dW, codes, d)
    return dict(dX=dX, dZ=dZ, dA=dA, db=db, dW=dW)


# ------------------------------------------------------------- packing ------

def pack2bit(codes: np.ndarray) -> np.ndarray:
    """Packed 2-bit codes, four per byte: the code of column c sits at bits
    2*(c mod 4) .. 2*(c mod 4)+1 of byte c // 4 of its row (least significant
    first).  The paper fixes only the width (2 bits, Sec. 2.1); the layout is
    this library's.  Returns uint8 array m x n/4."""
    C = np.asarray(codes, dtype=np.uint8)
    m, n = C.shape
    assert n % 4 == 0
    q = C.reshape(m, n // 4, 4).astype(np.uint32)
    byte = q[..., 0] | (q[..., 1] << 2) | (q[..., 2] << 4) | (q[..., 3] << 6)
    return byte.astype(np.uint8)


def unpack2bit(packed: np.ndarray, n: int) -> np.ndarray:
    """Codes of a packed m x n/4 array (inverse of pack2bit): code of column c =
    bits 2*(c mod 4) .. 2*(c mod 4)+1 of byte c // 4."""
    P = np.asarray(packed, dtype=np.uint8)
    m = P.shape[0]
    assert P.shape[1] * 4 == n
    out = np.empty((m, n), dtype=np.uint8)
    for i in range(4):
        out[:, i::4] = (P >> (2 * i)) & 3
    return out


def linear_forward_packed(packed, A, b, X, d, n):
    """Output of the layer from packed 2-bit codes (inference, Sec. 3.2 / App. A.2):
    Y = X W_hat^T with W_hat decoded from the unpacked codes."""
    return forward(X, decode(unpack2bit(packed, n), A, b, d))


# ------------------------------------------------------------ LC encode -----

def encode_values(W: np.ndarray, A: np.ndarray, b: np.ndarray, d: int) -> np.ndarray:
    """Continuous code vector of every group of a dense weight: the codeword
    relation w_g = A z + b of eq. lc_codebook (Sec. 2.2) solved for z, i.e.
        v[r, g*d + k] = sum_j Ainv[k, j] * (W[r, g*d + j] - b[j]),   Ainv = A^-1,
    in fp64 (A^-1 by LAPACK; the sum written out, so a non-finite weight gives
    the IEEE result of the written formula).  Raises for a singular A."""
    W = np.asarray(W, dtype=np.float64)
    m, n = W.shape
    assert n % d == 0
    Ainv = np.linalg.inv(np.asarray(A, dtype=np.float64))
    T = W.reshape(m, n // d, d) - np.asarray(b, dtype=np.float64)
    V = np.zeros_like(T)
    with np.errstate(invalid="ignore"):
        for k in range(d):
            for j in range(d):
                V[..., k] += Ainv[k, j] * T[..., j]
    return V.reshape(m, n)


def encode(W: np.ndarray, A: np.ndarray, b: np.ndarray, d: int) -> np.ndarray:
    """Codes of a dense weight under the map A, b: per group, clip(round(v), 0, 3)
    with v = A^-1 (w_g - b) (encode_values).  For A = s G with G orthogonal (the
    form of eq. init_ab) the squared distance ||w_g - A z - b||^2 = s^2 ||v - z||^2
    separates over the d coordinates, so these are the nearest codewords of
    eq. vq_assign; for other maps they are the rounding of A^-1 (w_g - b).
    Returns uint8 codes."""
    return quantize(encode_values(W, A, b, d))


# ------------------------------------------------------------ optimiser -----

def adamw_step(theta, grad, m1, m2, step: int, lr: float, beta1: float = 0.9,
               beta2: float = 0.999, eps: float = 1e-8, weight_decay: float = 0.0):
    """One AdamW update (the optimiser of Sec. 4.4, standard form with bias
    correction and decoupled weight decay).  Returns new (theta, m1, m2)."""
    theta = np.asarray(theta, dtype=np.float64)
    g = np.asarray(grad, dtype=np.float64)
    m1 = beta1 * np.asarray(m1, dtype=np.float64) + (1.0 - beta1) * g
    m2 = beta2 * np.asarray(m2, dtype=np.float64) + (1.0 - beta2) * g * g
    m_hat = m1 / (1.0 - beta1 ** step)
    v_hat = m2 / (1.0 - beta2 ** step)
    theta = theta - lr * weight_decay * theta - lr * m_hat / (np.sqrt(v_hat) + eps)
    return theta, m1, m2


# ------------------------------------------------------- init (Sec. 2.2) ----

def init_map(G: np.ndarray, bits: int = 2):
    """Initial map of eq. init_ab: A = s G, B = -s G mu 1, with mu = (2^b - 1)/2
    and s = sqrt(12 / (2^(2b) - 1)); G a d x d orthogonal matrix."""
    G = np.asarray(G, dtype=np.float64)
    d = G.shape[0]
    mu = (2 ** bits - 1) / 2.0
    s = np.sqrt(12.0 / (2 ** (2 * bits) - 1))
    return s * G, -s * G @ (mu * np.ones(d))

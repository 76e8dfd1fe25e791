"""LC-VQ linear layer (LC-QAT, arXiv 2606.10531) on MI355X (gfx950).

Thin torch binding of liblcvq.so: every function checks devices, dtypes and
contiguity, allocates outputs and workspace with torch, and passes raw device
pointers plus the current HIP stream to the C ABI.  All arithmetic runs in the
library's HIP kernels; there is no CPU or PyTorch fallback.
"""
from __future__ import annotations

import ctypes
import math

import torch

from . import _lib
from ._lib import (BF16, EST_DGE, EST_STE, F32, MASK_LATENT, MASK_ROUNDED, OP_BWD, OP_FWD, OP_FWD_PACKED,  # noqa: F401
                   SRC_CODES_U8, SRC_LATENT, SRC_PACKED2, LcvqError)

__all__ = ["linear_fwd", "linear_fwd_packed", "linear_bwd", "linear_bwd_dge", "xavier_quantizer", "xavier_init",
           "pack2bit", "dequant", "encode", "adamw_step", "workspace_bytes", "LcvqError", "MASK_ROUNDED", "MASK_LATENT",
           "SRC_LATENT", "SRC_CODES_U8", "SRC_PACKED2", "EST_STE", "EST_DGE"]

_DT = {torch.float32: F32, torch.bfloat16: BF16}


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype not in _DT:
        raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")
    return _DT[t.dtype]


def _dev(t: torch.Tensor, name: str) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _opt(t, name):
    return None if t is None else _dev(t, name)


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def workspace_bytes(op: int, N: int, m: int, n: int, d: int, dtype: torch.dtype) -> int:
    return int(_lib.load().lcvq_workspace_bytes(op, N, m, n, d, _DT[dtype]))


def _workspace(op, N, m, n, d, dtype, device, workspace):
    need = workspace_bytes(op, N, m, n, d, dtype)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=device)
    elif workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace has {workspace.numel() * workspace.element_size()} bytes, need {need}")
    return workspace


def pack2bit(src: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
    """Packed 2-bit codes (m x n/4 uint8) of a latent tensor (fp32/bf16) or of uint8 codes."""
    m, n = src.shape
    if src.dtype == torch.uint8:
        kind, sdt = SRC_CODES_U8, F32
    else:
        kind, sdt = SRC_LATENT, _dtype_code(src)
    if out is None:
        out = torch.empty((m, n // 4), dtype=torch.uint8, device=src.device)
    _lib.check(_lib.load().lcvq_pack2bit(_dev(src, "src"), kind, sdt, m, n, _dev(out, "out"),
                                         _stream(src.device)), "lcvq_pack2bit")
    return out


def dequant(src: torch.Tensor, A: torch.Tensor, b: torch.Tensor, d: int, n: int | None = None,
            src_kind: int | None = None, out_dtype: torch.dtype = torch.bfloat16,
            out: torch.Tensor | None = None) -> torch.Tensor:
    """Dense W_hat (m x n) from latents, uint8 codes or packed 2-bit codes (pass n for packed)."""
    if src_kind is None:
        src_kind = SRC_CODES_U8 if src.dtype == torch.uint8 else SRC_LATENT
    m = src.shape[0]
    if n is None:
        n = src.shape[1] * (4 if src_kind == SRC_PACKED2 else 1)
    sdt = _dtype_code(src) if src_kind == SRC_LATENT else F32
    if out is None:
        out = torch.empty((m, n), dtype=out_dtype, device=src.device)
    _lib.check(_lib.load().lcvq_dequant(m, n, d, src_kind, sdt, _dev(src, "src"), _dev(A, "A"), _dev(b, "b"),
                                        _dev(out, "out"), _DT[out.dtype], _stream(src.device)), "lcvq_dequant")
    return out


def encode(W: torch.Tensor, A: torch.Tensor, b: torch.Tensor, d: int, codes: bool = True, packed: bool = False):
    """LC encode of a dense weight W (m x n, fp32 or bf16): per group the codes
    clip(round(A^-1 (w_g - b)), 0, 3), the nearest codewords when A is a scaled
    orthogonal matrix.  Returns (codes m x n uint8 or None, packed m x n/4 uint8 or None)."""
    m, n = W.shape
    c = torch.empty((m, n), dtype=torch.uint8, device=W.device) if codes else None
    p = torch.empty((m, n // 4), dtype=torch.uint8, device=W.device) if packed else None
    _lib.check(_lib.load().lcvq_encode(m, n, d, _dev(W, "W"), _dtype_code(W), _dev(A, "A"), _dev(b, "b"),
                                       _opt(c, "codes"), _opt(p, "packed"), _stream(W.device)), "lcvq_encode")
    return c, p


def xavier_quantizer(m: int, n: int, bits: int = 2) -> tuple[float, float]:
    """(q_scale, q_shift) = (1 / s', t) of the Xavier reparameterisation (eq. xavier_preprocess,
    Sec. 3.4): s' = 2a / (2^b - 1), t = (2^b - 1) / 2, a = sqrt(6 / (m + n)); q_scale rounded to fp32."""
    a = math.sqrt(6.0 / (m + n))
    sp, t = 2.0 * a / (2 ** bits - 1), (2 ** bits - 1) / 2.0
    return float(torch.tensor(1.0 / sp, dtype=torch.float32)), t


def xavier_init(codes: torch.Tensor, m: int, n: int, d: int, src_kind: int | None = None,
                out_dtype: torch.dtype = torch.float32, bits: int = 2) -> torch.Tensor:
    """Initial proxy weights W_p = s' (W_z - t) (eq. xavier_preprocess) from uint8 or packed codes:
    lcvq_dequant with A = s' I and b = -s' t."""
    a = math.sqrt(6.0 / (m + n))
    sp, t = 2.0 * a / (2 ** bits - 1), (2 ** bits - 1) / 2.0
    A = torch.eye(d, dtype=torch.float32, device=codes.device) * sp
    b = torch.full((d,), -sp * t, dtype=torch.float32, device=codes.device)
    return dequant(codes, A, b, d, n=n, src_kind=src_kind, out_dtype=out_dtype)


def adamw_step(theta: torch.Tensor, grad: torch.Tensor, m1: torch.Tensor, m2: torch.Tensor, step: int,
               lr: float, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
               weight_decay: float = 0.0, shadow: torch.Tensor | None = None) -> None:
    """One in-place AdamW update of fp32 `theta`, `m1`, `m2` from `grad` (fp32 or bf16);
    `shadow` (fp32 or bf16, optional) receives the updated theta."""
    for t, nm in ((theta, "theta"), (m1, "m1"), (m2, "m2")):
        if t.dtype != torch.float32:
            raise TypeError(f"{nm} must be float32")
    numel = theta.numel()
    for t, nm in ((grad, "grad"), (m1, "m1"), (m2, "m2")) + (((shadow, "shadow"),) if shadow is not None else ()):
        if t.numel() != numel:
            raise ValueError(f"{nm} has {t.numel()} elements, theta has {numel}")
    sdt = _dtype_code(shadow) if shadow is not None else F32
    _lib.check(_lib.load().lcvq_adamw_step(_dev(theta, "theta"), _dev(grad, "grad"), _dtype_code(grad),
                                           _dev(m1, "m1"), _dev(m2, "m2"), _opt(shadow, "shadow"), sdt, numel,
                                           lr, beta1, beta2, eps, weight_decay, step, _stream(theta.device)),
               "lcvq_adamw_step")


def linear_fwd(Z: torch.Tensor, A: torch.Tensor, b: torch.Tensor, X: torch.Tensor, d: int,
               packed_out: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
               out: torch.Tensor | None = None, q_scale: float = 1.0, q_shift: float = 0.0) -> torch.Tensor:
    """Y = X W_hat^T (N x m) for latents Z (m x n), map A (d x d fp32), offset b (d fp32).

    q_scale, q_shift: the quantiser rounds Z * q_scale + q_shift (see xavier_quantizer);
    the default is the code domain."""
    m, n = Z.shape
    N = X.shape[0]
    dt = _dtype_code(X)
    if Z.dtype != X.dtype:
        raise TypeError("Z and X must share a dtype")
    if out is None:
        out = torch.empty((N, m), dtype=X.dtype, device=X.device)
    ws = _workspace(OP_FWD, N, m, n, d, X.dtype, X.device, workspace)
    tail = (_dev(A, "A"), _dev(b, "b"), _dev(X, "X"), _dev(out, "Y"), _opt(packed_out, "packed_out"),
            _dev(ws, "workspace"), ws.numel(), _stream(X.device))
    if q_scale == 1.0 and q_shift == 0.0:
        _lib.check(_lib.load().lcvq_linear_fwd(N, m, n, d, dt, _dev(Z, "Z"), *tail), "lcvq_linear_fwd")
    else:
        _lib.check(_lib.load().lcvq_linear_fwd_ex(N, m, n, d, dt, _dev(Z, "Z"), q_scale, q_shift, *tail),
                   "lcvq_linear_fwd_ex")
    return out


def linear_fwd_packed(packed: torch.Tensor, A: torch.Tensor, b: torch.Tensor, X: torch.Tensor, d: int,
                      out_dtype: torch.dtype = torch.bfloat16, workspace: torch.Tensor | None = None,
                      out: torch.Tensor | None = None) -> torch.Tensor:
    """Y = X W_hat^T (N x m, bf16 or fp32) from packed 2-bit codes (m x n/4 uint8) and bf16 X (N x n)."""
    m, n = packed.shape[0], packed.shape[1] * 4
    N = X.shape[0]
    if packed.dtype != torch.uint8:
        raise TypeError("packed codes must be uint8")
    if X.dtype != torch.bfloat16:
        raise TypeError("X must be bfloat16")
    if out is None:
        out = torch.empty((N, m), dtype=out_dtype, device=X.device)
    ws = _workspace(OP_FWD_PACKED, N, m, n, d, torch.bfloat16, X.device, workspace)
    _lib.check(_lib.load().lcvq_linear_fwd_packed(N, m, n, d, _dev(packed, "packed"), _dev(A, "A"), _dev(b, "b"),
                                                  _dev(X, "X"), _dev(out, "Y"), _DT[out.dtype],
                                                  _dev(ws, "workspace"), ws.numel(), _stream(X.device)),
               "lcvq_linear_fwd_packed")
    return out


def linear_bwd(Z: torch.Tensor, A: torch.Tensor, b: torch.Tensor, X: torch.Tensor, dY: torch.Tensor, d: int,
               mask_mode: int = MASK_ROUNDED, accumulate: bool = False, need_dX: bool = True,
               need_dZ: bool = True, need_map: bool = True, dz_dtype: torch.dtype | None = None,
               dX: torch.Tensor | None = None, dZ: torch.Tensor | None = None, dA: torch.Tensor | None = None,
               db: torch.Tensor | None = None, workspace: torch.Tensor | None = None, q_scale: float = 1.0,
               q_shift: float = 0.0):
    """Straight-through backward: returns (dX, dZ, dA, db); skipped outputs are None."""
    return _linear_bwd(None, Z, A, b, X, dY, d, mask_mode, accumulate, need_dX, need_dZ, need_map, dz_dtype,
                       dX, dZ, dA, db, workspace, q_scale, q_shift)


def linear_bwd_dge(Z: torch.Tensor, A: torch.Tensor, b: torch.Tensor, X: torch.Tensor, dY: torch.Tensor,
                   d: int, k: float = 5.0, cap: float = 3.0, mask_mode: int = MASK_LATENT,
                   accumulate: bool = False, need_dX: bool = True, need_dZ: bool = True, need_map: bool = True,
                   dz_dtype: torch.dtype | None = None, dX: torch.Tensor | None = None,
                   dZ: torch.Tensor | None = None, dA: torch.Tensor | None = None, db: torch.Tensor | None = None,
                   workspace: torch.Tensor | None = None, q_scale: float = 1.0, q_shift: float = 0.0):
    """Backward with the differentiable gradient estimator (k, slope cap): returns (dX, dZ, dA, db).

    The default mask is the latent one, [0 <= Z <= 3], which the chain rule
    gives through clip(f(Z), 0, 3)."""
    return _linear_bwd((float(k), float(cap)), Z, A, b, X, dY, d, mask_mode, accumulate, need_dX, need_dZ,
                       need_map, dz_dtype, dX, dZ, dA, db, workspace, q_scale, q_shift)


def _linear_bwd(dge, Z, A, b, X, dY, d, mask_mode, accumulate, need_dX, need_dZ, need_map, dz_dtype, dX, dZ, dA,
                db, workspace, q_scale=1.0, q_shift=0.0):
    m, n = Z.shape
    N = X.shape[0]
    dt = _dtype_code(X)
    dev = X.device
    if dz_dtype is None:
        dz_dtype = dZ.dtype if dZ is not None else Z.dtype
    if need_dX and dX is None:
        dX = torch.empty((N, n), dtype=X.dtype, device=dev)
    if need_dZ and dZ is None:
        dZ = (torch.zeros if accumulate else torch.empty)((m, n), dtype=dz_dtype, device=dev)
    if need_map and dA is None:
        dA = torch.zeros((d, d), dtype=torch.float32, device=dev)
        db = torch.zeros((d,), dtype=torch.float32, device=dev)
    ws = _workspace(OP_BWD, N, m, n, d, X.dtype, dev, workspace)
    head = (N, m, n, d, dt, _dev(Z, "Z"), _dev(A, "A"), _dev(b, "b"), _dev(X, "X"), _dev(dY, "dY"), mask_mode)
    tail = (1 if accumulate else 0, _opt(dX if need_dX else None, "dX"), _opt(dZ if need_dZ else None, "dZ"),
            _DT[dz_dtype], _opt(dA if need_map else None, "dA"), _opt(db if need_map else None, "db"),
            _dev(ws, "workspace"), ws.numel(), _stream(dev))
    if q_scale != 1.0 or q_shift != 0.0:
        est = (EST_STE, 0.0, 0.0) if dge is None else (EST_DGE, *dge)
        head_ex = head[:6] + (q_scale, q_shift) + head[6:]
        _lib.check(_lib.load().lcvq_linear_bwd_ex(*head_ex, *est, *tail), "lcvq_linear_bwd_ex")
    elif dge is None:
        _lib.check(_lib.load().lcvq_linear_bwd(*head, *tail), "lcvq_linear_bwd")
    else:
        _lib.check(_lib.load().lcvq_linear_bwd_dge(*head, *dge, *tail), "lcvq_linear_bwd_dge")
    return (dX if need_dX else None, dZ if need_dZ else None, dA if need_map else None,
            db if need_map else None)

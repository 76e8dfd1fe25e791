"""LC-VQ linear layer (LC-QAT, arXiv 2606.10531) on MI355X (gfx950).

Thin torch binding of liblcvq.so: every function checks devices, dtypes and
contiguity, allocates outputs and workspace with torch, and passes raw device
pointers plus the current HIP stream to the C ABI.  All arithmetic runs in the
library's HIP kernels; there is no CPU or PyTorch fallback.
"""
from __future__ import annotations

import ctypes

import torch

from . import _lib
from ._lib import (BF16, EST_DGE, EST_STE, F32, MASK_LATENT, MASK_ROUNDED, OP_BWD, OP_FWD, OP_FWD_PACKED,  # noqa: F401
                   SRC_CODES_U8, SRC_LATENT, SRC_PACKED2, LcvqError)

__all__ = ["linear_fwd", "linear_fwd_packed", "linear_fwd_packed_noalloc", "linear_bwd", "linear_bwd_dge", "xavier_quantizer", "xavier_init",
           "pack2bit", "dequant", "encode", "adamw_step", "workspace_bytes", "saved_bytes", "new_saved", "LcvqError", "MASK_ROUNDED", "MASK_LATENT",
           "SRC_LATENT", "SRC_CODES_U8", "SRC_PACKED2", "EST_STE", "EST_DGE"]

_DT = {torch.float32: F32, torch.bfloat16: BF16}


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype not in _DT:
        raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")
    return _DT[t.dtype]


def _check(t, name: str, shape=None, dtype=None) -> None:
    """Shape and dtype of one argument, checked before anything reaches the library
    (a mis-shaped buffer would be read or written out of bounds by the kernels, and
    a wrong dtype silently reinterpreted)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor, got {type(t).__name__}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if dtype is not None:
        ok = t.dtype in dtype if isinstance(dtype, tuple) else t.dtype == dtype
        if not ok:
            raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")


def _check_map(A, b, d: int) -> None:
    if d not in (4, 8):
        raise ValueError(f"group size d={d} (4 or 8)")
    _check(A, "A", (d, d), torch.float32)
    _check(b, "b", (d,), torch.float32)


def _check_2d(t, name: str) -> tuple:
    _check(t, name)
    if t.dim() != 2:
        raise ValueError(f"{name} must be 2-D, got shape {tuple(t.shape)}")
    return tuple(t.shape)


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


def saved_bytes(N: int, m: int, n: int, d: int, dtype: torch.dtype) -> int:
    """Size of the saved state of the training pair (0 for float32, which needs none)."""
    return int(_lib.load().lcvq_saved_bytes(N, m, n, d, _DT[dtype]))


def new_saved(N: int, m: int, n: int, d: int, dtype: torch.dtype, device) -> torch.Tensor:
    """A buffer for the saved state of linear_fwd(..., saved=...) / linear_bwd(..., saved=...)."""
    return torch.empty(max(saved_bytes(N, m, n, d, dtype), 16), dtype=torch.uint8, device=device)


def _saved_arg(saved, N, m, n, d, dtype):
    _check(saved, "saved", dtype=torch.uint8)
    if saved.dim() != 1:
        raise ValueError("saved must be a 1-D uint8 tensor")
    need = saved_bytes(N, m, n, d, dtype)
    if saved.numel() < need:
        raise ValueError(f"saved has {saved.numel()} bytes, need {need}")
    return _dev(saved, "saved"), saved.numel()


def workspace_bytes(op: int, N: int, m: int, n: int, d: int, dtype: torch.dtype) -> int:
    return int(_lib.load().lcvq_workspace_bytes(op, N, m, n, d, _DT[dtype]))


def _workspace(op, N, m, n, d, dtype, device, workspace):
    need = workspace_bytes(op, N, m, n, d, dtype)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=device)
    elif workspace.dtype != torch.uint8 or workspace.dim() != 1:
        raise TypeError(f"workspace must be a 1-D uint8 tensor (got {workspace.dtype}, {workspace.dim()}-D)")
    elif workspace.numel() < need:
        raise ValueError(f"workspace has {workspace.numel()} bytes, need {need}")
    return workspace


def pack2bit(src: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
    """Packed 2-bit codes (m x n/4 uint8) of a latent tensor (fp32/bf16) or of uint8 codes."""
    m, n = _check_2d(src, "src")
    if src.dtype == torch.uint8:
        kind, sdt = SRC_CODES_U8, F32
    else:
        kind, sdt = SRC_LATENT, _dtype_code(src)
    if n % 4 != 0:
        raise ValueError(f"n={n} is not a multiple of 4")
    if out is not None:
        _check(out, "out", (m, n // 4), torch.uint8)
    else:
        out = torch.empty((m, n // 4), dtype=torch.uint8, device=src.device)
    _lib.check(_lib.load().lcvq_pack2bit(_dev(src, "src"), kind, sdt, m, n, _dev(out, "out"),
                                         _stream(src.device)), "lcvq_pack2bit")
    return out


def dequant(src: torch.Tensor, A: torch.Tensor, b: torch.Tensor, d: int, n: int | None = None,
            src_kind: int | None = None, out_dtype: torch.dtype = torch.bfloat16,
            out: torch.Tensor | None = None) -> torch.Tensor:
    """Dense W_hat (m x n) from latents, uint8 codes or packed 2-bit codes (pass n for packed)."""
    _check_2d(src, "src")
    if src_kind is None:
        src_kind = SRC_CODES_U8 if src.dtype == torch.uint8 else SRC_LATENT
    m = src.shape[0]
    if n is None:
        n = src.shape[1] * (4 if src_kind == SRC_PACKED2 else 1)
    if src_kind == SRC_PACKED2:
        _check(src, "src", (m, n // 4), torch.uint8)
        if n % 4 != 0:
            raise ValueError(f"n={n} is not a multiple of 4")
    elif src_kind == SRC_CODES_U8:
        _check(src, "src", (m, n), torch.uint8)
    else:
        _check(src, "src", (m, n), (torch.float32, torch.bfloat16))
    _check_map(A, b, d)
    sdt = _dtype_code(src) if src_kind == SRC_LATENT else F32
    if out is not None:
        _check(out, "out", (m, n), (torch.float32, torch.bfloat16))
    else:
        out = torch.empty((m, n), dtype=out_dtype, device=src.device)
    _lib.check(_lib.load().lcvq_dequant(m, n, d, src_kind, sdt, _dev(src, "src"), _dev(A, "A"), _dev(b, "b"),
                                        _dev(out, "out"), _DT[out.dtype], _stream(src.device)), "lcvq_dequant")
    return out


def encode(W: torch.Tensor, A: torch.Tensor, b: torch.Tensor, d: int, codes: bool = True, packed: bool = False):
    """LC encode of a dense weight W (m x n, fp32 or bf16): per group the codes
    clip(round(A^-1 (w_g - b)), 0, 3), the nearest codewords when A is a scaled
    orthogonal matrix.  Returns (codes m x n uint8 or None, packed m x n/4 uint8 or None)."""
    m, n = _check_2d(W, "W")
    _check(W, "W", dtype=(torch.float32, torch.bfloat16))
    _check_map(A, b, d)
    c = torch.empty((m, n), dtype=torch.uint8, device=W.device) if codes else None
    p = torch.empty((m, n // 4), dtype=torch.uint8, device=W.device) if packed else None
    _lib.check(_lib.load().lcvq_encode(m, n, d, _dev(W, "W"), _dtype_code(W), _dev(A, "A"), _dev(b, "b"),
                                       _opt(c, "codes"), _opt(p, "packed"), _stream(W.device)), "lcvq_encode")
    return c, p


def xavier_quantizer(m: int, n: int) -> tuple[float, float]:
    """(q_scale, q_shift) = (1 / s', t) of the Xavier reparameterisation (Sec. 3.4,
    eq. xavier_preprocess) for 2-bit codes, from lcvq_xavier_quantizer."""
    qs, qb = ctypes.c_float(), ctypes.c_float()
    _lib.check(_lib.load().lcvq_xavier_quantizer(m, n, ctypes.byref(qs), ctypes.byref(qb)),
               "lcvq_xavier_quantizer")
    return qs.value, qb.value


def xavier_init(codes: torch.Tensor, m: int, n: int, src_kind: int | None = None,
                out_dtype: torch.dtype = torch.float32, out: torch.Tensor | None = None) -> torch.Tensor:
    """Initial proxy weights W_p = s' (W_z - t) (Sec. 3.4, eq. xavier_preprocess) of
    uint8 (m x n) or packed (m x n/4) codes, from lcvq_xavier_init."""
    if src_kind is None:
        src_kind = SRC_CODES_U8 if tuple(codes.shape) == (m, n) else SRC_PACKED2
    _check(codes, "codes", (m, n) if src_kind == SRC_CODES_U8 else (m, n // 4), torch.uint8)
    if out is not None:
        _check(out, "out", (m, n), (torch.float32, torch.bfloat16))
    else:
        out = torch.empty((m, n), dtype=out_dtype, device=codes.device)
    _lib.check(_lib.load().lcvq_xavier_init(m, n, src_kind, _dev(codes, "codes"), _dev(out, "out"), _DT[out.dtype],
                                            _stream(codes.device)), "lcvq_xavier_init")
    return out


def adamw_step(theta: torch.Tensor, grad: torch.Tensor, m1: torch.Tensor, m2: torch.Tensor, step: int,
               lr: float, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
               weight_decay: float = 0.0, shadow: torch.Tensor | None = None) -> None:
    """One in-place AdamW update of fp32 `theta`, `m1`, `m2` from `grad` (fp32 or bf16);
    `shadow` (fp32 or bf16, optional) receives the updated theta."""
    for t, nm in ((theta, "theta"), (m1, "m1"), (m2, "m2")):
        _check(t, nm, dtype=torch.float32)
    _check(grad, "grad", dtype=(torch.float32, torch.bfloat16))
    if shadow is not None:
        _check(shadow, "shadow", dtype=(torch.float32, torch.bfloat16))
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
               out: torch.Tensor | None = None, q_scale: float = 1.0, q_shift: float = 0.0,
               saved: torch.Tensor | None = None) -> torch.Tensor:
    """Y = X W_hat^T (N x m) for latents Z (m x n), map A (d x d fp32), offset b (d fp32).

    q_scale, q_shift: the quantiser rounds Z * q_scale + q_shift (see xavier_quantizer);
    the default is the code domain.  saved: a buffer from new_saved(); the forward then
    also writes what linear_bwd(..., saved=...) of the same layer needs (the training
    pair, lcvq_linear_fwd_train)."""
    m, n = _check_2d(Z, "Z")
    dt = _dtype_code(Z)
    N = _check_2d(X, "X")[0]
    _check(X, "X", (N, n), Z.dtype)
    _check_map(A, b, d)
    if packed_out is not None:
        if n % 4 != 0:
            raise ValueError(f"packed codes need n % 4 == 0 (n={n})")
        _check(packed_out, "packed_out", (m, n // 4), torch.uint8)
    if out is not None:
        _check(out, "out", (N, m), Z.dtype)
    else:
        out = torch.empty((N, m), dtype=X.dtype, device=X.device)
    ws = _workspace(OP_FWD, N, m, n, d, X.dtype, X.device, workspace)
    tail = (_dev(A, "A"), _dev(b, "b"), _dev(X, "X"), _dev(out, "Y"), _opt(packed_out, "packed_out"),
            _dev(ws, "workspace"), ws.numel(), _stream(X.device))
    if saved is not None:
        sp, sn = _saved_arg(saved, N, m, n, d, Z.dtype)
        _lib.check(_lib.load().lcvq_linear_fwd_train(N, m, n, d, dt, _dev(Z, "Z"), q_scale, q_shift, *tail[:5], sp, sn,
                                                     *tail[5:]), "lcvq_linear_fwd_train")
    elif q_scale == 1.0 and q_shift == 0.0:
        _lib.check(_lib.load().lcvq_linear_fwd(N, m, n, d, dt, _dev(Z, "Z"), *tail), "lcvq_linear_fwd")
    else:
        _lib.check(_lib.load().lcvq_linear_fwd_ex(N, m, n, d, dt, _dev(Z, "Z"), q_scale, q_shift, *tail),
                   "lcvq_linear_fwd_ex")
    return out


def linear_fwd_packed(packed: torch.Tensor, A: torch.Tensor, b: torch.Tensor, X: torch.Tensor, d: int,
                      out_dtype: torch.dtype = torch.bfloat16, workspace: torch.Tensor | None = None,
                      out: torch.Tensor | None = None) -> torch.Tensor:
    """Y = X W_hat^T (N x m, bf16 or fp32) from packed 2-bit codes (m x n/4 uint8) and bf16 X (N x n)."""
    m, n4 = _check_2d(packed, "packed")
    n = 4 * n4
    _check(packed, "packed", dtype=torch.uint8)
    N = _check_2d(X, "X")[0]
    _check(X, "X", (N, n), torch.bfloat16)
    _check_map(A, b, d)
    if out is not None:
        _check(out, "out", (N, m), (torch.float32, torch.bfloat16))
    else:
        out = torch.empty((N, m), dtype=out_dtype, device=X.device)
    ws = _workspace(OP_FWD_PACKED, N, m, n, d, torch.bfloat16, X.device, workspace)
    _lib.check(_lib.load().lcvq_linear_fwd_packed(N, m, n, d, _dev(packed, "packed"), _dev(A, "A"), _dev(b, "b"),
                                                  _dev(X, "X"), _dev(out, "Y"), _DT[out.dtype],
                                                  _dev(ws, "workspace"), ws.numel(), _stream(X.device)),
               "lcvq_linear_fwd_packed")
    return out


def linear_fwd_packed_noalloc(packed: torch.Tensor, A: torch.Tensor, b: torch.Tensor, X: torch.Tensor, d: int,
                              out: torch.Tensor) -> torch.Tensor:
    """linear_fwd_packed without a workspace: the library's fixed per-device scratch
    array takes its place (for callers that cannot allocate).  `out` (N x m, bf16 or
    fp32) is the caller's; calls that overlap on one device race."""
    m, n4 = _check_2d(packed, "packed")
    n = 4 * n4
    _check(packed, "packed", dtype=torch.uint8)
    N = _check_2d(X, "X")[0]
    _check(X, "X", (N, n), torch.bfloat16)
    _check_map(A, b, d)
    _check(out, "out", (N, m), (torch.float32, torch.bfloat16))
    _lib.check(_lib.load().lcvq_linear_fwd_packed_noalloc(N, m, n, d, _dev(packed, "packed"), _dev(A, "A"),
                                                          _dev(b, "b"), _dev(X, "X"), _dev(out, "Y"),
                                                          _DT[out.dtype], _stream(X.device)),
               "lcvq_linear_fwd_packed_noalloc")
    return out


def linear_bwd(Z: torch.Tensor, A: torch.Tensor, b: torch.Tensor, X: torch.Tensor, dY: torch.Tensor, d: int,
               mask_mode: int = MASK_ROUNDED, accumulate: bool = False, need_dX: bool = True,
               need_dZ: bool = True, need_map: bool = True, dz_dtype: torch.dtype | None = None,
               dX: torch.Tensor | None = None, dZ: torch.Tensor | None = None, dA: torch.Tensor | None = None,
               db: torch.Tensor | None = None, workspace: torch.Tensor | None = None, q_scale: float = 1.0,
               q_shift: float = 0.0, saved: torch.Tensor | None = None):
    """Straight-through backward: returns (dX, dZ, dA, db); skipped outputs are None.
    saved: the buffer a linear_fwd(..., saved=...) of the same layer and inputs filled."""
    return _linear_bwd(None, Z, A, b, X, dY, d, mask_mode, accumulate, need_dX, need_dZ, need_map, dz_dtype,
                       dX, dZ, dA, db, workspace, q_scale, q_shift, saved)


def linear_bwd_dge(Z: torch.Tensor, A: torch.Tensor, b: torch.Tensor, X: torch.Tensor, dY: torch.Tensor,
                   d: int, k: float = 5.0, cap: float = 3.0, mask_mode: int = MASK_LATENT,
                   accumulate: bool = False, need_dX: bool = True, need_dZ: bool = True, need_map: bool = True,
                   dz_dtype: torch.dtype | None = None, dX: torch.Tensor | None = None,
                   dZ: torch.Tensor | None = None, dA: torch.Tensor | None = None, db: torch.Tensor | None = None,
                   workspace: torch.Tensor | None = None, q_scale: float = 1.0, q_shift: float = 0.0,
                   saved: torch.Tensor | None = None):
    """Backward with the differentiable gradient estimator (k, slope cap): returns (dX, dZ, dA, db).

    The default mask is the latent one, [0 <= Z <= 3], which the chain rule
    gives through clip(f(Z), 0, 3)."""
    return _linear_bwd((float(k), float(cap)), Z, A, b, X, dY, d, mask_mode, accumulate, need_dX, need_dZ,
                       need_map, dz_dtype, dX, dZ, dA, db, workspace, q_scale, q_shift, saved)


def _linear_bwd(dge, Z, A, b, X, dY, d, mask_mode, accumulate, need_dX, need_dZ, need_map, dz_dtype, dX, dZ, dA,
                db, workspace, q_scale=1.0, q_shift=0.0, saved=None):
    m, n = _check_2d(Z, "Z")
    dt = _dtype_code(Z)
    N = _check_2d(X, "X")[0]
    _check(X, "X", (N, n), Z.dtype)
    _check(dY, "dY", (N, m), Z.dtype)
    _check_map(A, b, d)
    dev = X.device
    if dz_dtype is None:
        dz_dtype = dZ.dtype if dZ is not None else Z.dtype
    if dz_dtype not in (torch.float32, Z.dtype):
        raise TypeError(f"dZ dtype {dz_dtype}: float32 or the latent's dtype {Z.dtype}")
    if dX is not None:
        _check(dX, "dX", (N, n), Z.dtype)
    if dZ is not None:
        _check(dZ, "dZ", (m, n), dz_dtype)
    if (dA is None) != (db is None):
        raise ValueError("dA and db are given together or not at all")
    if dA is not None:
        _check(dA, "dA", (d, d), torch.float32)
        _check(db, "db", (d,), torch.float32)
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
    if saved is not None:
        sp, sn = _saved_arg(saved, N, m, n, d, Z.dtype)
        est = (EST_STE, 0.0, 0.0) if dge is None else (EST_DGE, *dge)
        head_ex = head[:6] + (q_scale, q_shift) + head[6:]
        _lib.check(_lib.load().lcvq_linear_bwd_train(*head_ex, *est, *tail[:6], sp, sn, *tail[6:]),
                   "lcvq_linear_bwd_train")
    elif q_scale != 1.0 or q_shift != 0.0:
        est = (EST_STE, 0.0, 0.0) if dge is None else (EST_DGE, *dge)
        head_ex = head[:6] + (q_scale, q_shift) + head[6:]
        _lib.check(_lib.load().lcvq_linear_bwd_ex(*head_ex, *est, *tail), "lcvq_linear_bwd_ex")
    elif dge is None:
        _lib.check(_lib.load().lcvq_linear_bwd(*head, *tail), "lcvq_linear_bwd")
    else:
        _lib.check(_lib.load().lcvq_linear_bwd_dge(*head, *dge, *tail), "lcvq_linear_bwd_dge")
    return (dX if need_dX else None, dZ if need_dZ else None, dA if need_map else None,
            db if need_map else None)

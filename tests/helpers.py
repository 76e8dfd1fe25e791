"""Host-side glue shared by the GPU tests: move seeded inputs to the device and
device results back to exact fp64 values for comparison with the oracle."""
import numpy as np

import oracle as orc


def to_dev(arr, dtype):
    import torch
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.uint16).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()


def to_host(t):
    """Exact fp64 values of a device tensor."""
    import torch
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return orc.widen(t.view(torch.int16).numpy().view(np.uint16), "bf16")
    return t.numpy().astype(np.float64)


def rel_fro(got, ref):
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def _ratio(num, den):
    """num / den elementwise; a zero reference block must be matched exactly."""
    out = np.where(den > 0, num / np.where(den > 0, den, 1.0), 0.0)
    return np.where((den == 0) & (num > 0), np.inf, out)


def local_rel(got, ref, tile=256):
    """The largest relative Frobenius error over the rows of a result, and over
    its tile x tile blocks (a 1-D result is one row).  A whole-matrix norm can
    hide an error confined to one row, one tile or a ragged tail; this does not."""
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    if got.shape != ref.shape:
        raise ValueError(f"shape mismatch {got.shape} vs {ref.shape}")
    if ref.ndim == 1:
        got, ref = got[None, :], ref[None, :]
    if ref.size == 0:
        return 0.0
    err2 = (got - ref) ** 2
    ref2 = ref ** 2
    worst = float(np.max(_ratio(np.sqrt(err2.sum(axis=1)), np.sqrt(ref2.sum(axis=1)))))
    R, C = ref.shape
    pr, pc = -R % tile, -C % tile
    e = np.pad(err2, ((0, pr), (0, pc))).reshape((R + pr) // tile, tile, (C + pc) // tile, tile).sum(axis=(1, 3))
    r = np.pad(ref2, ((0, pr), (0, pc))).reshape((R + pr) // tile, tile, (C + pc) // tile, tile).sum(axis=(1, 3))
    return max(worst, float(np.max(_ratio(np.sqrt(e), np.sqrt(r)))))


def assert_close(got, ref, tol, what=""):
    """Parity bar of a floating-point result: relative Frobenius error <= tol over
    the whole result, over every row and over every 256 x 256 tile."""
    g, loc = rel_fro(got, ref), local_rel(got, ref)
    assert g <= tol and loc <= tol, f"{what}: rel_fro {g:.3e}, worst row/tile {loc:.3e}, tolerance {tol:g}"


def unpack2bit(packed, n):
    p = np.asarray(packed, dtype=np.uint8)
    return np.stack([(p >> (2 * i)) & 3 for i in range(4)], axis=-1).reshape(p.shape[0], n)

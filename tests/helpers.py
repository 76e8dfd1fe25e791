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


def unpack2bit(packed, n):
    p = np.asarray(packed, dtype=np.uint8)
    return np.stack([(p >> (2 * i)) & 3 for i in range(4)], axis=-1).reshape(p.shape[0], n)

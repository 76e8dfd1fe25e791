"""Parity at the full sizes of the Llama-shaped workloads, through the C ABI,
in the same launch configuration as the 4096 x 4096 benchmark step:

  * 7B MLP: gate / up 11008 x 4096 and down 4096 x 11008, 8192 tokens;
  * 70B MLP: 28672 x 8192 and 8192 x 28672, 4096 tokens, plus the 2-bit pack
    of the final codes;
  * 7B decoder block: the 4096 x 4096 and 4096 x 11008 shapes at 16384 tokens.

Every matrix of a workload is drawn with its own index k (seeds of A, b, Z, X,
dY).  Codes and packed words are compared in full, bit for bit; Y and dX on
sampled token rows, dZ on sampled out-feature rows (each row is exact in the
oracle by itself); dA and db in full (fp64, over every token, row and group).
"""
import numpy as np
import pytest

import oracle as orc
import synth
from helpers import assert_close, rel_fro, to_dev, to_host

pytestmark = pytest.mark.gpu

TOL = 2e-2


@pytest.fixture(scope="module")
def lc():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_10531_amd as lc
    lc._lib.load()
    return lc


def _sample(count, k):
    return np.unique(np.concatenate([np.arange(64), synth.rng(7000 + k).integers(0, count, 192), [count - 1]]))


def _check_matrix(lc, N, m, n, d, k, pack):
    import torch
    print(f"\nworkload matrix N={N} m={m} n={n} d={d} k={k}", flush=True)
    inp = synth.layer_inputs(N, m, n, d, "bf16", k=k)
    Z, X, dY = to_dev(inp["Z"], "bf16"), to_dev(inp["X"], "bf16"), to_dev(inp["dY"], "bf16")
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    packed = torch.empty((m, n // 4), dtype=torch.uint8, device="cuda")
    Y = lc.linear_fwd(Z, A, b, X, d, packed_out=packed)
    dX, dZ, dA, db = lc.linear_bwd(Z, A, b, X, dY, d)
    P2 = lc.pack2bit(Z) if pack else None
    torch.cuda.synchronize()
    tok, rows = _sample(N, k), _sample(m, k + 100)
    Yh, dXh, dZh = to_host(Y[tok]), to_host(dX[tok]), to_host(dZ[rows])
    packed_h = packed.cpu().numpy()
    P2h = P2.cpu().numpy() if pack else None
    dAh, dbh = to_host(dA), to_host(db)
    del Z, X, dY, Y, dX, dZ, packed, P2
    torch.cuda.empty_cache()

    v = {key: orc.widen(inp[key], "bf16") for key in ("Z", "X", "dY")}
    A64, b64 = inp["A"].astype(np.float64), inp["b"].astype(np.float64)
    codes = orc.quantize(v["Z"])
    want = orc.pack2bit(codes)
    assert np.array_equal(packed_h, want)
    if pack:
        assert np.array_equal(P2h, want)
    W = orc.decode(codes, A64, b64, d)
    assert_close(Yh, orc.forward(v["X"][tok], W), TOL, 'Y')
    assert_close(dXh, orc.grad_input(v["dY"][tok], W), TOL, 'dX')
    del W
    mask = orc.ste_mask(v["Z"][rows])
    assert_close(dZh, orc.grad_latent(orc.grad_weight(v["dY"][:, rows], v["X"]), A64, d, mask), TOL, 'dZ')
    dA_ref, db_ref = orc.grad_map(orc.grad_weight(v["dY"], v["X"]), codes, d)
    assert_close(dAh, dA_ref, TOL, 'dA')
    assert_close(dbh, db_ref, TOL, 'db')


def _cases():
    out = []
    for name, pack in (("lcvq_mlp7b_n8192_bf16", False), ("lcvq_mlp70b_n4096_bf16", True)):
        w = synth.WORKLOADS[name]
        seen = set()
        for k, (m, n) in enumerate(w["mats"]):
            if (m, n) in seen:          # gate and up share a shape: one of them
                continue
            seen.add((m, n))
            out.append(pytest.param(w["N"], m, n, w["d"], k, pack, id=f"{name}-{m}x{n}"))
    w = synth.WORKLOADS["lcvq_block7b_n16384_bf16"]
    out.append(pytest.param(w["N"], 4096, 4096, w["d"], 0, False, id="lcvq_block7b_n16384_bf16-4096x4096"))
    out.append(pytest.param(w["N"], 4096, 11008, w["d"], 6, False, id="lcvq_block7b_n16384_bf16-4096x11008"))
    return out


@pytest.mark.parametrize("N,m,n,d,k,pack", _cases())
def test_workload_matrix_full_size(lc, N, m, n, d, k, pack):
    _check_matrix(lc, N, m, n, d, k, pack)

"""Run-to-run repeatability of the training step through the C ABI.

The products stage operands through LDS with explicit waits and barriers; a
wait that no longer covers a stage shows up as a result that changes from one
identical call to the next.  Every output is computed in a fixed order (dA and
db as per-block partial sums added up in a fixed order, no atomics), so Y, the
packed codes, dX, dZ, dA and db must all be the same bit for bit over repeated
calls on the same inputs.  The shapes cover the weight-gradient loop with no
full trip (256 tokens), a few trips and a ragged tail, and the 4096 x 4096 step
of the benchmark, under both estimators."""
import pytest

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


def _bits(t):
    import torch
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else (torch.uint8 if t.dtype == torch.uint8 else torch.int32))


CASES = [(256, 256, 256, 8, 40), (1024, 1024, 1024, 8, 40), (1000, 520, 1096, 4, 40), (4096, 4096, 4096, 8, 60)]


@pytest.mark.parametrize("N,m,n,d,reps", CASES)
@pytest.mark.parametrize("est", ["ste", "dge"])
def test_training_step_repeats_bit_for_bit(lc, N, m, n, d, reps, est):
    import torch
    print(f"\nrepeat N={N} m={m} n={n} d={d} est={est} reps={reps}", flush=True)
    inp = synth.layer_inputs(N, m, n, d, "bf16", k=N + m + n + d, z_lo=-1.0, z_hi=4.0)
    Z, X, dY = to_dev(inp["Z"], "bf16"), to_dev(inp["X"], "bf16"), to_dev(inp["dY"], "bf16")
    A, b = torch.from_numpy(inp["A"]).cuda(), torch.from_numpy(inp["b"]).cuda()
    saved = lc.new_saved(N, m, n, d, torch.bfloat16, "cuda")
    packed = torch.empty((m, n // 4), dtype=torch.uint8, device="cuda")
    Y = torch.empty((N, m), dtype=torch.bfloat16, device="cuda")
    dX = torch.empty((N, n), dtype=torch.bfloat16, device="cuda")
    dZ = torch.empty((m, n), dtype=torch.bfloat16, device="cuda")
    dA = torch.empty((d, d), dtype=torch.float32, device="cuda")
    db = torch.empty((d,), dtype=torch.float32, device="cuda")

    def step():
        lc.linear_fwd(Z, A, b, X, d, packed_out=packed, out=Y, saved=saved)
        if est == "ste":
            lc.linear_bwd(Z, A, b, X, dY, d, dX=dX, dZ=dZ, dA=dA, db=db, saved=saved)
        else:
            lc.linear_bwd_dge(Z, A, b, X, dY, d, k=5.0, cap=3.0, dX=dX, dZ=dZ, dA=dA, db=db, saved=saved)

    step()
    torch.cuda.synchronize()
    exact = {"Y": Y, "packed": packed, "dX": dX, "dZ": dZ, "dA": dA, "db": db}
    ref = {key: _bits(t).clone() for key, t in exact.items()}
    changed = {key: 0 for key in exact}
    for _ in range(reps):
        step()
        for key, t in exact.items():
            if not torch.equal(_bits(t), ref[key]):
                changed[key] += 1
    torch.cuda.synchronize()
    assert all(v == 0 for v in changed.values()), f"outputs changed between identical calls: {changed} of {reps}"

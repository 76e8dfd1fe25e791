"""AdamW step (lcvq_adamw_step) on the GPU against the fp64 oracle update."""
import numpy as np
import pytest

import oracle as orc
import synth

from helpers import to_dev, to_host

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _state(numel, seed, grad_dtype):
    r = synth.rng(seed)
    theta = r.uniform(-0.5, 3.5, numel).astype(np.float32)
    m1 = (0.01 * r.standard_normal(numel)).astype(np.float32)
    m2 = (1e-4 * r.random(numel)).astype(np.float32)
    g = r.standard_normal(numel).astype(np.float32) * 0.05
    if grad_dtype == "bf16":
        g = synth.bf16_bits(g)
    return theta, g, m1, m2


def _f32(x):
    return float(np.float32(x))


def _check(theta0, g, gdt, m10, m20, step, lr, wd, th, m1, m2):
    """fp32 state vs the fp64 update from the same inputs (hyper-parameters as the
    fp32 values the kernel receives): each moment within a few fp32 roundings of
    its terms, and the parameter update within 1e-5 plus the rounding of theta."""
    gw = orc.widen(g, gdt)
    b1, b2 = _f32(0.9), _f32(0.999)
    rt, r1, r2 = orc.adamw_step(theta0.astype(np.float64), gw, m10, m20, step, lr=_f32(lr), beta1=b1, beta2=b2,
                                eps=_f32(1e-8), weight_decay=_f32(wd))
    ulp = np.float64(2.0 ** -23)
    m10, m20 = np.asarray(m10, np.float64), np.asarray(m20, np.float64)
    assert np.all(np.abs(m1 - r1) <= 4 * ulp * (b1 * np.abs(m10) + (1 - b1) * np.abs(gw)) + 1e-38)
    assert np.all(np.abs(m2 - r2) <= 4 * ulp * np.abs(r2) + 1e-38)
    delta, rdelta = th.astype(np.float64) - theta0, rt - theta0
    # |theta| < 4 here: the two fp32 roundings of the new theta stay below 2^-21 absolute
    assert np.all(np.abs(delta - rdelta) <= 1e-5 * np.abs(rdelta) + 2.0 ** -21)


@pytest.mark.parametrize("numel", [1, 3, 4, 1000, 4097, 262147])
@pytest.mark.parametrize("gdt", ["f32", "bf16"])
def test_adamw_matches_oracle(numel, gdt):
    import paper_2606_10531_amd as lc
    theta0, g, m10, m20 = _state(numel, 11 + numel, gdt)
    th, m1, m2 = (torch.from_numpy(x.copy()).cuda() for x in (theta0, m10, m20))
    gd = to_dev(g, gdt)
    shadow = torch.empty(numel, dtype=torch.bfloat16, device="cuda")
    step, lr, wd = 3, 1e-2, 0.01
    lc.adamw_step(th, gd, m1, m2, step, lr, weight_decay=wd, shadow=shadow)
    torch.cuda.synchronize()
    thh = th.cpu().numpy()
    _check(theta0, g, gdt, m10, m20, step, lr, wd, thh, m1.cpu().numpy(), m2.cpu().numpy())
    # the bf16 copy is the round-to-nearest-even image of the fp32 result
    assert np.array_equal(shadow.cpu().view(torch.int16).numpy().view(np.uint16), synth.bf16_bits(thh))


def test_adamw_fp32_shadow_and_no_shadow_agree():
    import paper_2606_10531_amd as lc
    theta0, g, m10, m20 = _state(5003, 7, "f32")
    outs = []
    for with_shadow in (False, True):
        th, m1, m2 = (torch.from_numpy(x.copy()).cuda() for x in (theta0, m10, m20))
        sh = torch.empty(5003, dtype=torch.float32, device="cuda") if with_shadow else None
        lc.adamw_step(th, to_dev(g, "f32"), m1, m2, 1, 1e-3, shadow=sh)
        torch.cuda.synchronize()
        outs.append(th.cpu().numpy())
        if with_shadow:
            assert np.array_equal(sh.cpu().numpy(), outs[-1])
    assert np.array_equal(outs[0], outs[1])


def test_adamw_ten_steps_track_oracle():
    """Ten steps from zero moments, each checked against the oracle step taken from
    the state the GPU holds (per-step parity)."""
    import paper_2606_10531_amd as lc
    numel = 65536
    theta0, _, _, _ = _state(numel, 5, "f32")
    th = torch.from_numpy(theta0.copy()).cuda()
    m1 = torch.zeros(numel, device="cuda")
    m2 = torch.zeros(numel, device="cuda")
    for step in range(1, 11):
        g = (synth.rng(100 + step).standard_normal(numel) * 0.1).astype(np.float32)
        prev = (th.cpu().numpy(), m1.cpu().numpy(), m2.cpu().numpy())
        lc.adamw_step(th, to_dev(g, "f32"), m1, m2, step, 1e-4)
        torch.cuda.synchronize()
        _check(prev[0], g, "f32", prev[1], prev[2], step, 1e-4, 0.0, th.cpu().numpy(), m1.cpu().numpy(),
               m2.cpu().numpy())


def test_adamw_full_matrix_sampled():
    """A whole 11008 x 4096 latent (45 M parameters, bf16 gradient and shadow), checked on
    a seeded sample of elements."""
    import paper_2606_10531_amd as lc
    m, n = 11008, 4096
    numel = m * n
    theta0 = synth.draw_latent(m, n, 0, "f32").reshape(-1)
    g = synth.draw_activations(m, n, 9, "bf16").reshape(-1)
    th = torch.from_numpy(theta0.copy()).cuda()
    m1 = torch.zeros(numel, device="cuda")
    m2 = torch.zeros(numel, device="cuda")
    sh = torch.empty(numel, dtype=torch.bfloat16, device="cuda")
    lc.adamw_step(th, to_dev(g, "bf16"), m1, m2, 1, 1e-4, shadow=sh)
    torch.cuda.synchronize()
    idx = np.sort(synth.rng(3).choice(numel, 20000, replace=False))
    thh = th.cpu().numpy()
    _check(theta0[idx], g[idx], "bf16", np.zeros(idx.size), np.zeros(idx.size), 1, 1e-4, 0.0, thh[idx],
           m1.cpu().numpy()[idx], m2.cpu().numpy()[idx])
    assert np.array_equal(sh.cpu().view(torch.int16).numpy().view(np.uint16)[idx], synth.bf16_bits(thh[idx]))

"""The C ABI boundary without a GPU: the library loads, exports every entry
point declared in include/lcvq.h, and rejects bad arguments on the host before
anything is enqueued (so no call here reaches the HIP runtime)."""
import ctypes
import os
import re

import pytest

from paper_2606_10531_amd import _lib as L

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "lcvq.h")
FAKE = 0x10000            # 16-byte aligned, never dereferenced: validation fails first
MIS = 0x10002             # misaligned


@pytest.fixture(scope="module")
def lib():
    return L.load()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(lcvq_\w+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert set(names) >= {"lcvq_dequant", "lcvq_linear_fwd", "lcvq_linear_bwd", "lcvq_pack2bit",
                          "lcvq_workspace_bytes", "lcvq_status_string", "lcvq_last_error"}
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(L.SIGNATURES)


def test_status_strings(lib):
    for s in range(6):
        assert L.status_string(s)
    assert L.status_string(99) == "unknown status"


def test_workspace_bytes(lib):
    f = lib.lcvq_workspace_bytes
    assert f(L.OP_FWD, 16, 256, 256, 8, L.F32) > 0
    assert f(L.OP_FWD, 4096, 4096, 4096, 8, L.BF16) >= 4096 * 4096 * 2      # transformed activations
    assert f(L.OP_BWD, 4096, 4096, 4096, 8, L.BF16) >= 4096 * 4096 // 2     # codes, 4 bits each
    assert f(L.OP_FWD, 16, 256, 256, 5, L.F32) == 0
    assert f(L.OP_FWD, -1, 256, 256, 8, L.F32) == 0
    assert f(7, 16, 256, 256, 8, L.F32) == 0
    assert f(L.OP_FWD, 300, 264, 328, 8, L.BF16) >= f(L.OP_FWD, 256, 264, 328, 8, L.BF16)


def test_workspace_bytes_of_empty_problems(lib):
    """Zero sizes must not trip the host-side layout arithmetic (no division by zero)."""
    f = lib.lcvq_workspace_bytes
    for op in (L.OP_FWD, L.OP_BWD, L.OP_FWD_PACKED):
        for dt in (L.F32, L.BF16):
            for N, m, n in ((0, 64, 64), (16, 0, 64), (16, 64, 0), (0, 0, 0)):
                assert f(op, N, m, n, 8, dt) >= 0
    assert f(L.OP_FWD_PACKED, 16, 64, 64, 8, L.BF16) > 0
    assert f(L.OP_FWD_PACKED, 16, 64, 64, 8, L.F32) == 0          # bf16 only


def fwd(lib, N=16, m=64, n=64, d=8, dt=L.BF16, Z=FAKE, A=FAKE, b=FAKE, X=FAKE, Y=FAKE, packed=None,
        ws=FAKE, wsb=1 << 40):
    return lib.lcvq_linear_fwd(N, m, n, d, dt, Z, A, b, X, Y, packed, ws, wsb, None)


def bwd(lib, N=16, m=64, n=64, d=8, dt=L.BF16, mask=0, acc=0, dX=FAKE, dZ=FAKE, dzt=L.BF16, dA=FAKE,
        db=FAKE, ws=FAKE, wsb=1 << 40, X=FAKE, dY=FAKE):
    return lib.lcvq_linear_bwd(N, m, n, d, dt, FAKE, FAKE, FAKE, X, dY, mask, acc, dX, dZ, dzt, dA, db, ws,
                               wsb, None)


def test_fwd_validation(lib):
    assert fwd(lib, d=5) == L.EUNSUPPORTED
    assert fwd(lib, n=60, d=8) == L.EINVAL                 # n % d
    assert fwd(lib, N=-1) == L.EINVAL
    assert fwd(lib, dt=7) == L.EINVAL
    assert fwd(lib, m=60, n=64) == L.EUNSUPPORTED          # bf16 path: m % 8
    assert fwd(lib, m=60, n=64, dt=L.F32) != L.EUNSUPPORTED
    assert fwd(lib, Z=None) == L.EINVAL
    assert fwd(lib, X=None) == L.EINVAL
    assert fwd(lib, Y=MIS) == L.EALIGN
    assert fwd(lib, packed=MIS) == L.EALIGN
    assert fwd(lib, wsb=16) == L.EWORKSPACE
    assert fwd(lib, ws=None) == L.EWORKSPACE
    assert "workspace" in L.last_error()
    # an empty product is valid and enqueues nothing
    assert fwd(lib, N=0, Y=None, X=None) == L.OK
    assert fwd(lib, m=0, Y=None) == L.OK


def test_bwd_validation(lib):
    assert bwd(lib, d=3) == L.EUNSUPPORTED
    assert bwd(lib, mask=2) == L.EINVAL
    assert bwd(lib, acc=2) == L.EINVAL
    assert bwd(lib, dA=None) == L.EINVAL                   # dA and db go together
    assert bwd(lib, dt=L.F32, dzt=L.BF16) == L.EINVAL     # bf16 dZ needs the bf16 path
    assert bwd(lib, X=None) == L.EINVAL
    assert bwd(lib, dY=MIS) == L.EALIGN
    assert bwd(lib, dZ=MIS) == L.EALIGN
    assert bwd(lib, wsb=8) == L.EWORKSPACE
    assert bwd(lib, N=0, acc=1) == L.OK                    # accumulate into nothing: no work


def bwd_dge(lib, k=5.0, cap=3.0, N=16, m=64, n=64, d=8, dt=L.BF16, mask=1, acc=0, dX=FAKE, dZ=FAKE, dzt=L.BF16,
            dA=FAKE, db=FAKE, ws=FAKE, wsb=1 << 40, X=FAKE, dY=FAKE):
    return lib.lcvq_linear_bwd_dge(N, m, n, d, dt, FAKE, FAKE, FAKE, X, dY, mask, k, cap, acc, dX, dZ, dzt, dA,
                                   db, ws, wsb, None)


def test_bwd_dge_validation(lib):
    assert bwd_dge(lib, k=0.5) == L.EINVAL                 # k >= 1
    assert bwd_dge(lib, k=float("nan")) == L.EINVAL
    assert bwd_dge(lib, k=float("inf")) == L.EINVAL
    assert bwd_dge(lib, cap=0.0) == L.EINVAL               # cap > 0
    assert bwd_dge(lib, cap=-1.0) == L.EINVAL
    assert bwd_dge(lib, cap=float("inf")) == L.EINVAL
    assert "cap" in L.last_error()
    # the remaining checks are those of the straight-through entry point
    assert bwd_dge(lib, d=3) == L.EUNSUPPORTED
    assert bwd_dge(lib, mask=2) == L.EINVAL
    assert bwd_dge(lib, dA=None) == L.EINVAL
    assert bwd_dge(lib, dY=MIS) == L.EALIGN
    assert bwd_dge(lib, wsb=8) == L.EWORKSPACE
    assert bwd_dge(lib, N=0, acc=1) == L.OK
    assert bwd_dge(lib, k=1.0, N=0, acc=1) == L.OK


def fwd_packed(lib, N=16, m=64, n=64, d=8, P=FAKE, X=FAKE, Y=FAKE, ydt=L.BF16, ws=FAKE, wsb=1 << 40):
    return lib.lcvq_linear_fwd_packed(N, m, n, d, P, FAKE, FAKE, X, Y, ydt, ws, wsb, None)


def test_fwd_packed_validation(lib):
    assert fwd_packed(lib, d=5) == L.EUNSUPPORTED
    assert fwd_packed(lib, n=32) == L.EUNSUPPORTED               # n % 64
    assert "64" in L.last_error()
    assert fwd_packed(lib, m=60) == L.EUNSUPPORTED               # m % 8
    assert fwd_packed(lib, N=-1) == L.EINVAL
    assert fwd_packed(lib, ydt=7) == L.EINVAL
    assert fwd_packed(lib, P=None) == L.EINVAL
    assert fwd_packed(lib, X=None) == L.EINVAL
    assert fwd_packed(lib, Y=None) == L.EINVAL
    assert fwd_packed(lib, P=MIS) == L.EALIGN
    assert fwd_packed(lib, Y=MIS) == L.EALIGN
    assert fwd_packed(lib, wsb=16) == L.EWORKSPACE
    assert fwd_packed(lib, N=0, Y=None, X=None) == L.OK          # nothing to compute
    assert fwd_packed(lib, m=0, Y=None) == L.OK


def test_ex_validation(lib):
    def f(qs=0.5, qb=1.5, **kw):
        a = dict(N=16, m=64, n=64, d=8, dt=L.BF16)
        a.update(kw)
        return lib.lcvq_linear_fwd_ex(a["N"], a["m"], a["n"], a["d"], a["dt"], FAKE, qs, qb, FAKE, FAKE, FAKE, FAKE,
                                      None, FAKE, 1 << 40, None)

    def g(qs=0.5, qb=1.5, est=L.EST_STE, k=5.0, cap=3.0, mask=1, **kw):
        return lib.lcvq_linear_bwd_ex(16, 64, 64, kw.get("d", 8), L.BF16, FAKE, qs, qb, FAKE, FAKE, FAKE, FAKE, mask,
                                      est, k, cap, 0, FAKE, FAKE, L.BF16, FAKE, FAKE, FAKE, 1 << 40, None)
    for bad in (0.0, float("nan"), float("inf")):
        assert f(qs=bad) == L.EINVAL and g(qs=bad) == L.EINVAL
    assert f(qb=float("nan")) == L.EINVAL and g(qb=float("inf")) == L.EINVAL
    assert "quantiser" in L.last_error()
    assert g(est=2) == L.EINVAL
    assert g(est=L.EST_DGE, k=0.5) == L.EINVAL
    assert g(est=L.EST_DGE, cap=0.0) == L.EINVAL
    assert f(d=5) == L.EUNSUPPORTED and g(d=3) == L.EUNSUPPORTED
    assert g(mask=2) == L.EINVAL
    assert f(N=0) == L.OK                                   # nothing to compute


def test_encode_validation(lib):
    def e(m=64, n=64, d=8, W=FAKE, wdt=L.BF16, codes=FAKE, packed=None):
        return lib.lcvq_encode(m, n, d, W, wdt, FAKE, FAKE, codes, packed, None)
    assert e(d=5) == L.EUNSUPPORTED
    assert e(n=60) == L.EINVAL                              # n % d
    assert e(m=-1) == L.EINVAL
    assert e(wdt=7) == L.EINVAL
    assert e(codes=None, packed=None) == L.EINVAL           # nothing to write
    assert "output" in L.last_error()
    assert e(W=None) == L.EINVAL
    assert e(W=MIS) == L.EALIGN
    assert e(codes=None, packed=MIS) == L.EALIGN
    assert e(m=0) == L.OK and e(n=0) == L.OK                # empty: no launch


def test_pack_and_dequant_validation(lib):
    p = lib.lcvq_pack2bit
    assert p(FAKE, L.SRC_LATENT, L.BF16, 4, 6, FAKE, None) == L.EINVAL        # n % 4
    assert p(FAKE, L.SRC_PACKED2, L.BF16, 4, 8, FAKE, None) == L.EINVAL      # not a pack source
    assert p(FAKE, L.SRC_LATENT, 9, 4, 8, FAKE, None) == L.EINVAL
    assert p(None, L.SRC_LATENT, L.BF16, 4, 8, FAKE, None) == L.EINVAL
    assert p(MIS, L.SRC_LATENT, L.BF16, 4, 8, FAKE, None) == L.EALIGN
    assert p(None, L.SRC_LATENT, L.BF16, 0, 8, None, None) == L.OK
    q = lib.lcvq_dequant
    assert q(4, 8, 3, L.SRC_LATENT, L.BF16, FAKE, FAKE, FAKE, FAKE, L.BF16, None) == L.EUNSUPPORTED
    assert q(4, 12, 8, L.SRC_LATENT, L.BF16, FAKE, FAKE, FAKE, FAKE, L.BF16, None) == L.EINVAL
    assert q(4, 8, 8, 5, L.BF16, FAKE, FAKE, FAKE, FAKE, L.BF16, None) == L.EINVAL
    assert q(4, 8, 8, L.SRC_LATENT, L.BF16, FAKE, None, FAKE, FAKE, L.BF16, None) == L.EINVAL
    assert q(4, 8, 8, L.SRC_LATENT, L.BF16, FAKE, FAKE, FAKE, MIS, L.BF16, None) == L.EALIGN


def test_adamw_validation(lib):
    def a(theta=FAKE, grad=FAKE, gdt=L.BF16, m1=FAKE, m2=FAKE, sh=None, sdt=L.BF16, numel=64, lr=1e-3,
          b1=0.9, b2=0.999, eps=1e-8, wd=0.0, step=1):
        return lib.lcvq_adamw_step(theta, grad, gdt, m1, m2, sh, sdt, numel, lr, b1, b2, eps, wd, step, None)
    assert a(numel=-1) == L.EINVAL
    assert a(gdt=7) == L.EINVAL
    assert a(sh=FAKE, sdt=7) == L.EINVAL
    assert a(step=0) == L.EINVAL
    assert a(b1=1.0) == L.EINVAL
    assert a(b2=-0.1) == L.EINVAL
    assert a(eps=0.0) == L.EINVAL
    assert a(lr=-1.0) == L.EINVAL
    assert a(wd=float("nan")) == L.EINVAL
    assert a(m2=None) == L.EINVAL
    assert a(grad=MIS) == L.EALIGN
    assert a(sh=MIS) == L.EALIGN
    assert a(numel=0, theta=None) == L.OK        # empty: nothing to do


def test_binding_refuses_cpu_tensors():
    torch = pytest.importorskip("torch")
    import paper_2606_10531_amd as lc
    Z = torch.zeros(8, 8)
    with pytest.raises(ValueError, match="GPU"):
        lc.pack2bit(Z)


def test_token_bound(lib):
    # at most 2^22 - 256 tokens per layer call (the weight-gradient operands'
    # 32-bit buffer range); beyond it nothing is enqueued
    big = (1 << 22) - 255
    assert fwd(lib, N=big) == L.EUNSUPPORTED and "tokens" in L.last_error()
    assert bwd(lib, N=big) == L.EUNSUPPORTED
    assert fwd(lib, N=big, dt=L.F32) == L.EUNSUPPORTED
    assert fwd(lib, N=big - 1, wsb=16) == L.EWORKSPACE       # the largest N passes the bound


def test_xavier_quantizer_is_host_arithmetic(lib):
    """eq. xavier_preprocess: (1 / s', t) with s' = 2 sqrt(6 / (m + n)) / 3, t = 3 / 2,
    each rounded to fp32 (host-only call, no GPU needed)."""
    import numpy as np
    import oracle as orc
    qs, qb = ctypes.c_float(), ctypes.c_float()
    for m, n in ((4096, 4096), (28672, 8192), (1, 1)):
        assert lib.lcvq_xavier_quantizer(m, n, ctypes.byref(qs), ctypes.byref(qb)) == L.OK
        sp, t = orc.xavier_params(m, n)
        assert qs.value == float(np.float32(1.0 / sp)) and qb.value == 1.5 == t
    assert lib.lcvq_xavier_quantizer(0, 5, ctypes.byref(qs), ctypes.byref(qb)) == L.EINVAL
    assert lib.lcvq_xavier_quantizer(5, 5, None, ctypes.byref(qb)) == L.EINVAL


def test_xavier_init_validation(lib):
    def x(m=64, n=64, kind=L.SRC_CODES_U8, codes=FAKE, W=FAKE, odt=L.F32):
        return lib.lcvq_xavier_init(m, n, kind, codes, W, odt, None)
    assert x(m=0) == L.EINVAL
    assert x(kind=L.SRC_LATENT) == L.EINVAL
    assert x(n=62) == L.EINVAL                               # n % 4
    assert x(odt=7) == L.EINVAL
    assert x(codes=None) == L.EINVAL
    assert x(W=MIS) == L.EALIGN
    assert x(kind=L.SRC_PACKED2, codes=MIS) == L.EALIGN


def test_binding_checks_shapes_and_dtypes_before_any_call():
    """The torch binding validates every tensor against (N, m, n, d) and the
    activation dtype before it touches the device or the C ABI (checked here with
    CPU tensors: a well-formed call fails only at the device check)."""
    torch = pytest.importorskip("torch")
    import paper_2606_10531_amd as lc
    bf, f32 = torch.bfloat16, torch.float32
    N, m, n, d = 4, 16, 32, 8
    Z, X, dY = torch.zeros(m, n, dtype=bf), torch.zeros(N, n, dtype=bf), torch.zeros(N, m, dtype=bf)
    A, b = torch.zeros(d, d), torch.zeros(d)
    with pytest.raises(ValueError, match="GPU"):               # well formed: reaches the device check
        lc.linear_fwd(Z, A, b, X, d)
    with pytest.raises(ValueError, match="GPU"):
        lc.linear_bwd(Z, A, b, X, dY, d)
    bad_fwd = [dict(X=torch.zeros(N, n + 8, dtype=bf)), dict(X=torch.zeros(N, n, dtype=f32)),
               dict(A=torch.zeros(d, d + 1)), dict(A=torch.zeros(d, d, dtype=bf)), dict(b=torch.zeros(d + 1)),
               dict(out=torch.zeros(N, m + 8, dtype=bf)), dict(out=torch.zeros(N, m, dtype=f32)),
               dict(packed_out=torch.zeros(m, n // 4 + 1, dtype=torch.uint8)),
               dict(packed_out=torch.zeros(m, n // 4, dtype=torch.int8)),
               dict(workspace=torch.zeros(1 << 20, dtype=torch.int32))]
    for kw in bad_fwd:
        args = dict(Z=Z, A=A, b=b, X=X, d=d)
        args.update(kw)
        with pytest.raises((TypeError, ValueError)) as ei:
            lc.linear_fwd(**args)
        assert "GPU" not in str(ei.value), kw
    bad_bwd = [dict(dY=torch.zeros(N, m + 8, dtype=bf)), dict(dY=torch.zeros(N, m, dtype=f32)),
               dict(dX=torch.zeros(N, n, dtype=f32)), dict(dZ=torch.zeros(m, n + 8, dtype=bf)),
               dict(dZ=torch.zeros(m, n, dtype=torch.float16)), dict(dA=torch.zeros(d, d), db=None),
               dict(dA=torch.zeros(d, d), db=torch.zeros(d + 1)), dict(dA=torch.zeros(d, d, dtype=bf),
                                                                      db=torch.zeros(d))]
    for kw in bad_bwd:
        args = dict(Z=Z, A=A, b=b, X=X, dY=dY, d=d)
        args.update(kw)
        with pytest.raises((TypeError, ValueError)) as ei:
            lc.linear_bwd(**args)
        assert "GPU" not in str(ei.value), kw
    P = torch.zeros(m, n // 4, dtype=torch.uint8)
    with pytest.raises(TypeError):
        lc.linear_fwd_packed(P, A, b, torch.zeros(N, n, dtype=f32), d)
    with pytest.raises(ValueError, match="shape"):
        lc.linear_fwd_packed(P, A, b, torch.zeros(N, n + 4, dtype=bf), d)
    with pytest.raises(ValueError, match="shape"):
        lc.dequant(P, A, b, d, n=n + 4, src_kind=lc.SRC_PACKED2)
    with pytest.raises(ValueError, match="shape"):
        lc.xavier_init(P, m, n + 4, src_kind=lc.SRC_PACKED2)
    with pytest.raises(ValueError, match="shape"):
        lc.pack2bit(Z, out=torch.zeros(m, n, dtype=torch.uint8))


def test_training_pair_validation(lib):
    """Saved-state size and alignment are checked before anything is enqueued."""
    N, m, n, d = 16, 64, 64, 8
    need = lib.lcvq_saved_bytes(N, m, n, d, L.BF16)
    assert need >= m * n // 2 + n * 256 * 2                    # codes (4 bits) and X' (bf16, tokens padded)
    assert lib.lcvq_saved_bytes(N, m, n, d, L.F32) == 0
    assert lib.lcvq_saved_bytes(N, m, n, 5, L.BF16) == 0
    assert lib.lcvq_saved_bytes(-1, m, n, d, L.BF16) == 0

    def f(saved=FAKE, nbytes=None):
        return lib.lcvq_linear_fwd_train(N, m, n, d, L.BF16, FAKE, 1.0, 0.0, FAKE, FAKE, FAKE, FAKE, None, saved,
                                         need if nbytes is None else nbytes, FAKE, 1 << 40, None)

    def g(saved=FAKE, nbytes=None, est=L.EST_STE):
        return lib.lcvq_linear_bwd_train(N, m, n, d, L.BF16, FAKE, 1.0, 0.0, FAKE, FAKE, FAKE, FAKE, 0, est, 5.0, 3.0,
                                         0, FAKE, FAKE, L.BF16, FAKE, FAKE, saved,
                                         need if nbytes is None else nbytes, FAKE, 1 << 40, None)
    assert f(nbytes=need - 1) == L.EWORKSPACE and "saved" in L.last_error()
    assert f(saved=None) == L.EWORKSPACE
    assert f(saved=MIS) == L.EALIGN
    assert g(nbytes=need - 1) == L.EWORKSPACE
    assert g(saved=None) == L.EWORKSPACE
    assert g(saved=MIS) == L.EALIGN
    assert g(est=7) == L.EINVAL
    assert f(nbytes=0, saved=None) != L.OK

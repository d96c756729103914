"""Host-side checks of the C ABI: the library loads, exports every entry point
that include/fem.h declares, and rejects bad arguments before launching
anything (no GPU needed: every call here fails validation on the host)."""

import ctypes
import os
import re

import pytest

from paper_2602_07160_amd import binding

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "fem.h")

OK, NULLPTR, SHAPE, UNSUPPORTED, ALIGN, HIPERR, WORKSPACE = range(7)
BF16, F32 = 1, 0


def declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fem_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    return binding.load()


def test_exports_match_header(lib):
    names = declared()
    assert set(names) >= set(binding.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for s in range(7):
        assert binding.fem_status_str(s).startswith(
            ["FEM_OK", "FEM_ERR_NULLPTR", "FEM_ERR_SHAPE", "FEM_ERR_UNSUPPORTED",
             "FEM_ERR_ALIGN", "FEM_ERR_HIP", "FEM_ERR_WORKSPACE"][s])
    assert "UNKNOWN" in binding.fem_status_str(99)


# fake, never-dereferenced device addresses (validation fails first)
A = 1 << 20


def sm(lib, q=A, k=A, v=A, beta=A, out=A, B=1, H=1, T=8, d=64, dt=BF16):
    return lib.fem_softmax_fwd(q, k, v, beta, out, B, H, T, d, dt, None)


def ln(lib, q=A, k=A, v=A, beta=A, out=A, B=1, H=1, T=8, dk=64, dv=64, chunk=64, dt=BF16,
       ws=None, wsb=0):
    return lib.fem_linear_fwd(q, k, v, beta, out, B, H, T, dk, dv, chunk, dt, ws, wsb, None)


def test_softmax_validation(lib):
    assert sm(lib, q=None) == NULLPTR
    assert sm(lib, beta=None) == NULLPTR
    assert sm(lib, out=None) == NULLPTR
    assert sm(lib, T=0) == SHAPE
    assert sm(lib, B=-1) == SHAPE
    assert sm(lib, H=0) == SHAPE
    assert sm(lib, B=1 << 20, H=1 << 20, T=1 << 20) == SHAPE
    for d in (16, 48, 96, 256):
        assert sm(lib, d=d) == UNSUPPORTED
    assert sm(lib, d=300, dt=F32) == UNSUPPORTED
    assert sm(lib, dt=7) == UNSUPPORTED
    assert sm(lib, q=A + 2) == ALIGN
    assert sm(lib, out=A + 4) == ALIGN
    assert sm(lib, v=A + 8, dt=F32) == ALIGN


def test_linear_validation(lib):
    assert ln(lib, k=None) == NULLPTR
    assert ln(lib, T=0) == SHAPE
    assert ln(lib, dk=32) == UNSUPPORTED
    assert ln(lib, dv=128) == UNSUPPORTED
    for c in (0, 8, 48, 96, 256):
        assert ln(lib, chunk=c) == UNSUPPORTED, c
    # chunks 16, 32, 64 and 128 pass the chunk check (another argument fails)
    for c in (16, 32, 64, 128):
        assert ln(lib, chunk=c, dk=32) == UNSUPPORTED
        assert ln(lib, chunk=c, v=A + 2) == ALIGN
    assert ln(lib, dt=F32) == UNSUPPORTED
    assert ln(lib, v=A + 2) == ALIGN


def gt(lib, q=A, k=A, v=A, bmax=A, lam=A, gate=A, out=A, B=1, H=1, T=8, d=64, dt=BF16):
    return lib.fem_softmax_gated_fwd(q, k, v, bmax, lam, gate, out, B, H, T, d, dt, None)


def test_gated_validation(lib):
    assert gt(lib, lam=None) == NULLPTR
    assert gt(lib, bmax=None) == NULLPTR
    assert gt(lib, out=None) == NULLPTR
    assert gt(lib, T=0) == SHAPE
    assert gt(lib, d=48) == UNSUPPORTED
    assert gt(lib, dt=F32) == UNSUPPORTED
    assert gt(lib, lam=A + 4) == ALIGN
    assert gt(lib, gate=A + 8) == ALIGN
    assert gt(lib, gate=None, k=A + 2) == ALIGN


def ex(lib, q=A, k=A, v=A, beta=A, out=A, B=1, H=1, T=8, dqk=64, dv=64, flags=0, dt=BF16):
    return lib.fem_softmax_fwd_ex(q, k, v, beta, out, B, H, T, dqk, dv, flags, dt, None)


def test_ex_validation(lib):
    assert ex(lib, v=None) == NULLPTR
    assert ex(lib, T=-3) == SHAPE
    assert ex(lib, dv=0) == SHAPE
    assert ex(lib, flags=4) == UNSUPPORTED
    assert ex(lib, dt=F32) == UNSUPPORTED
    for dqk, dv in ((64, 128), (128, 32), (96, 48), (256, 128), (16, 16)):
        assert ex(lib, dqk=dqk, dv=dv) == UNSUPPORTED, (dqk, dv)
    assert ex(lib, out=A + 2, flags=3) == ALIGN
    assert ex(lib, dqk=128, dv=64, k=A + 8) == ALIGN


def dec(lib, q=A, k=A, v=A, lens=A, beta=A, out=A, B=1, H=1, L=8, dqk=64, dv=64, dt=BF16,
        ws=None, wsb=0):
    return lib.fem_softmax_decode(q, k, v, lens, beta, out, B, H, L, dqk, dv, dt, ws, wsb, None)


def test_decode_validation(lib):
    assert dec(lib, q=None) == NULLPTR
    assert dec(lib, out=None) == NULLPTR
    assert dec(lib, L=0) == SHAPE
    assert dec(lib, B=70000) == SHAPE
    assert dec(lib, dqk=32, dv=64) == UNSUPPORTED
    assert dec(lib, dt=F32) == UNSUPPORTED
    assert dec(lib, k=A + 4) == ALIGN


def gla(lib, q=A, k=A, v=A, g=A, beta=A, out=A, B=1, H=1, T=8, dk=64, dv=64, chunk=64, dt=BF16,
        ws=None, wsb=0):
    return lib.fem_gla_fwd(q, k, v, g, beta, out, B, H, T, dk, dv, chunk, dt, ws, wsb, None)


def test_gla_validation(lib):
    assert gla(lib, g=None) == NULLPTR
    assert gla(lib, T=0) == SHAPE
    assert gla(lib, dk=128) == UNSUPPORTED
    assert gla(lib, chunk=32) == UNSUPPORTED
    assert gla(lib, dt=F32) == UNSUPPORTED
    assert gla(lib, g=A + 4) == ALIGN


def test_train_and_backward_validation(lib):
    tr = lambda **kw: lib.fem_softmax_fwd_train(*[kw.get(n, A) for n in ("q", "k", "v", "b", "o", "l")],
                                                kw.get("B", 1), 1, 8, kw.get("d", 64), kw.get("dt", BF16), None)
    assert tr(l=None) == NULLPTR
    assert tr(d=96) == UNSUPPORTED
    assert tr(dt=F32) == UNSUPPORTED
    assert tr(o=A + 4) == ALIGN
    names = ("q", "k", "v", "b", "o", "l", "g", "dq", "dk", "dv", "db")
    bw = lambda **kw: lib.fem_softmax_bwd(*[kw.get(n, A) for n in names], kw.get("B", 1), 1, 8,
                                          kw.get("d", 64), kw.get("dt", BF16), kw.get("ws"),
                                          kw.get("wsb", 0), None)
    assert bw(db=None) == NULLPTR
    assert bw(g=None) == NULLPTR
    assert bw(B=0) == SHAPE
    assert bw(d=16) == UNSUPPORTED
    assert bw(dk=A + 8) == ALIGN
    # every size needs a workspace here: none, a short one, a misaligned one
    need = lib.fem_softmax_bwd_workspace_bytes(1, 1, 8, 64)
    assert need > 0
    assert bw() == WORKSPACE
    assert bw(ws=A, wsb=need - 1) == WORKSPACE
    assert bw(ws=A + 16, wsb=need) == ALIGN


# ---- workspace queries: the exact sizes documented in fem.h ----------------

def cdiv(a, b):
    return -(-a // b)


def want_decode(B, H, L, dqk, dv):
    blocks = cdiv(L, 64)
    s0 = max(1, min(cdiv(256, B * H), blocks))
    n = cdiv(blocks, s0)
    return 8 * B * H * cdiv(blocks, n) * (dv + 1)


def want_scan(B, H, T, gla, chunk=64):
    ntile = cdiv(T, max(chunk, 32))
    w = max(1, 512 // (B * H))
    c = cdiv(ntile, w)
    S = cdiv(ntile, c)
    return 0 if S == 1 else 2 * 4 * B * H * S * (4288 if gla else 4224)


def want_bwd(B, H, T, d):
    nbh, n = B * H, cdiv(T, 64)
    tp = 64 * n
    fl = nbh * T + 2 * nbh * d + 5 * nbh * n * d + nbh * T * d + nbh * tp
    return 256 + cdiv(4 * fl, 256) * 256 + 8 * nbh * tp * d


SIZES = [(1, 1, 1), (1, 1, 8), (1, 1, 63), (1, 1, 64), (1, 1, 65), (2, 3, 700), (4, 16, 8192),
         (8, 16, 4096), (1, 8, 16384), (1, 1, 100000), (64, 64, 128), (3, 5, 1000)]


def test_workspace_queries(lib):
    for B, H, T in SIZES:
        for dqk, dv in ((32, 32), (64, 64), (128, 128), (64, 32), (128, 64)):
            assert lib.fem_softmax_decode_workspace_bytes(B, H, T, dqk, dv) == \
                want_decode(B, H, T, dqk, dv), (B, H, T, dqk, dv)
        for c in (16, 32, 64, 128):
            assert lib.fem_linear_workspace_bytes(B, H, T, 64, 64, c) == \
                want_scan(B, H, T, False, c), (B, H, T, c)
        assert lib.fem_gla_workspace_bytes(B, H, T, 64, 64, 64) == want_scan(B, H, T, True)
        for d in (32, 64, 128):
            assert lib.fem_softmax_bwd_workspace_bytes(B, H, T, d) == want_bwd(B, H, T, d)
    # the headline and linear workloads
    assert lib.fem_softmax_bwd_workspace_bytes(8, 16, 4096, 128) == want_bwd(8, 16, 4096, 128)
    assert want_bwd(8, 16, 4096, 128) > 800e6
    assert lib.fem_linear_workspace_bytes(4, 16, 8192, 64, 64, 64) == 2 * 4 * 64 * 8 * 4224
    # arguments outside the supported set give 0
    assert lib.fem_linear_workspace_bytes(4, 16, 8192, 32, 64, 64) == 0
    assert lib.fem_linear_workspace_bytes(4, 16, 8192, 64, 64, 48) == 0
    assert lib.fem_gla_workspace_bytes(4, 16, 8192, 64, 64, 32) == 0
    assert lib.fem_linear_workspace_bytes(0, 16, 8192, 64, 64, 64) == 0
    assert lib.fem_softmax_decode_workspace_bytes(1, 1, 8, 32, 64) == 0
    assert lib.fem_softmax_bwd_workspace_bytes(1, 1, 8, 48) == 0
    assert binding.workspace_bytes("linear", 4, 16, 8192, 64, 64, 64) == want_scan(4, 16, 8192, False)


def test_workspace_errors(lib):
    need = lib.fem_linear_workspace_bytes(4, 16, 8192, 64, 64, 64)
    big = dict(B=4, H=16, T=8192)
    assert ln(lib, **big) == WORKSPACE
    assert ln(lib, **big, ws=A, wsb=need - 1) == WORKSPACE
    assert ln(lib, **big, ws=A + 128, wsb=need) == ALIGN
    assert gla(lib, **big) == WORKSPACE
    needd = lib.fem_softmax_decode_workspace_bytes(8, 16, 4096, 128, 128)
    assert needd > 0
    assert dec(lib, B=8, H=16, L=4096, dqk=128, dv=128) == WORKSPACE
    assert dec(lib, B=8, H=16, L=4096, dqk=128, dv=128, ws=A, wsb=needd - 8) == WORKSPACE
    # the argument checks come first
    assert ln(lib, **big, k=None) == NULLPTR
    assert ln(lib, **big, chunk=48) == UNSUPPORTED


def test_no_pool_in_library():
    """The library allocates nothing: no allocation or pool call in its sources."""
    csrc = os.path.join(os.path.dirname(HEADER), "..", "paper_2602_07160_amd", "csrc")
    for name in os.listdir(csrc):
        src = open(os.path.join(csrc, name)).read()
        for call in ("hipMalloc", "hipFree", "hipMemPool", "hipMallocAsync", "hipHostMalloc"):
            assert call not in src, (name, call)


def test_decode_noalloc_validation(lib):
    na = lambda **kw: lib.fem_softmax_decode_noalloc(
        kw.get("q", A), A, A, A, A, kw.get("out", A), kw.get("B", 1), kw.get("H", 1),
        kw.get("L", 8), kw.get("dqk", 64), kw.get("dv", 64), kw.get("dt", BF16), None)
    assert na(q=None) == NULLPTR
    assert na(L=0) == SHAPE
    assert na(dqk=32, dv=64) == UNSUPPORTED
    assert na(dt=F32) == UNSUPPORTED
    assert na(q=A + 2) == ALIGN
    # partials beyond the fixed 8 MiB array are refused before any launch
    assert want_decode(64, 128, 64, 128, 128) > 8 << 20
    assert na(B=64, H=128, L=64, dqk=128, dv=128) == WORKSPACE
    assert want_decode(63, 129, 64, 128, 128) <= 8 << 20

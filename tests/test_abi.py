"""C-ABI checks that need no GPU: the library loads, exports every symbol
include/laq.h declares, and rejects bad arguments on the host (before any
HIP call, so nothing is launched).  Pointers used here are never
dereferenced: each call fails validation first."""
import ctypes
import os
import re

import pytest

from paper_2605_08755_amd import laq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "laq.h")

FAKE = 0x100000  # 16-byte aligned, never dereferenced


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(laq_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    return laq.lib()


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert len(names) >= 7
    for n in names:
        assert hasattr(L, n), n
    assert set(laq.EXPORTS) == set(names)


def test_version_and_strings(L):
    assert L.laq_abi_version() == 1
    for s in range(0, 6):
        assert L.laq_status_string(s)
    assert L.laq_status_string(99) == b"unknown status"


def _quant(L, bits, w=FAKE, N=4, K=128, q=FAKE, s=FAKE, z=FAKE):
    f = L.laq_quantize_w3g128 if bits == 3 else L.laq_quantize_w4g128
    return f(ctypes.c_void_p(w), N, K, ctypes.c_void_p(q), ctypes.c_void_p(s), ctypes.c_void_p(z), None)


def _pack(L, bits, w=FAKE, s=FAKE, z=FAKE, N=4, K=128, q=FAKE):
    f = L.laq_pack_w3g128 if bits == 3 else L.laq_pack_w4g128
    return f(ctypes.c_void_p(w), ctypes.c_void_p(s), ctypes.c_void_p(z), N, K, ctypes.c_void_p(q), None)


def _lin(L, bits, x=FAKE, q=FAKE, s=FAKE, z=FAKE, y=FAKE, M=1, N=4, K=128):
    f = L.laq_linear_w3g128 if bits == 3 else L.laq_linear_w4g128
    return f(ctypes.c_void_p(x), ctypes.c_void_p(q), ctypes.c_void_p(s), ctypes.c_void_p(z),
             ctypes.c_void_p(y), M, N, K, None)


@pytest.mark.parametrize("bits", [3, 4])
def test_quantize_validation(L, bits):
    assert _quant(L, bits, w=0) == laq.LAQ_ERR_NULL_POINTER
    assert _quant(L, bits, q=0) == laq.LAQ_ERR_NULL_POINTER
    assert _quant(L, bits, s=0) == laq.LAQ_ERR_NULL_POINTER
    assert _quant(L, bits, z=0) == laq.LAQ_ERR_NULL_POINTER
    assert _quant(L, bits, N=0) == laq.LAQ_ERR_BAD_SHAPE
    assert _quant(L, bits, N=-3) == laq.LAQ_ERR_BAD_SHAPE
    assert _quant(L, bits, K=0) == laq.LAQ_ERR_BAD_SHAPE
    assert _quant(L, bits, K=64) == laq.LAQ_ERR_BAD_SHAPE
    assert _quant(L, bits, K=200) == laq.LAQ_ERR_BAD_SHAPE
    assert _quant(L, bits, N=1 << 31) == laq.LAQ_ERR_BAD_SHAPE
    assert _quant(L, bits, N=1 << 30, K=1 << 11) == laq.LAQ_ERR_BAD_SHAPE
    assert _quant(L, bits, w=FAKE + 8) == laq.LAQ_ERR_MISALIGNED
    assert _quant(L, bits, q=FAKE + 4) == laq.LAQ_ERR_MISALIGNED
    assert _quant(L, bits, s=FAKE + 1) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_quantize" in L.laq_last_error()


@pytest.mark.parametrize("bits", [3, 4])
def test_pack_validation(L, bits):
    for kw in ("w", "s", "z", "q"):
        assert _pack(L, bits, **{kw: 0}) == laq.LAQ_ERR_NULL_POINTER
    assert _pack(L, bits, N=0) == laq.LAQ_ERR_BAD_SHAPE
    assert _pack(L, bits, K=96) == laq.LAQ_ERR_BAD_SHAPE
    assert _pack(L, bits, K=1 << 25) == laq.LAQ_ERR_BAD_SHAPE
    assert _pack(L, bits, w=FAKE + 2) == laq.LAQ_ERR_MISALIGNED
    assert _pack(L, bits, q=FAKE + 4) == laq.LAQ_ERR_MISALIGNED
    assert _pack(L, bits, s=FAKE + 1) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_pack" in L.laq_last_error()


def _sw(L, bits, x=FAKE, q=FAKE, s=FAKE, z=FAKE, y=FAKE, M=1, N=4, K=128):
    f = L.laq_linear_swiglu_w3g128 if bits == 3 else L.laq_linear_swiglu_w4g128
    return f(ctypes.c_void_p(x), ctypes.c_void_p(q), ctypes.c_void_p(s), ctypes.c_void_p(z),
             ctypes.c_void_p(y), M, N, K, None)


@pytest.mark.parametrize("bits", [3, 4])
def test_linear_swiglu_validation(L, bits):
    for kw in ("x", "q", "s", "z", "y"):
        assert _sw(L, bits, **{kw: 0}) == laq.LAQ_ERR_NULL_POINTER
    assert _sw(L, bits, M=0) == laq.LAQ_ERR_BAD_M
    assert _sw(L, bits, M=5) == laq.LAQ_ERR_BAD_M
    assert _sw(L, bits, N=3) == laq.LAQ_ERR_BAD_SHAPE     # rows come in (gate, up) pairs
    assert _sw(L, bits, K=127) == laq.LAQ_ERR_BAD_SHAPE
    assert _sw(L, bits, K=16384 + 128) == laq.LAQ_ERR_BAD_SHAPE
    assert _sw(L, bits, M=2, K=8192 + 128) == laq.LAQ_ERR_BAD_SHAPE
    assert _sw(L, bits, M=3, K=4096 + 128) == laq.LAQ_ERR_BAD_SHAPE
    assert _sw(L, bits, x=FAKE + 2) == laq.LAQ_ERR_MISALIGNED
    assert _sw(L, bits, y=FAKE + 1) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_linear_swiglu" in L.laq_last_error()


def _nl(L, bits, swiglu=False, r=FAKE, d=FAKE, w=FAKE, eps=1e-6, ro=FAKE + 0x10000, q=FAKE, s=FAKE, z=FAKE,
        y=FAKE, N=4, K=128):
    f = {(3, False): L.laq_add_rmsnorm_linear_w3g128, (4, False): L.laq_add_rmsnorm_linear_w4g128,
         (3, True): L.laq_add_rmsnorm_linear_swiglu_w3g128, (4, True): L.laq_add_rmsnorm_linear_swiglu_w4g128}[
        (bits, swiglu)]
    return f(ctypes.c_void_p(r), ctypes.c_void_p(d), ctypes.c_void_p(w), ctypes.c_float(eps), ctypes.c_void_p(ro),
             ctypes.c_void_p(q), ctypes.c_void_p(s), ctypes.c_void_p(z), ctypes.c_void_p(y), N, K, None)


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("swiglu", [False, True])
def test_add_rmsnorm_linear_validation(L, bits, swiglu):
    for kw in ("r", "w", "q", "s", "z", "y"):
        assert _nl(L, bits, swiglu, **{kw: 0}) == laq.LAQ_ERR_NULL_POINTER
    assert _nl(L, bits, swiglu, N=0) == laq.LAQ_ERR_BAD_SHAPE
    assert _nl(L, bits, swiglu, K=127) == laq.LAQ_ERR_BAD_SHAPE
    assert _nl(L, bits, swiglu, K=8192 + 128) == laq.LAQ_ERR_BAD_SHAPE   # the row must fit one staging pass
    assert _nl(L, bits, swiglu, eps=-1.0) == laq.LAQ_ERR_BAD_SHAPE
    assert _nl(L, bits, swiglu, eps=float("inf")) == laq.LAQ_ERR_BAD_SHAPE
    assert _nl(L, bits, swiglu, ro=FAKE) == laq.LAQ_ERR_BAD_SHAPE         # residual_out == residual
    assert _nl(L, bits, swiglu, ro=FAKE + 4 * 128 - 16) == laq.LAQ_ERR_BAD_SHAPE  # overlapping
    if swiglu:
        assert _nl(L, bits, swiglu, N=3) == laq.LAQ_ERR_BAD_SHAPE
    for kw in ("r", "d", "w", "ro", "q"):
        assert _nl(L, bits, swiglu, **{kw: (FAKE + 0x20000 if kw == "ro" else FAKE) + 8}) == laq.LAQ_ERR_MISALIGNED
    assert _nl(L, bits, swiglu, s=FAKE + 1) == laq.LAQ_ERR_MISALIGNED
    assert _nl(L, bits, swiglu, y=FAKE + 1) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_add_rmsnorm_linear" in L.laq_last_error()


def _lres(L, bits, x=FAKE, q=FAKE, s=FAKE, z=FAKE, y=FAKE, ri=FAKE, ro=FAKE + 0x10000, N=2560, K=4096):
    f = L.laq_linear_residual_w3g128 if bits == 3 else L.laq_linear_residual_w4g128
    return f(ctypes.c_void_p(x), ctypes.c_void_p(q), ctypes.c_void_p(s), ctypes.c_void_p(z), ctypes.c_void_p(y),
             ctypes.c_void_p(ri), ctypes.c_void_p(ro), N, K, None)


@pytest.mark.parametrize("bits", [3, 4])
def test_linear_residual_validation(L, bits):
    for kw in ("x", "q", "s", "z", "ri", "ro"):
        assert _lres(L, bits, **{kw: 0}) == laq.LAQ_ERR_NULL_POINTER
    assert _lres(L, bits, y=0, N=0) == laq.LAQ_ERR_BAD_SHAPE          # y may be NULL (only the residual written)
    assert _lres(L, bits, y=FAKE + 1) == laq.LAQ_ERR_MISALIGNED
    assert _lres(L, bits, N=0) == laq.LAQ_ERR_BAD_SHAPE
    assert _lres(L, bits, K=1920) == laq.LAQ_ERR_BAD_SHAPE          # fewer than 16 groups
    assert _lres(L, bits, K=32768) == laq.LAQ_ERR_BAD_SHAPE         # activation tile past the LDS budget
    assert _lres(L, bits, ro=FAKE + 4 * 100) == laq.LAQ_ERR_BAD_SHAPE  # partial overlap
    assert _lres(L, bits, x=FAKE + 8) == laq.LAQ_ERR_MISALIGNED
    assert _lres(L, bits, s=FAKE + 1) == laq.LAQ_ERR_MISALIGNED
    assert _lres(L, bits, ri=FAKE + 2) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_linear_residual" in L.laq_last_error()


def _mlp(L, r=FAKE, d=FAKE, w=FAKE, eps=1e-6, ro=FAKE + 0x10000, gq=FAKE, gs=FAKE, gz=FAKE, dq=FAKE, ds=FAKE,
         dz=FAKE, y=FAKE, D=256, I=384, ws=FAKE, ws_bytes=1 << 20):
    return L.laq_add_rmsnorm_mlp_w3g128(
        ctypes.c_void_p(r), ctypes.c_void_p(d), ctypes.c_void_p(w), ctypes.c_float(eps), ctypes.c_void_p(ro),
        ctypes.c_void_p(gq), ctypes.c_void_p(gs), ctypes.c_void_p(gz), ctypes.c_void_p(dq), ctypes.c_void_p(ds),
        ctypes.c_void_p(dz), ctypes.c_void_p(y), D, I, ctypes.c_void_p(ws), ws_bytes, None)


def test_add_rmsnorm_mlp_validation(L):
    # workspace: fp32 partials [I/128][D] and team sums, then the counters
    S = 3
    T = 2  # about sqrt(S) teams
    assert L.laq_mlp_workspace_bytes(256, 384) == ((S + T) * 256 * 4 + (T + 1) * 4 + 15) // 16 * 16
    assert L.laq_mlp_workspace_bytes(2560, 9728) > 0
    assert L.laq_mlp_workspace_bytes(2560 + 128, 9728) == 0   # D past the register budget
    assert L.laq_mlp_workspace_bytes(256, 100) == 0
    for kw in ("r", "w", "gq", "gs", "gz", "dq", "ds", "dz", "y", "ws"):
        assert _mlp(L, **{kw: 0}) == laq.LAQ_ERR_NULL_POINTER
    assert _mlp(L, D=200) == laq.LAQ_ERR_BAD_SHAPE
    assert _mlp(L, I=0) == laq.LAQ_ERR_BAD_SHAPE
    assert _mlp(L, D=2688) == laq.LAQ_ERR_BAD_SHAPE
    assert _mlp(L, eps=-1.0) == laq.LAQ_ERR_BAD_SHAPE
    assert _mlp(L, ro=FAKE) == laq.LAQ_ERR_BAD_SHAPE                   # residual_out == residual
    assert _mlp(L, ws_bytes=L.laq_mlp_workspace_bytes(256, 384) - 16) == laq.LAQ_ERR_BAD_SHAPE
    for kw in ("r", "d", "w", "ro", "gq", "dq", "ws"):
        assert _mlp(L, **{kw: (FAKE + 0x20000 if kw == "ro" else FAKE) + 8}) == laq.LAQ_ERR_MISALIGNED
    for kw in ("gs", "ds", "y"):
        assert _mlp(L, **{kw: FAKE + 1}) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_add_rmsnorm_mlp" in L.laq_last_error()


@pytest.mark.parametrize("bits", [3, 4])
def test_linear_validation(L, bits):
    for kw in ("x", "q", "s", "z", "y"):
        assert _lin(L, bits, **{kw: 0}) == laq.LAQ_ERR_NULL_POINTER
    assert _lin(L, bits, M=0) == laq.LAQ_ERR_BAD_M
    assert _lin(L, bits, M=17) == laq.LAQ_ERR_BAD_M
    assert _lin(L, bits, M=-1) == laq.LAQ_ERR_BAD_M
    assert _lin(L, bits, N=0) == laq.LAQ_ERR_BAD_SHAPE
    assert _lin(L, bits, K=127) == laq.LAQ_ERR_BAD_SHAPE
    assert _lin(L, bits, K=384 + 32) == laq.LAQ_ERR_BAD_SHAPE
    assert _lin(L, bits, x=FAKE + 2) == laq.LAQ_ERR_MISALIGNED
    assert _lin(L, bits, q=FAKE + 8) == laq.LAQ_ERR_MISALIGNED
    assert _lin(L, bits, s=FAKE + 1) == laq.LAQ_ERR_MISALIGNED
    assert _lin(L, bits, y=FAKE + 1) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_linear" in L.laq_last_error()


@pytest.mark.parametrize("bits", [3, 4])
def test_group_validation(L, bits):
    f = L.laq_linear_group_w3g128 if bits == 3 else L.laq_linear_group_w4g128

    def calls(n, **kw):
        arr = (laq.LinearCall * max(n, 1))()
        for i in range(n):
            d = dict(x=FAKE, qweight=FAKE, scales=FAKE, zeros=FAKE, y=FAKE, N=4, K=128)
            if i == n - 1:
                d.update(kw)
            arr[i] = laq.LinearCall(d["x"], d["qweight"], d["scales"], d["zeros"], d["y"], d["N"], d["K"])
        return arr

    assert f(None, 1, 1, None) == laq.LAQ_ERR_NULL_POINTER
    assert f(calls(1), 0, 1, None) == laq.LAQ_ERR_BAD_SHAPE
    assert f(calls(9), 9, 1, None) == laq.LAQ_ERR_BAD_SHAPE
    assert f(calls(2), 2, 0, None) == laq.LAQ_ERR_BAD_M
    assert f(calls(2), 2, 17, None) == laq.LAQ_ERR_BAD_M
    for kw in ("x", "qweight", "scales", "zeros", "y"):
        assert f(calls(3, **{kw: 0}), 3, 1, None) == laq.LAQ_ERR_NULL_POINTER
    assert f(calls(2, K=100), 2, 1, None) == laq.LAQ_ERR_BAD_SHAPE
    assert f(calls(2, N=0), 2, 1, None) == laq.LAQ_ERR_BAD_SHAPE
    assert f(calls(2, x=FAKE + 2), 2, 1, None) == laq.LAQ_ERR_MISALIGNED
    assert f(calls(2, y=FAKE + 1), 2, 1, None) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_linear_group" in L.laq_last_error()


def _lin_ws(L, bits, x=FAKE, q=FAKE, s=FAKE, z=FAKE, y=FAKE, M=4, N=4, K=128, ws=FAKE, wsb=1024):
    f = L.laq_linear_ws_w3g128 if bits == 3 else L.laq_linear_ws_w4g128
    return f(ctypes.c_void_p(x), ctypes.c_void_p(q), ctypes.c_void_p(s), ctypes.c_void_p(z),
             ctypes.c_void_p(y), M, N, K, ctypes.c_void_p(ws), wsb, None)


@pytest.mark.parametrize("bits", [3, 4])
def test_linear_ws_validation(L, bits):
    for kw in ("x", "q", "s", "z", "y"):
        assert _lin_ws(L, bits, **{kw: 0}) == laq.LAQ_ERR_NULL_POINTER
    assert _lin_ws(L, bits, ws=0, wsb=16) == laq.LAQ_ERR_NULL_POINTER
    assert _lin_ws(L, bits, wsb=-1) == laq.LAQ_ERR_BAD_SHAPE
    assert _lin_ws(L, bits, M=0) == laq.LAQ_ERR_BAD_M
    assert _lin_ws(L, bits, M=17) == laq.LAQ_ERR_BAD_M
    assert _lin_ws(L, bits, K=200) == laq.LAQ_ERR_BAD_SHAPE
    assert _lin_ws(L, bits, x=FAKE + 2) == laq.LAQ_ERR_MISALIGNED
    assert _lin_ws(L, bits, y=FAKE + 1) == laq.LAQ_ERR_MISALIGNED
    assert _lin_ws(L, bits, ws=FAKE + 8) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_linear_ws" in L.laq_last_error()


def _lin_na(L, x=FAKE, q=FAKE, s=FAKE, z=FAKE, y=FAKE, M=2, N=4, K=128):
    return L.laq_linear_noalloc_w3g128(ctypes.c_void_p(x), ctypes.c_void_p(q), ctypes.c_void_p(s),
                                       ctypes.c_void_p(z), ctypes.c_void_p(y), M, N, K, None)


def test_linear_noalloc_validation(L):
    """The no-allocation linear validates like laq_linear_w3g128 and rejects,
    on the host, shapes whose split-K partial sums exceed its scratch array."""
    for kw in ("x", "q", "s", "z", "y"):
        assert _lin_na(L, **{kw: 0}) == laq.LAQ_ERR_NULL_POINTER
    assert _lin_na(L, M=0) == laq.LAQ_ERR_BAD_M
    assert _lin_na(L, M=17) == laq.LAQ_ERR_BAD_M
    assert _lin_na(L, K=200) == laq.LAQ_ERR_BAD_SHAPE
    assert _lin_na(L, x=FAKE + 2) == laq.LAQ_ERR_MISALIGNED
    assert _lin_na(L, y=FAKE + 1) == laq.LAQ_ERR_MISALIGNED
    # 410 K ranges x 16 x 16000 fp32 partials = 420 MB > 8 MiB of scratch
    need = L.laq_linear_workspace_bytes(16, 16000, 1 << 20)
    assert need > laq.NOALLOC_SCRATCH_BYTES
    assert _lin_na(L, M=16, N=16000, K=1 << 20) == laq.LAQ_ERR_BAD_SHAPE
    assert b"scratch" in L.laq_last_error()
    # the largest split of the Qwen3-32B stack (down projection, M = 16) fits
    assert 0 < L.laq_linear_workspace_bytes(16, 5120, 25600) <= laq.NOALLOC_SCRATCH_BYTES


def test_workspace_bytes(L):
    """The workspace holds S fp32 partial planes of M x N, one per K range of
    at most five quads (512-column blocks), when the row has at least 40 quads
    and fewer than 1024 row tiles (M >= 2); 0 otherwise and for invalid
    shapes."""
    f = L.laq_linear_workspace_bytes
    for (M, N, K) in [(16, 5120, 25600), (3, 100, 25088), (16, 3, 1 << 24), (8, 16368, 25600), (2, 5120, 20480),
                      (16, 1030, 20480)]:
        nq = -(-K // 512)
        b = f(M, N, K)
        assert b > 0 and b % (M * N * 4) == 0, (M, N, K)
        S = b // (M * N * 4)
        assert -(-nq // 5) <= S <= nq, (M, N, K, S)
        qs = -(-nq // S)  # quads per range
        assert -(-nq // qs) == S, (M, N, K, S)
    assert f(16, 5120, 25600) == 10 * 16 * 5120 * 4  # 80 blocks of four tiles x 10 ranges of 5 quads
    assert f(1, 5120, 25600) == 0         # one row: the VALU GEMV, no split
    assert f(16, 16384, 25600) == 0       # >= 1024 row tiles: blocks of several tiles
    assert f(16, 5120, 19968) == 0        # 39 quads
    assert f(16, 2560, 9728) == 0
    for (M, N, K) in [(0, 4, 128), (17, 4, 128), (4, 0, 128), (4, 4, 100), (4, 4, 1 << 25), (4, 1 << 31, 128)]:
        assert f(M, N, K) == 0


def test_shape_check_precedes_m_check(L):
    # a bad shape is reported even when M is also bad
    assert _lin(L, 3, M=0, K=100) == laq.LAQ_ERR_BAD_SHAPE


def test_packed_sizes():
    # 32 three-bit codes in three words: N*K*3/32 words; W4: N*K/8 words
    assert laq.packed_words(3, 1024, 1024) * 4 == 1024 * 1024 * 3 // 8
    assert laq.packed_words(4, 1024, 1024) * 4 == 1024 * 1024 // 2


# --- decode-step operations -------------------------------------------------
def _norm(L, r=FAKE, d=FAKE, w=FAKE, y=FAKE, M=1, D=2560, eps=1e-6):
    return L.laq_add_rmsnorm_f16(ctypes.c_void_p(r), ctypes.c_void_p(d) if d else None, ctypes.c_void_p(w),
                                 ctypes.c_void_p(y), M, D, eps, None)


def _rope(L, qkv=FAKE, qw=FAKE, kw=FAKE, cs=FAKE, pos=0, Hq=32, Hkv=8, hd=128, eps=1e-6, q=FAKE, kc=FAKE,
          vc=FAKE, S=1024):
    return L.laq_qk_norm_rope_f16(ctypes.c_void_p(qkv), ctypes.c_void_p(qw), ctypes.c_void_p(kw), ctypes.c_void_p(cs),
                                  pos, Hq, Hkv, hd, eps, ctypes.c_void_p(q), ctypes.c_void_p(kc), ctypes.c_void_p(vc),
                                  S, None)


def _attn(L, q=FAKE, kc=FAKE, vc=FAKE, Hq=32, Hkv=8, hd=128, Lp=100, S=1024, out=FAKE, ws=FAKE, wsb=1 << 20):
    return L.laq_decode_attention_f16(ctypes.c_void_p(q), ctypes.c_void_p(kc), ctypes.c_void_p(vc), Hq, Hkv, hd, Lp,
                                      S, ctypes.c_void_p(out), ctypes.c_void_p(ws), wsb, None)


def test_decode_ops_validation(L):
    for kw in ("r", "w", "y"):
        assert _norm(L, **{kw: 0}) == laq.LAQ_ERR_NULL_POINTER
    assert _norm(L, M=0) == laq.LAQ_ERR_BAD_SHAPE
    assert _norm(L, D=0) == laq.LAQ_ERR_BAD_SHAPE
    assert _norm(L, D=(1 << 20) + 1) == laq.LAQ_ERR_BAD_SHAPE
    assert _norm(L, eps=-1.0) == laq.LAQ_ERR_BAD_SHAPE
    assert _norm(L, eps=float("nan")) == laq.LAQ_ERR_BAD_SHAPE
    assert _norm(L, r=FAKE + 2) == laq.LAQ_ERR_MISALIGNED
    assert _norm(L, d=FAKE + 1) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_add_rmsnorm_f16" in L.laq_last_error()

    for kw in ("qkv", "qw", "kw", "cs", "q", "kc", "vc"):
        assert _rope(L, **{kw: 0}) == laq.LAQ_ERR_NULL_POINTER
    assert _rope(L, hd=64) == laq.LAQ_ERR_BAD_SHAPE
    assert _rope(L, Hq=24) == laq.LAQ_ERR_BAD_SHAPE      # ratio 3
    assert _rope(L, Hq=128) == laq.LAQ_ERR_BAD_SHAPE     # ratio 16
    assert _rope(L, Hkv=0) == laq.LAQ_ERR_BAD_SHAPE
    assert _rope(L, pos=1024) == laq.LAQ_ERR_BAD_SHAPE
    assert _rope(L, pos=-1) == laq.LAQ_ERR_BAD_SHAPE
    assert _rope(L, S=(1 << 21) + 1) == laq.LAQ_ERR_BAD_SHAPE
    assert _rope(L, kc=FAKE + 8) == laq.LAQ_ERR_MISALIGNED
    assert _rope(L, cs=FAKE + 2) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_qk_norm_rope_f16" in L.laq_last_error()

    for kw in ("q", "kc", "vc", "out", "ws"):
        assert _attn(L, **{kw: 0}) == laq.LAQ_ERR_NULL_POINTER
    assert _attn(L, hd=256) == laq.LAQ_ERR_BAD_SHAPE
    assert _attn(L, Hq=40) == laq.LAQ_ERR_BAD_SHAPE
    assert _attn(L, Lp=0) == laq.LAQ_ERR_BAD_SHAPE
    assert _attn(L, Lp=1025) == laq.LAQ_ERR_BAD_SHAPE
    need = L.laq_decode_attention_workspace_bytes(32, 100)
    assert need == 32 * 2 * 130 * 4  # two blocks of 64 positions, (m, l, 128 sums) in fp32
    assert _attn(L, wsb=need - 1) == laq.LAQ_ERR_BAD_SHAPE
    assert _attn(L, ws=FAKE + 8) == laq.LAQ_ERR_MISALIGNED
    assert _attn(L, vc=FAKE + 8) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_decode_attention_f16" in L.laq_last_error()
    assert L.laq_decode_attention_workspace_bytes(0, 5) == 0
    assert L.laq_decode_attention_workspace_bytes(8, 64) == 8 * 1 * 130 * 4
    assert L.laq_decode_attention_workspace_bytes(8, 65) == 8 * 2 * 130 * 4

    f = L.laq_silu_mul_f16
    assert f(None, ctypes.c_void_p(FAKE), 1, 8, None) == laq.LAQ_ERR_NULL_POINTER
    assert f(ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE), 0, 8, None) == laq.LAQ_ERR_BAD_SHAPE
    assert f(ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE), 1, 0, None) == laq.LAQ_ERR_BAD_SHAPE
    assert f(ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE), 65536, 8, None) == laq.LAQ_ERR_BAD_SHAPE
    assert f(ctypes.c_void_p(FAKE + 1), ctypes.c_void_p(FAKE), 1, 8, None) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_silu_mul_f16" in L.laq_last_error()


def _attn_qkv(L, qkv=FAKE, qw=FAKE, kw=FAKE, cs=FAKE, pos=100, Hq=32, Hkv=8, hd=128, eps=1e-6, kc=FAKE, vc=FAKE,
              S=1024, out=FAKE, ws=FAKE, wsb=1 << 24):
    P = ctypes.c_void_p
    return L.laq_decode_attention_qkv_f16(P(qkv), P(qw), P(kw), P(cs), pos, Hq, Hkv, hd, eps, P(kc), P(vc), S,
                                          P(out), P(ws), wsb, None)


def test_attention_qkv_validation(L):
    for kw in ("qkv", "qw", "kw", "cs", "kc", "vc", "out", "ws"):
        assert _attn_qkv(L, **{kw: 0}) == laq.LAQ_ERR_NULL_POINTER
    assert _attn_qkv(L, hd=64) == laq.LAQ_ERR_BAD_SHAPE
    assert _attn_qkv(L, Hq=24) == laq.LAQ_ERR_BAD_SHAPE
    assert _attn_qkv(L, pos=1024) == laq.LAQ_ERR_BAD_SHAPE
    assert _attn_qkv(L, pos=-1) == laq.LAQ_ERR_BAD_SHAPE
    assert _attn_qkv(L, eps=float("inf")) == laq.LAQ_ERR_BAD_SHAPE
    need = L.laq_decode_attention_qkv_workspace_bytes(32, 8, 101)
    assert _attn_qkv(L, wsb=need - 1) == laq.LAQ_ERR_BAD_SHAPE
    assert _attn_qkv(L, ws=FAKE + 4) == laq.LAQ_ERR_MISALIGNED
    assert _attn_qkv(L, kc=FAKE + 2) == laq.LAQ_ERR_MISALIGNED
    assert b"laq_decode_attention_qkv_f16" in L.laq_last_error()


def test_attention_qkv_workspace_bytes(L):
    """Tiles of 16 positions while Hkv * L < 4096, 32 below 32768, then 64;
    the query is the maximum over every context up to L, so a workspace
    sized for S_max serves every decoded position."""
    f = L.laq_decode_attention_qkv_workspace_bytes
    per = 130 * 4
    assert f(32, 8, 100) == 32 * 7 * per            # 100 positions in tiles of 16
    assert f(32, 8, 511) == 32 * 32 * per           # 511 in tiles of 16 (32 tiles)
    assert f(32, 8, 1024) == 32 * 32 * per          # 1024 in tiles of 32; 511 needed as many
    assert f(32, 8, 4095) == 32 * 128 * per         # 4095 in tiles of 32
    assert f(32, 8, 4096) == 32 * 128 * per         # 4096 in tiles of 64 (64 tiles) < 4095's 128
    assert f(32, 8, 1 << 20) == 32 * (1 << 14) * per
    for bad in ((0, 8, 10), (32, 0, 10), (32, 64, 10), (32, 8, 0), (32, 8, (1 << 21) + 1)):
        assert f(*bad) == 0
    prev = 0
    for Lp in range(1, 5000, 7):  # nondecreasing in L
        b = f(32, 8, Lp)
        assert b >= prev
        prev = b

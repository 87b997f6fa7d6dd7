"""CPU oracle for the W3G128 / W4G128 quantize + linear path.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
CPU-baseline leg of the benchmark, never by the library.  It shares no code
with the HIP path; the C source (laq_oracle.c) restates Eq. 1 of the paper and
the packed-format definition, and this module only marshals numpy arrays.
"""
import ctypes
import os

import numpy as np

from . import build as _build


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p)


class Oracle:
    """ctypes view of one build of laq_oracle.c (the default build, or a
    deliberately mutated copy used to show that the pins catch mistakes)."""

    def __init__(self, lib_path: str):
        L = ctypes.CDLL(lib_path)
        P = ctypes.c_void_p
        I64 = ctypes.c_int64
        L.laqo_quantize.argtypes = [P, I64, I64, ctypes.c_int, P, P, P]
        L.laqo_quantize.restype = None
        L.laqo_codes_from_params.argtypes = [P, I64, I64, ctypes.c_int, P, P, P]
        L.laqo_codes_from_params.restype = None
        L.laqo_pack.argtypes = [P, I64, I64, ctypes.c_int, P]
        L.laqo_pack.restype = ctypes.c_int
        L.laqo_unpack.argtypes = [P, I64, I64, ctypes.c_int, P]
        L.laqo_unpack.restype = None
        L.laqo_dequant.argtypes = [P, P, P, I64, I64, P]
        L.laqo_dequant.restype = None
        L.laqo_linear.argtypes = [P, I64, P, P, P, I64, I64, P]
        L.laqo_linear.restype = None
        L.laqo_f16_to_f32_array.argtypes = [P, I64, P]
        L.laqo_f16_to_f32_array.restype = None
        L.laqo_f32_to_f16_array.argtypes = [P, I64, P]
        L.laqo_f32_to_f16_array.restype = None
        L.laqo_num_threads.argtypes = []
        L.laqo_num_threads.restype = ctypes.c_int
        self.lib = L
        self.path = lib_path

    # -- fp16 helpers -------------------------------------------------------
    def f16_to_f32(self, h):
        h = np.ascontiguousarray(np.asarray(h, dtype=np.uint16))
        out = np.empty(h.shape, np.float32)
        self.lib.laqo_f16_to_f32_array(_p(h), h.size, _p(out))
        return out

    def f32_to_f16(self, v):
        v = np.ascontiguousarray(np.asarray(v, dtype=np.float32))
        out = np.empty(v.shape, np.uint16)
        self.lib.laqo_f32_to_f16_array(_p(v), v.size, _p(out))
        return out

    # -- quantize / pack ----------------------------------------------------
    def quantize(self, w, bits=3):
        """Eq. 1 with round-to-nearest min-max parameters per 128-group.

        w: fp16 [N][K] (np.float16 or its uint16 bits).  Returns (codes uint8
        [N][K], scales fp16 bits uint16 [N][K/128], zeros uint8 [N][K/128]).
        """
        w = np.ascontiguousarray(w)
        if w.dtype == np.float16:
            w = w.view(np.uint16)
        assert w.dtype == np.uint16 and w.ndim == 2
        N, K = w.shape
        assert K % 128 == 0 and K >= 128
        codes = np.empty((N, K), np.uint8)
        scales = np.empty((N, K // 128), np.uint16)
        zeros = np.empty((N, K // 128), np.uint8)
        self.lib.laqo_quantize(_p(w), N, K, bits, _p(codes), _p(scales), _p(zeros))
        return codes, scales, zeros

    def codes_from_params(self, w, scales, zeros, bits=3):
        """Eq. 1 with caller-supplied parameters: codes uint8 [N][K] from fp16
        w [N][K], fp16 scales (bits or np.float16) [N][K/128] and uint8 zeros."""
        w = np.ascontiguousarray(w)
        if w.dtype == np.float16:
            w = w.view(np.uint16)
        scales = np.ascontiguousarray(scales)
        if scales.dtype == np.float16:
            scales = scales.view(np.uint16)
        zeros = np.ascontiguousarray(zeros, dtype=np.uint8)
        assert w.dtype == np.uint16 and w.ndim == 2 and scales.dtype == np.uint16
        N, K = w.shape
        assert K % 128 == 0 and K >= 128
        assert scales.shape == (N, K // 128) and zeros.shape == (N, K // 128)
        codes = np.empty((N, K), np.uint8)
        self.lib.laqo_codes_from_params(_p(w), N, K, bits, _p(scales), _p(zeros), _p(codes))
        return codes

    def pack(self, codes, bits=3):
        """codes uint8 [N][K] -> qweight uint32 [N][bits][K/32] (library layout)."""
        codes = np.ascontiguousarray(codes, dtype=np.uint8)
        N, K = codes.shape
        q = np.empty((N, bits, K // 32), np.uint32)
        if self.lib.laqo_pack(_p(codes), N, K, bits, _p(q)) != 0:
            raise ValueError("code out of range for %d bits" % bits)
        return q

    def unpack(self, qweight, K, bits=3):
        qweight = np.ascontiguousarray(qweight, dtype=np.uint32)
        N = qweight.size // (bits * (K // 32))
        codes = np.empty((N, K), np.uint8)
        self.lib.laqo_unpack(_p(qweight), N, K, bits, _p(codes))
        return codes

    # -- dequant / linear ---------------------------------------------------
    def dequant(self, codes, scales, zeros):
        codes = np.ascontiguousarray(codes, dtype=np.uint8)
        scales = np.ascontiguousarray(scales, dtype=np.uint16)
        zeros = np.ascontiguousarray(zeros, dtype=np.uint8)
        N, K = codes.shape
        out = np.empty((N, K), np.float64)
        self.lib.laqo_dequant(_p(codes), _p(scales), _p(zeros), N, K, _p(out))
        return out

    def linear(self, x, codes, scales, zeros):
        """y[m][n] = sum_k x[m][k] * s[n][k/128] * (q[n][k] - z[n][k/128]), fp64."""
        x = np.ascontiguousarray(x)
        if x.dtype == np.float16:
            x = x.view(np.uint16)
        assert x.dtype == np.uint16
        codes = np.ascontiguousarray(codes, dtype=np.uint8)
        scales = np.ascontiguousarray(scales, dtype=np.uint16)
        zeros = np.ascontiguousarray(zeros, dtype=np.uint8)
        M, K = x.shape
        N = codes.shape[0]
        assert codes.shape == (N, K)
        y = np.empty((M, N), np.float64)
        self.lib.laqo_linear(_p(x), M, _p(codes), _p(scales), _p(zeros), N, K, _p(y))
        return y

    def num_threads(self):
        return self.lib.laqo_num_threads()


_default = None


def default() -> Oracle:
    global _default
    if _default is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _default = Oracle(_build.LIB)
    return _default


def quantize(w, bits=3):
    return default().quantize(w, bits)


def codes_from_params(w, scales, zeros, bits=3):
    return default().codes_from_params(w, scales, zeros, bits)


def pack(codes, bits=3):
    return default().pack(codes, bits)


def unpack(qweight, K, bits=3):
    return default().unpack(qweight, K, bits)


def dequant(codes, scales, zeros):
    return default().dequant(codes, scales, zeros)


def linear(x, codes, scales, zeros):
    return default().linear(x, codes, scales, zeros)


def f16_to_f32(h):
    return default().f16_to_f32(h)


def f32_to_f16(v):
    return default().f32_to_f16(v)


def num_threads():
    return default().num_threads()

"""laq_linear_noalloc_w3g128 (split-K partial sums in the library's own
per-GPU scratch array, nothing allocated) against laq_linear_ws_w3g128 with a
caller workspace, through the C ABI.  Two calls in a row, the second on a
smaller shape, then the first shape again: each result is bitwise equal to
the workspace entry point's and within the linear tolerance of the oracle
(sampled rows at the large shape)."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from oracle.compare import linear_check
from paper_2605_08755_amd import inputs, laq

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def say(*a):
    print("[gpu-case]", *a, flush=True)


def _case(M, N, K, cfg):
    w = inputs.weights(N, K, cfg=cfg)
    x = inputs.activations(M, K, cfg=cfg)
    codes, s, z = oracle.quantize(w, 3)
    q = torch.from_numpy(oracle.pack(codes, 3).view(np.int32)).to(DEV)
    return x, codes, s, z, q, torch.from_numpy(s.view(np.float16)).to(DEV), torch.from_numpy(z).to(DEV)


def _noalloc(xd, q, sd, zd, M, N, K):
    L = laq.lib()
    y = torch.full((M, N), float("nan"), dtype=torch.float16, device=DEV)
    st = L.laq_linear_noalloc_w3g128(ctypes.c_void_p(xd.data_ptr()), ctypes.c_void_p(q.data_ptr()),
                                     ctypes.c_void_p(sd.data_ptr()), ctypes.c_void_p(zd.data_ptr()),
                                     ctypes.c_void_p(y.data_ptr()), M, N, K,
                                     ctypes.c_void_p(torch.cuda.current_stream(DEV).cuda_stream))
    assert st == laq.LAQ_OK, L.laq_last_error()
    return y


def _ws(xd, q, sd, zd, M, N, K):
    L = laq.lib()
    nbytes = L.laq_linear_workspace_bytes(M, N, K)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=DEV)
    y = torch.full((M, N), float("nan"), dtype=torch.float16, device=DEV)
    st = L.laq_linear_ws_w3g128(ctypes.c_void_p(xd.data_ptr()), ctypes.c_void_p(q.data_ptr()),
                                ctypes.c_void_p(sd.data_ptr()), ctypes.c_void_p(zd.data_ptr()),
                                ctypes.c_void_p(y.data_ptr()), M, N, K, ctypes.c_void_p(ws.data_ptr()), nbytes,
                                ctypes.c_void_p(torch.cuda.current_stream(DEV).cuda_stream))
    assert st == laq.LAQ_OK, L.laq_last_error()
    return y, nbytes


def test_noalloc_matches_workspace_entry_point():
    # Qwen3-32B down projection at M = 16 (split K into ten ranges: 3.3 MB of
    # partial sums), then a smaller split shape, then a shape that never
    # splits, then the first shape again (the scratch keeps the last call's
    # contents; nothing may depend on them).
    shapes = [(16, 5120, 25600, 61), (4, 1000, 20480, 62), (3, 300, 1024, 63), (16, 5120, 25600, 61)]
    cache = {}
    rng = np.random.default_rng(5)
    for (M, N, K, cfg) in shapes:
        say("noalloc", M, N, K)
        if cfg not in cache:
            cache[cfg] = _case(M, N, K, cfg)
        x, codes, s, z, q, sd, zd = cache[cfg]
        xd = torch.from_numpy(x).to(DEV)
        y_ws, nbytes = _ws(xd, q, sd, zd, M, N, K)
        y_na = _noalloc(xd, q, sd, zd, M, N, K)
        torch.cuda.synchronize()
        assert nbytes <= laq.NOALLOC_SCRATCH_BYTES
        if N >= 1000:
            assert nbytes > 0, "shape expected to split K"
        assert torch.equal(y_na.view(torch.int16), y_ws.view(torch.int16)), (M, N, K)
        rows = np.sort(rng.choice(N, size=min(N, 128), replace=False))
        ref = oracle.linear(x, codes[rows], s[rows], z[rows])
        r = linear_check(y_na.cpu().numpy()[:, rows], ref)
        assert r["ok"], (M, N, K, r)

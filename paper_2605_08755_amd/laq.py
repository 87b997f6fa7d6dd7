"""Python binding of liblaq.so (the C ABI in include/laq.h).

Argument marshalling only: every step of quantize and linear runs in the HIP
kernels of liblaq.so.  torch provides device memory and the current stream.
There is no fallback: if the library is missing or a call fails, an
exception is raised.
"""
import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "liblaq.so")

LAQ_OK = 0
LAQ_ERR_NULL_POINTER = 1
LAQ_ERR_BAD_SHAPE = 2
LAQ_ERR_BAD_M = 3
LAQ_ERR_MISALIGNED = 4
LAQ_ERR_HIP = 5
MAX_M = 16
GROUP = 128

MAX_GROUP = 8
NOALLOC_SCRATCH_BYTES = 8 << 20  # LAQ_NOALLOC_SCRATCH_BYTES

EXPORTS = ("laq_abi_version", "laq_status_string", "laq_last_error", "laq_profile_next_launch",
           "laq_quantize_w3g128", "laq_pack_w3g128", "laq_linear_w3g128", "laq_linear_group_w3g128",
           "laq_quantize_w4g128", "laq_pack_w4g128", "laq_linear_w4g128", "laq_linear_group_w4g128",
           "laq_linear_workspace_bytes", "laq_linear_ws_w3g128", "laq_linear_ws_w4g128",
           "laq_add_rmsnorm_f16", "laq_qk_norm_rope_f16", "laq_decode_attention_workspace_bytes",
           "laq_decode_attention_f16", "laq_silu_mul_f16", "laq_linear_swiglu_w3g128",
           "laq_linear_swiglu_w4g128", "laq_linear_noalloc_w3g128", "laq_decode_attention_qkv_workspace_bytes",
           "laq_decode_attention_qkv_f16", "laq_add_rmsnorm_linear_w3g128", "laq_add_rmsnorm_linear_w4g128",
           "laq_add_rmsnorm_linear_swiglu_w3g128", "laq_add_rmsnorm_linear_swiglu_w4g128",
           "laq_mlp_workspace_bytes", "laq_add_rmsnorm_mlp_w3g128", "laq_linear_residual_w3g128",
           "laq_linear_residual_w4g128")
HEAD_DIM = 128


class LinearCall(ctypes.Structure):
    """laq_linear_call of include/laq.h."""
    _fields_ = [("x", ctypes.c_void_p), ("qweight", ctypes.c_void_p), ("scales", ctypes.c_void_p),
                ("zeros", ctypes.c_void_p), ("y", ctypes.c_void_p), ("N", ctypes.c_int64), ("K", ctypes.c_int64)]

_lib = None


class LaqError(RuntimeError):
    def __init__(self, status, message):
        super().__init__("laq status %d: %s" % (status, message))
        self.status = status


def lib():
    """Load liblaq.so (built by paper_2605_08755_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("liblaq.so not built: run `python -m paper_2605_08755_amd.build` "
                              "(there is no non-HIP fallback)")
        L = ctypes.CDLL(LIB_PATH)
        P, I64 = ctypes.c_void_p, ctypes.c_int64
        L.laq_abi_version.argtypes = []
        L.laq_abi_version.restype = ctypes.c_int32
        L.laq_status_string.argtypes = [ctypes.c_int32]
        L.laq_status_string.restype = ctypes.c_char_p
        L.laq_last_error.argtypes = []
        L.laq_last_error.restype = ctypes.c_char_p
        L.laq_profile_next_launch.argtypes = [P, P]
        L.laq_profile_next_launch.restype = ctypes.c_int32
        for name in ("laq_quantize_w3g128", "laq_quantize_w4g128"):
            f = getattr(L, name)
            f.argtypes = [P, I64, I64, P, P, P, P]
            f.restype = ctypes.c_int32
        for name in ("laq_pack_w3g128", "laq_pack_w4g128"):
            f = getattr(L, name)
            f.argtypes = [P, P, P, I64, I64, P, P]
            f.restype = ctypes.c_int32
        for name in ("laq_linear_group_w3g128", "laq_linear_group_w4g128"):
            f = getattr(L, name)
            f.argtypes = [ctypes.POINTER(LinearCall), ctypes.c_int32, I64, P]
            f.restype = ctypes.c_int32
        for name in ("laq_linear_w3g128", "laq_linear_w4g128", "laq_linear_swiglu_w3g128",
                     "laq_linear_swiglu_w4g128", "laq_linear_noalloc_w3g128"):
            f = getattr(L, name)
            f.argtypes = [P, P, P, P, P, I64, I64, I64, P]
            f.restype = ctypes.c_int32
        for name in ("laq_linear_ws_w3g128", "laq_linear_ws_w4g128"):
            f = getattr(L, name)
            f.argtypes = [P, P, P, P, P, I64, I64, I64, P, I64, P]
            f.restype = ctypes.c_int32
        L.laq_linear_workspace_bytes.argtypes = [I64, I64, I64]
        L.laq_linear_workspace_bytes.restype = I64
        F32 = ctypes.c_float
        L.laq_add_rmsnorm_f16.argtypes = [P, P, P, P, I64, I64, F32, P]
        L.laq_add_rmsnorm_f16.restype = ctypes.c_int32
        L.laq_qk_norm_rope_f16.argtypes = [P, P, P, P, I64, I64, I64, I64, F32, P, P, P, I64, P]
        L.laq_qk_norm_rope_f16.restype = ctypes.c_int32
        L.laq_decode_attention_workspace_bytes.argtypes = [I64, I64]
        L.laq_decode_attention_workspace_bytes.restype = I64
        L.laq_decode_attention_f16.argtypes = [P, P, P, I64, I64, I64, I64, I64, P, P, I64, P]
        L.laq_decode_attention_f16.restype = ctypes.c_int32
        L.laq_decode_attention_qkv_workspace_bytes.argtypes = [I64, I64, I64]
        L.laq_decode_attention_qkv_workspace_bytes.restype = I64
        L.laq_decode_attention_qkv_f16.argtypes = [P, P, P, P, I64, I64, I64, I64, F32, P, P, I64, P, P, I64, P]
        L.laq_decode_attention_qkv_f16.restype = ctypes.c_int32
        L.laq_silu_mul_f16.argtypes = [P, P, I64, I64, P]
        L.laq_silu_mul_f16.restype = ctypes.c_int32
        for name in ("laq_add_rmsnorm_linear_w3g128", "laq_add_rmsnorm_linear_w4g128",
                     "laq_add_rmsnorm_linear_swiglu_w3g128", "laq_add_rmsnorm_linear_swiglu_w4g128",
           "laq_mlp_workspace_bytes", "laq_add_rmsnorm_mlp_w3g128", "laq_linear_residual_w3g128",
           "laq_linear_residual_w4g128"):
            f = getattr(L, name)
            f.argtypes = [P, P, P, F32, P, P, P, P, P, I64, I64, P]
            f.restype = ctypes.c_int32
        for name in ("laq_linear_residual_w3g128", "laq_linear_residual_w4g128"):
            f = getattr(L, name)
            f.argtypes = [P, P, P, P, P, P, P, I64, I64, P]
            f.restype = ctypes.c_int32
        L.laq_mlp_workspace_bytes.argtypes = [I64, I64]
        L.laq_mlp_workspace_bytes.restype = I64
        L.laq_add_rmsnorm_mlp_w3g128.argtypes = [P, P, P, F32, P, P, P, P, P, P, P, P, I64, I64, P, I64, P]
        L.laq_add_rmsnorm_mlp_w3g128.restype = ctypes.c_int32
        _lib = L
    return _lib


def _check(status):
    if status != LAQ_OK:
        raise LaqError(status, lib().laq_last_error().decode())


def _stream(device):
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def profile_next_launch(start_event, stop_event):
    """Have the next quantize/linear call on this thread record the given
    torch.cuda.Event pair at its kernel's execution start and end."""
    _check(lib().laq_profile_next_launch(ctypes.c_void_p(start_event.cuda_event),
                                         ctypes.c_void_p(stop_event.cuda_event)))


def packed_words(bits, N, K):
    """Number of uint32 words of a packed [N][K] matrix."""
    return N * bits * (K // 32)


def quantize(w, bits=3, out=None):
    """Quantize fp16 [N][K] weights on the GPU (Eq. 1, RTN min-max per 128-group).

    Returns (qweight int32 [N][bits][K/32], scales fp16 [N][K/128],
    zeros uint8 [N][K/128]).  qweight holds uint32 bit patterns in an int32
    tensor (torch has no uint32 arithmetic).
    """
    import torch
    assert w.is_cuda and w.dtype == torch.float16 and w.dim() == 2 and w.is_contiguous()
    N, K = w.shape
    if out is None:
        qweight = torch.empty((N, bits, K // 32), dtype=torch.int32, device=w.device)
        scales = torch.empty((N, K // GROUP), dtype=torch.float16, device=w.device)
        zeros = torch.empty((N, K // GROUP), dtype=torch.uint8, device=w.device)
    else:
        qweight, scales, zeros = out
    fn = lib().laq_quantize_w3g128 if bits == 3 else lib().laq_quantize_w4g128
    _check(fn(_ptr(w), N, K, _ptr(qweight), _ptr(scales), _ptr(zeros), _stream(w.device)))
    return qweight, scales, zeros


def pack(w, scales, zeros, bits=3, out=None):
    """Eq. 1 with caller-supplied fp16 scales [N][K/128] and uint8 zero points
    [N][K/128] (e.g. trained ones); returns qweight int32 [N][bits][K/32]."""
    import torch
    assert w.is_cuda and w.dtype == torch.float16 and w.dim() == 2 and w.is_contiguous()
    N, K = w.shape
    assert scales.shape == (N, K // GROUP) and zeros.shape == (N, K // GROUP)
    assert scales.dtype == torch.float16 and zeros.dtype == torch.uint8
    assert scales.is_contiguous() and zeros.is_contiguous()
    qweight = torch.empty((N, bits, K // 32), dtype=torch.int32, device=w.device) if out is None else out
    fn = lib().laq_pack_w3g128 if bits == 3 else lib().laq_pack_w4g128
    _check(fn(_ptr(w), _ptr(scales), _ptr(zeros), N, K, _ptr(qweight), _stream(w.device)))
    return qweight


def workspace_bytes(M, N, K):
    """Workspace with which the linear splits K for this shape (0: never)."""
    return int(lib().laq_linear_workspace_bytes(M, N, K))


def linear(x, qweight, scales, zeros, bits=3, out=None, split_k=True):
    """y = x @ w_hat^T for fp16 x [M][K] (M <= 16) against packed weights.

    split_k: where the shape gains from splitting K across workgroups
    (laq_linear_workspace_bytes > 0), take a workspace from torch's allocator
    on the current stream and call the _ws entry point; False calls the plain
    entry point."""
    import torch
    assert x.is_cuda and x.dtype == torch.float16 and x.dim() == 2 and x.is_contiguous()
    M, K = x.shape
    N = scales.shape[0]
    assert qweight.numel() == packed_words(bits, N, K) and qweight.is_contiguous()
    assert scales.shape == (N, K // GROUP) and zeros.shape == (N, K // GROUP)
    assert scales.dtype == torch.float16 and zeros.dtype == torch.uint8
    y = torch.empty((M, N), dtype=torch.float16, device=x.device) if out is None else out
    nbytes = workspace_bytes(M, N, K) if split_k else 0
    if nbytes > 0:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=x.device)
        fn = lib().laq_linear_ws_w3g128 if bits == 3 else lib().laq_linear_ws_w4g128
        _check(fn(_ptr(x), _ptr(qweight), _ptr(scales), _ptr(zeros), _ptr(y), M, N, K, _ptr(ws), nbytes,
                  _stream(x.device)))
        return y
    fn = lib().laq_linear_w3g128 if bits == 3 else lib().laq_linear_w4g128
    _check(fn(_ptr(x), _ptr(qweight), _ptr(scales), _ptr(zeros), _ptr(y), M, N, K, _stream(x.device)))
    return y


def linear_noalloc_w3g128(x, qweight, scales, zeros, out=None):
    """The W3 linear with split-K partial sums in the library's own scratch
    array (laq_linear_noalloc_w3g128): no workspace is allocated for it."""
    import torch
    assert x.is_cuda and x.dtype == torch.float16 and x.dim() == 2 and x.is_contiguous()
    M, K = x.shape
    N = scales.shape[0]
    assert qweight.numel() == packed_words(3, N, K) and qweight.is_contiguous()
    assert scales.shape == (N, K // GROUP) and zeros.shape == (N, K // GROUP)
    assert scales.dtype == torch.float16 and zeros.dtype == torch.uint8
    y = torch.empty((M, N), dtype=torch.float16, device=x.device) if out is None else out
    _check(lib().laq_linear_noalloc_w3g128(_ptr(x), _ptr(qweight), _ptr(scales), _ptr(zeros), _ptr(y), M, N, K,
                                           _stream(x.device)))
    return y


def linear_residual(x, qweight, scales, zeros, residual_in, residual_out, bits=3, out=None, write_out=True):
    """One token's linear that also updates the residual stream: y = x @
    w_hat^T (fp16 [1][N], as `linear` computes it) and residual_out =
    residual_in + y (fp32 [1][N]; may be residual_in itself).  With
    write_out=False only residual_out is written and None is returned."""
    import torch
    assert x.is_cuda and x.dtype == torch.float16 and x.dim() == 2 and x.shape[0] == 1 and x.is_contiguous()
    K = x.shape[1]
    N = scales.shape[0]
    assert qweight.numel() == packed_words(bits, N, K) and qweight.is_contiguous()
    assert scales.shape == (N, K // GROUP) and zeros.shape == (N, K // GROUP)
    assert scales.dtype == torch.float16 and zeros.dtype == torch.uint8
    for r in (residual_in, residual_out):
        assert r.dtype == torch.float32 and r.numel() == N and r.is_contiguous()
    y = None
    if write_out:
        y = torch.empty((1, N), dtype=torch.float16, device=x.device) if out is None else out
    fn = lib().laq_linear_residual_w3g128 if bits == 3 else lib().laq_linear_residual_w4g128
    _check(fn(_ptr(x), _ptr(qweight), _ptr(scales), _ptr(zeros), _ptr(y) if y is not None else None,
              _ptr(residual_in), _ptr(residual_out), N, K, _stream(x.device)))
    return y


def linear_swiglu(x, qweight, scales, zeros, bits=3, out=None):
    """silu(gate) * up of the gate|up projection in one launch: fp16 x [M][K]
    (M <= 4) against packed weights whose rows alternate gate row j, up row j
    (N = 2 I rows); returns fp16 [M][I]."""
    import torch
    assert x.is_cuda and x.dtype == torch.float16 and x.dim() == 2 and x.is_contiguous()
    M, K = x.shape
    N = scales.shape[0]
    assert qweight.numel() == packed_words(bits, N, K) and qweight.is_contiguous()
    assert scales.shape == (N, K // GROUP) and zeros.shape == (N, K // GROUP)
    assert scales.dtype == torch.float16 and zeros.dtype == torch.uint8
    y = torch.empty((M, N // 2), dtype=torch.float16, device=x.device) if out is None else out
    fn = lib().laq_linear_swiglu_w3g128 if bits == 3 else lib().laq_linear_swiglu_w4g128
    _check(fn(_ptr(x), _ptr(qweight), _ptr(scales), _ptr(zeros), _ptr(y), M, N, K, _stream(x.device)))
    return y


def linear_group(calls, bits=3, outs=None):
    """Several independent linears with the same M in one launch.

    calls: sequence of (x, qweight, scales, zeros) as for `linear`; returns
    the list of y (or fills `outs`)."""
    import torch
    n = len(calls)
    assert 1 <= n <= MAX_GROUP
    arr = (LinearCall * n)()
    ys = []
    M = None
    for i, (x, qweight, scales, zeros) in enumerate(calls):
        assert x.is_cuda and x.dtype == torch.float16 and x.dim() == 2 and x.is_contiguous()
        Mi, K = x.shape
        M = Mi if M is None else M
        assert Mi == M, "every call of a group has the same M"
        N = scales.shape[0]
        assert qweight.numel() == packed_words(bits, N, K) and qweight.is_contiguous()
        assert scales.shape == (N, K // GROUP) and zeros.shape == (N, K // GROUP)
        assert scales.dtype == torch.float16 and zeros.dtype == torch.uint8
        y = torch.empty((M, N), dtype=torch.float16, device=x.device) if outs is None else outs[i]
        ys.append(y)
        arr[i] = LinearCall(x.data_ptr(), qweight.data_ptr(), scales.data_ptr(), zeros.data_ptr(), y.data_ptr(), N, K)
    fn = lib().laq_linear_group_w3g128 if bits == 3 else lib().laq_linear_group_w4g128
    _check(fn(arr, n, M, _stream(calls[0][0].device)))
    return ys


def quantize_w3g128(w, out=None):
    return quantize(w, 3, out)


def pack_w3g128(w, scales, zeros, out=None):
    return pack(w, scales, zeros, 3, out)


def pack_w4g128(w, scales, zeros, out=None):
    return pack(w, scales, zeros, 4, out)


def linear_w3g128(x, qweight, scales, zeros, out=None):
    return linear(x, qweight, scales, zeros, 3, out)


def quantize_w4g128(w, out=None):
    return quantize(w, 4, out)


def linear_w4g128(x, qweight, scales, zeros, out=None):
    return linear(x, qweight, scales, zeros, 4, out)


# ---------------------------------------------------------------------------
# decode-step operations (one token; head dimension 128)
# ---------------------------------------------------------------------------
def add_rmsnorm(residual, delta, weight, eps, out=None):
    """residual (fp32 [M][D], updated in place) += delta (fp16 [M][D] or None);
    returns fp16 RMSNorm(residual) * weight."""
    import torch
    assert residual.is_cuda and residual.dtype == torch.float32 and residual.dim() == 2 and residual.is_contiguous()
    M, D = residual.shape
    assert weight.dtype == torch.float16 and weight.numel() == D and weight.is_contiguous()
    if delta is not None:
        assert delta.dtype == torch.float16 and delta.shape == (M, D) and delta.is_contiguous()
    if out is None:
        out = torch.empty((M, D), dtype=torch.float16, device=residual.device)
    _check(lib().laq_add_rmsnorm_f16(_ptr(residual), _ptr(delta) if delta is not None else None, _ptr(weight),
                                     _ptr(out), M, D, float(eps), _stream(residual.device)))
    return out


def add_rmsnorm_linear(residual, delta, norm_weight, eps, qweight, scales, zeros, bits=3, swiglu=False, out=None,
                       residual_out=None):
    """One token's residual add + RMSNorm and the linear after it, in one
    kernel: r = residual + delta (fp32 [1][K]; delta fp16 or None), x =
    RMSNorm(r) * norm_weight, y = x w_hat^T (fp16 [1][N], or [1][N/2] =
    silu(gate) * up with swiglu).  r goes to residual_out (a separate fp32
    [1][K] buffer) when given; x is not materialized."""
    import torch
    assert residual.is_cuda and residual.dtype == torch.float32 and residual.is_contiguous()
    assert residual.dim() == 2 and residual.shape[0] == 1
    K = residual.shape[1]
    N = scales.shape[0]
    assert norm_weight.dtype == torch.float16 and norm_weight.numel() == K and norm_weight.is_contiguous()
    if delta is not None:
        assert delta.dtype == torch.float16 and delta.numel() == K and delta.is_contiguous()
    if residual_out is not None:
        assert residual_out.dtype == torch.float32 and residual_out.numel() == K and residual_out.is_contiguous()
    assert qweight.numel() == packed_words(bits, N, K) and qweight.is_contiguous()
    assert scales.shape == (N, K // GROUP) and zeros.shape == (N, K // GROUP)
    assert scales.dtype == torch.float16 and zeros.dtype == torch.uint8
    n_out = N // 2 if swiglu else N
    y = torch.empty((1, n_out), dtype=torch.float16, device=residual.device) if out is None else out
    fn = {(3, False): lib().laq_add_rmsnorm_linear_w3g128, (4, False): lib().laq_add_rmsnorm_linear_w4g128,
          (3, True): lib().laq_add_rmsnorm_linear_swiglu_w3g128,
          (4, True): lib().laq_add_rmsnorm_linear_swiglu_w4g128}[(bits, bool(swiglu))]
    _check(fn(_ptr(residual), _ptr(delta) if delta is not None else None, _ptr(norm_weight), float(eps),
              _ptr(residual_out) if residual_out is not None else None, _ptr(qweight), _ptr(scales), _ptr(zeros),
              _ptr(y), N, K, _stream(residual.device)))
    return y


def mlp_workspace_bytes(D, I):
    return int(lib().laq_mlp_workspace_bytes(D, I))


def mlp_workspace(D, I, device):
    """A zero-filled workspace for add_rmsnorm_mlp (its counters start at
    zero; every call leaves them zero)."""
    import torch
    n = mlp_workspace_bytes(D, I)
    if n <= 0:
        raise LaqError(LAQ_ERR_BAD_SHAPE, "merged MLP block: unsupported shape D=%d I=%d" % (D, I))
    return torch.zeros(n, dtype=torch.uint8, device=device)


def add_rmsnorm_mlp(residual, delta, norm_weight, eps, gate_up, down, workspace, out=None, residual_out=None):
    """One token's SwiGLU MLP block in one launch (W3G128): r = residual +
    delta, x = RMSNorm(r) * norm_weight, h = silu(x gate^T) * (x up^T), y =
    h down^T (fp16 [1][D]).  gate_up = (qweight, scales, zeros) of the 2I
    interleaved gate|up rows, down = (qweight, scales, zeros) of the D down
    rows; workspace from mlp_workspace(D, I)."""
    import torch
    assert residual.is_cuda and residual.dtype == torch.float32 and residual.is_contiguous()
    assert residual.dim() == 2 and residual.shape[0] == 1
    D = residual.shape[1]
    gq, gs, gz = gate_up
    dq, ds, dz = down
    I = gs.shape[0] // 2
    assert norm_weight.dtype == torch.float16 and norm_weight.numel() == D and norm_weight.is_contiguous()
    if delta is not None:
        assert delta.dtype == torch.float16 and delta.numel() == D and delta.is_contiguous()
    if residual_out is not None:
        assert residual_out.dtype == torch.float32 and residual_out.numel() == D and residual_out.is_contiguous()
    assert gq.numel() == packed_words(3, 2 * I, D) and gq.is_contiguous()
    assert gs.shape == (2 * I, D // GROUP) and gz.shape == (2 * I, D // GROUP)
    assert dq.numel() == packed_words(3, D, I) and dq.is_contiguous()
    assert ds.shape == (D, I // GROUP) and dz.shape == (D, I // GROUP)
    assert gs.dtype == torch.float16 and ds.dtype == torch.float16
    assert gz.dtype == torch.uint8 and dz.dtype == torch.uint8
    y = torch.empty((1, D), dtype=torch.float16, device=residual.device) if out is None else out
    _check(lib().laq_add_rmsnorm_mlp_w3g128(
        _ptr(residual), _ptr(delta) if delta is not None else None, _ptr(norm_weight), float(eps),
        _ptr(residual_out) if residual_out is not None else None, _ptr(gq), _ptr(gs), _ptr(gz), _ptr(dq), _ptr(ds),
        _ptr(dz), _ptr(y), D, I, _ptr(workspace), workspace.numel() * workspace.element_size(),
        _stream(residual.device)))
    return y


def qk_norm_rope(qkv, q_norm_weight, k_norm_weight, cos_sin, pos, Hq, Hkv, eps, k_cache, v_cache, q_out=None):
    """One token's q|k|v projection output -> normalized, rotated q (returned,
    fp16 [Hq][128]); k and v written to row pos of the caches [Hkv][S_max][128]."""
    import torch
    assert qkv.is_cuda and qkv.dtype == torch.float16 and qkv.is_contiguous() and qkv.numel() == (Hq + 2 * Hkv) * HEAD_DIM
    assert cos_sin.dtype == torch.float32 and cos_sin.dim() == 2 and cos_sin.shape[1] == HEAD_DIM and cos_sin.is_contiguous()
    S_max = k_cache.shape[1]
    assert k_cache.shape == (Hkv, S_max, HEAD_DIM) and v_cache.shape == k_cache.shape and cos_sin.shape[0] >= S_max
    assert k_cache.dtype == torch.float16 and v_cache.dtype == torch.float16
    if q_out is None:
        q_out = torch.empty((Hq, HEAD_DIM), dtype=torch.float16, device=qkv.device)
    _check(lib().laq_qk_norm_rope_f16(_ptr(qkv), _ptr(q_norm_weight), _ptr(k_norm_weight), _ptr(cos_sin), int(pos),
                                      Hq, Hkv, HEAD_DIM, float(eps), _ptr(q_out), _ptr(k_cache), _ptr(v_cache), S_max,
                                      _stream(qkv.device)))
    return q_out


def attention_workspace_bytes(Hq, L):
    return int(lib().laq_decode_attention_workspace_bytes(Hq, L))


def decode_attention(q, k_cache, v_cache, L, out=None, workspace=None):
    """Single-token attention over the first L cache positions; returns fp16 [Hq][128]."""
    import torch
    Hq = q.shape[0]
    Hkv, S_max, d = k_cache.shape
    assert q.dtype == torch.float16 and q.shape == (Hq, HEAD_DIM) and q.is_contiguous() and d == HEAD_DIM
    if out is None:
        out = torch.empty((Hq, HEAD_DIM), dtype=torch.float16, device=q.device)
    need = attention_workspace_bytes(Hq, L)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    _check(lib().laq_decode_attention_f16(_ptr(q), _ptr(k_cache), _ptr(v_cache), Hq, Hkv, HEAD_DIM, int(L), S_max,
                                          _ptr(out), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                          _stream(q.device)))
    return out


def attention_qkv_workspace_bytes(Hq, Hkv, L):
    return int(lib().laq_decode_attention_qkv_workspace_bytes(Hq, Hkv, L))


def decode_attention_qkv(qkv, q_norm_weight, k_norm_weight, cos_sin, pos, Hq, Hkv, eps, k_cache, v_cache,
                         out=None, workspace=None):
    """qk_norm_rope + decode_attention over positions 0..pos in two kernels:
    one token's q|k|v projection output -> attention output fp16 [Hq][128];
    k and v written to row pos of the caches [Hkv][S_max][128]."""
    import torch
    assert qkv.is_cuda and qkv.dtype == torch.float16 and qkv.is_contiguous() and qkv.numel() == (Hq + 2 * Hkv) * HEAD_DIM
    assert cos_sin.dtype == torch.float32 and cos_sin.dim() == 2 and cos_sin.shape[1] == HEAD_DIM and cos_sin.is_contiguous()
    S_max = k_cache.shape[1]
    assert k_cache.shape == (Hkv, S_max, HEAD_DIM) and v_cache.shape == k_cache.shape and cos_sin.shape[0] >= S_max
    assert k_cache.dtype == torch.float16 and v_cache.dtype == torch.float16
    if out is None:
        out = torch.empty((Hq, HEAD_DIM), dtype=torch.float16, device=qkv.device)
    need = attention_qkv_workspace_bytes(Hq, Hkv, pos + 1)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=qkv.device)
    _check(lib().laq_decode_attention_qkv_f16(_ptr(qkv), _ptr(q_norm_weight), _ptr(k_norm_weight), _ptr(cos_sin),
                                              int(pos), Hq, Hkv, HEAD_DIM, float(eps), _ptr(k_cache), _ptr(v_cache),
                                              S_max, _ptr(out), _ptr(workspace),
                                              workspace.numel() * workspace.element_size(), _stream(qkv.device)))
    return out


def silu_mul(gate_up, out=None):
    """fp16 [M][2I] gate | up -> fp16 [M][I] silu(gate) * up."""
    import torch
    assert gate_up.is_cuda and gate_up.dtype == torch.float16 and gate_up.dim() == 2 and gate_up.is_contiguous()
    M, I2 = gate_up.shape
    assert I2 % 2 == 0
    if out is None:
        out = torch.empty((M, I2 // 2), dtype=torch.float16, device=gate_up.device)
    _check(lib().laq_silu_mul_f16(_ptr(gate_up), _ptr(out), M, I2 // 2, _stream(gate_up.device)))
    return out

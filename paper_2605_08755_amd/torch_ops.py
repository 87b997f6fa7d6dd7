"""torch.library registrations of the C ABI (include/laq.h).

Registered as custom operators with fake (shape-only) implementations, the
library's calls can sit inside code that torch.compile traces or that a HIP
graph captures, as the quantized linears of a decode step do.  Argument
marshalling only: the real implementations call laq.py, which calls the HIP
kernels; there is no fallback.

    torch.ops.laq.linear(x, qweight, scales, zeros, bits)  -> y fp16 [M][N]
    torch.ops.laq.quantize(w, bits)                        -> (qweight, scales, zeros)
    torch.ops.laq.pack(w, scales, zeros, bits)             -> qweight
"""
from typing import Tuple

import torch

from . import laq

GROUP = laq.GROUP


@torch.library.custom_op("laq::linear", mutates_args=())
def linear(x: torch.Tensor, qweight: torch.Tensor, scales: torch.Tensor, zeros: torch.Tensor,
           bits: int) -> torch.Tensor:
    return laq.linear(x.contiguous(), qweight, scales, zeros, bits)


@linear.register_fake
def _linear_fake(x, qweight, scales, zeros, bits):
    torch._check(x.dim() == 2 and x.dtype == torch.float16)
    torch._check(x.shape[0] >= 1 and x.shape[0] <= laq.MAX_M)
    torch._check(scales.shape[1] * GROUP == x.shape[1])
    return x.new_empty((x.shape[0], scales.shape[0]))


@torch.library.custom_op("laq::quantize", mutates_args=())
def quantize(w: torch.Tensor, bits: int) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    return laq.quantize(w.contiguous(), bits)


@quantize.register_fake
def _quantize_fake(w, bits):
    torch._check(w.dim() == 2 and w.dtype == torch.float16 and w.shape[1] % GROUP == 0)
    N, K = w.shape
    return (w.new_empty((N, bits, K // 32), dtype=torch.int32),
            w.new_empty((N, K // GROUP), dtype=torch.float16),
            w.new_empty((N, K // GROUP), dtype=torch.uint8))


@torch.library.custom_op("laq::pack", mutates_args=())
def pack(w: torch.Tensor, scales: torch.Tensor, zeros: torch.Tensor, bits: int) -> torch.Tensor:
    return laq.pack(w.contiguous(), scales.contiguous(), zeros.contiguous(), bits)


@pack.register_fake
def _pack_fake(w, scales, zeros, bits):
    torch._check(w.dim() == 2 and w.dtype == torch.float16 and w.shape[1] % GROUP == 0)
    N, K = w.shape
    return w.new_empty((N, bits, K // 32), dtype=torch.int32)

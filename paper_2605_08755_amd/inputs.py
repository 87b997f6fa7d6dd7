"""Seeded synthetic inputs: weights, activations and the workload shapes.

This module holds random-number generation and shapes only -- none of the
quantization or GEMV arithmetic -- so that the HIP path and the CPU oracle can
be fed the very same inputs without sharing any code of the method.

Workloads (Qwen3-shaped decode linears; the paper evaluates Qwen3 models, Table 3):
  single    one 1024 x 1024 linear
  layer4b   the 7 projections of one Qwen3-4B decoder layer
  stack4b   36 such layers (the decode-step linear stack)
  stack32b  64 Qwen3-32B-shaped layers

Distributions: weights ~ N(0, 0.02) in fp32, each entry independently
multiplied by 10 with probability 0.01 (outliers), then rounded to fp16;
activations ~ N(0, 1) rounded to fp16.  The paper's checkpoints and
calibration data are not available, so these stand in for them.
"""
import numpy as np

ENTROPY = 260508755

# (name, N out, K in) per projection, in decoder order.
QWEN3_4B = (("q", 4096, 2560), ("k", 1024, 2560), ("v", 1024, 2560),
            ("o", 2560, 4096), ("gate", 9728, 2560), ("up", 9728, 2560),
            ("down", 2560, 9728))
QWEN3_32B = (("q", 8192, 5120), ("k", 1024, 5120), ("v", 1024, 5120),
             ("o", 5120, 8192), ("gate", 25600, 5120), ("up", 25600, 5120),
             ("down", 5120, 25600))

# Which activation each projection reads: q/k/v share the attention input,
# gate/up share the MLP input.
X_SLOT = {"q": 0, "k": 0, "v": 0, "o": 1, "gate": 2, "up": 2, "down": 3}

WORKLOADS = {
    "single": {"layers": 1, "projs": (("w", 1024, 1024),)},
    "layer4b": {"layers": 1, "projs": QWEN3_4B},
    "stack4b": {"layers": 36, "projs": QWEN3_4B},
    "stack32b": {"layers": 64, "projs": QWEN3_32B},
}

_T_WEIGHT, _T_ACT, _T_MASK = 0, 1, 2


def rng(cfg: int, layer: int, proj: int, tensor: int) -> np.random.Generator:
    ss = np.random.SeedSequence(entropy=ENTROPY, spawn_key=(cfg, layer, proj, tensor))
    return np.random.Generator(np.random.PCG64(ss))


def weights(N: int, K: int, cfg: int = 0, layer: int = 0, proj: int = 0,
            std: float = 0.02, outlier_p: float = 0.01, outlier_mul: float = 10.0) -> np.ndarray:
    """fp16 [N][K] weight matrix ~ N(0, std) with independent x10 outliers."""
    w = rng(cfg, layer, proj, _T_WEIGHT).standard_normal((N, K), dtype=np.float32)
    w *= np.float32(std)
    if outlier_p > 0:
        mask = rng(cfg, layer, proj, _T_MASK).random((N, K), dtype=np.float32) < outlier_p
        w[mask] *= np.float32(outlier_mul)
    return w.astype(np.float16)


def activations(M: int, K: int, cfg: int = 0, layer: int = 0, slot: int = 0) -> np.ndarray:
    """fp16 [M][K] activations ~ N(0, 1)."""
    x = rng(cfg, layer, 100 + slot, _T_ACT).standard_normal((M, K), dtype=np.float32)
    return x.astype(np.float16)


def weights_torch(N: int, K: int, seed: int, device, std: float = 0.02,
                  outlier_p: float = 0.01, outlier_mul: float = 10.0):
    """Same distribution as `weights`, drawn with torch's generator on `device`.

    Used where gigabytes of weights are needed (the 36- and 64-layer stacks),
    which numpy would take minutes to draw on the host.
    """
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(ENTROPY * 1000 + seed)
    w = torch.randn((N, K), generator=g, device=device, dtype=torch.float32)
    w.mul_(std)
    if outlier_p > 0:
        mask = torch.rand((N, K), generator=g, device=device) < outlier_p
        w[mask] *= outlier_mul
        del mask
    return w.to(torch.float16)


def activations_torch(M: int, K: int, seed: int, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(ENTROPY * 1000 + 500000 + seed)
    return torch.randn((M, K), generator=g, device=device, dtype=torch.float32).to(torch.float16)

"""CPU oracle for the decode-step operations around the quantized linears.

TEST INFRASTRUCTURE ONLY: imported by the test suite and the benchmark's
parity checks, never by the library, and sharing no code with the HIP path.

The paper measures decoding of its quantized Qwen3 models (Sec. 5, Table 3);
the operations between the linears are those of the model's decoder layer,
written here in float64 from their plain definitions:

  RMSNorm          y = x / sqrt(mean(x^2) + eps) * w
  rotary embedding  pair (x_i, x_{i+d/2}) rotated by pos * theta^(-2i/d),
                    i < d/2 (the half-split pairing of the Qwen3 layers)
  attention         softmax(q . k_t / sqrt(d)) over positions t, weights applied
                    to v_t; query head h reads key/value head h // (Hq / Hkv)
  SiLU-and-multiply silu(g) * u with silu(g) = g / (1 + exp(-g))

Every function takes numpy arrays of any float dtype and returns float64.
"""
import numpy as np


def rmsnorm(x, w, eps):
    """RMSNorm over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def add_rmsnorm(res, delta, w, eps):
    """Residual update r = res + delta, then y = RMSNorm(r) * w; returns (r, y)."""
    r = np.asarray(res, dtype=np.float64)
    if delta is not None:
        r = r + np.asarray(delta, dtype=np.float64)
    return r, rmsnorm(r, w, eps)


def rope_angles(pos, d, theta):
    """Rotation angle of pair i (i < d/2) at position pos."""
    i = np.arange(d // 2, dtype=np.float64)
    return float(pos) * theta ** (-2.0 * i / d)


def rope(x, pos, theta):
    """Rotary embedding of x [..., d] at position pos (half-split pairs)."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    a = rope_angles(pos, d, theta)
    c, s = np.cos(a), np.sin(a)
    x1, x2 = x[..., : d // 2], x[..., d // 2:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def qk_norm_rope(qkv, q_w, k_w, pos, Hq, Hkv, d, eps, theta):
    """Split one token's fused q|k|v projection [(Hq + 2 Hkv) d] into heads,
    RMSNorm each q and k head with its own weights, rotate q and k; v as is.
    Returns (q [Hq][d], k [Hkv][d], v [Hkv][d])."""
    qkv = np.asarray(qkv, dtype=np.float64).reshape(-1)
    q = qkv[: Hq * d].reshape(Hq, d)
    k = qkv[Hq * d: (Hq + Hkv) * d].reshape(Hkv, d)
    v = qkv[(Hq + Hkv) * d: (Hq + 2 * Hkv) * d].reshape(Hkv, d)
    q = rope(rmsnorm(q, q_w, eps), pos, theta)
    k = rope(rmsnorm(k, k_w, eps), pos, theta)
    return q, k, v


def decode_attention(q, K, V):
    """One query token: q [Hq][d], K, V [Hkv][L][d] -> out [Hq][d]."""
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    Hq, d = q.shape
    Hkv = K.shape[0]
    ratio = Hq // Hkv
    out = np.empty((Hq, d))
    for h in range(Hq):
        g = h // ratio
        s = K[g] @ q[h] / np.sqrt(d)
        p = np.exp(s - s.max())
        out[h] = (p / p.sum()) @ V[g]
    return out


def silu_mul(gu, I):
    """gu [M][2I] = gate | up halves -> silu(gate) * up [M][I]."""
    gu = np.asarray(gu, dtype=np.float64)
    g, u = gu[:, :I], gu[:, I: 2 * I]
    return g / (1.0 + np.exp(-g)) * u

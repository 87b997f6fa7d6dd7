"""Eq. 1's scale and zero point (Sec. 2; the readings of the group range and
of the fp16 scale), computed by the C oracle on 10^7 random W3 groups and
2 * 10^6 W4 groups, against an independent numpy re-derivation of the same
formula in IEEE float32 and binary16:

  lo = min(0, min w), hi = max(0, max w)
  s16 = RNE_fp16(fl32(fl32(hi) - fl32(lo)) / (2^b - 1)), 2^-24 if that is 0
  z   = clamp(rint(fl32(-lo) / fl32(s16)), 0, 2^b - 1)      (rint: ties to even)

Each group holds lo and hi at its first two positions and zeros elsewhere,
so its range is exactly (lo, hi).  |lo| and |hi| are drawn uniformly over the
bit patterns of the finite non-negative binary16 values (subnormals, every
exponent, 65504), with exact zeros mixed in; the scale bits and zero points
must agree on every group."""
import numpy as np
import pytest

import oracle

CHUNK = 1_000_000


def _magnitudes(rng, n):
    """Finite non-negative fp16 values, uniform over their bit patterns
    (0x0000 .. 0x7BFF), 1 % exact zeros."""
    bits = rng.integers(0, 0x7C00, size=n, dtype=np.uint16)
    bits[rng.random(n) < 0.01] = 0
    return bits.view(np.float16)


def _derive(lo, hi, bits):
    """The formula above in numpy float32 / float16 arithmetic."""
    qmax = np.float32(2 ** bits - 1)
    lo32, hi32 = lo.astype(np.float32), hi.astype(np.float32)
    s32 = (hi32 - lo32) / qmax
    s16 = s32.astype(np.float16)                       # round to nearest even
    s16 = np.where(s16 == 0, np.float16(2.0 ** -24), s16).astype(np.float16)
    q = (-lo32) / s16.astype(np.float32)
    z = np.clip(np.rint(q), 0, qmax).astype(np.uint8)
    return s16, z


@pytest.mark.parametrize("bits,chunks", [(3, 10), (4, 2)])
def test_scale_zero_formula_sweep(bits, chunks):
    rng = np.random.default_rng(0x5CA1E + bits)
    for _ in range(chunks):
        lo = -_magnitudes(rng, CHUNK)
        hi = _magnitudes(rng, CHUNK)
        w = np.zeros((CHUNK, 128), dtype=np.float16)
        w[:, 0] = lo
        w[:, 1] = hi
        _, s, z = oracle.quantize(w, bits)
        s_ref, z_ref = _derive(lo, hi, bits)
        bad = np.flatnonzero((s.reshape(-1).view(np.uint16) != s_ref.view(np.uint16)) | (z.reshape(-1) != z_ref))
        assert bad.size == 0, [(float(lo[i]), float(hi[i]), float(s.reshape(-1)[i]), float(s_ref[i]),
                                int(z.reshape(-1)[i]), int(z_ref[i])) for i in bad[:5]]
        del w


def test_sweep_generator_covers_the_range():
    """The drawn magnitudes reach subnormals, the largest finite value's
    binade and exact zeros (so the sweep exercises the 2^-24 floor and the
    clipping of z)."""
    m = _magnitudes(np.random.default_rng(1), CHUNK).astype(np.float32)
    assert (m == 0).any() and (m[m > 0] < 2.0 ** -14).any() and (m >= 32768).any()
    lo = -_magnitudes(np.random.default_rng(2), CHUNK)
    hi = _magnitudes(np.random.default_rng(3), CHUNK)
    s16, z = _derive(lo, hi, 3)
    assert (s16 == np.float16(2.0 ** -24)).any() and (z == 7).any() and (z == 0).any()

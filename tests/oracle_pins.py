"""Pins for the CPU oracle: checks against facts that do not come from the
oracle itself.

Each pin takes an `Oracle` (oracle.Oracle) and raises AssertionError when the
oracle disagrees with:
  - CPython's own IEEE binary16 codec (struct format 'e'), exhaustively or on
    all rounding edge cases -- an implementation independent of the oracle;
  - exact rational arithmetic (fractions.Fraction) applied to Eq. 1
    (Sec. 2): the chosen code must be a nearest quantization level, the scale
    a nearest fp16 to (hi-lo)/(2^b-1), the zero point a nearest integer to
    -lo/s;
  - closed forms: on-grid groups w = 2^e (j - z0) reconstruct exactly with
    s = 2^e, z = z0, q = j; hand-worked round-half-to-even ties;
  - the packed-format definition spelled out field by field;
  - numpy's float64 GEMV (a library routine) and exact rational sums for the
    linear.
The same functions run against deliberately mutated oracle builds
(test_oracle_mutants.py) to show that each plausible mistake fails a pin.
"""
import struct
from fractions import Fraction

import numpy as np

from paper_2605_08755_amd import inputs


# ---------------------------------------------------------------------------
# helpers independent of the oracle
# ---------------------------------------------------------------------------
def py_half_bits_to_float(bits: int) -> float:
    return struct.unpack("<e", struct.pack("<H", bits))[0]


def py_float_to_half_bits(v: float) -> int:
    try:
        return struct.unpack("<H", struct.pack("<e", v))[0]
    except OverflowError:
        return 0x7C00 if v > 0 else 0xFC00


def half_frac(bits: int) -> Fraction:
    return Fraction(py_half_bits_to_float(bits))


# ---------------------------------------------------------------------------
# fp16 conversions
# ---------------------------------------------------------------------------
def pin_f16_to_f32_exhaustive(o):
    allbits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = o.f16_to_f32(allbits)
    for b in range(65536):
        ref = py_half_bits_to_float(b)
        g = float(got[b])
        if ref != ref:
            assert g != g, hex(b)
        else:
            assert g == ref and bool(np.signbit(g)) == bool(b & 0x8000), (hex(b), g, ref)


def _f32_edge_values():
    vals = []
    finite = [b for b in range(0x7C00)]  # all non-negative finite halves
    hv = np.array([py_half_bits_to_float(b) for b in finite], dtype=np.float64)
    vals.extend(hv.tolist())
    # exact midpoints between consecutive halves (exact in fp32), and 1 fp32
    # ulp either side of them
    mids = (hv[:-1] + hv[1:]) / 2
    mids32 = mids.astype(np.float32)
    assert np.all(mids32.astype(np.float64) == mids)
    vals.extend(mids32.tolist())
    vals.extend(np.nextafter(mids32, np.float32(np.inf)).tolist())
    vals.extend(np.nextafter(mids32, np.float32(0)).tolist())
    vals.extend([65504.0, 65519.996, 65520.0, 65536.0, 1e30, 2.0 ** -25,
                 2.0 ** -25 * 1.0000001, 3 * 2.0 ** -26, 2.0 ** -26, 1e-30, 0.0])
    rng = np.random.default_rng(7)
    e = rng.integers(-30, 17, 20000)
    m = rng.random(20000) + 1.0
    vals.extend((m * np.exp2(e)).astype(np.float32).tolist())
    v = np.array(vals, dtype=np.float32)
    return np.concatenate([v, -v])


def pin_f32_to_f16_rne(o):
    v = _f32_edge_values()
    got = o.f32_to_f16(v)
    for x, g in zip(v.tolist(), got.tolist()):
        ref = py_float_to_half_bits(float(x))
        assert g == ref, (x, hex(g), hex(ref))


# ---------------------------------------------------------------------------
# quantization pins
# ---------------------------------------------------------------------------
def _levels(bits):
    return (1 << bits) - 1


def pin_ongrid_exact(o, bits=3, seed=0):
    """w = 2^e (j - z0), j uniform in 0..qmax with 0 and qmax both present:
    s = 2^e, z = z0, q = j and w_hat == w exactly."""
    qmax = _levels(bits)
    rng = np.random.default_rng(seed)
    rows = []
    expect = []
    for r in range(64):
        e = int(rng.integers(-14, 8))
        z0 = int(rng.integers(0, qmax + 1))
        rowq = []
        roww = []
        for g in range(2):
            j = rng.integers(0, qmax + 1, 128)
            j[rng.integers(0, 128)] = 0
            j[rng.integers(0, 128)] = qmax
            j[0], j[1] = 0, qmax
            rng.shuffle(j)
            roww.append(np.ldexp((j - z0).astype(np.float64), e))
            rowq.append(j)
        rows.append(np.concatenate(roww))
        expect.append((e, z0, np.concatenate(rowq)))
    w = np.array(rows).astype(np.float16)
    assert np.all(w.astype(np.float64) == np.array(rows))
    codes, scales, zeros = o.quantize(w, bits)
    for r, (e, z0, j) in enumerate(expect):
        assert np.all(scales[r] == py_float_to_half_bits(2.0 ** e)), (r, scales[r], e)
        assert np.all(zeros[r] == z0), (r, zeros[r], z0)
        assert np.array_equal(codes[r], j.astype(np.uint8)), r
    wh = o.dequant(codes, scales, zeros)
    assert np.array_equal(wh, w.astype(np.float64))


def pin_ties_handworked(o):
    """Round-half-to-even on exact ties, worked by hand from Eq. 1.

    W3: lo = -3/64, hi = 4/64 -> s = 1/64, z = 3.  w/s = 2.5 -> 2 -> q 5;
    1.5 -> 2 -> 5; -0.5 -> -0 -> 3; 0.5 -> 0 -> 3; 3.5 -> 4 -> 7;
    -2.5 -> -2 -> 1; -1.5 -> -2 -> 1; 4 -> 7; -3 -> 0; 0 -> 3.
    W4: lo = -7/64, hi = 8/64 -> s = 1/64, z = 7; same ratios give
    9, 9, 7, 7, 11, 5, 5, 11 (w/s=4), 4 (w/s=-3), 7.
    """
    ratios = [2.5, 1.5, -0.5, 0.5, 3.5, -2.5, -1.5, 4.0, -3.0, 0.0]
    for bits, lo_r, hi_r, exp in (
        (3, -3.0, 4.0, [5, 5, 3, 3, 7, 1, 1, 7, 0, 3]),
        (4, -7.0, 8.0, [9, 9, 7, 7, 11, 5, 5, 11, 4, 7]),
    ):
        g = np.zeros(128)
        g[0], g[1] = lo_r / 64, hi_r / 64
        g[2:2 + len(ratios)] = np.array(ratios) / 64
        w = g.astype(np.float16)[None, :]
        codes, scales, zeros = o.quantize(w, bits)
        assert scales[0, 0] == py_float_to_half_bits(1 / 64)
        assert zeros[0, 0] == (3 if bits == 3 else 7)
        assert codes[0, 0] == 0 and codes[0, 1] == _levels(bits)
        assert codes[0, 2:2 + len(ratios)].tolist() == exp, (bits, codes[0, 2:12].tolist())


def pin_special_groups(o, bits=3):
    qmax = _levels(bits)
    K = 128
    w = np.zeros((6, K), np.float16)
    # row 0: all zero -> smallest subnormal scale, z = 0, codes 0
    # row 1: constant positive -> lo = 0, z = 0, every code qmax
    w[1, :] = np.float16(0.75)
    # row 2: all negative -> hi = 0, z = qmax, minimum -> 0
    w[2, :] = -np.linspace(0.01, 0.5, K).astype(np.float16)
    # row 3: one outlier among zeros
    w[3, 17] = np.float16(-3.0)
    # row 4: tiny subnormal-range values (scale underflows fp16 normal range)
    w[4, :5] = np.array([6e-8, -6e-8, 1.2e-7, 0, -1.8e-7], np.float32).astype(np.float16)
    # row 5: single positive spike
    w[5, 100] = np.float16(1.0)
    codes, scales, zeros = o.quantize(w, bits)
    assert scales[0, 0] == 0x0001 and zeros[0, 0] == 0 and np.all(codes[0] == 0)
    assert zeros[1, 0] == 0 and np.all(codes[1] == qmax)
    assert zeros[2, 0] == qmax and codes[2, K - 1] == 0
    assert codes[3, 17] == 0 and np.all(np.delete(codes[3], 17) == zeros[3, 0])
    # row 4: scale is a subnormal half and the group reconstructs each value
    # to within s/2
    s4 = half_frac(int(scales[4, 0]))
    for k in range(5):
        wh = s4 * (int(codes[4, k]) - int(zeros[4, 0]))
        assert abs(Fraction(float(w[4, k])) - wh) <= s4 / 2
    assert codes[5, 100] == qmax and zeros[5, 0] == 0
    # every special group's (s, z) is the nearest-rounded function of the
    # exact, zero-widened range
    for r in range(w.shape[0]):
        _check_group_params_exact(w[r], int(scales[r, 0]), int(zeros[r, 0]), bits)
    # one-signed groups away from zero: the range still starts at 0
    pos = np.linspace(0.1, 0.5, K).astype(np.float16)[None, :]
    c, sc, zz = o.quantize(np.concatenate([pos, -pos]), bits)
    _check_group_params_exact(pos[0], int(sc[0, 0]), int(zz[0, 0]), bits)
    _check_group_params_exact(-pos[0], int(sc[1, 0]), int(zz[1, 0]), bits)
    assert zz[0, 0] == 0 and zz[1, 0] == qmax


def _allowed_round(v: Fraction, qmax: int, margin: Fraction):
    """Integers a correct round-half-to-even of v (clamped to 0..qmax) may
    give when v is only known to within `margin`."""
    fl = v.numerator // v.denominator
    fr = v - fl
    if abs(fr - Fraction(1, 2)) <= margin:
        cand = {fl, fl + 1}
    elif fr < Fraction(1, 2):
        cand = {fl}
    else:
        cand = {fl + 1}
    return {max(0, min(qmax, c)) for c in cand}


def _check_group_params_exact(w_row, s_bits, z, bits):
    """(s16, z) are nearest-rounded functions of the exact group (lo, hi)."""
    qmax = _levels(bits)
    vals = [Fraction(float(v)) for v in w_row]
    lo = min(min(vals), Fraction(0))
    hi = max(max(vals), Fraction(0))
    S = (hi - lo) / qmax
    s = half_frac(s_bits)
    assert s > 0
    if S <= Fraction(2) ** -25:
        # rounds to zero in fp16: the smallest subnormal is substituted
        assert s_bits == 0x0001, (float(S), hex(s_bits))
    else:
        ref_bits = py_float_to_half_bits(float(S))
        if s_bits != ref_bits:
            # allowed only next to a rounding midpoint (the fp32 rounding of
            # the range and of the quotient precede the fp16 rounding)
            ref = half_frac(ref_bits)
            mid = (s + ref) / 2
            assert abs(S - mid) <= S * Fraction(2) ** -21, (float(S), float(s), float(ref))
    assert z in _allowed_round(-lo / s, qmax, Fraction(2) ** -20), (float(-lo / s), z)


def pin_nearest_level(o, bits=3, N=48, K=512, seed=3):
    """Every code selects a nearest level s*(q-z) of Eq. 1 (exact check).

    Uses float64 ratios for the bulk and exact Fractions for the group
    parameters; an element may take either neighbour only when w/s lies
    within 2^-20 of a half-integer (where the fp32 quotient may round across).
    """
    qmax = _levels(bits)
    w = inputs.weights(N, K, cfg=90, layer=seed, proj=bits)
    codes, scales, zeros = o.quantize(w, bits)
    assert codes.max() <= qmax and zeros.max() <= qmax
    G = K // 128
    wf = w.astype(np.float64)
    s = np.array([[py_half_bits_to_float(int(b)) for b in row] for row in scales])
    for n in range(N):
        for g in range(G):
            _check_group_params_exact(w[n, g * 128:(g + 1) * 128], int(scales[n, g]), int(zeros[n, g]), bits)
    sk = np.repeat(s, 128, axis=1)
    zk = np.repeat(zeros.astype(np.float64), 128, axis=1)
    t = wf / sk + zk                     # real-valued position on the code axis
    q = codes.astype(np.float64)
    tc = np.clip(t, 0, qmax)
    dist = np.abs(tc - q)
    margin = 2.0 ** -20
    assert np.all(dist <= 0.5 + margin), float(dist.max())
    near_tie = np.abs(np.abs(tc - np.floor(tc)) - 0.5) <= margin
    strict = ~near_tie
    assert np.all(q[strict] == np.clip(np.floor(t[strict] + 0.5), 0, qmax))
    # reconstruction error of unclipped elements is at most s/2 (+ rounding)
    unclipped = (t >= -0.5) & (t <= qmax + 0.5)
    err = np.abs(wf - sk * (q - zk))
    assert np.all(err[unclipped] <= sk[unclipped] * (0.5 + margin))


def pin_group_permutation(o, bits=3, seed=11):
    """(s, z) depend only on the multiset of a group; codes follow elements."""
    w = inputs.weights(16, 256, cfg=91, layer=seed, proj=bits)
    rng = np.random.default_rng(seed)
    perm = np.concatenate([rng.permutation(128), 128 + rng.permutation(128)])
    c1, s1, z1 = o.quantize(w, bits)
    c2, s2, z2 = o.quantize(np.ascontiguousarray(w[:, perm]), bits)
    assert np.array_equal(s1, s2) and np.array_equal(z1, z2)
    assert np.array_equal(c1[:, perm], c2)


def pin_extremes(o, bits=3, seed=5):
    """The group minimum always maps to code 0 (RNE is odd-symmetric and
    negation is exact); the maximum maps to qmax unless -lo/s sits within
    qmax*2^-11 of a half-integer."""
    qmax = _levels(bits)
    w = inputs.weights(64, 256, cfg=92, layer=seed, proj=bits)
    codes, scales, zeros = o.quantize(w, bits)
    for n in range(64):
        for g in range(2):
            seg = w[n, g * 128:(g + 1) * 128].astype(np.float64)
            cs = codes[n, g * 128:(g + 1) * 128]
            lo, hi = min(seg.min(), 0.0), max(seg.max(), 0.0)
            if lo < 0:
                assert np.all(cs[seg == lo] == 0)
            if hi > 0:
                s = py_half_bits_to_float(int(scales[n, g]))
                r = -lo / s
                if abs(r - np.floor(r) - 0.5) > qmax * 2.0 ** -11:
                    assert np.all(cs[seg == hi] == qmax), (n, g)


# ---------------------------------------------------------------------------
# Eq. 1 with caller-supplied (s, z)
# ---------------------------------------------------------------------------
def pin_params_handworked(o):
    """Worked by hand from Eq. 1 with s = 1/64 (exact in fp16) and given z:
    w/s = 2.5 -> 2, 1.5 -> 2, -0.5 -> -0, 0.5 -> 0, 3.5 -> 4, -2.5 -> -2,
    -1.5 -> -2, 4, -3, 0, 10, -10; plus z, then clipped to 0..qmax.
    W3, z = 3: 5 5 3 3 7 1 1 7 0 3 7 0.  W4, z = 7: 9 9 7 7 11 5 5 11 4 7 15 0.
    A second group with s = 1/2 and z = 0 maps w = 0.75 -> rint(1.5) = 2,
    1.25 -> rint(2.5) = 2, -0.25 -> -0 -> 0, 3.0 -> 6 (W3) / 6 (W4)."""
    ratios = [2.5, 1.5, -0.5, 0.5, 3.5, -2.5, -1.5, 4.0, -3.0, 0.0, 10.0, -10.0]
    for bits, z0, exp in ((3, 3, [5, 5, 3, 3, 7, 1, 1, 7, 0, 3, 7, 0]),
                          (4, 7, [9, 9, 7, 7, 11, 5, 5, 11, 4, 7, 15, 0])):
        w = np.zeros((1, 256))
        w[0, :len(ratios)] = np.array(ratios) / 64
        w[0, 128:132] = [0.75, 1.25, -0.25, 3.0]
        w = w.astype(np.float16)
        scales = np.array([[py_float_to_half_bits(1 / 64), py_float_to_half_bits(0.5)]], np.uint16)
        zeros = np.array([[z0, 0]], np.uint8)
        c = o.codes_from_params(w, scales, zeros, bits)
        assert c[0, :len(ratios)].tolist() == exp, (bits, c[0, :len(ratios)].tolist())
        assert c[0, 128:132].tolist() == [2, 2, 0, 6], (bits, c[0, 128:132].tolist())
        assert np.all(c[0, len(ratios):128] == z0) and np.all(c[0, 132:] == 0)


def pin_params_exact(o, bits=3, seed=21):
    """Random weights, random positive fp16 scales (subnormal to large) and
    zero points: every code is clip(RNE(w/s) + z) of the exact rational
    quotient, either neighbour allowed only within the fp32 quotient's
    rounding of a tie."""
    qmax = _levels(bits)
    rng = np.random.default_rng(seed)
    N, K = 12, 384
    w = (rng.standard_normal((N, K)) * np.exp2(rng.integers(-12, 6, (N, 1)))).astype(np.float16)
    w[0, :4] = [np.float16(65504), np.float16(-65504), np.float16(6e-8), np.float16(-0.0)]
    exps = rng.integers(-24, 8, (N, K // 128))
    sv = np.ldexp(1.0 + rng.integers(0, 1024, exps.shape) / 1024.0, exps)
    scales = np.array([[py_float_to_half_bits(float(v)) for v in row] for row in sv], np.uint16)
    scales[scales == 0] = 1
    zeros = rng.integers(0, qmax + 1, (N, K // 128)).astype(np.uint8)
    c = o.codes_from_params(w, scales, zeros, bits)
    assert c.max() <= qmax
    for n in range(N):
        for k in range(K):
            g = k // 128
            v = Fraction(float(w[n, k])) / half_frac(int(scales[n, g])) + int(zeros[n, g])
            margin = abs(v) * Fraction(2) ** -22 + Fraction(2) ** -40
            assert int(c[n, k]) in _allowed_round(v, qmax, margin), (n, k, float(v), int(c[n, k]))


def pin_params_match_quantize(o, bits=3, seed=22):
    """Fed the scales and zero points that the min-max path chose, Eq. 1 gives
    back that path's codes."""
    w = inputs.weights(20, 512, cfg=93, layer=seed, proj=bits)
    codes, scales, zeros = o.quantize(w, bits)
    assert np.array_equal(o.codes_from_params(w, scales, zeros, bits), codes)


# ---------------------------------------------------------------------------
# packing pins
# ---------------------------------------------------------------------------
def _w3_words_spelled_out(q):
    """The W3 plane words of one 32-code chunk, field by field as defined."""
    q = [int(v) for v in q]
    words = []
    for p in range(3):
        b = 10 * p
        w = (q[b + 0] << 0 | q[b + 1] << 16 | q[b + 2] << 3 | q[b + 3] << 19 |
             q[b + 4] << 6 | q[b + 5] << 22 | q[b + 6] << 10 | q[b + 7] << 26 |
             q[b + 8] << 13 | q[b + 9] << 29 |
             ((q[30] >> p) & 1) << 9 | ((q[31] >> p) & 1) << 25)
        words.append(w)
    return words


def _w4_words_spelled_out(q):
    q = [int(v) for v in q]
    words = []
    for p in range(4):
        b = 8 * p
        w = (q[b + 0] << 0 | q[b + 1] << 16 | q[b + 2] << 4 | q[b + 3] << 20 |
             q[b + 4] << 8 | q[b + 5] << 24 | q[b + 6] << 12 | q[b + 7] << 28)
        words.append(w)
    return words


def pin_pack_fields(o, seed=1):
    rng = np.random.default_rng(seed)
    for bits, spell in ((3, _w3_words_spelled_out), (4, _w4_words_spelled_out)):
        N, K = 5, 256
        codes = rng.integers(0, 1 << bits, (N, K)).astype(np.uint8)
        # also single-code patterns at every position
        codes[0, :] = 0
        for i in range(32):
            codes[0, 32 * (i % 8) + i] = (1 << bits) - 1
        qw = o.pack(codes, bits)
        assert qw.shape == (N, bits, K // 32)
        for n in range(N):
            for c in range(K // 32):
                want = spell(codes[n, 32 * c:32 * c + 32])
                got = [int(qw[n, p, c]) for p in range(bits)]
                assert got == want, (bits, n, c, [hex(v) for v in got], [hex(v) for v in want])
        assert np.array_equal(o.unpack(qw, K, bits), codes)
    # every one of the 96 W3 bits is used by exactly one code bit
    codes = np.full((1, 32), 7, np.uint8)
    qw = o.pack(codes, 3)
    assert [int(v) for v in qw[0, :, 0]] == [0xFFFFFFFF] * 3


def pin_density(o, golden):
    """App. H: 32 three-bit weights in three 32-bit words; BLOCKHEIGHT =
    BLOCKWIDTH/32*3 packed rows per BLOCKWIDTH inputs; group size 128."""
    codes = np.zeros((3, golden["group_size"]), np.uint8)
    qw = o.pack(codes, 3)
    per_row_words = qw.shape[1] * qw.shape[2]
    assert per_row_words == golden["group_size"] // golden["codes_per_triple"] * golden["words_per_triple"]
    for bw in golden["blockwidths"]:
        c = np.zeros((1, bw), np.uint8)
        assert o.pack(c, 3).size == bw // 32 * 3
    c, s, z = o.quantize(np.zeros((2, 384), np.float16), 3)
    assert s.shape == (2, 384 // golden["group_size"])


# ---------------------------------------------------------------------------
# linear pins
# ---------------------------------------------------------------------------
def _numpy_dequant(codes, scales, zeros):
    s = np.array([[py_half_bits_to_float(int(b)) for b in row] for row in scales])
    return np.repeat(s, 128, axis=1) * (codes.astype(np.float64) - np.repeat(zeros.astype(np.float64), 128, axis=1))


def pin_linear_vs_numpy(o, bits=3, seed=4):
    """The oracle's fp64 linear equals numpy's float64 GEMM on w_hat (exact
    values), to 1e-12 of the output scale."""
    M, N, K = 5, 96, 640
    w = inputs.weights(N, K, cfg=93, layer=seed, proj=bits)
    x = inputs.activations(M, K, cfg=93, layer=seed)
    codes, scales, zeros = o.quantize(w, bits)
    wh = _numpy_dequant(codes, scales, zeros)
    assert np.array_equal(o.dequant(codes, scales, zeros), wh)
    y = o.linear(x, codes, scales, zeros)
    ref = x.astype(np.float64) @ wh.T
    scale = np.sqrt(np.mean(ref ** 2))
    assert np.max(np.abs(y - ref)) <= 1e-12 * scale, np.max(np.abs(y - ref)) / scale


def pin_linear_special(o, bits=3, seed=6):
    M, N, K = 3, 40, 384
    qmax = _levels(bits)
    w = inputs.weights(N, K, cfg=94, layer=seed, proj=bits)
    codes, scales, zeros = o.quantize(w, bits)
    wh = _numpy_dequant(codes, scales, zeros)
    # one-hot activation picks a single dequantized weight (one exact term)
    for k in (0, 127, 128, 300, K - 1):
        x = np.zeros((1, K), np.float16)
        x[0, k] = 1.0
        y = o.linear(x, codes, scales, zeros)
        assert np.array_equal(y[0], wh[:, k]), k
    # codes equal to the zero point give exactly zero
    c0 = np.repeat(zeros, 128, axis=1).astype(np.uint8)
    x = inputs.activations(M, K, cfg=94, layer=seed)
    assert np.all(o.linear(x, c0, scales, zeros) == 0.0)
    # scaling x by a power of two scales y exactly
    y1 = o.linear(x, codes, scales, zeros)
    y2 = o.linear((x.astype(np.float32) * 4).astype(np.float16), codes, scales, zeros)
    assert np.array_equal(y2, 4 * y1)
    # rows of a multi-row call equal single-row calls
    for m in range(M):
        assert np.array_equal(o.linear(x[m:m + 1], codes, scales, zeros)[0], y1[m])
    assert codes.max() <= qmax


def pin_linear_exact_fraction(o, seed=8):
    """Tiny case summed exactly in rationals: the fp64 oracle agrees to 1e-15."""
    M, N, K = 2, 3, 256
    w = inputs.weights(N, K, cfg=95, layer=seed)
    x = inputs.activations(M, K, cfg=95, layer=seed)
    codes, scales, zeros = o.quantize(w, 3)
    y = o.linear(x, codes, scales, zeros)
    for m in range(M):
        for n in range(N):
            acc = Fraction(0)
            for k in range(K):
                g = k // 128
                s = half_frac(int(scales[n, g]))
                acc += Fraction(float(x[m, k])) * s * (int(codes[n, k]) - int(zeros[n, g]))
            assert abs(Fraction(float(y[m, n])) - acc) <= Fraction(1, 10 ** 15) * (abs(acc) + 1), (m, n)


ALL_QUANT_PINS = (
    ("ongrid_w3", lambda o: pin_ongrid_exact(o, 3)),
    ("ongrid_w4", lambda o: pin_ongrid_exact(o, 4)),
    ("ties", pin_ties_handworked),
    ("special_w3", lambda o: pin_special_groups(o, 3)),
    ("special_w4", lambda o: pin_special_groups(o, 4)),
    ("nearest_w3", lambda o: pin_nearest_level(o, 3)),
    ("nearest_w4", lambda o: pin_nearest_level(o, 4)),
    ("permutation", pin_group_permutation),
    ("extremes", pin_extremes),
)
ALL_PARAMS_PINS = (
    ("params_handworked", pin_params_handworked),
    ("params_exact_w3", lambda o: pin_params_exact(o, 3)),
    ("params_exact_w4", lambda o: pin_params_exact(o, 4)),
    ("params_match_quantize_w3", lambda o: pin_params_match_quantize(o, 3)),
    ("params_match_quantize_w4", lambda o: pin_params_match_quantize(o, 4)),
)
ALL_PACK_PINS = (("pack_fields", pin_pack_fields),)
ALL_LINEAR_PINS = (
    ("linear_numpy_w3", lambda o: pin_linear_vs_numpy(o, 3)),
    ("linear_numpy_w4", lambda o: pin_linear_vs_numpy(o, 4)),
    ("linear_special", pin_linear_special),
    ("linear_fraction", pin_linear_exact_fraction),
)
ALL_FP16_PINS = (
    ("f16_to_f32", pin_f16_to_f32_exhaustive),
    ("f32_to_f16", pin_f32_to_f16_rne),
)

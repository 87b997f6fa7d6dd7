"""GPU parity: the HIP kernels (through the C ABI) against the CPU oracle.

Quantize: packed words, scale bits and zero bytes bit-exact.
Linear:   each fp16 output is an fp16 rounding of a value within
          1e-3 x RMS of the oracle's exact fp64 result (oracle/compare.py).
Inputs are seeded (paper_2605_08755_amd.inputs); the linear is fed the
oracle's own quantization, so its parity does not depend on the quantize
kernel.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from oracle.compare import linear_check
from paper_2605_08755_amd import inputs, laq

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def say(*a):
    print("[gpu-case]", *a, flush=True)


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def gpu_quantize(w16, bits):
    q, s, z = laq.quantize(to_dev(w16), bits)
    torch.cuda.synchronize()
    return (q.cpu().numpy().view(np.uint32), s.cpu().numpy().view(np.uint16), z.cpu().numpy())


def oracle_packed(w16, bits):
    codes, s, z = oracle.quantize(w16, bits)
    return codes, oracle.pack(codes, bits), s, z


def gpu_linear(x16, qw, s, z, bits):
    y = laq.linear(to_dev(x16), to_dev(qw.view(np.int32)), to_dev(s.view(np.float16)), to_dev(z), bits)
    torch.cuda.synchronize()
    return y.cpu().numpy()


# ---------------------------------------------------------------------------
# quantize
# ---------------------------------------------------------------------------
QSHAPES = [(1, 128), (17, 384), (33, 2560), (5, 9728), (1024, 1024), (300, 4096), (2, 25600)]


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("N,K", QSHAPES)
def test_quantize_bitexact(bits, N, K):
    say("quantize", bits, N, K)
    w = inputs.weights(N, K, cfg=10, layer=N, proj=K % 97)
    codes, qw, s, z = oracle_packed(w, bits)
    gq, gs, gz = gpu_quantize(w, bits)
    assert np.array_equal(gs, s), "scales differ"
    assert np.array_equal(gz, z), "zeros differ"
    assert np.array_equal(gq, qw), "packed codes differ"


@pytest.mark.parametrize("bits", [3, 4])
def test_quantize_special_groups(bits):
    say("quantize special", bits)
    qmax = (1 << bits) - 1
    K = 384
    rows = []
    rows.append(np.zeros(K))                                   # all zero
    rows.append(np.full(K, 0.75))                              # constant positive
    rows.append(-np.linspace(0.01, 0.5, K))                    # all negative
    r = np.zeros(K); r[17] = -3.0; rows.append(r)              # single outlier
    r = np.zeros(K); r[:5] = [6e-8, -6e-8, 1.2e-7, 0, -1.8e-7]; rows.append(r)  # subnormal range
    r = np.zeros(K); r[0], r[1] = -3 / 64, 4 / 64
    r[2:12] = np.array([2.5, 1.5, -0.5, 0.5, 3.5, -2.5, -1.5, 4.0, -3.0, 0.0]) / 64
    rows.append(r)                                             # exact ties (W3 grid)
    rng = np.random.default_rng(3)
    for e in (-14, -3, 5):                                     # on-grid groups
        z0 = int(rng.integers(0, qmax + 1))
        j = rng.integers(0, qmax + 1, K); j[0], j[1] = 0, qmax
        rows.append(np.ldexp((j - z0).astype(np.float64), e))
    rows.append(np.full(K, 65504.0))                           # largest half
    r = np.full(K, -65504.0); r[::2] = 65504.0; rows.append(r)  # widest range
    rows.append(np.full(K, -0.0))                              # negative zeros
    w = np.array(rows).astype(np.float16)
    codes, qw, s, z = oracle_packed(w, bits)
    gq, gs, gz = gpu_quantize(w, bits)
    assert np.array_equal(gs, s) and np.array_equal(gz, z) and np.array_equal(gq, qw)


def test_quantize_canary():
    """Writes stay inside the outputs: sentinels around them are untouched."""
    say("quantize canary")
    N, K = 37, 640
    w = to_dev(inputs.weights(N, K, cfg=11))
    words = laq.packed_words(3, N, K)
    G = K // 128
    qbuf = torch.full((words + 64,), 0x5A5A5A5A, dtype=torch.int32, device=DEV)
    sbuf = torch.full((N * G + 64,), 7.0, dtype=torch.float16, device=DEV)
    zbuf = torch.full((N * G + 64,), 0xEE, dtype=torch.uint8, device=DEV)
    laq.quantize(w, 3, out=(qbuf[:words], sbuf[:N * G].view(N, G), zbuf[:N * G].view(N, G)))
    torch.cuda.synchronize()
    assert torch.all(qbuf[words:] == 0x5A5A5A5A)
    assert torch.all(sbuf[N * G:] == 7.0)
    assert torch.all(zbuf[N * G:] == 0xEE)


# ---------------------------------------------------------------------------
# pack with caller-supplied scales and zero points (Eq. 1, trained parameters)
# ---------------------------------------------------------------------------
def random_params(N, K, bits, seed):
    """Positive fp16 scales from the subnormal range to 2^7, zero points 0..qmax."""
    rng = np.random.default_rng(seed)
    G = K // 128
    e = rng.integers(-24, 8, (N, G))
    sv = np.ldexp(1.0 + rng.integers(0, 1024, (N, G)) / 1024.0, e).astype(np.float16)
    sv[sv == 0] = np.float16(2.0 ** -24)
    z = rng.integers(0, (1 << bits), (N, G)).astype(np.uint8)
    return sv.view(np.uint16), z


def gpu_pack(w16, s, z, bits):
    qw = laq.pack(to_dev(w16), to_dev(s.view(np.float16)), to_dev(z), bits)
    torch.cuda.synchronize()
    return qw.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("N,K", QSHAPES)
def test_pack_bitexact(bits, N, K):
    say("pack", bits, N, K)
    w = inputs.weights(N, K, cfg=13, layer=N, proj=K % 89)
    s, z = random_params(N, K, bits, seed=N * 7 + K)
    ref = oracle.pack(oracle.codes_from_params(w, s, z, bits), bits)
    assert np.array_equal(gpu_pack(w, s, z, bits), ref)


@pytest.mark.parametrize("bits", [3, 4])
def test_pack_reproduces_quantize(bits):
    """Fed the parameters the min-max path wrote, pack gives its qweight."""
    say("pack vs quantize", bits)
    w = inputs.weights(129, 2560, cfg=14)
    gq, gs, gz = gpu_quantize(w, bits)
    assert np.array_equal(gpu_pack(w, gs, gz, bits), gq)


@pytest.mark.parametrize("bits", [3, 4])
def test_pack_special(bits):
    """Ties, clipping at both ends, extreme scales and weights."""
    say("pack special", bits)
    qmax = (1 << bits) - 1
    K = 256
    w = np.zeros((4, K))
    w[0, :12] = np.array([2.5, 1.5, -0.5, 0.5, 3.5, -2.5, -1.5, 4.0, -3.0, 0.0, 10.0, -10.0]) / 64
    w[1, :4] = [65504.0, -65504.0, 6e-8, -6e-8]
    w[2, :] = np.linspace(-8, 8, K)
    w[3, :] = -0.0
    w = w.astype(np.float16)
    s = np.array([[1 / 64, 0.5], [2.0 ** -24, 65504.0], [1.0, 2.0 ** -14], [0.25, 1.0]], np.float16).view(np.uint16)
    z = np.array([[3 % (qmax + 1), 0], [qmax, 0], [0, qmax], [1, qmax]], np.uint8)
    ref_codes = oracle.codes_from_params(w, s, z, bits)
    assert np.array_equal(gpu_pack(w, s, z, bits), oracle.pack(ref_codes, bits))


def test_pack_canary():
    """pack writes only qweight; scales and zeros are left as they were."""
    say("pack canary")
    N, K = 21, 768
    w = to_dev(inputs.weights(N, K, cfg=15))
    s, z = random_params(N, K, 3, seed=5)
    sd, zd = to_dev(s.view(np.float16)), to_dev(z)
    s0, z0 = sd.clone(), zd.clone()
    words = laq.packed_words(3, N, K)
    qbuf = torch.full((words + 64,), 0x3C3C3C3C, dtype=torch.int32, device=DEV)
    laq.pack(w, sd, zd, 3, out=qbuf[:words])
    torch.cuda.synchronize()
    assert torch.all(qbuf[words:] == 0x3C3C3C3C)
    assert torch.equal(sd, s0) and torch.equal(zd, z0)


# ---------------------------------------------------------------------------
# linear
# ---------------------------------------------------------------------------
LSHAPES = [(1, 128), (17, 384), (64, 128), (300, 2560), (1024, 1024), (4096, 1024), (257, 4096), (100, 9728), (3, 25600)]


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("M", [1, 2, 3, 4, 5, 8, 11, 16])
@pytest.mark.parametrize("N,K", LSHAPES)
def test_linear_parity(bits, M, N, K):
    say("linear", bits, M, N, K)
    w = inputs.weights(N, K, cfg=12, layer=M, proj=N % 89)
    x = inputs.activations(M, K, cfg=12, layer=N)
    codes, qw, s, z = oracle_packed(w, bits)
    y = gpu_linear(x, qw, s, z, bits)
    ref = oracle.linear(x, codes, s, z)
    r = linear_check(y, ref)
    assert r["ok"], r


@pytest.mark.parametrize("bits", [3, 4])
def test_linear_onehot_bitwise(bits):
    """x = e_k picks one exact term: y == fp16(w_hat[:, k]) bitwise."""
    say("linear onehot", bits)
    N, K = 200, 1280
    w = inputs.weights(N, K, cfg=13)
    codes, qw, s, z = oracle_packed(w, bits)
    wh = oracle.dequant(codes, s, z)
    for k in (0, 1, 29, 30, 31, 32, 127, 128, 555, K - 2, K - 1):
        x = np.zeros((1, K), np.float16)
        x[0, k] = 1.0
        y = gpu_linear(x, qw, s, z, bits)
        assert np.array_equal(y[0], wh[:, k].astype(np.float16)), k


@pytest.mark.parametrize("bits", [3, 4])
def test_linear_zero_codes_and_scaling(bits):
    say("linear zero/pow2", bits)
    M, N, K = 4, 130, 768
    w = inputs.weights(N, K, cfg=14)
    x = inputs.activations(M, K, cfg=14)
    codes, qw, s, z = oracle_packed(w, bits)
    # all-zero weights quantize to codes 0, zero point 0: y is exactly zero
    wz = np.zeros((N, K), np.float16)
    cz, qz, sz, zz = oracle_packed(wz, bits)
    assert np.all(gpu_linear(x, qz, sz, zz, bits) == 0)
    # codes equal to a nonzero zero point (a state quantize never produces):
    # the kernel forms sum x*q and z*sum x separately, so the result is the
    # fp32 rounding residue of that cancellation, bounded by a few fp32 ulps
    # of s*z*sum|x| per group (v_dot2_f32_f16 does not round each step to
    # nearest; see the design notes)
    c0 = np.repeat(z, 128, axis=1).astype(np.uint8)
    y0 = gpu_linear(x, oracle.pack(c0, bits), s, z, bits).astype(np.float64)
    sv = oracle.f16_to_f32(s).astype(np.float64)
    ax = np.abs(x.astype(np.float64)).reshape(M, K // 128, 128).sum(axis=2)      # [M][G]
    bound = (ax[:, None, :] * (sv * z)[None, :, :]).sum(axis=2) * 2.0 ** -16      # [M][N]
    assert np.all(np.abs(y0) <= bound + 2.0 ** -24), float(np.max(np.abs(y0) / (bound + 1e-30)))
    # y(4x) == 4 y(x) bitwise (power-of-two scaling is exact end to end)
    y1 = gpu_linear(x, qw, s, z, bits)
    y4 = gpu_linear((x.astype(np.float32) * 4).astype(np.float16), qw, s, z, bits)
    assert np.array_equal(y4, (y1.astype(np.float32) * 4).astype(np.float16))


@pytest.mark.parametrize("bits", [3, 4])
def test_linear_rows_consistent_and_deterministic(bits):
    say("linear rows/determinism", bits)
    N, K = 512, 2560
    w = inputs.weights(N, K, cfg=15)
    x = inputs.activations(16, K, cfg=15)
    codes, qw, s, z = oracle_packed(w, bits)
    y16 = gpu_linear(x, qw, s, z, bits)
    y16b = gpu_linear(x, qw, s, z, bits)
    assert np.array_equal(y16, y16b)
    ref = oracle.linear(x, codes, s, z)
    for m in (0, 7, 15):
        y1 = gpu_linear(x[m:m + 1], qw, s, z, bits)
        assert linear_check(y1[0], ref[m])["ok"]
        # both are within tolerance of the same exact value
        assert np.max(np.abs(y1[0].astype(np.float64) - y16[m])) <= 2e-3 * np.sqrt(np.mean(ref[m] ** 2)) + \
            np.max(np.abs(ref[m])) * 2 ** -10


def test_linear_canary():
    say("linear canary")
    M, N, K = 3, 77, 640
    w = inputs.weights(N, K, cfg=16)
    x = inputs.activations(M, K, cfg=16)
    codes, qw, s, z = oracle_packed(w, 3)
    ybuf = torch.full((M * N + 128,), 3.0, dtype=torch.float16, device=DEV)
    laq.linear(to_dev(x), to_dev(qw.view(np.int32)), to_dev(s.view(np.float16)), to_dev(z), 3,
               out=ybuf[:M * N].view(M, N))
    torch.cuda.synchronize()
    assert torch.all(ybuf[M * N:] == 3.0)
    r = linear_check(ybuf[:M * N].view(M, N).cpu().numpy(), oracle.linear(x, codes, s, z))
    assert r["ok"], r


def test_two_streams():
    say("two streams")
    M, N, K = 2, 2048, 2560
    w = inputs.weights(N, K, cfg=17)
    x = inputs.activations(M, K, cfg=17)
    codes, qw, s, z = oracle_packed(w, 3)
    ref = gpu_linear(x, qw, s, z, 3)
    xd, qd, sd, zd = to_dev(x), to_dev(qw.view(np.int32)), to_dev(s.view(np.float16)), to_dev(z)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    for st in (s1, s2, s1, s2):
        with torch.cuda.stream(st):
            outs.append(laq.linear(xd, qd, sd, zd, 3))
    torch.cuda.synchronize()
    for o in outs:
        assert np.array_equal(o.cpu().numpy(), ref)


# ---------------------------------------------------------------------------
# full-size shapes (the Qwen3-4B layer; Qwen3-32B projections on sampled rows)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("bits", [3, 4])
def test_layer4b_full(bits):
    """All seven Qwen3-4B projections at full size: GPU quantize bit-exact,
    GPU linear (M = 1 and 16) on the GPU-quantized weights vs the oracle."""
    for pi, (name, N, K) in enumerate(inputs.QWEN3_4B):
        say("layer4b", bits, name, N, K)
        w = inputs.weights(N, K, cfg=2, layer=0, proj=pi)
        codes, qw, s, z = oracle_packed(w, bits)
        gq, gs, gz = gpu_quantize(w, bits)
        assert np.array_equal(gs, s) and np.array_equal(gz, z) and np.array_equal(gq, qw), name
        for M in (1, 16):
            x = inputs.activations(M, K, cfg=2, layer=0, slot=inputs.X_SLOT[name])
            y = gpu_linear(x, gq, gs, gz, bits)
            r = linear_check(y, oracle.linear(x, codes, s, z))
            assert r["ok"], (name, M, r)


def test_stack32b_sampled():
    """Qwen3-32B projection shapes at full size on the GPU; the oracle checks
    every output of sampled rows (quantize is per row, so sampling rows of
    the weight matrix gives the same codes)."""
    rng = np.random.default_rng(32)
    for pi, (name, N, K) in enumerate(inputs.QWEN3_32B):
        if name in ("k", "v", "up"):
            continue
        say("stack32b", name, N, K)
        w = inputs.weights(N, K, cfg=5, layer=0, proj=pi)
        rows = np.sort(rng.choice(N, 96, replace=False))
        codes, qw, s, z = oracle_packed(np.ascontiguousarray(w[rows]), 3)
        wd = to_dev(w)
        q, sd, zd = laq.quantize(wd, 3)
        del wd
        torch.cuda.synchronize()
        assert np.array_equal(sd[rows].cpu().numpy().view(np.uint16), s)
        assert np.array_equal(zd[rows].cpu().numpy(), z)
        assert np.array_equal(q[rows].cpu().numpy().view(np.uint32), qw)
        for M in (1, 16):
            x = inputs.activations(M, K, cfg=5, layer=0, slot=inputs.X_SLOT[name])
            y = laq.linear(to_dev(x), q, sd, zd, 3)
            torch.cuda.synchronize()
            r = linear_check(y.cpu().numpy()[:, rows], oracle.linear(x, codes, s, z))
            assert r["ok"], (name, M, r)
        del q, sd, zd
        torch.cuda.empty_cache()


@pytest.mark.parametrize("bits", [3, 4])
def test_max_k(bits):
    """The largest K the ABI accepts (2^24): quantize and pack bit-exact, and
    the linear at M = 1 (K-tiled kernel: the activation row exceeds LDS), 2
    and 16 (matrix cores, many quad batches per wave) against the oracle."""
    K = 1 << 24
    N = 3
    say("max K", bits, N, K)
    rng = np.random.default_rng(77)
    w = (rng.standard_normal((N, K), dtype=np.float32) * 0.02).astype(np.float16)
    codes, qw, s, z = oracle_packed(w, bits)
    gq, gs, gz = gpu_quantize(w, bits)
    assert np.array_equal(gs, s) and np.array_equal(gz, z) and np.array_equal(gq, qw)
    assert np.array_equal(gpu_pack(w, s, z, bits), qw)
    for M in (1, 2, 16):
        x = rng.standard_normal((M, K), dtype=np.float32).astype(np.float16)
        y = gpu_linear(x, qw, s, z, bits)
        r = linear_check(y, oracle.linear(x, codes, s, z))
        assert r["ok"], (M, r)


QUAD_WAVE_SHAPES = [(17, 128), (300, 640), (1030, 2560), (257, 4992), (4100, 5120), (16400, 1152), (10256, 4992),
                    (257, 5248)]


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("N,K", QUAD_WAVE_SHAPES)
def test_matrix_core_quad_wave(bits, N, K):
    """Rows of at most 10 quads: one 16-row tile per block, one wave per quad.
    A single group (K = 128), a partial last quad (K = 640, five groups;
    K = 4992, 39 groups, ten quads), ten full quads (K = 5120), a ragged last
    tile (N = 17, 300, 1030, 257, 4100), at least 1024 tiles (N = 16400, the
    kernel keeps them up to M = 8), more waves than stay resident with the
    fragments read up front (N = 10256, K = 4992: 641 tiles x 10 waves, the
    64-register form), and K = 5248 (eleven quads: just past the kernel's
    limit).  M from 3 (four-row slab; rows of at most 24 groups
    included) to 16 (sixteen-row slab)."""
    say("mfma quad wave", bits, N, K)
    w = inputs.weights(N, K, cfg=22, layer=bits, proj=K % 97)
    codes, qw, s, z = oracle_packed(w, bits)
    for M in (3, 4, 5, 8, 9, 16):
        x = inputs.activations(M, K, cfg=22, layer=M)
        y = gpu_linear(x, qw, s, z, bits)
        r = linear_check(y, oracle.linear(x, codes, s, z))
        assert r["ok"], (M, r)


SHARE_SHAPES = [(16437, 2176), (16400, 128), (19456, 2560), (16389, 1664)]


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("N,K", SHARE_SHAPES)
def test_matrix_core_quad_share(bits, N, K):
    """At least 1024 tiles, rows of at most five quads, M > 4 (W4: M > 8, the
    one-tile blocks below that): three tiles per block sharing the quads'
    activation slabs (8 rows up to M = 8, 16 above).
    A last block with two real tiles and an idle one, the last tile ragged
    (N = 16437 = 1027 * 16 + 5, 1028 tiles) and a last quad of one group
    (K = 2176, 17 groups); a single group (K = 128); the Qwen3-4B gate|up
    shape; a last block with one real tile (N = 16389: 1025 tiles, ragged) and
    four quads (K = 1664, 13 groups).  Repeated calls are bit-identical."""
    say("mfma quad share", bits, N, K)
    w = inputs.weights(N, K, cfg=23, layer=bits, proj=K % 89)
    codes, qw, s, z = oracle_packed(w, bits)
    for M in (5, 8, 9, 16):
        x = inputs.activations(M, K, cfg=23, layer=M)
        y = gpu_linear(x, qw, s, z, bits)
        r = linear_check(y, oracle.linear(x, codes, s, z))
        assert r["ok"], (M, r)
        assert np.array_equal(gpu_linear(x, qw, s, z, bits).view(np.uint16), y.view(np.uint16)), M


@pytest.mark.parametrize("bits", [3, 4])
def test_matrix_core_two_tiles_ragged(bits):
    """Rows longer than 10 quads, enough 16-row tiles (>= 256) and long
    enough rows for each wave to take two tiles, with a last block holding a
    partial tile (N = 4100 = 256 * 16 + 4) and a partial last quad (K = 9728,
    76 groups: 19 quads)."""
    N, K = 4100, 9728
    say("mfma two tiles", bits, N, K)
    w = inputs.weights(N, K, cfg=16, layer=bits)
    codes, qw, s, z = oracle_packed(w, bits)
    for M in (3, 8, 16):
        x = inputs.activations(M, K, cfg=16, layer=M)
        y = gpu_linear(x, qw, s, z, bits)
        r = linear_check(y, oracle.linear(x, codes, s, z))
        assert r["ok"], (M, r)


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("N,K", [(16404, 640), (16400, 128), (16448, 2560)])
def test_matrix_core_shared_slab(bits, N, K):
    """Enough 16-row tiles (>= 1024) and M > 8 for blocks of four tiles
    sharing the activation slabs through LDS (K <= 2560: all quads in one
    round trip): a last block with a partial tile and idle waves (N = 16404 =
    1025 * 16 + 4), a partial last 4-group quad (K = 640, five groups) and a
    single group (K = 128).  M = 2, 3 and 8 take the other kernels on the
    same weights."""
    say("mfma shared slab", bits, N, K)
    w = inputs.weights(N, K, cfg=17, layer=bits, proj=K % 97)
    codes, qw, s, z = oracle_packed(w, bits)
    for M in (2, 3, 8, 9, 12, 16):
        x = inputs.activations(M, K, cfg=17, layer=M)
        y = gpu_linear(x, qw, s, z, bits)
        r = linear_check(y, oracle.linear(x, codes, s, z))
        assert r["ok"], (M, r)


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("K", [3072, 4096])
def test_matrix_core_walk_four_tiles(bits, K):
    """1024..3071 row tiles at M > 8 walk K in blocks of four tiles, the quad
    weights in three register sets in turn: K = 3072 (6 quads, the unrolled
    loop ends exactly) and 4096 (8 quads, two quads after the loop); N =
    16400 = 1025 * 16 (a last block with one tile).  M = 3 takes the
    one-wave-per-quad kernel on the same weights.  Sampled rows and the last
    rows."""
    N = 16400
    say("mfma walk four tiles", bits, N, K)
    rng = np.random.default_rng(K + bits)
    w = inputs.weights(N, K, cfg=19, layer=bits, proj=K % 97)
    rows = np.concatenate([np.sort(rng.choice(N - 16, 48, replace=False)), np.arange(N - 16, N)])
    codes, qw, s, z = oracle_packed(np.ascontiguousarray(w[rows]), bits)
    wd = to_dev(w)
    q, sd, zd = laq.quantize(wd, bits)
    del wd
    torch.cuda.synchronize()
    assert np.array_equal(q[rows].cpu().numpy().view(np.uint32), qw)
    for M in (3, 12, 16):
        x = inputs.activations(M, K, cfg=19, layer=M)
        y = laq.linear(to_dev(x), q, sd, zd, bits)
        torch.cuda.synchronize()
        r = linear_check(y.cpu().numpy()[:, rows], oracle.linear(x, codes, s, z))
        assert r["ok"], (M, r)
    del q, sd, zd


@pytest.mark.parametrize("M", [3, 5])
def test_matrix_core_two_tiles_per_wave_small_m(M):
    """Fewer than 1024 tiles, at least 256 of them and rows of more than 10
    quads: each wave takes two tiles, and its two KiB of partials reuse an
    activation slab of only M rows.  N = 4100 (ragged), K = 6144 (12 quads)."""
    N, K = 4100, 6144
    say("mfma two tiles per wave", M, N, K)
    w = inputs.weights(N, K, cfg=20, layer=M)
    x = inputs.activations(M, K, cfg=20, layer=M)
    codes, qw, s, z = oracle_packed(w, 3)
    y = gpu_linear(x, qw, s, z, 3)
    r = linear_check(y, oracle.linear(x, codes, s, z))
    assert r["ok"], r


def test_matrix_core_walk_ragged():
    """From 3072 row tiles at M > 8, blocks of eight tiles walk K one quad at
    a time (K > 2560): N = 49168 = 3073 * 16 (a last block with one tile),
    K = 3200 (25 groups: a partial last quad).  M = 3 and 8 take the
    one-wave-per-quad kernel on the same weights.  Quantize on the GPU; codes
    and outputs checked on sampled rows and the last rows."""
    N, K = 49168, 3200
    say("mfma walk ragged", N, K)
    rng = np.random.default_rng(49)
    w = inputs.weights(N, K, cfg=18, layer=3, proj=7)
    rows = np.concatenate([np.sort(rng.choice(N - 16, 80, replace=False)), np.arange(N - 16, N)])
    codes, qw, s, z = oracle_packed(np.ascontiguousarray(w[rows]), 3)
    wd = to_dev(w)
    q, sd, zd = laq.quantize(wd, 3)
    del wd
    torch.cuda.synchronize()
    assert np.array_equal(q[rows].cpu().numpy().view(np.uint32), qw)
    for M in (3, 8, 11, 16):
        x = inputs.activations(M, K, cfg=18, layer=M)
        y = laq.linear(to_dev(x), q, sd, zd, 3)
        torch.cuda.synchronize()
        r = linear_check(y.cpu().numpy()[:, rows], oracle.linear(x, codes, s, z))
        assert r["ok"], (M, r)
    del q, sd, zd
    torch.cuda.empty_cache()


SPLIT_SHAPES = [(5120, 25600), (100, 25088), (3, 20608), (1030, 20480)]


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("N,K", SPLIT_SHAPES)
def test_split_k(bits, N, K):
    """K split across workgroups of four row tiles (rows of >= 40 quads, fewer
    than 1024 tiles): the Qwen3-32B down projection (ranges of five quads), a
    partial last quad (K = 25088: 196 groups; K = 20608: 161), a last block
    with idle tiles (N = 100, 1030) and a single partial tile (N = 3), ranges
    of one quad; against the oracle, deterministic, and the plain entry point
    also within tolerance."""
    say("split K", bits, N, K)
    assert laq.workspace_bytes(16, N, K) > 0
    w = inputs.weights(N, K, cfg=19, layer=bits, proj=K % 83)
    codes, qw, s, z = oracle_packed(w, bits)
    qd, sd, zd = to_dev(qw.view(np.int32)), to_dev(s.view(np.float16)), to_dev(z)
    for M in (2, 3, 5, 8, 16):
        x = inputs.activations(M, K, cfg=19, layer=M)
        xd = to_dev(x)
        y1 = laq.linear(xd, qd, sd, zd, bits)
        y2 = laq.linear(xd, qd, sd, zd, bits)
        yp = laq.linear(xd, qd, sd, zd, bits, split_k=False)
        torch.cuda.synchronize()
        ref = oracle.linear(x, codes, s, z)
        assert torch.equal(y1, y2), M
        r = linear_check(y1.cpu().numpy(), ref)
        assert r["ok"], (M, r)
        r = linear_check(yp.cpu().numpy(), ref)
        assert r["ok"], (M, "plain", r)


def test_split_k_small_workspace():
    """A workspace smaller than laq_linear_workspace_bytes: the _ws call is
    the plain call, bit for bit."""
    N, K, M = 1030, 20480, 16
    say("split K small workspace", N, K, M)
    w = inputs.weights(N, K, cfg=20, layer=1)
    codes, qw, s, z = oracle_packed(w, 3)
    qd, sd, zd = to_dev(qw.view(np.int32)), to_dev(s.view(np.float16)), to_dev(z)
    xd = to_dev(inputs.activations(M, K, cfg=20, layer=2))
    need = laq.workspace_bytes(M, N, K)
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    y = torch.empty((M, N), dtype=torch.float16, device=DEV)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    st = laq.lib().laq_linear_ws_w3g128(ctypes.c_void_p(xd.data_ptr()), ctypes.c_void_p(qd.data_ptr()),
                                        ctypes.c_void_p(sd.data_ptr()), ctypes.c_void_p(zd.data_ptr()),
                                        ctypes.c_void_p(y.data_ptr()), M, N, K, ctypes.c_void_p(ws.data_ptr()),
                                        need - 16, stream)
    assert st == laq.LAQ_OK
    yp = laq.linear(xd, qd, sd, zd, 3, split_k=False)
    torch.cuda.synchronize()
    assert torch.equal(y, yp)


# ---------------------------------------------------------------------------
# grouped calls: several independent linears in one launch
# ---------------------------------------------------------------------------
def _group_case(bits, specs, M, cfg):
    """specs: list of (N, K, x_slot); calls sharing a slot share x."""
    xs = {}
    calls, refs = [], []
    for i, (N, K, slot) in enumerate(specs):
        if slot not in xs:
            xs[slot] = inputs.activations(M, K, cfg=cfg, layer=slot)
        x = xs[slot]
        w = inputs.weights(N, K, cfg=cfg, layer=i, proj=bits)
        codes, qw, s, z = oracle_packed(w, bits)
        calls.append((to_dev(x), to_dev(qw.view(np.int32)), to_dev(s.view(np.float16)), to_dev(z)))
        refs.append(oracle.linear(x, codes, s, z))
    ys = laq.linear_group(calls, bits)
    singles = [laq.linear(*c, bits) for c in calls]
    torch.cuda.synchronize()
    return [y.cpu().numpy() for y in ys], [y.cpu().numpy() for y in singles], refs


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("M", [1, 2, 3, 4, 8, 16])
def test_group_qkv(bits, M):
    """q, k, v of a Qwen3-4B layer (same activations) as one launch.  Up to
    M = 2 the grouped and the single calls run the same VALU kernel body and
    agree bit for bit; at M = 3 and 4 the group stays on the VALU kernel
    (its rows are short) while a single call takes the matrix cores."""
    say("group qkv", bits, M)
    ys, singles, refs = _group_case(bits, [(4096, 2560, 0), (1024, 2560, 0), (1024, 2560, 0)], M, cfg=40)
    for y, y1, ref in zip(ys, singles, refs):
        r = linear_check(y, ref)
        assert r["ok"], r
        if M <= 2:  # the same kernel body, bit for bit
            assert np.array_equal(y.view(np.uint16), y1.view(np.uint16))


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("M", [1, 2, 16])
def test_group_mixed(bits, M):
    """Eight calls of different shapes (the most a group takes): several K,
    ragged N, a single row, separate activations."""
    say("group mixed", bits, M)
    specs = [(2560, 4096, 0), (257, 9728, 1), (1, 128, 2), (300, 2560, 3), (17, 384, 4),
             (1024, 1024, 5), (96, 9728, 1), (64, 128, 6)]
    ys, singles, refs = _group_case(bits, specs, M, cfg=41)
    for y, y1, ref in zip(ys, singles, refs):
        r = linear_check(y, ref)
        assert r["ok"], r
        if M <= 2:
            assert np.array_equal(y.view(np.uint16), y1.view(np.uint16))


@pytest.mark.parametrize("bits", [3, 4])
def test_group_long_rows_one_row(bits):
    """M = 1 with a row longer than LDS holds: one launch per call, same results."""
    say("group long rows", bits)
    ys, singles, refs = _group_case(bits, [(5, 32768, 0), (3, 32768, 0)], 1, cfg=42)
    for y, y1, ref in zip(ys, singles, refs):
        assert linear_check(y, ref)["ok"]
        assert np.array_equal(y.view(np.uint16), y1.view(np.uint16))


# ---------------------------------------------------------------------------
# graph capture: every kernel path replayed several times, each replay equal
# (bitwise) to the eager call, with eager work of the same kernels between
# ---------------------------------------------------------------------------
GRAPH_CASES = [
    ("flat M=2 two rows per lane", 2, 300, 9728, 3),
    ("matrix cores one wave per quad M=5", 5, 1030, 4096, 4),
    ("matrix cores one wave per quad M=16", 16, 300, 5120, 3),
    ("matrix cores one wave per quad, 64 registers M=4", 4, 10256, 4992, 3),
    ("matrix cores one tile M=5", 5, 1030, 9728, 4),
    ("matrix cores four tiles M=16", 16, 16400, 2560, 3),
    ("matrix cores walk M=12", 12, 16400, 4096, 3),
    ("split K with workspace M=16", 16, 1030, 25600, 3),
]


@pytest.mark.parametrize("name,M,N,K,bits", GRAPH_CASES)
def test_graph_replay(name, M, N, K, bits):
    say("graph replay", name, M, N, K, bits)
    w = to_dev(inputs.weights(N, K, cfg=21, layer=M))
    x = to_dev(inputs.activations(M, K, cfg=21, layer=M))
    q, s, z = laq.quantize(w, bits)
    y_eager = laq.linear(x, q, s, z, bits)
    torch.cuda.synchronize()
    qg, sg, zg = torch.empty_like(q), torch.empty_like(s), torch.empty_like(z)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=torch.cuda.Stream()):
        laq.quantize(w, bits, out=(qg, sg, zg))
        y_graph = laq.linear(x, qg, sg, zg, bits)
    for _ in range(3):
        for t in (qg, sg, zg, y_graph):
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(qg, q) and torch.equal(sg, s) and torch.equal(zg, z), name
        assert torch.equal(y_graph.view(torch.int16), y_eager.view(torch.int16)), name
        # eager work of the same kernels between replays
        y2 = laq.linear(x, q, s, z, bits)
        torch.cuda.synchronize()
        assert torch.equal(y2.view(torch.int16), y_eager.view(torch.int16)), name
    del g

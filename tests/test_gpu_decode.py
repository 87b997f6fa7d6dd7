"""Decode-step operations on the GPU (through the C ABI) against the float64
oracle (oracle/decode.py), and one full Qwen3-4B-shaped decoder layer
(quantized linears + these operations) against the oracle's composition."""
import numpy as np
import pytest
import torch

import oracle
from oracle import decode as OD
from oracle.compare import linear_check
from paper_2605_08755_amd import inputs, laq

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
EPS = 1e-6
THETA = 1e6


def say(*a):
    print("[gpu-case]", *a, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def cos_sin_table(S, d=128, theta=THETA):
    """fp32 [S][d]: cos of the d/2 angles of each position, then their sin."""
    a = np.arange(S, dtype=np.float64)[:, None] * theta ** (-2.0 * np.arange(d // 2) / d)[None, :]
    return np.concatenate([np.cos(a), np.sin(a)], axis=1).astype(np.float32)


def f16(rng, shape, scale=1.0):
    return (rng.standard_normal(shape) * scale).astype(np.float16)


@pytest.mark.parametrize("M,D,with_delta", [(1, 2560, True), (3, 5120, True), (2, 100, True), (1, 2560, False)])
def test_add_rmsnorm(M, D, with_delta):
    say("add_rmsnorm", M, D, with_delta)
    rng = np.random.default_rng(D + M)
    res = rng.standard_normal((M, D)).astype(np.float32) * 3
    delta = f16(rng, (M, D)) if with_delta else None
    w = (1 + 0.1 * rng.standard_normal(D)).astype(np.float16)
    r_ref, y_ref = OD.add_rmsnorm(res, delta, w, EPS)
    rd = dev(res)
    y = laq.add_rmsnorm(rd, dev(delta) if with_delta else None, dev(w), EPS)
    torch.cuda.synchronize()
    assert np.allclose(rd.cpu().numpy(), r_ref, rtol=1e-6, atol=1e-6)
    r = linear_check(y.cpu().numpy(), y_ref)
    assert r["ok"], r


@pytest.mark.parametrize("Hq,Hkv,pos", [(32, 8, 0), (32, 8, 37), (32, 8, 1023), (8, 8, 5), (64, 8, 700)])
def test_qk_norm_rope(Hq, Hkv, pos):
    say("qk_norm_rope", Hq, Hkv, pos)
    S = 1024
    rng = np.random.default_rng(Hq * 7 + pos)
    qkv = f16(rng, (Hq + 2 * Hkv) * 128, 2.0)
    qw = (1 + 0.2 * rng.standard_normal(128)).astype(np.float16)
    kw = (1 + 0.2 * rng.standard_normal(128)).astype(np.float16)
    cs = cos_sin_table(S)
    canary = f16(rng, (Hkv, S, 128))
    kc, vc = dev(canary), dev(canary)
    q = laq.qk_norm_rope(dev(qkv), dev(qw), dev(kw), dev(cs), pos, Hq, Hkv, EPS, kc, vc)
    torch.cuda.synchronize()
    q_ref, k_ref, v_ref = OD.qk_norm_rope(qkv, qw, kw, pos, Hq, Hkv, 128, EPS, THETA)
    for got, ref in ((q.cpu().numpy(), q_ref), (kc.cpu().numpy()[:, pos], k_ref)):
        r = linear_check(got, ref)
        assert r["ok"], r
    kh, vh = kc.cpu().numpy(), vc.cpu().numpy()
    assert np.array_equal(vh[:, pos], qkv[(Hq + Hkv) * 128:].reshape(Hkv, 128))  # v copied exactly
    others = np.arange(S) != pos
    assert np.array_equal(kh[:, others], canary[:, others]) and np.array_equal(vh[:, others], canary[:, others])


@pytest.mark.parametrize("Hq,Hkv,L", [(32, 8, 1), (32, 8, 63), (32, 8, 64), (32, 8, 65), (32, 8, 1000),
                                      (8, 8, 130), (16, 8, 257), (64, 8, 999)])
def test_decode_attention(Hq, Hkv, L):
    say("decode_attention", Hq, Hkv, L)
    S = 1024
    rng = np.random.default_rng(L * 3 + Hq)
    K = f16(rng, (Hkv, S, 128))
    V = f16(rng, (Hkv, S, 128))
    q = f16(rng, (Hq, 128), 1.5)
    out = laq.decode_attention(dev(q), dev(K), dev(V), L)
    torch.cuda.synchronize()
    ref = OD.decode_attention(q, K[:, :L], V[:, :L])
    r = linear_check(out.cpu().numpy(), ref)
    assert r["ok"], r
    # deterministic
    out2 = laq.decode_attention(dev(q), dev(K), dev(V), L)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), out2.view(torch.int16))


@pytest.mark.parametrize("Hq,Hkv,pos,S", [(32, 8, 0, 64), (32, 8, 15, 64), (32, 8, 16, 64), (32, 8, 300, 1024),
                                           (32, 8, 511, 1024), (32, 8, 512, 1024), (32, 8, 1023, 1024),
                                           (32, 8, 4095, 4100), (32, 8, 4096, 4100), (8, 8, 63, 300),
                                           (8, 8, 64, 300), (16, 8, 257, 300), (64, 8, 999, 1024),
                                           (4, 2, 33, 40), (8, 1, 100, 128)])
def test_decode_attention_qkv(Hq, Hkv, pos, S):
    """laq_decode_attention_qkv_f16 (q/k RMSNorm + rotary embedding + cache
    append + attention in one pass over the cache) against the oracle's
    qk_norm_rope and attention (q rounded to fp16 as the separate call stores
    it), across every tile length (16, 32, 64 positions), tile boundaries,
    contexts of one position and query heads per key/value head of 1 to 8;
    the cache rows other than pos stay untouched."""
    say("decode_attention_qkv", Hq, Hkv, pos, S)
    rng = np.random.default_rng(Hq * 1000 + pos)
    qkv = f16(rng, (Hq + 2 * Hkv) * 128, 2.0)
    qw = (1 + 0.2 * rng.standard_normal(128)).astype(np.float16)
    kw = (1 + 0.2 * rng.standard_normal(128)).astype(np.float16)
    cs = cos_sin_table(S)
    Kc = f16(rng, (Hkv, S, 128))
    Vc = f16(rng, (Hkv, S, 128))
    kc, vc = dev(Kc), dev(Vc)
    out = laq.decode_attention_qkv(dev(qkv), dev(qw), dev(kw), dev(cs), pos, Hq, Hkv, EPS, kc, vc)
    torch.cuda.synchronize()
    q_ref, k_ref, v_ref = OD.qk_norm_rope(qkv, qw, kw, pos, Hq, Hkv, 128, EPS, THETA)
    kh, vh = kc.cpu().numpy(), vc.cpu().numpy()
    r = linear_check(kh[:, pos], k_ref)
    assert r["ok"], r
    assert np.array_equal(vh[:, pos], v_ref.astype(np.float16))
    others = np.arange(S) != pos
    assert np.array_equal(kh[:, others], Kc[:, others]) and np.array_equal(vh[:, others], Vc[:, others])
    ref = OD.decode_attention(q_ref.astype(np.float16), kh[:, :pos + 1], vh[:, :pos + 1])
    r = linear_check(out.cpu().numpy(), ref)
    assert r["ok"], r
    # deterministic, and the caches' row pos rewritten with the same values
    out2 = laq.decode_attention_qkv(dev(qkv), dev(qw), dev(kw), dev(cs), pos, Hq, Hkv, EPS, kc, vc)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), out2.view(torch.int16))
    assert np.array_equal(kc.cpu().numpy(), kh) and np.array_equal(vc.cpu().numpy(), vh)


@pytest.mark.parametrize("M,I", [(1, 9728), (2, 100), (1, 25600)])
def test_silu_mul(M, I):
    say("silu_mul", M, I)
    rng = np.random.default_rng(I + M)
    gu = f16(rng, (M, 2 * I), 3.0)
    y = laq.silu_mul(dev(gu))
    torch.cuda.synchronize()
    r = linear_check(y.cpu().numpy(), OD.silu_mul(gu, I))
    assert r["ok"], r


@pytest.mark.parametrize("M,I,K,bits", [(1, 9728, 2560, 3), (2, 100, 1024, 3), (3, 53, 4096, 4), (1, 37, 16384, 3),
                                         (4, 64, 128, 3), (1, 1, 640, 4)])
def test_linear_swiglu(M, I, K, bits):
    """Gate|up linear with SiLU-and-multiply in its output stage against the
    oracle's linear (fp64, unrounded) followed by its silu_mul, on weight rows
    interleaved gate j, up j."""
    say("linear_swiglu", M, I, K, bits)
    w = inputs.weights(2 * I, K, cfg=41, proj=bits)
    x = inputs.activations(M, K, cfg=41)
    codes, s, z = oracle.quantize(w, bits)
    y = laq.linear_swiglu(dev(x), dev(oracle.pack(codes, bits).view(np.int32)), dev(s.view(np.float16)), dev(z),
                          bits)
    torch.cuda.synchronize()
    full = np.asarray(oracle.linear(x, codes, s, z), dtype=np.float64)
    ref = OD.silu_mul(np.concatenate([full[:, 0::2], full[:, 1::2]], axis=1), I)
    r = linear_check(y.cpu().numpy(), ref)
    assert r["ok"], r


NORM_LINEAR_CASES = [(3, False, 6144, 2560, True), (4, False, 6144, 2560, True), (3, False, 4100, 4096, True),
                     (3, False, 300, 8192, True), (3, False, 25000, 2560, True), (3, False, 1031, 2560, False),
                     (3, True, 2 * 9728, 2560, True), (4, True, 2 * 37, 1024, True), (3, True, 2 * 150, 8192, False),
                     (3, False, 300, 128, True), (4, False, 517, 1024, False), (3, False, 40000, 2560, True)]


@pytest.mark.parametrize("bits,swiglu,N,K,with_delta", NORM_LINEAR_CASES)
def test_add_rmsnorm_linear(bits, swiglu, N, K, with_delta):
    """laq_add_rmsnorm_linear (residual add + RMSNorm computed by every block
    of the linear while it stages the row, then the linear; with swiglu the
    SiLU-and-multiply output stage) against the oracle: the new residual
    bitwise equal to residual + delta in fp32, the output against the
    oracle's linear (fp64) on the oracle's RMSNorm rounded to fp16, within the
    linear tolerance.  Rows of 1, 8, 20, 32 and 64 groups (256- and
    512-thread blocks), 25000 rows (two rows per lane), ragged N, no delta;
    the inputs are left untouched."""
    say("add_rmsnorm_linear", bits, swiglu, N, K, with_delta)
    rng = np.random.default_rng(N + K + bits)
    res = (rng.standard_normal((1, K)) * 3).astype(np.float32)
    delta = f16(rng, (1, K)) if with_delta else None
    w = (1 + 0.1 * rng.standard_normal(K)).astype(np.float16)
    wt = inputs.weights(N, K, cfg=44, layer=bits, proj=N % 97)
    codes, sc, z = oracle.quantize(wt, bits)
    rd, dd, wd = dev(res), (dev(delta) if with_delta else None), dev(w)
    ro = torch.full((1, K), float("nan"), dtype=torch.float32, device=DEV)
    y = laq.add_rmsnorm_linear(rd, dd, wd, EPS, dev(oracle.pack(codes, bits).view(np.int32)),
                               dev(sc.view(np.float16)), dev(z), bits, swiglu=swiglu, residual_out=ro)
    torch.cuda.synchronize()
    r_exp = res + (delta.astype(np.float32) if with_delta else np.float32(0))
    assert np.array_equal(ro.cpu().numpy(), r_exp)
    assert np.array_equal(rd.cpu().numpy(), res) and np.array_equal(wd.cpu().numpy(), w)
    _, x_ref = OD.add_rmsnorm(res, delta, w, EPS)
    full = np.asarray(oracle.linear(np.asarray(x_ref).astype(np.float16), codes, sc, z), dtype=np.float64)
    ref = OD.silu_mul(np.concatenate([full[:, 0::2], full[:, 1::2]], axis=1), N // 2) if swiglu else full
    r = linear_check(y.cpu().numpy(), ref)
    assert r["ok"], r
    # deterministic, and without residual_out
    y2 = laq.add_rmsnorm_linear(rd, dd, wd, EPS, dev(oracle.pack(codes, bits).view(np.int32)),
                                dev(sc.view(np.float16)), dev(z), bits, swiglu=swiglu)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16))


RESIDUAL_CASES = [(3, 2560, 4096), (3, 2560, 9728), (4, 2560, 4096), (3, 4100, 2048), (3, 1000, 8192),
                  (4, 517, 9728), (3, 33, 2560)]


@pytest.mark.parametrize("bits,N,K", RESIDUAL_CASES)
def test_linear_residual(bits, N, K):
    """laq_linear_residual (a batch-1 linear that also writes residual_in + y
    to the residual stream): y against the oracle's linear within the linear
    tolerance and bit for bit equal to the plain laq_linear call; the new
    residual bitwise equal to residual_in + y in fp32; in place as well, and
    with y NULL (the residual alone written, bit for bit the same).
    Qwen3-4B's o (2560 x 4096) and down (2560 x 9728, two rows per lane), a
    ragged 4100 x 2048, 1000 x 8192, W4, 33 rows."""
    say("linear_residual", bits, N, K)
    rng = np.random.default_rng(N + K + bits)
    x = inputs.activations(1, K, cfg=47, layer=bits)
    w = inputs.weights(N, K, cfg=47, layer=bits, proj=K % 89)
    codes, sc, z = oracle.quantize(w, bits)
    q, sd, zd = dev(oracle.pack(codes, bits).view(np.int32)), dev(sc.view(np.float16)), dev(z)
    res = (rng.standard_normal((1, N)) * 3).astype(np.float32)
    rd = dev(res)
    ro = torch.full((1, N), float("nan"), dtype=torch.float32, device=DEV)
    y = laq.linear_residual(dev(x), q, sd, zd, rd, ro, bits)
    y_plain = laq.linear(dev(x), q, sd, zd, bits)
    torch.cuda.synchronize()
    r = linear_check(y.cpu().numpy(), oracle.linear(x, codes, sc, z))
    assert r["ok"], r
    assert torch.equal(y.view(torch.int16), y_plain.view(torch.int16))
    expect = res + y.cpu().numpy().astype(np.float32)
    assert np.array_equal(ro.cpu().numpy(), expect)
    assert np.array_equal(rd.cpu().numpy(), res)
    ro2 = torch.full((1, N), float("nan"), dtype=torch.float32, device=DEV)
    assert laq.linear_residual(dev(x), q, sd, zd, rd, ro2, bits, write_out=False) is None  # y NULL: residual only
    laq.linear_residual(dev(x), q, sd, zd, rd, rd, bits)  # in place
    torch.cuda.synchronize()
    assert np.array_equal(ro2.cpu().numpy(), expect)
    assert np.array_equal(rd.cpu().numpy(), expect)


MLP_CASES = [(2560, 9728, True), (256, 384, True), (1024, 128, False), (1280, 128 * 77, True), (2560, 1152, False)]


@pytest.mark.parametrize("D,I,with_delta", MLP_CASES)
def test_add_rmsnorm_mlp(D, I, with_delta):
    """laq_add_rmsnorm_mlp_w3g128 (the SwiGLU MLP block in one launch: the
    norm prologue, gate|up with SiLU-and-multiply per slice of 128
    intermediates, the slice's share of down, partials added by the
    last-arriving workgroups) against the oracle's composition: the new
    residual bitwise equal to residual + delta, y against the oracle's down
    linear (fp64) on h = silu(gate) * up from the oracle's gate|up linear on
    the oracle's RMSNorm (x and h rounded to fp16 where the kernel rounds
    them), within the linear tolerance.  Qwen3-4B's D = 2560, I = 9728 (76
    slices in 9 teams), 3 slices (teams of 2 and 1), one slice, 77 slices (a
    last team of 5), no delta.  Then three more calls on the same workspace
    (its counters reset by each call) and three replays of a HIP-graph
    capture give y bit for bit."""
    say("add_rmsnorm_mlp", D, I, with_delta)
    rng = np.random.default_rng(D + I)
    res = (rng.standard_normal((1, D)) * 3).astype(np.float32)
    delta = f16(rng, (1, D)) if with_delta else None
    w = (1 + 0.1 * rng.standard_normal(D)).astype(np.float16)
    hgu, gu = _quantized(2 * I, D, 46, 0, I % 89, interleave_halves=True)
    hdn, dn = _quantized(D, I, 46, 1, D % 89)
    rd, dd, wd = dev(res), (dev(delta) if with_delta else None), dev(w)
    ro = torch.full((1, D), float("nan"), dtype=torch.float32, device=DEV)
    ws = laq.mlp_workspace(D, I, DEV)
    y = laq.add_rmsnorm_mlp(rd, dd, wd, EPS, gu, dn, ws, residual_out=ro)
    torch.cuda.synchronize()
    r_exp = res + (delta.astype(np.float32) if with_delta else np.float32(0))
    assert np.array_equal(ro.cpu().numpy(), r_exp)
    assert np.array_equal(rd.cpu().numpy(), res)
    _, x_ref = OD.add_rmsnorm(res, delta, w, EPS)
    full = np.asarray(oracle.linear(np.asarray(x_ref).astype(np.float16), *hgu), dtype=np.float64)
    h_ref = OD.silu_mul(np.concatenate([full[:, 0::2], full[:, 1::2]], axis=1), I)
    y_ref = oracle.linear(np.asarray(h_ref).astype(np.float16), *hdn)
    r = linear_check(y.cpu().numpy(), y_ref)
    assert r["ok"], r
    S = I // 128
    T = 1
    while T * T < S:
        T += 1
    T = -(-S // -(-S // T))  # teams of ceil(S / T) slices
    assert not ws[(S + T) * D * 4:].any()  # the counters are zero again
    for _ in range(3):
        y2 = laq.add_rmsnorm_mlp(rd, dd, wd, EPS, gu, dn, ws)
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), y2.view(torch.int16))
    out = torch.empty_like(y)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=torch.cuda.Stream()):
        laq.add_rmsnorm_mlp(rd, dd, wd, EPS, gu, dn, ws, out=out)
    for _ in range(3):
        out.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), y.view(torch.int16))
    del graph


def test_decoder_layer_4b():
    """One Qwen3-4B-shaped decoder layer at position pos = 300 with a filled
    cache: W3 linears and the decode operations on the GPU, against the oracle's
    linear (on the same codes) and decode operations, stage by stage on the
    GPU's own fp16 stage inputs and end to end on the residual."""
    say("decoder layer 4b")
    Hq, Hkv, D, I, S, pos = 32, 8, 2560, 9728, 512, 300
    rng = np.random.default_rng(11)
    w_in = (1 + 0.1 * rng.standard_normal(D)).astype(np.float16)
    w_post = (1 + 0.1 * rng.standard_normal(D)).astype(np.float16)
    qn = (1 + 0.1 * rng.standard_normal(128)).astype(np.float16)
    kn = (1 + 0.1 * rng.standard_normal(128)).astype(np.float16)
    proj = {}
    for name, N, K in (("qkv", (Hq + 2 * Hkv) * 128, D), ("o", D, Hq * 128), ("gateup", 2 * I, D), ("down", D, I)):
        w = inputs.weights(N, K, cfg=40, proj=len(proj))
        codes, s, z = oracle.quantize(w, 3)
        proj[name] = (codes, s, z, dev(oracle.pack(codes, 3).view(np.int32)), dev(s.view(np.float16)), dev(z))
    x0 = rng.standard_normal((1, D)).astype(np.float32)
    Kc = f16(rng, (Hkv, S, 128))
    Vc = f16(rng, (Hkv, S, 128))
    cs = cos_sin_table(S)

    res = dev(x0)
    kc, vc = dev(Kc), dev(Vc)
    h = laq.add_rmsnorm(res, None, dev(w_in), EPS)
    qkv = laq.linear(h, *proj["qkv"][3:], 3)
    q = laq.qk_norm_rope(qkv, dev(qn), dev(kn), dev(cs), pos, Hq, Hkv, EPS, kc, vc)
    a = laq.decode_attention(q, kc, vc, pos + 1)
    o = laq.linear(a.view(1, Hq * 128), *proj["o"][3:], 3)
    h2 = laq.add_rmsnorm(res, o, dev(w_post), EPS)
    gu = laq.linear(h2, *proj["gateup"][3:], 3)
    m = laq.silu_mul(gu)
    dn = laq.linear(m, *proj["down"][3:], 3)
    torch.cuda.synchronize()
    g = {k: t.cpu().numpy() for k, t in dict(h=h, qkv=qkv, q=q, a=a, o=o, h2=h2, gu=gu, m=m, dn=dn).items()}
    r_mid = res.cpu().numpy()

    def lin(xh, name):
        c, s, z = proj[name][:3]
        return oracle.linear(xh, c, s, z)

    # stage by stage: each GPU stage against the oracle on the GPU's own inputs
    checks = {
        "h": (g["h"], OD.add_rmsnorm(x0, None, w_in, EPS)[1]),
        "qkv": (g["qkv"], lin(g["h"], "qkv")),
        "q": (g["q"], OD.qk_norm_rope(g["qkv"], qn, kn, pos, Hq, Hkv, 128, EPS, THETA)[0]),
    }
    Kf, Vf = Kc.copy(), Vc.copy()
    _, k_new, v_new = OD.qk_norm_rope(g["qkv"], qn, kn, pos, Hq, Hkv, 128, EPS, THETA)
    Kf[:, pos] = kc.cpu().numpy()[:, pos]
    Vf[:, pos] = vc.cpu().numpy()[:, pos]
    assert linear_check(Kf[:, pos], k_new)["ok"] and np.array_equal(Vf[:, pos], v_new.astype(np.float16))
    checks["a"] = (g["a"], OD.decode_attention(g["q"], Kf[:, :pos + 1], Vf[:, :pos + 1]))
    checks["o"] = (g["o"], lin(g["a"].reshape(1, -1), "o"))
    r_ref, h2_ref = OD.add_rmsnorm(x0, g["o"], w_post, EPS)
    checks["h2"] = (g["h2"], h2_ref)
    checks["gu"] = (g["gu"], lin(g["h2"], "gateup"))
    checks["m"] = (g["m"], OD.silu_mul(g["gu"], I))
    checks["dn"] = (g["dn"], lin(g["m"], "down"))
    for name, (got, ref) in checks.items():
        r = linear_check(got, ref)
        assert r["ok"], (name, r)
    assert np.allclose(r_mid, r_ref, rtol=1e-6, atol=1e-5)


def _quantized(N, K, cfg, layer, proj, interleave_halves=False):
    """Oracle-quantized W3 weights of one projection: (codes, scales, zeros)
    on the host and (qweight, scales, zeros) on the GPU.  interleave_halves:
    rows reordered gate 0, up 0, gate 1, ... (quantization is per row)."""
    w = inputs.weights(N, K, cfg=cfg, layer=layer, proj=proj)
    if interleave_halves:
        w = np.stack([w[: N // 2], w[N // 2:]], axis=1).reshape(N, K)
    codes, s, z = oracle.quantize(w, 3)
    return (codes, s, z), (dev(oracle.pack(codes, 3).view(np.int32)), dev(s.view(np.float16)), dev(z))


@pytest.mark.parametrize("fused,fused_attention", [(False, False), (True, True), (False, True)])
def test_decode_step_vs_oracle(fused, fused_attention):
    """paper_2605_08755_amd.decode.DecodeStep over two Qwen3-4B-shaped layers
    plus an LM head (4096 vocabulary rows), W3 linears on oracle-quantized
    codes, at position 200 of a filled cache, against the oracle's
    composition: every stage of every layer (norms, q|k|v, the rotated q and
    the cache rows written, attention, o, gate|up or the fused gate|up +
    SiLU, down, the residual stream, the final norm and the logits) is
    checked against oracle/decode.py and the oracle's linear applied to the
    GPU's own fp16 input of that stage, within the linear tolerance (1e-3 x
    output RMS before the output's fp16 rounding; the fp32 residual stream
    to 1e-6 relative).  fused: the gate|up linear with SiLU-and-multiply in
    its output stage.  fused_attention: the q/k norm, rotary embedding, cache
    append and attention in one call (the rotated q is then not materialized:
    attention is checked against the oracle's q rounded to fp16).  Then the
    step (no recording) is captured in a HIP graph: three replays, with eager
    steps between them, each give logits bitwise equal to the checked eager
    step."""
    say("decode step vs oracle, fused =", fused, "fused attention =", fused_attention)
    from paper_2605_08755_amd import decode
    shape = dict(decode.QWEN3_4B, layers=2, vocab=4096)
    D, Hq, Hkv, I, S, V, pos = shape["hidden"], shape["heads"], shape["kv_heads"], shape["mlp"], 256, 4096, 200
    rng = np.random.default_rng(13 + fused)
    host, lins = [], []
    for l in range(2):
        hl, fl = {}, []
        for j, (name, N, K) in enumerate((("qkv", (Hq + 2 * Hkv) * 128, D), ("o", D, Hq * 128),
                                          ("gu", 2 * I, D), ("down", D, I))):
            hq, (q, s, z) = _quantized(N, K, 43, l, j, interleave_halves=fused and name == "gu")
            hl[name] = hq
            if name == "gu" and fused:
                f = lambda x, out, q=q, s=s, z=z: laq.linear_swiglu(x, q, s, z, 3, out=out)
                f.swiglu = True
            else:
                f = lambda x, out, q=q, s=s, z=z: laq.linear(x, q, s, z, 3, out=out)
            fl.append(f)
        host.append(hl)
        lins.append(fl)
    h_lm, (q_lm, s_lm, z_lm) = _quantized(V, D, 43, 9, 0)
    lm = lambda x, out: laq.linear(x, q_lm, s_lm, z_lm, 3, out=out)
    norms_h = [tuple((1 + 0.1 * rng.standard_normal(n)).astype(np.float16) for n in (D, D, 128, 128))
               for _ in range(2)]
    fin_h = (1 + 0.1 * rng.standard_normal(D)).astype(np.float16)
    kc_h = [f16(rng, (Hkv, S, 128)) for _ in range(2)]
    vc_h = [f16(rng, (Hkv, S, 128)) for _ in range(2)]
    x0_h = rng.standard_normal((1, D)).astype(np.float32)
    norms = [tuple(dev(a) for a in nl) for nl in norms_h]
    kcs, vcs = [dev(a) for a in kc_h], [dev(a) for a in vc_h]

    rec = []

    def recording(kind, l, f):
        def g(x, out):
            f(x, out)
            e = {"kind": kind, "layer": l, "x": x.clone(), "out": out.clone(), "res": step.residual.clone()}
            if kind == "o":
                e["q"] = step.q.clone()
            rec.append(e)
        g.swiglu = getattr(f, "swiglu", False)
        return g

    names = ("qkv", "o", "gu", "down")
    rec_lins = [tuple(recording(names[j], l, lins[l][j]) for j in range(4)) for l in range(2)]
    step = decode.DecodeStep(shape, rec_lins, norms, dev(fin_h), kcs, vcs, DEV, lm_head=recording("lm", 2, lm),
                             fused_attention=fused_attention)
    step.x0.copy_(dev(x0_h))
    logits = step.run(pos).clone()
    torch.cuda.synchronize()
    g = {(e["kind"], e["layer"]): {k: (v.cpu().numpy() if hasattr(v, "cpu") else v) for k, v in e.items()}
         for e in rec}
    assert len(g) == 9

    def check(name, got, ref):
        r = linear_check(got, ref)
        assert r["ok"], (name, r)

    def lin(xh, hq):
        return oracle.linear(xh, *hq)

    r_ref = x0_h.astype(np.float64)
    for l in range(2):
        w_in, w_post, qn, kn = norms_h[l]
        e_qkv, e_o, e_gu, e_dn = (g[(k, l)] for k in names)
        if l > 0:
            r_ref = g[("gu", l - 1)]["res"].astype(np.float64) + g[("down", l - 1)]["out"].astype(np.float64)
        assert np.allclose(e_qkv["res"], r_ref, rtol=1e-6, atol=1e-6), ("residual", l)
        check(("h", l), e_qkv["x"], OD.rmsnorm(e_qkv["res"], w_in, EPS))
        check(("qkv", l), e_qkv["out"], lin(e_qkv["x"], host[l]["qkv"]))
        q_ref, k_ref, v_ref = OD.qk_norm_rope(e_qkv["out"], qn, kn, pos, Hq, Hkv, 128, EPS, THETA)
        if fused_attention:
            q_att = q_ref.astype(np.float16)  # the rounding the fused call applies to q
        else:
            check(("q", l), e_o["q"], q_ref)
            q_att = e_o["q"]
        kc, vc = kcs[l].cpu().numpy(), vcs[l].cpu().numpy()
        check(("k cache row", l), kc[:, pos], k_ref)
        assert np.array_equal(vc[:, pos], v_ref.astype(np.float16)), ("v cache row", l)
        others = np.arange(S) != pos
        assert np.array_equal(kc[:, others], kc_h[l][:, others]) and np.array_equal(vc[:, others], vc_h[l][:, others])
        check(("attention", l), e_o["x"].reshape(Hq, 128),
              OD.decode_attention(q_att, kc[:, :pos + 1], vc[:, :pos + 1]))
        check(("o", l), e_o["out"], lin(e_o["x"], host[l]["o"]))
        assert np.allclose(e_gu["res"], e_o["res"].astype(np.float64) + e_o["out"].astype(np.float64),
                           rtol=1e-6, atol=1e-6), ("residual + o", l)
        check(("h2", l), e_gu["x"], OD.rmsnorm(e_gu["res"], w_post, EPS))
        gu_ref = lin(e_gu["x"], host[l]["gu"])
        if fused:
            # rows interleaved gate j, up j: the oracle's unrounded sums, then SiLU-and-multiply
            check(("gate|up + silu", l), e_gu["out"],
                  OD.silu_mul(np.concatenate([gu_ref[:, 0::2], gu_ref[:, 1::2]], axis=1), I))
            assert np.array_equal(e_dn["x"], e_gu["out"])
        else:
            check(("gate|up", l), e_gu["out"], gu_ref)
            check(("silu_mul", l), e_dn["x"], OD.silu_mul(e_gu["out"], I))
        check(("down", l), e_dn["out"], lin(e_dn["x"], host[l]["down"]))
    r_fin = g[("gu", 1)]["res"].astype(np.float64) + g[("down", 1)]["out"].astype(np.float64)
    assert np.allclose(step.residual.cpu().numpy(), r_fin, rtol=1e-6, atol=1e-6)
    check("final norm", g[("lm", 2)]["x"], OD.rmsnorm(r_fin, fin_h, EPS))
    check("logits", logits.cpu().numpy(), lin(g[("lm", 2)]["x"], h_lm))

    # the same step without recording, captured in a HIP graph
    gstep = decode.DecodeStep(shape, [tuple(f) for f in lins], norms, dev(fin_h), kcs, vcs, DEV, lm_head=lm,
                              fused_attention=fused_attention)
    gstep.x0.copy_(dev(x0_h))
    eager = gstep.run(pos).clone()
    torch.cuda.synchronize()
    assert torch.equal(eager.view(torch.int16), logits.view(torch.int16))
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=torch.cuda.Stream()):
        gstep.run(pos)
    for _ in range(3):
        gstep.logits.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(gstep.logits.view(torch.int16), logits.view(torch.int16))
        gstep.run(pos)  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(gstep.logits.view(torch.int16), logits.view(torch.int16))
    del graph


@pytest.mark.parametrize("merged_mlp", [False, True])
def test_decode_step_fused_norms_vs_oracle(merged_mlp):
    """DecodeStep with the norms before q|k|v, before gate|up and before the
    LM head inside those linears (laq.add_rmsnorm_linear; gate|up with the
    SiLU output stage) over two Qwen3-4B-shaped layers plus an LM head (4096
    rows), W3 on oracle-quantized codes, at position 200 of a filled cache:
    each fused call's new residual equals its input residual plus its delta
    (fp32), its output matches the oracle's linear on the oracle's RMSNorm of
    that residual, and attention, o and down match the oracle on the GPU's own
    stage inputs, within the linear tolerance; the logits of a HIP-graph
    capture of the step, replayed three times with eager steps between,
    equal the eager step's bit for bit.  merged_mlp: the MLP block (norm,
    gate|up, SiLU, down) as one laq.add_rmsnorm_mlp call, its output checked
    against the oracle's down linear on the oracle's h of the oracle's norm."""
    say("decode step with fused norms vs oracle, merged mlp =", merged_mlp)
    from paper_2605_08755_amd import decode
    shape = dict(decode.QWEN3_4B, layers=2, vocab=4096)
    D, Hq, Hkv, I, S, V, pos = shape["hidden"], shape["heads"], shape["kv_heads"], shape["mlp"], 256, 4096, 200
    rng = np.random.default_rng(29)
    rec = []

    def fused(kind, l, q, s, z, swiglu):
        def f(x, out):  # the plain linear (unused by the step when norm_linear is present)
            laq.linear(x, q, s, z, 3, out=out)

        def g(res, delta, w, eps, res_out, out):
            laq.add_rmsnorm_linear(res, delta, w, eps, q, s, z, 3, swiglu=swiglu, out=out, residual_out=res_out)
            rec.append({"kind": kind, "layer": l, "res": res.clone(), "delta": None if delta is None else delta.clone(),
                        "res_out": None if res_out is None else res_out.clone(), "out": out.clone()})
        f.norm_linear = g
        f.swiglu = swiglu
        return f

    def merged(l, gu, dn):
        f = fused("gu", l, *gu, True)

        def g(res, delta, w, eps, res_out, out):
            laq.add_rmsnorm_mlp(res, delta, w, eps, gu, dn, mlp_ws, out=out, residual_out=res_out)
            rec.append({"kind": "mlp", "layer": l, "res": res.clone(), "delta": delta.clone(),
                        "res_out": res_out.clone(), "out": out.clone()})
        f.norm_mlp = g
        return f

    mlp_ws = laq.mlp_workspace(2560, 9728, DEV)

    def plain(kind, l, q, s, z):
        def f(x, out):
            laq.linear(x, q, s, z, 3, out=out)
            rec.append({"kind": kind, "layer": l, "x": x.clone(), "out": out.clone()})
        return f

    host, lins, dev_w = [], [], {}
    for l in range(2):
        hl, fl = {}, []
        for j, (name, N, K) in enumerate((("qkv", (Hq + 2 * Hkv) * 128, D), ("o", D, Hq * 128),
                                          ("gu", 2 * I, D), ("down", D, I))):
            hq, (q, s, z) = _quantized(N, K, 45, l, j, interleave_halves=name == "gu")
            hl[name] = hq
            fl.append(fused(name, l, q, s, z, name == "gu") if name in ("qkv", "gu") else plain(name, l, q, s, z))
            dev_w[(name, l)] = (q, s, z)
        if merged_mlp:
            fl[2] = merged(l, dev_w[("gu", l)], dev_w[("down", l)])
        host.append(hl)
        lins.append(fl)
    h_lm, (q_lm, s_lm, z_lm) = _quantized(V, D, 45, 9, 0)
    norms_h = [tuple((1 + 0.1 * rng.standard_normal(n)).astype(np.float16) for n in (D, D, 128, 128))
               for _ in range(2)]
    fin_h = (1 + 0.1 * rng.standard_normal(D)).astype(np.float16)
    kc_h = [f16(rng, (Hkv, S, 128)) for _ in range(2)]
    vc_h = [f16(rng, (Hkv, S, 128)) for _ in range(2)]
    x0_h = rng.standard_normal((1, D)).astype(np.float32)
    norms = [tuple(dev(a) for a in nl) for nl in norms_h]
    kcs, vcs = [dev(a) for a in kc_h], [dev(a) for a in vc_h]
    step = decode.DecodeStep(shape, [tuple(f) for f in lins], norms, dev(fin_h), kcs, vcs, DEV,
                             lm_head=fused("lm", 2, q_lm, s_lm, z_lm, False))
    step.x0.copy_(dev(x0_h))
    logits = step.run(pos).clone()
    torch.cuda.synchronize()
    g = {(e["kind"], e["layer"]): {k: (v.cpu().numpy() if hasattr(v, "cpu") else v) for k, v in e.items()}
         for e in rec}
    assert len(g) == (7 if merged_mlp else 9)
    if merged_mlp:
        # the one-launch MLP block stands for the gate|up and down records
        for l in range(2):
            e = g.pop(("mlp", l))
            g[("gu", l)] = {k: e[k] for k in ("res", "delta", "res_out")}
            g[("down", l)] = {"out": e["out"]}

    def check(name, got, ref):
        r = linear_check(got, ref)
        assert r["ok"], (name, r)

    def normed(e, w):
        if e["delta"] is None:  # no delta: the residual stays put (no residual_out)
            assert e["res_out"] is None
            return np.asarray(OD.rmsnorm(e["res"], w, EPS)).astype(np.float16)
        r_out = e["res"] + e["delta"].astype(np.float32)
        assert np.array_equal(e["res_out"], r_out)
        return np.asarray(OD.rmsnorm(r_out, w, EPS)).astype(np.float16)

    def res_after(e):  # the residual stream after a norm
        return e["res"] if e["res_out"] is None else e["res_out"]

    assert np.array_equal(g[("qkv", 0)]["res"], x0_h) and g[("qkv", 0)]["delta"] is None
    for l in range(2):
        w_in, w_post, qn, kn = norms_h[l]
        e_qkv, e_o, e_gu, e_dn = (g[(k, l)] for k in ("qkv", "o", "gu", "down"))
        if l > 0:
            assert np.array_equal(e_qkv["res"], res_after(g[("gu", l - 1)]))
            assert np.array_equal(e_qkv["delta"], g[("down", l - 1)]["out"])
        check(("qkv", l), e_qkv["out"], oracle.linear(normed(e_qkv, w_in), *host[l]["qkv"]))
        q_ref, k_ref, v_ref = OD.qk_norm_rope(e_qkv["out"], qn, kn, pos, Hq, Hkv, 128, EPS, THETA)
        kc, vc = kcs[l].cpu().numpy(), vcs[l].cpu().numpy()
        check(("k cache row", l), kc[:, pos], k_ref)
        assert np.array_equal(vc[:, pos], v_ref.astype(np.float16))
        check(("attention", l), e_o["x"].reshape(Hq, 128),
              OD.decode_attention(q_ref.astype(np.float16), kc[:, :pos + 1], vc[:, :pos + 1]))
        check(("o", l), e_o["out"], oracle.linear(e_o["x"], *host[l]["o"]))
        assert np.array_equal(e_gu["res"], res_after(e_qkv)) and np.array_equal(e_gu["delta"], e_o["out"])
        full = np.asarray(oracle.linear(normed(e_gu, w_post), *host[l]["gu"]), dtype=np.float64)
        h_ref = OD.silu_mul(np.concatenate([full[:, 0::2], full[:, 1::2]], axis=1), I)
        if merged_mlp:
            check(("mlp block", l), e_dn["out"], oracle.linear(np.asarray(h_ref).astype(np.float16), *host[l]["down"]))
            continue
        check(("gate|up + silu", l), e_gu["out"], h_ref)
        assert np.array_equal(e_dn["x"], e_gu["out"])
        check(("down", l), e_dn["out"], oracle.linear(e_dn["x"], *host[l]["down"]))
    e_lm = g[("lm", 2)]
    assert np.array_equal(e_lm["res"], res_after(g[("gu", 1)])) and np.array_equal(e_lm["delta"], g[("down", 1)]["out"])
    check("logits", logits.cpu().numpy(), oracle.linear(normed(e_lm, fin_h), *h_lm))
    assert np.array_equal(step.residual.cpu().numpy(), res_after(e_lm))

    # HIP graph of the same step (recording wrappers copy tensors, which the graph captures too)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=torch.cuda.Stream()):
        step.run(pos)
    for _ in range(3):
        step.logits.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(step.logits.view(torch.int16), logits.view(torch.int16))
        step.run(pos)
        torch.cuda.synchronize()
        assert torch.equal(step.logits.view(torch.int16), logits.view(torch.int16))


def test_decode_step_residual_producers_vs_oracle():
    """DecodeStep with the norms inside q|k|v, gate|up (SiLU output stage) and
    the LM head, and with o and down adding their outputs to the residual
    stream themselves (laq.linear_residual), so that every norm runs with no
    delta: two Qwen3-4B-shaped layers plus an LM head (4096 rows), W3 on
    oracle-quantized codes, at position 200 of a filled cache.  Each
    producer's output matches the oracle's linear on its own input and its new
    residual equals its input residual plus that output (fp32, bit for bit);
    each norm's residual is the last producer's (the token's embedding first)
    and its linear matches the oracle's linear on the oracle's RMSNorm of it;
    attention matches the oracle; three replays of a HIP-graph capture give
    the eager logits bit for bit, and so do producers that write only the
    residual (y NULL)."""
    say("decode step with residual producers vs oracle")
    from paper_2605_08755_amd import decode
    shape = dict(decode.QWEN3_4B, layers=2, vocab=4096)
    D, Hq, Hkv, I, S, V, pos = shape["hidden"], shape["heads"], shape["kv_heads"], shape["mlp"], 256, 4096, 200
    rng = np.random.default_rng(31)
    rec = []
    no_y = False

    def norm_lin(kind, l, q, s, z, swiglu):
        def f(x, out):  # unused by the step (norm_linear is present)
            laq.linear(x, q, s, z, 3, out=out)

        def g(res, delta, w, eps, res_out, out):
            laq.add_rmsnorm_linear(res, delta, w, eps, q, s, z, 3, swiglu=swiglu, out=out, residual_out=res_out)
            rec.append({"kind": kind, "layer": l, "res": res.clone(), "delta": None if delta is None else delta.clone(),
                        "res_out": None if res_out is None else res_out.clone(), "out": out.clone()})
        f.norm_linear = g
        f.swiglu = swiglu
        return f

    def producer(kind, l, q, s, z):
        def f(x, out):  # unused by the step (residual_linear is present)
            laq.linear(x, q, s, z, 3, out=out)

        def g(x, r_in, r_out, out):
            if no_y:  # the residual alone (y NULL), as a step that reads nothing else
                laq.linear_residual(x, q, s, z, r_in, r_out, 3, write_out=False)
                return
            laq.linear_residual(x, q, s, z, r_in, r_out, 3, out=out)
            rec.append({"kind": kind, "layer": l, "x": x.clone(), "res_in": r_in.clone(), "res_out": r_out.clone(),
                        "out": out.clone()})
        f.residual_linear = g
        return f

    host, lins = [], []
    for l in range(2):
        hl, fl = {}, []
        for j, (name, N, K) in enumerate((("qkv", (Hq + 2 * Hkv) * 128, D), ("o", D, Hq * 128),
                                          ("gu", 2 * I, D), ("down", D, I))):
            hq, (q, s, z) = _quantized(N, K, 48, l, j, interleave_halves=name == "gu")
            hl[name] = hq
            fl.append(norm_lin(name, l, q, s, z, name == "gu") if name in ("qkv", "gu") else producer(name, l, q, s, z))
        host.append(hl)
        lins.append(fl)
    h_lm, (q_lm, s_lm, z_lm) = _quantized(V, D, 48, 9, 0)
    norms_h = [tuple((1 + 0.1 * rng.standard_normal(n)).astype(np.float16) for n in (D, D, 128, 128))
               for _ in range(2)]
    fin_h = (1 + 0.1 * rng.standard_normal(D)).astype(np.float16)
    kc_h = [f16(rng, (Hkv, S, 128)) for _ in range(2)]
    vc_h = [f16(rng, (Hkv, S, 128)) for _ in range(2)]
    x0_h = rng.standard_normal((1, D)).astype(np.float32)
    norms = [tuple(dev(a) for a in nl) for nl in norms_h]
    kcs, vcs = [dev(a) for a in kc_h], [dev(a) for a in vc_h]
    step = decode.DecodeStep(shape, [tuple(f) for f in lins], norms, dev(fin_h), kcs, vcs, DEV,
                             lm_head=norm_lin("lm", 2, q_lm, s_lm, z_lm, False))
    step.x0.copy_(dev(x0_h))
    logits = step.run(pos).clone()
    torch.cuda.synchronize()
    g = {(e["kind"], e["layer"]): {k: (v.cpu().numpy() if hasattr(v, "cpu") else v) for k, v in e.items()}
         for e in rec}
    assert len(g) == 9

    def check(name, got, ref):
        r = linear_check(got, ref)
        assert r["ok"], (name, r)

    def normed(e, w):
        assert e["delta"] is None and e["res_out"] is None  # no delta: the residual stays put
        return np.asarray(OD.rmsnorm(e["res"], w, EPS)).astype(np.float16)

    def produced(e, hq):
        check((e["kind"], e["layer"]), e["out"], oracle.linear(e["x"], *hq))
        assert np.array_equal(e["res_out"], e["res_in"] + e["out"].astype(np.float32)), e["kind"]

    res_prev = x0_h
    for l in range(2):
        w_in, w_post, qn, kn = norms_h[l]
        e_qkv, e_o, e_gu, e_dn = (g[(k, l)] for k in ("qkv", "o", "gu", "down"))
        assert np.array_equal(e_qkv["res"], res_prev)
        check(("qkv", l), e_qkv["out"], oracle.linear(normed(e_qkv, w_in), *host[l]["qkv"]))
        q_ref, k_ref, v_ref = OD.qk_norm_rope(e_qkv["out"], qn, kn, pos, Hq, Hkv, 128, EPS, THETA)
        kc, vc = kcs[l].cpu().numpy(), vcs[l].cpu().numpy()
        check(("k cache row", l), kc[:, pos], k_ref)
        assert np.array_equal(vc[:, pos], v_ref.astype(np.float16))
        check(("attention", l), e_o["x"].reshape(Hq, 128),
              OD.decode_attention(q_ref.astype(np.float16), kc[:, :pos + 1], vc[:, :pos + 1]))
        assert np.array_equal(e_o["res_in"], e_qkv["res"])
        produced(e_o, host[l]["o"])
        assert np.array_equal(e_gu["res"], e_o["res_out"])
        full = np.asarray(oracle.linear(normed(e_gu, w_post), *host[l]["gu"]), dtype=np.float64)
        check(("gate|up + silu", l), e_gu["out"], OD.silu_mul(np.concatenate([full[:, 0::2], full[:, 1::2]], axis=1), I))
        assert np.array_equal(e_dn["x"], e_gu["out"]) and np.array_equal(e_dn["res_in"], e_gu["res"])
        produced(e_dn, host[l]["down"])
        res_prev = e_dn["res_out"]
    e_lm = g[("lm", 2)]
    assert np.array_equal(e_lm["res"], res_prev)
    check("logits", logits.cpu().numpy(), oracle.linear(normed(e_lm, fin_h), *h_lm))

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=torch.cuda.Stream()):
        step.run(pos)
    for _ in range(3):
        step.logits.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(step.logits.view(torch.int16), logits.view(torch.int16))
        step.run(pos)
        torch.cuda.synchronize()
        assert torch.equal(step.logits.view(torch.int16), logits.view(torch.int16))
    # the producers writing only the residual (y NULL): the same logits
    no_y = True
    step.logits.zero_()
    step.run(pos)
    torch.cuda.synchronize()
    assert torch.equal(step.logits.view(torch.int16), logits.view(torch.int16))

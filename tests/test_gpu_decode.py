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


def test_decode_step_graph_replay():
    """paper_2605_08755_amd.decode.DecodeStep over two Qwen3-4B-shaped layers
    with W3 linears: HIP-graph replays equal the eager step bitwise, and the
    step equals the same calls issued one by one."""
    say("decode step graph")
    from paper_2605_08755_amd import decode
    shape = dict(decode.QWEN3_4B, layers=2)
    D, Hq, Hkv, I, S = shape["hidden"], shape["heads"], shape["kv_heads"], shape["mlp"], 256
    rng = np.random.default_rng(12)
    lins, norms, kcs, vcs = [], [], [], []
    for l in range(2):
        fs = []
        for j, (N, K) in enumerate((((Hq + 2 * Hkv) * 128, D), (D, Hq * 128), (2 * I, D), (D, I))):
            q, s, z = laq.quantize(dev(inputs.weights(N, K, cfg=41, layer=l, proj=j)), 3)
            fs.append(lambda x, out, q=q, s=s, z=z: laq.linear(x, q, s, z, 3, out=out))
        lins.append(tuple(fs))
        norms.append(tuple(dev((1 + 0.1 * rng.standard_normal(n)).astype(np.float16)) for n in (D, D, 128, 128)))
        kcs.append(dev(f16(rng, (Hkv, S, 128))))
        vcs.append(dev(f16(rng, (Hkv, S, 128))))
    fin = dev((1 + 0.1 * rng.standard_normal(D)).astype(np.float16))
    step = decode.DecodeStep(shape, lins, norms, fin, kcs, vcs, DEV)
    step.x0.copy_(dev(rng.standard_normal((1, D)).astype(np.float32)))
    pos = 200
    eager = step.run(pos).clone()
    torch.cuda.synchronize()
    assert torch.isfinite(eager.float()).all()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=torch.cuda.Stream()):
        step.run(pos)
    for _ in range(3):
        step.out.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(step.out.view(torch.int16), eager.view(torch.int16))
        step.run(pos)  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(step.out.view(torch.int16), eager.view(torch.int16))
    del g


def test_decode_step_fused_swiglu():
    """DecodeStep with the gate|up linear that applies SiLU-and-multiply in its
    output stage (weight rows interleaved gate j, up j) against the same step
    with the plain gate|up linear followed by silu_mul, over two Qwen3-4B-shaped
    layers.  The fused call skips the fp16 rounding of gate and up, so the two
    agree to the fp16 precision of the step, not bitwise."""
    say("decode step fused swiglu")
    from paper_2605_08755_amd import decode
    shape = dict(decode.QWEN3_4B, layers=2)
    D, Hq, Hkv, I, S = shape["hidden"], shape["heads"], shape["kv_heads"], shape["mlp"], 256
    rng = np.random.default_rng(13)
    plain, fused, norms, kcs, vcs = [], [], [], [], []
    for l in range(2):
        fs, ff = [], []
        for j, (N, K) in enumerate((((Hq + 2 * Hkv) * 128, D), (D, Hq * 128), (2 * I, D), (D, I))):
            w = dev(inputs.weights(N, K, cfg=42, layer=l, proj=j))
            q, s, z = laq.quantize(w, 3)
            fs.append(lambda x, out, q=q, s=s, z=z: laq.linear(x, q, s, z, 3, out=out))
            if j == 2:
                qi, si, zi = laq.quantize(torch.stack([w[:I], w[I:]], dim=1).reshape(N, K).contiguous(), 3)
                f = lambda x, out, q=qi, s=si, z=zi: laq.linear_swiglu(x, q, s, z, 3, out=out)
                f.swiglu = True
                ff.append(f)
            else:
                ff.append(fs[-1])
        plain.append(tuple(fs))
        fused.append(tuple(ff))
        norms.append(tuple(dev((1 + 0.1 * rng.standard_normal(n)).astype(np.float16)) for n in (D, D, 128, 128)))
        kcs.append(f16(rng, (Hkv, S, 128)))
        vcs.append(f16(rng, (Hkv, S, 128)))
    fin = dev((1 + 0.1 * rng.standard_normal(D)).astype(np.float16))
    x0 = dev(rng.standard_normal((1, D)).astype(np.float32))
    outs = []
    for lins in (plain, fused):
        step = decode.DecodeStep(shape, lins, norms, fin, [dev(a) for a in kcs], [dev(a) for a in vcs], DEV)
        step.x0.copy_(x0)
        outs.append(step.run(200).float().cpu().numpy())
        torch.cuda.synchronize()
    a, b = outs
    assert np.isfinite(b).all()
    rms = float(np.sqrt(np.mean(a ** 2)))
    assert float(np.abs(a - b).max()) <= 1e-2 * rms, (float(np.abs(a - b).max()), rms)

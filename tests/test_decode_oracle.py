"""Pins of the decode-step oracle (oracle/decode.py) against closed forms,
invariants and hand-worked values -- not against a retyped formula."""
import numpy as np

from oracle import decode as D


def test_rmsnorm_constant_vector_and_scale():
    # a constant vector c: mean(x^2) = c^2, so y = c / sqrt(c^2 + eps) * w
    for c, eps in ((3.0, 1e-6), (-0.5, 0.25), (2.0, 0.0)):
        w = np.linspace(-1, 2, 8)
        y = D.rmsnorm(np.full(8, c), w, eps)
        assert np.allclose(y, c / np.sqrt(c * c + eps) * w, rtol=1e-15, atol=0)
    # eps = 0: invariant under positive scaling of x, odd under negation
    x = np.random.default_rng(1).standard_normal(64)
    w = np.random.default_rng(2).standard_normal(64)
    assert np.allclose(D.rmsnorm(7.5 * x, w, 0.0), D.rmsnorm(x, w, 0.0), rtol=1e-14)
    assert np.allclose(D.rmsnorm(-x, w, 0.0), -D.rmsnorm(x, w, 0.0), rtol=1e-15)
    # unit RMS after normalisation with w = 1, eps = 0
    y = D.rmsnorm(x, np.ones(64), 0.0)
    assert abs(np.sqrt(np.mean(y * y)) - 1.0) < 1e-14


def test_add_rmsnorm_residual():
    r, y = D.add_rmsnorm(np.array([1.0, 2.0]), np.array([2.0, 2.0]), np.ones(2), 0.0)
    assert np.array_equal(r, [3.0, 4.0])
    assert np.allclose(y, np.array([3.0, 4.0]) / np.sqrt(12.5), rtol=1e-15)


def test_rope_worked_value_identity_and_composition():
    # d = 4, theta = 100: pair (x0, x2) turns by pos, pair (x1, x3) by pos / 10
    x = np.array([1.0, 0.0, 0.0, 0.0])
    assert np.allclose(D.rope(x, 1, 100.0), [np.cos(1), 0, np.sin(1), 0], rtol=0, atol=1e-15)
    x = np.array([0.0, 1.0, 0.0, 0.0])
    assert np.allclose(D.rope(x, 2, 100.0), [0, np.cos(0.2), 0, np.sin(0.2)], rtol=0, atol=1e-15)
    v = np.random.default_rng(3).standard_normal((3, 128))
    assert np.array_equal(D.rope(v, 0, 1e6), v)  # position 0: no rotation
    # rotations compose and preserve each pair's length
    a = D.rope(D.rope(v, 5, 1e6), 7, 1e6)
    assert np.allclose(a, D.rope(v, 12, 1e6), rtol=0, atol=1e-12)
    r = D.rope(v, 1234, 1e6)
    assert np.allclose(r[:, :64] ** 2 + r[:, 64:] ** 2, v[:, :64] ** 2 + v[:, 64:] ** 2, rtol=1e-12)


def test_qk_norm_rope_split():
    Hq, Hkv, d = 4, 2, 8
    rng = np.random.default_rng(4)
    qkv = rng.standard_normal((Hq + 2 * Hkv) * d)
    q, k, v = D.qk_norm_rope(qkv, np.ones(d), np.ones(d), 0, Hq, Hkv, d, 0.0, 1e4)
    # position 0 and unit weights: each q and k head has unit RMS; v untouched
    assert np.allclose(np.sqrt(np.mean(q * q, axis=1)), 1.0, rtol=1e-14)
    assert np.allclose(np.sqrt(np.mean(k * k, axis=1)), 1.0, rtol=1e-14)
    assert np.array_equal(v.reshape(-1), qkv[(Hq + Hkv) * d:])


def test_attention_special_cases():
    rng = np.random.default_rng(5)
    Hq, Hkv, L, d = 8, 2, 5, 16
    K = rng.standard_normal((Hkv, L, d))
    V = rng.standard_normal((Hkv, L, d))
    q = rng.standard_normal((Hq, d))
    # one position: the output is that position's value row
    out = D.decode_attention(q, K[:, :1], V[:, :1])
    assert np.allclose(out, np.repeat(V[:, 0], Hq // Hkv, axis=0), rtol=1e-15)
    # a zero query weighs all positions equally: the mean of the value rows
    out = D.decode_attention(np.zeros((Hq, d)), K, V)
    assert np.allclose(out, np.repeat(V.mean(axis=1), Hq // Hkv, axis=0), rtol=1e-14)
    # weights sum to one; query head h reads key/value head h // 4
    Vc = np.broadcast_to(np.arange(Hkv, dtype=np.float64)[:, None, None] + 1.0, (Hkv, L, d))
    out = D.decode_attention(q, K, Vc)
    assert np.allclose(out, (np.arange(Hq)[:, None] // (Hq // Hkv)) + 1.0, rtol=1e-14)
    # one dominant key: its value row is returned
    K2 = np.zeros((Hkv, L, d)); K2[:, 3, 0] = 1e3
    q2 = np.zeros((Hq, d)); q2[:, 0] = 1.0
    out = D.decode_attention(q2, K2, V)
    assert np.allclose(out, np.repeat(V[:, 3], Hq // Hkv, axis=0), rtol=1e-12)
    # order of positions does not matter
    perm = rng.permutation(L)
    assert np.allclose(D.decode_attention(q, K[:, perm], V[:, perm]), D.decode_attention(q, K, V), rtol=1e-13)


def test_silu_mul_values():
    gu = np.array([[0.0, np.log(3.0), 40.0, 1.5, -2.0, 2.0]])
    y = D.silu_mul(gu, 3)
    # silu(0) = 0; sigmoid(ln 3) = 3/4; silu(40) = 40 to double precision
    assert np.allclose(y, [[0.0, 0.75 * np.log(3.0) * -2.0, 40.0 * 2.0]], rtol=1e-15, atol=0)

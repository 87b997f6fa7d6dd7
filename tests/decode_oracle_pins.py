"""Pins of the decode-step oracle (oracle/decode.py): closed forms,
invariants and hand-worked values, each a function of the oracle module so
that the same pins also run against deliberately mutated copies of it
(tests/test_decode_oracle_mutants.py)."""
import numpy as np


def pin_rmsnorm_constant_vector_and_scale(D):
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


def pin_rmsnorm_worked_value(D):
    # x = (3, 4): mean(x^2) = 12.5; with eps = 3.5, sqrt(16) = 4 -> (0.75, 1) * w
    y = D.rmsnorm(np.array([3.0, 4.0]), np.array([2.0, -1.0]), 3.5)
    assert np.array_equal(y, [1.5, -1.0])
    # rows are normalised independently
    y = D.rmsnorm(np.array([[3.0, 4.0], [0.0, 5.0]]), np.ones(2), 0.0)
    assert np.allclose(y, [[3 / np.sqrt(12.5), 4 / np.sqrt(12.5)], [0.0, np.sqrt(2.0)]], rtol=1e-15, atol=0)


def pin_add_rmsnorm_residual(D):
    r, y = D.add_rmsnorm(np.array([1.0, 2.0]), np.array([2.0, 2.0]), np.ones(2), 0.0)
    assert np.array_equal(r, [3.0, 4.0])
    assert np.allclose(y, np.array([3.0, 4.0]) / np.sqrt(12.5), rtol=1e-15)
    r, y = D.add_rmsnorm(np.array([[1.0, -1.0]]), None, np.array([1.0, 3.0]), 0.0)
    assert np.array_equal(r, [[1.0, -1.0]]) and np.allclose(y, [[1.0, -3.0]], rtol=1e-15)


def pin_rope_worked_value_identity_and_composition(D):
    # d = 4, theta = 100: pair (x0, x2) turns by pos, pair (x1, x3) by pos / 10
    x = np.array([1.0, 0.0, 0.0, 0.0])
    assert np.allclose(D.rope(x, 1, 100.0), [np.cos(1), 0, np.sin(1), 0], rtol=0, atol=1e-15)
    x = np.array([0.0, 1.0, 0.0, 0.0])
    assert np.allclose(D.rope(x, 2, 100.0), [0, np.cos(0.2), 0, np.sin(0.2)], rtol=0, atol=1e-15)
    # the second member of a pair turns the other way round: (0, 1) -> (-sin, cos)
    x = np.array([0.0, 0.0, 1.0, 0.0])
    assert np.allclose(D.rope(x, 1, 100.0), [-np.sin(1), 0, np.cos(1), 0], rtol=0, atol=1e-15)
    v = np.random.default_rng(3).standard_normal((3, 128))
    assert np.array_equal(D.rope(v, 0, 1e6), v)  # position 0: no rotation
    # rotations compose and preserve each pair's length
    a = D.rope(D.rope(v, 5, 1e6), 7, 1e6)
    assert np.allclose(a, D.rope(v, 12, 1e6), rtol=0, atol=1e-12)
    r = D.rope(v, 1234, 1e6)
    assert np.allclose(r[:, :64] ** 2 + r[:, 64:] ** 2, v[:, :64] ** 2 + v[:, 64:] ** 2, rtol=1e-12)


def pin_qk_norm_rope_one_hot_heads(D):
    """Worked by hand: d = 8, theta = 100, pos = 2, so pair (i, i + 4) turns by
    2 * 100^(-i/4) = 2, 2/sqrt(10), 0.2, 0.2/sqrt(10).  Every q and k head is
    one-hot (a value c at one index): RMSNorm with eps = 0 turns it into
    sign(c) * sqrt(8) at that index, times that head's weight."""
    d, Hq, Hkv = 8, 2, 1
    a = [2.0, 2.0 / np.sqrt(10.0), 0.2, 0.2 / np.sqrt(10.0)]
    qkv = np.zeros((Hq + 2 * Hkv) * d)
    qkv[0 * d + 1] = 1.0    # q head 0: index 1 (first member of pair 1)
    qkv[1 * d + 6] = 2.0    # q head 1: index 6 (second member of pair 2)
    qkv[2 * d + 3] = -1.0   # k head 0: index 3 (first member of pair 3)
    qkv[3 * d:] = np.arange(1.0, 9.0)  # v head 0
    q_w = np.array([1.0, 2.0, 3.0, 4.0, 5.0, 6.0, 7.0, 8.0])
    k_w = np.array([-1.0, 0.5, 0.25, 3.0, 1.5, 2.5, 0.75, -2.0])
    q, k, v = D.qk_norm_rope(qkv, q_w, k_w, 2, Hq, Hkv, d, 0.0, 100.0)
    r8 = np.sqrt(8.0)
    q0 = np.zeros(d)
    q0[1], q0[5] = r8 * 2.0 * np.cos(a[1]), r8 * 2.0 * np.sin(a[1])
    q1 = np.zeros(d)
    q1[2], q1[6] = -r8 * 7.0 * np.sin(a[2]), r8 * 7.0 * np.cos(a[2])
    k0 = np.zeros(d)
    k0[3], k0[7] = -r8 * 3.0 * np.cos(a[3]), -r8 * 3.0 * np.sin(a[3])
    assert np.allclose(q, [q0, q1], rtol=0, atol=1e-14)
    assert np.allclose(k, [k0], rtol=0, atol=1e-14)
    assert np.array_equal(v, [np.arange(1.0, 9.0)])


def pin_qk_norm_rope_split(D):
    Hq, Hkv, d = 4, 2, 8
    rng = np.random.default_rng(4)
    qkv = rng.standard_normal((Hq + 2 * Hkv) * d)
    q, k, v = D.qk_norm_rope(qkv, np.ones(d), np.ones(d), 0, Hq, Hkv, d, 0.0, 1e4)
    # position 0 and unit weights: each q and k head has unit RMS and the
    # direction of its own slice of qkv; v untouched
    assert np.allclose(np.sqrt(np.mean(q * q, axis=1)), 1.0, rtol=1e-14)
    assert np.allclose(np.sqrt(np.mean(k * k, axis=1)), 1.0, rtol=1e-14)
    src = qkv.reshape(-1, d)
    for h in range(Hq):
        assert np.allclose(q[h] * np.sqrt(np.mean(src[h] ** 2)), src[h], rtol=1e-14)
    for h in range(Hkv):
        assert np.allclose(k[h] * np.sqrt(np.mean(src[Hq + h] ** 2)), src[Hq + h], rtol=1e-14)
    assert np.array_equal(v.reshape(-1), qkv[(Hq + Hkv) * d:])


def pin_attention_special_cases(D):
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


def pin_attention_worked_value(D):
    """d = 4: q . k = 2 and 0 over sqrt(4) give scores 1 and 0, weights
    e/(1+e) and 1/(1+e) on value rows e_0 and e_1."""
    q = np.array([[2.0, 0.0, 0.0, 0.0]])
    K = np.array([[[1.0, 0.0, 0.0, 0.0], [0.0, 0.0, 0.0, 0.0]]])
    V = np.array([[[1.0, 0.0, 0.0, 0.0], [0.0, 1.0, 0.0, 0.0]]])
    e = np.e
    out = D.decode_attention(q, K, V)
    assert np.allclose(out, [[e / (1 + e), 1 / (1 + e), 0.0, 0.0]], rtol=1e-15, atol=0)
    # two query heads per key/value head, heads 2, 3 on the second: scores
    # (3, 0)/2 for head 2 of a key (3, 0, 0, 0) against q (1, 0, 0, 0)
    q = np.array([[0.0] * 4, [0.0] * 4, [1.0, 0.0, 0.0, 0.0], [0.0] * 4])
    K = np.array([[[0.0] * 4, [0.0] * 4], [[3.0, 0.0, 0.0, 0.0], [0.0] * 4]])
    V = np.array([[[5.0, 0, 0, 0], [7.0, 0, 0, 0]], [[1.0, 0, 0, 0], [0.0, 0, 0, 0]]])
    out = D.decode_attention(q, K, V)
    w = np.exp(1.5) / (1 + np.exp(1.5))
    assert np.allclose(out[:, 0], [6.0, 6.0, w, 0.5], rtol=1e-15, atol=0)


def pin_silu_mul_values(D):
    gu = np.array([[0.0, np.log(3.0), 40.0, 1.5, -2.0, 2.0]])
    y = D.silu_mul(gu, 3)
    # silu(0) = 0; sigmoid(ln 3) = 3/4; silu(40) = 40 to double precision
    assert np.allclose(y, [[0.0, 0.75 * np.log(3.0) * -2.0, 40.0 * 2.0]], rtol=1e-15, atol=0)
    # silu(-ln 3) = -ln 3 / 4; the up half multiplies
    y = D.silu_mul(np.array([[-np.log(3.0), 0.5], [1.0, 3.0]]).reshape(2, 2), 1)
    assert np.allclose(y, [[-np.log(3.0) / 4 * 0.5], [3.0 / (1 + np.exp(-1.0))]], rtol=1e-15, atol=0)


ALL_DECODE_PINS = [(name, fn) for name, fn in sorted(globals().items()) if name.startswith("pin_")]

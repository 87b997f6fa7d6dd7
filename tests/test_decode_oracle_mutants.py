"""Mutation check of the decode-step oracle's pins, on the CPU.

Each case copies oracle/decode.py, plants one plausible mistake (a wrong head
offset, swapped norm weights, another rotary pairing, a wrong sign or scale,
another grouped-query head mapping) and runs every pin of
tests/decode_oracle_pins.py against the copy.  A pin set that lets a mutant
through is too weak.  Nothing here touches the real oracle."""
import importlib.util

import pytest

import decode_oracle_pins as P
from oracle import decode as D

MUTANTS = [
    ("k_from_q_region", "k = qkv[Hq * d: (Hq + Hkv) * d].reshape(Hkv, d)", "k = qkv[: Hkv * d].reshape(Hkv, d)"),
    ("v_from_k_region", "v = qkv[(Hq + Hkv) * d: (Hq + 2 * Hkv) * d].reshape(Hkv, d)",
     "v = qkv[Hq * d: (Hq + Hkv) * d].reshape(Hkv, d)"),
    ("qk_weights_swapped", "k = rope(rmsnorm(k, k_w, eps), pos, theta)", "k = rope(rmsnorm(k, q_w, eps), pos, theta)"),
    ("q_not_rotated", "q = rope(rmsnorm(q, q_w, eps), pos, theta)", "q = rmsnorm(q, q_w, eps)"),
    ("rope_interleaved_pairs", "x1, x2 = x[..., : d // 2], x[..., d // 2:]", "x1, x2 = x[..., 0::2], x[..., 1::2]"),
    ("rope_sign", "x1 * c - x2 * s", "x1 * c + x2 * s"),
    ("rope_angle_exponent", "theta ** (-2.0 * i / d)", "theta ** (-1.0 * i / d)"),
    ("rmsnorm_sum_not_mean", "np.mean(x * x, axis=-1, keepdims=True)", "np.sum(x * x, axis=-1, keepdims=True)"),
    ("rmsnorm_eps_outside_sqrt", "np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)",
     "(np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) + eps)"),
    ("residual_drops_delta", "r = r + np.asarray(delta, dtype=np.float64)", "r = r"),
    ("gqa_head_modulo", "g = h // ratio", "g = h % Hkv"),
    ("softmax_scale_d", "s = K[g] @ q[h] / np.sqrt(d)", "s = K[g] @ q[h] / d"),
    ("softmax_no_scale", "s = K[g] @ q[h] / np.sqrt(d)", "s = K[g] @ q[h]"),
    ("softmax_unnormalised", "out[h] = (p / p.sum()) @ V[g]", "out[h] = p @ V[g]"),
    ("silu_sign", "g / (1.0 + np.exp(-g)) * u", "g / (1.0 + np.exp(g)) * u"),
    ("silu_gate_up_swapped", "g, u = gu[:, :I], gu[:, I: 2 * I]", "u, g = gu[:, :I], gu[:, I: 2 * I]"),
]


def _load(path, name):
    spec = importlib.util.spec_from_file_location(name, path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_decode_mutant_is_caught(tmp_path, name, old, new):
    src = open(D.__file__).read()
    assert src.count(old) == 1, "mutation anchor not found exactly once: " + name
    path = tmp_path / ("decode_mutant_%s.py" % name)
    path.write_text(src.replace(old, new))
    m = _load(str(path), "decode_mutant_" + name)
    caught = []
    for pname, fn in P.ALL_DECODE_PINS:
        try:
            fn(m)
        except (AssertionError, ValueError, IndexError):
            caught.append(pname)
    assert caught, "no pin caught mutant " + name


def test_unmutated_copy_passes(tmp_path):
    """Control: the same loading procedure on the unmodified source passes."""
    path = tmp_path / "decode_copy.py"
    path.write_text(open(D.__file__).read())
    m = _load(str(path), "decode_copy")
    for pname, fn in P.ALL_DECODE_PINS:
        fn(m)

"""The CPU oracle against its pins (facts not derived from the oracle)."""
import json
import os

import pytest

import oracle
import oracle_pins as P

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_format.json")


@pytest.fixture(scope="module")
def o():
    return oracle.default()


@pytest.mark.parametrize("name,fn", P.ALL_FP16_PINS, ids=[n for n, _ in P.ALL_FP16_PINS])
def test_fp16_pins(o, name, fn):
    fn(o)


@pytest.mark.parametrize("name,fn", P.ALL_QUANT_PINS, ids=[n for n, _ in P.ALL_QUANT_PINS])
def test_quantize_pins(o, name, fn):
    fn(o)


@pytest.mark.parametrize("name,fn", P.ALL_PARAMS_PINS, ids=[n for n, _ in P.ALL_PARAMS_PINS])
def test_params_pins(o, name, fn):
    fn(o)


@pytest.mark.parametrize("name,fn", P.ALL_PACK_PINS, ids=[n for n, _ in P.ALL_PACK_PINS])
def test_pack_pins(o, name, fn):
    fn(o)


@pytest.mark.parametrize("name,fn", P.ALL_LINEAR_PINS, ids=[n for n, _ in P.ALL_LINEAR_PINS])
def test_linear_pins(o, name, fn):
    fn(o)


def test_paper_format_facts(o):
    with open(GOLDEN) as f:
        golden = json.load(f)
    assert golden["blockheight_at_256"] == 256 // 32 * 3
    assert golden["levels_w3"] == 8 and golden["levels_w4"] == 16
    assert golden["group_size"] % golden["inner_iteration_elements"] == 0
    P.pin_density(o, golden)

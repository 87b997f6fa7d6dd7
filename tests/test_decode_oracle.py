"""Pins of the decode-step oracle (oracle/decode.py) against closed forms,
invariants and hand-worked values -- not against a retyped formula."""
import pytest

import decode_oracle_pins as P
from oracle import decode as D


@pytest.mark.parametrize("name,fn", P.ALL_DECODE_PINS, ids=[p[0] for p in P.ALL_DECODE_PINS])
def test_decode_oracle_pin(name, fn):
    fn(D)

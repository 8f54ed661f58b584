"""The oracle against its committed fixture (tests/golden/tiny_attention.json,
written by tests/golden/make_golden.py from the oracle alone): a change to the
oracle's arithmetic shows up here as changed bits."""

import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))

import make_golden  # noqa: E402


def test_tiny_attention_matches_its_fixture_bit_for_bit():
    want = json.load(open(os.path.join(HERE, "golden", "tiny_attention.json")))
    got = make_golden.compute()
    assert got["rows"] == want["rows"] and got["dims"] == want["dims"]
    for mode in ("exact", "scaled_q"):
        assert got[mode]["out"] == want[mode]["out"], mode
        assert got[mode]["lse"] == want[mode]["lse"], mode

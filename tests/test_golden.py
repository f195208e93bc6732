"""The oracle still reproduces the Tiny fixture written by tests/golden/make_golden.py."""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))


def test_tiny_fixture_unchanged():
    import make_golden
    with open(os.path.join(HERE, "golden", "tiny_oracle.json")) as f:
        stored = json.load(f)
    assert make_golden.compute() == stored

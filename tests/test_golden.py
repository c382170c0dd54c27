"""The oracle and the seeded generators still produce the stored results
(tests/golden/seeded_outputs.txt, written by tests/golden/make_golden.py from
the oracle alone).  A change to either shows up here before it can silently
move the parity references or the benchmark's inputs."""
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))

import make_golden  # noqa: E402


def stored():
    vals = {}
    for line in open(os.path.join(HERE, "golden", "seeded_outputs.txt")):
        if line.strip() and not line.startswith("#"):
            k, v = line.split()
            vals[k] = v
    return vals


def test_oracle_and_generators_match_the_stored_results():
    assert make_golden.compute() == stored()

"""The seeded inputs are the same bytes as when the golden hashes were written
(tests/golden/input_sha256.json, by tests/golden/make_input_sha256.py): a change
in the generators, or in the random streams torch and numpy draw, fails here
instead of silently changing the benchmark's inputs.  CPU only."""
from __future__ import annotations

import json
import os

import pytest

from tests.golden import make_input_sha256 as M

GOLDEN = json.load(open(M.OUT))


@pytest.mark.parametrize("name", sorted(GOLDEN))
def test_inputs_match_golden_sha256(name):
    w = M.all_workloads()[name]
    got = M.workload_hashes(w)
    assert set(got) == set(GOLDEN[name])
    for key, h in GOLDEN[name].items():
        assert got[key] == h, f"{name}: {key} changed"

"""Regression record of the fp64 oracle (``tests/golden/oracle_small_cases.json``).

The stored outputs were written by ``tests/golden/make_golden.py``, which
calls only ``oracle/``; the paper prints no worked example, so these are not
paper values. Recomputing every case must reproduce them (to 1e-12, allowing
for another BLAS's summation order in the tiny matmuls; integer outputs
exactly), so that any change to the oracle's arithmetic is visible and has to
be justified."""

import json
import os

import numpy as np

from tests.golden.make_golden import OUT, cases


def _f(hexes):
    return np.array([float.fromhex(h) for h in hexes])


def test_oracle_reproduces_its_stored_outputs():
    stored = json.load(open(OUT))["cases"]
    now = cases()
    assert [c["name"] for c in stored] == [c["name"] for c in now]
    for old, new in zip(stored, now):
        assert old["inputs"] == new["inputs"], old["name"]
        for key in ("out", "w", "s", "cache"):
            if key in old:
                a, b = _f(old[key]), _f(new[key])
                np.testing.assert_allclose(b, a, rtol=1e-12, atol=1e-14, err_msg=f"{old['name']}:{key}")
        for key in ("idx", "perm", "offsets"):
            if key in old:
                assert old[key] == new[key], f"{old['name']}:{key}"


def test_golden_file_is_present_and_sized():
    assert os.path.getsize(OUT) < 100_000

"""The oracle against its stored regression fixture (tests/golden/c1_step.json,
written by tests/golden/make_golden.py from the oracle alone)."""
import importlib.util
import json
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))


def load_golden():
    with open(os.path.join(HERE, "golden", "c1_step.json")) as f:
        return json.load(f)


def test_oracle_reproduces_stored_c1_step():
    spec = importlib.util.spec_from_file_location("make_golden", os.path.join(HERE, "golden", "make_golden.py"))
    mg = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mg)
    want = load_golden()
    got = mg.golden()
    assert got["input_sha256"] == want["input_sha256"], "the seeded c1 inputs changed"
    assert got["P"] == want["P"] and got["R"] == want["R"] and got["sample_rows"] == want["sample_rows"]
    np.testing.assert_allclose(got["scores"], want["scores"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(np.array(got["o_sample"]), np.array(want["o_sample"]), rtol=1e-12, atol=1e-15)


def test_stored_c1_step_invariants():
    # the stored values themselves satisfy what the method fixes: the score mass of the
    # context equals (query tokens) x (query heads) (one critical layer, softmax over the
    # context), 38 = floor(0.3 x 128) rows per chunk, R = P then the 32 query rows
    g = load_golden()
    assert abs(sum(g["scores"]) - 32 * 8) < 1e-9
    P = np.array(g["P"])
    assert [int(((P >= 128 * c) & (P < 128 * (c + 1))).sum()) for c in range(4)] == [38] * 4
    assert g["R"] == g["P"] + list(range(512, 544))

"""The oracle's outputs on tiny seeded cases must not drift (CPU only).
The stored values were written by tests/golden/make_oracle_regression.py,
which calls only the oracle.  The paper's default hyperparameters are pinned
to Sec. 4.1 / Appendix B through tests/golden/paper_defaults.json."""
import json
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))


def test_oracle_regression(oracle_lib):
    import importlib.util
    spec = importlib.util.spec_from_file_location(
        "make_oracle_regression", os.path.join(HERE, "golden", "make_oracle_regression.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    with open(os.path.join(HERE, "golden", "oracle_regression.json")) as f:
        stored = json.load(f)["cases"]
    for want in stored:
        got = mod.run(tuple(want["case"]))
        assert got["proxies_sha256"] == want["proxies_sha256"]
        assert got["q_last_sha256"] == want["q_last_sha256"]
        assert got["idx"] == want["idx"]
        assert got["votes_sum"] == want["votes_sum"]
        np.testing.assert_allclose(got["mass_head"], want["mass_head"], rtol=1e-13)
        np.testing.assert_allclose(got["anchor_head"], want["anchor_head"], rtol=1e-13)


def test_paper_defaults():
    from paper_2607_22586_amd import workloads
    with open(os.path.join(HERE, "golden", "paper_defaults.json")) as f:
        ref = json.load(f)
    d = workloads.PAPER_DEFAULTS
    assert (d["P"], d["G"], d["gamma"], d["tau"], d["lam"]) == \
        (ref["P"], ref["G"], ref["gamma"], ref["tau"], ref["lambda"])
    assert ref["P"] == ref["G"] * ref["g"]

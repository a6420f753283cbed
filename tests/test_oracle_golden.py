"""The stored golden records are reproducible from the oracle (CPU): a change
of the oracle's arithmetic that alters them must come with a regenerated
fixture (tests/golden/make_screen_golden.py)."""
import importlib.util
import json
import os

HERE = os.path.dirname(os.path.abspath(__file__))


def test_golden_fixture_is_the_oracle_output(tmp_path, monkeypatch):
    spec = importlib.util.spec_from_file_location(
        "make_screen_golden", os.path.join(HERE, "golden", "make_screen_golden.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    stored = json.load(open(os.path.join(HERE, "golden", "screen_golden.json")))
    for dtype, case in stored["cases"].items():
        ref, cands = mod.build(dtype)
        assert len(cands) == len(case["records"])
        import oracle
        for c, want in zip(cands, case["records"]):
            s = oracle.screen(ref, c, dtype, case["atol"], case["rtol"])
            assert s["mismatches"] == want["mismatches"]
            assert s["nan_count"] == want["nan_count"]
            assert s["bitwise_equal"] == want["bitwise_equal"]
            assert s["sum_sq_ref"] == want["sum_sq_ref"]

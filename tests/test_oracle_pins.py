"""The CPU oracle against its pins (no GPU)."""
import numpy as np
import pytest

import oracle
import pins
from paper_2608_13144_amd import workload


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(oracle)


def test_jacobi_helper_closed_forms():
    pins.pin_jacobi_itself()


def test_certified_consistency_on_tiny_workload():
    pins.pin_lookup_certified_consistency(oracle, workload)


def test_golden_fixtures():
    """Hand-derived fixtures stored under tests/golden (each cites its passage)."""
    import json
    import os
    here = os.path.join(os.path.dirname(__file__), "golden")
    for name in sorted(os.listdir(here)):
        if not name.endswith(".json"):
            continue
        with open(os.path.join(here, name)) as f:
            fx = json.load(f)
        assert fx.get("cite"), name
        kind = fx["kind"]
        if kind == "certify":
            W = np.array(fx["W"], np.float32)
            b = None if fx.get("b") is None else np.array(fx["b"], np.float32)
            sigma = oracle.spectral_norm(W).sigma
            assert abs(sigma - fx["sigma"]) <= 1e-12 * fx["sigma"], name
            out = oracle.certify(np.array(fx["z"], np.float32), W, b, sigma)
            assert out.label.tolist() == fx["label"], name
            assert np.allclose(out.r64, fx["r"], rtol=1e-12, atol=0), name
        elif kind == "lookup":
            res = oracle.lookup(np.array(fx["zq"], np.float32), np.array(fx["z"], np.float32),
                                np.array(fx["r"], np.float32), np.array(fx["label"], np.int32))
            assert res.label.tolist() == fx["want_label"], name
            assert res.index.tolist() == fx["want_index"], name
        else:
            raise AssertionError(f"unknown fixture kind {kind}")

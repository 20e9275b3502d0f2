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


def test_stored_radius_never_exceeds_the_certificate():
    """The float32 radius is the float64 certificate rounded toward zero:
    r32 <= r64 < next float32 above r32 (both radius modes), so a query the
    float32 ball admits lies inside the certified ball (Lemma 5.1 holds for
    every radius up to r)."""
    import oracle
    from paper_2608_13144_amd import workload as wlmod
    wl = wlmod.make_workload("tiny-d64-c10", seed=0, n_cache=2000)
    sig = oracle.spectral_norm(wl.W).sigma
    for mode in ("conservative", "tight"):
        c = oracle.certify(wl.z, wl.W, wl.b, sig, radius_mode=mode)
        r32 = c.r.astype(np.float64)
        assert np.all(r32 <= c.r64)
        up = np.nextafter(c.r, np.float32(np.inf)).astype(np.float64)
        assert np.all(c.r64 < up)
        # about half the values round differently from round-to-nearest
        assert np.mean(c.r != c.r64.astype(np.float32)) > 0.2
    # exact values stay exact; 0 (a tie) stays 0; +inf (no constraint) stays +inf
    x = np.array([0.0, 0.5, 1.0 / 3.0, np.inf])
    f = oracle.to_f32_toward_zero(x)
    assert f[0] == 0.0 and f[1] == 0.5 and f[3] == np.inf
    assert f[2] < np.float32(1.0 / 3.0) or np.float64(np.float32(1.0 / 3.0)) < 1.0 / 3.0

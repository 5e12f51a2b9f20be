"""Where the decision tolerances come from.

The GPU path rounds at the same storage points as the oracle but sums its
products in another order (float32 MFMA accumulation vs float64).  These
tests measure how far a change of summation order alone moves the outputs
the decisions are taken on, using the brute-force reference evaluated once
with float64 and once with float32 matrix products, on the small bf16
model with gain jitter and the Zipf router bias.  The tolerances must lie
above that drift (with a factor of two: a gap is a difference of two
logits) -- and, for bf16 models, the drift must actually exceed the
float32-model route tolerance, else the looser bf16 tolerance is not
needed.
"""
import dataclasses

import numpy as np
import pytest

import oracle
import synth
from tests.bruteforce import Ref


@pytest.fixture(scope="module")
def drift():
    cfg = dataclasses.replace(synth.MID, n_layers=2)
    w = synth.make_weights(cfg, 0, 1, gain_jitter=0.1, zipf_s=1.1)
    tok = synth.text_tokens(cfg, 32)
    a, b = Ref(cfg, w), Ref(cfg, w, f32_products=True)
    ba, la, _ = a.verifier(tok)
    bb, lb, _ = b.verifier(tok)
    return dict(router=np.abs(a.router_logits - b.router_logits).max(axis=(1, 2)),
                logits=float(np.abs(la - lb).max()), b=float(np.abs(ba - bb).max()), cfg=cfg)


def test_route_tolerance_covers_summation_order_drift(drift):
    tol = oracle.route_tolerances(drift["cfg"])
    assert np.all(2 * drift["router"] < tol), (drift["router"], tol)


def test_bf16_route_drift_exceeds_float32_tolerance(drift):
    assert drift["router"].max() > oracle.ROUTE_TOL, drift["router"]


def test_argmax_tolerance_covers_summation_order_drift(drift):
    assert 2 * drift["logits"] < oracle.ARGMAX_TOL, drift["logits"]


def test_state_drift_within_bf16_comparison_tolerance(drift):
    # the GPU parity tests compare bf16-model states and logits at 2e-2
    assert drift["b"] < 2e-2 / 2, drift["b"]

"""Pins of the oracle's route follow: the rule that lets the oracle adopt a
top-k set chosen elsewhere (the GPU's) where that set is a near-tie of its
own.  A set is adopted exactly when it holds k distinct valid expert ids
and its lowest router logit is within the layer's tolerance of the best
logit it leaves out; otherwise the oracle keeps its own set and counts the
row as rejected.  The checks use the last row of the last layer, so an
adopted set changes nothing that later rows or layers would route on, and
compare an adopted set's effect with the brute-force reference evaluated
on the same forced selection."""
import numpy as np
import pytest

import oracle
import synth
from tests.bruteforce import Ref


@pytest.fixture(scope="module")
def case():
    cfg = synth.TINYU
    w = synth.make_weights(cfg, 0, 1, gain_jitter=0.1)
    orc = oracle.Oracle(cfg, w)
    n = 7
    tok = synth.text_tokens(cfg, n, seed=31)
    r = orc.verify_rows(orc.new_kv(16), tok, np.arange(n), want_routes=True,
                        want_router_logits=True)
    return cfg, w, orc, tok, r


def _run(orc, tok, follow, tol):
    cfg = orc.cfg
    t = np.full(cfg.n_layers, tol, np.float32)
    return orc.verify_rows(orc.new_kv(16), tok, np.arange(len(tok)), want_routes=True,
                           want_logits=True, follow_route=follow, route_tol=t)


def _variant(r, row_set):
    """The oracle's own routes with the last layer's last row replaced."""
    f = r["route_idx"].copy()
    f[-1, -1] = row_set
    return f


def _order(lg):
    return [int(e) for e in np.lexsort((np.arange(len(lg)), -lg))]


def test_own_routes_are_neither_followed_nor_rejected(case):
    cfg, w, orc, tok, r = case
    got = _run(orc, tok, r["route_idx"], 0.0)
    assert (got["route_followed"], got["route_rejected"]) == (0, 0)
    assert np.array_equal(got["b"], r["b"])


def test_neighbour_swap_adopted_exactly_when_gap_within_tolerance(case):
    """Swap the k-th chosen expert for the (k+1)-th best: that set's lowest
    logit lies exactly `gap` below the best left-out logit."""
    cfg, w, orc, tok, r = case
    k = cfg.top_k
    lg = r["router_logits"][-1, -1]
    order = _order(lg)
    gap = float(lg[order[k - 1]] - lg[order[k]])
    assert gap > 0
    swap = order[:k - 1] + [order[k]]
    f = _variant(r, swap)
    inside = _run(orc, tok, f, gap * 1.001 + 1e-7)
    assert (inside["route_followed"], inside["route_rejected"]) == (1, 0)
    assert sorted(inside["route_idx"][-1, -1].tolist()) == sorted(swap)
    outside = _run(orc, tok, f, gap * 0.999)
    assert (outside["route_followed"], outside["route_rejected"]) == (0, 1)
    assert outside["route_idx"][-1, -1].tolist() == r["route_idx"][-1, -1].tolist()
    assert np.array_equal(outside["b"], r["b"])
    # the adopted set is what the row is computed with: brute force on the
    # same forced selection
    ref = Ref(cfg, w)
    b_ref, lg_ref, _ = ref.verifier(tok, force={(cfg.n_layers - 1, len(tok) - 1): swap})
    np.testing.assert_allclose(inside["b"], b_ref, rtol=1e-4, atol=1e-4)
    assert not np.allclose(inside["b"][-1], r["b"][-1], rtol=0, atol=1e-6)
    np.testing.assert_array_equal(inside["b"][:-1], r["b"][:-1])


def test_far_set_rejected(case):
    """A set holding the lowest-logit expert is far from a near-tie."""
    cfg, w, orc, tok, r = case
    k = cfg.top_k
    lg = r["router_logits"][-1, -1]
    order = _order(lg)
    far = order[:k - 1] + [order[-1]]
    dist = float(lg[order[k - 1]] - lg[order[-1]])
    got = _run(orc, tok, _variant(r, far), 0.5 * dist)
    assert (got["route_followed"], got["route_rejected"]) == (0, 1)
    assert got["route_idx"][-1, -1].tolist() == r["route_idx"][-1, -1].tolist()
    # and adopted once the tolerance spans the distance (the rule is a
    # comparison of logits, not a rank test)
    got = _run(orc, tok, _variant(r, far), dist * 1.001 + 1e-7)
    assert (got["route_followed"], got["route_rejected"]) == (1, 0)


@pytest.mark.parametrize("bad", ["duplicate", "negative", "past_end"])
def test_invalid_sets_rejected_at_any_tolerance(case, bad):
    cfg, w, orc, tok, r = case
    own = r["route_idx"][-1, -1].tolist()
    s = list(own)
    if bad == "duplicate":
        s[-1] = s[0]
    elif bad == "negative":
        s[-1] = -1
    else:
        s[-1] = cfg.n_routed
    got = _run(orc, tok, _variant(r, s), np.inf)
    assert (got["route_followed"], got["route_rejected"]) == (0, 1)
    assert got["route_idx"][-1, -1].tolist() == own
    assert np.array_equal(got["b"], r["b"])


def test_reordered_own_set_is_the_same_selection(case):
    """The same experts in another order: adopted at zero tolerance, and the
    row's result does not change (experts are applied in id order)."""
    cfg, w, orc, tok, r = case
    own = r["route_idx"][-1, -1].tolist()
    got = _run(orc, tok, _variant(r, own[::-1]), 0.0)
    assert got["route_rejected"] == 0
    assert got["route_idx"][-1, -1].tolist() == own[::-1]
    assert np.array_equal(got["b"], r["b"])


def test_follow_requires_a_tolerance(case):
    cfg, w, orc, tok, r = case
    with pytest.raises(ValueError):
        orc.verify_rows(orc.new_kv(16), tok, np.arange(len(tok)), follow_route=r["route_idx"])

"""Replay of GPU speculative steps through the oracle.

The oracle runs its own draft chain and verify pass from its own state.
Wherever the GPU chose differently, the choice must be a near-tie of the
oracle's own scores (top-1/top-2 logit gap <= ARGMAX_TOL; router k-th vs
(k+1)-th gap <= the layer's routing tolerance, tests/tolerances.py) and the
GPU's value must lie in the oracle's near-tie set; the oracle then
continues on the GPU's choice.  Everything else -- every token, m, the
commit list and the cache bookkeeping -- must be equal, and floats must
agree to the stated tolerance.

The statistics count every decision and how many fell in the near-tie band
(graded only as "inside the near-tie set") and how many the oracle
followed; band_report() turns them into fractions that the tests print and
bound.  Where the GPU records its own k-th vs (k+1)-th router gaps, their
distance to the oracle's gaps (at most twice the router-logit deviation)
is tracked per layer and must stay within the layer's tolerance.
"""
from __future__ import annotations

import numpy as np

import oracle
import synth
from tests import tolerances


class Mismatch(AssertionError):
    pass


def near_tie_ok(logits_row: np.ndarray, tok: int, tol: float = oracle.ARGMAX_TOL) -> bool:
    return bool(logits_row[tok] >= logits_row.max() - tol)


def check_token(orc_logits_row, orc_tok, gpu_tok, what, stats):
    srt = np.sort(orc_logits_row)
    margin = float(srt[-1] - srt[-2])
    stats["tokens"] = stats.get("tokens", 0) + 1
    if margin <= oracle.ARGMAX_TOL:
        stats["token_band"] = stats.get("token_band", 0) + 1
    if orc_tok == gpu_tok:
        return gpu_tok
    if margin > oracle.ARGMAX_TOL or not near_tie_ok(orc_logits_row, gpu_tok):
        raise Mismatch(f"{what}: oracle {orc_tok} (margin {margin:.4f}) vs gpu {gpu_tok} "
                       f"(oracle logit {orc_logits_row[gpu_tok]:.4f} vs max {srt[-1]:.4f})")
    stats["followed_tokens"] = stats.get("followed_tokens", 0) + 1
    return gpu_tok


def draft_chain_follow(orc, st, K, gpu_drafts, stats, gpu_draft_logits=None, tol=None):
    """The oracle's draft chain; at each depth it checks the GPU's draft
    token and continues with it (gpu_drafts None: the oracle's own)."""
    n = st.n_rows
    hm = np.zeros(n, np.uint8)
    hm[n - 1] = 1
    r = orc.draft_rows(st.dkv, st.next_tok[:n], st.hid[:n], st.row_pos + np.arange(n),
                       head_mask=hm, want_logits=True)
    st.draft_len = st.row_pos + n
    lg = r["logits"][n - 1]
    u = r["u"][n - 1].copy()
    x = int(r["amax"][n - 1])
    if gpu_drafts is not None:
        x = check_token(lg, x, int(gpu_drafts[0]), "draft depth 1", stats)
    if gpu_draft_logits is not None:
        np.testing.assert_allclose(gpu_draft_logits[0], lg, rtol=tol, atol=tol)
    drafts = [x]
    for d in range(2, K + 1):
        p = st.row_pos + n - 1 + (d - 1)
        r = orc.draft_rows(st.dkv, [x], u[None, :], [p], head_mask=np.ones(1, np.uint8),
                           want_logits=True)
        lg = r["logits"][0]
        u = r["u"][0].copy()
        x = int(r["amax"][0])
        if gpu_drafts is not None:
            x = check_token(lg, x, int(gpu_drafts[d - 1]), f"draft depth {d}", stats)
        if gpu_draft_logits is not None:
            np.testing.assert_allclose(gpu_draft_logits[d - 1], lg, rtol=tol, atol=tol)
        drafts.append(x)
    return drafts


def count_routes(stats, gaps, rtol_l, n_followed):
    """gaps [L][n]: the oracle's k-th vs (k+1)-th router gaps of n rows."""
    stats["route_decisions"] = stats.get("route_decisions", 0) + int(gaps.size)
    stats["route_band"] = stats.get("route_band", 0) + int((gaps <= rtol_l[:, None]).sum())
    stats["followed_routes"] = stats.get("followed_routes", 0) + int(n_followed)


def track_gap_dev(stats, gpu_gap, orc_gap, rtol_l):
    """Per-layer max |gpu gap - oracle gap| (each gap is a difference of
    two order statistics of the router logits, so it moves by at most twice
    the logit deviation); must stay within the layer's tolerance."""
    d = np.abs(np.asarray(gpu_gap, np.float64) - np.asarray(orc_gap, np.float64)).max(axis=1)
    prev = stats.get("gap_dev")
    stats["gap_dev"] = d if prev is None else np.maximum(prev, d)
    bad = np.nonzero(d > rtol_l)[0]
    if len(bad):
        l = int(bad[0])
        raise Mismatch(f"router gap of layer {l} differs by {d[l]:.2e} > tolerance {rtol_l[l]:.2e}")


def band_report(stats):
    """Fractions of the decisions graded only by the near-tie band."""
    rd, td = stats.get("route_decisions", 0), stats.get("tokens", 0)
    out = dict(route_decisions=rd, tokens=td,
               route_band_frac=stats.get("route_band", 0) / rd if rd else 0.0,
               route_followed_frac=stats.get("followed_routes", 0) / rd if rd else 0.0,
               token_band_frac=stats.get("token_band", 0) / td if td else 0.0,
               token_followed_frac=stats.get("followed_tokens", 0) / td if td else 0.0)
    if stats.get("gap_dev") is not None:
        out["gap_dev_per_layer"] = [float(f"{x:.3g}") for x in stats["gap_dev"]]
    return out


# bounds on the end-to-end near-tie band.  End to end, the per-layer routing
# tolerances grow with depth (rounding accumulates over the layers), so at
# the full shape about half of the deep layers' decisions fall in the band;
# the layer-local check (local_step) grades those layers exactly instead.
MAX_ROUTE_BAND = 0.60
MAX_FOLLOWED = 0.15


def assert_band(stats):
    r = band_report(stats)
    assert r["route_band_frac"] <= MAX_ROUTE_BAND, r
    assert r["route_followed_frac"] <= MAX_FOLLOWED, r
    assert r["token_followed_frac"] <= MAX_FOLLOWED, r
    return r


def replay_step(orc, st, K, rec, stats, tol, forced=None, state_tol=None):
    """rec: the GPU's records of one step for one sequence: drafts [K],
    verify [K+1], m, commit [K+1], routes [L][K+1][k] (opt), route_gap
    [L][K+1] (opt), logits [K+1][V] (opt), hid [K+1][H] (opt), draft_logits
    [K][V] (opt).  tol: logits; state_tol: the final-norm states (default
    tol).  forced: the K tokens that replaced the drafts after drafting
    (rec["drafts"] then holds those; the drafted tokens themselves are
    checked through rec["draft_tokens_drafted"] when present)."""
    state_tol = tol if state_tol is None else state_tol
    if K > 0:
        gd = rec["drafts"] if forced is None else rec.get("draft_tokens_drafted")
        drafts = draft_chain_follow(orc, st, K, gd, stats, rec.get("draft_logits"), tol)
    else:
        drafts = []
    if forced is not None:
        drafts = [int(t) for t in forced]
    if K > 0 and [int(t) for t in rec["drafts"]] != drafts:
        raise Mismatch(f"verify inputs differ: gpu drafts {list(rec['drafts'])} vs {drafts}")
    toks = [st.pending] + drafts
    follow = rec.get("routes")
    rtol_l = tolerances.route_tol(orc.cfg)
    r = orc.verify_rows(st.kv, toks, st.kv_len + np.arange(K + 1), want_logits=True,
                        want_routes=True, follow_route=follow, route_tol=rtol_l)
    if r["route_rejected"]:
        # locate the first (layer, row) where the sets differ, without follow
        kv_copy = st.kv.copy()
        r0 = orc.verify_rows(kv_copy, toks, st.kv_len + np.arange(K + 1), want_routes=True)
        detail = []
        for l in range(follow.shape[0]):
            for i in range(follow.shape[1]):
                a_, b_ = sorted(r0["route_idx"][l, i].tolist()), sorted(follow[l, i].tolist())
                if a_ != b_:
                    detail.append(f"layer {l} row {i}: oracle {a_} gap {r0['route_gap'][l, i]:.2e} "
                                  f"gpu {b_}")
            if detail:
                break
        raise Mismatch(f"{r['route_rejected']} GPU routings are not top-k of the oracle's logits; "
                       f"first difference: {detail[:3]}")
    count_routes(stats, r["route_gap"], rtol_l, r["route_followed"])
    if follow is not None:
        ok = r["route_gap"] > rtol_l[:, None]
        if not np.array_equal(np.sort(r["route_idx"][ok], -1), np.sort(follow[ok], -1)):
            raise Mismatch("routing differs where the oracle's gap exceeds the tolerance")
    if rec.get("route_gap") is not None:
        track_gap_dev(stats, rec["route_gap"], r["route_gap"], rtol_l)
    v = [check_token(r["logits"][i], int(r["amax"][i]), int(rec["verify"][i]), f"verify row {i}",
                     stats) for i in range(K + 1)]
    if rec.get("logits") is not None:
        np.testing.assert_allclose(rec["logits"], r["logits"], rtol=tol, atol=tol)
    if rec.get("hid") is not None:
        np.testing.assert_allclose(rec["hid"], r["b"], rtol=tol, atol=state_tol)
    m, commit = oracle.accept(drafts, v)
    if m != int(rec["m"]) or commit != [int(t) for t in rec["commit"][:m + 1]]:
        raise Mismatch(f"accept: oracle m={m} commit={commit} vs gpu m={rec['m']} "
                       f"commit={list(rec['commit'])}")
    oracle.commit(st, m, commit, r["b"])
    stats["steps"] += 1
    return m


def new_stats():
    return dict(steps=0, followed_tokens=0, followed_routes=0, route_decisions=0, route_band=0,
                tokens=0, token_band=0, gap_dev=None)


def teacher_forced_check(orc, tok_prefix, vis_prefix, gen, stats, routes=None):
    """One causal oracle pass over the prefix and the generated tokens (the
    tokens the GPU produced are fed back in); the greedy token of the row
    before each generated token must be that token, or a near-tie of it
    (reading of several correct results).  routes [L][P+n-1][k]: the GPU's
    routing of every position of that pass, followed by the oracle where it
    is a near-tie of its own (elsewhere the two must agree).  Returns the
    number of tokens checked."""
    c = orc.cfg
    P, n = len(tok_prefix), len(gen)
    toks = np.concatenate([np.asarray(tok_prefix, np.int32), np.asarray(gen[:-1], np.int32)])
    emb = np.zeros((P + n - 1, c.hidden), c.wdtype)
    emb[:P] = vis_prefix
    hm = np.zeros(P + n - 1, np.uint8)
    hm[P - 1:] = 1
    kv = orc.new_kv(P + n)
    fr = None if routes is None else np.ascontiguousarray(routes[:, :P + n - 1])
    rtol_l = tolerances.route_tol(c)
    r = orc.verify_rows(kv, toks, np.arange(P + n - 1), emb=emb, head_mask=hm, want_logits=True,
                        want_routes=True, follow_route=fr,
                        route_tol=rtol_l if fr is not None else None)
    if r["route_rejected"]:
        raise Mismatch(f"{r['route_rejected']} routing decisions differ beyond the tolerance")
    count_routes(stats, r["route_gap"], rtol_l, r["route_followed"])
    for i in range(n):
        check_token(r["logits"][P - 1 + i], int(r["amax"][P - 1 + i]), int(gen[i]),
                    f"generated token {i}", stats)
    return n


# ---------------------------------------------------------------- layer-local
def _input_rows(orc, tok):
    c = orc.cfg
    E = orc.w["embed"]
    rows = np.stack([E[int(t)] for t in tok])
    return (synth.bf16_bits_to_f32(rows) if rows.dtype == np.uint16 else rows).astype(np.float32)


def _close(got, want, atol, rtol, what):
    try:
        np.testing.assert_allclose(got, want, rtol=rtol, atol=atol)
    except AssertionError as e:
        raise Mismatch(f"{what}: {str(e)[:600]}") from None


def local_step(orc, pre, rec, kv_post, dkv_post, K, stats):
    """Layer-local check of one step of one sequence: every part of the step
    recomputed by the oracle from the GPU's own inputs, so a difference can
    only come from that part's own rounding.

    pre: the sequence's state before the step -- kv_len, pending, n_rows,
    row_pos, hid [n_rows][H] (the GPU's final-norm states of the rows to
    catch up), next_tok [n_rows].  rec: the step's records (step_records,
    with layer_h).  kv_post [L][2][nh][cap][dh], dkv_post [2][nh][cap][dh]:
    the GPU's caches after the step, float32 (positions below kv_len,
    resp. row_pos, are those before the step).

    Draft: depth 1 over the catch-up rows from the GPU's states and draft
    cache, depth d >= 2 from the GPU's depth d-1 output state and token
    (rec["draft_u"]) and the GPU's draft cache (the rows its earlier depths
    wrote): draft logits, output states and the draft K/V of every row.
    Verify, layer by layer from the GPU's layer input: routing (exact but at
    near-ties within the layer tolerance), router gaps, layer output, the
    rows' K/V; the head from the GPU's last-layer output: final-norm states,
    logits, greedy tokens; acceptance from the GPU's tokens."""
    c = orc.cfg
    tl = tolerances.local_tol(c)
    L = c.n_layers
    drafted = rec.get("draft_tokens_drafted") or rec["drafts"]
    if K > 0:
        n, rp = int(pre["n_rows"]), int(pre["row_pos"])
        dk = np.ascontiguousarray(dkv_post.copy())
        hm = np.zeros(n, np.uint8)
        hm[n - 1] = 1
        r = orc.draft_rows(dk, pre["next_tok"][:n], pre["hid"][:n], rp + np.arange(n),
                           head_mask=hm, want_logits=True)
        lg = r["logits"][n - 1]
        if rec.get("draft_logits") is not None:
            t = tl["draft_logits"][0]
            _close(rec["draft_logits"][0], lg, t, t, "local draft logits depth 1")
        x = check_token(lg, int(r["amax"][n - 1]), int(drafted[0]), "local draft depth 1", stats)
        _close(dkv_post[:, :, rp:rp + n], dk[:, :, rp:rp + n], tl["kv_atol"], tl["kv_rtol"],
               "catch-up draft K/V")
        u = r["u"][n - 1:n]
        for d in range(2, K + 1):
            if rec.get("draft_u") is not None:
                gu = rec["draft_u"][d - 2][None, :]
                t = tl["draft_u"][d - 2]
                _close(gu, u, t, t, f"local draft state depth {d - 1}")
                u = gu
            p = rp + n - 1 + d - 1
            dk = np.ascontiguousarray(dkv_post.copy())   # the GPU's rows of earlier depths
            r = orc.draft_rows(dk, [x], u, [p], head_mask=np.ones(1, np.uint8), want_logits=True)
            _close(dkv_post[:, :, p:p + 1], dk[:, :, p:p + 1], tl["kv_atol"], tl["kv_rtol"],
                   f"draft K/V depth {d}")
            lg = r["logits"][0]
            if rec.get("draft_logits") is not None:
                t = tl["draft_logits"][d - 1]
                _close(rec["draft_logits"][d - 1], lg, t, t, f"local draft logits depth {d}")
            x = check_token(lg, int(r["amax"][0]), int(drafted[d - 1]), f"local draft depth {d}",
                            stats)
            u = r["u"]
    toks = [int(pre["pending"])] + [int(t) for t in rec["drafts"][:K]]
    pos = int(pre["kv_len"]) + np.arange(K + 1)
    lh = rec["layer_h"]
    _close(lh[0], _input_rows(orc, toks), 0.0, 0.0, "verify input rows")
    kvw = np.ascontiguousarray(kv_post.copy())
    for l in range(L):
        r = orc.verify_layer(l, kvw[l], lh[l], pos, follow_route=rec["routes"][l],
                             route_tol=float(tl["route"][l]))
        if r["route_rejected"]:
            raise Mismatch(f"layer {l}: GPU routing is not a top-k set of the oracle's logits "
                           f"within {tl['route'][l]:.2e} (layer-local)")
        count_routes(stats, r["route_gap"][None, :], tl["route"][l:l + 1], r["route_followed"])
        track_gap_dev_layer(stats, l, L, rec["route_gap"][l], r["route_gap"], tl["route"][l])
        _close(lh[l + 1], r["h"], tl["h"][l], tl["h"][l], f"layer {l} output")
        _close(kv_post[l][:, :, pos], kvw[l][:, :, pos], tl["kv_atol"], tl["kv_rtol"],
               f"layer {l} K/V")
    hd = orc.head(lh[L])
    _close(rec["hid"], hd["b"], tl["state"], tl["state"], "final-norm states")
    if rec.get("logits") is not None:
        _close(rec["logits"], hd["logits"], tl["logits"], tl["logits"], "logits")
        dev = float(np.abs(rec["logits"] - hd["logits"]).max())
        stats["logit_dev"] = max(stats.get("logit_dev", 0.0), dev)
    v = [check_token(hd["logits"][i], int(hd["amax"][i]), int(rec["verify"][i]),
                     f"local verify row {i}", stats) for i in range(K + 1)]
    m, commit = oracle.accept(toks[1:], v)
    if m != int(rec["m"]) or commit != [int(t) for t in rec["commit"][:m + 1]]:
        raise Mismatch(f"local accept: m={m} commit={commit} vs gpu m={rec['m']}")
    stats["steps"] = stats.get("steps", 0) + 1
    return m


def track_gap_dev_layer(stats, l, L, gpu_gap, orc_gap, tol):
    d = float(np.abs(np.asarray(gpu_gap, np.float64) - np.asarray(orc_gap, np.float64)).max())
    if stats.get("gap_dev") is None:
        stats["gap_dev"] = np.zeros(L)
    stats["gap_dev"][l] = max(stats["gap_dev"][l], d)
    if d > tol:
        raise Mismatch(f"layer {l}: router gap differs by {d:.2e} > {tol:.2e} (layer-local)")


# the layer-local check grades nearly every routing decision exactly
MAX_LOCAL_ROUTE_BAND = 0.10


def assert_local_band(stats):
    r = band_report(stats)
    assert r["route_band_frac"] <= MAX_LOCAL_ROUTE_BAND, r
    assert r["route_followed_frac"] <= MAX_LOCAL_ROUTE_BAND, r
    if stats.get("logit_dev") is not None:
        r["logit_dev"] = float(f"{stats['logit_dev']:.3g}")
    return r

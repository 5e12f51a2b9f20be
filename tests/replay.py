"""Replay of GPU speculative steps through the oracle.

The oracle runs its own draft chain and verify pass from its own state.
Wherever the GPU chose differently, the choice must be a near-tie of the
oracle's own scores (top-1/top-2 logit gap <= ARGMAX_TOL; router k-th vs
(k+1)-th gap <= the layer's routing tolerance, oracle.route_tolerances) and the GPU's value must lie in the oracle's
near-tie set; the oracle then continues on the GPU's choice.  Everything
else -- every token, m, the commit list and the cache bookkeeping -- must
be equal, and floats must agree to the stated tolerance.
"""
from __future__ import annotations

import numpy as np

import oracle


class Mismatch(AssertionError):
    pass


def near_tie_ok(logits_row: np.ndarray, tok: int, tol: float = oracle.ARGMAX_TOL) -> bool:
    return bool(logits_row[tok] >= logits_row.max() - tol)


def check_token(orc_logits_row, orc_tok, gpu_tok, what, stats):
    if orc_tok == gpu_tok:
        return gpu_tok
    srt = np.sort(orc_logits_row)
    margin = float(srt[-1] - srt[-2])
    if margin > oracle.ARGMAX_TOL or not near_tie_ok(orc_logits_row, gpu_tok):
        raise Mismatch(f"{what}: oracle {orc_tok} (margin {margin:.4f}) vs gpu {gpu_tok} "
                       f"(oracle logit {orc_logits_row[gpu_tok]:.4f} vs max {srt[-1]:.4f})")
    stats["followed_tokens"] += 1
    return gpu_tok


def draft_chain_follow(orc, st, K, gpu_drafts, stats, gpu_draft_logits=None, tol=None):
    """The oracle's draft chain; at each depth it checks the GPU's draft
    token and continues with it."""
    n = st.n_rows
    hm = np.zeros(n, np.uint8)
    hm[n - 1] = 1
    r = orc.draft_rows(st.dkv, st.next_tok[:n], st.hid[:n], st.row_pos + np.arange(n),
                       head_mask=hm, want_logits=True)
    st.draft_len = st.row_pos + n
    lg = r["logits"][n - 1]
    u = r["u"][n - 1].copy()
    x = check_token(lg, int(r["amax"][n - 1]), int(gpu_drafts[0]), "draft depth 1", stats)
    if gpu_draft_logits is not None:
        np.testing.assert_allclose(gpu_draft_logits[0], lg, rtol=tol, atol=tol)
    drafts = [x]
    for d in range(2, K + 1):
        p = st.row_pos + n - 1 + (d - 1)
        r = orc.draft_rows(st.dkv, [x], u[None, :], [p], head_mask=np.ones(1, np.uint8),
                           want_logits=True)
        lg = r["logits"][0]
        u = r["u"][0].copy()
        x = check_token(lg, int(r["amax"][0]), int(gpu_drafts[d - 1]), f"draft depth {d}", stats)
        if gpu_draft_logits is not None:
            np.testing.assert_allclose(gpu_draft_logits[d - 1], lg, rtol=tol, atol=tol)
        drafts.append(x)
    return drafts


def replay_step(orc, st, K, rec, stats, tol, forced=None, state_tol=None):
    """rec: the GPU's records of one step for one sequence: drafts [K],
    verify [K+1], m, commit [K+1], routes [L][K+1][k] (opt), logits
    [K+1][V] (opt), hid [K+1][H] (opt), draft_logits [K][V] (opt).
    tol: logits; state_tol: the final-norm states (default tol)."""
    state_tol = tol if state_tol is None else state_tol
    if K > 0:
        drafts = draft_chain_follow(orc, st, K, rec["drafts"], stats, rec.get("draft_logits"), tol)
    else:
        drafts = []
    if forced is not None:
        drafts = [int(t) for t in forced]
    if K > 0 and [int(t) for t in rec["drafts"]] != drafts:
        raise Mismatch(f"verify inputs differ: gpu drafts {list(rec['drafts'])} vs {drafts}")
    toks = [st.pending] + drafts
    follow = rec.get("routes")
    rtol_l = oracle.route_tolerances(orc.cfg)
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
    stats["followed_routes"] += r["route_followed"]
    if follow is not None:
        ok = r["route_gap"] > rtol_l[:, None]
        if not np.array_equal(np.sort(r["route_idx"][ok], -1), np.sort(follow[ok], -1)):
            raise Mismatch("routing differs where the oracle's gap exceeds the tolerance")
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
    return dict(steps=0, followed_tokens=0, followed_routes=0)


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
    r = orc.verify_rows(kv, toks, np.arange(P + n - 1), emb=emb, head_mask=hm, want_logits=True,
                        want_routes=fr is not None, follow_route=fr)
    if r["route_rejected"]:
        raise Mismatch(f"{r['route_rejected']} routing decisions differ beyond the tolerance")
    stats["followed_routes"] += r["route_followed"]
    for i in range(n):
        check_token(r["logits"][P - 1 + i], int(r["amax"][P - 1 + i]), int(gen[i]),
                    f"generated token {i}", stats)
    return n

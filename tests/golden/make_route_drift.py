"""Writes route_drift.json: how far a second, equally valid float32
evaluation of a bf16 model moves the quantities the parity tests take
decisions on.

For each model and workload below, the oracle runs twice on the same
inputs: once as the reference (float64 sums, rounded at the storage
points) and once in its float32-summation mode (every internal sum formed
in float32, sequentially).  The second run takes the reference run's
routing at every (row, layer), so the two differ by summation order alone
and not by a cascade of different expert choices -- the situation of the
GPU path, whose routing the oracle adopts at near-ties.  Each keeps its
own KV cache.  Recorded per model key, over every row of every workload:

  router[l]  max |delta router logit| in layer l,
  logits     max |delta token logit| over the LM-head rows,
  state      max |delta final-norm state b|.

A second, layer-local measurement ("local") gives every layer, the head
and the draft chain the reference run's own inputs: layer l from the
reference's input of layer l and its KV slab, the head (final norm, LM
head) from the reference's last-layer output, the draft chain (depths
1..3, each depth from the previous depth's output of the same run) from
the reference's final-norm states and draft cache.  It records per layer
the router-logit and layer-output drift, the drift of the K/V the layer
writes for its rows, the head's logit and state drift, and the draft
block's output-state and logit drift over every row of the sequence (one
application of the block per row, from the same states and input rows) --
the rounding of one layer, not an accumulation.  Every draft depth is one
application of that block, so the parity check uses this drift at every
depth.  The parity tests check the GPU path layer by
layer the same way (tests/replay.py, layer-local check).

The decision tolerances of the bf16 parity tests (tests/tolerances.py)
are derived from these numbers.  Only oracle/ and synth/ are used; run
from the repository root:  python tests/golden/make_route_drift.py [keys]
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "route_drift.json")


def _drift(orc, kv_cap, rows, preload=None):
    """Reference run, then the float32-summation run on the reference's
    routes; preload(kv) fills a synthetic cached context first."""
    def go(follow):
        kv = orc.new_kv(kv_cap)
        if preload is not None:
            preload(kv)
        res = []
        for i, (tok, emb, pos, head) in enumerate(rows):
            f = None if follow is None else follow[i]
            inf = np.full(orc.cfg.n_layers, np.inf, np.float32)
            r = orc.verify_rows(kv, tok, pos, emb=emb, head_mask=head, want_logits=True,
                                want_routes=True, want_router_logits=True, follow_route=f,
                                route_tol=inf if f is not None else None)
            if f is not None:
                assert r["route_rejected"] == 0
            res.append(r)
        return res
    oracle.set_sum32(False)
    ref = go(None)
    oracle.set_sum32(True)
    try:
        alt = go([r["route_idx"] for r in ref])
    finally:
        oracle.set_sum32(False)
    L = orc.cfg.n_layers
    router = np.zeros(L)
    lg = st = 0.0
    for a, b, (tok, emb, pos, head) in zip(ref, alt, rows):
        router = np.maximum(router, np.abs(a["router_logits"] - b["router_logits"]).max(axis=(1, 2)))
        hm = np.asarray(head, bool)
        if hm.any():
            lg = max(lg, float(np.abs(a["logits"][hm] - b["logits"][hm]).max()))
        st = max(st, float(np.abs(a["b"] - b["b"]).max()))
    return router, lg, st, sum(len(r[0]) for r in rows)


def _input_rows(orc, tok, emb):
    """The verifier's input rows: token embeddings, or the given rows."""
    c = orc.cfg
    E = orc.w["embed"]
    out = np.zeros((len(tok), c.hidden), np.float32)
    for r, t in enumerate(tok):
        row = E[int(t)] if t >= 0 else emb[r]
        out[r] = synth.bf16_bits_to_f32(row) if row.dtype == np.uint16 else row
    return out


def _local_drift(orc, kv_cap, rows, preload=None, dpreload=None, K=3):
    """Layer-local drift: every layer, the head and the draft block of the
    float32-summation mode started from the reference run's own inputs.
    The draft block runs in base form (state b_p, next input row) over
    every row the calls ran except the last, after dpreload (a synthetic
    cached draft context) when given."""
    c = orc.cfg
    L = c.n_layers
    kv = orc.new_kv(kv_cap)
    dkv = orc.new_dkv(kv_cap + K)
    if preload is not None:
        preload(kv)
    if dpreload is not None:
        dpreload(dkv)
    router, hdev = np.zeros(L), np.zeros(L)
    lg = st = kvd = 0.0
    dl = du = 0.0
    all_b, all_pos, all_tok, all_emb = [], [], [], []
    try:
        for tok, emb, pos, head in rows:
            h = _input_rows(orc, tok, emb)
            for l in range(L):
                snap = kv[l].copy()
                ref = orc.verify_layer(l, kv[l], h, pos)
                oracle.set_sum32(True)
                alt = orc.verify_layer(l, snap, h, pos, follow_route=ref["route_idx"],
                                       route_tol=np.inf)
                oracle.set_sum32(False)
                assert alt["route_rejected"] == 0
                router[l] = max(router[l], float(np.abs(ref["router_logits"] -
                                                        alt["router_logits"]).max()))
                hdev[l] = max(hdev[l], float(np.abs(ref["h"] - alt["h"]).max()))
                kvd = max(kvd, float(np.abs(kv[l][:, :, pos] - snap[:, :, pos]).max()))
                h = ref["h"]
            hm = np.asarray(head, bool)
            oracle.set_sum32(True)
            alt = orc.head(h[hm])
            oracle.set_sum32(False)
            ref = orc.head(h)
            lg = max(lg, float(np.abs(ref["logits"][hm] - alt["logits"]).max()))
            st = max(st, float(np.abs(ref["b"][hm] - alt["b"]).max()))
            all_b.append(ref["b"])
            all_pos.append(np.asarray(pos))
            all_tok.append(np.asarray(tok, np.int32))
            e = np.zeros((len(tok), c.hidden), c.wdtype) if emb is None else np.asarray(emb)
            all_emb.append(e)
        amax_last = int(ref["amax"][-1])
        b_all = np.concatenate(all_b)
        pos_all = np.concatenate(all_pos)
        tok_all = np.concatenate(all_tok)
        emb_all = np.concatenate(all_emb)
        T = len(pos_all)
        # next input row of every row: the following row's input, and the
        # greedy token after the last one
        nxt_tok = np.concatenate([tok_all[1:], [amax_last]]).astype(np.int32)
        nxt_emb = np.concatenate([emb_all[1:], np.zeros((1, c.hidden), c.wdtype)])
        # the draft block over every row of the sequence at once, from the
        # same inputs in both modes (states b, next input rows, the cache
        # before them): one application of the block per row, so its
        # rounding -- including the rare product input that lands on the
        # other side of a bf16 rounding boundary -- is sampled over many
        # rows; logits on every 4th row and the last
        if T > 1:
            hm = np.zeros(T - 1, np.uint8)
            hm[::4] = 1
            hm[-1] = 1
            outs = []
            for mode in (False, True):
                oracle.set_sum32(mode)
                dk = dkv.copy()
                outs.append(orc.draft_rows(dk, nxt_tok[:T - 1], b_all[:T - 1], pos_all[:T - 1],
                                           emb=nxt_emb[:T - 1], head_mask=hm, want_logits=True))
                oracle.set_sum32(False)
            h1 = hm.astype(bool)
            dl = max(dl, float(np.abs(outs[0]["logits"][h1] - outs[1]["logits"][h1]).max()))
            du = max(du, float(np.abs(outs[0]["u"] - outs[1]["u"]).max()))
    finally:
        oracle.set_sum32(False)
    return router, hdev, lg, st, dl, du, kvd


def _prefix_rows(cfg, n_vis, n_txt, n_ar, seed):
    """Prefix in one call (vision rows seed, tokens seed+100), then n_ar
    single rows of uniform tokens (teacher-forced; seed+200)."""
    P = n_vis + n_txt
    tok = np.full(P, -1, np.int32)
    emb = np.zeros((P, cfg.hidden), cfg.wdtype)
    if n_vis:
        emb[:n_vis] = synth.vision_prefix(cfg, n_vis, seed=seed)
    tok[n_vis:] = synth.text_tokens(cfg, n_txt, seed=seed + 100)
    head = np.zeros(P, np.uint8)
    head[P - 1] = 1
    rows = [(tok, emb, np.arange(P), head)]
    ar = synth.text_tokens(cfg, n_ar, seed=seed + 200)
    for i in range(n_ar):
        rows.append((ar[i:i + 1], None, [P + i], np.ones(1, np.uint8)))
    return rows, P + n_ar + 1


def _synthetic_rows(cfg, ctx, n_steps, K, b, seed):
    """A synthetic cached context of ctx positions (the batch-16/64 recipe,
    sequence b: verifier K/V, and draft K/V of positions 0..ctx-2), then
    n_steps verify passes of K+1 rows."""
    def preload(kv):
        for l in range(cfg.n_layers):
            for c in range(2):
                kv[l, c, :, :ctx] = synth.bf16_bits_to_f32(
                    synth.kv_values(cfg, l, b, c, ctx, 15, 70))

    def dpreload(dkv):
        for c in range(2):
            dkv[c, :, :ctx - 1] = synth.bf16_bits_to_f32(
                synth.kv_values(cfg, 0, b, c, ctx - 1, 15, 71))
    toks = synth.text_tokens(cfg, n_steps * (K + 1), seed=seed)
    rows = [(toks[i * (K + 1):(i + 1) * (K + 1)], None, ctx + i * (K + 1) + np.arange(K + 1),
             np.ones(K + 1, np.uint8)) for i in range(n_steps)]
    return rows, ctx + n_steps * (K + 1) + 1, preload, dpreload


# model key -> (config, weight options, workloads)
MODELS = {
    "tinyb": (synth.TINYB, dict(), [("prefix", dict(n_vis=6, n_txt=6, n_ar=12, seeds=(10, 11)))]),
    "mid": (synth.MID, dict(gain_jitter=0.1, zipf_s=1.1),
            [("prefix", dict(n_vis=16, n_txt=12, n_ar=16, seeds=(10, 11, 12))),
             ("prefix", dict(n_vis=8, n_txt=8, n_ar=12, seeds=(13, 14)))]),
    "full": (synth.FULL, dict(),
             [("prefix", dict(n_vis=256, n_txt=512, n_ar=8, seeds=(10,))),
              ("synthetic", dict(ctx=2048, n_steps=2, seqs=(0, 1)))]),
    "full_zipf": (synth.FULL, dict(zipf_s=1.1),
                  [("synthetic", dict(ctx=4096, n_steps=2, seqs=(0, 1)))]),
}


def _r(x):
    return float(f"{x:.4g}")


def measure_workload(orc, kind, p):
    """Drift of one workload: dict(recipe, rows, router [L], logits, state,
    local=dict(router [L], h [L], logits, state, draft_logits))."""
    cfg = orc.cfg
    L = cfg.n_layers
    router = np.zeros(L)
    lg = st = 0.0
    loc = dict(router=np.zeros(L), h=np.zeros(L), logits=0.0, state=0.0,
               draft_logits=0.0, draft_u=0.0, kv=0.0)
    n_rows = 0
    cases = []
    if kind == "prefix":
        for sd in p["seeds"]:
            rows, cap = _prefix_rows(cfg, p["n_vis"], p["n_txt"], p["n_ar"], sd)
            cases.append((rows, cap, None, None))
        recipe = (f"{len(p['seeds'])} x prefix {p['n_vis']} vision + {p['n_txt']} tokens "
                  f"then {p['n_ar']} single rows")
    else:
        K = 3
        for b in p["seqs"]:
            cases.append(_synthetic_rows(cfg, p["ctx"], p["n_steps"], K, b, 30 + b))
        recipe = (f"{len(p['seqs'])} x synthetic context {p['ctx']} then "
                  f"{p['n_steps']} verify passes of {K + 1} rows")
    for rows, cap, pre, dpre in cases:
        r, a, b, n = _drift(orc, cap, rows, preload=pre)
        router, lg, st, n_rows = np.maximum(router, r), max(lg, a), max(st, b), n_rows + n
        lr, lh, llg, lst, ldl, ldu, lkv = _local_drift(orc, cap, rows, preload=pre,
                                                       dpreload=dpre)
        loc["router"] = np.maximum(loc["router"], lr)
        loc["h"] = np.maximum(loc["h"], lh)
        loc["logits"] = max(loc["logits"], llg)
        loc["state"] = max(loc["state"], lst)
        loc["draft_logits"] = max(loc["draft_logits"], ldl)
        loc["draft_u"] = max(loc["draft_u"], ldu)
        loc["kv"] = max(loc["kv"], lkv)
    return {"recipe": recipe, "rows": n_rows, "router": [_r(x) for x in router],
            "logits": _r(lg), "state": _r(st),
            "local": {"router": [_r(x) for x in loc["router"]], "h": [_r(x) for x in loc["h"]],
                      "logits": _r(loc["logits"]), "state": _r(loc["state"]),
                      "draft_logits": _r(loc["draft_logits"]),
                      "draft_u": _r(loc["draft_u"]), "kv": _r(loc["kv"])}}


def measure(key, only=None):
    """All workloads of a model key (or only workload index `only`); the
    entry holds each workload's drift and the maximum over them."""
    cfg, wkw, work = MODELS[key]
    w = synth.make_weights(cfg, 0, 1, **wkw)
    orc = oracle.Oracle(cfg, w)
    parts = [measure_workload(orc, kind, p) for i, (kind, p) in enumerate(work)
             if only is None or i == only]
    loc = [x["local"] for x in parts]
    return {"config": cfg.name, "weights": wkw, "rows": sum(x["rows"] for x in parts),
            "workloads": parts,
            "router": [_r(x) for x in np.max([x["router"] for x in parts], axis=0)],
            "logits": max(x["logits"] for x in parts), "state": max(x["state"] for x in parts),
            "local": {"router": [_r(x) for x in np.max([x["router"] for x in loc], axis=0)],
                      "h": [_r(x) for x in np.max([x["h"] for x in loc], axis=0)],
                      "logits": max(x["logits"] for x in loc),
                      "state": max(x["state"] for x in loc),
                      "draft_logits": max(x["draft_logits"] for x in loc),
                      "draft_u": max(x["draft_u"] for x in loc),
                      "kv": max(x["kv"] for x in loc)}}


def main(keys):
    try:
        d = json.load(open(OUT))
    except OSError:
        d = {}
    for k in keys:
        t0 = time.time()
        d[k] = measure(k)
        print(k, json.dumps(d[k]), f"{time.time() - t0:.0f} s", flush=True)
        with open(OUT, "w") as fh:
            json.dump(d, fh, indent=1)


if __name__ == "__main__":
    main(sys.argv[1:] or list(MODELS))

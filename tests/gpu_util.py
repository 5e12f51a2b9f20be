"""Helpers shared by the GPU tests: model setup on both sides and step
records copied back from the device."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import synth
from paper_2609_03181_amd.session import Model, Session
from tests import tolerances


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def build_pair(name, max_batch, max_ctx, max_k, **wkw):
    cfg = synth.CONFIGS[name]
    w = synth.make_weights(cfg, 0, 1, **wkw)
    return cfg, w, Model(cfg, w, max_batch, max_ctx, max_k), oracle.Oracle(cfg, w)


def prefix_inputs(cfg, B, n_vis, n_txt, seed0=10):
    """Per-sequence prefixes: vision rows (seed seed0+b) then tokens (seed
    seed0+100+b).  Returns host arrays tok [B][P] (-1 = vision row) and
    vision [B][P][H] (storage dtype)."""
    P = n_vis + n_txt
    tok = np.full((B, P), -1, np.int32)
    vis = np.zeros((B, P, cfg.hidden), cfg.wdtype)
    for b in range(B):
        if n_vis:
            vis[b, :n_vis] = synth.vision_prefix(cfg, n_vis, seed=seed0 + b)
        tok[b, n_vis:] = synth.text_tokens(cfg, n_txt, seed=seed0 + 100 + b)
    return tok, vis


def to_dev_storage(arr, device="cuda"):
    a = np.ascontiguousarray(arr)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device)
    return torch.from_numpy(a).to(device)


def gpu_prefill(model, B, K, tok, vis, max_out, record=True, prefill_rows=0):
    s = Session(model, B, K, max_out, prefill_rows=prefill_rows, record=record)
    s.prefill(torch.from_numpy(tok), to_dev_storage(vis) if (tok < 0).any() else None)
    return s


def oracle_prefill(orc, cfg, tok_b, vis_b, cap, max_new, routes=None):
    """The oracle's prefill of one sequence; routes [L][P][k] (the GPU's
    prefill routing, Session.prefill_routes[:, b]) are followed at the
    oracle's near-ties (per-layer tolerances of tests/tolerances.py), and
    any other difference fails."""
    nv = int((tok_b < 0).sum())
    st = oracle.prefill(orc, cap, vis_b[:nv] if nv else None, tok_b[nv:], max_new=max_new,
                        follow_route=routes,
                        route_tol=tolerances.route_tol(cfg) if routes is not None else None)
    assert st.prefill_routes_rejected == 0, (
        f"{st.prefill_routes_rejected} prefill routings are not near-ties of the oracle's")
    return st


def step_records(s: Session):
    """Per-sequence records of the step just run (host copies)."""
    torch.cuda.synchronize()
    B, K = s.B, s.K
    recs = []
    d = s.draft_tok.cpu().numpy()
    v = s.verify_tok.cpu().numpy()
    m = s.accept_len.cpu().numpy()
    c = s.commit_tok.cpu().numpy()
    hid = s.hid.cpu().numpy()
    lg = s.logits.cpu().numpy() if s.logits is not None else None
    dl = s.draft_logits.cpu().numpy() if s.draft_logits is not None else None
    ri = s.route_idx.cpu().numpy() if s.route_idx is not None else None
    rg = s.route_gap.cpu().numpy() if s.route_gap is not None else None
    lh = s.layer_h.cpu().numpy() if s.layer_h is not None else None
    du = s.draft_u.cpu().numpy() if s.draft_u is not None else None
    dd = s.drafted_tok.cpu().numpy() if (s.record and s.override is not None) else None
    for b in range(B):
        rec = dict(drafts=d[b, :K].tolist(), verify=v[b].tolist(), m=int(m[b]),
                   commit=c[b].tolist(), hid=hid[b])
        if lg is not None:
            rec["logits"] = lg[b]
        if dl is not None and K > 0:
            rec["draft_logits"] = dl[b, :K]
        if ri is not None:
            rec["routes"] = ri[:, b * (K + 1):(b + 1) * (K + 1)]
        if rg is not None:
            rec["route_gap"] = rg[:, b * (K + 1):(b + 1) * (K + 1)]
        if lh is not None:
            rec["layer_h"] = lh[:, b * (K + 1):(b + 1) * (K + 1)]
        if du is not None and K > 0:
            rec["draft_u"] = du[b, :K]
        if dd is not None:
            rec["draft_tokens_drafted"] = dd[b, :K].tolist()
        recs.append(rec)
    return recs


def finished(s: Session) -> bool:
    return bool((s.n_out >= s.max_new).all().item())


def synthetic_context(cfg, B, ctx, seqs):
    """Synthetic cached context (the batch-16/64 recipe): verifier and draft
    K/V N(0,1) in the storage dtype (seed 15), last-commit states b N(0,1)
    (seed 15, stream 72), pending tokens uniform (seed 15, stream 73).  Only
    the sequences in `seqs` get K/V values (the others keep zero caches of
    the same lengths).  Returns kv {b: [L][2][nh][ctx][dh]}, dkv {b: ...},
    hid [B][H], pending [B]."""
    kv, dkv = {}, {}
    for b in seqs:
        n = int(ctx[b])
        kv[b] = np.stack([np.stack([synth.kv_values(cfg, l, b, c, n, 15, 70) for c in range(2)])
                          for l in range(cfg.n_layers)])
        dkv[b] = np.stack([synth.kv_values(cfg, 0, b, c, n - 1, 15, 71) for c in range(2)])
    hid = synth.normal(15, 72, (B, cfg.hidden))
    pend = synth.uniform_int(15, 73, B, 0, cfg.vocab)
    return kv, dkv, hid, pend


def load_synthetic(s: Session, cfg, ctx, kv, dkv, hid, pend):
    """Put a synthetic_context into a GPU session (state after a commit of
    one row at ctx-1)."""
    for b, a in kv.items():
        s.kv[:, b, :, :, :a.shape[3]] = to_dev_storage(a)
    for b, a in dkv.items():
        s.dkv[b, :, :, :a.shape[2]] = to_dev_storage(a)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    ctx = np.asarray(ctx, np.int32)
    s.kv_len.copy_(t(ctx))
    s.row_pos.copy_(t(ctx - 1))
    s.draft_len.copy_(t(ctx - 1))
    s.n_rows.fill_(1)
    s.pending.copy_(t(pend))
    s.next_tok[:, 0] = t(pend)
    s.hid[:, 0] = torch.from_numpy(np.ascontiguousarray(hid, np.float32)).cuda()
    s.n_out.fill_(0)


def oracle_synthetic_state(orc, cfg, b, ctx_b, cap, kv, dkv, hid, pend):
    """The oracle's state for sequence b of a synthetic_context."""
    f = (lambda a: synth.bf16_bits_to_f32(a)) if cfg.dtype == "bf16" else (lambda a: a)
    okv, odkv = orc.new_kv(cap), orc.new_dkv(cap)
    okv[:, :, :, :ctx_b] = f(kv[b])
    odkv[:, :, :ctx_b - 1] = f(dkv[b])
    p = int(pend[b])
    return oracle.SeqState(kv=okv, dkv=odkv, kv_len=ctx_b, pending=p,
                           hid=np.ascontiguousarray(hid[b:b + 1], np.float32),
                           next_tok=np.array([p], np.int32), n_rows=1, row_pos=ctx_b - 1,
                           draft_len=ctx_b - 1, out=[p])


def pre_state(s: Session, seqs):
    """The step state of the sequences in seqs before a step (host copies),
    for the layer-local check."""
    torch.cuda.synchronize()
    g = {k: getattr(s, k).cpu().numpy() for k in ("kv_len", "pending", "n_rows", "row_pos",
                                                   "hid", "next_tok")}
    return {b: dict(kv_len=int(g["kv_len"][b]), pending=int(g["pending"][b]),
                    n_rows=int(g["n_rows"][b]), row_pos=int(g["row_pos"][b]),
                    hid=g["hid"][b].copy(), next_tok=g["next_tok"][b].copy())
            for b in seqs}


def post_caches(s: Session, b, n_pos, cap):
    """Sequence b's verifier and draft caches after a step, positions
    0..n_pos-1, as float32 slabs of capacity cap (the oracle's layout)."""
    L = s.m.cfg.n_layers
    kv = s.kv[:, b, :, :, :n_pos].cpu().numpy()
    dkv = s.dkv[b, :, :, :n_pos].cpu().numpy()
    if s.m.bf16:
        kv = synth.bf16_bits_to_f32(kv.view(np.uint16))
        dkv = synth.bf16_bits_to_f32(dkv.view(np.uint16))
    okv = np.zeros((L,) + kv.shape[1:3] + (cap, kv.shape[-1]), np.float32)
    okv[..., :n_pos, :] = kv
    odkv = np.zeros(dkv.shape[:2] + (cap, dkv.shape[-1]), np.float32)
    odkv[..., :n_pos, :] = dkv
    return okv, odkv


def local_check(orc, s: Session, pre, recs, K, stats):
    """Layer-local check (replay.local_step) of the step just run for the
    sequences in pre."""
    from tests import replay
    for b, p in pre.items():
        n_pos = p["kv_len"] + K + 1
        kv, dkv = post_caches(s, b, n_pos, n_pos + K + 1)
        replay.local_step(orc, p, recs[b], kv, dkv, K, stats)

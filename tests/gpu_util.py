"""Helpers shared by the GPU tests: model setup on both sides and step
records copied back from the device."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import synth
from paper_2609_03181_amd.session import Model, Session


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


def oracle_prefill(orc, cfg, tok_b, vis_b, cap, max_new):
    nv = int((tok_b < 0).sum())
    return oracle.prefill(orc, cap, vis_b[:nv] if nv else None, tok_b[nv:], max_new=max_new)


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
    for b in range(B):
        rec = dict(drafts=d[b, :K].tolist(), verify=v[b].tolist(), m=int(m[b]),
                   commit=c[b].tolist(), hid=hid[b])
        if lg is not None:
            rec["logits"] = lg[b]
        if dl is not None and K > 0:
            rec["draft_logits"] = dl[b, :K]
        if ri is not None:
            rec["routes"] = ri[:, b * (K + 1):(b + 1) * (K + 1)]
        recs.append(rec)
    return recs


def finished(s: Session) -> bool:
    return bool((s.n_out >= s.max_new).all().item())

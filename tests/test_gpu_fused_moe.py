"""The small-batch MoE sub-layer in one launch (k_s_moe) against the
three-launch form (router, gate/up, down), bit for bit.

The fused kernel keeps every sum of the three kernels in the same order
(per-wave MFMA chains, wave-order block sums, fixed-point down sums), so
whole decode trajectories -- prefill of up to 16 rows per pass, draft,
verify, accept, commit, graph replay -- must agree in every output bit.
MTP_FUSED_MOE=0 (read when a context is created) selects the three-launch
form.  Full-shape cases cover one and four sequences (4 and 16 verify
rows), the others every router-strip and expert-count shape of the small
models (E = 8 with a partial strip, E = 16) and odd row counts."""
import numpy as np
import pytest
import torch

import synth
from paper_2609_03181_amd.session import Model, Session
from tests.gpu_util import build_pair, gpu_prefill, log, prefix_inputs

pytestmark = pytest.mark.gpu


def _trajectory(name, B, K, n_vis, n_txt, steps, graph, fused, monkeypatch, **wkw):
    monkeypatch.setenv("MTP_FUSED_MOE", fused)
    cfg, w, model, _ = build_pair(name, B, n_vis + n_txt + steps * (K + 1) + 8, 3, **wkw)
    tok, vis = prefix_inputs(cfg, B, n_vis, n_txt)
    s = gpu_prefill(model, B, K, tok, vis, steps * (K + 1) + 4, record=True)
    recs = []
    if graph:
        s.capture()
    for _ in range(steps):
        s.replay() if graph else s.step()
        torch.cuda.synchronize()
        recs.append({k: v.cpu().clone() for k, v in
                     dict(vt=s.verify_tok, hid=s.hid, lg=s.logits, mg=s.margin, ri=s.route_idx,
                          rg=s.route_gap, lh=s.layer_h, dl=s.draft_logits, du=s.draft_u,
                          acc=s.accept_len).items()})
    res = dict(recs=recs, kv=s.kv.cpu(), dkv=s.dkv.cpu(), out=s.out_tok.cpu(),
               n_out=s.n_out.cpu(), pre_routes=s.prefill_routes.cpu(), status=s.status())
    model.close()
    return res


def _check(a, b, label):
    assert a["status"] == 0 and b["status"] == 0, (a["status"], b["status"])
    for key in ("kv", "dkv", "out", "n_out", "pre_routes"):
        assert torch.equal(a[key], b[key]), (label, key)
    for i, (ra, rb) in enumerate(zip(a["recs"], b["recs"])):
        for key in ra:
            assert torch.equal(ra[key], rb[key]), (label, i, key)


@pytest.mark.parametrize("name,B,K,n_vis,n_txt,graph", [
    ("mid", 1, 3, 8, 8, False),    # 4 verify rows, E = 16 (one router strip)
    ("mid", 4, 3, 6, 6, True),     # 16 rows, graph replay
    ("mid", 5, 2, 6, 6, False),    # 15 rows
    ("mid", 3, 0, 6, 6, False),    # plain greedy decoding: 3 rows
    ("tinyb", 3, 3, 6, 6, False),  # E = 8: a partial router strip; 12 rows
])
def test_fused_moe_equals_three_launches(name, B, K, n_vis, n_txt, graph, monkeypatch):
    args = (name, B, K, n_vis, n_txt, 6, graph)
    a = _trajectory(*args, "0", monkeypatch, gain_jitter=0.1)
    b = _trajectory(*args, "1", monkeypatch, gain_jitter=0.1)
    _check(a, b, name)
    log(f"[fused moe] {name} B={B} K={K} graph={graph}: 6 steps bit-identical, "
        f"{int(a['n_out'].sum())} tokens")


@pytest.mark.parametrize("B", [1, 4])
def test_fused_moe_equals_three_launches_full_shape(B, monkeypatch):
    """Full shape (64 routed experts, 4 router strips, I = 896): 12-row
    prefill passes and graph-replayed steps of 4 and 16 verify rows."""
    args = ("full", B, 3, 6, 6, 4, True)
    a = _trajectory(*args, "0", monkeypatch)
    b = _trajectory(*args, "1", monkeypatch)
    _check(a, b, "full")
    log(f"[fused moe] full B={B}: 4 graph steps bit-identical")

"""The page loop at the full model shape: 32 synthetic pages (256 vision
rows N(0,1), seed 20+page, and the same 32 prompt tokens, seed 21), greedy
speculative decoding with K=3 to 2048 new tokens per page, the whole step
captured once in a HIP graph and replayed.  Pages 0-3 are checked token for
token against the oracle's greedy decode by a teacher-forced causal pass
over the GPU's tokens; near-ties of tokens and of routing decisions follow
the GPU (its routing of every checked position is recorded: the prefill's,
then that of each committed verify row).  The check covers the first
MTP_PAGES_CHECK_TOKENS tokens of each page (default: all 2048)."""
import os
import time

import numpy as np
import pytest

import oracle
import synth
from paper_2609_03181_amd.session import Model, Session
from tests import replay
from tests.gpu_util import log, to_dev_storage
import torch

pytestmark = pytest.mark.gpu

PAGES, N_VIS, N_TXT, N_NEW, K = 32, 256, 32, 2048, 3


def run_pages(model, tok, vis, n_check):
    """Runs the page loop; returns the session, the step count and the
    routes [L][P + n_check][k] of pages 0-3."""
    cfg = model.cfg
    P = tok.shape[1]
    s = Session(model, PAGES, K, N_NEW, prefill_rows=64, record=True)
    s.prefill(torch.from_numpy(tok), to_dev_storage(vis))
    routes = np.zeros((4, cfg.n_layers, P + n_check + K + 1, cfg.top_k), np.int32)
    routes[:, :, :P] = s.prefill_routes.cpu().numpy()[:, :4].transpose(1, 0, 2, 3)
    s.capture()
    steps = 0
    # first steps one replay at a time: the committed rows' routing of pages 0-3
    while int(s.n_out[:4].min().item()) < min(n_check + 1, N_NEW):
        s.replay()
        steps += 1
        ri = s.route_idx.cpu().numpy()
        m = s.accept_len.cpu().numpy()
        kv = s.kv_len.cpu().numpy()
        for q in range(4):
            kv0 = int(kv[q]) - int(m[q]) - 1
            for i in range(int(m[q]) + 1):
                if kv0 + i < routes.shape[2]:
                    routes[q, :, kv0 + i] = ri[:, q * (K + 1) + i]
        assert steps < 4 * N_NEW
    while not bool((s.n_out >= N_NEW).all().item()):
        for _ in range(64):
            s.replay()
        steps += 64
        assert steps < 4 * N_NEW
    assert s.status() == 0
    return s, steps, routes


def test_page_loop_matches_oracle_greedy_decode():
    cfg = synth.FULL
    n_check = int(os.environ.get("MTP_PAGES_CHECK_TOKENS", str(N_NEW)))
    log(f"[pages] weights; {PAGES} pages x {N_NEW} new tokens, checking {n_check} on pages 0-3")
    w = synth.make_weights(cfg, 0, 1)
    tok, vis = synth.page_inputs(cfg, PAGES, N_VIS, N_TXT)
    model = Model(cfg, w, PAGES, N_VIS + N_TXT + N_NEW + 4 * (K + 1) + 8, K)
    try:
        t0 = time.time()
        s, steps, routes = run_pages(model, tok, vis, n_check)
        outs = s.outputs()
        log(f"[pages] {steps} graph steps in {time.time() - t0:.1f} s")
        assert all(len(o) == N_NEW for o in outs)
        orc = oracle.Oracle(cfg, w)
        stats = replay.new_stats()
        for q in range(4):
            t1 = time.time()
            n = replay.teacher_forced_check(orc, tok[q], vis[q], np.array(outs[q][:n_check]),
                                            stats, routes=routes[q])
            log(f"[pages] page {q}: {n} tokens match ({time.time() - t1:.1f} s); near-tie "
                f"band so far: {replay.band_report(stats)}")
        log(f"[pages] near-tie band: {replay.assert_band(stats)}")
    finally:
        model.close()

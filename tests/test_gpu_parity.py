"""GPU parity of the HIP decode path against the CPU oracle, through the
C ABI.  Integers (tokens, routes, m, commit lists, lengths) must match
exactly except at the oracle's own near-ties (per-layer routing
tolerances and the token margin of tests/tolerances.py); floats to 1e-4
(fp32 model) or 2e-2 (bf16 logits).  Every replay prints and bounds the
fraction of decisions that fell in the near-tie band."""
import copy
import itertools

import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2609_03181_amd import _lib
from paper_2609_03181_amd.session import Session
from tests import replay, tolerances
from tests.gpu_util import (build_pair, finished, gpu_prefill, local_check, log, oracle_prefill,
                            pre_state, prefix_inputs, step_records, to_dev_storage)

pytestmark = pytest.mark.gpu



def _kv_close(s, st, b, n, tol):
    """GPU caches of sequence b versus the oracle's, positions < n."""
    L = s.m.cfg.n_layers
    kv = s.kv[:, b, :, :, :n].cpu()
    dkv = s.dkv[b, :, :, :max(st.draft_len, 0)].cpu()
    if s.m.bf16:
        kv = synth.bf16_bits_to_f32(kv.numpy().view(np.uint16))
        dkv = synth.bf16_bits_to_f32(dkv.numpy().view(np.uint16))
    else:
        kv, dkv = kv.numpy(), dkv.numpy()
    np.testing.assert_allclose(kv, st.kv[:L, :, :, :n], rtol=tol, atol=tol)
    np.testing.assert_allclose(dkv, st.dkv[:, :, :st.draft_len], rtol=tol, atol=tol)


def _run_and_replay(name, B, K, n_vis, n_txt, max_out, cap, wkw=None, check_kv=True):
    cfg, w, model, orc = build_pair(name, B, cap, max(K, 1), **(wkw or {}))
    tol, stol = tolerances.logit_tol(cfg), tolerances.state_tol(cfg)
    tok, vis = prefix_inputs(cfg, B, n_vis, n_txt)
    log(f"[{name}] prefill B={B} P={n_vis + n_txt} K={K}")
    s = gpu_prefill(model, B, K, tok, vis, max_out)
    assert s.status() == 0
    pr = s.prefill_routes.cpu().numpy()
    sts = [oracle_prefill(orc, cfg, tok[b], vis[b], cap, max_out, routes=pr[:, b])
           for b in range(B)]
    hid0 = s.hid.cpu().numpy()
    for b in range(B):
        t = replay.check_token(sts[b].last_logits, sts[b].pending, int(s.pending[b]),
                               "prefill token", replay.new_stats())
        if t != sts[b].pending:          # near-tie: continue on the GPU's token
            sts[b].pending = t
            sts[b].next_tok[0] = t
            sts[b].out[0] = t
        np.testing.assert_allclose(hid0[b, 0], sts[b].hid[0], rtol=stol, atol=stol)
        if check_kv:
            _kv_close(s, sts[b], b, sts[b].kv_len, tol)
    stats, lstats = replay.new_stats(), replay.new_stats()
    n_steps = 0
    while not finished(s):
        active = [b for b in range(B) if not sts[b].finished]
        pre = pre_state(s, active)
        s.step()
        recs = step_records(s)
        for b in active:
            replay.replay_step(orc, sts[b], K, recs[b], stats, tol, state_tol=stol)
        local_check(orc, s, pre, recs, K, lstats)
        n_steps += 1
        assert n_steps < 4 * max_out
    assert s.status() == 0
    outs = s.outputs()
    for b in range(B):
        assert outs[b] == sts[b].out[:max_out]
        assert int(s.kv_len[b]) == sts[b].kv_len
        if check_kv:
            _kv_close(s, sts[b], b, sts[b].kv_len, tol)
    log(f"[{name}] {n_steps} steps ok; end-to-end near-tie band: {replay.assert_band(stats)}; "
        f"layer-local: {replay.assert_local_band(lstats)}")
    return s, sts, stats


def test_tiny_config_spec_decode_matches_oracle():
    """Tiny fp32 case: 64 vision rows + 16 tokens, K=3, 32 new tokens."""
    _run_and_replay("tiny", 1, 3, 64, 16, 32, 128)


def test_tiny_untied_batch_spec_decode_matches_oracle():
    _run_and_replay("tinyu", 3, 3, 12, 9, 20, 96, dict(gain_jitter=0.1))


def test_mid_bf16_spec_decode_matches_oracle():
    """bf16 model with several tiles per dimension, a ragged vocabulary tail
    (8000), Zipf-biased routing, jittered gains; ragged commit lengths."""
    _run_and_replay("mid", 2, 3, 16, 12, 14, 96, dict(gain_jitter=0.1, zipf_s=1.1))


def test_mid_bf16_batch6_multi_group_path():
    """24 rows per pass: two 16-row groups, MoE down through slots, the
    separate grouping kernel."""
    _run_and_replay("mid", 6, 3, 8, 8, 8, 96, dict(gain_jitter=0.1, zipf_s=1.1))


def test_mid_bf16_batch17_ragged_groups():
    """68 rows per pass: five 16-row groups, the last one ragged (4 rows)."""
    _run_and_replay("mid", 17, 3, 4, 4, 5, 64, dict(gain_jitter=0.1), check_kv=False)


def test_k0_is_plain_greedy_on_gpu():
    _run_and_replay("tinyb", 2, 0, 6, 6, 12, 64)


def test_gpu_spec_equals_gpu_greedy_bitwise():
    cfg, w, model, orc = build_pair("mid", 2, 128, 3, gain_jitter=0.1)
    tok, vis = prefix_inputs(cfg, 2, 8, 8)
    outs = {}
    for K in (0, 1, 3):
        s = gpu_prefill(model, 2, K, tok, vis, 24, record=False)
        while not finished(s):
            s.step()
        outs[K] = (s.outputs(), s.kv[:, :, :, :, :40].clone())
    for K in (1, 3):
        assert outs[K][0] == outs[0][0]
        n = 16 + 23
        assert torch.equal(outs[K][1][..., :n, :], outs[0][1][..., :n, :])


def test_graph_replay_equals_eager():
    cfg, w, model, orc = build_pair("mid", 2, 128, 3)
    tok, vis = prefix_inputs(cfg, 2, 8, 8)
    eager = gpu_prefill(model, 2, 3, tok, vis, 20, record=False)
    graph = gpu_prefill(model, 2, 3, tok, vis, 20, record=False)
    graph.capture()
    torch.cuda.synchronize()
    for i in range(12):
        eager.step()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(eager.out_tok, graph.out_tok), i
        assert torch.equal(eager.kv_len, graph.kv_len), i
        assert torch.equal(eager.hid, graph.hid), i
    assert torch.equal(eager.kv, graph.kv) and torch.equal(eager.dkv, graph.dkv)


def test_forced_acceptance_reaches_every_m_and_is_lossless():
    """Drafts overwritten from the greedy trajectory (first m* correct,
    next one wrong): m must equal m* and the output the trajectory."""
    B, K, N = 4, 3, 30
    cfg, w, model, orc = build_pair("mid", B, 160, K)
    tok, vis = prefix_inputs(cfg, B, 8, 8)
    ar = gpu_prefill(model, B, 0, tok, vis, N + K + 2, record=False)
    while not finished(ar):
        ar.step()
    traj = ar.outputs()
    # the trajectory itself against the oracle (replayed greedy steps)
    st = oracle_prefill(orc, cfg, tok[0], vis[0], 160, N + K + 2)
    for t in traj[0][1:8]:
        r = orc.verify_rows(st.kv, [st.pending], [st.kv_len], want_logits=True)
        replay.check_token(r["logits"][0], int(r["amax"][0]), t, "trajectory", replay.new_stats())
        oracle.commit(st, 0, [t], r["b"])
    ms = synth.uniform_int(13, 70, 256, 0, K + 1)
    # forced table: step s of sequence b starts after len(out) tokens; with
    # m == m* the position is known in advance
    n_steps = 64
    table = np.zeros((n_steps, B, K), np.int32)
    m_star = np.zeros((n_steps, B), np.int32)
    for b in range(B):
        base = 1
        for s_ in range(n_steps):
            m = int(ms[(s_ * B + b) % len(ms)])
            d = [traj[b][min(base + t, len(traj[b]) - 1)] for t in range(K)]
            if m < K:
                d[m] = (d[m] + 1) % cfg.vocab
            table[s_, b] = d
            m_star[s_, b] = m
            base += m + 1
    sp = gpu_prefill(model, B, K, tok, vis, N, record=False)
    sp.set_forced_drafts(torch.from_numpy(table))
    seen = []
    for s_ in range(n_steps):
        if finished(sp):
            break
        active = (sp.n_out < N).cpu().numpy()       # finished sequences are frozen
        sp.step()
        got = sp.accept_len.cpu().numpy()
        assert np.array_equal(got[active], m_star[s_][active]), s_
        seen += got[active].tolist()
    assert set(seen) == set(range(K + 1))
    outs = sp.outputs()
    for b in range(B):
        assert outs[b] == traj[b][:N]


def forced_replay(name, B, K, n_vis, n_txt, n_steps, cap, wkw, check_kv=True):
    """Speculative steps whose drafts are replaced, step by step, from the
    oracle's own greedy continuation of the replayed state: the first m*
    drafts are the greedy tokens, the next is wrong, m* cycling over 0..K
    (seed 13).  The GPU's drafting itself (before the replacement) is
    compared with the oracle's draft chain, token and logits -- including
    the depth-1 catch-up over the m+1 rows of the previous commit, whose
    draft K/V is compared after every step."""
    cfg, w, model, orc = build_pair(name, B, cap, K, **wkw)
    tol, stol = tolerances.logit_tol(cfg), tolerances.state_tol(cfg)
    tok, vis = prefix_inputs(cfg, B, n_vis, n_txt)
    s = gpu_prefill(model, B, K, tok, vis, n_steps * (K + 1) + 4)
    pr = s.prefill_routes.cpu().numpy()
    sts = [oracle_prefill(orc, cfg, tok[b], vis[b], cap, 1 << 30, routes=pr[:, b])
           for b in range(B)]
    for b in range(B):
        t = replay.check_token(sts[b].last_logits, sts[b].pending, int(s.pending[b]),
                               "prefill token", replay.new_stats())
        sts[b].pending = t
        sts[b].next_tok[0] = t
        sts[b].out[0] = t
    ms = synth.uniform_int(13, 71, n_steps * B, 0, K + 1)
    stats, lstats = replay.new_stats(), replay.new_stats()
    seen = set()
    for i in range(n_steps):
        table = np.zeros((1, B, K), np.int32)
        m_star = []
        for b in range(B):
            ahead = copy.deepcopy(sts[b])
            ahead.max_new = 1 << 30
            traj = oracle.ar_decode(orc, ahead, len(ahead.out) + K)[len(sts[b].out):]
            m = int(ms[i * B + b])
            d = list(traj[:K])
            if m < K:
                d[m] = (d[m] + 1) % cfg.vocab
            table[0, b] = d
            m_star.append(m)
        s.set_forced_drafts(torch.from_numpy(table))
        pre = pre_state(s, range(B))
        s.step()
        recs = step_records(s)
        for b in range(B):
            got = replay.replay_step(orc, sts[b], K, recs[b], stats, tol,
                                     forced=table[0, b].tolist(), state_tol=stol)
            seen.add(got)
            if check_kv:
                _kv_close(s, sts[b], b, sts[b].kv_len, tol)
        local_check(orc, s, pre, recs, K, lstats)
        log(f"  step {i}: m* {m_star}, m {[r['m'] for r in recs]}")
    assert s.status() == 0
    assert seen == set(range(K + 1)), seen
    log(f"[{name} forced] {n_steps} steps, m seen {sorted(seen)}; end-to-end near-tie band: "
        f"{replay.assert_band(stats)}; layer-local: {replay.assert_local_band(lstats)}")


def test_mid_bf16_forced_acceptance_replayed_against_oracle():
    forced_replay("mid", 2, 3, 12, 10, 10, 96, dict(gain_jitter=0.1, zipf_s=1.1))


def test_tiny_forced_acceptance_replayed_against_oracle():
    forced_replay("tinyu", 2, 3, 8, 8, 10, 96, dict(gain_jitter=0.1))


def test_greedy_accept_exhaustive_on_gpu():
    V, K = 3, 3
    cases = [(d, v) for d in itertools.product(range(V), repeat=K)
             for v in itertools.product(range(V), repeat=K + 1)]
    B = len(cases)
    dr = torch.tensor([c[0] for c in cases], dtype=torch.int32, device="cuda")
    vf = torch.tensor([c[1] for c in cases], dtype=torch.int32, device="cuda")
    m = torch.zeros(B, dtype=torch.int32, device="cuda")
    cm = torch.zeros((B, K + 1), dtype=torch.int32, device="cuda")
    _lib.greedy_accept(B, K, dr.data_ptr(), vf.data_ptr(), m.data_ptr(), cm.data_ptr(),
                       torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    m, cm = m.cpu().numpy(), cm.cpu().numpy()
    for i, (d, v) in enumerate(cases):
        mm, commit = oracle.accept(d, v)
        assert m[i] == mm
        assert cm[i, :mm + 1].tolist() == commit
        assert (cm[i, mm + 1:] == -1).all()


def test_commit_rollback_bookkeeping_and_max_new_clamp():
    cfg, w, model, orc = build_pair("tiny", 8, 64, 3)
    B, K, max_out = 8, 3, 10
    rng = np.random.default_rng(0)
    kv_len = rng.integers(5, 40, B).astype(np.int32)
    m = rng.integers(0, K + 1, B).astype(np.int32)
    commit = np.full((B, K + 1), -1, np.int32)
    for b in range(B):
        commit[b, :m[b] + 1] = rng.integers(0, cfg.vocab, m[b] + 1)
    n_out = np.array([0, 3, 8, 9, 10, 7, 6, 2], np.int32)
    max_new = np.array([10, 10, 10, 10, 10, 9, 7, 10], np.int32)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    t = dict(kv=T(kv_len), nr=T(np.ones(B, np.int32)), rp=T(kv_len - 1),
             pend=T(np.zeros(B, np.int32)), nt=T(np.zeros((B, K + 1), np.int32)),
             out=T(np.full((B, max_out), -7, np.int32)), no=T(n_out))
    m_d, commit_d, max_new_d = T(m), T(commit), T(max_new)     # keep alive across the launch
    _lib.kv_commit_rollback(model.ctx, B, K, m_d.data_ptr(), commit_d.data_ptr(),
                            t["kv"].data_ptr(), t["nr"].data_ptr(), t["rp"].data_ptr(),
                            t["pend"].data_ptr(), t["nt"].data_ptr(), max_new_d.data_ptr(),
                            t["out"].data_ptr(), max_out, t["no"].data_ptr(),
                            torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in t.items()}
    for b in range(B):
        limit = min(max_new[b], max_out)
        if n_out[b] >= limit:                                  # finished: frozen
            assert g["kv"][b] == kv_len[b] and g["no"][b] == n_out[b]
            continue
        take = min(m[b] + 1, limit - n_out[b])
        assert g["kv"][b] == kv_len[b] + m[b] + 1
        assert g["nr"][b] == m[b] + 1 and g["rp"][b] == kv_len[b]
        assert g["pend"][b] == commit[b, m[b]]
        assert g["nt"][b, :m[b] + 1].tolist() == commit[b, :m[b] + 1].tolist()
        assert g["no"][b] == n_out[b] + take
        assert g["out"][b, n_out[b]:n_out[b] + take].tolist() == commit[b, :take].tolist()
        assert (g["out"][b, n_out[b] + take:] == -7).all()


def test_commit_rejects_out_of_range_accept_len():
    """An acceptance length outside [0, k] (acceptance equation: 0 <= m <=
    k) sets the context's status word and leaves the sequence unchanged."""
    cfg, w, model, orc = build_pair("tiny", 2, 64, 3)
    B, K, max_out = 2, 3, 8
    T = lambda a: torch.tensor(a, dtype=torch.int32, device="cuda")
    m = T([K + 1, -1])
    commit = T([[1, 2, 3, 4], [5, 6, 7, 8]])
    kv_len, nr, rp = T([10, 12]), T([1, 1]), T([9, 11])
    pend, nt = T([0, 0]), torch.zeros((B, K + 1), dtype=torch.int32, device="cuda")
    out, no = torch.full((B, max_out), -7, dtype=torch.int32, device="cuda"), T([0, 0])
    before = [t.clone() for t in (kv_len, nr, rp, pend, nt, out, no)]
    stream = torch.cuda.current_stream().cuda_stream
    _lib.kv_commit_rollback(model.ctx, B, K, m.data_ptr(), commit.data_ptr(), kv_len.data_ptr(),
                            nr.data_ptr(), rp.data_ptr(), pend.data_ptr(), nt.data_ptr(), None,
                            out.data_ptr(), max_out, no.data_ptr(), stream)
    torch.cuda.synchronize()
    assert _lib.mtp_status_read(model.ctx, None) == _lib.MTP_ERANGE
    for a, b in zip(before, (kv_len, nr, rp, pend, nt, out, no)):
        assert torch.equal(a, b)
    _lib.mtp_status_clear(model.ctx, None, stream)
    torch.cuda.synchronize()
    assert _lib.mtp_status_read(model.ctx, None) == _lib.MTP_OK
    assert _lib.mtp_context_bytes(model.ctx) >= 64 * (cfg.head_dim // 2) * 8


def test_capacity_overflow_sets_sticky_status_without_writes():
    cfg, w, model, orc = build_pair("tiny", 1, 40, 3)
    tok, vis = prefix_inputs(cfg, 1, 4, 4)
    s = gpu_prefill(model, 1, 3, tok, vis, 64, record=False)
    assert s.status() == 0
    s.kv_len.fill_(38)                      # rows at 38..41 pass max_ctx = 40
    before = s.kv.clone()
    s.verify()
    assert s.status() == _lib.MTP_ECAPACITY
    # valid rows (38, 39) wrote their K/V; nothing else changed
    diff = (s.kv != before).any(dim=(0, 1, 2, 3, 5)).cpu().numpy()
    assert set(np.nonzero(diff)[0].tolist()) <= {38, 39}
    _lib.mtp_status_clear(model.ctx, s.ws.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert s.status() == 0


def test_bad_token_sets_status():
    cfg, w, model, orc = build_pair("tiny", 1, 40, 3)
    tok, vis = prefix_inputs(cfg, 1, 4, 4)
    s = gpu_prefill(model, 1, 0, tok, vis, 64, record=False)
    s.pending.fill_(cfg.vocab + 5)
    s.verify()
    assert s.status() == _lib.MTP_ETOKEN


def test_host_argument_errors():
    cfg, w, model, orc = build_pair("tiny", 2, 40, 3)
    s = Session(model, 2, 3, 8, record=False)
    with pytest.raises(_lib.MtpError) as e:
        _lib.moe_verify_step(model.ctx, 3, 3, s.pending.data_ptr(), s.draft_tok.data_ptr(),
                             s.kv_len.data_ptr(), s.kv.data_ptr(), s.verify_tok.data_ptr(),
                             s.hid.data_ptr(), None, None, None, None, None, s.ws.data_ptr(),
                             s.ws_bytes, 0)
    assert e.value.code == _lib.MTP_EINVAL
    with pytest.raises(_lib.MtpError):
        _lib.mtp_draft_k(model.ctx, 2, 4, s.hid.data_ptr(), s.next_tok.data_ptr(),
                         s.n_rows.data_ptr(), s.row_pos.data_ptr(), s.dkv.data_ptr(),
                         s.draft_len.data_ptr(), s.draft_tok.data_ptr(), None, None, s.ws.data_ptr(),
                         s.ws_bytes, 0)
    with pytest.raises(_lib.MtpError):           # workspace too small
        _lib.moe_verify_step(model.ctx, 2, 3, s.pending.data_ptr(), s.draft_tok.data_ptr(),
                             s.kv_len.data_ptr(), s.kv.data_ptr(), s.verify_tok.data_ptr(),
                             s.hid.data_ptr(), None, None, None, None, None, s.ws.data_ptr(), 1024, 0)


def test_steps_after_prefill_do_not_depend_on_workspace_history():
    """The workspace is carved per call by its row count; a step after a
    prefill with larger chunks (other carve) must equal one after a prefill
    with the step's own row count, bit for bit (regression: attention
    split counters left non-zero by a differently carved call)."""
    cfg, w, model, orc = build_pair("mid", 1, 96, 3, gain_jitter=0.1)
    tok, _ = prefix_inputs(cfg, 1, 0, 40)
    res = []
    for rows in (4, 8, 16):
        s = Session(model, 1, 3, 16, prefill_rows=rows, record=True)
        s.prefill(torch.from_numpy(tok))
        for _ in range(2):
            s.step()
        torch.cuda.synchronize()
        res.append((s.draft_logits.cpu().numpy().copy(), s.logits.cpu().numpy().copy(),
                    s.outputs()))
    for r in res[1:]:
        assert np.array_equal(r[0], res[0][0])
        assert np.array_equal(r[1], res[0][1])
        assert r[2] == res[0][2]

"""GPU parity at the full model shape (12 layers, H=1280, 64+2 experts
top-6, V=129280, bf16), in the launch configuration bench.py times (the
whole step captured in a HIP graph and replayed), against the oracle:

* batch 1: the prompt (256 vision rows + 512 tokens) prefilled in one pass
  as the benchmark does, then graph-replayed steps whose drafts are
  replaced from the oracle's own greedy continuation so that every
  acceptance length 0..3 occurs (the catch-up of m+1 committed rows, its
  draft K/V and the multi-row commits are compared), then natural steps;
* batch 1, spec == greedy bit for bit for K = 1, 2, 3 against K = 0;
* batch 4: cached contexts U{512..1024} (seed 5), synthetic caches (16
  verify rows: one full row group);
* batch 16: cached contexts U{1024..2048} (seed 2), every sequence with a
  synthetic cache, acceptance forced by the benchmark's own table
  (P(m) = 0.2/0.2/0.25/0.35, seed 13); 8 sequences replayed, the shortest
  and the longest among them;
* batch 64: cached contexts U{512..4096} (seed 12), Zipf(1.1) router bias,
  every sequence with a synthetic cache; 8 sequences replayed;
* batch 1 at a long context: 30,000 cached positions of a 32,768-position
  cache (RoPE base 1e6; decode attention in 64 key splits of 512);
* a Gundam-mode page: 1156 vision rows + 64 prompt tokens prefilled in one
  pass, then graph-replayed steps.

Tolerances come from tests/tolerances.py (per-layer routing tolerances and
float tolerances derived from the measured float32-summation drift of
this model); every replay prints and bounds the near-tie band."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2609_03181_amd.session import Model, Session
from tests import replay, tolerances
from tests.gpu_util import (finished, gpu_prefill, local_check, log, oracle_prefill,
                            oracle_synthetic_state, pre_state, prefix_inputs, step_records,
                            to_dev_storage)

pytestmark = pytest.mark.gpu

CFG = synth.FULL
TOL = tolerances.logit_tol(CFG)
STATE_TOL = tolerances.state_tol(CFG)


@pytest.fixture(scope="module")
def plain():
    log("[full] weights (seed 0, draft seed 1)")
    w = synth.make_weights(CFG, 0, 1)
    model = Model(CFG, w, 16, 2048 + 64, 3)
    yield w, model, oracle.Oracle(CFG, w)
    model.close()


def _replay_steps(orc, s, sts, K, n_steps, stats, lstats, graph=True, forced=None):
    """Graph-replayed steps, each replayed through the oracle end to end
    (stats) and checked layer by layer (lstats) for the sequences in sts;
    forced [n_steps][B][K] drafts (the session's forced table) or None."""
    if graph and s.graph is None:
        s.capture()
    for i in range(n_steps):
        pre = pre_state(s, list(sts))
        if graph:
            s.replay()
        else:
            s.step()
        recs = step_records(s)
        for b, st in sts.items():
            replay.replay_step(orc, st, K, recs[b], stats, TOL, state_tol=STATE_TOL,
                               forced=None if forced is None else forced[i][b].tolist())
        local_check(orc, s, pre, recs, K, lstats)
        log(f"  step {i}: m = {[recs[b]['m'] for b in sts]}")
    assert s.status() == 0
    for b, st in sts.items():
        assert int(s.kv_len[b]) == st.kv_len


def fill_synthetic(s, cfg, ctx, keep):
    """Every sequence gets the synthetic cached context of the batch-16/64
    recipe (verifier and draft K/V N(0,1) -> bf16, seed 15; last-commit
    states N(0,1) and pending tokens, seed 15), uploaded one sequence at a
    time; the host copies of the sequences in `keep` are returned for the
    oracle.  The state is that after a commit of one row at ctx-1."""
    B = len(ctx)
    kv, dkv = {}, {}
    for b in range(B):
        n = int(ctx[b])
        kb = np.stack([np.stack([synth.kv_values(cfg, l, b, c, n, 15, 70) for c in range(2)])
                       for l in range(cfg.n_layers)])
        db = np.stack([synth.kv_values(cfg, 0, b, c, n - 1, 15, 71) for c in range(2)])
        s.kv[:, b, :, :, :n] = to_dev_storage(kb)
        s.dkv[b, :, :, :n - 1] = to_dev_storage(db)
        if b in keep:
            kv[b], dkv[b] = kb, db
    hid = synth.normal(15, 72, (B, cfg.hidden))
    pend = synth.uniform_int(15, 73, B, 0, cfg.vocab)
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
    return kv, dkv, hid, pend


def sampled_sequences(ctx, n=8):
    """The shortest, the longest and n-2 more spread over the batch."""
    B = len(ctx)
    pick = {int(np.argmin(ctx)), int(np.argmax(ctx))}
    for b in np.linspace(0, B - 1, n).astype(int):
        if len(pick) >= min(n, B):
            break
        pick.add(int(b))
    b = 0
    while len(pick) < min(n, B):
        pick.add(b)
        b += 1
    return sorted(pick)


def _synthetic_case(w, model, orc, B, lo, hi, seed, n_steps, forced=False, n_check=8):
    K = 3
    ctx = synth.context_lengths(B, lo, hi, seed)
    seqs = sampled_sequences(ctx, n_check)
    log(f"[full B={B}] ctx {int(ctx.min())}..{int(ctx.max())}, every cache filled, "
        f"replaying sequences {seqs}")
    s = Session(model, B, K, n_steps * (K + 1) + 4, record=True)
    kv, dkv, hid, pend = fill_synthetic(s, CFG, ctx, set(seqs))
    cap = int(ctx.max()) + n_steps * (K + 1) + 8
    sts = {b: oracle_synthetic_state(orc, CFG, b, int(ctx[b]), cap, kv, dkv, hid, pend)
           for b in seqs}
    del kv, dkv
    table = None
    if forced:
        import bench
        table = bench._forced_table(s, CFG, B, K, n_steps)
        s.set_forced_drafts(torch.from_numpy(table))
    stats, lstats = replay.new_stats(), replay.new_stats()
    _replay_steps(orc, s, sts, K, n_steps, stats, lstats, forced=table)
    log(f"[full B={B}] {n_steps} steps ok; end-to-end near-tie band: "
        f"{replay.assert_band(stats)}; layer-local: {replay.assert_local_band(lstats)}")
    return stats


def test_full_shape_batch1_one_pass_prefill_forced_and_natural_steps(plain):
    """The benchmark's batch-1 workload: one-pass prefill, graph steps."""
    w, model, orc = plain
    K, n_vis, n_txt = 3, 256, 512
    n_forced, n_nat = 8, 2
    P = n_vis + n_txt
    tok, vis = prefix_inputs(CFG, 1, n_vis, n_txt)
    log("[full B=1] GPU prefill of 768 rows in one pass")
    s = gpu_prefill(model, 1, K, tok, vis, (n_forced + n_nat) * (K + 1) + 4, prefill_rows=P)
    assert s.status() == 0
    log("[full B=1] oracle prefill")
    st = oracle_prefill(orc, CFG, tok[0], vis[0], P + (n_forced + n_nat) * (K + 1) + 8,
                        1 << 30, routes=s.prefill_routes.cpu().numpy()[:, 0])
    stats, lstats = replay.new_stats(), replay.new_stats()
    replay.count_routes(stats, st.prefill_route_gap, tolerances.route_tol(CFG),
                        st.prefill_routes_followed)
    log(f"[full B=1] prefill: {st.prefill_routes_followed} of {CFG.n_layers * P} routing "
        f"decisions followed at near-ties; band {replay.band_report(stats)}")
    t = replay.check_token(st.last_logits, st.pending, int(s.pending[0]), "prefill token", stats)
    st.pending = t
    st.next_tok[0] = t
    st.out[0] = t
    np.testing.assert_allclose(s.hid.cpu().numpy()[0, 0], st.hid[0], rtol=TOL, atol=STATE_TOL)
    # forced steps: drafts from the oracle's own greedy continuation
    import copy
    ms = [3, 2, 1, 0, 3, 1, 2, 0]
    s.set_forced_drafts(torch.zeros((1, 1, K), dtype=torch.int32))
    s.capture()
    seen = set()
    for i in range(n_forced):
        ahead = copy.deepcopy(st)
        ahead.max_new = 1 << 30
        traj = oracle.ar_decode(orc, ahead, len(ahead.out) + K)[len(st.out):]
        d = list(traj[:K])
        if ms[i] < K:
            d[ms[i]] = (d[ms[i]] + 1) % CFG.vocab
        s.update_forced_drafts(torch.tensor([[d]], dtype=torch.int32))
        pre = pre_state(s, [0])
        s.replay()
        recs = step_records(s)
        rec = recs[0]
        m = replay.replay_step(orc, st, K, rec, stats, TOL, state_tol=STATE_TOL, forced=d)
        local_check(orc, s, pre, recs, K, lstats)
        seen.add(m)
        log(f"  forced step {i}: m* {ms[i]}, m {m}")
    assert seen == set(range(K + 1)), seen
    kv = s.kv[:, 0, :, :, :st.kv_len].cpu().numpy().view(np.uint16)
    np.testing.assert_allclose(synth.bf16_bits_to_f32(kv), st.kv[:, :, :, :st.kv_len],
                               rtol=TOL, atol=TOL)
    dkv = s.dkv[0, :, :, :st.draft_len].cpu().numpy().view(np.uint16)
    np.testing.assert_allclose(synth.bf16_bits_to_f32(dkv), st.dkv[:, :, :st.draft_len],
                               rtol=TOL, atol=TOL)
    # natural steps (a fresh graph without the forced table)
    s.override = None
    s.graph = None
    _replay_steps(orc, s, {0: st}, K, n_nat, stats, lstats)
    log(f"[full B=1] {n_forced} forced + {n_nat} natural steps ok; end-to-end near-tie band "
        f"(prefill included): {replay.assert_band(stats)}; layer-local: "
        f"{replay.assert_local_band(lstats)}")


@pytest.mark.parametrize("n_txt", [64, 512])
def test_full_shape_gundam_prefix_one_pass(plain, n_txt):
    """Gundam-mode page (Table "Model specification": 256 + 100 n visual
    rows, n = 9 -> 1156, the largest) + n_txt prompt tokens prefilled in one
    pass, then graph-replayed steps: prefill token, state, every verifier
    K/V position and the draft cache against the oracle.  1220 rows (200
    row-tile x head blocks) run the key-split prefill attention, 1668 rows
    (the benchmark's page, 270 blocks) the one-block-per-row-tile form."""
    w, model, orc = plain
    K, n_vis, n_steps = 3, 1156, 3
    P = n_vis + n_txt
    tok, vis = prefix_inputs(CFG, 1, n_vis, n_txt)
    log(f"[gundam] GPU prefill of {P} rows in one pass")
    s = gpu_prefill(model, 1, K, tok, vis, n_steps * (K + 1) + 4, prefill_rows=P)
    assert s.status() == 0
    log("[gundam] oracle prefill")
    st = oracle_prefill(orc, CFG, tok[0], vis[0], P + n_steps * (K + 1) + 8, 1 << 30,
                        routes=s.prefill_routes.cpu().numpy()[:, 0])
    stats, lstats = replay.new_stats(), replay.new_stats()
    replay.count_routes(stats, st.prefill_route_gap, tolerances.route_tol(CFG),
                        st.prefill_routes_followed)
    t = replay.check_token(st.last_logits, st.pending, int(s.pending[0]), "prefill token", stats)
    st.pending = t
    st.next_tok[0] = t
    st.out[0] = t
    np.testing.assert_allclose(s.hid.cpu().numpy()[0, 0], st.hid[0], rtol=TOL, atol=STATE_TOL)
    kv = s.kv[:, 0, :, :, :P].cpu().numpy().view(np.uint16)
    np.testing.assert_allclose(synth.bf16_bits_to_f32(kv), st.kv[:, :, :, :P], rtol=TOL, atol=TOL)
    dkv = s.dkv[0, :, :, :P - 1].cpu().numpy().view(np.uint16)
    np.testing.assert_allclose(synth.bf16_bits_to_f32(dkv), st.dkv[:, :, :P - 1], rtol=TOL,
                               atol=TOL)
    _replay_steps(orc, s, {0: st}, K, n_steps, stats, lstats)
    log(f"[gundam] {P}-row prefill + {n_steps} steps ok; end-to-end near-tie band: "
        f"{replay.assert_band(stats)}; layer-local: {replay.assert_local_band(lstats)}")


def test_full_shape_batch1_spec_equals_greedy_bitwise(plain):
    """Losslessness on the GPU at full shape, bit for bit: with up to 16 rows
    a row's result does not depend on the other rows of its verify pass (the
    MoE down sums in exact fixed point), so speculative decoding with K = 1,
    2 and 3 emits exactly the tokens of plain greedy decoding (K = 0) and
    writes the same verifier K/V."""
    w, model, orc = plain
    n_vis, n_txt, n_new = 256, 512, 48
    tok, vis = prefix_inputs(CFG, 1, n_vis, n_txt)
    outs, kvs = {}, {}
    for K in (0, 1, 2, 3):
        s = gpu_prefill(model, 1, K, tok, vis, n_new, record=False, prefill_rows=n_vis + n_txt)
        s.capture()
        while not finished(s):
            s.replay()
        assert s.status() == 0
        outs[K] = s.outputs()[0]
        kvs[K] = (int(s.kv_len[0]), s.kv[:, 0].clone())
        log(f"[full B=1 bitwise] K={K}: {len(outs[K])} tokens, kv_len {kvs[K][0]}")
        del s
    n = min(v[0] for v in kvs.values())  # committed rows (later ones may be rejected drafts)
    assert n >= n_vis + n_txt + n_new - 4
    for K in (1, 2, 3):
        assert outs[K] == outs[0]
        assert torch.equal(kvs[K][1][..., :n, :], kvs[0][1][..., :n, :])


def test_full_shape_batch4_sixteen_rows_sampled_sequences(plain):
    """Batch 4: 16 verify rows, one full row group -- the streaming MoE
    gate/up stages 16 rows of 1280 (beyond its first 1024 16-byte chunks
    per block) and the RMSNorm prologues take four rows per wave."""
    w, model, orc = plain
    _synthetic_case(w, model, orc, 4, 512, 1024, 5, 3, n_check=4)


def test_full_shape_batch16_forced_acceptance(plain):
    """The benchmark's batch-16 workload: forced acceptance as timed."""
    w, model, orc = plain
    _synthetic_case(w, model, orc, 16, 1024, 2048, 2, 3, forced=True)


def test_full_shape_batch64_zipf():
    log("[full] weights with Zipf(1.1) router bias")
    w = synth.make_weights(CFG, 0, 1, zipf_s=1.1)
    model = Model(CFG, w, 64, 4096 + 64, 3)
    try:
        _synthetic_case(w, model, oracle.Oracle(CFG, w), 64, 512, 4096, 12, 2)
    finally:
        model.close()
        torch.cuda.empty_cache()


def test_full_shape_long_context_split_kv():
    """One sequence with 30,000 cached positions in a 32,768-position cache:
    decode attention over 64 key splits of 512 positions (the merge of the
    maximum split count), RoPE at positions near 30K."""
    log("[full] weights (seed 0, draft seed 1), long context")
    w = synth.make_weights(CFG, 0, 1)
    model = Model(CFG, w, 1, 32768, 3)
    try:
        _synthetic_case(w, model, oracle.Oracle(CFG, w), 1, 30000, 30000, 7, 2, n_check=1)
    finally:
        model.close()
        torch.cuda.empty_cache()

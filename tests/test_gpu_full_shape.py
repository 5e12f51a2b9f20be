"""GPU parity at the full model shape (12 layers, H=1280, 64+2 experts
top-6, V=129280, bf16), in the launch configuration bench.py times (the
whole step captured in a HIP graph and replayed), on sampled sequences the
oracle recomputes one by one:

* batch 1: real prefill of 256 vision rows + 512 prompt tokens, then steps;
* batch 4: cached contexts U{512..1024} (seed 5), synthetic caches (16
  verify rows: one full row group);
* batch 16: cached contexts U{1024..2048} (seed 2), synthetic caches;
* batch 64: cached contexts U{512..4096} (seed 12), Zipf(1.1) router bias,
  synthetic caches;
* batch 1 at a long context: 30,000 cached positions of a 32,768-position
  cache (RoPE base 1e6; decode attention in 64 key splits of 512).

For the synthetic-cache cases only the sampled sequences (shortest,
longest and one more) carry cache values; the others hold zero caches of
their lengths and are not checked.  Tolerances and near-tie handling as in
the small-shape parity tests."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2609_03181_amd.session import Model, Session
from tests import replay
from tests.gpu_util import (finished, gpu_prefill, load_synthetic, log, oracle_prefill,
                            oracle_synthetic_state, prefix_inputs, step_records,
                            synthetic_context)

pytestmark = pytest.mark.gpu

# Logits and final-norm states after 12 bf16 layers: the oracle itself,
# evaluated with float32 instead of float64 dot products on the same inputs
# and routes, moves logits by up to 2.3e-2 and states by up to 2.7e-2 here,
# so the comparison allows twice that (the 2e-2 of the small-shape tests is
# below this model's rounding-noise floor at full depth).
TOL = 5e-2
STATE_TOL = 5e-2
CFG = synth.FULL


@pytest.fixture(scope="module")
def plain():
    log("[full] weights (seed 0, draft seed 1)")
    w = synth.make_weights(CFG, 0, 1)
    model = Model(CFG, w, 16, 2048 + 64, 3)
    yield w, model, oracle.Oracle(CFG, w)
    model.close()


def _replay_steps(orc, s, sts, K, n_steps, graph=True):
    stats = replay.new_stats()
    if graph:
        s.capture()
    for i in range(n_steps):
        if graph:
            s.replay()
        else:
            s.step()
        recs = step_records(s)
        for b, st in sts.items():
            replay.replay_step(orc, st, K, recs[b], stats, TOL, state_tol=STATE_TOL)
        log(f"  step {i}: m = {[recs[b]['m'] for b in sts]}")
    assert s.status() == 0
    for b, st in sts.items():
        assert int(s.kv_len[b]) == st.kv_len
    return stats


def _synthetic_case(w, model, orc, B, lo, hi, seed, n_steps):
    K = 3
    ctx = synth.context_lengths(B, lo, hi, seed)
    seqs = sorted({int(np.argmin(ctx)), int(np.argmax(ctx)), B // 3})
    log(f"[full B={B}] ctx {int(ctx.min())}..{int(ctx.max())}, checking sequences {seqs}")
    kv, dkv, hid, pend = synthetic_context(CFG, B, ctx, seqs)
    s = Session(model, B, K, n_steps * (K + 1) + 4, record=True)
    load_synthetic(s, CFG, ctx, kv, dkv, hid, pend)
    cap = int(ctx.max()) + n_steps * (K + 1) + 8
    sts = {b: oracle_synthetic_state(orc, CFG, b, int(ctx[b]), cap, kv, dkv, hid, pend)
           for b in seqs}
    stats = _replay_steps(orc, s, sts, K, n_steps)
    log(f"[full B={B}] {n_steps} steps ok, followed near-ties: {stats}")


def test_full_shape_batch1_prefill_and_steps(plain):
    w, model, orc = plain
    K, n_vis, n_txt, n_steps = 3, 256, 512, 4
    tok, vis = prefix_inputs(CFG, 1, n_vis, n_txt)
    log("[full B=1] GPU prefill of 768 rows")
    s = gpu_prefill(model, 1, K, tok, vis, n_steps * (K + 1) + 4, prefill_rows=64)
    assert s.status() == 0
    log("[full B=1] oracle prefill")
    st = oracle_prefill(orc, CFG, tok[0], vis[0], n_vis + n_txt + n_steps * (K + 1) + 8,
                        1 << 30, routes=s.prefill_routes.cpu().numpy()[:, 0])
    log(f"[full B=1] prefill routes followed at near-ties: {st.prefill_routes_followed}")
    t = replay.check_token(st.last_logits, st.pending, int(s.pending[0]), "prefill token",
                           replay.new_stats())
    if t != st.pending:
        st.pending = t
        st.next_tok[0] = t
        st.out[0] = t
    np.testing.assert_allclose(s.hid.cpu().numpy()[0, 0], st.hid[0], rtol=TOL, atol=STATE_TOL)
    stats = _replay_steps(orc, s, {0: st}, K, n_steps)
    log(f"[full B=1] {n_steps} steps ok, followed near-ties: {stats}")


def test_full_shape_batch1_spec_equals_greedy_bitwise(plain):
    """Losslessness on the GPU at full shape, bit for bit: with up to 16 rows
    a row's result does not depend on the other rows of its verify pass (the
    MoE down sums in exact fixed point), so speculative decoding with K = 1
    and 3 emits exactly the tokens of plain greedy decoding (K = 0) and
    writes the same verifier K/V."""
    w, model, orc = plain
    n_vis, n_txt, n_new = 256, 512, 48
    tok, vis = prefix_inputs(CFG, 1, n_vis, n_txt)
    outs, kvs = {}, {}
    for K in (0, 1, 3):
        s = gpu_prefill(model, 1, K, tok, vis, n_new, record=False, prefill_rows=64)
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
    for K in (1, 3):
        assert outs[K] == outs[0]
        assert torch.equal(kvs[K][1][..., :n, :], kvs[0][1][..., :n, :])


def test_full_shape_batch4_sixteen_rows_sampled_sequences(plain):
    """Batch 4: 16 verify rows, one full row group -- the streaming MoE
    gate/up stages 16 rows of 1280 (beyond its first 1024 16-byte chunks
    per block) and the RMSNorm prologues take four rows per wave."""
    w, model, orc = plain
    _synthetic_case(w, model, orc, 4, 512, 1024, 5, 3)


def test_full_shape_batch16_sampled_sequences(plain):
    w, model, orc = plain
    _synthetic_case(w, model, orc, 16, 1024, 2048, 2, 3)


def test_full_shape_batch64_zipf_sampled_sequences():
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
        _synthetic_case(w, model, oracle.Oracle(CFG, w), 1, 30000, 30000, 7, 2)
    finally:
        model.close()
        torch.cuda.empty_cache()

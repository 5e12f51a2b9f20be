"""Pins of the CPU oracle against facts fixed by the paper and by the
mathematics: closed forms, special cases, brute force on tiny inputs,
losslessness and the acceptance rule.  None of these re-types the
oracle's own code path."""
import copy
import itertools
import json
import os

import numpy as np
import pytest

import oracle
import synth
from tests.bruteforce import Ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _model(name, **kw):
    cfg = synth.CONFIGS[name]
    w = synth.make_weights(cfg, 0, 1, **kw)
    return cfg, w, oracle.Oracle(cfg, w)


# ---------------------------------------------------------------- blocks

def test_bf16_round_ties_to_even():
    assert oracle.bf16_round(1.0 + 2.0 ** -8) == 1.0               # tie -> even (down)
    assert oracle.bf16_round(1.0 + 3 * 2.0 ** -8) == 1.0 + 2 ** -6   # tie -> even (up)
    assert oracle.bf16_round(1.0 + 2.0 ** -8 + 2.0 ** -20) == 1.0 + 2 ** -7
    assert oracle.bf16_round(-2.5) == -2.5


def test_rmsnorm_closed_forms():
    x = np.array([3.0, 4.0], np.float32)
    out = oracle.rmsnorm(x, np.ones(2), eps=0.0)
    np.testing.assert_allclose(out, x / np.sqrt(12.5), rtol=1e-7)
    c = np.full(64, -0.37, np.float32)
    g = np.linspace(0.5, 2.0, 64).astype(np.float32)
    np.testing.assert_allclose(oracle.rmsnorm(c, g, eps=0.0), -g, rtol=1e-6)
    # scale invariance
    r = np.random.default_rng(0).standard_normal(256).astype(np.float32)
    np.testing.assert_allclose(oracle.rmsnorm(r, g.repeat(4)[:256], 0.0),
                               oracle.rmsnorm(8 * r, g.repeat(4)[:256], 0.0), rtol=1e-6)


def test_rope_is_a_complex_rotation():
    rng = np.random.default_rng(1)
    dh, theta = 64, 1e4
    x = rng.standard_normal(dh).astype(np.float32)
    np.testing.assert_array_equal(oracle.rope(x, 0, theta), x)          # position 0
    for pos in (1, 17, 4095):
        got = oracle.rope(x, pos, theta)
        inv = theta ** (-2.0 * np.arange(dh // 2) / dh)
        z = (x[:32] + 1j * x[32:]) * np.exp(1j * pos * inv)
        np.testing.assert_allclose(got, np.concatenate([z.real, z.imag]), rtol=1e-5, atol=1e-6)
        assert abs(np.linalg.norm(got) - np.linalg.norm(x)) < 1e-5 * np.linalg.norm(x)
    # scores depend only on the relative position
    q = rng.standard_normal(dh).astype(np.float32)
    k = rng.standard_normal(dh).astype(np.float32)
    s1 = np.dot(oracle.rope(q, 100, theta), oracle.rope(k, 93, theta))
    s2 = np.dot(oracle.rope(q, 2007, theta), oracle.rope(k, 2000, theta))
    assert abs(s1 - s2) < 1e-4


def test_attention_special_cases():
    rng = np.random.default_rng(2)
    dh = 128
    q = rng.standard_normal(dh).astype(np.float32)
    K = rng.standard_normal((1, dh)).astype(np.float32)
    V = rng.standard_normal((1, dh)).astype(np.float32)
    np.testing.assert_allclose(oracle.attend(q, K, V), V[0], rtol=1e-7)     # one key -> v
    K = np.tile(rng.standard_normal(dh).astype(np.float32), (9, 1))
    V = rng.standard_normal((9, dh)).astype(np.float32)
    np.testing.assert_allclose(oracle.attend(q, K, V), V.mean(0), rtol=1e-5, atol=1e-6)
    K = rng.standard_normal((50, dh)).astype(np.float32)
    s = K.astype(np.float64) @ q / np.sqrt(dh)
    p = np.exp(s - s.max())
    np.testing.assert_allclose(oracle.attend(q, K, V := rng.standard_normal((50, dh)).astype(np.float32)),
                               (p / p.sum()) @ V, rtol=1e-5, atol=1e-6)


def test_router_uniform_logits_special_case():
    cfg, w, _ = _model("tinyu")
    w["router"] = np.zeros_like(w["router"])
    orc = oracle.Oracle(cfg, w)
    y = synth.normal(3, 3, (cfg.hidden,))
    lg, pr, tk, gap = orc.router(0, y)
    assert np.all(lg == 0)
    np.testing.assert_allclose(pr, 1.0 / cfg.n_routed, rtol=1e-7)
    assert tk.tolist() == list(range(cfg.top_k))      # ties go to the lower id
    assert gap == 0.0


@pytest.mark.parametrize("name,zipf", [("tinyu", 0.0), ("tinyb", 0.0), ("mid", 1.1)])
def test_moe_equals_bruteforce_over_all_experts(name, zipf):
    cfg, w, orc = _model(name, gain_jitter=0.1, zipf_s=zipf)
    ref = Ref(cfg, w)
    h = synth.normal(5, 5, (12, cfg.hidden))
    got, sel, rw, gap = orc.moe_sublayer(1, h)
    want, sel_ref, lg = ref.moe_block(h.astype(np.float64), 1)
    ok = gap > oracle.ROUTE_TOL
    assert ok.sum() >= 10
    assert np.array_equal(np.sort(sel[ok], 1), np.sort(sel_ref[ok], 1))
    tol = 2e-2 if cfg.dtype == "bf16" else 1e-5
    np.testing.assert_allclose(got[ok], want[ok], rtol=tol, atol=tol * 0.05)
    # gate weights are the softmax over all experts, not renormalised
    np.testing.assert_allclose(rw.sum(1) <= 1.0 + 1e-6, True)


def test_shared_experts_equal_one_wide_swiglu():
    cfg, w, _ = _model("tinyb")
    for key in ("exp_gu", "exp_down"):
        w[key] = np.zeros_like(w[key])          # routed experts contribute nothing
    orc = oracle.Oracle(cfg, w)
    ref = Ref(cfg, w)
    h = synth.normal(6, 6, (5, cfg.hidden))
    got, *_ = orc.moe_sublayer(0, h)
    y = ref.inp(ref.rms(h.astype(np.float64), ref.W("ffn_norm", 0)))
    S, I = cfg.n_shared, cfg.moe_inter
    gu = ref.W("sh_gu", 0)
    wide = ref.swiglu(y, gu[:S * I], gu[S * I:], ref.W("sh_down", 0))   # one 2I-wide SwiGLU
    np.testing.assert_allclose(got, h + wide, rtol=1e-2, atol=2e-4)


# ---------------------------------------------------------------- whole model

def _prefix(cfg, nv, nt):
    return synth.vision_prefix(cfg, nv), synth.text_tokens(cfg, nt)


@pytest.mark.parametrize("name", ["tinyu", "tinyb"])
def test_verifier_incremental_equals_full_sequence_bruteforce(name):
    """Prefill in two chunks plus row-by-row decode (KV cache) versus one
    causal pass over the whole sequence with dense experts."""
    cfg, w, orc = _model(name, gain_jitter=0.1)
    ref = Ref(cfg, w)
    vis, txt = _prefix(cfg, 8, 6)
    P = 14
    tok = np.concatenate([np.full(8, -1, np.int32), txt])
    emb = np.zeros((P, cfg.hidden), cfg.wdtype)
    emb[:8] = vis
    kv = orc.new_kv(64)
    r1 = orc.verify_rows(kv, tok[:9], np.arange(9), emb=emb[:9], want_routes=True)
    r2 = orc.verify_rows(kv, tok[9:], np.arange(9, P), emb=emb[9:], want_routes=True)
    extra = [int(t) for t in synth.text_tokens(cfg, 4, seed=99)]
    rows = [orc.verify_rows(kv, [t], [P + i], want_logits=True, want_routes=True)
            for i, t in enumerate(extra)]
    b = np.concatenate([r1["b"], r2["b"]] + [r["b"] for r in rows])
    full_tok = np.concatenate([tok, extra]).astype(np.int32)
    full_emb = np.zeros((P + 4, cfg.hidden), cfg.wdtype)
    full_emb[:P] = emb
    b_ref, lg_ref, routes_ref = ref.verifier(full_tok, full_emb)
    tol = 2e-2 if cfg.dtype == "bf16" else 1e-4
    np.testing.assert_allclose(b, b_ref, rtol=tol, atol=tol)
    for i, r in enumerate(rows):
        np.testing.assert_allclose(r["logits"][0], lg_ref[P + i], rtol=tol, atol=tol)
        if r["margin"][0] > oracle.ARGMAX_TOL:
            assert r["amax"][0] == int(np.argmax(lg_ref[P + i]))
    gaps = np.concatenate([r1["route_gap"], r2["route_gap"]] + [r["route_gap"] for r in rows], 1)
    idx = np.concatenate([r1["route_idx"], r2["route_idx"]] + [r["route_idx"] for r in rows], 1)
    ok = gaps > oracle.ROUTE_TOL
    assert np.array_equal(np.sort(idx[ok], -1), np.sort(routes_ref[ok], -1))


def test_rows_are_batch_invariant_bitwise():
    cfg, w, orc = _model("tinyb")
    vis, txt = _prefix(cfg, 4, 8)
    tok = np.concatenate([np.full(4, -1, np.int32), txt])
    emb = np.zeros((12, cfg.hidden), cfg.wdtype)
    emb[:4] = vis
    kv1, kv2 = orc.new_kv(32), orc.new_kv(32)
    a = orc.verify_rows(kv1, tok, np.arange(12), emb=emb, want_logits=True)
    bs = [orc.verify_rows(kv2, tok[i:i + 1], [i], emb=emb[i:i + 1], want_logits=True)
          for i in range(12)]
    assert np.array_equal(a["b"], np.concatenate([r["b"] for r in bs]))
    assert np.array_equal(a["logits"], np.concatenate([r["logits"] for r in bs]))
    assert np.array_equal(kv1, kv2)


@pytest.mark.parametrize("name", ["tinyu", "tinyb"])
def test_draft_rows_equal_parallel_grid_bruteforce(name):
    """Depth-1 draft rows run in parallel over the training grid equal the
    same rows run one at a time against the draft KV cache."""
    cfg, w, orc = _model(name, gain_jitter=0.1)
    ref = Ref(cfg, w)
    n = 10
    toks = synth.text_tokens(cfg, n, seed=21)
    a = synth.normal(22, 1, (n, cfg.hidden))
    u_ref, lg_ref = ref.draft(toks, None, a.astype(np.float64), np.arange(n))
    dkv1 = orc.new_dkv(32)
    par = orc.draft_rows(dkv1, toks, a, np.arange(n), want_logits=True)
    dkv2 = orc.new_dkv(32)
    seq = [orc.draft_rows(dkv2, toks[i:i + 1], a[i:i + 1], [i], want_logits=True) for i in range(n)]
    assert np.array_equal(par["u"], np.concatenate([s["u"] for s in seq]))
    assert np.array_equal(dkv1, dkv2)
    tol = 2e-2 if cfg.dtype == "bf16" else 1e-4
    np.testing.assert_allclose(par["u"], u_ref, rtol=tol, atol=tol)
    np.testing.assert_allclose(par["logits"], lg_ref, rtol=tol, atol=tol)


# ---------------------------------------------------------------- acceptance

def test_acceptance_rule_exhaustive():
    """Every draft/verify pattern over a 3-token vocabulary with K = 3."""
    V, K = 3, 3
    for dr in itertools.product(range(V), repeat=K):
        for vf in itertools.product(range(V), repeat=K + 1):
            m, commit = oracle.accept(dr, vf)
            # longest equality prefix
            want = 0
            while want < K and dr[want] == vf[want]:
                want += 1
            assert m == want
            assert commit == list(dr[:m]) + [vf[m]]
            # the committed tokens are the verifier's own greedy tokens:
            # accepted drafts equal v_1..v_m and the last is v_{m+1}
            assert commit == list(vf[:m + 1])
    assert oracle.accept([], [5]) == (0, [5])                    # K = 0


# ---------------------------------------------------------------- losslessness

def _start(name, nv=16, nt=8, cap=128, **kw):
    cfg, w, orc = _model(name, **kw)
    vis, txt = _prefix(cfg, nv, nt)
    st = oracle.prefill(orc, cap, vis, txt)
    return cfg, orc, st


@pytest.mark.parametrize("name", ["tiny", "tinyu", "tinyb"])
def test_speculative_equals_greedy_bitwise(name):
    cfg, orc, st = _start(name)
    ar_st = copy.deepcopy(st)
    ar = oracle.ar_decode(orc, ar_st, 24)
    for K in (0, 1, 3):
        s = copy.deepcopy(st)
        out, steps = oracle.spec_decode(orc, s, K, 24)
        assert out == ar
        n = s.kv_len
        assert np.array_equal(s.kv[:, :, :, :n], ar_st.kv[:, :, :, :n])
        if K == 0:
            assert all(x["m"] == 0 for x in steps) and len(steps) == 23


@pytest.mark.parametrize("name", ["tinyu", "tinyb"])
def test_forced_acceptance_hits_every_m_and_stays_lossless(name):
    """Drafts overwritten from the greedy trajectory: the first m* drafts
    are the greedy tokens, the next one is wrong; then m == m* exactly and
    the output is the greedy output."""
    cfg, orc, st = _start(name)
    K, n_new = 3, 40
    traj = oracle.ar_decode(orc, copy.deepcopy(st), n_new + K + 2)
    ms = [int(x) for x in synth.uniform_int(13, 70, 64, 0, K + 1)]

    def forced(i, s):
        base = len(s.out)                  # traj[base] is the token after pending
        m_star = ms[i % len(ms)]
        d = [traj[base + t] for t in range(K)]
        if m_star < K:
            d[m_star] = (d[m_star] + 1) % cfg.vocab
        return d

    s = copy.deepcopy(st)
    out, steps = oracle.spec_decode(orc, s, K, n_new, forced_fn=forced)
    assert out == traj[:n_new]
    got = [x["m"] for x in steps]
    assert got[:-1] == [ms[i % len(ms)] for i in range(len(got) - 1)]
    assert set(got) == set(range(K + 1))


def test_draft_chain_positions_follow_the_state_shift():
    """The chain that starts at row j = kv_len - 1 writes its depth-k draft
    row at p = j + k - 1; the catch-up rows are the committed rows."""
    cfg, orc, st = _start("tinyu")
    K = 3
    j = st.kv_len - 1
    before = st.dkv.copy()
    oracle.draft_chain(orc, st, K)
    touched = sorted(set(np.nonzero(np.any(st.dkv != before, axis=(0, 1, 3)))[0].tolist()))
    assert touched == [j + k - 1 for k in range(1, K + 1)]
    assert st.draft_len == j + 1
    # a step that accepts m drafts catches up m + 1 rows from the old length
    cfg, orc, st = _start("tinyu")
    traj = oracle.ar_decode(orc, copy.deepcopy(st), 12)
    old = st.kv_len
    info = oracle.spec_step(orc, st, K, forced=[traj[1], traj[2], (traj[3] + 1) % cfg.vocab])
    assert info["m"] == 2 and info["commit"] == traj[1:4]
    assert (st.n_rows, st.row_pos, st.kv_len) == (3, old, old + 3)
    assert st.next_tok.tolist() == traj[1:4] and st.pending == traj[3]


# ---------------------------------------------------------------- shapes, metrics

def test_full_shape_parameter_counts():
    """Table 'Model specification': about 3B total and 570M active decoder
    parameters (all 12 layers MoE; LM head counted, embedding not)."""
    cfg = synth.FULL
    shp = synth.weight_shapes(cfg)
    size = {k: int(np.prod(v)) for k, v in shp.items()}
    dec = [k for k in size if not k.startswith("d_")]
    total = sum(size[k] for k in dec)
    per_expert = 3 * cfg.hidden * cfg.moe_inter
    active = (total - size["embed"] - cfg.n_layers * (cfg.n_routed - cfg.top_k) * per_expert)
    assert 2.9e9 < total < 3.3e9, total
    assert 550e6 < active < 600e6, active


def test_efficiency_table_arithmetic():
    from paper_2609_03181_amd import metrics
    t = json.load(open(os.path.join(GOLDEN, "speculative_efficiency_table.json")))
    base = {r["mode"]: r["tok_s"] for r in t["rows"] if r["k"] == 0}
    for r in t["rows"]:
        if r["k"] == 0:
            continue
        S = metrics.speedup(r["tok_s"], base[r["mode"]])
        assert abs(S - r["S"]) <= 0.006
        assert abs(metrics.acceptance_rate(r["tau"], r["k"]) * 100 - r["acc_pct"]) <= 0.5 / r["k"] + 0.06
        assert abs(metrics.step_cost(r["tau"], S) - r["c"]) <= 0.006
    for mode, a in t["conditional_acceptance"].items():
        tau3 = [r["tau"] for r in t["rows"] if r["mode"] == mode and r["k"] == 3][0]
        assert abs(metrics.tau_from_conditional(a) - tau3) <= 0.006
    assert abs(base["graph"] / base["eager"] - t["graph_over_eager_k0"]) <= 0.006
    assert metrics.tau_from_accept_lengths([0, 3, 2]) == 8 / 3
    assert metrics.conditional_acceptance([0, 1, 3, 3], 3) == [0.75, 2 / 3, 1.0]


def test_argmax_ties_go_to_the_lowest_token_id():
    """A copy of the winning vocabulary row gives an exactly equal top
    logit (tied head); the greedy token must be the lower of the two ids."""
    cfg, w, orc = _model("tiny")
    inp = 11
    top = int(orc.verify_rows(orc.new_kv(8), [inp], [0])["amax"][0])
    for other in (top + 1 if top + 1 != inp else top + 2, max(top - 1, 0)):
        if other in (top, inp):
            continue
        w2 = dict(w)
        w2["embed"] = w["embed"].copy()
        w2["embed"][other] = w["embed"][top]
        r = oracle.Oracle(cfg, w2).verify_rows(orc.new_kv(8), [inp], [0], want_logits=True)
        lg = r["logits"][0]
        assert lg[other] == lg[top] == lg.max()
        assert r["amax"][0] == min(top, other) and r["margin"][0] == 0.0


def test_bf16_models_store_bf16_kv_and_inputs():
    """bf16 models keep the KV cache in bf16: every cached value is a
    bf16 number (its low 16 bits are zero)."""
    cfg, orc, st = _start("tinyb")
    for arr in (st.kv[:, :, :, :st.kv_len], st.dkv[:, :, :st.draft_len]):
        bits = np.ascontiguousarray(arr).view(np.uint32)
        assert np.all((bits & 0xFFFF) == 0)
        assert np.any(bits != 0)


@pytest.mark.parametrize("name", ["tinyu", "tinyb"])
def test_layer_by_layer_equals_whole_model_bitwise(name):
    """verify_layer over every layer, then head, gives exactly what one
    verify_rows call gives (the per-layer entry is the same computation cut
    at the layer boundaries), for a prefix call and then single rows."""
    cfg, w, orc = _model(name, gain_jitter=0.1)
    vis, txt = _prefix(cfg, 5, 7)
    P = 12
    tok = np.concatenate([np.full(5, -1, np.int32), txt])
    emb = np.zeros((P, cfg.hidden), cfg.wdtype)
    emb[:5] = vis
    kv_a, kv_b = orc.new_kv(32), orc.new_kv(32)
    calls = [(tok, emb, np.arange(P))] + [([int(t)], None, [P + i])
                                          for i, t in enumerate(synth.text_tokens(cfg, 3, seed=7))]
    E = orc.w["embed"]
    for t, e, pos in calls:
        whole = orc.verify_rows(kv_a, t, pos, emb=e, want_logits=True, want_routes=True)
        rows = [E[int(x)] if x >= 0 else e[r] for r, x in enumerate(t)]
        h = np.stack(rows)
        h = synth.bf16_bits_to_f32(h) if h.dtype == np.uint16 else h.astype(np.float32)
        for l in range(cfg.n_layers):
            r = orc.verify_layer(l, kv_b[l], h, pos)
            assert np.array_equal(r["route_idx"], whole["route_idx"][l])
            assert np.array_equal(r["route_gap"], whole["route_gap"][l])
            h = r["h"]
        hd = orc.head(h)
        assert np.array_equal(hd["b"], whole["b"])
        assert np.array_equal(hd["logits"], whole["logits"])
        assert np.array_equal(hd["amax"], whole["amax"])
        assert np.array_equal(kv_a, kv_b)

"""Pins of the oracle's draft-head objective (oracle/objective.py) against
what the paper and the mathematics fix, not against itself:

* the per-row CE and KL(Q||P) against scipy's log-softmax and relative
  entropy, and closed forms (uniform P: CE = log V; P = Q: KL = 0; a
  two-point pair);
* alpha_k of Eq. objective written out for K = 1, 2, 3 (beta = 0.6);
* the training grid's diagonal against the inference-time draft chain
  (Figure "FastMTP state-shift alignment": the chain that starts at the
  last prompt row j, drafting the true tokens, is the grid's diagonal
  p = j + k - 1, bit for bit);
* prompt rows keep their base state at every depth (their outputs are the
  same at every depth) and are not in the expectations."""
import numpy as np
import pytest
import scipy.special
import scipy.stats

import oracle
import synth
from oracle import objective as obj


def test_depth_weights_written_out():
    assert np.allclose(obj.depth_weights(1), [1.0])
    assert np.allclose(obj.depth_weights(2), [1 / 1.6, 0.6 / 1.6])
    assert np.allclose(obj.depth_weights(3), [1 / 1.96, 0.6 / 1.96, 0.36 / 1.96])
    assert abs(obj.depth_weights(7).sum() - 1.0) < 1e-15


def test_row_terms_against_scipy():
    rng = np.random.default_rng(3)
    n, V, H = 5, 97, 16
    lp = rng.normal(0, 3, (n, V))
    lq = rng.normal(0, 3, (n, V))
    u, b = rng.normal(size=(n, H)), rng.normal(size=(n, H))
    tgt = rng.integers(0, V, n)
    t = obj.row_terms(lp, lq, u, b, tgt)
    logp = scipy.special.log_softmax(lp, axis=1)
    q = scipy.special.softmax(lq, axis=1)
    p = scipy.special.softmax(lp, axis=1)
    assert np.allclose(t[:, 0], -logp[np.arange(n), tgt], rtol=1e-12, atol=1e-12)
    assert np.allclose(t[:, 1], [scipy.stats.entropy(q[i], p[i]) for i in range(n)], rtol=1e-10,
                       atol=1e-12)
    assert np.allclose(t[:, 2], np.linalg.norm(u - b, axis=1) ** 2, rtol=1e-12)


def test_row_terms_closed_forms():
    V = 50
    l0 = np.zeros((1, V))
    t = obj.row_terms(l0, l0, np.zeros((1, 4)), np.ones((1, 4)), np.array([7]))
    assert abs(t[0, 0] - np.log(V)) < 1e-12   # uniform P
    assert abs(t[0, 1]) < 1e-14               # P = Q
    assert abs(t[0, 2] - 4.0) < 1e-14
    # two-point distributions: q = (0.3, 0.7), p = (0.6, 0.4)
    lq = np.log(np.array([[0.3, 0.7]]))
    lp = np.log(np.array([[0.6, 0.4]]))
    t = obj.row_terms(lp, lq, np.zeros((1, 1)), np.zeros((1, 1)), np.array([1]))
    kl = 0.3 * np.log(0.3 / 0.6) + 0.7 * np.log(0.7 / 0.4)
    assert abs(t[0, 1] - kl) < 1e-12 and abs(t[0, 0] + np.log(0.4)) < 1e-12


def test_combine_written_out():
    means = np.array([[2.0, 0.5, 1.0], [3.0, 0.25, 2.0], [4.0, 1.0, 4.0]])
    a = np.array([1.0, 0.6, 0.36]) / 1.96
    want = (0.85 * (a * means[:, 0]).sum() + 0.45 * (a * means[:, 1]).sum()
            + 0.45 * (a * means[:, 2]).sum())
    assert abs(obj.combine(means) - want) < 1e-13
    assert abs(obj.combine(means[:1]) - (0.85 * 2 + 0.45 * 0.5 + 0.45 * 1.0)) < 1e-13


def _sequence(cfg, n_vis, n_prompt_txt, n_resp, seed=30):
    tok = np.concatenate([np.full(n_vis, -1, np.int32),
                          synth.text_tokens(cfg, n_prompt_txt + n_resp, seed=seed)])
    emb = np.zeros((len(tok), cfg.hidden), cfg.wdtype)
    if n_vis:
        emb[:n_vis] = synth.vision_prefix(cfg, n_vis, seed=seed + 1)
    return tok, emb


def _states(orc, tok, emb):
    """The verifier's post-norm states b_p of every row of the sequence."""
    kv = orc.new_kv(len(tok))
    return orc.verify_rows(kv, tok, np.arange(len(tok)), emb=emb)["b"]


@pytest.fixture(scope="module")
def grid():
    cfg = synth.CONFIGS["tinyb"]
    w = synth.make_weights(cfg, 0, 1, gain_jitter=0.1)
    orc = oracle.Oracle(cfg, w)
    tok, emb = _sequence(cfg, 4, 5, 9)
    b = _states(orc, tok, emb)
    n_prompt = 9
    return cfg, orc, tok, emb, b, n_prompt, obj.forward(orc, tok, emb, b, n_prompt, 3)


def test_diagonal_is_the_inference_chain(grid):
    """Depth k of the chain that starts at the last prompt row j sits at
    grid row j + k - 1: the same state, input token, position and attended
    cache rows, hence the same output bit for bit."""
    cfg, orc, tok, emb, b, n_prompt, r = grid
    j = n_prompt - 1
    dkv = orc.new_dkv(len(tok))
    # committed cache of the prompt in base form (state b_p, input row p+1)
    orc.draft_rows(dkv, tok[1:j + 1], b[:j], np.arange(j), emb=emb[1:j + 1])
    # the chain: catch-up row j, then depths 2..3 drafting the true tokens
    hm = np.ones(1, np.uint8)
    c = orc.draft_rows(dkv, tok[j + 1:j + 2], b[j:j + 1], [j], head_mask=hm, want_logits=True)
    chain_u, chain_l = [c["u"][0]], [c["logits"][0]]
    for d in range(2, 4):
        p = j + d - 1
        c = orc.draft_rows(dkv, tok[p + 1:p + 2], chain_u[-1][None, :], [p], head_mask=hm,
                           want_logits=True)
        chain_u.append(c["u"][0])
        chain_l.append(c["logits"][0])
    for k in range(1, 4):
        assert np.array_equal(r["u"][k - 1][j + k - 1], chain_u[k - 1]), k
        assert np.array_equal(r["logits"][k - 1][j + k - 1], chain_l[k - 1]), k


def test_prompt_rows_keep_their_base_state(grid):
    cfg, orc, tok, emb, b, n_prompt, r = grid
    for k in (2, 3):
        assert np.array_equal(r["u"][k - 1][:n_prompt], r["u"][0][:n_prompt])
        # response rows do shift (the test would not see a missing shift otherwise)
        assert not np.array_equal(r["u"][k - 1][n_prompt:], r["u"][0][n_prompt:])


def test_expectations_run_over_response_rows_with_targets(grid):
    cfg, orc, tok, emb, b, n_prompt, r = grid
    T = len(tok)
    rows = obj.loss_rows(T, n_prompt)
    assert rows[0] == n_prompt and rows[-1] == T - 3
    mask = np.zeros(T - 1, bool)
    mask[rows] = True
    assert not r["terms"][:, ~mask].any()
    assert np.allclose(r["means"], r["terms"][:, rows].mean(axis=1), rtol=0, atol=0)
    # the targets are the tokens two rows ahead: a row's CE equals -log P(x_{p+2})
    p = rows[2]
    lp = scipy.special.log_softmax(r["logits"][0][p].astype(np.float64))
    assert abs(r["terms"][0, p, 0] + lp[tok[p + 2]]) < 1e-9
    assert abs(r["loss"] - obj.combine(r["means"])) < 1e-15


def test_rejects_a_sequence_without_loss_rows(grid):
    cfg, orc, tok, emb, b, n_prompt, r = grid
    with pytest.raises(ValueError):
        obj.forward(orc, tok, emb, b, len(tok) - 2, 1)
    with pytest.raises(ValueError):
        obj.forward(orc, tok, emb, b, 0, 1)

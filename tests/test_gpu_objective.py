"""The draft-head objective forward on the GPU (mtp_objective) against the
oracle (oracle/objective.py) on the same sequence and the same verifier
states b.

Layer-local, as the decode-step checks: the oracle runs depth k from the
GPU's own depth k-1 outputs (u_in), so only one depth's rounding separates
the two.  Then
* u^(k) element-wise at the measured draft-state tolerance (the drift of
  the base-form draft pass over every row, tests/golden/route_drift.json);
* each row's CE, KL(Q||P) and MSE within a bound derived from the logit and
  state tolerances and the oracle's own values (below);
* the per-depth means and L within the mean of the row bounds.
The end-to-end difference (the oracle's own chain) is reported.

Bounds, with |d l| <= t (1 + |l|) for logits at tolerance t and
|d u_i| <= t_u (1 + |u_i|):
  CE = lse(l_P) - l_P[x]:          |dCE| <= 2 t_P (1 + max|l_P|)
  KL = sum_v q_v (l_Qv - l_Pv) - lse(l_Q) + lse(l_P):
       dKL/dl_P = p - q,  dKL/dl_Q = q (l_Q - l_P - KL)
                                   |dKL| <= 2 t_P (1 + max|l_P|)
                                          + t_Q (1 + max|l_Q|) sum_v q_v |l_Qv - l_Pv - KL|
  MSE = ||u - b||^2:               |dMSE| <= sum_i 2 |u_i - b_i| e_i + e_i^2,
                                   e_i = t_u (1 + |u_i|)."""
import dataclasses

import numpy as np
import pytest
import scipy.special
import torch

import oracle
import synth
from oracle import objective as obj
from paper_2609_03181_amd import _lib
from paper_2609_03181_amd.session import Model
from tests import tolerances
from tests.gpu_util import log, to_dev_storage

pytestmark = pytest.mark.gpu


def _sequence(cfg, n_vis, n_txt, seed=40):
    tok = np.concatenate([np.full(n_vis, -1, np.int32), synth.text_tokens(cfg, n_txt, seed=seed)])
    emb = np.zeros((len(tok), cfg.hidden), cfg.wdtype)
    if n_vis:
        emb[:n_vis] = synth.vision_prefix(cfg, n_vis, seed=seed + 1)
    return tok, emb


def _gpu(model, cfg, tok, emb, b, n_prompt, K):
    T, H = len(tok), cfg.hidden
    wsb = _lib.mtp_objective_workspace_bytes(model.ctx, T)
    ws = torch.zeros(wsb, dtype=torch.uint8, device="cuda")
    dkv = torch.zeros((K, 2, cfg.n_heads, model.max_ctx, cfg.head_dim),
                      dtype=model.storage_dtype, device="cuda")
    tok_d = torch.from_numpy(tok).cuda()
    vis_d = to_dev_storage(emb) if (tok < 0).any() else None
    b_d = torch.from_numpy(np.ascontiguousarray(b, np.float32)).cuda()
    terms = torch.zeros((K, T, 3), dtype=torch.float32, device="cuda")
    u = torch.zeros((K, T, H), dtype=torch.float32, device="cuda")
    loss = torch.zeros(3 * K + 1, dtype=torch.float64, device="cuda")
    p = lambda t: None if t is None else t.data_ptr()
    _lib.mtp_objective(model.ctx, T, n_prompt, K, p(tok_d), p(vis_d), p(b_d), p(dkv), p(terms),
                       p(u), p(loss), p(ws), wsb, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert _lib.mtp_status_read(model.ctx, ws.data_ptr()) == _lib.MTP_OK
    return terms.cpu().numpy(), u.cpu().numpy(), loss.cpu().numpy()


def _bounds(ref, k, rows, t_p, t_q, t_u, b):
    lp = ref["logits"][k][rows].astype(np.float64)
    lq = ref["q_logits"][rows].astype(np.float64)
    kl = ref["terms"][k, rows, 1]
    q = scipy.special.softmax(lq, axis=1)
    ce_b = 2 * t_p * (1 + np.abs(lp).max(axis=1))
    kl_b = ce_b + t_q * (1 + np.abs(lq).max(axis=1)) * (q * np.abs(lq - lp - kl[:, None])).sum(1)
    u = ref["u"][k][rows].astype(np.float64)
    e = t_u * (1 + np.abs(u))
    mse_b = (2 * np.abs(u - b[rows + 1]) * e + e * e).sum(axis=1)
    return np.stack([ce_b, kl_b, mse_b], axis=1) + 1e-6


def _check(name, n_vis, n_txt, n_prompt, K, vocab=None, **wkw):
    cfg = synth.CONFIGS[name]
    if vocab is not None:
        cfg = dataclasses.replace(cfg, vocab=vocab)
    w = synth.make_weights(cfg, 0, 1, **wkw)
    orc = oracle.Oracle(cfg, w)
    tok, emb = _sequence(cfg, n_vis, n_txt)
    T = len(tok)
    b = orc.verify_rows(orc.new_kv(T), tok, np.arange(T), emb=emb)["b"]
    model = Model(cfg, w, 1, T + 8, 3)
    g_terms, g_u, g_loss = _gpu(model, cfg, tok, emb, b, n_prompt, K)
    model.close()
    tl = tolerances.local_tol(cfg)
    t_u, t_p, t_q = float(tl["draft_u"][0]), float(tl["draft_logits"][0]), float(tl["logits"])
    ref = obj.forward(orc, tok, emb, b, n_prompt, K, u_in=g_u[:, :T - 1])
    rows = obj.loss_rows(T, n_prompt)
    mean_bound = np.zeros((K, 3))
    for k in range(K):
        np.testing.assert_allclose(g_u[k, :T - 1], ref["u"][k], rtol=t_u, atol=t_u,
                                   err_msg=f"{name} u depth {k + 1}")
        assert not g_u[k, T - 1].any()
        bd = _bounds(ref, k, rows, t_p, t_q, t_u, b.astype(np.float64))
        dev = np.abs(g_terms[k, rows] - ref["terms"][k, rows])
        assert (dev <= bd).all(), (name, k + 1, float((dev / bd).max()))
        mask = np.ones(T, bool)
        mask[rows] = False
        assert not g_terms[k, mask].any()
        mean_bound[k] = bd.mean(axis=0)
    g_means = g_loss[:3 * K].reshape(K, 3)
    assert (np.abs(g_means - ref["means"]) <= mean_bound).all(), (g_means, ref["means"])
    a = obj.depth_weights(K)
    l_bound = sum(wt * (a * mean_bound[:, j]).sum() for j, wt in enumerate(obj.WEIGHTS))
    assert abs(g_loss[3 * K] - ref["loss"]) <= l_bound, (g_loss[3 * K], ref["loss"], l_bound)
    e2e = obj.forward(orc, tok, emb, b, n_prompt, K)
    log(f"[objective] {name} T={T} n_prompt={n_prompt} K={K}: L gpu {g_loss[3 * K]:.6f} "
        f"oracle (GPU-fed chain) {ref['loss']:.6f} (bound {l_bound:.2e}); oracle's own chain "
        f"{e2e['loss']:.6f}; per-depth CE/KL/MSE {np.round(g_means, 4).tolist()}")


def test_objective_mid_bf16():
    _check("mid", 8, 40, 16, 3, gain_jitter=0.1)


def test_objective_odd_vocabulary():
    """A vocabulary that is not a multiple of 4 (the loss terms read the
    logit rows with 4-byte loads) nor of 16 (the LM head's last strip is
    ragged)."""
    _check("tinyb", 4, 22, 8, 2, vocab=3001)


def test_objective_tiny_f32_untied():
    _check("tinyu", 6, 26, 10, 3)


def test_objective_one_depth_and_a_short_sequence():
    _check("mid", 0, 6, 2, 1, gain_jitter=0.1)


def test_objective_mid_several_chunks():
    """1,323 draft rows: a 1,280-row pass and a 43-row pass per depth, so
    the states of a chunk's first row and the attended rows of the earlier
    chunk cross the chunk boundary."""
    _check("mid", 16, 1308, 40, 3, gain_jitter=0.1)


def test_objective_full_shape():
    """Full shape: 8 vision rows + 12 prompt tokens + 28 response tokens,
    K = 3 (the draft passes run in one 47-row chunk; LM head on every row)."""
    _check("full", 8, 40, 20, 3)


def test_objective_rejects_bad_arguments():
    cfg = synth.CONFIGS["mid"]
    w = synth.make_weights(cfg, 0, 1)
    model = Model(cfg, w, 1, 40, 3)
    T = 20
    wsb = _lib.mtp_objective_workspace_bytes(model.ctx, T)
    ws = torch.zeros(wsb, dtype=torch.uint8, device="cuda")
    dkv = torch.zeros((2, cfg.n_heads, 40, cfg.head_dim), dtype=model.storage_dtype, device="cuda")
    tok = torch.zeros(T, dtype=torch.int32, device="cuda")
    b = torch.zeros((T, cfg.hidden), dtype=torch.float32, device="cuda")
    loss = torch.zeros(4, dtype=torch.float64, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    for n_prompt, K, nb in ((0, 1, wsb), (T - 2, 1, wsb), (2, 0, wsb), (2, 9, wsb), (2, 1, wsb - 1)):
        with pytest.raises(_lib.MtpError) as e:
            _lib.mtp_objective(model.ctx, T, n_prompt, K, tok.data_ptr(), None, b.data_ptr(),
                               dkv.data_ptr(), None, None, loss.data_ptr(), ws.data_ptr(), nb, st)
        assert e.value.code == _lib.MTP_EINVAL
    assert _lib.mtp_objective_workspace_bytes(model.ctx, 41) == 0  # past max_ctx
    model.close()

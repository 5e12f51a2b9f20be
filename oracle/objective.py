"""Oracle of the FastMTP draft-head objective (forward only).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: imported by
``tests/`` and by the CPU leg of ``bench.py``, never by the GPU library.

Follows Section "Draft-head architecture" (the state-shift equation and
the training grid of positions x depths) and Section "Draft-head
objective" (Eq. draft-loss and Eq. objective).  One sequence of T rows:
row p is token x_p (or a vision row), b_p the verifier's post-norm state
after it (given: the verifier is frozen and its states detached).

* Depth k = 1..K runs the draft block over the rows p = 0..T-2 (row p's
  next input is row p+1) with causal attention among the rows of that
  depth, position p, and state
      a_p^(1) = b_p,
      a_p^(k) = u_{p-1}^(k-1)  (k > 1, response rows),
      a_p^(k) = b_p            (k > 1, prompt rows keep their base state);
  u_p^(k) is the draft output (after the tied final norm) and
  l_p^(k) = W_lm u_p^(k) its logits.
* Loss rows: response rows p (p >= n_prompt) whose target x_{p+2} exists
  (p <= T-3); prompt and padding rows are excluded.
* P_p^(k) = softmax(l_p^(k)), Q_p = softmax(W_lm b_{p+1}) (detached);
      CE_k  = mean_p  -log P_p^(k)(x_{p+2})
      KL_k  = mean_p  KL(Q_p || P_p^(k))
      MSE_k = mean_p  ||u_p^(k) - b_{p+1}||^2
      alpha_k = beta^(k-1) / sum_{r=1..K} beta^(r-1),  beta = 0.6
      L = 0.85 sum_k alpha_k CE_k + 0.45 sum_k alpha_k KL_k
          + 0.45 sum_k alpha_k MSE_k.
The loss arithmetic is float64 (numpy); the draft rows and the logits come
from the C oracle (float64 sums, rounded at the storage points)."""
from __future__ import annotations

import numpy as np

BETA = 0.6
WEIGHTS = (0.85, 0.45, 0.45)  # CE, KL, MSE


def depth_weights(K: int, beta: float = BETA) -> np.ndarray:
    """alpha_k = beta^(k-1) / sum_{r=1..K} beta^(r-1), k = 1..K."""
    p = beta ** np.arange(K, dtype=np.float64)
    return p / p.sum()


def loss_rows(n_rows: int, n_prompt: int) -> np.ndarray:
    """Indices p of the rows the expectations run over."""
    return np.arange(n_prompt, n_rows - 2)


def logsumexp(l: np.ndarray) -> np.ndarray:
    """Row-wise log sum exp (float64)."""
    l = np.asarray(l, np.float64)
    m = l.max(axis=-1, keepdims=True)
    return (m + np.log(np.exp(l - m).sum(axis=-1, keepdims=True)))[..., 0]


def row_terms(p_logits, q_logits, u, b_next, target):
    """Per-row CE, KL(Q||P) and MSE of rows given draft logits p_logits
    [n][V], verifier logits q_logits [n][V] (of b_{p+1}), draft states u
    [n][H], verifier states b_next [n][H] and targets [n]: float64 [n][3]."""
    lp = np.asarray(p_logits, np.float64)
    lq = np.asarray(q_logits, np.float64)
    logp = lp - logsumexp(lp)[:, None]
    logq = lq - logsumexp(lq)[:, None]
    ce = -logp[np.arange(len(target)), target]
    kl = (np.exp(logq) * (logq - logp)).sum(axis=1)
    d = np.asarray(u, np.float64) - np.asarray(b_next, np.float64)
    mse = (d * d).sum(axis=1)
    return np.stack([ce, kl, mse], axis=1)


def combine(means: np.ndarray, beta: float = BETA) -> float:
    """Eq. objective from the per-depth means [K][3] (CE, KL, MSE)."""
    a = depth_weights(means.shape[0], beta)
    return float(sum(wt * (a * means[:, j]).sum() for j, wt in enumerate(WEIGHTS)))


def depth_states(b, u_prev, k: int, n_prompt: int) -> np.ndarray:
    """States a_p^(k) of rows p = 0..T-2 (state-shift equation): b_p at
    depth 1 and on prompt rows, u_{p-1}^(k-1) on response rows after that."""
    T1 = b.shape[0] - 1
    a = np.array(b[:T1], dtype=np.float32, copy=True)
    if k > 1:
        p = np.arange(T1)
        resp = p >= max(n_prompt, 1)
        a[resp] = u_prev[p[resp] - 1]
    return a


def forward(orc, tok, emb, b, n_prompt: int, K: int, beta: float = BETA, u_in=None):
    """The objective of one sequence.  tok [T] (negative: vision row emb[p]),
    emb [T][H] storage dtype or None, b [T][H] the verifier's post-norm
    states.  u_in [K][T-1][H] (optional): the depth outputs to shift into
    the next depth instead of the oracle's own (the layer-local check feeds
    the GPU's).  Returns dict(u [K][T-1][H], logits [K][T-1][V], q_logits
    [T-1][V], terms [K][T-1][3] (zero outside the loss rows), means [K][3],
    loss)."""
    c = orc.cfg
    tok = np.asarray(tok, np.int32)
    T = len(tok)
    if not 1 <= n_prompt <= T - 3:
        raise ValueError("need 1 <= n_prompt <= n_rows - 3")
    b = np.asarray(b, np.float32)
    rows = loss_rows(T, n_prompt)
    q_logits = orc.lm_logits(b[1:])
    us, ls = [], []
    terms = np.zeros((K, T - 1, 3))
    u_prev = None
    for k in range(1, K + 1):
        a = depth_states(b, u_prev, k, n_prompt)
        dkv = orc.new_dkv(T)
        r = orc.draft_rows(dkv, tok[1:], a, np.arange(T - 1),
                           emb=None if emb is None else emb[1:],
                           head_mask=np.ones(T - 1, np.uint8), want_logits=True)
        us.append(r["u"])
        ls.append(r["logits"])
        terms[k - 1, rows] = row_terms(r["logits"][rows], q_logits[rows], r["u"][rows],
                                       b[rows + 1], tok[rows + 2])
        u_prev = r["u"] if u_in is None else np.asarray(u_in[k - 1], np.float32)
    means = terms[:, rows].mean(axis=1)
    return dict(u=np.stack(us), logits=np.stack(ls), q_logits=q_logits, terms=terms,
                means=means, loss=combine(means, beta))

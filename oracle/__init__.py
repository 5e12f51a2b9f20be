"""CPU oracle for the FastMTP greedy speculative-decode step.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by the smoke check and
by the CPU-baseline leg of ``bench.py``; never by the GPU library or its
binding.  It shares no code with the GPU path; only the seeded input
generator (``synth``) feeds both.

The C half (``oracle.c``) evaluates verifier rows and FastMTP draft rows.
This Python half holds the decoding loop written from the paper:

* the state-shift recursion of Section "Draft-head architecture": the
  chain that starts at row j has depth k at row p = j + k - 1, takes the
  state a = b_j at depth 1 and a = u^(k-1) after that, and predicts
  x_{j+k+1};
* greedy verification by the acceptance equation: m is the longest prefix
  on which every draft equals the verifier's greedy token; the step commits
  the m accepted drafts and then the verifier token v_{m+1} (a correction
  on a mismatch, a bonus when all K match); other candidates are dropped;
* the committed-token cache: committed draft rows are kept in base form
  (state b_p, next committed token), so the next step first catches up
  the m+1 rows it just committed.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "_oracle.so")
_lib = None

# Decision tolerances of the oracle's own checks (pins of the oracle
# against brute force): where two correct evaluations that sum in different
# orders may pick different integers.  The parity tests against the GPU
# path take their per-layer routing tolerances from a drift measurement
# (tests/tolerances.py) and pass them to verify_rows.
#   ROUTE_TOL   router k-th vs (k+1)-th logit gap (the gating margin the
#               workload statement fixes);
#   ARGMAX_TOL  top-1 vs top-2 token logit gap.
ROUTE_TOL = 1e-3
ARGMAX_TOL = 0.05


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11",
                               os.path.join(_HERE, "oracle.c"), "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "hidden", "n_heads", "head_dim", "n_routed", "top_k", "n_shared",
        "moe_inter", "draft_inter", "vocab", "tie_lm_head", "bf16")] + [
        ("rope_theta", ctypes.c_double), ("rms_eps", ctypes.c_double)]


_WFIELDS = ("embed", "lm_head", "final_norm", "attn_norm", "ffn_norm", "wqkv", "wo", "router",
            "exp_gu", "exp_down", "sh_gu", "sh_down", "router_bias", "d_enorm", "d_hnorm",
            "d_attn_norm", "d_ffn_norm", "d_eh_proj", "d_wqkv", "d_wo", "d_gu", "d_down")


class _Weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in _WFIELDS]


def _L():
    global _lib
    if _lib is None:
        # MTP_ORACLE_LIB: another build of oracle.c (the planted-mistake
        # check loads deliberately broken copies through it)
        path = os.environ.get("MTP_ORACLE_LIB") or _LIB_PATH
        if path == _LIB_PATH and not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(path)
        vp, i32, f32, dbl = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_double
        lib.orc_verify_rows.argtypes = [vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, vp,
                                        vp, vp, vp, vp, vp, vp, vp, vp, vp]
        lib.orc_verify_rows.restype = i32
        lib.orc_draft_rows.argtypes = [vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        lib.orc_draft_rows.restype = i32
        lib.orc_verify_layer.argtypes = [vp, vp, i32, vp, i32, i32, vp, vp, vp, f32, vp, vp,
                                         vp, vp]
        lib.orc_verify_layer.restype = i32
        lib.orc_head.argtypes = [vp, vp, i32, vp, vp, vp, vp, vp]
        lib.orc_lm_logits.argtypes = [vp, vp, i32, vp, vp]
        lib.orc_rmsnorm.argtypes = [vp, vp, i32, dbl, vp]
        lib.orc_rope.argtypes = [vp, i32, i32, dbl]
        lib.orc_attend.argtypes = [vp, vp, vp, i32, i32, vp]
        lib.orc_router.argtypes = [vp, vp, i32, vp, vp, vp, vp, vp]
        lib.orc_moe_sublayer.argtypes = [vp, vp, i32, i32, vp, vp, vp, vp, vp]
        lib.orc_set_sum32.argtypes = [i32]
        lib.orc_bf16_round.argtypes = [f32]
        lib.orc_bf16_round.restype = f32
        _lib = lib
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def _c(a, dt):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


class Oracle:
    """Model weights plus the row-level entry points of the C oracle."""

    def __init__(self, cfg, weights: dict):
        self.cfg = cfg
        self.w = {k: np.ascontiguousarray(v) for k, v in weights.items()}
        self.dims = _Dims(cfg.n_layers, cfg.hidden, cfg.n_heads, cfg.head_dim, cfg.n_routed,
                          cfg.top_k, cfg.n_shared, cfg.moe_inter, cfg.draft_inter, cfg.vocab,
                          int(cfg.tie_lm_head), int(cfg.dtype == "bf16"), cfg.rope_theta,
                          cfg.rms_eps)
        self.wts = _Weights(*[_p(self.w.get(n)) for n in _WFIELDS])

    # -- storage ---------------------------------------------------------
    def new_kv(self, cap: int) -> np.ndarray:
        c = self.cfg
        return np.zeros((c.n_layers, 2, c.n_heads, cap, c.head_dim), dtype=np.float32)

    def new_dkv(self, cap: int) -> np.ndarray:
        c = self.cfg
        return np.zeros((2, c.n_heads, cap, c.head_dim), dtype=np.float32)

    # -- rows ------------------------------------------------------------
    def verify_rows(self, kv, tok, pos, emb=None, head_mask=None, want_logits=False,
                    want_routes=False, follow_route=None, route_tol=None,
                    want_router_logits=False):
        """follow_route [L][n][k]: routes chosen elsewhere, adopted where
        they are a top-k set of the oracle's logits up to route_tol[l]
        (required with follow_route: per-layer tolerance)."""
        c = self.cfg
        tok = _c(tok, np.int32)
        pos = _c(pos, np.int32)
        n = len(tok)
        emb = _c(emb, c.wdtype)
        hm = None if head_mask is None else _c(head_mask, np.uint8)
        b = np.empty((n, c.hidden), np.float32)
        amax = np.full(n, -1, np.int32)
        margin = np.full(n, np.nan, np.float32)
        logits = np.empty((n, c.vocab), np.float32) if want_logits else None
        ri = rw = rg = None
        if want_routes:
            ri = np.empty((c.n_layers, n, c.top_k), np.int32)
            rw = np.empty((c.n_layers, n, c.top_k), np.float32)
            rg = np.empty((c.n_layers, n), np.float32)
        rl = (np.empty((c.n_layers, n, c.n_routed), np.float32) if want_router_logits
              else None)
        fr = _c(follow_route, np.int32)
        if follow_route is not None and route_tol is None:
            raise ValueError("follow_route needs a per-layer route_tol")
        rt = np.ascontiguousarray(np.broadcast_to(
            np.float32(ROUTE_TOL) if route_tol is None else np.asarray(route_tol, np.float32),
            (c.n_layers,)), np.float32)
        nf = ctypes.c_int(0)
        rc = _L().orc_verify_rows(ctypes.byref(self.dims), ctypes.byref(self.wts), _p(kv),
                                  kv.shape[3], n, _p(tok), _p(emb), _p(pos), _p(fr), _p(rt),
                                  ctypes.byref(nf), _p(b), _p(hm), _p(logits), _p(amax),
                                  _p(margin), _p(ri), _p(rw), _p(rg), _p(rl))
        if rc < 0:
            raise ValueError("oracle: position outside the KV capacity")
        return dict(b=b, amax=amax, margin=margin, logits=logits, route_idx=ri, route_w=rw,
                    route_gap=rg, route_rejected=rc, route_followed=nf.value, router_logits=rl)

    def verify_layer(self, layer, kv_l, h, pos, follow_route=None, route_tol=None):
        """One verifier layer from the layer input h [n][H] (float32) over
        the layer's KV slab kv_l [2][nh][cap][dh] (float32; the rows' K/V
        are written into it).  follow_route [n][k] with route_tol (a
        float): routes adopted at near-ties, as in verify_rows.  Returns the
        layer output and the layer's routing (route_idx [n][k], route_gap
        [n], router_logits [n][E]) and the follow counts."""
        c = self.cfg
        h = np.array(h, dtype=np.float32, copy=True, order="C")
        pos = _c(pos, np.int32)
        n = len(pos)
        assert kv_l.dtype == np.float32 and kv_l.flags.c_contiguous
        if follow_route is not None and route_tol is None:
            raise ValueError("follow_route needs route_tol")
        fr = _c(follow_route, np.int32)
        ri = np.empty((n, c.top_k), np.int32)
        rg = np.empty(n, np.float32)
        rl = np.empty((n, c.n_routed), np.float32)
        nf = ctypes.c_int(0)
        rc = _L().orc_verify_layer(ctypes.byref(self.dims), ctypes.byref(self.wts), layer,
                                   _p(kv_l), kv_l.shape[2], n, _p(pos), _p(h), _p(fr),
                                   float(route_tol or 0.0), ctypes.byref(nf), _p(ri), _p(rg),
                                   _p(rl))
        if rc < 0:
            raise ValueError("oracle: position outside the KV capacity")
        return dict(h=h, route_idx=ri, route_gap=rg, router_logits=rl, route_rejected=rc,
                    route_followed=nf.value)

    def head(self, h):
        """Final norm, LM head and greedy argmax of residual rows h [n][H]."""
        c = self.cfg
        h = _c(h, np.float32)
        n = h.shape[0]
        b = np.empty((n, c.hidden), np.float32)
        logits = np.empty((n, c.vocab), np.float32)
        amax = np.full(n, -1, np.int32)
        margin = np.full(n, np.nan, np.float32)
        _L().orc_head(ctypes.byref(self.dims), ctypes.byref(self.wts), n, _p(h), _p(b),
                      _p(logits), _p(amax), _p(margin))
        return dict(b=b, logits=logits, amax=amax, margin=margin)

    def draft_rows(self, dkv, tok, a, pos, emb=None, head_mask=None, want_logits=False):
        c = self.cfg
        tok = _c(tok, np.int32)
        pos = _c(pos, np.int32)
        a = _c(a, np.float32)
        n = len(tok)
        emb = _c(emb, c.wdtype)
        hm = None if head_mask is None else _c(head_mask, np.uint8)
        u = np.empty((n, c.hidden), np.float32)
        amax = np.full(n, -1, np.int32)
        margin = np.full(n, np.nan, np.float32)
        logits = np.empty((n, c.vocab), np.float32) if want_logits else None
        rc = _L().orc_draft_rows(ctypes.byref(self.dims), ctypes.byref(self.wts), _p(dkv),
                                 dkv.shape[2], n, _p(tok), _p(emb), _p(a), _p(pos), _p(u),
                                 _p(hm), _p(logits), _p(amax), _p(margin))
        if rc < 0:
            raise ValueError("oracle: position outside the draft KV capacity")
        return dict(u=u, amax=amax, margin=margin, logits=logits)

    def lm_logits(self, x):
        """LM-head logits of post-norm rows x [n][H] (no final norm)."""
        c = self.cfg
        x = _c(x, np.float32)
        logits = np.empty((x.shape[0], c.vocab), np.float32)
        _L().orc_lm_logits(ctypes.byref(self.dims), ctypes.byref(self.wts), x.shape[0], _p(x),
                           _p(logits))
        return logits

    # -- building blocks (for the pins) ------------------------------------
    def moe_sublayer(self, layer, h):
        c = self.cfg
        h = _c(h, np.float32)
        n = h.shape[0]
        out = np.empty_like(h)
        ri = np.empty((n, c.top_k), np.int32)
        rw = np.empty((n, c.top_k), np.float32)
        rg = np.empty(n, np.float32)
        _L().orc_moe_sublayer(ctypes.byref(self.dims), ctypes.byref(self.wts), layer, n, _p(h),
                              _p(out), _p(ri), _p(rw), _p(rg))
        return out, ri, rw, rg

    def router(self, layer, y):
        c = self.cfg
        y = _c(y, np.float32)
        lg = np.empty(c.n_routed, np.float32)
        pr = np.empty(c.n_routed, np.float32)
        tk = np.empty(c.top_k, np.int32)
        gap = np.empty(1, np.float32)
        _L().orc_router(ctypes.byref(self.dims), ctypes.byref(self.wts), layer, _p(y), _p(lg),
                        _p(pr), _p(tk), _p(gap))
        return lg, pr, tk, float(gap[0])


def rmsnorm(x, g, eps=1e-6):
    x = _c(x, np.float32)
    g = _c(g, np.float32)
    out = np.empty_like(x)
    _L().orc_rmsnorm(_p(x), _p(g), x.shape[-1], eps, _p(out))
    return out


def rope(x, pos, theta):
    x = np.array(x, dtype=np.float32, copy=True)
    _L().orc_rope(_p(x), x.shape[-1], int(pos), float(theta))
    return x


def attend(q, K, V):
    q, K, V = _c(q, np.float32), _c(K, np.float32), _c(V, np.float32)
    o = np.empty(q.shape[-1], np.float32)
    _L().orc_attend(_p(q), _p(K), _p(V), K.shape[0], q.shape[-1], _p(o))
    return o


def set_sum32(on: bool) -> None:
    """Sensitivity measurement only: weight dot products in float32
    (sequential) instead of float64 while on.  Reference values are always
    computed with it off."""
    _L().orc_set_sum32(int(bool(on)))


def bf16_round(x: float) -> float:
    return float(_L().orc_bf16_round(float(x)))


# ---------------------------------------------------------------------------
# greedy verification (acceptance equation)
# ---------------------------------------------------------------------------

def accept(draft, verify):
    """m = max({0} U {r <= K : draft_s == verify_s for all s <= r}); the
    step commits draft_1..draft_m and then verify_{m+1}.  ``draft`` holds
    K tokens, ``verify`` K+1 (verify[r] is the greedy token of the row that
    consumed the r-th input)."""
    K = len(draft)
    assert len(verify) == K + 1
    m = 0
    for r in range(1, K + 1):
        if all(int(draft[s - 1]) == int(verify[s - 1]) for s in range(1, r + 1)):
            m = r
    commit = [int(t) for t in draft[:m]] + [int(verify[m])]
    return m, commit


# ---------------------------------------------------------------------------
# per-sequence decoding state and the step
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class SeqState:
    kv: np.ndarray          # verifier KV [L][2][nh][cap][dh]
    dkv: np.ndarray         # draft KV [2][nh][cap][dh]
    kv_len: int             # positions the verifier has consumed
    pending: int            # committed token not yet consumed by the verifier
    hid: np.ndarray         # [n_rows][H] post-norm states of the rows to catch up
    next_tok: np.ndarray    # [n_rows] the committed token that follows each of them
    n_rows: int             # draft rows to catch up at the next step
    row_pos: int            # position of the first of them
    draft_len: int          # draft KV positions held in base form
    out: list               # generated tokens
    max_new: int = 1 << 30
    last_logits: np.ndarray | None = None   # logits of the last prefill row
    prefill_routes_followed: int = 0        # near-tie routes adopted from follow_route
    prefill_routes_rejected: int = 0        # given routes that were not near-ties
    prefill_route_gap: np.ndarray | None = None   # [L][P] k-th vs (k+1)-th router gaps

    @property
    def finished(self) -> bool:
        return len(self.out) >= self.max_new


def prefill(orc: Oracle, cap: int, vision, tokens, max_new: int = 1 << 30,
            follow_route=None, route_tol=None) -> SeqState:
    """Verifier over the prefix (vision rows then text tokens), greedy token
    of the last row, and the draft prefill: rows p = 0..P-2 in base form
    (state b_p, input row p+1 -- a vision row inside the visual prefix).
    follow_route [L][P][k]: routes chosen elsewhere, adopted where they are
    near-ties of the oracle's own up to route_tol[l] (see Oracle.verify_rows)."""
    c = orc.cfg
    nv = 0 if vision is None else len(vision)
    tokens = np.asarray(tokens, dtype=np.int32)
    P = nv + len(tokens)
    tok = np.concatenate([np.full(nv, -1, np.int32), tokens])
    emb = np.zeros((P, c.hidden), dtype=c.wdtype)
    if nv:
        emb[:nv] = vision
    kv, dkv = orc.new_kv(cap), orc.new_dkv(cap)
    hm = np.zeros(P, np.uint8)
    hm[P - 1] = 1
    r = orc.verify_rows(kv, tok, np.arange(P), emb=emb, head_mask=hm, want_logits=True,
                        want_routes=follow_route is not None, follow_route=follow_route,
                        route_tol=route_tol)
    pending = int(r["amax"][P - 1])
    if P >= 2:
        orc.draft_rows(dkv, tok[1:], r["b"][:P - 1], np.arange(P - 1), emb=emb[1:])
    return SeqState(kv=kv, dkv=dkv, kv_len=P, pending=pending, hid=r["b"][P - 1:P].copy(),
                    next_tok=np.array([pending], np.int32), n_rows=1, row_pos=P - 1,
                    draft_len=P - 1, out=[pending], max_new=max_new,
                    last_logits=r["logits"][P - 1].copy(),
                    prefill_routes_followed=r["route_followed"],
                    prefill_routes_rejected=r["route_rejected"],
                    prefill_route_gap=r["route_gap"])


def draft_chain(orc: Oracle, st: SeqState, K: int):
    """Depth 1 over the catch-up rows (the last one starts the chain), then
    depths 2..K one row each.  Returns the K draft tokens and per-depth
    details."""
    n = st.n_rows
    hm = np.zeros(n, np.uint8)
    hm[n - 1] = 1
    r = orc.draft_rows(st.dkv, st.next_tok[:n], st.hid[:n], st.row_pos + np.arange(n), head_mask=hm)
    st.draft_len = st.row_pos + n
    x, u = int(r["amax"][n - 1]), r["u"][n - 1].copy()
    drafts, margins = [x], [float(r["margin"][n - 1])]
    for d in range(2, K + 1):
        p = st.row_pos + n - 1 + (d - 1)
        r = orc.draft_rows(st.dkv, [x], u[None, :], [p], head_mask=np.ones(1, np.uint8))
        x, u = int(r["amax"][0]), r["u"][0].copy()
        drafts.append(x)
        margins.append(float(r["margin"][0]))
    return drafts, margins


def commit(st: SeqState, m: int, commit_tok, b_rows):
    """KV commit/rollback: the verifier rows 0..m become committed (their
    K/V already sit at their absolute positions), later rows are beyond the
    new length and are simply dropped; the next step catches up m+1 draft
    rows from the old length."""
    old = st.kv_len
    st.kv_len = old + m + 1
    st.hid = np.asarray(b_rows[:m + 1], np.float32).copy()
    st.next_tok = np.asarray(commit_tok, np.int32).copy()
    st.n_rows = m + 1
    st.row_pos = old
    st.pending = int(commit_tok[m])
    room = st.max_new - len(st.out)
    st.out.extend(int(t) for t in commit_tok[:max(room, 0)])


def spec_step(orc: Oracle, st: SeqState, K: int, forced=None, want_logits=False):
    """One greedy speculative step: draft K tokens, verify the K+1 rows
    [pending, drafts], accept, commit.  ``forced`` replaces the K draft
    tokens after drafting (benchmark timing mode)."""
    drafts, dmargins = draft_chain(orc, st, K) if K > 0 else ([], [])
    if forced is not None:
        drafts = [int(t) for t in forced]
    toks = [st.pending] + drafts
    r = orc.verify_rows(st.kv, toks, st.kv_len + np.arange(K + 1), want_logits=want_logits)
    v = [int(t) for t in r["amax"]]
    m, ct = accept(drafts, v)
    info = dict(drafts=drafts, draft_margin=dmargins, verify=v, verify_margin=r["margin"].copy(),
                m=m, commit=ct, kv_len_before=st.kv_len, logits=r["logits"], b=r["b"])
    commit(st, m, ct, r["b"])
    return info


def ar_step(orc: Oracle, st: SeqState):
    """Plain greedy decoding: the verifier consumes the pending token."""
    r = orc.verify_rows(st.kv, [st.pending], [st.kv_len])
    v = int(r["amax"][0])
    st.kv_len += 1
    st.pending = v
    if len(st.out) < st.max_new:
        st.out.append(v)
    return v


def ar_decode(orc: Oracle, st: SeqState, n_new: int):
    while len(st.out) < n_new:
        ar_step(orc, st)
    return list(st.out)


def spec_decode(orc: Oracle, st: SeqState, K: int, n_new: int, forced_fn=None):
    """Speculative decoding until n_new tokens are out.  forced_fn(step,
    st) may return K tokens that replace the drafts."""
    st.max_new = n_new
    steps = []
    i = 0
    while not st.finished:
        forced = forced_fn(i, st) if forced_fn else None
        steps.append(spec_step(orc, st, K, forced=forced))
        i += 1
    return list(st.out), steps

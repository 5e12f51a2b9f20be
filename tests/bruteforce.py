"""Brute-force numpy references used only to pin the oracle.

They compute the same model as the oracle by a different route:

* the whole sequence at once with a causal mask (no KV cache, no
  incremental positions);
* every routed expert evaluated densely on every row, then masked by the
  top-k selection (no gather of rows by expert);
* RoPE as a complex rotation (x_i + j x_{i+dh/2}) * exp(j pos theta_i),
  the form in Su et al.;
* float64 everywhere, with values rounded to the model's storage points
  (float32, and bf16 at matrix-product inputs of bf16 models) so the two
  sides can be compared tightly.
"""
from __future__ import annotations

import numpy as np

import synth


def _f32(x):
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def _bf16(x):
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


class Ref:
    """f32_products=True evaluates every matrix product in float32 (BLAS
    summation order) instead of float64; everything else is unchanged.  The
    difference between the two measures how far a change of summation
    order alone moves the model's outputs."""

    def __init__(self, cfg, w, f32_products: bool = False):
        self.cfg = cfg
        self.w = w
        self.bf = cfg.dtype == "bf16"
        self.f32_products = f32_products

    def mm(self, a, W):
        """a @ W.T"""
        if self.f32_products:
            return (np.asarray(a, np.float32) @ np.asarray(W, np.float32).T).astype(np.float64)
        return a @ W.T

    def W(self, name, *idx):
        a = self.w[name]
        for i in idx:
            a = a[i]
        if a.dtype == np.uint16:
            return synth.bf16_bits_to_f32(a).astype(np.float64)
        return a.astype(np.float64)

    def inp(self, x):                       # matrix-product input precision
        return _bf16(x) if self.bf else _f32(x)

    def rms(self, x, g):
        ms = np.mean(x * x, axis=-1, keepdims=True)
        return _f32(x / np.sqrt(ms + self.cfg.rms_eps) * g)

    def rope(self, x, pos):
        """x [n][heads][dh], pos [n]: complex rotation of (x_i, x_{i+dh/2})."""
        dh = x.shape[-1]
        half = dh // 2
        inv = self.cfg.rope_theta ** (-2.0 * np.arange(half) / dh)
        ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]
        rot = _f32(np.cos(ang)) + 1j * _f32(np.sin(ang))
        z = (x[..., :half] + 1j * x[..., half:]) * rot[:, None, :]
        return _f32(np.concatenate([z.real, z.imag], axis=-1))

    def attn_block(self, h, pos, g, wqkv, wo):
        """pre-norm causal self-attention over the full row set."""
        c = self.cfg
        n = h.shape[0]
        nh, dh = c.n_heads, c.head_dim
        a = self.inp(self.rms(h, g))
        qkv = _f32(self.mm(a, wqkv))
        q = qkv[:, :nh * dh].reshape(n, nh, dh)
        k = qkv[:, nh * dh:2 * nh * dh].reshape(n, nh, dh)
        v = qkv[:, 2 * nh * dh:].reshape(n, nh, dh)
        q = self.rope(q, pos)
        k = self.inp(self.rope(k, pos))
        v = self.inp(v)
        s = np.einsum("ihd,jhd->hij", q, k) / np.sqrt(dh)
        mask = np.asarray(pos)[None, :] <= np.asarray(pos)[:, None]
        s = np.where(mask[None], s, -np.inf)
        s = s - s.max(axis=-1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=-1, keepdims=True)
        o = self.inp(np.einsum("hij,jhd->ihd", p, v).reshape(n, nh * dh))
        return _f32(h + _f32(self.mm(o, wo)))

    def swiglu(self, y, wg, wu, wd):
        g = _f32(self.mm(y, wg))
        u = _f32(self.mm(y, wu))
        act = self.inp(g / (1.0 + np.exp(-g)) * u)
        return _f32(self.mm(act, wd))

    def moe_block(self, h, l, force=None):
        """dense evaluation of all routed experts, masked by top-k.
        force {row: expert ids}: that row's selection instead of its top-k."""
        c = self.cfg
        E, k, S, I = c.n_routed, c.top_k, c.n_shared, c.moe_inter
        y = self.inp(self.rms(h, self.W("ffn_norm", l)))
        lg = _f32(_f32(self.mm(y, self.W("router", l))) + self.w["router_bias"][l].astype(np.float64))
        z = lg - lg.max(axis=-1, keepdims=True)
        pr = _f32(np.exp(z) / np.exp(z).sum(axis=-1, keepdims=True))
        n = h.shape[0]
        mask = np.zeros((n, E))
        sel = np.zeros((n, k), dtype=np.int64)
        for r in range(n):
            order = np.lexsort((np.arange(E), -lg[r]))    # logit desc, then id asc
            sel[r] = order[:k] if not force or r not in force else force[r]
            mask[r, sel[r]] = 1.0
        out = np.zeros_like(h)
        shg, shd = self.W("sh_gu", l), self.W("sh_down", l)
        for s in range(S):
            out += self.swiglu(y, shg[s * I:(s + 1) * I], shg[(S + s) * I:(S + s + 1) * I],
                               shd[:, s * I:(s + 1) * I])
        for e in range(E):
            gu = self.W("exp_gu", l, e)
            fe = self.swiglu(y, gu[:I], gu[I:], self.W("exp_down", l, e))
            out += _f32(mask[:, e:e + 1] * pr[:, e:e + 1] * fe)
        return _f32(h + _f32(out)), sel, lg

    def embed_rows(self, tok, emb):
        c = self.cfg
        rows = np.zeros((len(tok), c.hidden))
        for r, t in enumerate(tok):
            if t >= 0:
                rows[r] = self.W("embed", int(t))
            else:
                e = emb[r]
                rows[r] = synth.bf16_bits_to_f32(e) if e.dtype == np.uint16 else e
        return rows

    def lm_logits(self, x):
        W = self.W("embed") if self.cfg.tie_lm_head else self.W("lm_head")
        return _f32(self.mm(self.inp(x), W))

    def verifier(self, tok, emb=None, force=None):
        """rows 0..n-1 at positions 0..n-1: returns b, logits, routes.
        force {(layer, row): expert ids} overrides those selections."""
        c = self.cfg
        h = self.embed_rows(tok, emb)
        pos = np.arange(len(tok))
        routes, router_logits = [], []
        for l in range(c.n_layers):
            h = self.attn_block(h, pos, self.W("attn_norm", l), self.W("wqkv", l), self.W("wo", l))
            fl = {r: e for (ll, r), e in (force or {}).items() if ll == l}
            h, sel, lg = self.moe_block(h, l, fl)
            routes.append(sel)
            router_logits.append(lg)
        b = self.rms(h, self.W("final_norm"))
        self.router_logits = np.stack(router_logits)    # [L][n][E] of the last call
        return b, self.lm_logits(b), np.stack(routes)

    def draft(self, next_tok, next_emb, a, pos):
        """draft rows with states a at positions pos (all rows attend
        causally to each other, as in the parallel training grid)."""
        e = self.embed_rows(next_tok, next_emb)
        cat = np.concatenate([self.inp(self.rms(e, self.W("d_enorm"))),
                              self.inp(self.rms(np.asarray(a, np.float64), self.W("d_hnorm")))],
                             axis=-1)
        z = _f32(self.mm(cat, self.W("d_eh_proj")))
        z = self.attn_block(z, pos, self.W("d_attn_norm"), self.W("d_wqkv"), self.W("d_wo"))
        F = self.cfg.draft_inter
        gu = self.W("d_gu")
        y = self.inp(self.rms(z, self.W("d_ffn_norm")))
        z = _f32(z + self.swiglu(y, gu[:F], gu[F:], self.W("d_down")))
        u = self.rms(z, self.W("final_norm"))
        return u, self.lm_logits(u)

"""Seeded synthetic inputs for the FastMTP speculative-decode step.

This module is the only code shared by the CPU oracle and the GPU path:
it produces model shapes, random-init weights, vision-prefix rows, token
ids, context lengths and synthetic KV caches from stated seeds.  It holds
none of the decoding arithmetic (no norm, matmul, softmax or argmax).

Weights follow the initialisation the workloads prescribe: every matrix
and embedding is N(0, 0.02); RMSNorm gains are 1 (optionally jittered for
tests that must see a gain bug); there are no biases.  bf16 tensors are
returned as uint16 bit patterns (round-to-nearest-even from the drawn
value).  Random numbers come from Philox4x32-10 in ``synth.c``.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "_synth.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile synth.c into _synth.so (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11",
             os.path.join(_HERE, "synth.c"), "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _L():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        u64, u32, i64, dbl, vp = (ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64,
                                  ctypes.c_double, ctypes.c_void_p)
        lib.synth_philox4x32.argtypes = [vp, vp, ctypes.c_int, vp]
        lib.synth_normal_f32.argtypes = [u64, u32, u64, u64, dbl, dbl, vp]
        lib.synth_normal_bf16.argtypes = [u64, u32, u64, u64, dbl, dbl, vp]
        lib.synth_uniform_int.argtypes = [u64, u32, u64, i64, u32, vp]
        lib.synth_uniform_f64.argtypes = [u64, u32, u64, vp]
        lib.synth_normal_at.argtypes = [u64, u32, u64]
        lib.synth_normal_at.restype = dbl
        _lib = lib
    return _lib


# --------------------------------------------------------------------------
# raw draws
# --------------------------------------------------------------------------

def philox4x32(ctr, key, rounds=10):
    c = np.asarray(ctr, dtype=np.uint32).copy()
    k = np.asarray(key, dtype=np.uint32).copy()
    out = np.zeros(4, dtype=np.uint32)
    _L().synth_philox4x32(c.ctypes.data, k.ctypes.data, rounds, out.ctypes.data)
    return out


def normal(seed: int, stream: int, shape, std: float = 1.0, mean: float = 0.0,
           dtype: str = "f32", start: int = 0) -> np.ndarray:
    """mean + std * N(0,1) elements start.. of (seed, stream); float32, or
    bf16 bits (uint16) when dtype == 'bf16'."""
    n = int(np.prod(shape)) if len(shape) else 1
    if dtype == "bf16":
        out = np.empty(shape, dtype=np.uint16)
        _L().synth_normal_bf16(seed, stream, start, n, mean, std, out.ctypes.data)
    else:
        out = np.empty(shape, dtype=np.float32)
        _L().synth_normal_f32(seed, stream, start, n, mean, std, out.ctypes.data)
    return out


def uniform_int(seed: int, stream: int, n: int, lo: int, span: int) -> np.ndarray:
    """n integers uniform in [lo, lo + span)."""
    out = np.empty(n, dtype=np.int32)
    _L().synth_uniform_int(seed, stream, n, lo, span, out.ctypes.data)
    return out


def uniform_f64(seed: int, stream: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.float64)
    _L().synth_uniform_f64(seed, stream, n, out.ctypes.data)
    return out


def bf16_bits_to_f32(u16: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32 (a storage-format change)."""
    return (np.asarray(u16, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------
# model shapes
# --------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class ModelCfg:
    name: str
    n_layers: int
    hidden: int
    n_heads: int
    head_dim: int
    n_routed: int
    top_k: int
    n_shared: int
    moe_inter: int
    draft_inter: int
    vocab: int
    tie_lm_head: bool
    dtype: str          # 'f32' or 'bf16'
    rope_theta: float
    rms_eps: float = 1e-6

    @property
    def wdtype(self):
        return np.uint16 if self.dtype == "bf16" else np.float32


# Tiny fp32 plumbing case: 2 layers, hidden 256, 4 heads x 64, 8 routed
# experts (top-2, width 128) + 1 shared, vocab 4096, tied LM head, RoPE
# base 1e4.  Draft FFN width = (top_k + shared) * width = 384.
TINY = ModelCfg("tiny", 2, 256, 4, 64, 8, 2, 1, 128, 384, 4096, True, "f32", 1e4)
# Full shape: DeepSeek-3B-MoE decoder (12 layers, d=1280, 10 heads x 128,
# 64 routed top-6 + 2 shared of width 896, vocab 129,280, RoPE base 1e6);
# draft FFN width (6 + 2) * 896 = 7168.
FULL = ModelCfg("full", 12, 1280, 10, 128, 64, 6, 2, 896, 7168, 129280, False, "bf16", 1e6)
# Mid-size bf16 shape for GPU parity cases the oracle finishes in seconds:
# several tiles in every dimension and a ragged vocabulary tail.
MID = ModelCfg("mid", 2, 512, 4, 128, 16, 4, 2, 256, 1536, 8000, False, "bf16", 1e6)
# Tiny bf16 shape (fast CPU tests of the bf16 rounding points).
TINYB = ModelCfg("tinyb", 2, 256, 2, 128, 8, 2, 2, 128, 512, 3000, False, "bf16", 1e6)

# Untied variant of the tiny case: with a tied head and random weights the
# greedy token equals the input token, so tests that need varied
# trajectories use this one.
TINYU = dataclasses.replace(TINY, name="tinyu", tie_lm_head=False)

CONFIGS = {c.name: c for c in (TINY, TINYU, FULL, MID, TINYB)}

# stream ids of the weight tensors
_STREAM = {
    "embed": 1, "lm_head": 2,
    "wqkv": 10, "wo": 11, "router": 12, "exp_gu": 13, "exp_down": 14,
    "sh_gu": 15, "sh_down": 16,
    "final_norm": 20, "attn_norm": 21, "ffn_norm": 22,
    "d_eh_proj": 30, "d_wqkv": 31, "d_wo": 32, "d_gu": 33, "d_down": 34,
    "d_enorm": 40, "d_hnorm": 41, "d_attn_norm": 42, "d_ffn_norm": 43,
}


def weight_shapes(cfg: ModelCfg) -> dict:
    """Every weight tensor and its shape.  Linear weights are [out][in].

    exp_gu[l][e] holds the gate rows (0..I-1) then the up rows (I..2I-1).
    sh_gu[l] holds the gate rows of all shared experts (expert s at rows
    s*I..s*I+I-1), then their up rows (S*I + s*I ...); sh_down[l] is
    [H][S*I] with expert s in columns s*I..s*I+I-1.
    """
    L, H, E, I, S, F, V = (cfg.n_layers, cfg.hidden, cfg.n_routed, cfg.moe_inter,
                           cfg.n_shared, cfg.draft_inter, cfg.vocab)
    nhd = cfg.n_heads * cfg.head_dim
    shp = {
        "embed": (V, H),
        "final_norm": (H,),
        "attn_norm": (L, H), "wqkv": (L, 3 * nhd, H), "wo": (L, H, nhd),
        "ffn_norm": (L, H), "router": (L, E, H),
        "exp_gu": (L, E, 2 * I, H), "exp_down": (L, E, H, I),
        "sh_gu": (L, 2 * S * I, H), "sh_down": (L, H, S * I),
        "d_enorm": (H,), "d_hnorm": (H,), "d_eh_proj": (H, 2 * H),
        "d_attn_norm": (H,), "d_wqkv": (3 * nhd, H), "d_wo": (H, nhd),
        "d_ffn_norm": (H,), "d_gu": (2 * F, H), "d_down": (H, F),
    }
    if not cfg.tie_lm_head:
        shp["lm_head"] = (V, H)
    return shp


_NORMS = ("final_norm", "attn_norm", "ffn_norm", "d_enorm", "d_hnorm", "d_attn_norm",
          "d_ffn_norm")
_DRAFT = ("d_enorm", "d_hnorm", "d_eh_proj", "d_attn_norm", "d_wqkv", "d_wo",
          "d_ffn_norm", "d_gu", "d_down")


def zipf_router_bias(cfg: ModelCfg, s: float = 1.1, seed_base: int = 14) -> np.ndarray:
    """Per-layer router-logit bias -s*ln(rank_e); rank_e is a seeded
    permutation of 1..E (seed seed_base + layer).  float32 [L][E]."""
    L, E = cfg.n_layers, cfg.n_routed
    out = np.zeros((L, E), dtype=np.float32)
    for l in range(L):
        u = uniform_f64(seed_base + l, 50, E)
        order = np.argsort(u, kind="stable")          # order[r] = expert with rank r+1
        rank = np.empty(E, dtype=np.int64)
        rank[order] = np.arange(1, E + 1)
        out[l] = (-s * np.log(rank.astype(np.float64))).astype(np.float32)
    return out


def make_weights(cfg: ModelCfg, seed: int = 0, draft_seed: int = 1,
                 gain_jitter: float = 0.0, zipf_s: float = 0.0,
                 zipf_seed: int = 14) -> dict:
    """Random-init weights: matrices N(0, 0.02) in the model dtype, norm
    gains float32 (1, or 1 + gain_jitter*N(0,1)), router bias float32
    [L][E] (zeros unless zipf_s > 0)."""
    w = {}
    for name, shape in weight_shapes(cfg).items():
        sd = draft_seed if name in _DRAFT else seed
        if name in _NORMS:
            if gain_jitter > 0:
                w[name] = normal(sd, _STREAM[name], shape, std=gain_jitter, mean=1.0)
            else:
                w[name] = np.ones(shape, dtype=np.float32)
        else:
            w[name] = normal(sd, _STREAM[name], shape, std=0.02, dtype=cfg.dtype)
    if zipf_s > 0:
        w["router_bias"] = zipf_router_bias(cfg, zipf_s, zipf_seed)
    else:
        w["router_bias"] = np.zeros((cfg.n_layers, cfg.n_routed), dtype=np.float32)
    return w


# --------------------------------------------------------------------------
# workload inputs
# --------------------------------------------------------------------------

def vision_prefix(cfg: ModelCfg, n: int, seed: int = 10, stream: int = 60) -> np.ndarray:
    """n vision-prefix rows N(0,1) of width H, in the model dtype."""
    return normal(seed, stream, (n, cfg.hidden), std=1.0, dtype=cfg.dtype)


def text_tokens(cfg: ModelCfg, n: int, seed: int = 11, stream: int = 61) -> np.ndarray:
    return uniform_int(seed, stream, n, 0, cfg.vocab)


def page_inputs(cfg: ModelCfg, pages: int, n_vis: int = 256, n_txt: int = 32):
    """The page-loop prefixes: page q is n_vis vision rows N(0,1) (seed
    20+q) followed by the same n_txt prompt tokens (seed 21).  Returns tok
    [pages][P] int32 (-1 = vision row) and vision [pages][P][H] (model
    dtype, zero at prompt rows)."""
    P = n_vis + n_txt
    tok = np.full((pages, P), -1, np.int32)
    vis = np.zeros((pages, P, cfg.hidden), cfg.wdtype)
    prompt = text_tokens(cfg, n_txt, seed=21)
    for q in range(pages):
        vis[q, :n_vis] = vision_prefix(cfg, n_vis, seed=20 + q)
        tok[q, n_vis:] = prompt
    return tok, vis


def context_lengths(b: int, lo: int, hi: int, seed: int) -> np.ndarray:
    """b lengths uniform over the integers lo..hi inclusive."""
    return uniform_int(seed, 62, b, lo, hi - lo + 1)


# Synthetic KV caches: the value at (layer l, sequence b, k/v c, head h,
# position p, dim d) is N(0,1) element
#   ((((l*BMAX + b)*2 + c)*nh + h)*PMAX + p)*dh + d
# of (seed, stream), BMAX = 1024, PMAX = 32768, so it does not depend on
# the batch size or on the allocated capacity.
_BMAX = 1024
_PMAX = 32768


def kv_values(cfg: ModelCfg, layer: int, b: int, c: int, n_pos: int, seed: int,
              stream: int) -> np.ndarray:
    """[nh][n_pos][dh] block (positions 0..n_pos-1) of a synthetic cache,
    in the model dtype."""
    nh, dh = cfg.n_heads, cfg.head_dim
    out = np.empty((nh, n_pos, dh), dtype=cfg.wdtype)
    for h in range(nh):
        base = ((((layer * _BMAX + b) * 2 + c) * nh + h) * _PMAX) * dh
        out[h] = normal(seed, stream, (n_pos, dh), dtype=cfg.dtype, start=base)
    return out

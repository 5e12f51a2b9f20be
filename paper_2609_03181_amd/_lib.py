"""ctypes binding of libmtp.so: the entry points of include/mtp.h under
the same names.  Argument marshalling only: every step of the decode path
runs in the library's HIP kernels.  Device pointers are passed as ints."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmtp.so")

(MTP_OK, MTP_EINVAL, MTP_ECAPACITY, MTP_EHIP, MTP_EUNSUPPORTED, MTP_ETOKEN,
 MTP_ERANGE, MTP_ESTALL) = 0, -1, -2, -3, -4, -5, -6, -7
MTP_F32, MTP_BF16 = 0, 1
STATUS_NAMES = {0: "MTP_OK", -1: "MTP_EINVAL", -2: "MTP_ECAPACITY", -3: "MTP_EHIP",
                -4: "MTP_EUNSUPPORTED", -5: "MTP_ETOKEN", -6: "MTP_ERANGE",
                -7: "MTP_ESTALL"}

# every symbol include/mtp.h declares
EXPORTS = ("mtp_create", "mtp_destroy", "mtp_context_bytes", "mtp_workspace_bytes",
           "mtp_status_read",
           "mtp_status_clear", "mtp_prefill", "mtp_draft_k", "moe_verify_step",
           "moe_verify_step_static", "mtp_objective_workspace_bytes", "mtp_objective",
           "greedy_accept", "kv_commit_rollback", "mtp_bench_override_drafts",
           "mtp_timing_start", "mtp_timing_stop")

# kernel classes of the timing hook (mtp_kernel_class)
KC_ATTN, KC_MOE_GU, KC_MOE_DOWN, KC_LM_HEAD, KC_QKV, KC_ROUTER, KC_DRAFT_FFN, KC_MOE = range(1, 9)


class MtpError(RuntimeError):
    def __init__(self, fn, code):
        super().__init__(f"{fn} returned {STATUS_NAMES.get(code, code)}")
        self.code = code


class MtpConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "hidden", "n_heads", "head_dim", "n_routed", "top_k", "n_shared",
        "moe_inter", "draft_inter", "vocab", "tie_lm_head", "dtype", "max_batch", "max_ctx",
        "max_k")] + [("rope_theta", ctypes.c_double), ("rms_eps", ctypes.c_double)]


WEIGHT_FIELDS = ("embed", "lm_head", "final_norm", "attn_norm", "ffn_norm", "wqkv", "wo",
                 "router", "router_bias", "exp_gu", "exp_down", "sh_gu", "sh_down", "d_enorm",
                 "d_hnorm", "d_attn_norm", "d_ffn_norm", "d_eh_proj", "d_wqkv", "d_wo", "d_gu",
                 "d_down")


class MtpWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in WEIGHT_FIELDS]


_lib = None


def load():
    """Loads the in-tree libmtp.so; raises when it is missing (there is no
    fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2609_03181_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    sig = {
        "mtp_create": ([P, P, P], I32),
        "mtp_destroy": ([P], None),
        "mtp_context_bytes": ([P], SZ),
        "mtp_workspace_bytes": ([P, I32, I32], SZ),
        "mtp_status_read": ([P, P, P], I32),
        "mtp_status_clear": ([P, P, P], I32),
        "mtp_prefill": ([P, I32, I32, I32, P, P, P, P, P, P, P, P, P, P, P, P, I32, P, P, P, SZ,
                         P], I32),
        "mtp_draft_k": ([P, I32, I32, P, P, P, P, P, P, P, P, P, P, SZ, P], I32),
        "moe_verify_step": ([P, I32, I32, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P], I32),
        "moe_verify_step_static": ([P, I32, I32, P, P, P, P, P, P, P, P, P, P, P, P], I32),
        "mtp_objective_workspace_bytes": ([P, I32], SZ),
        "mtp_objective": ([P, I32, I32, I32, P, P, P, P, P, P, P, P, SZ, P], I32),
        "greedy_accept": ([I32, I32, P, P, P, P, P], I32),
        "kv_commit_rollback": ([P, I32, I32, P, P, P, P, P, P, P, P, P, I32, P, P], I32),
        "mtp_bench_override_drafts": ([I32, I32, P, I32, P, P, P], I32),
        "mtp_timing_start": ([P, I32, I32], I32),
        "mtp_timing_stop": ([P, P, P], I32),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    _lib = lib
    return lib


def _check(name, rc):
    if rc != MTP_OK:
        raise MtpError(name, rc)


def mtp_create(cfg: MtpConfig, w: MtpWeights) -> int:
    out = ctypes.c_void_p()
    _check("mtp_create", load().mtp_create(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(out)))
    return out.value


def mtp_destroy(ctx: int) -> None:
    load().mtp_destroy(ctx)


def mtp_context_bytes(ctx: int) -> int:
    return int(load().mtp_context_bytes(ctx))


def mtp_workspace_bytes(ctx: int, batch: int, rows: int) -> int:
    return int(load().mtp_workspace_bytes(ctx, batch, rows))


def mtp_status_read(ctx: int, ws: int) -> int:
    st = ctypes.c_int32(0)
    _check("mtp_status_read", load().mtp_status_read(ctx, ws, ctypes.byref(st)))
    return st.value


def mtp_status_clear(ctx: int, ws: int, stream: int) -> None:
    _check("mtp_status_clear", load().mtp_status_clear(ctx, ws, stream))


def mtp_prefill(ctx, batch, k, n_rows, tok, vision, kv_cache, draft_kv, kv_len, draft_len, hid,
                next_tok, n_rows_out, row_pos, pending, out_tok, max_out, n_out, route_idx, ws,
                ws_bytes, stream):
    _check("mtp_prefill", load().mtp_prefill(
        ctx, batch, k, n_rows, tok, vision, kv_cache, draft_kv, kv_len, draft_len, hid, next_tok,
        n_rows_out, row_pos, pending, out_tok, max_out, n_out, route_idx, ws, ws_bytes, stream))


def mtp_draft_k(ctx, batch, k, hid, next_tok, n_rows, row_pos, draft_kv, draft_len, draft_tok,
                draft_logits, draft_u, ws, ws_bytes, stream):
    _check("mtp_draft_k", load().mtp_draft_k(ctx, batch, k, hid, next_tok, n_rows, row_pos,
                                             draft_kv, draft_len, draft_tok, draft_logits,
                                             draft_u, ws, ws_bytes, stream))


def moe_verify_step(ctx, batch, k, pending, draft_tok, kv_len, kv_cache, verify_tok, hid, logits,
                    margin, route_idx, route_gap, layer_h, ws, ws_bytes, stream):
    _check("moe_verify_step", load().moe_verify_step(
        ctx, batch, k, pending, draft_tok, kv_len, kv_cache, verify_tok, hid, logits, margin,
        route_idx, route_gap, layer_h, ws, ws_bytes, stream))


def moe_verify_step_static(ctx, batch, k, pending, draft_tok, kv_len, kv_cache, verify_tok, hid,
                           logits, margin, route_idx, route_gap, layer_h, stream):
    _check("moe_verify_step_static", load().moe_verify_step_static(
        ctx, batch, k, pending, draft_tok, kv_len, kv_cache, verify_tok, hid, logits, margin,
        route_idx, route_gap, layer_h, stream))


def mtp_objective_workspace_bytes(ctx, n_rows):
    return int(load().mtp_objective_workspace_bytes(ctx, n_rows))


def mtp_objective(ctx, n_rows, n_prompt, k, tok, vision, b_states, draft_kv, row_terms, u_out,
                  loss, ws, ws_bytes, stream):
    _check("mtp_objective", load().mtp_objective(ctx, n_rows, n_prompt, k, tok, vision, b_states,
                                                 draft_kv, row_terms, u_out, loss, ws, ws_bytes,
                                                 stream))


def greedy_accept(batch, k, draft_tok, verify_tok, accept_len, commit_tok, stream):
    _check("greedy_accept", load().greedy_accept(batch, k, draft_tok, verify_tok, accept_len,
                                                 commit_tok, stream))


def kv_commit_rollback(ctx, batch, k, accept_len, commit_tok, kv_len, n_rows, row_pos, pending,
                       next_tok, max_new, out_tok, max_out, n_out, stream):
    _check("kv_commit_rollback", load().kv_commit_rollback(
        ctx, batch, k, accept_len, commit_tok, kv_len, n_rows, row_pos, pending, next_tok,
        max_new, out_tok, max_out, n_out, stream))


def mtp_bench_override_drafts(batch, k, table, n_steps, step_ctr, draft_tok, stream):
    _check("mtp_bench_override_drafts", load().mtp_bench_override_drafts(
        batch, k, table, n_steps, step_ctr, draft_tok, stream))


def mtp_timing_start(ctx, kernel_class, max_launches):
    _check("mtp_timing_start", load().mtp_timing_start(ctx, kernel_class, max_launches))


def mtp_timing_stop(ctx):
    """-> (summed launch durations in ms, number of timed launches)"""
    ms, n = ctypes.c_float(0.0), ctypes.c_int32(0)
    _check("mtp_timing_stop", load().mtp_timing_stop(ctx, ctypes.byref(ms), ctypes.byref(n)))
    return float(ms.value), int(n.value)

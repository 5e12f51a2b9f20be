"""Device-side driver of the decode step: PyTorch allocates the buffers and
provides the stream; every computation is a libmtp.so call.

Model   -- weights uploaded to HBM plus the library context.
Session -- per-batch state (KV caches, step buffers, workspace), prefill,
           one speculative step (draft -> verify -> accept -> commit), and
           a HIP-graph capture of that step.
"""
from __future__ import annotations

import numpy as np
import torch

from . import _lib


def _dev_tensor(arr: np.ndarray, device) -> torch.Tensor:
    a = np.ascontiguousarray(arr)
    if a.dtype == np.uint16:                       # bf16 bit patterns
        return torch.from_numpy(a.view(np.int16)).to(device)
    return torch.from_numpy(a).to(device)


class Model:
    """Weights in HBM + an mtp context.  ``cfg`` is a synth.ModelCfg-like
    object (n_layers, hidden, ... , dtype 'f32'|'bf16')."""

    def __init__(self, cfg, weights: dict, max_batch: int, max_ctx: int, max_k: int,
                 device="cuda"):
        self.cfg = cfg
        self.device = torch.device(device)
        self.max_batch, self.max_ctx, self.max_k = max_batch, max_ctx, max_k
        self.t = {k: _dev_tensor(v, self.device) for k, v in weights.items()}
        self.bf16 = cfg.dtype == "bf16"
        c = _lib.MtpConfig(cfg.n_layers, cfg.hidden, cfg.n_heads, cfg.head_dim, cfg.n_routed,
                           cfg.top_k, cfg.n_shared, cfg.moe_inter, cfg.draft_inter, cfg.vocab,
                           int(cfg.tie_lm_head), _lib.MTP_BF16 if self.bf16 else _lib.MTP_F32,
                           max_batch, max_ctx, max_k, float(cfg.rope_theta), float(cfg.rms_eps))
        w = _lib.MtpWeights(*[self.t[n].data_ptr() if n in self.t else None
                              for n in _lib.WEIGHT_FIELDS])
        self.mcfg, self.mw = c, w
        self.ctx = _lib.mtp_create(c, w)

    @property
    def storage_dtype(self):
        return torch.int16 if self.bf16 else torch.float32

    def close(self):
        if self.ctx:
            _lib.mtp_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _p(t):
    return None if t is None else t.data_ptr()


class Session:
    """Decoding state of B sequences with draft depth K."""

    def __init__(self, model: Model, batch: int, k: int, max_out: int, prefill_rows: int = 0,
                 record: bool = False):
        c = model.cfg
        self.m, self.B, self.K, self.max_out = model, batch, k, max_out
        dev = model.device
        i32 = dict(dtype=torch.int32, device=dev)
        cap = model.max_ctx
        self.kv = torch.zeros((c.n_layers, batch, 2, c.n_heads, cap, c.head_dim),
                              dtype=model.storage_dtype, device=dev)
        self.dkv = torch.zeros((batch, 2, c.n_heads, cap, c.head_dim), dtype=model.storage_dtype,
                               device=dev)
        z = lambda *s: torch.zeros(s, **i32)
        self.kv_len, self.draft_len, self.n_rows, self.row_pos = z(batch), z(batch), z(batch), z(batch)
        self.pending, self.accept_len, self.n_out = z(batch), z(batch), z(batch)
        self.next_tok, self.verify_tok, self.commit_tok = z(batch, k + 1), z(batch, k + 1), z(batch, k + 1)
        self.draft_tok = z(batch, max(k, 1))
        self.out_tok = z(batch, max(max_out, 1))
        self.max_new = torch.full((batch,), max_out, **i32)
        self.hid = torch.zeros((batch, k + 1, c.hidden), dtype=torch.float32, device=dev)
        rows = max(k + 1, prefill_rows)
        self.ws_bytes = _lib.mtp_workspace_bytes(model.ctx, batch, rows)
        self.ws = torch.zeros(self.ws_bytes, dtype=torch.uint8, device=dev)
        # optional per-step records (tests)
        self.record = record
        if record:
            R = batch * (k + 1)
            self.logits = torch.zeros((batch, k + 1, c.vocab), dtype=torch.float32, device=dev)
            self.margin = torch.zeros((batch, k + 1), dtype=torch.float32, device=dev)
            self.route_idx = torch.zeros((c.n_layers, R, c.top_k), **i32)
            self.route_gap = torch.zeros((c.n_layers, R), dtype=torch.float32, device=dev)
            self.layer_h = torch.zeros((c.n_layers + 1, R, c.hidden), dtype=torch.float32,
                                       device=dev)
            self.draft_logits = torch.zeros((batch, max(k, 1), c.vocab), dtype=torch.float32,
                                            device=dev)
            self.drafted_tok = z(batch, max(k, 1))   # drafts before a forced override
            self.draft_u = torch.zeros((batch, max(k, 1), c.hidden), dtype=torch.float32,
                                       device=dev)
        else:
            self.logits = self.margin = self.route_idx = self.route_gap = None
            self.layer_h = None
            self.draft_u = None
            self.draft_logits = None
        self.override = None
        self.graph = None

    # ------------------------------------------------------------------
    @property
    def stream(self) -> int:
        return torch.cuda.current_stream(self.m.device).cuda_stream

    def status(self) -> int:
        torch.cuda.synchronize(self.m.device)
        return _lib.mtp_status_read(self.m.ctx, self.ws.data_ptr())

    def prefill(self, tok: torch.Tensor, vision: torch.Tensor | None = None):
        """tok [B][P] int32 (negative = vision row), vision [B][P][H] storage dtype."""
        B, P = tok.shape
        assert B == self.B
        tok = tok.to(self.m.device, torch.int32).contiguous()
        if vision is not None:
            vision = vision.to(self.m.device).contiguous()
        c = self.m.cfg
        # record mode keeps the prefill's routing ([L][B][P][k]) for checks
        self.prefill_routes = (torch.zeros((c.n_layers, B, P, c.top_k), dtype=torch.int32,
                                           device=self.m.device) if self.record else None)
        _lib.mtp_prefill(self.m.ctx, B, self.K, P, _p(tok), _p(vision), _p(self.kv), _p(self.dkv),
                         _p(self.kv_len), _p(self.draft_len), _p(self.hid), _p(self.next_tok),
                         _p(self.n_rows), _p(self.row_pos), _p(self.pending), _p(self.out_tok),
                         self.max_out, _p(self.n_out), _p(self.prefill_routes), _p(self.ws),
                         self.ws_bytes, self.stream)

    def set_forced_drafts(self, table: torch.Tensor):
        """Benchmark timing mode: table [n_steps][B][K] of draft tokens that
        replace the drafted ones, step by step."""
        self.override = (table.to(self.m.device, torch.int32).contiguous(),
                         torch.zeros(1, dtype=torch.int32, device=self.m.device))

    def update_forced_drafts(self, table: torch.Tensor):
        """Rewrites the forced-draft table in place (same shape) and restarts
        it at its first row, so a step captured in a graph picks it up."""
        t, ctr = self.override
        t.copy_(table.to(t.device, torch.int32))
        ctr.zero_()

    def draft(self):
        _lib.mtp_draft_k(self.m.ctx, self.B, self.K, _p(self.hid), _p(self.next_tok),
                         _p(self.n_rows), _p(self.row_pos), _p(self.dkv), _p(self.draft_len),
                         _p(self.draft_tok), _p(self.draft_logits), _p(self.draft_u),
                         _p(self.ws), self.ws_bytes, self.stream)
        if self.override is not None and self.K > 0:
            if self.record:
                self.drafted_tok.copy_(self.draft_tok)
            table, ctr = self.override
            _lib.mtp_bench_override_drafts(self.B, self.K, _p(table), table.shape[0], _p(ctr),
                                           _p(self.draft_tok), self.stream)

    def verify(self):
        _lib.moe_verify_step(self.m.ctx, self.B, self.K, _p(self.pending),
                             _p(self.draft_tok) if self.K > 0 else None, _p(self.kv_len),
                             _p(self.kv), _p(self.verify_tok), _p(self.hid), _p(self.logits),
                             _p(self.margin), _p(self.route_idx), _p(self.route_gap),
                             _p(self.layer_h), _p(self.ws), self.ws_bytes, self.stream)

    def accept(self):
        _lib.greedy_accept(self.B, self.K, _p(self.draft_tok) if self.K > 0 else None,
                           _p(self.verify_tok), _p(self.accept_len), _p(self.commit_tok),
                           self.stream)

    def commit(self):
        _lib.kv_commit_rollback(self.m.ctx, self.B, self.K, _p(self.accept_len),
                                _p(self.commit_tok), _p(self.kv_len), _p(self.n_rows),
                                _p(self.row_pos), _p(self.pending), _p(self.next_tok),
                                _p(self.max_new), _p(self.out_tok), self.max_out, _p(self.n_out),
                                self.stream)

    def step(self):
        """One greedy speculative step on the current stream."""
        self.draft()
        self.verify()
        self.accept()
        self.commit()

    def capture(self):
        """Captures one step into a HIP graph (replayed by replay())."""
        s = torch.cuda.Stream(self.m.device)
        s.wait_stream(torch.cuda.current_stream(self.m.device))
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            self.step()
        torch.cuda.current_stream(self.m.device).wait_stream(s)
        self.graph = g
        return g

    def replay(self):
        self.graph.replay()

    def outputs(self):
        torch.cuda.synchronize(self.m.device)
        n = self.n_out.cpu().numpy()
        o = self.out_tok.cpu().numpy()
        return [o[b, :n[b]].tolist() for b in range(self.B)]

"""Benchmark of the greedy speculative decode step on one MI355X.

A step is one pass of the whole hot path over the batch: FastMTP draft
(K=3 recursive applications of one block), one verifier pass over the K+1
rows of every sequence, greedy acceptance and the KV commit/rollback.
The headline workload is the full-shape B=1 case: 256 vision-prefix rows
+ 512 prompt tokens (real prefill), then verify steps; the value is
accepted tokens/s (tokens committed per second, bonus included).

Prints one JSON line.  Other workloads (--workload b16 / b64 / tiny) print
the same line for their configuration.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


WORKLOADS = {
    # full shape, batch 1, real prefill of 256 vision rows + 512 tokens
    "b1": dict(model="full", B=1, K=3, n_vis=256, n_txt=512, synthetic=False, forced=False,
               zipf=0.0),
    # full shape, batch 16, cached contexts U{1024..2048}, forced acceptance
    "b16": dict(model="full", B=16, K=3, ctx=(1024, 2048, 2), synthetic=True, forced=True,
                zipf=0.0),
    # full shape, batch 64, cached contexts U{512..4096}, Zipf-skewed routing
    "b64": dict(model="full", B=64, K=3, ctx=(512, 4096, 12), synthetic=True, forced=False,
                zipf=1.1),
    # tiny fp32 case
    "tiny": dict(model="tiny", B=1, K=3, n_vis=64, n_txt=16, synthetic=False, forced=False,
                 zipf=0.0),
}


def verify_bytes(cfg, B, K, kv_len, routes):
    """Algorithmic HBM bytes of one verify pass: every weight touched once
    (attention, router, shared experts, the distinct routed experts of each
    layer, final norm, LM head), each sequence's cached K/V read once, the
    new rows' K/V written once, the input embedding rows read once."""
    es = 2 if cfg.dtype == "bf16" else 4
    H, D, I, S, E = cfg.hidden, cfg.n_heads * cfg.head_dim, cfg.moe_inter, cfg.n_shared, cfg.n_routed
    per_layer = (3 * D * H + H * D + E * H + 3 * S * I * H) * es + 2 * H * 4
    expert = 3 * I * H * es
    U = [len(np.unique(routes[l])) for l in range(cfg.n_layers)]
    w = cfg.n_layers * per_layer + sum(U) * expert + cfg.vocab * H * es + H * 4
    kv_row = cfg.n_layers * 2 * D * es
    kv = sum(int(n) for n in kv_len) * kv_row + B * (K + 1) * kv_row
    emb = B * (K + 1) * H * es
    return w + kv + emb, U


def draft_bytes(cfg, B, K, draft_len, n_rows):
    es = 2 if cfg.dtype == "bf16" else 4
    H, D, F = cfg.hidden, cfg.n_heads * cfg.head_dim, cfg.draft_inter
    block = (2 * H * H + 3 * D * H + H * D + 3 * F * H) * es
    lm = cfg.vocab * H * es
    kv_row = 2 * D * es
    kv = sum(int(n) for n in draft_len) * kv_row * K
    return K * (block + lm) + kv


def cpu_baseline(cfg, w, K, ctx_len, budget_s=20.0):
    """The oracle as it stands, timed on this host: speculative steps of one
    sequence from a synthetic cache of ctx_len positions (B=1)."""
    import oracle
    import synth
    orc = oracle.Oracle(cfg, w)
    cap = ctx_len + 64 * (K + 1) + 8
    kv, dkv = orc.new_kv(cap), orc.new_dkv(cap)
    for l in range(cfg.n_layers):
        for c in range(2):
            kv[l, c, :, :ctx_len] = _f32(synth.kv_values(cfg, l, 0, c, ctx_len, 15, 70), cfg)
    for c in range(2):
        dkv[c, :, :ctx_len - 1] = _f32(synth.kv_values(cfg, 0, 0, c, ctx_len - 1, 15, 71), cfg)
    hid = synth.normal(15, 72, (1, cfg.hidden))
    pend = int(synth.uniform_int(15, 73, 1, 0, cfg.vocab)[0])
    st = oracle.SeqState(kv=kv, dkv=dkv, kv_len=ctx_len, pending=pend, hid=hid,
                         next_tok=np.array([pend], np.int32), n_rows=1, row_pos=ctx_len - 1,
                         draft_len=ctx_len - 1, out=[pend])
    t0 = time.perf_counter()
    steps = toks = 0
    while time.perf_counter() - t0 < budget_s and steps < 64:
        info = oracle.spec_step(orc, st, K)
        steps += 1
        toks += info["m"] + 1
    dt = time.perf_counter() - t0
    return dict(value=toks / dt, unit="accepted tokens/s", cores=os.cpu_count(), kind="oracle",
                sample=f"{steps} speculative steps (K={K}, B=1) of the same model from a "
                       f"synthetic {ctx_len}-position cache, {dt:.1f} s, "
                       f"OMP threads={os.environ.get('OMP_NUM_THREADS', 'all')}, "
                       f"cpu={platform.processor() or platform.machine()}")


def _f32(a, cfg):
    import synth
    return synth.bf16_bits_to_f32(a) if cfg.dtype == "bf16" else a


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="b1", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true", help="time eager launches, not a HIP graph")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}); the decode step has no "
              "cross-GPU path in this build", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_2609_03181_amd import metrics
    from paper_2609_03181_amd.session import Model, Session

    wl = WORKLOADS[args.workload]
    cfg = synth.CONFIGS[wl["model"]]
    B, K = wl["B"], wl["K"]
    total_steps = args.warmup + args.steps + 8
    t0 = time.time()
    w = synth.make_weights(cfg, 0, 1, zipf_s=wl["zipf"])
    log(f"weights {time.time() - t0:.1f}s")

    if wl["synthetic"]:
        lo, hi, seed = wl["ctx"]
        ctx = synth.context_lengths(B, lo, hi, seed)
        max_ctx = int(ctx.max()) + total_steps * (K + 1) + 8
    else:
        P = wl["n_vis"] + wl["n_txt"]
        ctx = np.full(B, P, np.int32)
        max_ctx = P + total_steps * (K + 1) + 8
    max_out = total_steps * (K + 1) + 4
    model = Model(cfg, w, B, max_ctx, K)
    s = Session(model, B, K, max_out, prefill_rows=64)
    log(f"upload {time.time() - t0:.1f}s")

    if wl["synthetic"]:
        _load_synthetic(s, cfg, ctx)
    else:
        tok = np.full((B, P), -1, np.int32)
        vis = np.zeros((B, P, cfg.hidden), cfg.wdtype)
        for b in range(B):
            vis[b, :wl["n_vis"]] = synth.vision_prefix(cfg, wl["n_vis"], seed=10 + b)
            tok[b, wl["n_vis"]:] = synth.text_tokens(cfg, wl["n_txt"], seed=11 + b)
        vv = torch.from_numpy(vis.view(np.int16) if cfg.dtype == "bf16" else vis)
        torch.cuda.synchronize()
        tp = time.perf_counter()
        s.prefill(torch.from_numpy(tok), vv)
        torch.cuda.synchronize()
        log(f"prefill {B}x{P} rows: {1e3 * (time.perf_counter() - tp):.1f} ms")
    if wl["forced"]:
        s.set_forced_drafts(torch.from_numpy(_forced_table(s, cfg, B, K, total_steps)))
    assert s.status() == 0

    # ---- timed region: graph replays of whole steps
    if not args.eager:
        s.capture()
    run = s.step if args.eager else s.replay
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    n0 = s.n_out.clone()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        run()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t_start
    accepted = int((s.n_out - n0).sum().item())
    ms_step = 1e3 * dt / args.steps
    value = accepted / dt

    # ---- per-call breakdown (eager, events on the launch stream)
    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)
    nb = 8
    times = {"draft": [], "verify": [], "accept+commit": []}
    route_sets = []
    s_rec = s
    s_rec.route_idx = torch.zeros((cfg.n_layers, B * (K + 1), cfg.top_k), dtype=torch.int32,
                                  device="cuda")
    kv_lens, d_lens, n_rows = [], [], []
    for _ in range(nb):
        kv_lens.append(s.kv_len.cpu().numpy().copy())
        d_lens.append(s.row_pos.cpu().numpy() + s.n_rows.cpu().numpy())
        e = [ev() for _ in range(4)]
        e[0].record(stream)
        s.draft()
        e[1].record(stream)
        s.verify()
        e[2].record(stream)
        s.accept()
        s.commit()
        e[3].record(stream)
        torch.cuda.synchronize()
        times["draft"].append(e[0].elapsed_time(e[1]))
        times["verify"].append(e[1].elapsed_time(e[2]))
        times["accept+commit"].append(e[2].elapsed_time(e[3]))
        route_sets.append(s.route_idx.cpu().numpy().copy())
    s_rec.route_idx = None
    vb, U = zip(*[verify_bytes(cfg, B, K, kv_lens[i], route_sets[i]) for i in range(nb)])
    verify_ms = float(np.median(times["verify"]))
    vbytes = float(np.mean(vb))
    dbytes = float(np.mean([draft_bytes(cfg, B, K, d_lens[i], None) for i in range(nb)]))
    achieved = vbytes / (verify_ms * 1e-3) / 1e9
    assert s.status() == 0

    out = {
        "metric": "accepted tokens/s per GPU",
        "value": round(value, 2),
        "unit": "accepted tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic (seeded random-init weights, N(0,1) vision prefix, uniform tokens)",
        "config": {"workload": _wl_name(args.workload, wl), "batch": B, "k": K,
                   "mode": "eager" if args.eager else "hipgraph",
                   "tau": round(accepted / (args.steps * B), 4),
                   "verify_steps_per_s": round(args.steps / dt, 2)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": None, "kernel": "moe_verify_step (whole verify pass)",
                     "bytes_per_launch": int(vbytes), "ms_per_launch": round(verify_ms, 4),
                     "experts_touched_per_layer": round(float(np.mean(U)), 2)},
        "breakdown_ms": {k: round(float(np.median(v)), 4) for k, v in times.items()},
        "draft_bytes_per_step": int(dbytes),
    }
    if not args.no_cpu_baseline:
        ctx_cpu = int(min(int(ctx[0]), 768))
        out["cpu_baseline"] = cpu_baseline(cfg, w, K, ctx_cpu)
    print(json.dumps(out), flush=True)


def _wl_name(name, wl):
    if name == "b1":
        return ("full-shape MoE decoder (12 layers, d=1280, 64+2 experts top-6, V=129280) + "
                "FastMTP K=3, batch 1, 256 vision + 512 prompt rows prefilled")
    if name == "b16":
        return "full shape, batch 16, cached ctx U{1024..2048}, forced acceptance 0.2/0.2/0.25/0.35"
    if name == "b64":
        return "full shape, batch 64, cached ctx U{512..4096}, Zipf(1.1) router bias"
    return "tiny fp32 case (2 layers, d=256, 8 experts top-2, V=4096), K=3, batch 1"


def _load_synthetic(s, cfg, ctx):
    """Synthetic cached context: verifier/draft KV N(0,1) (seed 15), last
    commit states b N(0,1), pending tokens uniform (the same recipe the
    oracle side uses)."""
    import torch
    import synth
    B = len(ctx)
    for l in range(cfg.n_layers):
        for b in range(B):
            for c in range(2):
                v = synth.kv_values(cfg, l, b, c, int(ctx[b]), 15, 70)
                s.kv[l, b, c, :, :ctx[b]] = torch.from_numpy(v.view(np.int16) if v.dtype == np.uint16 else v).cuda()
    for b in range(B):
        for c in range(2):
            v = synth.kv_values(cfg, 0, b, c, int(ctx[b]) - 1, 15, 71)
            s.dkv[b, c, :, :ctx[b] - 1] = torch.from_numpy(v.view(np.int16) if v.dtype == np.uint16 else v).cuda()
    hid = synth.normal(15, 72, (B, cfg.hidden))
    pend = synth.uniform_int(15, 73, B, 0, cfg.vocab)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    s.kv_len.copy_(t(ctx))
    s.row_pos.copy_(t(ctx - 1))
    s.draft_len.copy_(t(ctx - 1))
    s.n_rows.fill_(1)
    s.pending.copy_(t(pend))
    s.next_tok[:, 0] = t(pend)
    s.hid[:, 0] = torch.from_numpy(hid).cuda()
    s.n_out.fill_(0)


def _forced_table(s, cfg, B, K, n_steps):
    """Forced acceptance for timing: m* ~ {0:0.2, 1:0.2, 2:0.25, 3:0.35}
    (seed 13).  The greedy trajectory of every sequence comes from a
    natural K-draft run on a copy of the state (lossless, and computed with
    the same kernels and row count as the timed steps); at each step drafts
    1..m* are the next trajectory tokens and draft m*+1 is a wrong one, so
    exactly m* are accepted."""
    import torch
    from paper_2609_03181_amd.session import Session
    import synth
    need = n_steps * (K + 1) + K + 2
    tr = Session(s.m, B, K, need, prefill_rows=1)
    for name in ("kv", "dkv", "kv_len", "row_pos", "draft_len", "n_rows", "pending", "hid",
                 "next_tok"):
        getattr(tr, name).copy_(getattr(s, name))
    tr.n_out.fill_(0)
    tr.max_new.fill_(need)
    while bool((tr.n_out < need).any()):
        tr.step()
    traj = tr.out_tok.cpu().numpy()
    del tr
    torch.cuda.synchronize()
    u = synth.uniform_f64(13, 80, n_steps * B).reshape(n_steps, B)
    m_star = np.minimum(np.searchsorted(np.cumsum([0.2, 0.2, 0.25, 0.35]), u), K)
    table = np.zeros((n_steps, B, K), np.int32)
    for b in range(B):
        base = 0
        for i in range(n_steps):
            d = [int(traj[b, min(base + t, need - 1)]) for t in range(K)]
            m = int(m_star[i, b])
            if m < K:
                d[m] = (d[m] + 1) % cfg.vocab
            table[i, b] = d
            base += m + 1
    return table


if __name__ == "__main__":
    main()

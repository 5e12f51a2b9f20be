"""Decoding-efficiency metrics of the speculative-decoding evaluation
(Section "Speculative decoding", Table "Decoding efficiency").

* tau: mean tokens committed per speculative step, bonus token included;
* acceptance rate: the position-averaged (tau - 1) / k;
* speedup S: output tok/s over the k = 0 baseline of the same mode;
* step cost c = tau / S, in units of one autoregressive step;
* a_d: probability that draft depth d is accepted given that all
  shallower depths were, so tau = 1 + a_1 + a_1 a_2 + ... .
"""
from __future__ import annotations

from typing import Sequence


def speedup(tok_s: float, tok_s_k0: float) -> float:
    return tok_s / tok_s_k0


def acceptance_rate(tau: float, k: int) -> float:
    return (tau - 1.0) / k


def step_cost(tau: float, s: float) -> float:
    return tau / s


def tau_from_conditional(a: Sequence[float]) -> float:
    tau, run = 1.0, 1.0
    for ad in a:
        run *= ad
        tau += run
    return tau


def tau_from_accept_lengths(ms: Sequence[int]) -> float:
    """mean of (m + 1) over speculative steps (m accepted drafts + 1)."""
    return sum(m + 1 for m in ms) / len(ms)


def conditional_acceptance(ms: Sequence[int], k: int) -> list:
    """a_d = #(m >= d) / #(m >= d - 1), d = 1..k (nan where undefined)."""
    out = []
    for d in range(1, k + 1):
        den = sum(1 for m in ms if m >= d - 1)
        num = sum(1 for m in ms if m >= d)
        out.append(num / den if den else float("nan"))
    return out

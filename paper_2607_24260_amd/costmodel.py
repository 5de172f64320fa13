"""The paper's cost model of plan-guided execution (Sec. 4), as a reporter.

Memory-bound costs: W_main / W_prop are the weight-read costs of one
main-model / proposal forward, KV the cost of reading the full KV cache;
s is the retained-KV ratio (Eq. (4)) and h the acceptance rate (Eq. (5)); a
cycle proposes k tokens and verifies them with the full context.

* Eq. (3):  Cost_full = W_main + KV
* Eq. (6):  Cost_base = (1 + k h)(W_main + KV)     (same expected output)
* Eq. (7):  Cost_plan = k (W_prop + s KV) + (W_main + KV)
* Eq. (8)-(9): Cost_plan < Cost_base  <=>  (h - s) KV > W_prop - h W_main
* Eq. (11)-(13) (self-speculation, W_prop = W_main): (h - s) KV > (1 - h) W_main,
  which needs h > s, and KV_crit = (1 - h) W_main / (h - s)
* Eq. (14): phase slack  Delta = h (W_main + KV) - (W_prop + s KV)

``measured`` puts measured attention call times in place of the idealised
memory costs for the attention-only path this library implements (no weight
reads): T_view per proposal step on the selected view, T_full per full-context
decode step, T_verify per verify window.
"""
from __future__ import annotations

import math
from dataclasses import dataclass


def cost_full(W_main: float, KV: float) -> float:
    return W_main + KV


def cost_base(k: float, h: float, W_main: float, KV: float) -> float:
    return (1.0 + k * h) * (W_main + KV)


def cost_plan(k: float, s: float, W_prop: float, W_main: float, KV: float) -> float:
    return k * (W_prop + s * KV) + (W_main + KV)


def phase_slack(h: float, s: float, W_prop: float, W_main: float, KV: float) -> float:
    return h * (W_main + KV) - (W_prop + s * KV)


def kv_crit(h: float, s: float, W_main: float) -> float:
    """Break-even KV scale of self-speculation (Eq. (13)); inf when h <= s."""
    return (1.0 - h) * W_main / (h - s) if h > s else math.inf


def expected_acceptance(gamma: int, p_stop: float = 0.6) -> float:
    """h = E[min(X, gamma)] / gamma for accept lengths X with
    P(X = j) = p_stop (1 - p_stop)^j: E[min(X, gamma)] = sum_{j=1..gamma} P(X >= j)."""
    q = 1.0 - p_stop
    return sum(q ** j for j in range(1, gamma + 1)) / gamma


@dataclass
class Report:
    k: int
    h: float
    s: float
    ideal_ratio: float         # Cost_plan / Cost_base, attention only (W = 0)
    measured_ratio: float      # the same with measured call times
    h_minus_s: float

    def as_dict(self) -> dict:
        return {"k": self.k, "h": round(self.h, 5), "s": round(self.s, 5),
                "h_minus_s": round(self.h_minus_s, 5),
                "ideal_cost_ratio_attention": round(self.ideal_ratio, 4),
                "ideal_speedup_attention": round(1.0 / self.ideal_ratio, 3),
                "measured_cost_ratio_attention": round(self.measured_ratio, 4),
                "measured_speedup_attention": round(1.0 / self.measured_ratio, 3)}


def measured(k: int, h: float, s: float, T_view: float, T_full: float, T_verify: float) -> Report:
    """Attention-only cycle: k proposal steps on the view and one verify
    against (1 + k h) full-context decode steps for the same expected output."""
    ideal = cost_plan(k, s, 0.0, 0.0, 1.0) / cost_base(k, h, 0.0, 1.0)
    meas = (k * T_view + T_verify) / ((1.0 + k * h) * T_full)
    return Report(k, h, s, ideal, meas, h - s)

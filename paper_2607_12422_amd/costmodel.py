"""Speculation cost model and draft-cost analysis (host-side reporting).

Sec. 3 cost model: a speculative round that commits A tokens at draft cost
C_d and verify cost C_v is worthwhile only if (C_d + C_v) / A is below the
cost per token of the target model alone.

App. A.7 (repeated runs and draft-cost analysis): with measured iteration
time T0 and draft-side cost share rho_d, removing a fraction r of the draft
cost gives T(r) = T0 * (1 - r * rho_d) with the acceptance held fixed; the
predicted throughput is A / T(r), and the accepted tokens per round needed to
match a baseline of throughput X is X * T(r).
"""
from __future__ import annotations

from dataclasses import dataclass


def cost_per_token(c_draft: float, c_verify: float, accepted: float) -> float:
    """(C_d + C_v) / A of the Sec. 3 cost model."""
    return (c_draft + c_verify) / accepted


def draft_share(t_draft: float, t_verify: float) -> float:
    """rho_d: the draft pass's share of draft + verify time."""
    return t_draft / (t_draft + t_verify)


def reduced_iteration_time(t0: float, rho_d: float, r: float) -> float:
    """T(r) = T0 (1 - r rho_d), r in [0, 1]."""
    if not 0.0 <= r <= 1.0:
        raise ValueError("draft-cost reduction r must lie in [0, 1]")
    return t0 * (1.0 - r * rho_d)


@dataclass(frozen=True)
class DraftCostRow:
    reduction: float
    tokens_per_s: float
    need_vs: tuple          # accepted tokens per round needed to match each baseline


def draft_cost_table(accepted: float, tokens_per_s: float, t_draft: float,
                     t_verify: float, baselines=(), reductions=(0, .25, .5, .75, .9, 1.0)):
    """Rows of the draft-cost analysis.

    T0 = accepted / tokens_per_s (the measured iteration time); rho_d from the
    draft/verify pass times; each baseline is a throughput in tokens/s.
    """
    t0 = accepted / tokens_per_s
    rho = draft_share(t_draft, t_verify)
    rows = []
    for r in reductions:
        tr = reduced_iteration_time(t0, rho, r)
        rows.append(DraftCostRow(r, accepted / tr, tuple(b * tr for b in baselines)))
    return rows

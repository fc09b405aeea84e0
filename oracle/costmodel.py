"""Oracle of the speculative-decoding cost model (Sec. 3.1 Eq. 1-2, Sec. 4.1
Eq. 3-4).

TEST INFRASTRUCTURE ONLY: only ``tests/`` may use this module.  It shares no
code with the library's cost model.

Notation (per decoding step of a batch B at sequence length S):
  T_T       target decoding time (one token per sequence),
  T_D       draft decoding time per drafted token,
  T_select  KV-selection time per drafted token (Eq. 3; 0 for static
            selections such as StreamingLLM and SnapKV),
  T_V(g)    time to verify g speculated tokens,
  alpha     draft acceptance rate, gamma the speculation length.
"""
import math


def expected_tokens(gamma, alpha):
    """Eq. 1: Omega(gamma, alpha) = (1 - alpha^(gamma+1)) / (1 - alpha),
    continued to gamma + 1 at alpha = 1."""
    if alpha == 1.0:
        return float(gamma + 1)
    return (1.0 - alpha ** (gamma + 1)) / (1.0 - alpha)


def draft_time(t_draft, t_select=0.0):
    """Eq. 3: draft time with a KV budget, decoding plus selection."""
    return t_draft + t_select


def step_time(gamma, t_draft, t_verify, t_select=0.0):
    """T_Total^SD = gamma * T_D + T_V(gamma) (Sec. 3.1), T_D from Eq. 3."""
    return gamma * draft_time(t_draft, t_select) + t_verify


def latency_ratio(gamma, alpha, t_target, t_draft, t_verify, t_select=0.0):
    """Eq. 2 (with Eq. 3): T_Avg^SD / T_T = (gamma T_D / T_T + T_V / T_T) / Omega."""
    return step_time(gamma, t_draft, t_verify, t_select) / (
        expected_tokens(gamma, alpha) * t_target)


def best_gamma(alpha, t_target, t_draft, t_verify_by_gamma, t_select=0.0):
    """Eq. 4 over gamma (the budget and selection fixed): the gamma in
    1 .. len(t_verify_by_gamma) minimising Eq. 2, by trying each;
    t_verify_by_gamma[g - 1] = T_V(g).  Ties: the smaller gamma.
    Returns (gamma, ratio)."""
    best = None
    for g, tv in enumerate(t_verify_by_gamma, start=1):
        r = latency_ratio(g, alpha, t_target, t_draft, tv, t_select)
        if best is None or r < best[1]:
            best = (g, r)
    return best


def alpha_from_omega(gamma, omega, iters=200):
    """The alpha in [0, 1] with Omega(gamma, alpha) = omega (Eq. 1 is
    increasing in alpha from 1 to gamma + 1), by bisection."""
    if not 1.0 <= omega <= gamma + 1:
        return math.nan
    lo, hi = 0.0, 1.0
    for _ in range(iters):
        mid = 0.5 * (lo + hi)
        if expected_tokens(gamma, mid) < omega:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)

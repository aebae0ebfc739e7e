"""Stage performance model of the disaggregated Encoder -> Transformer ->
Decoder pipeline (paper: System Design, Hybrid-Strategy Instance Scheduling).

Each stage runs on instances that each occupy one GPU; g_E, g_T and g_D GPUs
go to the three stages with

    g_E + g_T + g_D <= G                      (GPU budget)
    S_M + S_A < C                             (per-GPU memory: model + activations)

A request's time in a stage is compute plus the time to move its activations:

    T_E = S_A,E I_E / P_E + S_A,E / B_E
    T_T = S_A,T I_T / P_T + S_A,T1 / B_T1 + S_A,T2 / B_T2
    T_D = S_A,D I_D / P_D + S_A,D / B_D

(S_A activation bytes, I compute intensity in FLOPs per byte -- so S_A I is
the stage's FLOPs --, P achieved FLOP/s, B bandwidth; the Transformer receives
from the encoder and sends to the decoder).  End-to-end throughput is set by
the slowest stage,

    QPS = min(g_E / T_E, g_T / T_T, g_D / T_D),

and a good allocation balances the three service rates.

Host-side planning code: it runs no kernels.  The DiT stage's time can be
calibrated with the measured per-step time of this library (the Transformer
stage runs n_steps DiT steps per request).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, Iterable, Optional, Sequence, Tuple

STAGES = ("E", "T", "D")


@dataclass(frozen=True)
class StageCost:
    """Per-request cost of one stage on one GPU (SI units: bytes, FLOPs/byte,
    FLOP/s, bytes/s).  `comm` lists the activation transfers the stage makes
    per request as (bytes, bytes/s) pairs (one for E and D; two for T, in and
    out)."""
    act_bytes: float                 # S_A
    intensity: float                 # I, FLOPs per activation byte
    perf: float                      # P, achieved FLOP/s
    comm: Tuple[Tuple[float, float], ...] = ()   # ((bytes, bytes/s), ...)
    model_bytes: float = 0.0         # S_M

    def time(self) -> float:
        """T = S_A I / P + sum(bytes / B) (the stage-time equations)."""
        t = self.act_bytes * self.intensity / self.perf
        for nbytes, bw in self.comm:
            t += nbytes / bw
        return t

    def fits(self, capacity_bytes: float) -> bool:
        """S_M + S_A < C."""
        return self.model_bytes + self.act_bytes < capacity_bytes


def qps(alloc: Dict[str, int], times: Dict[str, float]) -> float:
    """min over stages of g / T (requests per second); 0 when a stage has no GPU."""
    return min((alloc[s] / times[s]) if alloc[s] > 0 else 0.0 for s in STAGES)


def bottleneck(alloc: Dict[str, int], times: Dict[str, float]) -> str:
    """The stage whose service rate sets the throughput."""
    return min(STAGES, key=lambda s: (alloc[s] / times[s]) if alloc[s] > 0 else 0.0)


def allocations(G: int, min_per_stage: int = 1) -> Iterable[Dict[str, int]]:
    """Every (g_E, g_T, g_D) with g_E + g_T + g_D <= G and each >= min_per_stage."""
    for gE in range(min_per_stage, G + 1):
        for gT in range(min_per_stage, G - gE + 1):
            for gD in range(min_per_stage, G - gE - gT + 1):
                yield {"E": gE, "T": gT, "D": gD}


def best_allocation(G: int, times: Dict[str, float],
                    candidates: Optional[Sequence[Dict[str, int]]] = None) -> Tuple[Dict[str, int], float]:
    """Allocation of at most G GPUs with the highest QPS (ties: fewest GPUs,
    then the first in enumeration order).  `candidates` restricts the search,
    e.g. to a set of static configurations."""
    pool = list(candidates) if candidates is not None else list(allocations(G))
    best = max(pool, key=lambda a: (qps(a, times), -sum(a.values())))
    return best, qps(best, times)


def transformer_time(n_steps: int, step_seconds: float, act_in: Tuple[float, float] = (0.0, 1.0),
                     act_out: Tuple[float, float] = (0.0, 1.0)) -> float:
    """T_T calibrated with a measured DiT step time: n_steps steps of compute
    plus the two activation transfers ((bytes, bytes/s) in and out)."""
    return n_steps * step_seconds + act_in[0] / act_in[1] + act_out[0] / act_out[1]


def per_minute(q: float) -> float:
    """requests per second -> requests per minute (QPM)."""
    return 60.0 * q


def ratios(alloc: Dict[str, int]) -> str:
    return ":".join(str(alloc[s]) for s in STAGES)


def sweep(G: int, cases: Dict[str, Dict[str, float]]) -> Dict[str, Tuple[str, float, str]]:
    """For each named workload (stage times), the best allocation, its QPM and
    its bottleneck stage."""
    out = {}
    for name, times in cases.items():
        a, q = best_allocation(G, times)
        out[name] = (ratios(a), per_minute(q), bottleneck(a, times))
    return out


__all__ = ["StageCost", "qps", "bottleneck", "allocations", "best_allocation", "transformer_time", "per_minute",
           "ratios", "sweep", "STAGES"]

"""Routing telemetry and the HOT-set rebalancer (paper section IV-D).

Pure host logic, no device calls.  The library's native runtime
(mira_stack_*, mira_rebalance_plan) makes these decisions on the GPU path;
this module states them in plain Python as the reference its tests compare
the native planner with, and carries the settings (RebalanceConfig) the
Python stack passes to the runtime.

Telemetry (per layer and expert, over the current window of tokens): tokens
routed to the expert, and of those how many were served from a HOT slot, from
a STAGE slot or by a copy from the CPU store.  The window is reset after each
rebalancing pass; a short history of past windows is kept for probation.

Rebalancing pass (every `interval` tokens of a layer):
  1. victim score of every HOT expert: low routed volume in the window first,
     then the longest time since its last use (recency), then the lowest
     volume over the remembered windows (frequency);
  2. candidate score of every non-HOT expert with traffic in the window:
     routed volume plus `miss_weight` times its CPU-served tokens (high demand
     and a high cost of a miss); an expert is a candidate only after
     `probation` consecutive windows with traffic (the STAGE region is its
     probation area), so a burst does not buy residency;
  3. bounded swaps: at most `max_swaps` per layer and pass, each only while the
     candidate's score beats the victim's window volume by `margin`.
"""
from __future__ import annotations

from collections import deque
from dataclasses import dataclass, field


@dataclass
class ExpertStats:
    routed: int = 0        # tokens routed in the current window
    hot: int = 0           # ... served from a HOT slot
    stage: int = 0         # ... served from a STAGE slot
    cpu: int = 0           # ... served by a copy from the CPU store (a miss)
    last_use: int = -1     # token clock of the last use
    history: deque = field(default_factory=lambda: deque(maxlen=8))  # routed volume of past windows


class Telemetry:
    """Token-level accounting of one layer's experts."""

    def __init__(self, n_experts: int):
        self.stats = [ExpertStats() for _ in range(n_experts)]
        self.tokens = 0       # tokens of the current window
        self.clock = 0        # tokens since the start

    def record(self, expert: int, tokens: int, tier: str):
        s = self.stats[expert]
        s.routed += tokens
        if tier == "hot":
            s.hot += tokens
        elif tier == "stage":
            s.stage += tokens
        elif tier == "cpu":
            s.cpu += tokens
        else:
            raise ValueError(f"unknown tier {tier!r}")
        s.last_use = self.clock

    def advance(self, tokens: int):
        """The layer processed `tokens` more tokens."""
        self.tokens += tokens
        self.clock += tokens

    def close_window(self):
        for s in self.stats:
            s.history.append(s.routed)
            s.routed = s.hot = s.stage = s.cpu = 0
        self.tokens = 0


@dataclass
class RebalanceConfig:
    interval: int = 64      # tokens of a layer between passes
    max_swaps: int = 1      # swaps per layer and pass
    probation: int = 2      # consecutive windows with traffic before a promotion
    miss_weight: float = 1.0
    margin: int = 1         # a candidate must beat the victim's window volume by this much


@dataclass
class Swap:
    evict: int
    promote: int


class Rebalancer:
    """Decides, per layer, which HOT expert to evict for which candidate."""

    def __init__(self, cfg: RebalanceConfig):
        self.cfg = cfg

    def victim_key(self, tel: Telemetry, e: int):
        s = tel.stats[e]
        return (s.routed, s.last_use, sum(s.history))  # ascending = better victim

    def candidate_score(self, tel: Telemetry, e: int) -> float:
        s = tel.stats[e]
        return s.routed + self.cfg.miss_weight * s.cpu

    def on_probation(self, tel: Telemetry, e: int) -> bool:
        """True while the expert has not shown traffic in `probation`
        consecutive windows (the current one included)."""
        s = tel.stats[e]
        if s.routed == 0:
            return True
        need = self.cfg.probation - 1
        past = list(s.history)[-need:] if need > 0 else []
        return len(past) < need or any(v == 0 for v in past)

    def due(self, tel: Telemetry) -> bool:
        return tel.tokens >= self.cfg.interval

    def plan(self, tel: Telemetry, hot: set) -> list:
        """Swaps for one pass; the caller applies them and closes the window."""
        victims = sorted(hot, key=lambda e: (*self.victim_key(tel, e), e))
        cands = [e for e in range(len(tel.stats))
                 if e not in hot and tel.stats[e].routed > 0 and not self.on_probation(tel, e)]
        cands.sort(key=lambda e: (-self.candidate_score(tel, e), e))
        swaps = []
        for v, c in zip(victims, cands):
            if len(swaps) >= self.cfg.max_swaps:
                break
            if self.candidate_score(tel, c) < tel.stats[v].routed + self.cfg.margin:
                break
            swaps.append(Swap(evict=v, promote=c))
        return swaps

"""Oracle of the layer's model metrics and the host policies that act on
them.  TEST INFRASTRUCTURE ONLY (see the package docstring): nothing in the
product path imports this module.

* Section 4.2 (sample assignment caching): the Cache operator's metric, the
  number of samples whose assignment did not change since the cached one,
  and the cache update that stores the fresh assignment for the next epoch.
* Section 5.3 (caching results): caching is switched on once at least 96% of
  the samples are correctly cached and not before epoch 10, and switched off
  when that share falls below 90%.
* Section 3 (the recompile mechanism) with its implementation appendix:
  a model metric produced at the execution frontier drives a user trigger
  that alters the graph at the launch frontier, Delta_launch iterations
  later; Section 4.1 applies it to per-expert capacities computed from the
  observed per-expert assignment counts.

Readings taken here (each also stated where it is used):
C1 A sample is correctly cached when the set of experts the gate picks for
   it equals the cached set (order among the k picks does not matter).
C2 The caching decision is taken once per epoch from the epoch's totals of
   correctly cached samples and samples; the thresholds compare the exact
   fraction (integer arithmetic).
P1 Launch of iteration i first waits until at most Delta iterations are
   launched and unexecuted; the trigger then sees the counts of iteration
   i - 1 - Delta (none for i <= Delta, when the capacities stay as they are).
P2 The trigger recompiles when the counts it sees would overflow a current
   capacity (drops) or when a current capacity exceeds ceil(shrink * count)
   clamped to [cap_min, T]; a recompile sets every expert's capacity to
   ceil(grow * count), clamped the same way (grow <= shrink, so a recompile
   never leaves a capacity that the next identical metric would shrink).
   Iteration 0 uses the static capacity of Eq. 4.
P3 Drops of an iteration are sum_e max(0, counts_e - C_e); its capacity
   factor is sum_e C_e / (T k), 1.0 being exactly the demand on average.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

from .moe_oracle import capacity_dynamic

__all__ = ["cache_unchanged", "cache_update", "caching_decision",
           "capacity_policy_trigger", "simulate_capacity_policy"]


def cache_unchanged(fresh_ids: np.ndarray, cached_ids: np.ndarray) -> np.ndarray:
    """Per sample: True when the gate's fresh picks are the cached picks as
    a set (C1)."""
    fresh = np.asarray(fresh_ids)
    cached = np.asarray(cached_ids)
    return np.array([set(fresh[t].tolist()) == set(cached[t].tolist())
                     for t in range(fresh.shape[0])], dtype=bool)


def cache_update(fresh_ids: np.ndarray, cache: np.ndarray) -> Tuple[int, np.ndarray]:
    """The Cache operator on one mini-batch: count the correctly cached
    samples, then remember the fresh picks for the next epoch."""
    n = int(cache_unchanged(fresh_ids, cache).sum())
    return n, np.array(fresh_ids, dtype=np.int32, copy=True)


def caching_decision(enabled: bool, unchanged: int, samples: int, epoch: int,
                     on: Tuple[int, int] = (96, 100), off: Tuple[int, int] = (90, 100),
                     min_epoch: int = 10) -> bool:
    """Hysteresis of Section 5.3 (C2): switch on at unchanged/samples >= on
    once epoch >= min_epoch, switch off at unchanged/samples < off."""
    if samples <= 0:
        return enabled
    if enabled:
        return not (unchanged * off[1] < off[0] * samples)
    return epoch >= min_epoch and unchanged * on[1] >= on[0] * samples


def _ceil_mul(num: int, den: int, c: int) -> int:
    return (num * c + den - 1) // den


def capacity_policy_trigger(cap: Sequence[int], counts: Sequence[int], T: int,
                            grow: Tuple[int, int], shrink: Tuple[int, int],
                            cap_min: int) -> Tuple[List[int], bool]:
    """One trigger call (P2): returns (capacities for the next launch,
    whether a recompile happened)."""
    if grow[0] * shrink[1] > shrink[0] * grow[1]:
        raise ValueError("grow must not exceed shrink")
    cap = [int(c) for c in cap]
    counts = [int(c) for c in counts]
    over = any(c > C for c, C in zip(counts, cap))
    loose = any(C > min(T, max(cap_min, _ceil_mul(shrink[0], shrink[1], c)))
                for c, C in zip(counts, cap))
    if not (over or loose):
        return cap, False
    return [int(v) for v in capacity_dynamic(counts, T, grow[0], grow[1], cap_min)], True


def simulate_capacity_policy(counts_seq: Sequence[Sequence[int]], T: int, k: int,
                             delta: int, init_cap: Sequence[int],
                             grow: Tuple[int, int], shrink: Tuple[int, int],
                             cap_min: int = 0) -> Dict[str, np.ndarray]:
    """Run the policy over a sequence of per-iteration demand counts (P1-P3).

    Returns caps [N, E] (capacities each iteration ran with), recompile [N]
    (whether the trigger before iteration i recompiled), drops [N] and
    factor [N]."""
    N = len(counts_seq)
    cap = [int(c) for c in init_cap]
    caps, rec, drops, factor = [], [], [], []
    for i in range(N):
        changed = False
        src = i - 1 - delta
        if src >= 0:
            cap, changed = capacity_policy_trigger(cap, counts_seq[src], T, grow, shrink, cap_min)
        caps.append(list(cap))
        rec.append(changed)
        c = [int(v) for v in counts_seq[i]]
        drops.append(sum(max(0, ci - Ci) for ci, Ci in zip(c, cap)))
        factor.append(sum(cap) / float(T * k))
    return dict(caps=np.array(caps, dtype=np.int64), recompile=np.array(rec, dtype=bool),
                drops=np.array(drops, dtype=np.int64), factor=np.array(factor))

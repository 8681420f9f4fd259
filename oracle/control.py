"""Plain oracle for the cache's control plane: carbon model, replacement
policies on request traces, and the cache-size ILP.

TEST INFRASTRUCTURE. Only tests/ and the benchmark's CPU-baseline leg may
import this module. The product (paper_2505_23970_amd/control.py and
csrc/cache_policy.cpp) shares no code with it.

Carbon model, GreenCache §2.3 (Eqs. 1-3) and §3.2.1 (Eqs. 4-5):
  total carbon C = C_o + (T / LT) * C_e                         (Eq. 1)
  operational C_o = E * CI                                       (Eq. 2)
  embodied C_e = sum over GPU, CPU, memory, SSD                  (Eq. 3)
  cache embodied C_e,cache = S_alloc * (T / LT) * C_e,SSD^unit   (Eq. 4)
  C = E * CI + C_e,cache + (T / LT) * C_e,others                 (Eq. 5)
Units here: energy in kWh, CI in gCO2e/kWh, embodied carbon in kgCO2e
(converted to grams), times in hours, lifetimes in years (365 days).

Replacement policies, §5.5 (Eq. 7 LCS score, Eq. 8 multi-turn form) and the
FIFO / LRU baselines of §6.3.2 (Table tab:replacement), on the cache model stated in
include/greencache_ctl.h (the model is a reading: the paper states the score,
not the bookkeeping). Each eviction sorts every candidate entry by
(score, insertion time, key) and removes the first: slow and obviously right.

Cache-size ILP, §5.4.1 Eq. 6, with one cache size per time step chosen from a
discrete set: minimise the summed per-request carbon subject to at least
rho * N requests meeting the TTFT SLO and at least rho * N meeting the TPOT
SLO. Solved here by enumerating every assignment (tiny instances only).
"""
from __future__ import annotations

import itertools
import math

HOURS_PER_YEAR = 365.0 * 24.0


# ----------------------------------------------------------------- carbon model

def operational_g(energy_kwh, ci_g_per_kwh):
    """Eq. 2."""
    return energy_kwh * ci_g_per_kwh


def amortised_g(hours, lifetime_years, embodied_kg):
    """(T / LT) * C_e of Eq. 1, in grams."""
    return hours / (lifetime_years * HOURS_PER_YEAR) * embodied_kg * 1000.0


def cache_embodied_g(size_tb, hours, lifetime_years, ssd_kg_per_tb):
    """Eq. 4."""
    return size_tb * amortised_g(hours, lifetime_years, ssd_kg_per_tb)


def total_g(energy_kwh, ci, hours, size_tb, ssd_kg_per_tb, ssd_lifetime_years, others):
    """Eq. 5. others: iterable of (embodied_kg, lifetime_years) for GPU, CPU, memory."""
    return (operational_g(energy_kwh, ci) + cache_embodied_g(size_tb, hours, ssd_lifetime_years, ssd_kg_per_tb)
            + sum(amortised_g(hours, lt, kg) for kg, lt in others))


def request_carbon_g(power_w, ttft_s, ci, size_tb, ssd_kg_per_tb, ssd_lifetime_years, others):
    """The per-request term of Eq. 6: operational p * TTFT * CI, cache embodied
    TTFT / LT_SSD * S * C_unit, other embodied sum TTFT / LT_comp * C_comp."""
    hours = ttft_s / 3600.0
    energy_kwh = power_w * ttft_s / 3.6e6
    return total_g(energy_kwh, ci, hours, size_tb, ssd_kg_per_tb, ssd_lifetime_years, others)


# ----------------------------------------------------------------- replacement policies

FIFO, LRU, LCS, LCS_MULTITURN = 0, 1, 2, 3
MIN_AGE = 1e-6


class Cache:
    def __init__(self, policy, capacity_bytes, bytes_per_token):
        self.policy = policy
        self.capacity = capacity_bytes
        self.bpt = bytes_per_token
        self.entries = {}  # key -> dict(tokens, hits, acc, turn, t_ins, t_last)
        self.requests = self.hits = self.reused = self.prompt = 0
        self.insertions = self.evictions = 0

    def bytes(self):
        return sum(e["tokens"] * self.bpt for e in self.entries.values())

    def _rank(self, key, now):
        e = self.entries[key]
        if self.policy == FIFO:
            return (e["t_ins"], key)
        if self.policy == LRU:
            return (e["t_last"], key)
        age = max(now - e["t_ins"], MIN_AGE)
        size = float(e["tokens"] * self.bpt)
        if self.policy == LCS:
            score = (float(e["acc"]) * float(e["hits"])) / (size * age)
        else:
            score = (float(e["turn"]) * float(e["acc"])) / (size * age)
        return (score, e["t_ins"], key)

    def _fit(self, keep, now):
        if keep is not None and keep in self.entries:
            if self.entries[keep]["tokens"] * self.bpt > self.capacity:
                del self.entries[keep]
                self.evictions += 1
        while self.bytes() > self.capacity:
            cands = sorted((k for k in self.entries if k != keep), key=lambda k: self._rank(k, now))
            if not cands:
                break
            del self.entries[cands[0]]
            self.evictions += 1

    def access(self, key, context, prompt, total, turn, now):
        self.requests += 1
        self.prompt += prompt
        e = self.entries.get(key)
        reused = 0
        if e is not None:
            reused = min(context, e["tokens"])
            self.hits += 1
            self.reused += reused
            e["hits"] += 1
            e["acc"] += reused
            e["turn"] = turn
            e["t_last"] = now
            e["tokens"] = max(e["tokens"], total)
        else:
            self.entries[key] = dict(tokens=total, hits=0, acc=0, turn=turn, t_ins=now, t_last=now)
            self.insertions += 1
        self._fit(key, now)
        return reused

    def resize(self, capacity_bytes, now):
        self.capacity = capacity_bytes
        self._fit(None, now)


def replay(policy, capacity_bytes, bytes_per_token, requests):
    """requests: iterable of (key, context, prompt, total, turn, time). Returns
    (reused tokens per request, the cache)."""
    c = Cache(policy, capacity_bytes, bytes_per_token)
    out = [c.access(k, ctx, pr, tot, turn, t) for k, ctx, pr, tot, turn, t in requests]
    return out, c


# ----------------------------------------------------------------- cache-size ILP

def solve_sizes_bruteforce(cost, ok_ttft, ok_tpot, n_requests, rho):
    """cost[t][s]: carbon of time step t with size choice s; ok_*[t][s]: requests of
    step t meeting the SLO with choice s. Returns (best cost, choice per step) or
    (inf, None) when no assignment meets both attainment constraints. Ties: the
    lexicographically smallest choice vector."""
    T = len(cost)
    S = len(cost[0])
    need = rho * n_requests
    best, arg = math.inf, None
    for choice in itertools.product(range(S), repeat=T):
        if sum(ok_ttft[t][s] for t, s in enumerate(choice)) < need:
            continue
        if sum(ok_tpot[t][s] for t, s in enumerate(choice)) < need:
            continue
        c = sum(cost[t][s] for t, s in enumerate(choice))
        if c < best:
            best, arg = c, list(choice)
    return best, arg

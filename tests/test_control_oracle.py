"""The control-plane oracle (oracle/control.py) against pins that are not its own
code (CPU only): textbook replacement results, a hand-worked LCS example,
carbon-model invariants, and the paper's own 0-1 knapsack construction for the
cache-size ILP (appendix, NP-hardness proof) checked against a textbook DP."""
import json
import math
import os

import numpy as np
import pytest

from oracle import control as C0

HERE = os.path.dirname(os.path.abspath(__file__))
BELADY = [1, 2, 3, 4, 1, 2, 5, 1, 2, 3, 4, 5]


def unit_trace(keys):
    # unit-size entries: each request reuses its one token when cached
    return [(k, 1, 1, 1, 1, float(i)) for i, k in enumerate(keys)]


def faults(policy, frames, keys, C=C0):
    reused, _ = C.replay(policy, frames, 1, unit_trace(keys))
    return sum(1 for r in reused if r == 0)


def test_fifo_shows_beladys_anomaly(C=C0):
    """Belady, Nelson and Shedler (1969): FIFO on 1,2,3,4,1,2,5,1,2,3,4,5 faults 9
    times with 3 frames and 10 times with 4."""
    assert faults(C.FIFO, 3, BELADY, C) == 9
    assert faults(C.FIFO, 4, BELADY, C) == 10


def test_lru_textbook_fault_counts(C=C0):
    """LRU on the same string: 10 faults with 3 frames, 8 with 4."""
    assert faults(C.LRU, 3, BELADY, C) == 10
    assert faults(C.LRU, 4, BELADY, C) == 8


def test_lru_is_a_stack_algorithm(C=C0):
    """LRU's inclusion property: more capacity never loses a hit."""
    rng = np.random.default_rng(3)
    keys = list(rng.zipf(1.3, 400) % 40)
    hits = [400 - faults(C.LRU, c, keys, C) for c in range(1, 30)]
    assert all(a <= b for a, b in zip(hits, hits[1:]))


def test_lcs_hand_worked_example(C=C0):
    g = json.load(open(os.path.join(HERE, "golden", "lcs_example.json")))
    reqs = [(q["key"], q["context"], q["prompt"], q["total"], q["turn"], q["time"]) for q in g["requests"]]
    for name, pol in (("lcs", C.LCS), ("fifo", C.FIFO), ("lru", C.LRU)):
        reused, cache = C.replay(pol, 100, 1, reqs)
        assert reused == g["expected"][name]["reused"], name
        assert sorted(cache.entries) == g["expected"][name]["keys_after"], name


POLICY_NAMES = {"fifo": 0, "lru": 1, "lcs": 2, "lcs_multiturn": 3}


@pytest.mark.parametrize("case", range(5))
def test_hand_worked_sensitivity_cases(case, C=C0):
    """Each case separates the right score from a plausible wrong one (size, age,
    reused tokens, turn vs hits) or checks entry growth and partial reuse; the
    expected outcome is worked by hand in the golden file."""
    g = json.load(open(os.path.join(HERE, "golden", "lcs_example.json")))["cases"][case]
    reqs = [(q["key"], q["context"], q["prompt"], q["total"], q["turn"], q["time"]) for q in g["requests"]]
    reused, cache = C.replay(POLICY_NAMES[g["policy"]], g["capacity"], 1, reqs)
    if "resize" in g:
        cache.resize(g["resize"]["capacity"], g["resize"]["time"])
    if "expected_reused" in g:
        assert reused == g["expected_reused"], g["name"]
    assert sorted(cache.entries) == g["expected_keys_after"], g["name"]


def test_ilp_tpot_constraint_binds(C=C0):
    """Hand-worked: 2 steps of 10 requests, rho 0.9 (18 of 20 must meet each SLO).
    Step 0: choice 0 costs 1 with 10 TTFT / 2 TPOT successes, choice 1 costs 3 with
    10 / 10. Step 1: choice 0 costs 1 with 10 / 10, choice 1 costs 3 with 10 / 10.
    Choosing 0 twice (cost 2) meets TTFT (20) but not TPOT (12); the optimum is
    (1, 0) at cost 4."""
    best, choice = C.solve_sizes_bruteforce([[1.0, 3.0], [1.0, 3.0]], [[10, 10], [10, 10]],
                                            [[2, 10], [10, 10]], 20, 0.9)
    assert best == 4.0 and choice == [1, 0]


def test_lcs_without_hits_degenerates_to_fifo(C=C0):
    """Entries that were never hit all score 0; the tie-break (earlier insertion)
    then makes LCS evict exactly as FIFO does."""
    rng = np.random.default_rng(4)
    keys = list(rng.permutation(60))  # every key once: no hits at all
    reqs = [(int(k), 0, 5, 5 + int(k) % 7, 1, float(i)) for i, k in enumerate(keys)]
    _, a = C.replay(C.LCS, 200, 1, reqs)
    _, b = C.replay(C.FIFO, 200, 1, reqs)
    assert sorted(a.entries) == sorted(b.entries)


def test_multiturn_score_prefers_deeper_turns(C=C0):
    """Eq. 8: two entries equal in reuse, size and age; the one deeper in its
    conversation stays."""
    reqs = [(1, 0, 10, 20, 1, 0.0), (2, 0, 10, 20, 1, 0.0),
            (1, 20, 25, 20, 2, 1.0), (2, 20, 25, 20, 5, 1.0),
            (3, 0, 10, 20, 1, 2.0)]
    _, c = C.replay(C.LCS_MULTITURN, 40, 1, reqs)
    assert sorted(c.entries) == [2, 3]


def test_oversized_entry_is_dropped_without_evicting_others(C=C0):
    reqs = [(1, 0, 5, 10, 1, 0.0), (2, 0, 5, 50, 1, 1.0)]
    reused, c = C.replay(C.LRU, 20, 1, reqs)
    assert sorted(c.entries) == [1] and c.evictions == 1


def test_resize_evicts_by_policy(C=C0):
    reqs = [(1, 0, 5, 10, 1, 0.0), (2, 0, 5, 10, 1, 1.0), (1, 10, 12, 10, 2, 2.0)]
    _, c = C.replay(C.LRU, 30, 1, reqs)
    c.resize(10, 3.0)
    assert sorted(c.entries) == [1]


# ----------------------------------------------------------------- carbon model

def test_amortised_share_over_the_whole_lifetime_is_the_whole_embodied_carbon(C=C0):
    """Eq. 1: with T = LT the embodied term is C_e itself."""
    assert math.isclose(C.amortised_g(5 * C.HOURS_PER_YEAR, 5, 106.4), 106400.0, rel_tol=1e-12)


def test_carbon_is_additive_over_time_and_capacity(C=C0):
    a = C.cache_embodied_g(3, 2.0, 5, 30) + C.cache_embodied_g(3, 5.0, 5, 30)
    b = C.cache_embodied_g(3, 7.0, 5, 30)
    assert math.isclose(a, b, rel_tol=1e-12)
    assert math.isclose(C.cache_embodied_g(16, 1.0, 5, 30), 16 * C.cache_embodied_g(1, 1.0, 5, 30), rel_tol=1e-12)


def test_ssd_table_entry_per_terabyte(C=C0):
    """Table 1: up to 16 TB of SSD carry up to 480 kgCO2e; with 30 kg/TB the full
    16 TB over its 5-year lifetime amortise to exactly 480 kg."""
    assert math.isclose(C.cache_embodied_g(16, 5 * C.HOURS_PER_YEAR, 5, 480 / 16), 480e3, rel_tol=1e-12)


def test_zero_intensity_leaves_only_embodied_carbon_and_no_cache_leaves_none_of_its_own(C=C0):
    others = [(106.4, 5), (9.3, 5), (30.8, 5)]
    t = C.total_g(2.0, 0.0, 1.0, 0, 30, 5, others)
    assert math.isclose(t, sum(C.amortised_g(1.0, lt, kg) for kg, lt in others), rel_tol=1e-12)
    assert C.total_g(0.0, 124.0, 1.0, 0, 30, 5, []) == 0.0


def golden_fraction(expr):
    """A sum of fractions written in a golden file ("1/2 + 5/1314") as a float."""
    from fractions import Fraction
    return float(sum(Fraction(t.strip()) for t in expr.split("+")))


def test_carbon_hand_worked_examples(C=C0):
    """Per-request (Eq. ilp objective term) and per-interval (Eq. cache+other) carbon
    against values worked by hand in tests/golden/carbon_examples.json: the W*s to
    kWh conversion, the s to h conversion of the amortised terms, CI in g/kWh and
    embodied kg in g are each visible in one of the cases."""
    g = json.load(open(os.path.join(HERE, "golden", "carbon_examples.json")))
    p = g["platform"]
    others = [(p["gpu_kg"], p["lifetime_years"]), (p["cpu_kg"], p["lifetime_years"]),
              (p["mem_kg"], p["lifetime_years"])]
    for c in g["request_cases"]:
        got = C.request_carbon_g(c["power_w"], c["ttft_s"], c["ci"], c["size_tb"], p["ssd_kg_per_tb"],
                                 p["lifetime_years"], others if c["with_others"] else [])
        assert math.isclose(got, golden_fraction(c["expected"]), rel_tol=1e-12), c["name"]
    for c in g["interval_cases"]:
        got = C.total_g(c["energy_kwh"], c["ci"], c["hours"], c["size_tb"], p["ssd_kg_per_tb"],
                        p["lifetime_years"], others)
        assert math.isclose(got, golden_fraction(c["expected"]), rel_tol=1e-12), c["name"]


def test_operational_carbon_is_energy_times_intensity(C=C0):
    """Eq. carbon-op at values that are not 0: 0.25 kWh at 400 g/kWh is 100 g."""
    assert math.isclose(C.operational_g(0.25, 400.0), 100.0, rel_tol=1e-15)
    assert math.isclose(C.operational_g(3.0, 56.0), 168.0, rel_tol=1e-15)


# ----------------------------------------------------------------- cache-size ILP

def knapsack_min_weight(w, v, V):
    """Textbook DP: smallest total weight of a subset with total value >= V (inf if none)."""
    INF = math.inf
    best = [0.0] + [INF] * V           # best[x]: min weight reaching value >= x (capped at V)
    for wk, vk in zip(w, v):
        for x in range(V, -1, -1):
            src = max(0, x - vk)
            if best[src] + wk < best[x]:
                best[x] = best[src] + wk
    return best[V]


def greencache_from_knapsack(w, v, V):
    """The appendix construction: step k = item k, cache off/on; lambda_k = v_k
    requests, all meeting both SLOs when on and none when off; incremental carbon
    w_k when on; rho = V / sum(v)."""
    cost = [[0.0, float(wk)] for wk in w]
    ok = [[0, vk] for vk in v]
    N = sum(v)
    return cost, ok, ok, N, V / N


@pytest.mark.parametrize("seed", range(6))
def test_ilp_bruteforce_solves_the_knapsack_construction(seed, C=C0):
    rng = np.random.default_rng(seed)
    m = int(rng.integers(3, 9))
    w = [int(x) for x in rng.integers(1, 20, m)]
    v = [int(x) for x in rng.integers(1, 15, m)]
    V = int(rng.integers(1, sum(v) + 1))
    cost, ok1, ok2, N, rho = greencache_from_knapsack(w, v, V)
    best, choice = C.solve_sizes_bruteforce(cost, ok1, ok2, N, rho * (1 - 1e-12))
    assert math.isclose(best, knapsack_min_weight(w, v, V), rel_tol=0, abs_tol=1e-9)
    assert sum(v[k] for k in range(m) if choice[k]) >= V


def test_ilp_infeasible_when_no_choice_meets_the_slo(C=C0):
    best, choice = C.solve_sizes_bruteforce([[1.0, 2.0]], [[0, 3]], [[0, 2]], 4, 0.9)
    assert best == math.inf and choice is None


# ----------------------------------------------------------------- planted mistakes

MUTANTS = {
    "fifo_orders_by_last_access": ('return (e["t_ins"], key)', 'return (e["t_last"], key)'),
    "lru_orders_by_insertion": ('return (e["t_last"], key)', 'return (e["t_ins"], key)'),
    "lcs_drops_reused_tokens": ('score = (float(e["acc"]) * float(e["hits"])) / (size * age)',
                                'score = float(e["hits"]) / (size * age)'),
    "lcs_ignores_size": ('score = (float(e["acc"]) * float(e["hits"])) / (size * age)',
                         'score = (float(e["acc"]) * float(e["hits"])) / age'),
    "lcs_ignores_age": ('score = (float(e["acc"]) * float(e["hits"])) / (size * age)',
                        'score = (float(e["acc"]) * float(e["hits"])) / size'),
    "multiturn_uses_hits": ('score = (float(e["turn"]) * float(e["acc"])) / (size * age)',
                            'score = (float(e["hits"]) * float(e["acc"])) / (size * age)'),
    "tie_break_newest_first": ('return (score, e["t_ins"], key)', 'return (score, -e["t_ins"], key)'),
    "hit_reuses_whole_entry": ('reused = min(context, e["tokens"])', 'reused = e["tokens"]'),
    "entry_does_not_grow": ('e["tokens"] = max(e["tokens"], total)', 'pass'),
    "oversized_entry_evicts_others": ('if self.entries[keep]["tokens"] * self.bpt > self.capacity:',
                                      'if False:'),
    "lifetime_in_days": ('return hours / (lifetime_years * HOURS_PER_YEAR) * embodied_kg * 1000.0',
                         'return hours / (lifetime_years * 365.0) * embodied_kg * 1000.0'),
    "cache_size_dropped": ('return size_tb * amortised_g(hours, lifetime_years, ssd_kg_per_tb)',
                           'return amortised_g(hours, lifetime_years, ssd_kg_per_tb)'),
    "ilp_ignores_tpot": ('if sum(ok_tpot[t][s] for t, s in enumerate(choice)) < need:',
                         'if False:'),
    "ilp_maximises": ('if c < best:', 'if best == math.inf or c > best:'),
    "joules_to_kwh_off_by_1000": ('energy_kwh = power_w * ttft_s / 3.6e6', 'energy_kwh = power_w * ttft_s / 3.6e3'),
    "ttft_taken_as_hours": ('hours = ttft_s / 3600.0', 'hours = ttft_s'),
    "intensity_applied_in_kg": ('return energy_kwh * ci_g_per_kwh', 'return energy_kwh * ci_g_per_kwh / 1000.0'),
    "embodied_left_in_kg": ('return hours / (lifetime_years * HOURS_PER_YEAR) * embodied_kg * 1000.0',
                            'return hours / (lifetime_years * HOURS_PER_YEAR) * embodied_kg'),
    "request_drops_other_embodied": ('return total_g(energy_kwh, ci, hours, size_tb, ssd_kg_per_tb, ssd_lifetime_years, others)',
                                     'return total_g(energy_kwh, ci, hours, size_tb, ssd_kg_per_tb, ssd_lifetime_years, [])'),
}

PINS = [test_fifo_shows_beladys_anomaly, test_lru_textbook_fault_counts, test_lru_is_a_stack_algorithm,
        test_lcs_hand_worked_example, test_lcs_without_hits_degenerates_to_fifo,
        test_multiturn_score_prefers_deeper_turns, test_oversized_entry_is_dropped_without_evicting_others,
        test_resize_evicts_by_policy, test_ilp_tpot_constraint_binds,
        test_amortised_share_over_the_whole_lifetime_is_the_whole_embodied_carbon,
        test_carbon_is_additive_over_time_and_capacity, test_ssd_table_entry_per_terabyte,
        test_zero_intensity_leaves_only_embodied_carbon_and_no_cache_leaves_none_of_its_own,
        test_ilp_infeasible_when_no_choice_meets_the_slo, test_carbon_hand_worked_examples,
        test_operational_carbon_is_energy_times_intensity]


def _run_pins(C):
    failures = []
    for pin in PINS:
        try:
            pin(C=C)
        except Exception as e:  # noqa: BLE001 - a planted mistake may fail in any way
            failures.append(f"{pin.__name__}: {type(e).__name__}")
    for seed in range(6):
        try:
            test_ilp_bruteforce_solves_the_knapsack_construction(seed, C=C)
        except Exception as e:  # noqa: BLE001
            failures.append(f"knapsack[{seed}]: {type(e).__name__}")
    for case in range(5):
        try:
            test_hand_worked_sensitivity_cases(case, C=C)
        except Exception as e:  # noqa: BLE001
            failures.append(f"case[{case}]: {type(e).__name__}")
    return failures


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_control_pins_reject_planted_mistake(name, tmp_path):
    import importlib.util
    src = open(C0.__file__).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    path = tmp_path / f"control_{name}.py"
    path.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location(f"control_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    assert _run_pins(mod), f"planted mistake '{name}' passed every pin"


def test_unmodified_control_oracle_passes_every_pin():
    assert _run_pins(C0) == []

"""Control plane of the context cache (CPU): the carbon model, the replacement
model (native library libgreencache_ctl.so, C ABI in include/greencache_ctl.h)
and the hourly cache-size ILP.

GreenCache §2.3 (Eqs. 1-3) and §3.2.1 (Eqs. 4-5) price a serving interval as operational carbon
(energy x grid carbon intensity) plus the amortised embodied carbon of the
platform, with the cache's SSD share proportional to the allocated capacity.
§5.4.1 (Eq. 6) picks, per decision interval, the cache size that minimises the
summed per-request carbon while at least rho of all requests meet the TTFT SLO
and at least rho meet the TPOT SLO; the paper solves it with an ILP solver
(PuLP + CBC), here scipy's HiGHS interface. §5.5 (Eqs. 7-8) evicts the
entries with the Least Carbon Savings.

Units: power W, times s (TTFT) or h (intervals), energy kWh, carbon intensity
gCO2e/kWh, embodied carbon kgCO2e, lifetimes years of 365 days, sizes TB.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(HERE, "libgreencache_ctl.so")
EXPORTED = ("gc_cache_create", "gc_cache_destroy", "gc_cache_replay", "gc_cache_resize",
            "gc_cache_get_stats", "gc_cache_keys")
POLICIES = {"fifo": 0, "lru": 1, "lcs": 2, "lcs_multiturn": 3}
HOURS_PER_YEAR = 365.0 * 24.0

REQUEST_DTYPE = np.dtype([("key", "<i8"), ("context_tokens", "<i8"), ("prompt_tokens", "<i8"),
                          ("total_tokens", "<i8"), ("turn", "<i4"), ("reserved", "<i4"), ("time", "<f8")])


class Stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("requests", "hits", "reused_tokens", "prompt_tokens",
                                              "insertions", "evictions", "entries", "bytes")]


_lib = None


def load_library(path: str | None = None):
    """The replacement-model library; raises if it has not been built."""
    global _lib
    if path is None and _lib is not None:
        return _lib
    p = path or LIBRARY
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with `python -m paper_2505_23970_amd.build`")
    lib = ctypes.CDLL(p)
    i32, i64, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
    lib.gc_cache_create.restype = i32
    lib.gc_cache_create.argtypes = [i32, i64, i64, ctypes.POINTER(vp)]
    lib.gc_cache_destroy.restype = None
    lib.gc_cache_destroy.argtypes = [vp]
    lib.gc_cache_replay.restype = i32
    lib.gc_cache_replay.argtypes = [vp, vp, i64, vp]
    lib.gc_cache_resize.restype = i32
    lib.gc_cache_resize.argtypes = [vp, i64, ctypes.c_double]
    lib.gc_cache_get_stats.restype = i32
    lib.gc_cache_get_stats.argtypes = [vp, ctypes.POINTER(Stats)]
    lib.gc_cache_keys.restype = i32
    lib.gc_cache_keys.argtypes = [vp, vp, i64, ctypes.POINTER(i64)]
    if path is None:
        _lib = lib
    return lib


class CtlError(RuntimeError):
    pass


def _check(fn, st):
    if st != 0:
        raise CtlError(f"{fn} returned {st}")


class Cache:
    """A context cache of `capacity_bytes` under one replacement policy."""

    def __init__(self, policy: str, capacity_bytes: int, bytes_per_token: int):
        self._lib = load_library()
        h = ctypes.c_void_p()
        _check("gc_cache_create", self._lib.gc_cache_create(POLICIES[policy], int(capacity_bytes),
                                                            int(bytes_per_token), ctypes.byref(h)))
        self._h = h

    def close(self):
        if self._h:
            self._lib.gc_cache_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def replay(self, requests: np.ndarray) -> np.ndarray:
        """Replay a REQUEST_DTYPE array in order; returns the tokens each request reused."""
        r = np.ascontiguousarray(requests, dtype=REQUEST_DTYPE)
        out = np.zeros(len(r), np.int64)
        _check("gc_cache_replay", self._lib.gc_cache_replay(self._h, r.ctypes.data, len(r), out.ctypes.data))
        return out

    def resize(self, capacity_bytes: int, now: float):
        _check("gc_cache_resize", self._lib.gc_cache_resize(self._h, int(capacity_bytes), float(now)))

    def stats(self) -> dict:
        s = Stats()
        _check("gc_cache_get_stats", self._lib.gc_cache_get_stats(self._h, ctypes.byref(s)))
        return {n: int(getattr(s, n)) for n, _ in Stats._fields_}

    def keys(self) -> np.ndarray:
        cnt = ctypes.c_int64()
        _check("gc_cache_keys", self._lib.gc_cache_keys(self._h, None, 0, ctypes.byref(cnt)))
        out = np.zeros(cnt.value, np.int64)
        _check("gc_cache_keys", self._lib.gc_cache_keys(self._h, out.ctypes.data, len(out), ctypes.byref(cnt)))
        return out


def token_hit_rate(policy: str, capacity_bytes: int, bytes_per_token: int, trace: np.ndarray) -> float:
    """The paper's cache hit rate (§6.3.2, Table tab:replacement): reused tokens over all input tokens."""
    c = Cache(policy, capacity_bytes, bytes_per_token)
    reused = c.replay(trace)
    return float(reused.sum()) / float(np.sum(trace["prompt_tokens"]))


# ----------------------------------------------------------------- carbon model

@dataclasses.dataclass(frozen=True)
class Platform:
    """Embodied carbon of the serving platform (Table 1) and component lifetimes
    (5 years, §2.3). The SSD's embodied carbon is per allocated TB."""
    gpu_kg: float = 106.4
    cpu_kg: float = 9.3
    mem_kg: float = 30.8
    ssd_kg_per_tb: float = 480.0 / 16.0
    lifetime_years: float = 5.0
    ssd_lifetime_years: float = 5.0

    def others(self):
        return ((self.gpu_kg, self.lifetime_years), (self.cpu_kg, self.lifetime_years),
                (self.mem_kg, self.lifetime_years))


def operational_g(energy_kwh, ci):
    return np.asarray(energy_kwh, np.float64) * ci


def amortised_g(hours, lifetime_years, embodied_kg):
    return np.asarray(hours, np.float64) / (lifetime_years * HOURS_PER_YEAR) * (embodied_kg * 1000.0)


def interval_carbon_g(energy_kwh, ci, hours, size_tb, platform: Platform = Platform()):
    """Eq. 5: E x CI + S_alloc x (T / LT_SSD) x C_SSD,unit + (T / LT) x C_others."""
    others = sum(amortised_g(hours, lt, kg) for kg, lt in platform.others())
    return (operational_g(energy_kwh, ci) + np.asarray(size_tb, np.float64)
            * amortised_g(hours, platform.ssd_lifetime_years, platform.ssd_kg_per_tb) + others)


def request_carbon_g(power_w, ttft_s, ci, size_tb, platform: Platform = Platform()):
    """The per-request term of Eq. 6 (prefill phase): p x TTFT x CI + TTFT / LT_SSD
    x S x C_SSD,unit + sum over GPU, CPU, memory of TTFT / LT x C."""
    ttft = np.asarray(ttft_s, np.float64)
    return interval_carbon_g(np.asarray(power_w, np.float64) * ttft / 3.6e6, ci, ttft / 3600.0, size_tb, platform)


# ----------------------------------------------------------------- cache-size ILP

def profile_costs(profile: dict, platform: Platform = Platform(), cache_attribution: str = "ttft",
                  step_hours: float = 1.0) -> np.ndarray:
    """cost[t, s] = requests of step t x the per-request carbon at cache size s.

    cache_attribution "ttft" prices the SSD as Eq. 6 writes it (each request is
    charged TTFT / LT_SSD x S x C_SSD,unit); "interval" charges the allocated
    capacity for the whole decision interval instead (Eq. 4 with T = step_hours),
    which is what a provisioned cloud SSD costs whether or not requests run."""
    ci = np.asarray(profile["ci"], np.float64)[:, None]
    S = np.asarray(profile["sizes_tb"], np.float64)[None, :]
    n = np.asarray(profile["n"], np.float64)[:, None]
    if cache_attribution == "ttft":
        return n * request_carbon_g(profile["power"], profile["ttft"], ci, S, platform)
    if cache_attribution == "interval":
        per = request_carbon_g(profile["power"], profile["ttft"], ci, 0.0, platform)
        return n * per + S * amortised_g(step_hours, platform.ssd_lifetime_years, platform.ssd_kg_per_tb)
    raise ValueError(f"unknown cache_attribution {cache_attribution!r}")


def solve_cache_sizes(cost, ok_ttft, ok_tpot, n_requests, rho=0.9):
    """Eq. 6 with one size choice per step: binary x[t, s], sum_s x[t, s] = 1,
    minimise sum cost[t, s] x[t, s] subject to sum ok_ttft x >= rho N and
    sum ok_tpot x >= rho N. Returns (cost, choice per step) or (inf, None)."""
    from scipy.optimize import Bounds, LinearConstraint, milp
    cost = np.asarray(cost, np.float64)
    T, S = cost.shape
    A_one = np.zeros((T, T * S))
    for t in range(T):
        A_one[t, t * S:(t + 1) * S] = 1.0
    A_slo = np.vstack([np.asarray(ok_ttft, np.float64).ravel(), np.asarray(ok_tpot, np.float64).ravel()])
    need = rho * float(n_requests)
    res = milp(cost.ravel(), integrality=np.ones(T * S), bounds=Bounds(0, 1),
               constraints=[LinearConstraint(A_one, 1, 1), LinearConstraint(A_slo, need, np.inf)])
    if res.x is None or res.status != 0:
        return float("inf"), None
    x = np.rint(res.x).reshape(T, S)
    choice = [int(np.argmax(x[t])) for t in range(T)]
    return float(sum(cost[t, s] for t, s in enumerate(choice))), choice

"""Seeded synthetic inputs shaped like Qwen3-8B decode (random draws only).

This module holds none of the method's arithmetic: it draws keys, queries,
values, channel variances and ragged lengths, and is the one source of inputs
shared by the HIP path and the CPU oracle.

Per unit (one KV head of one sequence and layer), in this draw order from
``numpy.random.default_rng(SeedSequence(seed, spawn_key=(seed_key, session, layer, head)))``:
  1. sigma_c = exp(z_c), z_c ~ N(0, 1), c < 128   (log-normal channel scales)
  2. 4 outlier channels drawn without replacement; sigma_c *= 8 there
  3. queries q ~ N(0, 1), [G][D], stored fp32 or fp16
  4. (host path) keys K = sigma * eps, eps ~ N(0, 1), [n][D] fp32, then values V ~ N(0, 1) fp16
var_c = fp32(sigma_c^2) is the population variance of the generator (the
calibration statistic of Sec. 3.3, given identically to both sides).

Large workloads draw K and V on the GPU with torch's device generator,
seeded from the same tuple; the oracle always consumes copies of the device
values, never a re-draw.
"""
from __future__ import annotations

import dataclasses
import hashlib

import numpy as np

D = 128


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    seed_key: int            # first element of every seed tuple of this workload
    sessions: int
    layers: int
    kv_heads: int
    G: int
    n: int | None            # fixed length, or None for ragged
    n_range: tuple | None    # (lo, hi) inclusive for ragged lengths
    q_dtype: str             # "f32" | "f16"
    budgets: tuple           # water-filling budgets (code bits per key)
    uniform_r: tuple         # uniform-depth mode r values (4 planes each)
    k: int
    n_sink: int = 0
    n_local: int = 0

    @property
    def units(self) -> int:
        return self.sessions * self.layers * self.kv_heads


# The five workloads, by what they are.  The seed key keeps every draw of one
# workload independent of the others.
WORKLOADS = {
    "head4k": Config("single KV head, n=4096, fp32 query, B=48, k=64",
                     0, 1, 1, 1, 1, 4096, None, "f32", (48,), (), 64),
    "layer128k": Config("one Qwen3-8B layer, 8 KV heads x 4 query heads, n=131072, k=1024",
                        1, 1, 1, 8, 4, 131072, None, "f16", (40, 48, 80), (), 1024),
    "layer1m": Config("one Qwen3-8B layer, 8 KV heads x 4 query heads, n=2^20, k=2048",
                      2, 1, 1, 8, 4, 1 << 20, None, "f16", (48, 80), (16, 32), 2048),
    "ragged16": Config("16 resident sessions, ragged n in [65536, 524288], 8 KV heads x 4, B=40, k=1024",
                       3, 16, 1, 8, 4, None, (65536, 524288), "f16", (40,), (), 1024),
    "step4x1m": Config("full decode step: 4 sessions x 36 layers x 8 KV heads, n=2^20, B=48, k=2048, "
                       "4 sink + 32 local", 4, 4, 36, 8, 4, 1 << 20, None, "f16", (48,), (), 2048, 4, 32),
}


def unit_rng(seed_key: int, session: int, layer: int, head: int, seed: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(seed_key, session, layer, head)))


def torch_seed(seed_key: int, session: int, layer: int, head: int, stream: str, seed: int = 0) -> int:
    h = hashlib.sha256(f"{seed}/{seed_key}/{session}/{layer}/{head}/{stream}".encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def channel_sigma(rng: np.random.Generator, d: int = D, n_outliers: int = 4, mult: float = 8.0) -> np.ndarray:
    sigma = np.exp(rng.standard_normal(d))
    sigma[rng.choice(d, n_outliers, replace=False)] *= mult
    return sigma


def variance(sigma: np.ndarray) -> np.ndarray:
    return (sigma * sigma).astype(np.float32)


def queries(rng: np.random.Generator, G: int, q_dtype: str) -> np.ndarray:
    q = rng.standard_normal((G, D)).astype(np.float32)
    return q.astype(np.float16) if q_dtype == "f16" else q


def keys_host(rng: np.random.Generator, n: int, sigma: np.ndarray) -> np.ndarray:
    return (rng.standard_normal((n, D), dtype=np.float32) * sigma.astype(np.float32)).astype(np.float32)


def values_host(rng: np.random.Generator, n: int) -> np.ndarray:
    return rng.standard_normal((n, D), dtype=np.float32).astype(np.float16)


def mixing_rotation(cfg: Config, unit: int, seed: int = 0) -> np.ndarray:
    """A seeded random orthogonal D x D matrix for unit `unit` (QR of a Gaussian
    draw, column signs fixed by the triangular factor's diagonal), fp32.  Keys
    k R^T and queries q R^T keep every score q . k but spread the generator's
    independent channels over all raw channels: the covariance of a layer whose
    keys are not normalised per channel (the case for the rotated store)."""
    ids = list(unit_ids(cfg))
    rng = unit_rng(cfg.seed_key, *ids[unit], seed=seed + 7919)
    Q, T = np.linalg.qr(rng.standard_normal((D, D)))
    return (Q * np.sign(np.diag(T))).astype(np.float32)


def ragged_lengths(cfg: Config, seed: int = 0) -> np.ndarray:
    """Per-session lengths uniform in n_range (inclusive), one draw per session."""
    rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(cfg.seed_key, 10 ** 6)))
    lo, hi = cfg.n_range
    return rng.integers(lo, hi + 1, cfg.sessions).astype(np.int64)


def unit_lengths(cfg: Config, seed: int = 0) -> np.ndarray:
    """n for every unit, units ordered (session, layer, kv_head)."""
    per_session = ragged_lengths(cfg, seed) if cfg.n is None else np.full(cfg.sessions, cfg.n, np.int64)
    return np.repeat(per_session, cfg.layers * cfg.kv_heads)


def unit_ids(cfg: Config):
    for s in range(cfg.sessions):
        for l in range(cfg.layers):
            for h in range(cfg.kv_heads):
                yield s, l, h


@dataclasses.dataclass
class HostUnits:
    """Host arrays for a set of units (small configurations and tests)."""
    K: np.ndarray       # [U][n_max][D] fp32 (rows past n[u] are zero)
    V: np.ndarray       # [U][n_max][D] fp16
    q: np.ndarray       # [U][G][D] fp32 or fp16
    var: np.ndarray     # [U][D] fp32
    n: np.ndarray       # [U] int64


def host_units(cfg: Config, units=None, n_override: int | None = None, seed: int = 0) -> HostUnits:
    ids = list(unit_ids(cfg))
    lens = unit_lengths(cfg, seed)
    sel = range(len(ids)) if units is None else units
    sel = list(sel)
    ns = np.array([n_override if n_override is not None else lens[i] for i in sel], np.int64)
    nmax = int(ns.max()) if len(ns) else 0
    K = np.zeros((len(sel), nmax, D), np.float32)
    V = np.zeros((len(sel), nmax, D), np.float16)
    q = np.zeros((len(sel), cfg.G, D), np.float16 if cfg.q_dtype == "f16" else np.float32)
    var = np.zeros((len(sel), D), np.float32)
    for a, i in enumerate(sel):
        rng = unit_rng(cfg.seed_key, *ids[i], seed=seed)
        sig = channel_sigma(rng)
        var[a] = variance(sig)
        q[a] = queries(rng, cfg.G, cfg.q_dtype)
        K[a, :ns[a]] = keys_host(rng, int(ns[a]), sig)
        V[a, :ns[a]] = values_host(rng, int(ns[a]))
    return HostUnits(K, V, q, var, ns)


def device_units(cfg: Config, units=None, n_override: int | None = None, seed: int = 0, device="cuda",
                 with_values: bool = True, key_dtype=None):
    """Device tensors for large configurations: K [U][n_max][D] fp32 (or key_dtype), K16/V16 fp16 rows,
    q, var, n.  Keys and values come from torch's device generator, seeded per unit."""
    import torch

    ids = list(unit_ids(cfg))
    lens = unit_lengths(cfg, seed)
    sel = list(range(len(ids)) if units is None else units)
    ns = np.array([n_override if n_override is not None else lens[i] for i in sel], np.int64)
    nmax = int(ns.max()) if len(ns) else 0
    kd = torch.float32 if key_dtype is None else key_dtype
    K = torch.zeros((len(sel), nmax, D), dtype=kd, device=device)
    V = torch.zeros((len(sel), nmax, D), dtype=torch.float16, device=device) if with_values else None
    qd = np.float16 if cfg.q_dtype == "f16" else np.float32
    q = np.zeros((len(sel), cfg.G, D), qd)
    var = np.zeros((len(sel), D), np.float32)
    g = torch.Generator(device=device)
    for a, i in enumerate(sel):
        rng = unit_rng(cfg.seed_key, *ids[i], seed=seed)
        sig = channel_sigma(rng)
        var[a] = variance(sig)
        q[a] = queries(rng, cfg.G, cfg.q_dtype)
        g.manual_seed(torch_seed(cfg.seed_key, *ids[i], "K", seed))
        sig_t = torch.from_numpy(sig.astype(np.float32)).to(device)
        K[a, :ns[a]] = (torch.randn((int(ns[a]), D), generator=g, device=device, dtype=torch.float32) * sig_t).to(kd)
        if with_values:
            g.manual_seed(torch_seed(cfg.seed_key, *ids[i], "V", seed))
            V[a, :ns[a]] = torch.randn((int(ns[a]), D), generator=g, device=device, dtype=torch.float32).half()
    return {
        "K": K, "V": V,
        "q": torch.from_numpy(q).to(device), "var": torch.from_numpy(var).to(device),
        "n": torch.from_numpy(ns).to(device), "n_host": ns,
    }

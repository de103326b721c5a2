"""Seeded synthetic inputs for the capacity-bounded top-k MoE layer.

This module is shared by the CPU oracle (``oracle/``), the tests and the
benchmark.  It only *draws* inputs: it holds none of the layer's arithmetic
(no gating, routing, capacity, FFN or combine step lives here).

Storage conventions (the same ones the C-ABI library documents):

* every weight is stored output-features x input-features, the layout of a
  linear map ``y = x . W^T``:  ``w_g [E, d]``, ``w1 [E, f, d]``,
  ``w3 [E, f, d]`` (gated FFN only) and ``w2 [E, d, f]``;
* bf16 tensors are held as ``numpy.uint16`` bit patterns produced by
  round-to-nearest-even from float32 draws;
* fp32 tensors are ``numpy.float32``.

Every draw comes from a PCG64 stream keyed by (config seed, tensor id, chunk
index), so large tensors can be generated chunk-parallel and any tensor can
be regenerated on its own.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional, Tuple

import numpy as np

__all__ = [
    "Workload", "Inputs", "CONFIGS", "config", "make_inputs", "small",
    "to_bf16_bits", "TENSOR_IDS", "make_target", "drifting_assignments",
    "reassign_some",
]

# tensor ids used as SeedSequence spawn keys (fixed; never renumber)
TENSOR_IDS = {"x": 1, "w_g": 2, "bias": 3, "w1": 4, "w3": 5, "w2": 6,
              "dy": 7, "ids": 8, "cw": 9, "target": 10, "traj": 11,
              "reassign": 12}

_CHUNK = 1 << 22  # elements per independent PCG64 stream


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and recipe of one synthetic MoE-layer workload."""
    name: str
    T: int                 # tokens
    d: int                 # model width
    E: int                 # experts
    k: int                 # experts per token
    f: int                 # expert hidden width
    act: str               # "relu" | "gelu_tanh" | "swiglu"
    dtype: str             # "f32" | "bf16"
    gate: str = "linear"   # "linear" (x . w_g^T + b) | "cached" (ids/weights given)
    bias: str = "none"     # "none" | "zipf_log" | "normal"
    bias_scale: float = 0.0
    zipf_s: float = 1.2    # cached-id law, P(e) ~ (e+1)^-s
    renorm: int = 0        # 1: weights of the k picks renormalised to sum 1
    backward: bool = False
    # capacity runs: ("static", num, den) => alpha = num/den;
    # ("dynamic", num, den) => C_e = ceil(num/den * count_e); ("exact",1,1)
    capacity: Tuple[Tuple[str, int, int], ...] = (("static", 1, 1),)
    seed: int = 20220500
    x_std: float = 1.0
    w_std: float = 0.02

    @property
    def esize(self) -> int:
        return 4 if self.dtype == "f32" else 2


CONFIGS = {
    # 1: tiny fp32 layer, static alpha = 1.25, forward only
    "c1": Workload("c1", T=256, d=64, E=4, k=1, f=128, act="relu", dtype="f32",
                   capacity=(("static", 5, 4),), seed=20220500),
    # 2: balanced top-2, GELU(tanh), static alpha=1 then dynamic margin 1.1
    "c2": Workload("c2", T=8192, d=512, E=16, k=2, f=2048, act="gelu_tanh",
                   dtype="bf16", renorm=1,
                   capacity=(("static", 1, 1), ("dynamic", 11, 10)),
                   seed=20220501),
    # 3: Zipf-skewed Switch-style top-1, static alpha=2 vs dynamic margin 1.1
    "c3": Workload("c3", T=16384, d=1024, E=64, k=1, f=4096, act="relu",
                   dtype="bf16", bias="zipf_log", bias_scale=2.0,
                   capacity=(("static", 2, 1), ("dynamic", 11, 10)),
                   backward=True, seed=20220502),
    # 4: sample-assignment-caching path (gate bypassed), exact capacity
    "c4": Workload("c4", T=32768, d=2048, E=32, k=2, f=8192, act="relu",
                   dtype="bf16", gate="cached", zipf_s=1.2,
                   capacity=(("exact", 1, 1),), backward=True, seed=20220503),
    # 5: large SwiGLU layer, mildly imbalanced gate, dynamic margin 1.05
    "c5": Workload("c5", T=65536, d=4096, E=8, k=2, f=14336, act="swiglu",
                   dtype="bf16", bias="normal", bias_scale=0.5, renorm=1,
                   capacity=(("dynamic", 21, 20),), backward=True,
                   seed=20220504),
}


def config(name: str) -> Workload:
    return CONFIGS[name]


def small(base: str, **overrides) -> Workload:
    """A reduced copy of a named config (same recipe, smaller shapes)."""
    wl = CONFIGS[base]
    fields = dict(name=overrides.pop("name", base + "_small"))
    return dataclasses.replace(wl, **fields, **overrides)


@dataclasses.dataclass
class Inputs:
    wl: Workload
    x: np.ndarray                 # [T, d]  (uint16 bf16 bits or float32)
    w_g: Optional[np.ndarray]     # [E, d]  (None on the cached path)
    bias: Optional[np.ndarray]    # [E] float32 or None
    w1: np.ndarray                # [E, f, d]
    w3: Optional[np.ndarray]      # [E, f, d] (swiglu only)
    w2: np.ndarray                # [E, d, f]
    dy: Optional[np.ndarray]      # [T, d] upstream gradient (backward configs)
    ids: Optional[np.ndarray]     # [T, k] int32 cached expert ids
    cw: Optional[np.ndarray]      # [T, k] float32 cached combine weights


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + r) >> np.uint32(16)).astype(np.uint16)


def _rng(seed: int, tensor: str, chunk: int) -> np.random.Generator:
    ss = np.random.SeedSequence(entropy=seed, spawn_key=(TENSOR_IDS[tensor], chunk))
    return np.random.Generator(np.random.PCG64(ss))


def _normal(seed: int, tensor: str, shape, std: float, dtype: str,
            mean: float = 0.0) -> np.ndarray:
    """N(mean, std) draws of `shape`, fp32 or bf16 bits, chunk-parallel."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16 if dtype == "bf16" else np.float32)
    nchunks = (n + _CHUNK - 1) // _CHUNK

    def work(c):
        lo, hi = c * _CHUNK, min(n, (c + 1) * _CHUNK)
        v = _rng(seed, tensor, c).standard_normal(hi - lo, dtype=np.float32)
        if std != 1.0:
            v *= np.float32(std)
        if mean != 0.0:
            v += np.float32(mean)
        out[lo:hi] = to_bf16_bits(v) if dtype == "bf16" else v

    if nchunks == 1:
        work(0)
    else:
        with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(work, range(nchunks)))
    return out.reshape(shape)


def _bias(wl: Workload) -> Optional[np.ndarray]:
    if wl.bias == "none":
        return None
    if wl.bias == "zipf_log":
        # b_e = scale * log(1 / (e+1)^1.1), natural log, fp64 then fp32
        e = np.arange(wl.E, dtype=np.float64)
        return (wl.bias_scale * np.log(1.0 / (e + 1.0) ** 1.1)).astype(np.float32)
    if wl.bias == "normal":
        v = _rng(wl.seed, "bias", 0).standard_normal(wl.E, dtype=np.float32)
        return (v * np.float32(wl.bias_scale)).astype(np.float32)
    raise ValueError(wl.bias)


def _sample_distinct(rng: np.random.Generator, p: np.ndarray, T: int, k: int) -> np.ndarray:
    """[T,k] expert ids, k distinct per token, drawn one after another from
    p (renormalised over the experts not yet taken)."""
    E = len(p)
    u = rng.random((T, k))
    ids = np.empty((T, k), dtype=np.int32)
    taken = np.zeros((T, E), dtype=bool)
    for j in range(k):
        q = np.where(taken, 0.0, p[None, :])
        cdf = np.cumsum(q, axis=1)
        target = u[:, j] * cdf[:, -1]
        pick = (cdf <= target[:, None]).sum(axis=1)
        pick = np.minimum(pick, E - 1)
        # a pick can only land on a taken expert through the clamp above
        bad = taken[np.arange(T), pick]
        if bad.any():
            for t in np.nonzero(bad)[0]:
                pick[t] = int(np.nonzero(~taken[t])[0][-1])
        ids[:, j] = pick
        taken[np.arange(T), pick] = True
    return ids


def _cached_assignments(wl: Workload):
    """Cached [T,k] ids from P(e) ~ (e+1)^-s with distinct picks per token,
    and [T,k] weights uniform on [0,1) renormalised per token."""
    T, E, k = wl.T, wl.E, wl.k
    p = (np.arange(1, E + 1, dtype=np.float64)) ** (-wl.zipf_s)
    p /= p.sum()
    ids = _sample_distinct(_rng(wl.seed, "ids", 0), p, T, k)
    uw = _rng(wl.seed, "cw", 0).random((T, k))
    s = uw.sum(axis=1, keepdims=True)
    w = np.where(s > 0, uw / np.where(s > 0, s, 1.0), 1.0 / k).astype(np.float32)
    return ids, w


def make_inputs(wl: Workload) -> Inputs:
    """All inputs of `wl`, drawn in the fixed order x, w_g, b, w1, w3, w2,
    dy, cached ids/weights (each from its own keyed stream)."""
    dt = wl.dtype
    x = _normal(wl.seed, "x", (wl.T, wl.d), wl.x_std, dt)
    w_g = None
    if wl.gate == "linear":
        w_g = _normal(wl.seed, "w_g", (wl.E, wl.d), wl.w_std, dt)
    bias = _bias(wl) if wl.gate == "linear" else None
    w1 = _normal(wl.seed, "w1", (wl.E, wl.f, wl.d), wl.w_std, dt)
    w3 = (_normal(wl.seed, "w3", (wl.E, wl.f, wl.d), wl.w_std, dt)
          if wl.act == "swiglu" else None)
    w2 = _normal(wl.seed, "w2", (wl.E, wl.d, wl.f), wl.w_std, dt)
    dy = _normal(wl.seed, "dy", (wl.T, wl.d), 1.0, dt) if wl.backward else None
    ids = cw = None
    if wl.gate == "cached":
        ids, cw = _cached_assignments(wl)
    return Inputs(wl, x, w_g, bias, w1, w3, w2, dy, ids, cw)


def make_target(wl: Workload) -> np.ndarray:
    """A [T,d] regression target in the layer dtype, N(0,1) entries: the
    synthetic label of a squared-error task loss."""
    return _normal(wl.seed, "target", (wl.T, wl.d), 1.0, wl.dtype)


def drifting_assignments(seed: int, T: int, E: int, k: int, n_iter: int,
                         s_start: float = 1.2, s_end: float = 0.6,
                         swap_every: int = 5):
    """Expert picks of n_iter consecutive mini-batches whose per-expert load
    drifts: iteration i draws from P(e) ~ (rank_i(e) + 1)^-s_i with s_i going
    linearly from s_start to s_end (imbalance that fades as training goes on)
    and two experts adjacent in the ranking swapping places every swap_every
    iterations (popularity that moves between experts).  Returns a list of
    [T,k] int32 arrays, k distinct picks per token."""
    rng = _rng(seed, "traj", 0)
    rank = rng.permutation(E)
    out = []
    for i in range(n_iter):
        if i and swap_every and i % swap_every == 0 and E > 1:
            a = int(rng.integers(0, E - 1))
            rank[[a, a + 1]] = rank[[a + 1, a]]
        s = s_start + (s_end - s_start) * (i / max(1, n_iter - 1))
        p = np.empty(E)
        p[rank] = (np.arange(1, E + 1, dtype=np.float64)) ** (-s)
        p /= p.sum()
        out.append(_sample_distinct(_rng(seed, "traj", i + 1), p, T, k))
    return out


def reassign_some(seed: int, ids: np.ndarray, E: int, frac: float) -> np.ndarray:
    """A copy of [T,k] picks in which a seeded random subset of round(frac*T)
    tokens gets fresh picks drawn uniformly (k distinct; a redraw can repeat
    the old set by chance)."""
    T, k = ids.shape
    rng = _rng(seed, "reassign", 0)
    out = np.array(ids, dtype=np.int32, copy=True)
    n = int(round(frac * T))
    if n:
        who = rng.choice(T, size=n, replace=False)
        out[who] = _sample_distinct(rng, np.full(E, 1.0 / E), n, k)
    return out

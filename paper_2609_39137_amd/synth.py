"""Seeded synthetic inputs for the router step and the bias controller.

This module only draws random numbers and converts them to the storage formats
the router reads (bf16 bits, fp32).  It holds none of the method's arithmetic:
no logits, no sigmoid, no selection, no controller.  Both the GPU path and the
CPU oracle consume exactly the arrays produced here, so they see identical
bytes.

Seeds: ``numpy.random.default_rng(SeedSequence([2609, 39137, workload, stream,
step, block]))`` with stream 0 = router weight, 1 = mixture parameters,
2 = hidden-state noise, 3 = mixture component labels, 4 = drift of the mixture
weights.  Hidden states are drawn in blocks of ``BLOCK_ROWS`` rows so any row
can be regenerated on its own.

The paper trains on an unnamed corpus that is not available here; these
distributions stand in for the router's input (token hidden states) at the
shapes of the paper's Top-10/5/3-of-768 runs.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

BLOCK_ROWS = 256
SEED_ROOT = (2609, 39137)


def rng(*key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([*SEED_ROOT, *[int(k) for k in key]]))


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to bfloat16 (round to nearest, ties to even); returns the raw bits as uint16."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    if u.size and int(u.max()) >= 0xFFFF8000:  # NaN payloads the 32-bit sum would wrap: widen
        u = u.astype(np.uint64)
    lsb = (u >> 16) & 1
    return ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: router shape, input distribution, controller steps."""

    name: str
    wid: int  # seed key
    T: int
    d: int
    E: int
    K: int
    dtype: str  # "bf16" or "f32"
    x_kind: str  # "normal", "mixture", "mixture-drift"
    w_std: float
    steps: int

    @property
    def flops(self) -> float:
        return 2.0 * self.T * self.d * self.E


# The five workloads: a tiny fp32 closed loop, the Top-10-of-768 headline
# shape, the skewed Top-5 mixture, the drifting Top-3 mixture and a large
# d=4096 stand-in.  Hidden sizes follow the paper's model table; the expert
# count 768 and K in {10, 5, 3} follow its main comparison.
WORKLOADS = {
    "tiny-e64-k4": Workload("tiny-e64-k4", 0, 4096, 256, 64, 4, "f32", "normal", 0.02, 10),
    "top10-of-768": Workload("top10-of-768", 1, 16384, 2048, 768, 10, "bf16", "normal", 0.02, 1),
    "top5-of-768-mixture": Workload("top5-of-768-mixture", 2, 16384, 2048, 768, 5, "bf16", "mixture", 0.02, 100),
    "top3-of-768-drift": Workload("top3-of-768-drift", 3, 32768, 2048, 768, 3, "bf16", "mixture-drift", 0.02, 200),
    "large-d4096-top10": Workload("large-d4096-top10", 4, 65536, 4096, 768, 10, "bf16", "normal", 0.015, 1),
}
HEADLINE = "top10-of-768"

N_COMPONENTS = 32
MIX_SIGMA = 0.5
DIRICHLET_ALPHA = 0.3
DRIFT_STEP = 0.05


def _store(a: np.ndarray, dtype: str) -> np.ndarray:
    return to_bf16_bits(a) if dtype == "bf16" else np.ascontiguousarray(a, dtype=np.float32)


def router_weight(wl: Workload) -> np.ndarray:
    """Router matrix W [E][d]: N(0, w_std^2), fixed for the run (stream 0)."""
    g = rng(wl.wid, 0)
    return _store(g.standard_normal((wl.E, wl.d), dtype=np.float32) * np.float32(wl.w_std), wl.dtype)


def mixture_params(wl: Workload):
    """Component means mu [C][d] ~ N(0, I) and base weights pi ~ Dirichlet(0.3) (stream 1).

    The Top-3 drifting workload reuses the Top-5 workload's parameters.
    """
    g = rng(2, 1)
    mu = g.standard_normal((N_COMPONENTS, wl.d), dtype=np.float32)
    pi = g.dirichlet(np.full(N_COMPONENTS, DIRICHLET_ALPHA))
    return mu, pi


def mixture_weights(wl: Workload, step: int) -> np.ndarray:
    """Mixture weights at ``step``.

    Fixed for "mixture"; for "mixture-drift" a random walk: each step adds
    0.05 * N(0, I) (stream 4), clips at 0 and renormalises, resetting to uniform
    if everything clipped.
    """
    _, pi = mixture_params(wl)
    if wl.x_kind != "mixture-drift":
        return pi
    p = pi.copy()
    for t in range(1, step + 1):
        p = p + DRIFT_STEP * rng(wl.wid, 4, t).standard_normal(N_COMPONENTS)
        p = np.clip(p, 0.0, None)
        tot = p.sum()
        p = np.full(N_COMPONENTS, 1.0 / N_COMPONENTS) if tot <= 0 else p / tot
    return p


def hidden_block(wl: Workload, step: int, block: int, mix=None) -> np.ndarray:
    """fp32 hidden states of rows [block*256, block*256 + 256) (clipped to T)."""
    r0 = block * BLOCK_ROWS
    n = min(BLOCK_ROWS, wl.T - r0)
    eps = rng(wl.wid, 2, step, block).standard_normal((n, wl.d), dtype=np.float32)
    if wl.x_kind == "normal":
        return eps
    mu, p = mix if mix is not None else (mixture_params(wl)[0], mixture_weights(wl, step))
    labels = rng(wl.wid, 3, step, block).choice(N_COMPONENTS, size=n, p=p)
    return mu[labels] + np.float32(MIX_SIGMA) * eps


def hidden_states(wl: Workload, step: int = 0, rows: np.ndarray | None = None) -> np.ndarray:
    """Token hidden states x [T][d] (or the listed rows) in the workload's storage dtype."""
    mix = None
    if wl.x_kind != "normal":
        mix = (mixture_params(wl)[0], mixture_weights(wl, step))
    if rows is None:
        nblk = (wl.T + BLOCK_ROWS - 1) // BLOCK_ROWS
        out = np.empty((wl.T, wl.d), np.uint16 if wl.dtype == "bf16" else np.float32)
        for b in range(nblk):
            out[b * BLOCK_ROWS:(b + 1) * BLOCK_ROWS] = _store(hidden_block(wl, step, b, mix), wl.dtype)
        return out
    rows = np.asarray(rows, dtype=np.int64)
    out = np.empty((len(rows), wl.d), np.uint16 if wl.dtype == "bf16" else np.float32)
    cache = {}
    for j, r in enumerate(rows):
        b = int(r) // BLOCK_ROWS
        if b not in cache:
            cache[b] = _store(hidden_block(wl, step, b, mix), wl.dtype)
        out[j] = cache[b][int(r) - b * BLOCK_ROWS]
    return out


# --------------------------------------------------------------------------------------------
# Small synthetic cases for parity tests


def integer_router_inputs(T: int, d: int, E: int, seed: int, dtype: str = "bf16", w_shift: int = 6):
    """x in {-2..2} and W in {-2..2} * 2^-w_shift: every partial sum of W x is exact in fp32."""
    g = rng(9001, seed)
    x = g.integers(-2, 3, size=(T, d)).astype(np.float32)
    W = (g.integers(-2, 3, size=(E, d)).astype(np.float32) * np.float32(2.0 ** -w_shift))
    return _store(x, dtype), _store(W, dtype)


def normal_router_inputs(T: int, d: int, E: int, seed: int, dtype: str = "bf16", w_std: float = 0.02):
    g = rng(9002, seed)
    x = g.standard_normal((T, d), dtype=np.float32)
    W = g.standard_normal((E, d), dtype=np.float32) * np.float32(w_std)
    return _store(x, dtype), _store(W, dtype)


def scores(T: int, E: int, kind: str, seed: int) -> np.ndarray:
    """fp32 scores in [0, 1] shaped like router scores, drawn directly (no logits).

    kinds: "beta" (continuous, mean 0.5), "grid" (multiples of 1/8: heavy ties),
    "const" (every score 0.5), "edges" (a mix of 0, -0, 1, tiny subnormal-free
    values and grid values), "saturated" (mostly exactly 1.0 or 0.0).
    """
    g = rng(9003, seed, E)
    if kind == "beta":
        return g.beta(2.0, 2.0, size=(T, E)).astype(np.float32)
    if kind == "grid":
        return (g.integers(0, 9, size=(T, E)) / 8.0).astype(np.float32)
    if kind == "const":
        return np.full((T, E), 0.5, np.float32)
    if kind == "edges":
        choices = np.array([0.0, -0.0, 1.0, 0.5, 0.25, 1e-30, 0.999999940395355, 0.75], np.float32)
        a = choices[g.integers(0, len(choices), size=(T, E))]
        cont = g.random((T, E)).astype(np.float32)
        return np.where(g.random((T, E)) < 0.5, a, cont).astype(np.float32)
    if kind == "saturated":
        a = np.where(g.random((T, E)) < 0.5, np.float32(1.0), np.float32(0.0))
        return a.astype(np.float32)
    raise ValueError(kind)


def bias(E: int, kind: str, seed: int) -> np.ndarray:
    """Expert bias vectors: "zero", "small" (N(0, 0.01^2)), "grid" (multiples of 1/16), "large" (U(-1, 1))."""
    g = rng(9004, seed, E)
    if kind == "zero":
        return np.zeros(E, np.float32)
    if kind == "small":
        return (g.standard_normal(E) * 0.01).astype(np.float32)
    if kind == "grid":
        return (g.integers(-8, 9, size=E) / 16.0).astype(np.float32)
    if kind == "large":
        return g.uniform(-1.0, 1.0, size=E).astype(np.float32)
    raise ValueError(kind)


def count_stream(E: int, total: int, steps: int, kind: str, seed: int) -> np.ndarray:
    """Synthetic per-step load counts [steps][E] int32 for controller parity.

    kinds: "multinomial" (skewed Dirichlet(0.3) loads, fresh each step),
    "drift" (loads from a slowly drifting distribution), "sparse" (most experts
    empty), "mixed" (random small integers, including zero rows).
    """
    g = rng(9005, seed, E, steps)
    out = np.zeros((steps, E), np.int64)
    if kind == "multinomial":
        for t in range(steps):
            out[t] = g.multinomial(total, g.dirichlet(np.full(E, 0.3)))
    elif kind == "drift":
        p = g.dirichlet(np.full(E, 1.0))
        for t in range(steps):
            p = np.clip(p + 0.002 * g.standard_normal(E), 1e-6, None)
            p = p / p.sum()
            out[t] = g.multinomial(total, p)
    elif kind == "sparse":
        for t in range(steps):
            live = g.random(E) < 0.1
            p = np.where(live, g.random(E), 0.0)
            if p.sum() == 0:
                p[0] = 1.0
            out[t] = g.multinomial(total, p / p.sum())
    elif kind == "mixed":
        out = g.integers(0, 4, size=(steps, E))
        out[g.random(steps) < 0.1] = 0
    else:
        raise ValueError(kind)
    return out.astype(np.int32)


def integer_drift_inputs(T: int, d: int, E: int, step: int, seed: int, dtype: str = "bf16", w_shift: int = 6,
                         balanced: bool = False, drift_cols: int = 16, drift_amp: float = 2.0):
    """Integer-valued hidden states whose token groups drift from step to step, and a fixed integer router matrix.

    x has entries in {-2..2} (fresh each step, stream ``step``); the tokens
    fall into four groups, and group k's columns [k c, k c + c), c =
    ``drift_cols``, are set to a shared value round(A sin(2 pi (t + 3k) / 10)),
    A = ``drift_amp``, so the load moves between experts and back over the
    steps.  W has entries in {-2..2} * 2^-w_shift and does not depend on
    ``step``; with ``balanced`` every row is a permutation of the same
    multiset of values (equal norms, so no expert is favoured on average).
    Every partial sum of W x is a multiple of 2^-w_shift well inside fp32's
    exact range, so the logits are exact on any summation order.
    """
    g = rng(9010 if not balanced else 9020, seed, step)
    x = g.integers(-2, 3, size=(T, d)).astype(np.float32)
    grp = g.integers(0, 4, size=T)
    for k in range(4):
        c = float(np.round(drift_amp * np.sin(2.0 * np.pi * (step + 3 * k) / 10.0)))
        x[grp == k, drift_cols * k:drift_cols * k + drift_cols] = c
    if balanced:
        gw = rng(9021, seed)
        base = np.resize(np.array([-2, -1, 0, 1, 2], np.float32), d)
        W = np.stack([gw.permutation(base) for _ in range(E)]) * np.float32(2.0 ** -w_shift)
    else:
        gw = rng(9011, seed)
        W = gw.integers(-2, 3, size=(E, d)).astype(np.float32) * np.float32(2.0 ** -w_shift)
    return _store(x, dtype), _store(W, dtype)

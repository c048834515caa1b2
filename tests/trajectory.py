"""Oracle trajectories of Alg. 1 whose selections are decided the same way on any faithful fp32 implementation.

The GPU router computes the same exact logits as the oracle on
integer-valued inputs (every partial sum is exact in fp32), but its sigmoid
uses the hardware exp2 and reciprocal, so its scores can differ from the
oracle's libm sigmoid in the last bits.  A token's selection (set and rank
order) is then provably the same on both sides when every adjacent pair of
its oracle top-(K+1), ranked by (v desc, index asc) with v = fl32(s + b), is

* strictly apart: v_r - v_{r+1} > ``tol``, far above twice the score error
  (below 1e-6 for scores in (0, 1)) plus the rounding of the addition; or
* an exact logit tie with biases that are equal (then both sides compare
  equal values and the lower index wins) or at least two ulps of v apart
  (then rounding cannot merge or swap them).

Chains of such pairs keep their order (margins add up; equal logits are
transitive), so the top-K set and its rank order agree, hence the counts,
and by induction over the steps the whole bias trajectory.  The gate-weight
bits may still differ (they are ratios of the slightly different scores).
"""
from __future__ import annotations

import numpy as np

import oracle


def safe_tokens(s: np.ndarray, z: np.ndarray, b: np.ndarray, K: int, tol: float = 1e-5) -> np.ndarray:
    """Per token: True when the selection is decided identically for any scores within 1e-6 of ``s``."""
    T, E = s.shape
    v = (s + b[None, :]).astype(np.float32)
    order = np.lexsort((np.broadcast_to(np.arange(E), (T, E)), -v.astype(np.float64)), axis=1)
    top = order[:, :min(K + 1, E)]
    vt = np.take_along_axis(v, top, 1).astype(np.float64)
    zt = np.take_along_axis(z, top, 1)
    bt = b[top].astype(np.float64)
    strict = (vt[:, :-1] - vt[:, 1:]) > tol
    ulp = np.spacing(np.abs(vt[:, :-1]).astype(np.float32)).astype(np.float64)
    db = np.abs(bt[:, :-1] - bt[:, 1:])
    tie_ok = (zt[:, :-1] == zt[:, 1:]) & ((db == 0) | (db >= 2 * ulp))
    return (strict | tie_ok).all(1)


def oracle_step(x, W, state: oracle.ControllerState, K: int, Ki: float, Kd: float, center: bool = True):
    """One oracle iteration: route with the current bias, statistics, update (in place).

    Returns a dict with idx, w, counts, stats [MaxVio, MinVio], the update's
    diagnostics and the per-token safety flags of the selection."""
    s, z = oracle.router_scores(x, W, want_z=True)
    safe = safe_tokens(s, z, state.bias, K)
    idx, w, c = oracle.select(s, state.bias, K)
    stats = oracle.load_stats(c)
    status, diag = oracle.controller_diag(c, state, Ki, Kd, center=center)
    return {"idx": idx, "w": w, "counts": c, "stats": stats, "diag": diag, "status": status, "safe": safe}

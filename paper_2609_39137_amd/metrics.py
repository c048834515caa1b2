"""Load-balance metric families of the paper, aggregated on the host from the
per-step records the GPU path produces (MaxVio/MinVio per layer from
``idb_controller_update_layers`` or ``idb_load_stats``, biases at checkpoints).

* Per step, backbone values are averaged over the layers (Sec. 4.1).
* ``last1k`` and ``avg``: means of the per-step layer means over the final
  1000 steps and over the whole window; ``worst``: the largest MaxVio over
  layers and steps (Sec. 4.1, the results table).
* ``cumulative_excess``: the sum over steps of max(0, V_t - threshold), V_t the
  layer-mean MaxVio of step t, on unsmoothed observations (Sec. 5, the
  derivative-gain ablation uses threshold 1).
* ``bias_drift``: mean |b(t) - b(t - gap)| between checkpoints ``gap`` steps
  apart (Sec. 3, the EMA diagnostic uses 1000 steps).
"""
from __future__ import annotations

import numpy as np


class LoadRecord:
    """Per-step, per-layer MaxVio and MinVio ([steps][L] each), appended step by step."""

    def __init__(self):
        self._maxvio: list[np.ndarray] = []
        self._minvio: list[np.ndarray] = []

    def add(self, stats: np.ndarray) -> None:
        """``stats``: [L][2] (MaxVio, MinVio per layer) or [2] for one layer."""
        a = np.asarray(stats, dtype=np.float64).reshape(-1, 2)
        self._maxvio.append(a[:, 0].copy())
        self._minvio.append(a[:, 1].copy())

    @property
    def maxvio(self) -> np.ndarray:
        return np.stack(self._maxvio)

    @property
    def minvio(self) -> np.ndarray:
        return np.stack(self._minvio)

    def summary(self, last: int = 1000) -> dict:
        mx, mn = self.maxvio, self.minvio
        mx_mean, mn_mean = mx.mean(axis=1), mn.mean(axis=1)
        return {
            "maxvio_last": float(mx_mean[-last:].mean()),
            "maxvio_avg": float(mx_mean.mean()),
            "maxvio_worst": float(mx.max()),
            "minvio_last": float(mn_mean[-last:].mean()),
            "minvio_avg": float(mn_mean.mean()),
            "steps": int(mx.shape[0]),
            "layers": int(mx.shape[1]),
        }

    def cumulative_excess(self, threshold: float = 1.0, start: int = 0, stop: int | None = None) -> float:
        v = self.maxvio.mean(axis=1)[start:stop]
        return float(np.maximum(v - threshold, 0.0).sum())


def bias_drift(b_now: np.ndarray, b_then: np.ndarray) -> float:
    """Mean absolute bias change between two checkpoints (over experts, and layers if given [L][E])."""
    return float(np.mean(np.abs(np.asarray(b_now, np.float64) - np.asarray(b_then, np.float64))))

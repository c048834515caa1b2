"""CPU oracle for the ID Balancing router step and bias controller.

TEST INFRASTRUCTURE ONLY: the plain, slow reference that the GPU library is
checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may import this package.  It shares no code with
the GPU library; the arithmetic lives in ``idb_oracle.c`` (plain C, fp64 where
the paper fixes no precision) and this module only marshals numpy arrays.

Functions and the paper passage each follows (see ``idb_oracle.c`` for the
readings of points the paper leaves open):

* :func:`router_scores` -- logits ``z = W_r x`` and ``s = sigmoid(z)`` (Sec. 2.2)
* :func:`select` -- ``TopK(s + b)``, unbiased gate weights, load counts
  (Eq. pid-routing, Sec. 2.2, Eq. pid-error)
* :func:`router` -- both of the above in one pass
* :func:`controller` -- one ID bias update (Alg. 1, Eq. rapid-update) or the
  DeepSeek sign rule (Eq. pid-deepseek)
* :func:`load_stats` -- MaxVio / MinVio (Eq. vio)
* :func:`controller_diag` -- one update plus its diagnostics (active-gate
  fraction, busiest-10% share, inactive-expert ratio, mean |bias change|)
* :func:`topk_entropy`, :func:`full_entropy`, :func:`softmax_entropy` -- routing
  entropies (Sec. 4.3): top-K gate weights, clamped biased sigmoid scores, and
  the auxiliary-loss router's softmax probabilities
* :func:`qb_alpha`, :func:`qb_update` -- Quantile Balancing's cutoffs and
  target bias, with the EMA variant (Eq. pid-quantile, Eq. pid-quantile-def)
* :func:`aux_stats`, :func:`aux_router` -- the auxiliary-loss router's
  forward statistics f_i, P_i and the loss (Eq. pid-auxloss)
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libidb_oracle.so")
SRC_PATH = os.path.join(_HERE, "idb_oracle.c")
# A deliberately broken copy of the oracle can be loaded instead (mutation
# tests of the pins): IDB_ORACLE_LIB names a prebuilt library to use.
_OVERRIDE = os.environ.get("IDB_ORACLE_LIB")

DTYPE_BF16 = 0
DTYPE_F32 = 1
MODE_ERROR = 0
MODE_SIGN = 1
STATUS_OK = 0
STATUS_INVALID = 1
STATUS_EMPTY = 3

BUILD_CMD = ["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-shared", "-fPIC", "-o", LIB_PATH, SRC_PATH, "-lm"]


def build() -> str:
    """Compile the oracle's C library in place (plain gcc, no GPU code)."""
    subprocess.run(BUILD_CMD, check=True)
    return LIB_PATH


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if _OVERRIDE:
        _lib = _declare(ctypes.CDLL(_OVERRIDE))
        return _lib
    if not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(SRC_PATH):
        build()
    _lib = _declare(ctypes.CDLL(LIB_PATH))
    return _lib


def _declare(lib):
    P = ctypes.c_void_p
    i64, i32, f32, c_int = ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_int
    lib.oracle_num_threads.restype = c_int
    lib.oracle_set_num_threads.argtypes = [c_int]
    lib.oracle_router_scores.argtypes = [P, P, c_int, i64, i32, i32, P, i64, P, P]
    lib.oracle_select.argtypes = [P, P, i64, i32, i32, P, P, P, c_int]
    lib.oracle_router.argtypes = [P, P, c_int, P, i64, i32, i32, i32, P, P, P, c_int, P]
    lib.oracle_controller.argtypes = [P, i32, f32, f32, c_int, c_int, P, P, P, P]
    lib.oracle_controller.restype = c_int
    lib.oracle_load_stats.argtypes = [P, i32, P]
    lib.oracle_step_seconds.argtypes = [P, P, c_int, i64, i32, i32, i32, f32, f32, P, P, P, P, P, P, P, P]
    lib.oracle_step_seconds.restype = ctypes.c_double
    lib.oracle_controller_diag.argtypes = [P, i32, f32, f32, c_int, c_int, P, P, P, P, P]
    lib.oracle_controller_diag.restype = c_int
    lib.oracle_topk_entropy.argtypes = [P, i64, i32]
    lib.oracle_topk_entropy.restype = ctypes.c_double
    lib.oracle_full_entropy.argtypes = [P, P, i64, i32]
    lib.oracle_full_entropy.restype = ctypes.c_double
    lib.oracle_softmax_entropy.argtypes = [P, i64, i32]
    lib.oracle_softmax_entropy.restype = ctypes.c_double
    lib.oracle_qb_alpha.argtypes = [P, P, i64, i32, i32, P]
    lib.oracle_qb_update.argtypes = [P, P, i64, i32, i32, f32, P]
    lib.oracle_aux_stats.argtypes = [P, i64, i32, i32, ctypes.c_double, P, P, P, P, P, P]
    return lib


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data


def _dtype_code(x: np.ndarray) -> int:
    if x.dtype == np.uint16:
        return DTYPE_BF16  # raw bfloat16 bits
    if x.dtype == np.float32:
        return DTYPE_F32
    raise TypeError(f"oracle inputs must be bf16 bits (uint16) or float32, got {x.dtype}")


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's OpenMP loops from now on (timing only)."""
    _load().oracle_set_num_threads(int(n))


def router_scores(x: np.ndarray, W: np.ndarray, rows: np.ndarray | None = None, want_z: bool = False):
    """Scores ``s = sigmoid(W x)`` (fp32) for the listed token rows (all rows by default).

    ``x`` is [T][d], ``W`` is [E][d]; both bf16 bits (uint16) or float32.
    Returns ``s`` [n][E] float32, and also ``z`` [n][E] float64 when ``want_z``.
    """
    lib = _load()
    x = np.ascontiguousarray(x)
    W = np.ascontiguousarray(W)
    code = _dtype_code(x)
    assert _dtype_code(W) == code and x.shape[1] == W.shape[1]
    T, d = x.shape
    E = W.shape[0]
    r = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    n = T if r is None else len(r)
    s = np.empty((n, E), np.float32)
    z = np.empty((n, E), np.float64) if want_z else None
    lib.oracle_router_scores(_ptr(x), _ptr(W), code, T, d, E, _ptr(r), n, _ptr(z), _ptr(s))
    return (s, z) if want_z else s


def select(scores: np.ndarray, bias: np.ndarray, K: int, counts: np.ndarray | None = None):
    """Top-K by ``scores + bias`` with unbiased gate weights and load counts.

    Returns ``(idx [T][K] int32, w [T][K] float32, counts [E] int32)``.  When a
    ``counts`` array is passed it is accumulated into (microbatch summing).
    """
    lib = _load()
    s = np.ascontiguousarray(scores, dtype=np.float32)
    b = np.ascontiguousarray(bias, dtype=np.float32)
    T, E = s.shape
    assert b.shape == (E,) and 1 <= K <= E
    idx = np.empty((T, K), np.int32)
    w = np.empty((T, K), np.float32)
    acc = counts is not None
    c = counts if acc else np.empty(E, np.int32)
    assert c.dtype == np.int32 and c.flags.c_contiguous and c.shape == (E,)
    lib.oracle_select(_ptr(s), _ptr(b), T, E, K, _ptr(idx), _ptr(w), _ptr(c), int(acc))
    return idx, w, c


def router(x: np.ndarray, W: np.ndarray, bias: np.ndarray, K: int, want_scores: bool = False):
    """Whole router step from hidden states: ``(idx, w, counts[, s])``."""
    lib = _load()
    x = np.ascontiguousarray(x)
    W = np.ascontiguousarray(W)
    code = _dtype_code(x)
    assert _dtype_code(W) == code
    T, d = x.shape
    E = W.shape[0]
    b = np.ascontiguousarray(bias, dtype=np.float32)
    idx = np.empty((T, K), np.int32)
    w = np.empty((T, K), np.float32)
    c = np.empty(E, np.int32)
    s = np.empty((T, E), np.float32) if want_scores else None
    lib.oracle_router(_ptr(x), _ptr(W), code, _ptr(b), T, d, E, K, _ptr(idx), _ptr(w), _ptr(c), 0, _ptr(s))
    return (idx, w, c, s) if want_scores else (idx, w, c)


class ControllerState:
    """Controller state of Alg. 1: bias b, previous error e_prev, step, status."""

    def __init__(self, E: int):
        self.bias = np.zeros(E, np.float32)
        self.e_prev = np.zeros(E, np.float32)
        self.step = np.zeros(1, np.int64)
        self.status = np.zeros(1, np.int32)

    def copy(self) -> "ControllerState":
        c = ControllerState(len(self.bias))
        c.bias[:] = self.bias
        c.e_prev[:] = self.e_prev
        c.step[:] = self.step
        c.status[:] = self.status
        return c


def controller(counts: np.ndarray, state: ControllerState, Ki: float, Kd: float, mode: int = MODE_ERROR,
               center: bool = True) -> int:
    """One bias update in place; returns the status code (0 ok, 1 invalid, 3 empty)."""
    lib = _load()
    c = np.ascontiguousarray(counts, dtype=np.int32)
    E = len(c)
    assert state.bias.shape == (E,)
    return int(lib.oracle_controller(_ptr(c), E, float(Ki), float(Kd), int(mode), int(bool(center)),
                                     _ptr(state.bias), _ptr(state.e_prev), _ptr(state.step), _ptr(state.status)))


def load_stats(counts: np.ndarray) -> np.ndarray:
    """``[MaxVio, MinVio]`` as float64 (NaN for an empty batch)."""
    lib = _load()
    c = np.ascontiguousarray(counts, dtype=np.int32)
    out = np.empty(2, np.float64)
    lib.oracle_load_stats(_ptr(c), len(c), _ptr(out))
    return out


def step_seconds(x: np.ndarray, W: np.ndarray, K: int, Ki: float, Kd: float, state: ControllerState) -> float:
    """Wall-clock seconds of one oracle step (router + controller + stats)."""
    lib = _load()
    x = np.ascontiguousarray(x)
    W = np.ascontiguousarray(W)
    code = _dtype_code(x)
    T, d = x.shape
    E = W.shape[0]
    idx = np.empty((T, K), np.int32)
    w = np.empty((T, K), np.float32)
    c = np.empty(E, np.int32)
    stats = np.empty(2, np.float64)
    return float(lib.oracle_step_seconds(_ptr(x), _ptr(W), code, T, d, E, K, float(Ki), float(Kd),
                                         _ptr(state.bias), _ptr(state.e_prev), _ptr(state.step),
                                         _ptr(state.status), _ptr(idx), _ptr(w), _ptr(c), _ptr(stats)))


def qb_alpha(scores: np.ndarray, bias: np.ndarray, K: int) -> np.ndarray:
    """Quantile Balancing cutoffs (Eq. pid-quantile-def): per token the (K+1)-th largest fp32 ``s + b``."""
    lib = _load()
    s = np.ascontiguousarray(scores, dtype=np.float32)
    b = np.ascontiguousarray(bias, dtype=np.float32)
    T, E = s.shape
    assert 1 <= K < E and b.shape == (E,)
    alpha = np.empty(T, np.float32)
    lib.oracle_qb_alpha(_ptr(s), _ptr(b), T, E, K, _ptr(alpha))
    return alpha


def qb_update(scores: np.ndarray, alpha: np.ndarray, K: int, rho: float, bias: np.ndarray) -> np.ndarray:
    """Quantile Balancing's bias update (Eq. pid-quantile; EMA with ``rho`` > 0) in place on ``bias``."""
    lib = _load()
    s = np.ascontiguousarray(scores, dtype=np.float32)
    a = np.ascontiguousarray(alpha, dtype=np.float32)
    T, E = s.shape
    assert 1 <= K < E and a.shape == (T,) and bias.shape == (E,) and bias.dtype == np.float32
    assert bias.flags.c_contiguous
    lib.oracle_qb_update(_ptr(s), _ptr(a), T, E, K, float(rho), _ptr(bias))
    return bias


def controller_diag(counts: np.ndarray, state: ControllerState, Ki: float, Kd: float, mode: int = MODE_ERROR,
                    center: bool = True):
    """One bias update in place plus ``[active-gate fraction, busiest-10% share, inactive ratio, mean |db|]``."""
    lib = _load()
    c = np.ascontiguousarray(counts, dtype=np.int32)
    E = len(c)
    diag = np.empty(4, np.float64)
    st = lib.oracle_controller_diag(_ptr(c), E, float(Ki), float(Kd), int(mode), int(bool(center)),
                                    _ptr(state.bias), _ptr(state.e_prev), _ptr(state.step), _ptr(state.status),
                                    _ptr(diag))
    return int(st), diag


def topk_entropy(w: np.ndarray) -> float:
    """Mean over tokens of H_topK = -sum w log w (nats) for gate weights ``w`` [T][K]."""
    a = np.ascontiguousarray(w, dtype=np.float32)
    return float(_load().oracle_topk_entropy(_ptr(a), a.shape[0], a.shape[1]))


def full_entropy(scores: np.ndarray, bias: np.ndarray) -> float:
    """Mean over tokens of H_full over the clamped biased scores max(s + b, 0), normalised (nats)."""
    s = np.ascontiguousarray(scores, dtype=np.float32)
    b = np.ascontiguousarray(bias, dtype=np.float32)
    return float(_load().oracle_full_entropy(_ptr(s), _ptr(b), s.shape[0], s.shape[1]))


def softmax_entropy(z: np.ndarray) -> float:
    """Mean over tokens of H_full over the softmax probabilities of fp32 logits ``z`` [T][E] (nats; the
    auxiliary-loss router's full-pool entropy, Sec. 4.3)."""
    a = np.ascontiguousarray(z, dtype=np.float32)
    return float(_load().oracle_softmax_entropy(_ptr(a), a.shape[0], a.shape[1]))


def aux_stats(z: np.ndarray, K: int, alpha: float):
    """Auxiliary-loss forward statistics (Eq. pid-auxloss) from logits z [T][E].

    p = softmax(z) per token (fp64); Top-K ranked on the fp32-rounded logits,
    lowest index among equals; gate weights = selected p renormalised.
    Returns ``(idx [T][K] int32, w [T][K] float32, counts [E] int32,
    f [E] float64, P [E] float64, loss float)``.
    """
    lib = _load()
    zz = np.ascontiguousarray(z, dtype=np.float64)
    T, E = zz.shape
    assert 1 <= K <= E and T >= 1
    idx = np.empty((T, K), np.int32)
    w = np.empty((T, K), np.float32)
    c = np.empty(E, np.int32)
    f = np.empty(E, np.float64)
    P = np.empty(E, np.float64)
    loss = np.zeros(1, np.float64)
    lib.oracle_aux_stats(_ptr(zz), T, E, K, float(alpha), _ptr(idx), _ptr(w), _ptr(c), _ptr(f), _ptr(P),
                         _ptr(loss))
    return idx, w, c, f, P, float(loss[0])


def aux_router(x: np.ndarray, W: np.ndarray, K: int, alpha: float, rows: np.ndarray | None = None):
    """Logits from hidden states (R1), then :func:`aux_stats` of those rows."""
    _, z = router_scores(x, W, rows=rows, want_z=True)
    return aux_stats(z, K, alpha)

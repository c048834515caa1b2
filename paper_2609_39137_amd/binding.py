"""Python binding of the C ABI in ``include/idb.h`` (libidb.so).

Argument marshalling only: torch tensors supply device pointers and the
current HIP stream; every step of the router and controller runs in the HIP
kernels behind the ABI.  There is no fallback: if ``libidb.so`` is missing or
the arguments are rejected, the call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libidb.so")

IDB_OK = 0
IDB_ERR_INVALID_ARG = 1
IDB_ERR_UNSUPPORTED = 2
IDB_ERR_EMPTY_BATCH = 3
IDB_ERR_HIP = 4

IDB_DTYPE_BF16 = 0
IDB_DTYPE_F32 = 1
IDB_WEIGHT_ROW_MAJOR = 0
IDB_WEIGHT_PACKED = 1
IDB_INTEGRAL_ERROR = 0
IDB_INTEGRAL_SIGN = 1

EXPORTED = (
    "idb_router_workspace_bytes", "idb_router_forward", "idb_router_score_select", "idb_router_merge",
    "idb_router_variant_info", "idb_select_from_scores", "idb_controller_update", "idb_load_stats",
    "idb_status_string", "idb_last_error", "idb_router_packed_weight_bytes", "idb_router_pack_weight",
    "idb_controller_step", "idb_router_step", "idb_qb_router_workspace_bytes", "idb_qb_router_forward",
    "idb_qb_update", "idb_controller_update_layers", "idb_routing_entropy_workspace_bytes", "idb_routing_entropy",
    "idb_aux_router_workspace_bytes", "idb_aux_router_forward", "idb_router_merge_step",
    "idb_router_step_noalloc", "idb_routing_entropy_softmax", "idb_router_score_select_timed",
)


class IdbError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn}: status {status}: {msg}")
        self.status = status


class idb_controller_cfg(ctypes.Structure):
    _fields_ = [("E", ctypes.c_int32), ("Ki", ctypes.c_float), ("Kd", ctypes.c_float),
                ("integral_mode", ctypes.c_int32), ("center", ctypes.c_int32)]


class idb_controller_state(ctypes.Structure):
    _fields_ = [("bias", ctypes.c_void_p), ("e_prev", ctypes.c_void_p), ("step", ctypes.c_void_p),
                ("status", ctypes.c_void_p)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libidb.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_39137_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    router_args = [P, P, i32, i32, P, i64, i32, i32, i32, P, P, P, i32, P, P, sz, i32, P]
    L.idb_router_workspace_bytes.argtypes = [i64, i32, i32, i32, i32, i32]
    L.idb_router_workspace_bytes.restype = sz
    for name in ("idb_router_forward", "idb_router_score_select"):
        getattr(L, name).argtypes = router_args
        getattr(L, name).restype = ctypes.c_int
    L.idb_router_score_select_timed.argtypes = router_args + [P, P]
    L.idb_router_score_select_timed.restype = ctypes.c_int
    L.idb_router_merge.argtypes = [i64, i32, i32, i32, i32, P, P, P, P, sz, i32, P]
    L.idb_router_merge.restype = ctypes.c_int
    L.idb_router_packed_weight_bytes.argtypes = [i32, i32, i32]
    L.idb_router_packed_weight_bytes.restype = sz
    L.idb_router_pack_weight.argtypes = [P, i32, i32, i32, P, P]
    L.idb_router_pack_weight.restype = ctypes.c_int
    L.idb_router_variant_info.argtypes = [i64, i32, i32, i32, i32, i32, P]
    L.idb_router_variant_info.restype = ctypes.c_int
    L.idb_select_from_scores.argtypes = [P, P, i64, i32, i32, P, P, P, i32, P]
    L.idb_select_from_scores.restype = ctypes.c_int
    L.idb_controller_update.argtypes = [P, ctypes.POINTER(idb_controller_cfg), ctypes.POINTER(idb_controller_state), P]
    L.idb_controller_update.restype = ctypes.c_int
    L.idb_load_stats.argtypes = [P, i32, P, P]
    L.idb_load_stats.restype = ctypes.c_int
    L.idb_controller_step.argtypes = [P, ctypes.POINTER(idb_controller_cfg), ctypes.POINTER(idb_controller_state), P,
                                      P]
    L.idb_controller_step.restype = ctypes.c_int
    L.idb_router_step.argtypes = [P, P, i32, i32, i64, i32, i32, ctypes.POINTER(idb_controller_cfg),
                                  ctypes.POINTER(idb_controller_state), P, P, P, i32, P, P, sz, i32, P]
    L.idb_router_step.restype = ctypes.c_int
    L.idb_router_merge_step.argtypes = [i64, i32, i32, i32, ctypes.POINTER(idb_controller_cfg),
                                        ctypes.POINTER(idb_controller_state), P, P, P, P, P, sz, i32, P]
    L.idb_router_merge_step.restype = ctypes.c_int
    L.idb_router_step_noalloc.argtypes = [P, P, i32, i32, i64, i32, i32, ctypes.POINTER(idb_controller_cfg),
                                          ctypes.POINTER(idb_controller_state), P, P, P, i32, P, i32, P]
    L.idb_router_step_noalloc.restype = ctypes.c_int
    L.idb_qb_router_workspace_bytes.argtypes = [i64, i32, i32, i32, i32, i32]
    L.idb_qb_router_workspace_bytes.restype = sz
    L.idb_qb_router_forward.argtypes = [P, P, i32, i32, P, i64, i32, i32, i32, P, P, P, i32, P, P, P, sz, i32, P]
    L.idb_qb_router_forward.restype = ctypes.c_int
    L.idb_qb_update.argtypes = [P, P, i64, i32, i32, ctypes.c_float, P, P, P, P]
    L.idb_qb_update.restype = ctypes.c_int
    L.idb_controller_update_layers.argtypes = [P, i32, ctypes.POINTER(idb_controller_cfg),
                                               ctypes.POINTER(idb_controller_state), P, P, P]
    L.idb_controller_update_layers.restype = ctypes.c_int
    L.idb_routing_entropy_workspace_bytes.argtypes = []
    L.idb_routing_entropy_workspace_bytes.restype = sz
    L.idb_routing_entropy.argtypes = [P, i64, i32, P, P, i32, P, sz, P, P]
    L.idb_routing_entropy.restype = ctypes.c_int
    L.idb_routing_entropy_softmax.argtypes = [P, i64, i32, P, i32, P, sz, P, P]
    L.idb_routing_entropy_softmax.restype = ctypes.c_int
    L.idb_aux_router_workspace_bytes.argtypes = [i64, i32, i32, i32, i32, i32]
    L.idb_aux_router_workspace_bytes.restype = sz
    L.idb_aux_router_forward.argtypes = [P, P, i32, i32, i64, i32, i32, i32, ctypes.c_double, P, P, P, P, P, P, P,
                                         P, P, sz, i32, P]
    L.idb_aux_router_forward.restype = ctypes.c_int
    L.idb_status_string.argtypes = [ctypes.c_int]
    L.idb_status_string.restype = ctypes.c_char_p
    L.idb_last_error.argtypes = []
    L.idb_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def idb_status_string(status: int) -> str:
    return lib().idb_status_string(status).decode()


def idb_last_error() -> str:
    return lib().idb_last_error().decode()


def _check(fn: str, status: int) -> None:
    if status != IDB_OK:
        raise IdbError(fn, status, f"{idb_status_string(status)}: {idb_last_error()}")


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _ptr(t: torch.Tensor | None) -> int | None:
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("tensors passed to libidb must be contiguous device tensors")
    return t.data_ptr()


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return IDB_DTYPE_BF16
    if t.dtype == torch.float32:
        return IDB_DTYPE_F32
    raise TypeError(f"router inputs must be bfloat16 or float32, got {t.dtype}")


# ---------------------------------------------------------------------------- router


def idb_router_workspace_bytes(T: int, d: int, E: int, K: int, dtype: int, variant: int = 0) -> int:
    return int(lib().idb_router_workspace_bytes(T, d, E, K, dtype, variant))


def idb_router_variant_info(T: int, d: int, E: int, K: int, dtype: int, variant: int = 0) -> dict:
    out = (ctypes.c_int32 * 5)()
    _check("idb_router_variant_info", lib().idb_router_variant_info(T, d, E, K, dtype, variant, out))
    return {"tokens_per_wg": out[0], "slices": out[1], "waves": out[2], "experts_per_wave": out[3], "variant": out[4]}


def idb_router_packed_weight_bytes(E: int, d: int, dtype: int) -> int:
    return int(lib().idb_router_packed_weight_bytes(E, d, dtype))


def idb_router_pack_weight(W_g, W_packed, stream=None):
    """Write ``W_g`` [E][d] into ``W_packed`` (same shape and dtype) in the MFMA A-operand layout."""
    E, d = W_g.shape
    if W_packed.shape != W_g.shape or W_packed.dtype != W_g.dtype:
        raise ValueError("W_packed must match W_g in shape and dtype")
    st = lib().idb_router_pack_weight(_ptr(W_g), _dtype_code(W_g), E, d, _ptr(W_packed), _stream(stream))
    _check("idb_router_pack_weight", st)


def _router_call(fn: str, x, W_g, bias, K, expert_idx, gate_w, counts, accumulate, scores_dump, workspace,
                 variant, stream, weight_layout=IDB_WEIGHT_ROW_MAJOR, extra=()):
    T, d = x.shape
    E = W_g.shape[0]
    if W_g.shape[1] != d or W_g.dtype != x.dtype or bias.shape != (E,) or bias.dtype != torch.float32:
        raise ValueError("router operands disagree in shape or dtype")
    if expert_idx.shape != (T, K) or gate_w.shape != (T, K) or counts.shape != (E,):
        raise ValueError("router outputs have the wrong shape")
    if scores_dump is not None and (scores_dump.dtype != torch.float32 or scores_dump.numel() != T * E):
        raise ValueError("scores_dump must be a float32 tensor of T*E elements")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = getattr(lib(), fn)(_ptr(x), _ptr(W_g), _dtype_code(x), int(weight_layout), _ptr(bias), T, d, E, K,
                            _ptr(expert_idx),
                            _ptr(gate_w), _ptr(counts), int(bool(accumulate)), _ptr(scores_dump),
                            _ptr(workspace), ws_bytes, int(variant), _stream(stream), *extra)
    _check(fn, st)


def idb_router_forward(x, W_g, bias, K, expert_idx, gate_w, counts, accumulate=False, scores_dump=None,
                       workspace=None, variant=0, stream=None, weight_layout=IDB_WEIGHT_ROW_MAJOR):
    """Router step (gate contraction, sigmoid, biased Top-K, gate weights, counts) on ``stream``."""
    _router_call("idb_router_forward", x, W_g, bias, K, expert_idx, gate_w, counts, accumulate, scores_dump,
                 workspace, variant, stream, weight_layout)


def idb_router_score_select(x, W_g, bias, K, expert_idx, gate_w, counts, accumulate=False, scores_dump=None,
                            workspace=None, variant=0, stream=None, weight_layout=IDB_WEIGHT_ROW_MAJOR):
    _router_call("idb_router_score_select", x, W_g, bias, K, expert_idx, gate_w, counts, accumulate, scores_dump,
                 workspace, variant, stream, weight_layout)


def _event_handle(ev) -> int | None:
    """Raw HIP event of a ``torch.cuda.Event`` (recorded once, so it exists), or None."""
    if ev is None:
        return None
    if not getattr(ev, "cuda_event", 0):
        raise ValueError("record the event once before passing it (torch creates events on first record)")
    return int(ev.cuda_event)


def idb_router_score_select_timed(x, W_g, bias, K, expert_idx, gate_w, counts, start_event, stop_event,
                                  accumulate=False, scores_dump=None, workspace=None, variant=0, stream=None,
                                  weight_layout=IDB_WEIGHT_ROW_MAJOR):
    """:func:`idb_router_score_select` with the fused kernel's own start and end timestamps written into the
    two ``torch.cuda.Event`` objects (``enable_timing=True``, each recorded once beforehand)."""
    _router_call("idb_router_score_select_timed", x, W_g, bias, K, expert_idx, gate_w, counts, accumulate,
                 scores_dump, workspace, variant, stream, weight_layout,
                 extra=(_event_handle(start_event), _event_handle(stop_event)))


def idb_router_merge(T, d, E, K, dtype, expert_idx, gate_w, counts, workspace=None, variant=0, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib().idb_router_merge(T, d, E, K, dtype, _ptr(expert_idx), _ptr(gate_w), _ptr(counts), _ptr(workspace),
                                ws_bytes, int(variant), _stream(stream))
    _check("idb_router_merge", st)


# ---------------------------------------------------------------------------- selection


def idb_select_from_scores(scores, bias, K, expert_idx, gate_w, counts, accumulate=False, stream=None):
    T, E = scores.shape
    if scores.dtype != torch.float32 or bias.shape != (E,) or expert_idx.shape != (T, K) or counts.shape != (E,):
        raise ValueError("select operands have the wrong shape or dtype")
    st = lib().idb_select_from_scores(_ptr(scores), _ptr(bias), T, E, K, _ptr(expert_idx), _ptr(gate_w),
                                      _ptr(counts), int(bool(accumulate)), _stream(stream))
    _check("idb_select_from_scores", st)


# ---------------------------------------------------------------------------- controller


@dataclass
class ControllerCfg:
    E: int
    Ki: float = 6e-3
    Kd: float = 6e-3
    integral_mode: int = IDB_INTEGRAL_ERROR
    center: bool = True

    def c(self) -> idb_controller_cfg:
        return idb_controller_cfg(self.E, self.Ki, self.Kd, self.integral_mode, int(bool(self.center)))


class ControllerState:
    """Device-resident controller state (bias, e_prev, step, status), zero-initialised; with ``layers``, the
    state of that many MoE layers ([L][E] and [L])."""

    def __init__(self, E: int, device="cuda", layers: int | None = None):
        lead = () if layers is None else (layers,)
        self.bias = torch.zeros(lead + (E,), dtype=torch.float32, device=device)
        self.e_prev = torch.zeros(lead + (E,), dtype=torch.float32, device=device)
        self.step = torch.zeros(layers or 1, dtype=torch.int64, device=device)
        self.status = torch.zeros(layers or 1, dtype=torch.int32, device=device)

    def c(self) -> idb_controller_state:
        return idb_controller_state(_ptr(self.bias), _ptr(self.e_prev), _ptr(self.step), _ptr(self.status))

    _FIELDS = ("bias", "e_prev", "step", "status")

    def state_dict(self) -> dict:
        """Host copies of the full controller state (bias, e_prev, step, status; Alg. 1): a checkpoint.
        Synchronises with the device; restoring it continues the trajectory bit for bit."""
        return {k: getattr(self, k).detach().to("cpu", copy=True) for k in self._FIELDS}

    def load_state_dict(self, d: dict) -> None:
        """Restore a :meth:`state_dict` (same shapes and dtypes; copied into the existing device buffers, so
        pointers held elsewhere, e.g. by captured graphs, stay valid)."""
        for k in self._FIELDS:
            src, dst = d[k], getattr(self, k)
            if tuple(src.shape) != tuple(dst.shape) or src.dtype != dst.dtype:
                raise ValueError(f"{k}: expected {tuple(dst.shape)} {dst.dtype}, got {tuple(src.shape)} {src.dtype}")
        for k in self._FIELDS:
            getattr(self, k).copy_(d[k])


def idb_controller_update(counts, cfg: ControllerCfg, state: ControllerState, stream=None):
    """One ID controller update of ``state`` from ``counts`` on ``stream``."""
    c_cfg, c_state = cfg.c(), state.c()
    st = lib().idb_controller_update(_ptr(counts), ctypes.byref(c_cfg), ctypes.byref(c_state), _stream(stream))
    _check("idb_controller_update", st)


def idb_load_stats(counts, out, stream=None):
    """MaxVio, MinVio of ``counts`` into the device double[2] ``out``."""
    if out.dtype != torch.float64 or out.numel() != 2:
        raise ValueError("out must be a float64 tensor of 2 elements")
    st = lib().idb_load_stats(_ptr(counts), counts.numel(), _ptr(out), _stream(stream))
    _check("idb_load_stats", st)


def idb_controller_step(counts, cfg: ControllerCfg, state: ControllerState, out, stream=None):
    """MaxVio/MinVio of ``counts`` into ``out`` and one ID update of ``state``, in one launch."""
    if out.dtype != torch.float64 or out.numel() != 2:
        raise ValueError("out must be a float64 tensor of 2 elements")
    c_cfg, c_state = cfg.c(), state.c()
    st = lib().idb_controller_step(_ptr(counts), ctypes.byref(c_cfg), ctypes.byref(c_state), _ptr(out),
                                   _stream(stream))
    _check("idb_controller_step", st)


def idb_router_step(x, W_g, K, cfg: ControllerCfg, state: ControllerState, expert_idx, gate_w, counts,
                    accumulate=False, out=None, workspace=None, variant=0, stream=None,
                    weight_layout=IDB_WEIGHT_ROW_MAJOR):
    """One iteration for one batch: route with ``state.bias``, then MaxVio/MinVio into ``out`` (optional)
    and the ID update of ``state`` from the finished ``counts``."""
    T, d = x.shape
    E = cfg.E
    if W_g.shape != (E, d) or W_g.dtype != x.dtype or state.bias.shape != (E,):
        raise ValueError("router operands disagree in shape or dtype")
    if expert_idx.shape != (T, K) or gate_w.shape != (T, K) or counts.shape != (E,):
        raise ValueError("router outputs have the wrong shape")
    if out is not None and (out.dtype != torch.float64 or out.numel() != 2):
        raise ValueError("out must be a float64 tensor of 2 elements")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    c_cfg, c_state = cfg.c(), state.c()
    st = lib().idb_router_step(_ptr(x), _ptr(W_g), _dtype_code(x), int(weight_layout), T, d, K, ctypes.byref(c_cfg),
                               ctypes.byref(c_state), _ptr(expert_idx), _ptr(gate_w), _ptr(counts),
                               int(bool(accumulate)), _ptr(out), _ptr(workspace), ws_bytes, int(variant),
                               _stream(stream))
    _check("idb_router_step", st)


def idb_router_step_noalloc(x, W_g, K, cfg: ControllerCfg, state: ControllerState, expert_idx, gate_w, counts,
                            accumulate=False, out=None, variant=0, stream=None, weight_layout=IDB_WEIGHT_ROW_MAJOR):
    """:func:`idb_router_step` with the library's fixed device scratch as the workspace (allocates nothing)."""
    T, d = x.shape
    E = cfg.E
    if W_g.shape != (E, d) or W_g.dtype != x.dtype or state.bias.shape != (E,):
        raise ValueError("router operands disagree in shape or dtype")
    if expert_idx.shape != (T, K) or gate_w.shape != (T, K) or counts.shape != (E,):
        raise ValueError("router outputs have the wrong shape")
    if out is not None and (out.dtype != torch.float64 or out.numel() != 2):
        raise ValueError("out must be a float64 tensor of 2 elements")
    c_cfg, c_state = cfg.c(), state.c()
    st = lib().idb_router_step_noalloc(_ptr(x), _ptr(W_g), _dtype_code(x), int(weight_layout), T, d, K,
                                       ctypes.byref(c_cfg), ctypes.byref(c_state), _ptr(expert_idx), _ptr(gate_w),
                                       _ptr(counts), int(bool(accumulate)), _ptr(out), int(variant), _stream(stream))
    _check("idb_router_step_noalloc", st)


def idb_router_merge_step(T, d, K, dtype, cfg: ControllerCfg, state: ControllerState, expert_idx, gate_w, counts,
                          out=None, workspace=None, variant=0, stream=None):
    """The second launch of :func:`idb_router_step`, after :func:`idb_router_score_select` on the same stream:
    the slice merge with MaxVio/MinVio and the ID update in its last workgroup (or the controller step)."""
    E = cfg.E
    if expert_idx.shape != (T, K) or gate_w.shape != (T, K) or counts.shape != (E,):
        raise ValueError("router outputs have the wrong shape")
    if out is not None and (out.dtype != torch.float64 or out.numel() != 2):
        raise ValueError("out must be a float64 tensor of 2 elements")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    c_cfg, c_state = cfg.c(), state.c()
    st = lib().idb_router_merge_step(T, d, K, int(dtype), ctypes.byref(c_cfg), ctypes.byref(c_state),
                                     _ptr(expert_idx), _ptr(gate_w), _ptr(counts), _ptr(out), _ptr(workspace),
                                     ws_bytes, int(variant), _stream(stream))
    _check("idb_router_merge_step", st)


# ---------------------------------------------------------------------------- Quantile Balancing


def idb_qb_router_workspace_bytes(T: int, d: int, E: int, K: int, dtype: int, variant: int = 0) -> int:
    return int(lib().idb_qb_router_workspace_bytes(T, d, E, K, dtype, variant))


def idb_qb_router_forward(x, W_g, bias, K, expert_idx, gate_w, counts, scores_t, alpha, accumulate=False,
                          workspace=None, variant=0, stream=None, weight_layout=IDB_WEIGHT_ROW_MAJOR):
    """Router step that also writes Quantile Balancing's inputs: ``alpha`` [T] (cutoffs) and ``scores_t`` [E][T]."""
    T, d = x.shape
    E = W_g.shape[0]
    if W_g.shape[1] != d or W_g.dtype != x.dtype or bias.shape != (E,) or bias.dtype != torch.float32:
        raise ValueError("router operands disagree in shape or dtype")
    if expert_idx.shape != (T, K) or gate_w.shape != (T, K) or counts.shape != (E,):
        raise ValueError("router outputs have the wrong shape")
    if scores_t.shape != (E, T) or scores_t.dtype != torch.float32 or alpha.shape != (T,) or \
            alpha.dtype != torch.float32:
        raise ValueError("scores_t must be float32 [E][T] and alpha float32 [T]")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib().idb_qb_router_forward(_ptr(x), _ptr(W_g), _dtype_code(x), int(weight_layout), _ptr(bias), T, d, E, K,
                                     _ptr(expert_idx), _ptr(gate_w), _ptr(counts), int(bool(accumulate)),
                                     _ptr(scores_t), _ptr(alpha), _ptr(workspace), ws_bytes, int(variant),
                                     _stream(stream))
    _check("idb_qb_router_forward", st)


def idb_qb_update(scores_t, alpha, K, rho, bias, stream=None, counts=None, stats=None):
    """Quantile Balancing's bias update (exact per-expert quantile; EMA for ``rho`` > 0), ``bias`` in place;
    with ``counts`` and ``stats`` (fp64 [2]) also MaxVio/MinVio of the counts, in the same launch."""
    E, T = scores_t.shape
    if scores_t.dtype != torch.float32 or alpha.shape != (T,) or bias.shape != (E,) or bias.dtype != torch.float32:
        raise ValueError("Quantile Balancing operands have the wrong shape or dtype")
    if (counts is None) != (stats is None):
        raise ValueError("counts and stats go together")
    if counts is not None and (counts.shape != (E,) or counts.dtype != torch.int32 or stats.shape != (2,)
                               or stats.dtype != torch.float64):
        raise ValueError("counts must be int32 [E] and stats fp64 [2]")
    st = lib().idb_qb_update(_ptr(scores_t), _ptr(alpha), T, E, K, float(rho), _ptr(bias),
                             _ptr(counts) if counts is not None else None,
                             _ptr(stats) if stats is not None else None, _stream(stream))
    _check("idb_qb_update", st)


# ---------------------------------------------------------------------------- auxiliary-loss statistics


def idb_aux_router_workspace_bytes(T, d, E, K, dtype=IDB_DTYPE_BF16, variant=0) -> int:
    return int(lib().idb_aux_router_workspace_bytes(T, d, E, K, dtype, variant))


def idb_aux_router_forward(x, W_g, K, alpha, expert_idx, gate_w, counts, f, P, loss, workspace, logits_dump=None,
                           variant=0, stream=None, weight_layout=IDB_WEIGHT_ROW_MAJOR, stats=None):
    """Softmax router without bias and its auxiliary-loss statistics f, P and the loss (Eq. pid-auxloss);
    ``stats`` (float64 [2], optional) receives MaxVio/MinVio."""
    T, d = x.shape
    E = W_g.shape[0]
    if W_g.shape[1] != d or W_g.dtype != x.dtype:
        raise ValueError("router operands disagree in shape or dtype")
    if expert_idx.shape != (T, K) or gate_w.shape != (T, K) or counts.shape != (E,):
        raise ValueError("router outputs have the wrong shape")
    for name, t, shape in (("f", f, (E,)), ("P", P, (E,)), ("loss", loss, (1,))):
        if t.shape != shape or t.dtype != torch.float64:
            raise ValueError(f"{name} must be float64 of shape {shape}")
    if logits_dump is not None and (logits_dump.shape != (T, E) or logits_dump.dtype != torch.float32):
        raise ValueError("logits_dump must be float32 [T][E]")
    if stats is not None and (stats.shape != (2,) or stats.dtype != torch.float64):
        raise ValueError("stats must be float64 [2]")
    ws_bytes = workspace.numel() * workspace.element_size()
    st = lib().idb_aux_router_forward(_ptr(x), _ptr(W_g), _dtype_code(x), int(weight_layout), T, d, E, K,
                                      float(alpha), _ptr(expert_idx), _ptr(gate_w), _ptr(counts), _ptr(f), _ptr(P),
                                      _ptr(loss), _ptr(stats), _ptr(logits_dump), _ptr(workspace), ws_bytes,
                                      int(variant), _stream(stream))
    _check("idb_aux_router_forward", st)


# ---------------------------------------------------------------------------- layers and diagnostics


def idb_controller_update_layers(counts, cfg: ControllerCfg, state: ControllerState, stats=None, diag=None,
                                 stream=None):
    """All layers' updates in one launch: ``counts`` [L][E]; optional ``stats`` [L][2] and ``diag`` [L][4]."""
    L, E = counts.shape
    if E != cfg.E or state.bias.shape != (L, E) or state.step.shape != (L,):
        raise ValueError("layer state does not match counts")
    for t, n in ((stats, 2), (diag, 4)):
        if t is not None and (t.dtype != torch.float64 or t.shape != (L, n)):
            raise ValueError("stats must be float64 [L][2] and diag float64 [L][4]")
    c_cfg, c_state = cfg.c(), state.c()
    st = lib().idb_controller_update_layers(_ptr(counts), L, ctypes.byref(c_cfg), ctypes.byref(c_state), _ptr(stats),
                                            _ptr(diag), _stream(stream))
    _check("idb_controller_update_layers", st)


def idb_routing_entropy(gate_w, out, scores=None, bias=None, workspace=None, stream=None):
    """Mean top-K and full-pool routing entropies (nats) into the device double[2] ``out``."""
    T, K = gate_w.shape
    E = 0 if scores is None else scores.shape[1]
    if out.dtype != torch.float64 or out.numel() != 2:
        raise ValueError("out must be a float64 tensor of 2 elements")
    if scores is not None and (scores.shape[0] != T or bias is None or bias.shape != (E,)):
        raise ValueError("scores must be [T][E] with a bias of E")
    if workspace is None:
        workspace = torch.empty(int(lib().idb_routing_entropy_workspace_bytes()), dtype=torch.uint8,
                                device=gate_w.device)
    st = lib().idb_routing_entropy(_ptr(gate_w), T, K, _ptr(scores), _ptr(bias), E, _ptr(workspace),
                                   workspace.numel(), _ptr(out), _stream(stream))
    _check("idb_routing_entropy", st)


def idb_routing_entropy_softmax(gate_w, logits, out, workspace=None, stream=None):
    """Mean top-K entropy of ``gate_w`` and mean full-pool entropy of softmax(``logits``) (nats; the
    auxiliary-loss router's score family) into the device double[2] ``out``."""
    T, K = gate_w.shape
    if logits.dim() != 2 or logits.shape[0] != T or logits.dtype != torch.float32:
        raise ValueError("logits must be float32 [T][E]")
    if out.dtype != torch.float64 or out.numel() != 2:
        raise ValueError("out must be a float64 tensor of 2 elements")
    if workspace is None:
        workspace = torch.empty(int(lib().idb_routing_entropy_workspace_bytes()), dtype=torch.uint8,
                                device=gate_w.device)
    st = lib().idb_routing_entropy_softmax(_ptr(gate_w), T, K, _ptr(logits), logits.shape[1], _ptr(workspace),
                                           workspace.numel(), _ptr(out), _stream(stream))
    _check("idb_routing_entropy_softmax", st)

"""C ABI checks that need no GPU: the library loads, exports every function
include/idb.h declares, and rejects invalid arguments before any HIP call
(the pointers below are never dereferenced)."""
import ctypes
import os
import re

import pytest

from paper_2609_39137_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
A16 = 1 << 20  # a 16-byte aligned fake device address, never dereferenced


def header_functions():
    text = open(os.path.join(ROOT, "include", "idb.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(idb_[a-z_]+)\s*\(", text)))


def test_library_exports_every_header_function():
    names = header_functions()
    assert len(names) >= 10
    L = B.lib()
    for n in names:
        assert hasattr(L, n), f"libidb.so does not export {n}"
    assert set(names) == set(B.EXPORTED)


def router(T=128, d=256, E=768, K=10, dtype=B.IDB_DTYPE_BF16, x=A16, W=A16, bias=A16, idx=A16, w=A16, counts=A16,
           dump=None, ws=A16, ws_bytes=1 << 30, variant=0, fn="idb_router_forward", layout=0):
    extra = (None, None) if fn.endswith("_timed") else ()  # the timed call's two events
    return getattr(B.lib(), fn)(x, W, dtype, layout, bias, T, d, E, K, idx, w, counts, 0, dump, ws, ws_bytes, variant,
                                None, *extra)


@pytest.mark.parametrize("fn", ["idb_router_forward", "idb_router_score_select", "idb_router_score_select_timed"])
@pytest.mark.parametrize("kw,code", [
    (dict(T=0), B.IDB_ERR_INVALID_ARG),
    (dict(T=(1 << 26) + 1), B.IDB_ERR_INVALID_ARG),
    (dict(K=0), B.IDB_ERR_INVALID_ARG),
    (dict(K=769), B.IDB_ERR_INVALID_ARG),
    (dict(E=0), B.IDB_ERR_INVALID_ARG),
    (dict(d=0), B.IDB_ERR_INVALID_ARG),
    (dict(dtype=7), B.IDB_ERR_INVALID_ARG),
    (dict(x=None), B.IDB_ERR_INVALID_ARG),
    (dict(W=None), B.IDB_ERR_INVALID_ARG),
    (dict(bias=None), B.IDB_ERR_INVALID_ARG),
    (dict(idx=None), B.IDB_ERR_INVALID_ARG),
    (dict(counts=None), B.IDB_ERR_INVALID_ARG),
    (dict(x=A16 + 4), B.IDB_ERR_INVALID_ARG),
    (dict(W=A16 + 8), B.IDB_ERR_INVALID_ARG),
    (dict(bias=A16 + 2), B.IDB_ERR_INVALID_ARG),
    (dict(dump=A16 + 4), B.IDB_ERR_INVALID_ARG),
    (dict(ws=None, variant=1), B.IDB_ERR_INVALID_ARG),  # two slices: the workspace is required
    (dict(ws_bytes=16, variant=1), B.IDB_ERR_INVALID_ARG),
    (dict(variant=99), B.IDB_ERR_INVALID_ARG),
    (dict(layout=2), B.IDB_ERR_INVALID_ARG),
    (dict(variant=5), B.IDB_ERR_UNSUPPORTED),   # the fp32 tiling asked for bf16 input
    (dict(E=2048), B.IDB_ERR_UNSUPPORTED),
    (dict(E=100, K=4), B.IDB_ERR_UNSUPPORTED),
    (dict(K=33), B.IDB_ERR_UNSUPPORTED),
    (dict(d=96), B.IDB_ERR_UNSUPPORTED),
    (dict(d=48, dtype=B.IDB_DTYPE_F32, variant=5), B.IDB_ERR_UNSUPPORTED),
])
def test_router_rejects_invalid_arguments(fn, kw, code):
    assert router(fn=fn, **kw) == code
    assert B.idb_last_error() != ""


def test_pack_weight_rejects_invalid_arguments():
    L = B.lib()
    assert L.idb_router_pack_weight(None, 0, 768, 2048, A16, None) == B.IDB_ERR_INVALID_ARG
    assert L.idb_router_pack_weight(A16, 0, 768, 2048, None, None) == B.IDB_ERR_INVALID_ARG
    assert L.idb_router_pack_weight(A16, 0, 768, 2048, A16 + 4096, None) == B.IDB_ERR_INVALID_ARG  # overlap
    assert L.idb_router_pack_weight(A16 + 8, 0, 768, 2048, A16 + (1 << 26), None) == B.IDB_ERR_INVALID_ARG
    assert L.idb_router_pack_weight(A16, 0, 100, 2048, A16 + (1 << 26), None) == B.IDB_ERR_UNSUPPORTED
    assert L.idb_router_pack_weight(A16, 0, 768, 96, A16 + (1 << 26), None) == B.IDB_ERR_UNSUPPORTED
    assert B.idb_router_packed_weight_bytes(768, 2048, B.IDB_DTYPE_BF16) == 768 * 2048 * 2
    assert B.idb_router_packed_weight_bytes(64, 256, B.IDB_DTYPE_F32) == 64 * 256 * 4
    assert B.idb_router_packed_weight_bytes(100, 256, B.IDB_DTYPE_F32) == 0


def test_merge_rejects_invalid_arguments():
    L = B.lib()
    assert L.idb_router_merge(0, 256, 768, 10, 0, A16, A16, A16, A16, 1 << 30, 0, None) == B.IDB_ERR_INVALID_ARG
    assert L.idb_router_merge(128, 256, 768, 10, 0, None, A16, A16, A16, 1 << 30, 0, None) == B.IDB_ERR_INVALID_ARG
    assert L.idb_router_merge(128, 256, 768, 10, 0, A16, A16, A16, A16, 8, 1, None) == B.IDB_ERR_INVALID_ARG  # two slices


def test_workspace_and_variant_info():
    # 768 experts in bf16: the automatic tiling is the 16x16-tile kernel, two
    # 384-expert slices of 8 waves x 48 experts, 128 tokens per workgroup; the
    # slices' candidates are staged in the workspace.
    info = B.idb_router_variant_info(16384, 2048, 768, 10, B.IDB_DTYPE_BF16, 0)
    assert info == {"tokens_per_wg": 128, "slices": 2, "waves": 8, "experts_per_wave": 48, "variant": 6}
    # candidates (value, score, index) per token, slice and rank, then 256
    # bytes for the merge's ticket
    assert B.idb_router_workspace_bytes(16384, 2048, 768, 10, B.IDB_DTYPE_BF16, 0) == 3 * 16384 * 2 * 10 * 4 + 256
    # a single 768-expert slice needs no workspace
    info2 = B.idb_router_variant_info(16384, 2048, 768, 10, B.IDB_DTYPE_BF16, 2)
    assert info2["slices"] == 1 and info2["tokens_per_wg"] == 64 and info2["experts_per_wave"] == 96
    assert B.idb_router_workspace_bytes(16384, 2048, 768, 10, B.IDB_DTYPE_BF16, 2) == 0
    # fp32 input, 64 experts: one 128-expert slice, half padding
    info3 = B.idb_router_variant_info(4096, 256, 64, 4, B.IDB_DTYPE_F32, 0)
    assert info3["slices"] == 1 and info3["variant"] == 5
    assert B.idb_router_workspace_bytes(0, 256, 64, 4, B.IDB_DTYPE_F32, 0) == 0
    with pytest.raises(B.IdbError):
        B.idb_router_variant_info(128, 256, 768, 10, B.IDB_DTYPE_BF16, 5)


@pytest.mark.parametrize("args,code", [
    (dict(T=0), B.IDB_ERR_INVALID_ARG),
    (dict(K=0), B.IDB_ERR_INVALID_ARG),
    (dict(K=65, E=64), B.IDB_ERR_INVALID_ARG),
    (dict(E=1025, K=4), B.IDB_ERR_UNSUPPORTED),
    (dict(K=33, E=64), B.IDB_ERR_UNSUPPORTED),
    (dict(scores=None), B.IDB_ERR_INVALID_ARG),
    (dict(scores=A16 + 2), B.IDB_ERR_INVALID_ARG),
    (dict(counts=None), B.IDB_ERR_INVALID_ARG),
])
def test_select_rejects_invalid_arguments(args, code):
    a = dict(scores=A16, bias=A16, T=64, E=64, K=4, idx=A16, w=A16, counts=A16)
    a.update(args)
    st = B.lib().idb_select_from_scores(a["scores"], a["bias"], a["T"], a["E"], a["K"], a["idx"], a["w"],
                                        a["counts"], 0, None)
    assert st == code


def _state(**kw):
    s = dict(bias=A16, e_prev=A16, step=A16, status=A16)
    s.update(kw)
    return B.idb_controller_state(s["bias"], s["e_prev"], s["step"], s["status"])


@pytest.mark.parametrize("cfg,state,code", [
    (dict(E=0), {}, B.IDB_ERR_INVALID_ARG),
    (dict(E=1025), {}, B.IDB_ERR_INVALID_ARG),
    (dict(Ki=-1.0), {}, B.IDB_ERR_INVALID_ARG),
    (dict(Kd=float("nan")), {}, B.IDB_ERR_INVALID_ARG),
    (dict(Ki=float("inf")), {}, B.IDB_ERR_INVALID_ARG),
    (dict(integral_mode=2), {}, B.IDB_ERR_INVALID_ARG),
    (dict(center=2), {}, B.IDB_ERR_INVALID_ARG),
    (dict(), dict(bias=None), B.IDB_ERR_INVALID_ARG),
    (dict(), dict(step=A16 + 4), B.IDB_ERR_INVALID_ARG),
    (dict(), dict(e_prev=A16 + 2), B.IDB_ERR_INVALID_ARG),
])
def test_controller_rejects_invalid_arguments(cfg, state, code):
    c = dict(E=768, Ki=6e-3, Kd=6e-3, integral_mode=0, center=1)
    c.update(cfg)
    ccfg = B.idb_controller_cfg(c["E"], c["Ki"], c["Kd"], c["integral_mode"], c["center"])
    st = B.lib().idb_controller_update(A16, ctypes.byref(ccfg), ctypes.byref(_state(**state)), None)
    assert st == code


@pytest.mark.parametrize("kw,code", [
    (dict(cfg=None), B.IDB_ERR_INVALID_ARG),
    (dict(state=None), B.IDB_ERR_INVALID_ARG),
    (dict(E=0), B.IDB_ERR_INVALID_ARG),
    (dict(Ki=-1.0), B.IDB_ERR_INVALID_ARG),
    (dict(center=3), B.IDB_ERR_INVALID_ARG),
    (dict(bias=None), B.IDB_ERR_INVALID_ARG),
    (dict(bias=A16 + 2), B.IDB_ERR_INVALID_ARG),
    (dict(stats=A16 + 4), B.IDB_ERR_INVALID_ARG),
    (dict(T=0), B.IDB_ERR_INVALID_ARG),
    (dict(K=0), B.IDB_ERR_INVALID_ARG),
    (dict(x=None), B.IDB_ERR_INVALID_ARG),
    (dict(counts=None), B.IDB_ERR_INVALID_ARG),
    (dict(ws=None, variant=6), B.IDB_ERR_INVALID_ARG),
    (dict(ws_bytes=3 * 128 * 2 * 10 * 4, variant=6), B.IDB_ERR_INVALID_ARG),  # no room for the ticket
    (dict(E=100), B.IDB_ERR_UNSUPPORTED),
    (dict(K=33), B.IDB_ERR_UNSUPPORTED),
])
def test_router_step_rejects_invalid_arguments(kw, code):
    a = dict(x=A16, W=A16, T=128, d=256, K=10, E=768, Ki=6e-3, Kd=6e-3, center=1, bias=A16, stats=None,
             counts=A16, ws=A16, ws_bytes=1 << 30, variant=0, cfg=True, state=True)
    a.update(kw)
    ccfg = B.idb_controller_cfg(a["E"], a["Ki"], a["Kd"], 0, a["center"])
    cfg = ctypes.byref(ccfg) if a["cfg"] else None
    sts = _state(bias=a["bias"])
    state = ctypes.byref(sts) if a["state"] else None
    st = B.lib().idb_router_step(a["x"], a["W"], B.IDB_DTYPE_BF16, 0, a["T"], a["d"], a["K"], cfg, state, A16, A16,
                                 a["counts"], 0, a["stats"], a["ws"], a["ws_bytes"], a["variant"], None)
    assert st == code
    assert B.idb_last_error() != ""


def test_controller_and_stats_null_pointers():
    L = B.lib()
    ccfg = B.idb_controller_cfg(8, 0.1, 0.1, 0, 1)
    assert L.idb_controller_update(None, ctypes.byref(ccfg), ctypes.byref(_state()), None) == B.IDB_ERR_INVALID_ARG
    assert L.idb_controller_update(A16, None, ctypes.byref(_state()), None) == B.IDB_ERR_INVALID_ARG
    assert L.idb_load_stats(None, 8, A16, None) == B.IDB_ERR_INVALID_ARG
    assert L.idb_load_stats(A16, 0, A16, None) == B.IDB_ERR_INVALID_ARG
    assert L.idb_load_stats(A16, 8, A16 + 4, None) == B.IDB_ERR_INVALID_ARG


def test_status_strings():
    for s in range(5):
        assert B.idb_status_string(s) != "unknown status"
    assert B.idb_status_string(42) == "unknown status"


def test_binding_rejects_short_score_dump():
    # host-side check before any pointer is taken: the dump must hold T*E floats
    import torch
    T, d, E, K = 64, 256, 64, 4
    x = torch.zeros((T, d), dtype=torch.bfloat16)
    W = torch.zeros((E, d), dtype=torch.bfloat16)
    b = torch.zeros(E, dtype=torch.float32)
    idx = torch.zeros((T, K), dtype=torch.int32)
    w = torch.zeros((T, K), dtype=torch.float32)
    c = torch.zeros(E, dtype=torch.int32)
    with pytest.raises(ValueError, match="scores_dump"):
        B.idb_router_forward(x, W, b, K, idx, w, c, scores_dump=torch.zeros(T * E // 2, dtype=torch.float32))


@pytest.mark.parametrize("kw,code", [
    (dict(K=0), B.IDB_ERR_INVALID_ARG),
    (dict(E=32, K=32), B.IDB_ERR_INVALID_ARG),     # K + 1 > E
    (dict(K=32), B.IDB_ERR_UNSUPPORTED),           # K + 1 candidates above 32
    (dict(st=None), B.IDB_ERR_INVALID_ARG),
    (dict(alpha=None), B.IDB_ERR_INVALID_ARG),
    (dict(alpha=A16 + 2), B.IDB_ERR_INVALID_ARG),
    (dict(ws_bytes=3 * 128 * 2 * 10 * 4 + 256, variant=6), B.IDB_ERR_INVALID_ARG),  # sized for K, not K + 1
    (dict(x=None), B.IDB_ERR_INVALID_ARG),
    (dict(E=100), B.IDB_ERR_UNSUPPORTED),
])
def test_qb_router_rejects_invalid_arguments(kw, code):
    a = dict(x=A16, W=A16, T=128, d=256, E=768, K=10, st=A16, alpha=A16, ws=A16, ws_bytes=1 << 30, variant=0)
    a.update(kw)
    st = B.lib().idb_qb_router_forward(a["x"], a["W"], B.IDB_DTYPE_BF16, 0, A16, a["T"], a["d"], a["E"], a["K"],
                                       A16, A16, A16, 0, a["st"], a["alpha"], a["ws"], a["ws_bytes"], a["variant"],
                                       None)
    assert st == code
    assert B.idb_last_error() != ""


@pytest.mark.parametrize("kw,code", [
    (dict(st=None), B.IDB_ERR_INVALID_ARG),
    (dict(bias=None), B.IDB_ERR_INVALID_ARG),
    (dict(T=0), B.IDB_ERR_INVALID_ARG),
    (dict(E=1, K=0), B.IDB_ERR_INVALID_ARG),
    (dict(K=0), B.IDB_ERR_INVALID_ARG),
    (dict(K=768), B.IDB_ERR_INVALID_ARG),
    (dict(E=1025), B.IDB_ERR_INVALID_ARG),
    (dict(rho=1.0), B.IDB_ERR_INVALID_ARG),
    (dict(rho=-0.25), B.IDB_ERR_INVALID_ARG),
    (dict(rho=float("nan")), B.IDB_ERR_INVALID_ARG),
    (dict(alpha=A16 + 1), B.IDB_ERR_INVALID_ARG),
    (dict(counts=A16), B.IDB_ERR_INVALID_ARG),             # statistics output missing
    (dict(stats=A16), B.IDB_ERR_INVALID_ARG),              # counts missing
    (dict(counts=A16, stats=A16 + 4), B.IDB_ERR_INVALID_ARG),  # fp64 output not 8-byte aligned
    (dict(counts=A16 + 2, stats=A16), B.IDB_ERR_INVALID_ARG),  # misaligned counts
])
def test_qb_update_rejects_invalid_arguments(kw, code):
    a = dict(st=A16, alpha=A16, T=16384, E=768, K=10, rho=0.0, bias=A16)
    a.update(kw)
    assert B.lib().idb_qb_update(a["st"], a["alpha"], a["T"], a["E"], a["K"], a["rho"], a["bias"], a.get("counts"),
                                 a.get("stats"), None) == code


def test_qb_workspace_holds_k_plus_one_candidates():
    assert B.idb_qb_router_workspace_bytes(16384, 2048, 768, 10, B.IDB_DTYPE_BF16, 0) == \
        B.idb_router_workspace_bytes(16384, 2048, 768, 11, B.IDB_DTYPE_BF16, 0)
    assert B.idb_qb_router_workspace_bytes(16384, 2048, 768, 32, B.IDB_DTYPE_BF16, 0) == 0
    assert B.idb_qb_router_workspace_bytes(16384, 2048, 768, 10, B.IDB_DTYPE_BF16, 7) == 0  # one slice


def test_layers_and_entropy_reject_invalid_arguments():
    L = B.lib()
    ccfg = B.idb_controller_cfg(768, 6e-3, 6e-3, 0, 1)
    st = _state()
    assert L.idb_controller_update_layers(None, 4, ctypes.byref(ccfg), ctypes.byref(st), None, None, None) == \
        B.IDB_ERR_INVALID_ARG
    assert L.idb_controller_update_layers(A16, 0, ctypes.byref(ccfg), ctypes.byref(st), None, None, None) == \
        B.IDB_ERR_INVALID_ARG
    bad = B.idb_controller_cfg(768, -1.0, 6e-3, 0, 1)
    assert L.idb_controller_update_layers(A16, 4, ctypes.byref(bad), ctypes.byref(st), None, None, None) == \
        B.IDB_ERR_INVALID_ARG
    assert L.idb_controller_update_layers(A16, 4, ctypes.byref(ccfg), ctypes.byref(st), None, A16 + 4, None) == \
        B.IDB_ERR_INVALID_ARG
    ws = int(L.idb_routing_entropy_workspace_bytes())
    assert ws == 512 * 2 * 8
    assert L.idb_routing_entropy(A16, 0, 10, None, None, 0, A16, ws, A16, None) == B.IDB_ERR_INVALID_ARG
    assert L.idb_routing_entropy(A16, 100, 0, None, None, 0, A16, ws, A16, None) == B.IDB_ERR_INVALID_ARG
    assert L.idb_routing_entropy(A16, 100, 10, None, None, 0, A16, ws - 8, A16, None) == B.IDB_ERR_INVALID_ARG
    assert L.idb_routing_entropy(A16, 100, 10, A16, None, 768, A16, ws, A16, None) == B.IDB_ERR_INVALID_ARG
    assert L.idb_routing_entropy(None, 100, 10, None, None, 0, A16, ws, A16, None) == B.IDB_ERR_INVALID_ARG


@pytest.mark.parametrize("kw,code", [
    (dict(f=None), B.IDB_ERR_INVALID_ARG),
    (dict(P=None), B.IDB_ERR_INVALID_ARG),
    (dict(loss=None), B.IDB_ERR_INVALID_ARG),
    (dict(loss=A16 + 4), B.IDB_ERR_INVALID_ARG),          # fp64 output misaligned
    (dict(stats=A16 + 4), B.IDB_ERR_INVALID_ARG),
    (dict(variant=1), B.IDB_ERR_UNSUPPORTED),             # one slice at E <= 384, but no softmax mode
    (dict(alpha=float("inf")), B.IDB_ERR_INVALID_ARG),
    (dict(E=1024), B.IDB_ERR_UNSUPPORTED),                # no tiling covers 1024 experts in one slice
    (dict(variant=6), B.IDB_ERR_UNSUPPORTED),             # two 384-expert slices
    (dict(variant=5), B.IDB_ERR_UNSUPPORTED),             # fp32 tiling for bf16 inputs
    (dict(dtype=B.IDB_DTYPE_F32, E=256), B.IDB_ERR_UNSUPPORTED),  # fp32 tiling covers 128 experts
    (dict(ws_bytes=1024), B.IDB_ERR_INVALID_ARG),
    (dict(ws=None), B.IDB_ERR_INVALID_ARG),
    (dict(x=None), B.IDB_ERR_INVALID_ARG),
    (dict(K=0), B.IDB_ERR_INVALID_ARG),
    (dict(K=33), B.IDB_ERR_UNSUPPORTED),
])
def test_aux_router_rejects_invalid_arguments(kw, code):
    a = dict(x=A16, W=A16, dtype=B.IDB_DTYPE_BF16, T=128, d=256, E=768, K=10, alpha=0.05, f=A16, P=A16, loss=A16,
             stats=None, ws=A16, ws_bytes=1 << 30, variant=0)
    a.update(kw)
    st = B.lib().idb_aux_router_forward(a["x"], a["W"], a["dtype"], 0, a["T"], a["d"], a["E"], a["K"], a["alpha"],
                                        A16, A16, A16, a["f"], a["P"], a["loss"], a["stats"], None, a["ws"],
                                        a["ws_bytes"], a["variant"], None)
    assert st == code
    assert B.idb_last_error() != ""


def test_aux_workspace_and_tiling():
    # one-slice tilings only: 64 tokens x 768 experts per workgroup at the headline shape
    T, E = 16384, 768
    n = B.idb_aux_router_workspace_bytes(T, 2048, E, 10, B.IDB_DTYPE_BF16, 0)
    assert n >= 2 * (T // 64) * E * 4 + 16 * 24 + 4
    assert B.idb_aux_router_workspace_bytes(T, 2048, E, 10, B.IDB_DTYPE_BF16, 6) == 0
    assert B.idb_aux_router_workspace_bytes(T, 2048, 1024, 10, B.IDB_DTYPE_BF16, 0) == 0
    assert B.idb_aux_router_workspace_bytes(4096, 256, 64, 4, B.IDB_DTYPE_F32, 0) >= 32 * 64 * 4


def test_controller_state_dict_round_trip():
    # host-side checkpoint helpers (no kernel runs): exact bits, shape checks
    import torch
    a = B.ControllerState(768, "cpu", layers=3)
    a.bias.copy_(torch.linspace(-1, 1, 3 * 768).view(3, 768))
    a.bias[0, 5] = -0.0
    a.e_prev.fill_(0.25)
    a.step.fill_(7)
    a.status.fill_(3)
    d = a.state_dict()
    b = B.ControllerState(768, "cpu", layers=3)
    ptr = b.bias.data_ptr()
    b.load_state_dict(d)
    assert b.bias.data_ptr() == ptr  # restored in place
    for k in ("bias", "e_prev", "step", "status"):
        x, y = getattr(a, k), getattr(b, k)
        assert torch.equal(x.view(torch.int32) if x.dtype == torch.float32 else x,
                           y.view(torch.int32) if y.dtype == torch.float32 else y)
    d["bias"] = d["bias"][:2]
    with pytest.raises(ValueError, match="bias"):
        b.load_state_dict(d)


def test_merge_step_rejects_invalid_arguments():
    L = B.lib()
    cfg = B.idb_controller_cfg(768, 6e-3, 6e-3, 0, 1)
    st = B.idb_controller_state(A16, A16, A16, A16)
    args = dict(T=128, d=256, K=10, dtype=0, idx=A16, w=A16, counts=A16, out=A16, ws=A16, ws_bytes=1 << 30, variant=0)

    def call(**kw):
        a = dict(args, **kw)
        return L.idb_router_merge_step(a["T"], a["d"], a["K"], a["dtype"], ctypes.byref(cfg), ctypes.byref(st),
                                       a["idx"], a["w"], a["counts"], a["out"], a["ws"], a["ws_bytes"], a["variant"],
                                       None)
    assert call(T=0) == B.IDB_ERR_INVALID_ARG
    assert call(idx=None) == B.IDB_ERR_INVALID_ARG
    assert call(ws=None) == B.IDB_ERR_INVALID_ARG  # two slices: the candidates are in the workspace
    assert call(ws_bytes=64) == B.IDB_ERR_INVALID_ARG
    assert call(K=33) == B.IDB_ERR_UNSUPPORTED
    assert call(out=A16 + 4) == B.IDB_ERR_INVALID_ARG
    bad = B.idb_controller_state(None, A16, A16, A16)
    assert L.idb_router_merge_step(128, 256, 10, 0, ctypes.byref(cfg), ctypes.byref(bad), A16, A16, A16, A16, A16,
                                   1 << 30, 0, None) == B.IDB_ERR_INVALID_ARG


def test_noalloc_step_rejects_before_any_hip_call():
    L = B.lib()
    cfg = B.idb_controller_cfg(768, 6e-3, 6e-3, 0, 1)
    st = B.idb_controller_state(A16, A16, A16, A16)

    def call(T=128, d=256, K=10, x=A16, variant=0, state=st):
        return L.idb_router_step_noalloc(x, A16, 0, 0, T, d, K, ctypes.byref(cfg), ctypes.byref(state), A16, A16,
                                         A16, 0, None, variant, None)
    # 2 slices x 10 candidates x 12 bytes per token: 2^17 tokens need 31 MB, beyond the fixed scratch
    assert call(T=1 << 17) == B.IDB_ERR_UNSUPPORTED
    assert "scratch" in B.idb_last_error()
    assert call(T=0) == B.IDB_ERR_INVALID_ARG
    assert call(x=None) == B.IDB_ERR_INVALID_ARG
    assert call(K=33) == B.IDB_ERR_UNSUPPORTED
    assert call(state=B.idb_controller_state(A16, None, A16, A16)) == B.IDB_ERR_INVALID_ARG


def test_softmax_entropy_rejects_invalid_arguments():
    L = B.lib()
    ws = B.idb_routing_entropy_workspace_bytes() if hasattr(B, "idb_routing_entropy_workspace_bytes") else 1 << 20
    call = L.idb_routing_entropy_softmax
    assert call(A16, 128, 10, None, 768, A16, 1 << 20, A16, None) == B.IDB_ERR_INVALID_ARG   # no logits
    assert call(A16, 0, 10, A16, 768, A16, 1 << 20, A16, None) == B.IDB_ERR_INVALID_ARG     # T = 0
    assert call(A16, 128, 33, A16, 768, A16, 1 << 20, A16, None) == B.IDB_ERR_INVALID_ARG   # K > 32
    assert call(A16, 128, 10, A16, 2048, A16, 1 << 20, A16, None) == B.IDB_ERR_INVALID_ARG  # E > 1024
    assert call(A16, 128, 10, A16, 768, A16, 8, A16, None) == B.IDB_ERR_INVALID_ARG         # workspace too small
    assert call(A16, 128, 10, A16 + 2, 768, A16, 1 << 20, A16, None) == B.IDB_ERR_INVALID_ARG  # misaligned
    assert ws > 0

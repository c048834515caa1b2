"""Closed loops of Alg. 1 on the GPU.

* Given identical scores: each step draws fresh synthetic scores (the same
  arrays for both sides), routes them with the current bias, updates the bias
  from the counts and computes MaxVio/MinVio -- on the GPU through the C ABI and
  on the CPU oracle, independently.  Every step's selection, counts, bias,
  e_prev and statistics must be bit-identical: the whole bias trajectory is
  pinned.
* From hidden states (the tiny fp32 workload): the GPU loop runs its own
  router; each step its fused selection must equal the select kernel on its
  dumped scores, the scores must match the oracle's within rel 2e-3, and the
  free-running oracle loop must stay close (near-tie flips are reported).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_39137_amd import binding as B
from paper_2609_39137_amd import synth
from paper_2609_39137_amd.pipeline import RouterStep

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("T,E,K,steps,Ki,Kd,mode,center", [
    (2048, 768, 10, 30, 6e-3, 6e-3, 0, True),
    (4096, 768, 5, 40, 6e-3, 6e-3, 0, True),
    (4096, 768, 3, 40, 6e-3, 0.0, 0, True),
    (1024, 64, 4, 30, 1e-3, 0.0, 1, False),
    (1000, 100, 7, 25, 0.05, 0.1, 0, True),
])
def test_closed_loop_given_scores_is_bit_exact(T, E, K, steps, Ki, Kd, mode, center):
    cfg = B.ControllerCfg(E, Ki, Kd, mode, center)
    st = B.ControllerState(E, DEV)
    ref = oracle.ControllerState(E)
    idx = torch.empty((T, K), dtype=torch.int32, device=DEV)
    w = torch.empty((T, K), dtype=torch.float32, device=DEV)
    counts = torch.empty(E, dtype=torch.int32, device=DEV)
    stats = torch.empty(2, dtype=torch.float64, device=DEV)
    for t in range(steps):
        s = synth.scores(T, E, "beta", seed=1000 + t)
        # skew the load so the controller has work: a fixed per-expert tilt
        s = np.clip(s + (np.arange(E, dtype=np.float32) / E * 0.2)[None, :], 0, 1).astype(np.float32)
        B.idb_select_from_scores(torch.from_numpy(s).to(DEV), st.bias, K, idx, w, counts)
        B.idb_controller_update(counts, cfg, st)
        B.idb_load_stats(counts, stats)
        r_idx, r_w, r_c = oracle.select(s, ref.bias, K)
        oracle.controller(r_c, ref, Ki, Kd, mode=mode, center=center)
        np.testing.assert_array_equal(idx.cpu().numpy(), r_idx, err_msg=f"step {t}")
        np.testing.assert_array_equal(w.cpu().numpy().view(np.uint32), r_w.view(np.uint32))
        np.testing.assert_array_equal(counts.cpu().numpy(), r_c)
        np.testing.assert_array_equal(st.bias.cpu().numpy(), ref.bias, err_msg=f"bias step {t}")
        np.testing.assert_array_equal(st.e_prev.cpu().numpy(), ref.e_prev)
        np.testing.assert_array_equal(stats.cpu().numpy(), oracle.load_stats(r_c))
    assert int(st.step.item()) == steps


def test_tiny_workload_router_loop():
    wl = synth.WORKLOADS["tiny-e64-k4"]
    W = synth.router_weight(wl)
    Wt = torch.from_numpy(W).to(DEV)
    rs = RouterStep(wl.T, wl.d, wl.E, wl.K, torch.float32)
    ref = oracle.ControllerState(wl.E)
    dump = torch.empty((wl.T, wl.E), dtype=torch.float32, device=DEV)
    idx2 = torch.empty_like(rs.idx)
    w2 = torch.empty_like(rs.w)
    c2 = torch.empty_like(rs.counts)
    flips = 0
    for t in range(wl.steps):
        x = synth.hidden_states(wl, step=t)
        bias_before = rs.state.bias.clone()
        rs.route(torch.from_numpy(x).to(DEV), Wt, scores_dump=dump)
        B.idb_select_from_scores(dump, bias_before, wl.K, idx2, w2, c2)
        assert torch.equal(rs.idx, idx2) and torch.equal(rs.w, w2) and torch.equal(rs.counts, c2)
        rs.update()
        rs.load_stats()
        s_ref = oracle.router_scores(x, W)
        s = dump.cpu().numpy()
        assert np.all(np.abs(s.astype(np.float64) - s_ref) <= 2e-3 * np.abs(s_ref.astype(np.float64)))
        r_idx, r_w, r_c = oracle.select(s_ref, ref.bias, wl.K)
        oracle.controller(r_c, ref, 6e-3, 6e-3)
        flips += int((np.sort(rs.idx.cpu().numpy(), 1) != np.sort(r_idx, 1)).any(1).sum())
        counts = rs.counts.cpu().numpy()
        assert int(counts.sum()) == wl.T * wl.K
        mx, mn = rs.stats.cpu().numpy()
        assert 0 <= mx <= wl.E / wl.K - 1 and 0 <= mn <= 1
    # free-running oracle vs GPU: only near-tie flips may differ
    assert flips <= 0.01 * wl.T * wl.steps
    np.testing.assert_allclose(rs.state.bias.cpu().numpy(), ref.bias, atol=5e-4)
    print(f"tiny loop: {flips} token selections differ from the free-running oracle over {wl.steps} steps")


def _bf16(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(a.view(np.int16)).to(DEV).view(torch.bfloat16)


def _assert_same_step(f: RouterStep, s: RouterStep, msg):
    """The one-call step (f) against route + controller step (s): everything
    bit-identical (the controller step itself is pinned against the oracle on
    host-generated counts in test_gpu_controller.py)."""
    assert torch.equal(f.idx, s.idx), msg
    assert torch.equal(f.w.view(torch.int32), s.w.view(torch.int32)), msg
    assert torch.equal(f.counts, s.counts), msg
    for name in ("bias", "e_prev", "step", "status"):
        a, b = getattr(f.state, name), getattr(s.state, name)
        assert torch.equal(a.view(torch.int32) if a.dtype == torch.float32 else a,
                           b.view(torch.int32) if b.dtype == torch.float32 else b), f"{msg}: {name}"
    assert torch.equal(f.stats.view(torch.int64), s.stats.view(torch.int64)), msg
    assert int(f.state.status.item()) == 0, msg


@pytest.mark.parametrize("T,d,E,K,variant,packed", [
    (2048, 256, 768, 10, 0, True),    # two slices: the update runs in the merge's last workgroup
    (1000, 256, 768, 10, 6, False),   # ragged last token tile
    (2048, 256, 768, 10, 7, True),    # one slice: the controller is its own launch
    (513, 256, 1024, 32, 0, False),   # 4 slices x 32 candidates: the generic merge kernel
    (777, 128, 512, 8, 1, False),     # 32x32 tiles, a padded second slice
    (300, 256, 768, 10, 0, True),     # three token tiles: a three-workgroup merge
])
def test_router_step_equals_route_then_controller(T, d, E, K, variant, packed):
    x0, W = synth.normal_router_inputs(T, d, E, seed=77)
    Wt = _bf16(W)
    cfg = B.ControllerCfg(E, 6e-3, 6e-3)
    f = RouterStep(T, d, E, K, torch.bfloat16, cfg=cfg, variant=variant)
    s = RouterStep(T, d, E, K, torch.bfloat16, cfg=cfg, variant=variant)
    if packed:
        f.pack(Wt)
        s.pack(Wt)
    for t in range(5):
        x = _bf16(synth.normal_router_inputs(T, d, E, seed=100 + t)[0])
        # a component shared by every token skews the load, so the
        # controller has work to do
        x[:, :16] += 1.5
        f.step(x, None if packed else Wt)
        s.route(x, None if packed else Wt)
        s.update_and_stats()
        _assert_same_step(f, s, f"step {t}")
    assert int(f.state.step.item()) == 5


def test_router_step_accumulates_microbatches():
    T, d, E, K = 1024, 256, 768, 10
    _, W = synth.normal_router_inputs(T, d, E, seed=5)
    Wt = _bf16(W)
    f = RouterStep(T, d, E, K, torch.bfloat16)
    s = RouterStep(T, d, E, K, torch.bfloat16)
    for t in range(3):
        xa = _bf16(synth.normal_router_inputs(T, d, E, seed=200 + 2 * t)[0])
        xb = _bf16(synth.normal_router_inputs(T, d, E, seed=201 + 2 * t)[0])
        f.route(xa, Wt)
        f.step(xb, Wt, accumulate=True)
        s.route(xa, Wt)
        s.route(xb, Wt, accumulate=True)
        s.update_and_stats()
        assert int(f.counts.sum().item()) == 2 * T * K
        _assert_same_step(f, s, f"step {t}")


def test_router_step_graph_replays():
    """Captured in a graph and replayed: every replay equals the eager calls."""
    T, d, E, K = 2048, 256, 768, 10
    _, W = synth.normal_router_inputs(T, d, E, seed=9)
    Wt = _bf16(W)
    xs = [_bf16(synth.normal_router_inputs(T, d, E, seed=300 + t)[0]) for t in range(4)]
    x = torch.empty_like(xs[0])
    f = RouterStep(T, d, E, K, torch.bfloat16)
    s = RouterStep(T, d, E, K, torch.bfloat16)
    f.pack(Wt)
    s.pack(Wt)
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        f.step(x, None)
    for t, xt in enumerate(xs):
        x.copy_(xt)
        g.replay()
        s.route(xt, None)
        s.update_and_stats()
        torch.cuda.synchronize()
        _assert_same_step(f, s, f"replay {t}")


@pytest.mark.parametrize("T,d,E,K,variant", [(2048, 256, 768, 10, 6), (513, 256, 1024, 32, 0), (1000, 256, 768, 10, 7)])
def test_score_select_then_merge_step_equals_router_step(T, d, E, K, variant):
    """idb_router_score_select + idb_router_merge_step (the benchmark times the
    router kernel between them) give exactly idb_router_step's results."""
    _, W = synth.normal_router_inputs(T, d, E, seed=19)
    Wt = _bf16(W)
    cfg = B.ControllerCfg(E, 6e-3, 6e-3)
    f = RouterStep(T, d, E, K, torch.bfloat16, cfg=cfg, variant=variant)
    s = RouterStep(T, d, E, K, torch.bfloat16, cfg=cfg, variant=variant)
    for t in range(4):
        x = _bf16(synth.normal_router_inputs(T, d, E, seed=400 + t)[0])
        x[:, :16] += 1.5
        f.step(x, Wt)
        s.score_select(x, Wt)
        s.merge_step()
        _assert_same_step(f, s, f"step {t}")


@pytest.mark.parametrize("variant", [6, 7])
def test_timed_score_select_equals_untimed(variant):
    """idb_router_score_select_timed (the benchmark's live kernel timing) gives
    the untimed call's results bit for bit, and its events bracket the fused
    kernel: a positive interval, shorter than the whole call sequence around it."""
    T, d, E, K = 4096, 1024, 768, 10
    _, W = synth.normal_router_inputs(T, d, E, seed=23)
    Wt = _bf16(W)
    cfg = B.ControllerCfg(E, 6e-3, 6e-3)
    f = RouterStep(T, d, E, K, torch.bfloat16, cfg=cfg, variant=variant)
    s = RouterStep(T, d, E, K, torch.bfloat16, cfg=cfg, variant=variant)
    ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    outer = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    for e in ev:
        e.record()
    for t in range(3):
        x = _bf16(synth.normal_router_inputs(T, d, E, seed=500 + t)[0])
        x[:, :16] += 1.5
        f.score_select(x, Wt)
        f.merge_step()
        outer[0].record()
        s.score_select(x, Wt, events=ev)
        outer[1].record()
        s.merge_step()
        torch.cuda.synchronize()
        print(f"[timed] variant {variant} step {t}: kernel {ev[0].elapsed_time(ev[1]) * 1000:.1f} us, "
              f"call {outer[0].elapsed_time(outer[1]) * 1000:.1f} us", flush=True)
        _assert_same_step(f, s, f"step {t}")
        kernel_ms = ev[0].elapsed_time(ev[1])
        assert 0.0 < kernel_ms <= outer[0].elapsed_time(outer[1])

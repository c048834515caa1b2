"""idb_router_step_noalloc (the router step with the library's fixed device
scratch as its workspace) gives exactly the outputs of idb_router_step with a
caller workspace: two calls in a row on the same scratch, the second with a
smaller batch, on the two-slice tiling (scratch used by the slice merge and
its controller tail), the generic merge and the one-slice tiling (no
scratch).  Both sides start from the same controller state and run the same
inputs, so every output must be bit-identical."""
import numpy as np
import pytest
import torch

from paper_2609_39137_amd import binding as B
from paper_2609_39137_amd import synth
from paper_2609_39137_amd.pipeline import RouterStep

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _bf16(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(a.view(np.int16)).to(DEV).view(torch.bfloat16)


def _bits(t: torch.Tensor) -> np.ndarray:
    a = t.cpu().numpy()
    return a.view(np.uint32) if a.dtype == np.float32 else (a.view(np.uint64) if a.dtype == np.float64 else a)


@pytest.mark.parametrize("E,K,variant", [(768, 10, 6), (1024, 32, 6), (768, 10, 7)])
def test_noalloc_step_equals_workspace_step(E, K, variant):
    d = 256
    cfg = B.ControllerCfg(E, 6e-3, 6e-3)
    _, W = synth.normal_router_inputs(8, d, E, seed=41)
    Wt = _bf16(W)
    ref_state = B.ControllerState(E, DEV)
    new_state = B.ControllerState(E, DEV)
    for call, T in enumerate((4096, 1000)):  # the second call is smaller
        x = _bf16(synth.normal_router_inputs(T, d, E, seed=50 + call)[0])
        x[:, :16] += 1.0  # skew the load so the update has work
        print(f"[noalloc] E={E} K={K} variant={variant} call {call} T={T}", flush=True)
        ref = RouterStep(T, d, E, K, torch.bfloat16, cfg=cfg, variant=variant)
        ref.state = ref_state
        ref.step(x, Wt)
        idx = torch.full((T, K), -1, dtype=torch.int32, device=DEV)
        w = torch.full((T, K), -1.0, dtype=torch.float32, device=DEV)
        counts = torch.full((E,), 77, dtype=torch.int32, device=DEV)
        stats = torch.full((2,), -1.0, dtype=torch.float64, device=DEV)
        B.idb_router_step_noalloc(x, Wt, K, cfg, new_state, idx, w, counts, out=stats, variant=variant)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(_bits(idx), _bits(ref.idx))
        np.testing.assert_array_equal(_bits(w), _bits(ref.w))
        np.testing.assert_array_equal(_bits(counts), _bits(ref.counts))
        np.testing.assert_array_equal(_bits(stats), _bits(ref.stats))
        for name in ("bias", "e_prev", "step", "status"):
            np.testing.assert_array_equal(_bits(getattr(new_state, name)), _bits(getattr(ref_state, name)),
                                          err_msg=name)
        assert int(new_state.step.item()) == call + 1 and int(new_state.status.item()) == 0


def test_noalloc_rejects_shapes_beyond_the_scratch():
    E, K, d = 768, 10, 256
    cfg = B.ControllerCfg(E)
    st = B.ControllerState(E, DEV)
    T = 1 << 17  # 2 slices x 10 candidates x 12 bytes per token: 31 MB > 16 MB
    x = torch.empty((T, d), dtype=torch.bfloat16, device=DEV)
    W = torch.empty((E, d), dtype=torch.bfloat16, device=DEV)
    idx = torch.empty((T, K), dtype=torch.int32, device=DEV)
    w = torch.empty((T, K), dtype=torch.float32, device=DEV)
    counts = torch.full((E,), 5, dtype=torch.int32, device=DEV)
    with pytest.raises(B.IdbError) as ei:
        B.idb_router_step_noalloc(x, W, K, cfg, st, idx, w, counts)
    assert ei.value.status == B.IDB_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert torch.all(counts == 5)  # nothing was enqueued


def test_noalloc_step_captured_in_a_graph_replays_like_eager():
    """The callers this entry point serves capture it: a graph of one step
    replayed four times (fresh inputs copied in between, eager work and
    synchronisation between the replays) equals the eager workspace calls."""
    T, d, E, K = 2048, 256, 768, 10
    cfg = B.ControllerCfg(E, 6e-3, 6e-3)
    _, W = synth.normal_router_inputs(8, d, E, seed=43)
    Wt = _bf16(W)
    xs = [_bf16(synth.normal_router_inputs(T, d, E, seed=60 + t)[0]) for t in range(4)]
    x = torch.empty_like(xs[0])
    st = B.ControllerState(E, DEV)
    idx = torch.empty((T, K), dtype=torch.int32, device=DEV)
    w = torch.empty((T, K), dtype=torch.float32, device=DEV)
    counts = torch.empty(E, dtype=torch.int32, device=DEV)
    stats = torch.empty(2, dtype=torch.float64, device=DEV)
    ref = RouterStep(T, d, E, K, torch.bfloat16, cfg=cfg)
    side = torch.cuda.Stream()
    x.copy_(xs[0])
    # one eager call (on a throwaway state) before capture: the scratch
    # address is looked up on a device's first call
    B.idb_router_step_noalloc(x, Wt, K, cfg, B.ControllerState(E, DEV), idx, w, counts, out=stats)
    torch.cuda.synchronize()
    print(f"[noalloc] graph capture T={T} E={E} K={K}", flush=True)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        B.idb_router_step_noalloc(x, Wt, K, cfg, st, idx, w, counts, out=stats)
    for t, xt in enumerate(xs):
        x.copy_(xt)
        g.replay()
        ref.step(xt, Wt)
        torch.cuda.synchronize()
        for a, b in ((idx, ref.idx), (w, ref.w), (counts, ref.counts), (stats, ref.stats), (st.bias, ref.state.bias),
                     (st.e_prev, ref.state.e_prev), (st.step, ref.state.step)):
            np.testing.assert_array_equal(_bits(a), _bits(b), err_msg=f"replay {t}")

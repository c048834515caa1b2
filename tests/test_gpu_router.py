"""GPU parity of the fused router step (gate contraction, sigmoid, biased
Top-K, gate weights, counts; Sec. 2.2, Eq. pid-routing, Eq. pid-error) against
the CPU oracle on the same seeded inputs.

* Scores: the kernel's debug dump of the scores it selected with is within
  rel 2e-3 of the oracle's fp64-accumulated sigmoid scores (bf16 inputs, fp32
  accumulate).
* Selection given identical scores: the fused kernel's outputs equal those of
  the select-from-scores kernel run on its dumped scores (that kernel is itself
  bit-exact against the oracle on arbitrary scores, see test_gpu_select.py).
* Against the oracle directly: tokens whose oracle K-th / (K+1)-th biased
  scores are separated by more than the measured score error must select the
  oracle's experts; the rest (near ties) must be a valid Top-K within that
  error.  With integer-valued inputs the logits are exact on both sides and
  the selection must match the oracle exactly.
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


def to_dev(a: np.ndarray) -> torch.Tensor:
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(a).to(DEV)


def run_router(x, W, b, K, variant=0, dump=True, counts=None, accumulate=False):
    T, d = x.shape
    E = W.shape[0]
    xt, Wt, bt = to_dev(x), to_dev(W), torch.from_numpy(b).to(DEV)
    code = B.IDB_DTYPE_BF16 if x.dtype == np.uint16 else B.IDB_DTYPE_F32
    idx = torch.full((T, K), -7, dtype=torch.int32, device=DEV)
    w = torch.full((T, K), -7.0, dtype=torch.float32, device=DEV)
    c = counts if counts is not None else torch.full((E,), 999, dtype=torch.int32, device=DEV)
    ws = torch.empty(max(B.idb_router_workspace_bytes(T, d, E, K, code, variant), 16), dtype=torch.uint8, device=DEV)
    s = torch.full((T, E), -1.0, dtype=torch.float32, device=DEV) if dump else None
    B.idb_router_forward(xt, Wt, bt, K, idx, w, c, accumulate, s, ws, variant)
    out = [idx.cpu().numpy(), w.cpu().numpy(), c.cpu().numpy()]
    return out + [s.cpu().numpy() if dump else None]


def gpu_select(s, b, K):
    T, E = s.shape
    idx = torch.empty((T, K), dtype=torch.int32, device=DEV)
    w = torch.empty((T, K), dtype=torch.float32, device=DEV)
    c = torch.empty(E, dtype=torch.int32, device=DEV)
    B.idb_select_from_scores(torch.from_numpy(s).to(DEV), torch.from_numpy(b).to(DEV), K, idx, w, c)
    return idx.cpu().numpy(), w.cpu().numpy(), c.cpu().numpy()


def check_scores(s_gpu, s_ref, rtol=2e-3):
    err = np.abs(s_gpu.astype(np.float64) - s_ref.astype(np.float64))
    bound = rtol * np.abs(s_ref.astype(np.float64))
    assert np.all(err <= bound), f"max rel err {np.max(err / np.maximum(bound / rtol, 1e-30)):.3e}"
    return float(err.max())


def check_against_oracle(x, W, b, K, idx, w, c, s_gpu, rows=None, max_uncertain=0.01):
    """Margin-aware comparison of the GPU selection with the oracle's own."""
    s_ref = oracle.router_scores(x, W, rows=rows)
    g_idx, g_w = (idx, w) if rows is None else (idx[rows], w[rows])
    if s_gpu is not None:
        sg = s_gpu if rows is None else s_gpu[rows]
        eps = check_scores(sg, s_ref)
    else:
        eps = 1e-6
    tol = 2.0 * eps + 1e-7
    r_idx, r_w, _ = oracle.select(s_ref, b, K)
    v = (s_ref + b[None, :]).astype(np.float32).astype(np.float64)
    order = np.argsort(-v, axis=1, kind="stable")
    top = np.take_along_axis(v, order[:, :K + 1], 1)
    gaps = -np.diff(top, axis=1)  # adjacent gaps among the top K+1
    uncertain = 0
    for t in range(len(g_idx)):
        near_tie = K < v.shape[1] and gaps[t, K - 1] <= tol
        if near_tie:
            uncertain += 1
            vk = top[t, K - 1]
            assert np.all(v[t, g_idx[t]] >= vk - tol), f"token {t}: selection not a valid Top-K within {tol}"
            assert len(set(g_idx[t].tolist())) == K
            continue
        assert set(g_idx[t].tolist()) == set(r_idx[t].tolist()), f"token {t}"
        if np.all(gaps[t, :K - 1] > tol):
            assert g_idx[t].tolist() == r_idx[t].tolist(), f"token {t} rank order"
        perm = [g_idx[t].tolist().index(e) for e in r_idx[t]]
        np.testing.assert_allclose(g_w[t][perm], r_w[t], rtol=2e-5, atol=1e-7)
    assert uncertain <= max(1, max_uncertain * len(g_idx)), f"{uncertain} near-tie tokens"
    return uncertain


def check_invariants(idx, w, c, T, E, K):
    assert idx.min() >= 0 and idx.max() < E
    assert all(len(set(r)) == K for r in idx[: min(T, 4096)].tolist())
    np.testing.assert_array_equal(c, np.bincount(idx.ravel(), minlength=E))
    assert int(c.sum()) == T * K
    assert np.all(np.abs(w.astype(np.float64).sum(1) - 1.0) <= K * 2.0 ** -23)


@pytest.mark.parametrize("T,d,E,K,dtype", [
    (300, 256, 768, 10, "bf16"),
    (130, 2048, 768, 5, "bf16"),
    (257, 512, 768, 3, "bf16"),
    (200, 256, 256, 8, "bf16"),
    (97, 256, 64, 4, "bf16"),
    (1000, 256, 64, 4, "f32"),
    (129, 128, 800, 10, "bf16"),
])
def test_router_matches_oracle(T, d, E, K, dtype):
    x, W = synth.normal_router_inputs(T, d, E, seed=T, dtype=dtype, w_std=0.05)
    b = synth.bias(E, "small", seed=T)
    idx, w, c, s = run_router(x, W, b, K)
    check_invariants(idx, w, c, T, E, K)
    check_against_oracle(x, W, b, K, idx, w, c, s)
    # selection given identical scores: the select kernel on the dumped scores
    si, sw, sc = gpu_select(s, b, K)
    np.testing.assert_array_equal(idx, si)
    np.testing.assert_array_equal(w.view(np.uint32), sw.view(np.uint32))
    np.testing.assert_array_equal(c, sc)


@pytest.mark.parametrize("E,K", [(768, 10), (768, 3), (64, 4), (256, 16)])
def test_integer_inputs_select_exactly_like_oracle(E, K):
    # x in {-2..2}, W in {-2..2}/64: logits exact in fp32 and fp64, so with a
    # zero bias both sides rank by the same exact z (ties -> lowest index).
    T, d = 400, 256
    x, W = synth.integer_router_inputs(T, d, E, seed=E + K, dtype="bf16", w_shift=6)
    b = np.zeros(E, np.float32)
    idx, w, c, s = run_router(x, W, b, K)
    r_idx, r_w, r_c = oracle.router(x, W, b, K)
    np.testing.assert_array_equal(idx, r_idx)
    np.testing.assert_array_equal(c, r_c)
    np.testing.assert_allclose(w, r_w, rtol=2e-5)
    s_ref = oracle.router_scores(x, W)
    check_scores(s, s_ref, rtol=1e-6)


def test_all_variants_identical():
    T, d, E, K = 517, 512, 768, 10
    x, W = synth.normal_router_inputs(T, d, E, seed=3, w_std=0.05)
    b = synth.bias(E, "small", seed=4)
    ref = run_router(x, W, b, K, variant=1)
    # the 32x32-tile variants accumulate in the same order: identical outputs
    for v in (2, 3, 4):
        got = run_router(x, W, b, K, variant=v)
        for a, g in zip(ref, got):
            np.testing.assert_array_equal(a, g)
    # the 16x16-tile variant sums the contraction in another order: scores
    # agree to fp32 rounding, and its selection is exact on its own scores
    got6 = run_router(x, W, b, K, variant=6)
    check_scores(got6[3], ref[3], rtol=1e-5)
    check_invariants(*got6[:3], T, E, K)
    si, sw, sc = gpu_select(got6[3], b, K)
    np.testing.assert_array_equal(got6[0], si)
    np.testing.assert_array_equal(got6[1].view(np.uint32), sw.view(np.uint32))
    np.testing.assert_array_equal(got6[2], sc)
    # the two 16x16-tile variants accumulate in the same order
    got7 = run_router(x, W, b, K, variant=7)
    for a, g in zip(got6, got7):
        np.testing.assert_array_equal(a, g)
    again = run_router(x, W, b, K, variant=0)
    for a, g in zip(got6, again):
        np.testing.assert_array_equal(a, g)
    nodump = run_router(x, W, b, K, variant=0, dump=False)
    for a, g in zip(got6[:3], nodump[:3]):
        np.testing.assert_array_equal(a, g)


def test_microbatch_and_shard_accumulation_equals_whole_batch():
    T, d, E, K = 1024, 256, 768, 10
    x, W = synth.normal_router_inputs(T, d, E, seed=5, w_std=0.05)
    b = synth.bias(E, "small", seed=6)
    whole = run_router(x, W, b, K, dump=False)
    counts = torch.zeros(E, dtype=torch.int32, device=DEV)
    for lo, hi in ((0, 100), (100, 613), (613, 1024)):
        part = run_router(np.ascontiguousarray(x[lo:hi]), W, b, K, dump=False, counts=counts, accumulate=True)
        np.testing.assert_array_equal(part[0], whole[0][lo:hi])
    np.testing.assert_array_equal(counts.cpu().numpy(), whole[2])


@pytest.mark.parametrize("T,E,K", [(1, 768, 10), (1, 32, 32), (63, 32, 32), (100, 64, 1), (4097, 768, 10)])
def test_edge_shapes(T, E, K):
    d = 128
    x, W = synth.normal_router_inputs(T, d, E, seed=T + E + K, w_std=0.05)
    b = synth.bias(E, "large", seed=1)
    idx, w, c, s = run_router(x, W, b, K)
    check_invariants(idx, w, c, T, E, K)
    si, sw, sc = gpu_select(s, b, K)
    np.testing.assert_array_equal(idx, si)
    np.testing.assert_array_equal(w.view(np.uint32), sw.view(np.uint32))
    if K == E:
        assert np.all(c == T)
    check_against_oracle(x, W, b, K, idx, w, c, s, max_uncertain=0.02)


@pytest.mark.parametrize("E,K,variant", [(1024, 32, 4), (1024, 17, 3), (800, 10, 4), (768, 16, 1), (768, 32, 1),
                                         (1024, 32, 6), (800, 10, 6), (768, 24, 6), (1024, 20, 7), (800, 10, 7)])
def test_many_slices_and_large_k(E, K, variant):
    # up to 8 expert slices merged, K above the threshold path's 16 (every
    # list takes the per-token fallback), and E not a multiple of the slice
    T, d = 300, 256
    x, W = synth.normal_router_inputs(T, d, E, seed=E + K, w_std=0.05)
    b = synth.bias(E, "small", seed=K)
    idx, w, c, s = run_router(x, W, b, K, variant=variant)
    check_invariants(idx, w, c, T, E, K)
    si, sw, sc = gpu_select(s, b, K)
    np.testing.assert_array_equal(idx, si)
    np.testing.assert_array_equal(w.view(np.uint32), sw.view(np.uint32))
    np.testing.assert_array_equal(c, sc)
    check_against_oracle(x, W, b, K, idx, w, c, s, max_uncertain=0.02)


def test_tied_scores_fall_back_exactly():
    # identical tokens and a zero router matrix: every score is 0.5, every
    # token picks experts 0..K-1 (all candidate lists overflow).
    T, d, E, K = 300, 128, 768, 10
    x = synth.to_bf16_bits(np.ones((T, d), np.float32))
    W = synth.to_bf16_bits(np.zeros((E, d), np.float32))
    idx, w, c, s = run_router(x, W, np.zeros(E, np.float32), K)
    assert np.all(idx == np.arange(K)[None, :])
    assert np.all(w == np.float32(0.5) / np.float32(5.0))
    b = synth.bias(E, "grid", seed=2)  # heavy bias ties
    idx, w, c, s = run_router(x, W, b, K)
    r_idx, r_w, r_c = oracle.router(x, W, b, K)
    np.testing.assert_array_equal(idx, r_idx)
    np.testing.assert_array_equal(w, r_w)
    np.testing.assert_array_equal(c, r_c)


def test_overflowing_and_listed_tokens_share_waves():
    # every third token has x = 0, so all of its scores tie at 0.5 and its
    # candidate list overflows, while its neighbours in the same wave take
    # the list path; integer inputs keep every logit exact on both sides.
    T, d, E, K = 400, 256, 768, 10
    x, W = synth.integer_router_inputs(T, d, E, seed=31, dtype="bf16", w_shift=6)
    x = x.copy()
    x[::3] = 0
    b = np.zeros(E, np.float32)
    idx, w, c, s = run_router(x, W, b, K)
    r_idx, r_w, r_c = oracle.router(x, W, b, K)
    np.testing.assert_array_equal(idx, r_idx)
    np.testing.assert_array_equal(c, r_c)
    np.testing.assert_allclose(w, r_w, rtol=2e-5)
    assert np.all(idx[::3] == np.arange(K)[None, :])


def test_bias_steers_selection_but_not_weights():
    T, d, E, K = 256, 256, 768, 10
    x, W = synth.normal_router_inputs(T, d, E, seed=8, w_std=0.05)
    b = np.zeros(E, np.float32)
    b[100:110] = 10.0  # dominant bias: experts 100..109 always win
    idx, w, c, s = run_router(x, W, b, K)
    assert np.all(np.sort(idx, axis=1) == np.arange(100, 110)[None, :])
    sel = np.take_along_axis(s, idx, 1).astype(np.float64)
    np.testing.assert_allclose(w, sel / sel.sum(1, keepdims=True), rtol=1e-6)


@pytest.mark.parametrize("name", ["top10-of-768", "top5-of-768-mixture", "top3-of-768-drift", "large-d4096-top10",
                                  "tiny-e64-k4"])
def test_workload_full_size_sampled_rows(name):
    wl = synth.WORKLOADS[name]
    x = synth.hidden_states(wl, step=0)
    W = synth.router_weight(wl)
    b = synth.bias(wl.E, "small", seed=wl.wid)
    rs = RouterStep(wl.T, wl.d, wl.E, wl.K, torch.bfloat16 if wl.dtype == "bf16" else torch.float32)
    rs.state.bias.copy_(torch.from_numpy(b))
    dump = torch.empty((wl.T, wl.E), dtype=torch.float32, device=DEV) if wl.T * wl.E <= 64 << 20 else None
    rs.route(to_dev(x), to_dev(W), scores_dump=dump)
    idx, w, c = rs.idx.cpu().numpy(), rs.w.cpu().numpy(), rs.counts.cpu().numpy()
    check_invariants(idx, w, c, wl.T, wl.E, wl.K)
    rows = synth.rng(77, wl.wid).choice(wl.T, size=48, replace=False)
    rows = np.sort(np.concatenate([rows, [0, wl.T - 1]]))
    s = dump.cpu().numpy() if dump is not None else None
    check_against_oracle(x, W, b, wl.K, idx, w, c, s, rows=rows, max_uncertain=0.05)
    if s is not None:
        si, sw, sc = gpu_select(s, b, wl.K)
        np.testing.assert_array_equal(idx, si)
        np.testing.assert_array_equal(c, sc)


@pytest.mark.parametrize("name", ["top10-of-768", "top5-of-768-mixture", "top3-of-768-drift", "large-d4096-top10"])
def test_benchmarked_step_full_size(name):
    """The call the benchmark times, in its launch configuration, at the
    workload's full size: the packed router matrix and idb_router_step (the
    fused kernel on the two-slice tiling, then the slice merge whose last
    workgroup applies the ID update and writes MaxVio/MinVio), two steps in a
    row (the second routes with the bias the first one produced).  Sampled rows
    against the oracle's scores and selection (margin-aware, the fused kernel's
    scores taken from a dumping call on the same inputs); counts equal the
    bincount of the indices; the new bias, e_prev, step and MaxVio/MinVio are
    bit-identical to the oracle's controller on the step's counts."""
    wl = synth.WORKLOADS[name]
    W = synth.router_weight(wl)
    Wd = to_dev(W)
    cfg = B.ControllerCfg(wl.E, 6e-3, 6e-3)
    rs = RouterStep(wl.T, wl.d, wl.E, wl.K, torch.bfloat16, cfg=cfg)
    assert rs.info["variant"] == 6 and rs.info["slices"] == 2
    rs.pack(Wd)
    probe = RouterStep(wl.T, wl.d, wl.E, wl.K, torch.bfloat16)  # same tiling, for the score dump
    probe.pack(Wd)
    dump = torch.empty((wl.T, wl.E), dtype=torch.float32, device=DEV)
    ref = oracle.ControllerState(wl.E)
    for t in range(2):
        x = synth.hidden_states(wl, step=t)
        xd = to_dev(x)
        b = rs.state.bias.cpu().numpy().copy()
        print(f"[bench-step] {name} step {t}", flush=True)
        rs.step(xd, None)
        probe.state.bias.copy_(torch.from_numpy(b).to(DEV))  # the bias this step routed with
        probe.route(xd, None, scores_dump=dump)
        torch.cuda.synchronize()
        idx, w, c = rs.idx.cpu().numpy(), rs.w.cpu().numpy(), rs.counts.cpu().numpy()
        check_invariants(idx, w, c, wl.T, wl.E, wl.K)
        np.testing.assert_array_equal(probe.idx.cpu().numpy(), idx)  # same kernels, same bias
        rows = synth.rng(78 + t, wl.wid).choice(wl.T, size=48, replace=False)
        rows = np.sort(np.concatenate([rows, [0, wl.T - 1]]))
        s_rows = dump[torch.from_numpy(rows).to(DEV)].cpu().numpy()
        check_against_oracle(x[rows], W, b, wl.K, idx[rows], w[rows], c, s_rows, rows=None, max_uncertain=0.05)
        assert oracle.controller(c, ref, 6e-3, 6e-3) == 0
        np.testing.assert_array_equal(rs.state.bias.cpu().numpy().view(np.uint32), ref.bias.view(np.uint32))
        np.testing.assert_array_equal(rs.state.e_prev.cpu().numpy().view(np.uint32), ref.e_prev.view(np.uint32))
        assert int(rs.state.step.item()) == int(ref.step[0]) == t + 1
        np.testing.assert_array_equal(rs.stats.cpu().numpy().view(np.uint64), oracle.load_stats(c).view(np.uint64))
    assert np.abs(ref.bias).max() > 0


def test_headline_full_batch_against_oracle():
    """All 16384 rows of the Top-10-of-768 batch (d = 2048) against the oracle:
    scores within rel 2e-3 everywhere, the oracle's selection on every token
    outside near ties (at most 1%), counts = bincount of the indices."""
    wl = synth.WORKLOADS["top10-of-768"]
    x = synth.hidden_states(wl, step=0)
    W = synth.router_weight(wl)
    b = synth.bias(wl.E, "small", seed=wl.wid)
    rs = RouterStep(wl.T, wl.d, wl.E, wl.K, torch.bfloat16)
    rs.state.bias.copy_(torch.from_numpy(b))
    dump = torch.empty((wl.T, wl.E), dtype=torch.float32, device=DEV)
    rs.route(to_dev(x), to_dev(W), scores_dump=dump)
    idx, w, c = rs.idx.cpu().numpy(), rs.w.cpu().numpy(), rs.counts.cpu().numpy()
    check_invariants(idx, w, c, wl.T, wl.E, wl.K)
    n = check_against_oracle(x, W, b, wl.K, idx, w, c, dump.cpu().numpy(), rows=None, max_uncertain=0.01)
    print(f"headline full batch: {n} near-tie tokens of {wl.T}")


@pytest.mark.parametrize("T,d,E,K,dtype,variant", [
    (517, 512, 768, 10, "bf16", 1), (517, 512, 768, 10, "bf16", 2), (300, 256, 768, 5, "bf16", 3),
    (129, 128, 800, 10, "bf16", 4), (1000, 256, 64, 4, "f32", 5), (64, 2048, 256, 8, "bf16", 0),
    (517, 512, 768, 10, "bf16", 6), (300, 192, 800, 7, "bf16", 6), (200, 192, 800, 7, "bf16", 7),
])
def test_packed_weight_layout_is_bit_identical(T, d, E, K, dtype, variant):
    x, W = synth.normal_router_inputs(T, d, E, seed=11, dtype=dtype, w_std=0.05)
    b = synth.bias(E, "small", seed=12)
    ref = run_router(x, W, b, K, variant=variant)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    rs = RouterStep(T, d, E, K, tdt, variant=variant)
    rs.state.bias.copy_(torch.from_numpy(b))
    Wp = rs.pack(to_dev(W))
    assert not torch.equal(Wp.view(-1), to_dev(W).view(-1)) or E * d <= 64 * 32
    dump = torch.empty((T, E), dtype=torch.float32, device=DEV)
    rs.route(to_dev(x), None, scores_dump=dump)
    np.testing.assert_array_equal(rs.idx.cpu().numpy(), ref[0])
    np.testing.assert_array_equal(rs.w.cpu().numpy(), ref[1])
    np.testing.assert_array_equal(rs.counts.cpu().numpy(), ref[2])
    np.testing.assert_array_equal(dump.cpu().numpy(), ref[3])


def test_pack_weight_is_the_documented_permutation():
    # include/idb.h: piece (b, c, s) at byte ((b*NCH + c)*2 + s)*1024 holds, for
    # lane slot l, bytes [c*128 + 64 s + 16 (l/16), +16) of row 16 b + l%16
    E, d = 96, 256
    _, W = synth.normal_router_inputs(1, d, E, seed=13, dtype="bf16")
    Wt = to_dev(W)
    P = torch.empty_like(Wt)
    B.idb_router_pack_weight(Wt, P)
    got = P.cpu().view(torch.int16).numpy().view(np.uint8).reshape(-1)
    src = W.view(np.uint8).reshape(E, d * 2)
    nch = d * 2 // 128
    want = np.empty_like(got)
    for b in range(E // 16):
        for c in range(nch):
            for s in range(2):
                base = ((b * nch + c) * 2 + s) * 1024
                for l in range(64):
                    lo = c * 128 + 64 * s + 16 * (l // 16)
                    want[base + 16 * l: base + 16 * l + 16] = src[16 * b + l % 16, lo:lo + 16]
    np.testing.assert_array_equal(got, want)

@pytest.mark.parametrize("T,E,K,variant", [
    (1000, 768, 10, 6),   # two slices: the two-pointer merge
    (300, 768, 10, 3),    # three slices: the rank-counting tile merge
    (513, 1024, 32, 4),   # 8 slices x 32 candidates: the generic merge kernel
    (777, 512, 8, 1),     # 32x32 tiles, a padded second slice
])
def test_split_calls_equal_forward(T, E, K, variant):
    """score_select then merge, called separately, give exactly the outputs of
    the one-call forward, with and without accumulation."""
    d = 256
    x, W = synth.normal_router_inputs(T, d, E, seed=T + K, w_std=0.05)
    b = synth.bias(E, "small", seed=3)
    xt, Wt, bt = to_dev(x), to_dev(W), torch.from_numpy(b).to(DEV)
    code = B.IDB_DTYPE_BF16
    ws = torch.zeros(max(B.idb_router_workspace_bytes(T, d, E, K, code, variant), 16), dtype=torch.uint8,
                     device=DEV)
    outs = []
    for split in (False, True):
        idx = torch.full((T, K), -1, dtype=torch.int32, device=DEV)
        w = torch.full((T, K), -1.0, dtype=torch.float32, device=DEV)
        c = torch.full((E,), 7, dtype=torch.int32, device=DEV)
        for acc in (False, True):
            if split:
                B.idb_router_score_select(xt, Wt, bt, K, idx, w, c, acc, workspace=ws, variant=variant)
                B.idb_router_merge(T, d, E, K, code, idx, w, c, workspace=ws, variant=variant)
            else:
                B.idb_router_forward(xt, Wt, bt, K, idx, w, c, acc, workspace=ws, variant=variant)
        outs.append((idx.cpu().numpy(), w.cpu().numpy(), c.cpu().numpy()))
    (i0, w0, c0), (i1, w1, c1) = outs
    np.testing.assert_array_equal(i0, i1)
    np.testing.assert_array_equal(w0.view(np.uint32), w1.view(np.uint32))
    np.testing.assert_array_equal(c0, c1)
    assert int(c0.sum()) == 2 * T * K

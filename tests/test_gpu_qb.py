"""GPU parity of Quantile Balancing (Eq. pid-quantile, Eq. pid-quantile-def)
against the CPU oracle.

* The router's Quantile Balancing mode gives exactly the plain router's
  selection, gate weights and counts; its expert-major scores are the plain
  router's scores, transposed, bit for bit; its cutoffs are the (K+1)-th
  largest biased score fl32(s + b) of those scores (numpy's sort), bit for
  bit.
* The update kernel (exact radix select of each expert's k-th margin) equals
  the oracle's sort-based update bit for bit, for the plain target and the
  EMA variant, on continuous, tied and edge-case scores, across the LDS and
  the global-memory paths.
* A closed loop of Quantile Balancing steps from hidden states: every step
  the GPU's own outputs are consistent (expert-major scores = its dumped
  scores, cutoffs = their (K+1)-th largest biased value, counts = its
  selection, the new bias = numpy's inverted-CDF quantile of its margins),
  and a free-running oracle loop on the same hidden states stays within the
  scores' rounding: selections differ only at near ties, biases within
  1e-4.
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


def bits(t):
    return t.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("T,d,E,K,variant", [
    (1000, 256, 768, 10, 0),    # two slices: two-pointer merge of K+1 candidates
    (700, 256, 768, 10, 7),     # one slice: the cutoff from the fused epilogue
    (300, 256, 768, 5, 3),      # three slices: rank-counting merge
    (513, 128, 1024, 16, 4),    # 8 slices x 17 candidates: the generic merge kernel
    (777, 128, 512, 8, 1),      # 32x32 tiles, a padded second slice
    (4096, 256, 64, 4, 0),      # the tiny workload's shape, bf16
])
def test_qb_router_matches_plain_router_and_oracle_cutoffs(T, d, E, K, variant):
    x, W = synth.normal_router_inputs(T, d, E, seed=T + E, w_std=0.05)
    b = synth.bias(E, "small", seed=K)
    xt, Wt, bt = to_dev(x), to_dev(W), torch.from_numpy(b).to(DEV)
    code = B.IDB_DTYPE_BF16
    ws = torch.empty(max(B.idb_router_workspace_bytes(T, d, E, K, code, variant), 16), dtype=torch.uint8,
                     device=DEV)
    qws = torch.empty(max(B.idb_qb_router_workspace_bytes(T, d, E, K, code, variant), 16), dtype=torch.uint8,
                      device=DEV)
    idx0 = torch.empty((T, K), dtype=torch.int32, device=DEV)
    w0 = torch.empty((T, K), dtype=torch.float32, device=DEV)
    c0 = torch.empty(E, dtype=torch.int32, device=DEV)
    dump = torch.empty((T, E), dtype=torch.float32, device=DEV)
    B.idb_router_forward(xt, Wt, bt, K, idx0, w0, c0, scores_dump=dump, workspace=ws, variant=variant)
    idx = torch.empty_like(idx0)
    w = torch.empty_like(w0)
    c = torch.empty_like(c0)
    st = torch.empty((E, T), dtype=torch.float32, device=DEV)
    alpha = torch.empty(T, dtype=torch.float32, device=DEV)
    B.idb_qb_router_forward(xt, Wt, bt, K, idx, w, c, st, alpha, workspace=qws, variant=variant)
    assert torch.equal(idx, idx0) and torch.equal(c, c0)
    np.testing.assert_array_equal(bits(w), bits(w0))
    s = dump.cpu().numpy()
    np.testing.assert_array_equal(bits(st), np.ascontiguousarray(s.T).view(np.uint32))
    np.testing.assert_array_equal(bits(alpha), kth_biased(s, b, K).view(np.uint32))


def kth_biased(s, b, K):
    """The (K+1)-th largest fl32(s + b) per row, -0 written as +0 (numpy's sort)."""
    v = (s + b[None, :]).astype(np.float32)
    return (-np.sort(-v, axis=1)[:, K] + np.float32(0.0)).astype(np.float32)


def margin_quantile_target(s, alpha, K):
    """-(k-th smallest margin fl32(s - alpha), -0 read as +0), k = ceil(T (E - K) / E): numpy's inverted CDF."""
    T, E = s.shape
    d = ((s - alpha[:, None]).astype(np.float32) + np.float32(0.0)).astype(np.float32)
    k = -(-(T * (E - K)) // E)
    return (-np.sort(d, axis=0)[k - 1]).astype(np.float32)


@pytest.mark.parametrize("T,E,K,kind", [
    (1000, 768, 10, "beta"),
    (777, 96, 3, "grid"),        # heavy ties
    (333, 64, 5, "edges"),       # +-0, 1.0, tiny values
    (16384, 768, 10, "beta"),    # the headline shape
    (32768, 64, 3, "beta"),      # the largest batch held in LDS
    (40000, 32, 4, "grid"),      # beyond LDS: keys recomputed per pass
])
@pytest.mark.parametrize("rho", [0.0, 0.5, 0.9])
def test_qb_update_matches_oracle(T, E, K, kind, rho):
    s = synth.scores(T, E, kind, seed=T + K)
    b = synth.bias(E, "small", seed=E)
    alpha = oracle.qb_alpha(s, b, K)
    want = oracle.qb_update(s, alpha, K, rho, b.copy())
    st = torch.from_numpy(np.ascontiguousarray(s.T)).to(DEV)
    bt = torch.from_numpy(b.copy()).to(DEV)
    B.idb_qb_update(st, torch.from_numpy(alpha).to(DEV), K, rho, bt)
    np.testing.assert_array_equal(bits(bt), want.view(np.uint32))


@pytest.mark.parametrize("T,E,K", [(1000, 768, 10), (16384, 768, 10), (32768, 64, 3), (40000, 32, 4),
                                   (500, 1024, 8)])
def test_qb_update_writes_load_statistics_in_the_same_launch(T, E, K):
    # the first workgroup's MaxVio/MinVio (Eq. vio) equal the oracle's bit for
    # bit, and the bias is the same as without them (every kernel form: 512
    # and 1024 threads with keys in registers, keys recomputed from memory)
    s = synth.scores(T, E, "beta", seed=T + 3)
    b = synth.bias(E, "small", seed=E + 1)
    alpha = oracle.qb_alpha(s, b, K)
    st = torch.from_numpy(np.ascontiguousarray(s.T)).to(DEV)
    at = torch.from_numpy(alpha).to(DEV)
    rng = np.random.default_rng(E)
    for c in (rng.integers(0, 3 * T * K // E + 2, E).astype(np.int32), np.zeros(E, np.int32),
              np.full(E, 7, np.int32)):
        plain = torch.from_numpy(b.copy()).to(DEV)
        B.idb_qb_update(st, at, K, 0.5, plain)
        bt = torch.from_numpy(b.copy()).to(DEV)
        stats = torch.full((2,), -1.0, dtype=torch.float64, device=DEV)
        B.idb_qb_update(st, at, K, 0.5, bt, counts=torch.from_numpy(c).to(DEV), stats=stats)
        np.testing.assert_array_equal(bits(bt), bits(plain))
        want = np.asarray(oracle.load_stats(c), np.float64)
        got = stats.cpu().numpy()
        if c.sum() == 0:
            assert np.isnan(got).all() and np.isnan(want).all()  # empty batch
        else:
            np.testing.assert_array_equal(got.view(np.uint64), want.view(np.uint64))


def test_qb_closed_loop():
    """Quantile Balancing steps on the skewed mixture inputs (see the module
    notes): GPU-internal consistency every step, and a free-running oracle
    loop on the same hidden states close to the GPU's."""
    wl = synth.WORKLOADS["top5-of-768-mixture"]
    T, d, E, K = 2048, 256, wl.E, wl.K
    mu, pi = synth.mixture_params(wl)
    rng = np.random.default_rng(4)
    W = synth.to_bf16_bits(rng.standard_normal((E, d)).astype(np.float32) * np.float32(0.05))
    rs = RouterStep(T, d, E, K, torch.bfloat16)
    Wt = to_dev(W)
    rs.pack(Wt)
    ref_b = np.zeros(E, np.float32)
    dump = torch.empty((T, E), dtype=torch.float32, device=DEV)
    flips = 0
    for t in range(6):
        comp = rng.choice(len(pi), size=T, p=pi)
        x = synth.to_bf16_bits((mu[comp][:, :d] + np.float32(0.5) * rng.standard_normal((T, d))).astype(np.float32))
        xt = to_dev(x)
        b_gpu = rs.state.bias.cpu().numpy()
        rs.route(xt, None, scores_dump=dump)  # the scores the step will select with
        rs.qb_step(xt, None, rho=0.0)
        s = dump.cpu().numpy()
        idx, c = rs.idx.cpu().numpy(), rs.counts.cpu().numpy()
        np.testing.assert_array_equal(c, np.bincount(idx.ravel(), minlength=E))
        np.testing.assert_array_equal(bits(rs.scores_t), np.ascontiguousarray(s.T).view(np.uint32))
        alpha = kth_biased(s, b_gpu, K)
        np.testing.assert_array_equal(bits(rs.alpha), alpha.view(np.uint32))
        S = T * K
        np.testing.assert_array_equal(rs.stats.cpu().numpy(), [(E * int(c.max()) - S) / S, (S - E * int(c.min())) / S])
        np.testing.assert_array_equal(bits(rs.state.bias), margin_quantile_target(s, alpha, K).view(np.uint32),
                                      err_msg=f"bias step {t}")
        # the free-running oracle on its own scores of the same hidden states
        s_ref = oracle.router_scores(x, W)
        r_idx, _, _ = oracle.select(s_ref, ref_b, K)
        r_alpha = oracle.qb_alpha(s_ref, ref_b, K)
        oracle.qb_update(s_ref, r_alpha, K, 0.0, ref_b)
        flips += int((np.sort(idx, 1) != np.sort(r_idx, 1)).any(1).sum())
        np.testing.assert_allclose(rs.state.bias.cpu().numpy(), ref_b, atol=1e-4, err_msg=f"oracle bias step {t}")
    assert flips <= 0.01 * T * 6, flips

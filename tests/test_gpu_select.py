"""GPU parity of the selection stage given identical fp32 scores
(Eq. pid-routing; gate weights of Sec. 2.2; counts of Eq. pid-error):
expert indices, gate weights and counts must be bit-identical to the oracle's
on the same synthetic scores, including heavy ties, +-0, saturated scores,
ragged token counts, K > 16 and expert counts that are not multiples of 4."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_39137_amd import binding as B
from paper_2609_39137_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def gpu_select(s, b, K, counts=None):
    T, E = s.shape
    st = torch.from_numpy(s).to(DEV)
    bt = torch.from_numpy(b).to(DEV)
    idx = torch.empty((T, K), dtype=torch.int32, device=DEV)
    w = torch.empty((T, K), dtype=torch.float32, device=DEV)
    acc = counts is not None
    c = counts if acc else torch.full((E,), 12345, dtype=torch.int32, device=DEV)
    B.idb_select_from_scores(st, bt, K, idx, w, c, accumulate=acc)
    return idx.cpu().numpy(), w.cpu().numpy(), c.cpu().numpy()


def check(s, b, K):
    idx, w, c = gpu_select(s, b, K)
    ridx, rw, rc = oracle.select(s, b, K)
    np.testing.assert_array_equal(idx, ridx)
    np.testing.assert_array_equal(w.view(np.uint32), rw.view(np.uint32))
    np.testing.assert_array_equal(c, rc)


@pytest.mark.parametrize("E", [32, 64, 100, 256, 512, 768, 1024])
@pytest.mark.parametrize("kind", ["beta", "grid", "edges", "saturated"])
def test_select_matches_oracle(E, kind):
    for T, K, bkind in ((1, 1, "zero"), (17, 3, "small"), (333, 10, "grid"), (1000, min(16, E), "large"),
                        (257, min(17, E), "small"), (64, min(32, E), "grid")):
        s = synth.scores(T, E, kind, seed=T + E)
        b = synth.bias(E, bkind, seed=K)
        check(s, b, K)


def test_all_equal_scores_take_lowest_indices():
    s = synth.scores(50, 768, "const", seed=0)
    for K in (1, 10, 32):
        check(s, np.zeros(768, np.float32), K)
        idx, _, _ = gpu_select(s, np.zeros(768, np.float32), K)
        assert np.all(idx == np.arange(K)[None, :])


@pytest.mark.parametrize("E", [256, 512, 768, 1024])
def test_overflowing_and_listed_tokens_share_waves(E):
    # constant rows (every score tied: the list overflows) between rows of
    # distinct scores, so both paths run inside one wave
    s = synth.scores(200, E, "beta", seed=12)
    s[::4] = np.float32(0.25)
    b = np.zeros(E, np.float32)
    for K in (1, 10, 32):
        check(s, b, K)


def test_headline_shape_full_size():
    s = synth.scores(16384, 768, "beta", seed=1)
    b = synth.bias(768, "small", seed=2)
    check(s, b, 10)


def test_counts_accumulate_over_microbatches():
    s = synth.scores(3000, 768, "beta", seed=4)
    b = synth.bias(768, "small", seed=5)
    counts = torch.zeros(768, dtype=torch.int32, device=DEV)
    for lo, hi in ((0, 1000), (1000, 1001), (1001, 3000)):
        gpu_select(np.ascontiguousarray(s[lo:hi]), b, 5, counts=counts)
    _, _, rc = oracle.select(s, b, 5)
    np.testing.assert_array_equal(counts.cpu().numpy(), rc)


def test_gate_weights_sum_to_one_and_ignore_bias():
    s = synth.scores(2000, 768, "beta", seed=8)
    idx0, w0, _ = gpu_select(s, np.zeros(768, np.float32), 10)
    assert np.all(np.abs(w0.astype(np.float64).sum(1) - 1.0) <= 10 * 2.0 ** -23)
    # shifting every bias by the same dyadic constant keeps sets and weights
    # when the sums are exact: scores on a 2^-12 grid
    g = (np.round(s * 4096) / 4096).astype(np.float32)
    b = synth.bias(768, "grid", seed=9)
    i1, w1, _ = gpu_select(g, b, 10)
    i2, w2, _ = gpu_select(g, (b + np.float32(0.5)).astype(np.float32), 10)
    np.testing.assert_array_equal(i1, i2)
    np.testing.assert_array_equal(w1, w2)


@pytest.mark.parametrize("T,E,K", [(70001, 64, 4), (40001, 768, 10), (33000, 1024, 8)])
def test_more_tiles_than_workgroups(T, E, K):
    # more 64-token tiles than the launch has workgroups, so each walks
    # several (grid-stride), ragged last tile; with E a multiple of 256 the
    # full tiles take the load path without per-chunk conditions
    s = synth.scores(T, E, "beta", seed=21 + E)
    b = synth.bias(E, "small", seed=22 + E)
    check(s, b, K)


@pytest.mark.parametrize("E", [30, 770])
def test_expert_count_not_multiple_of_four(E):
    for T, K in ((129, 10), (40, 3)):
        s = synth.scores(T, E, "grid", seed=E + K)
        b = synth.bias(E, "small", seed=K)
        check(s, b, K)


def test_misaligned_score_rows():
    # a view starting one float into the allocation: rows are not 16-byte
    # aligned, which the register-resident kernel needs
    T, E, K = 300, 768, 10
    s = synth.scores(T, E, "beta", seed=31)
    b = synth.bias(E, "small", seed=32)
    base = torch.empty(T * E + 1, dtype=torch.float32, device=DEV)
    st = base[1:].view(T, E)
    st.copy_(torch.from_numpy(s))
    assert st.data_ptr() % 16 != 0
    idx = torch.empty((T, K), dtype=torch.int32, device=DEV)
    w = torch.empty((T, K), dtype=torch.float32, device=DEV)
    c = torch.empty(E, dtype=torch.int32, device=DEV)
    B.idb_select_from_scores(st, torch.from_numpy(b).to(DEV), K, idx, w, c, accumulate=False)
    ridx, rw, rc = oracle.select(s, b, K)
    np.testing.assert_array_equal(idx.cpu().numpy(), ridx)
    np.testing.assert_array_equal(w.cpu().numpy().view(np.uint32), rw.view(np.uint32))
    np.testing.assert_array_equal(c.cpu().numpy(), rc)


@pytest.mark.parametrize("E,K", [(768, 10), (768, 3), (64, 4), (256, 10), (768, 16), (770, 10)])
def test_rows_with_fewer_than_k_finite_biased_scores(E, K):
    # finite inputs whose sums overflow: s = b = -FLT_MAX gives s + b = -inf.
    # Rows where only 2 experts have a finite biased score must still select
    # K experts: the finite ones, then the -inf ones by lowest index (the
    # register kernel's overflow rounds and the epilogue's infinite-threshold
    # masks); ordinary rows share the waves.
    big = np.float32(-np.finfo(np.float32).max)
    s = synth.scores(130, E, "beta", seed=E + K)
    b = synth.bias(E, "small", seed=K)
    live = np.array([E // 3, E - 1])
    b_ovf = np.full(E, big, np.float32)
    b_ovf[live] = b[live]
    s[1::3] = big
    s[1::3, live] = np.float32(0.5)
    s[2::3, : E // 2] = big
    check(s, b_ovf, K)
    idx, _, _ = gpu_select(s, b_ovf, K)
    assert set(idx[1, :2].tolist()) == set(live.tolist())


@pytest.mark.parametrize("E,K", [(768, 16), (768, 10), (100, 12), (1024, 32)])
def test_signed_zero_scores_and_bias_tie(E, K):
    # every biased value is -0 or +0 (equal): the K lowest indices win, in
    # both the register kernel and the epilogue's threshold masks
    g = synth.rng(77, E, K)
    s = np.where(g.random((96, E)) < 0.5, np.float32(-0.0), np.float32(0.0)).astype(np.float32)
    b = np.where(g.random(E) < 0.5, np.float32(-0.0), np.float32(0.0)).astype(np.float32)
    # a third of the rows: -0 scores with -0 bias on the low experts, +0 on the rest
    s[::3, : E // 2] = np.float32(-0.0)
    b2 = b.copy()
    b2[: E // 2] = np.float32(-0.0)
    for bb in (b, b2):
        check(s, bb, K)
        idx, _, _ = gpu_select(s, bb, K)
        assert np.all(idx == np.arange(K)[None, :])

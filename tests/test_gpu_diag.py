"""GPU parity of the batched multi-layer controller with its diagnostics and of
the routing entropies, against the CPU oracle.

* idb_controller_update_layers: every layer's bias, e_prev, step and status
  bit-exact against the oracle's single-layer update on that layer, MaxVio /
  MinVio and the four diagnostics equal to the oracle's, over a trajectory of
  count streams, including layers with empty and invalid batches.
* idb_routing_entropy, on seeded gate weights and scores generated on the
  host (zero weights, clamped scores and an all-clamped token included):
  H_topK within rel 1e-9 of the oracle's (both fp64 logarithms, sums in
  different orders); H_full within the bound of the kernel's fp32 log2 per
  score: each term c log2 c is off by at most c 2^-21 (1 + |log2 c|) (a few
  ulp of the hardware log2, absolute near c = 1, relative elsewhere), so a
  token's entropy ln C - ln 2 (sum c log2 c) / C is off by at most
  ln 2 2^-21 (1 + sum c |log2 c| / C); the fp64 sums add rounding far below.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_39137_amd import binding as B
from paper_2609_39137_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("L,E,kind,mode,center", [
    (21, 768, "drift", B.IDB_INTEGRAL_ERROR, True),
    (3, 64, "sparse", B.IDB_INTEGRAL_ERROR, True),
    (5, 100, "drift", B.IDB_INTEGRAL_SIGN, False),
    (2, 1024, "sparse", B.IDB_INTEGRAL_ERROR, True),
])
def test_layers_update_and_diagnostics_match_oracle(L, E, kind, mode, center):
    Ki, Kd = (6e-3, 6e-3) if mode == B.IDB_INTEGRAL_ERROR else (1e-3, 0.0)
    cfg = B.ControllerCfg(E, Ki, Kd, mode, center)
    st = B.ControllerState(E, DEV, layers=L)
    refs = [oracle.ControllerState(E) for _ in range(L)]
    streams = [synth.count_stream(E, 16384 * 5, 8, kind, seed=100 + l) for l in range(L)]
    stats = torch.empty((L, 2), dtype=torch.float64, device=DEV)
    diag = torch.empty((L, 4), dtype=torch.float64, device=DEV)
    for t in range(8):
        counts = np.stack([streams[l][t] for l in range(L)]).astype(np.int32)
        if t == 3:
            counts[0] = 0          # an empty batch in layer 0
        if t == 5 and L > 1:
            counts[1, 7] = -1      # an invalid batch in layer 1
        B.idb_controller_update_layers(torch.from_numpy(counts).to(DEV), cfg, st, stats, diag)
        g_stats, g_diag = stats.cpu().numpy(), diag.cpu().numpy()
        for l in range(L):
            status, want_diag = oracle.controller_diag(counts[l], refs[l], Ki, Kd, mode, center)
            assert int(st.status[l].item()) == status, f"step {t} layer {l}"
            np.testing.assert_array_equal(st.bias[l].cpu().numpy().view(np.uint32), refs[l].bias.view(np.uint32))
            np.testing.assert_array_equal(st.e_prev[l].cpu().numpy().view(np.uint32), refs[l].e_prev.view(np.uint32))
            assert int(st.step[l].item()) == int(refs[l].step[0])
            np.testing.assert_array_equal(g_stats[l], oracle.load_stats(counts[l]))
            np.testing.assert_array_equal(g_diag[l], want_diag, err_msg=f"diag step {t} layer {l}")


def test_one_layer_equals_the_single_layer_update():
    E = 768
    cfg = B.ControllerCfg(E)
    one = B.ControllerState(E, DEV, layers=1)
    single = B.ControllerState(E, DEV)
    for t, c in enumerate(synth.count_stream(E, 163840, 5, "drift", seed=3)):
        ct = torch.from_numpy(c.astype(np.int32)).to(DEV)
        B.idb_controller_update_layers(ct.view(1, E), cfg, one)
        B.idb_controller_update(ct, cfg, single)
        assert torch.equal(one.bias[0].view(torch.int32), single.bias.view(torch.int32))
        assert torch.equal(one.e_prev[0].view(torch.int32), single.e_prev.view(torch.int32))


@pytest.mark.parametrize("T,E,K", [(2048, 768, 10), (1000, 64, 4), (300, 512, 3), (4097, 1024, 32)])
def test_routing_entropy_matches_oracle(T, E, K):
    r = synth.rng(T, E, K)
    w = r.random((T, K)).astype(np.float32) + np.float32(1e-3)
    w[::7, -1] = 0.0  # 0 log 0 = 0
    w = (w / w.sum(axis=1, keepdims=True)).astype(np.float32)
    s = synth.scores(T, E, "beta", seed=T + K)
    b = synth.bias(E, "small", seed=E)
    s[5] = -1.0  # every biased score of this token clamps to 0: H_full = 0
    wt, st, bt = (torch.from_numpy(a).to(DEV) for a in (w, s, b))
    out = torch.empty(2, dtype=torch.float64, device=DEV)
    B.idb_routing_entropy(wt, out, st, bt)
    got = out.cpu().numpy()
    np.testing.assert_allclose(got[0], oracle.topk_entropy(w), rtol=1e-9)
    c = np.maximum((s + b[None, :]).astype(np.float32), np.float32(0)).astype(np.float64)
    C = c.sum(axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        m = np.where(c > 0, c * np.abs(np.log2(np.where(c > 0, c, 1.0))), 0.0).sum(axis=1)
        per_token = np.where(C > 0, np.log(2.0) * 2.0 ** -21 * (1.0 + m / np.where(C > 0, C, 1.0)), 0.0)
    tol = per_token.mean() + 1e-12
    assert abs(got[1] - oracle.full_entropy(s, b)) <= tol
    B.idb_routing_entropy(wt, out)  # without scores: H_full is NaN
    got2 = out.cpu().numpy()
    assert got2[0] == got[0] and np.isnan(got2[1])


@pytest.mark.parametrize("T,E,K,scale", [(2048, 768, 10, 1.0), (1000, 64, 4, 3.0), (333, 1024, 32, 0.3),
                                         (129, 768, 10, 40.0)])
def test_softmax_routing_entropy_matches_oracle(T, E, K, scale):
    """H_full of the auxiliary-loss router over softmax(z) (Sec. 4.3).  Bound of
    the kernel's error per token: t_e = exp(x_e) (1 + d_e) with x_e = z_e - M,
    |d_e| <= (1.5 |x_e| + 1) 2^-23 (the rounded difference, the product with
    log2 e and the hardware exp2), and H = log Z - sum t x / Z moves by
    sum_e p_e d_e (1 - log p_e - H), plus sum_e p_e |x_e| 2^-24 from the
    rounded x in the second sum; the fp64 sums add far less."""
    r = synth.rng(T, E, K, 5)
    z = (r.standard_normal((T, E)) * scale).astype(np.float32)
    z[3] = np.float32(0.5)  # equal logits: H = log E
    w = r.random((T, K)).astype(np.float32) + np.float32(1e-3)
    w = (w / w.sum(axis=1, keepdims=True)).astype(np.float32)
    out = torch.empty(2, dtype=torch.float64, device=DEV)
    B.idb_routing_entropy_softmax(torch.from_numpy(w).to(DEV), torch.from_numpy(z).to(DEV), out)
    got = out.cpu().numpy()
    np.testing.assert_allclose(got[0], oracle.topk_entropy(w), rtol=1e-9)
    x = z.astype(np.float64) - z.max(axis=1, keepdims=True).astype(np.float64)
    p = np.exp(x)
    p /= p.sum(axis=1, keepdims=True)
    with np.errstate(divide="ignore", invalid="ignore"):
        lp = np.where(p > 0, np.log(np.where(p > 0, p, 1.0)), 0.0)
    H = -(p * lp).sum(axis=1, keepdims=True)
    d = (1.5 * np.abs(x) + 1.0) * 2.0 ** -23
    per_token = (p * d * np.abs(1.0 - lp - H)).sum(axis=1) + (p * np.abs(x)).sum(axis=1) * 2.0 ** -24
    tol = per_token.mean() + 1e-12
    want = oracle.softmax_entropy(z)
    assert abs(got[1] - want) <= tol, (got[1], want, tol)

"""Seeded random shapes through the C ABI, each against the oracle.

* Selection from given scores (Eq. pid-routing; gate weights of Sec. 2.2;
  counts of Eq. pid-error): any E in [2, 1024], K in [1, min(E, 32)], T in
  [1, 2500], every score and bias family; expert indices, gate weights and
  counts bit-identical to the oracle's.
* One router iteration (Alg. 1) with idb_router_step: E a multiple of 32 up
  to 1024, d a multiple of 64 up to 512, K up to 32, T up to 2048, integer
  inputs (exact logits on both sides) and a zero starting bias, so the
  selection is decided identically; error-scaled or DeepSeek's fixed-step
  integral, with or without centring: indices and counts exact, gate weights
  within the score error, and the new bias, e_prev and MaxVio/MinVio bit for
  bit equal to the oracle's controller on the same counts.
* One Quantile Balancing iteration: the same selection check, then the
  cutoffs, the new bias (EMA weight 0 or 0.5) and MaxVio/MinVio bit for bit
  against the oracle on the GPU's own expert-major scores.
* One routing with idb_router_forward on normally distributed inputs (bf16,
  and fp32 with d a multiple of 32) and a bias: scores within the accumulation error of the oracle's, the selection
  margin-aware against the oracle's, and bit-identical to the oracle's
  selection on the kernel's own fp32 scores.
* The auxiliary-loss router's forward statistics (E up to 768): on integer
  inputs selection, counts, f and MaxVio/MinVio exactly as the oracle's, P
  and the loss within the bound derived in tests/test_gpu_aux.py.
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


def _select_cases(n=120):
    g = np.random.default_rng(20261202)
    for i in range(n):
        E = int(g.integers(2, 1025))
        K = int(g.integers(1, min(E, 32) + 1))
        T = int(g.integers(1, 2501))
        kind = str(g.choice(["beta", "grid", "edges", "saturated"]))
        bkind = str(g.choice(["zero", "small", "large", "grid"]))
        yield T, E, K, kind, bkind, i


def _router_cases(n=48):
    g = np.random.default_rng(20261203)
    for i in range(n):
        E = 32 * int(g.integers(1, 33))
        K = int(g.integers(1, min(E, 32) + 1))
        d = 64 * int(g.integers(1, 9))
        T = int(g.integers(1, 2049))
        sign = bool(g.integers(0, 2))      # DeepSeek's fixed-step integral, else error-scaled
        center = bool(g.integers(0, 2))
        yield T, d, E, K, sign, center, i


@pytest.mark.parametrize("T,E,K,kind,bkind,seed", list(_select_cases()))
def test_select_random_shapes(T, E, K, kind, bkind, seed):
    s = synth.scores(T, E, kind, seed=1000 + seed)
    b = synth.bias(E, bkind, seed=2000 + seed)
    idx = torch.empty((T, K), dtype=torch.int32, device=DEV)
    w = torch.empty((T, K), dtype=torch.float32, device=DEV)
    c = torch.full((E,), 12345, dtype=torch.int32, device=DEV)
    B.idb_select_from_scores(torch.from_numpy(s).to(DEV), torch.from_numpy(b).to(DEV), K, idx, w, c)
    ridx, rw, rc = oracle.select(s, b, K)
    np.testing.assert_array_equal(idx.cpu().numpy(), ridx)
    np.testing.assert_array_equal(w.cpu().numpy().view(np.uint32), rw.view(np.uint32))
    np.testing.assert_array_equal(c.cpu().numpy(), rc)


@pytest.mark.parametrize("T,d,E,K,sign,center,seed", list(_router_cases()))
def test_router_step_random_shapes(T, d, E, K, sign, center, seed):
    Ki, Kd = 2.0 ** -7, 2.0 ** -6
    mode = B.IDB_INTEGRAL_SIGN if sign else B.IDB_INTEGRAL_ERROR
    x, W = synth.integer_router_inputs(T, d, E, seed=3000 + seed, dtype="bf16", w_shift=6)
    rs = RouterStep(T, d, E, K, torch.bfloat16, B.ControllerCfg(E, Ki, Kd, mode, center), device=DEV)
    xt = torch.from_numpy(x.view(np.int16)).to(DEV).view(torch.bfloat16)
    Wt = torch.from_numpy(W.view(np.int16)).to(DEV).view(torch.bfloat16)
    rs.step(xt, Wt)
    torch.cuda.synchronize()
    ref = oracle.ControllerState(E)
    r_idx, r_w, r_c = oracle.router(x, W, ref.bias, K)
    np.testing.assert_array_equal(rs.idx.cpu().numpy(), r_idx)
    np.testing.assert_array_equal(rs.counts.cpu().numpy(), r_c)
    np.testing.assert_allclose(rs.w.cpu().numpy(), r_w, rtol=2e-5)
    oracle.controller(r_c, ref, Ki, Kd, oracle.MODE_SIGN if sign else oracle.MODE_ERROR, center)
    np.testing.assert_array_equal(rs.state.bias.cpu().numpy(), ref.bias)
    np.testing.assert_array_equal(rs.state.e_prev.cpu().numpy(), ref.e_prev)
    np.testing.assert_array_equal(rs.stats.cpu().numpy(), oracle.load_stats(r_c))


def _qb_cases(n=24):
    g = np.random.default_rng(20261204)
    for i in range(n):
        E = 32 * int(g.integers(1, 33))
        K = int(g.integers(1, min(E - 1, 31) + 1))
        d = 64 * int(g.integers(1, 9))
        T = int(g.integers(1, 2049))
        rho = float(g.choice([0.0, 0.5]))
        yield T, d, E, K, rho, i


@pytest.mark.parametrize("T,d,E,K,rho,seed", list(_qb_cases()))
def test_qb_step_random_shapes(T, d, E, K, rho, seed):
    # one Quantile Balancing iteration (Eq. pid-quantile, pid-quantile-def)
    # from a zero bias on integer inputs: selection exact against the oracle;
    # the cutoffs, the new bias and MaxVio/MinVio bit for bit against the
    # oracle on the GPU's own expert-major scores
    x, W = synth.integer_router_inputs(T, d, E, seed=4000 + seed, dtype="bf16", w_shift=6)
    rs = RouterStep(T, d, E, K, torch.bfloat16, device=DEV)
    xt = torch.from_numpy(x.view(np.int16)).to(DEV).view(torch.bfloat16)
    Wt = torch.from_numpy(W.view(np.int16)).to(DEV).view(torch.bfloat16)
    rs.qb_step(xt, Wt, rho=rho)
    torch.cuda.synchronize()
    b0 = np.zeros(E, np.float32)
    r_idx, r_w, r_c = oracle.router(x, W, b0, K)
    np.testing.assert_array_equal(rs.idx.cpu().numpy(), r_idx)
    np.testing.assert_array_equal(rs.counts.cpu().numpy(), r_c)
    np.testing.assert_allclose(rs.w.cpu().numpy(), r_w, rtol=2e-5)
    s = np.ascontiguousarray(rs.scores_t.cpu().numpy().T)
    np.testing.assert_allclose(s, oracle.router_scores(x, W), rtol=2e-6)
    alpha = oracle.qb_alpha(s, b0, K)
    np.testing.assert_array_equal(rs.alpha.cpu().numpy().view(np.uint32), alpha.view(np.uint32))
    want = oracle.qb_update(s, alpha, K, rho, b0.copy())
    np.testing.assert_array_equal(rs.state.bias.cpu().numpy().view(np.uint32), want.view(np.uint32))
    np.testing.assert_array_equal(rs.stats.cpu().numpy(), oracle.load_stats(r_c))


def _aux_cases(n=24):
    g = np.random.default_rng(20261205)
    for i in range(n):
        E = 32 * int(g.integers(1, 25))  # one-slice tilings cover E <= 768
        K = int(g.integers(1, min(E, 32) + 1))
        d = 64 * int(g.integers(1, 9))
        T = int(g.integers(1, 2049))
        yield T, d, E, K, i


@pytest.mark.parametrize("T,d,E,K,seed", list(_aux_cases()))
def test_aux_router_random_shapes(T, d, E, K, seed):
    # the auxiliary-loss forward statistics (Eq. pid-auxloss) on integer
    # inputs: exact logits, so selection, counts, f and MaxVio/MinVio match
    # the oracle exactly and P and the loss lie within the derived bound
    from tests.test_gpu_aux import check_aux, run_aux

    x, W = synth.integer_router_inputs(T, d, E, seed=5000 + seed, dtype="bf16", w_shift=6)
    g = run_aux(x, W, K, 0.05)
    check_aux(x, W, K, 0.05, g, exact=True)


def _forward_cases(n=32, n_f32=12):
    g = np.random.default_rng(20261206)
    for i in range(n + n_f32):
        f32 = i >= n  # fp32 inputs (d a multiple of 32)
        E = 32 * int(g.integers(1, 9 if f32 else 33))
        K = int(g.integers(1, min(E, 32) + 1))
        d = (32 if f32 else 64) * int(g.integers(1, 9))
        T = int(g.integers(1, 1025 if f32 else 2049))
        bkind = str(g.choice(["zero", "small", "large", "grid"]))
        yield T, d, E, K, bkind, "f32" if f32 else "bf16", i


@pytest.mark.parametrize("T,d,E,K,bkind,dtype,seed", list(_forward_cases()))
def test_router_forward_random_shapes(T, d, E, K, bkind, dtype, seed):
    # normally distributed inputs and a biased selection (Eq. pid-routing):
    # the fused kernel's scores within the fp32 accumulation error of the
    # oracle's, its selection margin-aware against the oracle's, and, given
    # its own fp32 scores, indices, gate weights and counts bit-identical to
    # the oracle's selection
    from tests.test_gpu_router import check_against_oracle, check_invariants, run_router

    x, W = synth.normal_router_inputs(T, d, E, seed=6000 + seed, dtype=dtype, w_std=0.05)
    b = synth.bias(E, bkind, seed=7000 + seed)
    idx, w, c, s = run_router(x, W, b, K)
    check_invariants(idx, w, c, T, E, K)
    check_against_oracle(x, W, b, K, idx, w, c, s, max_uncertain=0.02)
    r_idx, r_w, r_c = oracle.select(s, b, K)
    np.testing.assert_array_equal(idx, r_idx)
    np.testing.assert_array_equal(w.view(np.uint32), r_w.view(np.uint32))
    np.testing.assert_array_equal(c, r_c)

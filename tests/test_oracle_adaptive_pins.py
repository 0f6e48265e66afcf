"""Pins of the oracle's Prox-RMSProp (Algorithm 1) and Prox-ADAM (Algorithm 2).

Each test checks the oracle against a fact the algorithms fix, not against a
retyping of its own formulas:
- constant gradients: Algorithm 2's bias corrections make m^_t = c and
  v^_t = c^2 for every t, so each step moves a weight by eta*c/(|c|+eps);
  Algorithm 1 has none, so v_t = (1 - beta^t) c^2 in closed form;
- the fixed point of the full-gradient iteration on 0.5*||w - a||^2, which
  is the soft-threshold S_{lambda*eps/(1-lambda)}(a) for both algorithms;
- invariance of the preconditioned step under power-of-two gradient scaling;
- beta1 = beta2 = 0 makes Algorithm 2 coincide with Algorithm 1 at beta = 0;
- the threshold eta*lambda acts on the unthresholded step exactly as the
  soft-threshold of Section 2.2;
- the stored-entry (CSR) form equals the dense form gathered on the pattern.
"""
import numpy as np
import pytest

import oracle
from oracle import ADAM, RMSPROP

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _dense_csr(w):
    """A 1 x K CSR holding every entry of w (zeros stored too)."""
    K = w.shape[0]
    return (np.array([0, K], np.int32), np.arange(K, dtype=np.int32), w.astype(np.float32))


def _row_step(solver, w, g, m, v, eta, lam, eps, b1, b2, t):
    rp, ci, vals = _dense_csr(w)
    Z, _, m2, v2 = oracle.prox_adaptive_dense(solver, rp, ci, vals, g[None, :], m, v, eta, lam,
                                              eps, b1, b2, t, w.shape[0])
    return Z[0], m2[0], v2[0]


def _signed_uniform(rng, n, lo, hi):
    return (rng.uniform(lo, hi, n) * rng.choice([-1.0, 1.0], n)).astype(np.float32)


def test_adam_constant_gradient_moves_by_eta_c_over_abs_c_plus_eps():
    rng = np.random.default_rng(11)
    K, T = 257, 30
    eta, eps, b1, b2 = 1e-3, 1e-8, 0.9, 0.999
    c = _signed_uniform(rng, K, 0.1, 2.0)
    w0 = rng.uniform(-1, 1, K).astype(np.float32)
    w, m, v = w0.copy(), None, None
    for t in range(1, T + 1):
        w, m, v = _row_step(ADAM, w, c, m, v, eta, 0.0, eps, b1, b2, t)
        cd = c.astype(np.float64)
        expect = w0.astype(np.float64) - t * eta * cd / (np.abs(cd) + eps)
        np.testing.assert_allclose(w, expect, rtol=0, atol=4e-6 + 2e-7 * t)


def test_rmsprop_constant_gradient_follows_closed_form_second_moment():
    rng = np.random.default_rng(12)
    K, T = 129, 25
    eta, eps, beta = 1e-3, 1e-8, 0.9
    c = _signed_uniform(rng, K, 0.1, 2.0)
    w0 = rng.uniform(-1, 1, K).astype(np.float32)
    w, v = w0.copy(), None
    expect = w0.astype(np.float64)
    cd = c.astype(np.float64)
    for t in range(1, T + 1):
        w, _, v = _row_step(RMSPROP, w, c, None, v, eta, 0.0, eps, 0.0, beta, t)
        vt = (1.0 - beta ** t) * cd * cd
        np.testing.assert_allclose(v, vt, rtol=4e-7 * t, atol=0)
        expect = expect - eta * cd / (np.sqrt(vt) + eps)
        np.testing.assert_allclose(w, expect, rtol=0, atol=4e-6 + 2e-7 * t)


@pytest.mark.parametrize("solver", [ADAM, RMSPROP])
@pytest.mark.parametrize("lam,eps", [(0.5, 0.1), (0.25, 0.3), (0.75, 0.02)])
def test_full_gradient_fixed_point_is_soft_threshold(solver, lam, eps):
    # f(w) = 0.5*||w - a||^2: at a fixed point with w != 0 the step
    # g/(|g|+eps) must cancel the threshold, |g| = lam*eps/(1-lam); with w = 0
    # it must not exceed it.  Both cases together: w* = S_{lam*eps/(1-lam)}(a).
    # every |a| at least 0.015 away from the thresholds 0.1, 0.1 and 0.06
    a = np.array([-0.3, 0.05, 0.25, 0.13, -0.07, 0.5, -0.12, 0.0, 0.075, -0.045], np.float32)
    thr = lam * eps / (1.0 - lam)
    ad = a.astype(np.float64)
    expect = np.sign(ad) * np.maximum(np.abs(ad) - thr, 0.0)
    w, m, v = np.zeros_like(a), None, None
    for t in range(1, 4001):
        g = (w - a).astype(np.float32)
        w, m, v = _row_step(solver, w, g, m, v, 0.01, lam, eps, 0.5, 0.6, t)
    np.testing.assert_allclose(w, expect, rtol=0, atol=2e-6)
    assert np.all((w == 0) == (expect == 0))


@pytest.mark.parametrize("k", [5, -7])
def test_adam_step_invariant_under_power_of_two_gradient_scaling(k):
    # with eps far below sqrt(v^) the step m^/(sqrt(v^)+eps) is scale free, and
    # every operation commutes with an exact power-of-two scale
    rng = np.random.default_rng(13)
    K = 300
    eps = 1e-30
    w = rng.normal(0, 0.1, K).astype(np.float32)
    ws = w.copy()
    m = v = ms = vs = None
    s = np.float32(2.0 ** k)
    for t in range(1, 4):
        g = _signed_uniform(rng, K, 0.01, 1.0)
        w, m, v = _row_step(ADAM, w, g, m, v, 1e-2, 0.3, eps, 0.9, 0.999, t)
        ws, ms, vs = _row_step(ADAM, ws, g * s, ms, vs, 1e-2, 0.3, eps, 0.9, 0.999, t)
        assert np.array_equal(w.view(np.int32), ws.view(np.int32))
        assert np.array_equal((m * s).view(np.int32), ms.view(np.int32))
        assert np.array_equal((v * s * s).view(np.int32), vs.view(np.int32))


def test_adam_with_zero_betas_is_rmsprop_with_zero_beta():
    rng = np.random.default_rng(14)
    K = 500
    w = rng.normal(0, 0.1, K).astype(np.float32)
    g = rng.normal(0, 1, K).astype(np.float32)
    v0 = rng.uniform(0, 1, K).astype(np.float32)
    wa, _, va = _row_step(ADAM, w, g, None, v0, 0.01, 0.2, 1e-3, 0.0, 0.0, 7)
    wr, _, vr = _row_step(RMSPROP, w, g, None, v0, 0.01, 0.2, 1e-3, 0.0, 0.0, 7)
    assert np.array_equal(wa.view(np.int32), wr.view(np.int32))
    assert np.array_equal(va.view(np.int32), vr.view(np.int32))


@pytest.mark.parametrize("solver", [ADAM, RMSPROP])
def test_threshold_is_soft_threshold_of_the_unregularised_step(solver):
    rng = np.random.default_rng(15)
    K = 4000
    eta, lam = 0.05, 0.4
    t_thr = eta * lam
    w = rng.normal(0, 0.05, K).astype(np.float32)
    g = rng.normal(0, 1, K).astype(np.float32)
    m0 = rng.normal(0, 0.3, K).astype(np.float32)
    v0 = rng.uniform(0, 1, K).astype(np.float32)
    z0, m1, v1 = _row_step(solver, w, g, m0, v0, eta, 0.0, 1e-3, 0.8, 0.9, 3)
    zl, m2, v2 = _row_step(solver, w, g, m0, v0, eta, lam, 1e-3, 0.8, 0.9, 3)
    # lambda does not enter the state
    assert np.array_equal(m1, m2) and np.array_equal(v1, v2)
    z0d = z0.astype(np.float64)
    st = np.sign(z0d) * np.maximum(np.abs(z0d) - t_thr, 0.0)
    ulp = np.spacing(np.abs(z0)).astype(np.float64)
    assert np.all(np.abs(zl - st) <= ulp)
    clear_keep = np.abs(z0d) > t_thr + ulp
    clear_drop = np.abs(z0d) < t_thr - ulp
    assert clear_keep.sum() > 100 and clear_drop.sum() > 100
    assert np.all(zl[clear_keep] != 0) and np.all(zl[clear_drop] == 0)
    assert np.all(np.sign(zl[clear_keep]) == np.sign(z0[clear_keep]))


@pytest.mark.parametrize("solver", [ADAM, RMSPROP])
def test_stored_entry_form_equals_dense_form_on_the_pattern(solver):
    rng = np.random.default_rng(16)
    N, K, nnz = 37, 53, 600
    flat = np.sort(rng.choice(N * K, nnz, replace=False))
    rows, cols = flat // K, flat % K
    rp = np.zeros(N + 1, np.int32)
    np.add.at(rp, rows + 1, 1)
    rp = np.cumsum(rp).astype(np.int32)
    ci = cols.astype(np.int32)
    vals = rng.normal(0, 0.1, nnz).astype(np.float32)
    G = rng.normal(0, 1, (N, K)).astype(np.float32)
    m = rng.normal(0, 0.2, (N, K)).astype(np.float32)
    v = rng.uniform(0, 0.5, (N, K)).astype(np.float32)
    Z, cnt, m2, v2 = oracle.prox_adaptive_dense(solver, rp, ci, vals, G, m, v, 0.02, 0.1, 1e-4,
                                                0.9, 0.99, 5, K)
    assert np.array_equal(cnt, np.count_nonzero(Z, axis=1))
    out, mc, vc = oracle.prox_adaptive_csr(solver, vals, G[rows, cols], m[rows, cols],
                                           v[rows, cols], 0.02, 0.1, 1e-4, 0.9, 0.99, 5)
    assert np.array_equal(out.view(np.int32), Z[rows, cols].view(np.int32))
    assert np.array_equal(vc.view(np.int32), v2[rows, cols].view(np.int32))
    if solver == ADAM:
        assert np.array_equal(mc.view(np.int32), m2[rows, cols].view(np.int32))


@pytest.mark.parametrize("kw", [dict(eps=0.0), dict(b2=1.0), dict(b1=1.0), dict(t=0),
                                dict(eta=0.0), dict(lam=-1.0), dict(solver=3)])
def test_oracle_rejects_arguments_outside_the_algorithms_inputs(kw):
    p = dict(solver=ADAM, eta=0.01, lam=0.1, eps=1e-8, b1=0.9, b2=0.999, t=1)
    p.update(kw)
    w = np.ones(4, np.float32)
    with pytest.raises(ValueError):
        _row_step(p["solver"], w, w, None, None, p["eta"], p["lam"], p["eps"], p["b1"], p["b2"],
                  p["t"])

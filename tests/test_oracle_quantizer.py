"""Pins of the oracle's offline quantizer (Appendix: offline quantizer derivation)."""

import numpy as np
import pytest
from scipy import stats
from scipy.integrate import quad

from oracle import quantizer


def test_m3_reduces_to_uniform_lloyd_max():
    # For m = 3, Y = u_j^2 ~ Beta(1/2, 1) so X = |u_j| is uniform on [0, 1];
    # the 8-level Lloyd-Max quantizer of U(0,1) is tau_t = t/8, a[t] = (2t+1)/16.
    tau, a, res = quantizer.lloyd_max(3)
    np.testing.assert_allclose(tau, np.arange(1, 8) / 8, rtol=0, atol=1e-15)
    np.testing.assert_allclose(a, (2 * np.arange(8) + 1) / 16, rtol=0, atol=1e-15)


def test_density_normalised_and_cdf_consistent():
    for m in (4, 8, 16):
        total, _ = quad(lambda x: quantizer.magnitude_pdf(x, m), 0, 1, epsabs=1e-13)
        assert abs(total - 1) < 1e-10
        for x in (0.1, 0.3, 0.6, 0.9):
            part, _ = quad(lambda t: quantizer.magnitude_pdf(t, m), 0, x, epsabs=1e-13)
            assert abs(part - float(quantizer.magnitude_cdf(x, m))) < 1e-10


def test_m8_fixed_point_conditions_by_quadrature():
    # Lloyd-Max optimality checked with plain numerical integration of the
    # density (independent of the Beta(1, .) route used by the oracle).
    m = 8
    tau, a, res = quantizer.lloyd_max(m)
    assert res < 1e-40
    edges = np.concatenate(([0.0], tau, [1.0]))
    for t in range(8):
        num, _ = quad(lambda x: x * quantizer.magnitude_pdf(x, m), edges[t], edges[t + 1],
                      epsabs=1e-15, epsrel=1e-13)
        den, _ = quad(lambda x: quantizer.magnitude_pdf(x, m), edges[t], edges[t + 1],
                      epsabs=1e-15, epsrel=1e-13)
        assert abs(num / den - a[t]) < 1e-12
    np.testing.assert_allclose(tau, 0.5 * (a[:-1] + a[1:]), rtol=0, atol=2e-16)
    # ordering: 0 < a0 < tau1 < a1 < ... < tau7 < a7 < 1
    inter = np.empty(15)
    inter[0::2] = a
    inter[1::2] = tau
    assert np.all(np.diff(inter) > 0) and inter[0] > 0 and inter[-1] < 1


def test_m8_matches_float64_iteration_and_beats_uniform_levels():
    tau, a, _ = quantizer.lloyd_max(8)
    t64, a64, _ = quantizer.lloyd_max_fp64(8)
    assert np.max(np.abs(tau - t64)) < 1e-13 and np.max(np.abs(a - a64)) < 1e-13
    # The optimum's error is below that of 8 equal-width cells with midpoint levels.
    u_tau = np.arange(1, 8) / 8
    u_a = (2 * np.arange(8) + 1) / 16
    assert quantizer.quantizer_mse(tau, a, 8) < quantizer.quantizer_mse(u_tau, u_a, 8)


def test_m8_is_a_local_minimum_of_mse():
    tau, a, _ = quantizer.lloyd_max(8)
    base = quantizer.quantizer_mse(tau, a, 8)
    rng = np.random.default_rng(0)
    for _ in range(4):
        dt = rng.normal(0, 2e-3, size=7)
        da = rng.normal(0, 2e-3, size=8)
        assert quantizer.quantizer_mse(tau + dt, a + da, 8) > base


def _haar(D, rng):
    g = rng.standard_normal((D, D))
    qm, r = np.linalg.qr(g)
    return qm * np.sign(np.diag(r))[None, :]


@pytest.mark.parametrize("D,m", [(32, 8), (128, 8)])
def test_beta_priors_under_haar_rotation(D, m):
    # Prop. "Rotation-induced Beta priors": for any fixed unit k_hat and Haar R,
    # z_b = r_b^2 ~ Beta(m/2, (D-m)/2) and (u_b)_j^2 ~ Beta(1/2, (m-1)/2).
    rng = np.random.default_rng(7)
    k_hat = rng.standard_normal(D)
    k_hat /= np.linalg.norm(k_hat)
    n_rot = 3000 if D == 32 else 600
    z, u2 = [], []
    for _ in range(n_rot):
        kt = _haar(D, rng) @ k_hat
        blocks = kt.reshape(D // m, m)
        r2 = np.sum(blocks * blocks, axis=1)
        z.append(r2)
        u2.append((blocks[:, 0] ** 2) / r2)
    z = np.concatenate(z)
    u2 = np.concatenate(u2)
    assert stats.kstest(z, stats.beta(m / 2, (D - m) / 2).cdf).pvalue > 1e-3
    assert stats.kstest(u2, stats.beta(0.5, (m - 1) / 2).cdf).pvalue > 1e-3
    # the density the quantizer is built on describes |u_j|
    assert stats.kstest(np.sqrt(u2), lambda x: quantizer.magnitude_cdf(x, m)).pvalue > 1e-3
    # and a wrong prior is rejected by the same samples
    assert stats.kstest(u2, stats.beta(0.5, m / 2).cdf).pvalue < 1e-3

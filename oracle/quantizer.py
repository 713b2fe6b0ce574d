"""Offline 3-bit magnitude quantizer for the 4-bit direction codes.

Paper: Appendix "Offline Quantizer Derivation from Rotation-Induced Priors",
Prop. "Rotation-induced Beta priors" (Eq. coord_beta_prop) and the
"Coordinate-Magnitude Quantizer" subsection with its Lloyd-Max updates.

For a Haar-random rotation, a unit direction u_b inside an m-dim subspace
is uniform on S^{m-1}, so each squared coordinate Y = u_j^2 follows
Beta(1/2, (m-1)/2).  The quantized quantity is X = |u_j| = sqrt(Y) on [0, 1].
Lloyd-Max alternates
    a[t]   <- E[X | tau_t <= X < tau_{t+1}]          (conditional means)
    tau_t  <- (a[t-1] + a[t]) / 2,  t = 1..L-1       (midpoints)
with tau_0 = 0 and tau_L = 1 until it stops moving.

Both expectations come straight from the Beta prior:
    P(lo <= X < hi)      = I_{hi^2}(1/2, (m-1)/2) - I_{lo^2}(1/2, (m-1)/2)
    E[X 1{lo <= X < hi}] = B(1, (m-1)/2) / B(1/2, (m-1)/2)
                           * (I_{hi^2}(1, (m-1)/2) - I_{lo^2}(1, (m-1)/2))
(the second because sqrt(y) * y^{-1/2} = y^0 turns the Beta(1/2, .) kernel
into a Beta(1, .) kernel), where I is the regularized incomplete beta.

The iteration is first run in float64 with SciPy, then polished by Newton's
method in 60-digit mpmath so that the returned float64 values are the
correctly rounded fixed point (unique: the density of X is log-concave).
"""

from functools import lru_cache

import numpy as np
from scipy.special import beta as _beta_fn
from scipy.special import betainc as _betainc

N_LEVELS = 8  # 3-bit magnitude bins


def magnitude_pdf(x, m):
    """Density of X = |u_j| for u uniform on S^{m-1}: 2 (1-x^2)^{(m-3)/2} / B(1/2,(m-1)/2)."""
    x = np.asarray(x, dtype=np.float64)
    return 2.0 * (1.0 - x * x) ** ((m - 3) / 2.0) / _beta_fn(0.5, (m - 1) / 2.0)


def magnitude_cdf(x, m):
    """P(X <= x) = P(Y <= x^2) with Y ~ Beta(1/2, (m-1)/2)."""
    x = np.asarray(x, dtype=np.float64)
    return _betainc(0.5, (m - 1) / 2.0, x * x)


def _partial_mean(x, m):
    """E[X 1{X < x}] via the Beta(1, (m-1)/2) kernel (see module docstring)."""
    b = (m - 1) / 2.0
    x = np.asarray(x, dtype=np.float64)
    return _beta_fn(1.0, b) / _beta_fn(0.5, b) * _betainc(1.0, b, x * x)


def conditional_means(tau_inner, m):
    """a[t] = E[X | tau_t <= X < tau_{t+1}] for the bins cut by tau_inner."""
    edges = np.concatenate(([0.0], np.asarray(tau_inner, dtype=np.float64), [1.0]))
    mass = np.diff(magnitude_cdf(edges, m))
    first = np.diff(_partial_mean(edges, m))
    return first / mass


def lloyd_max_fp64(m, levels=N_LEVELS, tol=1e-15, max_iter=200_000):
    """Plain float64 Lloyd-Max iteration, started from equal-mass thresholds."""
    # Start from quantiles of X: tau_t with P(X < tau_t) = t/L (bisection on the CDF).
    tau = np.empty(levels - 1)
    for t in range(1, levels):
        lo, hi = 0.0, 1.0
        for _ in range(200):
            mid = 0.5 * (lo + hi)
            if magnitude_cdf(mid, m) < t / levels:
                lo = mid
            else:
                hi = mid
        tau[t - 1] = 0.5 * (lo + hi)
    for it in range(max_iter):
        a = conditional_means(tau, m)
        new_tau = 0.5 * (a[:-1] + a[1:])
        delta = np.max(np.abs(new_tau - tau))
        tau = new_tau
        if delta < tol:
            break
    return tau, conditional_means(tau, m), it + 1


def _mp_fixed_point(tau0, m, dps=60, newton_steps=6):
    """Newton polish of tau = midpoints(a(tau)) in mpmath; returns mp values."""
    import mpmath as mp

    with mp.workdps(dps):
        b = mp.mpf(m - 1) / 2
        half = mp.mpf(1) / 2
        coef = mp.beta(1, b) / mp.beta(half, b)

        def means(tau):
            edges = [mp.mpf(0)] + list(tau) + [mp.mpf(1)]
            cdf = [mp.betainc(half, b, 0, e * e, regularized=True) for e in edges]
            pm = [coef * mp.betainc(1, b, 0, e * e, regularized=True) for e in edges]
            return [(pm[i + 1] - pm[i]) / (cdf[i + 1] - cdf[i]) for i in range(len(edges) - 1)]

        def residual(tau):
            a = means(tau)
            return mp.matrix([tau[i] - (a[i] + a[i + 1]) / 2 for i in range(len(tau))])

        tau = [mp.mpf(float(t)) for t in tau0]
        n = len(tau)
        h = mp.mpf(10) ** (-(dps // 2))
        for _ in range(newton_steps):
            r = residual(tau)
            jac = mp.matrix(n, n)
            for j in range(n):
                tp = list(tau)
                tp[j] += h
                rp = residual(tp)
                for i in range(n):
                    jac[i, j] = (rp[i] - r[i]) / h
            step = mp.lu_solve(jac, r)
            tau = [tau[i] - step[i] for i in range(n)]
            if max(abs(s) for s in step) < mp.mpf(10) ** (-(dps - 10)):
                break
        a = means(tau)
        res = max(abs(x) for x in residual(tau))
        return tau, a, res


@lru_cache(maxsize=None)
def lloyd_max(m=8, levels=N_LEVELS):
    """Correctly rounded float64 (tau[1..L-1], a[0..L-1]) for subspace dimension m.

    Returns (tau, a, residual) where residual is the mpmath fixed-point
    residual (|tau - midpoint(a(tau))|_inf) before rounding.
    """
    tau64, _, _ = lloyd_max_fp64(m, levels)
    tau_mp, a_mp, res = _mp_fixed_point(tau64, m)
    tau = np.array([float(t) for t in tau_mp], dtype=np.float64)
    a = np.array([float(x) for x in a_mp], dtype=np.float64)
    tau.setflags(write=False)
    a.setflags(write=False)
    return tau, a, float(res)


def quantizer_mse(tau, a, m):
    """E[(X - Q(X))^2] of the quantizer (tau, a) under the Beta-derived density."""
    from scipy.integrate import quad

    edges = np.concatenate(([0.0], tau, [1.0]))
    total = 0.0
    for t in range(len(a)):
        val, _ = quad(lambda x, t=t: (x - a[t]) ** 2 * magnitude_pdf(x, m),
                      edges[t], edges[t + 1], epsabs=1e-14, epsrel=1e-12)
        total += val
    return total

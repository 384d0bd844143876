"""The coefficient map in the form the flush kernel builds it, checked
against the oracle.

The oracle builds the state-dependent map literally in the basis-aligned
coordinates of the appendix "Low-Rank-Plus-Diagonal Approximation for the
Coefficient Map" (an orthogonal completion R of Omega, the full K x K metric,
a direct G x G solve).  The kernel never forms R or the K x K metric: it
works from the sketch U and the product U_p^T X of the first p sketch columns
with the state, uses a Cholesky factor of the p x p pivot Gram matrix in place
of Gram-Schmidt, and Woodbury's identity (Step 4 of that appendix) for the
G x G inverse, which gives C = F1 M + F2 Omega^T.  With w = d / (d + lambda)
the second factor is F2 = Diag(w) - F1 L_G^T Diag(w), so the kernel forms
C = F1 M' + Diag(w) Omega^T with the p x K correction
M' = M - L_G^T Diag(w) Omega^T.  This numpy model of both forms must give the
oracle's map.
"""
import numpy as np
import pytest
def factored_coef_map(X, Om, p, lam):
    """The map as the GPU flush builds it, from X = S^T [V][K], Omega [K][G]
    and the sketch U = X Omega: Cholesky of the pivot Gram U_p^T U_p = R^T R,
    L_G = U^T U_p R^{-1} / sqrt(mu), M = R^{-T} U_p^T X / sqrt(mu),
    d = max(diag(U^T U)/mu - |L_G|^2, 0), Woodbury for (L_G L_G^T + D)^{-1}
    with D = d + lambda, F1 = A^{-1} L_G, F2 = A^{-1} Diag(d); C = F1 M + F2 Omega^T."""
    U = X @ Om
    mu = (X ** 2).sum() / X.shape[1] or 1.0
    Up = U[:, :p]
    R = np.linalg.cholesky(Up.T @ Up).T  # upper: Up^T Up = R^T R
    Rinv = np.linalg.inv(R)
    LG = (U.T @ Up) @ Rinv / np.sqrt(mu)
    M = Rinv.T @ (Up.T @ X) / np.sqrt(mu)
    d = np.maximum((U ** 2).sum(0) / mu - (LG ** 2).sum(1), 0.0)
    Dinv = 1.0 / (d + lam)
    T = np.eye(p) + LG.T @ (Dinv[:, None] * LG)
    Ainv = np.diag(Dinv) - (Dinv[:, None] * LG) @ np.linalg.solve(T, LG.T * Dinv[None, :])
    F1 = Ainv @ LG
    F2 = Ainv * d[None, :]
    return F1 @ M + F2 @ Om.T, (M, F1, F2, LG, d * Dinv)


def kernel_form(X, Om, p, lam):
    """C = F1 M' + Diag(w) Omega^T with M' = M - L_G^T Diag(w) Omega^T, the
    form the flush forms, from the same factors."""
    _, (M, F1, F2, LG, w) = factored_coef_map(X, Om, p, lam)
    assert np.allclose(F2, np.diag(w) - F1 @ LG.T * w[None, :], rtol=1e-10, atol=1e-12)
    Mp = M - (LG * w[:, None]).T @ Om.T
    return F1 @ Mp + w[:, None] * Om.T


@pytest.mark.parametrize("K,V,G,p", [(8, 6, 5, 2), (16, 12, 8, 4), (12, 16, 4, 4)])
def test_factored_coef_map_equals_the_oracle(K, V, G, p):
    """F1 M + F2 Omega^T (Woodbury, no rotated coordinates) is the oracle's
    direct solve in the basis-aligned coordinates of the appendix."""
    from test_oracle_pins import coef_map_of, heads_omega

    rng = np.random.default_rng(K + V + G + p)
    S = rng.standard_normal((3, V, K)).astype(np.float32)
    om = heads_omega(1, K, G, seed=p)[0]
    want = coef_map_of(S, om, p, 0.1)
    for i in range(3):
        X, Om = S[i].astype(np.float64), om[0].astype(np.float64)
        got, _ = factored_coef_map(X, Om, p, 0.1)
        assert np.allclose(got, want[i], rtol=1e-6, atol=1e-7)
        assert np.allclose(kernel_form(X, Om, p, 0.1), want[i], rtol=1e-6, atol=1e-7)

"""The algebra the GPU kernels implement, checked against explicit products.

The kernels never form M_{1:t}; they use the WY form of Appendix "WY-Based
Effective-Query and Coefficient Computation" with window-local cumulative log
decays g_t (so decay ratios are exp(g_t - g_s) <= 1, never a division), plus
pseudo-values u_s that carry the erase into the buffer output, and a rank-W
flush.  This numpy model of those identities is compared with explicitly
multiplied K x K transition matrices; it imports neither the oracle nor the
kernels.
"""
import numpy as np
import pytest


def make(kind, K=6, V=5, W=6, G=3, seed=0):
    rng = np.random.default_rng(seed)
    k = rng.standard_normal((W, K)) * 0.5
    q = rng.standard_normal((W, K))
    v = rng.standard_normal((W, V))
    beta = rng.uniform(0.1, 0.9, W)
    logd = rng.uniform(-0.6, 0.0, (W, K) if kind == "kda" else (W, 1)) * np.ones((W, K))
    S0 = rng.standard_normal((K, V))
    C = np.linalg.qr(rng.standard_normal((K, G)))[0].T
    return k, q, v, beta, logd, S0, C


def M(kind, k, beta, logd):
    D = np.diag(np.exp(logd))
    return D if kind == "mamba2" else (np.eye(len(k)) - beta * np.outer(k, k)) @ D


@pytest.mark.parametrize("kind", ["mamba2", "gdn", "kda"])
def test_append_and_read_identities(kind):
    k, q, v, beta, logd, S0, C = make(kind)
    W, K = k.shape
    erase = kind != "mamba2"
    g = np.cumsum(logd, axis=0)                      # window-local cumulative log decay
    u, f, pis = [], [], []
    Mprod = np.eye(K)
    Z = np.zeros((K, v.shape[1]))                    # state the buffer alone would produce
    for t in range(W):
        Mt = M(kind, k[t], beta[t], logd[t])
        Mprod = Mt @ Mprod
        Z = Mt @ Z + beta[t] * np.outer(k[t], v[t])
        # append: b_{t,j} = <exp(g_t - g_j) * k_j, k_t>, then u_t, f_t (and pi_t)
        b = np.array([np.sum(np.exp(g[t] - g[j]) * k[j] * k[t]) for j in range(t)])
        if erase:
            u.append(beta[t] * (v[t] - sum(b[j] * u[j] for j in range(t))))
            f.append(beta[t] * (C @ (np.exp(g[t]) * k[t]) - sum(b[j] * f[j] for j in range(t))))
            pis.append(beta[t] * (np.exp(g[t]) * k[t] - sum(b[j] * pis[j] for j in range(t))))
        else:
            u.append(beta[t] * v[t])
        # read: a_{t,s} = <exp(g_t - g_s) * k_s, q_t>
        a = np.array([np.sum(np.exp(g[t] - g[s]) * k[s] * q[t]) for s in range(t + 1)])
        qt_eff = Mprod.T @ q[t]
        if erase:
            c = C @ (np.exp(g[t]) * q[t]) - sum(a[s] * f[s] for s in range(t + 1))
            q_wy = np.exp(g[t]) * q[t] - sum(a[s] * pis[s] for s in range(t + 1))
            np.testing.assert_allclose(q_wy, qt_eff, atol=1e-13)          # WY effective query
            np.testing.assert_allclose(Mprod, np.diag(np.exp(g[t])) - sum(
                np.outer(np.exp(g[t] - g[s]) * k[s], pis[s]) for s in range(t + 1)), atol=1e-13)
        else:
            c = np.exp(g[t][0]) * (C @ q[t])                               # scalar decay
        np.testing.assert_allclose(c, C @ qt_eff, atol=1e-13)              # projected factors are exact
        o_buf = sum(a[s] * u[s] for s in range(t + 1))
        np.testing.assert_allclose(o_buf, Z.T @ q[t], atol=1e-13)          # pseudo-value buffer output


@pytest.mark.parametrize("kind", ["mamba2", "gdn", "kda"])
@pytest.mark.parametrize("W", [1, 2, 6])
def test_rank_w_flush(kind, W):
    k, q, v, beta, logd, S0, C = make(kind, W=W, seed=W)
    K = k.shape[1]
    erase = kind != "mamba2"
    S = S0.copy()
    for t in range(W):
        S = M(kind, k[t], beta[t], logd[t]) @ S + beta[t] * np.outer(k[t], v[t])
    g = np.cumsum(logd, axis=0)
    u, pis = [], []
    for t in range(W):
        b = [np.sum(np.exp(g[t] - g[j]) * k[j] * k[t]) for j in range(t)]
        if erase:
            u.append(beta[t] * (v[t] - sum(b[j] * u[j] for j in range(t))))
            pis.append(beta[t] * (np.exp(g[t]) * k[t] - sum(b[j] * pis[j] for j in range(t))))
        else:
            u.append(beta[t] * v[t])
            pis.append(np.zeros(K))
    # in [V][K] storage: X_W = X_0 diag(e^{g_W}) + sum_s w_s l_s^T with w_s = u_s - X_0 pi_s
    X0 = S0.T
    L = np.stack([np.exp(g[-1] - g[s]) * k[s] for s in range(W)])        # W x K
    Wv = np.stack([u[s] - X0 @ pis[s] for s in range(W)], axis=1)        # V x W
    XW = X0 * np.exp(g[-1])[None, :] + Wv @ L
    np.testing.assert_allclose(XW, S.T, atol=1e-12)



@pytest.mark.parametrize("kind,seed", [("gdn", 0), ("kda", 1), ("gdn", 2)])
def test_inverse_rows_replace_the_recursions(kind, seed):
    """The ring stores rows of T^{-1}, T = I + Diag(beta) B with the couplings
    B_{s,j} = b_{s,j} (j < s) of eq. wy.  Each read computes gamma = T^{-T} b_t
    and stores row t as -beta_t gamma; the stored rows must be T^{-1} (an
    explicit inverse), and products with them must give the pseudo-values,
    the erase factors and the buffer term that the recursions define."""
    k, q, v, beta, logd, S0, C = make(kind, K=7, V=5, W=9, seed=seed)
    W, K = k.shape
    g = np.cumsum(logd, axis=0)
    Bc = np.zeros((W, W))
    for t in range(W):
        for j in range(t):
            Bc[t, j] = np.sum(np.exp(g[t] - g[j]) * k[j] * k[t])
    T = np.eye(W) + np.diag(beta) @ Bc
    Tinv = np.zeros((W, W))                       # rows as the reads append them
    for t in range(W):
        Tinv[t, t] = 1.0
        if t:
            gamma = Tinv[:t, :t].T @ Bc[t, :t]        # T_{<t}^{-T} b_t
            Tinv[t, :t] = -beta[t] * gamma
    np.testing.assert_allclose(Tinv, np.linalg.inv(T), atol=1e-12)
    # recursions of eq. wy (pi) and of the pseudo-values (u)
    u, pis = [], []
    for t in range(W):
        u.append(beta[t] * (v[t] - sum(Bc[t, j] * u[j] for j in range(t))))
        pis.append(beta[t] * (np.exp(g[t]) * k[t] - sum(Bc[t, j] * pis[j] for j in range(t))))
    np.testing.assert_allclose(Tinv @ (beta[:, None] * v), np.array(u), atol=1e-12)
    np.testing.assert_allclose(Tinv @ (beta[:, None] * np.exp(g) * k), np.array(pis), atol=1e-12)
    # a read at slot n: sum_s a_s u_s = sum_j alpha_j beta_j v_j with alpha = T^{-T} a
    for n in range(1, W):
        a = np.array([np.sum(np.exp(g[n] - g[s]) * k[s] * q[n]) for s in range(n)])
        alpha = Tinv[:n, :n].T @ a
        np.testing.assert_allclose(sum(a[s] * u[s] for s in range(n)),
                                   (alpha * beta[:n]) @ v[:n], atol=1e-12)


@pytest.mark.parametrize("kind,W,c", [("gdn", 9, 4), ("kda", 9, 4), ("gdn", 7, 3), ("kda", 8, 8), ("kda", 5, 2)])
def test_chunked_flush_from_stored_rows(kind, W, c):
    """A window flushed as chunks of c slots, each from the state the previous
    chunk left: T is unit lower triangular, so the rows of the window's T^{-1}
    that couple a chunk's slots among themselves (its diagonal block) are the
    inverse of the T that chunk alone would build (decays counted from the
    chunk's first slot), and each chunk is then a rank-c flush of its own.
    The chunked flush must reproduce the explicitly multiplied transitions."""
    k, q, v, beta, logd, S0, C = make(kind, K=7, V=5, W=W, seed=W + c)
    K = k.shape[1]
    S = S0.copy()
    for t in range(W):
        S = M(kind, k[t], beta[t], logd[t]) @ S + beta[t] * np.outer(k[t], v[t])
    g = np.cumsum(logd, axis=0)
    Bc = np.zeros((W, W))
    for t in range(W):
        for j in range(t):
            Bc[t, j] = np.sum(np.exp(g[t] - g[j]) * k[j] * k[t])
    Tinv = np.linalg.inv(np.eye(W) + np.diag(beta) @ Bc)     # the stored rows, whole window
    X = S0.T
    for s0 in range(0, W, c):
        sl = slice(s0, min(s0 + c, W))
        n = sl.stop - s0
        gc = np.cumsum(logd[sl], axis=0)                     # decays from the chunk's first slot
        Bl = np.zeros((n, n))
        for t in range(n):
            for j in range(t):
                Bl[t, j] = np.sum(np.exp(gc[t] - gc[j]) * k[s0 + j] * k[s0 + t])
        Ti = Tinv[sl, sl]
        np.testing.assert_allclose(Ti, np.linalg.inv(np.eye(n) + np.diag(beta[sl]) @ Bl), atol=1e-12)
        u = Ti @ (beta[sl, None] * v[sl])
        pis = Ti @ (beta[sl, None] * np.exp(gc) * k[sl])
        L = np.stack([np.exp(gc[-1] - gc[s]) * k[s0 + s] for s in range(n)])
        Wv = (u - (X @ pis.T).T).T                           # V x n: w_s = u_s - X pi_s
        X = X * np.exp(gc[-1])[None, :] + Wv @ L
    np.testing.assert_allclose(X, S.T, atol=1e-12)

"""Pins for the CPU oracle: it is checked against things other than itself.

Each test states what the paper or the mathematics fixes.  Together they are
chosen so that a plausible slip in the oracle (erase before decay, a dropped
self term, a transposed operand, a missing flush token, the sketch taken on
the wrong side of S) fails at least one of them.
"""
import numpy as np
import pytest

import oracle

KINDS = ["mamba2", "gdn", "kda"]


def tiny_inputs(kind, n=3, K=5, V=4, T=9, seed=0, unit_keys=False, beta_one=False, strong_decay=False):
    rng = np.random.default_rng(seed)
    S0 = rng.standard_normal((n, V, K)).astype(np.float32)
    q = rng.standard_normal((T, n, K)).astype(np.float32)
    k = rng.standard_normal((T, n, K)).astype(np.float32)
    if unit_keys:
        k = (k / np.linalg.norm(k, axis=-1, keepdims=True)).astype(np.float32)
    else:
        k = (0.6 * k).astype(np.float32)
    v = rng.standard_normal((T, n, V)).astype(np.float32)
    beta = np.ones((T, n), np.float32) if beta_one else rng.uniform(0.1, 0.9, (T, n)).astype(np.float32)
    lo = -1.5 if strong_decay else -0.4
    shape = (T, n, K) if kind == "kda" else (T, n)
    logd = rng.uniform(lo, 0.0, shape).astype(np.float32)
    return S0, q, k, v, beta, logd


def explicit_M(kind, k, beta, logd):
    """M_t as an explicit K x K matrix (Sec. 3.2): D_t, or (I - beta k k^T) D_t."""
    K = k.shape[0]
    d = np.exp(logd.astype(np.float64)) * np.ones(K)
    D = np.diag(d)
    if kind == "mamba2":
        return D
    kk = k.astype(np.float64)
    return (np.eye(K) - float(beta) * np.outer(kk, kk)) @ D


def brute_force_outputs(kind, S0, q, k, v, beta, logd):
    """o_n = S_n^T q_n with S_n = M_{1:n} S_0 + sum_m beta_m M_{m+1:n} k_m v_m^T,
    every ordered product formed explicitly (second form of eq. transition-update)."""
    T, n, K = q.shape
    V = v.shape[2]
    out = np.zeros((T, n, V))
    for i in range(n):
        Ms = [explicit_M(kind, k[t, i], beta[t, i], logd[t, i]) for t in range(T)]
        S_init = S0[i].astype(np.float64).T  # K x V
        for t in range(T):
            def prod(a, b):  # M_{a:b} = M_b ... M_a  (1-based, inclusive); identity when a > b
                P = np.eye(K)
                for j in range(a, b + 1):
                    P = Ms[j - 1] @ P
                return P
            S = prod(1, t + 1) @ S_init
            for m in range(1, t + 2):
                S = S + float(beta[m - 1, i]) * np.outer(prod(m + 1, t + 1) @ k[m - 1, i].astype(np.float64),
                                                         v[m - 1, i].astype(np.float64))
            out[t, i] = S.T @ q[t, i].astype(np.float64)
    return out


@pytest.mark.parametrize("kind", KINDS)
def test_recurrence_equals_explicit_products(kind):
    """O1 against the closed form with explicitly multiplied transition matrices."""
    S0, q, k, v, beta, logd = tiny_inputs(kind, seed=1)
    o, _ = oracle.recurrence(kind, S0, q, k, v, beta, logd)
    ref = brute_force_outputs(kind, S0, q, k, v, beta, logd)
    np.testing.assert_allclose(o, ref, rtol=1e-11, atol=1e-11)


def test_scalar_decay_is_decay_masked_attention():
    """Mamba-2 form (M_t = alpha_t I): the read is causal attention with a
    multiplicative decay mask plus the decayed initial-state read."""
    S0, q, k, v, beta, logd = tiny_inputs("mamba2", n=2, K=6, V=3, T=11, seed=2)
    o, _ = oracle.recurrence("mamba2", S0, q, k, v, beta, logd)
    T = q.shape[0]
    for i in range(S0.shape[0]):
        L = np.cumsum(logd[:, i].astype(np.float64))          # log prod_{j<=n} alpha_j
        mask = np.tril(np.exp(L[:, None] - L[None, :]))        # prod_{m<j<=n} alpha_j
        Q = q[:, i].astype(np.float64)
        Kx = k[:, i].astype(np.float64)
        Vx = v[:, i].astype(np.float64)
        att = (Q @ Kx.T) * mask * beta[:, i].astype(np.float64)[None, :]
        ref = att @ Vx + np.exp(L)[:, None] * (Q @ S0[i].astype(np.float64).T)
        np.testing.assert_allclose(o[:, i], ref, rtol=1e-11, atol=1e-11)
    assert T == 11


@pytest.mark.parametrize("kind", ["gdn", "kda"])
@pytest.mark.parametrize("beta_one", [False, True])
def test_delta_rule_retrieval(kind, beta_one):
    """The delta-rule write of token t leaves
    S_t^T k_t = (1 - beta_t |k_t|^2) (D_t S_{t-1})^T k_t + beta_t |k_t|^2 v_t,
    so with unit keys and beta_t = 1 the state returns v_t at key k_t.  This
    holds only if the erase acts after the decay (M_t = (I - beta k k^T) D_t)."""
    K, V, T = 6, 5, 7
    S0, q, k, v, beta, logd = tiny_inputs(kind, n=2, K=K, V=V, T=T, seed=3 + beta_one, unit_keys=True,
                                          beta_one=beta_one, strong_decay=True)
    _, S_prev = oracle.recurrence(kind, S0, q[:T - 1], k[:T - 1], v[:T - 1], beta[:T - 1], logd[:T - 1])
    _, S_last = oracle.recurrence(kind, S0, q, k, v, beta, logd)
    for i in range(2):
        kt = k[T - 1, i].astype(np.float64)
        nk = float(kt @ kt)
        b = float(beta[T - 1, i])
        d = np.exp(logd[T - 1, i].astype(np.float64)) * np.ones(K)
        lhs = S_last[i] @ kt                                     # S_t^T k_t  (storage is [V][K])
        rhs = (1 - b * nk) * (S_prev[i] @ (d * kt)) + b * nk * v[T - 1, i].astype(np.float64)
        np.testing.assert_allclose(lhs, rhs, rtol=1e-12, atol=1e-12)
        if beta_one:
            np.testing.assert_allclose(lhs, v[T - 1, i], rtol=0, atol=1e-6)


def orthonormal(K, G, seed):
    Q, R = np.linalg.qr(np.random.default_rng(seed).standard_normal((K, G)))
    return (Q * np.sign(np.diag(R))[None, :]).astype(np.float32)


def heads_omega(H, K, G, seed):
    om = np.stack([orthonormal(K, G, seed + h) for h in range(H)])
    return om, np.ascontiguousarray(om.transpose(0, 2, 1))


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("W", [3, 4])
def test_flush_equals_recurrence(kind, W):
    """Algorithm 1's flush replays the buffer exactly: after every W-th token
    the state and the output equal the plain recurrence."""
    T = 3 * W
    S0, q, k, v, beta, logd = tiny_inputs(kind, T=T, seed=5)
    om, C = heads_omega(2, 5, 2, 10)
    heads = np.array([0, 1, 0], np.int32)
    o_ex, S_ex = oracle.recurrence(kind, S0, q, k, v, beta, logd)
    r = oracle.sketchssm(kind, W, heads, om, C, S0, q, k, v, beta, logd)
    np.testing.assert_allclose(r.S_final, S_ex, rtol=1e-12, atol=1e-12)
    flush = np.arange(W - 1, T, W)
    np.testing.assert_allclose(r.o[flush], o_ex[flush], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("kind", KINDS)
def test_state_buffer_decomposition(kind):
    """Eq. m-reads: S_t^T q_t = S_0^T q~_t + o^buffer_t at every step."""
    W, T = 5, 12
    S0, q, k, v, beta, logd = tiny_inputs(kind, T=T, seed=6)
    om, C = heads_omega(1, 5, 2, 11)
    r = oracle.sketchssm(kind, W, np.zeros(3, np.int32), om, C, S0, q, k, v, beta, logd)
    o_ex, _ = oracle.recurrence(kind, S0, q, k, v, beta, logd)
    np.testing.assert_allclose(r.o_exact_windowed, o_ex, rtol=1e-11, atol=1e-11)
    # the buffer term is nonzero between flushes and the state term is not the whole output
    assert np.abs(r.o_buf).max() > 1e-3


@pytest.mark.parametrize("kind", KINDS)
def test_full_rank_identity_sketch_is_exact(kind):
    """r = K with Omega = I (so C = I): the sketch read is the exact state read."""
    K, V, W, T = 5, 3, 4, 13
    S0, q, k, v, beta, logd = tiny_inputs(kind, K=K, V=V, T=T, seed=7)
    om = np.eye(K, dtype=np.float32)[None]
    r = oracle.sketchssm(kind, W, np.zeros(3, np.int32), om, om.copy(), S0, q, k, v, beta, logd)
    o_ex, S_ex = oracle.recurrence(kind, S0, q, k, v, beta, logd)
    np.testing.assert_allclose(r.o, o_ex, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(r.U_final, r.S_final, rtol=1e-12, atol=1e-12)  # U = S^T I, storage [V][K]


@pytest.mark.parametrize("kind", KINDS)
def test_window_one_is_plain_recurrence(kind):
    """W = 1: every token is a flush, the sketch is never read."""
    S0, q, k, v, beta, logd = tiny_inputs(kind, T=6, seed=8)
    om, C = heads_omega(1, 5, 2, 12)
    r = oracle.sketchssm(kind, 1, np.zeros(3, np.int32), om, C, S0, q, k, v, beta, logd)
    o_ex, S_ex = oracle.recurrence(kind, S0, q, k, v, beta, logd)
    np.testing.assert_allclose(r.o, o_ex, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(r.S_final, S_ex, rtol=1e-12, atol=1e-12)


def test_sketch_projection_behaviour():
    """Sec. 3.3 with C = Omega^T and orthonormal Omega (K > G): a Mamba-2 query in
    span(Omega) is read exactly, a query orthogonal to it reads zero state."""
    K, V, G, W, T, n = 7, 4, 3, 6, 5, 2
    S0, q, k, v, beta, logd = tiny_inputs("mamba2", n=n, K=K, V=V, T=T, seed=9)
    om = orthonormal(K, G, 13)[None]
    C = np.ascontiguousarray(om.transpose(0, 2, 1))
    rng = np.random.default_rng(14)
    q_in = np.einsum("kg,tng->tnk", om[0].astype(np.float64), rng.standard_normal((T, n, G))).astype(np.float32)
    r = oracle.sketchssm("mamba2", W, np.zeros(n, np.int32), om, C, S0, q_in, k, v, beta, logd)
    np.testing.assert_allclose(r.o_state_hat, r.o_state, rtol=1e-6, atol=1e-6)  # limited by fp32 rounding of q
    P = np.eye(K) - om[0].astype(np.float64) @ om[0].astype(np.float64).T
    q_perp = np.einsum("kj,tnj->tnk", P, rng.standard_normal((T, n, K))).astype(np.float32)
    r = oracle.sketchssm("mamba2", W, np.zeros(n, np.int32), om, C, S0, q_perp, k, v, beta, logd)
    assert np.abs(r.o_state_hat).max() < 1e-6 * max(1.0, np.abs(r.o_state).max())
    assert np.abs(r.o_state).max() > 1e-2


@pytest.mark.parametrize("kind", KINDS)
def test_term_isolation_and_linearity(kind):
    """v = 0 removes the buffer term; S0 = 0 removes the state term in the first
    window; outputs are jointly linear in (S0, v) for fixed keys, queries, gates."""
    W, T = 4, 10
    S0, q, k, v, beta, logd = tiny_inputs(kind, T=T, seed=15)
    om, C = heads_omega(1, 5, 2, 16)
    hz = np.zeros(3, np.int32)
    r0 = oracle.sketchssm(kind, W, hz, om, C, S0, q, k, np.zeros_like(v), beta, logd)
    assert np.abs(r0.o_buf).max() == 0.0
    nf = [t for t in range(T) if (t + 1) % W != 0]
    np.testing.assert_allclose(r0.o[nf], r0.o_state_hat[nf], rtol=0, atol=0)
    rz = oracle.sketchssm(kind, W, hz, om, C, np.zeros_like(S0), q, k, v, beta, logd)
    assert np.abs(rz.o_state_hat[:W - 1]).max() == 0.0 and np.abs(rz.o_state[:W - 1]).max() == 0.0
    S1, _, _, v1, _, _ = tiny_inputs(kind, T=T, seed=17)
    a, b = 0.7, -1.3
    ra = oracle.sketchssm(kind, W, hz, om, C, S0, q, k, v, beta, logd)
    rb = oracle.sketchssm(kind, W, hz, om, C, S1, q, k, v1, beta, logd)
    rab = oracle.sketchssm(kind, W, hz, om, C, a * S0 + b * S1, q, k, a * v + b * v1, beta, logd)
    np.testing.assert_allclose(rab.o, a * ra.o + b * rb.o, rtol=1e-5, atol=1e-5)  # fp32 rounding of a*S0+b*S1


def test_storage_rounding_only_changes_state_at_fp32_level():
    """round_storage mirrors fp32 state/sketch storage; the result moves by at most fp32 rounding."""
    S0, q, k, v, beta, logd = tiny_inputs("gdn", T=12, seed=18)
    om, C = heads_omega(1, 5, 2, 19)
    hz = np.zeros(3, np.int32)
    r = oracle.sketchssm("gdn", 4, hz, om, C, S0, q, k, v, beta, logd)
    rr = oracle.sketchssm("gdn", 4, hz, om, C, S0, q, k, v, beta, logd, round_storage=True)
    rel = np.linalg.norm(rr.o - r.o) / np.linalg.norm(r.o)
    assert 0 < rel < 1e-6
    np.testing.assert_array_equal(rr.S_final, rr.S_final.astype(np.float32).astype(np.float64))


def test_bf16_sketch_storage_is_round_to_nearest_even():
    """The paper stores the sketch in BF16.  With that storage the oracle's
    sketch after a flush is torch's bfloat16 rounding (nearest, ties to even)
    of the fp32 sketch, and the flush leaves the state untouched by it."""
    import torch

    S0, q, k, v, beta, logd = tiny_inputs("gdn", n=3, K=8, V=6, T=8, seed=11)
    heads = np.zeros(3, np.int32)
    om, C = heads_omega(1, 8, 4, seed=5)
    a = oracle.sketchssm("gdn", 4, heads, om, C, S0, q, k, v, beta, logd, round_storage=True)
    b = oracle.sketchssm("gdn", 4, heads, om, C, S0, q, k, v, beta, logd, round_storage=True, sketch_bf16=True)
    want = torch.from_numpy(a.U_final.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(b.U_final, want)
    assert not np.array_equal(a.U_final, b.U_final)
    assert np.array_equal(a.S_final, b.S_final)


def test_bf16_sketch_is_the_one_read():
    """r = K, Omega = C = I, one token in the window (scalar decay): the
    sketch read is U (alpha_1 q) with U the bf16-rounded S_0^T (Sec. 3.3 read
    with the paper's storage)."""
    import torch

    S0, q, k, v, beta, logd = tiny_inputs("mamba2", n=2, K=6, V=5, T=1, seed=3)
    eye = np.broadcast_to(np.eye(6, dtype=np.float32), (1, 6, 6)).copy()
    r = oracle.sketchssm("mamba2", 4, np.zeros(2, np.int32), eye, eye, S0, q, k, v, beta, logd,
                         round_storage=True, sketch_bf16=True)
    U = torch.from_numpy(S0.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()  # [n][V][K]
    qt = np.exp(logd[0].astype(np.float64))[:, None] * q[0].astype(np.float64)
    want = np.einsum("nvk,nk->nv", U, qt)
    assert np.allclose(r.o_state_hat[0], want, rtol=1e-12, atol=1e-12)


# --- the state-dependent coefficient map (Sec. 4.1 eq. m-coeff; low-rank-plus-diagonal metric) ------
def coef_map_of(S_vk, om, pivots, ridge, lib=None):
    """The oracle's coefficient map for the states S_vk [n][V][K] (no flush:
    the map is the one built from the initial state)."""
    n, V, K = S_vk.shape
    G = om.shape[2]
    rng = np.random.default_rng(0)
    q = rng.standard_normal((1, n, K)).astype(np.float32)
    z = np.zeros((1, n, K), np.float32)
    r = oracle.sketchssm("mamba2", 4, np.zeros(n, np.int32), om, np.ascontiguousarray(om.transpose(0, 2, 1)),
                         S_vk.astype(np.float32), q, z, np.zeros((1, n, V), np.float32), np.zeros((1, n), np.float32),
                         np.zeros((1, n), np.float32), pivots=pivots, ridge=ridge, lib=lib)
    return r.coef_final


def low_rank_state(n, V, K, rank, seed):
    rng = np.random.default_rng(seed)
    return np.einsum("nvr,nkr->nvk", rng.standard_normal((n, V, rank)), rng.standard_normal((n, K, rank))).astype(np.float32)


def exact_ridge_map(S_vk, om, ridge):
    """(U^T U / mu + lambda I)^{-1} U^T S^T / mu with U = S^T Omega: the ridge
    solution under the exact state metric, solved by numpy."""
    X = S_vk.astype(np.float64)
    Om = om[0].astype(np.float64)
    out = []
    for Xi in X:
        U = Xi @ Om
        mu = (Xi ** 2).sum() / Xi.shape[1]
        out.append(np.linalg.solve(U.T @ U / mu + ridge * np.eye(U.shape[1]), U.T @ Xi / mu))
    return np.stack(out)


@pytest.mark.parametrize("pivots,rank", [(2, 2), (4, 3), (4, 4)])
def test_coef_map_is_the_exact_ridge_map_when_pivots_span_the_state(pivots, rank):
    """When S^T lies in the span of the first p sketch columns, the pivot
    metric reproduces the state metric (L L^T = H, d = 0), so the map is the
    ridge solution of eq. m-coeff under the exact metric."""
    K, V, G = 8, 6, 5
    S = low_rank_state(3, V, K, rank, seed=rank)
    om = heads_omega(1, K, G, seed=21)[0]
    got = coef_map_of(S, om, pivots, 0.1)
    # Omega is orthonormal to fp32 precision only; the oracle's basis completion
    # re-orthonormalises it, which moves the map at the 1e-8 level
    assert np.allclose(got, exact_ridge_map(S, om, 0.1), rtol=1e-6, atol=1e-7)


def test_coef_map_is_invariant_to_value_rotation_and_state_scale():
    """The metric H = S' S'^T / mu sees S only through S S^T and its norm, and
    Q spans the same value subspace after a rotation: the map must not move."""
    K, V, G = 7, 5, 4
    rng = np.random.default_rng(8)
    S = rng.standard_normal((2, V, K)).astype(np.float32)
    O, _ = np.linalg.qr(rng.standard_normal((V, V)))
    om = heads_omega(1, K, G, seed=3)[0]
    base = coef_map_of(S, om, 2, 0.1)
    rot = coef_map_of(np.einsum("uv,nvk->nuk", O, S.astype(np.float64)).astype(np.float32), om, 2, 0.1)
    scaled = coef_map_of((S * 8.0).astype(np.float32), om, 2, 0.1)
    assert np.allclose(rot, base, rtol=1e-5, atol=1e-6)   # the rotated state is rounded to fp32
    assert np.allclose(scaled, base, rtol=1e-12, atol=1e-12)


def test_coef_map_with_a_full_basis_tends_to_the_identity():
    """Omega = I (G = K): the ridge solve is (Hhat + lambda I)^{-1} Hhat, the
    identity as lambda -> 0, so the sketch read becomes exact."""
    K, V = 5, 7
    rng = np.random.default_rng(4)
    S = rng.standard_normal((2, V, K)).astype(np.float32)
    eye = np.eye(K, dtype=np.float32)[None]
    got = coef_map_of(S, eye, 3, 1e-9)
    assert np.allclose(got, np.broadcast_to(np.eye(K), got.shape), atol=1e-6)


def test_coef_map_of_a_zero_state_is_zero():
    """A zero state: mu = 1, no pivot columns, H = 0, so c = 0."""
    om = heads_omega(1, 6, 3, seed=2)[0]
    assert np.array_equal(coef_map_of(np.zeros((2, 4, 6), np.float32), om, 4, 0.1), np.zeros((2, 3, 6)))


def test_coef_map_pivots_are_the_leading_sketch_columns():
    """Q spans the first p sketch columns: reordering the other columns of
    Omega (or the first p among themselves) reorders the rows of the map and
    changes nothing else."""
    K, V, G, p = 8, 6, 6, 2
    rng = np.random.default_rng(12)
    S = rng.standard_normal((2, V, K)).astype(np.float32)
    om = heads_omega(1, K, G, seed=7)[0]
    base = coef_map_of(S, om, p, 0.1)
    perm = np.array([1, 0, 5, 2, 4, 3])
    moved = coef_map_of(S, np.ascontiguousarray(om[:, :, perm]), p, 0.1)
    assert np.allclose(moved, base[:, perm], rtol=1e-6, atol=1e-7)  # Omega orthonormal to fp32 only
    other = np.array([2, 0, 1, 3, 4, 5])  # a different pair leads: the map must change
    assert not np.allclose(coef_map_of(S, np.ascontiguousarray(om[:, :, other]), p, 0.1), base[:, other], atol=1e-6)


# --- the paper's coefficient-space forms and BF16 storage of f and the map -----------------------------
@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("pivots", [0, 4, oracle.EXACT])
def test_paper_path_equals_the_direct_forms(kind, pivots):
    """c_t through the projected erase factors (eq. app-projected-query with
    eq. wyread) equals C q~_t when nothing is rounded (App. C.2: the
    projected recursion is exact for a map that is fixed within the window)."""
    S0, q, k, v, beta, logd = tiny_inputs(kind, n=3, K=8, V=6, T=13, seed=21)
    heads = np.zeros(3, np.int32)
    om, C = heads_omega(1, 8, 5, seed=9)
    a = oracle.sketchssm(kind, 5, heads, om, C, S0, q, k, v, beta, logd, pivots=pivots, ridge=0.1)
    b = oracle.sketchssm(kind, 5, heads, om, C, S0, q, k, v, beta, logd, pivots=pivots, ridge=0.1, paper_path=True)
    np.testing.assert_allclose(b.o, a.o, rtol=1e-10, atol=1e-10 * np.abs(a.o).max())
    np.testing.assert_array_equal(b.coef_final, a.coef_final)
    np.testing.assert_array_equal(b.S_final, a.S_final)


def bf16_of(x):
    """torch's bfloat16 conversion (round to nearest, ties to even) of the fp32 value of x, as fp64."""
    import torch

    return torch.from_numpy(np.asarray(x, np.float64).astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("pivots", [4, oracle.EXACT])
def test_bf16_map_storage_is_round_to_nearest_even(kind, pivots, lib=None):
    """The paper stores the state-dependent map C (G x K per item) in BF16.
    The map is built from the fp32 state and its unrounded sketch, which bf16
    storage does not change (the flush replays raw inputs), so the stored map
    must be torch's bf16 rounding of the fp32-storage run's map, element for
    element: the dense matrix is rounded once, not factors of it."""
    S0, q, k, v, beta, logd = tiny_inputs(kind, n=3, K=8, V=6, T=12, seed=23)
    heads = np.zeros(3, np.int32)
    om, C = heads_omega(1, 8, 5, seed=12)
    a = oracle.sketchssm(kind, 5, heads, om, C, S0, q, k, v, beta, logd, pivots=pivots, round_storage=True, lib=lib)
    b = oracle.sketchssm(kind, 5, heads, om, C, S0, q, k, v, beta, logd, pivots=pivots, round_storage=True,
                         sketch_bf16=True, lib=lib)
    assert np.array_equal(b.S_final, a.S_final)
    assert np.array_equal(b.coef_final, bf16_of(a.coef_final))
    assert not np.array_equal(b.coef_final, a.coef_final)


@pytest.mark.parametrize("pivots", [4, oracle.EXACT])
def test_bf16_map_is_the_one_read(pivots, lib=None):
    """Scalar decay, tokens of the first window: the sketch read is
    U_bf16 (C_bf16 q~_t) with q~_t = (prod_{s<=t} alpha_s) q_t (Sec. 3.3,
    eq. m-coeff: c_t = C q~_t), with the stored (bf16) sketch and map."""
    S0, q, k, v, beta, logd = tiny_inputs("mamba2", n=2, K=8, V=6, T=4, seed=24)
    om, C = heads_omega(1, 8, 5, seed=13)
    r = oracle.sketchssm("mamba2", 6, np.zeros(2, np.int32), om, C, S0, q, k, v, beta, logd, pivots=pivots,
                         round_storage=True, sketch_bf16=True, lib=lib)
    qt = np.exp(np.cumsum(logd.astype(np.float64), axis=0))[:, :, None] * q.astype(np.float64)   # [T][n][K]
    want = np.einsum("nvg,ngk,tnk->tnv", r.U_final, r.coef_final, qt)
    assert np.allclose(r.o_state_hat, want, rtol=1e-12, atol=1e-12)
    assert np.array_equal(r.U_final, bf16_of(r.U_final)) and np.array_equal(r.coef_final, bf16_of(r.coef_final))


@pytest.mark.parametrize("kind", ["gdn", "kda"])
def test_bf16_f_is_rounded_when_stored_not_when_formed(kind, lib=None):
    """With S_0 = I (V = K) and Omega = C = I the sketch is exactly I in bf16,
    so the sketch read is c_t itself.  Through the projected erase factors
    (eqs. app-projected-query, wyread), c_t = C q~_t exactly when nothing is
    rounded.  Storing f_1 in bf16 (when token 1 is first read) and using the
    current f_t as formed moves c at token 1 by nothing, and at token 2 by
        c_2 - C q~_2 = -(a_{2,1} - a_{2,2} beta_2 b_{2,1}) (f^_1 - f_1),
    with f_1 = beta_1 C (d_[1] . k_1), f^_1 its bf16 rounding,
    a_{2,s} = <l_s(2), q_2>, b_{2,1} = <l_1(2), k_2>, l_s(t) = D_t..D_{s+1} k_s."""
    K = 6
    _, q, k, v, beta, logd = tiny_inputs(kind, n=2, K=K, V=K, T=2, seed=25)
    S0 = np.broadcast_to(np.eye(K, dtype=np.float32), (2, K, K)).copy()
    eye = np.eye(K, dtype=np.float32)[None]
    r = oracle.sketchssm(kind, 5, np.zeros(2, np.int32), eye, eye.copy(), S0, q, k, v, beta, logd,
                         round_storage=True, sketch_bf16=True, lib=lib)
    for i in range(2):
        M = [explicit_M(kind, k[t, i], beta[t, i], logd[t, i]) for t in range(2)]
        q1 = M[0].T @ q[0, i].astype(np.float64)
        q2 = M[0].T @ (M[1].T @ q[1, i].astype(np.float64))
        assert np.allclose(r.o_state_hat[0, i], q1, rtol=1e-13, atol=1e-13)
        d = [np.exp(logd[t, i].astype(np.float64)) * np.ones(K) for t in range(2)]
        k1, k2 = k[0, i].astype(np.float64), k[1, i].astype(np.float64)
        l1 = d[1] * k1                                  # l_1(2) = D_2 k_1
        a21, a22, b21 = l1 @ q[1, i], k2 @ q[1, i], l1 @ k2
        f1 = float(beta[0, i]) * d[0] * k1              # C = I, d_[1] = D_1
        want = -(a21 - a22 * float(beta[1, i]) * b21) * (bf16_of(f1) - f1)
        assert np.abs(want).max() > 1e-6                # f_1 is not representable in bf16 here
        assert np.allclose(r.o_state_hat[1, i] - q2, want, rtol=1e-9, atol=1e-13)


@pytest.mark.parametrize("rank_of_state", [None, 2])
def test_exact_map_is_the_closed_form(rank_of_state, lib=None):
    """The exact regularised map of eq. pivot-ridge, built literally with the
    dense metric H in the rotated coordinates, is (U^T U/mu + lambda I)^{-1}
    U^T S^T/mu: J^T H J = U^T U/mu and J^T H R = U^T S^T/mu because R^T R = I.
    Checked for full-rank and low-rank states."""
    K, V, G = 8, 6, 5
    if rank_of_state is None:
        S = np.random.default_rng(31).standard_normal((3, V, K)).astype(np.float32)
    else:
        S = low_rank_state(3, V, K, rank_of_state, seed=32)
    om = heads_omega(1, K, G, seed=33)[0]
    assert np.allclose(coef_map_of(S, om, oracle.EXACT, 0.1, lib=lib), exact_ridge_map(S, om, 0.1),
                       rtol=1e-6, atol=1e-7)
    if rank_of_state is None:  # the P = 4 metric is an approximation of H for a full-rank state
        assert not np.allclose(coef_map_of(S, om, 4, 0.1, lib=lib), exact_ridge_map(S, om, 0.1), atol=1e-3)

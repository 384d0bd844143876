"""Offline calibration (the package's `calibrate` module) against plain
definitions (`oracle.calibration`), closed forms and brute force, on the CPU.

Pins:
  - the sketching matrix attains the closed-form minimum of the offline loss
    (the discarded eigenvalues of C_z, App. A.1 eq. app-offline-solution),
    also with a singular E0, and no random or naive basis does better;
  - the offline map is the E0-weighted least-squares coefficient map;
  - the prefix-rank residuals of the QR formula (eq. alloc-qr) equal direct
    least squares for every rank, dependent sketch columns included, and the
    gradient-paired score equals its definition;
  - the Lagrangian allocation is feasible, its dual bound sits below the
    brute-force optimum and its certified gap covers the true gap; it is
    optimal on most tiny instances and its certified gap is small at model
    scale;
  - the layer driver's basis is E0-orthonormal, so every rank's offline map is
    a prefix of the stored map (what the kernels' per-head masking assumes);
  - G* as the allocation appendix defines it.
"""
import numpy as np
import pytest

from oracle import calibration as ref
from paper_2609_33051_amd import calibrate as cal


def samples(K=10, V=7, N=60, rank_S=None, seed=0):
    """States with a decaying spectrum (optionally of rank rank_S) and
    effective queries with a preferred subspace."""
    rng = np.random.default_rng(seed)
    r = K if rank_S is None else rank_S
    basis = np.linalg.qr(rng.standard_normal((K, K)))[0][:, :r]
    spec = 0.7 ** np.arange(r)
    X = np.stack([rng.standard_normal((V, r)) @ (spec[:, None] * basis.T) for _ in range(N)])  # S^T [V][K]
    mix = rng.standard_normal((K, K)) * (0.6 ** np.arange(K))[None, :]
    q = rng.standard_normal((N, K)) @ mix.T
    return X, q


@pytest.mark.parametrize("G,rank_S", [(1, None), (3, None), (5, None), (3, 6)])
def test_basis_attains_the_closed_form_loss(G, rank_S):
    X, q = samples(rank_S=rank_S, seed=G)
    b = cal.offline_basis(X, q, G)
    E0 = ref_metric = np.einsum("nvk,nvl->kl", X, X) / len(X)
    assert np.allclose(b.E0, ref_metric)
    loss = ref.offline_loss(b.omega, E0, q)
    assert loss == pytest.approx(b.loss, rel=1e-8, abs=1e-12)
    rng = np.random.default_rng(99)
    for _ in range(20):  # no other G-dimensional basis does better
        assert ref.offline_loss(rng.standard_normal((10, G)), E0, q) >= loss - 1e-10
    w, P = np.linalg.eigh(E0)
    assert ref.offline_loss(P[:, ::-1][:, :G], E0, q) >= loss - 1e-10   # leading directions of E0 alone
    w, P = np.linalg.eigh(q.T @ q)
    assert ref.offline_loss(P[:, ::-1][:, :G], E0, q) >= loss - 1e-10   # leading directions of the queries alone


def test_offline_map_is_the_weighted_least_squares_map():
    X, q = samples(seed=3)
    b = cal.offline_basis(X, q, 4)
    E_half = ref.sqrt_psd(b.E0)
    for qt in q[:10]:
        c = np.linalg.lstsq(E_half @ b.omega, E_half @ qt, rcond=None)[0]
        np.testing.assert_allclose(b.coef @ qt, c, rtol=1e-7, atol=1e-9)


def test_orthonormal_prefix_basis_keeps_every_prefix_span():
    X, q = samples(seed=4)
    om = cal.offline_basis(X, q, 5).omega
    om[:, 3] = om[:, 0] - 2 * om[:, 1]          # a dependent column
    Q = cal.orthonormal_prefix_basis(om)
    np.testing.assert_allclose(Q.T @ Q, np.eye(5), atol=1e-12)
    for g in range(1, 6):
        P = Q[:, :g] @ Q[:, :g].T
        np.testing.assert_allclose(P @ om[:, :g], om[:, :g], atol=1e-10)


@pytest.mark.parametrize("dependent", [False, True])
def test_rank_scores_equal_direct_least_squares(dependent):
    X, q = samples(N=25, seed=5)
    om = np.random.default_rng(6).standard_normal((10, 6))
    if dependent:
        om[:, 2] = om[:, 0] + om[:, 1]
    grads = np.random.default_rng(7).standard_normal((25, 7))
    eps, J = cal.rank_scores(X, q, om, grads)
    eps_r, J_r = ref.prefix_residuals(X, q, om, grads)
    np.testing.assert_allclose(eps, eps_r, rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(J, J_r, rtol=1e-9, atol=1e-11)
    assert np.all(np.diff(eps) <= 1e-12)          # a longer prefix never reconstructs worse


def tiny_instance(seed):
    rng = np.random.default_rng(seed)
    N, A, tau, full = 4, 5, 3.0, 20.0
    # curves that need not have diminishing returns
    S = np.sort(rng.exponential(1.0, (N, A)), axis=1)[:, ::-1] * rng.uniform(0.5, 3.0, (N, 1))
    if seed % 2:
        S[:, 2] *= 1.5
    return S, tau, full, float(rng.uniform(N * tau, N * full * 0.8))


def test_allocation_against_brute_force():
    """Lagrangian pricing plus improving single-head substitutions is a
    heuristic with a certificate: on every instance the table fits, the dual
    bound lies below the optimum and the certified gap covers the true one;
    on most tiny instances it is optimal."""
    hits = 0
    for seed in range(40):
        S, tau, full, budget = tiny_instance(seed)
        opt, _ = ref.brute_allocation(S, tau, full, budget)
        al = cal.allocate(S, tau, full, budget)
        assert al.traffic <= budget + 1e-9
        cost = sum(full if g == 0 else g * tau for g in al.ranks)
        assert cost == pytest.approx(al.traffic)
        obj = sum(0.0 if g == 0 else S[j, g - 1] for j, g in enumerate(al.ranks))
        assert obj == pytest.approx(al.objective)
        assert al.dual <= opt + 1e-9 <= al.objective + 2e-9
        assert (al.objective - opt) / max(al.objective, 1e-300) <= al.gap + 1e-9
        hits += al.objective <= opt * (1 + 1e-9) + 1e-12
    assert hits >= 30


def test_allocation_gap_is_small_at_model_scale():
    """With many heads (the paper allocates over whole models) the relaxation
    is tight: the certified gap of a 96-head, 24-rank instance is small."""
    rng = np.random.default_rng(12)
    N, A = 96, 24
    decay = rng.uniform(0.6, 0.95, (N, 1))
    S = rng.uniform(0.5, 5.0, (N, 1)) * decay ** np.arange(1, A + 1)[None, :]
    tau, full = 544.0, 65536.0
    al = cal.allocate(S, tau, full, cal.allocation_budget(N, 8.0, tau))
    assert al.traffic <= cal.allocation_budget(N, 8.0, tau)
    assert al.gap < 0.02


def test_allocation_prefers_full_reads_where_they_pay():
    """A head whose every rank keeps a large score goes dense when the budget
    allows; an easy head gets rank 1."""
    S = np.array([[100.0, 90.0, 80.0], [0.1, 0.05, 0.01], [1.0, 0.5, 0.2]])
    al = cal.allocate(S, 1.0, 5.0, 8.0)
    assert al.ranks[0] == 0 and al.ranks[1] == 1
    assert al.traffic <= 8.0


def test_max_rank_and_budget():
    assert cal.tau_sketch(128, 128, 16, True) == 2 * (128 + 128 + 16)
    assert cal.max_rank(128, 128, 16, True) == 120        # ceil(65536 / 544) - 1
    assert cal.max_rank(128, 64, 16, False) == 64         # capped by V
    assert cal.allocation_budget(32, 5.0, 544) == 32 * 5 * 544


def test_layer_calibration_prefix_maps():
    """calibrate_layer: per head, the stored map's first g rows are the rank-g
    offline map of the first g basis columns (E0-orthonormal columns), the
    table spends at most the budget, and a head whose states carry no energy
    outside one direction gets a small rank."""
    H, K, V, r = 3, 10, 7, 6
    X = np.stack([samples(K=K, V=V, N=40, seed=10 + h)[0] for h in range(H)])
    q = np.stack([samples(K=K, V=V, N=40, seed=20 + h)[1] for h in range(H)])
    X[2] = X[2][:, :, :] * 0.0 + np.einsum("nv,k->nvk", np.random.default_rng(1).standard_normal((40, V)),
                                            np.eye(K)[0])     # rank-one states
    out = cal.calibrate_layer(X, q, width=r, mean_rank=3.0, W=8, erase=True)
    assert out.omega.shape == (H, K, r) and out.coef.shape == (H, r, K)
    for h in range(H):
        E0 = np.einsum("nvk,nvl->kl", X[h], X[h]) / X.shape[1]
        om = out.omega[h].astype(np.float64)
        for g in range(1, r + 1):
            Cg = cal.offline_map(om[:, :g], E0)
            np.testing.assert_allclose(out.coef[h][:g], Cg, rtol=2e-4, atol=2e-5)
    tau = cal.tau_sketch(K, V, 8, True)
    cost = sum(4 * K * V if g == 0 else g * tau for g in out.head_ranks)
    assert cost <= cal.allocation_budget(H, 3.0, tau) + 1e-9
    assert out.head_ranks[2] in (1, 2)

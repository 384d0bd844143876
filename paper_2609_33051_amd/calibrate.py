"""Offline calibration: the sketching matrix and the per-head rank table.

Both run once, offline, on the host, as in the paper; their outputs (Omega,
the offline coefficient map, the rank table) are inputs of the decode path
(`SketchSSMLayer(omega=..., coef=..., head_ranks=...)`).  fp64 numpy.

Sketching matrix (Sec. 4.1, "Offline: sketching matrix"; App. A.1):
  E0  = E[S S^T]                  the average state geometry (K x K)
  z   = E0^{1/2} q~               state-weighted effective queries
  C_z = E[z z^T],  P_G = its leading G eigenvectors
  Omega* = E0^{-1/2} P_G          (pseudo-inverse on the support of E0)
  offline map  C = (Omega^T E0 Omega)^+ Omega^T E0
  The loss E[min_c |E0^{1/2}(q~ - Omega c)|^2] of Omega* is the sum of the
  discarded eigenvalues of C_z.

Rank scores (the allocation appendix, eq. alloc-qr and m-head-objective): for
a state S, effective query q~ and sketch U = S^T Omega, with U = Q R (thin QR),
the output residual of the rank-G prefix is
  |delta(G)|^2 = |o|^2 - |Q_{1:G}^T o|^2,   o = S^T q~,
and with an output gradient g the paired score is J(G) = E[(g^T delta(G))^2].

Allocation (the allocation appendix, eq. m-allocation and alloc-dual): each
head chooses a prefix rank in 1..G* or a full-state read (score 0, cost 4KV)
under a traffic budget N Gbar tau_sk, tau_sk = 2(V + K + eW); solved by a
Lagrangian relaxation (a traffic price mu, bisected until the traffic fits),
keeping the best feasible table met, then spending the remaining slack by
improving single-head substitutions; (P - D(mu)) / P certifies the gap.

Layouts follow the library: a state is stored transposed, [V][K] (S^T), so
S S^T = X^T X for the stored X.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def state_metric(states) -> np.ndarray:
    """E0 = E[S S^T] from stored states X = S^T, [N][V][K] -> [K][K]."""
    X = np.asarray(states, np.float64)
    return np.einsum("nvk,nvl->kl", X, X) / X.shape[0]


def _sym_power(E: np.ndarray, p: float, rtol: float = 1e-10) -> np.ndarray:
    """E^p for a symmetric PSD E; negative powers act on the support only."""
    w, Q = np.linalg.eigh((E + E.T) / 2)
    keep = w > rtol * max(w.max(), 0.0)
    wp = np.zeros_like(w)
    wp[keep] = w[keep] ** p
    return (Q * wp) @ Q.T


@dataclass
class OfflineBasis:
    omega: np.ndarray       # [K][G]  Omega* = E0^{-1/2} P_G
    coef: np.ndarray        # [G][K]  the offline map (Omega^T E0 Omega)^+ Omega^T E0
    eigvals: np.ndarray     # [K]     eigenvalues of C_z, descending
    E0: np.ndarray          # [K][K]

    @property
    def loss(self) -> float:
        """The offline loss of Omega*: the discarded eigenvalues of C_z."""
        return float(self.eigvals[self.omega.shape[1]:].sum())


def offline_map(omega: np.ndarray, E0: np.ndarray) -> np.ndarray:
    """C_offline = (Omega^T E0 Omega)^+ Omega^T E0, [G][K]."""
    om = np.asarray(omega, np.float64)
    return np.linalg.pinv(om.T @ E0 @ om) @ om.T @ E0


def offline_basis(states, queries, G: int) -> OfflineBasis:
    """Omega* for one head from calibration states [N][V][K] (stored S^T) and
    effective queries [M][K] (uncentered PCA of z = E0^{1/2} q~)."""
    E0 = state_metric(states)
    q = np.asarray(queries, np.float64)
    z = q @ _sym_power(E0, 0.5)                 # rows z_t^T (E0^{1/2} is symmetric)
    Cz = z.T @ z / q.shape[0]
    lam, P = np.linalg.eigh((Cz + Cz.T) / 2)
    order = np.argsort(lam)[::-1]
    lam, P = lam[order], P[:, order]
    omega = _sym_power(E0, -0.5) @ P[:, :G]
    return OfflineBasis(omega, offline_map(omega, E0), np.maximum(lam, 0.0), E0)


def orthonormal_prefix_basis(omega: np.ndarray) -> np.ndarray:
    """An orthonormal basis whose first g columns span the first g columns of
    `omega` for every g (QR with a positive diagonal; a dependent column is
    replaced by a unit vector orthogonal to the earlier ones).  The decode
    kernels' state-dependent map needs an orthonormal Omega (coef = Omega^T);
    the sketch's prefix spans, and so each rank's exact map, are unchanged."""
    om = np.asarray(omega, np.float64)
    K, G = om.shape
    out = np.zeros((K, G))
    m = 0
    for g in range(G):
        x = om[:, g].copy()
        for _ in range(2):
            x -= out[:, :m] @ (out[:, :m].T @ x)
        n = np.linalg.norm(x)
        if n <= 1e-10 * max(np.linalg.norm(om[:, g]), 1e-300):
            for e in range(K):  # a unit vector outside the span so far
                x = np.zeros(K)
                x[e] = 1.0
                for _ in range(2):
                    x -= out[:, :m] @ (out[:, :m].T @ x)
                n = np.linalg.norm(x)
                if n > 1e-6:
                    break
        out[:, m] = x / n
        m += 1
    return out


def rank_scores(states, queries, omega, grads=None):
    """Prefix-rank scores of one head over calibration pairs (state, query):
    eps[G] = E|delta(G)|^2 and, with output gradients [N][V], J[G] =
    E[(g^T delta(G))^2], for G = 0..Gmax (G = 0: nothing kept).
    states [N][V][K] (stored S^T), queries [N][K] (effective queries)."""
    X = np.asarray(states, np.float64)
    q = np.asarray(queries, np.float64)
    om = np.asarray(omega, np.float64)
    N, Gmax = X.shape[0], om.shape[1]
    eps = np.zeros(Gmax + 1)
    J = np.zeros(Gmax + 1) if grads is not None else None
    for t in range(N):
        o = X[t] @ q[t]                    # S^T q~
        U = X[t] @ om                      # S^T Omega, [V][Gmax]
        Q = _prefix_orthonormal(U)         # thin QR; a dependent prefix column adds a zero column
        proj = Q.T @ o
        eps += o @ o - np.concatenate([[0.0], np.cumsum(proj ** 2)])
        if grads is not None:
            gv = np.asarray(grads[t], np.float64)
            gq = Q.T @ gv
            J += (gv @ o - np.concatenate([[0.0], np.cumsum(gq * proj)])) ** 2
    eps /= N
    if J is not None:
        J /= N
    return np.maximum(eps, 0.0), J


def _prefix_orthonormal(U: np.ndarray) -> np.ndarray:
    """Columns q_g orthonormal with span(q_1..q_g) = span(u_1..u_g); where u_g
    depends on the earlier columns, q_g = 0 (Gram-Schmidt, twice per column)."""
    V, G = U.shape
    Q = np.zeros((V, G))
    scale = max(np.linalg.norm(U), 1e-300)
    for g in range(G):
        x = U[:, g].copy()
        for _ in range(2):
            x -= Q[:, :g] @ (Q[:, :g].T @ x)
        n = np.linalg.norm(x)
        if n > 1e-12 * scale:
            Q[:, g] = x / n
    return Q


def tau_sketch(K: int, V: int, W: int, erase: bool) -> int:
    """Read bytes per unit of sketch rank with BF16 storage: 2(V + K + eW)."""
    return 2 * (V + K + (W if erase else 0))


def max_rank(K: int, V: int, W: int, erase: bool) -> int:
    """G*: the largest rank strictly cheaper to read than the fp32 state."""
    return int(min(K, V, -(-4 * K * V // tau_sketch(K, V, W, erase)) - 1))


@dataclass
class Allocation:
    ranks: list            # per head: rank in 1..G*, or 0 = full-state read (dense fallback)
    objective: float       # P: the summed score of the table
    traffic: float         # its summed read bytes
    budget: float
    dual: float            # the best lower bound D(mu) met
    mu: float              # the price that gave it

    @property
    def gap(self) -> float:
        """(P - D) / P: relative distance from the optimum of the separable objective, at most."""
        return 0.0 if self.objective <= 0 else max(self.objective - self.dual, 0.0) / self.objective


def allocate(scores, tau_sk: float, full_cost: float, budget: float, iters: int = 200) -> Allocation:
    """Budgeted choice of one action per head.

    scores: [N][A] with scores[j][G-1] = J_j(G) for G = 1..A (ranks 1..A; A
    is G* or the storage width, whichever is smaller); the full-state read
    has score 0 and cost `full_cost`; rank G costs G tau_sk.  Returns the best
    feasible table (rank 0 = full read) with its objective, traffic and the
    best dual bound."""
    S = np.asarray(scores, np.float64)
    N, A = S.shape
    cost = np.concatenate([np.arange(1, A + 1) * float(tau_sk), [float(full_cost)]])
    score = np.concatenate([S, np.zeros((N, 1))], axis=1)          # action A = full read

    def choose(mu):
        pen = score + mu * cost[None, :]
        a = np.argmin(pen, axis=1)
        return a, float(pen[np.arange(N), a].sum() - mu * budget)

    def total(a):
        return float(cost[a].sum()), float(score[np.arange(N), a].sum())

    if N * cost.min() > budget:
        raise ValueError("the budget cannot pay for rank 1 on every head")
    best, best_obj, best_dual, best_mu = None, np.inf, -np.inf, 0.0

    def consider(a, mu, dual):
        nonlocal best, best_obj, best_dual, best_mu
        tr, ob = total(a)
        if dual > best_dual:
            best_dual, best_mu = dual, mu
        if tr <= budget and ob < best_obj:
            best, best_obj = a.copy(), ob

    a0, d0 = choose(0.0)
    consider(a0, 0.0, d0)
    if total(a0)[0] > budget:
        lo, hi = 0.0, 1.0
        while True:  # a price high enough that the cheapest actions win
            a, d = choose(hi)
            consider(a, hi, d)
            if total(a)[0] <= budget:
                break
            lo, hi = hi, hi * 2.0
        for _ in range(iters):
            mid = 0.5 * (lo + hi)
            a, d = choose(mid)
            consider(a, mid, d)
            if total(a)[0] <= budget:
                hi = mid
            else:
                lo = mid
    # spend the remaining slack: improving single-head substitutions, best first
    a = best.copy()
    while True:
        tr, ob = total(a)
        gain, move = 0.0, None
        for j in range(N):
            cur = a[j]
            for b in range(A + 1):
                if b == cur or tr - cost[cur] + cost[b] > budget:
                    continue
                dg = score[j, cur] - score[j, b]
                if dg > gain + 1e-15 * max(abs(ob), 1.0):
                    gain, move = dg, (j, b)
        if move is None:
            break
        a[move[0]] = move[1]
    tr, ob = total(a)
    ranks = [0 if x == A else int(x) + 1 for x in a]
    return Allocation(ranks, ob, tr, float(budget), best_dual, best_mu)


def allocation_budget(n_heads: int, mean_rank: float, tau_sk: float) -> float:
    """B = N Gbar tau_sk."""
    return n_heads * mean_rank * tau_sk


@dataclass
class LayerCalibration:
    omega: np.ndarray      # [H][K][width] fp32, each head's leading `width` basis columns
    coef: np.ndarray       # [H][width][K] fp32, the offline map of the full width
    head_ranks: list       # per head: rank 1..width, or 0 = dense fallback
    allocation: Allocation
    scores: np.ndarray     # [H][width] the per-rank scores the allocation used


def calibrate_layer(states, queries, width: int, mean_rank: float, W: int, erase: bool, grads=None,
                    ) -> LayerCalibration:
    """One layer's offline calibration in the decode path's layouts.

    states [H][N][V][K] (stored S^T), queries [H][N][K] (effective queries),
    grads [H][N][V] (output gradients) or None (then the gradient-free score
    eps(G) of the allocation appendix is used).  The basis of each head is its
    Omega* = E0^{-1/2} P_width; its columns are E0-orthonormal, so the
    offline map of the first g columns is the first g rows of the stored map,
    which is what a per-head rank table uses.  The allocation chooses, per
    head, a rank in 1..min(G*, width) or the full state under the budget
    H mean_rank tau_sk."""
    X = np.asarray(states, np.float64)
    q = np.asarray(queries, np.float64)
    H, _, V, K = X.shape
    A = min(max_rank(K, V, W, erase), width)
    omegas = np.zeros((H, K, width))
    coefs = np.zeros((H, width, K))
    scores = np.zeros((H, A))
    for h in range(H):
        b = offline_basis(X[h], q[h], width)
        omegas[h], coefs[h] = b.omega, b.coef
        eps, J = rank_scores(X[h], q[h], b.omega, None if grads is None else grads[h])
        scores[h] = (eps if J is None else J)[1:A + 1]
    tau = tau_sketch(K, V, W, erase)
    al = allocate(scores, tau, 4.0 * K * V, allocation_budget(H, mean_rank, tau))
    return LayerCalibration(omegas.astype(np.float32), coefs.astype(np.float32), al.ranks, al, scores)

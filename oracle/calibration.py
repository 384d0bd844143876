"""Plain definitions for checking the offline calibration (test
infrastructure only; the package never imports this module).

Each function restates its quantity from the paper's definition with no
shortcut, so a test can hold the faster calibration code to it:

offline_loss       eq. m-subspace-objective: the mean over samples of
                   min_c |E0^{1/2} (q~ - Omega c)|^2, each sample's inner
                   problem solved by least squares (App. A.1, steps 1-3)
prefix_residuals   the allocation appendix: for every prefix rank G, the
                   output residual delta(G) = o - U_G c with c the least-
                   squares coefficients of the first G sketch columns, its
                   mean square, and its mean squared pairing with a gradient
                   (eq. m-head-objective)
brute_allocation   eq. m-allocation by enumerating every table
"""
from __future__ import annotations

import itertools

import numpy as np


def sqrt_psd(E):
    """The symmetric square root of a PSD matrix, from its eigendecomposition."""
    w, Q = np.linalg.eigh((E + E.T) / 2)
    return (Q * np.sqrt(np.clip(w, 0.0, None))) @ Q.T


def offline_loss(omega, E0, queries):
    E_half = sqrt_psd(np.asarray(E0, np.float64))
    B = E_half @ np.asarray(omega, np.float64)
    tot = 0.0
    for q in np.asarray(queries, np.float64):
        z = E_half @ q
        c = np.linalg.lstsq(B, z, rcond=None)[0]
        tot += float(np.sum((z - B @ c) ** 2))
    return tot / len(queries)


def prefix_residuals(states, queries, omega, grads=None):
    """eps[G], J[G] for G = 0..Gmax from stored states X = S^T [N][V][K]."""
    X = np.asarray(states, np.float64)
    om = np.asarray(omega, np.float64)
    Gmax = om.shape[1]
    eps = np.zeros(Gmax + 1)
    J = np.zeros(Gmax + 1)
    for t in range(X.shape[0]):
        o = X[t] @ np.asarray(queries[t], np.float64)
        U = X[t] @ om
        for G in range(Gmax + 1):
            if G == 0:
                d = o
            else:
                c = np.linalg.lstsq(U[:, :G], o, rcond=None)[0]
                d = o - U[:, :G] @ c
            eps[G] += float(d @ d)
            if grads is not None:
                J[G] += float(np.asarray(grads[t], np.float64) @ d) ** 2
    n = X.shape[0]
    return eps / n, (J / n if grads is not None else None)


def brute_allocation(scores, tau_sk, full_cost, budget):
    """The best table by enumeration: every head picks a rank 1..A or the full
    read (rank 0 here, score 0, cost full_cost); rank G costs G tau_sk.
    Returns (objective, ranks) of a minimum, or (inf, None) if none fits."""
    S = np.asarray(scores, np.float64)
    N, A = S.shape
    best, arg = np.inf, None
    for choice in itertools.product(range(A + 1), repeat=N):  # A = the full read
        cost = sum(full_cost if a == A else (a + 1) * tau_sk for a in choice)
        if cost > budget:
            continue
        obj = sum(0.0 if a == A else S[j, a] for j, a in enumerate(choice))
        if obj < best:
            best, arg = obj, [0 if a == A else a + 1 for a in choice]
    return best, arg

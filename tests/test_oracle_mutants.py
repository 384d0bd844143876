"""Planted mistakes: each test copies the oracle source, introduces one plausible
slip, compiles the copy on the CPU and checks that the pins reject it.  This
shows the pins constrain every part of the oracle, not just its happy path."""
import numpy as np
import pytest

import oracle
from test_oracle_pins import brute_force_outputs, heads_omega, orthonormal, tiny_inputs

KINDS = ["mamba2", "gdn", "kda"]


def _close(a, b, tol=1e-9):
    return np.allclose(a, b, rtol=tol, atol=tol)


def pins_hold(lib) -> bool:
    """The pin battery of test_oracle_pins.py in compact form; False on the first failure."""
    for kind in KINDS:
        S0, q, k, v, beta, logd = tiny_inputs(kind, seed=1)
        o, _ = oracle.recurrence(kind, S0, q, k, v, beta, logd, lib=lib)
        if not _close(o, brute_force_outputs(kind, S0, q, k, v, beta, logd)):
            return False
        W, T = 4, 12
        S0, q, k, v, beta, logd = tiny_inputs(kind, T=T, seed=5)
        om, C = heads_omega(2, 5, 2, 10)
        heads = np.array([0, 1, 0], np.int32)
        o_ex, S_ex = oracle.recurrence(kind, S0, q, k, v, beta, logd, lib=lib)
        r = oracle.sketchssm(kind, W, heads, om, C, S0, q, k, v, beta, logd, lib=lib)
        if not _close(r.S_final, S_ex) or not _close(r.o_exact_windowed, o_ex):
            return False
        eye = np.eye(5, dtype=np.float32)[None]
        r = oracle.sketchssm(kind, W, np.zeros(3, np.int32), eye, eye.copy(), S0, q, k, v, beta, logd, lib=lib)
        if not _close(r.o, o_ex) or not _close(r.U_final, r.S_final):
            return False
    # sketch projection with a rectangular Omega (catches C / Omega transposes)
    K, V, G, W, T, n = 7, 4, 3, 6, 5, 2
    S0, q, k, v, beta, logd = tiny_inputs("mamba2", n=n, K=K, V=V, T=T, seed=9)
    om = orthonormal(K, G, 13)[None]
    C = np.ascontiguousarray(om.transpose(0, 2, 1))
    rng = np.random.default_rng(14)
    q_in = np.einsum("kg,tng->tnk", om[0].astype(np.float64), rng.standard_normal((T, n, G))).astype(np.float32)
    r = oracle.sketchssm("mamba2", W, np.zeros(n, np.int32), om, C, S0, q_in, k, v, beta, logd, lib=lib)
    if not np.allclose(r.o_state_hat, r.o_state, rtol=1e-6, atol=1e-6):
        return False
    # the state-dependent coefficient map
    from test_oracle_pins import coef_map_of, exact_ridge_map, low_rank_state
    Sl = low_rank_state(2, 6, 8, 2, seed=2)
    oml = heads_omega(1, 8, 5, seed=21)[0]
    if not np.allclose(coef_map_of(Sl, oml, 2, 0.1, lib=lib), exact_ridge_map(Sl, oml, 0.1), rtol=1e-6, atol=1e-7):
        return False
    Sg = np.random.default_rng(12).standard_normal((2, 6, 8)).astype(np.float32)
    omg = heads_omega(1, 8, 6, seed=7)[0]
    perm = np.array([1, 0, 5, 2, 4, 3])
    if not np.allclose(coef_map_of(Sg, np.ascontiguousarray(omg[:, :, perm]), 2, 0.1, lib=lib),
                       coef_map_of(Sg, omg, 2, 0.1, lib=lib)[:, perm], rtol=1e-6, atol=1e-7):
        return False
    eye = np.eye(5, dtype=np.float32)[None]
    Si = np.random.default_rng(4).standard_normal((2, 7, 5)).astype(np.float32)
    if not np.allclose(coef_map_of(Si, eye, 3, 1e-9, lib=lib), np.broadcast_to(np.eye(5), (2, 5, 5)), atol=1e-6):
        return False
    # the paper's coefficient-space forms (f_s) equal the direct ones
    for kind in ("gdn", "kda"):
        for piv in (0, 4):
            S0p, qp, kp, vp, bp, lp = tiny_inputs(kind, n=3, K=8, V=6, T=13, seed=21)
            omp, Cp = heads_omega(1, 8, 5, seed=9)
            z3 = np.zeros(3, np.int32)
            a = oracle.sketchssm(kind, 5, z3, omp, Cp, S0p, qp, kp, vp, bp, lp, pivots=piv, lib=lib)
            b = oracle.sketchssm(kind, 5, z3, omp, Cp, S0p, qp, kp, vp, bp, lp, pivots=piv, paper_path=True, lib=lib)
            if not np.allclose(b.o, a.o, rtol=1e-10, atol=1e-10 * np.abs(a.o).max()):
                return False
    # bf16 storage (the dense map rounded once, f rounded when stored) and the exact metric
    import test_oracle_pins as P
    try:
        for kind in KINDS:
            for piv in (4, oracle.EXACT):
                P.test_bf16_map_storage_is_round_to_nearest_even(kind, piv, lib=lib)
        P.test_bf16_map_is_the_one_read(4, lib=lib)
        for kind in ("gdn", "kda"):
            P.test_bf16_f_is_rounded_when_stored_not_when_formed(kind, lib=lib)
        P.test_exact_map_is_the_closed_form(None, lib=lib)
    except AssertionError:
        return False
    # the sketch must be refreshed from the updated state at each flush
    r = oracle.sketchssm("mamba2", 2, np.zeros(n, np.int32), om, C, S0, q_in, k, v, beta, logd, lib=lib)
    Uref = np.einsum("nvk,kg->nvg", r.S_final, om[0].astype(np.float64))
    if not _close(r.U_final, Uref):
        return False
    return True


MUTANTS = {
    "coef_ridge_dropped": [("w->A[(size_t)g * G + g2] = Hm[(size_t)g * K + g2] + (g == g2 ? lambda : 0.0);",
                            "w->A[(size_t)g * G + g2] = Hm[(size_t)g * K + g2];")],
    "coef_metric_not_normalised": [("      w->H[(size_t)i * K + i2] = acc / mu;", "      w->H[(size_t)i * K + i2] = acc;")],
    "coef_pivots_from_last_columns": [("      x[j] = U[(size_t)j * G + a];", "      x[j] = U[(size_t)j * G + (G - 1 - a)];")],
    "coef_diagonal_dropped": [("      double acc = (i == i2) ? w->d[i] : 0.0;", "      double acc = 0.0;")],
    "erase_sign": [("S[(size_t)kk * V + j] -= beta * (double)k[kk] * tmpV[j];",
                    "S[(size_t)kk * V + j] += beta * (double)k[kk] * tmpV[j];")],
    "erase_before_decay_in_update": [
        ("  for (int kk = 0; kk < K; ++kk) {\n    const double d = tok_decay(t, n, kk);\n"
         "    for (int j = 0; j < V; ++j) S[(size_t)kk * V + j] *= d;\n  }\n  if (has_erase(t->c)) {\n"
         "    /* tmpV = k^T (D S) */",
         "  if (has_erase(t->c)) {\n    /* tmpV = k^T (D S) */"),
        ("  for (int kk = 0; kk < K; ++kk)\n    for (int j = 0; j < V; ++j) S[(size_t)kk * V + j] += beta",
         "  for (int kk = 0; kk < K; ++kk) {\n    const double d = tok_decay(t, n, kk);\n"
         "    for (int j = 0; j < V; ++j) S[(size_t)kk * V + j] *= d;\n  }\n"
         "  for (int kk = 0; kk < K; ++kk)\n    for (int j = 0; j < V; ++j) S[(size_t)kk * V + j] += beta"),
    ],
    "effective_query_transposed_order": [("for (int s = len - 1; s >= 0; --s) apply_MT(&t, buf[s], x);",
                                          "for (int s = 0; s < len; ++s) apply_MT(&t, buf[s], x);")],
    "effective_query_without_erase": [("for (int s = len - 1; s >= 0; --s) apply_MT(&t, buf[s], x);",
                                       "for (int s = len - 1; s >= 0; --s) for (int kk = 0; kk < K; ++kk) "
                                       "x[kk] *= tok_decay(&t, buf[s], kk);")],
    "buffer_drops_self_term": [("for (int s = 0; s < len; ++s) {\n          const float* ks",
                                "for (int s = 0; s < len - 1; ++s) {\n          const float* ks")],
    "buffer_decay_off_by_one": [("for (int r = s + 1; r < len; ++r) apply_M(&t, buf[r], y);",
                                 "for (int r = s; r < len; ++r) apply_M(&t, buf[r], y);")],
    "buffer_drops_beta": [("const double w = tok_beta(&t, buf[s]) * a;", "const double w = a;")],
    "flush_drops_last_token": [("for (int s = 0; s < len; ++s) update_state(&t, buf[s], S0, tmp);",
                                "for (int s = 0; s < len - 1; ++s) update_state(&t, buf[s], S0, tmp);")],
    "coefficient_map_transposed": [("acc += (Cmi ? Cmi[(size_t)g * K + kk] : (double)Cm[(size_t)g * K + kk]) * x[kk];",
                                    "acc += (Cmi ? Cmi[(size_t)g * K + kk] : (double)Cm[(size_t)kk * G + g]) * x[kk];")],
    "sketch_omega_transposed": [("acc += S[(size_t)kk * V + j] * (double)omega[(size_t)kk * G + g];",
                                 "acc += S[(size_t)kk * V + j] * (double)omega[(size_t)g * K + kk];")],
    "kda_channel_index": [("[((size_t)n * c->n_items + t->item) * c->K + kk]",
                           "[((size_t)n * c->n_items + t->item) * c->K + (c->K - 1 - kk)]")],
    "wyread_drops_history": [("              ck -= fhat[(size_t)j * G + g] * ak[j];\n", "")],
    "wyread_drops_beta": [("            const double ft = bt * ck;", "            const double ft = ck;")],
    "projected_query_drops_self_term": [("            cvec[g] = cq - ft * akq;", "            cvec[g] = cq;")],
    "left_factor_decay_off_by_one": [("            for (int r = j + 1; r <= cur; ++r)", "            for (int r = j; r <= cur; ++r)")],
    "exact_map_uses_pivot_metric": [("  if (P > 0) {\n    /* Q: the first p columns", "  if (P != 0) {\n    /* Q: the first p columns")],
    "map_not_rounded_when_stored": [("{\n  store_sketch(c, Cm, n);\n}", "{\n  (void)c;\n  (void)Cm;\n  (void)n;\n}")],
    "map_built_from_rounded_sketch": [
        ("          make_sketch(K, V, G, S0, Om, U);\n          if (statedep && Cmi && cw.R) {\n"
         "            coef_map(c, K, V, G, S0, Om, U, Cmi, &cw);\n            store_map(c, Cmi, (size_t)G * K);\n"
         "          }\n          store_sketch(c, U, (size_t)V * G);",
         "          make_sketch(K, V, G, S0, Om, U);\n          store_sketch(c, U, (size_t)V * G);\n"
         "          if (statedep && Cmi && cw.R) {\n"
         "            coef_map(c, K, V, G, S0, Om, U, Cmi, &cw);\n            store_map(c, Cmi, (size_t)G * K);\n"
         "          }")],
    "current_f_rounded": [("            const double ft = bt * ck;",
                           "            const double ft = c->sketch_bf16 ? bf16_rne(bt * ck) : bt * ck;")],
    "f_not_rounded_when_stored": [("fhat[(size_t)cur * G + g] = c->sketch_bf16 ? bf16_rne(ft) : ft;",
                                   "fhat[(size_t)cur * G + g] = ft;")],
    "sketch_not_refreshed": [("        if (G > 0) {\n          make_sketch(K, V, G, S0, Om, U);\n"
                              "          if (statedep && Cmi && cw.R) {\n"
                              "            coef_map(c, K, V, G, S0, Om, U, Cmi, &cw);\n"
                              "            store_map(c, Cmi, (size_t)G * K);\n          }\n"
                              "          store_sketch(c, U, (size_t)V * G);\n        }\n"
                              "        for (int j = 0; j < V; ++j) {\n          if (o) o[oi + j] = ostate[j];",
                              "        for (int j = 0; j < V; ++j) {\n          if (o) o[oi + j] = ostate[j];")],
}


def test_unmodified_oracle_passes_the_battery():
    assert pins_hold(oracle._load())


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, tmp_path):
    src = oracle.source_text()
    for old, new in MUTANTS[name]:
        assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
        src = src.replace(old, new)
    lib = oracle.build_variant(src, str(tmp_path), name)
    assert not pins_hold(lib), f"planted mistake {name} passed every pin"

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
    # the sketch must be refreshed from the updated state at each flush
    r = oracle.sketchssm("mamba2", 2, np.zeros(n, np.int32), om, C, S0, q_in, k, v, beta, logd, lib=lib)
    Uref = np.einsum("nvk,kg->nvg", r.S_final, om[0].astype(np.float64))
    if not _close(r.U_final, Uref):
        return False
    return True


MUTANTS = {
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
    "coefficient_map_transposed": [("acc += (double)Cm[(size_t)g * K + kk] * x[kk];",
                                    "acc += (double)Cm[(size_t)kk * G + g] * x[kk];")],
    "sketch_omega_transposed": [("acc += S[(size_t)kk * V + j] * (double)omega[(size_t)kk * G + g];",
                                 "acc += S[(size_t)kk * V + j] * (double)omega[(size_t)g * K + kk];")],
    "kda_channel_index": [("[((size_t)n * c->n_items + t->item) * c->K + kk]",
                           "[((size_t)n * c->n_items + t->item) * c->K + (c->K - 1 - kk)]")],
    "sketch_not_refreshed": [("        if (G > 0) {\n          make_sketch(K, V, G, S0, Om, U);\n"
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

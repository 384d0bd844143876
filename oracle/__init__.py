"""Plain CPU oracle for the SketchSSM decode path (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports, links or calls it, and the two share no
code.

The arithmetic lives in ``sketchssm_oracle.c`` (fp64, one item at a time,
OpenMP over independent (request, head) items).  This module only compiles it
with gcc, loads it with ctypes and marshals numpy arrays.

Functions
---------
recurrence(kind, S_init, q, k, v, beta, log_decay)
    The plain per-token recurrence of Sec. 3.2 (eq. transition-update, first
    form) with the exact read o_t = S_t^T q_t at every token.
sketchssm(kind, W, heads, omega, coef, S_init, q, k, v, beta, log_decay)
    SketchSSM inference, Algorithm 1: sketch reads between flushes, exact
    replay of the buffered tokens at every W-th token.

Array conventions (all float32 inputs; bf16 inputs are passed as their exact
float32 values): states [n][V][K], per-step inputs [T][n][...], Omega
[H][K][G], coefficient map C [H][G][K].
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sketchssm_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

KINDS = {"mamba2": 0, "gdn": 1, "kda": 2}
EXACT = -1  # pivots value of the state-dependent map with the exact (dense) state metric


class _Cfg(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32),
        ("n_items", ctypes.c_int32),
        ("K", ctypes.c_int32),
        ("V", ctypes.c_int32),
        ("G", ctypes.c_int32),
        ("W", ctypes.c_int32),
        ("T", ctypes.c_int32),
        ("round_storage", ctypes.c_int32),
        ("sketch_bf16", ctypes.c_int32),
        ("pivots", ctypes.c_int32),
        ("ridge", ctypes.c_float),
        ("paper_path", ctypes.c_int32),
    ]


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (no HIP involved)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(
            ["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"],
            check=True,
        )
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _bind(lib):
    dp = ctypes.POINTER(ctypes.c_double)
    fp = ctypes.POINTER(ctypes.c_float)
    ip = ctypes.POINTER(ctypes.c_int32)
    lib.orc_recurrence.argtypes = [ctypes.POINTER(_Cfg), fp, fp, fp, fp, fp, fp, dp, dp]
    lib.orc_recurrence.restype = ctypes.c_int
    lib.orc_sketchssm.argtypes = [ctypes.POINTER(_Cfg), ip, fp, fp, fp, fp, fp, fp, fp, fp, dp, dp, dp, dp, dp, dp, dp]
    lib.orc_sketchssm.restype = ctypes.c_int
    lib.orc_max_threads.restype = ctypes.c_int
    lib.orc_set_threads.argtypes = [ctypes.c_int]
    return lib


def build_variant(source_text: str, out_dir: str, tag: str):
    """Compile a modified copy of the oracle source (used by the mutation
    tests, which plant a mistake on the CPU and check that a pin fails)."""
    src = os.path.join(out_dir, f"oracle_{tag}.c")
    lib = os.path.join(out_dir, f"liboracle_{tag}.so")
    with open(src, "w") as f:
        f.write(source_text)
    subprocess.run(["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-o", lib, src, "-lm"], check=True)
    return _bind(ctypes.CDLL(lib))


def source_text() -> str:
    with open(_SRC) as f:
        return f.read()


def _load():
    global _lib
    if _lib is None:
        _lib = _bind(ctypes.CDLL(build()))
    return _lib


def max_threads() -> int:
    return int(_load().orc_max_threads())


def set_threads(n: int) -> None:
    _load().orc_set_threads(int(n))


def _f32(a):
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def _out(shape, enabled=True):
    if not enabled:
        return None, None
    a = np.zeros(shape, dtype=np.float64)
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _check_inputs(kind, S_init, q, k, v, beta, log_decay):
    if kind not in KINDS:
        raise ValueError(f"unknown kind {kind!r}")
    n, V, K = S_init.shape
    T = q.shape[0]
    if q.shape != (T, n, K) or k.shape != (T, n, K) or v.shape != (T, n, V):
        raise ValueError("q/k/v shapes must be [T][n][K], [T][n][K], [T][n][V]")
    if beta.shape != (T, n):
        raise ValueError("beta must be [T][n]")
    want = (T, n, K) if kind == "kda" else (T, n)
    if log_decay.shape != want:
        raise ValueError(f"log_decay must be {want}")
    return n, K, V, T


def recurrence(kind, S_init, q, k, v, beta, log_decay, lib=None):
    """Plain recurrence.  Returns (o_exact [T][n][V], S_final [n][V][K]) in fp64."""
    lib = lib or _load()
    n, K, V, T = _check_inputs(kind, S_init, q, k, v, beta, log_decay)
    keep = [_f32(x) for x in (S_init, q, k, v, beta, log_decay)]
    o, op = _out((T, n, V))
    S, Sp = _out((n, V, K))
    cfg = _Cfg(KINDS[kind], n, K, V, 0, 1, T, 0, 0)
    rc = lib.orc_recurrence(ctypes.byref(cfg), *[p for _, p in keep], op, Sp)
    if rc != 0:
        raise RuntimeError(f"orc_recurrence failed ({rc})")
    return o, S


@dataclass
class SketchResult:
    o: np.ndarray            # [T][n][V] the method's output
    o_state_hat: np.ndarray  # [T][n][V] U c_t (non-flush), exact at flushes
    o_state: np.ndarray      # [T][n][V] S0^T q~_t (non-flush), exact at flushes
    o_buf: np.ndarray        # [T][n][V] buffer term (0 at flushes)
    S_final: np.ndarray      # [n][V][K]
    U_final: np.ndarray      # [n][V][G]
    coef_final: np.ndarray   # [n][G][K] the coefficient map in use at the end

    @property
    def o_exact_windowed(self) -> np.ndarray:
        """What an exact full-state read gives at every step."""
        return self.o_state + self.o_buf


def sketchssm(kind, W, heads, omega, coef, S_init, q, k, v, beta, log_decay, round_storage=False,
              diagnostics=True, lib=None, sketch_bf16=False, pivots=0, ridge=0.1, paper_path=False):
    """SketchSSM inference (Algorithm 1) in fp64.

    heads: [n] int, head index of every item (selects Omega / C); omega
    [H][K][G]; coef [H][G][K].  G = 0 (omega.shape[2] == 0) disables the
    sketch (o_state_hat is then 0 between flushes).  round_storage stores the
    state, the sketch and the state-dependent map as fp32; sketch_bf16 stores
    the sketch, the state-dependent map (the dense G x K matrix, rounded once
    per flush) and the projected erase factors f_s (rounded when first read)
    as bf16 (round to nearest, ties to even, through fp32), the paper's
    storage.  paper_path computes the coefficients through f_s (eq. wyread,
    app-projected-query; implied by sketch_bf16; without rounding it equals
    c = C q~).
    pivots != 0 replaces the given coef by the state-dependent coefficient
    map with ridge term `ridge` (lambda), rebuilt from the state at the start
    and at every flush: P > 0 pivots use the low-rank-plus-diagonal metric of
    eq. pivot-metric, pivots = EXACT the exact metric H (eq. pivot-ridge as
    written); coef_final returns the map in use at the end (as stored).
    """
    lib = lib or _load()
    n, K, V, T = _check_inputs(kind, S_init, q, k, v, beta, log_decay)
    heads = np.ascontiguousarray(heads, dtype=np.int32)
    if heads.shape != (n,):
        raise ValueError("heads must be [n]")
    omega = np.ascontiguousarray(omega, dtype=np.float32)
    coef = np.ascontiguousarray(coef, dtype=np.float32)
    H, K2, G = omega.shape
    if K2 != K or coef.shape != (H, G, K):
        raise ValueError("omega must be [H][K][G] and coef [H][G][K]")
    if n and (heads.min() < 0 or heads.max() >= H):
        raise ValueError("head index out of range")
    keep_o = _f32(omega)
    keep_c = _f32(coef)
    keep = [_f32(x) for x in (S_init, q, k, v, beta, log_decay)]
    o, op = _out((T, n, V))
    oh, ohp = _out((T, n, V), diagnostics)
    os_, osp = _out((T, n, V), diagnostics)
    ob, obp = _out((T, n, V), diagnostics)
    S, Sp = _out((n, V, K))
    U, Up = _out((n, V, G))
    Cf, Cfp = _out((n, G, K))
    cfg = _Cfg(KINDS[kind], n, K, V, G, int(W), T, 1 if round_storage else 0, 1 if sketch_bf16 else 0,
               int(pivots), float(ridge), 1 if paper_path else 0)
    rc = lib.orc_sketchssm(
        ctypes.byref(cfg),
        heads.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
        keep_o[1], keep_c[1],
        *[p for _, p in keep],
        op, ohp, osp, obp, Sp, Up, Cfp,
    )
    if rc != 0:
        raise RuntimeError(f"orc_sketchssm failed ({rc})")
    return SketchResult(o, oh, os_, ob, S, U, Cf)

"""Every kernel instance the library compiles runs against the oracle.

The library compiles the decode and flush kernels per family, (K, V) shape,
storage rank (8, 16, 32 or K), window class (up to 16 or 32 slots), io and
storage dtype and coefficient map (offline, P = 4 pivots for ranks 8..32, the
exact metric for ranks 8 and 16).  Each test below takes one family and
shape and runs, for every such instance, a tiny batch through one flush and a
few decode steps (windows of 7 and 20 tokens: W + 3 steps), checked against
the oracle with the parity bars of tests/harness.py.  Every instance thereby
runs at least once, whichever configurations the other tests exercise.
"""
import numpy as np
import pytest
import torch

from paper_2609_33051_amd import inputs
from harness import bars, format_report, oracle_of, parity_failures, parity_report, run_workload, to_np32

pytestmark = pytest.mark.gpu

STORAGE = (("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32"))  # (io, sketch)


def instances(K):
    for R in (8, 16, 32, K):
        for W in (7, 20):
            for io, sk in STORAGE:
                for piv in (0, 4, -1):
                    if piv == 4 and not 8 <= R <= 32:
                        continue
                    if piv == -1 and R not in (8, 16):
                        continue
                    yield R, W, io, sk, piv


@pytest.mark.parametrize("fam", ["mamba2", "gdn", "kda"])
@pytest.mark.parametrize("K,V", [(64, 64), (128, 64), (128, 128)])
def test_every_compiled_instance(fam, K, V):
    failures = []
    for R, W, io, sk, piv in instances(K):
        wl = inputs.tiny(fam, batch=2, heads=2, dk=K, dv=V, rank=R, window=W, steps=W + 3, io=io)
        print(f"[case] {fam} K={K} V={V} r={R} W={W} io={io} sketch={sk} pivots={piv}", flush=True)
        run, layer, S_sel, heads, (om, C) = run_workload(wl, sketch=sk, pivots=piv)
        ref = oracle_of(wl, run, S_sel, heads, om, C, W, sketch=sk, pivots=piv)
        n = wl.batch * wl.heads
        S_gpu = to_np32(layer.state().reshape(n, V, K))
        U_gpu = to_np32(layer.sketch_matrix().reshape(n, V, R))
        rep = parity_report(run.o_gpu, ref.o, S_gpu, ref.S_final, U_gpu, ref.U_final)
        print("  " + format_report(rep), flush=True)
        bad = parity_failures(rep, *bars(io, sk, piv))
        if bad:
            failures.append(f"r={R} W={W} io={io} sketch={sk} pivots={piv}: " + "; ".join(bad))
    assert not failures, "\n".join(failures)


@pytest.mark.parametrize("fam", ["mamba2", "gdn", "kda"])
@pytest.mark.parametrize("K,V", [(64, 64), (128, 64), (128, 128)])
def test_every_compiled_baseline_instance(fam, K, V):
    """The exact baseline's instances: the full-state read and its rank-0
    flush for both window classes, and the single-token update (window 1),
    for both io dtypes, against the oracle's exact windowed read."""
    failures = []
    for W in (1, 7, 20):
        for io in ("f32", "bf16"):
            wl = inputs.tiny(fam, batch=2, heads=2, dk=K, dv=V, rank=8, window=W, steps=W + 3, io=io)
            print(f"[case] baseline {fam} K={K} V={V} W={W} io={io}", flush=True)
            run, layer, S_sel, heads, (om, C) = run_workload(wl, baseline=True)
            ref = oracle_of(wl, run, S_sel, heads, om, C, W)
            n = wl.batch * wl.heads
            rep = parity_report(run.o_gpu, ref.o_exact_windowed, to_np32(layer.state().reshape(n, V, K)), ref.S_final)
            print("  " + format_report(rep), flush=True)
            bad = parity_failures(rep, *bars(io, "f32"))
            if bad:
                failures.append(f"W={W} io={io}: " + "; ".join(bad))
    assert not failures, "\n".join(failures)


@pytest.mark.parametrize("fam", ["mamba2", "gdn", "kda"])
@pytest.mark.parametrize("K,V", [(64, 64), (128, 64), (128, 128)])
def test_every_compiled_dense_fallback_instance(fam, K, V):
    """The decode instances compiled with the exact read of dense-fallback
    heads (launched for rank tables that have such heads): one head at the
    full storage width and one dense head, for every width, window class,
    storage and map, each head against its own oracle run."""
    from test_gpu_ragged import check_ragged
    for R in (8, 16, 32):
        for W in (7, 20):
            for io, sk in STORAGE:
                for piv in (0, 4, -1):
                    if piv == -1 and R not in (8, 16):
                        continue
                    wl = inputs.tiny(fam, batch=2, heads=2, dk=K, dv=V, rank=R, window=W, steps=W + 3, io=io)
                    check_ragged(wl, [R, 0], sketch=sk, pivots=piv)

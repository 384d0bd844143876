"""The parity bars catch single-item and single-channel mistakes (CPU only).

The GPU parity tests compare the kernels' outputs with the oracle through
harness.parity_report / parity_failures.  Here a stand-in for a GPU output
is made on the host from the oracle's own output (a float32 copy with
fp32-level noise), and mistakes are planted in that copy: one value channel
of one item at one step off by 10 %, one item's whole output off by 0.6 %, one
item's state or sketch off by 1 %.  Over a sampled batch the aggregate
(headline) relative L2 can stay under the bf16 bar for these, so each must
be caught by the per-item bars, whatever the storage dtype (with fp32
storage the tighter aggregate bar sees them as well).  No GPU is used.
"""
import numpy as np
import pytest

import oracle
from harness import bars, item_err, parity_failures, parity_report

from paper_2609_33051_amd import inputs


@pytest.fixture(scope="module")
def run():
    wl = inputs.tiny("gdn", batch=16, heads=3, dk=64, dv=64, rank=8, window=4, steps=6, io="bf16")
    om, C = inputs.omega(wl)
    S0 = inputs.initial_state(wl).reshape(wl.items, wl.dv, wl.dk).numpy()
    steps = [inputs.step_inputs(wl, t) for t in range(wl.steps)]

    def stack(key, width):
        return np.stack([s[key].float().reshape(wl.items, width).numpy() for s in steps])

    q, k, v = stack("q", wl.dk), stack("k", wl.dk), stack("v", wl.dv)
    beta, ld = stack("beta", 1)[..., 0], stack("log_decay", 1)[..., 0]
    heads = (np.arange(wl.items) % wl.heads).astype(np.int32)
    ref = oracle.sketchssm(wl.kind, wl.window, heads, om, C, S0, q, k, v, beta, ld, round_storage=True)
    rng = np.random.default_rng(5)

    def near(x):  # a result that agrees with the oracle to fp32 rounding
        x = np.asarray(x, np.float64)
        return (x * (1 + 1e-7 * rng.standard_normal(x.shape))).astype(np.float32)

    return ref, near(ref.o), near(ref.S_final), near(ref.U_final)


@pytest.mark.parametrize("io,sketch,pivots", [("f32", "f32", 0), ("bf16", "f32", 0), ("bf16", "f32", 4),
                                             ("bf16", "bf16", 0)])
def test_close_result_passes(run, io, sketch, pivots):
    ref, o, S, U = run
    rep = parity_report(o, ref.o, S, ref.S_final, U, ref.U_final)
    assert parity_failures(rep, *bars(io, sketch, pivots)) == []


@pytest.mark.parametrize("io,sketch", [("bf16", "f32"), ("bf16", "bf16")])
def test_one_channel_of_one_item_off_by_ten_percent(run, io, sketch):
    ref, o, S, U = run
    bad = o.copy()
    t, i = 3, 17
    c = int(np.argsort(np.abs(ref.o[t, i]))[ref.o.shape[2] // 2])  # a channel of typical size
    bad[t, i, c] = ref.o[t, i, c] * 1.1
    rep = parity_report(bad, ref.o, S, ref.S_final, U, ref.U_final)
    head, item = bars(io, sketch)
    if sketch == "bf16":  # under the bf16 bar the aggregate alone does not see it: the point of the per-item bar
        assert rep["o_step"] <= head
    assert rep["o_item"] > item, "the per-item bar catches it whatever the storage"
    assert any(f.startswith("o_item") for f in parity_failures(rep, head, item))


@pytest.mark.parametrize("io,sketch", [("bf16", "f32"), ("bf16", "bf16")])
def test_one_item_off_by_a_little_over_half_a_percent(run, io, sketch):
    ref, o, S, U = run
    bad = o.copy()
    sizes = np.linalg.norm(ref.o, axis=-1).mean(axis=0)
    i = int(np.argsort(sizes)[len(sizes) // 2])  # an item of typical size
    bad[:, i] = ref.o[:, i] * 1.006
    rep = parity_report(bad, ref.o, S, ref.S_final, U, ref.U_final)
    head, item = bars(io, sketch)
    if sketch == "bf16":
        assert rep["o_step"] <= head
    assert any(f.startswith("o_item") for f in parity_failures(rep, head, item))


@pytest.mark.parametrize("field", ["S", "U"])
def test_one_item_state_or_sketch_off(run, field):
    ref, o, S, U = run
    S2, U2 = S.copy(), U.copy()
    if field == "S":
        S2[9] = ref.S_final[9] * 1.01
    else:
        U2[9, :, 2] = ref.U_final[9, :, 2] * 1.05
    rep = parity_report(o, ref.o, S2, ref.S_final, U2, ref.U_final)
    fails = parity_failures(rep, *bars("bf16", "bf16"))
    assert any(f.startswith(field + "_item") for f in fails)


def test_item_err_is_per_item_against_the_typical_item():
    b = np.ones((2, 3, 4))
    b[:, 1] *= 1e-3          # a small item: its rounding-sized error must not look large
    a = b.copy()
    a[1, 2, 0] += 0.5        # one value of one item at step 1
    a[0, 1, 0] += 1e-6
    r = item_err(a, b)
    assert r.shape == (2, 3)
    typ = np.sqrt((2 * 4 + 4e-6) / 3)
    assert np.isclose(r[1, 2], 0.5 / typ) and r[1, 0] == 0.0
    assert np.isclose(r[0, 1], 1e-6 / typ)

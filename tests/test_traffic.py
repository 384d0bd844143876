"""The byte accounting reproduces the paper's printed traffic reductions."""
import csv
import os

import pytest

from paper_2609_33051_amd import traffic

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "traffic_reduction.csv")


def rows():
    with open(GOLDEN) as f:
        return list(csv.DictReader(line for line in f if not line.startswith("#")))


@pytest.mark.parametrize("row", rows(), ids=lambda r: f"{r['model']}-G{r['G']}")
def test_reduction_matches_printed_tables(row):
    K, V, e, W, G = (int(row[x]) for x in ("K", "V", "e", "W", "G"))
    assert round(traffic.paper_reduction(K, V, G, W, e), 2) == pytest.approx(float(row["printed"]), abs=1e-9)


def test_replay_reduction_printed():
    # Appendix "State Memory Traffic Reduction": 32/17 = 1.88x at W = 16
    assert round(traffic.paper_replay_reduction(16), 2) == 1.88


def test_reduction_limits():
    # G -> 0 leaves only the flush: reduction W; a sketch as large as the state is worse than ReplaySSM
    assert traffic.paper_reduction(128, 64, 0, 16, 0) == pytest.approx(16.0)
    assert traffic.paper_reduction(128, 64, 128, 16, 0) < traffic.paper_replay_reduction(16) * 1.5


def test_algorithmic_bytes_mamba2_decode():
    # Mamba-2 decode layer, bf16 io, fp32 U: per item the query (256 B), slots
    # 0..n of the ring (392 B each: k, v, beta, log decay), U (4 KiB) and o (256 B)
    s = traffic.Shape("mamba2", 128, 64, 16, 16, 2)
    wb = traffic.window_bytes(s)
    assert len(wb["nonflush"]) == 15
    assert traffic.decode_bytes(s, 0) == 256 + 392 + 4096 + 256
    assert wb["nonflush_mean"] == pytest.approx(256 + 8 * 392 + 4096 + 256)
    assert traffic.full_read_bytes(s, 0) - traffic.decode_bytes(s, 0) == 4 * 128 * 64 - 4 * 64 * 16


def test_algorithmic_bytes_gdn_decode():
    s = traffic.Shape("gdn", 128, 128, 16, 16, 2)
    # slot 0: q 256, current k, v 512 + beta 4 + log decay 4, derived f 64, U 8 KiB, o 512
    assert traffic.decode_bytes(s, 0) == 256 + 520 + 64 + 8192 + 512
    # each earlier slot adds raw k, v 512 + beta 4 + log decay 4 + f 64 = 584; from 2 to 3 earlier
    # slots the T^{-1} row reads grow from 1 + 0 to 2 + 1 + 0 values (8 B) and the stored row by 4 B
    assert traffic.decode_bytes(s, 3) - traffic.decode_bytes(s, 2) == 584 + 8 + 4


def test_ragged_bytes_reduce_to_the_uniform_and_dense_cases():
    T = traffic
    s = T.Shape("gdn", 128, 128, 16, 16, 2)
    for n in (0, 5, 14):
        # a full-width table is the uniform sketch read; an all-dense one the exact full read
        assert T.ragged_decode_bytes(s, n, [16, 16, 16]) == 3 * T.decode_bytes(s, n)
        assert T.ragged_decode_bytes(s, n, [0, 0]) == 2 * T.full_read_bytes(s, n)
        # a rank-5 head stores two fp32 panels (8 columns) of U and 5 f entries per slot
        sg = T.Shape("gdn", 128, 128, 5, 16, 2)
        assert T.ragged_decode_bytes(s, n, [5]) == T.decode_bytes(sg, n) + 4 * 128 * 3
    assert T.panel_cols(s, 5) == 8 and T.panel_cols(T.Shape("gdn", 128, 128, 16, 16, 2, 2), 5) == 8
    assert T.panel_cols(T.Shape("gdn", 128, 128, 16, 16, 2, 2), 9) == 16
    assert T.ragged_flush_bytes(s, 15, [16, 0]) == T.flush_bytes(s, 15) + T.flush_bytes(s, 15, 0)
    # with a state-dependent map a head stores the map rows below its rank: r x K at full width, g x K below it
    sm = T.Shape("gdn", 128, 128, 16, 16, 2, 2, pivots=4)
    assert T.ragged_flush_bytes(sm, 15, [16]) == T.flush_bytes(sm, 15)
    assert T.ragged_flush_bytes(sm, 15, [5]) == T.flush_bytes(sm, 15, 8) - 2 * (16 - 5) * 128
    # and reads those rows (its U up to the next whole bf16 panel: 8 columns)
    assert T.ragged_decode_bytes(sm, 3, [5]) == T.decode_bytes(T.Shape("gdn", 128, 128, 5, 16, 2, 2, pivots=4), 3) + 2 * 128 * 3


def test_bf16_storage_halves_f_and_the_map():
    """With the paper's storage the sketch, f and the state-dependent map are
    2-byte values, and the map a non-flush read takes is the dense G x K
    matrix: the 2GK bytes of T_G = 2G(V + K + eW) (state memory traffic
    appendix), beside the 2GV of the sketch."""
    T = traffic
    f32 = T.Shape("gdn", 128, 128, 16, 16, 2, 4, 4)
    b16 = T.Shape("gdn", 128, 128, 16, 16, 2, 2, 4)
    off = T.Shape("gdn", 128, 128, 16, 16, 2, 2, 0)
    assert b16.cmap_bytes == 2 * 16 * 128 and f32.cmap_bytes == 2 * b16.cmap_bytes and off.cmap_bytes == 0
    for n in (0, 7):
        assert T.decode_bytes(b16, n) - T.decode_bytes(off, n) == 2 * 16 * 128
    assert T.slot_read_bytes(f32) - T.slot_read_bytes(b16) == 2 * 16
    assert T.derived_write_bytes(f32, 5) - T.derived_write_bytes(b16, 5) == 2 * 16
    # the exact baseline keeps pi in fp32 whatever the sketch storage
    assert T.slot_read_bytes(f32, True) == T.slot_read_bytes(b16, True)


def test_profile_summary_reads_kernel_variants():
    """The profile summaries key each kernel-trace entry by entry point, sketch
    dtype and pivot count, read from the kernel's template arguments."""
    from paper_2609_33051_amd.profile_summary import kernel_variant
    assert kernel_variant("decode_kernel<1, 128, 128, 16, 16, unsigned short, unsigned short, 4, false>") == \
        ("decode", "bf16", 4)
    assert kernel_variant("decode_kernel<0, 128, 64, 16, 16, unsigned short, float, 0, true>") == ("decode", "f32", 0)
    assert kernel_variant("update_kernel<2, 128, 128, 16, 16, unsigned short, unsigned short, 0>") == \
        ("update", "bf16", 0)
    assert kernel_variant("full_read_kernel<1, 128, 128, 16, unsigned short>") == ("full_read", "f32", 0)
    assert kernel_variant("state_layout_kernel") is None

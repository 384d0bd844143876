"""The C-ABI library loads, exports every function its header declares, and
rejects invalid calls on the host before anything is enqueued.

No compute call is made here.  Every invalid call below carries a defect the
host validation reports; the fake device addresses used are never launched
on.  (The cases are skipped where a GPU is visible, so that a validation bug
could never turn into a launch on bogus addresses.)
"""
import ctypes
import os
import re

import pytest

from paper_2609_33051_amd import binding as B
from paper_2609_33051_amd import build as builder

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "sketchssm.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        builder.build()
    return B.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sketchssm_\w+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for f in ("sketchssm_update", "sketchssm_decode", "sketchssm_full_read_baseline"):
        assert f in names
    assert set(names) == set(B.FUNCTIONS)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = os.popen(f"nm -D --defined-only {B.LIB_PATH}").read()
    for name in declared_functions():
        assert re.search(rf"\bT {name}\b", out), name


def test_status_strings(lib):
    assert B.sketchssm_status_string(0) == "ok"
    assert "aligned" in B.sketchssm_status_string(-3)
    assert B.sketchssm_status_string(12345) == "unknown status"


def _gpu_visible():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


ADDR = 1 << 20  # a 16-byte aligned fake address, never dereferenced (every case fails validation)


def cfg(**kw):
    d = dict(kind="mamba2", batch=2, heads=4, dk=128, dv=64, rank=16, window=16, io="bf16", sketch="f32", pivots=0,
             ridge=0.1, head_ranks=None)
    d.update(kw)
    return B.make_config(d["kind"], d["batch"], d["heads"], d["dk"], d["dv"], d["rank"], d["window"], d["io"],
                         d["sketch"], d["pivots"], d["ridge"], head_ranks=d["head_ranks"])


def good_ring(**kw):
    d = dict(k=ADDR, v=ADDR, beta=ADDR, log_decay=ADDR, f=ADDR, pi=ADDR, tinv=ADDR)
    d.update(kw)
    return B.make_ring(**d)


def status(fn, *args):
    try:
        fn(*args)
    except B.SketchSSMError as e:
        return e.status
    return 0


@pytest.mark.skipif(_gpu_visible(), reason="host-validation cases use fake addresses; run on CPU only")
class TestValidation:
    def test_decode_rejections(self, lib):
        d = B.sketchssm_decode
        assert check_config_ok(lib)
        assert status(d, cfg(kind=7), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -1
        assert status(d, cfg(dk=96), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -2
        assert status(d, cfg(rank=12), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -2
        assert status(d, cfg(window=33), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -2
        assert status(d, cfg(window=1), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -1
        assert status(d, cfg(), ADDR, ADDR, good_ring(), 15, ADDR, ADDR) == -4
        assert status(d, cfg(), ADDR, ADDR, good_ring(), -1, ADDR, ADDR) == -4
        assert status(d, cfg(), ADDR + 4, ADDR, good_ring(), 0, ADDR, ADDR) == -3
        assert status(d, cfg(), ADDR, ADDR, good_ring(), 0, ADDR + 8, ADDR) == -3
        assert status(d, cfg(), ADDR, ADDR, good_ring(v=None), 0, ADDR, ADDR) == -1
        assert status(d, cfg(), ADDR, ADDR, good_ring(log_decay=ADDR + 4), 0, ADDR, ADDR) == -3
        assert status(d, cfg(kind="kda", dv=128), ADDR, ADDR, good_ring(tinv=None), 0, ADDR, ADDR) == -1
        assert status(d, cfg(), ADDR, ADDR, good_ring(), 0, None, ADDR) == -1
        assert status(d, cfg(kind="gdn", dv=128), ADDR, ADDR, good_ring(f=None), 0, ADDR, ADDR) == -1
        assert status(d, cfg(), None, ADDR, good_ring(), 0, ADDR, ADDR) == -1
        assert status(d, cfg(batch=0), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -1
        assert status(d, cfg(io=5), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -1
        assert status(d, cfg(sketch=3), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -1
        assert "sketch_dtype" in B.sketchssm_last_error()
        # state-dependent coefficient map: P = 4 only, rank 8..32, a 16-byte aligned cmap, ridge > 0
        assert status(d, cfg(pivots=3), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -2
        # the exact-metric map (pivots = -1) is compiled for ranks 8 and 16
        assert status(lambda *x: B.sketchssm_decode(*x, cmap=ADDR), cfg(pivots=-1, rank=32), ADDR, ADDR,
                      good_ring(), 0, ADDR, ADDR) == -2
        assert "exact" in B.sketchssm_last_error()
        assert status(d, cfg(pivots=-2), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -2
        assert status(d, cfg(pivots=4, rank=128), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -2
        assert status(d, cfg(pivots=4), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -1  # no cmap
        assert status(lambda *x: B.sketchssm_decode(*x, cmap=ADDR + 4), cfg(pivots=4), ADDR, ADDR, good_ring(), 0,
                      ADDR, ADDR) == -3
        assert status(d, cfg(pivots=4, ridge=-1.0), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -1
        # lambda = 0 would leave D = d + lambda singular where d = 0 (a zero state, columns past a head's rank)
        assert status(lambda *x: B.sketchssm_decode(*x, cmap=ADDR), cfg(pivots=4, ridge=0.0), ADDR, ADDR,
                      good_ring(), 0, ADDR, ADDR) == -1
        assert "ridge" in B.sketchssm_last_error()
        # with the offline map the caller's coef is required; with a state-dependent map it is not read
        assert status(d, cfg(), ADDR, None, good_ring(), 0, ADDR, ADDR) == -1
        assert "coef" in B.sketchssm_last_error()
        assert "n_buffered" in B.sketchssm_status_string(-4)

    def test_state_layout_rejections(self, lib):
        t, f = B.sketchssm_state_to_tiles, B.sketchssm_state_from_tiles
        big = ADDR + (1 << 24)   # past the 2*4*64*128*4-byte state at ADDR
        assert status(t, cfg(), None, big) == -1
        assert status(f, cfg(), ADDR, None) == -1
        assert status(t, cfg(), ADDR + 4, big) == -3
        assert status(t, cfg(), ADDR, ADDR + 4096) == -1          # overlapping ranges
        assert "overlap" in B.sketchssm_last_error()
        assert status(f, cfg(dk=96), ADDR, big) == -2
        assert status(t, cfg(batch=0), ADDR, big) == -1

    def test_update_rejections(self, lib):
        u = B.sketchssm_update
        assert status(u, cfg(), ADDR, ADDR, good_ring(), 16, ADDR, ADDR, ADDR) == -4
        assert status(u, cfg(), ADDR, ADDR, None, 3, None, ADDR, None) == -4          # sketch-only needs n = 0
        assert status(u, cfg(), ADDR, ADDR, good_ring(), 3, ADDR + 4, ADDR, None) == -3  # misaligned query
        assert status(u, cfg(rank=0), ADDR, None, None, 0, None, None, None) == -1   # sketch-only needs rank
        assert status(u, cfg(), None, ADDR, good_ring(), 15, ADDR, ADDR, ADDR) == -1
        assert status(u, cfg(), ADDR, None, good_ring(), 15, ADDR, ADDR, ADDR) == -1
        assert status(u, cfg(kind="kda", dv=128), ADDR, ADDR, good_ring(tinv=None), 15, ADDR, ADDR, ADDR) == -1
        assert status(u, cfg(), ADDR, ADDR, None, 15, ADDR, ADDR, ADDR) == -1  # ring needed when n > 0
        assert status(u, cfg(), ADDR, ADDR, good_ring(), 15, ADDR, ADDR, ADDR + 2) == -3
        assert status(u, cfg(sketch=-1), ADDR, ADDR, good_ring(), 15, ADDR, ADDR, ADDR) == -1
        assert status(u, cfg(pivots=4), ADDR, ADDR, good_ring(), 15, ADDR, ADDR, ADDR) == -1  # no cmap
        assert status(u, cfg(pivots=4, rank=0), ADDR, None, good_ring(), 15, ADDR, None, ADDR) == -2
        assert status(lambda *x: u(*x, cmap=ADDR), cfg(pivots=4, ridge=0.0), ADDR, ADDR, good_ring(), 15, ADDR, ADDR,
                      ADDR) == -1

    def test_full_read_rejections(self, lib):
        f = B.sketchssm_full_read_baseline
        assert status(f, cfg(kind="gdn", dv=128), ADDR, good_ring(pi=None), 0, ADDR, ADDR) == -1
        assert status(f, cfg(), ADDR, good_ring(), 15, ADDR, ADDR) == -4
        assert "n_buffered" in B.sketchssm_last_error()
        assert status(f, cfg(), None, good_ring(), 0, ADDR, ADDR) == -1
        assert status(f, cfg(dv=32), ADDR, good_ring(), 0, ADDR, ADDR) == -2

    def test_head_rank_table(self, lib):
        """Per-head rank tables are validated on the host; calls with nothing to
        do for their path return OK without a launch."""
        d, f, u = B.sketchssm_decode, B.sketchssm_full_read_baseline, B.sketchssm_update
        ok = [16, 0, 5, 8]
        assert status(d, cfg(head_ranks=[16, 0, 17, 8]), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -1
        assert "head_rank[2]" in B.sketchssm_last_error()
        assert status(d, cfg(head_ranks=[16, -1, 4, 8]), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -1
        assert status(d, cfg(rank=128, head_ranks=ok), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -2
        assert status(u, cfg(rank=0, head_ranks=[0, 0, 0, 0]), ADDR, None, good_ring(), 15, ADDR, None, ADDR) == -2
        assert status(f, cfg(rank=0, head_ranks=[0, 0, 0, 0]), ADDR, good_ring(), 0, ADDR, ADDR) == -2
        many = 300
        assert status(d, cfg(heads=many, head_ranks=[8] * many), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -2
        # dense-fallback heads are read from S by the decode: S (and, GDN/KDA, ring pi) required
        assert status(d, cfg(head_ranks=[0, 4, 0, 0]), ADDR, ADDR, good_ring(), 0, ADDR, ADDR) == -1
        assert "dense-fallback" in B.sketchssm_last_error()
        assert status(lambda *x: d(*x, S=ADDR + 4), cfg(head_ranks=[0, 4, 0, 0]), ADDR, ADDR, good_ring(), 0,
                      ADDR, ADDR) == -3
        assert status(lambda *x: d(*x, S=ADDR), cfg(kind="gdn", dv=128, head_ranks=[0, 4, 0, 0]), ADDR, ADDR,
                      good_ring(pi=None), 0, ADDR, ADDR) == -1
        # a sketch-only update with every head dense has nothing to build: OK without a launch
        assert status(u, cfg(head_ranks=[0, 0, 0, 0]), ADDR, ADDR, None, 0, None, ADDR, None) == 0
        # the rest of the validation still applies with a table
        assert status(d, cfg(head_ranks=[0, 0, 0, 0]), ADDR, ADDR, good_ring(), 15, ADDR, ADDR) == -4


def check_config_ok(lib):
    return B.sketchssm_check_config(cfg()) == 0 and B.sketchssm_check_config(cfg(rank=5)) == -2


def test_item_count_limit(lib):
    """B*H < 2^23: one slot of a derived ring field (up to 512 bytes per item)
    then spans less than 4 GiB, the range of the kernels' 32-bit slot strides."""
    assert B.sketchssm_check_config(cfg(batch=(1 << 23) - 1, heads=1)) == 0
    assert B.sketchssm_check_config(cfg(batch=1 << 22, heads=2)) == -2
    assert "items" in B.sketchssm_last_error()
    assert B.sketchssm_check_config(cfg(batch=1 << 20, heads=1 << 12)) == -2


def test_head_rank_table_marshalling():
    c = B.make_config("gdn", 2, 3, 128, 128, 16, 16, "bf16", head_ranks=[16, 0, 7])
    assert B.head_ranks(c) == [16, 0, 7]
    assert B.head_ranks(B.make_config("gdn", 2, 3, 128, 128, 16, 16, "bf16")) is None
    with pytest.raises(ValueError):
        B.make_config("gdn", 2, 3, 128, 128, 16, 16, "bf16", head_ranks=[16, 0])

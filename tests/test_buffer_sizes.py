"""The sizes query of the C ABI (sketchssm_buffer_sizes, sketchssm_ring_bytes)
against the layouts the header defines, for every family, dtype, map and
rank-table case, and the layer's allocations against the query.  CPU only:
no kernel is launched (the layer is built on the host without a state)."""
import itertools

import pytest
import torch

from paper_2609_33051_amd import binding as B
from paper_2609_33051_amd.layer import SketchSSMLayer


@pytest.fixture(scope="module", autouse=True)
def lib():
    from paper_2609_33051_amd import build as builder
    import os
    if not os.path.exists(B.LIB_PATH):
        builder.build()
    return B.load()


def expected(kind, Bt, H, K, V, r, W, io, sk, pivots, baseline, ranks):
    """Bytes per buffer, restated from the layouts in include/sketchssm.h."""
    iob, skb = (2 if io == "bf16" else 4), (2 if sk == "bf16" else 4)
    r = 0 if baseline else r
    erase = kind != "mamba2"
    dense = ranks is not None and 0 in ranks
    sketched = ranks is None or any(g > 0 for g in ranks)
    return {
        "S": Bt * H * V * K * 4, "U": Bt * H * V * r * skb, "omega": H * K * r * 4,
        "coef": 0 if pivots else H * r * K * 4, "cmap": Bt * H * r * K * skb if pivots and not baseline else 0,
        "q": Bt * H * K * iob, "o": Bt * H * V * 4,
        "ring_k": Bt * H * W * K * iob, "ring_v": Bt * H * W * V * iob, "ring_beta": Bt * H * W * 4,
        "ring_log_decay": Bt * H * W * (K if kind == "kda" else 1) * 4,
        "ring_f": W * H * Bt * r * skb if erase and not baseline and sketched else 0,
        "ring_pi": W * H * Bt * K * 4 if erase and (baseline or dense) else 0,
        "ring_tinv": W * H * Bt * W * 4 if erase else 0,
    }


CASES = list(itertools.product(["mamba2", "gdn", "kda"], ["f32", "bf16"], ["f32", "bf16"], [0, 4],
                               [False, True], [None, [16, 0, 5]]))


@pytest.mark.parametrize("kind,io,sk,pivots,baseline,ranks", CASES)
def test_sizes_follow_the_header_layouts(kind, io, sk, pivots, baseline, ranks):
    Bt, H, K, V, r, W = 5, 3, 128, (64 if kind == "mamba2" else 128), 16, 16
    cfg = B.make_config(kind, Bt, H, K, V, 0 if baseline else r, W, io, sk, 0 if baseline else pivots, 0.1,
                        head_ranks=None if baseline else ranks)
    got = B.sketchssm_buffer_sizes(cfg, baseline)
    want = expected(kind, Bt, H, K, V, r, W, io, sk, 0 if baseline else pivots, baseline, None if baseline else ranks)
    assert got == want
    assert B.sketchssm_ring_bytes(cfg, baseline) == sum(v for k, v in want.items() if k.startswith("ring_"))


@pytest.mark.parametrize("kind,io,sk,pivots,baseline,ranks", [c for c in CASES if c[1] == "bf16"])
def test_layer_allocates_what_the_library_reports(kind, io, sk, pivots, baseline, ranks):
    Bt, H, K, V, r, W = 5, 3, 128, (64 if kind == "mamba2" else 128), 16, 16
    om = torch.zeros((H, K, r))
    lay = SketchSSMLayer(kind, Bt, H, K, V, r, W, io, "cpu", baseline=baseline, omega=om,
                         coef=om.transpose(1, 2).contiguous(), sketch=sk, pivots=pivots, head_ranks=ranks)
    size = B.sketchssm_buffer_sizes(lay.cfg, baseline)
    held = {"S": lay.S, "U": lay.U, "cmap": lay.cmap, "ring_k": lay.rk, "ring_v": lay.rv, "ring_beta": lay.rbeta,
            "ring_log_decay": lay.rla, "ring_f": lay.rf, "ring_pi": lay.rpi, "ring_tinv": lay.rt, "o": lay.o}
    for name, t in held.items():
        nbytes = 0 if t is None else t.numel() * t.element_size()
        assert nbytes == size[name], name


def test_sizes_reject_what_the_calls_reject():
    assert B.sketchssm_ring_bytes(B.make_config("gdn", 2, 3, 96, 128, 16, 16, "bf16"), False) == 0
    with pytest.raises(B.SketchSSMError):
        B.sketchssm_buffer_sizes(B.make_config("gdn", 2, 3, 128, 128, 12, 16, "bf16"))
    with pytest.raises(B.SketchSSMError):
        B.sketchssm_buffer_sizes(B.make_config("gdn", 2, 3, 128, 128, 16, 16, "bf16", head_ranks=[16, 17, 0]))
    # the baseline layer ignores the rank
    assert B.sketchssm_ring_bytes(B.make_config("gdn", 2, 3, 128, 128, 12, 16, "bf16"), True) > 0


@pytest.mark.parametrize("K,R,skb", [(k, r, s) for k in (64, 128) for r in (8, 16, 32) for s in (4, 2)])
def test_map_panel_indices_stay_in_the_item(K, R, skb):
    """The dense map's index arithmetic, replayed on the host for one item:
    element (j, k) sits at ((k / c) * R + j) * c + k % c, c = 16 / skb.  The
    flush's stores (P = 4: four channels k0 .. k0 + 3 of row j from lane
    (j mod 16, k0 / 4 mod 4) of k tile k0 / 16; exact map: thread t writes
    panel t) cover rows j < G exactly once, and decode's loads (lane row rho,
    column j0 = lane mod 16, map row j = j0 + 16 p clamped to 0 at and past the
    head's rank G, panels rho * K / (4c) + i) stay below R * K for every G and
    read element (j, k) for the channels k the lane multiplies."""
    c = 16 // skb
    RP, CL, KQ = (R + 15) // 16, K // 4 // c, K // 4

    def at(j, k):
        return ((k // c) * R + j) * c + k % c

    for G in sorted({1, R // 2, R - 1, R}):
        pivot = []
        for kt in range(K // 16):
            for jt in range(RP):
                for lane in range(64):
                    j, k0 = 16 * jt + lane % 16, 16 * kt + 4 * (lane // 16)
                    if j < G:
                        base = ((k0 // c) * R + j) * c + k0 % c
                        pivot += [base + e for e in range(4)]
                        assert [base + e for e in range(4)] == [at(j, k0 + e) for e in range(4)]
        exact = [t * c + e for t in range(R * K // c) if t % R < G for e in range(c)]
        want = sorted(at(j, k) for j in range(G) for k in range(K))
        assert sorted(pivot) == want and sorted(exact) == want
        for lane in range(64):
            rho, j0 = lane // 16, lane % 16
            for p in range(RP):
                j = j0 + 16 * p
                jj = j if j < G else 0
                for i in range(CL):
                    first = ((rho * CL + i) * R + jj) * c
                    assert 0 <= first and first + c <= R * K
                    if j < G:
                        assert [first + e for e in range(c)] == [at(j, rho * KQ + i * c + e) for e in range(c)]

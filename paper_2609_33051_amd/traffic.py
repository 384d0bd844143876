"""Byte accounting for the decode path.

Two models live here.

paper_* -- the paper's state-memory traffic model (Appendix "State Memory
Traffic Reduction", Table tab:m-traffic): per state head per decode step,
Standard reads and writes the fp32 state (8KV bytes); ReplaySSM reads it every
step and writes it every W steps; SketchSSM reads a bf16 sketch, coefficient
map and (delta-rule families) projected erase vectors between flushes,
T_G = 2G(V + K + eW), and reads and writes the state once per window.  Ring
buffer traffic is excluded there.

algorithmic_* -- the bytes this implementation's kernels must move per
(request, head) item, ring buffer included (the ring is as large as the sketch
read at these shapes, so leaving it out would flatter the result).  Shared
per-head tensors (Omega, C) are amortised over the batch and not counted.
These are the numerators of the reported HBM roofline fractions.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, published peak


def paper_state_bytes(K: int, V: int) -> float:
    """D = 4KV: the fp32 state of one head."""
    return 4.0 * K * V


def paper_sketch_read_bytes(K: int, V: int, G: float, W: int, e: int) -> float:
    """T_G = 2G(V + K + eW): bf16 U, C and (e = 1) projected erase vectors."""
    return 2.0 * G * (V + K + e * W)


def paper_sketchssm_avg_read(K: int, V: int, G: float, W: int, e: int) -> float:
    """B_G = ((W - 1) T_G + D) / W."""
    return ((W - 1) * paper_sketch_read_bytes(K, V, G, W, e) + paper_state_bytes(K, V)) / W


def paper_reduction(K: int, V: int, G: float, W: int, e: int) -> float:
    """R_G = 8KV / ((W - 1) T_G / W + 8KV / W), reduction relative to Standard."""
    return 8.0 * K * V / ((W - 1) * paper_sketch_read_bytes(K, V, G, W, e) / W + 8.0 * K * V / W)


def paper_replay_reduction(W: int) -> float:
    """ReplaySSM: (D + D) / (D + D/W) = 2W / (W + 1)."""
    return 2.0 * W / (W + 1)


@dataclass(frozen=True)
class Shape:
    kind: str      # "mamba2" | "gdn" | "kda"
    dk: int
    dv: int
    rank: int
    window: int
    io_bytes: int  # 2 (bf16) or 4 (fp32)
    sketch_bytes: int = 4  # U element: 4 (fp32) or 2 (bf16)
    pivots: int = 0        # state-dependent coefficient map with this many pivots (0: offline map)

    @property
    def erase(self) -> bool:
        return self.kind in ("gdn", "kda")

    @property
    def cmap_bytes(self) -> int:
        """The per-item state-dependent map C (r x K), stored like U: the 2GK
        bytes of T_G with the paper's BF16 storage."""
        return self.sketch_bytes * self.rank * self.dk if self.pivots else 0

    @property
    def decay_bytes(self) -> int:
        """Per-token log decay / cumulative log decay: a scalar, or K values (KDA)."""
        return 4 * self.dk if self.kind == "kda" else 4


def slot_read_bytes(s: Shape, baseline: bool = False) -> int:
    """What a non-flush read takes from each earlier slot of the ring.

    Every kind: raw key and value, beta, log decay (K fp32 for KDA).
    GDN/KDA also: the projected erase vector f (r values stored like U,
    sketch read) or the erase factor pi (K fp32, exact baseline).  (The
    pseudo-values are solved from the raw values and the stored rows of
    T^{-1}, not stored.)"""
    raw = s.io_bytes * (s.dk + s.dv) + 4 + s.decay_bytes
    if not s.erase:
        return raw
    return raw + (4 * s.dk if baseline else s.sketch_bytes * s.rank)


def tinv_read_bytes(s: Shape, n: int) -> int:
    """GDN/KDA: the stored rows of T^{-1} (T = I + Diag(beta) B, B the
    couplings of eq. wy) of the n earlier slots (slot s holds s entries),
    which turn the buffer term into sums over the raw values."""
    return 2 * n * (n - 1) if s.erase else 0


def current_read_bytes(s: Shape) -> int:
    """The current token's raw inputs in ring slot n: k, v, beta, log decay."""
    return s.io_bytes * (s.dk + s.dv) + 4 + s.decay_bytes


def derived_write_bytes(s: Shape, n: int, baseline: bool = False) -> int:
    """Fields a read derives and stores for slot n: GDN/KDA f (or pi) and row
    n of T^{-1} (n entries).  Mamba-2: none."""
    if not s.erase:
        return 0
    extra = 4 * s.dk if baseline else s.sketch_bytes * s.rank
    return extra + 4 * n


def decode_bytes(s: Shape, n: int) -> int:
    """Sketch read at slot n: the query, n earlier slots, the current slot, the
    derived fields, U, the state-dependent map (if any) and o."""
    return (s.io_bytes * s.dk + n * slot_read_bytes(s) + current_read_bytes(s) + tinv_read_bytes(s, n)
            + derived_write_bytes(s, n) + s.sketch_bytes * s.dv * s.rank + s.cmap_bytes + 4 * s.dv)


def full_read_bytes(s: Shape, n: int) -> int:
    """Exact full-state read at slot n: as decode with S (4KV) in place of U."""
    return (s.io_bytes * s.dk + n * slot_read_bytes(s, True) + current_read_bytes(s) + tinv_read_bytes(s, n)
            + derived_write_bytes(s, n, True) + 4 * s.dk * s.dv + 4 * s.dv)


def flush_bytes(s: Shape, n_buffered: int, rank: int | None = None, map_rows: int | None = None) -> int:
    """Flush of the token in slot n_buffered: S read + write, the earlier
    slots (raw k, v, beta, log decay) and their rows of T^{-1}, the current
    slot, the query, the sketch write (rank columns), the state-dependent
    map's rows (if any; all r unless map_rows says fewer are stored) and o."""
    r = s.rank if rank is None else rank
    cmap = s.cmap_bytes if map_rows is None else s.sketch_bytes * map_rows * s.dk * (1 if s.pivots else 0)
    slot = s.io_bytes * (s.dk + s.dv) + 4 + s.decay_bytes
    tinv = 4 * n_buffered * (n_buffered - 1) // 2 if s.erase else 0
    return (8 * s.dk * s.dv + n_buffered * slot + tinv + current_read_bytes(s) + s.io_bytes * s.dk
            + s.sketch_bytes * s.dv * r + (cmap if r else 0) + 4 * s.dv)


def init_bytes(s: Shape) -> int:
    """Sketch construction from S alone: S read + U write."""
    return 4 * s.dk * s.dv + s.sketch_bytes * s.dv * s.rank


def window_bytes(s: Shape, baseline: bool = False) -> dict:
    """Per-item bytes over one window: W-1 non-flush reads and one flush."""
    W = s.window
    reads = [full_read_bytes(s, n) if baseline else decode_bytes(s, n) for n in range(W - 1)]
    fl = flush_bytes(s, W - 1, 0 if baseline else None)
    return {"nonflush": reads, "flush": fl, "total": sum(reads) + fl,
            "nonflush_mean": (sum(reads) / len(reads)) if reads else 0.0}


def panel_cols(s: Shape, g: int) -> int:
    """Sketch columns a rank-g head stores: whole panels of 16 bytes per value."""
    P = 16 // s.sketch_bytes
    return -(-g // P) * P


def ragged_decode_bytes(s: Shape, n: int, ranks) -> int:
    """Non-flush read at slot n of one batch row (all heads) under a per-head
    rank table with storage width s.rank: a sketched head (g > 0) moves the
    decode bytes of rank g (its U up to the next whole panel); a dense head
    (g = 0) moves the exact full-read bytes."""
    tot = 0
    for g in ranks:
        if g == 0:
            tot += full_read_bytes(s, n)
        else:
            sg = replace(s, rank=g)
            tot += decode_bytes(sg, n) + s.sketch_bytes * s.dv * (panel_cols(s, g) - g)
    return tot


def ragged_flush_bytes(s: Shape, n_buffered: int, ranks) -> int:
    """Flush of one batch row under a per-head rank table: each head's state
    read and write, its sketch columns (whole panels; none for a dense head)
    and, with a state-dependent map, its map's rows below its rank (the rows
    past it are not stored)."""
    return sum(flush_bytes(s, n_buffered, panel_cols(s, g) if g else 0, g) for g in ranks)

"""Device buffers of one linear-attention layer and its decode loop
(Algorithm 1, inference part), on top of the C ABI.

torch supplies device memory and the stream; every computation is a call
into libsketchssm.so.  Buffers (caller-owned, as the ABI requires):

  S      B*H*V*K fp32 full state X = S^T in the library's tile-major layout
         (16 x 16 tiles, 1 KB each); the constructor takes a row-layout state
         [B][H][V][K] and converts it, state() returns that layout again
  U      [B][H][r/P][V][P] sketch U = S^T Omega in panels of 16 bytes per
         value: P = 4 columns fp32, or P = 8 bf16 (sketch="bf16", the paper's
         storage); sketch_matrix() gives the [B][H][V][r] fp32 view
  omega  [H][K][r]     fp32 sketching matrix, coef [H][r][K] its coefficient map
         (Omega^T, the offline map); with pivots != 0 the map is
         state-dependent, rebuilt at every flush into cmap (the dense r x K
         map per item in 16-byte channel panels), stored like U: fp32, or bf16
         with sketch="bf16"
  ring   replay buffer of W slots per item:
         raw inputs k, v (io dtype), beta, log_decay ([..][K] for KDA), item-major
         [B][H][W][...], written into slot n by the token's producer (write_token);
         derived fields, slot-major and head-major [W][H][B][...]: rows of T^{-1} (GDN/KDA),
         f (sketch read; stored like U) or pi (baseline).
  head_ranks  optional per-head rank table (allocation of Sec. 4.2): head h
         uses the first head_ranks[h] columns of the rank-r storage; 0 keeps the
         head dense (the sketch read reads its state exactly, in the same
         launch; the ring then holds both f and pi).
"""
from __future__ import annotations

import torch

from . import binding as B


class SketchSSMLayer:
    def __init__(self, kind: str, batch: int, heads: int, dk: int, dv: int, rank: int, window: int,
                 io: str = "bf16", device="cuda", baseline: bool = False, S: torch.Tensor | None = None,
                 omega: torch.Tensor | None = None, coef: torch.Tensor | None = None, sketch: str = "f32",
                 pivots: int = 0, ridge: float = 0.1, head_ranks=None):
        self.kind, self.batch, self.heads, self.dk, self.dv = kind, batch, heads, dk, dv
        self.rank, self.window, self.io, self.baseline, self.sketch = rank, window, io, baseline, sketch
        self.pivots = 0 if baseline else pivots
        self.device = torch.device(device)
        iodt = torch.bfloat16 if io == "bf16" else torch.float32
        f32 = torch.float32
        Bt, H, K, V, W = batch, heads, dk, dv, window
        dev = self.device
        r = 0 if baseline else rank
        self.head_ranks = None if (baseline or head_ranks is None) else [int(x) for x in head_ranks]
        self.dense_heads = 0 if self.head_ranks is None else sum(1 for x in self.head_ranks if x == 0)
        self.cfg = B.make_config(kind, Bt, H, K, V, r, W, io, sketch, self.pivots, ridge, head_ranks=self.head_ranks)
        # every buffer is sized by the library (sketchssm_buffer_sizes) and
        # viewed with the shape its layout defines
        size = B.sketchssm_buffer_sizes(self.cfg, baseline)
        skdt = torch.bfloat16 if sketch == "bf16" else f32  # sketch, f and map share the storage dtype

        def buf(name, dtype, shape):
            nbytes = size[name]
            if nbytes == 0:
                return None
            t = torch.zeros(nbytes // torch.tensor([], dtype=dtype).element_size(), dtype=dtype, device=dev)
            return t.view(shape)

        # the state in the kernels' tile-major layout (S, if given, is row layout [B][H][V][K])
        self.S = buf("S", f32, (Bt, H, V * K))
        if S is not None:
            rows = S.to(device=dev, dtype=f32).reshape(Bt, H, V, K).contiguous()
            B.sketchssm_state_to_tiles(self.cfg, rows, self.S, self.stream())
        if not baseline:
            self.omega = omega.to(dev).contiguous()
            self.coef = coef.to(dev).contiguous()
            P = 8 if sketch == "bf16" else 4
            self.U = buf("U", skdt, (Bt, H, rank // P, V, P))
        else:
            self.omega = self.coef = self.U = None
        # state-dependent coefficient map (r x K per item), written by every update
        self.cmap = buf("cmap", skdt, (Bt, H, rank * K))
        # raw inputs, written by the producer of each token
        self.rk = buf("ring_k", iodt, (Bt, H, W, K))
        self.rv = buf("ring_v", iodt, (Bt, H, W, V))
        self.rbeta = buf("ring_beta", f32, (Bt, H, W))
        self.rla = buf("ring_log_decay", f32, (Bt, H, W, K) if kind == "kda" else (Bt, H, W))
        # derived fields, written by the library
        self.rt = buf("ring_tinv", f32, (W, H, Bt, W))
        self.rf = buf("ring_f", skdt, (W, H, Bt, rank))
        self.rpi = buf("ring_pi", f32, (W, H, Bt, K))
        self.ring = B.make_ring(k=self.rk, v=self.rv, beta=self.rbeta, log_decay=self.rla, f=self.rf,
                                pi=self.rpi, tinv=self.rt)
        self.o = torch.zeros((Bt, H, V), dtype=f32, device=dev)
        self.n = 0  # slot of the next token in the current window

    def sketch_matrix(self) -> torch.Tensor:
        """The sketch as [B][H][V][r] (a copy; U itself is stored in panels)."""
        Bt, H, V, r = self.batch, self.heads, self.dv, self.rank
        return self.U.permute(0, 1, 3, 2, 4).reshape(Bt, H, V, r).float()

    @staticmethod
    def stream() -> int:
        return torch.cuda.current_stream().cuda_stream

    def state(self) -> torch.Tensor:
        """The state in row layout [B][H][V][K] (X = S^T, K contiguous), a copy."""
        rows = torch.empty((self.batch, self.heads, self.dv, self.dk), dtype=torch.float32, device=self.device)
        B.sketchssm_state_from_tiles(self.cfg, self.S, rows, self.stream())
        return rows

    def init_sketch(self):
        """U = S^T Omega from S alone (after prefill); empties the window."""
        self.n = 0
        if not self.baseline:
            B.sketchssm_update(self.cfg, self.S, self.omega, None, 0, None, self.U, None, self.stream(), cmap=self.cmap)

    def write_token(self, inp: dict, slot: int | None = None):
        """The producer's side: the token's k, v, beta and log decay go into
        ring slot `slot` (default: the next slot of the window)."""
        s = self.n if slot is None else slot
        self.rk[:, :, s].copy_(inp["k"])
        self.rv[:, :, s].copy_(inp["v"])
        self.rbeta[:, :, s].copy_(inp["beta"])
        self.rla[:, :, s].copy_(inp["log_decay"])

    def read(self, q: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
        """One decode token whose inputs already sit in ring slot n: a non-flush
        read (sketch, or exact full read for the baseline) while the window is
        open, the flush on its W-th token."""
        o = self.o if out is None else out
        if self.n == self.window - 1:
            B.sketchssm_update(self.cfg, self.S, self.omega, self.ring, self.n, q, self.U, o, self.stream(),
                               cmap=self.cmap)
            self.n = 0
        elif self.baseline:
            B.sketchssm_full_read_baseline(self.cfg, self.S, self.ring, self.n, q, o, self.stream())
            self.n += 1
        else:
            B.sketchssm_decode(self.cfg, self.U, self.coef, self.ring, self.n, q, o, self.stream(), cmap=self.cmap,
                               S=self.S if self.dense_heads else None)
            self.n += 1
        return o

    def prepared_read(self, q: torch.Tensor, n: int, out: torch.Tensor | None = None) -> B.Prepared:
        """The read of ring slot `n` (as `read` would issue it with self.n == n)
        with its arguments marshalled once, on the current stream.  Replaying
        the W calls n = 0..W-1 in order is the same as W calls of `read`; the
        caller owns that order (self.n is not touched)."""
        o = self.o if out is None else out
        st = self.stream()
        if n == self.window - 1:
            return B.prepare_update(self.cfg, self.S, self.omega, self.ring, n, q, self.U, o, st, cmap=self.cmap)
        if self.baseline:
            return B.prepare_full_read_baseline(self.cfg, self.S, self.ring, n, q, o, st)
        return B.prepare_decode(self.cfg, self.U, self.coef, self.ring, n, q, o, st, cmap=self.cmap,
                                S=self.S if self.dense_heads else None)

    def step(self, inp: dict, out: torch.Tensor | None = None) -> torch.Tensor:
        """write_token + read."""
        self.write_token(inp)
        return self.read(inp["q"], out)

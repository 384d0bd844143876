"""Device buffers of one linear-attention layer and its decode loop
(Algorithm 1, inference part), on top of the C ABI.

torch supplies device memory and the stream; every computation is a call
into libsketchssm.so.  Buffers (caller-owned, as the ABI requires):

  S      [B][H][V][K]  fp32 full state (stored transposed: K contiguous)
  U      [B][H][V][r]  fp32 sketch  U = S^T Omega
  omega  [H][K][r]     fp32 sketching matrix, coef [H][r][K] its coefficient map
  ring   k [B][H][W][K] io, g [B][H][W] (KDA: [..][K]), beta [B][H][W];
         Mamba-2: v [B][H][W][V] io; GDN/KDA: u [B][H][W][V], bcoef [B][H][W][W],
         f [B][H][W][r] (sketch read) or pi [B][H][W][K] (exact baseline).
"""
from __future__ import annotations

import torch

from . import binding as B


class SketchSSMLayer:
    def __init__(self, kind: str, batch: int, heads: int, dk: int, dv: int, rank: int, window: int,
                 io: str = "bf16", device="cuda", baseline: bool = False, S: torch.Tensor | None = None,
                 omega: torch.Tensor | None = None, coef: torch.Tensor | None = None):
        self.kind, self.batch, self.heads, self.dk, self.dv = kind, batch, heads, dk, dv
        self.rank, self.window, self.io, self.baseline = rank, window, io, baseline
        self.device = torch.device(device)
        iodt = torch.bfloat16 if io == "bf16" else torch.float32
        f32 = torch.float32
        Bt, H, K, V, W = batch, heads, dk, dv, window
        erase = kind in ("gdn", "kda")
        dev = self.device
        self.S = S if S is not None else torch.zeros((Bt, H, V, K), dtype=f32, device=dev)
        r = 0 if baseline else rank
        self.cfg = B.make_config(kind, Bt, H, K, V, r, W, io)
        self.cfg_flush = B.make_config(kind, Bt, H, K, V, r, W, io)
        if not baseline:
            self.omega = omega.to(dev).contiguous()
            self.coef = coef.to(dev).contiguous()
            self.U = torch.zeros((Bt, H, V, rank), dtype=f32, device=dev)
        else:
            self.omega = self.coef = self.U = None
        self.rk = torch.zeros((Bt, H, W, K), dtype=iodt, device=dev)
        self.rg = torch.zeros((Bt, H, W, K) if kind == "kda" else (Bt, H, W), dtype=f32, device=dev)
        self.rbeta = torch.zeros((Bt, H, W), dtype=f32, device=dev)
        self.rv = torch.zeros((Bt, H, W, V), dtype=iodt, device=dev) if not erase else None
        self.ru = torch.zeros((Bt, H, W, V), dtype=f32, device=dev) if erase else None
        self.rb = torch.zeros((Bt, H, W, W), dtype=f32, device=dev) if erase else None
        self.rf = torch.zeros((Bt, H, W, rank), dtype=f32, device=dev) if (erase and not baseline) else None
        self.rpi = torch.zeros((Bt, H, W, K), dtype=f32, device=dev) if (erase and baseline) else None
        self.ring = B.make_ring(k=self.rk, v=self.rv, u=self.ru, f=self.rf, pi=self.rpi, g=self.rg,
                                beta=self.rbeta, bcoef=self.rb)
        self.o = torch.zeros((Bt, H, V), dtype=f32, device=dev)
        self.n = 0  # ring slots filled in the current window

    @staticmethod
    def stream() -> int:
        return torch.cuda.current_stream().cuda_stream

    def init_sketch(self):
        """U = S^T Omega from S alone (after prefill); empties the window."""
        self.n = 0
        if not self.baseline:
            B.sketchssm_update(self.cfg, self.S, self.omega, None, 0, None, self.U, None, self.stream())

    def step(self, inp: dict, out: torch.Tensor | None = None) -> torch.Tensor:
        """One decode token: a non-flush read (sketch, or exact full read for
        the baseline) while the window is open, the flush on its W-th token."""
        o = self.o if out is None else out
        st = B.make_step(inp["q"], inp["k"], inp["v"], inp["beta"], inp["log_decay"])
        if self.n == self.window - 1:
            B.sketchssm_update(self.cfg_flush, self.S, self.omega, self.ring, self.n, st, self.U, o, self.stream())
            self.n = 0
        elif self.baseline:
            B.sketchssm_full_read_baseline(self.cfg, self.S, self.ring, self.n, st, o, self.stream())
            self.n += 1
        else:
            B.sketchssm_decode(self.cfg, self.U, self.coef, self.ring, self.n, st, o, self.stream())
            self.n += 1
        return o

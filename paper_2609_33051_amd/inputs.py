"""Seeded synthetic inputs for the SketchSSM decode path.

This module draws inputs and nothing else: it holds none of the method's
arithmetic and is shared by the GPU path, the tests and the benchmark (the
CPU oracle receives copies of what it produces).

Workloads (shapes and value distributions of the paper's decode layers; the
models and calibration data themselves are not used):

  tiny_mamba2   scalar-decay linear attention in Mamba-2 form, all fp32.
                B=2 H=4 K=64 V=64 r=8 W=8, 64 steps.  q,k ~ N(0,1) then
                L2-normalised over K; v ~ N(0,1); log decay ~ U[-0.1, 0];
                write gate beta = 1; S0 = 0.1 N(0,1).
  mamba2_b256   Mamba-2 decode layer.  B=256 H=128 P=V=64 N=K=128 r=16 W=16,
                256 steps.  x,B,C ~ N(0,1) rounded to bf16 (v,k,q);
                dt = softplus(N(0,1)) per (b,h,t); A_h = -exp(U[0,2]) per head;
                beta = dt, log decay = dt * A_h (fp32); S0 = 0.1 N(0,1) fp32.
  gdn_b512      gated delta rule.  B=512 H=32 K=V=128 r=16 W=16, 256 steps.
                q,k ~ N(0,1), L2-normalised, bf16; v ~ N(0,1) bf16;
                beta = sigmoid(N(0,1)); log decay ~ U[-0.05, 0] per (b,h,t).
  kda_b512      as gdn_b512 with a per-channel log decay ~ U[-0.05, 0]^K.
  mamba2_b2048  Mamba-2 stress shape B=2048 H=128 V=64 K=128, 512 steps,
                ranks {8,16,32} x windows {16,32}.

Omega: per head, the Q factor of a seeded K x r_max Gaussian (column signs
fixed so diag(R) > 0), stored fp32; rank r uses its first r columns (a
prefix of an orthonormal basis is orthonormal).  The coefficient map is the
offline map of Sec. 3.3 at E0 = I, i.e. C = Omega^T.

Per-step tensors come from torch.Generator streams keyed on
(seed, workload, tensor, step), drawn on the device the caller names (the CPU
and GPU generators give different, equally seeded streams; a test always
feeds both sides from one draw).
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import numpy as np
import torch

SEED = 2609


@dataclass(frozen=True)
class Workload:
    name: str
    family: str          # "mamba2_form" | "mamba2" | "gdn" | "kda"
    batch: int
    heads: int
    dk: int
    dv: int
    rank: int
    window: int
    steps: int
    io: str              # "f32" | "bf16"
    ranks: tuple = field(default=())
    windows: tuple = field(default=())

    @property
    def kind(self) -> str:
        return "mamba2" if self.family in ("mamba2_form", "mamba2") else self.family

    @property
    def items(self) -> int:
        return self.batch * self.heads

    def with_(self, **kw) -> "Workload":
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)


WORKLOADS = {
    "tiny_mamba2": Workload("tiny_mamba2", "mamba2_form", 2, 4, 64, 64, 8, 8, 64, "f32"),
    "mamba2_b256": Workload("mamba2_b256", "mamba2", 256, 128, 128, 64, 16, 16, 256, "bf16"),
    "gdn_b512": Workload("gdn_b512", "gdn", 512, 32, 128, 128, 16, 16, 256, "bf16"),
    "kda_b512": Workload("kda_b512", "kda", 512, 32, 128, 128, 16, 16, 256, "bf16"),
    "mamba2_b2048": Workload("mamba2_b2048", "mamba2", 2048, 128, 128, 64, 16, 16, 512, "bf16",
                             ranks=(8, 16, 32), windows=(16, 32)),
}

_STREAMS = {"S0": 1, "q": 2, "k": 3, "v": 4, "gate": 5, "decay": 6, "omega": 7, "A": 8}


def _seed(wl_name: str, stream: str, step: int = 0, seed: int = SEED) -> int:
    h = hashlib.sha256(f"{seed}:{wl_name}:{stream}:{step}".encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def _gen(device, wl: Workload, stream: str, step: int = 0, seed: int = SEED) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(_seed(wl.name, stream, step, seed))
    return g


def io_dtype(wl: Workload) -> torch.dtype:
    return torch.bfloat16 if wl.io == "bf16" else torch.float32


def omega(wl: Workload, rank: int | None = None, seed: int = SEED):
    """(omega [H][K][r], coef [H][r][K]) as float32 numpy arrays, C = Omega^T."""
    rmax = max((wl.rank,) + tuple(wl.ranks))
    r = wl.rank if rank is None else rank
    if r > rmax:
        raise ValueError("rank above the workload's largest rank")
    rng = np.random.default_rng([seed, _STREAMS["omega"], len(wl.name), wl.dk, rmax] + list(wl.name.encode()))
    om = np.empty((wl.heads, wl.dk, rmax), np.float32)
    for h in range(wl.heads):
        Q, R = np.linalg.qr(rng.standard_normal((wl.dk, rmax)))
        om[h] = (Q * np.sign(np.diag(R))[None, :]).astype(np.float32)
    om = np.ascontiguousarray(om[:, :, :r])
    return om, np.ascontiguousarray(om.transpose(0, 2, 1))


def identity_omega(wl: Workload):
    """Omega = I (r = K), C = I: the closed-form case where the sketch read is exact."""
    om = np.broadcast_to(np.eye(wl.dk, dtype=np.float32), (wl.heads, wl.dk, wl.dk)).copy()
    return om, om.copy()


def mamba2_A(wl: Workload, seed: int = SEED) -> np.ndarray:
    """A_h = -exp(U[0, 2]) per head (fp32)."""
    rng = np.random.default_rng([seed, _STREAMS["A"]] + list(wl.name.encode()))
    return (-np.exp(rng.uniform(0.0, 2.0, wl.heads))).astype(np.float32)


def initial_state(wl: Workload, device="cpu", seed: int = SEED) -> torch.Tensor:
    """S0 = 0.1 N(0,1), fp32, [B][H][V][K] (K contiguous)."""
    g = _gen(device, wl, "S0", 0, seed)
    S = torch.randn((wl.batch, wl.heads, wl.dv, wl.dk), generator=g, device=device, dtype=torch.float32)
    return S.mul_(0.1)


def step_inputs(wl: Workload, step: int, device="cpu", seed: int = SEED) -> dict:
    """One decode token for every (b, h): q, k [B][H][K], v [B][H][V] in the io
    dtype; beta [B][H] and log_decay [B][H] (or [B][H][K] for KDA) in fp32."""
    B, H, K, V = wl.batch, wl.heads, wl.dk, wl.dv
    f32 = torch.float32

    def normal(stream, shape):
        return torch.randn(shape, generator=_gen(device, wl, stream, step, seed), device=device, dtype=f32)

    def uniform(stream, shape, lo, hi):
        u = torch.rand(shape, generator=_gen(device, wl, stream, step, seed), device=device, dtype=f32)
        return u * (hi - lo) + lo

    q = normal("q", (B, H, K))
    k = normal("k", (B, H, K))
    v = normal("v", (B, H, V))
    if wl.family in ("mamba2_form", "gdn", "kda"):
        q = q / q.norm(dim=-1, keepdim=True)
        k = k / k.norm(dim=-1, keepdim=True)
    dt = io_dtype(wl)
    q, k, v = q.to(dt), k.to(dt), v.to(dt)
    if wl.family == "mamba2_form":
        beta = torch.ones((B, H), device=device, dtype=f32)
        log_decay = uniform("decay", (B, H), -0.1, 0.0)
    elif wl.family == "mamba2":
        dtv = torch.nn.functional.softplus(normal("gate", (B, H)))
        A = torch.as_tensor(mamba2_A(wl, seed), device=device)
        beta = dtv
        log_decay = dtv * A[None, :]
    elif wl.family == "gdn":
        beta = torch.sigmoid(normal("gate", (B, H)))
        log_decay = uniform("decay", (B, H), -0.05, 0.0)
    elif wl.family == "kda":
        beta = torch.sigmoid(normal("gate", (B, H)))
        log_decay = uniform("decay", (B, H, K), -0.05, 0.0)
    else:
        raise ValueError(wl.family)
    return {"q": q.contiguous(), "k": k.contiguous(), "v": v.contiguous(),
            "beta": beta.contiguous(), "log_decay": log_decay.contiguous()}


def tiny(family: str, batch=2, heads=3, dk=64, dv=64, rank=8, window=8, steps=24, io="f32",
         name: str | None = None) -> Workload:
    """A small workload of any family, for parity cases the oracle finishes quickly."""
    return Workload(name or f"tiny_{family}_{dk}x{dv}_r{rank}_w{window}_{io}", family, batch, heads, dk, dv,
                    rank, window, steps, io)


def ragged_ranks(wl: Workload, seed: int = SEED) -> list[int]:
    """A seeded per-head rank table for workload `wl` with storage width
    wl.rank, shaped like the allocations of Sec. 4.2 (a spread of ranks from
    1 to the width, and a small share of dense-fallback heads): one head in
    ten (at least one) is dense (rank 0); the others draw their rank
    uniformly from 1..wl.rank.  (No calibration data is used.)"""
    rng = np.random.default_rng(_seed(wl.name, "head_ranks", 0, seed))
    H = wl.heads
    ranks = rng.integers(1, wl.rank + 1, size=H)
    dense = rng.choice(H, size=max(1, H // 10), replace=False)
    ranks[dense] = 0
    return [int(x) for x in ranks]

"""Shared machinery for the GPU parity tests: run a workload through the HIP
path (C ABI via the layer helper) and through the CPU oracle on the same
seeded inputs, and compare them."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2609_33051_amd import inputs
from paper_2609_33051_amd.layer import SketchSSMLayer


def to_np32(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float32).numpy()


def rel_l2(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a - b))


class Run:
    """GPU outputs (for all items or a sampled subset) plus the oracle inputs."""

    def __init__(self):
        self.o_gpu = []      # per step, [n_sel][V]
        self.inp = {"q": [], "k": [], "v": [], "beta": [], "log_decay": []}


def run_workload(wl, rank=None, window=None, steps=None, omega_coef=None, sel=None, baseline=False,
                 device="cuda", seed=inputs.SEED, S0=None, keep_layer=False, sketch="f32", pivots=0, head_ranks=None):
    """Run `steps` decode tokens of workload `wl` on the GPU.

    sel: flat item indices (b*H + h) whose outputs and inputs are kept for the
    oracle (None = all).  Returns (Run, layer, S0 subset, heads subset)."""
    rank = wl.rank if rank is None else rank
    window = wl.window if window is None else window
    steps = wl.steps if steps is None else steps
    if omega_coef is None:
        omega_coef = inputs.omega(wl, rank, seed)
    om, C = omega_coef
    S = inputs.initial_state(wl, device, seed) if S0 is None else S0.to(device).clone()
    n_items = wl.batch * wl.heads
    sel_t = None if sel is None else torch.as_tensor(sel, device=device, dtype=torch.long)
    S_sel = to_np32(S.reshape(n_items, wl.dv, wl.dk) if sel is None else S.reshape(n_items, wl.dv, wl.dk)[sel_t])
    layer = SketchSSMLayer(wl.kind, wl.batch, wl.heads, wl.dk, wl.dv, rank, window, wl.io, device,
                           baseline=baseline, S=S, omega=torch.as_tensor(om), coef=torch.as_tensor(C), sketch=sketch,
                           pivots=pivots, head_ranks=head_ranks)
    layer.init_sketch()
    run = Run()
    for t in range(steps):
        inp = inputs.step_inputs(wl, t, device, seed)
        o = layer.step(inp)
        flat = o.reshape(n_items, wl.dv)
        run.o_gpu.append(to_np32(flat if sel is None else flat[sel_t]))
        for key in run.inp:
            x = inp[key].reshape(n_items, -1) if inp[key].dim() > 2 or key in ("q", "k", "v") else inp[key].reshape(n_items)
            run.inp[key].append(to_np32(x if sel is None else x[sel_t]))
    torch.cuda.synchronize()
    heads = (np.arange(n_items) % wl.heads) if sel is None else (np.asarray(sel) % wl.heads)
    return run, layer, S_sel, heads.astype(np.int32), (om, C)


def oracle_of(wl, run, S_sel, heads, om, C, window=None, sketch="f32", pivots=0):
    window = wl.window if window is None else window
    q = np.stack(run.inp["q"])
    k = np.stack(run.inp["k"])
    v = np.stack(run.inp["v"])
    beta = np.stack(run.inp["beta"])
    logd = np.stack(run.inp["log_decay"])
    return oracle.sketchssm(wl.kind, window, heads, om, C, S_sel, q, k, v, beta, logd, round_storage=True,
                            sketch_bf16=(sketch == "bf16"), pivots=pivots, ridge=0.1)


def max_step_rel(o_gpu_list, o_ref):
    return max(rel_l2(o_gpu_list[t], o_ref[t]) for t in range(len(o_gpu_list)))

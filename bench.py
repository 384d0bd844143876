#!/usr/bin/env python3
"""Decode-path benchmark: decode steps/s per layer and state-access GB/s
(fraction of the MI355X HBM roofline) at batch B, on one GPU.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--layers L]

A step is one decode token of one linear-attention layer for the whole batch
(B requests x H heads): a non-flush sketch read (sketchssm_decode) while the
window is open, the flush (sketchssm_update) on its W-th token.  The token's
k, v, beta and log decay sit in its replay-buffer slot, where the layer's
projections write them; one window of such tokens is written before timing
and reused, so the timed region holds exactly the hot path's kernels.  K is rounded
up to whole windows, so the timed region holds both in the method's ratio.
L independent layers (own state, sketch and ring) are stepped in turn, as a
hybrid model interleaves its recurrent layers; this keeps the working set far
above the 256 MB last-level cache so the reads come from HBM.  Inputs are
seeded synthetic tensors, generated before timing and resident in HBM.

Reported (one JSON line):
  value          decode steps/s per layer over the timed region
  roofline       the non-flush read kernel (the dominant one): algorithmic
                 bytes per launch / mean launch time from HIP events recorded
                 on the launch stream, against the 8 TB/s HBM peak
  kernels        the same for the flush and the window-averaged figures
  ragged         a per-head rank table over the same storage width (seeded,
                 with dense-fallback heads read exactly beside the sketch read)
  full_read      the exact full-state-read (ReplaySSM-style) baseline path
  cpu_baseline   the CPU oracle timed on a bounded sample of the same
                 workload on the host cores, scaled to steps/s per layer
  exact_map      the flush with the state-dependent map built under the exact
                 state metric beside the P = 4 one (the paper's Table 2 ratio)

The timed tokens are split into rounds of whole windows (up to seven, as
the paper times its kernels); besides the whole-region `value`, the median
over rounds of each round's steps/s is reported.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

METRIC = "decode steps/s per layer + state-access GB/s (% HBM roofline) at batch B"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=672, help="timed tokens per layer (rounded up to whole windows)")
    p.add_argument("--warmup", type=int, default=32, help="untimed tokens per layer (rounded up to whole windows)")
    p.add_argument("--rounds", type=int, default=7, help="timing rounds of whole windows the median is taken over")
    p.add_argument("--workload", default="mamba2_b256")
    p.add_argument("--rank", type=int, default=None)
    p.add_argument("--window", type=int, default=None)
    p.add_argument("--layers", type=int, default=4)
    p.add_argument("--sketch", choices=("f32", "bf16"), default="f32",
                   help="storage of the sketch U for the headline path (bf16: the paper's storage)")
    p.add_argument("--pivots", type=int, choices=(0, 4), default=0,
                   help="coefficient map of the headline path: 0 = offline (C = Omega^T), 4 = state-dependent")
    p.add_argument("--no-paper-storage", action="store_true",
                   help="skip the extra timed passes with the paper's storage and method beside the headline")
    p.add_argument("--no-full-read", action="store_true", help="skip the exact baseline path")
    p.add_argument("--no-ragged", action="store_true",
                   help="skip the pass with a per-head rank table (seeded, with dense-fallback heads)")
    p.add_argument("--no-standard", action="store_true",
                   help="skip the Standard recurrence (window 1, no sketch: S read and written every token)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU time of the oracle sample")
    p.add_argument("--no-ceilings", action="store_true",
                   help="skip timing torch's plain streaming kernels (read, copy, in place) the kernels are compared with")
    p.add_argument("--copy-calibration", action="store_true",
                   help="also run a plain 1 GiB device copy (scales HBM byte counters)")
    return p.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the decode path has no cross-GPU work "
              "(items shard with zero exchange); run it per GPU with --gpus 1.", file=sys.stderr)
        return 2

    import torch

    from paper_2609_33051_amd import inputs, traffic
    from paper_2609_33051_amd import binding as B
    from paper_2609_33051_amd.layer import SketchSSMLayer

    if not torch.cuda.is_available():
        print("bench.py needs an MI355X GPU", file=sys.stderr)
        return 2
    B.load()  # fails loudly if the HIP library is not built
    dev = torch.device("cuda:0")
    wl = inputs.WORKLOADS[args.workload]
    rank = wl.rank if args.rank is None else args.rank
    W = wl.window if args.window is None else args.window
    wl = wl.with_(rank=rank, window=W)
    K_steps = -(-args.steps // W) * W
    warm = -(-args.warmup // W) * W
    L = args.layers
    io_bytes = 2 if wl.io == "bf16" else 4
    shape = traffic.Shape(wl.kind, wl.dk, wl.dv, rank, W, io_bytes, 2 if args.sketch == "bf16" else 4, args.pivots)
    items = wl.items

    om, C = inputs.omega(wl, rank)
    om_t, C_t = torch.as_tensor(om), torch.as_tensor(C)
    # one window of resident inputs per rotated layer (its own queries and ring
    # contents, so no layer's reads are served from another's cached data)
    pools = [[inputs.step_inputs(wl, t, dev, seed=inputs.SEED + 100 * li) for t in range(W)] for li in range(L)]

    def make_layers(baseline, sketch, pivots, head_ranks=None):
        layers = []
        for li in range(L):
            S = inputs.initial_state(wl, dev, seed=inputs.SEED + li)
            lay = SketchSSMLayer(wl.kind, wl.batch, wl.heads, wl.dk, wl.dv, rank, W, wl.io, dev,
                                 baseline=baseline, S=S, omega=om_t, coef=C_t, sketch=sketch, pivots=pivots,
                                 head_ranks=head_ranks)
            lay.init_sketch()
            for slot in range(W):  # the producer's writes: one window of tokens, resident in the ring
                lay.write_token(pools[li][slot], slot)
            layers.append(lay)
        torch.cuda.synchronize()
        return layers

    def run(layers, n_tokens, events=None, win_events=None):
        """n_tokens decode tokens through every layer, from calls marshalled
        once per (slot, layer).  The L launches of one token are the same
        kernel at the same slot, back to back on one stream; with `events`, a
        pre-created pair of HIP events brackets each such group, and with
        `win_events` one event marks every window boundary."""
        plan = [[lay.prepared_read(pools[li][t]["q"], t) for li, lay in enumerate(layers)] for t in range(W)]
        stream = torch.cuda.current_stream()
        for t in range(n_tokens):
            if win_events is not None and t % W == 0:
                win_events[t // W].record(stream)
            if events is not None:
                events[t][1].record(stream)
            for call in plan[t % W]:
                call()
            if events is not None:
                events[t][2].record(stream)
        if win_events is not None:
            win_events[-1].record(stream)
        for lay in layers:
            lay.n = n_tokens % W

    n_win = K_steps // W
    n_rounds = max(1, min(args.rounds, n_win))

    def round_rates(win_events):
        """Steps/s per layer of each round (whole windows, launch gaps included)."""
        wt = [win_events[i].elapsed_time(win_events[i + 1]) * 1e-3 for i in range(n_win)]
        per = n_win // n_rounds
        out = []
        for r in range(n_rounds):
            ws = wt[r * per:(r + 1) * per] if r < n_rounds - 1 else wt[r * per:]
            out.append(len(ws) * W * L / sum(ws))
        return out

    def timed(baseline, sketch=args.sketch, pivots=args.pivots, head_ranks=None):
        layers = make_layers(baseline, sketch, pivots, head_ranks)
        stream = torch.cuda.current_stream()
        events = [(t % W, torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for t in range(K_steps)]
        win_events = [torch.cuda.Event(enable_timing=True) for _ in range(n_win + 1)]
        for _, e0, e1 in events:  # create the HIP events before the timed region
            e0.record(stream)
            e1.record(stream)
        for e in win_events:
            e.record(stream)
        run(layers, warm, None)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        run(layers, K_steps, events, win_events)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        per_n = {}  # slot -> per-launch seconds, one entry per token (group of L launches)
        for n, e0, e1 in events:
            per_n.setdefault(n, []).append(e0.elapsed_time(e1) * 1e-3 / L)
        rates = round_rates(win_events)
        del layers
        torch.cuda.empty_cache()
        return elapsed, per_n, rates

    def kernel_stats(per_n, sketch, pivots):
        """Decode and flush figures from per-slot launch times (seconds)."""
        sh = traffic.Shape(wl.kind, wl.dk, wl.dv, rank, W, io_bytes, 2 if sketch == "bf16" else 4, pivots)
        dec_n = [n for n in per_n if n < W - 1]
        dec_time = sum(sum(per_n[n]) for n in dec_n)
        dec_launches = sum(len(per_n[n]) for n in dec_n)
        dec_bytes = sum(traffic.decode_bytes(sh, n) * items * len(per_n[n]) for n in dec_n)
        fl = per_n.get(W - 1, [])
        fl_mean = sum(fl) / len(fl)
        fl_bytes = traffic.flush_bytes(sh, W - 1) * items
        flops = items * (2 * wl.dv * wl.dk * W * (2 if sh.erase else 1) + 2 * wl.dv * wl.dk * rank)
        win = sum(sum(v) / len(v) for v in per_n.values())
        dec_all = sorted(x for n in dec_n for x in per_n[n])
        return {"dec_mean": dec_time / dec_launches, "dec_bytes": dec_bytes / dec_launches,
                "dec_median": statistics.median(dec_all), "fl_median": statistics.median(fl),
                "dec_gbps": dec_bytes / dec_time / 1e9, "fl_mean": fl_mean, "fl_bytes": fl_bytes,
                "fl_gbps": fl_bytes / fl_mean / 1e9, "fl_tflops": flops / fl_mean / 1e12, "window": win,
                "per_slot": {int(n): round(sum(v) / len(v) * 1e6, 2) for n, v in sorted(per_n.items()) if n < W - 1}}

    # ---- the SketchSSM path
    elapsed, per_n, rates = timed(False)
    layer_steps = K_steps * L
    value = layer_steps / elapsed
    ks = kernel_stats(per_n, args.sketch, args.pivots)
    traffic_rec = recorded_traffic("decode", wl, rank, W, args.sketch, args.pivots)
    dec_mean_s, dec_bytes_per_launch, dec_gbps = ks["dec_mean"], ks["dec_bytes"], ks["dec_gbps"]
    fl_mean_s, fl_bytes, window_s = ks["fl_mean"], ks["fl_bytes"], ks["window"]

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": K_steps,
        "warmup": warm,
        "steps_requested": args.steps,
        "warmup_requested": args.warmup,
        "steps_note": "tokens per layer, rounded up to whole windows of W so that every timed window holds its flush",
        "rounds": n_rounds,
        "value_median_of_rounds": round(statistics.median(rates), 2),
        "value_rounds": [round(x, 1) for x in rates],
        "ms_per_step": round(elapsed / layer_steps * 1e3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "kind": wl.kind, "batch": wl.batch, "heads": wl.heads, "dk": wl.dk,
                   "dv": wl.dv, "rank": rank, "window": W, "io": wl.io, "state": "f32", "sketch": args.sketch,
                   "pivots": args.pivots,
                   "layers_rotated": L},
        "roofline": {
            "kernel": "decode_kernel (sketchssm_decode)",
            "bound": "hbm",
            "achieved": round(dec_gbps, 1),
            "peak": traffic.HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(dec_gbps / traffic.HBM_PEAK_GBPS, 4),
            "traffic": traffic_rec and traffic_rec["bytes_per_launch"],
            "bytes_per_launch": int(dec_bytes_per_launch),
            "mean_launch_us": round(dec_mean_s * 1e6, 2),
            "median_launch_us": round(ks["dec_median"] * 1e6, 2),
        },
        "state_access_gbps": round(dec_gbps, 1),
        "kernels": {
            "decode": {"mean_us": round(dec_mean_s * 1e6, 2), "median_us": round(ks["dec_median"] * 1e6, 2),
                       "gbps": round(dec_gbps, 1), "per_slot_us": ks["per_slot"]},
            "flush": {"mean_us": round(fl_mean_s * 1e6, 2), "median_us": round(ks["fl_median"] * 1e6, 2),
                      "bytes": fl_bytes,
                      "gbps": round(ks["fl_gbps"], 1),
                      "mfma_tflops": round(ks["fl_tflops"], 2), "mfma_peak_tflops": 157.3},
            "window_us": round(window_s * 1e6, 1),
            "window_avg_steps_per_s": round(W / window_s, 1),
        },
    }

    # ---- beside an offline-map fp32 headline, same inputs: the paper's sketch
    # storage (bf16 U), its method (bf16 U and map with the state-dependent
    # P = 4 map) and the same with the exact-metric map (flush cost, Table 2)
    legs = [("paper_storage", "bf16", 0), ("paper_method", "bf16", 4)]
    if rank in (8, 16):
        legs.append(("exact_map", "bf16", -1))
    if args.sketch == "f32" and args.pivots == 0 and not args.no_paper_storage:
        for key, sk_, pv in legs:
            e_p, per_p, rates_p = timed(False, sk_, pv)
            kp = kernel_stats(per_p, sk_, pv)
            tr = recorded_traffic("decode", wl, rank, W, sk_, pv)
            out[key] = {
                "sketch": sk_, "pivots": pv, "value": round(layer_steps / e_p, 2), "unit": "steps/s",
                "value_median_of_rounds": round(statistics.median(rates_p), 2),
                "decode_mean_us": round(kp["dec_mean"] * 1e6, 2), "decode_bytes_per_launch": int(kp["dec_bytes"]),
                "decode_gbps": round(kp["dec_gbps"], 1),
                "decode_frac": round(kp["dec_gbps"] / traffic.HBM_PEAK_GBPS, 4),
                "decode_traffic": tr and tr["bytes_per_launch"],
                "flush_mean_us": round(kp["fl_mean"] * 1e6, 2), "flush_median_us": round(kp["fl_median"] * 1e6, 2),
                "flush_bytes": kp["fl_bytes"], "flush_gbps": round(kp["fl_gbps"], 1),
                "window_avg_steps_per_s": round(W / kp["window"], 1),
            }
        if "exact_map" in out and "paper_method" in out:
            out["exact_map"]["flush_ratio_exact_vs_p4"] = round(
                out["exact_map"]["flush_median_us"] / out["paper_method"]["flush_median_us"], 3)
        if "paper_storage" in out and "paper_method" in out:
            out["paper_method"]["flush_overhead_vs_offline_map"] = round(
                out["paper_method"]["flush_median_us"] / out["paper_storage"]["flush_median_us"] - 1, 4)

    # ---- a per-head rank table (Sec. 4.2) over the same storage width: a
    # seeded synthetic allocation with dense-fallback heads, whose non-flush
    # reads are exact full-state reads issued beside the sketch read
    if not args.no_ragged and rank in (8, 16, 32) and wl.heads <= 256:
        ranks = inputs.ragged_ranks(wl)
        e_r, per_r, _ = timed(False, args.sketch, args.pivots, head_ranks=ranks)
        rd_n = [n for n in per_r if n < W - 1]
        rd_time = sum(sum(per_r[n]) for n in rd_n)
        rd_launch = rd_time / sum(len(per_r[n]) for n in rd_n)
        rd_bytes = sum(traffic.ragged_decode_bytes(shape, n, ranks) * wl.batch * len(per_r[n]) for n in rd_n)
        rf = per_r.get(W - 1, [])
        rf_mean = sum(rf) / len(rf)
        win_r = sum(sum(v) / len(v) for v in per_r.values())
        out["ragged"] = {
            "head_ranks": ranks, "dense_heads": sum(1 for g in ranks if g == 0),
            "mean_rank": round(sum(ranks) / len(ranks), 3), "value": round(layer_steps / e_r, 2), "unit": "steps/s",
            "read_mean_us": round(rd_launch * 1e6, 2),
            "read_bytes_per_step": int(rd_bytes / sum(len(per_r[n]) for n in rd_n)),
            "read_gbps": round(rd_bytes / rd_time / 1e9, 1),
            "read_frac": round(rd_bytes / rd_time / 1e9 / traffic.HBM_PEAK_GBPS, 4),
            "flush_mean_us": round(rf_mean * 1e6, 2),
            "flush_gbps": round(traffic.ragged_flush_bytes(shape, W - 1, ranks) * wl.batch / rf_mean / 1e9, 1),
            "window_avg_steps_per_s": round(W / win_r, 1),
        }

    # ---- the exact full-state-read baseline (same inputs; flush with rank 0)
    if not args.no_full_read:
        e_b, per_b, rates_b = timed(True)
        fr_n = [n for n in per_b if n < W - 1]
        fr_time = sum(sum(per_b[n]) for n in fr_n)
        fr_bytes = sum(traffic.full_read_bytes(shape, n) * items * len(per_b[n]) for n in fr_n)
        fr_launch = fr_time / sum(len(per_b[n]) for n in fr_n)
        fb = per_b.get(W - 1, [])
        win_b = sum(sum(v) / len(v) for v in per_b.values())
        out["full_read"] = {
            "value": round(layer_steps / e_b, 2), "unit": "steps/s",
            "read_mean_us": round(fr_launch * 1e6, 2), "read_gbps": round(fr_bytes / fr_time / 1e9, 1),
            "read_frac": round(fr_bytes / fr_time / 1e9 / traffic.HBM_PEAK_GBPS, 4),
            "flush_mean_us": round(sum(fb) / len(fb) * 1e6, 2),
            "window_avg_steps_per_s": round(W / win_b, 1),
            "value_median_of_rounds": round(statistics.median(rates_b), 2),
            "speedup_sketch_vs_full_read": round(value / (layer_steps / e_b), 3),
            "read_bytes_ratio_window_mean": round(traffic.window_bytes(shape, baseline=True)["nonflush_mean"]
                                                  / traffic.window_bytes(shape)["nonflush_mean"], 3),
        }
    # ---- Standard decoding: every token reads and writes the whole state (window 1, rank 0)
    if not args.no_standard:
        layers = []
        for li in range(L):
            S = inputs.initial_state(wl, dev, seed=inputs.SEED + li)
            lay = SketchSSMLayer(wl.kind, wl.batch, wl.heads, wl.dk, wl.dv, 0, 1, wl.io, dev, baseline=True, S=S)
            lay.write_token(pools[li][0], 0)
            layers.append(lay)
        plan = [lay.prepared_read(pools[li][0]["q"], 0) for li, lay in enumerate(layers)]
        stream = torch.cuda.current_stream()
        for _ in range(warm):
            for call in plan:
                call()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K_steps)]
        for e0, e1 in ev:
            e0.record(stream)
            e1.record(stream)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for e0, e1 in ev:
            e0.record(stream)
            for call in plan:
                call()
            e1.record(stream)
        torch.cuda.synchronize()
        e_s = time.perf_counter() - t0
        st_launch = sum(e0.elapsed_time(e1) for e0, e1 in ev) * 1e-3 / (K_steps * L)
        sh1 = traffic.Shape(wl.kind, wl.dk, wl.dv, 0, 1, io_bytes)
        st_bytes = traffic.flush_bytes(sh1, 0, 0) * items
        std_value = layer_steps / e_s
        out["standard"] = {
            "value": round(std_value, 2), "unit": "steps/s", "launch_mean_us": round(st_launch * 1e6, 2),
            "bytes_per_launch": st_bytes, "gbps": round(st_bytes / st_launch / 1e9, 1),
            "frac": round(st_bytes / st_launch / 1e9 / traffic.HBM_PEAK_GBPS, 4),
            "speedup_sketch_vs_standard": round(value / std_value, 3),
        }
        for key in ("paper_storage", "paper_method"):
            if key in out:
                out[key]["speedup_vs_standard"] = round(out[key]["value"] / std_value, 3)
        del layers, plan
        torch.cuda.empty_cache()

    out["traffic_model"] = {
        "paper_R_G_bf16": round(traffic.paper_reduction(wl.dk, wl.dv, rank, W, 1 if shape.erase else 0), 3),
        "state_vs_sketch_read": round(wl.dk / rank, 3),
        "decode_bytes_per_item_mean": traffic.window_bytes(shape)["nonflush_mean"],
        "full_read_bytes_per_item_mean": traffic.window_bytes(shape, baseline=True)["nonflush_mean"],
    }

    # ---- what torch's plain streaming kernels reach on this part, measured in
    # the same run (HIP events, median of 7): a read-only pass, a copy and an
    # in-place rewrite, 1 GiB each way (beyond the 256 MB last-level cache).
    # Reference rates, not bounds: the flush streams faster than torch's copy.
    if not args.no_ceilings:
        ce = torch_streams(dev)
        out["torch_streams"] = ce
        out["roofline"]["frac_of_torch_read"] = round(dec_gbps / ce["read_gbps"], 4)
        out["kernels"]["flush"]["frac_of_torch_copy"] = round(ks["fl_gbps"] / ce["copy_gbps"], 4)
        out["kernels"]["flush"]["frac_of_torch_inplace"] = round(ks["fl_gbps"] / ce["inplace_gbps"], 4)
        if "standard" in out:
            out["standard"]["frac_of_torch_inplace"] = round(out["standard"]["gbps"] / ce["inplace_gbps"], 4)

    if args.copy_calibration:
        n = 1 << 28  # 1 GiB of fp32
        a = torch.empty(n, dtype=torch.float32, device=dev).fill_(1.0)
        b = torch.empty_like(a)
        for _ in range(3):  # a streaming kernel named neg_kernel: reads 1 GiB, writes 1 GiB
            torch.neg(a, out=b)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = 2 * n * 4

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, rank, W, args.cpu_seconds, dev)

    print(json.dumps(out), flush=True)
    return 0


def recorded_traffic(entry, wl, rank, W, sketch="f32", pivots=0):
    """HBM bytes per launch of the `entry` kernel ("decode", ...) on this
    workload, from the FETCH_SIZE and WRITE_SIZE counter runs recorded under
    profiles/, each scaled by the factor a plain copy kernel's counters gave
    in the same runs.  None when no run was recorded for this configuration
    or the kernel's sources have changed since (their digest differs)."""
    from paper_2609_33051_amd import build as hip_build

    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        table = json.load(f)
    unit = f"{entry}_{wl.kind}"
    rec = table.get(f"{unit}:{wl.name}:r{rank}:w{W}" + (":bf16" if sketch == "bf16" else "")
                    + (f":p{pivots}" if pivots else ""))
    if rec is None or rec.get("digest") != hip_build.source_digest(unit):
        return None
    b = rec["fetch_kib"] * 1024 * rec["fetch_scale"] + rec["write_kib"] * 1024 * rec["write_scale"]
    return {"bytes_per_launch": int(round(b)), "record": rec}


def torch_streams(dev, reps=7):
    """Bandwidth of plain streaming kernels on 1 GiB operands: row sums of a
    16384 x 16384 fp32 matrix (reads 1 GiB; of torch's reductions the one that
    streams fastest here), torch.neg (reads 1 GiB, writes 1 GiB elsewhere) and
    its in-place form (reads and rewrites the same 1 GiB, as the flush does with
    the state), timed with HIP events on the current stream, median of `reps`
    launches after a warmup."""
    import torch

    n = 1 << 28
    a = torch.empty(n, dtype=torch.float32, device=dev).fill_(1.0)
    b = torch.empty_like(a)
    s = torch.empty(1 << 14, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def med(fn):
        fn()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3)
        return statistics.median(ts)

    t_read = med(lambda: torch.sum(a.view(1 << 14, 1 << 14), dim=1, out=s))
    t_copy = med(lambda: torch.neg(a, out=b))
    t_inpl = med(lambda: a.neg_())
    del a, b
    torch.cuda.empty_cache()
    return {"read_gbps": round(4 * n / t_read / 1e9, 1), "copy_gbps": round(8 * n / t_copy / 1e9, 1),
            "inplace_gbps": round(8 * n / t_inpl / 1e9, 1),
            "read_kernel": "torch.sum(dim=1) of a 16384 x 16384 fp32 matrix", "copy_kernel": "torch.neg, 1 GiB fp32 in and out",
            "inplace_kernel": "torch.neg_ on 1 GiB fp32 (read and rewritten in place)",
            "read_frac_of_peak": round(4 * n / t_read / 1e9 / 8000.0, 4),
            "copy_frac_of_peak": round(8 * n / t_copy / 1e9 / 8000.0, 4)}


def cpu_model() -> str | None:
    """The host CPU's model name (/proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(wl, rank, W, target_s, dev):
    """The oracle (plain fp64 C, items spread over the host threads) on the
    first n_sel items of the workload (all of them when one window of all
    takes under about a third of `target_s`), for as many consecutive windows
    as fill about `target_s` seconds (the state carries from window to
    window), scaled linearly to all items (items are independent) and
    reported as steps/s per layer.  A one-thread figure on a sixteenth of
    that sample is reported beside it."""
    import numpy as np
    import torch

    import oracle
    from paper_2609_33051_amd import inputs

    items = wl.items
    threads = oracle.max_threads()
    om, C = inputs.omega(wl, rank)
    pool = [inputs.step_inputs(wl, t, dev) for t in range(W)]
    S_all = inputs.initial_state(wl, dev).reshape(items, wl.dv, wl.dk)

    def host(x, w, n):
        return x.reshape(items, w)[:n].to("cpu", torch.float32).numpy()

    def sample(n):
        q = np.stack([host(p["q"], wl.dk, n) for p in pool])
        k = np.stack([host(p["k"], wl.dk, n) for p in pool])
        v = np.stack([host(p["v"], wl.dv, n) for p in pool])
        beta = np.stack([host(p["beta"], 1, n)[:, 0] for p in pool])
        ld = np.stack([host(p["log_decay"], wl.dk if wl.kind == "kda" else 1, n) for p in pool])
        if wl.kind != "kda":
            ld = ld[:, :, 0]
        heads = (np.arange(n) % wl.heads).astype(np.int32)
        return heads, q, k, v, beta, ld, S_all[:n].cpu().numpy()

    def windows(n_win, data, S):
        heads, q, k, v, beta, ld, _ = data
        t0 = time.perf_counter()
        for _ in range(n_win):
            S = oracle.sketchssm(wl.kind, W, heads, om, C, S, q, k, v, beta, ld, round_storage=True,
                                 diagnostics=False).S_final
        return time.perf_counter() - t0, S

    # calibrate on a small slice, then size the sample
    n_cal = min(items, 2048)
    cal = sample(n_cal)
    dt_cal, _ = windows(1, cal, cal[-1])
    per_item_window = dt_cal / n_cal
    n_sel = int(min(items, max(n_cal, target_s / 3 / max(per_item_window, 1e-9))))
    data = sample(n_sel)
    dt, S1 = windows(1, data, data[-1])
    n_win = 1
    if dt < 0.5 * target_s:  # too short to time alone: run enough further windows
        n_win = int(min(64, max(1, round(target_s / max(dt, 1e-3)))))
        dt, _ = windows(n_win, data, S1)
    steps = n_win * W
    value = steps / dt * n_sel / items
    # one thread, a sixteenth of the sample, one window
    n1 = max(1, n_sel // 16)
    heads, q, k, v, beta, ld, S0 = data
    one = (heads[:n1], q[:, :n1], k[:, :n1], v[:, :n1], beta[:, :n1], ld[:, :n1], S0[:n1])
    oracle.set_threads(1)
    try:
        dt1, _ = windows(1, one, one[-1])
    finally:
        oracle.set_threads(threads)
    value1 = W / dt1 * n1 / items
    return {"value": round(value, 4), "unit": "steps/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "nproc": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0)),
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
            "sample": f"{n_sel} of {items} (request, head) items x {n_win} consecutive windows of {W} steps "
                      f"({steps} decode steps), {dt:.1f} s wall on {threads} threads, scaled linearly to all items",
            "one_thread": {"value": round(value1, 5), "sample": f"{n1} items x one window, {dt1:.1f} s"}}


if __name__ == "__main__":
    sys.exit(main())

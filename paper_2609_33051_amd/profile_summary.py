"""Summarise rocprofv3 CSV output of a bench.py run into short text records.

    python -m paper_2609_33051_amd.profile_summary --trace DIR --fetch DIR --write DIR \
        --workload mamba2_b256 --command "..." --out profiles/

--trace is the output directory of `rocprofv3 --kernel-trace --stats
--output-format csv`, --fetch / --write those of two `--pmc FETCH_SIZE` and
`--pmc WRITE_SIZE` runs of a bench.py command with --copy-calibration, whose
1 GiB fp32 copy fixes the scale of each counter (bytes it reads or writes
divided by what the counter reports for it).

Writes <entry>_<workload>.txt per kernel of this library that ran (duration
statistics, counter means per dispatch, scaled bytes, algorithmic bytes) and
merges the per-launch counter records into traffic.json, keyed
"<entry>_<kind>:<workload>:r<rank>:w<window>" with the kernel's source digest,
for bench.py's roofline `traffic` field.
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import re
import sys

COPY_BYTES = 1 << 30  # the calibration copy: 2^28 fp32 read and written


def _rows(d, suffix):
    fs = glob.glob(os.path.join(d, "*" + suffix))
    if len(fs) != 1:
        raise SystemExit(f"expected one *{suffix} under {d}, found {fs}")
    with open(fs[0]) as f:
        return list(csv.DictReader(f))


def _short(name: str) -> str:
    name = name.replace("void ", "")
    m = re.match(r"([\w:]+)(<[^()]*>)?", name)
    return (m.group(1).split("::")[-1] + (m.group(2) or "")) if m else name[:80]


def _entry(short: str) -> str | None:
    for e in ("decode", "full_read", "update"):
        if short.startswith(f"{e}_kernel<"):
            return e
    return None


def kernel_variant(short: str) -> tuple[str, str, int] | None:
    """(entry, sketch dtype, pivots) of a kernel-trace name such as
    decode_kernel<1, 128, 128, 16, 16, unsigned short, float, 0, false>:
    update's template arguments end with io, sketch, pivots; decode's with io,
    sketch, pivots, dense (its dense-fallback instance); full_read has no sketch."""
    e = _entry(short)
    if e is None:
        return None
    targs = short[short.index("<") + 1:short.rindex(">")].split(", ")
    if targs[-1] in ("true", "false"):
        targs = targs[:-1]
    if e == "full_read":
        return e, "f32", 0
    return e, ("bf16" if targs[-2] == "unsigned short" else "f32"), int(targs[-1])


def _counter(d, counter):
    """(per-kernel list of values in KiB, copy-kernel value) from one pmc run."""
    per, copy = {}, []
    for r in sorted(_rows(d, "_counter_collection.csv"), key=lambda r: int(r["Dispatch_Id"])):
        if r["Counter_Name"] != counter:
            continue
        s = _short(r["Kernel_Name"])
        v = float(r["Counter_Value"])
        per.setdefault(s, []).append(v)
        if "neg_kernel" in r["Kernel_Name"]:
            copy.append(v)  # bench.py --copy-calibration: 2^28 fp32 negated, 1 GiB in, 1 GiB out
    if not copy:
        raise SystemExit(f"no calibration copy kernel found in {d} (run bench.py with --copy-calibration)")
    return per, sum(copy) / len(copy)


XCDS, SIMDS = 8, 1024  # MI355X: GRBM_GUI_ACTIVE is summed over the 8 XCDs; 256 CUs x 4 SIMDs


def _mfma_lines(d, kernel):
    """Matrix-core utilisation per group of dispatches with the same MFMA op
    count (the initial sketch and the flush differ): busy cycles of all SIMDs
    over (active cycles per XCD x SIMDs), and fp32 MFMA flops (512 per op)."""
    per = {}
    for r in _rows(d, "_counter_collection.csv"):
        if _short(r["Kernel_Name"]) != kernel:
            continue
        per.setdefault(r["Dispatch_Id"], {})[r["Counter_Name"]] = float(r["Counter_Value"])
    groups = {}
    for c in per.values():
        groups.setdefault(c.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0.0), []).append(c)
    out = []
    for mops, cs in sorted(groups.items()):
        busy = sum(c["SQ_VALU_MFMA_BUSY_CYCLES"] for c in cs) / len(cs)
        active = sum(c["GRBM_GUI_ACTIVE"] for c in cs) / len(cs) / XCDS
        out.append(f"    {len(cs)} dispatches with {mops:.0f} MFMA MOPS ({mops * 512 / 1e9:.2f} GFLOP fp32, 512 flops per MOP): "
                   f"MFMA busy {100 * busy / (active * SIMDS):.1f} % of {active:.0f} active cycles per SIMD")
    return out


def _split_lines(d, layers):
    """Initial-sketch and flush durations of one update kernel, from its
    dispatches in launch order (the first `layers` are initial sketches)."""
    init, fl = d[:layers], d[layers:]
    out = []
    if init:
        out.append(f"    initial sketches: {len(init)} dispatches, average {sum(init) / len(init):.2f} us")
    if fl:
        srt = sorted(fl)
        out.append(f"    flushes: {len(fl)} dispatches, average {sum(fl) / len(fl):.2f} us, "
                   f"median {srt[len(srt) // 2]:.2f} us, min {srt[0]:.2f} us, max {srt[-1]:.2f} us")
    return out


def main(argv=None):
    p = argparse.ArgumentParser()
    p.add_argument("--trace", required=True)
    p.add_argument("--fetch", required=True)
    p.add_argument("--write", required=True)
    p.add_argument("--workload", required=True)
    p.add_argument("--rank", type=int, default=None)
    p.add_argument("--window", type=int, default=None)
    p.add_argument("--command", required=True, help="the rocprofv3 commands, as run")
    p.add_argument("--mfma", default=None,
                   help="output of a --pmc SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_BUSY_CYCLES "
                        "GRBM_GUI_ACTIVE run (matrix-core utilisation of the update kernel)")
    p.add_argument("--mfma-command", default="", help="the command of the --mfma run")
    p.add_argument("--out", required=True)
    p.add_argument("--layers", type=int, default=4, help="layers the bench run rotated (initial sketches per leg)")
    a = p.parse_args(argv)

    from . import build as hip_build
    from . import inputs, traffic

    wl = inputs.WORKLOADS[a.workload]
    rank = wl.rank if a.rank is None else a.rank
    W = wl.window if a.window is None else a.window
    items = wl.items

    def algo(entry, sketch, pivots):
        sh = traffic.Shape(wl.kind, wl.dk, wl.dv, rank, W, 2 if wl.io == "bf16" else 4, 2 if sketch == "bf16" else 4,
                           pivots)
        if entry == "decode":
            return sum(traffic.decode_bytes(sh, n) for n in range(W - 1)) / (W - 1) * items
        if entry == "full_read":
            return sum(traffic.full_read_bytes(sh, n) for n in range(W - 1)) / (W - 1) * items
        if entry == "flush":
            return traffic.flush_bytes(sh, W - 1) * items
        return None

    stats = {}
    for r in _rows(a.trace, "_kernel_stats.csv"):
        s = _short(r["Name"])
        stats[s] = r
    # per-dispatch durations in launch order: the first `layers` dispatches of
    # an update kernel with a sketch are the initial sketches of the bench's
    # layers (no state write), the rest are flushes
    durs = {}
    for r in sorted(_rows(a.trace, "_kernel_trace.csv"), key=lambda r: int(r["Dispatch_Id"])):
        durs.setdefault(_short(r["Kernel_Name"]), []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    p_layers = a.layers
    fetch, copy_f = _counter(a.fetch, "FETCH_SIZE")
    write, copy_w = _counter(a.write, "WRITE_SIZE")
    f_scale = COPY_BYTES / (copy_f * 1024)
    w_scale = COPY_BYTES / (copy_w * 1024)

    os.makedirs(a.out, exist_ok=True)
    tpath = os.path.join(a.out, "traffic.json")
    table = json.load(open(tpath)) if os.path.exists(tpath) else {}
    for s, r in sorted(stats.items()):
        v = kernel_variant(s)
        if v is None:
            continue
        e, sketch, pivots = v
        unit = f"{e}_{wl.kind}"
        digest = hip_build.source_digest(unit)
        tag = (":bf16" if sketch == "bf16" else "") + (f":p{pivots}" if pivots else "")
        ab = algo(e, sketch, pivots)
        fv, wv = fetch.get(s, []), write.get(s, [])
        split = e == "update" and not re.search(r"<\d+, \d+, \d+, 0,", s)  # with a sketch: initial sketches first
        if split:
            ab = algo("flush", sketch, pivots)
            fv, wv = fv[p_layers:], wv[p_layers:]
        lines = [
            f"# {s} on {a.workload} (rank {rank}, window {W})",
            "",
            "Commands (from the repository root of the run; CSV output):",
            *[f"    {c}" for c in a.command.split(" ;; ")],
            "",
            f"source digest of {unit}: {digest}",
            "",
            "kernel trace (--kernel-trace --stats):",
            f"    calls {r['Calls']}, average {float(r['AverageNs']) / 1e3:.2f} us, "
            f"min {float(r['MinNs']) / 1e3:.2f} us, max {float(r['MaxNs']) / 1e3:.2f} us, "
            f"{float(r['Percentage']):.2f} % of GPU kernel time",
            *(_split_lines(durs.get(s, []), p_layers) if split else []),
            "",
            "counters per dispatch (KiB as reported; scaled by the calibration copy of 1 GiB:",
            f"    FETCH_SIZE read {copy_f:.1f} KiB for it -> scale {f_scale:.4f};"
            f" WRITE_SIZE wrote {copy_w:.1f} KiB -> scale {w_scale:.4f})",
        ]
        if fv and wv:
            fm, wm = sum(fv) / len(fv), sum(wv) / len(wv)
            hbm = fm * 1024 * f_scale + wm * 1024 * w_scale
            lines += [
                f"    FETCH_SIZE dispatches {len(fv)}, mean {fm:.1f}, min {min(fv):.1f}, max {max(fv):.1f}",
                f"    WRITE_SIZE dispatches {len(wv)}, mean {wm:.1f}, min {min(wv):.1f}, max {max(wv):.1f}",
                f"    HBM bytes per launch (scaled): read {fm * 1024 * f_scale / 1e6:.2f} MB + "
                f"write {wm * 1024 * w_scale / 1e6:.2f} MB = {hbm / 1e6:.2f} MB",
            ]
            if split:
                lines.append(f"    (flush dispatches only: the first {p_layers} dispatches, the initial sketches, excluded)")
            if ab is not None:
                what = "per flush" if split else f"per launch (mean over slots 0..{W - 2})"
                lines.append(f"    algorithmic bytes {what}: {ab / 1e6:.2f} MB"
                             f" -> measured / algorithmic = {hbm / ab:.3f}")
                table[f"{unit}:{a.workload}:r{rank}:w{W}{tag}"] = {
                    "kernel": s, "digest": digest, "fetch_kib": round(fm, 1), "write_kib": round(wm, 1),
                    "fetch_scale": round(f_scale, 6), "write_scale": round(w_scale, 6),
                    "dispatches": len(fv), "algorithmic_bytes": int(ab),
                }

        if a.mfma and e == "update":
            m = _mfma_lines(a.mfma, s)
            if m:
                lines += ["", "matrix cores (" + a.mfma_command + "):"] + m
        name = f"{e}_{a.workload}" + ("" if rank == wl.rank and W == wl.window else f"_r{rank}_w{W}")
        if sketch == "bf16":
            name += "_bf16sketch"
        if pivots:
            name += "_exactmap" if pivots < 0 else f"_pivots{pivots}"
        if "<" in s and e == "update" and re.search(r"<\d+, \d+, \d+, 0,", s):
            name += "_rank0"
        with open(os.path.join(a.out, name + ".txt"), "w") as f:
            f.write("\n".join(lines) + "\n")
        print("wrote", name + ".txt")
    with open(tpath, "w") as f:
        json.dump(table, f, indent=1, sort_keys=True)
        f.write("\n")
    return 0


if __name__ == "__main__":
    sys.exit(main())

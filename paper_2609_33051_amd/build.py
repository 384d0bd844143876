"""Compile libsketchssm.so for gfx950 with hipcc (in-tree, no JIT cache).

    python -m paper_2609_33051_amd.build [--force] [--jobs N]

Every translation unit under csrc/ is compiled to an object in _build/ (in
parallel), then linked into paper_2609_33051_amd/libsketchssm.so.  Without
--force only units whose sources or headers changed are recompiled.
"""
from __future__ import annotations

import argparse
import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libsketchssm.so")
INCLUDE = os.path.join(os.path.dirname(PKG), "include")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 math stays off: the compiler's v_pk_*_f32 forms are not used
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", "-Wno-unused-result",
]


def sources():
    return [os.path.join(CSRC, "abi.hip")] + sorted(glob.glob(os.path.join(CSRC, "units", "*.hip")))


def headers():
    return glob.glob(os.path.join(CSRC, "*.h")) + glob.glob(os.path.join(INCLUDE, "*.h"))


KERNEL_HEADERS = {"decode": "decode.h", "full_read": "decode.h", "update": "update.h"}


def unit_sources(unit: str) -> list[str]:
    """The files whose text decides the machine code of one unit's kernels
    (unit = "decode_mamba2", "update_gdn", ...): its translation units (the
    dispatcher and one per shape), the shared device and argument headers,
    the launch table and the kernel's own header."""
    entry = unit.rsplit("_", 1)[0]
    names = ["device.h", "args.h", "dispatch.h", KERNEL_HEADERS[entry]]
    units = sorted(glob.glob(os.path.join(CSRC, "units", unit + ".hip")) + glob.glob(os.path.join(CSRC, "units", unit + "_*.hip")))
    return units + [os.path.join(CSRC, n) for n in names]


def source_digest(unit: str) -> str:
    """sha256 over unit_sources(unit), with the build flags: a recorded
    measurement of a kernel is current only while this digest is unchanged."""
    import hashlib
    h = hashlib.sha256(" ".join(FLAGS[1:-2]).encode())
    for f in unit_sources(unit):
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def _obj(src):
    return os.path.join(BUILD, os.path.splitext(os.path.basename(src))[0] + ".o")


def _stale(src, newest_header):
    o = _obj(src)
    return not os.path.exists(o) or os.path.getmtime(o) < max(os.path.getmtime(src), newest_header)


def _compile(src, extra):
    o = _obj(src)
    cmd = [HIPCC, *FLAGS, *extra, "-c", src, "-o", o + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        return src, r.stdout + r.stderr
    os.replace(o + ".tmp", o)
    return src, None


def build(force: bool = False, jobs: int | None = None, extra=()) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    newest = max(os.path.getmtime(h) for h in headers())
    todo = [s for s in srcs if force or _stale(s, newest)]
    jobs = jobs or min(8, os.cpu_count() or 1)
    if todo:
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            errs = [(s, e) for s, e in ex.map(lambda s: _compile(s, list(extra)), todo) if e]
        if errs:
            msg = "\n".join(f"--- {s}\n{e}" for s, e in errs)
            raise RuntimeError(f"hipcc failed:\n{msg}")
    if todo or not os.path.exists(LIB):
        tmp = LIB + f".tmp{os.getpid()}"
        cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *[_obj(s) for s in srcs]]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
        os.replace(tmp, LIB)
    return LIB


def main(argv=None):
    p = argparse.ArgumentParser()
    p.add_argument("--force", action="store_true")
    p.add_argument("--jobs", type=int, default=None)
    args = p.parse_args(argv)
    print(build(force=args.force, jobs=args.jobs))


if __name__ == "__main__":
    sys.exit(main())

"""ctypes binding of libsketchssm.so (include/sketchssm.h).

Argument marshalling only: every step of the path runs in the HIP kernels.
The functions keep the C names and take device pointers either as integers
or as torch tensors (their data_ptr()); `stream` is a hipStream_t handle
(torch.cuda.current_stream().cuda_stream) or None for the default stream.
A non-OK status raises SketchSSMError with the library's message.  There is
no fallback: if the library is not built, loading raises.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libsketchssm.so")

MAMBA2, GDN, KDA = 0, 1, 2
KIND_IDS = {"mamba2": MAMBA2, "gdn": GDN, "kda": KDA}
F32, BF16 = 0, 1

STATUS = {0: "SKSSM_OK", -1: "SKSSM_EINVAL", -2: "SKSSM_EUNSUPPORTED", -3: "SKSSM_EALIGN",
          -4: "SKSSM_ESTATE", -5: "SKSSM_EHIP"}

FUNCTIONS = ("sketchssm_update", "sketchssm_decode", "sketchssm_full_read_baseline",
             "sketchssm_state_to_tiles", "sketchssm_state_from_tiles", "sketchssm_buffer_sizes",
             "sketchssm_ring_bytes", "sketchssm_status_string", "sketchssm_last_error", "sketchssm_check_config")


class SketchSSMError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in
                ("kind", "batch", "heads", "dk", "dv", "rank", "window", "io_dtype", "sketch_dtype", "pivots")] + [
                   ("ridge", ctypes.c_float), ("head_rank", ctypes.POINTER(ctypes.c_int32))]


BUFFERS = ("S", "U", "omega", "coef", "cmap", "q", "o", "ring_k", "ring_v", "ring_beta", "ring_log_decay",
           "ring_f", "ring_pi", "ring_tinv")


class BufferSizes(ctypes.Structure):
    _fields_ = [(name, ctypes.c_size_t) for name in BUFFERS]


class Ring(ctypes.Structure):
    _fields_ = [(name, ctypes.c_void_p) for name in
                ("k", "v", "beta", "log_decay", "f", "pi", "tinv")]


_lib = None


def load(path: str | None = None):
    """Load the library: `path`, else $SKETCHSSM_LIBRARY, else the in-tree build."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or os.environ.get("SKETCHSSM_LIBRARY") or LIB_PATH
    if not os.path.exists(path):
        raise FileNotFoundError(f"{path} is not built; run `python -m paper_2609_33051_amd.build`")
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    cfgp = ctypes.POINTER(Config)
    ringp = ctypes.POINTER(Ring)
    lib.sketchssm_update.argtypes = [cfgp, P, P, ringp, ctypes.c_int32, P, P, P, P, P]
    lib.sketchssm_decode.argtypes = [cfgp, P, P, P, P, ringp, ctypes.c_int32, P, P, P]
    lib.sketchssm_full_read_baseline.argtypes = [cfgp, P, ringp, ctypes.c_int32, P, P, P]
    lib.sketchssm_state_to_tiles.argtypes = [cfgp, P, P, P]
    lib.sketchssm_state_from_tiles.argtypes = [cfgp, P, P, P]
    for f in ("sketchssm_update", "sketchssm_decode", "sketchssm_full_read_baseline", "sketchssm_check_config",
              "sketchssm_state_to_tiles", "sketchssm_state_from_tiles"):
        getattr(lib, f).restype = ctypes.c_int
    lib.sketchssm_check_config.argtypes = [cfgp]
    lib.sketchssm_buffer_sizes.argtypes = [cfgp, ctypes.c_int32, ctypes.POINTER(BufferSizes)]
    lib.sketchssm_buffer_sizes.restype = ctypes.c_int
    lib.sketchssm_ring_bytes.argtypes = [cfgp, ctypes.c_int32]
    lib.sketchssm_ring_bytes.restype = ctypes.c_size_t
    lib.sketchssm_status_string.argtypes = [ctypes.c_int]
    lib.sketchssm_status_string.restype = ctypes.c_char_p
    lib.sketchssm_last_error.argtypes = []
    lib.sketchssm_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def ptr(x) -> int | None:
    """Device address of a tensor (or an int / None passed through)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _dtype(x) -> int:
    return {"f32": F32, "bf16": BF16}[x] if isinstance(x, str) else int(x)


def make_config(kind, batch, heads, dk, dv, rank, window, io, sketch="f32", pivots=0, ridge=0.1,
                head_ranks=None) -> Config:
    """head_ranks: optional per-head rank table (H ints, 0 = dense fallback);
    `rank` is then the storage width.  The table is copied into host memory
    owned by the returned Config."""
    k = KIND_IDS[kind] if isinstance(kind, str) else int(kind)
    cfg = Config(k, batch, heads, dk, dv, rank, window, _dtype(io), _dtype(sketch), int(pivots), float(ridge), None)
    if head_ranks is not None:
        vals = [int(x) for x in head_ranks]
        if len(vals) != heads:
            raise ValueError(f"head_ranks has {len(vals)} entries for {heads} heads")
        arr = (ctypes.c_int32 * heads)(*vals)
        cfg.head_rank = ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32))
        cfg._head_rank_storage = arr
    return cfg


def head_ranks(cfg: Config) -> list[int] | None:
    """The per-head rank table of a Config, or None."""
    return None if not cfg.head_rank else [cfg.head_rank[h] for h in range(cfg.heads)]


def make_ring(k=None, v=None, beta=None, log_decay=None, f=None, pi=None, tinv=None) -> Ring:
    return Ring(ptr(k), ptr(v), ptr(beta), ptr(log_decay), ptr(f), ptr(pi), ptr(tinv))


def _check(rc: int):
    if rc != 0:
        raise SketchSSMError(rc, load().sketchssm_last_error().decode())


class Prepared:
    """One entry-point call with its arguments marshalled once, so that a
    caller replaying the same launch (a decode loop over resident buffers)
    pays only the foreign call.  The Config and Ring it points to are kept
    alive with it."""

    __slots__ = ("fn", "args", "keep")

    def __init__(self, fn, args, keep):
        self.fn, self.args, self.keep = fn, args, keep

    def __call__(self):
        rc = self.fn(*self.args)
        if rc:
            _check(rc)


def _vp(x):
    p = ptr(x)
    return None if p is None else ctypes.c_void_p(p)


def prepare_update(cfg: Config, S, omega, ring: Ring | None, n_buffered: int, q, U, o, stream=None,
                   cmap=None) -> Prepared:
    lib = load()
    args = (ctypes.byref(cfg), _vp(S), _vp(omega), ctypes.byref(ring) if ring else None, ctypes.c_int32(n_buffered),
            _vp(q), _vp(U), _vp(cmap), _vp(o), _vp(stream))
    return Prepared(lib.sketchssm_update, args, (cfg, ring))


def prepare_decode(cfg: Config, U, coef, ring: Ring, n_buffered: int, q, o, stream=None, cmap=None,
                   S=None) -> Prepared:
    lib = load()
    args = (ctypes.byref(cfg), _vp(U), _vp(coef), _vp(cmap), _vp(S), ctypes.byref(ring), ctypes.c_int32(n_buffered),
            _vp(q), _vp(o), _vp(stream))
    return Prepared(lib.sketchssm_decode, args, (cfg, ring))


def prepare_full_read_baseline(cfg: Config, S, ring: Ring, n_buffered: int, q, o, stream=None) -> Prepared:
    lib = load()
    args = (ctypes.byref(cfg), _vp(S), ctypes.byref(ring), ctypes.c_int32(n_buffered), _vp(q), _vp(o), _vp(stream))
    return Prepared(lib.sketchssm_full_read_baseline, args, (cfg, ring))


def sketchssm_update(cfg: Config, S, omega, ring: Ring | None, n_buffered: int, q, U, o, stream=None, cmap=None):
    lib = load()
    _check(lib.sketchssm_update(ctypes.byref(cfg), ptr(S), ptr(omega), ctypes.byref(ring) if ring else None,
                                int(n_buffered), ptr(q), ptr(U), ptr(cmap), ptr(o), stream))


def sketchssm_decode(cfg: Config, U, coef, ring: Ring, n_buffered: int, q, o, stream=None, cmap=None, S=None):
    lib = load()
    _check(lib.sketchssm_decode(ctypes.byref(cfg), ptr(U), ptr(coef), ptr(cmap), ptr(S),
                                ctypes.byref(ring) if ring else None, int(n_buffered), ptr(q), ptr(o), stream))


def sketchssm_full_read_baseline(cfg: Config, S, ring: Ring, n_buffered: int, q, o, stream=None):
    lib = load()
    _check(lib.sketchssm_full_read_baseline(ctypes.byref(cfg), ptr(S), ctypes.byref(ring) if ring else None,
                                            int(n_buffered), ptr(q), ptr(o), stream))


def sketchssm_state_to_tiles(cfg: Config, S_rows, S, stream=None):
    """Row layout X[B][H][V][K] -> the tile-major state the other calls use."""
    _check(load().sketchssm_state_to_tiles(ctypes.byref(cfg), ptr(S_rows), ptr(S), stream))


def sketchssm_state_from_tiles(cfg: Config, S, S_rows, stream=None):
    """Tile-major state -> row layout X[B][H][V][K]."""
    _check(load().sketchssm_state_from_tiles(ctypes.byref(cfg), ptr(S), ptr(S_rows), stream))


def sketchssm_buffer_sizes(cfg: Config, baseline: bool = False) -> dict:
    """Bytes of every caller-owned buffer of a layer (the library's sizes query)."""
    out = BufferSizes()
    _check(load().sketchssm_buffer_sizes(ctypes.byref(cfg), 1 if baseline else 0, ctypes.byref(out)))
    return {name: int(getattr(out, name)) for name in BUFFERS}


def sketchssm_ring_bytes(cfg: Config, baseline: bool = False) -> int:
    return int(load().sketchssm_ring_bytes(ctypes.byref(cfg), 1 if baseline else 0))


def sketchssm_check_config(cfg: Config) -> int:
    return int(load().sketchssm_check_config(ctypes.byref(cfg)))


def sketchssm_status_string(status: int) -> str:
    return load().sketchssm_status_string(int(status)).decode()


def sketchssm_last_error() -> str:
    return load().sketchssm_last_error().decode()

// Host side of the C ABI declared in include/sketchssm.h: argument
// validation (before anything is enqueued), dispatch to the compiled kernel
// of the shape, and error reporting.  No allocation, no synchronisation.
#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>

#include "../../include/sketchssm.h"
#include "args.h"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

constexpr int64_t kMaxItems = (int64_t)1 << 23;

bool aligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Shape checks common to every entry point.
int check_shape(const skssm_config* c, bool need_rank, bool allow_rank0) {
  if (!c) return fail(SKSSM_EINVAL, "cfg is NULL");
  if (c->kind < SKSSM_MAMBA2 || c->kind > SKSSM_KDA) return fail(SKSSM_EINVAL, "unknown kind %d", c->kind);
  if (c->batch < 1 || c->heads < 1) return fail(SKSSM_EINVAL, "batch and heads must be >= 1");
  // one slot of a derived ring field (at most 512 bytes per item) must span
  // less than 4 GiB: the kernels step between slots with 32-bit byte strides
  if ((int64_t)c->batch * c->heads >= kMaxItems)
    return fail(SKSSM_EUNSUPPORTED, "batch*heads = %lld: at most %lld items", (long long)c->batch * c->heads,
                (long long)kMaxItems - 1);
  if (c->io_dtype != SKSSM_F32 && c->io_dtype != SKSSM_BF16) return fail(SKSSM_EINVAL, "unknown io_dtype %d", c->io_dtype);
  if (c->sketch_dtype != SKSSM_F32 && c->sketch_dtype != SKSSM_BF16)
    return fail(SKSSM_EINVAL, "unknown sketch_dtype %d", c->sketch_dtype);
  if (c->pivots != 0 && c->pivots != 4 && c->pivots != SKSSM_EXACT_MAP)
    return fail(SKSSM_EUNSUPPORTED, "pivots %d: 0, 4 or SKSSM_EXACT_MAP (-1) are compiled", c->pivots);
  // lambda > 0 keeps the map's diagonal D = d + lambda invertible where d = 0
  // (a zero state, sketch columns past a head's rank); the paper uses 0.1
  if (c->pivots && !(c->ridge > 0.f && c->ridge < 1e30f))
    return fail(SKSSM_EINVAL, "ridge must be finite and > 0 with a state-dependent map");
  if (c->window < 1 || c->window > 32) return fail(SKSSM_EUNSUPPORTED, "window %d outside 1..32", c->window);
  const bool kv_ok = (c->dk == 64 && c->dv == 64) || (c->dk == 128 && c->dv == 64) || (c->dk == 128 && c->dv == 128);
  if (!kv_ok) return fail(SKSSM_EUNSUPPORTED, "(dk, dv) = (%d, %d) not compiled", c->dk, c->dv);
  if (need_rank) {
    const bool r_ok = c->rank == 8 || c->rank == 16 || c->rank == 32 || c->rank == c->dk || (allow_rank0 && c->rank == 0);
    if (!r_ok) return fail(c->rank < 0 ? SKSSM_EINVAL : SKSSM_EUNSUPPORTED, "rank %d not supported", c->rank);
  }
  return SKSSM_OK;
}

// State-dependent maps: P = 4 pivots for ranks 8..32, the exact metric for
// ranks 8 and 16 (the storage width with a rank table).
int check_map_rank(const skssm_config* c) {
  if (c->pivots == SKSSM_EXACT_MAP && c->rank != 8 && c->rank != 16)
    return fail(SKSSM_EUNSUPPORTED, "the exact-metric map is compiled for rank 8 and 16");
  if (c->rank < 8 || c->rank > 32) return fail(SKSSM_EUNSUPPORTED, "state-dependent maps need rank 8..32");
  return SKSSM_OK;
}

// Ring fields read or written by a call: the raw inputs always, the derived
// fields of the family, and f (`derived_f`, sketch read) or pi
// (`derived_pi`, exact baseline).
int check_ring(const skssm_config* c, const skssm_ring* r, bool derived_f, bool derived_pi) {
  if (!r) return fail(SKSSM_EINVAL, "ring is NULL");
  if (!r->k || !r->v || !r->beta || !r->log_decay) return fail(SKSSM_EINVAL, "ring k/v/beta/log_decay is NULL");
  if (!aligned(r->k) || !aligned(r->v) || !aligned(r->beta) || !aligned(r->log_decay))
    return fail(SKSSM_EALIGN, "ring input field not 16-byte aligned");
  if (c->kind != SKSSM_MAMBA2) {
    if (!r->tinv) return fail(SKSSM_EINVAL, "ring tinv is NULL (GDN/KDA)");
    if (!aligned(r->tinv)) return fail(SKSSM_EALIGN, "ring tinv not aligned");
    if (derived_f && !r->f) return fail(SKSSM_EINVAL, "ring f is NULL (GDN/KDA sketch read)");
    if (derived_f && !aligned(r->f)) return fail(SKSSM_EALIGN, "ring f not aligned");
    if (derived_pi && !r->pi) return fail(SKSSM_EINVAL, "ring pi is NULL (GDN/KDA baseline)");
    if (derived_pi && !aligned(r->pi)) return fail(SKSSM_EALIGN, "ring pi not aligned");
  }
  return SKSSM_OK;
}

// Per-head rank table (cfg->head_rank): validated here and copied into the
// kernel arguments.  Counts the dense-fallback and the sketched heads.
struct Ranks {
  int ragged = 0, dense = 0, sketched = 0;
  uint8_t h[skssm::kMaxRaggedHeads] = {};
  uint8_t order[skssm::kMaxRaggedHeads] = {};  // dense heads first, then the sketched ones
};

int check_ranks(const skssm_config* c, Ranks& rk) {
  rk = Ranks{};
  if (!c->head_rank) {
    rk.sketched = c->heads;
    return SKSSM_OK;
  }
  if (c->heads > skssm::kMaxRaggedHeads)
    return fail(SKSSM_EUNSUPPORTED, "a per-head rank table supports at most %d heads", skssm::kMaxRaggedHeads);
  if (c->rank != 8 && c->rank != 16 && c->rank != 32)
    return fail(SKSSM_EUNSUPPORTED, "with a per-head rank table, rank (the storage width) must be 8, 16 or 32");
  for (int h = 0; h < c->heads; ++h) {
    const int32_t g = c->head_rank[h];
    if (g < 0 || g > c->rank) return fail(SKSSM_EINVAL, "head_rank[%d] = %d outside 0..%d", h, g, c->rank);
    rk.h[h] = (uint8_t)g;
    if (g == 0) ++rk.dense; else ++rk.sketched;
  }
  int d = 0, k = rk.dense;
  for (int h = 0; h < c->heads; ++h) rk.order[rk.h[h] == 0 ? d++ : k++] = (uint8_t)h;
  rk.ragged = 1;
  return SKSSM_OK;
}

// The decode launches the dense heads' workgroups first: each reads a whole
// state and takes several times as long as a sketch read, so starting them
// early keeps them from trailing the launch.
void put_order(skssm::DecodeArgs& a, const Ranks& rk) {
  a.ndense = rk.dense;
  for (int h = 0; h < skssm::kMaxRaggedHeads; ++h) a.hlist[h] = rk.order[h];
}

template <class A> void put_ranks(A& a, const Ranks& rk) {
  a.ragged = rk.ragged;
  for (int h = 0; h < skssm::kMaxRaggedHeads; ++h) a.hrank[h] = rk.h[h];
}

int launched(int rc, const char* what) {
  if (rc == -2) return fail(SKSSM_EUNSUPPORTED, "%s: no kernel compiled for this shape", what);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(SKSSM_EHIP, "%s: %s", what, hipGetErrorString(e));
  g_err[0] = '\0';
  return SKSSM_OK;
}

skssm::DecodeArgs decode_args(const skssm_config* c, const skssm_ring* r, int32_t n, const void* q, float* o) {
  skssm::DecodeArgs a{};
  a.B = c->batch;
  a.H = c->heads;
  a.W = c->window;
  a.n = n;
  a.q = q;
  a.rk = r->k;
  a.rv = r->v;
  a.rbeta = r->beta;
  a.rla = r->log_decay;
  a.rf = r->f;
  a.rpi = r->pi;
  a.rt = r->tinv;
  a.o = o;
  return a;
}

int state_layout(const skssm_config* cfg, const float* src, float* dst, void* stream, int to_tiles,
                        const char* what) {
  int rc = check_shape(cfg, false, true);
  if (rc) return rc;
  if (!src || !dst) return fail(SKSSM_EINVAL, "%s: source and destination are required", what);
  if (!aligned(src) || !aligned(dst)) return fail(SKSSM_EALIGN, "%s: source/destination not aligned", what);
  const size_t items = (size_t)cfg->batch * cfg->heads;
  const size_t bytes = items * cfg->dk * cfg->dv * sizeof(float);
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  if (s0 < d0 + bytes && d0 < s0 + bytes) return fail(SKSSM_EINVAL, "%s: source and destination overlap", what);
  return launched(skssm::run_state_layout(src, dst, items, cfg->dk, cfg->dv, to_tiles, stream), what);
}

}  // namespace

extern "C" {

const char* sketchssm_status_string(int status) {
  switch (status) {
    case SKSSM_OK: return "ok";
    case SKSSM_EINVAL: return "invalid argument";
    case SKSSM_EUNSUPPORTED: return "unsupported shape";
    case SKSSM_EALIGN: return "pointer not 16-byte aligned";
    case SKSSM_ESTATE: return "n_buffered out of range";
    case SKSSM_EHIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* sketchssm_last_error(void) { return g_err; }

int sketchssm_check_config(const skssm_config* cfg) { return check_shape(cfg, true, false); }

int sketchssm_update(const skssm_config* cfg, float* S, const float* omega, const skssm_ring* ring,
                     int32_t n_buffered, const void* q, void* U, void* cmap, float* o, void* stream) {
  int rc = check_shape(cfg, true, true);
  if (rc) return rc;
  Ranks rk;
  if ((rc = check_ranks(cfg, rk))) return rc;
  if (cfg->pivots) {
    if ((rc = check_map_rank(cfg))) return rc;
    if (!cmap) return fail(SKSSM_EINVAL, "cmap is required when pivots > 0");
    if (!aligned(cmap)) return fail(SKSSM_EALIGN, "cmap not aligned");
  }
  if (!S) return fail(SKSSM_EINVAL, "S is NULL");
  if (!aligned(S)) return fail(SKSSM_EALIGN, "S not aligned");
  if (cfg->rank > 0) {
    if (!U || !omega) return fail(SKSSM_EINVAL, "U and omega are required when rank > 0");
    if (!aligned(U) || !aligned(omega)) return fail(SKSSM_EALIGN, "U/omega not aligned");
  }
  if (o && !aligned(o)) return fail(SKSSM_EALIGN, "o not aligned");
  skssm::UpdateArgs a{};
  a.B = cfg->batch;
  a.H = cfg->heads;
  a.W = cfg->window;
  a.n = n_buffered;
  put_ranks(a, rk);
  a.S = S;
  a.omega = omega;
  a.U = cfg->rank > 0 ? U : nullptr;
  a.cmap = cfg->pivots ? cmap : nullptr;
  a.ridge = cfg->ridge;
  if (q) {
    if (n_buffered < 0 || n_buffered > cfg->window - 1)
      return fail(SKSSM_ESTATE, "n_buffered %d outside 0..%d", n_buffered, cfg->window - 1);
    if (!aligned(q)) return fail(SKSSM_EALIGN, "q not aligned");
    if ((rc = check_ring(cfg, ring, false, false))) return rc;
    a.nt = n_buffered + 1;
    a.q = q;
    a.rk = ring->k;
    a.rv = ring->v;
    a.rbeta = ring->beta;
    a.rla = ring->log_decay;
    a.rt = ring->tinv;
    a.o = o;
  } else {
    if (n_buffered != 0) return fail(SKSSM_ESTATE, "sketch-only update needs n_buffered = 0");
    if (cfg->rank == 0 || !U) return fail(SKSSM_EINVAL, "sketch-only update needs rank > 0 and U");
    a.nt = 0;
    a.o = nullptr;
    if (rk.sketched == 0) {  // every head is dense: no sketch to build
      g_err[0] = '\0';
      return SKSSM_OK;
    }
  }
  int r;
  switch (cfg->kind) {
    case SKSSM_MAMBA2: r = skssm::run_update_mamba2(a, cfg->dk, cfg->dv, cfg->rank, cfg->io_dtype, cfg->sketch_dtype, cfg->pivots, stream); break;
    case SKSSM_GDN: r = skssm::run_update_gdn(a, cfg->dk, cfg->dv, cfg->rank, cfg->io_dtype, cfg->sketch_dtype, cfg->pivots, stream); break;
    default: r = skssm::run_update_kda(a, cfg->dk, cfg->dv, cfg->rank, cfg->io_dtype, cfg->sketch_dtype, cfg->pivots, stream); break;
  }
  return launched(r, "sketchssm_update");
}

int sketchssm_decode(const skssm_config* cfg, const void* U, const float* coef, const void* cmap, const float* S,
                     const skssm_ring* ring, int32_t n_buffered, const void* q, float* o, void* stream) {
  int rc = check_shape(cfg, true, false);
  if (rc) return rc;
  Ranks rk;
  if ((rc = check_ranks(cfg, rk))) return rc;
  if (cfg->pivots) {
    if ((rc = check_map_rank(cfg))) return rc;
    if (!cmap) return fail(SKSSM_EINVAL, "cmap is required when pivots > 0");
    if (!aligned(cmap)) return fail(SKSSM_EALIGN, "cmap not aligned");
  }
  if (cfg->window < 2) return fail(SKSSM_EINVAL, "decode needs window >= 2 (window 1 flushes every token)");
  if (n_buffered < 0 || n_buffered > cfg->window - 2)
    return fail(SKSSM_ESTATE, "n_buffered %d outside 0..%d", n_buffered, cfg->window - 2);
  if (!U || !o || !q) return fail(SKSSM_EINVAL, "U, q and o are required");
  if (!cfg->pivots && !coef) return fail(SKSSM_EINVAL, "coef is required with the offline map (pivots = 0)");
  if (!aligned(U) || !aligned(o) || !aligned(q) || (coef && !aligned(coef)))
    return fail(SKSSM_EALIGN, "U/coef/q/o not aligned");
  if (rk.dense) {  // dense-fallback heads read the state (and keep pi in the ring)
    if (!S) return fail(SKSSM_EINVAL, "S is required when the rank table has dense-fallback heads");
    if (!aligned(S)) return fail(SKSSM_EALIGN, "S not aligned");
  }
  if ((rc = check_ring(cfg, ring, rk.sketched > 0, rk.dense > 0))) return rc;
  skssm::DecodeArgs a = decode_args(cfg, ring, n_buffered, q, o);
  put_ranks(a, rk);
  put_order(a, rk);
  a.S = rk.dense ? S : nullptr;
  a.U = U;
  a.coef = cfg->pivots ? nullptr : coef;
  a.cmap = cfg->pivots ? cmap : nullptr;
  int r;
  switch (cfg->kind) {
    case SKSSM_MAMBA2: r = skssm::run_decode_mamba2(a, cfg->dk, cfg->dv, cfg->rank, cfg->io_dtype, cfg->sketch_dtype, cfg->pivots, stream); break;
    case SKSSM_GDN: r = skssm::run_decode_gdn(a, cfg->dk, cfg->dv, cfg->rank, cfg->io_dtype, cfg->sketch_dtype, cfg->pivots, stream); break;
    default: r = skssm::run_decode_kda(a, cfg->dk, cfg->dv, cfg->rank, cfg->io_dtype, cfg->sketch_dtype, cfg->pivots, stream); break;
  }
  return launched(r, "sketchssm_decode");
}

int sketchssm_full_read_baseline(const skssm_config* cfg, const float* S, const skssm_ring* ring,
                                 int32_t n_buffered, const void* q, float* o, void* stream) {
  int rc = check_shape(cfg, false, false);
  if (rc) return rc;
  Ranks rk;
  if ((rc = check_ranks(cfg, rk))) return rc;
  if (cfg->window < 2) return fail(SKSSM_EINVAL, "baseline read needs window >= 2");
  if (n_buffered < 0 || n_buffered > cfg->window - 2)
    return fail(SKSSM_ESTATE, "n_buffered %d outside 0..%d", n_buffered, cfg->window - 2);
  if (!S || !o || !q) return fail(SKSSM_EINVAL, "S, q and o are required");
  if (!aligned(S) || !aligned(o) || !aligned(q)) return fail(SKSSM_EALIGN, "S/q/o not aligned");
  if ((rc = check_ring(cfg, ring, false, true))) return rc;
  skssm::DecodeArgs a = decode_args(cfg, ring, n_buffered, q, o);
  a.S = S;
  int r;
  switch (cfg->kind) {
    case SKSSM_MAMBA2: r = skssm::run_full_read_mamba2(a, cfg->dk, cfg->dv, cfg->io_dtype, stream); break;
    case SKSSM_GDN: r = skssm::run_full_read_gdn(a, cfg->dk, cfg->dv, cfg->io_dtype, stream); break;
    default: r = skssm::run_full_read_kda(a, cfg->dk, cfg->dv, cfg->io_dtype, stream); break;
  }
  return launched(r, "sketchssm_full_read_baseline");
}

int sketchssm_buffer_sizes(const skssm_config* cfg, int32_t baseline, skssm_buffer_sizes* out) {
  if (!out) return fail(SKSSM_EINVAL, "out is NULL");
  *out = skssm_buffer_sizes{};
  int rc = check_shape(cfg, !baseline, !baseline);
  if (rc) return rc;
  Ranks rk;
  if (!baseline && (rc = check_ranks(cfg, rk))) return rc;
  const size_t B = (size_t)cfg->batch, H = (size_t)cfg->heads, K = (size_t)cfg->dk, V = (size_t)cfg->dv;
  const size_t W = (size_t)cfg->window, r = baseline ? 0 : (size_t)cfg->rank;
  const size_t io = cfg->io_dtype == SKSSM_BF16 ? 2 : 4, sk = cfg->sketch_dtype == SKSSM_BF16 ? 2 : 4;
  const bool erase = cfg->kind != SKSSM_MAMBA2;
  out->S = B * H * V * K * 4;
  out->U = B * H * V * r * sk;
  out->omega = H * K * r * 4;
  out->coef = cfg->pivots ? 0 : H * r * K * 4;
  out->cmap = cfg->pivots && !baseline ? B * H * r * K * sk : 0;
  out->q = B * H * K * io;
  out->o = B * H * V * 4;
  out->ring_k = B * H * W * K * io;
  out->ring_v = B * H * W * V * io;
  out->ring_beta = B * H * W * 4;
  out->ring_log_decay = B * H * W * (cfg->kind == SKSSM_KDA ? K : 1) * 4;
  if (erase) {
    out->ring_tinv = W * H * B * W * 4;
    out->ring_f = (!baseline && rk.sketched > 0) ? W * H * B * r * sk : 0;
    out->ring_pi = (baseline || rk.dense > 0) ? W * H * B * K * 4 : 0;
  }
  g_err[0] = '\0';
  return SKSSM_OK;
}

size_t sketchssm_ring_bytes(const skssm_config* cfg, int32_t baseline) {
  skssm_buffer_sizes z;
  if (sketchssm_buffer_sizes(cfg, baseline, &z) != SKSSM_OK) return 0;
  return z.ring_k + z.ring_v + z.ring_beta + z.ring_log_decay + z.ring_f + z.ring_pi + z.ring_tinv;
}

int sketchssm_state_to_tiles(const skssm_config* cfg, const float* S_rows, float* S, void* stream) {
  return state_layout(cfg, S_rows, S, stream, 1, "sketchssm_state_to_tiles");
}

int sketchssm_state_from_tiles(const skssm_config* cfg, const float* S, float* S_rows, void* stream) {
  return state_layout(cfg, S, S_rows, stream, 0, "sketchssm_state_from_tiles");
}

}  // extern "C"

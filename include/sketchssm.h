/*
 * sketchssm.h -- C ABI of the SketchSSM decode hot path on MI355X (gfx950).
 *
 * SketchSSM (arXiv 2609.33051) serves the linear-attention layers of hybrid
 * models (Mamba-2 scalar decay, GDN gated delta rule, KDA channel-wise decay)
 * during decoding.  Every (request b, head h) keeps a full fp32 recurrent
 * state S.  Algorithm 1 splits the decode loop into windows of W tokens:
 *
 *   - W-1 non-flush steps append the token's update inputs to a replay buffer
 *     and read the output from a compact sketch, o_t = U c_t + o_t^buffer
 *     (Sec. 3.3, eq. equantion-sketch), never touching S;
 *   - one flush step applies every buffered update to S exactly, emits the
 *     exact output o_W = S_W^T q_W and rebuilds the sketch U = S_W^T Omega
 *     from the same single read of S (Sec. 4.1, "Per-window: Sketch").
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Layout.  The paper writes S as K x V with o = S^T q; this library stores
 * its transpose, S[B][H][V][K] fp32 with K contiguous, so a row S[b][h][v][:]
 * is contiguous.  All other per-item tensors are [B][H][...] row-major with
 * the item index b*H + h.  The sketch U[B][H][V][r] is fp32 (U[.., v, g] is
 * the output of basis query g at value channel v).  Omega[H][K][r] and the
 * coefficient map coef[H][r][K] (C, shared by the batch) are fp32.
 *
 * Memory.  Every pointer is a device pointer owned by the caller; the library
 * never allocates, frees or synchronises, keeps no per-call state and is
 * re-entrant.  All work is enqueued on `stream` (a hipStream_t; NULL = the
 * default stream).  Pointers must be 16-byte aligned.
 *
 * Errors.  Arguments are validated on the host before any launch; a negative
 * skssm_status is returned and nothing is enqueued.  A launch failure returns
 * SKSSM_EHIP with the HIP error text available from sketchssm_last_error()
 * (thread-local).  Outputs are unspecified after a non-OK return.  Nothing
 * aborts and no exception crosses the ABI.
 *
 * Supported shapes.  (dk, dv) in {(64,64), (128,64), (128,128)};
 * rank in {8, 16, 32, dk} (0 where stated); window 1..32; io dtype fp32 or
 * bf16 for q, k, v and the ring's raw keys and values.
 */
#ifndef SKETCHSSM_H
#define SKETCHSSM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SKSSM_OK = 0,
  SKSSM_EINVAL = -1,       /* null pointer, bad enum value, bad size          */
  SKSSM_EUNSUPPORTED = -2, /* valid but not compiled: (dk, dv, rank, window)  */
  SKSSM_EALIGN = -3,       /* a pointer is not 16-byte aligned                */
  SKSSM_ESTATE = -4,       /* n_buffered outside the range the call allows    */
  SKSSM_EHIP = -5          /* the HIP runtime reported an error               */
} skssm_status;

typedef enum {
  SKSSM_MAMBA2 = 0, /* M_t = alpha_t I            (scalar decay, no erase)       */
  SKSSM_GDN = 1,    /* M_t = (I - beta k k^T) alpha_t     (gated delta rule)     */
  SKSSM_KDA = 2     /* M_t = (I - beta k k^T) Diag(alpha_t)  (channel decay)     */
} skssm_kind;

typedef enum { SKSSM_F32 = 0, SKSSM_BF16 = 1 } skssm_dtype;

/* Shape of one linear-attention layer. */
typedef struct {
  int32_t kind;     /* skssm_kind                                           */
  int32_t batch;    /* B requests                                           */
  int32_t heads;    /* H heads                                              */
  int32_t dk;       /* K key channels  (Mamba-2 d_state N)                  */
  int32_t dv;       /* V value channels (Mamba-2 headdim P)                 */
  int32_t rank;     /* r sketch columns (the paper's G)                     */
  int32_t window;   /* W tokens per window = ring capacity                  */
  int32_t io_dtype; /* skssm_dtype of q, k, v and ring.k / ring.v           */
} skssm_config;

/* One decode token for every (b, h).  Mamba-2 maps q = C_t, k = B_t,
 * v = x_t, beta = dt and log_decay = dt * A_h (Sec. 3.2, M_t = D_t). */
typedef struct {
  const void* q;          /* [B][H][K] io_dtype                                  */
  const void* k;          /* [B][H][K] io_dtype                                  */
  const void* v;          /* [B][H][V] io_dtype                                  */
  const float* beta;      /* [B][H] write gate beta_t                            */
  const float* log_decay; /* [B][H] (MAMBA2, GDN) or [B][H][K] (KDA), log alpha <= 0 */
} skssm_step;

/* Replay buffer ("ring"), W slots per (b, h), slot-major: field[B][H][W][...].
 * Slot s holds the s-th token of the current window (0-based).  Besides the
 * raw update inputs the ring keeps fields derived when a token is appended,
 * so that later reads are parallel reductions over slots (Appendix C):
 *   g      window-local cumulative log decay, g_s = sum_{j<=s} log alpha_j,
 *          so every decay ratio is exp(g_t - g_s) <= 1 (never a division);
 *   bcoef  b_{s,j} = <exp(g_s - g_j) k_j, k_s>, j < s      (erase couplings);
 *   u      pseudo-values u_s = beta_s (v_s - sum_{j<s} b_{s,j} u_j), which
 *          carry the erase into the buffer output o^buf = sum_s a_{t,s} u_s;
 *   f      projected erase factors f_s = C pi_s in R^r (eq. wyread), read by
 *          sketchssm_decode;
 *   pi     erase factors pi_s in R^K (eq. wy), read by the exact baseline.
 * Unused fields may be NULL. */
typedef struct {
  void* k;      /* [W][K] io_dtype raw keys                          all kinds   */
  void* v;      /* [W][V] io_dtype raw values                        MAMBA2      */
  float* u;     /* [W][V] pseudo-values                              GDN, KDA    */
  float* f;     /* [W][rank] projected erase factors                 GDN, KDA (decode)   */
  float* pi;    /* [W][K] erase factors                              GDN, KDA (baseline) */
  float* g;     /* [W] (MAMBA2, GDN) or [W][K] (KDA) cumulative log decay        */
  float* beta;  /* [W] write gates                                   all kinds   */
  float* bcoef; /* [W][W] row s holds b_{s,j} for j < s              GDN, KDA    */
} skssm_ring;

/*
 * sketchssm_update -- flush step, initial sketch, or Standard step.
 * Algorithm 1 (flush) and Sec. 4.1: the single full-state read per window.
 *
 *   step != NULL: the token `step` completes the window after n_buffered
 *     (0..W-1) ring slots.  Reads S once, applies the n_buffered + 1 updates
 *     exactly (rank-(n_buffered+1) form of eq. update, on matrix cores),
 *     writes o = S_W^T q_W (if o != NULL), U = S_W^T Omega (if rank > 0) and
 *     S_W back in place.  The caller then restarts the window (next
 *     n_buffered = 0); the ring needs no clearing.  window = 1 with rank = 0
 *     is the Standard recurrence (one read and one write of S per token).
 *   step == NULL: builds U = S^T Omega from S alone (initial sketch after
 *     prefill, Algorithm 1 "Construct the initial U"); n_buffered must be 0,
 *     S is not written and o is ignored.
 *
 * S      [B][H][V][K] fp32, read and (step != NULL) written in place.
 * omega  [H][K][rank] fp32 (may be NULL when rank == 0).
 * ring   read-only here; only the fields of `kind` (k, g, beta; v for MAMBA2;
 *        u and bcoef for GDN/KDA) are read, slots 0..n_buffered-1.
 * U      [B][H][V][rank] fp32 output (may be NULL when rank == 0).
 * o      [B][H][V] fp32 output or NULL.
 * rank may be 0 here (no sketch: the flush of the exact baseline).
 */
int sketchssm_update(const skssm_config* cfg, float* S, const float* omega, const skssm_ring* ring,
                     int32_t n_buffered, const skssm_step* step, float* U, float* o, void* stream);

/*
 * sketchssm_decode -- non-flush step (Algorithm 1, t < W): appends `step` at
 * ring slot n_buffered (0..W-2) and writes
 *     o = U c_t + o_t^buffer,
 *     c_t = C (e^{g_t} . q_t) - sum_{s<=t} a_{t,s} f_s        (eq. app-projected-query)
 *     o_t^buffer = sum_{s<=t} a_{t,s} u_s,  a_{t,s} = <exp(g_t - g_s) k_s, q_t>
 * (for MAMBA2 f_s = 0 and u_s = beta_s v_s, so c_t = e^{g_t} C q_t).  S is
 * never read.  U [B][H][V][rank] fp32 and coef [H][rank][K] fp32 (C; Omega^T
 * for the offline map of Sec. 4.1 at E0 = I) are read; the ring slot
 * n_buffered is written (k, g, beta; v for MAMBA2; u, f and the bcoef row for
 * GDN/KDA).  o [B][H][V] fp32.  rank must be > 0 and window >= 2.
 */
int sketchssm_decode(const skssm_config* cfg, const float* U, const float* coef, const skssm_ring* ring,
                     int32_t n_buffered, const skssm_step* step, float* o, void* stream);

/*
 * sketchssm_full_read_baseline -- exact non-flush step that reads all of S
 * (ReplaySSM-style; the reference the sketch read is measured against):
 *     o = S_0^T q~_t + o_t^buffer,  q~_t = e^{g_t} . q_t - sum_{s<=t} a_{t,s} pi_s
 * (eq. m-reads with the effective query of eq. app-effective-query-wy).
 * Appends `step` at slot n_buffered (0..W-2): k, g, beta (v for MAMBA2;
 * u, pi and the bcoef row for GDN/KDA).  S [B][H][V][K] is only read.
 * Flushes of this path use sketchssm_update with rank = 0.  cfg->rank is
 * ignored.
 */
int sketchssm_full_read_baseline(const skssm_config* cfg, const float* S, const skssm_ring* ring,
                                 int32_t n_buffered, const skssm_step* step, float* o, void* stream);

/* Static text for a status code. */
const char* sketchssm_status_string(int status);
/* Detail of the last failure on this thread (validation message or HIP error text). */
const char* sketchssm_last_error(void);
/* SKSSM_OK if every entry point supports cfg's shape (window/rank limits per call as above). */
int sketchssm_check_config(const skssm_config* cfg);

#ifdef __cplusplus
}
#endif
#endif /* SKETCHSSM_H */

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
 *     from the same single read of S (Sec. 4.1, per-window sketch).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Layout.  The paper writes S as K x V with o = S^T q; this library keeps
 * its transpose X = S^T (V x K per item, fp32) in a tile-major layout: item
 * b*H + h holds (V/16) x (K/16) tiles of 16 x 16, tile (vt, kt) at offset
 * (vt * K/16 + kt) * 256 floats, and within a tile X[16 vt + r][16 kt + c]
 * at 4 (r + 16 (c / 4)) + c % 4.  That is the register layout of the flush's
 * matrix-core accumulators, so every state load and store moves 1 KB
 * contiguous.  sketchssm_state_to_tiles / sketchssm_state_from_tiles convert
 * from and to the row layout X[B][H][V][K].  All other per-item tensors are
 * [B][H][...] row-major with the item index b*H + h.  The sketch is stored in panels of 16 bytes per
 * value channel, U[B][H][r/P][V][P] with P = 4 columns (fp32) or P = 8
 * (bf16, the paper's sketch storage; cfg.sketch_dtype): element (v, g) of
 * the paper's V x r sketch (the output of basis query g at value channel v)
 * sits at U[b][h][g/P][v][g%P], so each panel of the read is one contiguous,
 * coalesced run.  A bf16 sketch is rounded from fp32 to nearest, ties to
 * even.  Omega[H][K][r] and the coefficient map coef[H][r][K] (C, shared by
 * the batch) are fp32.
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

/* skssm_config.pivots of the state-dependent map with the exact state metric. */
enum { SKSSM_EXACT_MAP = -1 };

/* Shape of one linear-attention layer. */
typedef struct {
  int32_t kind;     /* skssm_kind                                           */
  int32_t batch;    /* B requests (B * H < 2^23: SKSSM_EUNSUPPORTED beyond)  */
  int32_t heads;    /* H heads                                              */
  int32_t dk;       /* K key channels  (Mamba-2 d_state N)                  */
  int32_t dv;       /* V value channels (Mamba-2 headdim P)                 */
  int32_t rank;     /* r sketch columns (the paper's G)                     */
  int32_t window;   /* W tokens per window = ring capacity                  */
  int32_t io_dtype; /* skssm_dtype of q, k, v and ring.k / ring.v           */
  int32_t sketch_dtype; /* skssm_dtype of U, ring.f and cmap (0 = fp32; BF16, the
                           paper's storage of the sketch, the coefficient map and
                           the projected erase vectors, halves their reads;
                           rounded to nearest even when stored)                 */
  int32_t pivots;   /* 0: the coefficient map is `coef` (offline, shared per head);
                       4: the state-dependent map (Sec. 4.1, eq. m-coeff) with the
                       P = 4 low-rank-plus-diagonal state metric (appendix on the
                       coefficient map, eq. pivot-metric), rebuilt from the state
                       by every sketchssm_update into `cmap` (rank 8..32);
                       SKSSM_EXACT_MAP (-1): the same map with the exact state
                       metric H (eq. pivot-ridge; Table 2's "Exact"), which for
                       an orthonormal Omega is (U^T U/mu + lambda I)^{-1} U^T S^T/mu
                       (rank 8 or 16)                                           */
  float ridge;      /* lambda > 0 of the state-dependent map (the paper uses 0.1) */
  const int32_t* head_rank; /* per-head rank table (host memory, read during the call),
                       or NULL: every head has rank `rank`.  With a table (the
                       allocation of Sec. 4.2 and the allocation appendix), entry h
                       is head h's rank G_h in 0..rank, and `rank` (8, 16 or 32) is
                       the storage width: U, omega, coef, f and cmap keep the layouts
                       of width `rank`, a head uses its first G_h columns (U panels
                       up to the next whole panel; the tail of a partly used panel
                       is written as zeros), and the unused panels, f entries and map
                       rows are neither read nor written.  G_h = 0 is a dense-fallback
                       head: it keeps the full state; sketchssm_decode reads its state
                       exactly (as sketchssm_full_read_baseline does, in the same
                       launch) and its flush writes no sketch.  heads <= 256;
                       omega's columns past G_h are ignored.
                       sketchssm_full_read_baseline reads every head exactly and
                       ignores the table (after validating it).                  */
} skssm_config;

/* Replay buffer ("ring"): W slots per (b, h) item.  Slot s holds the s-th
 * token of the current window (0-based).  Two layouts, by who writes:
 *   - raw inputs (k, v, beta, log_decay), written by the producer and only
 *     read here, are item-major, field[B][H][W][...]: the window of an item
 *     is one contiguous block, so a read fetches four consecutive slots per
 *     load instruction and the flush stages the window in one sweep;
 *   - derived fields (f, pi, tinv), written by each read for its own
 *     slot, are slot-major and head-major within a slot, field[W][H][B][...]:
 *     one step's writes for all items form one contiguous region, and the
 *     items one head's reads touch together (consecutive requests) are
 *     adjacent, so they cover whole cache lines.
 *
 * Raw update inputs of token s are written into slot s by the token's
 * producer (the layer's projections) before the call that consumes it;
 * appending to the buffer is therefore free.  Mamba-2 maps k = B_t,
 * v = x_t, beta = dt and log_decay = dt * A_h (Sec. 3.2, M_t = D_t); the
 * query C_t is passed to each call.
 *
 * Every read rebuilds the window-local cumulative log decays
 * g_s = sum_{j<=s} log alpha_j from log_decay (per channel for KDA), so every
 * decay ratio is exp(g_t - g_s) <= 1, never a division.  The library derives
 * and stores the remaining fields when a token is read for the first time
 * (the WY appendix), so later reads are parallel reductions over slots.
 * With the couplings of eq. wy, b_{s,j} = <exp(g_s - g_j) k_j, k_s> (j < s),
 * T = I + Diag(beta) B is unit lower triangular; the erase factors are
 * pi = T^{-1} (beta . e^g . k) and the pseudo-values that carry the erase
 * into the buffer output are u = T^{-1} (beta . v) (stacked over slots).
 *   tinv   row s of T^{-1}: entries j < s (the unit diagonal is implicit).
 *          Row s is -beta_s gamma^T with gamma = T^{-T} b_{s,.}, which the
 *          read of token s computes anyway;
 *   f      projected erase factors f_s = C pi_s in R^r (eq. wyread), read by
 *          sketchssm_decode;
 *   pi     erase factors pi_s in R^K (eq. wy), read by the exact baseline.
 * u is never stored: sum_s a_{t,s} u_s = sum_j alpha_j beta_j v_j with
 * alpha = T^{-T} a_{t,.}, one product with the stored rows per read; the
 * flush forms u itself.  Entries of tinv at or above the diagonal, and rows
 * of slots not yet read in this window, are never used (the ring needs no
 * clearing).
 * Unused fields may be NULL. */
typedef struct {
  const void* k;          /* [B][H][W][K] io_dtype raw keys (producer)              all kinds */
  const void* v;          /* [B][H][W][V] io_dtype raw values (producer)            all kinds */
  const float* beta;      /* [B][H][W] write gates (producer)                       all kinds */
  const float* log_decay; /* [B][H][W] (MAMBA2, GDN) or [B][H][W][K] (KDA), <= 0 (producer) */
  void* f;                /* [W][H][B][rank] projected erase factors, sketch_dtype   GDN, KDA (sketch read) */
  float* pi;              /* [W][H][B][K] erase factors                GDN, KDA (baseline)    */
  float* tinv;            /* [W][H][B][W]: slot s holds (T^{-1})_{s,j}, j < s      GDN, KDA  */
} skssm_ring;

/*
 * sketchssm_update -- flush step, initial sketch, or Standard step.
 * Algorithm 1 (flush) and Sec. 4.1: the single full-state read per window.
 *
 *   q != NULL: the token in ring slot n_buffered (0..W-1) completes the
 *     window; slots 0..n_buffered-1 hold its earlier tokens.  Reads S once,
 *     applies the n_buffered + 1 updates exactly (rank-(n_buffered+1) form of
 *     eq. update, on matrix cores), writes o = S_W^T q (if o != NULL),
 *     U = S_W^T Omega (if rank > 0) and S_W back in place.  The caller then
 *     starts the next window at slot 0; the ring needs no clearing.
 *     window = 1 with rank = 0 is the Standard recurrence (one read and one
 *     write of S per token); a single token at rank 0 runs as the rank-1
 *     recurrence on the vector units, the state streamed through registers.
 *   q == NULL: builds U = S^T Omega from S alone (the initial sketch after
 *     prefill, the initialisation step of Algorithm 1); n_buffered must be 0,
 *     S is not written and o is ignored.
 *
 * S      B*H*V*K fp32 in the tile-major layout, read and (q != NULL) written in place.
 * omega  [H][K][rank] fp32 (may be NULL when rank == 0).
 * ring   read-only here: k, v, beta, log_decay of slots 0..n_buffered;
 *        tinv (GDN, KDA) of slots 0..n_buffered-1.
 * q      [B][H][K] io_dtype, the current query.
 * U      [B][H][rank/P][V][P] output in cfg.sketch_dtype, panel layout (may be NULL when rank == 0).
 * cmap   cfg.pivots != 0: the state-dependent coefficient map C (rank x K per
 *        item, Sec. 4.1 eq. m-coeff with the ridge term of eq. pivot-ridge),
 *        built from S_W and its sketch and written in cfg.sketch_dtype as the
 *        dense matrix in 16-byte channel panels, [B][H][K/CP][rank][CP] with
 *        CP = 4 (fp32) or 8 (bf16) channels: element (j, k) of item i at
 *        i rank K + ((k / CP) rank + j) CP + k % CP.  Rows past a head's rank
 *        are not written.  Ignored (may be NULL) when pivots = 0.
 * o      [B][H][V] fp32 output or NULL.
 * rank may be 0 here (no sketch: the flush of the exact baseline).
 *
 * Occupancy: a flush with pivots = 0 (and the Mamba-2 single-token update)
 * launches with unused dynamic LDS so that at most three (two) of its
 * workgroups are resident per CU, which streams the in-place state faster
 * than more would; other kernels on the device are not affected, except that
 * a kernel running concurrently on the same CUs finds that LDS taken.
 */
int sketchssm_update(const skssm_config* cfg, float* S, const float* omega, const skssm_ring* ring,
                     int32_t n_buffered, const void* q, void* U, void* cmap, float* o, void* stream);

/*
 * sketchssm_decode -- non-flush step (Algorithm 1, t < W) for the token in
 * ring slot n_buffered (0..W-2), every head of the layer:
 *     o = U c_t + o_t^buffer,
 *     c_t = C (e^{g_t} . q_t) - sum_{s<=t} a_{t,s} f_s        (eq. app-projected-query)
 *     o_t^buffer = sum_{s<=t} a_{t,s} u_s,  a_{t,s} = <exp(g_t - g_s) k_s, q_t>
 * (for MAMBA2 f_s = 0 and u_s = beta_s v_s, so c_t = e^{g_t} C q_t).  The
 * state of a sketched head is never read.  U [B][H][rank/P][V][P]
 * (cfg.sketch_dtype) and the map C are read: coef [H][rank][K] fp32 (the
 * offline map of Sec. 4.1, Omega^T at E0 = I) or, with a state-dependent map,
 * the item's own cmap; for GDN/KDA the derived fields of slot n_buffered (f,
 * tinv) are written.
 * S (tile-major, fp32) is read only for the dense-fallback heads of a per-head
 * rank table (cfg.head_rank entries 0), whose output is the exact read of
 * sketchssm_full_read_baseline (their slot gets pi instead of f, so ring.pi
 * is then required); S may be NULL when no head is dense.
 * With cfg.pivots != 0 the map is the state-dependent one that the last
 * sketchssm_update wrote to cmap (the paper's 2 rank K bytes per item with bf16
 * storage); coef is then not read and may be NULL.  q [B][H][K] io_dtype;
 * o [B][H][V] fp32.  rank must be > 0, window >= 2.
 */
int sketchssm_decode(const skssm_config* cfg, const void* U, const float* coef, const void* cmap, const float* S,
                     const skssm_ring* ring, int32_t n_buffered, const void* q, float* o, void* stream);

/*
 * sketchssm_full_read_baseline -- exact non-flush step that reads all of S
 * (ReplaySSM-style; the reference the sketch read is measured against):
 *     o = S_0^T q~_t + o_t^buffer,  q~_t = e^{g_t} . q_t - sum_{s<=t} a_{t,s} pi_s
 * (eq. m-reads with the effective query of eq. app-effective-query-wy), for
 * the token in ring slot n_buffered (0..W-2).  For GDN/KDA the derived fields
 * of that slot (pi, tinv) are written.  S (tile-major) is only
 * read.  Flushes of this path use sketchssm_update with rank = 0.
 * cfg->rank is ignored.
 */
int sketchssm_full_read_baseline(const skssm_config* cfg, const float* S, const skssm_ring* ring,
                                 int32_t n_buffered, const void* q, float* o, void* stream);

/*
 * sketchssm_state_to_tiles / sketchssm_state_from_tiles -- convert states
 * between the row layout X[B][H][V][K] (X = S^T, K contiguous; how a caller
 * or a prefill usually holds them) and the tile-major layout every other
 * entry point reads and writes (see Layout).  Both arrays are B*H*V*K fp32
 * device memory owned by the caller, 16-byte aligned, and must not overlap
 * (SKSSM_EINVAL).  One kernel launch on `stream`; cfg->rank is ignored.
 */
int sketchssm_state_to_tiles(const skssm_config* cfg, const float* S_rows, float* S, void* stream);
int sketchssm_state_from_tiles(const skssm_config* cfg, const float* S, float* S_rows, void* stream);

/*
 * Buffer sizes -- the bytes of every caller-owned buffer of one layer with
 * configuration cfg, as the layouts above define them, so that a caller can
 * allocate without restating them (Algorithm 1's memory objects: the fp32
 * state, the sketch and coefficient map, and the replay buffer).
 *
 * baseline = 0: the layer of the sketch path (sketchssm_update /
 *   sketchssm_decode).  The derived ring fields are tinv and f for GDN/KDA,
 *   plus pi when the rank table has dense-fallback heads.
 * baseline = 1: the layer of the exact full-read path
 *   (sketchssm_full_read_baseline, with flushes by sketchssm_update at rank
 *   0): no sketch, map or f; pi and tinv for GDN/KDA.  cfg->rank and
 *   cfg->head_rank are ignored.
 * Fields the configuration does not use are 0.  A field's size depends only
 * on cfg, never on a pointer.  Returns SKSSM_OK, or a negative status for a
 * configuration the calls would reject (out may be partly written then).
 */
typedef struct {
  size_t S;         /* state, B*H*V*K fp32 (tile-major)                           */
  size_t U;         /* sketch, B*H*V*rank in sketch_dtype                          */
  size_t omega;     /* sketching matrix, H*K*rank fp32                             */
  size_t coef;      /* offline map, H*rank*K fp32 (pivots = 0)                     */
  size_t cmap;      /* state-dependent map, B*H*rank*K in sketch_dtype (pivots != 0) */
  size_t q;         /* one query, B*H*K io_dtype                                   */
  size_t o;         /* one output, B*H*V fp32                                      */
  size_t ring_k;    /* [B][H][W][K] io_dtype                                       */
  size_t ring_v;    /* [B][H][W][V] io_dtype                                       */
  size_t ring_beta; /* [B][H][W] fp32                                              */
  size_t ring_log_decay; /* [B][H][W] fp32, or [B][H][W][K] for KDA                */
  size_t ring_f;    /* [W][H][B][rank] sketch_dtype (GDN/KDA sketch path)         */
  size_t ring_pi;   /* [W][H][B][K] fp32 (GDN/KDA exact reads)                     */
  size_t ring_tinv; /* [W][H][B][W] fp32 (GDN/KDA)                                 */
} skssm_buffer_sizes;

int sketchssm_buffer_sizes(const skssm_config* cfg, int32_t baseline, skssm_buffer_sizes* out);

/* Total bytes of the replay buffer's fields (the ring_* sizes above), or 0
 * for a configuration the calls would reject. */
size_t sketchssm_ring_bytes(const skssm_config* cfg, int32_t baseline);

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

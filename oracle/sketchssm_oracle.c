/*
 * Plain CPU oracle for the SketchSSM decode path.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously-correct
 * reference that the GPU kernels are checked against.  Only the test suite,
 * the smoke check and the CPU-baseline leg of the benchmark may load it; the
 * product path never links, loads or calls it.  It shares no code, header,
 * table or helper with the HIP implementation.
 *
 * Everything is computed in fp64 from the plain definitions of the paper,
 * one independent (request, head) item at a time:
 *
 *   - Notation follows the paper (Sec. 3.2): the state S is K x V, the read
 *     is o = S^T q, the decay D_t is diagonal (scalar for Mamba-2 and GDN,
 *     per channel for KDA), the transition is M_t = D_t for Mamba-2 and
 *     M_t = (I - beta_t k_t k_t^T) D_t for GDN and KDA (eq. transition-update).
 *   - Storage orientation at this interface: states are passed as [V][K]
 *     (the transpose of the paper's K x V), sketches as [V][G].
 *   - No WY factorisation, no cumulative log-decays, no pseudo-values, no
 *     rank-W GEMM: effective queries are formed by applying M_s^T one token
 *     at a time, buffer outputs by applying M_j to each buffered key one token
 *     at a time (eq. m-reads), and flushes replay the buffered tokens one at a
 *     time through the update (eq. transition-update, Algorithm 1).
 *   - The only optional deviations from pure fp64 are `round_storage`, which
 *     rounds the full state, the sketch and the coefficient map to fp32 at
 *     the points where the method writes them back (the paper keeps the state
 *     in FP32 storage, Appendix "Detailed Evaluation Setup"), and
 *     `sketch_bf16`, which rounds to bf16 what the paper stores in BF16
 *     (Appendix "State Memory Traffic Reduction"): the sketch U, the
 *     state-dependent coefficient map C (the dense G x K matrix, rounded once
 *     when a flush writes it) and the projected erase factors f_s (rounded
 *     when slot s is first read; the current token's f_t is used as
 *     computed).  Arithmetic stays fp64.  The f_s only exist on the
 *     `paper_path` (the paper's coefficient-space forms), which bf16 storage
 *     therefore selects; without rounding it equals the direct form c = C q~
 *     (pinned).
 *
 * Pins (see tests/test_oracle_pins.py): brute-force closed forms of the
 * recurrence on tiny inputs, the delta-rule retrieval invariant, the
 * state/buffer decomposition (Sec. 3.2), r = K with Omega = I, W = 1,
 * projection behaviour of the sketch (Sec. 3.3), term isolation and
 * linearity.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_MAMBA2 = 0, ORC_GDN = 1, ORC_KDA = 2 };

typedef struct {
  int32_t kind;          /* ORC_MAMBA2 | ORC_GDN | ORC_KDA                  */
  int32_t n_items;       /* independent (request, head) items               */
  int32_t K, V;          /* key and value channels                          */
  int32_t G;             /* sketch rank (columns of Omega); 0 = no sketch   */
  int32_t W;             /* window: tokens applied per flush                */
  int32_t T;             /* decode steps                                    */
  int32_t round_storage; /* 1: state and sketch stored as fp32              */
  int32_t sketch_bf16;   /* 1: sketch, coefficient map and projected erase
                            factors stored as bf16 (the paper's storage;
                            implies paper_path)                              */
  int32_t pivots;        /* 0: the given map C; P > 0: the state-dependent
                            map with the P-pivot metric; -1: the state-
                            dependent map with the exact metric H            */
  float ridge;           /* lambda of the state-dependent map               */
  int32_t paper_path;    /* 1: coefficients through the projected erase
                            factors f_s (eq. wyread, app-projected-query);
                            0: c = C q~ from the effective query              */
} orc_cfg;

/* Per-item views of the per-step inputs.  Step inputs are laid out
 * [T][n_items][...]; log_decay is [T][n_items] (scalar decay) or
 * [T][n_items][K] (KDA). */
typedef struct {
  const orc_cfg* c;
  int item;
  const float *q, *k, *v, *beta, *log_decay;
} orc_tok;

static const float* tok_q(const orc_tok* t, int n) { return t->q + ((size_t)n * t->c->n_items + t->item) * t->c->K; }
static const float* tok_k(const orc_tok* t, int n) { return t->k + ((size_t)n * t->c->n_items + t->item) * t->c->K; }
static const float* tok_v(const orc_tok* t, int n) { return t->v + ((size_t)n * t->c->n_items + t->item) * t->c->V; }
static double tok_beta(const orc_tok* t, int n) { return (double)t->beta[(size_t)n * t->c->n_items + t->item]; }

/* Diagonal of D_n: alpha = exp(log decay), per channel. */
static double tok_decay(const orc_tok* t, int n, int kk)
{
  const orc_cfg* c = t->c;
  if (c->kind == ORC_KDA)
    return exp((double)t->log_decay[((size_t)n * c->n_items + t->item) * c->K + kk]);
  return exp((double)t->log_decay[(size_t)n * c->n_items + t->item]);
}

static int has_erase(const orc_cfg* c) { return c->kind == ORC_GDN || c->kind == ORC_KDA; }

/* y <- M_n y = (I - beta k k^T) D_n y   (GDN/KDA), or D_n y (Mamba-2). */
static void apply_M(const orc_tok* t, int n, double* y)
{
  const int K = t->c->K;
  for (int kk = 0; kk < K; ++kk) y[kk] *= tok_decay(t, n, kk);
  if (has_erase(t->c)) {
    const float* k = tok_k(t, n);
    double dot = 0.0;
    for (int kk = 0; kk < K; ++kk) dot += (double)k[kk] * y[kk];
    const double bd = tok_beta(t, n) * dot;
    for (int kk = 0; kk < K; ++kk) y[kk] -= bd * (double)k[kk];
  }
}

/* x <- M_n^T x = D_n (I - beta k k^T) x   (GDN/KDA), or D_n x (Mamba-2). */
static void apply_MT(const orc_tok* t, int n, double* x)
{
  const int K = t->c->K;
  if (has_erase(t->c)) {
    const float* k = tok_k(t, n);
    double dot = 0.0;
    for (int kk = 0; kk < K; ++kk) dot += (double)k[kk] * x[kk];
    const double bd = tok_beta(t, n) * dot;
    for (int kk = 0; kk < K; ++kk) x[kk] -= bd * (double)k[kk];
  }
  for (int kk = 0; kk < K; ++kk) x[kk] *= tok_decay(t, n, kk);
}

/* S <- M_n S + beta_n k_n v_n^T, S is K x V (paper orientation), S[kk*V+v].
 * The erase acts after the decay: (I - beta k k^T)(D_n S). */
static void update_state(const orc_tok* t, int n, double* S, double* tmpV)
{
  const int K = t->c->K, V = t->c->V;
  const float* k = tok_k(t, n);
  const float* v = tok_v(t, n);
  const double beta = tok_beta(t, n);
  for (int kk = 0; kk < K; ++kk) {
    const double d = tok_decay(t, n, kk);
    for (int j = 0; j < V; ++j) S[(size_t)kk * V + j] *= d;
  }
  if (has_erase(t->c)) {
    /* tmpV = k^T (D S) */
    for (int j = 0; j < V; ++j) tmpV[j] = 0.0;
    for (int kk = 0; kk < K; ++kk)
      for (int j = 0; j < V; ++j) tmpV[j] += (double)k[kk] * S[(size_t)kk * V + j];
    for (int kk = 0; kk < K; ++kk)
      for (int j = 0; j < V; ++j) S[(size_t)kk * V + j] -= beta * (double)k[kk] * tmpV[j];
  }
  for (int kk = 0; kk < K; ++kk)
    for (int j = 0; j < V; ++j) S[(size_t)kk * V + j] += beta * (double)k[kk] * (double)v[j];
}

/* out = S^T x  (V entries). */
static void read_state(int K, int V, const double* S, const double* x, double* out)
{
  for (int j = 0; j < V; ++j) out[j] = 0.0;
  for (int kk = 0; kk < K; ++kk)
    for (int j = 0; j < V; ++j) out[j] += S[(size_t)kk * V + j] * x[kk];
}

static void round_f32(double* a, size_t n)
{
  for (size_t i = 0; i < n; ++i) a[i] = (double)(float)a[i];
}

/* The paper stores the sketch in BF16 (8-bit significand): round the value
 * to fp32 and then to bf16, to nearest with ties to even. */
static double bf16_rne(double x)
{
  float f = (float)x;
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  if ((u & 0x7f800000u) != 0x7f800000u) { /* finite: add half an ulp of bf16, ties to even */
    u += 0x7fffu + ((u >> 16) & 1u);
    u &= 0xffff0000u;
  }
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

static void store_sketch(const orc_cfg* c, double* U, size_t n)
{
  if (c->sketch_bf16) {
    for (size_t i = 0; i < n; ++i) U[i] = bf16_rne(U[i]);
  } else if (c->round_storage) {
    round_f32(U, n);
  }
}

/* The state-dependent map C (G x K) as a flush stores it: like the sketch. */
static void store_map(const orc_cfg* c, double* Cm, size_t n)
{
  store_sketch(c, Cm, n);
}

/* U = S^T Omega  (V x G), Omega is this head's K x G block. */
static void make_sketch(int K, int V, int G, const double* S, const float* omega, double* U)
{
  for (int j = 0; j < V; ++j)
    for (int g = 0; g < G; ++g) {
      double acc = 0.0;
      for (int kk = 0; kk < K; ++kk) acc += S[(size_t)kk * V + j] * (double)omega[(size_t)kk * G + g];
      U[(size_t)j * G + g] = acc;
    }
}

/* ------------------------------------------------------------------------ */
/* State-dependent coefficient map (Sec. 4.1, eq. m-coeff, solved with the   */
/* ridge term of the appendix "Low-Rank-Plus-Diagonal Approximation for the  */
/* Coefficient Map", eq. pivot-ridge), in the paper's basis-aligned          */
/* coordinates and order of steps:                                           */
/*   R       orthogonal K x K whose first G rows are Omega^T (Omega completed  */
/*           by Gram-Schmidt over the unit vectors), J = first G coordinates */
/*   S'      = R S,  mu = |S'|_F^2 / K (1 for a zero state),  H = S' S'^T/mu */
/* exact metric (pivots < 0): Hm = H, the dense state metric;                */
/* P pivots (eq. pivot-metric):                                              */
/*   Q       orthonormal basis of the first p = min(G, P) columns of U       */
/*           (Gram-Schmidt; a column dependent on the earlier ones is dropped)*/
/*   L       = S' Q / sqrt(mu),  d_i = max(H_ii - |L_i|^2, 0)                */
/*   Hm      = Hhat = L L^T + Diag(d)                                        */
/* then c = (J^T Hm J + lambda I)^{-1} J^T Hm x,  x = R q~, so c = Cm q~ with */
/* Cm = (J^T Hm J + lambda I)^{-1} J^T Hm R (G x K), solved directly by      */
/* Gaussian elimination with partial pivoting.                               */
/* ------------------------------------------------------------------------ */
typedef struct {
  double *R, *Sp, *H, *Q, *L, *d, *Hh, *A, *B;
} orc_cmap_work;

static int cmap_work_alloc(orc_cmap_work* w, int K, int V, int G)
{
  w->R = (double*)malloc(sizeof(double) * (size_t)K * K);
  w->Sp = (double*)malloc(sizeof(double) * (size_t)K * V);
  w->H = (double*)malloc(sizeof(double) * (size_t)K * K);
  w->Q = (double*)malloc(sizeof(double) * (size_t)V * (G > 0 ? G : 1));
  w->L = (double*)malloc(sizeof(double) * (size_t)K * (G > 0 ? G : 1));
  w->d = (double*)malloc(sizeof(double) * (size_t)K);
  w->Hh = (double*)malloc(sizeof(double) * (size_t)K * K);
  w->A = (double*)malloc(sizeof(double) * (size_t)G * G + 1);
  w->B = (double*)malloc(sizeof(double) * (size_t)G * K + 1);
  return w->R && w->Sp && w->H && w->Q && w->L && w->d && w->Hh && w->A && w->B;
}

static void cmap_work_free(orc_cmap_work* w)
{
  free(w->R); free(w->Sp); free(w->H); free(w->Q); free(w->L); free(w->d); free(w->Hh); free(w->A); free(w->B);
}

/* Orthonormalise column vector x (length n, stride 1) against the m rows
 * basis[0..m-1] (each length n); returns 1 and normalises x when it has a
 * part outside their span, 0 when it is dependent on them. */
static int gram_schmidt(double* x, const double* basis, int m, int n, double scale)
{
  for (int pass = 0; pass < 2; ++pass) /* twice, for a clean orthogonalisation */
    for (int r = 0; r < m; ++r) {
      double dot = 0.0;
      for (int i = 0; i < n; ++i) dot += basis[(size_t)r * n + i] * x[i];
      for (int i = 0; i < n; ++i) x[i] -= dot * basis[(size_t)r * n + i];
    }
  double nrm = 0.0;
  for (int i = 0; i < n; ++i) nrm += x[i] * x[i];
  nrm = sqrt(nrm);
  if (!(nrm > 1e-12 * scale)) return 0;
  for (int i = 0; i < n; ++i) x[i] /= nrm;
  return 1;
}

static void coef_map(const orc_cfg* c, int K, int V, int G, const double* S, const float* Om, const double* U,
                     double* Cm, orc_cmap_work* w)
{
  const int P = c->pivots, p = G < P ? G : P;
  const double lambda = (double)c->ridge;
  /* R: rows 0..G-1 = the columns of Omega, then unit vectors outside their span */
  int m = 0;
  double x[1024];
  for (int g = 0; g < G; ++g) {
    for (int kk = 0; kk < K; ++kk) x[kk] = (double)Om[(size_t)kk * G + g];
    if (gram_schmidt(x, w->R, m, K, 1.0)) memcpy(w->R + (size_t)m++ * K, x, sizeof(double) * K);
  }
  for (int e = 0; e < K && m < K; ++e) {
    for (int kk = 0; kk < K; ++kk) x[kk] = (kk == e) ? 1.0 : 0.0;
    if (gram_schmidt(x, w->R, m, K, 1.0)) memcpy(w->R + (size_t)m++ * K, x, sizeof(double) * K);
  }
  /* S' = R S, mu, H */
  double fro = 0.0;
  for (int i = 0; i < K; ++i)
    for (int j = 0; j < V; ++j) {
      double acc = 0.0;
      for (int kk = 0; kk < K; ++kk) acc += w->R[(size_t)i * K + kk] * S[(size_t)kk * V + j];
      w->Sp[(size_t)i * V + j] = acc;
      fro += acc * acc;
    }
  const double mu = fro > 0.0 ? fro / K : 1.0;
  for (int i = 0; i < K; ++i)
    for (int i2 = 0; i2 < K; ++i2) {
      double acc = 0.0;
      for (int j = 0; j < V; ++j) acc += w->Sp[(size_t)i * V + j] * w->Sp[(size_t)i2 * V + j];
      w->H[(size_t)i * K + i2] = acc / mu;
    }
  const double* Hm = w->H; /* the exact metric (pivots < 0) */
  if (P > 0) {
    /* Q: the first p columns of U, orthonormalised (stored as rows of length V) */
    int pq = 0;
    for (int a = 0; a < p; ++a) {
      double nrm = 0.0;
      for (int j = 0; j < V; ++j) {
        x[j] = U[(size_t)j * G + a];
        nrm += x[j] * x[j];
      }
      if (nrm > 0.0 && gram_schmidt(x, w->Q, pq, V, sqrt(nrm))) memcpy(w->Q + (size_t)pq++ * V, x, sizeof(double) * V);
    }
    /* L = S' Q / sqrt(mu) (K x pq), d, Hhat */
    const double rs = 1.0 / sqrt(mu);
    for (int i = 0; i < K; ++i)
      for (int a = 0; a < pq; ++a) {
        double acc = 0.0;
        for (int j = 0; j < V; ++j) acc += w->Sp[(size_t)i * V + j] * w->Q[(size_t)a * V + j];
        w->L[(size_t)i * pq + a] = acc * rs;
      }
    for (int i = 0; i < K; ++i) {
      double l2 = 0.0;
      for (int a = 0; a < pq; ++a) l2 += w->L[(size_t)i * pq + a] * w->L[(size_t)i * pq + a];
      const double r = w->H[(size_t)i * K + i] - l2;
      w->d[i] = r > 0.0 ? r : 0.0;
    }
    for (int i = 0; i < K; ++i)
      for (int i2 = 0; i2 < K; ++i2) {
        double acc = (i == i2) ? w->d[i] : 0.0;
        for (int a = 0; a < pq; ++a) acc += w->L[(size_t)i * pq + a] * w->L[(size_t)i2 * pq + a];
        w->Hh[(size_t)i * K + i2] = acc;
      }
    Hm = w->Hh;
  }
  /* A = J^T Hm J + lambda I (G x G);  B = J^T Hm R (G x K) */
  for (int g = 0; g < G; ++g) {
    for (int g2 = 0; g2 < G; ++g2) w->A[(size_t)g * G + g2] = Hm[(size_t)g * K + g2] + (g == g2 ? lambda : 0.0);
    for (int kk = 0; kk < K; ++kk) {
      double acc = 0.0;
      for (int i = 0; i < K; ++i) acc += Hm[(size_t)g * K + i] * w->R[(size_t)i * K + kk];
      w->B[(size_t)g * K + kk] = acc;
    }
  }
  /* Cm = A^{-1} B: Gaussian elimination with partial pivoting on [A | B] */
  for (int col = 0; col < G; ++col) {
    int piv = col;
    for (int r = col + 1; r < G; ++r)
      if (fabs(w->A[(size_t)r * G + col]) > fabs(w->A[(size_t)piv * G + col])) piv = r;
    if (piv != col) {
      for (int j = 0; j < G; ++j) {
        const double t = w->A[(size_t)col * G + j];
        w->A[(size_t)col * G + j] = w->A[(size_t)piv * G + j];
        w->A[(size_t)piv * G + j] = t;
      }
      for (int j = 0; j < K; ++j) {
        const double t = w->B[(size_t)col * K + j];
        w->B[(size_t)col * K + j] = w->B[(size_t)piv * K + j];
        w->B[(size_t)piv * K + j] = t;
      }
    }
    const double inv = 1.0 / w->A[(size_t)col * G + col];
    for (int r = 0; r < G; ++r) {
      if (r == col) continue;
      const double f = w->A[(size_t)r * G + col] * inv;
      if (f == 0.0) continue;
      for (int j = col; j < G; ++j) w->A[(size_t)r * G + j] -= f * w->A[(size_t)col * G + j];
      for (int j = 0; j < K; ++j) w->B[(size_t)r * K + j] -= f * w->B[(size_t)col * K + j];
    }
  }
  for (int g = 0; g < G; ++g) {
    const double inv = 1.0 / w->A[(size_t)g * G + g];
    for (int kk = 0; kk < K; ++kk) Cm[(size_t)g * K + kk] = w->B[(size_t)g * K + kk] * inv;
  }
}

static void load_state(int K, int V, const float* S_vk, double* S)
{
  for (int j = 0; j < V; ++j)
    for (int kk = 0; kk < K; ++kk) S[(size_t)kk * V + j] = (double)S_vk[(size_t)j * K + kk];
}

static void store_state(int K, int V, const double* S, double* S_vk)
{
  for (int j = 0; j < V; ++j)
    for (int kk = 0; kk < K; ++kk) S_vk[(size_t)j * K + kk] = S[(size_t)kk * V + j];
}

/* ------------------------------------------------------------------------ */
/* O1: the plain recurrence, one token at a time (eq. transition-update and  */
/* m-reads, first forms).  o_exact[n] = S_n^T q_n, S_final = S_T.            */
/* ------------------------------------------------------------------------ */
int orc_recurrence(const orc_cfg* c, const float* S_init, const float* q, const float* k, const float* v,
                   const float* beta, const float* log_decay, double* o_exact, double* S_final)
{
  if (!c || c->K <= 0 || c->V <= 0 || c->n_items <= 0 || c->T < 0) return -1;
  if (c->K > 1024 || c->V > 1024) return -1;
  const int K = c->K, V = c->V, NI = c->n_items;
  int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int i = 0; i < NI; ++i) {
    double* S = (double*)malloc(sizeof(double) * (size_t)K * V);
    double* tmp = (double*)malloc(sizeof(double) * (size_t)(K + V));
    if (!S || !tmp) {
      err = -2;
      free(S);
      free(tmp);
      continue;
    }
    orc_tok t = {c, i, q, k, v, beta, log_decay};
    load_state(K, V, S_init + (size_t)i * V * K, S);
    for (int n = 0; n < c->T; ++n) {
      update_state(&t, n, S, tmp);
      double xq[1024];
      const float* qn = tok_q(&t, n);
      for (int kk = 0; kk < K; ++kk) xq[kk] = (double)qn[kk];
      if (o_exact) read_state(K, V, S, xq, o_exact + ((size_t)n * NI + i) * V);
    }
    if (S_final) store_state(K, V, S, S_final + (size_t)i * V * K);
    free(S);
    free(tmp);
  }
  return err;
}

/* ------------------------------------------------------------------------ */
/* O2: SketchSSM inference (Algorithm 1) for every item.                    */
/*                                                                          */
/* Window-local time t = 1..W.  At a non-flush step (t < W):                 */
/*   q~_t   = M_1^T ... M_t^T q_t                 (effective query)          */
/*   c_t    = C q~_t                              (coefficient vector)       */
/*   o^state_hat = U c_t,   o^state = S0^T q~_t   (sketch and exact reads)   */
/*   o^buf  = sum_{s<=t} beta_s <M_{s+1:t} k_s, q_t> v_s                     */
/*   o_t    = o^state_hat + o^buf                                            */
/* At the flush (t = W): replay the W buffered tokens into S0 one at a time, */
/* o_t = S0^T q_t exactly, U = S0^T Omega, clear the buffer.                 */
/*                                                                          */
/* Per-item head index: heads[i] selects Omega [H][K][G] and C [H][G][K].    */
/* Outputs (any may be NULL):                                                */
/*   o            [T][n][V]  the method's output                             */
/*   o_state_hat  [T][n][V]  U c_t at non-flush steps, S0^T q at flushes     */
/*   o_state      [T][n][V]  S0^T q~_t at non-flush steps, S0^T q at flushes */
/*   o_buf        [T][n][V]  buffer term (0 at flushes)                      */
/*   S_final      [n][V][K]  the full state after the last flush             */
/*   U_final      [n][V][G]  the sketch after the last flush                 */
/*   coef_final   [n][G][K]  the coefficient map in use after the last flush */
/* With c->pivots != 0 the map is state-dependent: built from the state and  */
/* its (unrounded) sketch at the start and at every flush (coef_map above)   */
/* and stored (store_map: rounded like the sketch); otherwise it is the      */
/* given C of the item's head.                                               */
/* The exact windowed output (what a full-state read would give) is         */
/* o_state + o_buf at every step.                                           */
/* ------------------------------------------------------------------------ */
int orc_sketchssm(const orc_cfg* c, const int32_t* heads, const float* omega, const float* coef,
                  const float* S_init, const float* q, const float* k, const float* v, const float* beta,
                  const float* log_decay, double* o, double* o_state_hat, double* o_state, double* o_buf,
                  double* S_final, double* U_final, double* coef_final)
{
  if (!c || c->K <= 0 || c->V <= 0 || c->n_items <= 0 || c->T < 0 || c->W < 1 || c->G < 0) return -1;
  if (c->K > 1024 || c->V > 1024 || c->G > 1024 || c->pivots < -1 || c->pivots > 4) return -1;
  const int K = c->K, V = c->V, G = c->G, NI = c->n_items, W = c->W;
  const int fpath = (c->paper_path || c->sketch_bf16) && has_erase(c) && G > 0;
  if (fpath && W > 64) return -1;
  int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int i = 0; i < NI; ++i) {
    const int h = heads ? heads[i] : 0;
    const float* Om = omega ? omega + (size_t)h * K * G : NULL;
    const float* Cm = coef ? coef + (size_t)h * G * K : NULL;
    double* S0 = (double*)malloc(sizeof(double) * (size_t)K * V);
    double* U = (double*)malloc(sizeof(double) * ((size_t)V * (G > 0 ? G : 1)));
    const int statedep = c->pivots != 0 && G > 0;
    double* Cmi = statedep ? (double*)malloc(sizeof(double) * (size_t)G * K) : NULL;
    orc_cmap_work cw = {0};
    if (statedep && (!Cmi || !cmap_work_alloc(&cw, K, V, G))) {
#pragma omp atomic write
      err = -2;
    }
    double* tmp = (double*)malloc(sizeof(double) * (size_t)(K + V));
    int* buf = (int*)malloc(sizeof(int) * (size_t)W);
    double* fhat = (double*)malloc(sizeof(double) * (size_t)W * (G > 0 ? G : 1)); /* stored f_s of the window */
    if (!S0 || !U || !tmp || !buf || !fhat) {
      err = -2;
      free(S0); free(U); free(tmp); free(buf); free(fhat);
      continue;
    }
    orc_tok t = {c, i, q, k, v, beta, log_decay};
    load_state(K, V, S_init + (size_t)i * V * K, S0);
    /* Initialise the sketch from the prefill state (Algorithm 1). */
    if (G > 0) {
      make_sketch(K, V, G, S0, Om, U);
      if (statedep && Cmi && cw.R) {
        coef_map(c, K, V, G, S0, Om, U, Cmi, &cw);
        store_map(c, Cmi, (size_t)G * K);
      }
      store_sketch(c, U, (size_t)V * G);
    }
    int len = 0; /* tokens in the buffer B */
    double x[1024], y[1024], cvec[1024], ohat[1024], ostate[1024], obuf[1024];
    for (int n = 0; n < c->T; ++n) {
      buf[len++] = n; /* append the current update inputs to B */
      const size_t oi = ((size_t)n * NI + i) * V;
      const float* qn = tok_q(&t, n);
      if (len < W) {
        /* effective query q~ = M_1^T (M_2^T ( ... M_t^T q)) */
        for (int kk = 0; kk < K; ++kk) x[kk] = (double)qn[kk];
        for (int s = len - 1; s >= 0; --s) apply_MT(&t, buf[s], x);
        /* exact state read and sketch read */
        read_state(K, V, S0, x, ostate);
        for (int j = 0; j < V; ++j) ohat[j] = 0.0;
        if (fpath) {
          /* coefficient space (eq. app-projected-query, with f_s from eq. wyread):
           *   f_t = beta_t (C (d_[t] . k_t) - sum_{j<t} f_j <l_j(t), k_t>)
           *   c_t = C (d_[t] . q_t) - sum_{s<t} f_s <l_s(t), q_t> - f_t <k_t, q_t>
           * with l_j(t) = D_t ... D_{j+1} k_j and d_[t] the decay product of the
           * window so far; each f_s is stored (bf16 with the paper's storage)
           * when formed, and later steps use the stored value */
          const int cur = len - 1, tn = buf[cur];
          const float* kt = tok_k(&t, tn);
          double dq[1024], dk[1024], aq[64], ak[64];
          for (int kk = 0; kk < K; ++kk) {
            dq[kk] = (double)qn[kk];
            dk[kk] = (double)kt[kk];
          }
          for (int s = 0; s < len; ++s)
            for (int kk = 0; kk < K; ++kk) {
              const double dd = tok_decay(&t, buf[s], kk);
              dq[kk] *= dd;
              dk[kk] *= dd;
            }
          for (int j = 0; j < cur; ++j) {
            const float* kj = tok_k(&t, buf[j]);
            for (int kk = 0; kk < K; ++kk) y[kk] = (double)kj[kk];
            for (int r = j + 1; r <= cur; ++r)
              for (int kk = 0; kk < K; ++kk) y[kk] *= tok_decay(&t, buf[r], kk);
            double sq = 0.0, sk = 0.0;
            for (int kk = 0; kk < K; ++kk) {
              sq += y[kk] * (double)qn[kk];
              sk += y[kk] * (double)kt[kk];
            }
            aq[j] = sq;
            ak[j] = sk;
          }
          double akq = 0.0;
          for (int kk = 0; kk < K; ++kk) akq += (double)kt[kk] * (double)qn[kk];
          const double bt = tok_beta(&t, tn);
          for (int g = 0; g < G; ++g) {
            double cq = 0.0, ck = 0.0;
            for (int kk = 0; kk < K; ++kk) {
              const double cg = Cmi ? Cmi[(size_t)g * K + kk] : (double)Cm[(size_t)g * K + kk];
              cq += cg * dq[kk];
              ck += cg * dk[kk];
            }
            for (int j = 0; j < cur; ++j) {
              ck -= fhat[(size_t)j * G + g] * ak[j];
              cq -= fhat[(size_t)j * G + g] * aq[j];
            }
            const double ft = bt * ck;
            cvec[g] = cq - ft * akq;
            fhat[(size_t)cur * G + g] = c->sketch_bf16 ? bf16_rne(ft) : ft;
          }
        } else if (G > 0) {
          for (int g = 0; g < G; ++g) {
            double acc = 0.0;
            for (int kk = 0; kk < K; ++kk)
              acc += (Cmi ? Cmi[(size_t)g * K + kk] : (double)Cm[(size_t)g * K + kk]) * x[kk];
            cvec[g] = acc;
          }
        }
        if (G > 0) {
          for (int j = 0; j < V; ++j) {
            double acc = 0.0;
            for (int g = 0; g < G; ++g) acc += U[(size_t)j * G + g] * cvec[g];
            ohat[j] = acc;
          }
        }
        /* buffer output: sum_s beta_s <M_{s+1:t} k_s, q_t> v_s */
        for (int j = 0; j < V; ++j) obuf[j] = 0.0;
        for (int s = 0; s < len; ++s) {
          const float* ks = tok_k(&t, buf[s]);
          for (int kk = 0; kk < K; ++kk) y[kk] = (double)ks[kk];
          for (int r = s + 1; r < len; ++r) apply_M(&t, buf[r], y);
          double a = 0.0;
          for (int kk = 0; kk < K; ++kk) a += y[kk] * (double)qn[kk];
          const double w = tok_beta(&t, buf[s]) * a;
          const float* vs = tok_v(&t, buf[s]);
          for (int j = 0; j < V; ++j) obuf[j] += w * (double)vs[j];
        }
        for (int j = 0; j < V; ++j) {
          if (o) o[oi + j] = ohat[j] + obuf[j];
          if (o_state_hat) o_state_hat[oi + j] = ohat[j];
          if (o_state) o_state[oi + j] = ostate[j];
          if (o_buf) o_buf[oi + j] = obuf[j];
        }
      } else {
        /* flush: apply every buffered update exactly, in order */
        for (int s = 0; s < len; ++s) update_state(&t, buf[s], S0, tmp);
        if (c->round_storage) round_f32(S0, (size_t)K * V);
        for (int kk = 0; kk < K; ++kk) x[kk] = (double)qn[kk];
        read_state(K, V, S0, x, ostate);
        if (G > 0) {
          make_sketch(K, V, G, S0, Om, U);
          if (statedep && Cmi && cw.R) {
            coef_map(c, K, V, G, S0, Om, U, Cmi, &cw);
            store_map(c, Cmi, (size_t)G * K);
          }
          store_sketch(c, U, (size_t)V * G);
        }
        for (int j = 0; j < V; ++j) {
          if (o) o[oi + j] = ostate[j];
          if (o_state_hat) o_state_hat[oi + j] = ostate[j];
          if (o_state) o_state[oi + j] = ostate[j];
          if (o_buf) o_buf[oi + j] = 0.0;
        }
        len = 0; /* clear B */
      }
    }
    if (S_final) store_state(K, V, S0, S_final + (size_t)i * V * K);
    if (U_final && G > 0) memcpy(U_final + (size_t)i * V * G, U, sizeof(double) * (size_t)V * G);
    if (coef_final && G > 0) {
      for (size_t e = 0; e < (size_t)G * K; ++e)
        coef_final[(size_t)i * G * K + e] = Cmi ? Cmi[e] : (double)Cm[e];
    }
    if (statedep) cmap_work_free(&cw);
    free(Cmi);
    free(S0); free(U); free(tmp); free(buf); free(fhat);
  }
  return err;
}

int orc_max_threads(void)
{
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void orc_set_threads(int n)
{
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

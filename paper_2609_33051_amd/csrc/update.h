// Flush step of SketchSSM (Algorithm 1, t = W; Sec. 4.1, per-window sketch)
// and the initial sketch: one read and one write of the full state.
//
// With the window's tokens in ring slots 0..n (slot n: the current token),
// cumulative log decays g_s and c_s = exp(g_n - g_s):
//   L[s]   = exp(g_n - g_s) . k_s                  (left factors l_s(W), Appendix C.1)
//   pi_s   = beta_s (e^{g_s} . k_s - sum_{j<s} b_{s,j} pi_j)           (eq. wy)
//          = sum_{j<=s} (T^{-1})_{s,j} beta_j e^{g_j} . k_j,  T = I + Diag(beta) B
//            (rows s < n of T^{-1} come from the ring; row n's couplings
//            b_{n,j} are formed here)
//   w_s    = u_s - X_0 pi_s                         (true write vectors; Mamba-2: beta_s v_s)
//   X_W    = X_0 Diag(e^{g_n}) + sum_s w_s L[s]^T   (eq. update in rank-(n+1) form)
//   o_W    = X_W q_W,   U = X_W Omega
// where X = S^T is the stored [V][K] state.  For a scalar decay c_s is one
// number per slot and moves to the value side (w_s L[s]^T = (c_s w_s) k_s^T),
// so the raw keys are the matrix-core operand.  The two contractions over the
// state (X_0 Pi^T, K-deep; the rank-(n+1) update, slot-deep) and the sketch
// projection X_W Omega run on fp32 matrix cores (v_mfma_f32_16x16x4f32).
//
// Mapping: one workgroup (4 waves) per (request, head) item.  The window's
// slots are staged into LDS with wide loads (row layout: four slots per load
// instruction, wave w taking slot groups w, w + 4, ...).  Each wave owns
// 16-column value tiles of X^T (K rows x 16 values), held in MFMA
// accumulator layout: lane l holds X[v0 + l%16][16 kt + 4 (l/16) + i],
// i = 0..3.  The state is stored in exactly this order (tile-major: tile
// (v0/16, kt) is 1 KB contiguous with lane l's four values at 4 l), so each
// load and store instruction moves 1 KB contiguous; both are non-temporal,
// as the state is touched once per flush.  Because the
// contraction index of the K-deep products may be visited in any order, the
// same registers serve as the B operand of X_0 Pi^T and X_W Omega (step i of
// k-tile kt contracts over k = 16 kt + 4 g + i for lane group g) and as the
// accumulator of the rank update, so the state never leaves registers
// between its load and its store.
#pragma once

#include "args.h"
#include "device.h"

namespace skssm {

__device__ __forceinline__ floatx4 mfma4(float a, float b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

template <typename IO> __device__ __forceinline__ float load1(const IO* p);
template <> __device__ __forceinline__ float load1<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float load1<bf16_t>(const bf16_t* p) { return bf16_lo((uint32_t)*p); }

// The state-dependent coefficient map (Sec. 4.1, eq. m-coeff with the ridge
// term and the low-rank-plus-diagonal metric of the appendix on the P = 4
// pivot approximation), from the partial sums the tiles left behind:
//   mu   = |S|_F^2 / K (1 for a zero state)
//   U_p  = the first P sketch columns,  U_p^T U_p = R^T R (Cholesky; a column
//          dependent on the earlier ones is dropped: its row of R^{-1} is 0)
//   L_G  = U^T U_p R^{-1} / sqrt(mu)             (G x P; Q = U_p R^{-1})
//   M    = R^{-T} U_p^T S^T / sqrt(mu)           (P x K, i.e. Q^T S^T / sqrt(mu))
//   d    = max(diag(U^T U) / mu - |L_G rows|^2, 0),  D = d + lambda
//   T    = I + L_G^T D^{-1} L_G                  (Woodbury: only T is inverted)
//   F1   = D^{-1} L_G T^{-1}  (= A^{-1} L_G),  F2 = A^{-1} Diag(d),
//   A^{-1} = D^{-1} - D^{-1} L_G T^{-1} L_G^T D^{-1}
// so the map is C = F1 M + F2 Omega^T (G x K).  With w = d / (d + lambda),
// F2 = Diag(w) - F1 L_G^T Diag(w), hence
//   C = F1 M' + Diag(w) Omega^T,   M' = M - L_G^T Diag(w) Omega^T   (P x K):
// thread k forms column k of M' beside that of M, and the flush forms
// C^T = M'^T F1^T on the matrix cores (one 16x16x4 step per block) plus
// w_j Omega[k][j] per element, then stores the dense map per item in the
// sketch's dtype (bf16 with the paper's storage, rounded to nearest even) in
// 16-byte channel panels cmap[B][H][K/CPW][G][CPW].  Rows past the head's
// rank are not stored.  Every thread of the workgroup calls this.
template <int K, int R, int P, int MT, int RT, int LSZ, int USZ, int OPJ, typename SK>
__device__ __forceinline__ void coef_map_tail(const UpdateArgs& a, size_t item, int wave, int lane, int tid, int rh,
                                              const floatx4 (&nacc)[MT], const floatx4 (&gram)[RT],
                                              const float (&dsq)[RT], float msq,
                                              float* Ls, float* Us, float* cmS, const float* OmL, float* Fext) {
  static_assert(LSZ >= 4 * K * P && USZ >= 4 * R * 5, "staging buffers too small for the map's partial sums");
  static_assert(MT % 4 == 0, "the four waves split the k tiles evenly");
  constexpr int FBP = P + 1;                           // row pitch of F1 (odd: lanes of a read spread over banks)
  constexpr bool FB_ALIAS = LSZ >= P * K + 16 * RT * FBP;
  const int lr = lane & 15, lg = lane >> 4;
  // the squared sketch columns summed over the four lane rows (the Gram
  // products already summed over this wave's values)
  float dq[RT];
#pragma unroll
  for (int jt = 0; jt < RT; ++jt) dq[jt] = cross_row_sum(dsq[jt]);
  msq = wave_sum(msq);
  lds_barrier();  // every wave is done with the window staging (Ls, Us), reused below
  float* cmN = Ls;  // [wave][K][P]
  float* cmG = Us;  // [wave][R][5]
  if (lg == 0) {
#pragma unroll
    for (int kt = 0; kt < MT; ++kt)
      *reinterpret_cast<float4*>(&cmN[(wave * K + 16 * kt + lr) * P]) = make_float4(nacc[kt][0], nacc[kt][1], nacc[kt][2], nacc[kt][3]);
  }
  // row j of cmG: U_j . U_a for the pivots a < P, then |U_j|^2
#pragma unroll
  for (int jt = 0; jt < RT; ++jt) {
    if (lr < P) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = 16 * jt + 4 * lg + i;
        if (j < R) cmG[(wave * R + j) * 5 + lr] = gram[jt][i];
      }
    }
    if (lg == 0 && 16 * jt + lr < R) cmG[(wave * R + 16 * jt + lr) * 5 + 4] = dq[jt];
  }
  if (lane == 0) cmS[wave] = msq;
  lds_barrier();

  float F1[P] = {};  // wave 0, lane g < R: row g of F1
  if (wave == 0) {
    const float fro = cmS[0] + cmS[1] + cmS[2] + cmS[3];
    const float mu = fro > 0.f ? fro / K : 1.f;
    // the algebra is one serial chain on one wave while the other waves wait:
    // hardware reciprocal, square root and reciprocal square root (1 ulp) keep it short
    const float rs = __builtin_amdgcn_rsqf(mu);
    // pivot Gram, Cholesky with dropping, R^{-1} (all lanes, uniform)
    float Gp[P][P], Rm[P][P], Ri[P][P];
#pragma unroll
    for (int x = 0; x < P; ++x)
#pragma unroll
      for (int y = 0; y < P; ++y) {
        Gp[x][y] = cmG[(0 * R + x) * 5 + y] + cmG[(1 * R + x) * 5 + y] + cmG[(2 * R + x) * 5 + y] + cmG[(3 * R + x) * 5 + y];
        Rm[x][y] = 0.f;
        Ri[x][y] = 0.f;
      }
#pragma unroll
    for (int x = 0; x < P; ++x) {
      float sd = Gp[x][x];
#pragma unroll
      for (int b = 0; b < x; ++b) sd -= Rm[b][x] * Rm[b][x];
      if (Gp[x][x] > 0.f && sd > 1e-6f * Gp[x][x]) {
        const float rxx = __builtin_amdgcn_sqrtf(sd), irx = __builtin_amdgcn_rcpf(rxx);
        Rm[x][x] = rxx;
#pragma unroll
        for (int y = x + 1; y < P; ++y) {
          float e = Gp[x][y];
#pragma unroll
          for (int b = 0; b < x; ++b) e -= Rm[b][x] * Rm[b][y];
          Rm[x][y] = e * irx;
        }
      }
    }
#pragma unroll
    for (int x = 0; x < P; ++x)
      if (Rm[x][x] > 0.f) Ri[x][x] = __builtin_amdgcn_rcpf(Rm[x][x]);
#pragma unroll
    for (int x = 0; x < P; ++x) {
#pragma unroll
      for (int y = x + 1; y < P; ++y) {
        if (Rm[y][y] > 0.f) {
          float e = 0.f;
#pragma unroll
          for (int b = x; b < y; ++b) e += Ri[x][b] * Rm[b][y];
          Ri[x][y] = -e * Ri[y][y];
        }
      }
    }
    // lane g < R: row g of L_G, d, D^{-1}
    const int g = lane;
    float LG[P] = {}, dg = 0.f, dinv = 0.f;
    if (g < R) {
      float Bg[P], diag = 0.f;
#pragma unroll
      for (int b = 0; b < P; ++b)
        Bg[b] = cmG[(0 * R + g) * 5 + b] + cmG[(1 * R + g) * 5 + b] + cmG[(2 * R + g) * 5 + b] + cmG[(3 * R + g) * 5 + b];
      diag = cmG[(0 * R + g) * 5 + 4] + cmG[(1 * R + g) * 5 + 4] + cmG[(2 * R + g) * 5 + 4] + cmG[(3 * R + g) * 5 + 4];
      float l2 = 0.f;
#pragma unroll
      for (int c = 0; c < P; ++c) {
        float e = 0.f;
#pragma unroll
        for (int b = 0; b < P; ++b) e += Bg[b] * Ri[b][c];
        LG[c] = e * rs;
        l2 += LG[c] * LG[c];
      }
      dg = fmaxf(diag / mu - l2, 0.f);
      dinv = __builtin_amdgcn_rcpf(dg + a.ridge);  // ridge > 0 (the ABI rejects others)
    }
    // T = I + L_G^T D^{-1} L_G (sum over the lanes g), then its inverse
    float Tm[P][P];
#pragma unroll
    for (int x = 0; x < P; ++x)
#pragma unroll
      for (int y = x; y < P; ++y) {
        const float e = wave_sum(LG[x] * dinv * LG[y]);
        Tm[x][y] = e + (x == y ? 1.f : 0.f);
        Tm[y][x] = Tm[x][y];
      }
    float Ti[P][P];
#pragma unroll
    for (int x = 0; x < P; ++x)
#pragma unroll
      for (int y = 0; y < P; ++y) Ti[x][y] = (x == y) ? 1.f : 0.f;
#pragma unroll
    for (int c = 0; c < P; ++c) {  // Gauss-Jordan on the SPD T (pivots >= 1)
      const float inv = __builtin_amdgcn_rcpf(Tm[c][c]);
#pragma unroll
      for (int y = 0; y < P; ++y) {
        Tm[c][y] *= inv;
        Ti[c][y] *= inv;
      }
#pragma unroll
      for (int x = 0; x < P; ++x) {
        if (x == c) continue;
        const float f = Tm[x][c];
#pragma unroll
        for (int y = 0; y < P; ++y) {
          Tm[x][y] -= f * Tm[c][y];
          Ti[x][y] -= f * Ti[c][y];
        }
      }
    }
    // F1 row g; L_G and w = D^{-1} d of every g for the correction M' = M - L_G^T Diag(w) Omega^T
#pragma unroll
    for (int c = 0; c < P; ++c) {
      float e = 0.f;
#pragma unroll
      for (int b = 0; b < P; ++b) e += LG[b] * Ti[b][c];
      F1[c] = dinv * e;
    }
    float* sL = cmS + 8 + 16;  // [R][P] L_G, then [R] w = D^{-1} d
    if (g < R) {
#pragma unroll
      for (int c = 0; c < P; ++c) sL[g * P + c] = LG[c];
      sL[R * P + g] = dinv * dg;
    }
    if (lane == 0) {
#pragma unroll
      for (int x = 0; x < P; ++x)
#pragma unroll
        for (int y = 0; y < P; ++y) cmS[8 + x * P + y] = Ri[x][y] * rs;
    }
  }
  lds_barrier();
  // M' = R^{-T} N^T / sqrt(mu) - L_G^T Diag(w) Omega^T: thread k sums the four
  // waves' N rows for column k of M, then subtracts sum_h L_G[h] w_h Omega[k][h]
  // (Omega's columns past the head's rank are zero in LDS, and so is w there)
  const float* sL = cmS + 8 + 16;  // [R][P] L_G, then [R] w
  float Mk[P] = {};
  if (tid < K) {
    const int k = tid;
    float Nk[P];
#pragma unroll
    for (int b = 0; b < P; ++b)
      Nk[b] = cmN[(0 * K + k) * P + b] + cmN[(1 * K + k) * P + b] + cmN[(2 * K + k) * P + b] + cmN[(3 * K + k) * P + b];
#pragma unroll
    for (int x = 0; x < P; ++x) {
#pragma unroll
      for (int b = 0; b < P; ++b) Mk[x] += cmS[8 + b * P + x] * Nk[b];
    }
#pragma unroll
    for (int h4 = 0; h4 < R; h4 += 4) {
      const float4 o4 = *reinterpret_cast<const float4*>(&OmL[k * OPJ + h4]);
      const float oh[4] = {o4.x, o4.y, o4.z, o4.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float wo = sL[R * P + h4 + e] * oh[e];
#pragma unroll
        for (int x = 0; x < P; ++x) Mk[x] -= sL[(h4 + e) * P + x] * wo;
      }
    }
  }
  lds_barrier();  // the waves' N rows are consumed: M'^T and F1 take their place
  float* Mb = Ls;                              // [K][P]   M'^T
  float* Fb = FB_ALIAS ? Ls + P * K : Fext;    // [16 RT][FBP]  row j = F1 row j, zero past R
  if (tid < K) *reinterpret_cast<float4*>(&Mb[tid * P]) = make_float4(Mk[0], Mk[1], Mk[2], Mk[3]);
  if (wave == 0 && lane < 16 * RT) {
    float* fr = Fb + lane * FBP;
#pragma unroll
    for (int c = 0; c < P; ++c) fr[c] = lane < R ? F1[c] : 0.f;
  }
  lds_barrier();
  // C^T = M'^T F1^T + (Diag(w) Omega^T)^T: wave w takes k tiles w, w + 4, ...;
  // lane (lr, lg) ends with C[16 jt + lr][16 kt + 4 lg + i], i = 0..3
  constexpr int CPW = 16 / (int)sizeof(SK);
  SK* cm = static_cast<SK*>(a.cmap) + item * (size_t)(R * K);
#pragma unroll
  for (int kq = 0; kq < MT / 4; ++kq) {
    const int kt = wave + 4 * kq;
#pragma unroll
    for (int jt = 0; jt < RT; ++jt) {
      const int j = 16 * jt + lr, k0 = 16 * kt + 4 * lg;
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = mfma4(Mb[(16 * kt + lr) * P + lg], Fb[(16 * jt + lr) * FBP + lg], acc);
      const float wj = j < R ? sL[R * P + j] : 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[i] += wj * OmL[(k0 + i) * OPJ + j];
      if (j < rh) st_elem4<SK>(cm + ((size_t)(k0 / CPW) * R + j) * CPW + k0 % CPW, acc[0], acc[1], acc[2], acc[3]);
    }
  }
}

// The state-dependent map with the exact state metric (eq. pivot-ridge with
// the dense H; Table 2's "Exact"): with Omega orthonormal and R^T R = I,
// J^T H J = U^T U / mu and J^T H R = U^T S^T / mu, so
//   C = (U^T U / mu + lambda I)^{-1} N / mu,   N = U^T X = U^T S^T (G x K).
// The sketch pass leaves per-wave partial products of N^T = U^T X and the
// Gram U^T U (matrix cores, contraction over the wave's value tiles) and of
// |S|_F^2.  They are summed over the waves in LDS in a fixed order (wave 0
// stores, waves 1..3 add in turn), the Gram system is factored by Cholesky
// on one wave (lane = row), every channel's column of the map is solved by
// forward and back substitution (thread k), and the dense map is stored like
// the pivot map's (16-byte channel panels).  G <= 16.  Every thread calls this.
template <int K, int R, typename SK>
__device__ __forceinline__ void coef_map_exact_tail(const UpdateArgs& a, size_t item, int wave, int lane, int tid,
                                                    int rh, const floatx4 (&nacc)[K / 16], const floatx4& gacc,
                                                    float msq, float* Ls, float* Us, float* cmS) {
  constexpr int MT = K / 16, NP = K + 4, GP = R + 1;
  static_assert(R <= 16, "the exact map is compiled for ranks up to 16");
  const int lr = lane & 15, lg = lane >> 4;
  float* Ns = Ls;            // [R][NP]   N, then the map
  float* Gs = Us;            // [R][GP]   U^T U
  float* Lm = Us + R * GP;   // [R][GP]   its Cholesky factor; then 1 / diagonal at Lm[j * GP + j]
  msq = wave_sum(msq);
  // rows j = 4 lg + i of N^T and of the Gram live in lane group lg
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    lds_barrier();  // w = 0: every wave is done with the pass's scratch in Ls
    if (wave == w) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = 4 * lg + i;
        if (j < R) {
#pragma unroll
          for (int kt = 0; kt < MT; ++kt) {
            float* p = &Ns[j * NP + 16 * kt + lr];
            *p = (w == 0 ? 0.f : *p) + nacc[kt][i];
          }
          if (lr < R) {
            float* p = &Gs[j * GP + lr];
            *p = (w == 0 ? 0.f : *p) + gacc[i];
          }
        }
      }
      if (lane == 0) cmS[w] = msq;
    }
  }
  lds_barrier();
  const float fro = cmS[0] + cmS[1] + cmS[2] + cmS[3];
  const float mu = fro > 0.f ? fro / K : 1.f;
  const float imu = 1.f / mu;
  if (wave == 0) {
    // Cholesky of A = U^T U / mu + lambda I: lane j holds row j
    float ar[R];
#pragma unroll
    for (int g = 0; g < R; ++g) ar[g] = (lane < R ? Gs[lane * GP + g] * imu : 0.f) + (lane == g ? a.ridge : 0.f);
    float lrow[R];
#pragma unroll
    for (int c = 0; c < R; ++c) {
      const float piv = lane_bcast(ar[c], c);          // A_cc after the updates of columns < c (> 0: SPD)
      const float ip = __builtin_amdgcn_rsqf(piv);
      const float l = ar[c] * ip;                      // L_jc for j >= c
      lrow[c] = lane >= c ? l : 0.f;
#pragma unroll
      for (int g = c + 1; g < R; ++g) ar[g] -= l * lane_bcast(l, g);
    }
    if (lane < R) {
#pragma unroll
      for (int c = 0; c < R; ++c) Lm[lane * GP + c] = c == lane ? 1.f / lrow[c] : lrow[c];
    }
  }
  lds_barrier();
  // column k of the map: L y = N_k / mu, L^T c = y.  Each row's reads of L
  // stay within its own step (scheduling barrier): hoisting the whole
  // triangle's reads ahead held 136 values live at rank 16 and took the
  // kernel from 80 to 162 registers.
  if (tid < K) {
    const int k = tid;
    float y[R];
#pragma unroll
    for (int j = 0; j < R; ++j) {
      float e = Ns[j * NP + k] * imu;
#pragma unroll
      for (int c = 0; c < j; ++c) e -= Lm[j * GP + c] * y[c];
      y[j] = e * Lm[j * GP + j];
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int j = R - 1; j >= 0; --j) {
      float e = y[j];
#pragma unroll
      for (int c = j + 1; c < R; ++c) e -= Lm[c * GP + j] * y[c];
      y[j] = e * Lm[j * GP + j];
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int j = 0; j < R; ++j) Ns[j * NP + k] = y[j];
  }
  lds_barrier();
  // the dense map in 16-byte channel panels: thread (kp, j), j fastest
  constexpr int CPW = 16 / (int)sizeof(SK);
  SK* cm = static_cast<SK*>(a.cmap) + item * (size_t)(R * K);
#pragma unroll
  for (int t = tid; t < R * K / CPW; t += 256) {
    const int j = t % R, kp = t / R;
    if (j < rh) {
      const float* src = &Ns[j * NP + kp * CPW];
#pragma unroll
      for (int e = 0; e < CPW; e += 4) st_elem4<SK>(cm + (size_t)t * CPW + e, src[e], src[e + 1], src[e + 2], src[e + 3]);
    }
  }
}

// The rank update of one 16-value tile of X = S^T from the factors of a window
// (or a chunk of one) staged in LDS, eq. wy: lane (lr, lg) holds
// X[v][16 kt + 4 lg + i] in x[kt][i], v = 16 vt + lr, and
//   X^T <- Diag(e^{g_n}) X^T + (keys or L)^T W^T,
// with w_s = c_s (u_s - (Pi X^T)[s]) (GDN), u_s - (Pi X^T)[s] (KDA, whose decays
// are in L and ds) or c_s beta_s v_s (Mamba-2), slot s = 16 st + 4 lg + i.
template <int KIND, int MT, int ST, int LP, int PP, int UP>
__device__ __forceinline__ void rank_update_tile(floatx4 (&x)[MT], int v, int lr, int lg, float egn, const float* Ls,
                                                 const float* PiT, const float* Us, const float* bsl, const float* csc,
                                                 const float* ds) {
  constexpr bool ERASE = KIND != MAMBA2;
  constexpr bool CHAN = KIND == KDA;
  floatx4 wv[ST];
#pragma unroll
  for (int st = 0; st < ST; ++st) {
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    if constexpr (ERASE) {
      // (Pi X^T)[s] in four independent accumulation chains
      floatx4 pc[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) pc[i] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kt = 0; kt < MT; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          pc[i] = mfma4(PiT[(16 * kt + 4 * lg + i) * PP + 16 * st + lr], x[kt][i], pc[i]);
      acc = (pc[0] + pc[1]) + (pc[2] + pc[3]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int s = 16 * st + 4 * lg + i;
      float w = Us[s * UP + v] - acc[i];
      if constexpr (!ERASE) w *= bsl[s] * csc[s];
      if constexpr (ERASE && !CHAN) w *= csc[s];
      wv[st][i] = w;
    }
  }
#pragma unroll
  for (int kt = 0; kt < MT; ++kt) {
    floatx4 acc;
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = x[kt][i] * (CHAN ? ds[16 * kt + 4 * lg + i] : egn);
#pragma unroll
    for (int st = 0; st < ST; ++st)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc = mfma4(Ls[(16 * st + 4 * lg + i) * LP + 16 * kt + lr], wv[st][i], acc);
    x[kt] = acc;
  }
}

// Three workgroups per CU, or four for the state-dependent maps (P = 4 and
// exact) at window 16 and rank <= 16: their flush spends part of each
// workgroup's life off the memory bus (the map's products and algebra), so
// occupancy pays there, even with the few registers the per-channel-decay
// instances then spill.
template <int KIND, int K, int V, int R, int WMAX, typename IO, typename SK, int P>
__global__ __launch_bounds__(256, (P != 0 && WMAX == 16 && R <= 16) ? 4 : 3) void update_kernel(const UpdateArgs a) {
  constexpr bool ERASE = KIND != MAMBA2;
  constexpr bool CHAN = KIND == KDA;
  constexpr int MT = K / 16;          // k tiles
  constexpr int VT = V / 16;          // value tiles
  constexpr int VTW = (VT + 3) / 4;   // value tiles per wave
  // The erase families flush a window of up to 32 slots as chunks of 16 on
  // the register-resident state: T is unit lower triangular, so the rows of
  // T^{-1} that couple a chunk's slots among themselves are the inverse of
  // that chunk's own T, and a chunk started from the state the previous one
  // left is a window of its own (decays taken from the chunk's first slot).
  // The staging and registers are then those of a 16-slot window.
  constexpr int SP = ERASE ? 16 : WMAX;  // staged slot rows (16 or 32)
  constexpr int CH = WMAX / SP;          // chunks per flush
  constexpr int ST = SP / 16;         // slot tiles
  constexpr int NG = SP / 4;          // slot groups of four
  constexpr int RT = (R + 15) / 16;   // sketch tiles
  constexpr int KPL = K / 16;         // key channels per lane (row layout)
  constexpr int VR = V / 16;          // value channels per lane (row layout)
  constexpr int LP = K + 4;           // LDS pitches chosen so that the 4 lane
  constexpr int PP = SP + 4;          // groups of an operand read land in
  constexpr int UP = V + 4;           // different banks
  constexpr int KW = (K + 63) / 64;   // waves that carry channel work

  __shared__ __align__(16) float Ls[SP * LP];                 // keys k_s (KDA: then L[s]), [s][k]
  __shared__ __align__(16) float PiT[ERASE ? K * PP : 4];     // Pi^T[k][s]
  __shared__ __align__(16) float Us[SP * UP];                 // raw v_s (Mamba-2) or u_s
  __shared__ float Bs[ERASE ? SP * SP : 1];                   // (T^{-1})_{s,j}, j < s < n
  __shared__ float bpart[ERASE ? KW * SP : 1];                // partial sums of b_{n,j}
  __shared__ __align__(16) float qs[K];
  __shared__ __align__(16) float ds[CHAN ? K : 4];            // e^{g_n} per channel (KDA)
  __shared__ float csc[SP];                                   // c_s = e^{g_n - g_s} (scalar decay)
  __shared__ float bsl[SP], gsl[SP];                          // beta_s, g_s (0 past slot n)

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lg = lane >> 4;   // MFMA lane coordinates
  const int row = lg, col = lr;               // row-layout coordinates (same lanes)
  const int H = a.H, W = a.W, nw = a.n;  // nw: the window's current slot
  const size_t item = blockIdx.x;  // b * H + h (B*H <= 2^30)
  const int h = (int)(blockIdx.x % (uint32_t)H);
  const bool flush = a.nt > 0;
  // slot s of an item: raw ring fields at (item * W + s) * width, derived
  // fields at (s * B*H + dp) * width, dp = h * B + b
  const size_t NI = (size_t)a.B * H, dp = (size_t)h * a.B + blockIdx.x / (uint32_t)H;

  // Omega of this head goes to LDS (rows padded to whole 16-column tiles plus
  // four words, so the four lane groups of an operand read hit different banks)
  // when it is small; the full-rank case reads it from global memory.
  constexpr bool OM_LDS = R > 0 && R <= 32;
  constexpr int OPJ = 16 * RT + 4;
  constexpr int OQ = OM_LDS ? (K * R / 4 + 255) / 256 : 1;  // float4 of Omega per thread
  __shared__ __align__(16) float OmL[OM_LDS ? K * OPJ : 4];
  // this head's rank (per-head rank table): the sketch uses Omega's first rh
  // columns (the rest are zeroed in LDS, so U's columns past rh come out 0 and
  // the state-dependent map's rows past rh too); rh = 0: a dense-fallback head
  const int rh = a.ragged ? arg_byte(a.hrank, h) : R;
  const bool want_U = R > 0 && a.U != nullptr && rh > 0;

  // state-dependent coefficient map (P = 4 pivots, or the exact metric, P < 0):
  // per-wave scratch for the block transposes of X and of the sketch columns,
  // and the small factors shared by the workgroup
  constexpr bool EXACT = P < 0;
  static_assert(P == 0 || (P == 4 && R >= 8 && R <= 32) || (EXACT && R >= 8 && R <= 16),
                "state-dependent maps: P = 4 with rank 8..32, or the exact metric with rank 8..16");
  constexpr int XP = 20;                                        // row pitch of a transposed 16 x 16 block
  // When the key staging Ls has room, that scratch lives in Ls: every tile is
  // then updated first and sketched after a barrier, once Ls is dead.  This
  // keeps the kernel's LDS that of the offline-map flush (four workgroups per CU).
  // Each tile's sketch columns go through the same per-wave block as X's
  // (one after the other).
  constexpr bool CM_ALIAS = P != 0 && SP * LP >= 4 * 16 * XP;
  __shared__ __align__(16) float cmXs[P != 0 && !CM_ALIAS ? 4 * 16 * XP : 4];
  float* const cmX = CM_ALIAS ? Ls : cmXs;                 // [wave][16 values][16 keys]
  float* const cmU = cmX;                                  // [wave][16 values][16 sketch columns], before X's blocks
  __shared__ __align__(16) float cmS[P != 0 ? 8 + 16 + 5 * R : 4];  // mu parts, R^{-1}/sqrt(mu), L_G and w
  // F1 of the map, in its own LDS only where the key staging has no room
  constexpr bool CMF_OWN = P > 0 && SP * LP < P * K + 16 * RT * (P + 1);
  __shared__ __align__(16) float cmF[CMF_OWN ? 16 * RT * (P + 1) : 4];
  static_assert(!EXACT || (SP * LP >= R * (K + 4) && SP * UP >= 2 * R * (R + 1)),
                "the exact map's sums must fit the window staging");
  floatx4 nacc[P != 0 ? MT : 1];   // N^T (rows 4 lg + i: pivots a < 4, or every sketch column), this wave's values
  floatx4 gram[P > 0 ? RT : 1];    // sketch Gram U^T U_p: lane (lr, lg), i: row 16 jt + 4 lg + i, column lr < P; this wave's values
  float dsq[P > 0 ? RT : 1];       // squared sketch column 16 jt + lr over this lane row's values
  [[maybe_unused]] floatx4 gacc = {0.f, 0.f, 0.f, 0.f};  // exact: U^T U (rows 4 lg + i, column lr), this wave's values
  float msq = 0.f;                 // this lane's share of |S|_F^2
  if constexpr (P != 0) {
#pragma unroll
    for (int kt = 0; kt < MT; ++kt) nacc[kt] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  if constexpr (P > 0) {
#pragma unroll
    for (int jt = 0; jt < RT; ++jt) {
      gram[jt] = floatx4{0.f, 0.f, 0.f, 0.f};
      dsq[jt] = 0.f;
    }
  }

  // ---- every small load first (window, query, rows of T^{-1}, Omega), then the
  // state: the staged values reach LDS while the state read is still in flight
  float egn = 1.f, gn = 0.f, bn = 0.f;  // the chunk's e^{g_n} (scalar decay), g_n, beta_n (from LDS after the staging)
  Raw<IO, 1> qr;  // this thread's query channel, raw (converted at the staging, so no wait here)
  constexpr int BQ = ERASE ? (SP * SP + 255) / 256 : 1;
  Vec<4> omv[OQ];
  floatx4 xs[VTW][MT];
#pragma unroll
  for (int ch = 0; ch < CH; ++ch) {
    const int sb = 16 * ch;                                 // the chunk's first slot in the ring
    // the chunk's current slot (counted from sb), and whether the chunk holds
    // the window's current slot (then it is the last one)
    const int n = CH == 1 ? nw : !flush ? 0 : (nw - sb < SP ? nw - sb : SP - 1);
    const bool last = CH == 1 || !flush || nw < sb + SP;
    float bl = 0.f, ll = 0.f;             // wave 0, lane s: beta_s and (scalar decay) log alpha_s
    float gk[CHAN ? SP : 1];              // KDA: g_s of channel tid
    Raw<IO, KPL> kr[NG / 4];              // ring keys, row layout (slot 4 (wave + 4 gq) + row)
    Raw<IO, VR> vr[NG / 4];               // raw values
    float bv[BQ];
    if (flush) {
      // per-slot scalars: lane s of wave 0 loads slot s; every slot load is
      // issued before any is used (slots past n re-read slot n, in bounds, and
      // are masked afterwards), so no load waits on a branch
      if (tid < SP) {
        const size_t si = item * W + sb + (tid < n ? tid : n);
        bl = a.rbeta[si];
        if constexpr (!CHAN) ll = a.rla[si];
      }
      if constexpr (CHAN) {
        if (tid < K) {
#pragma unroll
          for (int s = 0; s < SP; ++s) gk[s] = a.rla[(item * W + sb + (s < n ? s : n)) * K + tid];
        }
      }
#pragma unroll
      for (int gq = 0; gq < NG / 4; ++gq) {
        const int s = 4 * (wave + 4 * gq) + row;
        const size_t si = item * W + sb + s;
        if (s <= n) {
          kr[gq].load(static_cast<const IO*>(a.rk) + si * K + col * KPL);
          vr[gq].load(static_cast<const IO*>(a.rv) + si * V + col * VR);
        }
      }
      if (ch == 0) qr.load(static_cast<const IO*>(a.q) + item * K + (tid < K ? tid : K - 1));
      if constexpr (ERASE) {
#pragma unroll
        for (int c = 0; c < BQ; ++c) {
          const int idx = tid + 256 * c;
          const int s = idx / SP, j = idx % SP;
          bv[c] = (idx < SP * SP && s < n && j < s) ? a.rt[((size_t)(sb + s) * NI + dp) * W + sb + j] : 0.f;
        }
      }
    }
    if constexpr (OM_LDS) {
      if (ch == 0 && want_U) {
#pragma unroll
        for (int c = 0; c < OQ; ++c) {
          const int i = tid + 256 * c;
#pragma unroll
          for (int e = 0; e < 4; ++e) omv[c].e[e] = 0.f;
          if (i < K * R / 4 && 4 * (i % (R / 4)) < rh) omv[c].load(a.omega + (size_t)h * K * R + 4 * i);
        }
      }
    }

    // ---- the single read of the state (unconditional where every wave owns
    // VTW tiles, so that waiting for the staged loads never waits for these)
    if (ch == 0) {
#pragma unroll
      for (int t = 0; t < VTW; ++t) {
        const int vt = wave + 4 * t;
        if (VT % 4 == 0 || vt < VT) {
          // tile (vt, kt) of the state is 1 KB contiguous, lane l's float4 at 4 l
          const float* src = a.S + item * V * K + (size_t)(vt * MT) * 256 + 4 * lane;
#pragma unroll
          for (int kt = 0; kt < MT; ++kt) {
            const float4 x = ld_nt(reinterpret_cast<const float4*>(src + 256 * kt));
            xs[t][kt] = floatx4{x.x, x.y, x.z, x.w};
          }
        }
      }
    }
    compiler_fence();

    // ---- staged values into LDS
    if constexpr (OM_LDS) {
      if (ch == 0 && want_U) {
#pragma unroll
        for (int c = 0; c < OQ; ++c) {
          const int i = tid + 256 * c;
          if (i < K * R / 4) {
            Vec<4> w = omv[c];
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (4 * (i % (R / 4)) + e >= rh) w.e[e] = 0.f;
            w.store(&OmL[(i / (R / 4)) * OPJ + 4 * (i % (R / 4))]);
          }
        }
        if constexpr (R < 16 * RT) {  // zero columns R..16 RT-1
          constexpr int ZQ = (16 * RT - R) / 4;
          for (int i = tid; i < K * ZQ; i += 256)
            *reinterpret_cast<float4*>(&OmL[(i / ZQ) * OPJ + R + 4 * (i % ZQ)]) = make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
    }
    if (flush) {
#pragma unroll
      for (int gq = 0; gq < NG / 4; ++gq) {
        const int s = 4 * (wave + 4 * gq) + row;
        float ksv[KPL], vsv[VR];
#pragma unroll
        for (int m = 0; m < KPL; ++m) ksv[m] = 0.f;
#pragma unroll
        for (int m = 0; m < VR; ++m) vsv[m] = 0.f;
        if (s <= n) {
#pragma unroll
          for (int m = 0; m < KPL; ++m) ksv[m] = kr[gq].get(m);
          // raw values (Mamba-2 scales them by beta_s c_s where they are used)
#pragma unroll
          for (int m = 0; m < VR; ++m) vsv[m] = vr[gq].get(m);
        }
#pragma unroll
        for (int m = 0; m < KPL; m += 4)
          *reinterpret_cast<float4*>(&Ls[s * LP + col * KPL + m]) = make_float4(ksv[m], ksv[m + 1], ksv[m + 2], ksv[m + 3]);
#pragma unroll
        for (int m = 0; m < VR; m += 4)
          *reinterpret_cast<float4*>(&Us[s * UP + col * VR + m]) = make_float4(vsv[m], vsv[m + 1], vsv[m + 2], vsv[m + 3]);
      }
      if (ch == 0 && tid < K) qs[tid] = qr.get(0);
      if (tid < 64) {
        // wave 0: beta_s, g_s = sum_{j<=s} log alpha_j (inclusive scan over the
        // lanes) and c_s = e^{g_n - g_s}, slots past n zero
        const int sl = tid;
        const bool live = sl <= n && sl < SP;
        float g = (!CHAN && live) ? ll : 0.f;
#pragma unroll
        for (int d = 1; d < SP; d <<= 1) {
          const float u = __shfl_up(g, d);
          if (sl >= d) g += u;
        }
        const float gnn = __shfl(g, n);
        if (sl < SP) {
          bsl[sl] = live ? bl : 0.f;
          gsl[sl] = live ? g : 0.f;
          if constexpr (!CHAN) csc[sl] = live ? fast_exp(gnn - g) : 0.f;
        }
      }
      if constexpr (ERASE) {
#pragma unroll
        for (int c = 0; c < BQ; ++c) {
          const int idx = tid + 256 * c;
          if (idx < SP * SP) Bs[idx] = bv[c];
        }
      }
    }
    lds_barrier();
    if (flush) {  // the current slot's scalars, for every thread
      gn = gsl[n];
      bn = bsl[n];
      if constexpr (!CHAN) egn = fast_exp(gn);
    }

    if (flush) {
      if constexpr (ERASE) {
        // ---- channel work: thread tid owns channel k = tid.  Ls holds raw keys.
        // The pseudo-values of slots before n need only the stored rows of T^{-1},
        // so the waves that own no channel form them meanwhile.
        static_assert(K + V <= 256, "channel waves and value waves must be disjoint");
        float pi[SP], kn = 0.f;
        if (tid < K) {
          const int kk = tid;
          kn = Ls[n * LP + kk];
          float gnk = gn;
          if constexpr (CHAN) {
            // g_s of channel tid: running sum of the chunk's log alphas
            float acc = 0.f;
#pragma unroll
            for (int s = 0; s < SP; ++s) {
              acc += s <= n ? gk[s] : 0.f;
              gk[s] = s <= n ? acc : 0.f;
            }
#pragma unroll
            for (int s = 0; s < SP; ++s)
              if (s == n) gnk = gk[s];
          }
          // erase factors pi_s = sum_{j<=s} (T^{-1})_{s,j} beta_j e^{g_j} k_j, s < n
          // (eq. wy with T^{-1} from the ring): independent sums, no recursion
          float xk[SP];
#pragma unroll
          for (int s = 0; s < SP; ++s) xk[s] = s < n ? bsl[s] * fast_exp(CHAN ? gk[s] : gsl[s]) * Ls[s * LP + kk] : 0.f;
#pragma unroll
          for (int s = 0; s < SP; ++s) {
            pi[s] = 0.f;
            if (s < n) {
              float acc = xk[s];
#pragma unroll
              for (int j = 0; j < s; ++j) acc += Bs[s * SP + j] * xk[j];
              pi[s] = acc;
            }
          }
          // b_{n,s} = <exp(g_n - g_s) . k_s, k_n>: partial sums over this wave's channels
#pragma unroll
          for (int s = 0; s < SP; ++s) {
            if (s < n) {
              const float e = CHAN ? fast_exp(gnk - gk[s]) : csc[s];
              const float bsum = wave_sum(e * Ls[s * LP + kk] * kn);
              if (lane == 0) bpart[wave * SP + s] = bsum;
            }
          }
          if constexpr (CHAN) {
            // left factors L[s] = exp(g_n - g_s) k_s replace the keys in place
            ds[kk] = fast_exp(gnk);
#pragma unroll
            for (int s = 0; s < SP; ++s)
              if (s < n) Ls[s * LP + kk] *= fast_exp(gnk - gk[s]);
          }
        } else if (tid >= 256 - V) {
          // pseudo-values u_s = sum_{j<=s} (T^{-1})_{s,j} beta_j v_j, s < n, in
          // place over the raw values (thread owns value channel v)
          const int v = tid - (256 - V);
          float xv[SP];
#pragma unroll
          for (int s = 0; s < SP; ++s) xv[s] = s < n ? bsl[s] * Us[s * UP + v] : 0.f;
#pragma unroll
          for (int s = 0; s < SP; ++s) {
            if (s < n) {
              float acc = xv[s];
#pragma unroll
              for (int j = 0; j < s; ++j) acc += Bs[s * SP + j] * xv[j];
              Us[s * UP + v] = acc;
            }
          }
        }
        lds_barrier();
        // ---- slot n: row n of the couplings comes from every wave's partial sums
        if (tid < V) {
          const int v = tid;
          float acc = Us[n * UP + v];
#pragma unroll
          for (int j = 0; j < SP; ++j) {
            if (j < n) {
              float bj = 0.f;
#pragma unroll
              for (int w = 0; w < KW; ++w) bj += bpart[w * SP + j];
              acc -= bj * Us[j * UP + v];
            }
          }
          Us[n * UP + v] = bn * acc;
        }
        if (tid < K) {
          const int kk = tid;
          float gnk = gn;
          if constexpr (CHAN) {
#pragma unroll
            for (int s = 0; s < SP; ++s)
              if (s == n) gnk = gk[s];
          }
          float acc = fast_exp(gnk) * kn;
#pragma unroll
          for (int j = 0; j < SP; ++j) {
            if (j < n) {
              float bj = 0.f;
#pragma unroll
              for (int w = 0; w < KW; ++w) bj += bpart[w * SP + j];
              acc -= bj * pi[j];
            }
          }
          const float pin = bn * acc;
#pragma unroll
          for (int s = 0; s < SP; ++s) PiT[kk * PP + s] = (s < n) ? pi[s] : (s == n ? pin : 0.f);
        }
        lds_barrier();
      }
    }
    if (last) break;
    // an earlier chunk: its update, before the next chunk's staging reuses the LDS
#pragma unroll
    for (int t = 0; t < VTW; ++t)
      if (wave + 4 * t < VT)
        rank_update_tile<KIND, MT, ST, LP, PP, UP>(xs[t], 16 * (wave + 4 * t) + lr, lr, lg, egn, Ls, PiT, Us, bsl, csc, ds);
    lds_barrier();
  }

  // ---- matrix-core phase, one 16-column value tile at a time (with a
  // state-dependent map: pass 0 updates and stores every tile, pass 1
  // sketches them)
  constexpr int PASSES = P != 0 ? 2 : 1;
  float msc = 1.f;  // pass 1: the power of two the map's partial sums scale the state by
  float xmax = 0.f;  // pass 0: this lane's largest state magnitude (state-dependent map)
#pragma unroll
  for (int ps = 0; ps < PASSES; ++ps) {
  if constexpr (P != 0) {
  if (ps == 1) {
    // The map is invariant to the state's scale.  Its partial sums (|S|^2,
    // the Gram of the sketch, N) are quadratic in the state, so they are
    // formed from the state scaled by 2^-e, e the exponent of the item's
    // largest magnitude (exact; the scaled largest magnitude is in [0.5, 1)):
    // a state that has decayed far (below ~1e-19) would otherwise square
    // into fp32's denormal range and break the map's algebra.
    const float m0 = wave_max(xmax);
    if (lane == 0) cmS[4 + wave] = m0;
    lds_barrier();  // also: every wave is done with Ls before the map's scratch reuses it
    const float m = fmaxf(fmaxf(cmS[4], cmS[5]), fmaxf(cmS[6], cmS[7]));
    int e = 0;
    (void)frexpf(m, &e);
    msc = m > 0.f ? ldexpf(1.f, -e) : 1.f;
  }
  }
#pragma unroll
  for (int t = 0; t < VTW; ++t) {
    const int vt = wave + 4 * t;
    if (vt >= VT) continue;
    const int v = 16 * vt + lr;
    if (flush && ps == 0) {
      rank_update_tile<KIND, MT, ST, LP, PP, UP>(xs[t], v, lr, lg, egn, Ls, PiT, Us, bsl, csc, ds);
      // exact output o_W[v] = sum_k X_W[v][k] q_W[k]
      if (a.o) {
        float p = 0.f;
#pragma unroll
        for (int kt = 0; kt < MT; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) p += xs[t][kt][i] * qs[16 * kt + 4 * lg + i];
        p = cross_row_sum(p);
        if (lg == 0) a.o[item * V + v] = p;
      }
      // the state is final: store it before the sketch and map products
      {
        float* dst = a.S + item * V * K + (size_t)(vt * MT) * 256 + 4 * lane;
#pragma unroll
        for (int kt = 0; kt < MT; ++kt)
          st_nt(reinterpret_cast<float4*>(dst + 256 * kt), make_float4(xs[t][kt][0], xs[t][kt][1], xs[t][kt][2], xs[t][kt][3]));
      }
    }
    if constexpr (P != 0) {
      if (ps == 0) {  // the tile is final (updated, or as loaded for the initial sketch)
#pragma unroll
        for (int kt = 0; kt < MT; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) xmax = fmaxf(xmax, fabsf(xs[t][kt][i]));
      }
    }
    // sketch U^T = Omega^T X^T  (rows j = 16 jt + 4 lg + i of the C layout)
    if constexpr (R > 0) {
      if (want_U && ps == PASSES - 1) {
        const float* om = a.omega + (size_t)h * K * R;
        float aop[4] = {0.f, 0.f, 0.f, 0.f};            // U_p^T (exact: U^T) as the A operand of N^T = U_p^T X
#pragma unroll
        for (int jt = 0; jt < RT; ++jt) {
          const int jj = 16 * jt + lr;
          floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kt = 0; kt < MT; ++kt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              float w;
              if constexpr (OM_LDS)
                w = OmL[(16 * kt + 4 * lg + i) * OPJ + jj];
              else
                w = (jj < R) ? om[(16 * kt + 4 * lg + i) * R + jj] : 0.f;
              acc = mfma4(w, xs[t][kt][i], acc);
            }
          if constexpr (P != 0) {
            // every sketch column of the tile's 16 values goes through LDS, so
            // that U^T becomes an operand with the value index as the
            // contraction index: ut[st] = U[v = 4 st + lg][16 jt + lr], scaled
            float* cu = cmU + wave * 16 * XP;
            wave_lds_sync();
            *reinterpret_cast<float4*>(&cu[lr * XP + 4 * lg]) =
                make_float4(acc[0] * msc, acc[1] * msc, acc[2] * msc, acc[3] * msc);
            wave_lds_sync();
            float ut[4];
#pragma unroll
            for (int st = 0; st < 4; ++st) ut[st] = cu[(4 * st + lg) * XP + lr];
            if constexpr (EXACT) {
              // the whole Gram U^T U (R <= 16: one block)
#pragma unroll
              for (int st = 0; st < 4; ++st) {
                aop[st] = ut[st];
                gacc = mfma4(ut[st], ut[st], gacc);
              }
            } else {
              // the Gram against the first P columns (tile 0's, kept from
              // jt = 0) on the matrix cores, and the squared columns
              if (jt == 0) {
#pragma unroll
                for (int st = 0; st < 4; ++st) aop[st] = lr < P ? ut[st] : 0.f;
              }
#pragma unroll
              for (int st = 0; st < 4; ++st) {
                gram[jt] = mfma4(ut[st], aop[st], gram[jt]);
                dsq[jt] += ut[st] * ut[st];
              }
            }
          }
          // columns 16 jt + 4 lg .. +3 of value v; panels of 16 bytes per value:
          // fp32 U[B][H][R/4][V][4], bf16 U[B][H][R/8][V][8]
          // (panels past this head's rank are not stored; the tail of its last
          // panel holds zeros)
          constexpr int PWU = 16 / (int)sizeof(SK);
          if (16 * jt + 4 * lg < R && ((16 * jt + 4 * lg) / PWU) * PWU < rh) {
            SK* Ui = static_cast<SK*>(a.U) + item * (size_t)V * R;
            if constexpr (sizeof(SK) == 4) {
              reinterpret_cast<float4*>(Ui)[(4 * jt + lg) * V + v] = make_float4(acc[0], acc[1], acc[2], acc[3]);
            } else {
              const uint2 w = make_uint2(bf16_bits_rne(acc[0]) | (bf16_bits_rne(acc[1]) << 16),
                                         bf16_bits_rne(acc[2]) | (bf16_bits_rne(acc[3]) << 16));
              reinterpret_cast<uint2*>(Ui)[((2 * jt + (lg >> 1)) * V + v) * 2 + (lg & 1)] = w;
            }
          }
        }
        if constexpr (P != 0) {
          // N^T = U_p^T X (exact map: U^T X) over this tile's 16 values on the matrix cores: each 16 x 16
          // block of X goes through LDS so that the value index becomes the
          // contraction index (lane group), then four 16x16x4 steps
          float* cx = cmX + wave * 16 * XP;
#pragma unroll
          for (int kt = 0; kt < MT; ++kt) {
            wave_lds_sync();
            const float4 xsc = make_float4(xs[t][kt][0] * msc, xs[t][kt][1] * msc, xs[t][kt][2] * msc,
                                           xs[t][kt][3] * msc);
            *reinterpret_cast<float4*>(&cx[lr * XP + 4 * lg]) = xsc;
            wave_lds_sync();
#pragma unroll
            for (int st = 0; st < 4; ++st) nacc[kt] = mfma4(aop[st], cx[(4 * st + lg) * XP + lr], nacc[kt]);
            // one accumulation per element (a four-term sum here keeps the scaled
            // values live across the syncs: 22 more registers for Mamba-2)
#pragma unroll
            for (int i = 0; i < 4; ++i) msq += (xs[t][kt][i] * msc) * (xs[t][kt][i] * msc);
          }
        }
      }
    }
  }
  }

  if constexpr (P > 0) {
    if (want_U)
      coef_map_tail<K, R, P, MT, RT, SP * LP, SP * UP, OPJ, SK>(a, item, wave, lane, tid, rh, nacc, gram, dsq, msq, Ls, Us,
                                                                 cmS, OmL, cmF);
  }
  if constexpr (EXACT) {
    if (want_U) coef_map_exact_tail<K, R, SK>(a, item, wave, lane, tid, rh, nacc, gacc, msq, Ls, Us, cmS);
  }
}


// One token and no sketch: the whole-state recurrence (Sec. 3.2, eq.
// transition-update: decay, then erase, then write) applied to S read once
// and written once, and o = S^T q from the updated state (eq. read).  This is
// the update with a single buffered token at rank 0, i.e. the window-1
// decoding a conventional recurrent layer does.  The window's machinery
// (staged slots, rows of T^{-1}, rank-W products on the matrix cores) reduces
// to one rank-1 update per state element, so the state streams through
// registers: in the tile-major layout lane (lr, lg) of a wave holds
// X[16 vt + lr][16 kt + 4 lg + i] (X = S^T), and the two contractions over
// keys (X k for the erase, X q for the output) are per-lane partial sums and
// one cross-row sum.  In X's terms the update is
//   X <- X Diag(alpha) + beta (v - X Diag(alpha) k) k^T     (GDN, KDA)
//   X <- alpha X + beta v k^T                               (Mamba-2).
template <int KIND, int K, int V, typename IO>
__global__ __launch_bounds__(256) void token_kernel(const UpdateArgs a) {
  constexpr bool ERASE = KIND != MAMBA2;
  constexpr bool CHAN = KIND == KDA;
  constexpr int MT = K / 16, VT = V / 16, VTW = (VT + 3) / 4;
  __shared__ __align__(16) float ks[K];              // k
  __shared__ __align__(16) float qs[K];              // q
  __shared__ __align__(16) float as[CHAN ? K : 4];   // per-channel decay alpha (KDA)
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lg = lane >> 4;
  const size_t item = blockIdx.x;                    // b * H + h
  const size_t cur = item * (size_t)a.W + a.n;       // the token's raw ring slot

  // ---- the token's small loads, then the single read of the state
  float kk = 0.f, qq = 0.f, lk = 0.f;
  if (tid < K) {
    kk = load1<IO>(static_cast<const IO*>(a.rk) + cur * K + tid);
    qq = load1<IO>(static_cast<const IO*>(a.q) + item * K + tid);
    if constexpr (CHAN) lk = a.rla[cur * K + tid];
  }
  const float beta = a.rbeta[cur];
  const float ls = CHAN ? 0.f : a.rla[cur];
  float vv[VTW];
#pragma unroll
  for (int t = 0; t < VTW; ++t) {
    const int vt = wave + 4 * t;
    vv[t] = vt < VT ? load1<IO>(static_cast<const IO*>(a.rv) + cur * V + 16 * vt + lr) : 0.f;
  }
  floatx4 xs[VTW][MT];
#pragma unroll
  for (int t = 0; t < VTW; ++t) {
    const int vt = wave + 4 * t;
    if (vt < VT) {
      const float* src = a.S + item * V * K + (size_t)(vt * MT) * 256 + 4 * lane;
#pragma unroll
      for (int kt = 0; kt < MT; ++kt) {
        const float4 x = ld_nt(reinterpret_cast<const float4*>(src + 256 * kt));
        xs[t][kt] = floatx4{x.x, x.y, x.z, x.w};
      }
    }
  }
  compiler_fence();
  if (tid < K) {
    ks[tid] = kk;
    qs[tid] = qq;
    if constexpr (CHAN) as[tid] = fast_exp(lk);
  }
  lds_barrier();  // LDS only: the state loads stay in flight
  const float alpha = CHAN ? 1.f : fast_exp(ls);

#pragma unroll
  for (int t = 0; t < VTW; ++t) {
    const int vt = wave + 4 * t;
    if (vt >= VT) continue;
    // k, q and alpha are re-read from LDS per tile: kept in registers across
    // the wave's tiles they would double its registers
    compiler_fence();
    // w = beta (v - X Diag(alpha) k), or beta v without the erase
    float w = beta * vv[t];
    if constexpr (ERASE) {
      float y = 0.f;
#pragma unroll
      for (int kt = 0; kt < MT; ++kt) {
        const float4 k4 = *reinterpret_cast<const float4*>(&ks[16 * kt + 4 * lg]);
        float4 d4 = make_float4(alpha, alpha, alpha, alpha);
        if constexpr (CHAN) d4 = *reinterpret_cast<const float4*>(&as[16 * kt + 4 * lg]);
        y += xs[t][kt][0] * (d4.x * k4.x) + xs[t][kt][1] * (d4.y * k4.y) + xs[t][kt][2] * (d4.z * k4.z) +
             xs[t][kt][3] * (d4.w * k4.w);
      }
      w = beta * (vv[t] - cross_row_sum(y));
    }
    compiler_fence();  // k is read again below rather than held across the cross-row sum
    // X <- X Diag(alpha) + w k^T, then o = X q
    float p = 0.f;
#pragma unroll
    for (int kt = 0; kt < MT; ++kt) {
      const float4 k4 = *reinterpret_cast<const float4*>(&ks[16 * kt + 4 * lg]);
      const float4 q4 = *reinterpret_cast<const float4*>(&qs[16 * kt + 4 * lg]);
      float4 d4 = make_float4(alpha, alpha, alpha, alpha);
      if constexpr (CHAN) d4 = *reinterpret_cast<const float4*>(&as[16 * kt + 4 * lg]);
      floatx4 x = xs[t][kt];
      x[0] = x[0] * d4.x + w * k4.x;
      x[1] = x[1] * d4.y + w * k4.y;
      x[2] = x[2] * d4.z + w * k4.z;
      x[3] = x[3] * d4.w + w * k4.w;
      p += x[0] * q4.x + x[1] * q4.y + x[2] * q4.z + x[3] * q4.w;
      xs[t][kt] = x;
    }
    p = cross_row_sum(p);
    if (a.o && lg == 0) a.o[item * V + 16 * vt + lr] = p;
    float* dst = a.S + item * V * K + (size_t)(vt * MT) * 256 + 4 * lane;
#pragma unroll
    for (int kt = 0; kt < MT; ++kt)
      st_nt(reinterpret_cast<float4*>(dst + 256 * kt), make_float4(xs[t][kt][0], xs[t][kt][1], xs[t][kt][2], xs[t][kt][3]));
  }
}

}  // namespace skssm

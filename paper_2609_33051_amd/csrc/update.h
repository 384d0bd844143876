// Flush step of SketchSSM (Algorithm 1, t = W; Sec. 4.1, per-window sketch)
// and the initial sketch: one read and one write of the full state.
//
// With n ring slots plus the current token (nt = n + 1 tokens) and the
// window-local cumulative log decay g (g_n of the last token):
//   L[s]   = exp(g_n - g_s) . k_s                  (left factors l_s(W), Appendix C.1)
//   pi_s   = beta_s (e^{g_s} . k_s - sum_{j<s} b_{s,j} pi_j)           (eq. wy)
//   w_s    = u_s - X_0 pi_s                         (true write vectors; Mamba-2: beta_s v_s)
//   X_W    = X_0 Diag(e^{g_n}) + sum_s w_s L[s]^T   (eq. update in rank-nt form)
//   o_W    = X_W q_W,   U = X_W Omega
// where X = S^T is the stored [V][K] state.  The two contractions over the
// state (X_0 Pi^T, K-deep; the rank-nt update, W-deep) and the sketch
// projection X_W Omega run on fp32 matrix cores (v_mfma_f32_16x16x4f32).
//
// Mapping: one workgroup (4 waves) per (request, head) item; each wave owns
// 16-column value tiles of X^T (K rows x 16 values).  The state tile is held
// in MFMA accumulator layout: lane l holds X[v0 + l%16][16 kt + 4 (l/16) + i],
// i = 0..3, a 16-byte contiguous piece of a state row.  Because the
// contraction index of the K-deep products may be visited in any order, the
// same registers serve as the B operand of X_0 Pi^T and X_W Omega (step i of
// k-tile kt contracts over k = 16 kt + 4 g + i for lane group g) and as the
// accumulator of the rank-nt update, so the state never leaves registers
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

template <int KIND, int K, int V, int R, int WMAX, typename IO>
__global__ __launch_bounds__(256) void update_kernel(const UpdateArgs a) {
  constexpr bool ERASE = KIND != MAMBA2;
  constexpr bool CHAN = KIND == KDA;
  constexpr int MT = K / 16;          // k tiles
  constexpr int VT = V / 16;          // value tiles
  constexpr int VTW = (VT + 3) / 4;   // value tiles per wave
  constexpr int SP = WMAX;            // slot rows (16 or 32)
  constexpr int ST = SP / 16;         // slot tiles
  constexpr int RT = (R + 15) / 16;   // sketch tiles
  constexpr int LP = K + 4;           // LDS pitches chosen so that the 4 lane
  constexpr int PP = SP + 4;          // groups of an operand read land in
  constexpr int UP = V + 4;           // different banks
  constexpr int KW = (K + 63) / 64;   // waves that carry channel work

  __shared__ __align__(16) float Ls[SP * LP];                 // L[s][k]
  __shared__ __align__(16) float PiT[ERASE ? K * PP : 4];     // Pi^T[k][s]
  __shared__ __align__(16) float Us[SP * UP];                 // w-vector source: u_s[v]
  __shared__ float Bs[ERASE ? SP * SP : 1];                   // b_{s,j}
  __shared__ float bpart[ERASE ? KW * SP : 1];                // partial sums of b_{n,j}
  __shared__ __align__(16) float qs[K];
  __shared__ __align__(16) float ds[K];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lg = lane >> 4;
  const int H = a.H, W = a.W, n = a.n;
  const size_t item = blockIdx.x;
  const int h = (int)(item % (size_t)H);
  const bool flush = a.nt > 0;
  const size_t NI = (size_t)a.B * H;  // slot s of item: ring field + (s * NI + item) * width

  // ---- the single read of the state: issue every tile load first
  floatx4 xs[VTW][MT];
#pragma unroll
  for (int t = 0; t < VTW; ++t) {
    const int vt = wave + 4 * t;
    if (vt < VT) {
      const float* src = a.S + (item * V + 16 * vt + lr) * K + 4 * lg;
#pragma unroll
      for (int kt = 0; kt < MT; ++kt) {
        const float4 x = *reinterpret_cast<const float4*>(src + 16 * kt);
        xs[t][kt] = floatx4{x.x, x.y, x.z, x.w};
      }
    }
  }

  if (flush) {
    // ---- channel work: thread tid owns channel k = tid.  Slots 0..n of the
    // ring hold the window's tokens (slot n: the current one).
    float gk[SP], kc[SP], gn = 0.f;
    if (tid < K) {
      const int kk = tid;
      float acc = 0.f;  // running cumulative log decay (scalar decay)
#pragma unroll
      for (int s = 0; s < SP; ++s) {
        gk[s] = 0.f;
        kc[s] = 0.f;
        if (s <= n) {
          const size_t si = (size_t)s * NI + item;
          kc[s] = load1<IO>(static_cast<const IO*>(a.rk) + si * K + kk);
          if constexpr (CHAN) {
            gk[s] = (s < n) ? a.rg[si * K + kk] : ((n > 0 ? a.rg[(si - NI) * K + kk] : 0.f) + a.rla[si * K + kk]);
          } else {
            acc += a.rla[si];
            gk[s] = acc;
          }
          if (s == n) gn = gk[s];
        }
      }
      qs[kk] = load1<IO>(static_cast<const IO*>(a.q) + item * K + kk);
      ds[kk] = fast_exp(gn);
      const float kn = load1<IO>(static_cast<const IO*>(a.rk) + ((size_t)n * NI + item) * K + kk);
#pragma unroll
      for (int s = 0; s < SP; ++s) {
        const float l = (s <= n) ? fast_exp(gn - gk[s]) * kc[s] : 0.f;
        Ls[s * LP + kk] = l;
        if constexpr (ERASE) {
          // b_{n,s} = <exp(g_n - g_s) . k_s, k_n>: reduce over the channels of this wave
          if (s < n) {
            const float bsum = wave_sum(l * kn);
            if (lane == 0) bpart[wave * SP + s] = bsum;
          }
        }
      }
    }
    // ---- value-side staging: u_s (Mamba-2: beta_s v_s), b_{s,j}
    for (int idx = tid; idx < SP * V; idx += 256) {
      const int s = idx / V, v = idx % V;
      float val = 0.f;
      const size_t si = (size_t)s * NI + item;
      if constexpr (ERASE) {
        if (s < n) val = a.ru[si * V + v];
      } else {
        if (s <= n) val = a.rbeta[si] * load1<IO>(static_cast<const IO*>(a.rv) + si * V + v);
      }
      Us[s * UP + v] = val;
    }
    if constexpr (ERASE) {
      for (int idx = tid; idx < SP * SP; idx += 256) {
        const int s = idx / SP, j = idx % SP;
        Bs[idx] = (s < n && j < s) ? a.rb[((size_t)s * NI + item) * W + j] : 0.f;
      }
    }
    __syncthreads();

    if constexpr (ERASE) {
      const size_t cur = (size_t)n * NI + item;
      const float beta_n = a.rbeta[cur];
      // pseudo-value of the current token from the per-wave partial sums of b_{n,j}
      if (tid < V) {
        const int v = tid;
        float acc = load1<IO>(static_cast<const IO*>(a.rv) + cur * V + v);
#pragma unroll
        for (int j = 0; j < SP; ++j) {
          if (j < n) {
            float bj = 0.f;
#pragma unroll
            for (int w = 0; w < KW; ++w) bj += bpart[w * SP + j];
            acc -= bj * Us[j * UP + v];
          }
        }
        Us[n * UP + v] = beta_n * acc;   // u_n
      }
      if (tid < K) {
        // erase factors pi_s of this channel, s = 0..n (forward substitution)
        const int kk = tid;
        float pi[SP];
#pragma unroll
        for (int s = 0; s < SP; ++s) {
          pi[s] = 0.f;
          if (s <= n) {
            const float bet = a.rbeta[(size_t)s * NI + item];
            float acc = fast_exp(gk[s]) * kc[s];
#pragma unroll
            for (int j = 0; j < s; ++j) {
              float bj;
              if (s < n) {
                bj = Bs[s * SP + j];
              } else {
                bj = 0.f;
#pragma unroll
                for (int w = 0; w < KW; ++w) bj += bpart[w * SP + j];
              }
              acc -= bj * pi[j];
            }
            pi[s] = bet * acc;
          }
          PiT[kk * PP + s] = pi[s];
        }
      }
      __syncthreads();
    }
  }

  // ---- matrix-core phase, one 16-column value tile at a time
#pragma unroll
  for (int t = 0; t < VTW; ++t) {
    const int vt = wave + 4 * t;
    if (vt >= VT) continue;
    const int v = 16 * vt + lr;
    if (flush) {
      // w-vectors W^T[s][v] = u_s[v] - (Pi X_0^T)[s][v]   (C layout: s = 16 st + 4 lg + i)
      floatx4 wv[ST];
#pragma unroll
      for (int st = 0; st < ST; ++st) {
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
        if constexpr (ERASE) {
#pragma unroll
          for (int kt = 0; kt < MT; ++kt)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              acc = mfma4(PiT[(16 * kt + 4 * lg + i) * PP + 16 * st + lr], xs[t][kt][i], acc);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) wv[st][i] = Us[(16 * st + 4 * lg + i) * UP + v] - acc[i];
      }
      // X_W^T = Diag(e^{g_n}) X_0^T + L^T W^T   (accumulates onto the decayed state)
#pragma unroll
      for (int kt = 0; kt < MT; ++kt) {
        floatx4 acc;
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = xs[t][kt][i] * ds[16 * kt + 4 * lg + i];
#pragma unroll
        for (int st = 0; st < ST; ++st)
#pragma unroll
          for (int i = 0; i < 4; ++i) acc = mfma4(Ls[(16 * st + 4 * lg + i) * LP + 16 * kt + lr], wv[st][i], acc);
        xs[t][kt] = acc;
      }
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
    }
    // sketch U^T = Omega^T X^T  (rows j = 16 jt + 4 lg + i of the C layout)
    if constexpr (R > 0) {
      if (a.U) {
        const float* om = a.omega + (size_t)h * K * R;
#pragma unroll
        for (int jt = 0; jt < RT; ++jt) {
          const int jj = 16 * jt + lr;
          floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kt = 0; kt < MT; ++kt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float w = (jj < R) ? om[(16 * kt + 4 * lg + i) * R + jj] : 0.f;
              acc = mfma4(w, xs[t][kt][i], acc);
            }
          // 4-column panel 4 jt + lg of U[B][H][R/4][V][4]
          if (16 * jt + 4 * lg < R)
            reinterpret_cast<float4*>(a.U + item * (size_t)V * R)[(4 * jt + lg) * V + v] =
                make_float4(acc[0], acc[1], acc[2], acc[3]);
        }
      }
    }
    if (flush) {
      float* dst = a.S + (item * V + v) * K + 4 * lg;
#pragma unroll
      for (int kt = 0; kt < MT; ++kt)
        *reinterpret_cast<float4*>(dst + 16 * kt) = make_float4(xs[t][kt][0], xs[t][kt][1], xs[t][kt][2], xs[t][kt][3]);
    }
  }
}

}  // namespace skssm

// Flush step of SketchSSM (Algorithm 1, t = W; Sec. 4.1, per-window sketch)
// and the initial sketch: one read and one write of the full state.
//
// With the window's tokens in ring slots 0..n (slot n: the current token),
// cumulative log decays g_s and c_s = exp(g_n - g_s):
//   L[s]   = exp(g_n - g_s) . k_s                  (left factors l_s(W), Appendix C.1)
//   pi_s   = beta_s (e^{g_s} . k_s - sum_{j<s} b_{s,j} pi_j)           (eq. wy)
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
// i = 0..3, a 16-byte contiguous piece of a state row.  Because the
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

template <int KIND, int K, int V, int R, int WMAX, typename IO>
__global__ __launch_bounds__(256) void update_kernel(const UpdateArgs a) {
  constexpr bool ERASE = KIND != MAMBA2;
  constexpr bool CHAN = KIND == KDA;
  constexpr int MT = K / 16;          // k tiles
  constexpr int VT = V / 16;          // value tiles
  constexpr int VTW = (VT + 3) / 4;   // value tiles per wave
  constexpr int SP = WMAX;            // slot rows (16 or 32)
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
  __shared__ __align__(16) float Us[SP * UP];                 // c_s beta_s v_s (Mamba-2) or u_s
  __shared__ float Bs[ERASE ? SP * SP : 1];                   // b_{s,j}
  __shared__ float bpart[ERASE ? KW * SP : 1];                // partial sums of b_{n,j}
  __shared__ __align__(16) float qs[K];
  __shared__ __align__(16) float ds[CHAN ? K : 4];            // e^{g_n} per channel (KDA)
  __shared__ float csc[SP];                                   // c_s (scalar decay)

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lg = lane >> 4;   // MFMA lane coordinates
  const int row = lg, col = lr;               // row-layout coordinates (same lanes)
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

  float egn = 1.f;  // e^{g_n} (scalar decay)
  if (flush) {
    // ---- per-slot scalars, uniform in every wave: beta_s and (scalar decay)
    // the cumulative log decay g_s, summed in slot order
    float bsv[SP], gsv[SP];
    {
      float acc = 0.f;
#pragma unroll
      for (int s = 0; s < SP; ++s) {
        bsv[s] = 0.f;
        gsv[s] = 0.f;
        if (s <= n) {
          const size_t si = (size_t)s * NI + item;
          bsv[s] = a.rbeta[si];
          if constexpr (!CHAN) {
            acc += a.rla[si];
            gsv[s] = acc;
          }
        }
      }
    }
    float gn = 0.f, bn = 0.f;
#pragma unroll
    for (int s = 0; s < SP; ++s)
      if (s == n) {
        gn = gsv[s];
        bn = bsv[s];
      }
    if constexpr (!CHAN) egn = fast_exp(gn);
    // KDA: per-channel cumulative log decays, thread tid owns channel tid
    float gk[CHAN ? SP : 1];
    if constexpr (CHAN) {
      if (tid < K) {
#pragma unroll
        for (int s = 0; s < SP; ++s) {
          gk[s] = 0.f;
          if (s <= n) {
            const size_t si = (size_t)s * NI + item;
            gk[s] = (s < n) ? a.rg[si * K + tid] : ((n > 0 ? a.rg[(si - NI) * K + tid] : 0.f) + a.rla[si * K + tid]);
          }
        }
      }
    }

    // ---- stage the window with wide loads: row r of wave w holds slot 4 gi + r
#pragma unroll
    for (int gq = 0; gq < NG / 4; ++gq) {
      const int gi = wave + 4 * gq;  // slot group of this wave (wave-uniform)
      const int s = 4 * gi + row;
      const size_t si = (size_t)s * NI + item;
      float ksv[KPL], vsv[VR];
#pragma unroll
      for (int m = 0; m < KPL; ++m) ksv[m] = 0.f;
#pragma unroll
      for (int m = 0; m < VR; ++m) vsv[m] = 0.f;
      if (s <= n) {
        Raw<IO, KPL> kr;
        kr.load(static_cast<const IO*>(a.rk) + si * K + col * KPL);
#pragma unroll
        for (int m = 0; m < KPL; ++m) ksv[m] = kr.get(m);
        if (ERASE && s < n) {
          Vec<VR> ur;
          ur.load(a.ru + si * V + col * VR);
#pragma unroll
          for (int m = 0; m < VR; ++m) vsv[m] = ur.e[m];
        } else {
          // raw value: Mamba-2 scales it into c_s beta_s v_s; GDN/KDA keep v_n
          // in row n until u_n is formed
          Raw<IO, VR> vr;
          vr.load(static_cast<const IO*>(a.rv) + si * V + col * VR);
          float sc = 1.f;
          if constexpr (!ERASE) {
            // select this row's slot from the wave-uniform tables (compile-time indices only)
            float gs = 0.f, bs = 0.f;
#pragma unroll
            for (int j = 0; j < SP; ++j)
              if (j == s) {
                gs = gsv[j];
                bs = bsv[j];
              }
            sc = bs * fast_exp(gn - gs);
          }
#pragma unroll
          for (int m = 0; m < VR; ++m) vsv[m] = sc * vr.get(m);
        }
      }
#pragma unroll
      for (int m = 0; m < KPL; m += 4)
        *reinterpret_cast<float4*>(&Ls[s * LP + col * KPL + m]) = make_float4(ksv[m], ksv[m + 1], ksv[m + 2], ksv[m + 3]);
#pragma unroll
      for (int m = 0; m < VR; m += 4)
        *reinterpret_cast<float4*>(&Us[s * UP + col * VR + m]) = make_float4(vsv[m], vsv[m + 1], vsv[m + 2], vsv[m + 3]);
    }
    if (tid < K) qs[tid] = load1<IO>(static_cast<const IO*>(a.q) + item * K + tid);
    if constexpr (!CHAN) {
      if (tid < SP) {
        float c = 0.f;
#pragma unroll
        for (int j = 0; j < SP; ++j)
          if (j == tid && j <= n) c = fast_exp(gn - gsv[j]);
        csc[tid] = c;
      }
    }
    if constexpr (ERASE) {
      for (int idx = tid; idx < SP * SP; idx += 256) {
        const int s = idx / SP, j = idx % SP;
        Bs[idx] = (s < n && j < s) ? a.rb[((size_t)s * NI + item) * W + j] : 0.f;
      }
    }
    __syncthreads();

    if constexpr (ERASE) {
      // ---- channel work: thread tid owns channel k = tid.  Ls holds raw keys.
      float pi[SP], kn = 0.f;
      if (tid < K) {
        const int kk = tid;
        kn = Ls[n * LP + kk];
        float gnk = gn;
        if constexpr (CHAN) {
#pragma unroll
          for (int s = 0; s < SP; ++s)
            if (s == n) gnk = gk[s];
        }
        // erase factors pi_s, s < n, by forward substitution over the stored couplings
#pragma unroll
        for (int s = 0; s < SP; ++s) {
          pi[s] = 0.f;
          if (s < n) {
            float acc = fast_exp(CHAN ? gk[s] : gsv[s]) * Ls[s * LP + kk];
#pragma unroll
            for (int j = 0; j < s; ++j) acc -= Bs[s * SP + j] * pi[j];
            pi[s] = bsv[s] * acc;
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
      }
      __syncthreads();
      // ---- the current token: u_n and pi_n need b_{n,j} from every wave
      if (tid < V) {
        const int v = tid;
        float acc = Us[n * UP + v];  // raw v_n
#pragma unroll
        for (int j = 0; j < SP; ++j) {
          if (j < n) {
            float bj = 0.f;
#pragma unroll
            for (int w = 0; w < KW; ++w) bj += bpart[w * SP + j];
            acc -= bj * Us[j * UP + v];
          }
        }
        Us[n * UP + v] = bn * acc;  // u_n
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
      // value-side factors of the rank update, C layout: slot s = 16 st + 4 lg + i
      floatx4 wv[ST];
#pragma unroll
      for (int st = 0; st < ST; ++st) {
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
        if constexpr (ERASE) {
          // w_s = u_s - (Pi X_0^T)[s]; four independent accumulation chains
          floatx4 pc[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) pc[i] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kt = 0; kt < MT; ++kt)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              pc[i] = mfma4(PiT[(16 * kt + 4 * lg + i) * PP + 16 * st + lr], xs[t][kt][i], pc[i]);
          acc = (pc[0] + pc[1]) + (pc[2] + pc[3]);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int s = 16 * st + 4 * lg + i;
          float w = Us[s * UP + v] - acc[i];
          if constexpr (ERASE && !CHAN) w *= csc[s];  // GDN: c_s w_s
          wv[st][i] = w;
        }
      }
      // X_W^T = Diag(e^{g_n}) X_0^T + (keys or L)^T W^T, accumulated onto the decayed state
#pragma unroll
      for (int kt = 0; kt < MT; ++kt) {
        floatx4 acc;
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = xs[t][kt][i] * (CHAN ? ds[16 * kt + 4 * lg + i] : egn);
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
          // four independent accumulation chains over the K-deep contraction
          floatx4 uc[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) uc[i] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kt = 0; kt < MT; ++kt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float w = (jj < R) ? om[(16 * kt + 4 * lg + i) * R + jj] : 0.f;
              uc[i] = mfma4(w, xs[t][kt][i], uc[i]);
            }
          const floatx4 acc = (uc[0] + uc[1]) + (uc[2] + uc[3]);
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

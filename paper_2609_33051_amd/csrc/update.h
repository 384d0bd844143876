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

template <int KIND, int K, int V, int R, int WMAX, typename IO, typename SK>
__global__ __launch_bounds__(256, 3) void update_kernel(const UpdateArgs a) {
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
  // slot s of an item: raw ring fields at (item * W + s) * width, derived
  // fields at (s * B*H + item) * width
  const size_t NI = (size_t)a.B * H;

  // Omega of this head goes to LDS (rows padded to whole 16-column tiles plus
  // four words, so the four lane groups of an operand read hit different banks)
  // when it is small; the full-rank case reads it from global memory.
  constexpr bool OM_LDS = R > 0 && R <= 32;
  constexpr int OPJ = 16 * RT + 4;
  constexpr int OQ = OM_LDS ? (K * R / 4 + 255) / 256 : 1;  // float4 of Omega per thread
  __shared__ __align__(16) float OmL[OM_LDS ? K * OPJ : 4];
  const bool want_U = R > 0 && a.U != nullptr;

  // ---- every small load first (window, query, couplings, Omega), then the
  // state: the staged values reach LDS while the state read is still in flight
  float egn = 1.f, gn = 0.f, bn = 0.f;  // e^{g_n} (scalar decay), g_n, beta_n
  float bsv[SP], gsv[SP];               // beta_s and (scalar decay) g_s, wave-uniform
  float gk[CHAN ? SP : 1];              // KDA: g_s of channel tid
  Raw<IO, KPL> kr[NG / 4];              // ring keys, row layout (slot 4 (wave + 4 gq) + row)
  Vec<ERASE ? VR : 1> ur[NG / 4];       // GDN/KDA: pseudo-values u_s (s < n)
  Raw<IO, VR> vr[NG / 4];               // raw values (Mamba-2: all slots; GDN/KDA: slot n)
  float qv = 0.f;
  constexpr int BQ = ERASE ? (SP * SP + 255) / 256 : 1;
  float bv[BQ];
  Vec<4> omv[OQ];
  if (flush) {
    {
      float acc = 0.f;
#pragma unroll
      for (int s = 0; s < SP; ++s) {
        bsv[s] = 0.f;
        gsv[s] = 0.f;
        if (s <= n) {
          const size_t si = item * W + s;
          bsv[s] = a.rbeta[si];
          if constexpr (!CHAN) {
            acc += a.rla[si];
            gsv[s] = acc;
          }
        }
      }
    }
#pragma unroll
    for (int s = 0; s < SP; ++s)
      if (s == n) {
        gn = gsv[s];
        bn = bsv[s];
      }
    if constexpr (!CHAN) egn = fast_exp(gn);
    if constexpr (CHAN) {
      if (tid < K) {
#pragma unroll
        for (int s = 0; s < SP; ++s) {
          gk[s] = 0.f;
          if (s <= n) {
            const size_t si = item * W + s;
            const size_t sd = (size_t)s * NI + item;
            gk[s] = (s < n) ? a.rg[sd * K + tid] : ((n > 0 ? a.rg[(sd - NI) * K + tid] : 0.f) + a.rla[si * K + tid]);
          }
        }
      }
    }
#pragma unroll
    for (int gq = 0; gq < NG / 4; ++gq) {
      const int s = 4 * (wave + 4 * gq) + row;
      const size_t si = item * W + s;
      if (s <= n) {
        kr[gq].load(static_cast<const IO*>(a.rk) + si * K + col * KPL);
        if (ERASE && s < n) {
          if constexpr (ERASE) ur[gq].load(a.ru + ((size_t)s * NI + item) * V + col * VR);
        } else {
          vr[gq].load(static_cast<const IO*>(a.rv) + si * V + col * VR);
        }
      }
    }
    if (tid < K) qv = load1<IO>(static_cast<const IO*>(a.q) + item * K + tid);
    if constexpr (ERASE) {
#pragma unroll
      for (int c = 0; c < BQ; ++c) {
        const int idx = tid + 256 * c;
        const int s = idx / SP, j = idx % SP;
        bv[c] = (idx < SP * SP && s < n && j < s) ? a.rb[((size_t)s * NI + item) * W + j] : 0.f;
      }
    }
  }
  if constexpr (OM_LDS) {
    if (want_U) {
#pragma unroll
      for (int c = 0; c < OQ; ++c) {
        const int i = tid + 256 * c;
        if (i < K * R / 4) omv[c].load(a.omega + (size_t)h * K * R + 4 * i);
      }
    }
  }

  // ---- the single read of the state
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
  compiler_fence();

  // ---- staged values into LDS
  if constexpr (OM_LDS) {
    if (want_U) {
#pragma unroll
      for (int c = 0; c < OQ; ++c) {
        const int i = tid + 256 * c;
        if (i < K * R / 4)
          omv[c].store(&OmL[(i / (R / 4)) * OPJ + 4 * (i % (R / 4))]);
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
        if (ERASE && s < n) {
          if constexpr (ERASE) {
#pragma unroll
            for (int m = 0; m < VR; ++m) vsv[m] = ur[gq].e[m];
          }
        } else {
          // raw value: Mamba-2 scales it into c_s beta_s v_s; GDN/KDA keep v_n
          // in row n until u_n is formed
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
          for (int m = 0; m < VR; ++m) vsv[m] = sc * vr[gq].get(m);
        }
      }
#pragma unroll
      for (int m = 0; m < KPL; m += 4)
        *reinterpret_cast<float4*>(&Ls[s * LP + col * KPL + m]) = make_float4(ksv[m], ksv[m + 1], ksv[m + 2], ksv[m + 3]);
#pragma unroll
      for (int m = 0; m < VR; m += 4)
        *reinterpret_cast<float4*>(&Us[s * UP + col * VR + m]) = make_float4(vsv[m], vsv[m + 1], vsv[m + 2], vsv[m + 3]);
    }
    if (tid < K) qs[tid] = qv;
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
#pragma unroll
      for (int c = 0; c < BQ; ++c) {
        const int idx = tid + 256 * c;
        if (idx < SP * SP) Bs[idx] = bv[c];
      }
    }
  }
  lds_barrier();

  if (flush) {
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
      lds_barrier();
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
      lds_barrier();
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
      if (want_U) {
        const float* om = a.omega + (size_t)h * K * R;
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
          // columns 16 jt + 4 lg .. +3 of value v; panels of 16 bytes per value:
          // fp32 U[B][H][R/4][V][4], bf16 U[B][H][R/8][V][8]
          if (16 * jt + 4 * lg < R) {
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

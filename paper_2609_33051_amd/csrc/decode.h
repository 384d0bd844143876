// Non-flush read of SketchSSM (Algorithm 1, t < W) and the exact
// full-state-read baseline, both appending the token to the replay buffer.
//
// Per (request, head) item, with t = n + 1 tokens in the window:
//   g_t      = g_{t-1} + log alpha_t                       (cumulative log decay)
//   a_{t,s}  = <exp(g_t - g_s) . k_s, q_t>,  s <= t       (Appendix C.2, key reuse)
//   b_{t,j}  = <exp(g_t - g_j) . k_j, k_t>,  j <  t       (erase couplings)
//   u_t      = beta_t (v_t - sum_j b_{t,j} u_j)           (pseudo-values; Mamba-2: beta_t v_t)
//   f_t      = beta_t (C (e^{g_t} . k_t) - sum_j b_{t,j} f_j)      (eq. wyread)
//   c_t      = C (e^{g_t} . q_t) - sum_{s<=t} a_{t,s} f_s          (eq. app-projected-query)
//   o_t      = U c_t + sum_{s<=t} a_{t,s} u_s              (eq. equantion-sketch + buffer term)
// The exact baseline replaces f by the full erase factors pi (eq. wy) and
// U c_t by S_0^T q~_t with q~_t = e^{g_t} . q_t - sum_s a_{t,s} pi_s.
//
// Mapping: one wave per item.  Keys, decays and erase factors of the ring
// are read in the row layout (4 slots per load, 16-lane DPP dot products);
// the sketch U, the values / pseudo-values and the output use the value
// layout.  No matrix cores: every contraction here is a matrix-vector product.
#pragma once

#include "args.h"
#include "device.h"

namespace skssm {

template <int KIND, int K, int V, int WMAX, typename IO>
struct RowLoads {
  static constexpr bool ERASE = KIND != MAMBA2;
  static constexpr bool CHAN = KIND == KDA;
  static constexpr int KPL = K / 16;
  static constexpr int VPL = V / 64;
  static constexpr int NG = WMAX / 4;
  static constexpr int GD = CHAN ? KPL : 1;

  Raw<IO, KPL> q_raw, k_raw;  // current token, row layout (same in every row)
  Raw<IO, VPL> v_raw;         // current token, value layout
  float beta_t;
  float la[GD];               // log alpha_t
  float gprev[GD];            // g_{t-1}
  Raw<IO, KPL> ks[NG];        // ring keys of slot 4*gi + row
  float gs[NG][GD];           // ring cumulative log decay of slot 4*gi + row
  float bs[NG];               // ring beta of slot 4*gi + row (Mamba-2)

  __device__ __forceinline__ void load(const DecodeArgs& a, size_t item, int row, int col, int lane) {
    const int n = a.n, W = a.W;
    const size_t slot0 = item * (size_t)W;
    q_raw.load(static_cast<const IO*>(a.q) + item * K + col * KPL);
    k_raw.load(static_cast<const IO*>(a.k) + item * K + col * KPL);
    v_raw.load(static_cast<const IO*>(a.v) + item * V + lane * VPL);
    beta_t = a.beta[item];
    if constexpr (CHAN) {
      Vec<KPL> t;
      t.load(a.logd + item * K + col * KPL);
#pragma unroll
      for (int m = 0; m < KPL; ++m) la[m] = t.e[m];
    } else {
      la[0] = a.logd[item];
    }
#pragma unroll
    for (int m = 0; m < GD; ++m) gprev[m] = 0.f;
    if (n > 0) {
      if constexpr (CHAN) {
        Vec<KPL> t;
        t.load(a.rg + (slot0 + n - 1) * K + col * KPL);
#pragma unroll
        for (int m = 0; m < KPL; ++m) gprev[m] = t.e[m];
      } else {
        gprev[0] = a.rg[slot0 + n - 1];
      }
    }
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) {
      const int s = 4 * gi + row;
      ks[gi].zero();
#pragma unroll
      for (int m = 0; m < GD; ++m) gs[gi][m] = 0.f;
      bs[gi] = 0.f;
      if (4 * gi < n && s < n) {
        ks[gi].load(static_cast<const IO*>(a.rk) + (slot0 + s) * K + col * KPL);
        if constexpr (CHAN) {
          Vec<KPL> t;
          t.load(a.rg + (slot0 + s) * K + col * KPL);
#pragma unroll
          for (int m = 0; m < KPL; ++m) gs[gi][m] = t.e[m];
        } else {
          gs[gi][0] = a.rg[slot0 + s];
        }
        if constexpr (!ERASE) bs[gi] = a.rbeta[slot0 + s];
      }
    }
  }
};

// Dot products of the current query / key with every buffered key.
// Returns, in the row layout, av[gi] = a_{t,s} (Mamba-2: a_{t,s} beta_s) and
// bv[gi] = b_{t,s} for s = 4*gi + row (0 for s >= n), plus at = <k_t, q_t>.
template <class L>
__device__ __forceinline__ void slot_dots(const L& r, int n, int row, const float (&qv)[L::KPL],
                                          const float (&kv)[L::KPL], const float (&gt)[L::GD],
                                          float (&av)[L::NG], float (&bv)[L::NG], float& at) {
  float p = 0.f;
#pragma unroll
  for (int m = 0; m < L::KPL; ++m) p += kv[m] * qv[m];
  at = row_sum16(p);
#pragma unroll
  for (int gi = 0; gi < L::NG; ++gi) {
    float pa = 0.f, pb = 0.f;
    if (4 * gi < n) {
#pragma unroll
      for (int m = 0; m < L::KPL; ++m) {
        float kk = r.ks[gi].get(m);
        if constexpr (L::CHAN) kk *= fast_exp(gt[m] - r.gs[gi][m]);
        pa += kk * qv[m];
        if constexpr (L::ERASE) pb += kk * kv[m];
      }
      pa = row_sum16(pa);
      if constexpr (L::ERASE) pb = row_sum16(pb);
      if constexpr (!L::CHAN) {
        const float e = fast_exp(gt[0] - r.gs[gi][0]);
        pa *= e;
        pb *= e;
      }
      if (4 * gi + row >= n) {
        pa = 0.f;
        pb = 0.f;
      }
      if constexpr (!L::ERASE) pa *= r.bs[gi];
    }
    av[gi] = pa;
    bv[gi] = pb;
  }
}

template <int KIND, int K, int V, int R, int WMAX, typename IO>
__global__ __launch_bounds__(256) void decode_kernel(const DecodeArgs a) {
  using L = RowLoads<KIND, K, V, WMAX, IO>;
  constexpr bool ERASE = L::ERASE, CHAN = L::CHAN;
  constexpr int KPL = L::KPL, VPL = L::VPL, NG = L::NG, GD = L::GD;
  constexpr int RP = (R + 15) / 16;  // sketch components per lane in the row layout
  constexpr int CP = K + 4;          // padded LDS row pitch of C
  constexpr int KQ = K / 4;          // channels each row covers in C x
  constexpr int WS = 2 * K + R;      // per-wave LDS scratch: x_q, x_k, c
  constexpr bool U_PRELOAD = R <= 32;
  constexpr int UR = U_PRELOAD ? R : 1;

  __shared__ __align__(16) float c_lds[R * CP];
  __shared__ __align__(16) float wscr[4 * WS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row = lane >> 4, col = lane & 15;
  const int H = a.H, W = a.W, n = a.n;
  const int h = blockIdx.x % H;
  const int b = (blockIdx.x / H) * 4 + wave;
  const bool valid = b < a.B;
  const size_t item = (size_t)(valid ? b : 0) * H + h;
  const size_t slot0 = item * (size_t)W;

  // ---- issue every global load of this item first
  L r;
  float fs[NG][RP];                  // ring f of slot 4*gi + row, component col + 16p
  float us[ERASE ? WMAX : 1][VPL];   // ring u (value layout)
  Raw<IO, VPL> vs[ERASE ? 1 : WMAX]; // ring v (value layout)
  float Ur[VPL][UR];
  if (valid) {
    r.load(a, item, row, col, lane);
    if constexpr (ERASE) {
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) {
        const int s = 4 * gi + row;
#pragma unroll
        for (int p = 0; p < RP; ++p) {
          const int j = col + 16 * p;
          fs[gi][p] = (4 * gi < n && s < n && j < R) ? a.rf[(slot0 + s) * R + j] : 0.f;
        }
      }
#pragma unroll
      for (int s = 0; s < WMAX; ++s) {
        if (s < n) {
          Vec<VPL> t;
          t.load(a.ru + (slot0 + s) * V + lane * VPL);
#pragma unroll
          for (int vv = 0; vv < VPL; ++vv) us[s][vv] = t.e[vv];
        } else {
#pragma unroll
          for (int vv = 0; vv < VPL; ++vv) us[s][vv] = 0.f;
        }
      }
    } else {
#pragma unroll
      for (int s = 0; s < WMAX; ++s) {
        vs[s].zero();
        if (s < n) vs[s].load(static_cast<const IO*>(a.rv) + (slot0 + s) * V + lane * VPL);
      }
    }
    if constexpr (U_PRELOAD) {
#pragma unroll
      for (int vv = 0; vv < VPL; ++vv) {
        Vec<R> t;
        t.load(a.U + (item * V + lane * VPL + vv) * R);
#pragma unroll
        for (int j = 0; j < R; ++j) Ur[vv][j] = t.e[j];
      }
    }
  }

  // ---- stage this head's coefficient map C (R x K) in LDS
  {
    const float4* src = reinterpret_cast<const float4*>(a.coef + (size_t)h * R * K);
    for (int i = tid; i < R * K / 4; i += 256) {
      const int j = (4 * i) / K, kk = (4 * i) % K;
      *reinterpret_cast<float4*>(&c_lds[j * CP + kk]) = src[i];
    }
  }
  __syncthreads();
  if (!valid) return;

  float* xq_l = wscr + wave * WS;
  float* xk_l = xq_l + K;
  float* c_l = xq_l + 2 * K;

  float qv[KPL], kv[KPL], gt[GD];
#pragma unroll
  for (int m = 0; m < KPL; ++m) {
    qv[m] = r.q_raw.get(m);
    kv[m] = r.k_raw.get(m);
  }
#pragma unroll
  for (int m = 0; m < GD; ++m) gt[m] = r.gprev[m] + r.la[m];

  float av[NG], bv[NG], at;
  slot_dots(r, n, row, qv, kv, gt, av, bv, at);

  // wave-uniform copies of a_{t,s} (and b_{t,s}) for the value-layout sums
  float a_u[WMAX], b_u[ERASE ? WMAX : 1];
#pragma unroll
  for (int gi = 0; gi < NG; ++gi)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      a_u[4 * gi + r4] = (4 * gi < n) ? lane_bcast(av[gi], 16 * r4) : 0.f;
      if constexpr (ERASE) b_u[4 * gi + r4] = (4 * gi < n) ? lane_bcast(bv[gi], 16 * r4) : 0.f;
    }

  // ---- pseudo-value of the current token (value layout)
  float ut[VPL];
#pragma unroll
  for (int vv = 0; vv < VPL; ++vv) {
    float acc = r.v_raw.get(vv);
    if constexpr (ERASE) {
#pragma unroll
      for (int s = 0; s < WMAX; ++s)
        if (s < n) acc -= b_u[s] * us[s][vv];
    }
    ut[vv] = r.beta_t * acc;
  }

  // ---- C (e^{g_t} . q_t) and C (e^{g_t} . k_t): each row covers K/4 channels
  {
    float xq[KPL], xk[KPL];
#pragma unroll
    for (int m = 0; m < KPL; ++m) {
      const float e = CHAN ? fast_exp(gt[m]) : 1.f;
      xq[m] = e * qv[m];
      xk[m] = e * kv[m];
    }
    if (row == 0) {
#pragma unroll
      for (int m = 0; m < KPL; ++m) {
        xq_l[col * KPL + m] = xq[m];
        if constexpr (ERASE) xk_l[col * KPL + m] = xk[m];
      }
    }
  }
  wave_lds_sync();
  const float eg = CHAN ? 1.f : fast_exp(gt[0]);
  float cfin[RP], ft[RP];
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    const int j = col + 16 * p;
    float sq = 0.f, sk = 0.f;
    if (j < R) {
      const float* cr = c_lds + j * CP + row * KQ;
      const float* xqr = xq_l + row * KQ;
      const float* xkr = xk_l + row * KQ;
#pragma unroll
      for (int m = 0; m < KQ; m += 4) {
        const float4 cc = *reinterpret_cast<const float4*>(cr + m);
        const float4 xx = *reinterpret_cast<const float4*>(xqr + m);
        sq += cc.x * xx.x + cc.y * xx.y + cc.z * xx.z + cc.w * xx.w;
        if constexpr (ERASE) {
          const float4 yy = *reinterpret_cast<const float4*>(xkr + m);
          sk += cc.x * yy.x + cc.y * yy.y + cc.z * yy.z + cc.w * yy.w;
        }
      }
    }
    sq = cross_row_sum(sq);
    if constexpr (ERASE) {
      sk = cross_row_sum(sk);
      float sb = 0.f, sa = 0.f;
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) {
        sb += bv[gi] * fs[gi][p];
        sa += av[gi] * fs[gi][p];
      }
      sb = cross_row_sum(sb);
      sa = cross_row_sum(sa);
      ft[p] = r.beta_t * (eg * sk - sb);
      cfin[p] = eg * sq - sa - at * ft[p];
    } else {
      ft[p] = 0.f;
      cfin[p] = eg * sq;
    }
  }
  if (row == 0) {
#pragma unroll
    for (int p = 0; p < RP; ++p)
      if (col + 16 * p < R) c_l[col + 16 * p] = cfin[p];
  }
  wave_lds_sync();

  // ---- o = U c + sum_s a_{t,s} u_s  (value layout)
  float ov[VPL];
#pragma unroll
  for (int vv = 0; vv < VPL; ++vv) {
    float acc = 0.f;
    if constexpr (U_PRELOAD) {
#pragma unroll
      for (int j = 0; j < R; j += 4) {
        const float4 c4 = *reinterpret_cast<const float4*>(c_l + j);
        acc += Ur[vv][j] * c4.x + Ur[vv][j + 1] * c4.y + Ur[vv][j + 2] * c4.z + Ur[vv][j + 3] * c4.w;
      }
    } else {
      const float* up = a.U + (item * V + lane * VPL + vv) * R;
#pragma unroll 4
      for (int j = 0; j < R; j += 4) {
        const float4 u4 = *reinterpret_cast<const float4*>(up + j);
        const float4 c4 = *reinterpret_cast<const float4*>(c_l + j);
        acc += u4.x * c4.x + u4.y * c4.y + u4.z * c4.z + u4.w * c4.w;
      }
    }
    if constexpr (ERASE) {
#pragma unroll
      for (int s = 0; s < WMAX; ++s)
        if (s < n) acc += a_u[s] * us[s][vv];
      acc += at * ut[vv];
    } else {
#pragma unroll
      for (int s = 0; s < WMAX; ++s)
        if (s < n) acc += a_u[s] * vs[s].get(vv);
      acc += at * ut[vv];
    }
    ov[vv] = acc;
  }
  {
    Vec<VPL> t;
#pragma unroll
    for (int vv = 0; vv < VPL; ++vv) t.e[vv] = ov[vv];
    t.store(a.o + item * V + lane * VPL);
  }

  // ---- append the token at ring slot n
  const size_t sl = slot0 + n;
  if (row == 0) {
    r.k_raw.store(static_cast<IO*>(a.rk) + sl * K + col * KPL);
    if constexpr (CHAN) {
      Vec<KPL> t;
#pragma unroll
      for (int m = 0; m < KPL; ++m) t.e[m] = gt[m];
      t.store(a.rg + sl * K + col * KPL);
    }
  }
  if (lane == 0) {
    if constexpr (!CHAN) a.rg[sl] = gt[0];
    a.rbeta[sl] = r.beta_t;
  }
  if constexpr (ERASE) {
    Vec<VPL> t;
#pragma unroll
    for (int vv = 0; vv < VPL; ++vv) t.e[vv] = ut[vv];
    t.store(a.ru + sl * V + lane * VPL);
    if (row == 0) {
#pragma unroll
      for (int p = 0; p < RP; ++p)
        if (col + 16 * p < R) a.rf[sl * R + col + 16 * p] = ft[p];
    }
    if (col == 0) {
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) {
        const int s = 4 * gi + row;
        if (4 * gi < n && s < n) a.rb[sl * W + s] = bv[gi];
      }
    }
  } else {
    r.v_raw.store(static_cast<IO*>(a.rv) + sl * V + lane * VPL);
  }
}

template <int KIND, int K, int V, int WMAX, typename IO>
__global__ __launch_bounds__(256) void full_read_kernel(const DecodeArgs a) {
  using L = RowLoads<KIND, K, V, WMAX, IO>;
  constexpr bool ERASE = L::ERASE, CHAN = L::CHAN;
  constexpr int KPL = L::KPL, VPL = L::VPL, NG = L::NG, GD = L::GD;

  __shared__ __align__(16) float os_lds[4 * V];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row = lane >> 4, col = lane & 15;
  const int W = a.W, n = a.n;
  const size_t n_items = (size_t)a.B * a.H;
  const size_t item = (size_t)blockIdx.x * 4 + wave;
  if (item >= n_items) return;  // wave-uniform; no block barrier in this kernel
  const size_t slot0 = item * (size_t)W;

  L r;
  r.load(a, item, row, col, lane);
  float ps[ERASE ? NG : 1][KPL];     // ring pi of slot 4*gi + row (row layout)
  float us[ERASE ? WMAX : 1][VPL];
  Raw<IO, VPL> vs[ERASE ? 1 : WMAX];
  if constexpr (ERASE) {
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) {
      const int s = 4 * gi + row;
      Vec<KPL> t;
#pragma unroll
      for (int m = 0; m < KPL; ++m) t.e[m] = 0.f;
      if (4 * gi < n && s < n) t.load(a.rpi + (slot0 + s) * K + col * KPL);
#pragma unroll
      for (int m = 0; m < KPL; ++m) ps[gi][m] = t.e[m];
    }
#pragma unroll
    for (int s = 0; s < WMAX; ++s) {
      Vec<VPL> t;
#pragma unroll
      for (int vv = 0; vv < VPL; ++vv) t.e[vv] = 0.f;
      if (s < n) t.load(a.ru + (slot0 + s) * V + lane * VPL);
#pragma unroll
      for (int vv = 0; vv < VPL; ++vv) us[s][vv] = t.e[vv];
    }
  } else {
#pragma unroll
    for (int s = 0; s < WMAX; ++s) {
      vs[s].zero();
      if (s < n) vs[s].load(static_cast<const IO*>(a.rv) + (slot0 + s) * V + lane * VPL);
    }
  }

  float qv[KPL], kv[KPL], gt[GD];
#pragma unroll
  for (int m = 0; m < KPL; ++m) {
    qv[m] = r.q_raw.get(m);
    kv[m] = r.k_raw.get(m);
  }
#pragma unroll
  for (int m = 0; m < GD; ++m) gt[m] = r.gprev[m] + r.la[m];

  float av[NG], bv[NG], at;
  slot_dots(r, n, row, qv, kv, gt, av, bv, at);
  float a_u[WMAX], b_u[ERASE ? WMAX : 1];
#pragma unroll
  for (int gi = 0; gi < NG; ++gi)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      a_u[4 * gi + r4] = (4 * gi < n) ? lane_bcast(av[gi], 16 * r4) : 0.f;
      if constexpr (ERASE) b_u[4 * gi + r4] = (4 * gi < n) ? lane_bcast(bv[gi], 16 * r4) : 0.f;
    }

  // ---- effective query q~_t and erase factor pi_t (row layout, all rows equal)
  float qe[KPL], pit[KPL];
#pragma unroll
  for (int m = 0; m < KPL; ++m) {
    const float e = fast_exp(CHAN ? gt[m] : gt[0]);
    if constexpr (ERASE) {
      float sb = 0.f, sa = 0.f;
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) {
        sb += bv[gi] * ps[gi][m];
        sa += av[gi] * ps[gi][m];
      }
      sb = cross_row_sum(sb);
      sa = cross_row_sum(sa);
      pit[m] = r.beta_t * (e * kv[m] - sb);
      qe[m] = e * qv[m] - sa - at * pit[m];
    } else {
      pit[m] = 0.f;
      qe[m] = e * qv[m];
    }
  }

  // ---- o^state = S_0^T q~_t : rows v = 4*vi + row of S, K channels over 16 lanes
  float* os_l = os_lds + wave * V;
#pragma unroll
  for (int vi = 0; vi < V / 4; ++vi) {
    const int v = 4 * vi + row;
    Vec<KPL> x;
    x.load(a.S + (item * V + v) * K + col * KPL);
    float d = 0.f;
#pragma unroll
    for (int m = 0; m < KPL; ++m) d += x.e[m] * qe[m];
    d = row_sum16(d);
    if (col == 0) os_l[v] = d;
  }
  wave_lds_sync();

  float ut[VPL], ov[VPL];
#pragma unroll
  for (int vv = 0; vv < VPL; ++vv) {
    float acc = r.v_raw.get(vv);
    if constexpr (ERASE) {
#pragma unroll
      for (int s = 0; s < WMAX; ++s)
        if (s < n) acc -= b_u[s] * us[s][vv];
    }
    ut[vv] = r.beta_t * acc;
    float o = os_l[lane * VPL + vv] + at * ut[vv];
    if constexpr (ERASE) {
#pragma unroll
      for (int s = 0; s < WMAX; ++s)
        if (s < n) o += a_u[s] * us[s][vv];
    } else {
#pragma unroll
      for (int s = 0; s < WMAX; ++s)
        if (s < n) o += a_u[s] * vs[s].get(vv);
    }
    ov[vv] = o;
  }
  {
    Vec<VPL> t;
#pragma unroll
    for (int vv = 0; vv < VPL; ++vv) t.e[vv] = ov[vv];
    t.store(a.o + item * V + lane * VPL);
  }

  const size_t sl = slot0 + n;
  if (row == 0) {
    r.k_raw.store(static_cast<IO*>(a.rk) + sl * K + col * KPL);
    if constexpr (CHAN) {
      Vec<KPL> t;
#pragma unroll
      for (int m = 0; m < KPL; ++m) t.e[m] = gt[m];
      t.store(a.rg + sl * K + col * KPL);
    }
    if constexpr (ERASE) {
      Vec<KPL> t;
#pragma unroll
      for (int m = 0; m < KPL; ++m) t.e[m] = pit[m];
      t.store(a.rpi + sl * K + col * KPL);
    }
  }
  if (lane == 0) {
    if constexpr (!CHAN) a.rg[sl] = gt[0];
    a.rbeta[sl] = r.beta_t;
  }
  if constexpr (ERASE) {
    Vec<VPL> t;
#pragma unroll
    for (int vv = 0; vv < VPL; ++vv) t.e[vv] = ut[vv];
    t.store(a.ru + sl * V + lane * VPL);
    if (col == 0) {
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) {
        const int s = 4 * gi + row;
        if (4 * gi < n && s < n) a.rb[sl * W + s] = bv[gi];
      }
    }
  } else {
    r.v_raw.store(static_cast<IO*>(a.rv) + sl * V + lane * VPL);
  }
}

}  // namespace skssm

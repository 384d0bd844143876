// Non-flush read of SketchSSM (Algorithm 1, t < W) and the exact
// full-state-read baseline.
//
// Per (request, head) item, with the current token in ring slot n (t = n + 1
// tokens in the window):
//   g_t      = sum_{j<=t} log alpha_j                      (window-local cumulative log decay)
//   a_{t,s}  = <exp(g_t - g_s) . k_s, q_t>,  s <= t       (Appendix C.2, key reuse)
//   b_{t,j}  = <exp(g_t - g_j) . k_j, k_t>,  j <  t       (erase couplings)
//   u_t      = beta_t (v_t - sum_j b_{t,j} u_j)           (pseudo-values; Mamba-2: beta_t v_t)
//   f_t      = beta_t (C (e^{g_t} . k_t) - sum_j b_{t,j} f_j)      (eq. wyread)
//   c_t      = C (e^{g_t} . q_t) - sum_{s<=t} a_{t,s} f_s          (eq. app-projected-query)
//   o_t      = U c_t + sum_{s<=t} a_{t,s} u_s              (eq. equantion-sketch + buffer term)
// The exact baseline replaces f by the full erase factors pi (eq. wy) and
// U c_t by S_0^T q~_t with q~_t = e^{g_t} . q_t - sum_s a_{t,s} pi_s.
//
// The token's raw update inputs (k, v, beta, log alpha) were written into
// ring slot n by their producer, so appending costs no copy: the kernels read
// them there and store only derived fields (GDN/KDA: u, f or pi, the row of
// couplings b; KDA: the cumulative log decay).  For scalar decays the
// cumulative log decays are rebuilt on the fly from the ring's log alphas.
//
// Mapping: one wave per item; the item index is wave-uniform, so per-item
// base addresses live in scalar registers.  Everything read from the replay
// buffer uses the row layout: row r of the wave holds ring slot 4 gi + r, so
// one load instruction fetches four slots and the slot sums of the buffer
// term reduce inside each row before a single cross-row sum.  The sketch and
// the output use the value layout (lane l owns v = l + 64 j); the sketch sits
// in 4-column panels U[B][H][r/4][V][4], one float4 per lane per panel, 1 KB
// contiguous per load.  The buffer term crosses from the row layout to the
// value layout through a small LDS transpose.  No matrix cores: every
// contraction here is a matrix-vector product.
#pragma once

#include "args.h"
#include "device.h"

namespace skssm {

// Loads shared by the sketch read and the exact baseline (row layout).
template <int KIND, int K, int V, int WMAX, typename IO>
struct RowLoads {
  static constexpr bool ERASE = KIND != MAMBA2;
  static constexpr bool CHAN = KIND == KDA;
  static constexpr int KPL = K / 16;  // key channels per lane
  static constexpr int VR = V / 16;   // value channels per lane
  static constexpr int NG = WMAX / 4; // groups of four slots
  static constexpr int GD = CHAN ? KPL : 1;
  static constexpr int JP = (WMAX + 15) / 16;  // columns of T^{-1} per lane: j = col + 16 p

  Raw<IO, KPL> q_raw, k_raw;          // current query and key (same in every row)
  Raw<IO, VR> v_raw;                  // current value (same in every row)
  float beta_t;
  float la[GD];                       // log alpha_t
  float gprev[GD];                    // g_{t-1}, rebuilt from the ring's log alphas
  Raw<IO, KPL> ks[NG];                // ring keys of slot 4 gi + row, s < n
  float gs[NG][GD];                   // log alpha, then cumulative log decay, of slot 4 gi + row
  Raw<IO, VR> vs[NG];                 // ring raw values
  float bs[NG];                       // ring beta
  float tv[ERASE ? NG : 1][JP];       // ring (T^{-1})_{s,j}, s = 4 gi + row, j = col + 16 p (unmasked)

  // `item` is wave-uniform.  Slot s of a raw ring field (k, v, beta, log
  // alpha) of width w sits at field + (item * W + s) * w, the W slots of an
  // item contiguous; slot s of a derived field (f, pi, rows of T^{-1}) at
  // field + (s * B*H + dp) * w with dp = h * B + b: one slot of all items
  // contiguous, head-major within the slot.
  __device__ __forceinline__ void load(const DecodeArgs& a, size_t item, size_t dp, int row, int col) {
    const int n = a.n;
    const size_t W = (size_t)a.W, NI = (size_t)a.B * a.H;
    if constexpr (ERASE) {
      // rows of T^{-1}: issued first and without branches (row and column
      // clamped into the ring, masked at use), so they share the first wait;
      // slots are a 32-bit byte stride apart (the ABI bounds B*H)
      const int smax = n > 0 ? n - 1 : 0;
      const uint32_t slot_bytes = (uint32_t)(NI * W * sizeof(float));
#pragma unroll
      for (int p = 0; p < JP; ++p) {
        const int j = col + 16 * p;
        const char* lb = reinterpret_cast<const char*>(a.rt + dp * W + (j < a.W ? j : a.W - 1));
#pragma unroll
        for (int gi = 0; gi < NG; ++gi) {
          const int s = 4 * gi + row;
          tv[gi][p] = *reinterpret_cast<const float*>(lb + (uint64_t)(uint32_t)(s < smax ? s : smax) * slot_bytes);
        }
      }
    }
    const uint32_t koff = (uint32_t)(col * KPL), voff = (uint32_t)(col * VR);
    const size_t cur = item * W + n;                 // slot n of this item (raw fields)
    q_raw.load_nt(static_cast<const IO*>(a.q) + item * K + koff);
    k_raw.load_nt(static_cast<const IO*>(a.rk) + cur * K + koff);
    v_raw.load_nt(static_cast<const IO*>(a.rv) + cur * V + voff);
    beta_t = a.rbeta[cur];
    if constexpr (CHAN) {
      Vec<KPL> t;
      t.load_nt(a.rla + cur * K + koff);
#pragma unroll
      for (int m = 0; m < KPL; ++m) la[m] = t.e[m];
    } else {
      la[0] = a.rla[cur];
    }
#pragma unroll
    for (int m = 0; m < GD; ++m) gprev[m] = 0.f;
    const size_t rowslot = item * W + row;           // slot `row` of this item (raw fields)
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) {
      const int s = 4 * gi + row;
      const size_t si = rowslot + 4 * gi;
      ks[gi].zero();
      vs[gi].zero();
      bs[gi] = 0.f;
#pragma unroll
      for (int m = 0; m < GD; ++m) gs[gi][m] = 0.f;
      if (4 * gi < n && s < n) {  // per lane (rows), so it masks lanes rather than branching
        ks[gi].load_nt(static_cast<const IO*>(a.rk) + si * K + koff);
        vs[gi].load_nt(static_cast<const IO*>(a.rv) + si * V + voff);
        bs[gi] = a.rbeta[si];
        // log alpha_s for now; made cumulative in prefix_decay()
        if constexpr (CHAN) {
          Vec<KPL> t;
          t.load_nt(a.rla + si * K + koff);
#pragma unroll
          for (int m = 0; m < KPL; ++m) gs[gi][m] = t.e[m];
        } else {
          gs[gi][0] = a.rla[si];
        }
      }
    }
  }

  // Turn the per-slot log alphas into cumulative log decays
  // g_s = sum_{j<=s} log alpha_j (slots in order), and g_{t-1}.  Slots >= n
  // hold zeros, so sums over whole groups are sums over the window.
  __device__ __forceinline__ void prefix_decay(int n, int row) {
    // per channel (KDA) or per slot: inclusive scan over the 4 rows of a
    // group (rows_scan), then the running total of the earlier groups
    float tot[GD];
#pragma unroll
    for (int m = 0; m < GD; ++m) tot[m] = 0.f;
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) {
      if (4 * gi < n) {
#pragma unroll
        for (int m = 0; m < GD; ++m) {
          float grp;
          const float z = rows_scan(gs[gi][m], row, grp);
          gs[gi][m] = tot[m] + z;
          tot[m] += grp;
        }
      }
    }
#pragma unroll
    for (int m = 0; m < GD; ++m) gprev[m] = tot[m];
  }
};

// Dot products of the current query / key with every buffered key.
// Returns, in the row layout, av[gi] = a_{t,s} and bv[gi] = b_{t,s} for
// s = 4 gi + row (0 for s >= n), plus at = <k_t, q_t>.
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
    }
    av[gi] = pa;
    bv[gi] = pb;
  }
}

// Coefficients of the buffer term on the raw values (GDN/KDA).  With the
// couplings B_{s,j} = b_{s,j} (j < s) of eq. wy, T = I + Diag(beta) B is unit
// lower triangular and the pseudo-values are u = T^{-1} (beta . v), so
//   sum_{s<n} a_{t,s} u_s = sum_j alpha_j beta_j v_j,   alpha = T^{-T} a_{t,.}
//   sum_{j<n} b_{t,j} u_j = sum_j gamma_j beta_j v_j,   gamma = T^{-T} b_{t,.}
// The ring holds the rows of T^{-1}, so both are products with stored rows:
// lane (row, col) multiplies (T^{-1})_{s,j} (s = 4 gi + row, j = col + 16 p)
// by a_s and b_s and the 4 rows are summed, leaving alpha_j and gamma_j in
// column j.  A pass through LDS (sc: 2 WMAX floats) returns them to the row
// layout as ca = alpha . beta and cg = gamma . beta (slot 4 gi + row);
// gcol keeps gamma_j in column j for the new row of T^{-1}.
template <class L>
__device__ __forceinline__ void erase_coefs(int n, int row, int col, const L& r, const float (&av)[L::NG],
                                            const float (&bv)[L::NG], float* sc, float (&ca)[L::NG],
                                            float (&cg)[L::NG], float (&gcol)[L::JP]) {
  constexpr int NG = L::NG, JP = L::JP, WM = 4 * NG;
  float acol[JP];
#pragma unroll
  for (int p = 0; p < JP; ++p) {
    const int j = col + 16 * p;
    float pa = 0.f, pg = 0.f;
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) {
      const int s = 4 * gi + row;
      // selected, never multiplied away: entries past row n-1 or on and
      // above the diagonal are stale ring contents (slots >= n have a_s = b_s = 0)
      const float t = (s < n && j < s) ? r.tv[gi][p] : (j == s ? 1.f : 0.f);
      pa += t * av[gi];
      pg += t * bv[gi];
    }
    acol[p] = cross_row_sum(pa);
    gcol[p] = cross_row_sum(pg);
  }
  // column j -> slot j = 4 gi + row: sc[(j % 4) NG + j / 4], so a lane reads its NG values contiguously
  if (row == 0) {
#pragma unroll
    for (int p = 0; p < JP; ++p) {
      const int j = col + 16 * p;
      if (j < WM) {
        sc[(j & 3) * NG + (j >> 2)] = acol[p];
        sc[WM + (j & 3) * NG + (j >> 2)] = gcol[p];
      }
    }
  }
  wave_lds_sync();
  Vec<NG> va, vg;
  va.load(sc + row * NG);
  vg.load(sc + WM + row * NG);
#pragma unroll
  for (int gi = 0; gi < NG; ++gi) {
    ca[gi] = va.e[gi] * r.bs[gi];
    cg[gi] = vg.e[gi] * r.bs[gi];
  }
}

// Buffer term and current pseudo-value in the row layout (every row ends
// with the full sums), from per-slot coefficients on the raw values:
// ob = sum_s ca_s v_s + a_{t,t} u_t and u_t = beta_t (v_t - sum_s cg_s v_s)
// (Mamba-2: ca_s = a_{t,s} beta_s, no cg, u_t = beta_t v_t).
template <class L>
__device__ __forceinline__ void buffer_term(const L& r, const float (&ca)[L::NG], const float (&cg)[L::NG],
                                            float at, float (&ut)[L::VR], float (&ob)[L::VR]) {
#pragma unroll
  for (int m = 0; m < L::VR; ++m) {
    float sa = 0.f, sb = 0.f;
#pragma unroll
    for (int gi = 0; gi < L::NG; ++gi) {
      const float x = r.vs[gi].get(m);
      sa += ca[gi] * x;
      if constexpr (L::ERASE) sb += cg[gi] * x;
    }
    sa = cross_row_sum(sa);
    if constexpr (L::ERASE) {
      sb = cross_row_sum(sb);
      ut[m] = r.beta_t * (r.v_raw.get(m) - sb);
    } else {
      ut[m] = r.beta_t * r.v_raw.get(m);
    }
    ob[m] = sa + at * ut[m];
  }
}

// Per-slot coefficients of the buffer term for any kind (see erase_coefs).
template <class L>
__device__ __forceinline__ void buffer_coefs(int n, int row, int col, const L& r, const float (&av)[L::NG],
                                             const float (&bv)[L::NG], float* sc, float (&ca)[L::NG],
                                             float (&cg)[L::NG], float (&gcol)[L::JP]) {
  if constexpr (L::ERASE) {
    erase_coefs<L>(n, row, col, r, av, bv, sc, ca, cg, gcol);
  } else {
#pragma unroll
    for (int gi = 0; gi < L::NG; ++gi) {
      ca[gi] = av[gi] * r.bs[gi];
      cg[gi] = 0.f;
    }
#pragma unroll
    for (int p = 0; p < L::JP; ++p) gcol[p] = 0.f;
  }
}

// Row n of T^{-1} for the token at ring slot n (GDN/KDA), stored for later
// reads and the flush: (T^{-1})_{n,j} = -beta_n gamma_j, j < n, because row n
// of T T^{-1} = I reads (T^{-1})_{n,.} = -beta_n b_{n,.} T^{-1}.  Mamba-2
// derives nothing.
template <class L>
__device__ __forceinline__ void append_derived(const DecodeArgs& a, size_t dp, int row, int col,
                                               const L& r, const float (&gcol)[L::JP]) {
  if constexpr (L::ERASE) {
    const int n = a.n;
    if (row == 0) {
      float* dst = a.rt + ((size_t)n * a.B * a.H + dp) * a.W;
#pragma unroll
      for (int p = 0; p < L::JP; ++p) {
        const int j = col + 16 * p;
        if (j < n) dst[j] = -r.beta_t * gcol[p];
      }
    }
  }
}

// The exact full-state read of one item by one wave (no workgroup barrier):
//   o = S_0^T q~_t + o_t^buffer,  q~_t = e^{g_t} . q_t - sum_s a_{t,s} pi_s
// (eq. app-effective-query-wy), storing pi_t and row n of T^{-1} for the
// token.  dp: the item's position in the derived ring fields (h * B + b).
// ws: the wave's 2V + 2 WMAX + K floats of LDS.
template <int KIND, int K, int V, int WMAX, typename IO>
__device__ __forceinline__ void full_read_item(const DecodeArgs& a, size_t item, size_t dp, int lane, float* ws) {
  using L = RowLoads<KIND, K, V, WMAX, IO>;
  constexpr bool ERASE = L::ERASE, CHAN = L::CHAN;
  constexpr int KPL = L::KPL, VR = L::VR, NG = L::NG, GD = L::GD;
  constexpr int VPL = V / 64;
  const int row = lane >> 4, col = lane & 15;
  const int n = a.n;
  const size_t NI = (size_t)a.B * a.H;
  const uint32_t koff = (uint32_t)(col * KPL);

  L r;
  r.load(a, item, dp, row, col);
  float ps[ERASE ? NG : 1][KPL];     // ring pi of slot 4 gi + row (row layout)
  if constexpr (ERASE) {
    // slot clamped below n and the value selected (no guarded load)
    const int smax = n > 0 ? n - 1 : 0;
    const uint32_t slot_bytes = (uint32_t)(NI * K * sizeof(float));
    const char* lb = reinterpret_cast<const char*>(a.rpi + dp * K + koff);
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) {
      const int s = 4 * gi + row;
      Vec<KPL> t;
      t.load(reinterpret_cast<const float*>(lb + (uint64_t)(uint32_t)(s < smax ? s : smax) * slot_bytes));
#pragma unroll
      for (int m = 0; m < KPL; ++m) ps[gi][m] = s < n ? t.e[m] : 0.f;
    }
  }

  float* os_l = ws;
  float* ob_l = os_l + V;
  float* b_l = ob_l + V;

  r.prefix_decay(n, row);
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
  float ca[NG], cg[NG], gcol[L::JP];
  buffer_coefs<L>(n, row, col, r, av, bv, b_l, ca, cg, gcol);
  float ut[VR], ob[VR];
  buffer_term(r, ca, cg, at, ut, ob);

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

  // ---- o^state = S_0^T q~_t over the state's 16 x 16 tiles.  Tile (vt, kt)
  // is 1 KB contiguous with lane l holding X[16 vt + l%16][16 kt + 4 (l/16) + i]
  // (the flush's register layout), so every load moves 1 KB: q~ goes through
  // LDS to those channels, each lane sums over the K tiles, and the four lane
  // rows are summed.
  constexpr int MT = K / 16, VT = V / 16;
  float* qe_l = b_l + 2 * WMAX;                   // K floats
  if (row == 0) {
#pragma unroll
    for (int m = 0; m < KPL; ++m) qe_l[koff + m] = qe[m];
  }
  wave_lds_sync();
  float4 qf[MT];
#pragma unroll
  for (int kt = 0; kt < MT; ++kt) qf[kt] = *reinterpret_cast<const float4*>(qe_l + 16 * kt + 4 * row);
  const float* Sb = a.S + item * (size_t)V * K + 4 * lane;
#pragma unroll
  for (int vt = 0; vt < VT; ++vt) {
    float d = 0.f;
#pragma unroll
    for (int kt = 0; kt < MT; ++kt) {
      const float4 x = ld_nt(reinterpret_cast<const float4*>(Sb + (uint32_t)((vt * MT + kt) * 256)));
      d += x.x * qf[kt].x + x.y * qf[kt].y + x.z * qf[kt].z + x.w * qf[kt].w;
    }
    d = cross_row_sum(d);
    if (row == 0) os_l[16 * vt + col] = d;
  }
  if (row == 0) {
#pragma unroll
    for (int m = 0; m < VR; ++m) ob_l[col * VR + m] = ob[m];
  }
  wave_lds_sync();
  float* ob_g = a.o + item * V;
#pragma unroll
  for (int vv = 0; vv < VPL; ++vv) ob_g[lane + 64 * vv] = os_l[lane + 64 * vv] + ob_l[lane + 64 * vv];

  append_derived<L>(a, dp, row, col, r, gcol);
  if constexpr (ERASE) {
    if (row == 0) {
      Vec<KPL> t;
#pragma unroll
      for (int m = 0; m < KPL; ++m) t.e[m] = pit[m];
      t.store(a.rpi + ((size_t)n * NI + dp) * K + koff);
    }
  }
}

// Ring f of slots 4 gi + row (components col + 16 p) for the read of slot n:
// the slot is clamped below n and the load made unconditionally, the value
// then masked by a select (a guarded load would compile to a branch whose
// join waits for every load in flight).  bf16: lanes j and j^1 read the same
// 32-bit word.  Slots are a 32-bit byte stride apart (the ABI bounds B*H).
template <int NG, int RP, typename SK>
__device__ __forceinline__ void load_ring_f(const DecodeArgs& a, size_t dp, int n, int row, int col, int rh, int R,
                                            const SK* rf, float (&fs)[NG][RP]) {
  const int smax = n > 0 ? n - 1 : 0;
  const uint32_t slot_bytes = (uint32_t)((size_t)a.B * a.H * R * sizeof(SK));
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    const int j = col + 16 * p;
    const char* lb = reinterpret_cast<const char*>(rf + dp * R) + (sizeof(SK) == 2 ? 4 * (j >> 1) : 4 * j);
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) {
      const int s = 4 * gi + row;
      const uint32_t w = *reinterpret_cast<const uint32_t*>(lb + (uint64_t)(uint32_t)(s < smax ? s : smax) * slot_bytes);
      const float fv = sizeof(SK) == 2 ? ((j & 1) ? bf16_hi(w) : bf16_lo(w)) : __uint_as_float(w);
      fs[gi][p] = (s < n && j < rh) ? fv : 0.f;
    }
  }
}

// The item's state-dependent coefficient map C (R x K in the sketch dtype),
// stored in 16-byte channel panels cmap[B][H][K/CPW][R][CPW] (element (j, k)
// at ((k / CPW) R + j) CPW + k % CPW, CPW = 4 fp32 or 8 bf16 channels): for
// this lane's rows j = col + 16 p, its K/4 channels row K/4 .. as CL panels.
// Rows at or past the head's rank re-read row 0 (fetched anyway) and are not
// used; the load itself is unconditional.
template <int K, int R, int RP, int CL, typename SK>
__device__ __forceinline__ void load_map_rows(const DecodeArgs& a, size_t item, int row, int col, int rh,
                                              Raw<SK, 16 / sizeof(SK)> (&cm)[RP][CL]) {
  constexpr int CPW = 16 / (int)sizeof(SK);
  const SK* base = static_cast<const SK*>(a.cmap) + item * (size_t)(R * K);
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    const int j = col + 16 * p;
    const int jj = j < rh ? j : 0;
#pragma unroll
    for (int i = 0; i < CL; ++i) cm[p][i].load_nt(base + (uint32_t)(((row * CL + i) * R + jj) * CPW));
  }
}

// DENSE: compiled with the exact read for dense-fallback heads (launched only
// for rank tables that have some); without it the kernel needs fewer registers.
template <int KIND, int K, int V, int R, int WMAX, typename IO, typename SK, int P, bool DENSE>
__global__ __launch_bounds__(256) void decode_kernel(const DecodeArgs a) {
  using L = RowLoads<KIND, K, V, WMAX, IO>;
  constexpr bool ERASE = L::ERASE, CHAN = L::CHAN;
  constexpr int KPL = L::KPL, VR = L::VR, NG = L::NG, GD = L::GD;
  constexpr int VPL = V / 64;                    // value channels per lane (value layout)
  constexpr int RP = (R + 15) / 16;              // sketch components per lane (row layout)
  constexpr int PW = 16 / (int)sizeof(SK);       // sketch columns per panel: 16 bytes per value
  constexpr int NP = R / PW;                     // sketch panels
  constexpr int CP = K + 4;                      // padded LDS row pitch of C
  constexpr int KQ = K / 4;                      // channels each row covers in C x
  constexpr int WS = 2 * K + R + V + 2 * WMAX;   // per-wave LDS: x_q, x_k, c, o_buf, alpha/gamma transposition
  constexpr bool U_PRELOAD = R <= 32;
  constexpr int UP = U_PRELOAD ? NP : 1;

  __shared__ __align__(16) float c_lds[P != 0 ? 4 : R * CP];
  __shared__ __align__(16) float wscr[4 * WS];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int row = lane >> 4, col = lane & 15;
  const int H = a.H, n = a.n;
  // workgroup -> (head, batch tile): head fastest; with a per-head rank table
  // the dense heads' workgroups come first, in the head order hlist
  int h = blockIdx.x % H, tile = blockIdx.x / H;
  if (a.ragged) {
    const int T = gridDim.x / H, nd = a.ndense, w = blockIdx.x;
    if (w < nd * T) {
      h = arg_byte(a.hlist, w % nd);
      tile = w / nd;
    } else {
      const int ns = H - nd, w2 = w - nd * T;
      h = arg_byte(a.hlist, nd + w2 % ns);
      tile = w2 / ns;
    }
  }
  const int b = tile * 4 + wave;
  const bool valid = b < a.B;
  const size_t item = (size_t)(valid ? b : 0) * H + h;
  const size_t dp = (size_t)h * a.B + (valid ? b : 0);  // position in the derived ring fields
  const SK* Ub = static_cast<const SK*>(a.U) + item * (size_t)V * R;
  // this head's rank: its first rh sketch columns, coefficient rows and f
  // entries are used; a dense-fallback head (rh = 0) is read elsewhere
  const int rh = a.ragged ? arg_byte(a.hrank, h) : R;
  if (rh == 0) {
    // dense-fallback head: the exact full-state read of its items, one per
    // wave (the whole workgroup shares the head and takes this branch, so no
    // barrier is skipped)
    static_assert(WS >= 2 * V + 2 * WMAX + K, "per-wave LDS too small for the full read");
    if constexpr (DENSE) {
      if (valid) full_read_item<KIND, K, V, WMAX, IO>(a, item, dp, lane, wscr + wave * WS);
    }
    return;
  }

  // ---- the offline map C first (shared by the head's items, staged in
  // LDS), then every global load of this item; a state-dependent map (P != 0)
  // is per item and read into registers like the other per-item data
  constexpr bool SMAP = P != 0;
  constexpr int CQ = SMAP ? 1 : (R * K / 4 + 255) / 256;  // float4 of C per thread
  [[maybe_unused]] Vec<4> cv[CQ];
  if constexpr (!SMAP) {
#pragma unroll
    for (int c = 0; c < CQ; ++c) {
      const int i = tid + 256 * c;
#pragma unroll
      for (int e = 0; e < 4; ++e) cv[c].e[e] = 0.f;
      if ((CQ * 256 == R * K / 4 || i < R * K / 4) && (4 * i) / K < rh) cv[c].load(a.coef + (size_t)h * R * K + 4 * i);
    }
  }
  compiler_fence();
  // Every load of the item follows (the sketch panels after the slot
  // products), with no wave-uniform guard: a wave past
  // the batch reads item 0 of its head (and returns after the barrier);
  // derived-field slots and sketch panels past what the step uses are clamped
  // to ones that exist and their values masked by selects.  A load under a
  // wave-uniform guard compiles to a branch whose join waits for the loads in
  // flight, which serialises the item's memory accesses.  The raw ring slots
  // are guarded per lane (slot 4 gi + row < n), which masks lanes instead.
  L r;
  r.load(a, item, dp, row, col);
  float fs[ERASE ? NG : 1][RP];      // ring f of slot 4 gi + row, component col + 16 p
  Raw<SK, PW> Ur[VPL][UP];           // sketch panels (value layout), loaded after the slot dot products
  // the item's state-dependent map (P != 0): this lane's channels of its rows
  constexpr int CPW = 16 / (int)sizeof(SK);      // channels per 16-byte map panel
  constexpr int CL = SMAP ? KQ / CPW : 1;        // map panels per lane and row
  [[maybe_unused]] Raw<SK, 16 / sizeof(SK)> cmr[SMAP ? RP : 1][CL];
  // f and the map are used only after the C products: with a per-channel
  // decay (KDA) they are loaded with the sketch panels, after the slot
  // products, which keeps the kernel within 128 registers (four waves per
  // SIMD); the other kinds load them here, first
  constexpr bool LATE_FM = CHAN;
  if constexpr (!LATE_FM) {
    if constexpr (ERASE) load_ring_f<NG, RP>(a, dp, n, row, col, rh, R, static_cast<const SK*>(a.rf), fs);
    if constexpr (SMAP) load_map_rows<K, R, RP, CL>(a, item, row, col, rh, cmr);
  }

  // ---- this head's offline map C (R x K) into LDS; its loads were issued
  // first, so the LDS-only barrier leaves the item's own loads in flight
  if constexpr (!SMAP) {
#pragma unroll
    for (int c = 0; c < CQ; ++c) {
      const int i = tid + 256 * c;
      if (CQ * 256 == R * K / 4 || i < R * K / 4) cv[c].store(&c_lds[((4 * i) / K) * CP + (4 * i) % K]);
    }
    lds_barrier();
  }
  if (!valid) return;

  float* xq_l = wscr + wave * WS;
  float* xk_l = xq_l + K;
  float* c_l = xq_l + 2 * K;
  float* ob_l = c_l + R;
  float* b_l = ob_l + V;

  r.prefix_decay(n, row);
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
  // the sketch panels: issued once the ring keys and decays are consumed, so
  // their registers are not live across the slot products (KDA then fits four
  // waves per SIMD); the buffer term and C products cover their latency.
  // Panels past the head's rank re-read panel 0 and are zeroed.
  if constexpr (U_PRELOAD) {
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int vv = 0; vv < VPL; ++vv) {
        const int pp = p * PW < rh ? p : 0;
        Ur[vv][p].load_nt(Ub + (uint32_t)((pp * V + lane + 64 * vv) * PW));
        Ur[vv][p].keep_if(p * PW < rh);
      }
  }
  if constexpr (LATE_FM) {
    if constexpr (ERASE) load_ring_f<NG, RP>(a, dp, n, row, col, rh, R, static_cast<const SK*>(a.rf), fs);
    if constexpr (SMAP) load_map_rows<K, R, RP, CL>(a, item, row, col, rh, cmr);
  }
  float ca[NG], cg[NG], gcol[L::JP];
  buffer_coefs<L>(n, row, col, r, av, bv, b_l, ca, cg, gcol);
  float ut[VR], ob[VR];
  buffer_term(r, ca, cg, at, ut, ob);

  // ---- C (e^{g_t} . q_t) and C (e^{g_t} . k_t): each row covers K/4 channels
  if (row == 0) {
#pragma unroll
    for (int m = 0; m < KPL; ++m) {
      const float e = CHAN ? fast_exp(gt[m]) : 1.f;
      xq_l[col * KPL + m] = e * qv[m];
      if constexpr (ERASE) xk_l[col * KPL + m] = e * kv[m];
    }
#pragma unroll
    for (int m = 0; m < VR; ++m) ob_l[col * VR + m] = ob[m];
  }
  wave_lds_sync();
  const float eg = CHAN ? 1.f : fast_exp(gt[0]);
  float cfin[RP], ft[RP], sqv[RP], skv[RP];
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    const int j = col + 16 * p;
    float sq = 0.f, sk = 0.f;
    if (j < rh) {
      const float* xqr = xq_l + row * KQ;
      const float* xkr = xk_l + row * KQ;
      if constexpr (SMAP) {
        // the item's map: row j over this lane's channels, from registers
#pragma unroll
        for (int i = 0; i < CL; ++i)
#pragma unroll
          for (int e = 0; e < CPW; e += 4) {
            const Raw<SK, 16 / sizeof(SK)>& cr = cmr[p][i];
            const float4 xx = *reinterpret_cast<const float4*>(xqr + i * CPW + e);
            sq += cr.get(e) * xx.x + cr.get(e + 1) * xx.y + cr.get(e + 2) * xx.z + cr.get(e + 3) * xx.w;
            if constexpr (ERASE) {
              const float4 yy = *reinterpret_cast<const float4*>(xkr + i * CPW + e);
              sk += cr.get(e) * yy.x + cr.get(e + 1) * yy.y + cr.get(e + 2) * yy.z + cr.get(e + 3) * yy.w;
            }
          }
      } else {
        const float* cr = c_lds + j * CP + row * KQ;
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
    }
    sqv[p] = cross_row_sum(sq);
    skv[p] = ERASE ? cross_row_sum(sk) : 0.f;
  }
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    const float sq = sqv[p], sk = skv[p];
    if constexpr (ERASE) {
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

  // ---- o = U c + buffer term  (value layout)
  float* ob_g = a.o + item * V;
#pragma unroll
  for (int vv = 0; vv < VPL; ++vv) {
    float acc = ob_l[lane + 64 * vv];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      if (p * PW >= rh) break;  // panels past this head's rank are not stored
      Raw<SK, PW> u;
      if constexpr (U_PRELOAD) u = Ur[vv][p];
      else u.load_nt(Ub + (uint32_t)((p * V + lane + 64 * vv) * PW));
#pragma unroll
      for (int i = 0; i < PW; i += 4) {
        const float4 c4 = *reinterpret_cast<const float4*>(c_l + PW * p + i);
        acc += u.get(i) * c4.x + u.get(i + 1) * c4.y + u.get(i + 2) * c4.z + u.get(i + 3) * c4.w;
      }
    }
    ob_g[lane + 64 * vv] = acc;
  }

  // ---- derived fields of the token at ring slot n
  append_derived<L>(a, dp, row, col, r, gcol);
  if constexpr (ERASE) {
    if (row == 0) {
      const size_t sl = (size_t)n * a.B * H + dp;
#pragma unroll
      for (int p = 0; p < RP; ++p) {
        const int j = col + 16 * p;
        SK* dst = static_cast<SK*>(a.rf) + sl * R;
        if constexpr (sizeof(SK) == 2) {
          // bf16: even lanes store their value and their neighbour's as one 32-bit word
          const float nb = dpp<0xB1>(ft[p]);  // quad_perm [1,0,3,2]: lane j ^ 1
          if (!(j & 1)) {
            if (j + 1 < rh)
              reinterpret_cast<uint32_t*>(dst)[j >> 1] = bf16_bits_rne(ft[p]) | (bf16_bits_rne(nb) << 16);
            else if (j < rh)
              st_elem<SK>(dst + j, ft[p]);
          }
        } else {
          if (j < rh) st_elem<SK>(dst + j, ft[p]);
        }
      }
    }
  }
}

template <int KIND, int K, int V, int WMAX, typename IO>
__global__ __launch_bounds__(256) void full_read_kernel(const DecodeArgs a) {
  constexpr int WS = 2 * V + 2 * WMAX + K;  // per-wave LDS: o^state, o_buf, alpha/gamma transposition, q~
  __shared__ __align__(16) float wscr[4 * WS];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const size_t NI = (size_t)a.B * a.H;
  // XCD x runs a contiguous share of the items (neighbouring items share the
  // cache lines of the per-slot scalars); plain order when the grid does not split
  const uint32_t G = gridDim.x, wg = blockIdx.x;
  const uint32_t lwg = (G % 8 == 0) ? (wg % 8) * (G / 8) + wg / 8 : wg;
  const size_t item = (size_t)lwg * 4 + wave;
  if (item >= NI) return;  // wave-uniform; no block barrier in this kernel
  const uint32_t b = (uint32_t)item / (uint32_t)a.H, h = (uint32_t)item - b * (uint32_t)a.H;  // B*H <= 2^30
  full_read_item<KIND, K, V, WMAX, IO>(a, item, (size_t)h * a.B + b, lane, wscr + wave * WS);
}

}  // namespace skssm

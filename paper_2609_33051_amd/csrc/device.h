// Device helpers shared by the SketchSSM kernels (gfx950, wave64).
//
// Lane layouts used by the kernels:
//   row layout    the wave is 4 rows of 16 lanes (DPP rows).  A K-vector is
//                 spread over the 16 lanes of a row, K/16 consecutive channels
//                 per lane; the 4 rows either hold copies or 4 different
//                 ring slots, so one wide load fetches 4 slots at once and a
//                 16-lane DPP reduction finishes 4 dot products together.
//   value layout  lane l owns value channels l + 64 j, j < V/64, so a load
//                 instruction over the value axis reads one contiguous run.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace skssm {

enum Kind { MAMBA2 = 0, GDN = 1, KDA = 2 };

typedef uint16_t bf16_t;
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t uintx4 __attribute__((ext_vector_type(4)));
typedef uint32_t uintx2 __attribute__((ext_vector_type(2)));

// Non-temporal loads (the nt bit): for data a launch reads once (the sketch,
// the ring, the state).  Reads marked this way stream past the caches and
// raise the achieved HBM bandwidth of one-shot reads by several percent;
// data shared across workgroups (C, Omega) keeps ordinary loads.
__device__ __forceinline__ float4 ld_nt(const float4* p) {
  const floatx4 t = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(p));
  return make_float4(t.x, t.y, t.z, t.w);
}
__device__ __forceinline__ uint4 ld_nt(const uint4* p) {
  const uintx4 t = __builtin_nontemporal_load(reinterpret_cast<const uintx4*>(p));
  return make_uint4(t.x, t.y, t.z, t.w);
}
__device__ __forceinline__ uint2 ld_nt(const uint2* p) {
  const uintx2 t = __builtin_nontemporal_load(reinterpret_cast<const uintx2*>(p));
  return make_uint2(t.x, t.y);
}
__device__ __forceinline__ float ld_nt(const float* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st_nt(float4* p, float4 v) {
  __builtin_nontemporal_store(floatx4{v.x, v.y, v.z, v.w}, reinterpret_cast<floatx4*>(p));
}
__device__ __forceinline__ uint32_t ld_nt(const uint32_t* p) { return __builtin_nontemporal_load(p); }

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// One io element kept in a full 32-bit register (raw bits, zero-extended for
// bf16): loads need no packing into register halves, so the compiler does not
// have to wait for them early.
template <typename IO> __device__ __forceinline__ uint32_t ld_bits(const IO* p, uint32_t off);
template <> __device__ __forceinline__ uint32_t ld_bits<float>(const float* p, uint32_t off) {
  return __float_as_uint(p[off]);
}
template <> __device__ __forceinline__ uint32_t ld_bits<bf16_t>(const bf16_t* p, uint32_t off) {
  return (uint32_t)p[off];
}
template <typename IO> __device__ __forceinline__ void st_bits(IO* p, uint32_t off, uint32_t x);
template <> __device__ __forceinline__ void st_bits<float>(float* p, uint32_t off, uint32_t x) {
  p[off] = __uint_as_float(x);
}
template <> __device__ __forceinline__ void st_bits<bf16_t>(bf16_t* p, uint32_t off, uint32_t x) {
  p[off] = (bf16_t)x;
}
// fp32 -> bf16 bits, round to nearest with ties to even (NaN payloads are
// truncated, infinities kept).
__device__ __forceinline__ uint32_t bf16_bits_rne(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7f800000u) != 0x7f800000u) u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// One stored element of a field kept in T (fp32, or bf16 rounded to nearest
// even), as fp32; and four consecutive ones (16-byte / 8-byte aligned).
template <typename T> __device__ __forceinline__ float ld_elem(const T* p);
template <> __device__ __forceinline__ float ld_elem<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ld_elem<bf16_t>(const bf16_t* p) { return bf16_lo((uint32_t)*p); }
template <typename T> __device__ __forceinline__ void st_elem(T* p, float x);
template <> __device__ __forceinline__ void st_elem<float>(float* p, float x) { *p = x; }
template <> __device__ __forceinline__ void st_elem<bf16_t>(bf16_t* p, float x) { *p = (bf16_t)bf16_bits_rne(x); }
template <typename T> __device__ __forceinline__ void st_elem4(T* p, float a, float b, float c, float d);
template <> __device__ __forceinline__ void st_elem4<float>(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
template <> __device__ __forceinline__ void st_elem4<bf16_t>(bf16_t* p, float a, float b, float c, float d) {
  *reinterpret_cast<uint2*>(p) = make_uint2(bf16_bits_rne(a) | (bf16_bits_rne(b) << 16),
                                            bf16_bits_rne(c) | (bf16_bits_rne(d) << 16));
}

template <typename IO> __device__ __forceinline__ float bits_f32(uint32_t x) {
  if constexpr (sizeof(IO) == 2) return bf16_lo(x);
  else return __uint_as_float(x);
}

// N raw elements of the io dtype, moved with the widest aligned accesses.
template <typename IO, int N> struct Raw;

template <int N> struct Raw<float, N> {
  float e[N];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < N; ++i) e[i] = 0.f;
  }
  // zero the values unless `keep` (a select, so a load before it stays unconditional)
  __device__ __forceinline__ void keep_if(bool keep) {
#pragma unroll
    for (int i = 0; i < N; ++i) e[i] = keep ? e[i] : 0.f;
  }
  __device__ __forceinline__ void load(const float* p) {
    if constexpr (N % 4 == 0) {
#pragma unroll
      for (int i = 0; i < N / 4; ++i) {
        const float4 t = reinterpret_cast<const float4*>(p)[i];
        e[4 * i] = t.x; e[4 * i + 1] = t.y; e[4 * i + 2] = t.z; e[4 * i + 3] = t.w;
      }
    } else if constexpr (N == 2) {
      const float2 t = *reinterpret_cast<const float2*>(p);
      e[0] = t.x; e[1] = t.y;
    } else {
      static_assert(N == 1, "unsupported width");
      e[0] = *p;
    }
  }
  __device__ __forceinline__ void load_nt(const float* p) {
    if constexpr (N % 4 == 0) {
#pragma unroll
      for (int i = 0; i < N / 4; ++i) {
        const float4 t = ld_nt(reinterpret_cast<const float4*>(p) + i);
        e[4 * i] = t.x; e[4 * i + 1] = t.y; e[4 * i + 2] = t.z; e[4 * i + 3] = t.w;
      }
    } else if constexpr (N == 1) {
      e[0] = ld_nt(p);
    } else {
      load(p);
    }
  }
  __device__ __forceinline__ void store(float* p) const {
    if constexpr (N % 4 == 0) {
#pragma unroll
      for (int i = 0; i < N / 4; ++i)
        reinterpret_cast<float4*>(p)[i] = make_float4(e[4 * i], e[4 * i + 1], e[4 * i + 2], e[4 * i + 3]);
    } else if constexpr (N == 2) {
      *reinterpret_cast<float2*>(p) = make_float2(e[0], e[1]);
    } else {
      *p = e[0];
    }
  }
  __device__ __forceinline__ float get(int i) const { return e[i]; }
};

template <int N> struct Raw<bf16_t, N> {
  static constexpr int NW = (N + 1) / 2;
  uint32_t w[NW];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < NW; ++i) w[i] = 0u;
  }
  __device__ __forceinline__ void keep_if(bool keep) {
#pragma unroll
    for (int i = 0; i < NW; ++i) w[i] = keep ? w[i] : 0u;
  }
  __device__ __forceinline__ void load(const bf16_t* p) {
    if constexpr (N % 8 == 0) {
#pragma unroll
      for (int i = 0; i < N / 8; ++i) {
        const uint4 t = reinterpret_cast<const uint4*>(p)[i];
        w[4 * i] = t.x; w[4 * i + 1] = t.y; w[4 * i + 2] = t.z; w[4 * i + 3] = t.w;
      }
    } else if constexpr (N == 4) {
      const uint2 t = *reinterpret_cast<const uint2*>(p);
      w[0] = t.x; w[1] = t.y;
    } else if constexpr (N == 2) {
      w[0] = *reinterpret_cast<const uint32_t*>(p);
    } else {
      static_assert(N == 1, "unsupported width");
      w[0] = (uint32_t)(*p);
    }
  }
  __device__ __forceinline__ void load_nt(const bf16_t* p) {
    if constexpr (N % 8 == 0) {
#pragma unroll
      for (int i = 0; i < N / 8; ++i) {
        const uint4 t = ld_nt(reinterpret_cast<const uint4*>(p) + i);
        w[4 * i] = t.x; w[4 * i + 1] = t.y; w[4 * i + 2] = t.z; w[4 * i + 3] = t.w;
      }
    } else if constexpr (N == 4) {
      const uint2 t = ld_nt(reinterpret_cast<const uint2*>(p));
      w[0] = t.x; w[1] = t.y;
    } else if constexpr (N == 2) {
      w[0] = ld_nt(reinterpret_cast<const uint32_t*>(p));
    } else {
      load(p);
    }
  }
  __device__ __forceinline__ void store(bf16_t* p) const {
    if constexpr (N % 8 == 0) {
#pragma unroll
      for (int i = 0; i < N / 8; ++i)
        reinterpret_cast<uint4*>(p)[i] = make_uint4(w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]);
    } else if constexpr (N == 4) {
      *reinterpret_cast<uint2*>(p) = make_uint2(w[0], w[1]);
    } else if constexpr (N == 2) {
      *reinterpret_cast<uint32_t*>(p) = w[0];
    } else {
      *p = (bf16_t)(w[0] & 0xFFFFu);
    }
  }
  __device__ __forceinline__ float get(int i) const {
    return (i & 1) ? bf16_hi(w[i >> 1]) : bf16_lo(w[i >> 1]);
  }
};

template <int N> struct Vec {
  float e[N];
  __device__ __forceinline__ void load(const float* p) {
    Raw<float, N> r;
    r.load(p);
#pragma unroll
    for (int i = 0; i < N; ++i) e[i] = r.e[i];
  }
  __device__ __forceinline__ void load_nt(const float* p) {
    Raw<float, N> r;
    r.load_nt(p);
#pragma unroll
    for (int i = 0; i < N; ++i) e[i] = r.e[i];
  }
  __device__ __forceinline__ void store(float* p) const {
    Raw<float, N> r;
#pragma unroll
    for (int i = 0; i < N; ++i) r.e[i] = e[i];
    r.store(p);
  }
};

// ---- cross-lane reductions -------------------------------------------------

template <int CTRL> __device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}

// Sum over the 16 lanes of a DPP row; every lane of the row receives it.
__device__ __forceinline__ float row_sum16(float x) {
  x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp<0x141>(x);  // row_half_mirror
  x += dpp<0x140>(x);  // row_mirror
  return x;
}

// Sum over a quad of lanes (lane & ~3 .. lane | 3).
__device__ __forceinline__ float quad_sum(float x) {
  x += dpp<0xB1>(x);  // quad_perm [1,0,3,2]
  x += dpp<0x4E>(x);  // quad_perm [2,3,0,1]
  return x;
}

// The row exchanges are gfx950's permlane swaps: swapping a register with a
// copy of itself leaves the partner row's value in one of the two results,
// so a pair sum is one swap and one add (no LDS round trip).
__device__ __forceinline__ float pair_rows_sum(float x) {  // rows (0,1) and (2,3)
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float half_waves_sum(float x) {  // lanes l and l ^ 32
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Sum over the 4 rows (lanes l, l^16, l^32, l^48); every lane receives it.
__device__ __forceinline__ float cross_row_sum(float x) { return half_waves_sum(pair_rows_sum(x)); }

// Inclusive scan over the 4 rows (row r receives x_0 + ... + x_r of its
// column) and the total of all four rows.
__device__ __forceinline__ float rows_scan(float x, int row, float& total) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  // r[0] holds the even row of the pair, r[1] the odd one, in both rows of the pair
  const float ev = __uint_as_float(r[0]), od = __uint_as_float(r[1]);
  const float pair = ev + od;
  const float in_pair = (row & 1) ? pair : ev;
  const auto h = __builtin_amdgcn_permlane32_swap(__float_as_uint(pair), __float_as_uint(pair), false, false);
  const float lo = __uint_as_float(h[0]), hi = __uint_as_float(h[1]);  // pair totals of rows 0-1 and 2-3
  total = lo + hi;
  return in_pair + (row >= 2 ? lo : 0.f);
}

__device__ __forceinline__ float wave_sum(float x) { return cross_row_sum(row_sum16(x)); }

// Maximum over the 64 lanes of a wave; every lane receives it.
__device__ __forceinline__ float wave_max(float x) {
  x = fmaxf(x, dpp<0xB1>(x));   // quad_perm [1,0,3,2]
  x = fmaxf(x, dpp<0x4E>(x));   // quad_perm [2,3,0,1]
  x = fmaxf(x, dpp<0x141>(x));  // row_half_mirror
  x = fmaxf(x, dpp<0x140>(x));  // row_mirror
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  const auto h = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(h[0]), __uint_as_float(h[1]));
}

// Entry i of a byte table in the kernel's by-value arguments, for a
// wave-uniform i: read as its aligned 32-bit word, which is a scalar load.
// There is no scalar byte load on this target, so indexing the table
// directly becomes a vector load whose wait delays every load after it.
__device__ __forceinline__ int arg_byte(const uint8_t* table, int i) {
  const uint32_t w = reinterpret_cast<const uint32_t*>(table)[i >> 2];
  return (int)((w >> (8 * (i & 3))) & 0xffu);
}

__device__ __forceinline__ float lane_bcast(float x, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), lane));
}

// Order LDS traffic between lanes of one wave (writes before later reads).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Workgroup barrier for LDS traffic only: waits for this wave's LDS (and
// scalar) operations, then meets the other waves.  Unlike __syncthreads it
// leaves this wave's global loads in flight, so a kernel can keep a large
// read outstanding while its waves exchange staged data through LDS.  The
// memory clobber keeps the compiler from moving memory operations across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Compiler-only fence: memory operations stay on their side of it.
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

__device__ __forceinline__ float fast_exp(float x) { return __expf(x); }

}  // namespace skssm

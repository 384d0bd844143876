// Maps a runtime shape to its compiled kernel instantiation and launches it.
// Compiled shapes: (K, V) in {(64,64), (128,64), (128,128)}; R in {8, 16, 32, K}
// (update also R = 0); windows up to 16 or 32 slots; fp32 or bf16 io; fp32 or
// bf16 sketch.
#pragma once

#include <hip/hip_runtime.h>

#include "decode.h"
#include "update.h"

namespace skssm {

constexpr int kUnsupported = -2;

// LDS of one gfx950 CU, shared by the workgroups resident on it.
constexpr size_t kLdsPerCU = 160 * 1024;

// Dynamic LDS (unused by the kernel) that holds a kernel to at most `cap`
// resident workgroups per CU: each then takes more than a (cap + 1)-th of the
// CU's LDS.  Zero where the kernel's static LDS already does that, or if its
// attributes cannot be read (the launch then runs uncapped).
template <typename Kernel>
size_t lds_for_cap(Kernel kern, int cap) {
  hipFuncAttributes at;
  if (hipFuncGetAttributes(&at, reinterpret_cast<const void*>(kern)) != hipSuccess) return 0;
  const size_t need = kLdsPerCU / (size_t)(cap + 1) + 1024;
  return need > at.sharedSizeBytes ? need - at.sharedSizeBytes : 0;
}

// Resident workgroups per CU for the kernels that read each item's state and
// write it back in place (the flush with the offline map or none, and the
// single-token update).  With more of these streams resident per CU the
// in-place stream measured slower: the flush took 431 / 456 us (Mamba-2 at six
// per CU, GDN at four; B = 256 / 512) against 387 / 435 us at three, and the
// Mamba-2 single-token update 391 us at eight against 342 us at two.  The
// flushes that build a state-dependent map and the decode do arithmetic or
// wait on latency between their loads and keep their occupancy (capping them
// measured slower), as does the initial sketch (a read of the state, run once
// after prefill).
constexpr int kFlushPerCU = 3;
constexpr int kTokenPerCU = 2;

template <int KIND, int K, int V, int R, int WM, typename IO, typename SK, int P>
int launch_decode(const DecodeArgs& a, hipStream_t s) {
  const unsigned tiles = (unsigned)((a.B + 3) / 4);
  if (a.ndense > 0)
    hipLaunchKernelGGL((decode_kernel<KIND, K, V, R, WM, IO, SK, P, true>), dim3((unsigned)a.H * tiles), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((decode_kernel<KIND, K, V, R, WM, IO, SK, P, false>), dim3((unsigned)a.H * tiles), dim3(256), 0, s, a);
  return 0;
}

template <int KIND, int K, int V, int WM, typename IO>
int launch_full_read(const DecodeArgs& a, hipStream_t s) {
  const size_t items = (size_t)a.B * a.H;
  hipLaunchKernelGGL((full_read_kernel<KIND, K, V, WM, IO>), dim3((unsigned)((items + 3) / 4)), dim3(256), 0, s, a);
  return 0;
}

template <int KIND, int K, int V, int R, int WM, typename IO, typename SK, int P>
int launch_update(const UpdateArgs& a, hipStream_t s) {
  const size_t items = (size_t)a.B * a.H;
  static const size_t cap = P == 0 ? lds_for_cap(&update_kernel<KIND, K, V, R, WM, IO, SK, P>, kFlushPerCU) : 0;
  hipLaunchKernelGGL((update_kernel<KIND, K, V, R, WM, IO, SK, P>), dim3((unsigned)items), dim3(256), a.nt > 0 ? cap : 0,
                     s, a);
  return 0;
}

// State-dependent maps: piv = 4 (P = 4 pivots) is compiled for ranks 8..32,
// piv = -1 (the exact metric, flush only: decode reads either map the same
// way) for ranks 8 and 16.
template <int R> constexpr bool kPivotRank = R >= 8 && R <= 32;
template <int R> constexpr bool kExactRank = R == 8 || R == 16;

template <int KIND, int K, int V, int R, int WM, int P>
int decode_t(const DecodeArgs& a, int io, int sk, hipStream_t s) {
  if (io) return sk ? launch_decode<KIND, K, V, R, WM, bf16_t, bf16_t, P>(a, s) : launch_decode<KIND, K, V, R, WM, bf16_t, float, P>(a, s);
  return sk ? launch_decode<KIND, K, V, R, WM, float, bf16_t, P>(a, s) : launch_decode<KIND, K, V, R, WM, float, float, P>(a, s);
}

template <int KIND, int K, int V, int R>
int decode_w(const DecodeArgs& a, int io, int sk, int piv, hipStream_t s) {
  if constexpr (kPivotRank<R>) {
    if (piv) return a.W <= 16 ? decode_t<KIND, K, V, R, 16, 4>(a, io, sk, s) : decode_t<KIND, K, V, R, 32, 4>(a, io, sk, s);
  } else {
    if (piv) return kUnsupported;
  }
  return a.W <= 16 ? decode_t<KIND, K, V, R, 16, 0>(a, io, sk, s) : decode_t<KIND, K, V, R, 32, 0>(a, io, sk, s);
}

// One (kind, K, V) shape; explicitly instantiated in its own translation unit.
template <int KIND, int K, int V>
int decode_r(const DecodeArgs& a, int R, int io, int sk, int piv, hipStream_t s) {
  switch (R) {
    case 8: return decode_w<KIND, K, V, 8>(a, io, sk, piv, s);
    case 16: return decode_w<KIND, K, V, 16>(a, io, sk, piv, s);
    case 32: return decode_w<KIND, K, V, 32>(a, io, sk, piv, s);
    case K: return decode_w<KIND, K, V, K>(a, io, sk, piv, s);
    default: return kUnsupported;
  }
}

template <int KIND>
int run_decode(const DecodeArgs& a, int K, int V, int R, int io, int sk, int piv, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (K == 64 && V == 64) return decode_r<KIND, 64, 64>(a, R, io, sk, piv, s);
  if (K == 128 && V == 64) return decode_r<KIND, 128, 64>(a, R, io, sk, piv, s);
  if (K == 128 && V == 128) return decode_r<KIND, 128, 128>(a, R, io, sk, piv, s);
  return kUnsupported;
}

template <int KIND, int K, int V>
int full_read_w(const DecodeArgs& a, int io, hipStream_t s) {
  if (a.W <= 16)
    return io ? launch_full_read<KIND, K, V, 16, bf16_t>(a, s) : launch_full_read<KIND, K, V, 16, float>(a, s);
  return io ? launch_full_read<KIND, K, V, 32, bf16_t>(a, s) : launch_full_read<KIND, K, V, 32, float>(a, s);
}

template <int KIND>
int run_full_read(const DecodeArgs& a, int K, int V, int io, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (K == 64 && V == 64) return full_read_w<KIND, 64, 64>(a, io, s);
  if (K == 128 && V == 64) return full_read_w<KIND, 128, 64>(a, io, s);
  if (K == 128 && V == 128) return full_read_w<KIND, 128, 128>(a, io, s);
  return kUnsupported;
}

template <int KIND, int K, int V, typename IO>
int launch_token(const UpdateArgs& a, hipStream_t s) {
  const size_t items = (size_t)a.B * a.H;
  // (the erase families' single-token update holds more registers per lane and
  // measured the same at two to five resident workgroups per CU)
  static const size_t cap = KIND == MAMBA2 ? lds_for_cap(&token_kernel<KIND, K, V, IO>, kTokenPerCU) : 0;
  hipLaunchKernelGGL((token_kernel<KIND, K, V, IO>), dim3((unsigned)items), dim3(256), cap, s, a);
  return 0;
}

template <int KIND, int K, int V, int R, int WM, int P>
int update_t(const UpdateArgs& a, int io, int sk, hipStream_t s) {
  if constexpr (R == 0) {  // no sketch: its dtype does not matter
    // a single token (window-1 decoding, or a window flushed after its first
    // token): the rank-1 update streams the state through registers
    if (a.nt == 1) return io ? launch_token<KIND, K, V, bf16_t>(a, s) : launch_token<KIND, K, V, float>(a, s);
    return io ? launch_update<KIND, K, V, 0, WM, bf16_t, float, 0>(a, s) : launch_update<KIND, K, V, 0, WM, float, float, 0>(a, s);
  } else {
    if (io) return sk ? launch_update<KIND, K, V, R, WM, bf16_t, bf16_t, P>(a, s) : launch_update<KIND, K, V, R, WM, bf16_t, float, P>(a, s);
    return sk ? launch_update<KIND, K, V, R, WM, float, bf16_t, P>(a, s) : launch_update<KIND, K, V, R, WM, float, float, P>(a, s);
  }
}

template <int KIND, int K, int V, int R>
int update_w(const UpdateArgs& a, int io, int sk, int piv, hipStream_t s) {
  if constexpr (kExactRank<R>) {
    if (piv < 0) return a.W <= 16 ? update_t<KIND, K, V, R, 16, -1>(a, io, sk, s) : update_t<KIND, K, V, R, 32, -1>(a, io, sk, s);
  }
  if constexpr (kPivotRank<R>) {
    if (piv > 0) return a.W <= 16 ? update_t<KIND, K, V, R, 16, 4>(a, io, sk, s) : update_t<KIND, K, V, R, 32, 4>(a, io, sk, s);
  }
  if (piv) return kUnsupported;
  return a.W <= 16 ? update_t<KIND, K, V, R, 16, 0>(a, io, sk, s) : update_t<KIND, K, V, R, 32, 0>(a, io, sk, s);
}

// One (kind, K, V) shape; explicitly instantiated in its own translation unit.
template <int KIND, int K, int V>
int update_r(const UpdateArgs& a, int R, int io, int sk, int piv, hipStream_t s) {
  switch (R) {
    case 0: return update_w<KIND, K, V, 0>(a, io, sk, piv, s);
    case 8: return update_w<KIND, K, V, 8>(a, io, sk, piv, s);
    case 16: return update_w<KIND, K, V, 16>(a, io, sk, piv, s);
    case 32: return update_w<KIND, K, V, 32>(a, io, sk, piv, s);
    case K: return update_w<KIND, K, V, K>(a, io, sk, piv, s);
    default: return kUnsupported;
  }
}

template <int KIND>
int run_update(const UpdateArgs& a, int K, int V, int R, int io, int sk, int piv, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (K == 64 && V == 64) return update_r<KIND, 64, 64>(a, R, io, sk, piv, s);
  if (K == 128 && V == 64) return update_r<KIND, 128, 64>(a, R, io, sk, piv, s);
  if (K == 128 && V == 128) return update_r<KIND, 128, 128>(a, R, io, sk, piv, s);
  return kUnsupported;
}

}  // namespace skssm

// Kernel argument blocks (passed by value to the kernels).
//
// Replay buffer (ring): slot s of item i (= b*H + h) of a field of width w
// sits at field + (i * W + s) * w for the raw inputs (item-major) and at
// field + (s * B*H + h * B + b) * w for the derived fields (slot-major,
// head-major within a slot, so the four items of a decode workgroup, one head
// and four consecutive requests, are adjacent).
// Raw inputs of token s (k, v, beta, log decay) are written into slot s by
// the producer of the token; the kernels derive and store the rest.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace skssm {

// Per-head rank table (head_rank in the config), by value: hrank[h] = G_h
// (0 = dense fallback) when `ragged`; otherwise every head has the class rank.
constexpr int kMaxRaggedHeads = 256;

struct DecodeArgs {
  int B, H, W, n;                 // batch, heads, window, slot of the current token
  int ragged;                     // hrank holds the per-head ranks
  alignas(4) uint8_t hrank[kMaxRaggedHeads];
  int ndense;                     // dense-fallback heads (ragged)
  alignas(4) uint8_t hlist[kMaxRaggedHeads];  // heads in launch order: the dense ones first (ragged)
  const void* q;                  // [B][H][K] io, current query
  const void* U;                  // [B][H][R/P][V][P], P = 4 (fp32) or 8 (bf16)  (sketch read)
  const float* coef;              // [H][R][K]           (sketch read, offline map; NULL with a state-dependent map)
  const void* cmap;               // [B][H][K/CPW][R][CPW] state-dependent map, sketch dtype, CPW = 16 B / element (or NULL)
  const float* S;                 // [B][H][V][K]        (exact baseline)
  const void* rk;                 // ring [B][H][W][K] io      raw keys
  const void* rv;                 // ring [B][H][W][V] io      raw values
  const float* rbeta;             // ring [B][H][W]            write gates
  const float* rla;               // ring [B][H][W] or [..][K] log decays
  void* rf;                       // ring [W][H][B][R]  projected erase factors, sketch dtype (GDN/KDA sketch read)
  float* rpi;                     // ring [W][H][B][K]  erase factors (GDN/KDA baseline)
  float* rt;                      // ring [W][H][B][W]  rows of T^{-1} (GDN/KDA)
  float* o;                       // [B][H][V]
};

struct UpdateArgs {
  int B, H, W, n;                 // n = slot of the current token (tokens applied: n + 1)
  int ragged;                     // hrank holds the per-head ranks
  alignas(4) uint8_t hrank[kMaxRaggedHeads];
  int nt;                         // n + 1, or 0 (sketch only)
  float* S;                       // [B][H][V][K]
  const float* omega;             // [H][K][R]
  const void* q;                  // [B][H][K] io, current query (NULL when nt == 0)
  const void* rk;
  const void* rv;
  const float* rbeta;
  const float* rla;
  const float* rt;                // GDN/KDA rows of T^{-1}, slots < n
  void* U;                        // [B][H][R/P][V][P], P = 4 (fp32) or 8 (bf16), or NULL
  void* cmap;                     // [B][H][K/CPW][R][CPW] state-dependent map, sketch dtype, or NULL
  float ridge;                    // its lambda
  float* o;                       // [B][H][V] or NULL
};

// Host-side entry points of the per-family translation units.  Each returns
// 0 after a launch, or -2 when the shape has no compiled kernel.
int run_decode_mamba2(const DecodeArgs& a, int K, int V, int R, int io, int sk, int piv, void* stream);
int run_decode_gdn(const DecodeArgs& a, int K, int V, int R, int io, int sk, int piv, void* stream);
int run_decode_kda(const DecodeArgs& a, int K, int V, int R, int io, int sk, int piv, void* stream);
int run_full_read_mamba2(const DecodeArgs& a, int K, int V, int io, void* stream);
int run_full_read_gdn(const DecodeArgs& a, int K, int V, int io, void* stream);
int run_full_read_kda(const DecodeArgs& a, int K, int V, int io, void* stream);
int run_update_mamba2(const UpdateArgs& a, int K, int V, int R, int io, int sk, int piv, void* stream);
int run_update_gdn(const UpdateArgs& a, int K, int V, int R, int io, int sk, int piv, void* stream);
int run_update_kda(const UpdateArgs& a, int K, int V, int R, int io, int sk, int piv, void* stream);
// State layout conversion (row layout <-> tile-major), items states of V x K.
int run_state_layout(const float* src, float* dst, size_t items, int K, int V, int to_tiles, void* stream);

}  // namespace skssm

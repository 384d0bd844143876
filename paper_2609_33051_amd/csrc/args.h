// Kernel argument blocks (passed by value to the kernels).
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace skssm {

struct DecodeArgs {
  int B, H, W, n;                 // batch, heads, window, slot being appended
  const void* q;                  // [B][H][K] io
  const void* k;                  // [B][H][K] io
  const void* v;                  // [B][H][V] io
  const float* beta;              // [B][H]
  const float* logd;              // [B][H] or [B][H][K]
  const float* U;                 // [B][H][V][R]       (sketch read)
  const float* coef;              // [H][R][K]          (sketch read)
  const float* S;                 // [B][H][V][K]       (exact baseline)
  void* rk;                       // ring [B][H][W][K] io
  void* rv;                       // ring [B][H][W][V] io   (Mamba-2)
  float* ru;                      // ring [B][H][W][V]      (GDN/KDA)
  float* rf;                      // ring [B][H][W][R]      (GDN/KDA sketch read)
  float* rpi;                     // ring [B][H][W][K]      (GDN/KDA baseline)
  float* rg;                      // ring [B][H][W] or [B][H][W][K]
  float* rbeta;                   // ring [B][H][W]
  float* rb;                      // ring [B][H][W][W]      (GDN/KDA)
  float* o;                       // [B][H][V]
};

struct UpdateArgs {
  int B, H, W, n;                 // n = ring slots already filled (0..W-1)
  int nt;                         // tokens applied: n + 1, or 0 (sketch only)
  float* S;                       // [B][H][V][K]
  const float* omega;             // [H][K][R]
  const void* rk;
  const void* rv;
  const float* ru;
  const float* rg;
  const float* rbeta;
  const float* rb;
  const void* q;                  // current token (NULL when nt == 0)
  const void* k;
  const void* v;
  const float* beta;
  const float* logd;
  float* U;                       // [B][H][V][R] or NULL
  float* o;                       // [B][H][V] or NULL
};

// Host-side entry points of the per-family translation units.  Each returns
// 0 after a launch, or -2 when the shape has no compiled kernel.
int run_decode_mamba2(const DecodeArgs& a, int K, int V, int R, int io, void* stream);
int run_decode_gdn(const DecodeArgs& a, int K, int V, int R, int io, void* stream);
int run_decode_kda(const DecodeArgs& a, int K, int V, int R, int io, void* stream);
int run_full_read_mamba2(const DecodeArgs& a, int K, int V, int io, void* stream);
int run_full_read_gdn(const DecodeArgs& a, int K, int V, int io, void* stream);
int run_full_read_kda(const DecodeArgs& a, int K, int V, int io, void* stream);
int run_update_mamba2(const UpdateArgs& a, int K, int V, int R, int io, void* stream);
int run_update_gdn(const UpdateArgs& a, int K, int V, int R, int io, void* stream);
int run_update_kda(const UpdateArgs& a, int K, int V, int R, int io, void* stream);

}  // namespace skssm

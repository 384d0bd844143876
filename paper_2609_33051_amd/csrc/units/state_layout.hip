// Conversion of the recurrent state between the row layout X[v][k] (X = S^T,
// the transpose of the paper's K x V state, per item) and the tile-major
// layout the kernels read and write: 16 x 16 tiles (vt, kt), vt-major, each
// 1 KB contiguous with lane l of a wave holding X[16 vt + l%16][16 kt +
// 4 (l/16) + i] at 4 l + i (the register layout of the flush's MFMA
// accumulators).  A pure permutation of float4s: one thread per float4.
#include <hip/hip_runtime.h>

#include "../args.h"

namespace skssm {

__global__ __launch_bounds__(256) void state_layout_kernel(const float4* src, float4* dst, size_t n4, int K, int V,
                                                           int to_tiles) {
  const uint32_t MT = (uint32_t)K / 16;
  const size_t per = (size_t)V * K / 4;  // float4s per item
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (size_t)gridDim.x * 256) {
    const size_t item = i / per;
    const uint32_t j = (uint32_t)(i - item * per);           // tiled float4 index within the item
    const uint32_t blk = j >> 6, l = j & 63, vt = blk / MT, kt = blk - vt * MT;
    const uint32_t v = 16 * vt + (l & 15), k = 16 * kt + 4 * (l >> 4);
    const size_t r = item * per + (v * (uint32_t)K + k) / 4;  // row-layout float4 index
    if (to_tiles)
      dst[i] = src[r];
    else
      dst[r] = src[i];
  }
}

int run_state_layout(const float* src, float* dst, size_t items, int K, int V, int to_tiles, void* stream) {
  if (K % 16 || V % 16) return -2;
  const size_t n4 = items * (size_t)V * K / 4;
  const size_t blocks = (n4 + 255) / 256;
  const unsigned grid = (unsigned)(blocks < 16384 ? blocks : 16384);  // grid-stride beyond
  hipLaunchKernelGGL(state_layout_kernel, dim3(grid), dim3(256), 0, static_cast<hipStream_t>(stream),
                     reinterpret_cast<const float4*>(src), reinterpret_cast<float4*>(dst), n4, K, V, to_tiles);
  return 0;
}

}  // namespace skssm

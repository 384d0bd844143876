// Instantiations: non-flush sketch read, mamba2.
#include "../dispatch.h"
namespace skssm {
int run_decode_mamba2(const DecodeArgs& a, int K, int V, int R, int io, int sk, void* stream) {
  return run_decode<MAMBA2>(a, K, V, R, io, sk, stream);
}
}  // namespace skssm

// Instantiations: non-flush sketch read, kda.
#include "../dispatch.h"
namespace skssm {
int run_decode_kda(const DecodeArgs& a, int K, int V, int R, int io, int sk, void* stream) {
  return run_decode<KDA>(a, K, V, R, io, sk, stream);
}
}  // namespace skssm

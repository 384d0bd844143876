// Instantiations: non-flush sketch read, gdn.
#include "../dispatch.h"
namespace skssm {
int run_decode_gdn(const DecodeArgs& a, int K, int V, int R, int io, int sk, void* stream) {
  return run_decode<GDN>(a, K, V, R, io, sk, stream);
}
}  // namespace skssm

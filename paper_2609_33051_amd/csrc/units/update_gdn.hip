// Instantiations: flush / initial sketch, gdn.
#include "../dispatch.h"
namespace skssm {
int run_update_gdn(const UpdateArgs& a, int K, int V, int R, int io, int sk, void* stream) {
  return run_update<GDN>(a, K, V, R, io, sk, stream);
}
}  // namespace skssm

// Instantiations: flush / initial sketch, kda.
#include "../dispatch.h"
namespace skssm {
int run_update_kda(const UpdateArgs& a, int K, int V, int R, int io, int sk, void* stream) {
  return run_update<KDA>(a, K, V, R, io, sk, stream);
}
}  // namespace skssm

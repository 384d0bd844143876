// Instantiations: flush / initial sketch, mamba2.
#include "../dispatch.h"
namespace skssm {
int run_update_mamba2(const UpdateArgs& a, int K, int V, int R, int io, int sk, void* stream) {
  return run_update<MAMBA2>(a, K, V, R, io, sk, stream);
}
}  // namespace skssm

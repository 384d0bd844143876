// Instantiations: exact full-state-read baseline, kda.
#include "../dispatch.h"
namespace skssm {
int run_full_read_kda(const DecodeArgs& a, int K, int V, int io, void* stream) {
  return run_full_read<KDA>(a, K, V, io, stream);
}
}  // namespace skssm

// Instantiations: exact full-state-read baseline, mamba2.
#include "../dispatch.h"
namespace skssm {
int run_full_read_mamba2(const DecodeArgs& a, int K, int V, int io, void* stream) {
  return run_full_read<MAMBA2>(a, K, V, io, stream);
}
}  // namespace skssm

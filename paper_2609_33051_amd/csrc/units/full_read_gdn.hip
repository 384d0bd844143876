// Instantiations: exact full-state-read baseline, gdn.
#include "../dispatch.h"
namespace skssm {
int run_full_read_gdn(const DecodeArgs& a, int K, int V, int io, void* stream) {
  return run_full_read<GDN>(a, K, V, io, stream);
}
}  // namespace skssm

// Instantiations: non-flush sketch read, mamba2, K = 64, V = 64.
#include "../dispatch.h"
namespace skssm {
template int decode_r<MAMBA2, 64, 64>(const DecodeArgs&, int, int, int, int, hipStream_t);
}  // namespace skssm

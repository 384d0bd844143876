// Instantiations: non-flush sketch read, mamba2, K = 128, V = 128.
#include "../dispatch.h"
namespace skssm {
template int decode_r<MAMBA2, 128, 128>(const DecodeArgs&, int, int, int, int, hipStream_t);
}  // namespace skssm

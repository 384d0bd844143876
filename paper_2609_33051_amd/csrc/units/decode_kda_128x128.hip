// Instantiations: non-flush sketch read, kda, K = 128, V = 128.
#include "../dispatch.h"
namespace skssm {
template int decode_r<KDA, 128, 128>(const DecodeArgs&, int, int, int, int, hipStream_t);
}  // namespace skssm

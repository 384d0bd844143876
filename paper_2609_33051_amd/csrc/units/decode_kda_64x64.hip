// Instantiations: non-flush sketch read, kda, K = 64, V = 64.
#include "../dispatch.h"
namespace skssm {
template int decode_r<KDA, 64, 64>(const DecodeArgs&, int, int, int, int, hipStream_t);
}  // namespace skssm

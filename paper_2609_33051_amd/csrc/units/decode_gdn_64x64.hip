// Instantiations: non-flush sketch read, gdn, K = 64, V = 64.
#include "../dispatch.h"
namespace skssm {
template int decode_r<GDN, 64, 64>(const DecodeArgs&, int, int, int, int, hipStream_t);
}  // namespace skssm

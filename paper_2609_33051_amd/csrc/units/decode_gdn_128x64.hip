// Instantiations: non-flush sketch read, gdn, K = 128, V = 64.
#include "../dispatch.h"
namespace skssm {
template int decode_r<GDN, 128, 64>(const DecodeArgs&, int, int, int, int, hipStream_t);
}  // namespace skssm

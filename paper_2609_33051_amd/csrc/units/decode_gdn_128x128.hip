// Instantiations: non-flush sketch read, gdn, K = 128, V = 128.
#include "../dispatch.h"
namespace skssm {
template int decode_r<GDN, 128, 128>(const DecodeArgs&, int, int, int, int, hipStream_t);
}  // namespace skssm

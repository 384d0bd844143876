// Instantiations: flush / initial sketch, gdn, K = 128, V = 128.
#include "../dispatch.h"
namespace skssm {
template int update_r<GDN, 128, 128>(const UpdateArgs&, int, int, int, int, hipStream_t);
}  // namespace skssm

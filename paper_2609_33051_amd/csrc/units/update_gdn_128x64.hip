// Instantiations: flush / initial sketch, gdn, K = 128, V = 64.
#include "../dispatch.h"
namespace skssm {
template int update_r<GDN, 128, 64>(const UpdateArgs&, int, int, int, int, hipStream_t);
}  // namespace skssm

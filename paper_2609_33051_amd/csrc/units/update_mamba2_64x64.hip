// Instantiations: flush / initial sketch, mamba2, K = 64, V = 64.
#include "../dispatch.h"
namespace skssm {
template int update_r<MAMBA2, 64, 64>(const UpdateArgs&, int, int, int, int, hipStream_t);
}  // namespace skssm

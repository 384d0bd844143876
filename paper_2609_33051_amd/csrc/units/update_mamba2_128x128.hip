// Instantiations: flush / initial sketch, mamba2, K = 128, V = 128.
#include "../dispatch.h"
namespace skssm {
template int update_r<MAMBA2, 128, 128>(const UpdateArgs&, int, int, int, int, hipStream_t);
}  // namespace skssm

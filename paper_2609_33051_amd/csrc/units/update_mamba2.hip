// Dispatch of the flush / initial sketch kernels, mamba2; the shapes are compiled in
// update_mamba2_<K>x<V>.hip.
#include "../dispatch.h"
namespace skssm {
extern template int update_r<MAMBA2, 64, 64>(const UpdateArgs&, int, int, int, int, hipStream_t);
extern template int update_r<MAMBA2, 128, 64>(const UpdateArgs&, int, int, int, int, hipStream_t);
extern template int update_r<MAMBA2, 128, 128>(const UpdateArgs&, int, int, int, int, hipStream_t);
int run_update_mamba2(const UpdateArgs& a, int K, int V, int R, int io, int sk, int piv, void* stream) {
  return run_update<MAMBA2>(a, K, V, R, io, sk, piv, stream);
}
}  // namespace skssm

// Dispatch of the flush / initial sketch kernels, kda; the shapes are compiled in
// update_kda_<K>x<V>.hip.
#include "../dispatch.h"
namespace skssm {
extern template int update_r<KDA, 64, 64>(const UpdateArgs&, int, int, int, int, hipStream_t);
extern template int update_r<KDA, 128, 64>(const UpdateArgs&, int, int, int, int, hipStream_t);
extern template int update_r<KDA, 128, 128>(const UpdateArgs&, int, int, int, int, hipStream_t);
int run_update_kda(const UpdateArgs& a, int K, int V, int R, int io, int sk, int piv, void* stream) {
  return run_update<KDA>(a, K, V, R, io, sk, piv, stream);
}
}  // namespace skssm

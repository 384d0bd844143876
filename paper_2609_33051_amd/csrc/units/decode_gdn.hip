// Dispatch of the non-flush sketch read kernels, gdn; the shapes are compiled in
// decode_gdn_<K>x<V>.hip.
#include "../dispatch.h"
namespace skssm {
extern template int decode_r<GDN, 64, 64>(const DecodeArgs&, int, int, int, int, hipStream_t);
extern template int decode_r<GDN, 128, 64>(const DecodeArgs&, int, int, int, int, hipStream_t);
extern template int decode_r<GDN, 128, 128>(const DecodeArgs&, int, int, int, int, hipStream_t);
int run_decode_gdn(const DecodeArgs& a, int K, int V, int R, int io, int sk, int piv, void* stream) {
  return run_decode<GDN>(a, K, V, R, io, sk, piv, stream);
}
}  // namespace skssm

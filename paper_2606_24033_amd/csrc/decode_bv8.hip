// Packed decode instantiation for value code width 8 (see decode_impl.h).
#include "decode_impl.h"

namespace bgtq {
hipError_t launch_split_bv8(const Dims& d, const void* layout, const void* q, const int32_t* ctx_len,
                            const CachePtrs& c, float* out, const DecodeWs& ws, hipStream_t s) {
  return split_detail::launch_split_bv_impl<8>(d, layout, q, ctx_len, c, out, ws, s);
}
}  // namespace bgtq

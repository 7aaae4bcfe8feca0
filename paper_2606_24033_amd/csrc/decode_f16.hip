// The fp16 comparator decode (decode_impl.h, k_f16_mfma).
#include "decode_impl.h"

namespace bgtq {
hipError_t launch_decode_fp16(const Dims& d, const void* q, const int32_t* ctx_len, const void* k16,
                              const void* v16, float* out, const DecodeWs& ws, hipStream_t s) {
  return split_detail::launch_f16_mfma_impl(d, q, ctx_len, k16, v16, out, ws, s);
}
}  // namespace bgtq

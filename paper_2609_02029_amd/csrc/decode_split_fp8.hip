// decode_split_fp8.hip -- decode split kernels for fp8-E4M3 caches (the
// matrix-core kernel of decode_mfma.h; all head dims and group sizes).
#include "decode_split.h"

namespace hwkv {
template hipError_t launch_decode_split_fmt<HWKV_KV_FP8_E4M3>(int, int, const DecodeArgs &, int,
                                                              hipStream_t, hipEvent_t, hipEvent_t);
}  // namespace hwkv

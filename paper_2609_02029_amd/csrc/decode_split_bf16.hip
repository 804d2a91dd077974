// decode_split_bf16.hip -- decode split kernels for bf16 caches (all head
// dims and group sizes).
#include "decode_split.h"

namespace hwkv {
template hipError_t launch_decode_split_fmt<HWKV_KV_BF16>(int, int, const DecodeArgs &, int,
                                                          hipStream_t, hipEvent_t, hipEvent_t);
}  // namespace hwkv

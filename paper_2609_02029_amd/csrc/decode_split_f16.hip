// decode_split_f16.hip -- decode split kernels for IEEE binary16 caches (all head
// dims and group sizes).
#include "decode_split.h"

namespace hwkv {
template hipError_t launch_decode_split_fmt<HWKV_KV_F16>(int, int, const DecodeArgs &, int,
                                                         hipStream_t, hipEvent_t, hipEvent_t);
}  // namespace hwkv

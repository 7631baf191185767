// The decode kernels for bf16 K/V caches, and the entry points that pick the
// instantiation for a call's K/V element type.
#include "decode_impl.h"

namespace dsa {

hipError_t launch_decode(const Derived& d, const DecodeArgs& a, hipStream_t st, hipEvent_t t0,
                         hipEvent_t t1) {
  if (a.kv_dtype == DSA_KV_FP8_E4M3) return launch_kv_fp8(d, a, st, t0, t1, false);
  return launch_kv<KvBf16>(d, a, st, t0, t1, false);
}

hipError_t launch_step(const Derived& d, const DecodeArgs& a, hipStream_t st, hipEvent_t t0,
                       hipEvent_t t1) {
  if (a.kv_dtype == DSA_KV_FP8_E4M3) return launch_kv_fp8(d, a, st, t0, t1, true);
  return launch_kv<KvBf16>(d, a, st, t0, t1, true);
}

}  // namespace dsa

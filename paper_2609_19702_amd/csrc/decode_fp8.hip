// The decode kernels for fp8 (OCP E4M3) K/V caches.
#include "decode_impl.h"

namespace dsa {

hipError_t launch_kv_fp8(const Derived& d, const DecodeArgs& a, hipStream_t st, hipEvent_t t0,
                         hipEvent_t t1, bool fused) {
  return launch_kv<KvFp8>(d, a, st, t0, t1, fused);
}

}  // namespace dsa

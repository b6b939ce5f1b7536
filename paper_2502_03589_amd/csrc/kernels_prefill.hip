// Prefill attention on quantized Q/K/V/P (Sec. 5.3 with L_Q = L_KV; Eq. 2-4).
#include "hack_internal.hpp"

namespace hack {

hipError_t launch_prefill(const hack_kv_layout& lay, const CacheView& c, const __half* q, int num_q_heads,
                          int batch, int len, int causal, float* out, hipStream_t stream) {
  (void)lay; (void)c; (void)q; (void)num_q_heads; (void)batch; (void)len; (void)causal; (void)out; (void)stream;
  return hipErrorNotSupported;
}

}  // namespace hack

// Prefill path entry.  Large batches currently run the same fused
// dequantize x matrix-vector kernels as decode (correct for any bucket size,
// weights read once per bucket).
#include "internal.h"

namespace moeq {

hipError_t launch_gateup_prefill(const DecodeArgs& a, hipStream_t s) { return launch_gateup_decode(a, s); }

hipError_t launch_down_prefill(const DecodeArgs& a, hipStream_t s) { return launch_down_decode(a, s); }

}  // namespace moeq

// Prefill path entry.  Large batches currently run the same fused
// dequantize x matrix-vector kernels as decode (correct for any bucket size,
// weights read once per bucket).
#include "internal.h"

namespace moeq {

hipError_t launch_prefill(const DecodeArgs& a, hipStream_t s) { return launch_decode(a, s); }

}  // namespace moeq

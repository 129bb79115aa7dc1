// Expert importance for pruning (Section 3.1 of arXiv 2509.25689).
//
// Statistics of the unpruned router over calibration tokens: an expert's
// activation frequency f_e (tokens that selected it / tokens) and its mean
// routing score when selected, sbar_e; importance I_e = alpha f_e +
// (1 - alpha) sbar_e; the ceil(rE) most important experts are kept.
//
// The routing and the bucketing are the forward's own kernels (route.hip);
// with renormalisation off and scale 1 the router's weights are the sigmoid
// scores.  Each expert then sums its bucket's scores in float32 in token
// order (the bucket lists its tokens ascending), so the result does not
// depend on scheduling.  f_e and sbar_e are float32 quotients; I_e is formed
// in float64 with explicitly rounded operations (no contraction), and the
// ranking is by I_e descending, lower id first on ties.
#include "internal.h"

namespace moeq {

namespace {

__global__ __launch_bounds__(256) void fill_u8_kernel(uint8_t* p, int n, uint8_t v) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}

// Host values handed to the device through the kernel arguments, which the
// launch copies: the caller's buffer may change as soon as the launch returns.
constexpr int kArgFloats = 256;
struct HostFloats {
  float v[kArgFloats];
};
__global__ __launch_bounds__(kArgFloats) void store_floats_kernel(float* dst, int n, HostFloats src) {
  const int i = threadIdx.x;
  if (i < n) dst[i] = src.v[i];
}

__global__ __launch_bounds__(256) void expert_stats_kernel(const int32_t* offsets, const int32_t* perm,
                                                           const float* w, int E, int n, double alpha,
                                                           double* importance, int32_t* counts) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= E) return;
  const int b = offsets[e], c = offsets[e + 1] - b;
  float sum = 0.0f;
  for (int p = 0; p < c; ++p) sum = __fadd_rn(sum, w[perm[b + p]]);
  const float f = __fdiv_rn((float)c, (float)n);
  const float sbar = c > 0 ? __fdiv_rn(sum, (float)c) : 0.0f;
  const double t1 = __dmul_rn(alpha, (double)f);
  const double t2 = __dmul_rn(__dsub_rn(1.0, alpha), (double)sbar);
  importance[e] = __dadd_rn(t1, t2);
  if (counts) counts[e] = c;
}

// one workgroup: rank of every expert among all E, kept if rank < keep
__global__ __launch_bounds__(1024) void select_kernel(const double* importance, int E, int keep, uint8_t* mask) {
  __shared__ double imp[kMaxExperts];
  for (int e = threadIdx.x; e < E; e += 1024) imp[e] = importance[e];
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += 1024) {
    const double v = imp[e];
    int rank = 0;
    for (int o = 0; o < E; ++o) rank += (imp[o] > v || (imp[o] == v && o < e)) ? 1 : 0;
    mask[e] = rank < keep ? 1 : 0;
  }
}

}  // namespace

hipError_t launch_fill_u8(uint8_t* p, int n, uint8_t v, hipStream_t s) {
  fill_u8_kernel<<<(n + 255) / 256, 256, 0, s>>>(p, n, v);
  return hipGetLastError();
}

hipError_t launch_store_host_floats(float* dst, const float* src, int n, hipStream_t s) {
  for (int i = 0; i < n; i += kArgFloats) {
    HostFloats h{};
    const int m = n - i < kArgFloats ? n - i : kArgFloats;
    for (int j = 0; j < m; ++j) h.v[j] = src ? src[i + j] : 0.0f;
    store_floats_kernel<<<1, kArgFloats, 0, s>>>(dst + i, m, h);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_expert_importance(const int32_t* offsets, const int32_t* perm, const float* w, int E, int n,
                                    double alpha, int keep, double* importance, uint8_t* mask, int32_t* counts,
                                    hipStream_t s) {
  expert_stats_kernel<<<(E + 255) / 256, 256, 0, s>>>(offsets, perm, w, E, n, alpha, importance, counts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  select_kernel<<<1, 1024, 0, s>>>(importance, E, keep, mask);
  return hipGetLastError();
}

}  // namespace moeq

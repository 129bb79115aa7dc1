// Router gate: the affinities the router of Sections 3.1 and 3.2 turns into
// scores, logits = x W_r^T, with x bfloat16 [n x H], W_r float32 [E x H] and
// logits float32 [n x E].  Products and sums are float32 and every logit is
// accumulated in an order fixed by (n <= kGateFewTokens, H), so a forward is
// deterministic.
//
// Few tokens (decode): one workgroup per expert.  Thread t owns the float4
// columns t, t + 256, ... of the expert's row, keeps one partial sum per
// token, and the 256 partials are reduced by a fixed tree (DPP within a
// wave, then the four waves in order).  The row of W_r is streamed once.
//
// Many tokens (prefill): 64 tokens x 64 experts per workgroup, 32-wide K
// slices of x and W_r staged k-major in LDS, 4 x 4 logits per thread, each
// a single fused multiply-add chain over k = 0 .. H-1.
#include "internal.h"
#include "layout.h"

namespace moeq {

namespace {

__device__ __forceinline__ float wave_sum(float v) {
  v += __shfl_xor(v, 1, 64);
  v += __shfl_xor(v, 2, 64);
  v += __shfl_xor(v, 4, 64);
  v += __shfl_xor(v, 8, 64);
  v += __shfl_xor(v, 16, 64);
  v += __shfl_xor(v, 32, 64);
  return v;
}

// grid = E workgroups of 256 threads; H a multiple of 128, n <= kGateFewTokens
__global__ __launch_bounds__(256) void gate_few_kernel(const uint16_t* x, const float* w, int n, int H, int E,
                                                      float* logits) {
  __shared__ float part[4][kGateFewTokens];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int e = blockIdx.x;
  const int C = H / 4;  // float4 columns
  const MOEQ_GLOBAL f32x4* wr = gptr(reinterpret_cast<const f32x4*>(w + (size_t)e * H));
  const MOEQ_GLOBAL u32x2* xg = gptr(reinterpret_cast<const u32x2*>(x));
  float acc[kGateFewTokens];
#pragma unroll
  for (int t = 0; t < kGateFewTokens; ++t) acc[t] = 0.0f;
  // H <= 8192 gives at most 8 columns per thread: load them all, then use them
  constexpr int kMaxCols = 8;
  f32x4 wv[kMaxCols];
#pragma unroll
  for (int i = 0; i < kMaxCols; ++i) {
    const int c = tid + 256 * i;
    wv[i] = c < C ? __builtin_nontemporal_load(wr + c) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  }
#pragma unroll
  for (int t = 0; t < kGateFewTokens; ++t) {
    if (t < n) {
      float a = 0.0f;
#pragma unroll
      for (int i = 0; i < kMaxCols; ++i) {
        const int c = tid + 256 * i;
        if (c < C) {
          const u32x2 p = xg[(size_t)t * C + c];
          a = fmaf(bf16_lo(p.x), wv[i].x, a);
          a = fmaf(bf16_hi(p.x), wv[i].y, a);
          a = fmaf(bf16_lo(p.y), wv[i].z, a);
          a = fmaf(bf16_hi(p.y), wv[i].w, a);
        }
      }
      acc[t] = a;
    }
  }
#pragma unroll
  for (int t = 0; t < kGateFewTokens; ++t) {
    if (t < n) {
      const float v = wave_sum(acc[t]);
      if (lane == 0) part[wave][t] = v;
    }
  }
  __syncthreads();
  if (tid < n) logits[(size_t)tid * E + e] = ((part[0][tid] + part[1][tid]) + part[2][tid]) + part[3][tid];
}

constexpr int kTB = 64, kTK = 32, kTP = kTB + 4;

// grid = (ceil(E / 64), ceil(n / 64)) workgroups of 256 threads; H a multiple of 32
__global__ __launch_bounds__(256) void gate_tiled_kernel(const uint16_t* x, const float* w, int n, int H, int E,
                                                        float* logits) {
  __shared__ __align__(16) float xs[kTK][kTP];
  __shared__ __align__(16) float ws[kTK][kTP];
  const int tid = threadIdx.x;
  const int e0 = blockIdx.x * kTB, t0 = blockIdx.y * kTB;
  const int ty = tid >> 4, tx = tid & 15;  // logits (t0 + 4 ty + i, e0 + 4 tx + j)
  // x loader: token tid / 4, k = 8 (tid % 4) .. + 7 (one 16-byte load)
  const int xl_t = tid >> 2, xl_k = (tid & 3) * 8;
  const MOEQ_GLOBAL u32x4* xrow =
      gptr(reinterpret_cast<const u32x4*>(x + (size_t)min(t0 + xl_t, n - 1) * H + xl_k));
  // W loader: experts tid / 8 and tid / 8 + 32, k = 4 (tid % 8) .. + 3
  const int wl_e = tid >> 3, wl_k = (tid & 7) * 4;
  const MOEQ_GLOBAL f32x4* wrow0 =
      gptr(reinterpret_cast<const f32x4*>(w + (size_t)min(e0 + wl_e, E - 1) * H + wl_k));
  const MOEQ_GLOBAL f32x4* wrow1 =
      gptr(reinterpret_cast<const f32x4*>(w + (size_t)min(e0 + wl_e + 32, E - 1) * H + wl_k));
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0f;
  for (int k0 = 0; k0 < H; k0 += kTK) {
    const u32x4 xv = xrow[k0 / 8];
    const f32x4 w0 = wrow0[k0 / 4], w1 = wrow1[k0 / 4];
    __syncthreads();
    xs[xl_k + 0][xl_t] = bf16_lo(xv.x);
    xs[xl_k + 1][xl_t] = bf16_hi(xv.x);
    xs[xl_k + 2][xl_t] = bf16_lo(xv.y);
    xs[xl_k + 3][xl_t] = bf16_hi(xv.y);
    xs[xl_k + 4][xl_t] = bf16_lo(xv.z);
    xs[xl_k + 5][xl_t] = bf16_hi(xv.z);
    xs[xl_k + 6][xl_t] = bf16_lo(xv.w);
    xs[xl_k + 7][xl_t] = bf16_hi(xv.w);
    ws[wl_k + 0][wl_e] = w0.x;
    ws[wl_k + 1][wl_e] = w0.y;
    ws[wl_k + 2][wl_e] = w0.z;
    ws[wl_k + 3][wl_e] = w0.w;
    ws[wl_k + 0][wl_e + 32] = w1.x;
    ws[wl_k + 1][wl_e + 32] = w1.y;
    ws[wl_k + 2][wl_e + 32] = w1.z;
    ws[wl_k + 3][wl_e + 32] = w1.w;
    __syncthreads();
#pragma unroll 8
    for (int k = 0; k < kTK; ++k) {
      const f32x4 a = *reinterpret_cast<const f32x4*>(&xs[k][ty * 4]);
      const f32x4 b = *reinterpret_cast<const f32x4*>(&ws[k][tx * 4]);
      const float av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = t0 + ty * 4 + i;
    if (t >= n) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = e0 + tx * 4 + j;
      if (e < E) logits[(size_t)t * E + e] = acc[i][j];
    }
  }
}

}  // namespace

hipError_t launch_router_gate(const uint16_t* x, const float* w, int n, int H, int E, float* logits,
                              hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n <= kGateFewTokens) {
    gate_few_kernel<<<E, 256, 0, s>>>(x, w, n, H, E, logits);
  } else {
    dim3 grid((E + kTB - 1) / kTB, (n + kTB - 1) / kTB);
    gate_tiled_kernel<<<grid, 256, 0, s>>>(x, w, n, H, E, logits);
  }
  return hipGetLastError();
}

}  // namespace moeq

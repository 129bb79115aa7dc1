// Measured roofline denominators (include/moeq_peaks.h): a streaming read of
// device memory and a register-only loop of binary16 matrix instructions.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "moeq_peaks.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kReadThreads = 256;
constexpr int kReadUnroll = 8;  // 16-byte loads in flight per thread
constexpr size_t kBytesPerWg = (size_t)kReadThreads * kReadUnroll * 16;

// Workgroup w reads the contiguous bytes [w * kBytesPerWg, +kBytesPerWg):
// load i of thread t is the 16 bytes at (i * 256 + t) * 16, so every load
// instruction of a wave covers 1 KiB contiguously; all kReadUnroll loads are
// issued before the first is used.  The tail workgroup checks bounds.
__global__ __launch_bounds__(kReadThreads) void stream_read_kernel(const u32x4* src, size_t n16, uint32_t* sink) {
  const size_t base = (size_t)blockIdx.x * (kReadThreads * kReadUnroll) + threadIdx.x;
  u32x4 v[kReadUnroll];
#pragma unroll
  for (int i = 0; i < kReadUnroll; ++i) {
    const size_t j = base + (size_t)i * kReadThreads;
    v[i] = j < n16 ? __builtin_nontemporal_load(src + j) : u32x4{0u, 0u, 0u, 0u};
  }
  uint32_t x = 0;
#pragma unroll
  for (int i = 0; i < kReadUnroll; ++i) x ^= v[i].x ^ v[i].y ^ v[i].z ^ v[i].w;
  __shared__ uint32_t red[kReadThreads / 64];
  for (int off = 32; off > 0; off >>= 1) x ^= __shfl_xor(x, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

// 4 independent accumulator chains per wave of v_mfma_f32_32x32x16_f16 (the
// shape the grouped GEMMs issue), so that the issue of one MFMA never waits
// on the result of the previous one.
constexpr int kChains = 4;
__global__ __launch_bounds__(256) void mfma_loop_kernel(int iters, float* sink) {
  const int lane = threadIdx.x & 63;
  half8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (_Float16)(0.001f * (float)((lane + i) & 7));
    b[i] = (_Float16)(0.001f * (float)((lane * 3 + i) & 7));
  }
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[c][v] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += acc[c][v];
  sink[(size_t)blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace

extern "C" {

int moeq_peaks_read_workgroups(size_t n_bytes) { return (int)((n_bytes + kBytesPerWg - 1) / kBytesPerWg); }

int moeq_peaks_stream_read(const void* src, size_t n_bytes, uint32_t* sink, void* stream) {
  if (!src || !sink || (n_bytes & 15) || ((uintptr_t)src & 15)) return (int)hipErrorInvalidValue;
  const int grid = moeq_peaks_read_workgroups(n_bytes);
  if (grid == 0) return 0;
  stream_read_kernel<<<grid, kReadThreads, 0, (hipStream_t)stream>>>((const u32x4*)src, n_bytes / 16, sink);
  return (int)hipGetLastError();
}

int moeq_peaks_mfma(int workgroups, int iters, float* sink, void* stream) {
  if (!sink || workgroups < 1 || iters < 1) return (int)hipErrorInvalidValue;
  mfma_loop_kernel<<<workgroups, 256, 0, (hipStream_t)stream>>>(iters, sink);
  return (int)hipGetLastError();
}

double moeq_peaks_mfma_flops(int workgroups, int iters) {
  return (double)workgroups * 4.0 * iters * kChains * 2.0 * 32 * 32 * 16;
}

}  // extern "C"

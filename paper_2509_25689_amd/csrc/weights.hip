// Weight-format kernels: canonical packing -> device layout (repack), device
// layout -> float32 through each decoder the products use (diagnostics), and
// float32 -> canonical packing (quantize).
//
// The format is the symmetric block format standing in for the paper's
// per-tensor low-bit formats (Section 3.3): weight = d * (c - 2^(b-1)), one
// binary16 scale d per 32 weights, b-bit codes packed least significant bit
// first within each block.
#include "internal.h"
#include "layout.h"

namespace moeq {

namespace {

// codes of one block (32 values < 2^b) -> its b device dwords
template <int B>
__device__ void encode_block(const uint8_t* c, uint32_t* w) {
  for (int d = 0; d < B; ++d) w[d] = 0u;
  if constexpr (B == 8) {
    uint8_t lo[32], hi[32];
    for (int i = 0; i < 32; ++i) {
      lo[i] = c[i] & 15;
      hi[i] = c[i] >> 4;
    }
    encode_block<4>(lo, w);
    encode_block<4>(hi, w + 4);
  } else if constexpr (B == 6) {
    for (int d = 0; d < 6; ++d)
      for (int f = 0; f < 2; ++f)
        w[d] |= (uint32_t)c[4 * d + 2 * f] << (6 * f) | (uint32_t)c[4 * d + 2 * f + 1] << (16 + 6 * f);
    for (int m = 0; m < 4; ++m) {
      const uint32_t c0 = c[24 + 2 * m], c1 = c[25 + 2 * m];
      w[m] |= (c0 & 15u) << 12 | (c1 & 15u) << 28;
      const int sh = 12 + 2 * (m & 1);
      w[4 + m / 2] |= (c0 >> 4) << sh | (c1 >> 4) << (16 + sh);
    }
  } else if constexpr (B == 5) {
    for (int d = 0; d < 5; ++d)
      for (int f = 0; f < 3; ++f)
        w[d] |= (uint32_t)c[6 * d + 2 * f] << (5 * f) | (uint32_t)c[6 * d + 2 * f + 1] << (16 + 5 * f);
    for (int q = 0; q < 5; ++q)
      w[q] |= ((uint32_t)(c[30] >> q) & 1u) << 15 | ((uint32_t)(c[31] >> q) & 1u) << 31;
  } else if constexpr (B == 4) {
    for (int d = 0; d < 4; ++d)
      for (int s = 0; s < 4; ++s)
        w[d] |= (uint32_t)c[8 * d + 2 * s] << (4 * s) | (uint32_t)c[8 * d + 2 * s + 1] << (16 + 4 * s);
  } else if constexpr (B == 2) {
    for (int d = 0; d < 2; ++d)
      for (int s = 0; s < 8; ++s)
        w[d] |= (uint32_t)c[16 * d + 2 * s] << (2 * s) |
                (uint32_t)c[16 * d + 2 * s + 1] << (16 + 2 * s);
  } else {
    for (int d = 0; d < 3; ++d)
      for (int f = 0; f < 5; ++f)
        w[d] |= (uint32_t)c[10 * d + 2 * f] << (3 * f) |
                (uint32_t)c[10 * d + 2 * f + 1] << (16 + 3 * f);
    for (int q = 0; q < 3; ++q)
      w[q] |= ((uint32_t)(c[30] >> q) & 1u) << 15 | ((uint32_t)(c[31] >> q) & 1u) << 31;
  }
}

// one thread per (row, unit): read 4 canonical blocks, write b 16-byte chunks
template <int B>
__global__ __launch_bounds__(256) void repack_kernel(const uint8_t* canon, int rows, int K,
                                                     uint32_t* dev) {
  const int U = K / kUnit;
  const long long gid = (long long)blockIdx.x * 256 + threadIdx.x;
  if (gid >= (long long)rows * U) return;
  const int r = (int)(gid / U), u = (int)(gid % U);
  const uint8_t* src = canon + ((size_t)r * (K / kBlock) + 4 * u) * 4 * B;  // 16*B bytes
  uint8_t c[kUnit];
  for (int i = 0; i < kUnit; ++i) {
    const int bit = i * B;
    const uint32_t lo = src[bit >> 3], hi = (bit >> 3) + 1 < 16 * B ? src[(bit >> 3) + 1] : 0u;
    c[i] = (uint8_t)(((lo | hi << 8) >> (bit & 7)) & ((1u << B) - 1u));
  }
  uint32_t w[4 * B];
  for (int q = 0; q < 4; ++q) encode_block<B>(c + 32 * q, w + q * B);
  uint32_t* row = dev + (size_t)r * B * U * 4;
  for (int j = 0; j < B; ++j)
    for (int e = 0; e < 4; ++e) row[((size_t)j * U + u) * 4 + e] = w[4 * j + e];
}

// one thread per (row, unit): the bfloat16-form unpacking of block_pairs
// (the 5/6/8-bit matrix-vector kernels), then
// d * (c - 2^(b-1)) exactly
template <int B>
__global__ __launch_bounds__(256) void dequant_kernel(TensorDev t, float* out) {
  const int U = t.K / kUnit;
  const long long gid = (long long)blockIdx.x * 256 + threadIdx.x;
  if (gid >= (long long)t.rows * U) return;
  const int r = (int)(gid / U), u = (int)(gid % U);
  uint32_t w[4 * B];
  load_unit<B>(t.codes + (size_t)r * B * U * 4, U, u, w);
  const uint16_t* sc = t.scales + (size_t)r * (t.K / kBlock) + 4 * u;
  const float z = (float)(1 << (B - 1)), unit = (float)(1 << (B <= 7 ? 7 - B : 0));
  float* o = out + (size_t)r * t.K + kUnit * u;
  const PairConsts pk = pair_consts();
  for (int q = 0; q < 4; ++q) {
    const float d = half_to_float(sc[q]);
    if constexpr (B == 8) {
      uint32_t pl[16], ph[16];
      block_pairs<4>(w + 8 * q, pk, pl);
      block_pairs<4>(w + 8 * q + 4, pk, ph);
      for (int P = 0; P < 16; ++P) {
        const float c0 = (bf16_lo(ph[P]) - 128.0f) * 2.0f + (bf16_lo(pl[P]) - 128.0f) / 8.0f;
        const float c1 = (bf16_hi(ph[P]) - 128.0f) * 2.0f + (bf16_hi(pl[P]) - 128.0f) / 8.0f;
        o[32 * q + 2 * P] = d * (c0 - z);
        o[32 * q + 2 * P + 1] = d * (c1 - z);
      }
    } else {
      uint32_t p[16];
      block_pairs<B>(w + q * B, pk, p);
      for (int P = 0; P < 16; ++P) {
        const float c0 = (bf16_lo(p[P]) - 128.0f) / unit, c1 = (bf16_hi(p[P]) - 128.0f) / unit;
        o[32 * q + 2 * P] = d * (c0 - z);
        o[32 * q + 2 * P + 1] = d * (c1 - z);
      }
    }
  }
}

// one thread per (row, unit): the binary16-subnormal code pairs of
// block_pairs_sub (the one-token gate/up and the 2-4-bit down matrix-vector
// kernels).  Pair P's two halves are c * 2^(k-24) with k = sub_shift<B>(P);
// c is rebuilt exactly as that value times 2^(24-k), then d * (c - 2^(b-1)).
template <int B>
__global__ __launch_bounds__(256) void dequant_sub_kernel(TensorDev t, float* out) {
  const int U = t.K / kUnit;
  const long long gid = (long long)blockIdx.x * 256 + threadIdx.x;
  if (gid >= (long long)t.rows * U) return;
  const int r = (int)(gid / U), u = (int)(gid % U);
  uint32_t w[4 * B];
  load_unit<B>(t.codes + (size_t)r * B * U * 4, U, u, w);
  const uint16_t* sc = t.scales + (size_t)r * (t.K / kBlock) + 4 * u;
  const float z = (float)(1 << (B - 1));
  float* o = out + (size_t)r * t.K + kUnit * u;
  for (int q = 0; q < 4; ++q) {
    const float d = half_to_float(sc[q]);
    uint32_t p[16];
    block_pairs_sub<B>(w + q * B, p);
#pragma unroll
    for (int P = 0; P < 16; ++P) {
      const float up = __builtin_amdgcn_ldexpf(1.0f, 24 - sub_shift<B>(P));
      const float c0 = half_to_float(p[P] & 0xFFFFu) * up, c1 = half_to_float(p[P] >> 16) * up;
      o[32 * q + 2 * P] = d * (c0 - z);
      o[32 * q + 2 * P + 1] = d * (c1 - z);
    }
  }
}

// float64 -> binary16 bit pattern, round to nearest even; v >= 0
__device__ uint16_t half_rne_from_double(double v) {
  if (!(v > 0.0)) return 0;
  if (v >= 65520.0) return 0x7C00;  // at or above the midpoint to 2^16: infinity
  int ex;
  frexp(v, &ex);
  int e2 = ex - 1;  // v in [2^e2, 2^(e2+1))
  if (e2 < -14) return (uint16_t)rint(ldexp(v, 24));  // subnormal, units of 2^-24 (1024 = min normal)
  double m = rint(ldexp(v, 10 - e2));               // in [1024, 2048]
  if (m == 2048.0) {
    m = 1024.0;
    ++e2;
  }
  return (uint16_t)(((e2 + 15) << 10) | ((int)m - 1024));
}

// one thread per block of 32
__global__ __launch_bounds__(256) void quantize_kernel(const float* w, int rows, int K, int bits,
                                                       uint8_t* codes, uint16_t* scales) {
  const int nb = K / kBlock;
  const long long gid = (long long)blockIdx.x * 256 + threadIdx.x;
  if (gid >= (long long)rows * nb) return;
  const float* src = w + gid * kBlock;  // row-major, blocks contiguous
  float amax = 0.0f;
  for (int i = 0; i < kBlock; ++i) amax = fmaxf(amax, fabsf(src[i]));
  const int qm = (1 << (bits - 1)) - 1, z = 1 << (bits - 1);
  const uint16_t hb = half_rne_from_double((double)amax / (double)qm);
  scales[gid] = hb;
  const double d = (double)half_to_float(hb);
  uint32_t acc[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};  // 32 * bits <= 256 bits
  for (int i = 0; i < kBlock; ++i) {
    int q = 0;
    if (d > 0.0) {
      const double qq = rint((double)src[i] / d);
      q = (int)fmin(fmax(qq, (double)-qm), (double)qm);
    }
    const uint32_t c = (uint32_t)(q + z);
    const int bit = i * bits;
    acc[bit >> 5] |= c << (bit & 31);
    if ((bit & 31) + bits > 32) acc[(bit >> 5) + 1] |= c >> (32 - (bit & 31));
  }
  uint8_t* dst = codes + gid * 4 * bits;
  for (int i = 0; i < 4 * bits; ++i) dst[i] = (uint8_t)(acc[i >> 2] >> (8 * (i & 3)));
}

}  // namespace

hipError_t launch_repack(const uint8_t* canon, int rows, int K, int bits, uint32_t* dev,
                         hipStream_t s) {
  const long long n = (long long)rows * (K / kUnit);
  const int grid = (int)((n + 255) / 256);
  switch (bits) {
    case 2: repack_kernel<2><<<grid, 256, 0, s>>>(canon, rows, K, dev); break;
    case 3: repack_kernel<3><<<grid, 256, 0, s>>>(canon, rows, K, dev); break;
    case 4: repack_kernel<4><<<grid, 256, 0, s>>>(canon, rows, K, dev); break;
    case 5: repack_kernel<5><<<grid, 256, 0, s>>>(canon, rows, K, dev); break;
    case 6: repack_kernel<6><<<grid, 256, 0, s>>>(canon, rows, K, dev); break;
    case 8: repack_kernel<8><<<grid, 256, 0, s>>>(canon, rows, K, dev); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

namespace {
__device__ __forceinline__ uint32_t scale_key(uint32_t v) {
  const uint32_t mag = v & 0x7FFFu;
  return (v & 0x8000u) || mag == 0 || mag >= 0x7C00u ? 0xFFFFu : mag;
}

// 8 scales per thread and load, a workgroup maximum in LDS, one atomic per
// workgroup
__global__ __launch_bounds__(256) void scale_key_max_kernel(const uint16_t* sc, size_t n, uint32_t* out) {
  __shared__ uint32_t wmax[4];
  uint32_t m = 0;
  const size_t n8 = n / 8;
  const u32x4* s8 = reinterpret_cast<const u32x4*>(sc);
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n8; i += (size_t)gridDim.x * 256) {
    const u32x4 v = s8[i];
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) m = max(m, max(scale_key(w[j] & 0xFFFFu), scale_key(w[j] >> 16)));
  }
  for (size_t i = n8 * 8 + (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256)
    m = max(m, scale_key(sc[i]));
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off, 64));
  if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    m = max(max(wmax[0], wmax[1]), max(wmax[2], wmax[3]));
    if (m) atomicMax(out, m);
  }
}
}  // namespace

hipError_t launch_scale_key_max(const uint16_t* scales, size_t n, uint32_t* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  // the scales are 256-byte aligned in the layer's store (16-byte loads)
  const size_t want = (n / 8 + 255) / 256 + 1;
  const int grid = (int)(want < 256 ? want : 256);
  scale_key_max_kernel<<<grid, 256, 0, s>>>(scales, n, out);
  return hipGetLastError();
}

hipError_t launch_dequant_sub(const TensorDev& t, float* out, hipStream_t s) {
  const long long n = (long long)t.rows * (t.K / kUnit);
  const int grid = (int)((n + 255) / 256);
  switch (t.bits) {
    case 2: dequant_sub_kernel<2><<<grid, 256, 0, s>>>(t, out); break;
    case 3: dequant_sub_kernel<3><<<grid, 256, 0, s>>>(t, out); break;
    case 4: dequant_sub_kernel<4><<<grid, 256, 0, s>>>(t, out); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_dequant(const TensorDev& t, float* out, hipStream_t s) {
  const long long n = (long long)t.rows * (t.K / kUnit);
  const int grid = (int)((n + 255) / 256);
  switch (t.bits) {
    case 2: dequant_kernel<2><<<grid, 256, 0, s>>>(t, out); break;
    case 3: dequant_kernel<3><<<grid, 256, 0, s>>>(t, out); break;
    case 4: dequant_kernel<4><<<grid, 256, 0, s>>>(t, out); break;
    case 5: dequant_kernel<5><<<grid, 256, 0, s>>>(t, out); break;
    case 6: dequant_kernel<6><<<grid, 256, 0, s>>>(t, out); break;
    case 8: dequant_kernel<8><<<grid, 256, 0, s>>>(t, out); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_quantize(const float* w, int rows, int K, int bits, uint8_t* codes,
                           uint16_t* scales, hipStream_t s) {
  const long long n = (long long)rows * (K / kBlock);
  quantize_kernel<<<(int)((n + 255) / 256), 256, 0, s>>>(w, rows, K, bits, codes, scales);
  return hipGetLastError();
}

}  // namespace moeq

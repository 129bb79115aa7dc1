// Device layout of the quantized weights and the code-to-bfloat16 unpacking
// shared by the repack, dequantize and matrix-vector kernels.
//
// The value of a weight is d * (c - 2^(b-1)) with a binary16 block scale d
// and a b-bit code c (the symmetric block format this library uses for the
// per-tensor low bit widths of Section 3.3).  On the device a row is cut into
// units of 128 weights (four blocks of 32).  A unit is 4*b dwords; block q of
// the unit is dwords [q*b, q*b + b), encoded so that two codes -- those of
// weights 2i and 2i+1 -- sit at the same offset of the low and high 16-bit
// halves of one dword:
//
//   b = 4: dword d (0..3) holds weights 8d..8d+7: weight 8d+2s in bits
//          [4s, 4s+4), weight 8d+2s+1 in bits [16+4s, 20+4s), s = 0..3
//   b = 2: dword d (0..1) holds weights 16d..16d+15: weight 16d+2s in bits
//          [2s, 2s+2), weight 16d+2s+1 in bits [16+2s, 18+2s), s = 0..7
//   b = 3: dword d (0..2) holds weights 10d..10d+9: weight 10d+2f in bits
//          [3f, 3f+3), weight 10d+2f+1 in bits [16+3f, 19+3f), f = 0..4;
//          bit q of weight 30 is bit 15 of dword q, bit q of weight 31 is
//          bit 31 of dword q (q = 0..2)
//
// Unpacking moves a code pair to the top of the 7-bit bfloat16 mantissa and
// ORs in the exponent of 128 (one shift and one v_and_or_b32 per pair): the
// dword is then two bfloat16 values 128 + c * 2^(7-b), exact, ready for
// v_dot2_f32_bf16 against a pair of activations.  Since
//   sum_i (128 + 2^(7-b) c_i) x_i = 2^(7-b) * sum_i (c_i - z) x_i + 192 * sum_i x_i
// with z = 2^(b-1), a block's contribution is
//   d * 2^(b-7) * (dot - 192 * X),     X = sum of the block's 32 activations.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moeq {

constexpr uint32_t kBf16Base = 0x43004300u;  // bfloat16 128.0 in both halves

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Global (not generic) address space: pointers read from the descriptor
// table would otherwise become flat loads, which also count against the LDS
// wait counter and serialize HBM streaming with LDS reads.
#define MOEQ_GLOBAL __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ const MOEQ_GLOBAL T* gptr(const T* p) {
  return (const MOEQ_GLOBAL T*)p;
}

// (a & m) | c as one v_and_or_b32.  gfx9 VOP3 cannot encode literals, so the
// constants are passed in VGPRs (see the masks below) and the instruction is
// written out; the compiler otherwise splits it into v_and + v_or.
__device__ __forceinline__ uint32_t and_or(uint32_t a, uint32_t m, uint32_t c) {
  uint32_t r;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(m), "v"(c));
  return r;
}

// Masks and the bfloat16 base held in registers for and_or.
struct PairConsts {
  uint32_t base, m2, m3, m4, b30, b31, b32;
};
__device__ __forceinline__ PairConsts pair_consts() {
  PairConsts k;
  // opaque moves keep the constants in VGPRs
  asm("v_mov_b32 %0, 0x43004300" : "=v"(k.base));
  asm("v_mov_b32 %0, 0x00600060" : "=v"(k.m2));
  asm("v_mov_b32 %0, 0x00700070" : "=v"(k.m3));
  asm("v_mov_b32 %0, 0x00780078" : "=v"(k.m4));
  asm("v_mov_b32 %0, 0x00100010" : "=v"(k.b30));
  asm("v_mov_b32 %0, 0x00200020" : "=v"(k.b31));
  asm("v_mov_b32 %0, 0x00400040" : "=v"(k.b32));
  return k;
}

// shift a dword left (s > 0) or right (s < 0); s is a compile-time constant
template <int S>
__device__ __forceinline__ uint32_t shl(uint32_t v) {
  if constexpr (S >= 0)
    return v << S;
  else
    return v >> (-S);
}

// The 16 code pairs of one block (P = pair index = weights 2P, 2P+1), each as
// two bfloat16 values 128 + c * 2^(7-b).
template <int B>
__device__ __forceinline__ void block_pairs(const uint32_t* w, const PairConsts& k, uint32_t (&p)[16]);

template <>
__device__ __forceinline__ void block_pairs<4>(const uint32_t* w, const PairConsts& k, uint32_t (&p)[16]) {
  // mask m4: bits [3,7) of each half
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    p[4 * d + 0] = and_or(shl<3>(w[d]), k.m4, k.base);
    p[4 * d + 1] = and_or(shl<-1>(w[d]), k.m4, k.base);
    p[4 * d + 2] = and_or(shl<-5>(w[d]), k.m4, k.base);
    p[4 * d + 3] = and_or(shl<-9>(w[d]), k.m4, k.base);
  }
}

template <>
__device__ __forceinline__ void block_pairs<2>(const uint32_t* w, const PairConsts& k, uint32_t (&p)[16]) {
  // mask m2: bits [5,7) of each half
#pragma unroll
  for (int d = 0; d < 2; ++d) {
    p[8 * d + 0] = and_or(shl<5>(w[d]), k.m2, k.base);
    p[8 * d + 1] = and_or(shl<3>(w[d]), k.m2, k.base);
    p[8 * d + 2] = and_or(shl<1>(w[d]), k.m2, k.base);
    p[8 * d + 3] = and_or(shl<-1>(w[d]), k.m2, k.base);
    p[8 * d + 4] = and_or(shl<-3>(w[d]), k.m2, k.base);
    p[8 * d + 5] = and_or(shl<-5>(w[d]), k.m2, k.base);
    p[8 * d + 6] = and_or(shl<-7>(w[d]), k.m2, k.base);
    p[8 * d + 7] = and_or(shl<-9>(w[d]), k.m2, k.base);
  }
}

template <>
__device__ __forceinline__ void block_pairs<3>(const uint32_t* w, const PairConsts& k, uint32_t (&p)[16]) {
  // mask m3: bits [4,7) of each half
#pragma unroll
  for (int d = 0; d < 3; ++d) {
    p[5 * d + 0] = and_or(shl<4>(w[d]), k.m3, k.base);
    p[5 * d + 1] = and_or(shl<1>(w[d]), k.m3, k.base);
    p[5 * d + 2] = and_or(shl<-2>(w[d]), k.m3, k.base);
    p[5 * d + 3] = and_or(shl<-5>(w[d]), k.m3, k.base);
    p[5 * d + 4] = and_or(shl<-8>(w[d]), k.m3, k.base);
  }
  uint32_t t = and_or(shl<-11>(w[0]), k.b30, k.base);
  t = and_or(shl<-10>(w[1]), k.b31, t);
  p[15] = and_or(shl<-9>(w[2]), k.b32, t);
}

// 5-bit blocks: dword d (0..4) holds pairs 3d + f (f = 0..2), the even code
// of a pair at bits [5f, 5f+5) of the low half, the odd one in the high half;
// pair 15 (codes 30, 31) is spread over bit 15 (code 30) and bit 31 (code 31)
// of the five dwords, bit q of each code in dword q.
template <>
__device__ __forceinline__ void block_pairs<5>(const uint32_t* w, const PairConsts& k, uint32_t (&p)[16]) {
  uint32_t m5, b0, b1;
  asm("v_mov_b32 %0, 0x007C007C" : "=v"(m5));  // bits [2,7) of each half
  asm("v_mov_b32 %0, 0x00040004" : "=v"(b0));
  asm("v_mov_b32 %0, 0x00080008" : "=v"(b1));
#pragma unroll
  for (int d = 0; d < 5; ++d) {
    p[3 * d + 0] = and_or(shl<2>(w[d]), m5, k.base);
    p[3 * d + 1] = and_or(shl<-3>(w[d]), m5, k.base);
    p[3 * d + 2] = and_or(shl<-8>(w[d]), m5, k.base);
  }
  // bit q of the spare bits goes to mantissa bit 2 + q of each half
  uint32_t t = and_or(shl<-13>(w[0]), b0, k.base);
  t = and_or(shl<-12>(w[1]), b1, t);
  t = and_or(shl<-11>(w[2]), k.b30, t);
  t = and_or(shl<-10>(w[3]), k.b31, t);
  p[15] = and_or(shl<-9>(w[4]), k.b32, t);
}

// 6-bit blocks: dword d (0..5) holds pairs 2d + f (f = 0, 1) at bits
// [6f, 6f+6) of each half; pairs 12 + m (m = 0..3) keep their codes' low
// four bits in bits [12,16) of each half of dword m and their top two bits in
// bits [12 + 2(m&1), 14 + 2(m&1)) of each half of dword 4 + m/2.
template <>
__device__ __forceinline__ void block_pairs<6>(const uint32_t* w, const PairConsts& k, uint32_t (&p)[16]) {
  uint32_t m6, lo4;
  asm("v_mov_b32 %0, 0x007E007E" : "=v"(m6));   // bits [1,7) of each half
  asm("v_mov_b32 %0, 0x001E001E" : "=v"(lo4));  // bits [1,5)
#pragma unroll
  for (int d = 0; d < 6; ++d) {
    p[2 * d + 0] = and_or(shl<1>(w[d]), m6, k.base);
    p[2 * d + 1] = and_or(shl<-5>(w[d]), m6, k.base);
  }
  // top two bits to mantissa bits [5,7) (mask m2)
  p[12] = and_or(shl<-7>(w[4]), k.m2, and_or(shl<-11>(w[0]), lo4, k.base));
  p[13] = and_or(shl<-9>(w[4]), k.m2, and_or(shl<-11>(w[1]), lo4, k.base));
  p[14] = and_or(shl<-7>(w[5]), k.m2, and_or(shl<-11>(w[2]), lo4, k.base));
  p[15] = and_or(shl<-9>(w[5]), k.m2, and_or(shl<-11>(w[3]), lo4, k.base));
}

// Code pairs as binary16 subnormals (widths 2-4, the gate/up and down
// GEMVs): a dword masked so that only one code pair remains, at bit
// offset k of each half, with the exponent fields zero, is two binary16 values
// c * 2^(k - 24), exact, for v_dot2_f32_f16 (which keeps subnormal inputs).
// The layout puts several pairs at offsets inside the 10-bit mantissa, so most
// pairs need a mask alone and the others one shift per dword:
//   b = 4: offsets 0, 4 of w and of w >> 8           (k = 0, 4, 0, 4)
//   b = 3: offsets 0, 3, 6 of w and 0, 3 of w >> 9  (k = 0, 3, 6, 0, 3);
//          the spare pair 15 is gathered at offset 0
//   b = 2: offsets 0, 2, 4, 6, 8 of w and 0, 2, 4 of w >> 10
// The dot of a block keeps one sum per offset k and scales the sums by 2^-k
// when the block is done; there is no offset to cancel.
template <int B>
constexpr int sub_shift(int P) {  // k of pair P (0..15)
  if constexpr (B == 4) return (P & 1) ? 4 : 0;
  if constexpr (B == 3) return P == 15 ? 0 : (P % 5 == 1 || P % 5 == 4) ? 3 : (P % 5 == 2) ? 6 : 0;
  return P % 8 < 5 ? 2 * (P % 8) : 2 * (P % 8 - 5);
}
template <int B>
constexpr int sub_step() { return B == 4 ? 4 : B == 3 ? 3 : 2; }  // offsets are multiples of it
template <int B>
constexpr int sub_classes() { return B == 4 ? 2 : B == 3 ? 3 : 5; }  // distinct offsets

template <int B>
__device__ __forceinline__ void block_pairs_sub(const uint32_t* w, uint32_t (&p)[16]) {
  static_assert(B >= 2 && B <= 4, "subnormal pairs exist for widths 2-4");
  if constexpr (B == 4) {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const uint32_t s = w[d] >> 8;
      p[4 * d + 0] = w[d] & 0x000F000Fu;
      p[4 * d + 1] = w[d] & 0x00F000F0u;
      p[4 * d + 2] = s & 0x000F000Fu;
      p[4 * d + 3] = s & 0x00F000F0u;
    }
  } else if constexpr (B == 3) {
#pragma unroll
    for (int d = 0; d < 3; ++d) {
      const uint32_t s = w[d] >> 9;
      p[5 * d + 0] = w[d] & 0x00070007u;
      p[5 * d + 1] = w[d] & 0x00380038u;
      p[5 * d + 2] = w[d] & 0x01C001C0u;
      p[5 * d + 3] = s & 0x00070007u;
      p[5 * d + 4] = s & 0x00380038u;
    }
    // bit q of codes 30 and 31 is bit 15 / 31 of dword q
    uint32_t t = (w[0] >> 15) & 0x00010001u;
    t = and_or(w[1] >> 14, 0x00020002u, t);
    p[15] = and_or(w[2] >> 13, 0x00040004u, t);
  } else {
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      const uint32_t s = w[d] >> 10;
      p[8 * d + 0] = w[d] & 0x00030003u;
      p[8 * d + 1] = w[d] & 0x000C000Cu;
      p[8 * d + 2] = w[d] & 0x00300030u;
      p[8 * d + 3] = w[d] & 0x00C000C0u;
      p[8 * d + 4] = w[d] & 0x03000300u;
      p[8 * d + 5] = s & 0x00030003u;
      p[8 * d + 6] = s & 0x000C000Cu;
      p[8 * d + 7] = s & 0x00300030u;
    }
  }
}

// 8-bit blocks are two 4-bit planes: dwords 0..3 encode the codes' low
// nibbles and dwords 4..7 their high nibbles, each plane exactly as a 4-bit
// block.  The 8-bit value d (c - 128) = 16 d (hi - 8) + d (lo - 8) + 8 d.

// Load unit u of a row (4*B dwords) with B coalesced 16-byte loads.
//   row: the row's first dword; U: units per row.
template <int B>
__device__ __forceinline__ void load_unit(const uint32_t* row, int U, int u, uint32_t (&w)[4 * B]) {
  const MOEQ_GLOBAL u32x4* r4 = gptr(reinterpret_cast<const u32x4*>(row));
#pragma unroll
  for (int j = 0; j < B; ++j) {
    const u32x4 v = __builtin_nontemporal_load(r4 + (size_t)j * U + u);
    w[4 * j + 0] = v.x;
    w[4 * j + 1] = v.y;
    w[4 * j + 2] = v.z;
    w[4 * j + 3] = v.w;
  }
}

__device__ __forceinline__ float half_to_float(uint32_t h16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)h16);
}

__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xFFFF0000u); }

// float -> bfloat16 bits, round to nearest even (finite inputs)
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

}  // namespace moeq

// Decode path: fused dequantize x matrix-vector products for small batches.
//
// Per token the layer (Fig. 1, middle, of arXiv 2509.25689) evaluates the k
// routed experts it chose and the shared expert(s), each a SwiGLU network
// h = silu(W_gate x) * (W_up x), o = W_down h, and sums the outputs with the
// routing weights.  The work per token is about 2 * sum_i k_i P_i FLOPs
// (Section 3.2), but at batch sizes of a few tokens every weight byte is used
// once, so the path is bound by streaming the packed weights from HBM.
//
// Work decomposition.  A workgroup handles one (expert slot, row tile) pair:
// the slot is a shared expert or one entry of the device-built list of active
// experts (no host synchronization: slots beyond the active count exit at
// once).  Inside, lanes are split into groups of LPR lanes; a group owns one
// row, each lane one 128-weight unit of it (coalesced 16-byte loads of the
// packed codes, see layout.h).  The weights of the wave's rows are loaded to
// registers once and reused for every token of the expert's bucket, whose
// activations are staged in LDS in chunks of TM tokens together with their
// per-block sums.  The dot products accumulate in float32; the per-block
// scale and zero point are applied once per block; the group reduces its partial sums with cross-lane shuffles in a
// fixed order, so results are deterministic.
//
// gate/up kernel: writes h (float32) for every assignment in bucket order.
// Arithmetic of the 2-4-bit kernels.  The one-token gate/up kernel and the
// down kernel stage their activations (x, exactly, and h) in binary16 after a
// power-of-two prescale per block of 32 (11 significant bits at any
// magnitude), mask the code pairs out of the packed dwords as binary16
// subnormals (layout.h) and run the dot products on v_dot2_f32_f16.  The
// gate/up kernel for buckets of 2-64 tokens stages x in bfloat16 as given and
// multiplies it with the codes unpacked to bfloat16 (v_dot2_f32_bf16): there,
// converting four tokens' x per workgroup costs more than the cheaper unpack
// saves.
// down kernel: the result, times the token's routing weight, is written as
// one partial row per (token, slot).
// combine kernel: y_t = sum_j partial(t, j) (j in slot order) + shared.
#include "internal.h"
#include "layout.h"
#include "route_wave.h"

namespace moeq {

namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

constexpr int kXStride = 68;  // dwords per staged unit: 64 + 4 padding against LDS bank conflicts

// Pipeline shape of the down GEMV: each wave walks kDownSteps row steps with
// kDownBuf register buffers, i.e. NBUF - 1 steps of codes in flight while
// one is reduced; MinBlocks bounds registers for occupancy.
#ifndef MOEQ_DOWN_STEPS
#define MOEQ_DOWN_STEPS 4
#endif
#ifndef MOEQ_DOWN_BUF
#define MOEQ_DOWN_BUF 1
#endif
#ifndef MOEQ_DOWN_MINBLOCKS
#define MOEQ_DOWN_MINBLOCKS 4
#endif
// the down kernel for 2-64 tokens (the values above serve one token)
#ifndef MOEQ_DOWNM_STEPS
#define MOEQ_DOWNM_STEPS 4
#endif
#ifndef MOEQ_DOWNM_BUF
#define MOEQ_DOWNM_BUF 1
#endif
static_assert(MOEQ_DOWN_STEPS % MOEQ_DOWN_BUF == 0, "steps per wave must be a multiple of the pipeline depth");
constexpr int kDownSteps = MOEQ_DOWN_STEPS, kDownBuf = MOEQ_DOWN_BUF;
constexpr int kDownStepsM = MOEQ_DOWNM_STEPS, kDownBufM = MOEQ_DOWNM_BUF;
static_assert(MOEQ_DOWNM_STEPS % MOEQ_DOWNM_BUF == 0, "steps per wave must be a multiple of the pipeline depth");
constexpr int kDownMinBlocks = MOEQ_DOWN_MINBLOCKS;

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a),
                                         __builtin_bit_cast(bf16x2, b), c, false);
}
__device__ __forceinline__ float dot2h(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, a), __builtin_bit_cast(f16x2, b), c, false);
}

// Which expert and tokens a slot covers.
struct Slot {
  int desc;     // descriptor row (expert id, or E + s for shared expert s)
  int M;        // tokens in the bucket
  int base;     // first activation row (h) of the bucket
  int shared;   // shared expert index, or -1
};

// The slot's bucket; M = -1 for a slot beyond the active count.
__device__ __forceinline__ Slot slot_info(const DecodeArgs& a, int slot) {
  Slot s;
  if (slot < a.S) {
    s.desc = a.E + slot;
    s.M = a.n;
    s.base = a.n * a.k + slot * a.n;
    s.shared = slot;
    return s;
  }
  const int i = slot - a.S;
  s.shared = -1;
  if (i >= a.active[0]) {
    s.desc = 0;
    s.M = -1;
    s.base = 0;
    return s;
  }
  const int e = a.active[1 + i];
  s.desc = e;
  s.base = a.offsets[e];
  s.M = a.offsets[e + 1] - s.base;
  return s;
}

// One block's contribution for one token: d * sum_i (c_i - z) x_i, from the
// block's code pairs p, the token's 16 activation dwords at xl (and their lo
// parts at xl + lo_offset when NX = 2) and the block sum X.
template <int NX>
__device__ __forceinline__ float block_dot(const uint32_t (&p)[16], const uint32_t* xl, int lo_offset,
                                           float ds, float X, float acc_out) {
  float acc = 0.0f;
  const u32x4* x4 = reinterpret_cast<const u32x4*>(xl);
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const u32x4 xv = x4[c];
    acc = dot2(p[4 * c + 0], xv.x, acc);
    acc = dot2(p[4 * c + 1], xv.y, acc);
    acc = dot2(p[4 * c + 2], xv.z, acc);
    acc = dot2(p[4 * c + 3], xv.w, acc);
  }
  if constexpr (NX == 2) {
    const u32x4* l4 = reinterpret_cast<const u32x4*>(xl + lo_offset);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const u32x4 xv = l4[c];
      acc = dot2(p[4 * c + 0], xv.x, acc);
      acc = dot2(p[4 * c + 1], xv.y, acc);
      acc = dot2(p[4 * c + 2], xv.z, acc);
      acc = dot2(p[4 * c + 3], xv.w, acc);
    }
  }
  return fmaf(ds, fmaf(-192.0f, X, acc), acc_out);
}

// block q's scale (binary16, 4 per unit in sc) times 2^24, for subnormal pairs
__device__ __forceinline__ float block_scale_sub(u32x2 sc, int q) {
  const uint32_t s16 = ((q < 2 ? sc.x : sc.y) >> (16 * (q & 1))) & 0xFFFFu;
  return half_to_float(s16) * 16777216.0f;
}

// One block's contribution for one token from its subnormal code pairs p
// (pair P = c * 2^(k_P - 24)), the token's 16 binary16 activation dwords at xl
// (prescaled by 2^-e) and xf = (X, 2^e), X the sum of the staged values:
//   d 2^e (2^24 sum_k 2^-k dot_k - z X) = (d 2^24) 2^e (dot - z 2^-24 X).
template <int B>
__device__ __forceinline__ float block_dot_sub(const uint32_t (&p)[16], const uint32_t* xl, float ds, float2 xf,
                                               float acc_out) {
  constexpr int NC = sub_classes<B>(), ST = sub_step<B>();
  float acc[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) acc[c] = 0.0f;
  const u32x4* x4 = reinterpret_cast<const u32x4*>(xl);
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const u32x4 xv = x4[c];
    acc[sub_shift<B>(4 * c + 0) / ST] = dot2h(p[4 * c + 0], xv.x, acc[sub_shift<B>(4 * c + 0) / ST]);
    acc[sub_shift<B>(4 * c + 1) / ST] = dot2h(p[4 * c + 1], xv.y, acc[sub_shift<B>(4 * c + 1) / ST]);
    acc[sub_shift<B>(4 * c + 2) / ST] = dot2h(p[4 * c + 2], xv.z, acc[sub_shift<B>(4 * c + 2) / ST]);
    acc[sub_shift<B>(4 * c + 3) / ST] = dot2h(p[4 * c + 3], xv.w, acc[sub_shift<B>(4 * c + 3) / ST]);
  }
  float dot = acc[NC - 1];
#pragma unroll
  for (int c = NC - 2; c >= 0; --c) dot = fmaf(dot, 1.0f / (float)(1 << ST), acc[c]);
  constexpr float zs = (float)(1 << (B - 1)) * 0x1p-24f;
  return fmaf(ds * xf.y, fmaf(-zs, xf.x, dot), acc_out);
}

// One thread's 16-byte piece (8 values) of a block of 32, whose four pieces
// are held by four consecutive threads of one wave (all active): binary16
// after the block's power-of-two prescale 2^-e, e from the block's largest
// magnitude so that it lands in [2^14, 2^15) (no overflow, 11 significant
// bits at any scale; e >= -100 keeps 2^-e finite for an all-zero block).
// The piece goes to dst; the block's first thread (first) writes
// (X, 2^e) to *xf, X the sum of the staged values.
__device__ __forceinline__ void stage_piece(const float (&f)[8], uint32_t* dst, float2* xf, bool first) {
  float am = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i) am = fmaxf(am, fabsf(f[i]));
  am = fmaxf(am, __shfl_xor(am, 1, 64));
  am = fmaxf(am, __shfl_xor(am, 2, 64));
  const int e = max((int)((__float_as_uint(am) >> 23) & 0xFFu) - 141, -100);
  const float sc = __builtin_amdgcn_ldexpf(1.0f, -e);
  uint32_t hv[4];
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const _Float16 h0 = (_Float16)(f[2 * i] * sc), h1 = (_Float16)(f[2 * i + 1] * sc);
    hv[i] = (uint32_t)__builtin_bit_cast(uint16_t, h0) | (uint32_t)__builtin_bit_cast(uint16_t, h1) << 16;
    sum += (float)h0 + (float)h1;
  }
  sum += __shfl_xor(sum, 1, 64);
  sum += __shfl_xor(sum, 2, 64);
  *reinterpret_cast<u32x4*>(dst) = u32x4{hv[0], hv[1], hv[2], hv[3]};
  if (first) *xf = make_float2(sum, __builtin_amdgcn_ldexpf(1.0f, e));
}

// the 8 bfloat16 values of a 16-byte piece as float
__device__ __forceinline__ void bf16x8_to_f32(const u32x4 v, float (&f)[8]) {
  f[0] = bf16_lo(v.x); f[1] = bf16_hi(v.x); f[2] = bf16_lo(v.y); f[3] = bf16_hi(v.y);
  f[4] = bf16_lo(v.z); f[5] = bf16_hi(v.z); f[6] = bf16_lo(v.w); f[7] = bf16_hi(v.w);
}

template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROW_MASK, 0xF, false));
}

// Sum over a group of LPR lanes (16, 32 or 64) with DPP adds in a fixed order:
// quad butterflies, row rotations, then row broadcasts.  The group's last
// lane holds the total.
template <int LPR>
__device__ __forceinline__ float group_sum(float v) {
  v += dpp_f<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f<0x124>(v);  // row_ror:4
  v += dpp_f<0x128>(v);  // row_ror:8
  if constexpr (LPR >= 32) v += dpp_f<0x142, 0xA>(v);  // row_bcast:15 into rows 1, 3
  if constexpr (LPR >= 64) v += dpp_f<0x143, 0xC>(v);  // row_bcast:31 into rows 2, 3
  return v;
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + expf(-g)); }

// ---------------------------------------------------------------------------
// down x routing weight for one (slot, row tile), down width BD; the same
// two-buffer walk over each wave's row steps.
template <int BD>
struct DownRows {
  uint32_t w[4 * BD];
  u32x2 s;
};

template <int BD>
__device__ __forceinline__ void load_down(DownRows<BD>& b, const TensorDev& td, int row, int U, int u, int I) {
  load_unit<BD>(td.codes + (size_t)row * BD * U * 4, U, u, b.w);
  b.s = *gptr(reinterpret_cast<const u32x2*>(td.scales + (size_t)row * (I / kBlock) + 4 * u));
}

template <int BD, int LPR, int TM>
__device__ __forceinline__ void compute_down(const DownRows<BD>& b, bool active, const uint32_t* xu,
                                             const float2* su4, int xts, int sts, int mc, int u,
                                             const Slot sl, int m0, int row, const DecodeArgs& a) {
  float o[TM];
#pragma unroll
  for (int m = 0; m < TM; ++m) o[m] = 0.0f;
  if (active) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t p[16];
      block_pairs_sub<BD>(b.w + q * BD, p);
      const float dd = block_scale_sub(b.s, q);
#pragma unroll
      for (int m = 0; m < TM; ++m)
        if (m < mc) o[m] = block_dot_sub<BD>(p, xu + m * xts + 16 * q, dd, su4[m * sts + q], o[m]);
    }
  }
#pragma unroll
  for (int m = 0; m < TM; ++m) {
    if (m < mc) {
      const float os = group_sum<LPR>(o[m]);
      if (u == LPR - 1) {
        int prow;
        float wv;
        if (sl.shared >= 0) {
          prow = a.n * a.k + sl.shared * a.n + m0 + m;
          wv = 1.0f;
        } else {
          prow = a.perm[sl.base + m0 + m];
          wv = a.w[prow];
        }
        a.partial[(size_t)prow * a.H + row] = wv * os;
      }
    }
  }
}

template <int BD, int LPR, int TM, int RW, int NBUF>
__device__ __forceinline__ void down_body(const DecodeArgs& a, const Slot sl, const TensorDev& td,
                                          uint32_t* smem) {
  const int H = a.H, I = a.I, U = I / kUnit;
  const int xts = U * kXStride, sts = U * 4;  // per-token LDS strides (dwords, float pairs)
  uint32_t* xl = smem;
  float2* xs = reinterpret_cast<float2*>(smem + TM * xts);

  constexpr int GPW = 64 / LPR;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int grp = lane / LPR, u = lane % LPR;
  const bool uok = u < U;
  const int row0 = blockIdx.x * (4 * GPW * RW) + wave * (GPW * RW) + grp;  // + step * GPW

  DownRows<BD> buf[NBUF];
  for (int m0 = 0; m0 < sl.M; m0 += TM) {
    const int mc = min(TM, sl.M - m0);
    asm volatile("" ::: "memory");  // weight loads stay inside the chunk loop
#pragma unroll
    for (int st = 0; st < NBUF; ++st)
      if (st < RW && uok && row0 + st * GPW < H) load_down(buf[st], td, row0 + st * GPW, U, u, I);
    __syncthreads();
    // stage h rows in binary16 with per-block prescales
    for (int m = 0; m < mc; ++m) {
      const MOEQ_GLOBAL f32x4* src = gptr(reinterpret_cast<const f32x4*>(a.h + (size_t)(sl.base + m0 + m) * I));
      for (int q = threadIdx.x; q < I / 8; q += 256) {
        const f32x4 v0 = src[2 * q], v1 = src[2 * q + 1];
        const float f[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
        const int uu = q >> 4, cq = q & 15;
        stage_piece(f, xl + m * xts + uu * kXStride + cq * 4, xs + m * sts + uu * 4 + (cq >> 2), (cq & 3) == 0);
      }
    }
    __syncthreads();
    const uint32_t* xu = xl + u * kXStride;
    const float2* su4 = xs + u * 4;
#pragma unroll 1
    for (int g0 = 0; g0 < RW; g0 += NBUF) {
      asm volatile("" ::: "memory");
#pragma unroll
      for (int b = 0; b < NBUF; ++b) {
        const int st = g0 + b;
        const int r = row0 + st * GPW;
        if (r < H) compute_down<BD, LPR, TM>(buf[b], uok, xu, su4, xts, sts, mc, u, sl, m0, r, a);
        const int rn = row0 + (st + NBUF) * GPW;
        if (st + NBUF < RW && uok && rn < H) load_down(buf[b], td, rn, U, u, I);
      }
    }
  }
}

// grid = (row tiles of H, S + max_active), 256 threads
template <int LPR, int TM, int RW, int NBUF>
__global__ __launch_bounds__(256, TM == 1 ? kDownMinBlocks : 2) void down_kernel(DecodeArgs a) {
  extern __shared__ uint32_t smem[];
  const Slot sl = slot_info(a, blockIdx.y);
  if (sl.M < 0 || sl.M > a.gemm_above) return;  // (large buckets: the grouped GEMMs)
  const TensorDev td = a.desc[sl.desc * 3 + 2];
  if (!td.codes) return;
  switch (td.bits) {
    case 2: down_body<2, LPR, TM, RW, NBUF>(a, sl, td, smem); break;
    case 3: down_body<3, LPR, TM, RW, NBUF>(a, sl, td, smem); break;
    case 4: down_body<4, LPR, TM, RW, NBUF>(a, sl, td, smem); break;
    default: break;
  }
}

// ---------------------------------------------------------------------------
// One token: down x routing weight and the combine in one pass, for layers
// whose down tensors are 2-4 bits wide with at most 16 units per row: one
// width BD, or (BD = 0) widths that differ between tensors, where every
// unit is fetched as four chunk loads, those past the slot's width from 16
// zero bytes that stay in the vector cache, and the slot's width picks the
// decoder.  A workgroup of NT threads owns NT / 16 rows of y across every slot (the
// token's k choices in choice order, then the shared experts): a group of 16
// lanes owns one row, lane u unit u of that row in every slot, with D slots'
// codes in flight.  The lane accumulates w_j * (its partial dot of slot j) in
// slot order and the group sums its lanes with DPP in a fixed order: no
// partial rows, no combine launch.  All h rows are staged once per workgroup
// (binary16 with per-block prescales, as in the down kernel), their loads
// issued in batches so a batch costs one memory round trip.
struct DownSlot {
  const uint32_t* codes;
  const uint16_t* scales;
  float w;
  int hrow;
  int bits;
};

// w_j-free partial dot of one slot's unit: sum over its 4 blocks
template <int B>
__device__ __forceinline__ float down1_unit_dot(const uint32_t* w, u32x2 sc, const uint32_t* xu,
                                                const float2* su4) {
  float o = 0.0f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t pr[16];
    block_pairs_sub<B>(w + q * B, pr);
    o = block_dot_sub<B>(pr, xu + 16 * q, block_scale_sub(sc, q), su4[q], o);
  }
  return o;
}

constexpr int kDown1Batch = 6;  // staged 32-byte pieces per thread per round trip

template <int BD, int NT, int D>
__global__ __launch_bounds__(NT) void down1_kernel(DecodeArgs a) {
  extern __shared__ uint32_t smem[];
  __shared__ DownSlot slots[kMaxTopK + kMaxShared];
  const int H = a.H, I = a.I, U = I / kUnit, k = a.k, NS = a.k + a.S;
  const int xts = U * kXStride, sts = U * 4;
  uint32_t* xl = smem;
  float2* xs = reinterpret_cast<float2*>(smem + NS * xts);
  if ((int)threadIdx.x < NS) {
    const int j = threadIdx.x;
    DownSlot v;
    if (j < k) {
      // choice j of the token: its bucket of one holds h row offsets[e]
      const int e = a.idx[j];
      const TensorDev t = a.desc[e * 3 + 2];
      v.codes = t.codes;
      v.scales = t.scales;
      v.w = a.w[j];
      v.hrow = a.offsets[e];
      v.bits = t.bits;
    } else {
      const TensorDev t = a.desc[(a.E + (j - k)) * 3 + 2];
      v.codes = t.codes;
      v.scales = t.scales;
      v.w = 1.0f;
      v.hrow = k + (j - k);
      v.bits = t.bits;
    }
    slots[j] = v;
  }
  __syncthreads();

  const int u = threadIdx.x & 15;
  const int row = blockIdx.x * (NT / 16) + (threadIdx.x >> 4);
  const int rowc = min(row, H - 1), uc = min(u, U - 1);
  constexpr int BL = BD == 0 ? 4 : BD;  // chunks loaded per unit
  auto load_slot = [&](DownRows<BL>& b, int j) {
    const DownSlot& sl = slots[min(j, NS - 1)];
    if constexpr (BD == 0) {
      const int bits = sl.bits;
      const MOEQ_GLOBAL u32x4* r4 =
          gptr(reinterpret_cast<const u32x4*>(sl.codes + (size_t)rowc * bits * U * 4)) + uc;
      const MOEQ_GLOBAL u32x4* z4 = gptr(reinterpret_cast<const u32x4*>(a.zeros));
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const u32x4 v = __builtin_nontemporal_load(c < bits ? r4 + (size_t)c * U : z4);
        b.w[4 * c + 0] = v.x;
        b.w[4 * c + 1] = v.y;
        b.w[4 * c + 2] = v.z;
        b.w[4 * c + 3] = v.w;
      }
    } else {
      load_unit<BD>(sl.codes + (size_t)rowc * BD * U * 4, U, uc, b.w);
    }
    b.s = *gptr(reinterpret_cast<const u32x2*>(sl.scales + (size_t)rowc * (I / kBlock) + 4 * uc));
  };
  DownRows<BL> buf[D];
#pragma unroll
  for (int i = 0; i < D - 1; ++i) load_slot(buf[i], i);

  // stage every slot's h row: piece p (8 values) of slot p / (I / 8); a
  // batch's loads all go out before its first piece is converted
  const int PPS = I / 8, NP = NS * PPS;
  for (int p0 = 0; p0 < NP; p0 += NT * kDown1Batch) {
    f32x4 v[kDown1Batch][2];
#pragma unroll
    for (int i = 0; i < kDown1Batch; ++i) {
      if (p0 + i * NT < NP) {
        // pieces past the end repeat the last block's (same values, same place)
        int p = p0 + i * NT + (int)threadIdx.x;
        p = p < NP ? p : NP - 4 + (p & 3);
        const MOEQ_GLOBAL f32x4* src =
            gptr(reinterpret_cast<const f32x4*>(a.h + (size_t)slots[p / PPS].hrow * I)) + 2 * (p % PPS);
        v[i][0] = src[0];
        v[i][1] = src[1];
      }
    }
#pragma unroll
    for (int i = 0; i < kDown1Batch; ++i) {
      if (p0 + i * NT < NP) {
        int p = p0 + i * NT + (int)threadIdx.x;
        p = p < NP ? p : NP - 4 + (p & 3);
        const int m = p / PPS, c = p % PPS;
        const float f[8] = {v[i][0].x, v[i][0].y, v[i][0].z, v[i][0].w,
                            v[i][1].x, v[i][1].y, v[i][1].z, v[i][1].w};
        const int uu = c >> 4, cq = c & 15;
        stage_piece(f, xl + m * xts + uu * kXStride + cq * 4, xs + m * sts + uu * 4 + (cq >> 2), (cq & 3) == 0);
      }
    }
  }
  __syncthreads();

  const uint32_t* xu = xl + uc * kXStride;
  const float2* su4 = xs + uc * 4;
  float acc = 0.0f;
#pragma unroll 1
  for (int j0 = 0; j0 < NS; j0 += D) {
    asm volatile("" ::: "memory");
#pragma unroll
    for (int b = 0; b < D; ++b) {
      const int j = j0 + b;
      if (j < NS) {
        // slot j + D - 1 goes out before slot j is reduced
        load_slot(buf[(b + D - 1) % D], j + D - 1);
        float o;
        if constexpr (BD == 0) {
          switch (__builtin_amdgcn_readfirstlane(slots[j].bits)) {
            case 2: o = down1_unit_dot<2>(buf[b].w, buf[b].s, xu + j * xts, su4 + j * sts); break;
            case 3: o = down1_unit_dot<3>(buf[b].w, buf[b].s, xu + j * xts, su4 + j * sts); break;
            default: o = down1_unit_dot<4>(buf[b].w, buf[b].s, xu + j * xts, su4 + j * sts); break;
          }
        } else {
          o = down1_unit_dot<BD>(buf[b].w, buf[b].s, xu + j * xts, su4 + j * sts);
        }
        acc = fmaf(slots[j].w, u < U ? o : 0.0f, acc);
      }
    }
  }
  const float ys = group_sum<16>(acc);
  if (u == 15 && row < H) a.y[row] = ys;
}

// ---------------------------------------------------------------------------
// y_t = sum_j partial(t*k + j) + sum_s partial(n*k + s*n + t), fixed order;
// the loads of eight partial rows are issued together.
__global__ __launch_bounds__(256) void combine_kernel(DecodeArgs a) {
  const int H4 = a.H / 4;
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long long)a.n * H4) return;
  const int t = (int)(i / H4), c = (int)(i % H4);
  const float4* p = reinterpret_cast<const float4*>(a.partial);
  const int rows = a.k + a.S;
  float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  for (int j0 = 0; j0 < rows; j0 += 8) {
    float4 v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int j = j0 + q;
      if (j < rows) {
        const size_t r = j < a.k ? (size_t)t * a.k + j : (size_t)a.n * a.k + (size_t)(j - a.k) * a.n + t;
        v[q] = p[r * H4 + c];
      }
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      if (j0 + q < rows) {
        acc.x += v[q].x; acc.y += v[q].y; acc.z += v[q].z; acc.w += v[q].w;
      }
    }
  }
  reinterpret_cast<float4*>(a.y)[i] = acc;
}

// ---------------------------------------------------------------------------
// Buckets of one token: gate/up + SwiGLU with 16 lanes per row pair.  Lanes 0-7 of a
// 16-lane group stream the gate row and lanes 8-15 the up row; lane j of a
// half walks the units j, j + 8, j + 16, ... of its row, so all lanes are
// busy for any number of units, and the per-row work (sums, activation,
// store) is spread over several units per lane.  The codes of unit i + 1 are
// in flight while unit i is reduced.  A half sums its lanes with DPP (quad
// butterflies, then the half-row mirror); the up half's last lane receives
// the gate total across the row (row_ror:8) and writes h.
template <int B>
struct UnitBuf {
  uint32_t w[4 * B];
  u32x2 s;
};

template <int B>
__device__ __forceinline__ void load_unit_buf(UnitBuf<B>& b, const TensorDev& t, int row, int U, int u, int K) {
  load_unit<B>(t.codes + (size_t)row * B * U * 4, U, u, b.w);
  b.s = *gptr(reinterpret_cast<const u32x2*>(t.scales + (size_t)row * (K / kBlock) + 4 * u));
}

// d * sum (c - z) x over one 128-weight unit, for the token staged at xu / su4
template <int B>
__device__ __forceinline__ float unit_dot(const UnitBuf<B>& b, const uint32_t* xu, const float2* su4, float acc) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t p[16];
    block_pairs_sub<B>(b.w + q * B, p);
    acc = block_dot_sub<B>(p, xu + 16 * q, block_scale_sub(b.s, q), su4[q], acc);
  }
  return acc;
}

__device__ __forceinline__ float half_sum8(float v) {
  v += dpp_f<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f<0x141>(v);  // row_half_mirror: the other quad of the half row
  return v;
}

// the half's partial dot over its units (units j, j + 8, ... of row `row`);
// GU1_DEPTH units are in flight while one is reduced
#ifndef MOEQ_GU1_DEPTH
#define MOEQ_GU1_DEPTH 2
#endif
#ifndef MOEQ_GU1_MINBLOCKS
#define MOEQ_GU1_MINBLOCKS 5
#endif
template <int B>
__device__ __forceinline__ float row_half_dot(const TensorDev& t, int row, int U, int j, int H, const uint32_t* xl,
                                              const float2* xs, const UnitBuf<B>& first) {
  constexpr int NB = MOEQ_GU1_DEPTH;
  const int UPL = (U + 7) / 8;
  UnitBuf<B> buf[NB];
  buf[0] = first;
#pragma unroll
  for (int i = 1; i < NB - 1; ++i) load_unit_buf<B>(buf[i], t, row, U, min(j + 8 * min(i, UPL - 1), U - 1), H);
  float acc = 0.0f;
#pragma unroll 1
  for (int i0 = 0; i0 < UPL; i0 += NB) {
    asm volatile("" ::: "memory");
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int i = i0 + b;
      if (i < UPL) {
        // unit i + NB - 1 (clamped to the last valid one) goes out before unit i is reduced
        load_unit_buf<B>(buf[(b + NB - 1) % NB], t, row, U, min(j + 8 * min(i + NB - 1, UPL - 1), U - 1), H);
        const int u = j + 8 * i;
        if (u < U) acc = unit_dot<B>(buf[b], xl + u * kXStride, xs + u * 4, acc);
      }
    }
  }
  return acc;
}

// the token's x into LDS in binary16 with per-block prescales (16-byte
// pieces, 4 per block)
__device__ __forceinline__ void stage_x1(const DecodeArgs& a, const Slot sl, uint32_t* xl, float2* xs) {
  const int H = a.H;
  // (one token: token 0, without reading the bucket permutation, which the
  // routing workgroup of gateup1_route_kernel may still be writing)
  const int t = sl.shared >= 0 || a.n == 1 ? 0 : a.perm[sl.base] / a.k;
  const MOEQ_GLOBAL u32x4* src = gptr(reinterpret_cast<const u32x4*>(a.x + (size_t)t * H));
  for (int q = threadIdx.x; q < H / 8; q += 256) {
    float f[8];
    bf16x8_to_f32(src[q], f);
    const int uu = q >> 4, cq = q & 15;
    stage_piece(f, xl + uu * kXStride + cq * 4, xs + uu * 4 + (cq >> 2), (cq & 3) == 0);
  }
}

// token 0's x staged by threads [t0, t0 + nt) of the workgroup (nt a multiple
// of 64, t0 of 64: the four pieces of a block stay in four lanes of a wave)
__device__ __forceinline__ void stage_x1_token0(const DecodeArgs& a, int t0, int nt, uint32_t* xl, float2* xs) {
  const int H = a.H;
  const MOEQ_GLOBAL u32x4* src = gptr(reinterpret_cast<const u32x4*>(a.x));
  for (int q = (int)threadIdx.x - t0; q < H / 8; q += nt) {
    float f[8];
    bf16x8_to_f32(src[q], f);
    const int uu = q >> 4, cq = q & 15;
    stage_piece(f, xl + uu * kXStride + cq * 4, xs + uu * 4 + (cq >> 2), (cq & 3) == 0);
  }
}

// Each lane requests its first unit before x is staged, so the staging
// latency overlaps the weight traffic (STAGED: x is in LDS already).
template <int BG, int BU, bool STAGED = false>
__device__ __forceinline__ void gateup1_body(const DecodeArgs& a, const Slot sl, const TensorDev& tg,
                                             const TensorDev& tu, uint32_t* xl, float2* xs) {
  const int H = a.H, I = a.I, U = H / kUnit;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = blockIdx.x * 16 + wave * 4 + (lane >> 4);
  const bool up = (lane & 8) != 0;
  const int j = lane & 7;
  const int rowc = min(row, I - 1);
  float v;
  if constexpr (BG == BU) {
    const TensorDev& t = up ? tu : tg;
    UnitBuf<BG> first;
    load_unit_buf<BG>(first, t, rowc, U, min(j, U - 1), H);
    if constexpr (!STAGED) {
      stage_x1(a, sl, xl, xs);
      __syncthreads();
    }
    v = row_half_dot<BG>(t, rowc, U, j, H, xl, xs, first);
  } else {
    UnitBuf<BG> fg;
    UnitBuf<BU> fu;
    if (up)
      load_unit_buf<BU>(fu, tu, rowc, U, min(j, U - 1), H);
    else
      load_unit_buf<BG>(fg, tg, rowc, U, min(j, U - 1), H);
    if constexpr (!STAGED) {
      stage_x1(a, sl, xl, xs);
      __syncthreads();
    }
    if (up)
      v = row_half_dot<BU>(tu, rowc, U, j, H, xl, xs, fu);
    else
      v = row_half_dot<BG>(tg, rowc, U, j, H, xl, xs, fg);
  }
  v = half_sum8(v);
  const float other = dpp_f<0x128>(v);  // row_ror:8: the other half's total
  if ((lane & 15) == 15 && row < I) a.h[(size_t)sl.base * a.I + row] = silu(other) * v;
}

// one workgroup's share of the gate/up of a bucket of one token
template <bool STAGED = false>
__device__ __forceinline__ void gateup1_slot(const DecodeArgs& a, const Slot& sl, uint32_t* smem) {
  if (sl.M != 1) return;  // the buckets of one token, of any batch
  const TensorDev tg = a.desc[sl.desc * 3 + 0], tu = a.desc[sl.desc * 3 + 1];
  if (!tg.codes || !tu.codes) return;
  const int U = a.H / kUnit;
  uint32_t* xl = smem;
  float2* xs = reinterpret_cast<float2*>(smem + U * kXStride);
  switch (tg.bits * 8 + tu.bits) {
    case 2 * 8 + 2: gateup1_body<2, 2, STAGED>(a, sl, tg, tu, xl, xs); break;
    case 2 * 8 + 3: gateup1_body<2, 3, STAGED>(a, sl, tg, tu, xl, xs); break;
    case 2 * 8 + 4: gateup1_body<2, 4, STAGED>(a, sl, tg, tu, xl, xs); break;
    case 3 * 8 + 2: gateup1_body<3, 2, STAGED>(a, sl, tg, tu, xl, xs); break;
    case 3 * 8 + 3: gateup1_body<3, 3, STAGED>(a, sl, tg, tu, xl, xs); break;
    case 3 * 8 + 4: gateup1_body<3, 4, STAGED>(a, sl, tg, tu, xl, xs); break;
    case 4 * 8 + 2: gateup1_body<4, 2, STAGED>(a, sl, tg, tu, xl, xs); break;
    case 4 * 8 + 3: gateup1_body<4, 3, STAGED>(a, sl, tg, tu, xl, xs); break;
    case 4 * 8 + 4: gateup1_body<4, 4, STAGED>(a, sl, tg, tu, xl, xs); break;
    default: break;
  }
}

// grid = (I / 16, S + max_active), 256 threads; the buckets of one token
__global__ __launch_bounds__(256, MOEQ_GU1_MINBLOCKS) void gateup1_kernel(DecodeArgs a) {
  extern __shared__ uint32_t smem[];
  gateup1_slot(a, slot_info(a, blockIdx.y), smem);
}

// The same for a forward of one token that needs no routing launch: wave 0
// of every workgroup of a routed slot routes the token itself (the routing
// kernels' selection, deterministic, so every workgroup finds the same
// experts; waves 1-3 stage x meanwhile) while the shared experts'
// workgroups start at once.  Routed slot
// i is the i-th chosen expert in ascending id order, as the bucketing lists
// them.  Workgroup (0, S) also writes what the routing launch would have:
// idx and w in choice order, offsets, the active list and the permutation,
// which the down kernel and any 5/6/8-bit gate/up kernel read after this
// launch.  grid = (I / 16, S + k), 256 threads.
template <int EPL>
__global__ __launch_bounds__(256, MOEQ_GU1_MINBLOCKS) void gateup1_route_kernel(DecodeArgs a, RouterParams rp,
                                                                                Workspace ws) {
  extern __shared__ uint32_t smem[];
  __shared__ float gs_l[64];
  __shared__ int32_t chosen[kMaxTopK];
  Slot sl;
  if ((int)blockIdx.y < a.S) {
    sl = slot_info(a, blockIdx.y);
  } else {
    if (threadIdx.x < 64) {
      // (slots past the choices, which the creation checks rule out, read
      // expert 0's descriptor: in range, skipped if it holds no tensor)
      if (threadIdx.x < kMaxTopK) chosen[threadIdx.x] = 0;
      const bool out = blockIdx.x == 0 && (int)blockIdx.y == a.S;
      const LaneChoice<EPL> ch =
          route_token_wave<EPL>(rp, 0, gs_l, out ? ws.idx : nullptr, out ? ws.w : nullptr, nullptr);
      const int lane = threadIdx.x, E = rp.E_row;
      const int cnt = __popc(ch.bits);
      const int below = wave_incl_sum(cnt) - cnt;  // chosen ids of the lanes below
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        const int e = lane * EPL + i;
        const int r = below + __popc(ch.bits & ((1u << i) - 1u));
        const bool c = (ch.bits >> i) & 1u;
        if (c) chosen[r] = e;
        if (out) {
          if (e < E) ws.offsets[e] = r;
          if (c) {
            ws.active[1 + r] = e;
            ws.perm[r] = ch.order[i];
          }
        }
      }
      if (out && lane == 0) {
        ws.offsets[E] = rp.k;
        ws.active[0] = rp.k;
      }
    } else {
      // waves 1-3 stage the token's x meanwhile
      const int U = a.H / kUnit;
      stage_x1_token0(a, 64, 192, smem, reinterpret_cast<float2*>(smem + U * kXStride));
    }
    __syncthreads();
    const int i = blockIdx.y - a.S;
    sl.desc = chosen[i];
    sl.base = i;
    sl.M = 1;
    sl.shared = -1;
    gateup1_slot<true>(a, sl, smem);
    return;
  }
  gateup1_slot(a, sl, smem);
}

// ---------------------------------------------------------------------------
// Buckets of 2 or more tokens, in the one-token kernel's layout (16 lanes per
// row pair, lane j of a half walking the units j, j + 8, ... of its row, code
// pairs as binary16 subnormals), TM tokens staged per pass: each unit's code
// pairs are unpacked once and multiplied with every staged token.  Measured
// at 16 tokens: 2 tokens per pass (four workgroups per compute unit) 427 us
// per step, 3 per pass 427, 4 per pass (two workgroups per CU) 451, against
// 446 for a kernel that gave a whole wave to each row and staged 4 tokens
// in bfloat16.

// token t's x into LDS at xl / xs (binary16 with per-block prescales)
__device__ __forceinline__ void stage_x_token(const DecodeArgs& a, int t, uint32_t* xl, float2* xs) {
  const int H = a.H;
  const MOEQ_GLOBAL u32x4* src = gptr(reinterpret_cast<const u32x4*>(a.x + (size_t)t * H));
  for (int q = threadIdx.x; q < H / 8; q += 256) {
    float f[8];
    bf16x8_to_f32(src[q], f);
    const int uu = q >> 4, cq = q & 15;
    stage_piece(f, xl + uu * kXStride + cq * 4, xs + uu * 4 + (cq >> 2), (cq & 3) == 0);
  }
}

// the half's partial dots over its units for the mc <= TM staged tokens
template <int B, int TM>
__device__ __forceinline__ void row_half_dot_tm(const TensorDev& t, int row, int U, int j, int H, const uint32_t* xl,
                                                const float2* xs, int xts, int sts, int mc,
                                                const UnitBuf<B>& first, float (&acc)[TM]) {
  constexpr int NB = MOEQ_GU1_DEPTH;
  const int UPL = (U + 7) / 8;
  UnitBuf<B> buf[NB];
  buf[0] = first;
#pragma unroll
  for (int i = 1; i < NB - 1; ++i) load_unit_buf<B>(buf[i], t, row, U, min(j + 8 * min(i, UPL - 1), U - 1), H);
#pragma unroll
  for (int m = 0; m < TM; ++m) acc[m] = 0.0f;
#pragma unroll 1
  for (int i0 = 0; i0 < UPL; i0 += NB) {
    asm volatile("" ::: "memory");
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int i = i0 + b;
      if (i < UPL) {
        load_unit_buf<B>(buf[(b + NB - 1) % NB], t, row, U, min(j + 8 * min(i + NB - 1, UPL - 1), U - 1), H);
        const int u = j + 8 * i;
        if (u < U) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            uint32_t p[16];
            block_pairs_sub<B>(buf[b].w + q * B, p);
            const float ds = block_scale_sub(buf[b].s, q);
#pragma unroll
            for (int m = 0; m < TM; ++m)
              if (m < mc)
                acc[m] = block_dot_sub<B>(p, xl + m * xts + u * kXStride + 16 * q, ds, xs[m * sts + u * 4 + q],
                                          acc[m]);
          }
        }
      }
    }
  }
}

template <int BG, int BU, int TM>
__device__ __forceinline__ void gateupn_body(const DecodeArgs& a, const Slot sl, const TensorDev& tg,
                                             const TensorDev& tu, uint32_t* smem) {
  const int H = a.H, I = a.I, U = H / kUnit;
  const int xts = U * kXStride, sts = U * 4;  // per-token LDS strides (dwords, float2)
  uint32_t* xl = smem;
  float2* xs = reinterpret_cast<float2*>(smem + TM * xts);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = blockIdx.x * 16 + wave * 4 + (lane >> 4);
  const bool up = (lane & 8) != 0;
  const int j = lane & 7;
  const int rowc = min(row, I - 1);
  for (int m0 = 0; m0 < sl.M; m0 += TM) {
    const int mc = min(TM, sl.M - m0);
    // the first unit is requested before x is staged
    UnitBuf<BG> fg;
    UnitBuf<BU> fu;
    if constexpr (BG == BU) {
      load_unit_buf<BG>(fg, up ? tu : tg, rowc, U, min(j, U - 1), H);
    } else {
      if (up)
        load_unit_buf<BU>(fu, tu, rowc, U, min(j, U - 1), H);
      else
        load_unit_buf<BG>(fg, tg, rowc, U, min(j, U - 1), H);
    }
    if (m0 > 0) __syncthreads();  // the previous pass has read its x
    for (int m = 0; m < mc; ++m) {
      const int t = sl.shared >= 0 ? m0 + m : a.perm[sl.base + m0 + m] / a.k;
      stage_x_token(a, t, xl + m * xts, xs + m * sts);
    }
    __syncthreads();
    float acc[TM];
    if constexpr (BG == BU) {
      row_half_dot_tm<BG, TM>(up ? tu : tg, rowc, U, j, H, xl, xs, xts, sts, mc, fg, acc);
    } else {
      if (up)
        row_half_dot_tm<BU, TM>(tu, rowc, U, j, H, xl, xs, xts, sts, mc, fu, acc);
      else
        row_half_dot_tm<BG, TM>(tg, rowc, U, j, H, xl, xs, xts, sts, mc, fg, acc);
    }
#pragma unroll
    for (int m = 0; m < TM; ++m) {
      if (m < mc) {
        const float v = half_sum8(acc[m]);
        const float other = dpp_f<0x128>(v);  // row_ror:8: the gate half's total
        if ((lane & 15) == 15 && row < I) a.h[(size_t)(sl.base + m0 + m) * I + row] = silu(other) * v;
      }
    }
  }
}

// grid = (I / 16, S + max_active), 256 threads; buckets of 2 .. gemm_above tokens
template <int TM>
__global__ __launch_bounds__(256, TM <= 2 ? 4 : 2) void gateupn_kernel(DecodeArgs a) {
  extern __shared__ uint32_t smem[];
  const Slot sl = slot_info(a, blockIdx.y);
  if (sl.M < 2 || sl.M > a.gemm_above) return;
  const TensorDev tg = a.desc[sl.desc * 3 + 0], tu = a.desc[sl.desc * 3 + 1];
  if (!tg.codes || !tu.codes) return;
  switch (tg.bits * 8 + tu.bits) {
    case 2 * 8 + 2: gateupn_body<2, 2, TM>(a, sl, tg, tu, smem); break;
    case 2 * 8 + 3: gateupn_body<2, 3, TM>(a, sl, tg, tu, smem); break;
    case 2 * 8 + 4: gateupn_body<2, 4, TM>(a, sl, tg, tu, smem); break;
    case 3 * 8 + 2: gateupn_body<3, 2, TM>(a, sl, tg, tu, smem); break;
    case 3 * 8 + 3: gateupn_body<3, 3, TM>(a, sl, tg, tu, smem); break;
    case 3 * 8 + 4: gateupn_body<3, 4, TM>(a, sl, tg, tu, smem); break;
    case 4 * 8 + 2: gateupn_body<4, 2, TM>(a, sl, tg, tu, smem); break;
    case 4 * 8 + 3: gateupn_body<4, 3, TM>(a, sl, tg, tu, smem); break;
    case 4 * 8 + 4: gateupn_body<4, 4, TM>(a, sl, tg, tu, smem); break;
    default: break;
  }
}

// ---------------------------------------------------------------------------
// Wide tensors (5, 6 and 8 bits).  The kernels above skip a slot whose gate or
// up (down) tensor is wide; these take exactly those slots.  LPR lanes per
// row (8, 16 or 32): lane j walks the units j, j + LPR, ... of its row with the
// next unit in flight, for up to TM tokens per pass (1 for a single token,
// else 4).  Gate, up and down are reduced one tensor at a time, so a wave
// decodes one width at a time.  Few slots (shared experts only) take more
// lanes per row, so that the grid still covers the chip.
__device__ __forceinline__ bool wide_bits(int b) { return b > 4; }

template <int B>
struct WideUnit {
  uint32_t w[4 * B];
  u32x2 s;
};

template <int B>
__device__ __forceinline__ void wide_load(WideUnit<B>& b, const TensorDev& t, int row, int U, int u, int K) {
  load_unit<B>(t.codes + (size_t)row * B * U * 4, U, u, b.w);
  b.s = *gptr(reinterpret_cast<const u32x2*>(t.scales + (size_t)row * (K / kBlock) + 4 * u));
}

// acc[m] += d * sum (c - z) x_m over one unit, for the mc staged tokens
template <int B, int NX, int TM>
__device__ __forceinline__ void wide_unit_dot(const WideUnit<B>& b, const uint32_t* xu, int xts, int lo,
                                              const float* su4, int sts, int mc, float (&acc)[TM]) {
  const PairConsts pk = pair_consts();
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float d = half_to_float(((q < 2 ? b.s.x : b.s.y) >> (16 * (q & 1))) & 0xFFFFu);
    if constexpr (B == 8) {
      // two 4-bit planes: d (c - 128) = 16 d (hi - 8) + d (lo - 8) + 8 d
      uint32_t p[16];
      block_pairs<4>(b.w + 8 * q + 4, pk, p);
#pragma unroll
      for (int m = 0; m < TM; ++m)
        if (m < mc) acc[m] = block_dot<NX>(p, xu + m * xts + 16 * q, lo, 2.0f * d, su4[m * sts + q], acc[m]);
      block_pairs<4>(b.w + 8 * q, pk, p);
#pragma unroll
      for (int m = 0; m < TM; ++m) {
        if (m < mc) {
          const float X = su4[m * sts + q];
          acc[m] = fmaf(8.0f * d, X, block_dot<NX>(p, xu + m * xts + 16 * q, lo, 0.125f * d, X, acc[m]));
        }
      }
    } else {
      uint32_t p[16];
      block_pairs<B>(b.w + q * B, pk, p);
      const float ds = d * (1.0f / (float)(1 << (7 - B)));
#pragma unroll
      for (int m = 0; m < TM; ++m)
        if (m < mc) acc[m] = block_dot<NX>(p, xu + m * xts + 16 * q, lo, ds, su4[m * sts + q], acc[m]);
    }
  }
}

template <int TM>
struct WideAcc {
  float v[TM];
};

// The staged tokens live in the kernel's dynamic LDS; naming it here (not
// through a pointer argument) keeps the accesses LDS instructions.
extern __shared__ uint32_t wide_lds[];

// This lane's share (units j, j + 8, ...) of row `row` against the staged
// tokens.  Not inlined: one function per width keeps each width's registers
// to itself (inlined together, the allocator merges all six).
template <int B, int NX, int TM, int LPR>
__device__ __noinline__ WideAcc<TM> wide_row_dot(const TensorDev t, int row, int U, int K, int j, int xts, int lo,
                                                 int sts, int mc) {
  const uint32_t* xl = wide_lds;
  const float* xs = reinterpret_cast<const float*>(wide_lds + TM * xts);
  WideAcc<TM> r;
#pragma unroll
  for (int m = 0; m < TM; ++m) r.v[m] = 0.0f;
  const int UPL = (U + LPR - 1) / LPR;
  WideUnit<B> buf[2];
  wide_load<B>(buf[0], t, row, U, min(j, U - 1), K);
#pragma unroll 1
  for (int i0 = 0; i0 < UPL; i0 += 2) {
    asm volatile("" ::: "memory");
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int i = i0 + b;
      if (i < UPL) {
        // the next unit (clamped to the last valid one) goes out before this one is reduced
        wide_load<B>(buf[1 - b], t, row, U, min(j + LPR * min(i + 1, UPL - 1), U - 1), K);
        const int u = j + LPR * i;
        if (u < U) wide_unit_dot<B, NX, TM>(buf[b], xl + u * kXStride, xts, lo, xs + u * 4, sts, mc, r.v);
      }
    }
  }
  return r;
}

template <int NX, int TM, int LPR>
__device__ __forceinline__ WideAcc<TM> wide_row_dot_any(const TensorDev& t, int row, int U, int K, int j, int xts,
                                                        int lo, int sts, int mc) {
  switch (t.bits) {
    case 2: return wide_row_dot<2, NX, TM, LPR>(t, row, U, K, j, xts, lo, sts, mc);
    case 3: return wide_row_dot<3, NX, TM, LPR>(t, row, U, K, j, xts, lo, sts, mc);
    case 4: return wide_row_dot<4, NX, TM, LPR>(t, row, U, K, j, xts, lo, sts, mc);
    case 5: return wide_row_dot<5, NX, TM, LPR>(t, row, U, K, j, xts, lo, sts, mc);
    case 6: return wide_row_dot<6, NX, TM, LPR>(t, row, U, K, j, xts, lo, sts, mc);
    default: return wide_row_dot<8, NX, TM, LPR>(t, row, U, K, j, xts, lo, sts, mc);
  }
}

// sum over the LPR lanes of a row group; the group's last lane holds it
template <int LPR>
__device__ __forceinline__ float wide_sum(float v) {
  if constexpr (LPR == 8)
    return half_sum8(v);
  else
    return group_sum<LPR>(v);
}

// grid = (ceil(I / (4 * 64 / LPR)), slots), 256 threads
template <int TM, int LPR>
__global__ __launch_bounds__(256) void wide_gateup_kernel(DecodeArgs a) {
  const Slot sl = slot_info(a, blockIdx.y);
  if (sl.M < 0 || sl.M > a.gemm_above) return;  // (large buckets: the grouped GEMMs)
  const TensorDev tg = a.desc[sl.desc * 3 + 0], tu = a.desc[sl.desc * 3 + 1];
  if (!tg.codes || !tu.codes) return;
  if (!wide_bits(tg.bits) && !wide_bits(tu.bits)) return;
  const int H = a.H, I = a.I, U = H / kUnit;
  const int xts = U * kXStride, sts = U * 4;
  uint32_t* xl = wide_lds;
  float* xs = reinterpret_cast<float*>(wide_lds + TM * xts);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  constexpr int RPW = 64 / LPR;  // rows per wave
  const int row = blockIdx.x * 4 * RPW + wave * RPW + lane / LPR, j = lane % LPR;
  const int rowc = min(row, I - 1);
  for (int m0 = 0; m0 < sl.M; m0 += TM) {
    const int mc = min(TM, sl.M - m0);
    __syncthreads();
    for (int m = 0; m < mc; ++m) {
      const int t = sl.shared >= 0 ? m0 + m : a.perm[sl.base + m0 + m] / a.k;
      const MOEQ_GLOBAL u32x4* src = gptr(reinterpret_cast<const u32x4*>(a.x + (size_t)t * H));
      for (int q = threadIdx.x; q < H / 8; q += 256) {
        const u32x4 v = src[q];
        float s = 0.0f;
        s += bf16_lo(v.x); s += bf16_hi(v.x); s += bf16_lo(v.y); s += bf16_hi(v.y);
        s += bf16_lo(v.z); s += bf16_hi(v.z); s += bf16_lo(v.w); s += bf16_hi(v.w);
        s += __shfl_xor(s, 1, 64);
        s += __shfl_xor(s, 2, 64);
        const int uu = q >> 4, cq = q & 15;
        *reinterpret_cast<u32x4*>(xl + m * xts + uu * kXStride + cq * 4) = v;
        if ((cq & 3) == 0) xs[m * sts + uu * 4 + (cq >> 2)] = s;
      }
    }
    __syncthreads();
    const WideAcc<TM> g = wide_row_dot_any<1, TM, LPR>(tg, rowc, U, H, j, xts, 0, sts, mc);
    const WideAcc<TM> u = wide_row_dot_any<1, TM, LPR>(tu, rowc, U, H, j, xts, 0, sts, mc);
#pragma unroll
    for (int m = 0; m < TM; ++m) {
      if (m < mc) {
        const float gs = wide_sum<LPR>(g.v[m]), us = wide_sum<LPR>(u.v[m]);
        if (j == LPR - 1 && row < I) a.h[(size_t)(sl.base + m0 + m) * I + row] = silu(gs) * us;
      }
    }
  }
}

// grid = (ceil(H / (4 * 64 / LPR)), slots), 256 threads
template <int TM, int LPR>
__global__ __launch_bounds__(256) void wide_down_kernel(DecodeArgs a) {
  const Slot sl = slot_info(a, blockIdx.y);
  if (sl.M < 0 || sl.M > a.gemm_above) return;  // (large buckets: the grouped GEMMs)
  const TensorDev td = a.desc[sl.desc * 3 + 2];
  if (!td.codes || !wide_bits(td.bits)) return;
  const int H = a.H, I = a.I, U = I / kUnit;
  const int xts = 2 * U * kXStride, sts = U * 4, lo = U * kXStride;
  uint32_t* xl = wide_lds;
  float* xs = reinterpret_cast<float*>(wide_lds + TM * xts);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  constexpr int RPW = 64 / LPR;  // rows per wave
  const int row = blockIdx.x * 4 * RPW + wave * RPW + lane / LPR, j = lane % LPR;
  const int rowc = min(row, H - 1);
  for (int m0 = 0; m0 < sl.M; m0 += TM) {
    const int mc = min(TM, sl.M - m0);
    __syncthreads();
    // h rows as bfloat16 hi + lo pairs; block sums of hi + lo
    for (int m = 0; m < mc; ++m) {
      const MOEQ_GLOBAL f32x4* src = gptr(reinterpret_cast<const f32x4*>(a.h + (size_t)(sl.base + m0 + m) * I));
      for (int q = threadIdx.x; q < I / 8; q += 256) {
        const f32x4 v0 = src[2 * q], v1 = src[2 * q + 1];
        const float f[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
        uint32_t hi[4], lw[4];
        float s = 0.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t h0 = bf16_rne(f[2 * i]), h1 = bf16_rne(f[2 * i + 1]);
          const uint32_t l0 = bf16_rne(f[2 * i] - __uint_as_float(h0 << 16));
          const uint32_t l1 = bf16_rne(f[2 * i + 1] - __uint_as_float(h1 << 16));
          hi[i] = h0 | h1 << 16;
          lw[i] = l0 | l1 << 16;
          s += __uint_as_float(h0 << 16) + __uint_as_float(l0 << 16);
          s += __uint_as_float(h1 << 16) + __uint_as_float(l1 << 16);
        }
        s += __shfl_xor(s, 1, 64);
        s += __shfl_xor(s, 2, 64);
        const int uu = q >> 4, cq = q & 15;
        uint32_t* dst = xl + m * xts + uu * kXStride + cq * 4;
        *reinterpret_cast<u32x4*>(dst) = u32x4{hi[0], hi[1], hi[2], hi[3]};
        *reinterpret_cast<u32x4*>(dst + lo) = u32x4{lw[0], lw[1], lw[2], lw[3]};
        if ((cq & 3) == 0) xs[m * sts + uu * 4 + (cq >> 2)] = s;
      }
    }
    __syncthreads();
    const WideAcc<TM> o = wide_row_dot_any<2, TM, LPR>(td, rowc, U, I, j, xts, lo, sts, mc);
#pragma unroll
    for (int m = 0; m < TM; ++m) {
      if (m < mc) {
        const float os = wide_sum<LPR>(o.v[m]);
        if (j == LPR - 1 && row < H) {
          int prow;
          float wv;
          if (sl.shared >= 0) {
            prow = a.n * a.k + sl.shared * a.n + m0 + m;
            wv = 1.0f;
          } else {
            prow = a.perm[sl.base + m0 + m];
            wv = a.w[prow];
          }
          a.partial[(size_t)prow * H + row] = wv * os;
        }
      }
    }
  }
}

// launches a kernel whose dynamic LDS may exceed the 64 KiB default
template <typename K>
hipError_t launch_lds(K kernel, dim3 grid, size_t lds, hipStream_t s, const DecodeArgs& a, int threads = 256) {
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  kernel<<<grid, threads, lds, s>>>(a);
  return hipGetLastError();
}

template <int TM, int LPR>
hipError_t launch_wide_gateup_tm(const DecodeArgs& a, hipStream_t s) {
  const int U = a.H / kUnit;
  const size_t lds = (size_t)TM * (U * kXStride + U * 4) * 4;
  const int rows_wg = 4 * (64 / LPR);
  dim3 grid((a.I + rows_wg - 1) / rows_wg, a.wide_gateup == 1 ? a.S : a.S + a.max_active);
  return launch_lds(wide_gateup_kernel<TM, LPR>, grid, lds, s, a);
}

template <int TM, int LPR>
hipError_t launch_wide_down_tm(const DecodeArgs& a, hipStream_t s) {
  const int U = a.I / kUnit;
  const size_t lds = (size_t)TM * (2 * U * kXStride + U * 4) * 4;
  const int rows_wg = 4 * (64 / LPR);
  dim3 grid((a.H + rows_wg - 1) / rows_wg, a.wide_down == 1 ? a.S : a.S + a.max_active);
  return launch_lds(wide_down_kernel<TM, LPR>, grid, lds, s, a);
}

// shared experts only: more lanes per row (as many as the units allow, up
// to 32 for gate/up and 16 for down) keep enough workgroups for a few slots
hipError_t launch_wide_gateup(const DecodeArgs& a, hipStream_t s) {
  if (!a.wide_gateup) return hipSuccess;
  const bool few = a.wide_gateup == 1 && a.H / kUnit >= 32;
  if (a.n == 1) return few ? launch_wide_gateup_tm<1, 32>(a, s) : launch_wide_gateup_tm<1, 8>(a, s);
  return few ? launch_wide_gateup_tm<4, 32>(a, s) : launch_wide_gateup_tm<4, 8>(a, s);
}

hipError_t launch_wide_down(const DecodeArgs& a, hipStream_t s) {
  if (!a.wide_down) return hipSuccess;
  const bool few = a.wide_down == 1 && a.I / kUnit >= 16;
  if (a.n == 1) return few ? launch_wide_down_tm<1, 16>(a, s) : launch_wide_down_tm<1, 8>(a, s);
  return few ? launch_wide_down_tm<4, 16>(a, s) : launch_wide_down_tm<4, 8>(a, s);
}

// Rows per wave step of the down GEMV are 64 / LPR; a workgroup covers
// 4 * (64 / LPR) * steps rows of one slot.

template <int LPR, int TM>
hipError_t launch_down_lpr_tm(const DecodeArgs& a, hipStream_t s) {
  const int slots = a.S + a.max_active;
  const int U = a.I / kUnit;
  const size_t lds = (size_t)TM * (U * kXStride + U * 8) * 4;
  constexpr int RW = TM == 1 ? kDownSteps : kDownStepsM, NB = TM == 1 ? kDownBuf : kDownBufM;
  const int rows_wg = 4 * (64 / LPR) * RW;
  dim3 grid((a.H + rows_wg - 1) / rows_wg, slots);
  return launch_lds(down_kernel<LPR, TM, RW, NB>, grid, lds, s, a);
}

template <int TM>
hipError_t launch_down_tm(const DecodeArgs& a, hipStream_t s) {
  const int U = a.I / kUnit;
  if (U > 32) return launch_down_lpr_tm<64, TM>(a, s);
  if (U > 16) return launch_down_lpr_tm<32, TM>(a, s);
  return launch_down_lpr_tm<16, TM>(a, s);
}

}  // namespace

// Gate/up: buckets of one token (every bucket when n = 1) take the
// one-token kernel, the others (n > 1) the kernel that stages 4 tokens at a
// time.  Down: one kernel per batch size (measured: splitting it the same way
// gains nothing at 16 tokens and costs 3 % at 64).
hipError_t launch_gateup_decode_single(const DecodeArgs& a, hipStream_t s) {
  const int U = a.H / kUnit;
  const size_t lds = (size_t)(U * kXStride + U * 8) * 4;
  dim3 grid((a.I + 15) / 16, a.S + a.max_active);
  gateup1_kernel<<<grid, 256, lds, s>>>(a);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? launch_wide_gateup(a, s) : e;
}

// tokens staged per pass of the 2-64-token gate/up kernel
#ifndef MOEQ_GATEUPN_TOKENS
#define MOEQ_GATEUPN_TOKENS 2
#endif
hipError_t launch_gateup_decode_multi(const DecodeArgs& a, hipStream_t s2) {
  constexpr int TM = MOEQ_GATEUPN_TOKENS;
  const int U = a.H / kUnit;
  const size_t lds = (size_t)TM * (U * kXStride + U * 8) * 4;
  dim3 grid((a.I + 15) / 16, a.S + a.max_active);
  return launch_lds(gateupn_kernel<TM>, grid, lds, s2, a);
}

bool gateup1_routes(const RouterParams& rp) { return !rp.kept_ids && !rp.x && rp.E_row <= 256 && rp.k <= kMaxTopK; }

hipError_t launch_gateup_decode_routing(const DecodeArgs& a, const RouterParams& rp, const Workspace& ws,
                                        hipStream_t s) {
  const int U = a.H / kUnit;
  const size_t lds = (size_t)(U * kXStride + U * 8) * 4;
  dim3 grid((a.I + 15) / 16, a.S + rp.k);
  if (rp.E_row <= 64)
    gateup1_route_kernel<1><<<grid, 256, lds, s>>>(a, rp, ws);
  else if (rp.E_row <= 128)
    gateup1_route_kernel<2><<<grid, 256, lds, s>>>(a, rp, ws);
  else
    gateup1_route_kernel<4><<<grid, 256, lds, s>>>(a, rp, ws);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? launch_wide_gateup(a, s) : e;
}

hipError_t launch_gateup_decode(const DecodeArgs& a, hipStream_t s) {
  hipError_t e = launch_gateup_decode_single(a, s);
  if (e == hipSuccess && a.n > 1) e = launch_gateup_decode_multi(a, s);
  return e;
}

namespace {
// threads per workgroup (NT / 16 rows) and slots in flight per lane (D) of
// the one-token down + combine kernel
#ifndef MOEQ_DOWN1_THREADS
#define MOEQ_DOWN1_THREADS 512
#endif
#ifndef MOEQ_DOWN1_DEPTH
#define MOEQ_DOWN1_DEPTH 3
#endif
size_t down1_lds(const DecodeArgs& a) {
  const size_t U = a.I / kUnit, NS = a.k + a.S;
  return NS * (U * kXStride * 4 + U * 4 * sizeof(float2));
}

template <int BD>
hipError_t launch_down1_b(const DecodeArgs& a, hipStream_t s) {
  constexpr int NT = MOEQ_DOWN1_THREADS, R = NT / 16;
  down1_kernel<BD, NT, MOEQ_DOWN1_DEPTH><<<(a.H + R - 1) / R, NT, down1_lds(a), s>>>(a);
  return hipGetLastError();
}
}  // namespace

bool down_combines(const DecodeArgs& a) {
  return a.n == 1 && a.wide_down == 0 && a.down_bits <= 4 && a.I / kUnit <= 16 &&
         down1_lds(a) <= 65536;
}

hipError_t launch_down_decode(const DecodeArgs& a, hipStream_t s) {
  if (down_combines(a)) {
    switch (a.down_bits) {
      case 0: return launch_down1_b<0>(a, s);  // widths differ between tensors
      case 2: return launch_down1_b<2>(a, s);
      case 3: return launch_down1_b<3>(a, s);
      default: return launch_down1_b<4>(a, s);
    }
  }
  const hipError_t e = a.n == 1 ? launch_down_tm<1>(a, s) : launch_down_tm<4>(a, s);
  return e == hipSuccess ? launch_wide_down(a, s) : e;
}

hipError_t launch_combine(const DecodeArgs& a, hipStream_t s) {
  const long long items = (long long)a.n * (a.H / 4);
  combine_kernel<<<(int)((items + 255) / 256), 256, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace moeq

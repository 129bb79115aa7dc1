// Prefill path: grouped GEMM on the matrix cores for many tokens.
//
// Every active expert (and the shared expert, whose bucket is all n tokens)
// multiplies its bucket of tokens by its weights, so the layer becomes a set
// of independent GEMMs of very different heights (routing is skewed).  The
// bucketing permutation lists each expert's tokens contiguously; a small
// kernel cuts every bucket into m-tiles of kGemmBM rows and writes the tile
// list, so the GEMM grids never depend on a host synchronization.
//
// Arithmetic: activations (bf16, exact in binary16 after a per-token
// power-of-two prescale), dequantized weights fp16(d * (c - z)) (one rounding)
// and the SwiGLU activations h (binary16 after a per-row power-of-two
// prescale) enter v_mfma_f32_16x16x32_f16 with float32 accumulation.  The
// packed-weight tile of each K step is decoded once per workgroup into LDS.
//
// Workgroup tile: 128 rows (tokens) x 128 output features (per projection;
// gate/up computes both projections of the same features so SwiGLU is fused
// into the epilogue), K step 64, four waves in a 2 x 2 arrangement, each
// owning a 64 x 64 block of 4 x 4 MFMA tiles.  The next K step's global data
// is loaded into registers while the current step's MFMAs run.  Workgroup ids
// are remapped so that consecutive tiles of one expert land on one XCD and
// share its L2.
#include "internal.h"
#include "layout.h"

namespace moeq {

namespace {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x4v __attribute__((ext_vector_type(4)));

constexpr int BM = kGemmBM, BN = 128, BK = 64;
constexpr int LDS_STRIDE = BK + 8;  // halves per LDS row (padding against bank conflicts)

// ---- tile list: slot order = shared experts, then active experts ----
__global__ __launch_bounds__(1024) void prefill_tiles_kernel(DecodeArgs a) {
  __shared__ int32_t cnt[kMaxShared + kMaxExperts + 1];
  __shared__ int32_t off[kMaxShared + kMaxExperts + 2];
  const int tid = threadIdx.x;
  const int nslots = a.S + a.active[0];
  for (int s = tid; s < nslots; s += 1024) {
    int M;
    if (s < a.S) {
      M = a.n;
    } else {
      const int e = a.active[1 + s - a.S];
      M = a.offsets[e + 1] - a.offsets[e];
    }
    cnt[s] = (M + BM - 1) / BM;
  }
  // rows of h whose running maxima the gate/up epilogue accumulates
  const int rows = a.n * (a.k + a.S);
  for (int r = tid; r < rows; r += 1024) a.rowmax[r] = 0u;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int s = 0; s < nslots; ++s) {
      off[s] = run;
      run += cnt[s];
    }
    off[nslots] = run;
    a.tiles[0] = min(run, a.max_mtiles);
  }
  __syncthreads();
  for (int s = tid; s < nslots; s += 1024)
    for (int i = 0; i < cnt[s]; ++i) {
      const int t = off[s] + i;
      if (t < a.max_mtiles) {
        a.tiles[1 + 2 * t] = s;
        a.tiles[2 + 2 * t] = i * BM;
      }
    }
}

struct SlotInfo {
  int desc, M, base, shared;
};

__device__ __forceinline__ SlotInfo slot_of(const DecodeArgs& a, int s) {
  SlotInfo r;
  if (s < a.S) {
    r.desc = a.E + s;
    r.M = a.n;
    r.base = a.n * a.k + s * a.n;
    r.shared = s;
  } else {
    const int e = a.active[1 + s - a.S];
    r.desc = e;
    r.base = a.offsets[e];
    r.M = a.offsets[e + 1] - r.base;
    r.shared = -1;
  }
  return r;
}

// Workgroup id -> logical id: the hardware deals workgroups to the 8 XCDs
// round-robin; consecutive logical ids are made to share an XCD.
__device__ __forceinline__ int xcd_logical(int hw, int total) {
  constexpr int X = 8;
  const int xcd = hw % X, idx = hw / X;
  const int per = total / X, extra = total % X;
  // XCDs [0, extra) own per + 1 ids, the rest own per
  return xcd < extra ? xcd * (per + 1) + idx : extra * (per + 1) + (xcd - extra) * per + idx;
}

// ---- weight tile decode: one thread, one row, two blocks (64 weights) ----
// Writes fp16(d * (c - z)) for k = [32*q0, 32*q0 + 64) of the row's unit u.
template <int B>
struct HalfUnit {
  uint32_t w[2 * B];
  uint32_t sc;  // two binary16 scales
};

template <int B>
__device__ __forceinline__ void load_half_unit(HalfUnit<B>& h, const TensorDev& t, int row, int kb0) {
  // kb0: first of the two blocks (even); unit u = kb0 / 4, half hs = (kb0 / 2) % 2
  const int K = t.K, U = K / kUnit, u = kb0 / 4, hs = (kb0 / 2) & 1;
  const MOEQ_GLOBAL u32x4* r4 = gptr(reinterpret_cast<const u32x4*>(t.codes + (size_t)row * B * U * 4));
  const int d0 = hs * 2 * B;  // first dword of the half unit
  if constexpr (B == 4) {
    const u32x4 v0 = __builtin_nontemporal_load(r4 + (size_t)(d0 / 4) * U + u);
    const u32x4 v1 = __builtin_nontemporal_load(r4 + (size_t)(d0 / 4 + 1) * U + u);
    h.w[0] = v0.x; h.w[1] = v0.y; h.w[2] = v0.z; h.w[3] = v0.w;
    h.w[4] = v1.x; h.w[5] = v1.y; h.w[6] = v1.z; h.w[7] = v1.w;
  } else if constexpr (B == 2) {
    const u32x4 v0 = __builtin_nontemporal_load(r4 + (size_t)(d0 / 4) * U + u);
    h.w[0] = v0.x; h.w[1] = v0.y; h.w[2] = v0.z; h.w[3] = v0.w;
  } else {
    // six dwords from two chunks: [0,6) or [6,12)
    const u32x4 v0 = __builtin_nontemporal_load(r4 + (size_t)(d0 / 4) * U + u);
    const u32x4 v1 = __builtin_nontemporal_load(r4 + (size_t)(d0 / 4 + 1) * U + u);
    if (hs == 0) {
      h.w[0] = v0.x; h.w[1] = v0.y; h.w[2] = v0.z; h.w[3] = v0.w; h.w[4] = v1.x; h.w[5] = v1.y;
    } else {
      h.w[0] = v0.z; h.w[1] = v0.w; h.w[2] = v1.x; h.w[3] = v1.y; h.w[4] = v1.z; h.w[5] = v1.w;
    }
  }
  h.sc = *gptr(reinterpret_cast<const uint32_t*>(t.scales + (size_t)row * (K / kBlock) + kb0));
}

// (c_lo, c_hi) at bit offset s of each half -> binary16 pair d * (c - z), exact
// code extraction through the 1024 + c binary16 bit trick, then one rounding.
template <int B, int S>
__device__ __forceinline__ uint32_t dq_pair(uint32_t w, uint32_t mask, uint32_t base, half2_t zb, half2_t d2) {
  const uint32_t v = and_or(w >> S, mask, base);
  const half2_t c = __builtin_bit_cast(half2_t, v) + zb;  // c - z, exact
  return __builtin_bit_cast(uint32_t, c * d2);          // rounded once
}

template <int B>
__device__ __forceinline__ void decode_half_unit(const HalfUnit<B>& h, _Float16* dst) {
  uint32_t mask, base;
  asm("v_mov_b32 %0, 0x64006400" : "=v"(base));
  if constexpr (B == 4) asm("v_mov_b32 %0, 0x000F000F" : "=v"(mask));
  if constexpr (B == 3) asm("v_mov_b32 %0, 0x00070007" : "=v"(mask));
  if constexpr (B == 2) asm("v_mov_b32 %0, 0x00030003" : "=v"(mask));
  const _Float16 zf = (_Float16)(-(1024.0f + (float)(1 << (B - 1))));
  const half2_t zb = {zf, zf};
#pragma unroll
  for (int blk = 0; blk < 2; ++blk) {
    const _Float16 d = __builtin_bit_cast(_Float16, (uint16_t)(h.sc >> (16 * blk)));
    const half2_t d2 = {d, d};
    const uint32_t* w = h.w + blk * B;
    uint32_t p[16];
    if constexpr (B == 4) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        p[4 * q + 0] = dq_pair<4, 0>(w[q], mask, base, zb, d2);
        p[4 * q + 1] = dq_pair<4, 4>(w[q], mask, base, zb, d2);
        p[4 * q + 2] = dq_pair<4, 8>(w[q], mask, base, zb, d2);
        p[4 * q + 3] = dq_pair<4, 12>(w[q], mask, base, zb, d2);
      }
    } else if constexpr (B == 2) {
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        p[8 * q + 0] = dq_pair<2, 0>(w[q], mask, base, zb, d2);
        p[8 * q + 1] = dq_pair<2, 2>(w[q], mask, base, zb, d2);
        p[8 * q + 2] = dq_pair<2, 4>(w[q], mask, base, zb, d2);
        p[8 * q + 3] = dq_pair<2, 6>(w[q], mask, base, zb, d2);
        p[8 * q + 4] = dq_pair<2, 8>(w[q], mask, base, zb, d2);
        p[8 * q + 5] = dq_pair<2, 10>(w[q], mask, base, zb, d2);
        p[8 * q + 6] = dq_pair<2, 12>(w[q], mask, base, zb, d2);
        p[8 * q + 7] = dq_pair<2, 14>(w[q], mask, base, zb, d2);
      }
    } else {
#pragma unroll
      for (int q = 0; q < 3; ++q) {
        p[5 * q + 0] = dq_pair<3, 0>(w[q], mask, base, zb, d2);
        p[5 * q + 1] = dq_pair<3, 3>(w[q], mask, base, zb, d2);
        p[5 * q + 2] = dq_pair<3, 6>(w[q], mask, base, zb, d2);
        p[5 * q + 3] = dq_pair<3, 9>(w[q], mask, base, zb, d2);
        p[5 * q + 4] = dq_pair<3, 12>(w[q], mask, base, zb, d2);
      }
      // weights 30, 31: bit q of each in bit 15 / 31 of dword q
      uint32_t m1, m2, m4;
      asm("v_mov_b32 %0, 0x00010001" : "=v"(m1));
      asm("v_mov_b32 %0, 0x00020002" : "=v"(m2));
      asm("v_mov_b32 %0, 0x00040004" : "=v"(m4));
      uint32_t t = and_or(w[0] >> 15, m1, base);
      t = and_or(w[1] >> 14, m2, t);
      t = and_or(w[2] >> 13, m4, t);
      const half2_t c = __builtin_bit_cast(half2_t, t) + zb;
      p[15] = __builtin_bit_cast(uint32_t, c * d2);
    }
    u32x4* o = reinterpret_cast<u32x4*>(dst + blk * 32);
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = u32x4{p[4 * i], p[4 * i + 1], p[4 * i + 2], p[4 * i + 3]};
  }
}

// ---- activation tile rows ----
// bf16 x (32 values) -> binary16 * 2^-e, into dst
__device__ __forceinline__ void convert_x32(const u32x4 (&v)[4], int e, _Float16* dst) {
  const float sc = __builtin_amdgcn_ldexpf(1.0f, -e);
  uint32_t o[16];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t q[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const half2_t hv = {(_Float16)(bf16_lo(q[j]) * sc), (_Float16)(bf16_hi(q[j]) * sc)};
      o[4 * i + j] = __builtin_bit_cast(uint32_t, hv);
    }
  }
  u32x4* d = reinterpret_cast<u32x4*>(dst);
#pragma unroll
  for (int i = 0; i < 4; ++i) d[i] = u32x4{o[4 * i], o[4 * i + 1], o[4 * i + 2], o[4 * i + 3]};
}

__device__ __forceinline__ half8 lds_frag(const _Float16* p) {
  return *reinterpret_cast<const half8*>(p);
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + expf(-g)); }

// ---------------------------------------------------------------------------
// gate/up grouped GEMM + SwiGLU.  Thread roles in the load phase: thread t
// decodes half a unit of row (t & 127) of tensor (t >> 7) and converts 32
// activations of tile row (t >> 1).
template <int BG, int BU>
__device__ void gateup_gemm_body(const DecodeArgs& a, const SlotInfo& sl, int m0, int n0,
                                 const TensorDev& tg, const TensorDev& tu, _Float16* lds) {
  _Float16* As = lds;                        // [BM][LDS_STRIDE]
  _Float16* Ws = lds + BM * LDS_STRIDE;      // [2][BN][LDS_STRIDE]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int H = a.H, I = a.I;
  // load-phase roles
  const int wt = tid >> 7, wrow = n0 + (tid & 127);
  const int arow = tid >> 1, akh = tid & 1;
  const bool arow_ok = m0 + arow < sl.M;
  int tok = 0, xe = 0;
  if (arow_ok) {
    tok = sl.shared >= 0 ? m0 + arow : a.perm[sl.base + m0 + arow] / a.k;
    xe = a.xexp[tok];
  }
  const MOEQ_GLOBAL u32x4* xrow = gptr(reinterpret_cast<const u32x4*>(a.x + (size_t)tok * H));

  f32x4v accg[4][4], accu[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) accg[i][c] = accu[i][c] = f32x4v{0.f, 0.f, 0.f, 0.f};

  HalfUnit<BG> hg;
  HalfUnit<BU> hu;
  u32x4 xv[4];
  auto fetch = [&](int k0) {
    if (wt == 0)
      load_half_unit<BG>(hg, tg, wrow, k0 / 32);
    else
      load_half_unit<BU>(hu, tu, wrow, k0 / 32);
    if (arow_ok) {
#pragma unroll
      for (int i = 0; i < 4; ++i) xv[i] = xrow[(k0 + 32 * akh) / 8 + i];
    }
  };
  fetch(0);
  const int nk = H / BK;
  for (int ks = 0; ks < nk; ++ks) {
    // registers -> LDS
    if (wt == 0)
      decode_half_unit<BG>(hg, Ws + (tid & 127) * LDS_STRIDE);
    else
      decode_half_unit<BU>(hu, Ws + (BN + (tid & 127)) * LDS_STRIDE);
    {
      _Float16* dst = As + arow * LDS_STRIDE + 32 * akh;
      if (arow_ok) {
        convert_x32(xv, xe, dst);
      } else {
        u32x4* d = reinterpret_cast<u32x4*>(dst);
#pragma unroll
        for (int i = 0; i < 4; ++i) d[i] = u32x4{0u, 0u, 0u, 0u};
      }
    }
    __syncthreads();
    if (ks + 1 < nk) fetch((ks + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int kof = kk * 32 + (lane >> 4) * 8;
      half8 af[4], bg[4], bu[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = lds_frag(As + (wm * 64 + 16 * i + (lane & 15)) * LDS_STRIDE + kof);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        bg[c] = lds_frag(Ws + (wn * 64 + 16 * c + (lane & 15)) * LDS_STRIDE + kof);
        bu[c] = lds_frag(Ws + (BN + wn * 64 + 16 * c + (lane & 15)) * LDS_STRIDE + kof);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          accg[i][c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[i], bg[c], accg[i][c], 0, 0, 0);
          accu[i][c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[i], bu[c], accu[i][c], 0, 0, 0);
        }
    }
    __syncthreads();
  }

  // epilogue: undo the activation prescale, SwiGLU, store h, track row maxima
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = wm * 64 + 16 * i + (lane >> 4) * 4 + j;
      const bool ok = m0 + r < sl.M;
      float sc = 1.0f;
      if (ok) {
        const int t = sl.shared >= 0 ? m0 + r : a.perm[sl.base + m0 + r] / a.k;
        sc = __builtin_amdgcn_ldexpf(1.0f, a.xexp[t]);
      }
      float rmax = 0.0f;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int col = n0 + wn * 64 + 16 * c + (lane & 15);
        const float hv = silu(accg[i][c][j] * sc) * (accu[i][c][j] * sc);
        if (ok) a.h[(size_t)(sl.base + m0 + r) * I + col] = hv;
        rmax = fmaxf(rmax, fabsf(hv));
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) rmax = fmaxf(rmax, __shfl_xor(rmax, off, 64));
      if (ok && (lane & 15) == 0) atomicMax(a.rowmax + sl.base + m0 + r, __float_as_uint(rmax));
    }
  }
}

__global__ __launch_bounds__(256, 2) void gateup_gemm_kernel(DecodeArgs a) {
  extern __shared__ _Float16 lds_h[];
  const int nN = a.I / BN;
  const int L = xcd_logical(blockIdx.x, gridDim.x);
  const int mt = L / nN, nt = L % nN;
  if (mt >= a.tiles[0]) return;
  const SlotInfo sl = slot_of(a, a.tiles[1 + 2 * mt]);
  const int m0 = a.tiles[2 + 2 * mt];
  const TensorDev tg = a.desc[sl.desc * 3 + 0], tu = a.desc[sl.desc * 3 + 1];
  if (!tg.codes || !tu.codes) return;
  switch (tg.bits * 8 + tu.bits) {
    case 2 * 8 + 2: gateup_gemm_body<2, 2>(a, sl, m0, nt * BN, tg, tu, lds_h); break;
    case 2 * 8 + 3: gateup_gemm_body<2, 3>(a, sl, m0, nt * BN, tg, tu, lds_h); break;
    case 2 * 8 + 4: gateup_gemm_body<2, 4>(a, sl, m0, nt * BN, tg, tu, lds_h); break;
    case 3 * 8 + 2: gateup_gemm_body<3, 2>(a, sl, m0, nt * BN, tg, tu, lds_h); break;
    case 3 * 8 + 3: gateup_gemm_body<3, 3>(a, sl, m0, nt * BN, tg, tu, lds_h); break;
    case 3 * 8 + 4: gateup_gemm_body<3, 4>(a, sl, m0, nt * BN, tg, tu, lds_h); break;
    case 4 * 8 + 2: gateup_gemm_body<4, 2>(a, sl, m0, nt * BN, tg, tu, lds_h); break;
    case 4 * 8 + 3: gateup_gemm_body<4, 3>(a, sl, m0, nt * BN, tg, tu, lds_h); break;
    case 4 * 8 + 4: gateup_gemm_body<4, 4>(a, sl, m0, nt * BN, tg, tu, lds_h); break;
    default: break;
  }
}

// ---------------------------------------------------------------------------
// down grouped GEMM x routing weight -> partial rows.  Load-phase roles:
// waves 0-1 decode the weight tile (thread t: row t, both halves of K step),
// waves 2-3 convert the activation tile (thread t - 128: row t - 128).
template <int BD>
__device__ void down_gemm_body(const DecodeArgs& a, const SlotInfo& sl, int m0, int n0,
                               const TensorDev& td, _Float16* lds) {
  _Float16* As = lds;                    // [BM][LDS_STRIDE]
  _Float16* Ws = lds + BM * LDS_STRIDE;  // [BN][LDS_STRIDE]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int H = a.H, I = a.I;
  const bool wrole = tid < 128;
  const int r = tid & 127;  // weight row (n0 + r) or activation row (m0 + r)
  const bool arow_ok = !wrole && m0 + r < sl.M;
  int he = 0;
  if (arow_ok) he = max(0, (int)((a.rowmax[sl.base + m0 + r] >> 23) & 0xFFu) - 127 - 14);
  const MOEQ_GLOBAL f32x4v* hrow =
      gptr(reinterpret_cast<const f32x4v*>(a.h + (size_t)(sl.base + m0 + (arow_ok ? r : 0)) * I));

  f32x4v acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[i][c] = f32x4v{0.f, 0.f, 0.f, 0.f};

  HalfUnit<BD> h0, h1;
  f32x4v hv[16];
  auto fetch = [&](int k0) {
    if (wrole) {
      load_half_unit<BD>(h0, td, n0 + r, k0 / 32);
    } else if (arow_ok) {
#pragma unroll
      for (int i = 0; i < 16; ++i) hv[i] = hrow[k0 / 4 + i];
    }
  };
  fetch(0);
  const int nk = I / BK;
  for (int ks = 0; ks < nk; ++ks) {
    if (wrole) {
      decode_half_unit<BD>(h0, Ws + r * LDS_STRIDE);
    } else {
      _Float16* dst = As + r * LDS_STRIDE;
      uint32_t o[32];
      const float sc = __builtin_amdgcn_ldexpf(1.0f, -he);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const half2_t p0 = {(_Float16)(hv[i][0] * sc), (_Float16)(hv[i][1] * sc)};
        const half2_t p1 = {(_Float16)(hv[i][2] * sc), (_Float16)(hv[i][3] * sc)};
        o[2 * i] = arow_ok ? __builtin_bit_cast(uint32_t, p0) : 0u;
        o[2 * i + 1] = arow_ok ? __builtin_bit_cast(uint32_t, p1) : 0u;
      }
      u32x4* d = reinterpret_cast<u32x4*>(dst);
#pragma unroll
      for (int i = 0; i < 8; ++i) d[i] = u32x4{o[4 * i], o[4 * i + 1], o[4 * i + 2], o[4 * i + 3]};
    }
    __syncthreads();
    if (ks + 1 < nk) fetch((ks + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int kof = kk * 32 + (lane >> 4) * 8;
      half8 af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = lds_frag(As + (wm * 64 + 16 * i + (lane & 15)) * LDS_STRIDE + kof);
#pragma unroll
      for (int c = 0; c < 4; ++c) bf[c] = lds_frag(Ws + (wn * 64 + 16 * c + (lane & 15)) * LDS_STRIDE + kof);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int c = 0; c < 4; ++c)
          acc[i][c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[i], bf[c], acc[i][c], 0, 0, 0);
    }
    __syncthreads();
  }
  (void)h1;

  // epilogue: undo the row prescale, scale by the routing weight, store partials
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int rr = wm * 64 + 16 * i + (lane >> 4) * 4 + j;
      if (m0 + rr >= sl.M) continue;
      const int e = max(0, (int)((a.rowmax[sl.base + m0 + rr] >> 23) & 0xFFu) - 127 - 14);
      int prow;
      float wv;
      if (sl.shared >= 0) {
        prow = a.n * a.k + sl.shared * a.n + m0 + rr;
        wv = 1.0f;
      } else {
        prow = a.perm[sl.base + m0 + rr];
        wv = a.w[prow];
      }
      const float sc = __builtin_amdgcn_ldexpf(wv, e);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int col = n0 + wn * 64 + 16 * c + (lane & 15);
        a.partial[(size_t)prow * H + col] = acc[i][c][j] * sc;
      }
    }
  }
}

__global__ __launch_bounds__(256, 2) void down_gemm_kernel(DecodeArgs a) {
  extern __shared__ _Float16 lds_h[];
  const int nN = a.H / BN;
  const int L = xcd_logical(blockIdx.x, gridDim.x);
  const int mt = L / nN, nt = L % nN;
  if (mt >= a.tiles[0]) return;
  const SlotInfo sl = slot_of(a, a.tiles[1 + 2 * mt]);
  const int m0 = a.tiles[2 + 2 * mt];
  const TensorDev td = a.desc[sl.desc * 3 + 2];
  if (!td.codes) return;
  switch (td.bits) {
    case 2: down_gemm_body<2>(a, sl, m0, nt * BN, td, lds_h); break;
    case 3: down_gemm_body<3>(a, sl, m0, nt * BN, td, lds_h); break;
    case 4: down_gemm_body<4>(a, sl, m0, nt * BN, td, lds_h); break;
    default: break;
  }
}

}  // namespace

int prefill_max_mtiles(int n, int k, int S, int n_kept) {
  const long long nk = (long long)n * k;
  const long long routed = (nk + BM - 1) / BM + (nk < n_kept ? nk : n_kept);
  return (int)(routed + (long long)S * ((n + BM - 1) / BM));
}

hipError_t launch_gateup_prefill(const DecodeArgs& a, hipStream_t s) {
  prefill_tiles_kernel<<<1, 1024, 0, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t lds = (size_t)(BM + 2 * BN) * LDS_STRIDE * sizeof(_Float16);
  const int grid = a.max_mtiles * (a.I / BN);
  gateup_gemm_kernel<<<grid, 256, lds, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_down_prefill(const DecodeArgs& a, hipStream_t s) {
  const size_t lds = (size_t)(BM + BN) * LDS_STRIDE * sizeof(_Float16);
  const int grid = a.max_mtiles * (a.H / BN);
  down_gemm_kernel<<<grid, 256, lds, s>>>(a);
  return hipGetLastError();
}

}  // namespace moeq

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
// owning a 64 x 64 block of 4 x 4 MFMA tiles.  LDS holds two decoded K steps
// and registers the raw data of the next two, so the decode of one step and
// the loads of later ones overlap the current step's MFMAs.  Workgroup ids
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
// The raw codes of half a unit (2*B dwords starting at dword 2*B*hs of the
// unit) come from the two 16-byte chunks c0 = (2*B*hs)/4 and c1 = min(c0+1,
// B-1) of the unit; they are kept as loaded (no selection at load time, so
// the loads stay in flight) and picked apart when the tile is decoded.
struct Raw {
  u32x4 a, b;
  uint32_t sc;  // the two binary16 scales of the half unit
};

// Row-base pointer of a tensor row in the device layout.
__device__ __forceinline__ const MOEQ_GLOBAL u32x4* row_chunks(const TensorDev& t, int bits, int row) {
  const int U = t.K / kUnit;
  return gptr(reinterpret_cast<const u32x4*>(t.codes + (size_t)row * bits * U * 4));
}

// Half unit hs of unit u of a row (its blocks 4u + 2hs, 4u + 2hs + 1).
__device__ __forceinline__ Raw load_raw(const MOEQ_GLOBAL u32x4* rc, const MOEQ_GLOBAL uint32_t* rs, int U,
                                        int bits, int u, int hs) {
  const int c0 = (2 * bits * hs) >> 2;
  const int c1 = min(c0 + 1, bits - 1);
  Raw r;
  r.a = rc[(size_t)c0 * U + u];
  r.b = rc[(size_t)c1 * U + u];
  r.sc = rs[2 * u + hs];
  return r;
}

// (c_lo, c_hi) at bit offset s of each half -> binary16 pair d * (c - z), exact
// code extraction through the 1024 + c binary16 bit trick, then one rounding.
template <int S>
__device__ __forceinline__ uint32_t dq_pair(uint32_t w, uint32_t mask, uint32_t base, half2_t zb, half2_t d2) {
  const uint32_t v = and_or(w >> S, mask, base);
  const half2_t c = __builtin_bit_cast(half2_t, v) + zb;  // c - z, exact
  return __builtin_bit_cast(uint32_t, c * d2);          // rounded once
}

// Decodes the half unit in r (width B, half HS) to 64 binary16 values at dst.
template <int B, int HS>
__device__ __forceinline__ void decode_raw(const Raw& r, _Float16* dst) {
  const uint32_t all[8] = {r.a.x, r.a.y, r.a.z, r.a.w, r.b.x, r.b.y, r.b.z, r.b.w};
  constexpr int o = (B == 3 && HS) ? 2 : 0;  // first dword of the half unit within chunk c0
  uint32_t mask, base;
  asm("v_mov_b32 %0, 0x64006400" : "=v"(base));
  if constexpr (B == 4) asm("v_mov_b32 %0, 0x000F000F" : "=v"(mask));
  if constexpr (B == 3) asm("v_mov_b32 %0, 0x00070007" : "=v"(mask));
  if constexpr (B == 2) asm("v_mov_b32 %0, 0x00030003" : "=v"(mask));
  const _Float16 zf = (_Float16)(-(1024.0f + (float)(1 << (B - 1))));
  const half2_t zb = {zf, zf};
#pragma unroll
  for (int blk = 0; blk < 2; ++blk) {
    const _Float16 d = __builtin_bit_cast(_Float16, (uint16_t)(r.sc >> (16 * blk)));
    const half2_t d2 = {d, d};
    const uint32_t* w = all + o + blk * B;
    uint32_t p[16];
    if constexpr (B == 4) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        p[4 * q + 0] = dq_pair<0>(w[q], mask, base, zb, d2);
        p[4 * q + 1] = dq_pair<4>(w[q], mask, base, zb, d2);
        p[4 * q + 2] = dq_pair<8>(w[q], mask, base, zb, d2);
        p[4 * q + 3] = dq_pair<12>(w[q], mask, base, zb, d2);
      }
    } else if constexpr (B == 2) {
#pragma unroll
      for (int q = 0; q < 2; ++q) {
#pragma unroll
        for (int f = 0; f < 8; ++f) p[8 * q + f] = dq_pair<0>(w[q] >> (2 * f), mask, base, zb, d2);
      }
    } else {
#pragma unroll
      for (int q = 0; q < 3; ++q) {
#pragma unroll
        for (int f = 0; f < 5; ++f) p[5 * q + f] = dq_pair<0>(w[q] >> (3 * f), mask, base, zb, d2);
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
    u32x4* out = reinterpret_cast<u32x4*>(dst + blk * 32);
#pragma unroll
    for (int i = 0; i < 4; ++i) out[i] = u32x4{p[4 * i], p[4 * i + 1], p[4 * i + 2], p[4 * i + 3]};
  }
}

// ---- activation tile rows ----
// 32 binary16 values (already prescaled) from registers into an LDS row
__device__ __forceinline__ void store_row32(const u32x4 (&v)[4], _Float16* dst) {
  u32x4* d = reinterpret_cast<u32x4*>(dst);
#pragma unroll
  for (int i = 0; i < 4; ++i) d[i] = v[i];
}

__device__ __forceinline__ half8 lds_frag(const _Float16* p) {
  return *reinterpret_cast<const half8*>(p);
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + expf(-g)); }

// ---------------------------------------------------------------------------
// gate/up grouped GEMM + SwiGLU.  Thread roles in the load phase: thread t
// decodes half a unit of row (t & 127) of tensor (t >> 7) and converts 32
// activations of tile row (t >> 1).
// Field copies of the kernel arguments the GEMM bodies use (passing the
// argument struct by reference would place it in scratch memory).
struct GemmArgs {
  const uint16_t* x;
  const uint16_t* x16;
  uint16_t* h16;
  const int32_t* perm;
  const int32_t* xexp;
  const float* w;
  float* h;
  float* partial;
  uint32_t* rowmax;
  int n, H, I, k;
};

__device__ __forceinline__ GemmArgs gemm_args(const DecodeArgs& a) {
  GemmArgs g;
  g.x = a.x;
  g.x16 = a.x16;
  g.h16 = a.h16;
  g.perm = a.perm;
  g.xexp = a.xexp;
  g.w = a.w;
  g.h = a.h;
  g.partial = a.partial;
  g.rowmax = a.rowmax;
  g.n = a.n;
  g.H = a.H;
  g.I = a.I;
  g.k = a.k;
  return g;
}

// A/B fragments of one K step (two MFMA K slices of 32) of a wave's 64 x 64
// block, for NT weight tensors that share the activation fragments.
template <int NT>
struct Frags {
  half8 a[2][4];
  half8 b[2][NT][4];
};

template <int NT>
__device__ __forceinline__ void read_frags(const _Float16* A, const _Float16* W, int lane, int wm, int wn,
                                           Frags<NT>& f) {
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const int kof = kk * 32 + (lane >> 4) * 8;
#pragma unroll
    for (int i = 0; i < 4; ++i) f.a[kk][i] = lds_frag(A + (wm * 64 + 16 * i + (lane & 15)) * LDS_STRIDE + kof);
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int c = 0; c < 4; ++c)
        f.b[kk][t][c] = lds_frag(W + (t * BN + wn * 64 + 16 * c + (lane & 15)) * LDS_STRIDE + kof);
  }
}

template <int NT>
__device__ __forceinline__ void mfmas(const Frags<NT>& f, f32x4v (&acc)[NT][4][4]) {
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc[t][i][c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(f.a[kk][i], f.b[kk][t][c], acc[t][i][c], 0, 0, 0);
}

// Scheduling hint for one pipelined K step: the fragment reads first, then
// the step's MFMAs each followed by a few VALU instructions of the next
// step's decode (and its LDS writes), so that the matrix core and the vector
// ALU work at the same time; the loads of a later step go in the middle.
template <int NMFMA, int NREAD, int NVALU, int NWRITE>
__device__ __forceinline__ void interleave_hint() {
  __builtin_amdgcn_sched_group_barrier(0x100, NREAD, 0);  // DS read
#pragma unroll
  for (int i = 0; i < NMFMA; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);      // MFMA
    __builtin_amdgcn_sched_group_barrier(0x002, NVALU, 0);  // VALU
    if (i % (NMFMA / NWRITE) == NMFMA / NWRITE - 1) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // DS write
    if (i == NMFMA / 2) __builtin_amdgcn_sched_group_barrier(0x020, 16, 0);  // VMEM read
  }
}

// The pipelined K loop of the gate/up GEMM for a wave whose weight rows have
// width B.  LDS holds two decoded K steps (double buffer), registers hold the
// raw data of the next two steps.  While step s is multiplied, step s+1 is
// decoded into the other LDS buffer and the loads of step s+3 go into the
// register slot just consumed.  Step s uses register slot and LDS buffer
// s % 2, and half unit s % 2 of unit s / 2.  nk is even (H is a multiple of
// 128); loads and decodes are unconditional (the last ones repeat the final
// steps into buffers nobody reads again) so that every K step is one basic
// block and the wait counts stay exact.
template <int B>
__device__ __forceinline__ void gateup_loop(const MOEQ_GLOBAL u32x4* rc, const MOEQ_GLOBAL uint32_t* rs, int U,
                                            const MOEQ_GLOBAL u32x4* xrow, _Float16* wdst, _Float16* adst,
                                            const _Float16* As, const _Float16* Ws, int lane, int wm, int wn,
                                            int nk, f32x4v (&acc)[2][4][4]) {
  Raw hw[2];
  u32x4 xv[2][4];
#define GU_LOAD(slot, st)                                                                       \
  do {                                                                                          \
    hw[slot] = load_raw(rc, rs, U, B, (st) >> 1, slot);                                         \
    _Pragma("unroll") for (int i_ = 0; i_ < 4; ++i_) xv[slot][i_] = xrow[(st) * (BK / 8) + i_]; \
  } while (0)
#define GU_DECODE(slot)                                                        \
  do {                                                                         \
    decode_raw<B, slot>(hw[slot], wdst + (slot) * (2 * BN * LDS_STRIDE));       \
    store_row32(xv[slot], adst + (slot) * (BM * LDS_STRIDE));                  \
  } while (0)
#define GU_STEP(P, st_next)                                                                    \
  do {                                                                                         \
    Frags<2> f;                                                                                \
    read_frags<2>(As + (P) * (BM * LDS_STRIDE), Ws + (P) * (2 * BN * LDS_STRIDE), lane, wm, wn, f); \
    GU_DECODE(1 - (P));                                                                        \
    GU_LOAD(1 - (P), st_next);                                                                 \
    mfmas<2>(f, acc);                                                                          \
    interleave_hint<64, 24, 4, 12>();                                                          \
    __syncthreads();                                                                           \
  } while (0)
  GU_LOAD(0, 0);
  GU_LOAD(1, 1);
  GU_DECODE(0);
  GU_LOAD(0, min(2, nk - 2));
  __syncthreads();
  for (int s0 = 0; s0 < nk; s0 += 2) {
    GU_STEP(0, min(s0 + 3, nk - 1));  // step s0; decodes s0 + 1, loads s0 + 3
    GU_STEP(1, min(s0 + 4, nk - 2));  // step s0 + 1; decodes s0 + 2, loads s0 + 4
  }
#undef GU_LOAD
#undef GU_DECODE
#undef GU_STEP
}

__device__ void gateup_gemm_body(const GemmArgs a, const SlotInfo sl, int m0, int n0,
                                 const TensorDev tg, const TensorDev tu, _Float16* lds) {
  _Float16* As = lds;                            // [2][BM][LDS_STRIDE]
  _Float16* Ws = lds + 2 * BM * LDS_STRIDE;      // [2][2][BN][LDS_STRIDE]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int H = a.H, I = a.I, U = H / kUnit;
  const MOEQ_GLOBAL int32_t* perm = gptr(a.perm);
  const MOEQ_GLOBAL int32_t* xexp = gptr(a.xexp);
  // Load-phase roles.  Weights: waves 0-1 take gate rows, waves 2-3 up rows
  // (so the tensor, hence the width, is wave-uniform); thread t decodes half a
  // unit of row t & 127.  Activations (the prescaled binary16 copy of x): thread
  // t moves 32 values of tile row t >> 1.  Rows past the bucket read token row
  // 0: they only feed output rows that are never stored.
  const int wt = __builtin_amdgcn_readfirstlane(tid >> 7);
  const TensorDev t = wt ? tu : tg;
  const int bits = __builtin_amdgcn_readfirstlane(t.bits);
  const int wrow = n0 + (tid & 127);
  const MOEQ_GLOBAL u32x4* rc = row_chunks(t, bits, wrow);
  const MOEQ_GLOBAL uint32_t* rs = gptr(reinterpret_cast<const uint32_t*>(t.scales + (size_t)wrow * (H / kBlock)));
  _Float16* wdst = Ws + (wt * BN + (tid & 127)) * LDS_STRIDE;
  const int arow = tid >> 1, akh = tid & 1;
  int tok = 0;
  if (m0 + arow < sl.M) tok = sl.shared >= 0 ? m0 + arow : perm[sl.base + m0 + arow] / a.k;
  const MOEQ_GLOBAL u32x4* xrow = gptr(reinterpret_cast<const u32x4*>(a.x16 + (size_t)tok * H)) + 4 * akh;
  _Float16* adst = As + arow * LDS_STRIDE + 32 * akh;

  f32x4v acc[2][4][4];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[q][i][c] = f32x4v{0.f, 0.f, 0.f, 0.f};

  const int nk = H / BK;
  if (bits == 2)
    gateup_loop<2>(rc, rs, U, xrow, wdst, adst, As, Ws, lane, wm, wn, nk, acc);
  else if (bits == 3)
    gateup_loop<3>(rc, rs, U, xrow, wdst, adst, As, Ws, lane, wm, wn, nk, acc);
  else
    gateup_loop<4>(rc, rs, U, xrow, wdst, adst, As, Ws, lane, wm, wn, nk, acc);

  // epilogue: undo the activation prescale, SwiGLU, store h, track row maxima
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = wm * 64 + 16 * i + (lane >> 4) * 4 + j;
      const bool ok = m0 + r < sl.M;
      float sc = 1.0f;
      if (ok) {
        const int tk = sl.shared >= 0 ? m0 + r : perm[sl.base + m0 + r] / a.k;
        sc = __builtin_amdgcn_ldexpf(1.0f, xexp[tk]);
      }
      float rmax = 0.0f;
      MOEQ_GLOBAL float* hout = (MOEQ_GLOBAL float*)(a.h + (size_t)(sl.base + m0 + r) * I);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int col = n0 + wn * 64 + 16 * c + (lane & 15);
        const float hv = silu(acc[0][i][c][j] * sc) * (acc[1][i][c][j] * sc);
        if (ok) hout[col] = hv;
        rmax = fmaxf(rmax, fabsf(hv));
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) rmax = fmaxf(rmax, __shfl_xor(rmax, off, 64));
      if (ok && (lane & 15) == 0) atomicMax(a.rowmax + sl.base + m0 + r, __float_as_uint(rmax));
    }
  }
}

__global__ __launch_bounds__(256, 1) void gateup_gemm_kernel(DecodeArgs a) {
  extern __shared__ _Float16 lds_h[];
  const int nN = a.I / BN;
  const int L = xcd_logical(blockIdx.x, gridDim.x);
  const int mt = L / nN, nt = L % nN;
  if (mt >= a.tiles[0]) return;
  const SlotInfo sl = slot_of(a, a.tiles[1 + 2 * mt]);
  const int m0 = a.tiles[2 + 2 * mt];
  const TensorDev tg = a.desc[sl.desc * 3 + 0], tu = a.desc[sl.desc * 3 + 1];
  if (!tg.codes || !tu.codes) return;
  if (tg.bits < 2 || tg.bits > 4 || tu.bits < 2 || tu.bits > 4) return;
  gateup_gemm_body(gemm_args(a), sl, m0, nt * BN, tg, tu, lds_h);
}

// ---------------------------------------------------------------------------
// h -> binary16 rows prescaled by 2^-e, e from the row's maximum |h|, so
// that the largest value stays below 2^15 (one rounding to nearest even).
// One wave per row of h.
__global__ __launch_bounds__(256) void h16_kernel(const float* h, const uint32_t* rowmax, int rows, int I,
                                                 uint16_t* h16) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= rows) return;
  const int e = max(0, (int)((rowmax[row] >> 23) & 0xFFu) - 127 - 14);
  const float sc = __builtin_amdgcn_ldexpf(1.0f, -e);
  const MOEQ_GLOBAL f32x4v* src = gptr(reinterpret_cast<const f32x4v*>(h + (size_t)row * I));
  MOEQ_GLOBAL u32x2* dst = (MOEQ_GLOBAL u32x2*)(h16 + (size_t)row * I);
  for (int c = lane; c < I / 4; c += 64) {
    const f32x4v v = __builtin_nontemporal_load(src + c);
    const half2_t p0 = {(_Float16)(v[0] * sc), (_Float16)(v[1] * sc)};
    const half2_t p1 = {(_Float16)(v[2] * sc), (_Float16)(v[3] * sc)};
    dst[c] = u32x2{__builtin_bit_cast(uint32_t, p0), __builtin_bit_cast(uint32_t, p1)};
  }
}

// down grouped GEMM x routing weight -> partial rows.  Load-phase roles:
// thread t decodes block t >> 7 of the K step of weight row n0 + (t & 127)
// and moves the 32 binary16 activations of half t >> 7 of the K step of tile
// row t & 127.

// Block q = 2*hs + half of unit u (32 weights, B dwords at dword q*B of the
// unit): chunks c0 = q*B/4 and min(c0+1, B-1), and the block's scale.
struct RawBlk {
  u32x4 a, b;
  uint32_t sc;
};

__device__ __forceinline__ RawBlk load_blk(const MOEQ_GLOBAL u32x4* rc, const MOEQ_GLOBAL uint16_t* rs, int U,
                                           int bits, int u, int q) {
  const int c0 = (q * bits) >> 2;
  const int c1 = min(c0 + 1, bits - 1);
  RawBlk r;
  r.a = rc[(size_t)c0 * U + u];
  r.b = rc[(size_t)c1 * U + u];
  r.sc = rs[4 * u + q];
  return r;
}

// Decodes one block (width B) whose first dword is dword o (0..3, wave-
// uniform) of the loaded pair of chunks.
template <int B>
__device__ __forceinline__ void decode_blk(const RawBlk& r, int o, _Float16* dst) {
  const uint32_t all[8] = {r.a.x, r.a.y, r.a.z, r.a.w, r.b.x, r.b.y, r.b.z, r.b.w};
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < B; ++i)
    w[i] = o == 0 ? all[i] : o == 1 ? all[i + 1] : o == 2 ? all[i + 2] : all[i + 3];
  uint32_t mask, base;
  asm("v_mov_b32 %0, 0x64006400" : "=v"(base));
  if constexpr (B == 4) asm("v_mov_b32 %0, 0x000F000F" : "=v"(mask));
  if constexpr (B == 3) asm("v_mov_b32 %0, 0x00070007" : "=v"(mask));
  if constexpr (B == 2) asm("v_mov_b32 %0, 0x00030003" : "=v"(mask));
  const _Float16 zf = (_Float16)(-(1024.0f + (float)(1 << (B - 1))));
  const half2_t zb = {zf, zf};
  const _Float16 d = __builtin_bit_cast(_Float16, (uint16_t)r.sc);
  const half2_t d2 = {d, d};
  uint32_t p[16];
  if constexpr (B == 4) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int f = 0; f < 4; ++f) p[4 * q + f] = dq_pair<0>(w[q] >> (4 * f), mask, base, zb, d2);
  } else if constexpr (B == 2) {
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int f = 0; f < 8; ++f) p[8 * q + f] = dq_pair<0>(w[q] >> (2 * f), mask, base, zb, d2);
  } else {
#pragma unroll
    for (int q = 0; q < 3; ++q)
#pragma unroll
      for (int f = 0; f < 5; ++f) p[5 * q + f] = dq_pair<0>(w[q] >> (3 * f), mask, base, zb, d2);
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
  u32x4* out = reinterpret_cast<u32x4*>(dst);
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = u32x4{p[4 * i], p[4 * i + 1], p[4 * i + 2], p[4 * i + 3]};
}

// The pipelined K loop of the down GEMM for width B (same scheme as the
// gate/up loop).
template <int B>
__device__ __forceinline__ void down_loop(const MOEQ_GLOBAL u32x4* rc, const MOEQ_GLOBAL uint16_t* rs, int U, int half,
                                          const MOEQ_GLOBAL u32x4* hrow, _Float16* wdst, _Float16* adst,
                                          const _Float16* As, const _Float16* Ws, int lane, int wm, int wn, int nk,
                                          f32x4v (&acc)[1][4][4]) {
  // first dword of block q = 2*hs + half inside its chunk pair
  const int o0 = (half * B) & 3, o1 = ((2 + half) * B) & 3;
  RawBlk hr[2];
  u32x4 hv[2][4];
#define DN_LOAD(slot, st)                                                                        \
  do {                                                                                           \
    hr[slot] = load_blk(rc, rs, U, B, (st) >> 1, 2 * (slot) + half);                             \
    _Pragma("unroll") for (int i_ = 0; i_ < 4; ++i_) hv[slot][i_] = hrow[(st) * (BK / 8) + i_];  \
  } while (0)
#define DN_DECODE(slot)                                                                 \
  do {                                                                                  \
    decode_blk<B>(hr[slot], (slot) ? o1 : o0, wdst + (slot) * (BN * LDS_STRIDE));       \
    store_row32(hv[slot], adst + (slot) * (BM * LDS_STRIDE));                           \
  } while (0)
#define DN_STEP(P, st_next)                                                                   \
  do {                                                                                        \
    Frags<1> f;                                                                               \
    read_frags<1>(As + (P) * (BM * LDS_STRIDE), Ws + (P) * (BN * LDS_STRIDE), lane, wm, wn, f); \
    DN_DECODE(1 - (P));                                                                       \
    DN_LOAD(1 - (P), st_next);                                                                \
    mfmas<1>(f, acc);                                                                         \
    interleave_hint<32, 16, 4, 8>();                                                          \
    __syncthreads();                                                                          \
  } while (0)
  DN_LOAD(0, 0);
  DN_LOAD(1, 1);
  DN_DECODE(0);
  DN_LOAD(0, min(2, nk - 2));
  __syncthreads();
  for (int s0 = 0; s0 < nk; s0 += 2) {
    DN_STEP(0, min(s0 + 3, nk - 1));
    DN_STEP(1, min(s0 + 4, nk - 2));
  }
#undef DN_LOAD
#undef DN_DECODE
#undef DN_STEP
}

__device__ void down_gemm_body(const GemmArgs a, const SlotInfo sl, int m0, int n0,
                               const TensorDev td, _Float16* lds) {
  _Float16* As = lds;                        // [2][BM][LDS_STRIDE]
  _Float16* Ws = lds + 2 * BM * LDS_STRIDE;  // [2][BN][LDS_STRIDE]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int H = a.H, I = a.I, U = I / kUnit;
  const int r = tid & 127;
  const int half = __builtin_amdgcn_readfirstlane(tid >> 7);  // wave-uniform
  const int bits = __builtin_amdgcn_readfirstlane(td.bits);
  const MOEQ_GLOBAL u32x4* rc = row_chunks(td, bits, n0 + r);
  const MOEQ_GLOBAL uint16_t* rs = gptr(td.scales + (size_t)(n0 + r) * (I / kBlock));
  _Float16* wdst = Ws + r * LDS_STRIDE + 32 * half;
  const bool arow_ok = m0 + r < sl.M;
  const MOEQ_GLOBAL uint32_t* rowmax = gptr((const uint32_t*)a.rowmax);
  const MOEQ_GLOBAL int32_t* perm = gptr(a.perm);
  // rows past the bucket read activation row 0 of the slot (never stored)
  const MOEQ_GLOBAL u32x4* hrow =
      gptr(reinterpret_cast<const u32x4*>(a.h16 + (size_t)(sl.base + m0 + (arow_ok ? r : 0)) * I)) + 4 * half;
  _Float16* adst = As + r * LDS_STRIDE + 32 * half;

  f32x4v acc[1][4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[0][i][c] = f32x4v{0.f, 0.f, 0.f, 0.f};

  const int nk = I / BK;
  if (bits == 2)
    down_loop<2>(rc, rs, U, half, hrow, wdst, adst, As, Ws, lane, wm, wn, nk, acc);
  else if (bits == 3)
    down_loop<3>(rc, rs, U, half, hrow, wdst, adst, As, Ws, lane, wm, wn, nk, acc);
  else
    down_loop<4>(rc, rs, U, half, hrow, wdst, adst, As, Ws, lane, wm, wn, nk, acc);

  // epilogue: undo the row prescale, scale by the routing weight, store partials
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int rr = wm * 64 + 16 * i + (lane >> 4) * 4 + j;
      if (m0 + rr >= sl.M) continue;
      const int e = max(0, (int)((rowmax[sl.base + m0 + rr] >> 23) & 0xFFu) - 127 - 14);
      int prow;
      float wv;
      if (sl.shared >= 0) {
        prow = a.n * a.k + sl.shared * a.n + m0 + rr;
        wv = 1.0f;
      } else {
        prow = perm[sl.base + m0 + rr];
        wv = gptr(a.w)[prow];
      }
      const float sc = __builtin_amdgcn_ldexpf(wv, e);
      MOEQ_GLOBAL float* prow_out = (MOEQ_GLOBAL float*)(a.partial + (size_t)prow * H);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int col = n0 + wn * 64 + 16 * c + (lane & 15);
        prow_out[col] = acc[0][i][c][j] * sc;
      }
    }
  }
}

__global__ __launch_bounds__(256, 1) void down_gemm_kernel(DecodeArgs a) {
  extern __shared__ _Float16 lds_h[];
  const int nN = a.H / BN;
  const int L = xcd_logical(blockIdx.x, gridDim.x);
  const int mt = L / nN, nt = L % nN;
  if (mt >= a.tiles[0]) return;
  const SlotInfo sl = slot_of(a, a.tiles[1 + 2 * mt]);
  const int m0 = a.tiles[2 + 2 * mt];
  const TensorDev td = a.desc[sl.desc * 3 + 2];
  if (!td.codes) return;
  if (td.bits < 2 || td.bits > 4) return;
  down_gemm_body(gemm_args(a), sl, m0, nt * BN, td, lds_h);
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
  const size_t lds = (size_t)2 * (BM + 2 * BN) * LDS_STRIDE * sizeof(_Float16);
  static bool attr = false;
  if (!attr) {
    e = hipFuncSetAttribute((const void*)gateup_gemm_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int grid = a.max_mtiles * (a.I / BN);
  gateup_gemm_kernel<<<grid, 256, lds, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_down_prefill(const DecodeArgs& a, hipStream_t s) {
  const int rows = a.n * (a.k + a.S);
  h16_kernel<<<(rows + 3) / 4, 256, 0, s>>>(a.h, a.rowmax, rows, a.I, a.h16);
  hipError_t e0 = hipGetLastError();
  if (e0 != hipSuccess) return e0;
  const size_t lds = (size_t)2 * (BM + BN) * LDS_STRIDE * sizeof(_Float16);
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)down_gemm_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int grid = a.max_mtiles * (a.H / BN);
  down_gemm_kernel<<<grid, 256, lds, s>>>(a);
  return hipGetLastError();
}

}  // namespace moeq

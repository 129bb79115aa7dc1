// Prefill path: grouped GEMM on the matrix cores for many tokens.
//
// Every active expert (and the shared expert, whose bucket is all n tokens)
// multiplies its bucket of tokens by its weights, so the layer becomes a set
// of independent GEMMs of very different heights (routing is skewed).  The
// bucketing permutation lists each expert's tokens contiguously; a small
// kernel cuts every bucket into tiles of up to 128 tokens and writes the
// tile list, so the GEMM grids never depend on a host synchronization.
//
// Arithmetic: activations (bf16, exact in binary16 after a per-token
// power-of-two prescale), dequantized weights fp16(d * (c - z)) (one rounding)
// and the SwiGLU activations h (binary16 after a per-row power-of-two
// prescale) enter binary16 matrix instructions with float32 accumulation.
//
// 2-4-bit tensors whose block scales are positive, finite and within the
// register decoder's bound, with rows of an even number of 128-weight units
// (every tensor of the workloads measured here), take the register-decoded
// GEMMs below (v_mfma_f32_32x32x16_f16, tiles of up to 128 tokens): the
// packed weights are decoded in registers straight into the matrix operand.
// Every other tensor (5, 6 or 8 bits, scales outside the bound, or an odd
// unit count) takes the LDS-decoded GEMMs (gateup_gemm8_kernel,
// down_gemm8_kernel, v_mfma_f32_16x16x32_f16): 128 tokens x 128 weight rows
// per workgroup, the weight tile of each K step decoded once into LDS.
// Workgroups are mapped to tiles from counts the device wrote, whatever the
// worst-case size of the grid: each XCD takes an equal run of list
// positions, the LDS-decoded tiles in slot order (one expert's tiles share
// its L2), the register-decoded ones sorted by work and dealt to the XCDs
// in turn (equal work per XCD).
#include <atomic>

#include "internal.h"
#include "layout.h"

namespace moeq {

namespace {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x4v __attribute__((ext_vector_type(4)));

constexpr int BM = kGemmBM, BN = 128, BK = 64;
// halves per LDS row: 16 halves of padding (measured best of 8, 16, 24, 40)
constexpr int LDS_STRIDE = BK + 16;

constexpr int kXcds = 8;  // the hardware deals workgroup ids to them round-robin
#ifndef MOEQ_RD_DEAL
#define MOEQ_RD_DEAL 1
#endif
constexpr int kRdDeal = MOEQ_RD_DEAL;  // register-decoded tiles dealt to an XCD at a time

// ---- tile lists: slot order = shared experts, then active experts; every
// bucket of M rows becomes ceil(M / 128) tiles of up to 128 rows.  tiles_all
// (the LDS-decoded GEMMs) keeps slot order, large and small buckets
// interleaved, so every XCD's share mixes both.  tiles_rd (the
// register-decoded GEMMs) holds a run of tiles_rd[0] positions per XCD (empty
// ones -1): the tiles sorted by work (full tiles in slot order, then the
// remainders by decreasing row count) and dealt to the XCDs in turn in groups
// of kRdDeal, so every XCD gets nearly the same work and runs its largest
// tiles first (kRdDeal = 0: slot order).  Also clears the running maxima of
// the h rows.
__global__ __launch_bounds__(1024) void prefill_tiles_kernel(DecodeArgs a) {
  constexpr int kCls = kRdTile / 32;  // remainder classes by 32-row steps
  // per-slot counts scanned over the slots: LDS-decoded tiles, full
  // register-decoded tiles, register-decoded tiles, remainders of each class
  constexpr int NF = 3 + kCls;
  constexpr int kSlots = kMaxShared + kMaxExperts;
  static_assert(kSlots <= 2 * 1024, "two slots per thread");
  __shared__ int32_t off[kSlots];   // first LDS-decoded tile of the slot
  __shared__ int32_t foff[kSlots];  // sorted index of its first full register-decoded tile
  __shared__ int32_t soff[kSlots];  // its first register-decoded tile in slot order
  __shared__ int32_t rpos[kSlots];  // sorted index of its remainder tile, or -1
  __shared__ int32_t nfull[kSlots];
  __shared__ int32_t ncnt[kSlots];
  __shared__ int32_t wsum[16][NF];
  __shared__ int32_t total[NF];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nslots = a.S + a.active[0];
  for (int t = tid; t < a.max_rtiles; t += 1024) a.tiles_rd[1 + 2 * t] = -1;
  // rows of h whose running maxima the gate/up epilogue accumulates
  const int rows = a.n * (a.k + a.S);
  for (int r = tid; r < rows; r += 1024) a.rowmax[r] = 0u;

  // thread tid holds slots 2 tid and 2 tid + 1
  int val[2][NF], cls[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int sl = 2 * tid + h;
    int M = 0;
    if (sl < a.S) {
      M = a.n;
    } else if (sl < nslots) {
      const int e = a.active[1 + sl - a.S];
      M = a.offsets[e + 1] - a.offsets[e];
    }
    if (M <= a.gemm_above) M = 0;  // (small buckets of a decode forward: the GEMV kernels)
    const int rem = M % kRdTile;
    cls[h] = (rem + 31) / 32;
    val[h][0] = (M + BM - 1) / BM;
    val[h][1] = M / kRdTile;
    val[h][2] = M / kRdTile + (rem ? 1 : 0);
#pragma unroll
    for (int c = 1; c <= kCls; ++c) val[h][2 + c] = cls[h] == c ? 1 : 0;
  }
  // exclusive prefix sums over the slots: within the wave by shuffles, then
  // over the 16 wave totals
  int ps[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) ps[f] = val[0][f] + val[1][f];
#pragma unroll
  for (int d = 1; d < 64; d *= 2)
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      const int t = __shfl_up(ps[f], d, 64);
      if (lane >= d) ps[f] += t;
    }
  if (lane == 63)
#pragma unroll
    for (int f = 0; f < NF; ++f) wsum[wave][f] = ps[f];
  __syncthreads();
  if (tid == 0) {
    for (int f = 0; f < NF; ++f) {
      int run = 0;
      for (int w = 0; w < 16; ++w) {
        const int v = wsum[w][f];
        wsum[w][f] = run;
        run += v;
      }
      total[f] = run;
    }
  }
  __syncthreads();
  int ex[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) ex[f] = ps[f] - val[0][f] - val[1][f] + wsum[wave][f];
  // sorted order: full tiles in slot order, then the remainders by class,
  // largest first, in slot order within a class
  int base[kCls + 1];
  base[kCls] = total[1];
#pragma unroll
  for (int c = kCls; c > 1; --c) base[c - 1] = base[c] + total[2 + c];
  const int T = base[1] + total[3];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int sl = 2 * tid + h;
    if (sl < nslots) {
      off[sl] = ex[0];
      foff[sl] = ex[1];
      soff[sl] = ex[2];
      int r = -1;
#pragma unroll
      for (int c = 1; c <= kCls; ++c)
        if (cls[h] == c) r = base[c] + ex[2 + c];
      rpos[sl] = r;
      ncnt[sl] = val[h][0];
      nfull[sl] = val[h][1];
    }
#pragma unroll
    for (int f = 0; f < NF; ++f) ex[f] += val[h][f];
  }
  int B = kRdDeal ? kRdDeal * ((T + kRdDeal * kXcds - 1) / (kRdDeal * kXcds)) : (T + kXcds - 1) / kXcds;
  B = min(B, a.max_rtiles / kXcds);
  if (tid == 0) {
    a.tiles_all[0] = min(total[0], a.max_mtiles);
    a.tiles_rd[0] = B;
  }
  __syncthreads();
  for (int s = tid; s < nslots; s += 1024) {
    for (int i = 0; i < ncnt[s]; ++i) {
      const int t = off[s] + i;
      if (t < a.max_mtiles) {
        a.tiles_all[1 + 2 * t] = s;
        a.tiles_all[2 + 2 * t] = i * BM;
      }
    }
    for (int i = 0; i <= nfull[s]; ++i) {
      int si;  // sorted index
      if (i < nfull[s])
        si = foff[s] + i;
      else if (rpos[s] >= 0)
        si = rpos[s];
      else
        break;
      int t;
      if (kRdDeal) {
        const int q = si / kRdDeal, x = q % kXcds;
        t = x * B + kRdDeal * (q / kXcds) + si % kRdDeal;
      } else {
        t = soff[s] + i;
      }
      if (t < kXcds * B) {
        a.tiles_rd[1 + 2 * t] = s;
        a.tiles_rd[2 + 2 * t] = i * kRdTile;
      }
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

// Workgroup -> (m-tile, n-tile) for T m-tiles of nN n-tiles each.  The
// hardware deals workgroup ids to the 8 XCDs round-robin; XCD x takes the
// m-tiles [x B, x B + B), B = ceil(T / 8), all n-tiles of an m-tile in a row,
// so one m-tile's activations stay in one L2 and every XCD gets the same
// share of the T tiles present, however large the grid (which covers
// 8 ceil(Tmax / 8) m-tiles).  False for a workgroup without a tile.
__device__ __forceinline__ bool tile_of_wg(int hw, int T, int nN, int* mt, int* nt) {
  const int x = hw % kXcds, j = hw / kXcds;
  const int B = (T + kXcds - 1) / kXcds;
  const int lm = j / nN;
  if (lm >= B) return false;
  *mt = x * B + lm;
  *nt = j % nN;
  return *mt < T;
}
inline int tile_grid(int max_tiles, int nN) { return (max_tiles + kXcds - 1) / kXcds * kXcds * nN; }

// Workgroup -> (list position, n-tile) in the register-decoded tile list:
// XCD x takes the B = tiles_rd[0] positions [x B, x B + B), all n-tiles of a
// position in a row.  False for a workgroup past the run or at an empty
// position.
__device__ __forceinline__ bool rd_tile_of_wg(const int32_t* tiles, int hw, int nN, int* mt, int* nt) {
  const int x = hw % kXcds, j = hw / kXcds;
  const int lm = j / nN;
  if (lm >= tiles[0]) return false;
  *mt = x * tiles[0] + lm;
  *nt = j % nN;
  return tiles[1 + 2 * *mt] >= 0;
}

// The register-decoded GEMMs take a tensor of 2-4 bits whose scales the
// create-time scan found positive, finite and small enough and whose rows
// hold an even number of units (flags); the LDS-decoded GEMMs take every
// other tensor.
__device__ __forceinline__ bool rd_ok(const TensorDev& t) {
  return t.bits <= 4 && !(t.flags & kTensorOffRegisterDecoder);
}

// Row-base pointer of a tensor row in the device layout.
__device__ __forceinline__ const MOEQ_GLOBAL u32x4* row_chunks(const TensorDev& t, int bits, int row) {
  const int U = t.K / kUnit;
  return gptr(reinterpret_cast<const u32x4*>(t.codes + (size_t)row * bits * U * 4));
}

// (c_lo, c_hi) at bit offset s of each half -> binary16 pair d * (c - z), exact
// code extraction through the 1024 + c binary16 bit trick, then one rounding.
template <int S>
__device__ __forceinline__ uint32_t dq_pair(uint32_t w, uint32_t mask, uint32_t base, half2_t zb, half2_t d2) {
  const uint32_t v = and_or(w >> S, mask, base);
  const half2_t c = __builtin_bit_cast(half2_t, v) + zb;  // c - z, exact
  return __builtin_bit_cast(uint32_t, c * d2);          // rounded once
}

__device__ __forceinline__ half8 lds_frag(const _Float16* p) {
  return *reinterpret_cast<const half8*>(p);
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + expf(-g)); }

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
  const uint32_t* zeros;
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
  g.zeros = a.zeros;
  g.n = a.n;
  g.H = a.H;
  g.I = a.I;
  g.k = a.k;
  return g;
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

// ---------------------------------------------------------------------------
// h -> binary16 rows prescaled by 2^-e, e from the row's maximum |h|, so
// that the largest value lands in [2^14, 2^15) at any magnitude (one rounding
// to nearest even; e >= -100 keeps 2^-e finite for an all-zero row).  The
// down epilogue recomputes the same e.
// One wave per row of h.
__global__ __launch_bounds__(256) void h16_kernel(const float* h, const uint32_t* rowmax, int rows, int I,
                                                 uint16_t* h16) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= rows) return;
  const int e = max((int)((rowmax[row] >> 23) & 0xFFu) - 127 - 14, -100);
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

// ---- weight tile decode: one thread, one row, one block (32 weights) ----
// Block q of unit u (B dwords at dword q*B of the unit): the 16-byte chunks
// c0 = q*B/4 and min(c0+1, B-1), kept as loaded (no selection at load time,
// so the loads stay in flight), and the aligned pair of binary16 scales that
// holds the block's.
struct RawBlk {
  u32x4 a, b;
  uint32_t sc;
};

// Block Q of unit u: its first chunk, and the next one only when the block
// runs past the end of the first (Q and B are compile-time, so a block that
// sits in one chunk issues one load).
template <int B, int Q>
__device__ __forceinline__ RawBlk load_blk(const MOEQ_GLOBAL u32x4* rc, const MOEQ_GLOBAL uint16_t* rs, int U,
                                           int u) {
  constexpr int c0 = (Q * B) >> 2;
  constexpr bool two = ((Q * B) & 3) + B > 4;
  RawBlk r;
  r.a = rc[(size_t)c0 * U + u];
  if constexpr (two)
    r.b = rc[(size_t)(c0 + 1) * U + u];
  else
    r.b = u32x4{0u, 0u, 0u, 0u};
  // the aligned pair of binary16 scales holding block Q's (Q even: low half)
  r.sc = *reinterpret_cast<const MOEQ_GLOBAL uint32_t*>(rs + 4 * u + (Q & 2));
  return r;
}

// Decodes one block (width B) whose first dword is dword o (0..3, wave-
// uniform) of the loaded pair of chunks; its scale is the high half of the
// loaded scale pair when o_half_shift (odd block index).
template <int B>
__device__ __forceinline__ void decode_blk(const RawBlk& r, int o, bool o_half_shift, _Float16* dst) {
  const uint32_t all[8] = {r.a.x, r.a.y, r.a.z, r.a.w, r.b.x, r.b.y, r.b.z, r.b.w};
  // a block starts at dword o = (q * B) % 4 of its first chunk: o + B <= 8
  // for every width here (B = 6 has o in {0, 2}, B = 8 has o = 0)
  uint32_t w[B];
#pragma unroll
  for (int i = 0; i < B; ++i) {
    if constexpr (B == 8)
      w[i] = all[i];
    else if constexpr (B == 6)
      w[i] = o == 0 ? all[i] : all[i + 2];
    else
      w[i] = o == 0 ? all[i] : o == 1 ? all[i + 1] : o == 2 ? all[i + 2] : all[i + 3];
  }
  uint32_t mask, base;
  asm("v_mov_b32 %0, 0x64006400" : "=v"(base));
  if constexpr (B == 4 || B == 8) asm("v_mov_b32 %0, 0x000F000F" : "=v"(mask));
  if constexpr (B == 3) asm("v_mov_b32 %0, 0x00070007" : "=v"(mask));
  if constexpr (B == 2) asm("v_mov_b32 %0, 0x00030003" : "=v"(mask));
  if constexpr (B == 5) asm("v_mov_b32 %0, 0x001F001F" : "=v"(mask));
  if constexpr (B == 6) asm("v_mov_b32 %0, 0x003F003F" : "=v"(mask));
  const _Float16 zf = (_Float16)(-(1024.0f + (float)(1 << (B - 1))));
  const half2_t zb = {zf, zf};
  const _Float16 d = __builtin_bit_cast(_Float16, (uint16_t)(o_half_shift ? r.sc >> 16 : r.sc));
  const half2_t d2 = {d, d};
  uint32_t p[16];
  if constexpr (B == 8) {
    // low nibbles in dwords 0..3 and high nibbles in 4..7, each a 4-bit
    // block: 1024 + c is the low nibble under the base with the high
    // nibble placed at bits [4, 8)
    uint32_t hm;
    asm("v_mov_b32 %0, 0x00F000F0" : "=v"(hm));
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        const uint32_t hs = f == 0 ? w[4 + q] << 4 : w[4 + q] >> (4 * f - 4);
        const uint32_t t = and_or(hs, hm, and_or(w[q] >> (4 * f), mask, base));
        const half2_t c = __builtin_bit_cast(half2_t, t) + zb;
        p[4 * q + f] = __builtin_bit_cast(uint32_t, c * d2);
      }
  } else if constexpr (B == 6) {
#pragma unroll
    for (int q = 0; q < 6; ++q)
#pragma unroll
      for (int f = 0; f < 2; ++f) p[2 * q + f] = dq_pair<0>(w[q] >> (6 * f), mask, base, zb, d2);
    uint32_t lo4, hi2;
    asm("v_mov_b32 %0, 0x000F000F" : "=v"(lo4));
    asm("v_mov_b32 %0, 0x00300030" : "=v"(hi2));
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const uint32_t t = and_or(w[4 + m / 2] >> (8 + 2 * (m & 1)), hi2, and_or(w[m] >> 12, lo4, base));
      const half2_t c = __builtin_bit_cast(half2_t, t) + zb;
      p[12 + m] = __builtin_bit_cast(uint32_t, c * d2);
    }
  } else if constexpr (B == 5) {
#pragma unroll
    for (int q = 0; q < 5; ++q)
#pragma unroll
      for (int f = 0; f < 3; ++f) p[3 * q + f] = dq_pair<0>(w[q] >> (5 * f), mask, base, zb, d2);
    // bit q of codes 30 and 31 sits at bit 15 (31) of dword q
    uint32_t m0, m1, m2, m3, m4;
    asm("v_mov_b32 %0, 0x00010001" : "=v"(m0));
    asm("v_mov_b32 %0, 0x00020002" : "=v"(m1));
    asm("v_mov_b32 %0, 0x00040004" : "=v"(m2));
    asm("v_mov_b32 %0, 0x00080008" : "=v"(m3));
    asm("v_mov_b32 %0, 0x00100010" : "=v"(m4));
    uint32_t t = and_or(w[0] >> 15, m0, base);
    t = and_or(w[1] >> 14, m1, t);
    t = and_or(w[2] >> 13, m2, t);
    t = and_or(w[3] >> 12, m3, t);
    t = and_or(w[4] >> 11, m4, t);
    const half2_t c = __builtin_bit_cast(half2_t, t) + zb;
    p[15] = __builtin_bit_cast(uint32_t, c * d2);
  } else if constexpr (B == 4) {
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

// ---------------------------------------------------------------------------
// Eight waves per workgroup (two per SIMD): the same 128 x 128 tile and K
// step of 64, each wave owning 64 rows x 32 columns per tensor (2 x 4 wave
// grid), so that while one wave of a SIMD waits on LDS or a barrier the other
// issues MFMAs.  Weight roles: a thread decodes one 32-weight block per K
// step (block 2*hs + BLK of its row's unit, BLK wave-uniform and a template
// argument, hs = step parity), activation roles move 16 or 32 binary16
// values.  Register slot and LDS buffer s % 2 hold step s; loads run two
// steps ahead; the last loads repeat the final steps (their decodes land in a
// buffer nobody reads again).
template <int NT>
__device__ __forceinline__ void read_frags8(const _Float16* A, const _Float16* W, int lane, int wm, int wn,
                                            half8 (&fa)[2][4], half8 (&fb)[2][NT][2]) {
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const int kof = kk * 32 + (lane >> 4) * 8;
#pragma unroll
    for (int i = 0; i < 4; ++i) fa[kk][i] = lds_frag(A + (wm * 64 + 16 * i + (lane & 15)) * LDS_STRIDE + kof);
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int c = 0; c < 2; ++c)
        fb[kk][t][c] = lds_frag(W + (t * BN + wn * 32 + 16 * c + (lane & 15)) * LDS_STRIDE + kof);
  }
}

template <int NT>
__device__ __forceinline__ void mfmas8(const half8 (&fa)[2][4], const half8 (&fb)[2][NT][2], f32x4v (&acc)[NT][4][2]) {
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc[t][i][c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[kk][i], fb[kk][t][c], acc[t][i][c], 0, 0, 0);
}

// One K loop.  DW: this wave decodes weight blocks (width B, block BLK of the
// half unit); NA: u32x4 activation pieces this thread moves per step (0, 2
// or 4).
template <int NT, int B, int BLK, bool DW, int NA>
__device__ __forceinline__ void gemm_loop8(const MOEQ_GLOBAL u32x4* rc, const MOEQ_GLOBAL uint16_t* rs, int U,
                                           const MOEQ_GLOBAL u32x4* arow, _Float16* wdst, _Float16* adst,
                                           const _Float16* As, const _Float16* Ws, int lane, int wm, int wn, int nk,
                                           f32x4v (&acc)[NT][4][2]) {
  RawBlk hw[2];
  u32x4 xv[2][NA > 0 ? NA : 1];
#define L8(slot, st)                                                                        \
  do {                                                                                      \
    if constexpr (DW) hw[slot] = load_blk<B, 2 * (slot) + BLK>(rc, rs, U, (st) >> 1);        \
    _Pragma("unroll") for (int i_ = 0; i_ < NA; ++i_) xv[slot][i_] = arow[(st) * 8 + i_];   \
  } while (0)
#define D8(slot)                                                                                         \
  do {                                                                                                   \
    if constexpr (DW) decode_blk<B>(hw[slot], ((2 * (slot) + BLK) * B) & 3, BLK != 0, wdst + (slot) * (NT * BN * LDS_STRIDE)); \
    u32x4* ad_ = reinterpret_cast<u32x4*>(adst + (slot) * (BM * LDS_STRIDE));                            \
    _Pragma("unroll") for (int i_ = 0; i_ < NA; ++i_) ad_[i_] = xv[slot][i_];                            \
  } while (0)
  // The gate/up loop runs its MFMAs interleaved with the decode by the
  // scheduling hint; the down loop (half the decode work, and waves that only
  // move activations) is faster left to the compiler's own schedule.
  constexpr bool kHint = NT == 2;
#define STEP8(P, st_next)                                                                         \
  do {                                                                                            \
    half8 fa[2][4], fb[2][NT][2];                                                                 \
    read_frags8<NT>(As + (P) * (BM * LDS_STRIDE), Ws + (P) * (NT * BN * LDS_STRIDE), lane, wm, wn, fa, fb); \
    D8(1 - (P));                                                                                  \
    L8(1 - (P), st_next);                                                                         \
    mfmas8<NT>(fa, fb, acc);                                                                      \
    if constexpr (kHint) interleave_hint<16 * NT, 8 + 4 * NT, 2, 4>();                            \
    __syncthreads();                                                                              \
  } while (0)
  L8(0, 0);
  L8(1, 1);
  D8(0);
  L8(0, min(2, nk - 2));
  __syncthreads();
  for (int s0 = 0; s0 < nk; s0 += 2) {
    STEP8(0, min(s0 + 3, nk - 1));
    STEP8(1, min(s0 + 4, nk - 2));
  }
#undef L8
#undef D8
#undef STEP8
}

__device__ void gateup_gemm_body8(const GemmArgs a, const SlotInfo sl, int m0, int n0, const TensorDev tg,
                                  const TensorDev tu, _Float16* lds) {
  _Float16* As = lds;                            // [2][BM][LDS_STRIDE]
  _Float16* Ws = lds + 2 * BM * LDS_STRIDE;      // [2][2][BN][LDS_STRIDE]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int H = a.H, I = a.I, U = H / kUnit;
  const MOEQ_GLOBAL int32_t* perm = gptr(a.perm);
  const MOEQ_GLOBAL int32_t* xexp = gptr(a.xexp);
  // weights: waves 0-3 gate rows, 4-7 up rows; waves 2w and 2w + 1 take
  // block BLK = w % 2 of each half unit.  Activations: thread t moves 16
  // values (quarter t % 4) of tile row t / 4.
  const int wt = __builtin_amdgcn_readfirstlane(tid >> 8);
  const int blk = __builtin_amdgcn_readfirstlane((tid >> 7) & 1);
  const TensorDev t = wt ? tu : tg;
  const int bits = __builtin_amdgcn_readfirstlane(t.bits);
  const int wrow = n0 + (tid & 127);
  const MOEQ_GLOBAL u32x4* rc = row_chunks(t, bits, wrow);
  const MOEQ_GLOBAL uint16_t* rs = gptr(t.scales + (size_t)wrow * (H / kBlock));
  _Float16* wdst = Ws + (wt * BN + (tid & 127)) * LDS_STRIDE + 32 * blk;
  const int ar = tid >> 2, aq = tid & 3;
  int tok = 0;
  if (m0 + ar < sl.M) tok = sl.shared >= 0 ? m0 + ar : perm[sl.base + m0 + ar] / a.k;
  const MOEQ_GLOBAL u32x4* arow = gptr(reinterpret_cast<const u32x4*>(a.x16 + (size_t)tok * H)) + 2 * aq;
  _Float16* adst = As + ar * LDS_STRIDE + 16 * aq;

  f32x4v acc[2][4][2];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int c = 0; c < 2; ++c) acc[q][i][c] = f32x4v{0.f, 0.f, 0.f, 0.f};
  const int nk = H / BK;
#define GU8(B, BL) gemm_loop8<2, B, BL, true, 2>(rc, rs, U, arow, wdst, adst, As, Ws, lane, wm, wn, nk, acc)
  if (bits == 2) {
    if (blk) GU8(2, 1); else GU8(2, 0);
  } else if (bits == 3) {
    if (blk) GU8(3, 1); else GU8(3, 0);
  } else if (bits == 4) {
    if (blk) GU8(4, 1); else GU8(4, 0);
  } else if (bits == 5) {
    if (blk) GU8(5, 1); else GU8(5, 0);
  } else if (bits == 6) {
    if (blk) GU8(6, 1); else GU8(6, 0);
  } else {
    if (blk) GU8(8, 1); else GU8(8, 0);
  }
#undef GU8

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
      for (int c = 0; c < 2; ++c) {
        const int col = n0 + wn * 32 + 16 * c + (lane & 15);
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

// The tiles whose gate or up tensor the register decoder cannot take (5, 6
// or 8 bits wide, or scales outside its range; the other of the two may be
// any width); the other tiles take gateup_rd_kernel.
__global__ __launch_bounds__(512, 1) void gateup_gemm8_kernel(DecodeArgs a) {
  extern __shared__ _Float16 lds_h[];
  const int nN = a.I / BN;
  int mt, nt, slot, m0;
  if (!tile_of_wg(blockIdx.x, a.tiles_all[0], nN, &mt, &nt)) return;
  slot = a.tiles_all[1 + 2 * mt];
  m0 = a.tiles_all[2 + 2 * mt];
  const SlotInfo sl = slot_of(a, slot);
  const TensorDev tg = a.desc[sl.desc * 3 + 0], tu = a.desc[sl.desc * 3 + 1];
  if (!tg.codes || !tu.codes) return;
  if (rd_ok(tg) && rd_ok(tu)) return;
  gateup_gemm_body8(gemm_args(a), sl, m0, nt * BN, tg, tu, lds_h);
}

__device__ void down_gemm_body8(const GemmArgs a, const SlotInfo sl, int m0, int n0, const TensorDev td,
                                _Float16* lds) {
  _Float16* As = lds;                        // [2][BM][LDS_STRIDE]
  _Float16* Ws = lds + 2 * BM * LDS_STRIDE;  // [2][BN][LDS_STRIDE]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int H = a.H, I = a.I, U = I / kUnit;
  // waves 0-3 decode weight blocks (block BLK = (t >> 7) % 2 of row t % 128),
  // waves 4-7 move the activations (32 values of tile row (t - 256) / 2)
  const bool wrole = __builtin_amdgcn_readfirstlane(wave) < 4;
  const int blk = __builtin_amdgcn_readfirstlane((tid >> 7) & 1);
  const int bits = __builtin_amdgcn_readfirstlane(td.bits);
  const int wrow = n0 + (tid & 127);
  const MOEQ_GLOBAL u32x4* rc = row_chunks(td, bits, wrow);
  const MOEQ_GLOBAL uint16_t* rs = gptr(td.scales + (size_t)wrow * (I / kBlock));
  _Float16* wdst = Ws + (tid & 127) * LDS_STRIDE + 32 * blk;
  const int at = tid & 255, ar = at >> 1, ah = at & 1;
  const bool aok = m0 + ar < sl.M;
  // rows past the bucket read activation row 0 of the slot (never stored)
  const MOEQ_GLOBAL u32x4* arow =
      gptr(reinterpret_cast<const u32x4*>(a.h16 + (size_t)(sl.base + m0 + (aok ? ar : 0)) * I)) + 4 * ah;
  _Float16* adst = As + ar * LDS_STRIDE + 32 * ah;
  const MOEQ_GLOBAL uint32_t* rowmax = gptr((const uint32_t*)a.rowmax);
  const MOEQ_GLOBAL int32_t* perm = gptr(a.perm);

  f32x4v acc[1][4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int c = 0; c < 2; ++c) acc[0][i][c] = f32x4v{0.f, 0.f, 0.f, 0.f};
  const int nk = I / BK;
#define DN8(B, BL) gemm_loop8<1, B, BL, true, 0>(rc, rs, U, arow, wdst, adst, As, Ws, lane, wm, wn, nk, acc)
  if (!wrole) {
    gemm_loop8<1, 4, 0, false, 4>(rc, rs, U, arow, wdst, adst, As, Ws, lane, wm, wn, nk, acc);
  } else {
    if (bits == 2) {
      if (blk) DN8(2, 1); else DN8(2, 0);
    } else if (bits == 3) {
      if (blk) DN8(3, 1); else DN8(3, 0);
    } else if (bits == 4) {
      if (blk) DN8(4, 1); else DN8(4, 0);
    } else if (bits == 5) {
      if (blk) DN8(5, 1); else DN8(5, 0);
    } else if (bits == 6) {
      if (blk) DN8(6, 1); else DN8(6, 0);
    } else {
      if (blk) DN8(8, 1); else DN8(8, 0);
    }
  }
#undef DN8

  // epilogue: undo the row prescale, scale by the routing weight, store partials
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int rr = wm * 64 + 16 * i + (lane >> 4) * 4 + j;
      if (m0 + rr >= sl.M) continue;
      const int e = max((int)((rowmax[sl.base + m0 + rr] >> 23) & 0xFFu) - 127 - 14, -100);
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
      for (int c = 0; c < 2; ++c) {
        const int col = n0 + wn * 32 + 16 * c + (lane & 15);
        prow_out[col] = acc[0][i][c][j] * sc;
      }
    }
  }
}

// The tiles whose down tensor the register decoder cannot take (5, 6 or 8
// bits wide, or scales outside its range; the other tiles take
// down_rd_kernel).  Four waves per SIMD (128 registers): two workgroups share
// a compute unit (2 x 80 KB of LDS) and overlap their K-step chains.
__global__ __launch_bounds__(512, 4) void down_gemm8_kernel(DecodeArgs a) {
  extern __shared__ _Float16 lds_h[];
  const int nN = a.H / BN;
  int mt, nt, slot, m0;
  if (!tile_of_wg(blockIdx.x, a.tiles_all[0], nN, &mt, &nt)) return;
  slot = a.tiles_all[1 + 2 * mt];
  m0 = a.tiles_all[2 + 2 * mt];
  const SlotInfo sl = slot_of(a, slot);
  const TensorDev td = a.desc[sl.desc * 3 + 2];
  if (!td.codes) return;
  if (rd_ok(td)) return;
  down_gemm_body8(gemm_args(a), sl, m0, nt * BN, td, lds_h);
}

// ---------------------------------------------------------------------------
// Register-decoded grouped GEMM for 2-4-bit weights (gate/up with SwiGLU, and
// down).
//
// Weights are the MFMA's first operand (32 weight rows x 16 k) and tokens
// its second (16 k x 32 tokens) of v_mfma_f32_32x32x16_f16 (on gfx950 it
// runs at twice the rate of the 16 x 16 x 32 shape), so a bucket of M tokens
// costs ceil(M / 32) token tiles per 32 weight rows.  A workgroup of eight
// waves owns up to 128 tokens of one expert bucket and 256 weight rows; each
// wave owns one row tile of 32 and all the tokens (1-4 token tiles), so one
// decoded weight fragment feeds up to four matrix instructions.  One
// workgroup per compute unit (two waves per SIMD).
//
// Weights never pass through LDS.  Lane l of a wave (row r = l % 32 of its
// row tile, k-half g = l / 32) loads, for each K stage of 512 weights (4
// units of 128), units 4U + 2g and 4U + 2g + 1 of its row: the two lanes of
// a row read 64 contiguous bytes per chunk plane.  It decodes them in
// registers straight into the operand layout, binary16 d * (c - 2^(b-1))
// with one rounding: at k step t (0..7) of sub-stage q (block q of each
// unit), the 8 operand values of lane (r, g) are weights 32 q + 8 (t % 4) ..
// + 7 of unit 4U + 2g + t / 4.  The activation operand of lane (c, g) must
// hold the same k values, which the LDS tile provides: activations go through
// LDS in sub-stages of 128 k values (block q of the stage's four units), 128
// token rows of 16 pieces of 16 bytes, piece p = 4 u + m (unit u of the
// stage, piece m of its block) stored at position p ^ (row % 16) of its row
// (no bank conflicts for the 16-byte fragment reads).  Four LDS buffers:
// sub-stage s + 2 is requested when s begins and stored when it ends.
//
// gate/up: waves 0-3 own 32 gate rows each, waves 4-7 the same features' up
// rows (each wave works on one tensor, so on one width); the up waves hand
// their accumulators to the gate waves through LDS for the SwiGLU epilogue.
// down: eight waves of 32 output features of one tensor.  The K loop is
// instantiated per width and per token-tile count, so a small bucket does
// not spend matrix instructions on empty tiles, and the loop has no branches.
constexpr int RD_T = kRdTile;         // tokens per workgroup tile
#ifndef MOEQ_RD_WAVES
#define MOEQ_RD_WAVES 8
#endif
constexpr int RD_WAVES = MOEQ_RD_WAVES;
constexpr int RD_THREADS = 64 * RD_WAVES;
constexpr int RD_NTMAX = RD_T / 32;   // token tiles of 32 per workgroup tile
#ifndef MOEQ_RD_RT
#define MOEQ_RD_RT (RD_T >= 128 && RD_WAVES == 8 ? 1 : 2)
#endif
constexpr int RD_RT = MOEQ_RD_RT;  // row tiles of 32 per wave
constexpr int RD_WROWS = 32 * RD_RT;  // weight rows per wave
constexpr int RD_ROWS = RD_WAVES * RD_WROWS;  // weight rows per workgroup
constexpr int RD_SUB = RD_T * 256;    // bytes of one activation sub-stage
constexpr int RD_NBUF = 4;            // activation sub-stages resident in LDS
constexpr int RD_APT = RD_SUB / 16 / RD_THREADS;  // 16-byte staging pieces per thread and sub-stage
constexpr int RD_RPJ = RD_THREADS / 16;  // token rows per staging piece index
static_assert(32 % RD_RPJ == 0, "the staging pieces of a token tile are whole");
// staging pieces per thread for NT token tiles
template <int NT>
constexpr int rd_apt() { return NT * 32 / RD_RPJ; }
constexpr size_t RD_LDS = (size_t)RD_NBUF * RD_SUB;
static_assert(RD_WAVES * RD_WROWS == RD_ROWS, "the waves cover the workgroup's rows");
static_assert(RD_LDS >= (size_t)(RD_WAVES / 2) * RD_RT * RD_NTMAX * 64 * 64,
              "the SwiGLU hand-over must fit the activation buffers");
static_assert(RD_LDS <= 160 * 1024, "the activation buffers fit a compute unit's LDS");

typedef float f32x16 __attribute__((ext_vector_type(16)));

// this lane's unit of one weight row: B chunks of 16 bytes and the unit's
// four binary16 scales
template <int B>
struct RdUnit {
  u32x4 c[B];
  u32x2 s;
};

template <int B>
__device__ __forceinline__ uint32_t rd_dword(const RdUnit<B>& u, int i) {
  return u.c[i >> 2][i & 3];
}

// Register decode of the code pairs (weights 2i and 2i + 1 sit in the low
// and high halves of a dword).  The pair is shifted and masked to bit
// P = 10 - b of each half with the exponent field zero: two binary16
// subnormals c * 2^(P - 24), exact.  One packed fused multiply-add with
// D = d * 2^(24 - P) and C = -2^(b-1) d then forms c d - z d = d (c - z) and
// rounds it once: the binary16 value of d * (c - z).  D and C are exact for a
// positive finite d <= rd_scale_limit(b), which the create-time scan
// guarantees for every tensor these kernels take.
template <int B>
constexpr int rd_at() { return 10 - B; }

struct RdConsts {
  uint32_t mask;  // the width's code mask at bit P of both halves
};

template <int B>
__device__ __forceinline__ RdConsts rd_consts() {
  constexpr uint32_t m = ((1u << B) - 1u) << rd_at<B>();
  RdConsts k;
  k.mask = m | (m << 16);
  return k;
}

struct RdScale {
  half2_t D, C;  // d * 2^(24 - P) and -2^(b-1) d in both halves
};

template <int B, int Q>
__device__ __forceinline__ RdScale rd_scale(const RdUnit<B>& u) {
  const uint32_t sp = Q < 2 ? u.s.x : u.s.y;
  const _Float16 d = __builtin_bit_cast(_Float16, (uint16_t)((Q & 1) ? sp >> 16 : sp));
  const _Float16 D = __builtin_amdgcn_ldexph(d, 24 - rd_at<B>());
  const _Float16 C = d * (_Float16)(-(float)(1 << (B - 1)));
  return RdScale{half2_t{D, D}, half2_t{C, C}};
}

// code pair at bit offset S of each half of w -> binary16 d * (c - z) pair
template <int B, int S>
__device__ __forceinline__ uint32_t rd_pair(uint32_t w, const RdConsts& k, const RdScale& sc) {
  constexpr int P = rd_at<B>();
  const uint32_t v = (S >= P ? w >> (S - P) : w << (P - S)) & k.mask;
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_fma(__builtin_bit_cast(half2_t, v), sc.D, sc.C));
}

// Operand piece M (weights 8M .. 8M + 7) of block Q of this lane's unit.
template <int B, int Q, int M>
__device__ __forceinline__ half8 rd_piece(const RdUnit<B>& u, const RdConsts& k) {
  const RdScale sc = rd_scale<B, Q>(u);
  uint32_t p[4];
  if constexpr (B == 4) {
    const uint32_t w = rd_dword(u, 4 * Q + M);
    p[0] = rd_pair<B, 0>(w, k, sc);
    p[1] = rd_pair<B, 4>(w, k, sc);
    p[2] = rd_pair<B, 8>(w, k, sc);
    p[3] = rd_pair<B, 12>(w, k, sc);
  } else if constexpr (B == 2) {
    const uint32_t w = rd_dword(u, 2 * Q + M / 2);
    constexpr int o = 8 * (M & 1);
    p[0] = rd_pair<B, o + 0>(w, k, sc);
    p[1] = rd_pair<B, o + 2>(w, k, sc);
    p[2] = rd_pair<B, o + 4>(w, k, sc);
    p[3] = rd_pair<B, o + 6>(w, k, sc);
  } else {
    // pairs 4M .. 4M + 3 of the block; pair P < 15 sits in dword P / 5 at
    // offset 3 (P % 5), pair 15 is bit q of each code in bit 15 / 31 of dword q
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int P = 4 * M + i;
      if (P < 15) {
        const uint32_t w = rd_dword(u, 3 * Q + P / 5);
        switch (P % 5) {
          case 0: p[i] = rd_pair<B, 0>(w, k, sc); break;
          case 1: p[i] = rd_pair<B, 3>(w, k, sc); break;
          case 2: p[i] = rd_pair<B, 6>(w, k, sc); break;
          case 3: p[i] = rd_pair<B, 9>(w, k, sc); break;
          default: p[i] = rd_pair<B, 12>(w, k, sc); break;
        }
      } else {
        constexpr int A = rd_at<B>();
        constexpr uint32_t b0 = (1u << A) | (1u << (A + 16));
        uint32_t t = (rd_dword(u, 3 * Q) >> (15 - A)) & b0;
        t = and_or(rd_dword(u, 3 * Q + 1) >> (14 - A), b0 << 1, t);
        t = and_or(rd_dword(u, 3 * Q + 2) >> (13 - A), b0 << 2, t);
        p[i] = __builtin_bit_cast(uint32_t, __builtin_elementwise_fma(__builtin_bit_cast(half2_t, t), sc.D, sc.C));
      }
    }
  }
  return __builtin_bit_cast(half8, u32x4{p[0], p[1], p[2], p[3]});
}

// The K loop of one wave.  ACT: the wave owns weight rows (else it only
// stages activations, e.g. rows past the end of the tensor).  rc/rs: per row
// tile, this lane's row chunk base and scale pairs; arow: the activation rows
// this thread stages (row j * RD_RPJ + tid / 16 of the tile), as 16-byte pieces;
// su/sm: the unit and piece of the thread's staging slot; zero: 16 zeroed
// bytes, 16-byte aligned (the scales of units past the row).
//
// Prefetch depths: AL register sets of activation pieces (sub-stage s + AL
// is requested when s begins) and a ring of WL stages of weight registers
// (each chunk is requested 4 WL - 2 sub-stages before the sub-stage that
// first uses it, as soon as the ring slot's previous stage has finished with
// it).
template <int B, int NT, bool ACT, int AL, int WL>
__device__ __forceinline__ void rd_kloop(const MOEQ_GLOBAL u32x4* const (&rc)[RD_RT],
                                         const MOEQ_GLOBAL u32x2* const (&rs)[RD_RT], int Uk,
                                         const MOEQ_GLOBAL u32x4* const (&arow)[RD_APT], int su, int sm,
                                         const MOEQ_GLOBAL uint32_t* zero, char* lds, int tid, int lane,
                                         f32x16 (&acc)[RD_RT][NT]) {
  static_assert(WL >= 1 && AL >= 2 && (4 * WL) % AL == 0, "staging sets cycle within the unrolled stages");
  const int NS = (Uk + 3) / 4;                  // K stages of 4 units
  const int NSp = (NS + WL - 1) / WL * WL;      // stages run (a stage past NS has zero weights)
  const int NSUB = 4 * NS;                      // activation sub-stages
  const int g = lane >> 5;
  const RdConsts kc = rd_consts<B>();
  RdUnit<B> raw[WL][RD_RT][2];                  // [ring slot][row tile][unit 2g, 2g + 1 of the stage]
  // fragment read offset of k step t (bytes within a sub-stage buffer):
  // row c = lane % 32, piece (8 g + t) ^ (c % 16) = 8 (g ^ (c / 8 % 2)) + (t ^ (c % 8)),
  // i.e. fbase ^ 16 t with fbase's bits 4-6 holding c % 8
  const int fbase = (lane & 31) * 256 + (((g ^ ((lane >> 3) & 1)) << 7) | ((lane & 7) << 4));
  char* wdst = lds + tid * 16;

  // the staging pieces of sub-stage s (stage s / 4, block s % 4)
  // (only the NT token tiles that are multiplied are staged)
  auto aload = [&](u32x4 (&v)[RD_APT], int s) {
    const int unit = min(4 * (s >> 2) + su, Uk - 1);
    const int off = unit * 16 + 4 * (s & 3) + sm;
#pragma unroll
    for (int j = 0; j < rd_apt<NT>(); ++j) v[j] = arow[j][off];
  };
  auto astore = [&](const u32x4 (&v)[RD_APT], int buf) {
#pragma unroll
    for (int j = 0; j < rd_apt<NT>(); ++j)
      *reinterpret_cast<u32x4*>(wdst + buf * RD_SUB + j * (RD_THREADS * 16)) = v[j];
  };
  // chunk j / scale half h of this lane's two units in stage V, every row
  // tile, into one ring slot.  Plain (not streaming) loads: a stage reads 64
  // bytes of each row's chunk plane, half of a 128-byte line whose other half
  // the next stage reads, so the line has to stay in L2 until then
  // (streaming loads here cost 20%).
  auto rload_chunk = [&](RdUnit<B> (&dst)[RD_RT][2], int j, int V) {
    if constexpr (ACT) {
#pragma unroll
      for (int v = 0; v < 2; ++v) {
        const int uc = min(4 * V + 2 * g + v, Uk - 1);
#pragma unroll
        for (int r = 0; r < RD_RT; ++r) dst[r][v].c[j] = rc[r][(size_t)j * Uk + uc];
      }
    }
  };
  // the chunks that sub-stage f of stage V uses first (4 bits: chunk f;
  // 3 bits: chunk f for f < 3, used again in sub-stage f + 1; 2 bits: chunk
  // f / 2 for even f, used in f and f + 1)
  auto rload_first = [&](RdUnit<B> (&dst)[RD_RT][2], int f, int V) {
    if constexpr (B == 4) rload_chunk(dst, f, V);
    if constexpr (B == 3) {
      if (f < 3) rload_chunk(dst, f, V);
    }
    if constexpr (B == 2) {
      if ((f & 1) == 0) rload_chunk(dst, f >> 1, V);
    }
  };
  // the scales of this lane's two units of stage V (units 2g and 2g + 1 of
  // the stage, four binary16 scales each: 16 contiguous bytes, as rows hold
  // an even number of units), one load per row tile, requested in sub-stage
  // 1 of the stage before and moved into the stage's ring slot at its end.
  // A stage past the row reads 16 zero bytes, so its weights decode to zeros
  // (the choice is made on the address, so no instruction waits for the
  // loaded value).
  u32x4 sn[RD_RT];
  auto sload = [&](int V) {
    if constexpr (ACT) {
      const int unit = 4 * V + 2 * g;
#pragma unroll
      for (int r = 0; r < RD_RT; ++r) {
        const MOEQ_GLOBAL u32x4* src = unit < Uk ? reinterpret_cast<const MOEQ_GLOBAL u32x4*>(rs[r] + unit)
                                                 : reinterpret_cast<const MOEQ_GLOBAL u32x4*>(zero);
        sn[r] = *src;
      }
    }
  };
  auto sput = [&](RdUnit<B> (&dst)[RD_RT][2]) {
    if constexpr (ACT) {
#pragma unroll
      for (int r = 0; r < RD_RT; ++r) {
        dst[r][0].s = u32x2{sn[r].x, sn[r].y};
        dst[r][1].s = u32x2{sn[r].z, sn[r].w};
      }
    }
  };

  // prologue: the chunks whose request point (4 V + f - (4 WL - 2) - 1)
  // lies before the first sub-stage, in that order; sub-stage 0 stored,
  // sub-stages 1 .. AL - 1 in flight
#pragma unroll
  for (int V = 0; V < WL; ++V)
#pragma unroll
    for (int f = 0; f < 4; ++f)
      if (4 * V + f < 4 * WL - 1) rload_first(raw[V], f, V);
  sload(0);
  sput(raw[0]);
  u32x4 xs[AL][RD_APT];
  aload(xs[0], 0);
  astore(xs[0], 0);
#pragma unroll
  for (int i = 1; i < AL; ++i) aload(xs[i], min(i, NSUB - 1));
  __syncthreads();

  // k step TS of sub-stage Q (ring slot W): operands into FA / FB (fragment
  // reads from LDS and the weight decode), then the matrix products of a
  // step whose operands are ready.  The steps of a sub-stage are
  // software-pipelined: the operands of step t + 1 are prepared among the
  // products of step t, and a scheduling barrier keeps the compiler from
  // hoisting later steps' decodes (which costs registers and spills).
  half8 fa0[RD_RT], fb0[NT], fa1[RD_RT], fb1[NT];
#define RD_OPERANDS(W, Q, TS, FA, FB)                                                                   \
  do {                                                                                                  \
    if constexpr (ACT) {                                                                                \
      _Pragma("unroll") for (int T = 0; T < NT; ++T) FB[T] =                                            \
          *reinterpret_cast<const half8*>(lds + (Q) * RD_SUB + T * (32 * 256) + (fbase ^ (16 * (TS))));  \
      _Pragma("unroll") for (int r = 0; r < RD_RT; ++r) FA[r] =                                         \
          rd_piece<B, Q, (TS) & 3>(raw[W][r][(TS) >> 2], kc);                                           \
    }                                                                                                   \
  } while (0)
#define RD_PRODUCTS(FA, FB)                                                                             \
  do {                                                                                                  \
    if constexpr (ACT) {                                                                                \
      _Pragma("unroll") for (int T = 0; T < NT; ++T)                                                    \
      _Pragma("unroll") for (int r = 0; r < RD_RT; ++r) acc[r][T] =                                     \
          __builtin_amdgcn_mfma_f32_32x32x16_f16(FA[r], FB[T], acc[r][T], 0, 0, 0);                     \
    }                                                                                                   \
  } while (0)
#define RD_KSTEPS(W, Q)                                                                                 \
  do {                                                                                                  \
    RD_OPERANDS(W, Q, 0, fa0, fb0);                                                                     \
    RD_OPERANDS(W, Q, 1, fa1, fb1);                                                                     \
    RD_PRODUCTS(fa0, fb0);                                                                              \
    __builtin_amdgcn_sched_barrier(0);                                                                  \
    RD_OPERANDS(W, Q, 2, fa0, fb0);                                                                     \
    RD_PRODUCTS(fa1, fb1);                                                                              \
    __builtin_amdgcn_sched_barrier(0);                                                                  \
    RD_OPERANDS(W, Q, 3, fa1, fb1);                                                                     \
    RD_PRODUCTS(fa0, fb0);                                                                              \
    __builtin_amdgcn_sched_barrier(0);                                                                  \
    RD_OPERANDS(W, Q, 4, fa0, fb0);                                                                     \
    RD_PRODUCTS(fa1, fb1);                                                                              \
    __builtin_amdgcn_sched_barrier(0);                                                                  \
    RD_OPERANDS(W, Q, 5, fa1, fb1);                                                                     \
    RD_PRODUCTS(fa0, fb0);                                                                              \
    __builtin_amdgcn_sched_barrier(0);                                                                  \
    RD_OPERANDS(W, Q, 6, fa0, fb0);                                                                     \
    RD_PRODUCTS(fa1, fb1);                                                                              \
    __builtin_amdgcn_sched_barrier(0);                                                                  \
    RD_OPERANDS(W, Q, 7, fa1, fb1);                                                                     \
    RD_PRODUCTS(fa0, fb0);                                                                              \
    __builtin_amdgcn_sched_barrier(0);                                                                  \
    RD_PRODUCTS(fa1, fb1);                                                                              \
  } while (0)

  // sub-stage s = 4 (U + W) + Q in LDS buffer Q, weights in ring slot W:
  // request sub-stage s + AL into the staging set that held s (stored at the
  // end of s - 1), multiply sub-stage s, store sub-stage s + 1 (requested
  // when s + 1 - AL began) into buffer (Q + 1) % 4 (free: its sub-stage s - 3
  // was read before earlier barriers), and request the chunks that
  // sub-stage Q - 1 of a stage uses first for stage U + W + WL (Q = 0: the
  // chunks of sub-stage 3 for stage U + W + WL - 1), whose ring registers
  // this sub-stage freed; sub-stage 1 requests the next stage's scales,
  // sub-stage 3 moves them into its ring slot.  No branches: past the last
  // sub-stage or stage the loads repeat the last one (clamped) and the stores
  // go to buffers nobody reads again, so the compiler counts the outstanding
  // loads exactly.
#define RD_SUBSTAGE(W, Q)                                                                               \
  do {                                                                                                  \
    aload(xs[(4 * (W) + (Q)) % AL], min(4 * (U + (W)) + (Q) + AL, NSUB - 1));                           \
    RD_KSTEPS(W, Q);                                                                                    \
    astore(xs[(4 * (W) + (Q) + 1) % AL], ((Q) + 1) & 3);                                                \
    if constexpr ((Q) == 0)                                                                             \
      rload_first(raw[((W) + WL - 1) % WL], 3, min(U + (W) + WL - 1, NSp));                             \
    else                                                                                                \
      rload_first(raw[W], (Q) - 1, min(U + (W) + WL, NSp));                                             \
    if constexpr ((Q) == 1) sload(min(U + (W) + 1, NSp));                                               \
    if constexpr ((Q) == 3) sput(raw[((W) + 1) % WL]);                                                  \
    __syncthreads();                                                                                    \
  } while (0)

  for (int U = 0; U < NSp; U += WL) {
    RD_SUBSTAGE(0, 0);
    RD_SUBSTAGE(0, 1);
    RD_SUBSTAGE(0, 2);
    RD_SUBSTAGE(0, 3);
    if constexpr (WL == 2) {
      RD_SUBSTAGE(1, 0);
      RD_SUBSTAGE(1, 1);
      RD_SUBSTAGE(1, 2);
      RD_SUBSTAGE(1, 3);
    }
  }
#undef RD_SUBSTAGE
#undef RD_KSTEPS
#undef RD_PRODUCTS
#undef RD_OPERANDS
}

// Prefetch depths of the K loop (deeper settings, with the registers the
// smaller token-tile counts leave free, measured no faster: the loads are
// limited by the requests each compute unit can keep in flight, not by
// their latency).
#ifndef MOEQ_RD_AL
#define MOEQ_RD_AL 2
#endif
#ifndef MOEQ_RD_WL
#define MOEQ_RD_WL 1
#endif

// Width dispatch of one wave's K loop (B is uniform per wave: one tensor).
template <int NT>
__device__ __forceinline__ void rd_kloop_any(int bits, bool act, const MOEQ_GLOBAL u32x4* const (&rc)[RD_RT],
                                             const MOEQ_GLOBAL u32x2* const (&rs)[RD_RT], int Uk,
                                             const MOEQ_GLOBAL u32x4* const (&arow)[RD_APT], int su, int sm,
                                             const MOEQ_GLOBAL uint32_t* zero, char* lds, int tid, int lane,
                                             f32x16 (&acc)[RD_RT][NT]) {
  constexpr int AL = MOEQ_RD_AL, WL = MOEQ_RD_WL;
  if (!act)
    rd_kloop<2, NT, false, AL, WL>(rc, rs, Uk, arow, su, sm, zero, lds, tid, lane, acc);
  else if (bits == 2)
    rd_kloop<2, NT, true, AL, WL>(rc, rs, Uk, arow, su, sm, zero, lds, tid, lane, acc);
  else if (bits == 3)
    rd_kloop<3, NT, true, AL, WL>(rc, rs, Uk, arow, su, sm, zero, lds, tid, lane, acc);
  else
    rd_kloop<4, NT, true, AL, WL>(rc, rs, Uk, arow, su, sm, zero, lds, tid, lane, acc);
}

// Accumulator element v (0..15) of lane l in a 32 x 32 tile: row (weight row)
// 8 (v / 4) + 4 (l / 32) + v % 4, column (token) l % 32.
__device__ __forceinline__ int rd_acc_row(int v, int lane) { return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3); }

// Gate/up tile: features [f0, f0 + 256) of one slot, tokens [m0, m0 + 64)
// of its bucket (Mt of them real).  NT token tiles of 32 are multiplied.
template <int NT>
__device__ void rd_gateup_tile(const GemmArgs& a, const SlotInfo& sl, int m0, int Mt, int f0, const TensorDev& tg,
                               const TensorDev& tu, char* lds) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int H = a.H, I = a.I, Uk = H / kUnit;
  constexpr int HW = RD_WAVES / 2;   // waves per projection
  const TensorDev& t = wave < HW ? tg : tu;
  const int bits = __builtin_amdgcn_readfirstlane(t.bits);
  const int row0 = f0 + (wave % HW) * RD_WROWS;
  const bool act = row0 < I;   // I is a multiple of 128: a wave's features are all in or all out
  const MOEQ_GLOBAL u32x4* rc[RD_RT];
  const MOEQ_GLOBAL u32x2* rs[RD_RT];
#pragma unroll
  for (int r = 0; r < RD_RT; ++r) {
    const int row = act ? row0 + 32 * r + (lane & 31) : 0;
    rc[r] = gptr(reinterpret_cast<const u32x4*>(t.codes + (size_t)row * bits * Uk * 4));
    rs[r] = gptr(reinterpret_cast<const u32x2*>(t.scales + (size_t)row * (H / kBlock)));
  }
  // staging slots of this thread: rows j * RD_RPJ + tid / 16 (the NT token
  // tiles multiplied), piece (tid % 16) ^ (row % 16)
  const MOEQ_GLOBAL int32_t* perm = gptr(a.perm);
  const MOEQ_GLOBAL u32x4* arow[RD_APT] = {};
#pragma unroll
  for (int j = 0; j < rd_apt<NT>(); ++j) {
    int ar = j * RD_RPJ + (tid >> 4);
    ar = ar < Mt ? ar : 0;
    const int tok = sl.shared >= 0 ? m0 + ar : perm[sl.base + m0 + ar] / a.k;
    arow[j] = gptr(reinterpret_cast<const u32x4*>(a.x16 + (size_t)tok * H));
  }
  const int lp = (tid & 15) ^ ((tid >> 4) & 15);
  f32x16 acc[RD_RT][NT];
#pragma unroll
  for (int r = 0; r < RD_RT; ++r)
#pragma unroll
    for (int T = 0; T < NT; ++T)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[r][T][v] = 0.f;
  rd_kloop_any<NT>(bits, act, rc, rs, Uk, arow, lp >> 2, lp & 3, gptr(a.zeros), lds, tid, lane, acc);

  // SwiGLU: the up waves hand their accumulators to the gate waves of the
  // same features (the buffers are free after the loop's last barrier)
  f32x16* xch = reinterpret_cast<f32x16*>(lds);
  if (wave >= HW && act) {
#pragma unroll
    for (int r = 0; r < RD_RT; ++r)
#pragma unroll
      for (int T = 0; T < NT; ++T) xch[(((wave - HW) * RD_RT + r) * RD_NTMAX + T) * 64 + lane] = acc[r][T];
  }
  __syncthreads();
  if (wave >= HW || !act) return;
  const MOEQ_GLOBAL int32_t* xexp = gptr(a.xexp);
#pragma unroll
  for (int T = 0; T < NT; ++T) {
    const int rr = T * 32 + (lane & 31);
    const bool ok = rr < Mt;
    float sc = 1.0f;
    if (ok) {
      const int tk = sl.shared >= 0 ? m0 + rr : perm[sl.base + m0 + rr] / a.k;
      sc = __builtin_amdgcn_ldexpf(1.0f, xexp[tk]);
    }
    MOEQ_GLOBAL float* hout = (MOEQ_GLOBAL float*)(a.h + (size_t)(sl.base + m0 + rr) * I + row0);
    float rmax = 0.0f;
#pragma unroll
    for (int r = 0; r < RD_RT; ++r) {
      const f32x16 u = xch[((wave * RD_RT + r) * RD_NTMAX + T) * 64 + lane];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        f32x4 hv;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int v = 4 * q + i;
          hv[i] = silu(acc[r][T][v] * sc) * (u[v] * sc);
          rmax = fmaxf(rmax, fabsf(hv[i]));
        }
        if (ok) *reinterpret_cast<MOEQ_GLOBAL f32x4*>(hout + 32 * r + rd_acc_row(4 * q, lane)) = hv;
      }
    }
    rmax = fmaxf(rmax, __shfl_xor(rmax, 32, 64));
    if (ok && lane < 32) atomicMax(a.rowmax + sl.base + m0 + rr, __float_as_uint(rmax));
  }
}

// Down tile: output features [n0, n0 + 512) (rows of the down tensor) of one
// slot, tokens [m0, m0 + 64); results times the routing weight are the
// slot's partial rows.
template <int NT>
__device__ void rd_down_tile(const GemmArgs& a, const SlotInfo& sl, int m0, int Mt, int n0, const TensorDev& td,
                             char* lds) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int H = a.H, I = a.I, Uk = I / kUnit;
  const int bits = __builtin_amdgcn_readfirstlane(td.bits);
  const int row0 = n0 + wave * RD_WROWS;
  const bool act = row0 < H;   // H is a multiple of 128 and of 64: a wave's rows are all in or all out
  const MOEQ_GLOBAL u32x4* rc[RD_RT];
  const MOEQ_GLOBAL u32x2* rs[RD_RT];
#pragma unroll
  for (int r = 0; r < RD_RT; ++r) {
    const int row = act ? row0 + 32 * r + (lane & 31) : 0;
    rc[r] = gptr(reinterpret_cast<const u32x4*>(td.codes + (size_t)row * bits * Uk * 4));
    rs[r] = gptr(reinterpret_cast<const u32x2*>(td.scales + (size_t)row * (I / kBlock)));
  }
  const MOEQ_GLOBAL u32x4* arow[RD_APT] = {};
#pragma unroll
  for (int j = 0; j < rd_apt<NT>(); ++j) {
    int ar = j * RD_RPJ + (tid >> 4);
    ar = ar < Mt ? ar : 0;
    arow[j] = gptr(reinterpret_cast<const u32x4*>(a.h16 + (size_t)(sl.base + m0 + ar) * I));
  }
  const int lp = (tid & 15) ^ ((tid >> 4) & 15);
  f32x16 acc[RD_RT][NT];
#pragma unroll
  for (int r = 0; r < RD_RT; ++r)
#pragma unroll
    for (int T = 0; T < NT; ++T)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[r][T][v] = 0.f;
  rd_kloop_any<NT>(bits, act, rc, rs, Uk, arow, lp >> 2, lp & 3, gptr(a.zeros), lds, tid, lane, acc);
  if (!act) return;

  const MOEQ_GLOBAL uint32_t* rowmax = gptr((const uint32_t*)a.rowmax);
  const MOEQ_GLOBAL int32_t* perm = gptr(a.perm);
#pragma unroll
  for (int T = 0; T < NT; ++T) {
    const int rr = T * 32 + (lane & 31);
    if (rr >= Mt) continue;
    const int e = max((int)((rowmax[sl.base + m0 + rr] >> 23) & 0xFFu) - 127 - 14, -100);
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
    MOEQ_GLOBAL float* pout = (MOEQ_GLOBAL float*)(a.partial + (size_t)prow * H + row0);
#pragma unroll
    for (int r = 0; r < RD_RT; ++r)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        f32x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = acc[r][T][4 * q + i] * sc;
        *reinterpret_cast<MOEQ_GLOBAL f32x4*>(pout + 32 * r + rd_acc_row(4 * q, lane)) = v;
      }
  }
}

// grid: tile_grid(max m-tiles, n-tiles); tiles of slots whose gate and up
// (down) tensors are both 2-4 bits wide
__global__ __launch_bounds__(RD_THREADS, 1) void gateup_rd_kernel(DecodeArgs a) {
  extern __shared__ __attribute__((aligned(16))) char lds_c[];
  const int nN = (a.I + RD_ROWS / 2 - 1) / (RD_ROWS / 2);
  int mt, nt;
  if (!rd_tile_of_wg(a.tiles_rd, blockIdx.x, nN, &mt, &nt)) return;
  const SlotInfo sl = slot_of(a, a.tiles_rd[1 + 2 * mt]);
  const int m0 = a.tiles_rd[2 + 2 * mt];
  const TensorDev tg = a.desc[sl.desc * 3 + 0], tu = a.desc[sl.desc * 3 + 1];
  if (!tg.codes || !tu.codes || !rd_ok(tg) || !rd_ok(tu)) return;
  const int Mt = min(RD_T, sl.M - m0);
  const GemmArgs g = gemm_args(a);
  const int f0 = nt * (RD_ROWS / 2);
  if (Mt <= 32)
    rd_gateup_tile<1>(g, sl, m0, Mt, f0, tg, tu, lds_c);
  else if (RD_NTMAX == 2 || Mt <= 64)
    rd_gateup_tile<2>(g, sl, m0, Mt, f0, tg, tu, lds_c);
  else if constexpr (RD_NTMAX == 4) {
    if (Mt <= 96)
      rd_gateup_tile<3>(g, sl, m0, Mt, f0, tg, tu, lds_c);
    else
      rd_gateup_tile<4>(g, sl, m0, Mt, f0, tg, tu, lds_c);
  }
}

__global__ __launch_bounds__(RD_THREADS, 1) void down_rd_kernel(DecodeArgs a) {
  extern __shared__ __attribute__((aligned(16))) char lds_c[];
  const int nN = (a.H + RD_ROWS - 1) / RD_ROWS;
  int mt, nt;
  if (!rd_tile_of_wg(a.tiles_rd, blockIdx.x, nN, &mt, &nt)) return;
  const SlotInfo sl = slot_of(a, a.tiles_rd[1 + 2 * mt]);
  const int m0 = a.tiles_rd[2 + 2 * mt];
  const TensorDev td = a.desc[sl.desc * 3 + 2];
  if (!td.codes || !rd_ok(td)) return;
  const int Mt = min(RD_T, sl.M - m0);
  const GemmArgs g = gemm_args(a);
  const int n0 = nt * RD_ROWS;
  if (Mt <= 32)
    rd_down_tile<1>(g, sl, m0, Mt, n0, td, lds_c);
  else if (RD_NTMAX == 2 || Mt <= 64)
    rd_down_tile<2>(g, sl, m0, Mt, n0, td, lds_c);
  else if constexpr (RD_NTMAX == 4) {
    if (Mt <= 96)
      rd_down_tile<3>(g, sl, m0, Mt, n0, td, lds_c);
    else
      rd_down_tile<4>(g, sl, m0, Mt, n0, td, lds_c);
  }
}

// Diagnostic: one tensor through the grouped GEMMs' decoders, one thread per
// (row, unit): binary16 d * (c - z) bit patterns in natural weight order
// (rd_piece for the tensors the register-decoded GEMMs take, decode_blk for
// the others, as the LDS-decoded GEMMs do).
template <int B>
__global__ __launch_bounds__(256) void dequant_gemm_kernel(TensorDev t, uint16_t* out) {
  const int U = t.K / kUnit;
  const long long gid = (long long)blockIdx.x * 256 + threadIdx.x;
  if (gid >= (long long)t.rows * U) return;
  const int r = (int)(gid / U), u = (int)(gid % U);
  const MOEQ_GLOBAL u32x4* rc = row_chunks(t, B, r);
  const MOEQ_GLOBAL uint16_t* rs = gptr(t.scales + (size_t)r * (t.K / kBlock));
  u32x4* o = reinterpret_cast<u32x4*>(out + (size_t)r * t.K + kUnit * u);
  if (rd_ok(t)) {
    if constexpr (B <= 4) {
    RdUnit<B> un;
#pragma unroll
    for (int j = 0; j < B; ++j) un.c[j] = rc[(size_t)j * U + u];
    un.s = *reinterpret_cast<const MOEQ_GLOBAL u32x2*>(rs + 4 * u);
    const RdConsts kc = rd_consts<B>();
#define DQG(Q, M) o[4 * (Q) + (M)] = __builtin_bit_cast(u32x4, rd_piece<B, Q, M>(un, kc))
    DQG(0, 0); DQG(0, 1); DQG(0, 2); DQG(0, 3);
    DQG(1, 0); DQG(1, 1); DQG(1, 2); DQG(1, 3);
    DQG(2, 0); DQG(2, 1); DQG(2, 2); DQG(2, 3);
    DQG(3, 0); DQG(3, 1); DQG(3, 2); DQG(3, 3);
#undef DQG
    }
  } else {
    __attribute__((aligned(16))) _Float16 blk[32];
#define DQW(Q)                                                                    \
  do {                                                                            \
    const RawBlk rb = load_blk<B, Q>(rc, rs, U, u);                               \
    decode_blk<B>(rb, ((Q) * B) & 3, ((Q) & 1) != 0, blk);                        \
    _Pragma("unroll") for (int i = 0; i < 4; ++i) o[4 * (Q) + i] = reinterpret_cast<const u32x4*>(blk)[i]; \
  } while (0)
    DQW(0); DQW(1); DQW(2); DQW(3);
#undef DQW
  }
}

}  // namespace

int prefill_max_tiles(int n, int k, int S, int n_kept, int rows) {
  const long long nk = (long long)n * k;
  const long long routed = (nk + rows - 1) / rows + (nk < n_kept ? nk : n_kept);
  return (int)(routed + (long long)S * ((n + rows - 1) / rows));
}

int prefill_max_mtiles(int n, int k, int S, int n_kept) { return prefill_max_tiles(n, k, S, n_kept, BM); }
// capacity of the register-decoded list: 8 runs of the longest run any count
// of tiles up to the largest needs
int prefill_max_rtiles(int n, int k, int S, int n_kept) {
  const int T = prefill_max_tiles(n, k, S, n_kept, kRdTile);
  const int g = kRdDeal ? kRdDeal * kXcds : kXcds;
  return (T + g - 1) / g * g;
}

namespace {

// Raises a GEMM kernel's dynamic LDS limit (once per device and kernel), then
// launches it.
constexpr int kMaxDevices = 64;
template <typename K>
hipError_t launch_gemm(K kernel, std::atomic<uint64_t>& done, int block, int grid, size_t lds, hipStream_t s,
                       const DecodeArgs& a) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev < kMaxDevices ? 1ull << dev : 0ull;
  if (!bit || !(done.load(std::memory_order_acquire) & bit)) {
    e = hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    done.fetch_or(bit, std::memory_order_release);
  }
  kernel<<<grid, block, lds, s>>>(a);
  return hipGetLastError();
}

std::atomic<uint64_t> g_attr_gu_rd{0}, g_attr_dn_rd{0}, g_attr_gu_w{0}, g_attr_dn_w{0};

}  // namespace

hipError_t launch_dequant_gemm(const TensorDev& t, uint16_t* out, hipStream_t s) {
  const long long n = (long long)t.rows * (t.K / kUnit);
  const int grid = (int)((n + 255) / 256);
  switch (t.bits) {
    case 2: dequant_gemm_kernel<2><<<grid, 256, 0, s>>>(t, out); break;
    case 3: dequant_gemm_kernel<3><<<grid, 256, 0, s>>>(t, out); break;
    case 4: dequant_gemm_kernel<4><<<grid, 256, 0, s>>>(t, out); break;
    case 5: dequant_gemm_kernel<5><<<grid, 256, 0, s>>>(t, out); break;
    case 6: dequant_gemm_kernel<6><<<grid, 256, 0, s>>>(t, out); break;
    case 8: dequant_gemm_kernel<8><<<grid, 256, 0, s>>>(t, out); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_prefill_tiles(const DecodeArgs& a, hipStream_t s) {
  prefill_tiles_kernel<<<1, 1024, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_gateup_prefill(const DecodeArgs& a, hipStream_t s) {
  hipError_t e = launch_gemm(gateup_rd_kernel, g_attr_gu_rd, RD_THREADS, tile_grid(a.max_rtiles, (a.I + RD_ROWS / 2 - 1) / (RD_ROWS / 2)),
                             RD_LDS, s, a);
  if (e == hipSuccess && a.lds_gateup) {
    const size_t lds = (size_t)2 * (BM + 2 * BN) * LDS_STRIDE * sizeof(_Float16);
    e = launch_gemm(gateup_gemm8_kernel, g_attr_gu_w, 512, tile_grid(a.max_mtiles, a.I / BN), lds, s, a);
  }
  return e;
}

hipError_t launch_down_prefill(const DecodeArgs& a, hipStream_t s) {
  const int rows = a.n * (a.k + a.S);
  h16_kernel<<<(rows + 3) / 4, 256, 0, s>>>(a.h, a.rowmax, rows, a.I, a.h16);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_gemm(down_rd_kernel, g_attr_dn_rd, RD_THREADS, tile_grid(a.max_rtiles, (a.H + RD_ROWS - 1) / RD_ROWS),
                  RD_LDS, s, a);
  if (e == hipSuccess && a.lds_down) {
    const size_t lds = (size_t)2 * (BM + BN) * LDS_STRIDE * sizeof(_Float16);
    e = launch_gemm(down_gemm8_kernel, g_attr_dn_w, 512, tile_grid(a.max_mtiles, a.H / BN), lds, s, a);
  }
  return e;
}

}  // namespace moeq

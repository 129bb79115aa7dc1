// Prefill path: grouped GEMM on the matrix cores for many tokens.
//
// Every active expert (and the shared expert, whose bucket is all n tokens)
// multiplies its bucket of tokens by its weights, so the layer becomes a set
// of independent GEMMs of very different heights (routing is skewed).  The
// bucketing permutation lists each expert's tokens contiguously; a small
// kernel cuts every bucket into m-tiles of kGemmBM (128) rows, a remainder
// of at most 64 rows into a 64-row tile for the gate/up GEMM, and writes the
// tile lists, so the GEMM grids never depend on a host synchronization.
//
// Arithmetic: activations (bf16, exact in binary16 after a per-token
// power-of-two prescale), dequantized weights fp16(d * (c - z)) (one rounding)
// and the SwiGLU activations h (binary16 after a per-row power-of-two
// prescale) enter v_mfma_f32_16x16x32_f16 with float32 accumulation.  The
// packed-weight tile of each K step is decoded once per workgroup into LDS.
//
// Workgroup tile: 128 rows (tokens) x 128 output features (per projection;
// gate/up computes both projections of the same features so SwiGLU is fused
// into the epilogue), K step 64, eight waves (two per SIMD) in a 2 x 4
// arrangement, each owning 64 rows x 32 columns of 16 x 16 MFMA tiles.  LDS
// holds two decoded K steps and registers the raw data of the next two, so
// the decode of one step and the loads of later ones overlap the current
// step's MFMAs.  Workgroups are mapped to tiles from the tile count on the
// device: each XCD takes an equal run of consecutive m-tiles (one expert's
// tiles share its L2), whatever the worst-case size of the grid.
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

// ---- tile lists: slot order = shared experts, then active experts ----
// For the gate/up GEMM of 2-4-bit tensors a bucket of M rows becomes M / 128
// full 128-row tiles; a remainder of more than 64 rows takes one more
// 128-row tile, one of 1..64 rows a 64-row tile in the second list.  The
// third list cuts every bucket into ceil(M / 128) 128-row tiles (the GEMMs
// without a 64-row variant), large and small buckets interleaved in slot
// order, so every XCD's share mixes both.
__global__ __launch_bounds__(1024) void prefill_tiles_kernel(DecodeArgs a) {
  __shared__ int32_t cnt[kMaxShared + kMaxExperts + 1];   // 128-row tiles
  __shared__ int32_t scnt[kMaxShared + kMaxExperts + 1];  // 64-row tile (0 or 1)
  __shared__ int32_t off[kMaxShared + kMaxExperts + 2];
  __shared__ int32_t soff[kMaxShared + kMaxExperts + 2];
  __shared__ int32_t aoff[kMaxShared + kMaxExperts + 2];
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
    const int r = M % BM;
    cnt[s] = M / BM + (r > BM / 2 ? 1 : 0);
    scnt[s] = r > 0 && r <= BM / 2 ? 1 : 0;
  }
  // rows of h whose running maxima the gate/up epilogue accumulates
  const int rows = a.n * (a.k + a.S);
  for (int r = tid; r < rows; r += 1024) a.rowmax[r] = 0u;
  __syncthreads();
  if (tid == 0) {
    int run = 0, srun = 0, arun = 0;
    for (int s = 0; s < nslots; ++s) {
      off[s] = run;
      soff[s] = srun;
      aoff[s] = arun;
      run += cnt[s];
      srun += scnt[s];
      arun += cnt[s] + scnt[s];
    }
    a.tiles[0] = min(run, a.max_mtiles);
    a.tiles_small[0] = min(srun, a.max_small);
    a.tiles_all[0] = min(arun, a.max_mtiles);
  }
  __syncthreads();
  for (int s = tid; s < nslots; s += 1024) {
    const int nb = cnt[s];
    for (int i = 0; i < nb; ++i) {
      const int t = off[s] + i;
      if (t < a.max_mtiles) {
        a.tiles[1 + 2 * t] = s;
        a.tiles[2 + 2 * t] = i * BM;
      }
    }
    if (scnt[s] && soff[s] < a.max_small) {
      a.tiles_small[1 + 2 * soff[s]] = s;
      a.tiles_small[2 + 2 * soff[s]] = nb * BM;
    }
    for (int i = 0; i < nb + scnt[s]; ++i) {
      const int t = aoff[s] + i;
      if (t < a.max_mtiles) {
        a.tiles_all[1 + 2 * t] = s;
        a.tiles_all[2 + 2 * t] = i * BM;
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
constexpr int kXcds = 8;
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

template <bool WIDE>
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
  } else if (!WIDE || bits == 4) {
    if (blk) GU8(4, 1); else GU8(4, 0);
  } else if constexpr (WIDE) {
    if (bits == 5) {
      if (blk) GU8(5, 1); else GU8(5, 0);
    } else if (bits == 6) {
      if (blk) GU8(6, 1); else GU8(6, 0);
    } else {
      if (blk) GU8(8, 1); else GU8(8, 0);
    }
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

// Launched with WIDE = true: the tiles with a 5, 6 or 8-bit gate or up
// tensor (the other of the two may be narrower).  The 2-4-bit tiles take the
// raw-staged gateup_rs_kernel; WIDE = false, their register-path variant, is
// not launched.
template <bool WIDE>
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
  if ((tg.bits > 4 || tu.bits > 4) != WIDE) return;
  gateup_gemm_body8<WIDE>(gemm_args(a), sl, m0, nt * BN, tg, tu, lds_h);
}

template <bool WIDE>
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
  } else if constexpr (!WIDE) {
    if (bits == 2) {
      if (blk) DN8(2, 1); else DN8(2, 0);
    } else if (bits == 3) {
      if (blk) DN8(3, 1); else DN8(3, 0);
    } else {
      if (blk) DN8(4, 1); else DN8(4, 0);
    }
  } else {
    if (bits == 5) {
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

// WIDE = false takes the tiles whose down tensor is 2-4 bits wide, WIDE = true
// the 5, 6 and 8-bit ones.  Four waves per SIMD (128 registers): two
// workgroups share a compute unit (2 x 80 KB of LDS) and overlap their K-step
// chains.
template <bool WIDE>
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
  if ((td.bits > 4) != WIDE) return;
  down_gemm_body8<WIDE>(gemm_args(a), sl, m0, nt * BN, td, lds_h);
}

// ---------------------------------------------------------------------------
// Raw-staged grouped GEMM for 2-4 bit weights.
//
// In the kernels above every lane loads one 16-byte chunk of a different
// weight row per K step: each load brings a whole cache line from L2 and
// uses a quarter of it or less, and the line is gone before the same thread
// needs its neighbour, so the L1 miss traffic, not the matrix cores, sets
// the pace.  Here the decode waves load the packed codes (and scales) of 4
// units (512 k, 8 K steps) of all 128 weight rows of the tile at once, 4
// lanes per row and chunk plane (64 contiguous bytes), store them in LDS,
// and each K step decodes its block from LDS into the binary16 tile.
//
// Used for gate/up (the down GEMM, with a quarter of the K steps per tile,
// measured faster with the per-thread loads above).  The loop is written for
// NT tensors of 128 / NT rows each.  Tile: 128 tokens x 128 weight rows (64
// features of each projection, rows 0-63 gate and 64-127 up).  Waves
// 0-3 load and decode (wave w: rows 64 (w % 2) .. +63, block half w / 2 of
// each half unit, so every wave works on one tensor and one width), waves
// 4-7 move activations (32 values of tile row (t - 256) / 2 per step).
// The eight waves share the MFMAs: 2 x 4 waves of 64 tokens x 16 features
// per projection.
constexpr int RS_ROWS = 128;
constexpr int RS_RAW = 4 * 16 + 4;   // dwords per staged row: 4 chunk planes x 4 units (+ padding)
constexpr int RS_SCL = 10;           // dwords per staged row of scales: 16 binary16 (+ padding; even, so
                                     // the 8-byte stores stay aligned)
// LDS of a tile of bmt tokens: A [2][bmt], W [2][128], raw and scale stages
constexpr size_t rs_lds(int bmt) {
  return (size_t)2 * (bmt + RS_ROWS) * LDS_STRIDE * 2 + (size_t)2 * RS_ROWS * RS_RAW * 4 +
         (size_t)2 * RS_ROWS * RS_SCL * 4;
}
static_assert(rs_lds(BM) <= 160 * 1024, "the raw-staged tile must fit the LDS of a compute unit");

// one raw stage (4 units) of this lane: 2B chunk pieces and 2 scale pieces
template <int B>
struct RsStage {
  u32x4 c[2 * B];
  u32x2 s[2];
};

// Piece m of a wave's tensor (RPT rows, WPT waves per tensor, h = this wave's
// index among them): row ((lane / 4) + 16 m) mod RPT, unit lane % 4, chunk
// plane m / (RPT / 16); the wave takes m = WPT i + h.
template <int B, int NT>
__device__ __forceinline__ void rs_load(RsStage<B>& st, const TensorDev& t, int n0, int U, int K, int u0, int lane,
                                        int h) {
  constexpr int RPT = RS_ROWS / NT, WPT = 4 / NT;
  const int uu = min(u0 + (lane & 3), U - 1);
#pragma unroll
  for (int i = 0; i < 2 * B; ++i) {
    const int m = WPT * i + h;
    const int r = ((lane >> 2) + 16 * m) % RPT, j = m / (RPT / 16);
    const MOEQ_GLOBAL u32x4* rc = gptr(reinterpret_cast<const u32x4*>(t.codes + (size_t)(n0 + r) * B * U * 4));
    st.c[i] = rc[(size_t)j * U + uu];
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int m = WPT * i + h;
    const int r = ((lane >> 2) + 16 * m) % RPT;
    st.s[i] = *gptr(reinterpret_cast<const u32x2*>(t.scales + (size_t)(n0 + r) * (K / kBlock)) + uu);
  }
}

template <int B, int NT>
__device__ __forceinline__ void rs_store(const RsStage<B>& st, uint32_t* raw, uint32_t* scl, int tt, int lane, int h) {
  constexpr int RPT = RS_ROWS / NT, WPT = 4 / NT;
#pragma unroll
  for (int i = 0; i < 2 * B; ++i) {
    const int m = WPT * i + h;
    const int r = ((lane >> 2) + 16 * m) % RPT, j = m / (RPT / 16);
    *reinterpret_cast<u32x4*>(raw + (tt * RPT + r) * RS_RAW + j * 16 + (lane & 3) * 4) = st.c[i];
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int m = WPT * i + h;
    const int r = ((lane >> 2) + 16 * m) % RPT;
    *reinterpret_cast<u32x2*>(scl + (tt * RPT + r) * RS_SCL + (lane & 3) * 2) = st.s[i];
  }
}

// Block Q of staged unit ul of LDS row `row` (the chunks it occupies and the
// aligned pair of scales holding its own).
template <int B, int Q>
__device__ __forceinline__ RawBlk rs_block(const uint32_t* raw, const uint32_t* scl, int row, int ul) {
  constexpr int c0 = (Q * B) >> 2;
  constexpr bool two = ((Q * B) & 3) + B > 4;
  RawBlk r;
  const uint32_t* base = raw + row * RS_RAW + ul * 4;
  r.a = *reinterpret_cast<const u32x4*>(base + c0 * 16);
  if constexpr (two)
    r.b = *reinterpret_cast<const u32x4*>(base + (c0 + 1) * 16);
  else
    r.b = u32x4{0u, 0u, 0u, 0u};
  r.sc = scl[row * RS_SCL + ul * 2 + (Q >> 1)];
  return r;
}

// MI: 16-row MFMA tiles per wave along the tokens (4 for 128-token tiles, 2
// for 64-token tiles)
template <int NT, int C, int MI>
__device__ __forceinline__ void read_frags_rs(const _Float16* A, const _Float16* W, int lane, int wm, int wn,
                                              half8 (&fa)[2][MI], half8 (&fb)[2][NT][C]) {
  constexpr int RPT = RS_ROWS / NT;
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const int kof = kk * 32 + (lane >> 4) * 8;
#pragma unroll
    for (int i = 0; i < MI; ++i) fa[kk][i] = lds_frag(A + (wm * 16 * MI + 16 * i + (lane & 15)) * LDS_STRIDE + kof);
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int c = 0; c < C; ++c)
        fb[kk][t][c] = lds_frag(W + (t * RPT + wn * 16 * C + 16 * c + (lane & 15)) * LDS_STRIDE + kof);
  }
}

template <int NT, int C, int MI>
__device__ __forceinline__ void mfmas_rs(const half8 (&fa)[2][MI], const half8 (&fb)[2][NT][C],
                                         f32x4v (&acc)[NT][MI][C]) {
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < MI; ++i)
          acc[t][i][c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[kk][i], fb[kk][t][c], acc[t][i][c], 0, 0, 0);
}

// One K loop.  DW: this wave stages and decodes weights of width B (block
// half BLK of its rows; its tensor t, index h among the tensor's waves),
// else it moves MI pieces of activations per step.  LDS: A [2][32 MI], W
// [2][128] (binary16 rows of LDS_STRIDE), raw [2][128][RS_RAW], scales
// [2][128][RS_SCL].  Raw stage t (K steps 8t .. 8t + 7) is stored to LDS at
// step 8t - 2 and requested one stage earlier, at step 8t - 10 (the prologue
// loads stage 0 and requests stage 1), so its loads have a whole stage to
// arrive; step s + 1 is decoded during step s.
template <int NT, int C, int B, int BLK, bool DW, int MI>
__device__ __forceinline__ void gemm_loop_rs(const TensorDev& t, int tt, int h, int n0, int U, int K,
                                             const MOEQ_GLOBAL u32x4* arow, _Float16* adst, _Float16* As, _Float16* Ws,
                                             uint32_t* raw, uint32_t* scl, int lane, int wm, int wn, int nk,
                                             f32x4v (&acc)[NT][MI][C]) {
  constexpr int ABUF = 32 * MI * LDS_STRIDE;  // halves per A buffer
  const int wrow = tt * 64 + lane;     // decode row: rows 64 (w % 2) + lane
  const int ts = NT == 2 ? tt : 0;     // the staged tensor of this wave
  RsStage<B> st;
  u32x4 xv[2][MI];
  // decode step s into W buffer s % 2 (S2: s % 2, compile-time)
#define RS_DECODE(S2, s)                                                                                   \
  do {                                                                                                     \
    if constexpr (DW) {                                                                                    \
      const int sb_ = ((s) >> 3) & 1, ul_ = ((s) >> 1) & 3;                                               \
      const RawBlk rb_ = rs_block<B, 2 * (S2) + BLK>(raw + sb_ * RS_ROWS * RS_RAW, scl + sb_ * RS_ROWS * RS_SCL, \
                                                     wrow, ul_);                                           \
      decode_blk<B>(rb_, ((2 * (S2) + BLK) * B) & 3, BLK != 0,                                            \
                    Ws + (S2) * (RS_ROWS * LDS_STRIDE) + wrow * LDS_STRIDE + 32 * BLK);                    \
    }                                                                                                      \
  } while (0)
#define RS_AMOVE(S2)                                                                                       \
  do {                                                                                                     \
    if constexpr (!DW) {                                                                                   \
      u32x4* ad_ = reinterpret_cast<u32x4*>(adst + (S2) * ABUF);                                          \
      _Pragma("unroll") for (int i_ = 0; i_ < MI; ++i_) ad_[i_] = xv[S2][i_];                              \
    }                                                                                                      \
  } while (0)
#define RS_ALOAD(S2, s)                                                                                    \
  do {                                                                                                     \
    if constexpr (!DW) {                                                                                   \
      _Pragma("unroll") for (int i_ = 0; i_ < MI; ++i_) xv[S2][i_] = arow[(s) * 8 + i_];                   \
    }                                                                                                      \
  } while (0)
  // raw stage handling at the end of step s's work: store stage (s / 8) + 1
  // at step s % 8 == 6, then request stage (s / 8) + 2
#define RS_STAGE(s)                                                                                        \
  do {                                                                                                     \
    if constexpr (DW) {                                                                                    \
      if (((s) & 7) == 6 && (s) + 2 < nk) {                                                                \
        const int nb_ = (((s) >> 3) + 1) & 1;                                                              \
        rs_store<B, NT>(st, raw + nb_ * RS_ROWS * RS_RAW, scl + nb_ * RS_ROWS * RS_SCL, ts, lane, h);       \
        if (8 * (((s) >> 3) + 2) < nk) rs_load<B, NT>(st, t, n0, U, K, 4 * (((s) >> 3) + 2), lane, h);     \
      }                                                                                                    \
    }                                                                                                      \
  } while (0)
#define RS_STEP(P, s)                                                                                      \
  do {                                                                                                     \
    half8 fa[2][MI], fb[2][NT][C];                                                                         \
    read_frags_rs<NT, C, MI>(As + (P) * ABUF, Ws + (P) * (RS_ROWS * LDS_STRIDE), lane, wm, wn, fa, fb);   \
    RS_DECODE(1 - (P), (s) + 1);                                                                           \
    RS_AMOVE(1 - (P));                                                                                     \
    RS_ALOAD(1 - (P), min((s) + 3, nk - 1));                                                               \
    RS_STAGE(s);                                                                                           \
    mfmas_rs<NT, C, MI>(fa, fb, acc);                                                                      \
    __syncthreads();                                                                                       \
  } while (0)
  // prologue: stage 0 stored, stage 1 requested; steps 0 (decoded) and 1 (loaded)
  if constexpr (DW) {
    rs_load<B, NT>(st, t, n0, U, K, 0, lane, h);
    rs_store<B, NT>(st, raw, scl, ts, lane, h);
    if (8 < nk) rs_load<B, NT>(st, t, n0, U, K, 4, lane, h);
  }
  RS_ALOAD(0, 0);
  RS_ALOAD(1, min(1, nk - 1));
  __syncthreads();
  RS_DECODE(0, 0);
  RS_AMOVE(0);
  RS_ALOAD(0, min(2, nk - 1));
  __syncthreads();
  for (int s0 = 0; s0 < nk; s0 += 2) {
    RS_STEP(0, s0);
    RS_STEP(1, s0 + 1);
  }
#undef RS_DECODE
#undef RS_AMOVE
#undef RS_ALOAD
#undef RS_STAGE
#undef RS_STEP
}

// Tile of BMT tokens (128 or 64).  The 256 movers take piece t % TPR of tile
// row t / TPR (TPR = 2 or 4 movers per row, MI 16-byte pieces each per step).
template <int BMT>
__device__ void gateup_rs_body(const GemmArgs a, const SlotInfo sl, int m0, int n0, const TensorDev tg,
                               const TensorDev tu, _Float16* lds) {
  constexpr int MI = BMT / 32, TPR = 8 / MI;
  _Float16* As = lds;
  _Float16* Ws = lds + 2 * BMT * LDS_STRIDE;
  uint32_t* raw = reinterpret_cast<uint32_t*>(Ws + 2 * RS_ROWS * LDS_STRIDE);
  uint32_t* scl = raw + 2 * RS_ROWS * RS_RAW;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int H = a.H, I = a.I, U = H / kUnit;
  const MOEQ_GLOBAL int32_t* perm = gptr(a.perm);
  const MOEQ_GLOBAL int32_t* xexp = gptr(a.xexp);
  const bool dw = __builtin_amdgcn_readfirstlane(wave) < 4;
  const int tt = wave & 1, h = (wave >> 1) & 1, blk = (wave >> 1) & 1;
  const TensorDev t = tt ? tu : tg;
  const int bits = __builtin_amdgcn_readfirstlane(t.bits);
  const int ar = (tid & 255) / TPR, aq = (tid & 255) % TPR;
  int tok = 0;
  if (m0 + ar < sl.M) tok = sl.shared >= 0 ? m0 + ar : perm[sl.base + m0 + ar] / a.k;
  const MOEQ_GLOBAL u32x4* arow = gptr(reinterpret_cast<const u32x4*>(a.x16 + (size_t)tok * H)) + MI * aq;
  _Float16* adst = As + ar * LDS_STRIDE + 8 * MI * aq;

  f32x4v acc[2][MI][1];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int i = 0; i < MI; ++i) acc[q][i][0] = f32x4v{0.f, 0.f, 0.f, 0.f};
  const int nk = H / BK;
#define GURS(B, BL) \
  gemm_loop_rs<2, 1, B, BL, true, MI>(t, tt, h, n0, U, H, arow, adst, As, Ws, raw, scl, lane, wm, wn, nk, acc)
  if (!dw) {
    gemm_loop_rs<2, 1, 2, 0, false, MI>(t, tt, h, n0, U, H, arow, adst, As, Ws, raw, scl, lane, wm, wn, nk, acc);
  } else if (bits == 2) {
    if (blk) GURS(2, 1); else GURS(2, 0);
  } else if (bits == 3) {
    if (blk) GURS(3, 1); else GURS(3, 0);
  } else {
    if (blk) GURS(4, 1); else GURS(4, 0);
  }
#undef GURS

  // epilogue: undo the activation prescale, SwiGLU, store h, track row maxima
#pragma unroll
  for (int i = 0; i < MI; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = wm * 16 * MI + 16 * i + (lane >> 4) * 4 + j;
      const bool ok = m0 + r < sl.M;
      float sc = 1.0f;
      if (ok) {
        const int tk = sl.shared >= 0 ? m0 + r : perm[sl.base + m0 + r] / a.k;
        sc = __builtin_amdgcn_ldexpf(1.0f, xexp[tk]);
      }
      MOEQ_GLOBAL float* hout = (MOEQ_GLOBAL float*)(a.h + (size_t)(sl.base + m0 + r) * I);
      const int col = n0 + wn * 16 + (lane & 15);
      const float hv = silu(acc[0][i][0][j] * sc) * (acc[1][i][0][j] * sc);
      if (ok) hout[col] = hv;
      float rmax = fabsf(hv);
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) rmax = fmaxf(rmax, __shfl_xor(rmax, off, 64));
      if (ok && (lane & 15) == 0) atomicMax(a.rowmax + sl.base + m0 + r, __float_as_uint(rmax));
    }
  }
}

// grid = m-tiles x (I / 64); tiles whose gate and up tensors are 2-4 bits
// wide, from the 128-row list (BMT = 128) or the 64-row list (BMT = 64)
template <int BMT>
__global__ __launch_bounds__(512, 1) void gateup_rs_kernel(DecodeArgs a) {
  extern __shared__ _Float16 lds_h[];
  const int nN = a.I / 64;
  const int32_t* tl = BMT == BM ? a.tiles : a.tiles_small;
  int mt, nt;
  if (!tile_of_wg(blockIdx.x, tl[0], nN, &mt, &nt)) return;
  const SlotInfo sl = slot_of(a, tl[1 + 2 * mt]);
  const int m0 = tl[2 + 2 * mt];
  const TensorDev tg = a.desc[sl.desc * 3 + 0], tu = a.desc[sl.desc * 3 + 1];
  if (!tg.codes || !tu.codes) return;
  if (tg.bits > 4 || tu.bits > 4) return;
  gateup_rs_body<BMT>(gemm_args(a), sl, m0, nt * 64, tg, tu, lds_h);
}

}  // namespace

int prefill_max_mtiles(int n, int k, int S, int n_kept) {
  const long long nk = (long long)n * k;
  const long long routed = (nk + BM - 1) / BM + (nk < n_kept ? nk : n_kept);
  return (int)(routed + (long long)S * ((n + BM - 1) / BM));
}

int prefill_max_small(int n, int k, int S, int n_kept) {
  const long long nk = (long long)n * k;
  return (int)((nk < n_kept ? nk : n_kept) + S);
}

namespace {

// sets the LDS limit of a GEMM kernel once per process, then launches it
template <typename K>
hipError_t launch_gemm(K kernel, bool& attr, int grid, size_t lds, hipStream_t s, const DecodeArgs& a) {
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr = true;
  }
  kernel<<<grid, 512, lds, s>>>(a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_prefill_tiles(const DecodeArgs& a, hipStream_t s) {
  prefill_tiles_kernel<<<1, 1024, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_gateup_prefill_big(const DecodeArgs& a, hipStream_t s) {
  const size_t lds = (size_t)2 * (BM + 2 * BN) * LDS_STRIDE * sizeof(_Float16);
  const int grid = tile_grid(a.max_mtiles, a.I / BN);
  static bool attr_n = false, attr_w = false;
  hipError_t e = launch_gemm(gateup_rs_kernel<BM>, attr_n, tile_grid(a.max_mtiles, a.I / 64), rs_lds(BM), s, a);
  if (e == hipSuccess && a.wide_gateup) e = launch_gemm(gateup_gemm8_kernel<true>, attr_w, grid, lds, s, a);
  return e;
}

hipError_t launch_gateup_prefill_small(const DecodeArgs& a, hipStream_t s2) {
  static bool attr_s = false;
  return launch_gemm(gateup_rs_kernel<BM / 2>, attr_s, tile_grid(a.max_small, a.I / 64), rs_lds(BM / 2), s2, a);
}

hipError_t launch_gateup_prefill(const DecodeArgs& a, hipStream_t s) {
  hipError_t e = launch_prefill_tiles(a, s);
  if (e == hipSuccess) e = launch_gateup_prefill_big(a, s);
  if (e == hipSuccess) e = launch_gateup_prefill_small(a, s);
  return e;
}

hipError_t launch_down_prefill(const DecodeArgs& a, hipStream_t s) {
  const int rows = a.n * (a.k + a.S);
  h16_kernel<<<(rows + 3) / 4, 256, 0, s>>>(a.h, a.rowmax, rows, a.I, a.h16);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t lds = (size_t)2 * (BM + BN) * LDS_STRIDE * sizeof(_Float16);
  const int grid = tile_grid(a.max_mtiles, a.H / BN);
  static bool attr_n = false, attr_w = false;
  e = launch_gemm(down_gemm8_kernel<false>, attr_n, grid, lds, s, a);
  if (e == hipSuccess && a.wide_down) e = launch_gemm(down_gemm8_kernel<true>, attr_w, grid, lds, s, a);
  return e;
}

}  // namespace moeq

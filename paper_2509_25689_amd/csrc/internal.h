// Internal declarations shared by the host runtime (api.cpp) and the HIP
// kernel files.  Not part of the public interface (include/moeq.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdint.h>

#include "moeq.h"

namespace moeq {

// Records the calling thread's error text (moeq_last_error) and returns st.
moeq_status vset_error(moeq_status st, const char* fmt, va_list ap);

// Weights per device unit: four blocks of 32.  A lane of a GEMV wave owns one
// unit of a row at a time; hidden and inter must be multiples of this.
constexpr int kUnit = 128;
constexpr int kBlock = 32;
constexpr int kMaxExperts = 1024;
constexpr int kMaxTopK = 32;
constexpr int kMaxShared = 4;
constexpr int kChunk = 64;          // tokens per bucketing chunk (one bit per token in a 64-bit mask)
constexpr int kDecodeMaxTokens = 64;
constexpr int kDefaultDecodeMax = 64;

// One stored tensor in the device layout.
//   codes:  rows * (K/128) units of 16*bits bytes.  Row r's unit u, 16-byte
//           chunk j lives at byte ((r*bits + j) * U + u) * 16 with U = K/128,
//           so that chunk j of consecutive units is contiguous (one coalesced
//           load per wave per chunk).  Inside a unit, block q (q = 0..3) is the
//           dwords [q*bits, q*bits + bits) of the unit's 4*bits dwords, encoded
//           as in encode_block() (weights.hip).
//   scales: row-major [rows x K/32] binary16 (the canonical array, unchanged).
struct TensorDev {
  const uint32_t* codes;
  const uint16_t* scales;
  int32_t bits;
  int32_t rows;
  int32_t K;
  int32_t flags;  // kTensor* bits
};

// TensorDev.flags: the grouped GEMMs' register-decoded kernels cannot take
// the tensor, because some block scale is not a positive finite binary16 at
// most rd_scale_limit(bits) (they form d * (c - z) from d * 2^(14 + b)) or
// its rows hold an odd number of 128-weight units (they load the scales of
// two units at once); its tiles go to the LDS-decoded kernels instead.
constexpr int32_t kTensorOffRegisterDecoder = 1;
// Largest binary16 bit pattern of a scale d with d * 2^(14 + b) finite.
constexpr uint32_t rd_scale_limit(int b) { return 0x7BFFu - ((uint32_t)(14 + b) << 10); }

struct RouterParams {
  const float* logits;    // [n x E_row]
  const uint8_t* mask;    // [E_row] device copy
  const float* bias;      // [E_row] device copy (zeros when none was given)
  // router experts: E_row (original ids) or, when kept_ids is set, the E
  // kept experts in ascending id order (groups formed over them alone)
  const int32_t* kept_ids;
  int32_t E_row;
  int32_t E, G, TG, k, topn, norm;
  float scale;
  // optional (many-token path): activations whose per-token binary exponent
  // prescale for half precision is written to xexp, and the prescaled
  // binary16 copy x * 2^-xexp to x16
  const uint16_t* x;      // bf16 [n x H] or null
  int32_t H;
  int32_t* xexp;          // [n]
  uint16_t* x16;          // binary16 [n x H]
};

// Workspace views (device pointers) for one forward.
struct Workspace {
  int32_t* idx;        // [T*k]   chosen experts, token-major
  float* w;            // [T*k]   combine weights
  int32_t* offsets;    // [E+1]
  int32_t* perm;       // [T*k]   bucket order -> t*k + j
  int32_t* active;     // [1+E]   count, then active expert ids ascending
  int32_t* chunk_cnt;  // [C*E]   per-chunk counts, then per-chunk bucket bases
  int32_t* rank;       // [T*k]   rank of an assignment inside its chunk and expert
  float* h;            // [(T*k + T*S) x I] SwiGLU activations, bucket order then shared
  float* partial;      // [(T*k + T*S) x H] per-assignment expert outputs, t*k + j then shared
  int32_t* xexp;       // [T]     per-token exponent e: x * 2^-e fits binary16
  uint32_t* rowmax;    // [T*k + T*S] max |h| of each activation row (float bits)
  int32_t* tiles_all;  // [1 + 2*max_mtiles] count, then (slot, first row) of every bucket's
                       // tiles of up to 128 rows, slot order
  int32_t* tiles_rd;   // [1 + 2*max_rtiles] the same for tiles of up to 64 rows
  uint16_t* x16;       // [T x H]  binary16 x * 2^-xexp (many-token path)
  uint16_t* h16;       // [(T*k + T*S) x I] binary16 h * 2^-(row exponent) (many-token path)
  uint32_t* zeros;     // [64]    zeroed at create, never written again
};

// ---- launchers (return hipSuccess or the launch error) ----
// route.hip
hipError_t launch_route_bucket_small(const RouterParams& rp, const int32_t* idx_in, int n,
                                     const Workspace& ws, hipStream_t s);
hipError_t launch_route_tokens(const RouterParams& rp, int n, int32_t* idx, float* w,
                               hipStream_t s);
hipError_t launch_bucket_chunked(const int32_t* idx, int n, int k, int E, const Workspace& ws,
                                 hipStream_t s);
// weights.hip
hipError_t launch_repack(const uint8_t* canon_codes, int rows, int K, int bits,
                         uint32_t* dev_codes, hipStream_t s);
hipError_t launch_dequant(const TensorDev& t, float* out, hipStream_t s);
// widths 2-4: the binary16-subnormal pair decoder rebuilt to float32
hipError_t launch_dequant_sub(const TensorDev& t, float* out, hipStream_t s);
// *out = max over the n binary16 scales of key(s): the magnitude bits of a
// positive finite scale, 0xFFFF for a zero, negative or non-finite one
// (atomic maximum: *out must start at 0)
hipError_t launch_scale_key_max(const uint16_t* scales, size_t n, uint32_t* out, hipStream_t s);
hipError_t launch_quantize(const float* w, int rows, int K, int bits, uint8_t* codes,
                           uint16_t* scales, hipStream_t s);
// decode.hip
struct DecodeArgs {
  const TensorDev* desc;  // [(E + S) * 3]
  const uint16_t* x;      // bf16 [n x H]
  const int32_t* active;
  const int32_t* offsets;
  const int32_t* perm;
  const float* w;
  float* h;
  float* partial;
  float* y;
  int32_t n, H, I, E, S, k;
  int32_t max_active;     // routed slots launched: min(n*k, kept experts)
  // many-token path
  const int32_t* xexp;
  uint32_t* rowmax;
  int32_t max_mtiles;
  int32_t* tiles_all;
  int32_t max_rtiles;
  int32_t* tiles_rd;
  const uint16_t* x16;
  uint16_t* h16;
  const uint32_t* zeros;  // 256 zero bytes
  const int32_t* idx;     // [n*k] chosen experts, token-major
  // width shared by every kept routed and shared down tensor (2-4), else 0
  int32_t down_bits;
  // slots with a 5/6/8-bit gate or up (down) tensor: 0 none, 1 shared
  // experts only, 2 routed experts too
  int32_t wide_gateup, wide_down;
  // many-token path: some kept or shared gate/up (down) tensor is wider than
  // 4 bits or off the register decoder, so the LDS-decoded GEMM runs too
  int32_t lds_gateup, lds_down;
  // buckets of more rows take the grouped GEMMs (prefill path: 0, every
  // bucket; decode path: the large buckets of a skewed routing), the others
  // the dequant-GEMV kernels
  int32_t gemm_above;
};
hipError_t launch_gateup_decode(const DecodeArgs& a, hipStream_t s);
// the same work split over two streams: the one-token buckets (and the wide
// kernels) on s, the buckets of 2-64 tokens on s2 (n > 1; the caller orders
// s2 after the routing and joins it back into s)
hipError_t launch_gateup_decode_single(const DecodeArgs& a, hipStream_t s);
hipError_t launch_gateup_decode_multi(const DecodeArgs& a, hipStream_t s2);
// One token without a routing launch: the gate/up workgroups route the
// token themselves and one of them writes the routing and bucket outputs
// (gateup1_routes: the mask-based router with at most 256 experts)
bool gateup1_routes(const RouterParams& rp);
hipError_t launch_gateup_decode_routing(const DecodeArgs& a, const RouterParams& rp, const Workspace& ws,
                                        hipStream_t s);
// down x routing weight; for one token with 2-4-bit down tensors (down_combines)
// it also sums the slots into y, and the combine is not launched
hipError_t launch_down_decode(const DecodeArgs& a, hipStream_t s);
bool down_combines(const DecodeArgs& a);
hipError_t launch_combine(const DecodeArgs& a, hipStream_t s);
// gate.hip: logits = x W_r^T (bf16 x [n x H], float32 W_r [E x H]); up to
// kGateFewTokens tokens take the streaming kernel, more the tiled one
constexpr int kGateFewTokens = 8;
hipError_t launch_router_gate(const uint16_t* x, const float* w, int n, int H, int E, float* logits,
                              hipStream_t s);
// prune.hip
hipError_t launch_fill_u8(uint8_t* p, int n, uint8_t v, hipStream_t s);
// dst[0..n) = src[0..n) (HOST floats, NULL = zeros), passed by value in the
// kernel arguments: src may be reused as soon as this returns
hipError_t launch_store_host_floats(float* dst, const float* src, int n, hipStream_t s);
hipError_t launch_expert_importance(const int32_t* offsets, const int32_t* perm, const float* w, int E, int n,
                                    double alpha, int keep, double* importance, uint8_t* mask, int32_t* counts,
                                    hipStream_t s);
// prefill.hip
constexpr int kGemmBM = 128;  // tokens per m-tile of the LDS-decoded (5/6/8-bit) GEMMs
#ifndef MOEQ_RD_TILE
#define MOEQ_RD_TILE 128
#endif
constexpr int kRdTile = MOEQ_RD_TILE;  // tokens per tile of the register-decoded (2-4-bit) GEMMs
int prefill_max_mtiles(int n, int k, int S, int n_kept);
int prefill_max_rtiles(int n, int k, int S, int n_kept);
// the tile list (and cleared h row maxima), then the gate/up GEMMs, then
// h in binary16 and the down GEMMs
hipError_t launch_prefill_tiles(const DecodeArgs& a, hipStream_t s);
hipError_t launch_gateup_prefill(const DecodeArgs& a, hipStream_t s);
hipError_t launch_down_prefill(const DecodeArgs& a, hipStream_t s);
// the grouped GEMMs' weight decoder: binary16 d * (c - 2^(b-1)) bit patterns
hipError_t launch_dequant_gemm(const TensorDev& t, uint16_t* out, hipStream_t s);

}  // namespace moeq

// Router and token-to-expert bucketing kernels.
//
// Router (Sections 3.1 and 3.2 of arXiv 2509.25689, with the DeepSeek-V3
// routing function its model uses): for every token, sigmoid affinities over
// all E experts; experts removed by pruning are masked out; each of the G
// contiguous expert groups is scored by the float32 sum of its `topn` best
// kept (biased) scores; the `TG` best groups are kept; the `k` best kept
// experts inside them are chosen, best first; their unbiased scores are
// renormalised (optionally) and multiplied by the routed scale.  Ties go to
// the lower group id, then the lower expert id.  One wavefront routes one
// token: the selection is a sequence of wave-wide arg-max reductions over a
// total order, so it is deterministic and independent of scheduling.
//
// Bucketing: a stable counting sort of the (token, slot) assignments by
// expert.  Within a chunk of 64 tokens each expert keeps a 64-bit mask of the
// tokens that chose it (a token's experts are distinct), which gives per-chunk
// counts and every assignment's rank inside its expert; a scan over chunks and
// experts turns those into global positions.  Integer-only and deterministic.
#include "internal.h"

namespace moeq {

namespace {

constexpr int kWaves = 4;

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// (va, ia) comes before (vb, ib) in the selection order: larger value first,
// lower index first among equal values.
__device__ __forceinline__ bool before(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

__device__ __forceinline__ void wave_argmax(float& v, int& i) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    float ov = __shfl_xor(v, off, 64);
    int oi = __shfl_xor(i, off, 64);
    if (before(ov, oi, v, i)) {
      v = ov;
      i = oi;
    }
  }
}

// Route token t with the calling wavefront.  s_l / b_l: this wave's LDS rows
// of E floats; gs_l: G floats.  Writes idx/w for the token to idx_g/w_g
// (global) and, if idx_s is not null, the ids to idx_s (LDS).
__device__ void route_token_wave(const RouterParams& rp, int t, float* s_l, float* b_l,
                                 float* gs_l, int32_t* idx_g, float* w_g, int32_t* idx_s) {
  const int lane = threadIdx.x & 63;
  const int E = rp.E, G = rp.G, per = rp.E / rp.G;
  const float* lg = rp.logits + (size_t)t * E;
  for (int e = lane; e < E; e += 64) {
    // sigmoid evaluated in double precision, rounded once to float
    float s = (float)(1.0 / (1.0 + exp(-(double)lg[e])));
    if (!(s == s)) s = 0.0f;  // a NaN logit must not leave the index range undefined
    s_l[e] = s;
    b_l[e] = rp.mask[e] ? s + rp.bias[e] : -INFINITY;
  }
  wave_sync();

  // group scores: lane g sums its group's `topn` best kept scores, best first
  for (int g = lane; g < G; g += 64) {
    float acc = 0.0f, pv = INFINITY;
    int pi = -1, taken = 0;
    for (int r = 0; r < rp.topn; ++r) {
      float bv = -INFINITY;
      int bi = INT_MAX;
      for (int e = g * per; e < (g + 1) * per; ++e) {
        float v = b_l[e];
        if (v == -INFINITY) continue;
        if (before(pv, pi, v, e) && before(v, e, bv, bi)) {
          bv = v;
          bi = e;
        }
      }
      if (bi == INT_MAX) break;
      acc = acc + bv;
      ++taken;
      pv = bv;
      pi = bi;
    }
    gs_l[g] = taken ? acc : -INFINITY;
  }
  wave_sync();

  // group selection, computed redundantly by every lane (G <= 64)
  uint64_t gsel = 0;
  for (int r = 0; r < rp.TG; ++r) {
    float bv = 0.0f;
    int bi = -1;
    for (int g = 0; g < G; ++g) {
      if ((gsel >> g) & 1) continue;
      float v = gs_l[g];
      if (bi < 0 || before(v, g, bv, bi)) {
        bv = v;
        bi = g;
      }
    }
    gsel |= 1ull << bi;
  }

  // expert selection: k rounds of "best remaining" over the kept experts of
  // the chosen groups; round r finds the r-th element of the sorted order
  float pv = INFINITY, sum = 0.0f, my_s = 0.0f;
  int pi = -1, my_i = 0;
  for (int r = 0; r < rp.k; ++r) {
    float bv = -INFINITY;
    int bi = INT_MAX;
    for (int e = lane; e < E; e += 64) {
      if (!((gsel >> (e / per)) & 1)) continue;
      float v = b_l[e];
      if (v == -INFINITY) continue;
      if (before(pv, pi, v, e) && before(v, e, bv, bi)) {
        bv = v;
        bi = e;
      }
    }
    wave_argmax(bv, bi);
    // creation checks guarantee k candidates; never leave the index range
    if (bi == INT_MAX) bi = pi < 0 ? 0 : pi;
    const float sv = s_l[bi];
    sum = sum + sv;
    if (lane == r) {
      my_i = bi;
      my_s = sv;
    }
    pv = bv;
    pi = bi;
  }
  if (lane < rp.k) {
    float wv;
    if (rp.norm)
      wv = sum == 0.0f ? 0.0f : my_s / sum * rp.scale;
    else
      wv = my_s * rp.scale;
    idx_g[(size_t)t * rp.k + lane] = my_i;
    w_g[(size_t)t * rp.k + lane] = wv;
    if (idx_s) idx_s[t * rp.k + lane] = my_i;
  }
}

// Exclusive scan of cnt[0..E) by one wavefront into off[0..E] (off[E] = total),
// plus the ascending list of experts with cnt > 0 into active[1..], count in
// active[0].  Each lane owns a contiguous run of experts.
__device__ void wave_scan_experts(const int* cnt, int E, int32_t* off_lds, int32_t* off_g,
                                  int32_t* active_g) {
  const int lane = threadIdx.x & 63;
  const int epl = (E + 63) / 64;
  const int e0 = lane * epl, e1 = min(E, e0 + epl);
  int local = 0, nact = 0;
  for (int e = e0; e < e1; ++e) {
    local += cnt[e];
    nact += cnt[e] > 0;
  }
  int incl = local, iact = nact;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    int v = __shfl_up(incl, d, 64);
    int a = __shfl_up(iact, d, 64);
    if (lane >= d) {
      incl += v;
      iact += a;
    }
  }
  int run = incl - local, arun = iact - nact;
  for (int e = e0; e < e1; ++e) {
    if (off_lds) off_lds[e] = run;
    off_g[e] = run;
    if (cnt[e] > 0) active_g[1 + arun++] = e;
    run += cnt[e];
  }
  if (lane == 63) {
    off_g[E] = incl;
    if (off_lds) off_lds[E] = incl;
    active_g[0] = iact;
  }
}

// ---- small batches (n <= 64): route + bucket in one workgroup ----
__global__ __launch_bounds__(256) void route_bucket_small_kernel(RouterParams rp,
                                                                 const int32_t* idx_in, int n,
                                                                 Workspace ws) {
  __shared__ float s_l[kWaves][kMaxExperts];
  __shared__ float b_l[kWaves][kMaxExperts];
  __shared__ float gs_l[kWaves][64];
  __shared__ int32_t idx_l[kDecodeMaxTokens * kMaxTopK];
  __shared__ unsigned long long emask[kMaxExperts];
  __shared__ int32_t cnt[kMaxExperts];
  __shared__ int32_t off[kMaxExperts + 1];

  const int tid = threadIdx.x, wave = tid >> 6;
  const int E = rp.E, k = rp.k, nk = n * k;
  for (int e = tid; e < E; e += 256) emask[e] = 0ull;
  if (idx_in) {
    for (int a = tid; a < nk; a += 256) idx_l[a] = idx_in[a];
  } else {
    for (int t = wave; t < n; t += kWaves)
      route_token_wave(rp, t, s_l[wave], b_l[wave], gs_l[wave], ws.idx, ws.w, idx_l);
  }
  __syncthreads();
  // ids outside [0, E) (possible only for caller-provided ids) are ignored
  for (int a = tid; a < nk; a += 256)
    if ((unsigned)idx_l[a] < (unsigned)E) atomicOr(&emask[idx_l[a]], 1ull << (a / k));
  __syncthreads();
  for (int e = tid; e < E; e += 256) cnt[e] = __popcll(emask[e]);
  __syncthreads();
  if (wave == 0) wave_scan_experts(cnt, E, off, ws.offsets, ws.active);
  __syncthreads();
  for (int a = tid; a < nk; a += 256) {
    const int e = idx_l[a], t = a / k;
    if ((unsigned)e >= (unsigned)E) continue;
    const unsigned long long below = (t == 0) ? 0ull : (emask[e] & ((1ull << t) - 1ull));
    ws.perm[off[e] + __popcll(below)] = a;
  }
}

// ---- large batches: one token per wavefront ----
__global__ __launch_bounds__(256) void route_tokens_kernel(RouterParams rp, int n, int32_t* idx,
                                                           float* w) {
  __shared__ float s_l[kWaves][kMaxExperts];
  __shared__ float b_l[kWaves][kMaxExperts];
  __shared__ float gs_l[kWaves][64];
  const int wave = threadIdx.x >> 6;
  const int t = blockIdx.x * kWaves + wave;
  if (t < n) route_token_wave(rp, t, s_l[wave], b_l[wave], gs_l[wave], idx, w, nullptr);
}

// chunk c = tokens [64c, 64c+64): per-expert counts and in-chunk ranks
__global__ __launch_bounds__(256) void bucket_count_kernel(const int32_t* idx, int n, int k, int E,
                                                           int32_t* chunk_cnt, int32_t* rank) {
  __shared__ unsigned long long emask[kMaxExperts];
  const int c = blockIdx.x, tid = threadIdx.x;
  const int t0 = c * kChunk, t1 = min(n, t0 + kChunk);
  for (int e = tid; e < E; e += 256) emask[e] = 0ull;
  __syncthreads();
  for (int a = t0 * k + tid; a < t1 * k; a += 256)
    if ((unsigned)idx[a] < (unsigned)E) atomicOr(&emask[idx[a]], 1ull << (a / k - t0));
  __syncthreads();
  for (int e = tid; e < E; e += 256) chunk_cnt[(size_t)c * E + e] = __popcll(emask[e]);
  for (int a = t0 * k + tid; a < t1 * k; a += 256) {
    const int tl = a / k - t0, e = idx[a];
    if ((unsigned)e >= (unsigned)E) continue;
    const unsigned long long below = tl == 0 ? 0ull : (emask[e] & ((1ull << tl) - 1ull));
    rank[a] = __popcll(below);
  }
}

// one workgroup: per-expert scan over chunks, then over experts
__global__ __launch_bounds__(1024) void bucket_scan_kernel(int n_chunks, int E, int32_t* chunk_cnt,
                                                           int32_t* offsets, int32_t* active) {
  __shared__ int32_t total[kMaxExperts];
  __shared__ int32_t off[kMaxExperts + 1];
  const int tid = threadIdx.x;
  for (int e = tid; e < E; e += 1024) {
    int run = 0;
    for (int c = 0; c < n_chunks; ++c) {
      const int v = chunk_cnt[(size_t)c * E + e];
      chunk_cnt[(size_t)c * E + e] = run;
      run += v;
    }
    total[e] = run;
  }
  __syncthreads();
  if (tid < 64) wave_scan_experts(total, E, off, offsets, active);
  __syncthreads();
  for (int e = tid; e < E; e += 1024)
    for (int c = 0; c < n_chunks; ++c) chunk_cnt[(size_t)c * E + e] += off[e];
}

__global__ __launch_bounds__(256) void bucket_scatter_kernel(const int32_t* idx, int n, int k, int E,
                                                             const int32_t* chunk_cnt,
                                                             const int32_t* rank, int32_t* perm) {
  const int a = blockIdx.x * 256 + threadIdx.x;
  if (a >= n * k) return;
  const int c = (a / k) / kChunk, e = idx[a];
  if ((unsigned)e >= (unsigned)E) return;
  perm[chunk_cnt[(size_t)c * E + e] + rank[a]] = a;
}

}  // namespace

hipError_t launch_route_bucket_small(const RouterParams& rp, const int32_t* idx_in, int n,
                                     const Workspace& ws, hipStream_t s) {
  route_bucket_small_kernel<<<1, 256, 0, s>>>(rp, idx_in, n, ws);
  return hipGetLastError();
}

hipError_t launch_route_tokens(const RouterParams& rp, int n, int32_t* idx, float* w,
                               hipStream_t s) {
  route_tokens_kernel<<<(n + kWaves - 1) / kWaves, 256, 0, s>>>(rp, n, idx, w);
  return hipGetLastError();
}

hipError_t launch_bucket_chunked(const int32_t* idx, int n, int k, int E, const Workspace& ws,
                                 hipStream_t s) {
  const int chunks = (n + kChunk - 1) / kChunk;
  bucket_count_kernel<<<chunks, 256, 0, s>>>(idx, n, k, E, ws.chunk_cnt, ws.rank);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  bucket_scan_kernel<<<1, 1024, 0, s>>>(chunks, E, ws.chunk_cnt, ws.offsets, ws.active);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  bucket_scatter_kernel<<<(n * k + 255) / 256, 256, 0, s>>>(idx, n, k, E, ws.chunk_cnt, ws.rank,
                                                            ws.perm);
  return hipGetLastError();
}

}  // namespace moeq

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
#include "layout.h"
#include "route_wave.h"

namespace moeq {

namespace {

constexpr int kWaves = 4;        // tokens per workgroup of the many-token router

// Experts per lane for E experts (the kernels are instantiated per value).
int experts_per_lane(int E) { return E <= 64 ? 1 : E <= 128 ? 2 : E <= 256 ? 4 : E <= 512 ? 8 : 16; }

// Exclusive scan of cnt[0..E) by one wavefront into off[0..E] (off[E] = total),
// plus the ascending list of experts with cnt > 0 into active[1..], count in
// active[0].  Lane l owns experts [l*EPL, l*EPL + EPL), EPL*64 >= E.
template <int EPL>
__device__ void wave_scan_experts(const int* cnt, int E, int32_t* off_lds, int32_t* off_g,
                                  int32_t* active_g) {
  const int lane = threadIdx.x & 63;
  int c[EPL];
  int local = 0, nact = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane * EPL + i;
    c[i] = e < E ? cnt[e] : 0;
    local += c[i];
    nact += c[i] > 0;
  }
  const int incl = wave_incl_sum(local), iact = wave_incl_sum(nact);
  int run = incl - local, arun = iact - nact;
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane * EPL + i;
    if (e < E) {
      if (off_lds) off_lds[e] = run;
      off_g[e] = run;
      if (c[i] > 0) active_g[1 + arun++] = e;
      run += c[i];
    }
  }
  if (lane == 63) {
    off_g[E] = incl;
    if (off_lds) off_lds[E] = incl;
    active_g[0] = iact;
  }
}

// ---- small batches (n <= 64): route + bucket in one workgroup ----
// threads of the small-batch workgroup: fewer for wide lanes (register room)
template <int EPL>
constexpr int small_threads() { return EPL >= 8 ? 512 : 1024; }

template <int EPL>
__global__ __launch_bounds__(small_threads<EPL>()) void route_bucket_small_kernel(RouterParams rp,
                                                                  const int32_t* idx_in, int n,
                                                                  Workspace ws) {
  constexpr int NT = small_threads<EPL>(), NW = NT / 64;
  __shared__ float gs_l[NW][64];
  __shared__ int32_t idx_l[kDecodeMaxTokens * kMaxTopK];
  __shared__ unsigned long long emask[kMaxExperts];
  __shared__ int32_t cnt[kMaxExperts];
  __shared__ int32_t off[kMaxExperts + 1];

  const int tid = threadIdx.x, wave = tid >> 6;
  // buckets are over the original expert ids
  const int E = rp.E_row, k = rp.k, nk = n * k;
  for (int e = tid; e < E; e += NT) emask[e] = 0ull;
  if (idx_in) {
    for (int a = tid; a < nk; a += NT) idx_l[a] = idx_in[a];
  } else {
    for (int t = wave; t < n; t += NW) route_token_wave<EPL>(rp, t, gs_l[wave], ws.idx, ws.w, idx_l);
  }
  __syncthreads();
  // ids outside [0, E) (possible only for caller-provided ids) are ignored
  for (int a = tid; a < nk; a += NT)
    if ((unsigned)idx_l[a] < (unsigned)E) atomicOr(&emask[idx_l[a]], 1ull << (a / k));
  __syncthreads();
  for (int e = tid; e < E; e += NT) cnt[e] = __popcll(emask[e]);
  __syncthreads();
  if (wave == 0) wave_scan_experts<EPL>(cnt, E, off, ws.offsets, ws.active);
  __syncthreads();
  for (int a = tid; a < nk; a += NT) {
    const int e = idx_l[a], t = a / k;
    if ((unsigned)e >= (unsigned)E) continue;
    const unsigned long long below = (t == 0) ? 0ull : (emask[e] & ((1ull << t) - 1ull));
    ws.perm[off[e] + __popcll(below)] = a;
  }
}

// ---- one token: one wavefront routes it and writes the buckets directly ----
// Every chosen expert holds one assignment: offsets[e] is the number of
// chosen ids below e, the active list is the chosen ids in ascending order,
// and perm at an id's ascending rank is its slot.  The result equals the
// counting sort's.  Without kept_ids the lanes own the original ids, and the
// ranks come from each lane's choice bits and a prefix sum over the lanes.
template <int EPL>
__global__ __launch_bounds__(64) void route_bucket_one_kernel(RouterParams rp, Workspace ws) {
  __shared__ float gs_l[64];
  __shared__ int32_t ids[kMaxTopK];
  const LaneChoice<EPL> ch = route_token_wave<EPL>(rp, 0, gs_l, ws.idx, ws.w, ids);
  const int lane = threadIdx.x, k = rp.k, E = rp.E_row;
  if (!rp.kept_ids) {
    const int cnt = __popc(ch.bits);
    const int below = wave_incl_sum(cnt) - cnt;  // chosen ids of the lanes below
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = lane * EPL + i;
      const int r = below + __popc(ch.bits & ((1u << i) - 1u));
      if (e < E) ws.offsets[e] = r;
      if ((ch.bits >> i) & 1u) {
        ws.active[1 + r] = e;
        ws.perm[r] = ch.order[i];
      }
    }
    if (lane == 0) {
      ws.offsets[E] = k;
      ws.active[0] = k;
    }
    return;
  }
  wave_sync();
  if (lane < k) {
    const int mine = ids[lane];
    int r = 0;
    for (int j = 0; j < k; ++j) r += ids[j] < mine;
    ws.active[1 + r] = mine;
    ws.perm[r] = lane;
  }
  for (int e = lane; e <= E; e += 64) {
    int c = 0;
    for (int j = 0; j < k; ++j) c += ids[j] < e;
    ws.offsets[e] = c;
  }
  if (lane == 0) ws.active[0] = k;
}

// ---- large batches: one token per wavefront ----
template <int EPL>
__global__ __launch_bounds__(256) void route_tokens_kernel(RouterParams rp, int n, int32_t* idx,
                                                           float* w) {
  __shared__ float gs_l[kWaves][64];
  const int wave = threadIdx.x >> 6;
  const int t = blockIdx.x * kWaves + wave;
  if (t < n) route_token_wave<EPL>(rp, t, gs_l[wave], idx, w, nullptr);
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
template <int EPL>
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
  if (tid < 64) wave_scan_experts<EPL>(total, E, off, offsets, active);
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
  // lanes own enough experts for both the router's and the buckets' id range
  if (!idx_in && n == 1) {
    switch (experts_per_lane(rp.E_row)) {
      case 1: route_bucket_one_kernel<1><<<1, 64, 0, s>>>(rp, ws); break;
      case 2: route_bucket_one_kernel<2><<<1, 64, 0, s>>>(rp, ws); break;
      case 4: route_bucket_one_kernel<4><<<1, 64, 0, s>>>(rp, ws); break;
      case 8: route_bucket_one_kernel<8><<<1, 64, 0, s>>>(rp, ws); break;
      default: route_bucket_one_kernel<16><<<1, 64, 0, s>>>(rp, ws); break;
    }
    return hipGetLastError();
  }
  switch (experts_per_lane(rp.E_row)) {
    case 1: route_bucket_small_kernel<1><<<1, small_threads<1>(), 0, s>>>(rp, idx_in, n, ws); break;
    case 2: route_bucket_small_kernel<2><<<1, small_threads<2>(), 0, s>>>(rp, idx_in, n, ws); break;
    case 4: route_bucket_small_kernel<4><<<1, small_threads<4>(), 0, s>>>(rp, idx_in, n, ws); break;
    case 8: route_bucket_small_kernel<8><<<1, small_threads<8>(), 0, s>>>(rp, idx_in, n, ws); break;
    default: route_bucket_small_kernel<16><<<1, small_threads<16>(), 0, s>>>(rp, idx_in, n, ws); break;
  }
  return hipGetLastError();
}

hipError_t launch_route_tokens(const RouterParams& rp, int n, int32_t* idx, float* w,
                               hipStream_t s) {
  const int grid = (n + kWaves - 1) / kWaves;
  switch (experts_per_lane(rp.E_row)) {
    case 1: route_tokens_kernel<1><<<grid, 256, 0, s>>>(rp, n, idx, w); break;
    case 2: route_tokens_kernel<2><<<grid, 256, 0, s>>>(rp, n, idx, w); break;
    case 4: route_tokens_kernel<4><<<grid, 256, 0, s>>>(rp, n, idx, w); break;
    case 8: route_tokens_kernel<8><<<grid, 256, 0, s>>>(rp, n, idx, w); break;
    default: route_tokens_kernel<16><<<grid, 256, 0, s>>>(rp, n, idx, w); break;
  }
  return hipGetLastError();
}

hipError_t launch_bucket_chunked(const int32_t* idx, int n, int k, int E, const Workspace& ws,
                                 hipStream_t s) {
  const int chunks = (n + kChunk - 1) / kChunk;
  bucket_count_kernel<<<chunks, 256, 0, s>>>(idx, n, k, E, ws.chunk_cnt, ws.rank);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  switch (experts_per_lane(E)) {
    case 1: bucket_scan_kernel<1><<<1, 1024, 0, s>>>(chunks, E, ws.chunk_cnt, ws.offsets, ws.active); break;
    case 2: bucket_scan_kernel<2><<<1, 1024, 0, s>>>(chunks, E, ws.chunk_cnt, ws.offsets, ws.active); break;
    case 4: bucket_scan_kernel<4><<<1, 1024, 0, s>>>(chunks, E, ws.chunk_cnt, ws.offsets, ws.active); break;
    case 8: bucket_scan_kernel<8><<<1, 1024, 0, s>>>(chunks, E, ws.chunk_cnt, ws.offsets, ws.active); break;
    default: bucket_scan_kernel<16><<<1, 1024, 0, s>>>(chunks, E, ws.chunk_cnt, ws.offsets, ws.active); break;
  }
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  bucket_scatter_kernel<<<(n * k + 255) / 256, 256, 0, s>>>(idx, n, k, E, ws.chunk_cnt, ws.rank,
                                                            ws.perm);
  return hipGetLastError();
}

}  // namespace moeq

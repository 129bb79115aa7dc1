// Host runtime of the C interface declared in include/moeq.h: validation,
// the device weight store, the workspace and the per-forward dispatch.
//
// Every argument check runs before the first HIP runtime call of an entry
// point, so validation behaves identically without a GPU.  Device memory is
// owned by the layer and released by moeq_destroy (or on a failed create).
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"

// decode forwards of at least MOEQ_HYBRID_FROM tokens send the buckets of
// more than MOEQ_HYBRID_ABOVE rows to the grouped GEMMs
#ifndef MOEQ_HYBRID_FROM
#define MOEQ_HYBRID_FROM 24
#endif
#ifndef MOEQ_HYBRID_ABOVE
#define MOEQ_HYBRID_ABOVE 2
#endif

using namespace moeq;

namespace {
thread_local std::string g_last_error;

// One auxiliary stream per device (default priority, non-blocking), shared by
// every layer on that device and created on first use.  A forward forks part
// of its work onto it and joins it back with the layer's own two events, so
// layers never wait on each other's auxiliary work except by sharing this
// queue.
constexpr int kMaxDevices = 64;
std::mutex g_aux_mu;
hipStream_t g_aux[kMaxDevices] = {};

hipError_t aux_stream(int dev, hipStream_t* out) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_aux_mu);
  if (!g_aux[dev]) {
    const hipError_t e = hipStreamCreateWithFlags(&g_aux[dev], hipStreamNonBlocking);
    if (e != hipSuccess) return e;
  }
  *out = g_aux[dev];
  return hipSuccess;
}
}  // namespace

moeq_status moeq::vset_error(moeq_status st, const char* fmt, va_list ap) {
  char buf[512];
  vsnprintf(buf, sizeof buf, fmt, ap);
  g_last_error = buf;
  return st;
}

namespace {

moeq_status fail(moeq_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vset_error(st, fmt, ap);
  va_end(ap);
  return st;
}

moeq_status ok() { return MOEQ_OK; }

moeq_status hip_fail(hipError_t e, const char* what) {
  return fail(e == hipErrorOutOfMemory ? MOEQ_ERR_OUT_OF_MEMORY : MOEQ_ERR_DEVICE, "%s: %s", what,
              hipGetErrorString(e));
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

struct TensorPlan {
  size_t codes_off, scales_off;
  int rows, K, bits;
};

}  // namespace

struct moeq_layer {
  moeq_config cfg{};
  int device = 0;
  int path = MOEQ_PATH_AUTO;
  int decode_max = kDefaultDecodeMax;
  int n_kept = 0;
  uint64_t weight_bytes = 0;   // codes + scales as stored
  uint64_t ws_bytes = 0;
  std::vector<TensorDev> desc_host;  // [(E + S) * 3]
  void* store = nullptr;
  TensorDev* desc = nullptr;
  uint8_t* mask = nullptr;
  float* bias = nullptr;
  int wide_gateup = 0, wide_down = 0;  // 0: no 5/6/8-bit tensor, 1: shared experts only, 2: routed too
  int lds_gateup = 0, lds_down = 0;    // some gate/up (down) tensor takes the LDS-decoded GEMM
  int down_bits = 0;                   // width of every kept and shared down tensor when they agree
  int32_t* kept_ids = nullptr;  // kept experts ascending, when the router regroups them
  float* router_w = nullptr;    // float32 [n_experts x hidden] gate weight, when set
  float* gate_logits = nullptr; // float32 [max_tokens x n_experts], logits the forward computes
  void* ws_mem = nullptr;
  Workspace ws{};
  hipEvent_t stage_events[MOEQ_STAGE_EVENTS] = {};
  // the device's auxiliary stream (shared, not owned) and two events: for
  // 2-64 tokens the gate/up GEMVs of one-token buckets and of larger buckets
  // run side by side
  hipStream_t aux = nullptr;
  hipEvent_t fork_ev = nullptr, join_ev = nullptr;
  bool timing = false;
};

namespace {

void release(moeq_layer* L) {
  if (!L) return;
  if (L->fork_ev) hipEventDestroy(L->fork_ev);
  if (L->join_ev) hipEventDestroy(L->join_ev);
  hipFree(L->store);
  hipFree(L->desc);
  hipFree(L->mask);
  hipFree(L->bias);
  hipFree(L->kept_ids);
  hipFree(L->router_w);
  hipFree(L->gate_logits);
  hipFree(L->ws_mem);
  delete L;
}

moeq_status check_config(const moeq_config* c) {
  if (!c) return fail(MOEQ_ERR_INVALID_ARG, "cfg is NULL");
  if (c->hidden <= 0 || c->inter <= 0 || c->hidden % kBlock || c->inter % kBlock)
    return fail(MOEQ_ERR_INVALID_ARG, "hidden (%d) and inter (%d) must be positive multiples of 32",
                c->hidden, c->inter);
  if (c->hidden % kUnit || c->inter % kUnit)
    return fail(MOEQ_ERR_UNSUPPORTED, "hidden (%d) and inter (%d) must be multiples of 128",
                c->hidden, c->inter);
  if (c->hidden > 8192 || c->inter > 8192)
    return fail(MOEQ_ERR_UNSUPPORTED, "hidden and inter are limited to 8192 (got %d, %d)", c->hidden,
                c->inter);
  if (c->n_experts < 1 || c->n_experts > kMaxExperts)
    return fail(MOEQ_ERR_INVALID_ARG, "n_experts %d outside 1..%d", c->n_experts, kMaxExperts);
  if (c->n_group < 1 || c->n_group > 64 || c->n_experts % c->n_group)
    return fail(MOEQ_ERR_INVALID_ARG, "n_group %d must be 1..64 and divide n_experts %d", c->n_group,
                c->n_experts);
  if (c->topk_group < 1 || c->topk_group > c->n_group)
    return fail(MOEQ_ERR_INVALID_ARG, "topk_group %d outside 1..n_group", c->topk_group);
  if (c->top_k < 1 || c->top_k > kMaxTopK || c->top_k > c->n_experts)
    return fail(MOEQ_ERR_INVALID_ARG, "top_k %d outside 1..%d", c->top_k, kMaxTopK);
  if (c->group_topn < 1 || c->group_topn > c->n_experts / c->n_group)
    return fail(MOEQ_ERR_INVALID_ARG, "group_topn %d outside 1..experts per group", c->group_topn);
  if (c->norm_topk != 0 && c->norm_topk != 1)
    return fail(MOEQ_ERR_INVALID_ARG, "norm_topk must be 0 or 1");
  if (!isfinite(c->routed_scale))
    return fail(MOEQ_ERR_INVALID_ARG, "routed_scale must be finite");
  if (c->n_shared < 0 || c->n_shared > kMaxShared)
    return fail(MOEQ_ERR_INVALID_ARG, "n_shared %d outside 0..%d", c->n_shared, kMaxShared);
  if (c->max_tokens < 1 || c->max_tokens > (1 << 20))
    return fail(MOEQ_ERR_INVALID_ARG, "max_tokens %d outside 1..2^20", c->max_tokens);
  if (c->regroup != 0 && c->regroup != 1) return fail(MOEQ_ERR_INVALID_ARG, "regroup must be 0 or 1");
  if (c->decode_max_tokens < 0 || c->decode_max_tokens > kDecodeMaxTokens)
    return fail(MOEQ_ERR_INVALID_ARG, "decode_max_tokens %d outside 0..%d", c->decode_max_tokens,
                kDecodeMaxTokens);
  return ok();
}

bool valid_bits(int b) { return (b >= 2 && b <= 6) || b == 8; }

moeq_status check_tensor(const moeq_qtensor& t, const char* who, int e, int p) {
  if (!valid_bits(t.bits))
    return fail(MOEQ_ERR_INVALID_ARG, "%s %d proj %d: bits %d not in {2,3,4,5,6,8}", who, e, p, t.bits);
  if (!t.codes || !t.scales) return fail(MOEQ_ERR_INVALID_ARG, "%s %d proj %d: NULL codes or scales", who, e, p);
  return ok();
}

// Worst case of the grouped selection: the topk_group non-empty groups with
// the fewest kept experts must still hold top_k of them.
moeq_status check_routing(const moeq_config* c, const uint8_t* mask, int* n_kept) {
  const int per = c->n_experts / c->n_group;
  std::vector<int> counts;
  int kept = 0;
  for (int g = 0; g < c->n_group; ++g) {
    int n = 0;
    for (int e = g * per; e < (g + 1) * per; ++e) n += mask[e] != 0;
    kept += n;
    if (n > 0) counts.push_back(n);
  }
  *n_kept = kept;
  if (c->regroup) {
    // the kept experts form n_group equal groups of their own
    if (kept % c->n_group)
      return fail(MOEQ_ERR_INVALID_ARG, "regroup needs the kept count (%d) to be a multiple of n_group %d", kept,
                  c->n_group);
    if (c->group_topn > kept / c->n_group)
      return fail(MOEQ_ERR_INVALID_ARG, "group_topn %d exceeds the %d experts of a regrouped group", c->group_topn,
                  kept / c->n_group);
    if (c->topk_group * (kept / c->n_group) < c->top_k)
      return fail(MOEQ_ERR_INVALID_ARG, "topk_group regrouped groups of %d experts hold fewer than top_k %d",
                  kept / c->n_group, c->top_k);
    return ok();
  }
  if ((int)counts.size() < c->topk_group)
    return fail(MOEQ_ERR_INVALID_ARG, "only %d groups have kept experts; topk_group is %d",
                (int)counts.size(), c->topk_group);
  std::sort(counts.begin(), counts.end());
  int worst = 0;
  for (int i = 0; i < c->topk_group; ++i) worst += counts[i];
  if (worst < c->top_k)
    return fail(MOEQ_ERR_INVALID_ARG,
                "the %d smallest non-empty groups hold %d kept experts, fewer than top_k %d",
                c->topk_group, worst, c->top_k);
  return ok();
}

RouterParams router_params(const moeq_layer* L, const float* logits, const void* x = nullptr) {
  RouterParams rp;
  rp.x = (const uint16_t*)x;
  rp.H = L->cfg.hidden;
  rp.xexp = L->ws.xexp;
  rp.x16 = L->ws.x16;
  rp.logits = logits;
  rp.mask = L->mask;
  rp.kept_ids = L->kept_ids;
  rp.E_row = L->cfg.n_experts;
  rp.bias = L->bias;
  rp.E = L->kept_ids ? L->n_kept : L->cfg.n_experts;
  rp.G = L->cfg.n_group;
  rp.TG = L->cfg.topk_group;
  rp.k = L->cfg.top_k;
  rp.topn = L->cfg.group_topn;
  rp.norm = L->cfg.norm_topk;
  rp.scale = L->cfg.routed_scale;
  return rp;
}

moeq_status check_device(const moeq_layer* L) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != L->device)
    return fail(MOEQ_ERR_INVALID_ARG, "layer lives on device %d but device %d is current", L->device, dev);
  return ok();
}

// Route (+ bucket) n tokens into the workspace: the first stage of a forward.
// With x given, the router also records each token's binary16 prescale.
hipError_t route_and_bucket(moeq_layer* L, const float* logits, int n, hipStream_t s,
                            const void* x = nullptr) {
  const RouterParams rp = router_params(L, logits, x);
  if (n <= kDecodeMaxTokens) return launch_route_bucket_small(rp, nullptr, n, L->ws, s);
  hipError_t e = launch_route_tokens(rp, n, L->ws.idx, L->ws.w, s);
  if (e != hipSuccess) return e;
  return launch_bucket_chunked(L->ws.idx, n, L->cfg.top_k, L->cfg.n_experts, L->ws, s);
}

}  // namespace

extern "C" {

const char* moeq_last_error(void) { return g_last_error.c_str(); }

moeq_status moeq_layer_create(const moeq_config* cfg, const uint8_t* expert_mask,
                              const float* score_bias, const moeq_qtensor* routed,
                              const moeq_qtensor* shared, int32_t weights_location,
                              moeq_layer** out) {
  if (!out) return fail(MOEQ_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  moeq_status st = check_config(cfg);
  if (st != MOEQ_OK) return st;
  if (!expert_mask) return fail(MOEQ_ERR_INVALID_ARG, "expert_mask is NULL");
  if (weights_location != MOEQ_WEIGHTS_HOST && weights_location != MOEQ_WEIGHTS_DEVICE)
    return fail(MOEQ_ERR_INVALID_ARG, "weights_location %d is neither HOST nor DEVICE", weights_location);
  const int E = cfg->n_experts, S = cfg->n_shared, H = cfg->hidden, I = cfg->inter;
  int n_kept = 0;
  st = check_routing(cfg, expert_mask, &n_kept);
  if (st != MOEQ_OK) return st;
  if (score_bias)
    for (int e = 0; e < E; ++e)
      if (!isfinite(score_bias[e]) || fabsf(score_bias[e]) > 1e30f)
        return fail(MOEQ_ERR_INVALID_ARG, "score_bias[%d] is not a finite value of magnitude <= 1e30", e);
  if (!routed) return fail(MOEQ_ERR_INVALID_ARG, "routed is NULL");
  if (S > 0 && !shared) return fail(MOEQ_ERR_INVALID_ARG, "shared is NULL but n_shared = %d", S);
  for (int e = 0; e < E; ++e)
    if (expert_mask[e])
      for (int p = 0; p < 3; ++p)
        if ((st = check_tensor(routed[e * 3 + p], "expert", e, p)) != MOEQ_OK) return st;
  for (int s = 0; s < S; ++s)
    for (int p = 0; p < 3; ++p)
      if ((st = check_tensor(shared[s * 3 + p], "shared expert", s, p)) != MOEQ_OK) return st;

  // ---- plan the weight store: one allocation, 256-byte aligned tensors ----
  std::vector<TensorPlan> plan((size_t)(E + S) * 3);
  size_t off = 0, max_codes = 0;
  uint64_t wbytes = 0;
  auto plan_tensor = [&](int slot, int p, const moeq_qtensor& t) {
    TensorPlan& tp = plan[(size_t)slot * 3 + p];
    tp.rows = p == MOEQ_PROJ_DOWN ? H : I;
    tp.K = p == MOEQ_PROJ_DOWN ? I : H;
    tp.bits = t.bits;
    const size_t cb = (size_t)tp.rows * tp.K * t.bits / 8, sb = (size_t)tp.rows * (tp.K / kBlock) * 2;
    tp.codes_off = off;
    off = align_up(off + cb, 256);
    tp.scales_off = off;
    off = align_up(off + sb, 256);
    max_codes = cb > max_codes ? cb : max_codes;
    wbytes += cb + sb;
  };
  for (int e = 0; e < E; ++e)
    if (expert_mask[e])
      for (int p = 0; p < 3; ++p) plan_tensor(e, p, routed[e * 3 + p]);
  for (int s = 0; s < S; ++s)
    for (int p = 0; p < 3; ++p) plan_tensor(E + s, p, shared[s * 3 + p]);

  // ---- workspace sizes ----
  const int T = cfg->max_tokens, k = cfg->top_k;
  const size_t nk = (size_t)T * k, rows_h = nk + (size_t)T * S;
  const size_t chunks = (T + kChunk - 1) / kChunk;
  size_t wo = 0;
  auto ws_take = [&](size_t bytes) {
    const size_t at = wo;
    wo = align_up(wo + bytes, 256);
    return at;
  };
  const int max_mtiles = prefill_max_mtiles(T, k, S, n_kept), max_rtiles = prefill_max_rtiles(T, k, S, n_kept);
  const size_t o_idx = ws_take(nk * 4), o_w = ws_take(nk * 4), o_off = ws_take((size_t)(E + 1) * 4),
               o_perm = ws_take(nk * 4), o_act = ws_take((size_t)(E + 1) * 4),
               o_cc = ws_take(chunks * E * 4), o_rank = ws_take(nk * 4),
               o_h = ws_take(rows_h * I * 4), o_part = ws_take(rows_h * H * 4),
               o_xexp = ws_take((size_t)T * 4), o_rmax = ws_take(rows_h * 4),
               o_tiles = ws_take((size_t)(1 + 2 * max_mtiles) * 4), o_rtiles = ws_take((size_t)(1 + 2 * max_rtiles) * 4),
               o_x16 = ws_take((size_t)T * H * 2), o_h16 = ws_take(rows_h * I * 2), o_zero = ws_take(256);

  // ---- device work ----
  moeq_layer* L = new moeq_layer();
  L->cfg = *cfg;
  L->n_kept = n_kept;
  L->decode_max = cfg->decode_max_tokens ? cfg->decode_max_tokens : kDefaultDecodeMax;
  L->weight_bytes = wbytes;
  L->ws_bytes = wo;
  auto wide = [](const moeq_qtensor& t) { return t.bits > 4; };
  for (int s = 0; s < S; ++s) {
    if (wide(shared[s * 3 + 0]) || wide(shared[s * 3 + 1])) L->wide_gateup = 1;
    if (wide(shared[s * 3 + 2])) L->wide_down = 1;
  }
  int db = -1;
  auto agree = [&db](int b) { db = db == -1 || db == b ? b : 0; };
  for (int s = 0; s < S; ++s) agree(shared[s * 3 + 2].bits);
  for (int e = 0; e < E; ++e)
    if (expert_mask[e]) {
      if (wide(routed[e * 3 + 0]) || wide(routed[e * 3 + 1])) L->wide_gateup = 2;
      if (wide(routed[e * 3 + 2])) L->wide_down = 2;
      agree(routed[e * 3 + 2].bits);
    }
  L->down_bits = db > 0 ? db : 0;
  hipError_t he = hipGetDevice(&L->device);
  if (he != hipSuccess) {
    release(L);
    return hip_fail(he, "hipGetDevice");
  }
  uint8_t* staging = nullptr;
  uint32_t* scale_keys = nullptr;  // per descriptor: the largest scale key (launch_scale_key_max)
  auto bail = [&](hipError_t e, const char* what) {
    hipStreamSynchronize(nullptr);
    hipFree(staging);
    hipFree(scale_keys);
    release(L);
    return hip_fail(e, what);
  };
  if ((he = hipMalloc(&L->store, off ? off : 256)) != hipSuccess) return bail(he, "hipMalloc(weights)");
  if ((he = hipMalloc(&L->ws_mem, wo)) != hipSuccess) return bail(he, "hipMalloc(workspace)");
  if ((he = hipMalloc((void**)&L->desc, sizeof(TensorDev) * plan.size())) != hipSuccess)
    return bail(he, "hipMalloc(descriptors)");
  if ((he = hipMalloc((void**)&L->mask, E)) != hipSuccess) return bail(he, "hipMalloc(mask)");
  if (cfg->regroup) {
    std::vector<int32_t> ids;
    for (int e = 0; e < E; ++e)
      if (expert_mask[e]) ids.push_back(e);
    if ((he = hipMalloc((void**)&L->kept_ids, ids.size() * 4)) != hipSuccess) return bail(he, "hipMalloc(kept ids)");
    if ((he = hipMemcpy(L->kept_ids, ids.data(), ids.size() * 4, hipMemcpyHostToDevice)) != hipSuccess)
      return bail(he, "hipMemcpy(kept ids)");
  }
  if ((he = hipMalloc((void**)&L->bias, sizeof(float) * E)) != hipSuccess) return bail(he, "hipMalloc(bias)");
  if (weights_location == MOEQ_WEIGHTS_HOST && max_codes &&
      (he = hipMalloc((void**)&staging, max_codes)) != hipSuccess)
    return bail(he, "hipMalloc(staging)");
  if ((he = hipMalloc((void**)&scale_keys, sizeof(uint32_t) * plan.size())) != hipSuccess ||
      (he = hipMemset(scale_keys, 0, sizeof(uint32_t) * plan.size())) != hipSuccess)
    return bail(he, "scale keys");

  uint8_t* base = (uint8_t*)L->store;
  L->desc_host.assign(plan.size(), TensorDev{nullptr, nullptr, 0, 0, 0, 0});
  auto upload = [&](int slot, int p, const moeq_qtensor& t) -> hipError_t {
    const TensorPlan& tp = plan[(size_t)slot * 3 + p];
    const size_t cb = (size_t)tp.rows * tp.K * tp.bits / 8, sb = (size_t)tp.rows * (tp.K / kBlock) * 2;
    const uint8_t* src = (const uint8_t*)t.codes;
    hipError_t e;
    if (weights_location == MOEQ_WEIGHTS_HOST) {
      // staging is reused: the null-stream copy waits for the previous repack
      if ((e = hipMemcpy(staging, src, cb, hipMemcpyHostToDevice)) != hipSuccess) return e;
      src = staging;
    }
    if ((e = launch_repack(src, tp.rows, tp.K, tp.bits, (uint32_t*)(base + tp.codes_off), 0)) != hipSuccess)
      return e;
    if ((e = hipMemcpy(base + tp.scales_off, t.scales, sb,
                       weights_location == MOEQ_WEIGHTS_HOST ? hipMemcpyHostToDevice
                                                             : hipMemcpyDeviceToDevice)) != hipSuccess)
      return e;
    if ((e = launch_scale_key_max((const uint16_t*)(base + tp.scales_off), sb / 2,
                                  scale_keys + (size_t)slot * 3 + p, 0)) != hipSuccess)
      return e;
    TensorDev& d = L->desc_host[(size_t)slot * 3 + p];
    d.codes = (const uint32_t*)(base + tp.codes_off);
    d.scales = (const uint16_t*)(base + tp.scales_off);
    d.bits = tp.bits;
    d.rows = tp.rows;
    d.K = tp.K;
    return hipSuccess;
  };
  for (int e = 0; e < E; ++e)
    if (expert_mask[e])
      for (int p = 0; p < 3; ++p)
        if ((he = upload(e, p, routed[e * 3 + p])) != hipSuccess) return bail(he, "weight upload");
  for (int s = 0; s < S; ++s)
    for (int p = 0; p < 3; ++p)
      if ((he = upload(E + s, p, shared[s * 3 + p])) != hipSuccess) return bail(he, "weight upload");

  // tensors the grouped GEMMs' register decoder cannot take (wider than 4
  // bits, a scale outside (0, rd_scale_limit(bits)], or rows of an odd number
  // of 128-weight units)
  {
    std::vector<uint32_t> keys(plan.size());
    if ((he = hipMemcpy(keys.data(), scale_keys, sizeof(uint32_t) * plan.size(), hipMemcpyDeviceToHost)) !=
        hipSuccess)
      return bail(he, "scale keys");
    for (size_t i = 0; i < plan.size(); ++i) {
      TensorDev& d = L->desc_host[i];
      if (!d.codes) continue;
      if (d.bits <= 4 && (keys[i] > rd_scale_limit(d.bits) || (d.K / kUnit) % 2 != 0))
        d.flags |= kTensorOffRegisterDecoder;
      if (d.bits > 4 || (d.flags & kTensorOffRegisterDecoder)) {
        if (i % 3 == 2)
          L->lds_down = 1;
        else
          L->lds_gateup = 1;
      }
    }
  }
  std::vector<float> bias_h(E, 0.0f);
  if (score_bias) memcpy(bias_h.data(), score_bias, sizeof(float) * E);
  if ((he = hipMemcpy(L->desc, L->desc_host.data(), sizeof(TensorDev) * plan.size(),
                      hipMemcpyHostToDevice)) != hipSuccess ||
      (he = hipMemcpy(L->mask, expert_mask, E, hipMemcpyHostToDevice)) != hipSuccess ||
      (he = hipMemcpy(L->bias, bias_h.data(), sizeof(float) * E, hipMemcpyHostToDevice)) != hipSuccess)
    return bail(he, "hipMemcpy(tables)");
  // every copy and repack kernel above ran on the null stream
  if ((he = hipStreamSynchronize(nullptr)) != hipSuccess) return bail(he, "create");
  hipFree(staging);
  staging = nullptr;
  hipFree(scale_keys);
  scale_keys = nullptr;

  uint8_t* w = (uint8_t*)L->ws_mem;
  L->ws.idx = (int32_t*)(w + o_idx);
  L->ws.w = (float*)(w + o_w);
  L->ws.offsets = (int32_t*)(w + o_off);
  L->ws.perm = (int32_t*)(w + o_perm);
  L->ws.active = (int32_t*)(w + o_act);
  L->ws.chunk_cnt = (int32_t*)(w + o_cc);
  L->ws.rank = (int32_t*)(w + o_rank);
  L->ws.h = (float*)(w + o_h);
  L->ws.partial = (float*)(w + o_part);
  L->ws.xexp = (int32_t*)(w + o_xexp);
  L->ws.rowmax = (uint32_t*)(w + o_rmax);
  L->ws.tiles_all = (int32_t*)(w + o_tiles);
  L->ws.tiles_rd = (int32_t*)(w + o_rtiles);
  L->ws.x16 = (uint16_t*)(w + o_x16);
  L->ws.h16 = (uint16_t*)(w + o_h16);
  L->ws.zeros = (uint32_t*)(w + o_zero);
  if ((he = hipMemset(L->ws.zeros, 0, 256)) != hipSuccess || (he = hipStreamSynchronize(nullptr)) != hipSuccess)
    return bail(he, "hipMemset(zeros)");
  if ((he = aux_stream(L->device, &L->aux)) != hipSuccess) return bail(he, "hipStreamCreate (auxiliary)");
  if ((he = hipEventCreateWithFlags(&L->fork_ev, hipEventDisableTiming)) != hipSuccess ||
      (he = hipEventCreateWithFlags(&L->join_ev, hipEventDisableTiming)) != hipSuccess)
    return bail(he, "hipEventCreate");
  *out = L;
  return ok();
}

void moeq_destroy(moeq_layer* L) {
  if (!L) return;
  // the handle does not know every stream its forwards ran on (nor does
  // hipFree wait for them by itself on every runtime), so the whole device
  // is drained before its memory is released
  hipDeviceSynchronize();
  release(L);
}

moeq_status moeq_set_path(moeq_layer* L, int32_t path) {
  if (!L) return fail(MOEQ_ERR_INVALID_ARG, "layer is NULL");
  if (path != MOEQ_PATH_AUTO && path != MOEQ_PATH_DECODE && path != MOEQ_PATH_PREFILL)
    return fail(MOEQ_ERR_INVALID_ARG, "path %d is not AUTO, DECODE or PREFILL", path);
  L->path = path;
  return ok();
}

moeq_status moeq_layer_bytes(const moeq_layer* L, uint64_t* weight_bytes, uint64_t* workspace_bytes) {
  if (!L) return fail(MOEQ_ERR_INVALID_ARG, "layer is NULL");
  if (weight_bytes) *weight_bytes = L->weight_bytes;
  if (workspace_bytes) *workspace_bytes = L->ws_bytes;
  return ok();
}

moeq_status moeq_forward(moeq_layer* L, const void* x, const float* logits, int32_t n, float* y,
                         void* stream) {
  if (!L) return fail(MOEQ_ERR_INVALID_ARG, "layer is NULL");
  if (n < 0) return fail(MOEQ_ERR_INVALID_ARG, "n_tokens %d is negative", n);
  if (n > L->cfg.max_tokens)
    return fail(MOEQ_ERR_CAPACITY, "n_tokens %d exceeds max_tokens %d", n, L->cfg.max_tokens);
  if (n == 0) return ok();
  if (!x || !y) return fail(MOEQ_ERR_INVALID_ARG, "x and y must not be NULL");
  if (!logits && !L->router_w)
    return fail(MOEQ_ERR_INVALID_ARG, "logits is NULL and no router weight is set");
  if (!aligned16(x) || !aligned16(y) || (logits && !aligned16(logits)))
    return fail(MOEQ_ERR_INVALID_ARG, "x, logits and y must be 16-byte aligned");
  moeq_status st = check_device(L);
  if (st != MOEQ_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  DecodeArgs a;
  a.desc = L->desc;
  a.x = (const uint16_t*)x;
  a.active = L->ws.active;
  a.offsets = L->ws.offsets;
  a.perm = L->ws.perm;
  a.w = L->ws.w;
  a.h = L->ws.h;
  a.partial = L->ws.partial;
  a.y = y;
  a.n = n;
  a.H = L->cfg.hidden;
  a.I = L->cfg.inter;
  a.E = L->cfg.n_experts;
  a.S = L->cfg.n_shared;
  a.k = L->cfg.top_k;
  const long long nk = (long long)n * a.k;
  a.max_active = (int)(nk < L->n_kept ? nk : L->n_kept);
  a.xexp = L->ws.xexp;
  a.rowmax = L->ws.rowmax;
  a.max_mtiles = prefill_max_mtiles(n, a.k, a.S, L->n_kept);
  a.tiles_all = L->ws.tiles_all;
  a.max_rtiles = prefill_max_rtiles(n, a.k, a.S, L->n_kept);
  a.tiles_rd = L->ws.tiles_rd;
  a.x16 = L->ws.x16;
  a.h16 = L->ws.h16;
  a.zeros = L->ws.zeros;
  a.wide_gateup = L->wide_gateup;
  a.wide_down = L->wide_down;
  a.lds_gateup = L->lds_gateup;
  a.lds_down = L->lds_down;
  a.idx = L->ws.idx;
  a.down_bits = L->down_bits;
  const bool prefill =
      L->path == MOEQ_PATH_PREFILL || (L->path == MOEQ_PATH_AUTO && n > L->decode_max);
  // decode forwards of several tokens: the buckets of more than
  // MOEQ_HYBRID_ABOVE rows (the large buckets of a skewed routing) take the
  // grouped GEMMs, which read an expert's weights once for all its tokens
  const bool hybrid = !prefill && n >= MOEQ_HYBRID_FROM;
  a.gemm_above = prefill ? 0 : hybrid ? MOEQ_HYBRID_ABOVE : kDecodeMaxTokens;
  hipError_t e = hipSuccess;
  auto mark = [&](int i) {
    if (L->timing && e == hipSuccess) e = hipEventRecord(L->stage_events[i], s);
  };
  mark(0);
  if (!logits) {
    if (e == hipSuccess)
      e = launch_router_gate(a.x, L->router_w, n, a.H, a.E, L->gate_logits, s);
    logits = L->gate_logits;
  }
  // one token: the gate/up workgroups route the token themselves
  const RouterParams rp1 = router_params(L, logits);
  const bool self_routed = !prefill && n == 1 && gateup1_routes(rp1);
  if (e == hipSuccess && !self_routed) e = route_and_bucket(L, logits, n, s, prefill || hybrid ? x : nullptr);
  mark(1);
  if (e == hipSuccess) {
    if (prefill) {
      e = launch_prefill_tiles(a, s);
      if (e == hipSuccess) e = launch_gateup_prefill(a, s);
    } else if (n > 1) {
      if (hybrid) e = launch_prefill_tiles(a, s);
      // fork: the buckets of 2-64 tokens on the layer's second stream, then join
      if (e == hipSuccess) e = hipEventRecord(L->fork_ev, s);
      if (e == hipSuccess) e = hipStreamWaitEvent(L->aux, L->fork_ev, 0);
      if (e == hipSuccess) e = launch_gateup_decode_multi(a, L->aux);
      if (e == hipSuccess) e = hipEventRecord(L->join_ev, L->aux);
      if (e == hipSuccess) e = launch_gateup_decode_single(a, s);
      if (e == hipSuccess && hybrid) e = launch_gateup_prefill(a, s);
      if (e == hipSuccess) e = hipStreamWaitEvent(s, L->join_ev, 0);
    } else if (self_routed) {
      e = launch_gateup_decode_routing(a, rp1, L->ws, s);
    } else {
      e = launch_gateup_decode(a, s);
    }
  }
  mark(2);
  if (e == hipSuccess) e = prefill ? launch_down_prefill(a, s) : launch_down_decode(a, s);
  if (e == hipSuccess && hybrid) e = launch_down_prefill(a, s);
  mark(3);
  if (e == hipSuccess && (prefill || !down_combines(a))) e = launch_combine(a, s);
  mark(4);
  if (e != hipSuccess) return hip_fail(e, prefill ? "forward (prefill path)" : "forward (decode path)");
  return ok();
}

moeq_status moeq_set_router_weight(moeq_layer* L, const float* w, int32_t location) {
  if (!L) return fail(MOEQ_ERR_INVALID_ARG, "layer is NULL");
  if (location != MOEQ_WEIGHTS_HOST && location != MOEQ_WEIGHTS_DEVICE)
    return fail(MOEQ_ERR_INVALID_ARG, "location %d is neither HOST nor DEVICE", location);
  const int E = L->cfg.n_experts, H = L->cfg.hidden;
  const size_t wb = (size_t)E * H * 4;
  if (w && location == MOEQ_WEIGHTS_HOST)
    for (size_t i = 0; i < (size_t)E * H; ++i)
      if (!isfinite(w[i])) return fail(MOEQ_ERR_INVALID_ARG, "router weight element %zu is not finite", i);
  moeq_status st = check_device(L);
  if (st != MOEQ_OK) return st;
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "set_router_weight");
  if (!w) {
    hipFree(L->router_w);
    hipFree(L->gate_logits);
    L->router_w = nullptr;
    L->gate_logits = nullptr;
    return ok();
  }
  if (!L->router_w) {
    float *rw = nullptr, *lg = nullptr;
    if ((e = hipMalloc((void**)&rw, wb)) != hipSuccess) return hip_fail(e, "hipMalloc(router weight)");
    if ((e = hipMalloc((void**)&lg, (size_t)L->cfg.max_tokens * E * 4)) != hipSuccess) {
      hipFree(rw);
      return hip_fail(e, "hipMalloc(router logits)");
    }
    L->router_w = rw;
    L->gate_logits = lg;
  }
  e = hipMemcpy(L->router_w, w, wb, location == MOEQ_WEIGHTS_HOST ? hipMemcpyHostToDevice : hipMemcpyDeviceToDevice);
  if (e != hipSuccess || (e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(e, "hipMemcpy(router weight)");
  return ok();
}

moeq_status moeq_router_logits(moeq_layer* L, const void* x, int32_t n, float* logits, void* stream) {
  if (!L) return fail(MOEQ_ERR_INVALID_ARG, "layer is NULL");
  if (n < 0 || n > L->cfg.max_tokens)
    return fail(n < 0 ? MOEQ_ERR_INVALID_ARG : MOEQ_ERR_CAPACITY, "n_tokens %d outside 0..max_tokens", n);
  if (n == 0) return ok();
  if (!x || !logits) return fail(MOEQ_ERR_INVALID_ARG, "x and logits must not be NULL");
  if (!aligned16(x)) return fail(MOEQ_ERR_INVALID_ARG, "x must be 16-byte aligned");
  if (!L->router_w) return fail(MOEQ_ERR_INVALID_ARG, "no router weight is set");
  moeq_status st = check_device(L);
  if (st != MOEQ_OK) return st;
  const hipError_t e = launch_router_gate((const uint16_t*)x, L->router_w, n, L->cfg.hidden, L->cfg.n_experts,
                                          logits, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "router gate launch");
}

// Scratch of moeq_expert_importance_noalloc (16 MiB; see below).
static __device__ __align__(256) uint8_t scratch[(size_t)16 << 20];

namespace {

// Scratch of the router-statistics pass over n tokens (layout shared by both
// entry points): idx, w, per-chunk counts, ranks, offsets, permutation,
// active list, the all-kept mask and the bias, each 256-byte aligned.
struct ImportanceScratch {
  size_t o_idx, o_w, o_cc, o_rank, o_off, o_perm, o_act, o_mask, o_bias, total;
};

ImportanceScratch importance_scratch(size_t n_tokens, int k, int E) {
  const size_t nk = n_tokens * k, chunks = (n_tokens + kChunk - 1) / kChunk;
  ImportanceScratch l{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, 256);
    return at;
  };
  l.o_idx = take(nk * 4);
  l.o_w = take(nk * 4);
  l.o_cc = take(chunks * E * 4);
  l.o_rank = take(nk * 4);
  l.o_off = take((size_t)(E + 1) * 4);
  l.o_perm = take(nk * 4);
  l.o_act = take((size_t)(E + 1) * 4);
  l.o_mask = take(E);
  l.o_bias = take((size_t)E * 4);
  l.total = off;
  return l;
}

// Argument checks shared by both entry points (host only, before any HIP call).
moeq_status importance_check(const moeq_config* cfg, const float* score_bias, const float* logits, int32_t n_tokens,
                             double alpha, double retain, const double* importance, const uint8_t* mask) {
  moeq_status st = check_config(cfg);
  if (st != MOEQ_OK) return st;
  const int E = cfg->n_experts;
  if (n_tokens < 1 || n_tokens > (1 << 24))
    return fail(MOEQ_ERR_INVALID_ARG, "n_tokens %d outside 1..2^24", n_tokens);
  if (!logits || !importance || !mask)
    return fail(MOEQ_ERR_INVALID_ARG, "logits, importance and mask must not be NULL");
  if (!(alpha >= 0.0 && alpha <= 1.0)) return fail(MOEQ_ERR_INVALID_ARG, "alpha must lie in [0, 1]");
  if (!(retain > 0.0 && retain <= 1.0)) return fail(MOEQ_ERR_INVALID_ARG, "retain must lie in (0, 1]");
  if (score_bias)
    for (int e = 0; e < E; ++e)
      if (!isfinite(score_bias[e]) || fabsf(score_bias[e]) > 1e30f)
        return fail(MOEQ_ERR_INVALID_ARG, "score_bias[%d] is not a finite value of magnitude <= 1e30", e);
  std::vector<uint8_t> all(E, 1);
  int kept = 0;
  return check_routing(cfg, all.data(), &kept);
}

// The pass itself on caller-provided scratch `buf` (layout importance_scratch):
// route with every expert kept, bucket, per-expert statistics, mask.
hipError_t importance_run(const moeq_config* cfg, const float* score_bias, const float* logits, int32_t n_tokens,
                          double alpha, double retain, double* importance, uint8_t* mask, int32_t* counts,
                          hipStream_t s, uint8_t* buf, const ImportanceScratch& l) {
  const int E = cfg->n_experts, k = cfg->top_k;
  int keep = (int)std::ceil(retain * (double)E - 1e-9);
  keep = keep < 1 ? 1 : keep > E ? E : keep;
  Workspace ws{};
  ws.idx = (int32_t*)(buf + l.o_idx);
  ws.w = (float*)(buf + l.o_w);
  ws.chunk_cnt = (int32_t*)(buf + l.o_cc);
  ws.rank = (int32_t*)(buf + l.o_rank);
  ws.offsets = (int32_t*)(buf + l.o_off);
  ws.perm = (int32_t*)(buf + l.o_perm);
  ws.active = (int32_t*)(buf + l.o_act);
  uint8_t* all_kept = buf + l.o_mask;
  float* bias = (float*)(buf + l.o_bias);
  hipError_t e = launch_fill_u8(all_kept, E, 1, s);
  // the bias travels in kernel arguments, so score_bias is free on return
  if (e == hipSuccess) e = launch_store_host_floats(bias, score_bias, E, s);
  RouterParams rp{};
  rp.logits = logits;
  rp.mask = all_kept;
  rp.bias = bias;
  rp.kept_ids = nullptr;
  rp.E_row = E;
  rp.E = E;
  rp.G = cfg->n_group;
  rp.TG = cfg->topk_group;
  rp.k = k;
  rp.topn = cfg->group_topn;
  rp.norm = 0;       // weights = sigmoid scores
  rp.scale = 1.0f;
  rp.x = nullptr;
  if (e == hipSuccess) e = launch_route_tokens(rp, n_tokens, ws.idx, ws.w, s);
  if (e == hipSuccess) e = launch_bucket_chunked(ws.idx, n_tokens, k, E, ws, s);
  if (e == hipSuccess)
    e = launch_expert_importance(ws.offsets, ws.perm, ws.w, E, n_tokens, alpha, keep, importance, mask, counts, s);
  return e;
}

// ---- scratch of moeq_expert_importance_noalloc: the file-scope device array ----
// Each device the library runs on holds its own copy for the life of the
// process.  In host code `scratch` is only a stand-in for the symbol: its
// device address comes from hipGetSymbolAddress, looked up once per device
// with that device current, and only that address is ever handed to kernels.
constexpr size_t kStaticScratchBytes = sizeof(scratch);
std::mutex g_scratch_mu;
uint8_t* g_scratch_ptr[kMaxDevices] = {};

hipError_t static_scratch(int dev, uint8_t** out) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = (uint8_t*)p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

moeq_status moeq_expert_importance(const moeq_config* cfg, const float* score_bias, const float* logits,
                                   int32_t n_tokens, double alpha, double retain, double* importance,
                                   uint8_t* mask, int32_t* counts, void* stream) {
  moeq_status st = importance_check(cfg, score_bias, logits, n_tokens, alpha, retain, importance, mask);
  if (st != MOEQ_OK) return st;
  const ImportanceScratch l = importance_scratch((size_t)n_tokens, cfg->top_k, cfg->n_experts);
  hipStream_t s = (hipStream_t)stream;
  uint8_t* buf = nullptr;
  hipError_t e = hipMallocAsync((void**)&buf, l.total, s);
  if (e != hipSuccess) return hip_fail(e, "hipMallocAsync (importance scratch)");
  e = importance_run(cfg, score_bias, logits, n_tokens, alpha, retain, importance, mask, counts, s, buf, l);
  const hipError_t ef = hipFreeAsync(buf, s);
  if (e != hipSuccess) return hip_fail(e, "expert importance");
  if (ef != hipSuccess) return hip_fail(ef, "hipFreeAsync (importance scratch)");
  return ok();
}

moeq_status moeq_expert_importance_noalloc(const moeq_config* cfg, const float* score_bias, const float* logits,
                                           int32_t n_tokens, double alpha, double retain, double* importance,
                                           uint8_t* mask, int32_t* counts, void* stream) {
  moeq_status st = importance_check(cfg, score_bias, logits, n_tokens, alpha, retain, importance, mask);
  if (st != MOEQ_OK) return st;
  const ImportanceScratch l = importance_scratch((size_t)n_tokens, cfg->top_k, cfg->n_experts);
  if (l.total > kStaticScratchBytes)
    return fail(MOEQ_ERR_CAPACITY,
                "%d tokens at top_k %d over %d experts need %zu bytes of scratch; the static scratch holds %zu",
                n_tokens, cfg->top_k, cfg->n_experts, l.total, kStaticScratchBytes);
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  uint8_t* buf = nullptr;
  if ((e = static_scratch(dev, &buf)) != hipSuccess) return hip_fail(e, "hipGetSymbolAddress (static scratch)");
  e = importance_run(cfg, score_bias, logits, n_tokens, alpha, retain, importance, mask, counts,
                     (hipStream_t)stream, buf, l);
  return e == hipSuccess ? ok() : hip_fail(e, "expert importance");
}

moeq_status moeq_set_stage_events(moeq_layer* L, void* const* events, int32_t count) {
  if (!L) return fail(MOEQ_ERR_INVALID_ARG, "layer is NULL");
  if (count == 0) {
    L->timing = false;
    return ok();
  }
  if (count != MOEQ_STAGE_EVENTS || !events)
    return fail(MOEQ_ERR_INVALID_ARG, "need %d events (got %d)", MOEQ_STAGE_EVENTS, count);
  for (int i = 0; i < MOEQ_STAGE_EVENTS; ++i)
    if (!events[i]) return fail(MOEQ_ERR_INVALID_ARG, "event %d is NULL", i);
  for (int i = 0; i < MOEQ_STAGE_EVENTS; ++i) L->stage_events[i] = (hipEvent_t)events[i];
  L->timing = true;
  return ok();
}

moeq_status moeq_route(moeq_layer* L, const float* logits, int32_t n, int32_t* idx, float* w,
                       void* stream) {
  if (!L) return fail(MOEQ_ERR_INVALID_ARG, "layer is NULL");
  if (n < 0 || n > L->cfg.max_tokens)
    return fail(n < 0 ? MOEQ_ERR_INVALID_ARG : MOEQ_ERR_CAPACITY, "n_tokens %d outside 0..max_tokens", n);
  if (n == 0) return ok();
  if (!logits || !idx || !w) return fail(MOEQ_ERR_INVALID_ARG, "logits, idx and w must not be NULL");
  moeq_status st = check_device(L);
  if (st != MOEQ_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = route_and_bucket(L, logits, n, s);
  if (e != hipSuccess) return hip_fail(e, "route launch");
  const size_t bytes = (size_t)n * L->cfg.top_k * 4;
  if ((e = hipMemcpyAsync(idx, L->ws.idx, bytes, hipMemcpyDeviceToDevice, s)) != hipSuccess ||
      (e = hipMemcpyAsync(w, L->ws.w, bytes, hipMemcpyDeviceToDevice, s)) != hipSuccess)
    return hip_fail(e, "route copy-out");
  return ok();
}

moeq_status moeq_bucket(moeq_layer* L, const int32_t* idx, int32_t n, int32_t* offsets, int32_t* perm,
                        void* stream) {
  if (!L) return fail(MOEQ_ERR_INVALID_ARG, "layer is NULL");
  if (n < 0 || n > L->cfg.max_tokens)
    return fail(n < 0 ? MOEQ_ERR_INVALID_ARG : MOEQ_ERR_CAPACITY, "n_tokens %d outside 0..max_tokens", n);
  if (!idx || !offsets || !perm) return fail(MOEQ_ERR_INVALID_ARG, "idx, offsets and perm must not be NULL");
  moeq_status st = check_device(L);
  if (st != MOEQ_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  const int E = L->cfg.n_experts, k = L->cfg.top_k;
  hipError_t e;
  if (n == 0) {
    e = hipMemsetAsync(offsets, 0, (size_t)(E + 1) * 4, s);
    return e == hipSuccess ? ok() : hip_fail(e, "bucket");
  }
  if (n <= kDecodeMaxTokens)
    e = launch_route_bucket_small(router_params(L, nullptr), idx, n, L->ws, s);
  else
    e = launch_bucket_chunked(idx, n, k, E, L->ws, s);
  if (e != hipSuccess) return hip_fail(e, "bucket launch");
  if ((e = hipMemcpyAsync(offsets, L->ws.offsets, (size_t)(E + 1) * 4, hipMemcpyDeviceToDevice, s)) !=
          hipSuccess ||
      (e = hipMemcpyAsync(perm, L->ws.perm, (size_t)n * k * 4, hipMemcpyDeviceToDevice, s)) != hipSuccess)
    return hip_fail(e, "bucket copy-out");
  return ok();
}

moeq_status moeq_dequant(moeq_layer* L, int32_t expert, int32_t proj, float* out, void* stream) {
  return moeq_dequant_as(L, expert, proj, MOEQ_DECODER_EXACT, out, stream);
}

moeq_status moeq_dequant_as(moeq_layer* L, int32_t expert, int32_t proj, int32_t decoder, void* out,
                            void* stream) {
  if (!L) return fail(MOEQ_ERR_INVALID_ARG, "layer is NULL");
  if (decoder != MOEQ_DECODER_EXACT && decoder != MOEQ_DECODER_GEMV_SUBNORMAL && decoder != MOEQ_DECODER_GEMM_F16)
    return fail(MOEQ_ERR_INVALID_ARG, "decoder %d is not one of MOEQ_DECODER_*", decoder);
  if (proj < 0 || proj > 2) return fail(MOEQ_ERR_INVALID_ARG, "proj %d outside 0..2", proj);
  const int E = L->cfg.n_experts, S = L->cfg.n_shared;
  int slot;
  if (expert >= 0 && expert < E)
    slot = expert;
  else if (expert < 0 && -1 - expert < S)
    slot = E + (-1 - expert);
  else
    return fail(MOEQ_ERR_INVALID_ARG, "expert %d is neither a routed id nor -1-s for a shared expert", expert);
  const TensorDev& t = L->desc_host[(size_t)slot * 3 + proj];
  if (!t.codes) return fail(MOEQ_ERR_INVALID_ARG, "expert %d was pruned", expert);
  if (!out) return fail(MOEQ_ERR_INVALID_ARG, "out is NULL");
  if (decoder == MOEQ_DECODER_GEMV_SUBNORMAL && t.bits > 4)
    return fail(MOEQ_ERR_UNSUPPORTED, "the subnormal-pair decoder serves widths 2-4 (tensor has %d bits)", t.bits);
  moeq_status st = check_device(L);
  if (st != MOEQ_OK) return st;
  hipError_t e;
  if (decoder == MOEQ_DECODER_EXACT)
    e = launch_dequant(t, (float*)out, (hipStream_t)stream);
  else if (decoder == MOEQ_DECODER_GEMV_SUBNORMAL)
    e = launch_dequant_sub(t, (float*)out, (hipStream_t)stream);
  else
    e = launch_dequant_gemm(t, (uint16_t*)out, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "dequant launch");
}

moeq_status moeq_quantize(const float* w, int32_t rows, int32_t K, int32_t bits, void* codes,
                          uint16_t* scales, void* stream) {
  if (!w || !codes || !scales) return fail(MOEQ_ERR_INVALID_ARG, "w, codes and scales must not be NULL");
  if (rows < 0 || K < 0 || K % kBlock) return fail(MOEQ_ERR_INVALID_ARG, "rows %d / K %d invalid", rows, K);
  if (!valid_bits(bits)) return fail(MOEQ_ERR_INVALID_ARG, "bits %d not in {2,3,4,5,6,8}", bits);
  if (rows == 0 || K == 0) return ok();
  hipError_t e = launch_quantize(w, rows, K, bits, (uint8_t*)codes, scales, (hipStream_t)stream);
  return e == hipSuccess ? ok() : hip_fail(e, "quantize launch");
}

}  // extern "C"

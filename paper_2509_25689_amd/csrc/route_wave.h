// The one-wavefront router (Sections 3.1 and 3.2 of arXiv 2509.25689, with
// the DeepSeek-V3 routing function its model uses): the routing kernels and
// the one-token gate/up kernel, which routes its token itself, share it.
// See route.hip for the routing function and its tie order.
#pragma once

#include "internal.h"
#include "layout.h"

namespace moeq {

namespace {

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

// Order-preserving float -> uint32 map; keys compare like the selection
// order: larger score first, then lower id.  0 = no candidate.
__device__ __forceinline__ uint32_t ord_f32(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ uint64_t sel_key(float v, int e) {
  return ((uint64_t)ord_f32(v) << 32) | (uint64_t)(~(uint32_t)e);
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint64_t dpp64(uint64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, CTRL, ROW_MASK, 0xF, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), CTRL, ROW_MASK, 0xF, false);
  return ((uint64_t)hi << 32) | lo;
}

// Maximum of a 64-bit key over the wavefront, returned to every lane:
// row prefix maxima (row_shr 1, 2, 4, 8), then row broadcasts into lane 63.
__device__ __forceinline__ uint64_t wave_max_key(uint64_t k) {
  uint64_t t;
  t = dpp64<0x111, 0xF>(k); k = t > k ? t : k;
  t = dpp64<0x112, 0xF>(k); k = t > k ? t : k;
  t = dpp64<0x114, 0xF>(k); k = t > k ? t : k;
  t = dpp64<0x118, 0xF>(k); k = t > k ? t : k;
  t = dpp64<0x142, 0xA>(k); k = t > k ? t : k;   // row_bcast:15
  t = dpp64<0x143, 0xC>(k); k = t > k ? t : k;   // row_bcast:31
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)k, 63);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(k >> 32), 63);
  return ((uint64_t)hi << 32) | lo;
}

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Maximum of an unsigned key over the wavefront, returned to every lane
// (0 is the identity, so each step folds into one v_max_u32 with DPP).
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false));  // row_shr:1
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false));  // row_shr:2
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false));  // row_shr:4
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false));  // row_shr:8
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false));  // row_bcast:15
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false));  // row_bcast:31
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Inclusive prefix sum over the wavefront.
__device__ __forceinline__ int wave_incl_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);  // row_bcast:15
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return v;
}

// Which of the lane's experts the selection chose: bit i of `bits` for
// expert lane*EPL + i, chosen as the token's j-th expert with j = order[i].
template <int EPL>
struct LaneChoice {
  uint32_t bits;
  int order[EPL];
};

// Route token t with the calling wavefront.  Lane l owns experts
// [l*EPL, l*EPL + EPL).  gs_l: this wave's LDS row of >= G floats.  Writes
// idx/w for the token to idx_g/w_g and the ids to idx_s, each if not null.
// Returns the lane's share of the choice (router expert indices).
template <int EPL>
__device__ LaneChoice<EPL> route_token_wave(const RouterParams& rp, int t, float* gs_l, int32_t* idx_g,
                                            float* w_g, int32_t* idx_s) {
  const int lane = threadIdx.x & 63;
  if (rp.x) {
    // binary exponent prescale for half precision: e puts the row's largest
    // |x| in [2^14, 2^15) (e >= -100 keeps 2^-e finite for an all-zero row),
    // and the prescaled binary16 copy of the row (exact unless a value lies
    // more than 2^28 below the largest, then rounded to nearest even)
    const MOEQ_GLOBAL u32x4* xr = gptr(reinterpret_cast<const u32x4*>(rp.x + (size_t)t * rp.H));
    const int C = rp.H / 8;
    // XB pieces per lane requested together in each pass (indices past the
    // row read its last piece again: loads that do not depend on a
    // condition go out before the first is used)
    constexpr int XB = EPL >= 8 ? 4 : 8;
    uint32_t mx = 0;
    for (int c0 = lane; c0 < C; c0 += 64 * XB) {
      u32x4 v[XB];
#pragma unroll
      for (int b = 0; b < XB; ++b) v[b] = xr[min(c0 + 64 * b, C - 1)];
#pragma unroll
      for (int b = 0; b < XB; ++b) {
        const uint32_t q[4] = {v[b].x, v[b].y, v[b].z, v[b].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) mx = max(mx, max(q[j] & 0x7FFFu, (q[j] >> 16) & 0x7FFFu));
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, off, 64));
    const int e = max((int)((mx >> 7) & 0xFFu) - 127 - 14, -100);
    if (lane == 0) rp.xexp[t] = e;
    const float sc = __builtin_amdgcn_ldexpf(1.0f, -e);
    MOEQ_GLOBAL u32x4* hr = (MOEQ_GLOBAL u32x4*)(rp.x16 + (size_t)t * rp.H);
    for (int c0 = lane; c0 < C; c0 += 64 * XB) {
      u32x4 v[XB];
#pragma unroll
      for (int b = 0; b < XB; ++b) v[b] = xr[min(c0 + 64 * b, C - 1)];
#pragma unroll
      for (int b = 0; b < XB; ++b) {
        const uint32_t q[4] = {v[b].x, v[b].y, v[b].z, v[b].w};
        uint32_t o[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float lo = __uint_as_float(q[j] << 16) * sc, hi = __uint_as_float(q[j] & 0xFFFF0000u) * sc;
          o[j] = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)lo) |
                 ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)hi) << 16);
        }
        if (c0 + 64 * b < C) hr[c0 + 64 * b] = u32x4{o[0], o[1], o[2], o[3]};
      }
    }
  }
  const int E = rp.E, G = rp.G, per = rp.E / rp.G;
  const float* lg = rp.logits + (size_t)t * rp.E_row;
  float s[EPL], b[EPL];
  // every load is issued before the first is used, unconditionally (a
  // conditional load makes the compiler wait for all outstanding ones), so
  // the inputs take one memory round trip (two with kept_ids); lanes past E
  // read the last expert and discard it
  float lv[EPL], bv[EPL];
  bool kv[EPL];
  int eo[EPL];  // original expert ids
  if (rp.kept_ids) {
#pragma unroll
    for (int i = 0; i < EPL; ++i) eo[i] = rp.kept_ids[min(lane * EPL + i, E - 1)];
  } else {
#pragma unroll
    for (int i = 0; i < EPL; ++i) eo[i] = min(lane * EPL + i, E - 1);
  }
  uint8_t mk[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    lv[i] = lg[eo[i]];
    bv[i] = rp.bias[eo[i]];
    mk[i] = rp.mask[eo[i]];
  }
#pragma unroll
  for (int i = 0; i < EPL; ++i) kv[i] = (rp.kept_ids != nullptr) | (mk[i] != 0);
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane * EPL + i;
    s[i] = 0.0f;
    b[i] = -INFINITY;
    if (e < E) {
      // sigmoid evaluated in double precision, rounded once to float
      float v = (float)(1.0 / (1.0 + exp(-(double)lv[i])));
      if (!(v == v)) v = 0.0f;  // a NaN logit must not leave the index range undefined
      s[i] = v;
      if (kv[i]) b[i] = v + bv[i];
    }
  }

  // ---- group scores: float32 sum of each group's topn best kept scores ----
  const int lpg = per / EPL;  // lanes per group on the fast path
  const bool fast = per % EPL == 0 && (lpg & (lpg - 1)) == 0 && rp.topn <= 2;
  if (fast) {
    float a = -INFINITY, c = -INFINITY;  // best and second best of this lane
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      if (b[i] > a) {
        c = a;
        a = b[i];
      } else if (b[i] > c) {
        c = b[i];
      }
    }
    // partners: quad butterflies, then the mirror lane of the half row and
    // of the row (each step pairs lanes whose partial groups are disjoint
    // halves of the next larger group), then shuffles beyond 16 lanes
    auto merge = [&](float oa, float oc) {
      const float lo = fminf(a, oa);
      a = fmaxf(a, oa);
      c = fmaxf(lo, fmaxf(c, oc));
    };
    if (lpg > 1) merge(dpp_f32<0xB1>(a), dpp_f32<0xB1>(c));    // quad_perm [1,0,3,2]
    if (lpg > 2) merge(dpp_f32<0x4E>(a), dpp_f32<0x4E>(c));    // quad_perm [2,3,0,1]
    if (lpg > 4) merge(dpp_f32<0x141>(a), dpp_f32<0x141>(c));  // row_half_mirror
    if (lpg > 8) merge(dpp_f32<0x140>(a), dpp_f32<0x140>(c));  // row_mirror
    for (int off = 16; off < lpg; off <<= 1) merge(__shfl_xor(a, off, 64), __shfl_xor(c, off, 64));
    float gsc = a;
    if (rp.topn == 2 && c != -INFINITY) gsc = a + c;  // 0 + a + c in float32, best first
    if (lane % lpg == 0 && lane / lpg < G) gs_l[lane / lpg] = gsc;
  } else {
    // any group size and topn: per group, topn rounds of a wave-wide arg-max
    for (int g = 0; g < G; ++g) {
      float acc = 0.0f;
      int taken = 0;
      uint64_t prev = ~0ull;
      for (int r = 0; r < rp.topn; ++r) {
        uint64_t kb = 0;
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
          const int e = lane * EPL + i;
          const uint64_t kk = (e < E && e / per == g && b[i] != -INFINITY) ? sel_key(b[i], e) : 0ull;
          if (kk < prev && kk > kb) kb = kk;
        }
        kb = wave_max_key(kb);
        if (kb == 0) break;
        const int e = (int)~(uint32_t)kb;
        float bv = 0.0f;
#pragma unroll
        for (int i = 0; i < EPL; ++i)
          if (e % EPL == i) bv = b[i];
        acc = acc + __shfl(bv, e / EPL, 64);
        ++taken;
        prev = kb;
      }
      if (lane == 0) gs_l[g] = taken ? acc : -INFINITY;
    }
  }
  wave_sync();

  // ---- group selection: group g is kept if fewer than TG groups precede it ----
  bool keep = false;
  if (lane < G) {
    const float mine = gs_l[lane];
    int rank = 0;
    for (int g = 0; g < G; ++g) rank += before(gs_l[g], g, mine, lane);
    keep = rank < rp.TG;
  }
  const uint64_t gsel = __ballot(keep);

  // ---- expert selection ----
  // Each lane sorts its own candidates (biased score descending, lower id
  // first); then k rounds of: wave-wide max of every lane's current head
  // key, the lowest lane holding it wins (lane l owns ids [l*EPL, l*EPL+EPL),
  // so that is the lowest id among equal scores), the winner advances.
  int gi[EPL];  // group of each of the lane's experts
  if (per % EPL == 0) {
    const int g0 = lane * EPL / per;
#pragma unroll
    for (int i = 0; i < EPL; ++i) gi[i] = g0;
  } else {
#pragma unroll
    for (int i = 0; i < EPL; ++i) gi[i] = (lane * EPL + i) / per;
  }
  float cv[EPL], cs[EPL];
  int ci[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane * EPL + i;
    const bool ok = e < E && b[i] != -INFINITY && ((gsel >> gi[i]) & 1);
    cv[i] = ok ? b[i] : -INFINITY;
    cs[i] = s[i];
    ci[i] = i;
  }
#pragma unroll
  for (int i = 1; i < EPL; ++i)
#pragma unroll
    for (int j = i; j > 0; --j) {
      // insertion step: move element j up while it comes before element j-1
      const bool sw = cv[j] > cv[j - 1] || (cv[j] == cv[j - 1] && ci[j] < ci[j - 1]);
      const float tv = cv[j], ts = cs[j];
      const int ti = ci[j];
      cv[j] = sw ? cv[j - 1] : cv[j];
      cs[j] = sw ? cs[j - 1] : cs[j];
      ci[j] = sw ? ci[j - 1] : ci[j];
      cv[j - 1] = sw ? tv : cv[j - 1];
      cs[j - 1] = sw ? ts : cs[j - 1];
      ci[j - 1] = sw ? ti : ci[j - 1];
    }
  // keys: order-preserving map of the score, 0 = no candidate left
  uint32_t key[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) key[i] = cv[i] == -INFINITY ? 0u : ord_f32(cv[i]);
  LaneChoice<EPL> ch;
  ch.bits = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i) ch.order[i] = 0;
  // the lane's head: its pos-th sorted candidate (pos = EPL: none left)
  int pos = 0;
  uint32_t hk = key[0];
  float hs = cs[0];
  int hi = ci[0];
  float sum = 0.0f, my_s = 0.0f;
  int my_i = 0, last = 0;
  // branch-free rounds (selects, not exec masks), unrolled by 8: each round
  // is a short dependency chain, and taken branches would dominate it
  auto round = [&](int r) {
    const uint32_t m = wave_max_u32(hk);
    const uint64_t hold = __ballot((hk == m) & (m != 0u));
    // creation checks guarantee k candidates; never leave the index range
    // (the lane reads are unconditional; the selects follow them)
    const int wl = hold ? (int)__builtin_ctzll(hold) : 0;
    const int li = __builtin_amdgcn_readlane(hi, wl);
    const float sr = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, hs), wl));
    const float sv = hold ? sr : 0.0f;
    const int e = hold ? wl * EPL + li : last;
    const bool win = hold && lane == wl;
    ch.bits |= win ? 1u << hi : 0u;
#pragma unroll
    for (int i = 0; i < EPL; ++i) ch.order[i] = win && i == hi ? r : ch.order[i];
    const int np = pos + 1;
    uint32_t nk = 0u;
    float ns = hs;
    int ni = hi;
#pragma unroll
    for (int i = 1; i < EPL; ++i) {
      nk = np == i ? key[i] : nk;
      ns = np == i ? cs[i] : ns;
      ni = np == i ? ci[i] : ni;
    }
    pos = win ? np : pos;
    hk = win ? nk : hk;
    hs = win ? ns : hs;
    hi = win ? ni : hi;
    sum = sum + sv;
    my_i = lane == r ? e : my_i;
    my_s = lane == r ? sv : my_s;
    last = e;
  };
  int r = 0;
  for (; r + 8 <= rp.k; r += 8) {
#pragma unroll
    for (int q = 0; q < 8; ++q) round(r + q);
  }
  for (; r < rp.k; ++r) round(r);
  if (lane < rp.k) {
    float wv;
    if (rp.norm)
      wv = sum == 0.0f ? 0.0f : my_s / sum * rp.scale;
    else
      wv = my_s * rp.scale;
    const int id = rp.kept_ids ? rp.kept_ids[my_i] : my_i;  // back to original ids
    if (idx_g) idx_g[(size_t)t * rp.k + lane] = id;
    if (w_g) w_g[(size_t)t * rp.k + lane] = wv;
    if (idx_s) idx_s[t * rp.k + lane] = id;
  }
  wave_sync();  // gs_l is reused by this wave's next token
  return ch;
}

}  // namespace

}  // namespace moeq

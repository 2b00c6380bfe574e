// Top-k expert routing and the canonical token -> row permutation of the
// MoE layer (the paper's MoE rollout layer, Sec. 3.3 / Sec. 4.1; the router
// itself is not specified there: top-k of the logits with ties to the lower
// expert index, softmax weights over the selected logits).
//
// Three workgroup bodies (launched alone by route.hip, or fused with the
// activation quantiser and the channel selection by the layer):
//   route_topk_body      E <= 256 and few tokens: one workgroup per token,
//                        every expert's rank counted in parallel, rank r < k
//                        is slot r; many tokens or larger E: one wavefront
//                        per token, k rounds of a wave-wide arg-max.  Then
//                        the softmax weights.
//   route_rank_body      per block of 256 tokens: expert bitmasks in LDS give
//                        every (token, slot) its rank among the block's tokens
//                        of the same expert, and per-block expert counts.
//   route_scatter_body   scan of the counts -> expert offsets; row =
//                        offset[e] + rows of e in earlier blocks + rank
//                        (256 or more threads).
// No atomic slot claims: the row order (expert asc, token asc) is a pure
// function of the routing, so the permutation is bit-reproducible.
#pragma once
#include <type_traits>

#include "common.h"

namespace qdr {


constexpr int kTokBlock = 256;
constexpr int kMaxE = 1024;
constexpr int kMaxK = 32;

// (value desc, index asc)
__device__ __forceinline__ bool better(float v1, int e1, float v2, int e2) {
  return v1 > v2 || (v1 == v2 && e1 < e2);
}

// Order-preserving 64-bit key of (value desc, index asc): a larger key takes
// an earlier slot.  The float bits map to an unsigned order (negative values
// flipped), -0 counts as +0 (they compare equal), and the low word holds the
// complement of the expert index.  No real logit maps to key 0, which pads.
__device__ __forceinline__ uint64_t topk_key(float v, int e) {
  uint32_t b = __float_as_uint(v);
  if (b == 0x80000000u) b = 0u;
  const uint32_t o = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return ((uint64_t)o << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)e);
}

// Top-k for E <= 256 experts, one workgroup per token: lane l of every wave
// holds experts l, l + 64, ...; wave w broadcasts the keys of experts
// l + 64 j with l in [16 w, 16 w + 16) in turn from their lanes and counts,
// for each of its lane's experts, how many of those have a larger key; the
// four partial counts summed in LDS give each expert's rank, and rank r < k
// is slot r.  No serial reduction rounds.
constexpr int kRankMaxE = 256;
__device__ __forceinline__ void route_topk_rank_body(int bid, const float *__restrict__ logits,
                                                     int64_t T, int E, int k, int renorm,
                                                     int32_t *__restrict__ ids,
                                                     float *__restrict__ wts) {
  __shared__ int rk[kRankMaxE];
  __shared__ float slot_v[kMaxK];
  __shared__ int slot_e[kMaxK];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int64_t t = bid;
  if (t >= T) return;                           // whole workgroup
  const int per = (E + 63) >> 6;                // <= 4, uniform
  for (int e = threadIdx.x; e < E; e += blockDim.x) rk[e] = 0;
  float v[4];
  uint64_t key[4];
  int r[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = lane + 64 * j;
    const bool ok = j < per && e < E;
    v[j] = ok ? logits[t * E + e] : 0.0f;
    key[j] = ok ? topk_key(v[j], e) : 0ull;
    r[j] = 0;
  }
  const int wu = __builtin_amdgcn_readfirstlane(wid);
#pragma unroll
  for (int j2 = 0; j2 < 4; ++j2) {
    if (j2 >= per) break;
    const uint32_t kh = (uint32_t)(key[j2] >> 32), kl = (uint32_t)key[j2];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int i = 16 * wu + q;
      const uint64_t u = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)kh, i) << 32) |
                         (uint32_t)__builtin_amdgcn_readlane((int)kl, i);
#pragma unroll
      for (int j = 0; j < 4; ++j) r[j] += u > key[j] ? 1 : 0;
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = lane + 64 * j;
    if (j < per && e < E) atomicAdd(&rk[e], r[j]);
  }
  __syncthreads();
  if (wid == 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = lane + 64 * j;
      if (j < per && e < E && rk[e] < k) {
        slot_v[rk[e]] = v[j];
        slot_e[rk[e]] = e;
      }
    }
  }
  __syncthreads();
  if (wid != 0) return;
  const float top_v = slot_v[0];
  float denom = 0.0f;
  if (renorm) {
    for (int s = 0; s < k; ++s) denom += expf(slot_v[s] - top_v);   // slot order 0..k-1
  } else {                 // full softmax denominator over all E experts
    float part = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (j < per && lane + 64 * j < E) part += expf(v[j] - top_v);
    for (int o = 32; o > 0; o >>= 1) part += __shfl_xor(part, o, 64);
    denom = part;
  }
  if (lane < k) {
    ids[t * k + lane] = slot_e[lane];
    wts[t * k + lane] = expf(slot_v[lane] - top_v) / denom;
  }
}

// Top-k for E <= 256 experts and many tokens: one wavefront per token, four
// tokens per workgroup.  k rounds of a wave-wide arg-max of the 64-bit keys
// (within rows of 16 lanes by DPP moves, across rows by two shuffles); all
// keys differ, so each round's maximum sits in exactly one lane and slot, and
// the expert found in round s takes slot s.  (Counting every expert's rank
// against all E broadcast keys instead takes 2.5x the time at E = 128,
// k = 8.)  Same arithmetic as the rank body above (softmax terms in slot
// order).
constexpr int64_t kTopkWaveMinT = 1024;
// PER = ceil(E / 64) experts per lane
template <int PER>
__device__ __forceinline__ void route_topk_wave_body(int bid, const float *__restrict__ logits,
                                                     int64_t T, int E, int k, int renorm,
                                                     int32_t *__restrict__ ids,
                                                     float *__restrict__ wts) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int64_t t = (int64_t)bid * 4 + wid;
  if (t >= T) return;                           // whole wave; no barriers below
  float v[PER];
  uint64_t key[PER];
  int r[PER];
  bool ok[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int e = lane + 64 * j;
    ok[j] = e < E;
    v[j] = ok[j] ? logits[t * E + e] : 0.0f;
    key[j] = ok[j] ? topk_key(v[j], e) : 0ull;
    r[j] = 0;
  }
  // r[j]: the round that found expert lane + 64 j, or k (not selected)
  {
    uint64_t kk[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      kk[j] = key[j];
      r[j] = k;
    }
    for (int rd = 0; rd < k; ++rd) {
      uint64_t m = kk[0];
#pragma unroll
      for (int j = 1; j < PER; ++j) m = kk[j] > m ? kk[j] : m;
      auto step_dpp = [&](auto ctrl_c) __attribute__((always_inline)) {
        constexpr int C = decltype(ctrl_c)::value;
        const uint32_t h = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(m >> 32), C, 0xF, 0xF, false);
        const uint32_t l = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)m, C, 0xF, 0xF, false);
        const uint64_t o = ((uint64_t)h << 32) | l;
        m = o > m ? o : m;
      };
      step_dpp(std::integral_constant<int, 0xB1>{});    // quad_perm [1,0,3,2]
      step_dpp(std::integral_constant<int, 0x4E>{});    // quad_perm [2,3,0,1]
      step_dpp(std::integral_constant<int, 0x124>{});   // row_ror 4
      step_dpp(std::integral_constant<int, 0x128>{});   // row_ror 8
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const uint32_t h = (uint32_t)__shfl_xor((int)(uint32_t)(m >> 32), o, 64);
        const uint32_t l = (uint32_t)__shfl_xor((int)(uint32_t)m, o, 64);
        const uint64_t x = ((uint64_t)h << 32) | l;
        m = x > m ? x : m;
      }
      // unused slots hold key 0, below every real key (k <= E)
#pragma unroll
      for (int j = 0; j < PER; ++j)
        if (kk[j] == m) {
          r[j] = rd;
          kk[j] = 0ull;
        }
    }
  }
  // the value of slot s, broadcast from the lane holding the expert of rank s
  auto slot_value = [&](int sl) {
    float val = 0.0f;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const uint64_t b = __ballot(ok[j] && r[j] == sl);
      if (b) val = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v[j]), __ffsll((long long)b) - 1));
    }
    return val;
  };
  const float top_v = slot_value(0);
  float denom = 0.0f;
  if (renorm) {
    for (int sl = 0; sl < k; ++sl) denom += expf(slot_value(sl) - top_v);   // slot order
  } else {                 // full softmax denominator over all E experts
    float part = 0.0f;
#pragma unroll
    for (int j = 0; j < PER; ++j)
      if (ok[j]) part += expf(v[j] - top_v);
    for (int o = 32; o > 0; o >>= 1) part += __shfl_xor(part, o, 64);
    denom = part;
  }
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    if (ok[j] && r[j] < k) {
      ids[t * k + r[j]] = lane + 64 * j;
      wts[t * k + r[j]] = expf(v[j] - top_v) / denom;
    }
  }
}

// workgroups the top-k step needs for T tokens and E experts
inline int topk_groups(int64_t T, int E) {
  return (int)(E <= kRankMaxE && T < kTopkWaveMinT ? T : (T + 3) / 4);
}

// E <= 256: the rank body (T < 1024) or the wave body above.  Otherwise one
// wavefront per token, four tokens per workgroup (workgroup index bid): k
// rounds of a wave-wide arg-max (any E up to kMaxE).
__device__ __forceinline__ void route_topk_body(int bid, const float *__restrict__ logits,
                                                int64_t T, int E, int k, int renorm,
                                                int32_t *__restrict__ ids,
                                                float *__restrict__ wts) {
  if (E <= kRankMaxE) {
    if (T < kTopkWaveMinT) {
      route_topk_rank_body(bid, logits, T, E, k, renorm, ids, wts);
    } else {
      switch ((E + 63) >> 6) {
        case 1: route_topk_wave_body<1>(bid, logits, T, E, k, renorm, ids, wts); break;
        case 2: route_topk_wave_body<2>(bid, logits, T, E, k, renorm, ids, wts); break;
        case 3: route_topk_wave_body<3>(bid, logits, T, E, k, renorm, ids, wts); break;
        default: route_topk_wave_body<4>(bid, logits, T, E, k, renorm, ids, wts); break;
      }
    }
    return;
  }
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int64_t t = (int64_t)bid * 4 + wid;
  if (t >= T) return;
  const int per_lane = (E + 63) / 64;
  float v[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    int e = lane + 64 * j;
    v[j] = (j < per_lane && e < E) ? logits[t * E + e] : -INFINITY;
  }
  uint32_t used = 0u;
  float top_v = 0.0f, denom = 0.0f, my_v = 0.0f;
  int my_e = 0;
  for (int s = 0; s < k; ++s) {
    // best unused candidate of this lane
    float bv = -INFINITY;
    int be = 0x7fffffff;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      int e = lane + 64 * j;
      if (j < per_lane && e < E && !((used >> j) & 1u) && better(v[j], e, bv, be)) {
        bv = v[j];
        be = e;
      }
    }
    // wave-wide arg-max; the order is total, so every lane ends with the winner
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      float ov = __shfl_xor(bv, o, 64);
      int oe = __shfl_xor(be, o, 64);
      if (better(ov, oe, bv, be)) {
        bv = ov;
        be = oe;
      }
    }
    if ((be & 63) == lane) used |= 1u << (be >> 6);
    if (s == 0) top_v = bv;
    if (renorm) denom += expf(bv - top_v);        // slot order 0..k-1
    if (lane == s) {
      my_v = bv;
      my_e = be;
    }
  }
  if (!renorm) {           // full softmax denominator over all E experts
    float part = 0.0f;
    for (int j = 0; j < per_lane; ++j) {
      int e = lane + 64 * j;
      if (e < E) part += expf(v[j] - top_v);
    }
    for (int o = 32; o > 0; o >>= 1) part += __shfl_xor(part, o, 64);
    denom = part;
  }
  if (lane < k) {
    ids[t * k + lane] = my_e;
    wts[t * k + lane] = expf(my_v - top_v) / denom;
  }
}

// Per block of 256 tokens: expert bitmasks in LDS give every (token, slot)
// its rank among the block's tokens routed to the same expert, and the
// block's per-expert counts.
// (mask: kMaxE x 8 words and before: kMaxE x 8 bytes of LDS, from the caller)
constexpr int kRankLdsBytes = kMaxE * (kTokBlock / 32) * 5;
__device__ __forceinline__ void route_rank_rows(int bid, int64_t T, int E, int k,
                                                const int32_t *__restrict__ ids,
                                                int32_t *__restrict__ counts,
                                                int32_t *__restrict__ ranks,
                                                uint32_t (*mask)[kTokBlock / 32],
                                                uint8_t (*before)[kTokBlock / 32]) {
  // before[e][w]: tokens of e in earlier words
  const int64_t t0 = (int64_t)bid * kTokBlock;
  for (int i = threadIdx.x; i < E * (kTokBlock / 32); i += blockDim.x) (&mask[0][0])[i] = 0u;
  __syncthreads();
  const int tl = threadIdx.x;
  const int64_t t = t0 + tl;
  // this token's experts, loaded once (k <= 8 in registers)
  int idr[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) idr[s] = (t < T && s < k) ? ids[t * k + s] : 0;
  if (t < T) {
#pragma unroll
    for (int s = 0; s < 8; ++s)
      if (s < k) atomicOr(&mask[idr[s]][tl >> 5], 1u << (tl & 31));
    for (int s = 8; s < k; ++s) atomicOr(&mask[ids[t * k + s]][tl >> 5], 1u << (tl & 31));
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    int c = 0;
#pragma unroll
    for (int w = 0; w < kTokBlock / 32; ++w) {
      before[e][w] = (uint8_t)c;          // < 256: at most 224 tokens before word 7
      c += __popc(mask[e][w]);
    }
    counts[(int64_t)bid * E + e] = c;
  }
  __syncthreads();
  if (t < T) {
    const uint32_t low = (1u << (tl & 31)) - 1u;
    const int wd = tl >> 5;
#pragma unroll
    for (int s = 0; s < 8; ++s)
      if (s < k)
        ranks[t * k + s] = (int)before[idr[s]][wd] + __popc(mask[idr[s]][wd] & low);
    for (int s = 8; s < k; ++s) {
      const int e = ids[t * k + s];
      ranks[t * k + s] = (int)before[e][wd] + __popc(mask[e][wd] & low);
    }
  }
}

// route_rank_rows with LDS arrays of its own
__device__ __forceinline__ void route_rank_body(int bid, int64_t T, int E, int k,
                                                const int32_t *__restrict__ ids,
                                                int32_t *__restrict__ counts,
                                                int32_t *__restrict__ ranks) {
  __shared__ uint32_t mask[kMaxE][kTokBlock / 32];
  __shared__ uint8_t before[kMaxE][kTokBlock / 32];
  route_rank_rows(bid, T, E, k, ids, counts, ranks, mask, before);
}

__device__ __forceinline__ void route_scatter_body(
    int bid, int64_t T, int E, int k, int nblk, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ counts, const int32_t *__restrict__ ranks,
    int32_t *__restrict__ offsets, int32_t *__restrict__ row_token,
    int32_t *__restrict__ inv_row) {
  __shared__ int32_t base[kMaxE];
  __shared__ int32_t total[kMaxE];
  const int b = bid;
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    // eight token blocks' counts in flight at a time
    int tot = 0, pre = 0;
    for (int b0 = 0; b0 < nblk; b0 += 8) {
      int c[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int bj = b0 + j < nblk ? b0 + j : nblk - 1;   // in bounds, unpredicated
        const int v = counts[(int64_t)bj * E + e];
        c[j] = b0 + j < nblk ? v : 0;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        tot += c[j];
        if (b0 + j < b) pre += c[j];
      }
    }
    total[e] = tot;
    base[e] = pre;
  }
  __syncthreads();
  {
    // exclusive scan over experts (E <= 1024): threads 0..255 hold four
    // consecutive experts each, scanned across lanes and the four waves
    __shared__ int wsum[4];
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    int c[4], tsum = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * tid + q;
      c[q] = (tid < 256 && e < E) ? total[e] : 0;
      tsum += c[q];
    }
    int xs = tsum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(xs, o, 64);
      if (lane >= o) xs += y;
    }
    if (tid < 256 && lane == 63) wsum[wid] = xs;
    __syncthreads();
    if (tid < 256) {
      int ex = xs - tsum;
      for (int ww = 0; ww < wid; ++ww) ex += wsum[ww];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = 4 * tid + q;
        if (e < E) total[e] = ex;
        ex += c[q];
      }
    }
    if (tid == 0 && b == 0) offsets[E] = wsum[0] + wsum[1] + wsum[2] + wsum[3];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    if (b == 0) offsets[e] = total[e];
    base[e] += total[e];
  }
  __syncthreads();
  const int64_t t = (int64_t)b * kTokBlock + threadIdx.x;
  if (threadIdx.x < kTokBlock && t < T) {
    for (int s = 0; s < k; ++s) {
      const int e = ids[t * k + s];
      const int row = base[e] + ranks[t * k + s];
      row_token[row] = (int32_t)t;
      inv_row[t * k + s] = row;
    }
  }
}

}  // namespace qdr

// Device bodies of the RAC selection (Eq. (channel-select)) and the masked
// residual quantisation (Eq. (residual-recon)): launched alone by rac.hip, or
// fused with the routing work by the layer.
#pragma once
#include "common.h"

namespace qdc {

using namespace qd;

__device__ __forceinline__ void load_bf16x16(const uint16_t *p, float (&x)[16]) {
  const uint4 *q = reinterpret_cast<const uint4 *>(p);
  uint4 a = q[0], b = q[1];
  uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    x[2 * j] = __uint_as_float(w[j] << 16);
    x[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
  }
}

// residual r = fl(x_hat - x) of one 16-block from its codes and scale
__device__ __forceinline__ void block_residual(const float (&x)[16], uint2 cw, uint32_t sb,
                                               float s_dec, float (&r)[16]) {
  const float sbf = e4m3_to_f32(sb);
  float ev[16];
  e2m1_word_values(cw.x, ev);
  e2m1_word_values(cw.y, ev + 8);
#pragma unroll
  for (int i = 0; i < 16; ++i) r[i] = (ev[i] * sbf) * s_dec - x[i];   // as dequant_value
}

// Block-wide exclusive scan of one int per thread (1024 threads).
__device__ int block_exclusive_scan(int v, int *sh /* 1024 + 32 ints */, int &total) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  // inclusive scan inside the wave
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[1024 + wid] = x;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    const int nwv = (int)(blockDim.x >> 6);
    for (int w = 0; w < nwv; ++w) {
      int c = sh[1024 + w];
      sh[1024 + w] = run;
      run += c;
    }
    sh[1024 + 16] = run;
  }
  __syncthreads();
  int res = x - v + sh[1024 + wid];
  total = sh[1024 + 16];
  __syncthreads();
  return res;
}

// Selection for K <= 16384 channels: radix select on 4-bit digits from the
// highest non-zero digit of the largest score down.  Digit counts come from
// wave ballots (no atomics: most channels share their leading digits, which
// would serialise histogram atomics).  Each wave posts its 16 counts, one
// barrier, and every wave then derives the same digit from the posted
// counts (double-buffered, so one barrier per digit).  Thread i owns
// channels i, i + 256, ... in registers.  Channels above the threshold theta
// are taken, then channels equal to it in ascending order until K_s (a
// popcount scan over a bitmap of the equal ones); a popcount scan of the
// selection bitmap emits S in ascending order.
constexpr int kSelThreads = 256;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSelMaxK = 16384;
constexpr int kSelBuckets = 2304;        // 11-bit keys (0..2048), 9 per thread
constexpr int kSelCand = 512;            // candidates ranked directly

// Monotone 11-bit key of a score: 0 for 0, else 1 + 32 e + m with e the
// position of the leading one and m the five bits below it.
__device__ __forceinline__ int sel_key(uint64_t v) {
  if (v == 0ull) return 0;
  const int e = 63 - __clzll((long long)v);
  const uint32_t m = e >= 5 ? (uint32_t)(v >> (e - 5)) & 31u : (uint32_t)(v << (5 - e)) & 31u;
  return 1 + 32 * e + (int)m;
}

template <int PER>
__device__ __forceinline__ void rac_select_body(const uint64_t *__restrict__ scores, int K, int Ks,
                                                int32_t *__restrict__ sel_idx,
                                                uint32_t *__restrict__ bitmap) {
  __shared__ int cnt[2][kSelWaves][16];     // [pass parity][wave][digit]
  __shared__ uint32_t gt[16384 / 32], eq[16384 / 32];
  __shared__ int sh[1024 + 32];
  __shared__ uint64_t s_max[kSelWaves];
  __shared__ int hist[kSelBuckets];
  __shared__ uint64_t cand_s[kSelCand];
  __shared__ int cand_i[kSelCand];
  __shared__ int s_cut[4];                  // bucket, count above it, candidates
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int nw = (K + 31) / 32;
  uint64_t sv[PER];
  bool live[PER];
  uint64_t mx = 0ull;
  for (int i = tid; i < kSelBuckets; i += kSelThreads) hist[i] = 0;
  if (tid == 0) s_cut[2] = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int j = tid + kSelThreads * i;
    live[i] = j < K;
    sv[i] = live[i] ? scores[j] : 0ull;
    mx = sv[i] > mx ? sv[i] : mx;
  }
  for (int w = tid; w < nw; w += kSelThreads) {
    gt[w] = 0u;
    eq[w] = 0u;
  }
  // ---- fast path: histogram of 11-bit keys, the bucket b* holding the
  // K_s-th largest score, and a direct ranking of b*'s channels (by score
  // desc, index asc); taken if b* holds at most kSelCand channels
  bool fast = false;
  if (Ks > 0) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < PER; ++i)
      if (live[i]) atomicAdd(&hist[sel_key(sv[i])], 1);
    __syncthreads();
    // thread t sums keys [kSelBuckets - 9 (t + 1), kSelBuckets - 9 t), top down
    const int hi = kSelBuckets - 9 * tid;
    int c = 0;
#pragma unroll
    for (int q = 1; q <= 9; ++q) c += hist[hi - q];
    int tot;
    int above = block_exclusive_scan(c, sh, tot);
    if (above < Ks && above + c >= Ks) {
      for (int q = 1; q <= 9; ++q) {
        const int h = hist[hi - q];
        if (above + h >= Ks) {
          s_cut[0] = hi - q;
          s_cut[1] = above;
          break;
        }
        above += h;
      }
    }
    __syncthreads();
    const int bstar = s_cut[0];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      if (live[i] && sel_key(sv[i]) == bstar) {
        const int slot = atomicAdd(&s_cut[2], 1);
        if (slot < kSelCand) {
          cand_s[slot] = sv[i];
          cand_i[slot] = tid + kSelThreads * i;
        }
      }
    }
    __syncthreads();
    const int nc = s_cut[2];
    fast = nc <= kSelCand;
    if (fast) {
      const int need = Ks - s_cut[1];          // channels to take from b*
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int j = tid + kSelThreads * i;
        if (live[i] && sel_key(sv[i]) > bstar) atomicOr(&gt[j >> 5], 1u << (j & 31));
      }
      for (int q = tid; q < nc; q += kSelThreads) {
        const uint64_t v = cand_s[q];
        const int jq = cand_i[q];
        int r = 0;
        for (int o = 0; o < nc; ++o) {
          const uint64_t u = cand_s[o];
          r += (u > v) || (u == v && cand_i[o] < jq);
        }
        if (r < need) atomicOr(&gt[jq >> 5], 1u << (jq & 31));
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t y = __shfl_xor(mx, o, 64);
    mx = y > mx ? y : mx;
  }
  if (lane == 0) s_max[wid] = mx;
  __syncthreads();
  mx = 0ull;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) mx = s_max[w] > mx ? s_max[w] : mx;
  // theta = the K_s-th largest score; every wave tracks (prefix, remaining)
  uint64_t pre = 0ull, msk = 0ull;
  int rem = Ks;
  if (!fast && Ks > 0 && mx != 0ull) {
    const int top = (63 - __clzll((long long)mx)) >> 2;
    for (int d = top, par = 0; d >= 0; --d, par ^= 1) {
      // per-lane digit counts packed as 16-bit fields: digit q lives in
      // word q >> 2, bits 16 (q & 3) .. +15; summed over the wave's lanes
      // (at most 64 * PER < 2^16 per digit)
      uint64_t pk[4] = {0ull, 0ull, 0ull, 0ull};
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const bool m = live[i] && (sv[i] & msk) == pre;
        const int dig = (int)((sv[i] >> (4 * d)) & 15ull);
        const uint64_t inc = m ? (1ull << (16 * (dig & 3))) : 0ull;
#pragma unroll
        for (int q = 0; q < 4; ++q) pk[q] += (dig >> 2) == q ? inc : 0ull;
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1)
#pragma unroll
        for (int q = 0; q < 4; ++q) pk[q] += __shfl_xor(pk[q], o, 64);
      // lane b < 16: this wave's count of digit b
      int mine = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if ((lane >> 2) == q) mine = (int)((pk[q] >> (16 * (lane & 3))) & 0xFFFFull);
      if (lane < 16) cnt[par][wid][lane] = mine;
      __syncthreads();
      // lane l < 16 holds digit 15 - l; an inclusive scan over the lanes
      // counts the candidates at or above each digit
      const int b = 15 - (lane & 15);
      int c = 0;
#pragma unroll
      for (int w = 0; w < kSelWaves; ++w) c += cnt[par][w][b];
      c = lane < 16 ? c : 0;
      int incl = c;
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        const int y = __shfl_up(incl, o, 64);
        if (lane >= o) incl += y;
      }
      const uint64_t hit = __ballot(lane < 16 && incl >= rem);
      const int L = __ffsll((long long)hit) - 1;
      const int above = __shfl(incl - c, L, 64);
      pre |= (uint64_t)(15 - L) << (4 * d);
      rem -= above;
      msk |= 15ull << (4 * d);
    }
  }
  const uint64_t theta = pre;
  const int take_eq = (Ks > 0 && !fast) ? rem : 0;   // channels equal to theta to keep
  if (Ks > 0 && !fast) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int j = tid + kSelThreads * i;
      if (live[i]) {
        if (sv[i] > theta) atomicOr(&gt[j >> 5], 1u << (j & 31));
        else if (sv[i] == theta) atomicOr(&eq[j >> 5], 1u << (j & 31));
      }
    }
  }
  __syncthreads();
  // nw <= 512 words: two per thread (2 tid, 2 tid + 1), scanned as a pair
  uint32_t e2[2], w2[2];
  int ce = 0;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int w = 2 * tid + q;
    e2[q] = w < nw ? eq[w] : 0u;
    w2[q] = w < nw ? gt[w] : 0u;
    ce += __popc(e2[q]);
  }
  int tot;
  int eq_before = block_exclusive_scan(ce, sh, tot);
  int cw = 0;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    int need = take_eq - eq_before;
    uint32_t m = e2[q];
    eq_before += __popc(m);
    while (need > 0 && m) {
      w2[q] |= m & (0u - m);        // lowest remaining equal channel
      m &= m - 1u;
      --need;
    }
    cw += __popc(w2[q]);
  }
  int pos = block_exclusive_scan(cw, sh, tot);
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int w = 2 * tid + q;
    if (w < nw) {
      bitmap[w] = w2[q];
      uint32_t m = w2[q];
      while (m) {
        sel_idx[pos++] = w * 32 + (__ffs(m) - 1);
        m &= m - 1u;
      }
    }
  }
}

// Selection by rank for K <= kRankSelMaxK, one 1024-thread workgroup per
// 16-channel block (the layer's fused path for few rows per expert).
// Workgroup g ranks channels 16 g .. 16 g + 15 against all K channels in
// (score desc, index asc) order: rank(c) = #{j : s_j > s_c, or s_j == s_c
// and j < c}.  The ranks are a permutation of 0..K-1, so the channels of
// rank < K_s are exactly the K_s the threshold selection above takes (top
// K_s by score, ties to the lower index).  The workgroup stores its 16 bits
// of the bitmap, then (rcodes not NULL) quantises the residual of its column
// block for every row and masks it (the block arithmetic of rac_resq_body).  64 threads
// share a channel: thread (part p, channel o) counts over the channels
// j = p (mod 64) of a copy of the scores in LDS, so the four parts of a
// wave read four consecutive scores per step.
constexpr int kRankSelMaxK = 4096;
constexpr int kRankSelThreads = 1024;

__device__ __forceinline__ void rac_rank_select_body(
    int g, const uint64_t *__restrict__ scores, int K, int Ks, uint32_t *__restrict__ bitmap,
    const uint16_t *__restrict__ x, const uint8_t *__restrict__ xcodes,
    const uint8_t *__restrict__ xscales, const float *__restrict__ xgs, int64_t T,
    const float *__restrict__ ramax, uint8_t *__restrict__ rcodes, uint8_t *__restrict__ rscales,
    float *__restrict__ rgs) {
  constexpr int NT = kRankSelThreads, NP = NT / 16, NW = NT / 64;
  __shared__ uint64_t sk[kRankSelMaxK];
  __shared__ int red[NW][16];
  __shared__ uint32_t s_bits;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  for (int i = tid; i < K; i += NT) sk[i] = scores[i];
  __syncthreads();
  const int own = tid & 15, part = tid >> 4;
  const int c = 16 * g + own;
  const uint64_t sc = c < K ? sk[c] : 0ull;
  int r = 0;
  int j = part;
  for (; j + NP * 3 < K; j += NP * 4) {
    uint64_t u[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) u[q] = sk[j + NP * q];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int jq = j + NP * q;
      r += (int)((u[q] > sc) | ((u[q] == sc) & (jq < c)));
    }
  }
  for (; j < K; j += NP) {
    const uint64_t u = sk[j];
    r += (int)((u > sc) | ((u == sc) & (j < c)));
  }
  // sum over the four parts of the wave (lanes own + 16 i), then the waves
  r += __shfl_xor(r, 16, 64);
  r += __shfl_xor(r, 32, 64);
  if (lane < 16) red[wid][own] = r;
  __syncthreads();
  if (wid == 0) {
    int rank = 0;
    if (lane < 16)
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) rank += red[ww][own];
    const uint32_t b = (uint32_t)__ballot(lane < 16 && c < K && rank < Ks) & 0xFFFFu;
    if (lane == 0) {
      reinterpret_cast<uint16_t *>(bitmap)[g] = (uint16_t)b;
      s_bits = b;
    }
  }
  __syncthreads();
  if (!rcodes) return;                  // selection only (the compact residual follows)
  // the masked residual of column block g
  const uint32_t m16 = s_bits;
  const float amax_r = ramax[0];
  float s_enc, s_dec;
  tensor_scale(amax_r, s_enc, s_dec);
  const bool zero_tensor = !(amax_r >= kZeroAmax);
  if (g == 0 && tid == 0) {
    rgs[0] = s_enc;
    rgs[1] = s_dec;
  }
  const float xs_dec = xgs[1];
  const int64_t nbc = K >> 4;
  uint32_t mlo = 0u, mhi = 0u;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    if ((m16 >> i) & 1u) mlo |= 15u << (4 * i);
    if ((m16 >> (i + 8)) & 1u) mhi |= 15u << (4 * i);
  }
  for (int64_t t = tid; t < T; t += NT) {
    const int64_t bi = t * nbc + g;
    uint32_t lo = 0u, hi = 0u, sb = 0u;
    if (m16) {
      float v[16], rr[16];
      load_bf16x16(x + bi * 16, v);
      block_residual(v, reinterpret_cast<const uint2 *>(xcodes)[bi], xscales[bi], xs_dec, rr);
      sb = quantize_block(rr, s_enc, zero_tensor, lo, hi);
      lo &= mlo;
      hi &= mhi;
    }
    reinterpret_cast<uint2 *>(rcodes)[bi] = make_uint2(lo, hi);
    rscales[bi] = (uint8_t)sb;
  }
}

// S in ascending order from the selection bitmap (K <= 8192, at most one
// word per thread of a 256-thread workgroup) into `out` (LDS or global).
// Every thread of the workgroup calls it; sh: 1024 + 32 ints of LDS.
__device__ __forceinline__ void rac_list_selected(const uint32_t *__restrict__ bitmap, int K,
                                                  int32_t *out, int *sh) {
  const int tid = threadIdx.x;
  const int nw = (K + 31) >> 5;
  uint32_t m = tid < nw ? bitmap[tid] : 0u;
  if (tid == nw - 1 && (K & 31)) m &= (1u << (K & 31)) - 1u;
  int tot;
  int pos = block_exclusive_scan(__popc(m), sh, tot);
  while (m) {
    out[pos++] = tid * 32 + (__ffs(m) - 1);
    m &= m - 1u;
  }
}

// Masked residual quantisation: one thread per 16-element block of [T][K];
// workgroup bid of nblk.
__device__ __forceinline__ void rac_resq_body(
    int bid, int nblk, const uint16_t *__restrict__ x, const uint8_t *__restrict__ xcodes,
    const uint8_t *__restrict__ xscales, const float *__restrict__ xgs, int64_t T, int64_t K,
    const float *__restrict__ ramax, const uint32_t *__restrict__ bitmap,
    uint8_t *__restrict__ rcodes, uint8_t *__restrict__ rscales, float *__restrict__ rgs) {
  const float amax_r = ramax[0];
  float s_enc, s_dec;
  tensor_scale(amax_r, s_enc, s_dec);
  const bool zero_tensor = !(amax_r >= kZeroAmax);
  if (bid == 0 && threadIdx.x == 0) {
    rgs[0] = s_enc;
    rgs[1] = s_dec;
  }
  const float xs_dec = xgs[1];
  const int64_t nbc = K >> 4;
  const int64_t total = T * nbc;
  const int64_t stride = (int64_t)nblk * blockDim.x;
  for (int64_t b = (int64_t)bid * blockDim.x + threadIdx.x; b < total; b += stride) {
    const int64_t cb = b % nbc;
    const uint32_t m16 = (bitmap[cb >> 1] >> (16 * (cb & 1))) & 0xFFFFu;
    uint32_t lo = 0u, hi = 0u, sb = 0u;
    if (m16) {
      const int64_t t = b / nbc;
      float v[16], r[16];
      load_bf16x16(x + t * K + cb * 16, v);
      uint2 cw = reinterpret_cast<const uint2 *>(xcodes)[b];
      block_residual(v, cw, xscales[b], xs_dec, r);
      sb = quantize_block(r, s_enc, zero_tensor, lo, hi);
      uint32_t mlo = 0u, mhi = 0u;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        if ((m16 >> i) & 1u) mlo |= 15u << (4 * i);
        if ((m16 >> (i + 8)) & 1u) mhi |= 15u << (4 * i);
      }
      lo &= mlo;
      hi &= mhi;
    }
    reinterpret_cast<uint2 *>(rcodes)[b] = make_uint2(lo, hi);
    rscales[b] = (uint8_t)sb;
  }
}

// The masked residual at the selected channels only, compacted per token:
// out[t][j] = e2m1 * e4m3 value (no tensor scale, exact in f16) of channel
// sel[j] in the residual quantised over all channels (the same block
// arithmetic as rac_resq_body, evaluated for the blocks that hold a selected
// channel), 0 for Ks <= j < width.  Also writes the residual's tensor scale.
// Work item i of T * width; workgroup bid of nblk.
__device__ __forceinline__ void rac_compact_body(
    int bid, int nblk, const uint16_t *__restrict__ x, const uint8_t *__restrict__ xcodes,
    const uint8_t *__restrict__ xscales, const float *__restrict__ xgs, int64_t T, int64_t K,
    const float *__restrict__ ramax, const int32_t *__restrict__ sel, int Ks, int width,
    uint16_t *__restrict__ out, float *__restrict__ rgs) {
  const float amax_r = ramax[0];
  float s_enc, s_dec;
  tensor_scale(amax_r, s_enc, s_dec);
  const bool zero_tensor = !(amax_r >= kZeroAmax);
  if (bid == 0 && threadIdx.x == 0) {
    rgs[0] = s_enc;
    rgs[1] = s_dec;
  }
  const float xs_dec = xgs[1];
  const int64_t nbc = K >> 4;
  const int64_t total = T * width;
  const int64_t stride = (int64_t)nblk * blockDim.x;
  for (int64_t i = (int64_t)bid * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int64_t t = i / width;
    const int j = (int)(i - t * width);
    float v = 0.0f;
    if (j < Ks) {
      const int c = sel[j];
      const int64_t b = t * nbc + (c >> 4);
      float xv[16], r[16];
      load_bf16x16(x + b * 16, xv);
      block_residual(xv, reinterpret_cast<const uint2 *>(xcodes)[b], xscales[b], xs_dec, r);
      uint32_t lo, hi;
      const uint32_t sb = quantize_block(r, s_enc, zero_tensor, lo, hi);
      const int e = c & 15;
      const uint32_t code = ((e < 8 ? lo : hi) >> (4 * (e & 7))) & 15u;
      v = e2m1_value(code) * e4m3_to_f32(sb);
      if (code & 8u) v = -v;
    }
    out[i] = __builtin_bit_cast(uint16_t, (_Float16)v);
  }
}

}  // namespace qdc

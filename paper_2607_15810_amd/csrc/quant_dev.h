// Device bodies of the activation quantiser Q_A (Sec. 2.2 "FP4"; Eq.
// (act-error-def)) with the fused RAC statistics (Eq. (residual-def),
// Eq. (channel-score)): launched alone by quant.hip, or fused with the
// routing work by the layer.
#pragma once
#include "common.h"

namespace qdq {

using namespace qd;

template <typename T> struct Loader;
// load_raw brings 16 consecutive elements starting at element index i
// (16-aligned) into registers as stored; unpack widens them to float, so a
// caller can keep the next block's load in flight while it works on this one.
template <> struct Loader<uint16_t> {   // bf16 storage
  struct Raw {
    uint4 a, b;
  };
  __device__ static void load_raw(const void *base, int64_t i, Raw &r) {
    const uint4 *p = reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(base) + i);
    r.a = p[0];
    r.b = p[1];
  }
  __device__ static void unpack(const Raw &r, float (&x)[16]) {
    const uint32_t w[8] = {r.a.x, r.a.y, r.a.z, r.a.w, r.b.x, r.b.y, r.b.z, r.b.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      x[2 * j] = __uint_as_float(w[j] << 16);
      x[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
    }
  }
  __device__ static void load16(const void *base, int64_t i, float (&x)[16]) {
    Raw r;
    load_raw(base, i, r);
    unpack(r, x);
  }
};
template <> struct Loader<float> {
  struct Raw {
    float4 q[4];
  };
  __device__ static void load_raw(const void *base, int64_t i, Raw &r) {
    const float4 *p = reinterpret_cast<const float4 *>(static_cast<const float *>(base) + i);
#pragma unroll
    for (int j = 0; j < 4; ++j) r.q[j] = p[j];
  }
  __device__ static void unpack(const Raw &r, float (&x)[16]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[4 * j] = r.q[j].x; x[4 * j + 1] = r.q[j].y; x[4 * j + 2] = r.q[j].z;
      x[4 * j + 3] = r.q[j].w;
    }
  }
  __device__ static void load16(const void *base, int64_t i, float (&x)[16]) {
    Raw r;
    load_raw(base, i, r);
    unpack(r, x);
  }
};

// Per-workgroup max|x| over a flat array of n16 16-element blocks; also zeroes
// the RAC statistics buffers when given (they are accumulated by the next
// kernel on the same stream).
// Workgroup bid of nblk.
template <typename T>
__device__ __forceinline__ void amax_partial_body(int bid, int nblk, const void *__restrict__ x,
                                                  int64_t n16, float *__restrict__ part,
                                                  uint64_t *__restrict__ zero_u64,
                                                  int64_t n_zero_u64,
                                                  float *__restrict__ zero_f32) {
  __shared__ float red[16];
  float m = 0.0f;
  const int64_t stride = (int64_t)nblk * blockDim.x;
  for (int64_t b = (int64_t)bid * blockDim.x + threadIdx.x; b < n16; b += stride) {
    float v[16];
    Loader<T>::load16(x, b * 16, v);
#pragma unroll
    for (int i = 0; i < 16; ++i) m = fmaxf(m, fabsf(v[i]));
  }
  if (zero_u64) {
    for (int64_t i = (int64_t)bid * blockDim.x + threadIdx.x; i < n_zero_u64; i += stride)
      zero_u64[i] = 0ull;
  }
  if (zero_f32 && bid == 0 && threadIdx.x == 0) zero_f32[0] = 0.0f;
  m = block_max(m, red);
  if (threadIdx.x == 0) part[bid] = m;
}

// Q_A over [rows][cols] on a (gx, gy) grid of workgroups; this is
// workgroup (bx, by).  Thread (tx, ty) of a 16x16 workgroup owns column block
// (bx*16 + tx) and rows ty, ty+16*gy, ...  With RAC the same pass forms
// r = x_hat - x and accumulates the fixed-point channel scores (u64, order
// independent) and max|r|.
// The LDS it uses comes from the caller: red (16 floats) and, with RAC, part
// (16 x 272 u64), so that a kernel fusing it with other work can overlay
// the two bodies' arrays.
constexpr int kQuantPartCols = 16 * 17;
constexpr int kQuantLdsBytes = 16 * kQuantPartCols * 8 + 16 * 4;
template <typename T, bool RAC>
__device__ __forceinline__ void quantize_act_rows(
    int bx, int by, int gy, const void *__restrict__ x, int64_t rows, int64_t cols,
    const float *__restrict__ amax_part, int n_part, uint8_t *__restrict__ codes,
    uint8_t *__restrict__ scales, float *__restrict__ gscale, uint64_t *__restrict__ scores,
    float *__restrict__ ramax, uint64_t (*part)[kQuantPartCols], float *red) {
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  // tensor amax from the partial maxima
  const float amax = block_max(partials_max(amax_part, n_part), red);
  float s_enc, s_dec;
  tensor_scale(amax, s_enc, s_dec);
  const bool zero_tensor = !(amax >= kZeroAmax);
  if (bx == 0 && by == 0 && threadIdx.x == 0) {
    gscale[0] = s_enc;
    gscale[1] = s_dec;
  }
  const int64_t nbc = cols >> 4;
  const int64_t cb = (int64_t)bx * 16 + tx;
  const bool active = cb < nbc;

  int F = 0;
  if (RAC) {
    int e;
    frexpf(amax, &e);
    F = 36 - 2 * e;
  }
  // per-thread score sums: exact integer sums in double (cheaper per term
  // than 64-bit integer shifts), at most kScoreMaxRows terms each
  double accd[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) accd[i] = 0.0;
  float rmax = 0.0f;

  if (active) {
    const int64_t step = (int64_t)gy * 16;
    int64_t r = (int64_t)by * 16 + ty;
    // with RAC (the longer row body) the thread's next row is loaded while
    // this one is quantised
    typename Loader<T>::Raw cur = {}, nxt = {};
    if (RAC && r < rows) Loader<T>::load_raw(x, r * cols + cb * 16, cur);
    for (; r < rows; r += step) {
      if (!RAC) Loader<T>::load_raw(x, r * cols + cb * 16, cur);
      else if (r + step < rows) Loader<T>::load_raw(x, (r + step) * cols + cb * 16, nxt);
      float v[16];
      Loader<T>::unpack(cur, v);
      uint32_t lo, hi;
      uint32_t sb = quantize_block(v, s_enc, zero_tensor, lo, hi);
      reinterpret_cast<uint2 *>(codes + r * (cols >> 1))[cb] = make_uint2(lo, hi);
      scales[r * nbc + cb] = (uint8_t)sb;
      if (RAC) {
        // x_hat = fl(fl(e2m1 * e4m3) * s_dec), as dequant_value
        const float sbf = e4m3_to_f32(sb);
        float ev[16];
        e2m1_word_values(lo, ev);
        e2m1_word_values(hi, ev + 8);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          float xh = (ev[i] * sbf) * s_dec;
          float rr = xh - v[i];
          rmax = fmaxf(rmax, fabsf(rr));
          accd[i] += fixed_point_term_f64(rr * rr, F);   // each term < 2^37
        }
      }
      if (RAC) cur = nxt;
    }
  }
  if (RAC) {
    // reduce the per-thread sums over ty, then one atomic per channel
    // (channel 16 tx + i of row ty at 17 i + tx: consecutive tx are
    // adjacent when written, and consecutive channels 17 apart when read)
#pragma unroll
    for (int i = 0; i < 16; ++i) part[ty][17 * i + tx] = score_sum_u64(accd[i]);
    __syncthreads();
    uint64_t s = 0;
    const int rd = 17 * (threadIdx.x & 15) + (threadIdx.x >> 4);
#pragma unroll
    for (int j = 0; j < 16; ++j) s += part[j][rd];
    const int64_t ch = (int64_t)bx * 256 + threadIdx.x;
    if (ch < cols && s != 0ull) atomicAdd((unsigned long long *)&scores[ch], (unsigned long long)s);
    float m = block_max(rmax, red);
    if (threadIdx.x == 0 && m > 0.0f)
      atomic_max_pos(ramax, m);
  }
}

// quantize_act_rows with LDS arrays of its own
template <typename T, bool RAC>
__device__ __forceinline__ void quantize_act_body(
    int bx, int by, int gy, const void *__restrict__ x, int64_t rows, int64_t cols,
    const float *__restrict__ amax_part, int n_part, uint8_t *__restrict__ codes,
    uint8_t *__restrict__ scales, float *__restrict__ gscale, uint64_t *__restrict__ scores,
    float *__restrict__ ramax) {
  __shared__ float red[16];
  __shared__ uint64_t part[RAC ? 16 : 1][kQuantPartCols];
  quantize_act_rows<T, RAC>(bx, by, gy, x, rows, cols, amax_part, n_part, codes, scales, gscale,
                            scores, ramax, part, red);
}

constexpr int kAmaxPartials = 1024;     // per-call partial maxima (workspace)

// workgroups of the amax pass over n16 16-element blocks
inline int amax_grid(int64_t n16) {
  int64_t g = (n16 + 255) / 256;
  return (int)(g < kAmaxPartials ? (g < 1 ? 1 : g) : kAmaxPartials);
}

// (gx, gy) grid of the quantiser: 16 column blocks per workgroup along x;
// with RAC at most 1024 workgroups (one u64 atomic per channel and workgroup)
inline void quant_grid(int64_t rows, int64_t cols, bool rac, int &gx, int &gy) {
  const int64_t nbc = cols / 16;
  gx = (int)((nbc + 15) / 16);
  int64_t g = (rows + 15) / 16;
  const int64_t cap = rac ? 1024 : 4096;
  int64_t lim = cap / gx;
  if (lim < 1) lim = 1;
  if (g > lim) g = lim;
  // at most kScoreMaxRows rows per thread (the exact double score sums)
  const int64_t need = (rows + 16 * kScoreMaxRows - 1) / (16 * kScoreMaxRows);
  if (g < need) g = need;
  gy = (int)g;
}

}  // namespace qdq

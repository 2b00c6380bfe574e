// Device bodies of the activation quantiser Q_A (Sec. 2.2 "FP4"; Eq.
// (act-error-def)) with the fused RAC statistics (Eq. (residual-def),
// Eq. (channel-score)): launched alone by quant.hip, or fused with the
// routing work by the layer.
#pragma once
#include "common.h"

namespace qdq {

using namespace qd;

template <typename T> struct Loader;
template <> struct Loader<uint16_t> {   // bf16 storage
  // 16 consecutive elements starting at element index i (16-aligned)
  __device__ static void load16(const void *base, int64_t i, float (&x)[16]) {
    const uint4 *p = reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(base) + i);
    uint4 a = p[0], b = p[1];
    uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      x[2 * j] = __uint_as_float(w[j] << 16);
      x[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
    }
  }
};
template <> struct Loader<float> {
  __device__ static void load16(const void *base, int64_t i, float (&x)[16]) {
    const float4 *p = reinterpret_cast<const float4 *>(static_cast<const float *>(base) + i);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float4 v = p[j];
      x[4 * j] = v.x; x[4 * j + 1] = v.y; x[4 * j + 2] = v.z; x[4 * j + 3] = v.w;
    }
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

// trunc(sq * 2^F) as uint64 for a finite float sq >= 0, exactly (what the
// float64 product and truncation give): sq = m * 2^x with m the integer
// significand, so the result is m shifted by x + F.
__device__ __forceinline__ uint64_t fixed_point_term(float sq, int F) {
  const uint32_t bits = __float_as_uint(sq);
  const uint32_t be = bits >> 23;
  const uint64_t m = be ? ((bits & 0x7FFFFFu) | 0x800000u) : (bits & 0x7FFFFFu);
  const int sh = (be ? (int)be - 150 : -149) + F;
  if (sh >= 0) return m << sh;
  return sh > -64 ? m >> (-sh) : 0ull;
}

// Q_A over [rows][cols] on a (gx, gy) grid of workgroups; this is
// workgroup (bx, by).  Thread (tx, ty) of a 16x16 workgroup owns column block
// (bx*16 + tx) and rows ty, ty+16*gy, ...  With RAC the same pass forms
// r = x_hat - x and accumulates the fixed-point channel scores (u64, order
// independent) and max|r|.
template <typename T, bool RAC>
__device__ __forceinline__ void quantize_act_body(
    int bx, int by, int gy, const void *__restrict__ x, int64_t rows, int64_t cols,
    const float *__restrict__ amax_part, int n_part, uint8_t *__restrict__ codes,
    uint8_t *__restrict__ scales, float *__restrict__ gscale, uint64_t *__restrict__ scores,
    float *__restrict__ ramax) {
  __shared__ float red[16];
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
  uint64_t acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0ull;
  float rmax = 0.0f;

  if (active) {
    for (int64_t r = (int64_t)by * 16 + ty; r < rows; r += (int64_t)gy * 16) {
      float v[16];
      Loader<T>::load16(x, r * cols + cb * 16, v);
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
          acc[i] += fixed_point_term(rr * rr, F);   // each term < 2^37
        }
      }
    }
  }
  if (RAC) {
    // reduce the per-thread sums over ty, then one atomic per channel
    // (channel 16 tx + i of row ty at 17 i + tx: consecutive tx are
    // adjacent when written, and consecutive channels 17 apart when read)
    __shared__ uint64_t part[16][16 * 17];
#pragma unroll
    for (int i = 0; i < 16; ++i) part[ty][17 * i + tx] = acc[i];
    __syncthreads();
    uint64_t s = 0;
    const int rd = 17 * (threadIdx.x & 15) + (threadIdx.x >> 4);
#pragma unroll
    for (int j = 0; j < 16; ++j) s += part[j][rd];
    const int64_t ch = (int64_t)bx * 256 + threadIdx.x;
    if (ch < cols && s != 0ull) atomicAdd((unsigned long long *)&scores[ch], (unsigned long long)s);
    float m = block_max(rmax, red);
    if (threadIdx.x == 0 && m > 0.0f)
      atomicMax(reinterpret_cast<unsigned int *>(ramax), __float_as_uint(m));
  }
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
  gy = (int)g;
}

}  // namespace qdq

// Shared device helpers for the gfx950 kernels of libquads.so.
//
// Number formats (paper, Sec. 2.2 "FP4" paragraph): E2M1 element codes
// (magnitudes 0, .5, 1, 1.5, 2, 3, 4, 6; sign in bit 3), one E4M3FN scale per
// 16 consecutive elements, and an FP32 tensor scale pair {s_enc, s_dec}.
// Every helper here is exact or rounds once to nearest even, so the GPU
// reproduces the quantiser's codes bit for bit.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "../../include/quads.h"

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace qd {

constexpr int kBlock = 16;              // NVFP4 block length
constexpr float kZeroAmax = 7.8886090522101181e-31f;   // 2^-100

// ---------------------------------------------------------------- bf16
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) {
  return __uint_as_float(b << 16);
}
// Round to nearest even; inputs are finite.
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// ---------------------------------------------------------------- E4M3FN
// t in [0, 448]: nearest E4M3FN code, ties to the even code.
__device__ __forceinline__ uint32_t e4m3_encode_pos(float t) {
  if (t < 0.015625f) {                    // below 2^-6: multiples of 2^-9
    return (uint32_t)__builtin_rintf(t * 512.0f);   // 0..8 (8 is 2^-6)
  }
  uint32_t u = __float_as_uint(t);
  uint32_t r = u + 0x7FFFFu + ((u >> 20) & 1u);     // keep 3 mantissa bits
  return (((r >> 23) - 120u) << 3) | ((r >> 20) & 7u);
}
__device__ __forceinline__ float e4m3_to_f32(uint32_t b) {   // sign bit 0
  uint32_t e = (b >> 3) & 15u, m = b & 7u;
  if (e == 0) return (float)m * 0.001953125f;                 // m * 2^-9
  return __uint_as_float(((e + 120u) << 23) | (m << 20));
}

// ---------------------------------------------------------------- E2M1
// |v| -> magnitude index, round to nearest, ties to even, saturating at 6.
__device__ __forceinline__ uint32_t e2m1_mag(float a) {
  return (uint32_t)(a > 0.25f) + (uint32_t)(a >= 0.75f) + (uint32_t)(a > 1.25f) +
         (uint32_t)(a >= 1.75f) + (uint32_t)(a > 2.5f) + (uint32_t)(a >= 3.5f) +
         (uint32_t)(a > 5.0f);
}
// magnitude index -> value (exact float)
__device__ __forceinline__ float e2m1_value(uint32_t c) {
  c &= 7u;
  if (c == 0) return 0.0f;
  uint32_t m = (c > 1u) ? (c & 1u) : 0u;
  return __uint_as_float(((126u + (c >> 1)) << 23) | (m << 22));
}

// ---------------------------------------------------------------- scales
// Tensor scale pair from the tensor amax (zero-tensor guard below 2^-100).
__device__ __forceinline__ void tensor_scale(float amax, float &s_enc, float &s_dec) {
  if (!(amax >= kZeroAmax)) { s_enc = 1.0f; s_dec = 1.0f; return; }
  s_enc = 2688.0f / amax;
  s_dec = 1.0f / s_enc;
}

// Quantise one 16-element block held in registers.  Writes 8 packed code
// bytes (two uint32) and returns the E4M3 scale byte.  Used by every
// quantiser in the library so their arithmetic is one sequence:
//   t = fl(fl(a_b / 6) * s_enc), sb = E4M3(min(t, 448)),
//   enc = s_enc / value(sb) (0 if sb == 0), v = fl(x * enc), code = RNE(|v|).
__device__ __forceinline__ uint32_t quantize_block(const float (&x)[16], float s_enc,
                                                   bool zero_tensor, uint32_t &lo,
                                                   uint32_t &hi) {
  float ab = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) ab = fmaxf(ab, fabsf(x[i]));
  uint32_t sb = 0;
  float enc = 0.0f;
  if (!zero_tensor) {
    float t = (ab / 6.0f) * s_enc;
    t = fminf(t, 448.0f);
    sb = e4m3_encode_pos(t);
    float sbf = e4m3_to_f32(sb);
    enc = (sb == 0) ? 0.0f : s_enc / sbf;
  }
  // code = E2M1_RNE(|v|) (ties to even, saturating at 6) with the sign of
  // v, which is the sign of x (enc >= 0): the hardware conversion with a
  // unit scale, two elements per instruction, element 2j in the low nibble
  // (checked against e2m1_mag on every rounding threshold and 2M values)
  uint32_t lo_w = 0u, hi_w = 0u;
  lo_w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(lo_w, x[0] * enc, x[1] * enc, 1.0f, 0);
  lo_w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(lo_w, x[2] * enc, x[3] * enc, 1.0f, 1);
  lo_w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(lo_w, x[4] * enc, x[5] * enc, 1.0f, 2);
  lo_w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(lo_w, x[6] * enc, x[7] * enc, 1.0f, 3);
  hi_w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(hi_w, x[8] * enc, x[9] * enc, 1.0f, 0);
  hi_w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(hi_w, x[10] * enc, x[11] * enc, 1.0f, 1);
  hi_w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(hi_w, x[12] * enc, x[13] * enc, 1.0f, 2);
  hi_w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(hi_w, x[14] * enc, x[15] * enc, 1.0f, 3);
  lo = lo_w;
  hi = hi_w;
  return sb;
}

// Q8 value of one code: fl(fl(e2m1 * sbf) * s_dec); the first product is exact.
// The 8 codes of a word (element j in bits 4j .. 4j+3) as their exact signed
// E2M1 values: the hardware conversion with a unit scale, two per
// instruction.
typedef float f32x2_pair __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void e2m1_word_values(uint32_t w, float *v) {
  const f32x2_pair p0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 0);
  const f32x2_pair p1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 1);
  const f32x2_pair p2 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 2);
  const f32x2_pair p3 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 3);
  v[0] = p0[0]; v[1] = p0[1]; v[2] = p1[0]; v[3] = p1[1];
  v[4] = p2[0]; v[5] = p2[1]; v[6] = p3[0]; v[7] = p3[1];
}

__device__ __forceinline__ float dequant_value(uint32_t code, float sbf, float s_dec) {
  float p = e2m1_value(code) * sbf;
  p = (code & 8u) ? -p : p;
  return p * s_dec;
}

// ---------------------------------------------------------------- MFMA operand decode
// E4M3 scale byte -> f16 bit pattern of value/256 (exact, possibly subnormal):
// shifting the 7 magnitude bits into an f16 exponent/mantissa field keeps the
// value up to a factor 2^-8 for normals and subnormals alike.
__device__ __forceinline__ uint32_t scale_pair_f16(uint32_t s0, uint32_t s1) {
  return (s0 << 7) | (s1 << 23);
}

// 8 E2M1 codes (one uint32, element 0 in bits 3:0) and one f16 scale factor
// (value/256) -> 8 exact f16 operands e2m1 * e4m3.  The scaled convert
// multiplies by a power of two only (256 here); the E4M3 mantissa enters
// through one exact packed f16 multiply.
__device__ __forceinline__ f16x8 decode8(uint32_t codes, f16x2 sc) {
  f16x2 p0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, 256.0f, 0);
  f16x2 p1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, 256.0f, 1);
  f16x2 p2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, 256.0f, 2);
  f16x2 p3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, 256.0f, 3);
  p0 *= sc; p1 *= sc; p2 *= sc; p3 *= sc;
  f16x8 r;
  r[0] = p0[0]; r[1] = p0[1]; r[2] = p1[0]; r[3] = p1[1];
  r[4] = p2[0]; r[5] = p2[1]; r[6] = p3[0]; r[7] = p3[1];
  return r;
}

// The two E4M3 scale bytes 2c, 2c+1 of a scale dword as an f16 pair
// (value/256 each, as scale_pair_f16): one byte permute and one shift.
__device__ __forceinline__ f16x2 scale_pair_of(uint32_t sdw, int c) {
  const uint32_t v = __builtin_amdgcn_perm(0u, sdw, c ? 0x0C030C02u : 0x0C010C00u);
  return __builtin_bit_cast(f16x2, v << 7);
}
// decode8 with the scale taken from the low (hi = false) or high half of a
// pair; the half is selected by the packed multiply's operand selection
__device__ __forceinline__ f16x8 decode8_sel(uint32_t codes, f16x2 pair, bool hi) {
  const f16x2 sc = hi ? __builtin_shufflevector(pair, pair, 1, 1)
                      : __builtin_shufflevector(pair, pair, 0, 0);
  return decode8(codes, sc);
}

__device__ __forceinline__ f16x2 splat_lo(uint32_t pair) {
  uint32_t v = (pair & 0xFFFFu) | (pair << 16);
  return __builtin_bit_cast(f16x2, v);
}
__device__ __forceinline__ f16x2 splat_hi(uint32_t pair) {
  uint32_t v = (pair >> 16) | (pair & 0xFFFF0000u);
  return __builtin_bit_cast(f16x2, v);
}

// ---------------------------------------------------------------- reductions
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// The channel-score term trunc(sq * 2^F) (what the float64 product and
// truncation give), for a finite sq >= 0 whose term is below 2^37, computed in
// floating point: sq * 2^F is exact in float wherever it is >= 1 (a
// power-of-two scaling of a normal value into the normal range), anything
// below 1 truncates to 0 either way, and the integer result is exact in
// double, where sums of up to kScoreMaxRows such terms stay exact.
// score_sum_u64 converts such a sum; its clamp only keeps the sum of a
// non-finite input's terms in range.
constexpr int64_t kScoreMaxRows = 1 << 16;
__device__ __forceinline__ double fixed_point_term_f64(float sq, int F) {
  return (double)truncf(ldexpf(sq, F));
}
__device__ __forceinline__ uint64_t score_sum_u64(double d) {
  return (uint64_t)fmin(d, 9007199254740992.0);   // 2^53
}

// max(*addr, m) for finite m >= 0 into a float >= 0 that many workgroups
// update at the end of a kernel: the device-coherent value is read first and
// the atomic is issued only when m exceeds it.  The stored value only grows
// during the kernel, so a skipped update is already covered; at one address
// this removes most of the serialised atomics.
__device__ __forceinline__ void atomic_max_pos(float *addr, float m) {
  unsigned int *a = reinterpret_cast<unsigned int *>(addr);
  const unsigned int cur = __hip_atomic_load(a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (__float_as_uint(m) > cur) atomicMax(a, __float_as_uint(m));
}

// This thread's max over the n partial maxima (>= 0) at p, taken in steps of
// blockDim.x: sixteen independent loads in flight per thread, so one round
// trip to memory covers up to sixteen values per thread (the partials are read
// once at the start of a kernel, where that latency is the kernel's critical
// path).
__device__ __forceinline__ float partials_max(const float *__restrict__ p, int64_t n) {
  float m = 0.0f;
  const int64_t st = blockDim.x;
  for (int64_t i = threadIdx.x; i < n; i += 16 * st) {
    float v[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) v[j] = i + j * st < n ? p[i + j * st] : 0.0f;
#pragma unroll
    for (int j = 0; j < 16; ++j) m = fmaxf(m, v[j]);
  }
  return m;
}

// Block-wide max over blockDim.x threads (multiple of 64, <= 1024).
__device__ __forceinline__ float block_max(float v, float *red /* >= 16 floats */) {
  v = wave_max(v);
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  if (lane == 0) red[wid] = v;
  __syncthreads();
  const int nw = blockDim.x >> 6;
  float r = (threadIdx.x < (unsigned)nw) ? red[threadIdx.x] : 0.0f;
  if (wid == 0) r = wave_max(r);
  if (threadIdx.x == 0) red[0] = r;
  __syncthreads();
  r = red[0];
  __syncthreads();
  return r;
}

}  // namespace qd

// ---------------------------------------------------------------- host-side helpers
namespace qdh {

inline bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

// Returns QD_ERR_HIP if the environment asks for an injected launch failure
// (QD_FAULT_INJECT=launch); lets host-only tests reach the error path.
qd_status fault_injected();

qd_status check_launch();

inline hipStream_t S(void *s) { return reinterpret_cast<hipStream_t>(s); }

inline size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

qd_status check_nvfp4(const qd_nvfp4 *t, int64_t groups, int64_t rows, int64_t cols);

}  // namespace qdh

// Internal launchers shared between translation units.
namespace qdi {
// Reduce n non-negative floats to their maximum, written to out[0] (1 workgroup).
void launch_reduce_max(const float *in, int64_t n, float *out, hipStream_t s);
// Fill n int32 with a value (a kernel, so it is safe inside captured graphs).
void launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s);
// Whether moe_w4a4_grouped_gemm on these sizes contracts the residual from
// its compact form (rq_sel).
bool gemm_wants_rq_sel(int64_t rows, int32_t E, int64_t N, int64_t K, int32_t Ks,
                       int32_t epilogue);
// Whether the grouped GEMM on these sizes takes the residual in bitmap mode
// (the decode kernel, K <= 4096).
bool gemm_takes_bitmap(int64_t rows, int32_t E, int64_t N, int64_t K, int32_t Ks,
                       int32_t epilogue);
// The number of amax partials the grouped GEMM's kernel on these sizes
// writes (its grid; moe_w4a4_grouped_gemm_amax_count is an upper bound over
// the kernels that could run); sfrag: the weights carry fragment-ordered
// scales; bitmap: the residual comes in bitmap mode.
int64_t gemm_amax_written(int64_t rows, int32_t E, int64_t N, int64_t K, int32_t Ks,
                          int32_t epilogue, bool sfrag, bool bitmap);
// moe_w4a4_grouped_gemm in bitmap mode: bitmap [K / 32] marks the selected
// channels S in place of a list; the decode kernel writes S in ascending
// order to sel_out.  QD_ERR_UNSUPPORTED where gemm_takes_bitmap is false.
qd_status grouped_gemm_bitmap(const qd_nvfp4 *a, const int32_t *row_token,
                              const int32_t *expert_offsets, int32_t E, int64_t rows,
                              const qd_nvfp4 *w, const qd_nvfp4 *rq, const uint32_t *bitmap,
                              int32_t Ks, int32_t *sel_out, int32_t epilogue, void *out,
                              float *amax_partials, hipStream_t stream);
// Bytes of the staged A operand the grouped GEMM reads on these sizes (the
// tile kernel with the residual, gathered rows and the A-scale ring): codes
// [K / 64][rows][32 B] then scales [K / 256][rows][16 B]; 0 where it reads the
// gathered rows directly.  gemm_stage_reserve: an upper bound over K_s >= 1.
int64_t gemm_stage_bytes(int64_t rows, int32_t E, int64_t N, int64_t K, int32_t Ks,
                         int32_t epilogue);
int64_t gemm_stage_reserve(int64_t rows, int32_t E, int64_t N, int64_t K, int32_t epilogue);
// moe_w4a4_grouped_gemm with the A operand also given staged (a_stg, as
// gemm_stage_bytes describes; the kernel falls back to the gathered rows
// where it does not use it).
qd_status grouped_gemm_staged(const qd_nvfp4 *a, const int32_t *row_token,
                              const int32_t *expert_offsets, int32_t E, int64_t rows,
                              const qd_nvfp4 *w, const qd_nvfp4 *rq, const int32_t *sel_idx,
                              int32_t Ks, const void *rq_sel, int32_t epilogue, void *out,
                              float *amax_partials, const uint8_t *a_stg, hipStream_t stream);
}  // namespace qdi

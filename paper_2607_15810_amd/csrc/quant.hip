// NVFP4 quantisation kernels: Q_A (activations, with the fused RAC channel
// statistics), Q_W (weights, one tensor scale per expert matrix) and the
// dequantiser used by the trainer-side fake-quant.
//
// Paper: Sec. 2.2 (the NVFP4 format), Eq. (act-error-def) / Eq. (residual-def)
// (activation QDQ and its residual), Eq. (weight-error-def) and
// Eq. (w4a16-qat-forward) (weight QDQ shared with the trainer), Eq.
// (channel-score) (per-channel residual norm, accumulated in the same pass).
#include "quant_dev.h"

namespace {

using namespace qd;
using qdq::Loader;

using qdq::kAmaxPartials;
using qdq::amax_grid;

template <typename T>
__global__ __launch_bounds__(256) void amax_partial_kernel(const void *__restrict__ x,
                                                           int64_t n16, float *__restrict__ part,
                                                           uint64_t *__restrict__ zero_u64,
                                                           int64_t n_zero_u64,
                                                           float *__restrict__ zero_f32) {
  qdq::amax_partial_body<T>(blockIdx.x, gridDim.x, x, n16, part, zero_u64, n_zero_u64, zero_f32);
}

template <typename T, bool RAC>
__global__ __launch_bounds__(256) void quantize_act_kernel(
    const void *__restrict__ x, int64_t rows, int64_t cols, const float *__restrict__ amax_part,
    int n_part, uint8_t *__restrict__ codes, uint8_t *__restrict__ scales,
    float *__restrict__ gscale, uint64_t *__restrict__ scores, float *__restrict__ ramax) {
  qdq::quantize_act_body<T, RAC>(blockIdx.x, blockIdx.y, gridDim.y, x, rows, cols, amax_part,
                                 n_part, codes, scales, gscale, scores, ramax);
}

// Weight amax per group: grid (P, G); part[g * P + p].
__global__ __launch_bounds__(256) void amax_group_kernel(const uint16_t *__restrict__ w,
                                                         int64_t n16_per_group,
                                                         float *__restrict__ part) {
  __shared__ float red[16];
  const int64_t g = blockIdx.y;
  const void *base = w + g * n16_per_group * 16;
  float m = 0.0f;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b < n16_per_group; b += stride) {
    float v[16];
    Loader<uint16_t>::load16(base, b * 16, v);
#pragma unroll
    for (int i = 0; i < 16; ++i) m = fmaxf(m, fabsf(v[i]));
  }
  m = block_max(m, red);
  if (threadIdx.x == 0) part[g * gridDim.x + blockIdx.x] = m;
}

// Q_W: grid (tiles, G); each thread quantises one 16-element block of group g.
__global__ __launch_bounds__(256) void quantize_weight_kernel(
    const uint16_t *__restrict__ w, int64_t n16_per_group, const float *__restrict__ part,
    int n_part, uint8_t *__restrict__ codes, uint8_t *__restrict__ scales,
    float *__restrict__ gscale) {
  __shared__ float red[16];
  const int64_t g = blockIdx.y;
  const float amax = block_max(partials_max(part + g * n_part, n_part), red);
  float s_enc, s_dec;
  tensor_scale(amax, s_enc, s_dec);
  const bool zero_tensor = !(amax >= kZeroAmax);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    gscale[2 * g] = s_enc;
    gscale[2 * g + 1] = s_dec;
  }
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b < n16_per_group; b += stride) {
    const int64_t gb = g * n16_per_group + b;
    float v[16];
    Loader<uint16_t>::load16(w, gb * 16, v);
    uint32_t lo, hi;
    uint32_t sb = quantize_block(v, s_enc, zero_tensor, lo, hi);
    reinterpret_cast<uint2 *>(codes)[gb] = make_uint2(lo, hi);
    scales[gb] = (uint8_t)sb;
  }
}

// Dequantise: one thread per 16-element block.
template <bool UNSCALED, bool BF16_OUT>
__global__ __launch_bounds__(256) void dequantize_kernel(
    const uint8_t *__restrict__ codes, const uint8_t *__restrict__ scales,
    const float *__restrict__ gscale, int64_t n16_per_group, int64_t groups, void *__restrict__ out) {
  const int64_t total = n16_per_group * groups;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b < total; b += stride) {
    const int64_t g = b / n16_per_group;
    const float s_dec = gscale[2 * g + 1];
    const float sbf = e4m3_to_f32(scales[b]);
    uint2 cw = reinterpret_cast<const uint2 *>(codes)[b];
    float v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      uint32_t c = ((i < 8 ? cw.x : cw.y) >> (4 * (i & 7))) & 15u;
      float p = e2m1_value(c) * sbf;
      p = (c & 8u) ? -p : p;
      v[i] = UNSCALED ? p : p * s_dec;
    }
    if (BF16_OUT) {
      uint32_t w[8];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        w[j] = f32_to_bf16_bits(v[2 * j]) | (f32_to_bf16_bits(v[2 * j + 1]) << 16);
      uint4 *o = reinterpret_cast<uint4 *>(static_cast<uint16_t *>(out) + b * 16);
      o[0] = make_uint4(w[0], w[1], w[2], w[3]);
      o[1] = make_uint4(w[4], w[5], w[6], w[7]);
    } else {
      float4 *o = reinterpret_cast<float4 *>(static_cast<float *>(out) + b * 16);
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = make_float4(v[4 * j], v[4 * j + 1], v[4 * j + 2], v[4 * j + 3]);
    }
  }
}

}  // namespace

extern "C" size_t nvfp4_quantize_act_workspace(int64_t rows, int64_t cols) {
  (void)rows; (void)cols;
  return (size_t)kAmaxPartials * sizeof(float) + 256;
}

// Up to this many amax partials the quantiser's workgroups read them directly
// (eight loads in flight per thread); more are reduced by a launch of their own.
constexpr int64_t kDirectPartials = 8192;

extern "C" qd_status nvfp4_quantize_act(const void *x, int x_dtype, int64_t rows, int64_t cols,
                                        const float *amax_partials, int64_t n_partials,
                                        const qd_nvfp4 *out, uint64_t *rac_scores,
                                        float *rac_ramax, void *ws, size_t ws_bytes,
                                        void *stream) {
  if (rows < 0 || cols <= 0 || cols % 16) return QD_ERR_SHAPE;
  if (x_dtype != QD_DTYPE_BF16 && x_dtype != QD_DTYPE_F32) return QD_ERR_DTYPE;
  qd_status st = qdh::check_nvfp4(out, 1, rows, cols);
  if (st) return st;
  if (rows == 0) return QD_OK;
  if (!x) return QD_ERR_NULL;
  if (!qdh::aligned16(x)) return QD_ERR_ALIGN;
  const bool rac = rac_scores != nullptr;
  if (rac && (!rac_ramax)) return QD_ERR_NULL;
  if (rac && (amax_partials || x_dtype != QD_DTYPE_BF16)) return QD_ERR_UNSUPPORTED;
  if (amax_partials && n_partials <= 0) return QD_ERR_SHAPE;
  if (!ws) return QD_ERR_WORKSPACE;
  if (ws_bytes < nvfp4_quantize_act_workspace(rows, cols)) return QD_ERR_WORKSPACE;
  if (!qdh::aligned16(ws) || (rac && !qdh::aligned16(rac_scores))) return QD_ERR_ALIGN;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  if (rows == 0) return QD_OK;

  hipStream_t s = qdh::S(stream);
  float *part = static_cast<float *>(ws);
  const int64_t n16 = rows * cols / 16;
  const float *ap;
  int np;
  if (!amax_partials) {
    const int g = amax_grid(n16);
    if (x_dtype == QD_DTYPE_BF16)
      hipLaunchKernelGGL(amax_partial_kernel<uint16_t>, dim3(g), dim3(256), 0, s, x, n16, part,
                         rac_scores, rac ? cols : 0, rac_ramax);
    else
      hipLaunchKernelGGL(amax_partial_kernel<float>, dim3(g), dim3(256), 0, s, x, n16, part,
                         nullptr, 0, nullptr);
    ap = part;
    np = g;
  } else if (n_partials > kDirectPartials) {
    qdi::launch_reduce_max(amax_partials, n_partials, part, s);
    ap = part;
    np = 1;
  } else {
    ap = amax_partials;
    np = (int)n_partials;
  }
  int gx, gy;
  qdq::quant_grid(rows, cols, rac, gx, gy);
  dim3 grid(gx, (unsigned)gy);
  if (x_dtype == QD_DTYPE_BF16) {
    if (rac)
      hipLaunchKernelGGL((quantize_act_kernel<uint16_t, true>), grid, dim3(256), 0, s, x, rows,
                         cols, ap, np, out->codes, out->scales, out->gscale, rac_scores, rac_ramax);
    else
      hipLaunchKernelGGL((quantize_act_kernel<uint16_t, false>), grid, dim3(256), 0, s, x, rows,
                         cols, ap, np, out->codes, out->scales, out->gscale, nullptr, nullptr);
  } else {
    hipLaunchKernelGGL((quantize_act_kernel<float, false>), grid, dim3(256), 0, s, x, rows, cols,
                       ap, np, out->codes, out->scales, out->gscale, nullptr, nullptr);
  }
  return qdh::check_launch();
}

extern "C" size_t nvfp4_quantize_weight_workspace(int64_t groups, int64_t rows, int64_t cols) {
  (void)rows; (void)cols;
  return (size_t)(groups > 0 ? groups : 1) * 64 * sizeof(float) + 256;
}

extern "C" qd_status nvfp4_quantize_weight(const void *w, int64_t groups, int64_t rows,
                                           int64_t cols, const qd_nvfp4 *out, void *ws,
                                           size_t ws_bytes, void *stream) {
  if (groups < 1 || rows < 0 || cols <= 0 || cols % 16) return QD_ERR_SHAPE;
  qd_status st = qdh::check_nvfp4(out, groups, rows, cols);
  if (st) return st;
  if (rows == 0) return QD_OK;
  if (!w) return QD_ERR_NULL;
  if (!qdh::aligned16(w)) return QD_ERR_ALIGN;
  if (!ws || ws_bytes < nvfp4_quantize_weight_workspace(groups, rows, cols)) return QD_ERR_WORKSPACE;
  if (!qdh::aligned16(ws)) return QD_ERR_ALIGN;
  if (groups > 65535) return QD_ERR_UNSUPPORTED;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  if (rows == 0) return QD_OK;
  hipStream_t s = qdh::S(stream);
  const int64_t n16 = rows * cols / 16;
  float *part = static_cast<float *>(ws);
  const int P = 64;
  hipLaunchKernelGGL(amax_group_kernel, dim3(P, (unsigned)groups), dim3(256), 0, s,
                     static_cast<const uint16_t *>(w), n16, part);
  int64_t tiles = (n16 + 255) / 256;
  if (tiles > 1024) tiles = 1024;
  hipLaunchKernelGGL(quantize_weight_kernel, dim3((unsigned)tiles, (unsigned)groups), dim3(256), 0,
                     s, static_cast<const uint16_t *>(w), n16, part, P, out->codes, out->scales,
                     out->gscale);
  return qdh::check_launch();
}

extern "C" qd_status nvfp4_dequantize(const qd_nvfp4 *in, int unscaled, void *out, int out_dtype,
                                      void *stream) {
  if (!in) return QD_ERR_NULL;
  qd_status st = qdh::check_nvfp4(in, in->groups, in->rows, in->cols);
  if (st) return st;
  if (in->rows == 0) return QD_OK;
  if (!out) return QD_ERR_NULL;
  if (out_dtype != QD_DTYPE_BF16 && out_dtype != QD_DTYPE_F32) return QD_ERR_DTYPE;
  if (!qdh::aligned16(out)) return QD_ERR_ALIGN;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  if (in->rows == 0) return QD_OK;
  hipStream_t s = qdh::S(stream);
  const int64_t n16 = in->rows * in->cols / 16;
  int64_t g = (n16 * in->groups + 255) / 256;
  if (g > 8192) g = 8192;
  dim3 grid((unsigned)g);
  if (unscaled) {
    if (out_dtype == QD_DTYPE_BF16)
      hipLaunchKernelGGL((dequantize_kernel<true, true>), grid, dim3(256), 0, s, in->codes,
                         in->scales, in->gscale, n16, in->groups, out);
    else
      hipLaunchKernelGGL((dequantize_kernel<true, false>), grid, dim3(256), 0, s, in->codes,
                         in->scales, in->gscale, n16, in->groups, out);
  } else {
    if (out_dtype == QD_DTYPE_BF16)
      hipLaunchKernelGGL((dequantize_kernel<false, true>), grid, dim3(256), 0, s, in->codes,
                         in->scales, in->gscale, n16, in->groups, out);
    else
      hipLaunchKernelGGL((dequantize_kernel<false, false>), grid, dim3(256), 0, s, in->codes,
                         in->scales, in->gscale, n16, in->groups, out);
  }
  return qdh::check_launch();
}

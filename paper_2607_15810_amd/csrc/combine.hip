// Unpermute and combine: the weighted sum of a token's k expert outputs,
// the last step of the MoE layer (routing weights from moe_route_permute).
//   y[t][n] = bf16( sum_{s=0..k-1} w[t][s] * z[inv_row[t][s]][n] ), f32, slot order.
// Grid (column block of 2048, token; tokens beyond 65535 loop over the grid's
// second dimension), column blocks innermost so that the blocks running
// together share their tokens' rows: each thread owns 8 consecutive
// columns (16 bytes of bf16), so every z row is read with full 16-byte
// loads.  The token's k rows and weights are staged in LDS first and, for
// k <= 8, all k loads of a thread are in flight together; the sum still runs
// in slot order.
#include "common.h"

namespace {

using namespace qd;

constexpr int kCombineMaxK = 32;

__global__ __launch_bounds__(256) void combine_kernel(const uint16_t *__restrict__ z,
                                                      const int32_t *__restrict__ inv_row,
                                                      const float *__restrict__ wts, int k,
                                                      int64_t H, int64_t T,
                                                      uint16_t *__restrict__ y) {
  __shared__ int64_t srow[kCombineMaxK];
  __shared__ float sw[kCombineMaxK];
  const int64_t nc = H >> 3;
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int64_t t = blockIdx.y; t < T; t += gridDim.y) {
    if (t != blockIdx.y) __syncthreads();   // the previous token's rows are read
    if (threadIdx.x < k) {
      srow[threadIdx.x] = (int64_t)inv_row[t * k + threadIdx.x] * H;
      sw[threadIdx.x] = wts[t * k + threadIdx.x];
    }
    __syncthreads();
    if (c >= nc) continue;
    float acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.0f;
    auto add = [&](uint4 v, float wv) {
      const uint32_t q[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] += wv * bf16_bits_to_f32(q[i] & 0xFFFFu);
        acc[2 * i + 1] += wv * bf16_bits_to_f32(q[i] >> 16);
      }
    };
    if (k <= 8) {
      uint4 v[8];
#pragma unroll
      for (int s = 0; s < 8; ++s)
        if (s < k) v[s] = reinterpret_cast<const uint4 *>(z + srow[s])[c];
#pragma unroll
      for (int s = 0; s < 8; ++s)
        if (s < k) add(v[s], sw[s]);
    } else {
      for (int s = 0; s < k; ++s) add(reinterpret_cast<const uint4 *>(z + srow[s])[c], sw[s]);
    }
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      o[i] = f32_to_bf16_bits(acc[2 * i]) | (f32_to_bf16_bits(acc[2 * i + 1]) << 16);
    reinterpret_cast<uint4 *>(y + t * H)[c] = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

}  // namespace

extern "C" qd_status moe_unpermute_combine(const void *z, const int32_t *inv_row,
                                           const float *topk_w, int64_t T, int32_t k, int64_t H,
                                           void *y, void *stream) {
  if (T < 0 || k < 1 || k > kCombineMaxK || H <= 0 || H % 8 != 0) return QD_ERR_SHAPE;
  if (T == 0) return QD_OK;
  if (!z || !inv_row || !topk_w || !y) return QD_ERR_NULL;
  if (!qdh::aligned16(z) || !qdh::aligned16(y) || ((uintptr_t)inv_row & 3u) ||
      ((uintptr_t)topk_w & 3u))
    return QD_ERR_ALIGN;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  if (T == 0) return QD_OK;
  const int64_t ncb = (H / 8 + 255) / 256;
  if (ncb > 0x7fffffffLL) return QD_ERR_UNSUPPORTED;
  const unsigned gy = (unsigned)(T < 65535 ? T : 65535);
  hipLaunchKernelGGL(combine_kernel, dim3((unsigned)ncb, gy), dim3(256), 0, qdh::S(stream),
                     static_cast<const uint16_t *>(z), inv_row, topk_w, k, H, T,
                     static_cast<uint16_t *>(y));
  return qdh::check_launch();
}

// moe_route_permute: top-k routing and the token -> row permutation of the
// MoE layer (Sec. 3.3 / Sec. 4.1; readings in route_dev.h), three kernels.
#include "route_dev.h"

namespace {

using qdr::kTokBlock;
using qdr::kMaxE;
using qdr::kMaxK;

__global__ __launch_bounds__(256) void route_topk_kernel(const float *__restrict__ logits,
                                                         int64_t T, int E, int k, int renorm,
                                                         int32_t *__restrict__ ids,
                                                         float *__restrict__ wts) {
  qdr::route_topk_body(blockIdx.x, logits, T, E, k, renorm, ids, wts);
}
__global__ __launch_bounds__(256) void route_rank_kernel(int64_t T, int E, int k,
                                                         const int32_t *__restrict__ ids,
                                                         int32_t *__restrict__ counts,
                                                         int32_t *__restrict__ ranks) {
  qdr::route_rank_body(blockIdx.x, T, E, k, ids, counts, ranks);
}
__global__ __launch_bounds__(256) void route_scatter_kernel(
    int64_t T, int E, int k, int nblk, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ counts, const int32_t *__restrict__ ranks,
    int32_t *__restrict__ offsets, int32_t *__restrict__ row_token,
    int32_t *__restrict__ inv_row) {
  qdr::route_scatter_body(blockIdx.x, T, E, k, nblk, ids, counts, ranks, offsets, row_token,
                          inv_row);
}

}  // namespace

extern "C" size_t moe_route_permute_workspace(int64_t T, int32_t E, int32_t k) {
  const int64_t nblk = (T + kTokBlock - 1) / kTokBlock;
  return qdh::align_up((size_t)(nblk > 0 ? nblk : 1) * (E > 0 ? E : 1) * 4) +
         qdh::align_up((size_t)(T > 0 ? T : 1) * (k > 0 ? k : 1) * 4);
}

extern "C" qd_status moe_route_permute(const float *logits, int64_t T, int32_t E, int32_t k,
                                       int32_t renorm, int32_t *topk_ids, float *topk_w,
                                       int32_t *expert_offsets, int32_t *row_token,
                                       int32_t *inv_row, void *ws, size_t ws_bytes,
                                       void *stream) {
  if (T < 0 || E < 1 || E > kMaxE || k < 1 || k > E || k > kMaxK) return QD_ERR_SHAPE;
  if (!expert_offsets) return QD_ERR_NULL;
  if (T > 0 && (!logits || !topk_ids || !topk_w || !row_token || !inv_row)) return QD_ERR_NULL;
  if (T * (int64_t)k > 0x7fffffffLL) return QD_ERR_SHAPE;
  if (!ws || ws_bytes < moe_route_permute_workspace(T, E, k)) return QD_ERR_WORKSPACE;
  if (!qdh::aligned16(logits) || !qdh::aligned16(topk_ids) || !qdh::aligned16(topk_w) ||
      !qdh::aligned16(expert_offsets) || !qdh::aligned16(row_token) ||
      !qdh::aligned16(inv_row) || !qdh::aligned16(ws))
    return QD_ERR_ALIGN;   // (NULL is aligned)
  if (qdh::fault_injected()) return QD_ERR_HIP;
  hipStream_t s = qdh::S(stream);
  if (T == 0) {
    // offsets of an empty batch are all zero
    qdi::launch_fill_i32(expert_offsets, E + 1, 0, s);
    return qdh::check_launch();
  }
  const int nblk = (int)((T + kTokBlock - 1) / kTokBlock);
  int32_t *counts = static_cast<int32_t *>(ws);
  int32_t *ranks = reinterpret_cast<int32_t *>(static_cast<char *>(ws) +
                                               qdh::align_up((size_t)nblk * E * 4));
  hipLaunchKernelGGL(route_topk_kernel, dim3((unsigned)qdr::topk_groups(T, E)), dim3(256), 0, s, logits,
                     T, E, k, renorm, topk_ids, topk_w);
  hipLaunchKernelGGL(route_rank_kernel, dim3(nblk), dim3(256), 0, s, T, E, k, topk_ids, counts,
                     ranks);
  hipLaunchKernelGGL(route_scatter_kernel, dim3(nblk), dim3(256), 0, s, T, E, k, nblk,
                     topk_ids, counts, ranks, expert_offsets, row_token, inv_row);
  return qdh::check_launch();
}

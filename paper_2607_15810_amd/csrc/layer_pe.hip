// The MoE layer with one RAC channel set per expert at the W13 input: each
// expert ranks the channels by the residual scores of its own rows (a
// variant of Sec. 3.3, Eq. (channel-score)/(channel-select)), and its rows
// subtract the residual at its own set (Eq. (residual-recon)).  Composed of
// the library's boundary calls on one stream; the intermediates live in the
// caller's workspace.
#include "common.h"

namespace {

struct PeLayout {
  int64_t ids, wts, offs, row_token, inv_row, route_ws, xq_c, xq_s, xq_g, q1_ws, scores, ramax,
      sel, rq_c, rq_s, rq_g, rq_rows, sel_ws, h, h_amax, hq_c, hq_s, hq_g, q2_ws, z, total;
};

PeLayout pe_layout(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I, int32_t Ks) {
  PeLayout L{};
  const int64_t R = T * k;
  int64_t o = 0;
  auto take = [&](int64_t bytes) {
    const int64_t at = o;
    o += (int64_t)qdh::align_up((size_t)(bytes > 0 ? bytes : 1));
    return at;
  };
  L.ids = take(R * 4);
  L.wts = take(R * 4);
  L.offs = take((int64_t)(E + 1) * 4);
  L.row_token = take(R * 4);
  L.inv_row = take(R * 4);
  L.route_ws = take((int64_t)moe_route_permute_workspace(T, E, k));
  L.xq_c = take(T * H / 2);
  L.xq_s = take(T * H / 16);
  L.xq_g = take(8);
  L.q1_ws = take((int64_t)nvfp4_quantize_act_workspace(T, H));
  L.scores = take((int64_t)E * H * 8);
  L.ramax = take(4);
  L.sel = take((int64_t)E * Ks * 4);
  L.rq_c = take(T * H / 2);
  L.rq_s = take(T * H / 16);
  L.rq_g = take(8);
  L.rq_rows = take(R * (int64_t)rac_selected_width(Ks) * 2);
  L.sel_ws = take((int64_t)rac_select_channels_per_expert_workspace(T, H, E));
  L.h = take(R * I * 2);
  L.h_amax = take(std::max<int64_t>(moe_w4a4_grouped_gemm_per_expert_amax_count(R, 2 * I, H, E, Ks,
                                                                               QD_EPI_SWIGLU), 1) * 4);
  L.hq_c = take(R * I / 2);
  L.hq_s = take(R * I / 16);
  L.hq_g = take(8);
  L.q2_ws = take((int64_t)nvfp4_quantize_act_workspace(R, I));
  L.z = take(R * H * 2);
  L.total = o;
  return L;
}

}  // namespace

extern "C" size_t qd_moe_layer_per_expert_workspace(int64_t T, int64_t H, int32_t E, int32_t k,
                                                    int64_t I, int32_t Ks) {
  if (T < 0 || H <= 0 || E < 1 || k < 1 || I <= 0 || Ks < 1) return 0;
  return (size_t)pe_layout(T, H, E, k, I, Ks).total;
}

extern "C" qd_status qd_moe_layer_forward_per_expert(const void *x, const float *logits, int64_t T,
                                                     int64_t H, int32_t E, int32_t k, int64_t I,
                                                     int32_t Ks, int32_t renorm,
                                                     const qd_nvfp4 *w13, const qd_nvfp4 *w2,
                                                     void *y, void *ws, size_t ws_bytes,
                                                     void *stream) {
  if (!w13 || !w2) return QD_ERR_NULL;
  if (T < 0 || H <= 0 || H % 16 || I <= 0 || I % 16 || E < 1 || k < 1 || k > E) return QD_ERR_SHAPE;
  if (Ks < 1 || Ks > H) return QD_ERR_SHAPE;
  if (T * (int64_t)k > 0x7fffffffLL) return QD_ERR_SHAPE;
  qd_status st = qdh::check_nvfp4(w13, E, 2 * I, H);
  if (st) return st;
  st = qdh::check_nvfp4(w2, E, H, I);
  if (st) return st;
  if (T == 0) return QD_OK;
  if (!x || !logits || !y) return QD_ERR_NULL;
  if (!ws) return QD_ERR_WORKSPACE;
  const PeLayout L = pe_layout(T, H, E, k, I, Ks);
  if (ws_bytes < (size_t)L.total) return QD_ERR_WORKSPACE;
  if (!qdh::aligned16(ws) || !qdh::aligned16(x) || !qdh::aligned16(y) || !qdh::aligned16(logits))
    return QD_ERR_ALIGN;
  const int64_t R = T * k;
  // the per-expert GEMM must apply at these sizes before anything runs
  if (moe_w4a4_grouped_gemm_per_expert_amax_count(R, 2 * I, H, E, Ks, QD_EPI_SWIGLU) <= 0)
    return QD_ERR_UNSUPPORTED;
  char *b = static_cast<char *>(ws);
  int32_t *ids = reinterpret_cast<int32_t *>(b + L.ids);
  float *wts = reinterpret_cast<float *>(b + L.wts);
  int32_t *offs = reinterpret_cast<int32_t *>(b + L.offs);
  int32_t *row_token = reinterpret_cast<int32_t *>(b + L.row_token);
  int32_t *inv_row = reinterpret_cast<int32_t *>(b + L.inv_row);
  st = moe_route_permute(logits, T, E, k, renorm, ids, wts, offs, row_token, inv_row,
                         b + L.route_ws, moe_route_permute_workspace(T, E, k), stream);
  if (st) return st;
  const qd_nvfp4 xq{reinterpret_cast<uint8_t *>(b + L.xq_c), reinterpret_cast<uint8_t *>(b + L.xq_s),
                    reinterpret_cast<float *>(b + L.xq_g), 1, T, H, nullptr};
  st = nvfp4_quantize_act(x, QD_DTYPE_BF16, T, H, nullptr, 0, &xq, nullptr, nullptr, b + L.q1_ws,
                          nvfp4_quantize_act_workspace(T, H), stream);
  if (st) return st;
  const qd_nvfp4 rq{reinterpret_cast<uint8_t *>(b + L.rq_c), reinterpret_cast<uint8_t *>(b + L.rq_s),
                    reinterpret_cast<float *>(b + L.rq_g), 1, T, H, nullptr};
  int32_t *sel = reinterpret_cast<int32_t *>(b + L.sel);
  void *rq_rows = b + L.rq_rows;
  st = rac_select_channels_per_expert(x, &xq, Ks, row_token, offs, E, R,
                                      reinterpret_cast<uint64_t *>(b + L.scores),
                                      reinterpret_cast<float *>(b + L.ramax), sel, &rq, rq_rows,
                                      b + L.sel_ws,
                                      rac_select_channels_per_expert_workspace(T, H, E), stream);
  if (st) return st;
  void *h = b + L.h;
  float *hamax = reinterpret_cast<float *>(b + L.h_amax);
  st = moe_w4a4_grouped_gemm_per_expert(&xq, row_token, offs, E, R, w13, &rq, sel, Ks, rq_rows,
                                        QD_EPI_SWIGLU, h, hamax, stream);
  if (st) return st;
  const qd_nvfp4 hq{reinterpret_cast<uint8_t *>(b + L.hq_c), reinterpret_cast<uint8_t *>(b + L.hq_s),
                    reinterpret_cast<float *>(b + L.hq_g), 1, R, I, nullptr};
  st = nvfp4_quantize_act(h, QD_DTYPE_BF16, R, I, hamax,
                          moe_w4a4_grouped_gemm_per_expert_amax_count(R, 2 * I, H, E, Ks,
                                                                      QD_EPI_SWIGLU),
                          &hq, nullptr, nullptr, b + L.q2_ws, nvfp4_quantize_act_workspace(R, I),
                          stream);
  if (st) return st;
  void *z = b + L.z;
  st = moe_w4a4_grouped_gemm(&hq, nullptr, offs, E, R, w2, nullptr, nullptr, 0, nullptr,
                             QD_EPI_NONE, z, nullptr, stream);
  if (st) return st;
  return moe_unpermute_combine(z, inv_row, wts, T, k, H, y, stream);
}

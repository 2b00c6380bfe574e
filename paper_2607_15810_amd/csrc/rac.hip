// Residual Activation Compensation (paper, Sec. 3.3):
//   Eq. (channel-score)  s_j = ||dX_q[:, j]||_2 over the token batch,
//   Eq. (channel-select) S = TopK(s_j), chosen online every forward,
//   Eq. (residual-recon) X~ = Q_A(X) - M_S (.) Q_A(dX_q).
//
// Kernels:
//   rac_amax_kernel / rac_scores_kernel  the score pass when the quantiser did
//                        not fuse it (reads x and its NVFP4 codes, recomputes
//                        r = x_hat - x, fixed-point u64 sums).
//   rac_select_ballot_kernel / rac_select_kernel  one workgroup: the K_s
//                        largest u64 scores (ties to the lower channel) by a
//                        radix select (4-bit digits counted with wave ballots for
//                        K <= 16384, 8-bit LDS histograms above); ascending list
//                        and a channel bitmap.
//   rac_resq_kernel      residual quantised over all channels with its own
//                        tensor scale (max|r|), then masked to S.
//   rac_residual_gemm_kernel  the residual contraction over S alone (f32 out).
#include "rac_dev.h"

namespace {

using namespace qd;
using qdc::load_bf16x16;
using qdc::block_residual;
using qdc::block_exclusive_scan;

constexpr int kMaxK = 65536;

__global__ __launch_bounds__(256) void rac_amax_kernel(const uint16_t *__restrict__ x,
                                                       int64_t n16, float *__restrict__ part,
                                                       uint64_t *__restrict__ scores, int64_t K,
                                                       float *__restrict__ ramax) {
  __shared__ float red[16];
  float m = 0.0f;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b < n16; b += stride) {
    float v[16];
    load_bf16x16(x + b * 16, v);
#pragma unroll
    for (int i = 0; i < 16; ++i) m = fmaxf(m, fabsf(v[i]));
  }
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < K; i += stride)
    scores[i] = 0ull;
  if (blockIdx.x == 0 && threadIdx.x == 0) ramax[0] = 0.0f;
  m = block_max(m, red);
  if (threadIdx.x == 0) part[blockIdx.x] = m;
}

// Same workgroup shape as the fused quantiser: 16 column blocks x 16 rows.
__global__ __launch_bounds__(256) void rac_scores_kernel(
    const uint16_t *__restrict__ x, const uint8_t *__restrict__ codes,
    const uint8_t *__restrict__ scales, const float *__restrict__ gscale, int64_t T, int64_t K,
    const float *__restrict__ part, int n_part, uint64_t *__restrict__ scores,
    float *__restrict__ ramax) {
  __shared__ float red[16];
  __shared__ uint64_t acc_s[16][256];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const float amax = block_max(partials_max(part, n_part), red);
  int e;
  frexpf(amax, &e);
  const int F = 36 - 2 * e;
  const float s_dec = gscale[1];
  const int64_t nbc = K >> 4;
  const int64_t cb = (int64_t)blockIdx.x * 16 + tx;
  // exact integer sums in double, moved into the u64 sums every
  // kScoreMaxRows rows of the thread
  uint64_t acc[16];
  double accd[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    acc[i] = 0ull;
    accd[i] = 0.0;
  }
  int nrow = 0;
  float rmax = 0.0f;
  if (cb < nbc) {
    for (int64_t t = (int64_t)blockIdx.y * 16 + ty; t < T; t += (int64_t)gridDim.y * 16) {
      float v[16], r[16];
      load_bf16x16(x + t * K + cb * 16, v);
      uint2 cw = reinterpret_cast<const uint2 *>(codes + t * (K >> 1))[cb];
      block_residual(v, cw, scales[t * nbc + cb], s_dec, r);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        rmax = fmaxf(rmax, fabsf(r[i]));
        accd[i] += fixed_point_term_f64(r[i] * r[i], F);
      }
      if (++nrow == kScoreMaxRows) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          acc[i] += score_sum_u64(accd[i]);
          accd[i] = 0.0;
        }
        nrow = 0;
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) acc_s[ty][tx * 16 + i] = acc[i] + score_sum_u64(accd[i]);
  __syncthreads();
  uint64_t s = 0;
#pragma unroll
  for (int j = 0; j < 16; ++j) s += acc_s[j][threadIdx.x];
  const int64_t ch = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (ch < K && s != 0ull) atomicAdd((unsigned long long *)&scores[ch], (unsigned long long)s);
  float m = block_max(rmax, red);
  if (threadIdx.x == 0 && m > 0.0f)
    atomic_max_pos(ramax, m);
}

// One workgroup of 1024 threads.  Radix select over 8-bit digits of the u64
// keys finds the K_s-th largest score theta; channels above theta are taken,
// then channels equal to theta in ascending index order until K_s.  Thread i
// owns channels [i*per, (i+1)*per); with K <= 16384 they stay in registers.
template <bool REG>
__global__ __launch_bounds__(1024) void rac_select_kernel(const uint64_t *__restrict__ scores,
                                                          int K, int Ks,
                                                          int32_t *__restrict__ sel_idx,
                                                          uint32_t *__restrict__ bitmap) {
  __shared__ int hist[256];
  __shared__ int sh[1024 + 32];
  __shared__ uint64_t s_prefix;
  __shared__ int s_remaining;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  constexpr int PER = REG ? 16 : 64;      // channels per thread (K <= 1024 * PER)
  const int per = (K + 1023) / 1024;
  const int j0 = tid * per;
  const int n = max(0, min(K, j0 + per) - j0);
  uint64_t sv[16];
  if (REG) {
#pragma unroll
    for (int i = 0; i < 16; ++i) sv[i] = i < n ? scores[j0 + i] : 0ull;
  }
  auto key = [&](int i) -> uint64_t { return REG ? sv[i] : scores[j0 + i]; };
  for (int w = tid; w < (K + 31) / 32; w += 1024) bitmap[w] = 0u;
  if (tid == 0) {
    s_prefix = 0ull;
    s_remaining = Ks;
  }
  __syncthreads();
  if (Ks > 0) {
    uint64_t msk = 0ull;
    for (int d = 7; d >= 0; --d) {
      if (tid < 256) hist[tid] = 0;
      __syncthreads();
      const uint64_t pre = s_prefix;
      const int rem = s_remaining;
      if (REG) {
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (i < n && (sv[i] & msk) == pre) atomicAdd(&hist[(int)((sv[i] >> (8 * d)) & 255ull)], 1);
      } else {
        for (int i = 0; i < n; ++i) {
          const uint64_t v = key(i);
          if ((v & msk) == pre) atomicAdd(&hist[(int)((v >> (8 * d)) & 255ull)], 1);
        }
      }
      __syncthreads();
      if (wid == 0) {
        // lane l owns bins 255-4l .. 252-4l (descending digit order)
        const int b = 255 - 4 * lane;
        const int c0 = hist[b], c1 = hist[b - 1], c2 = hist[b - 2], c3 = hist[b - 3];
        const int lsum = c0 + c1 + c2 + c3;
        int incl = lsum;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_up(incl, o, 64);
          if (lane >= o) incl += y;
        }
        const int excl = incl - lsum;
        if (excl < rem && rem <= incl) {
          int above = excl, dig;
          if (above + c0 >= rem) dig = b;
          else if ((above += c0) + c1 >= rem) dig = b - 1;
          else if ((above += c1) + c2 >= rem) dig = b - 2;
          else { above += c2; dig = b - 3; }
          s_prefix = pre | ((uint64_t)dig << (8 * d));
          s_remaining = rem - above;
        }
      }
      msk |= 255ull << (8 * d);
      __syncthreads();
    }
  }
  const uint64_t theta = s_prefix;
  const int take_eq = s_remaining;          // channels equal to theta to keep
  // rank the channels equal to theta by index
  int n_eq = 0;
  if (Ks > 0) {
#pragma unroll
    for (int i = 0; i < PER; ++i)
      if (i < n) n_eq += (key(i) == theta);
  }
  int tot;
  const int eq_before = block_exclusive_scan(n_eq, sh, tot);
  int n_sel = 0;
  {
    int eq_seen = eq_before;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      if (i >= n) break;
      const uint64_t v = key(i);
      bool take = false;
      if (Ks > 0) {
        if (v > theta) take = true;
        else if (v == theta) take = eq_seen++ < take_eq;
      }
      n_sel += take;
    }
  }
  int pos = block_exclusive_scan(n_sel, sh, tot);
  {
    int eq_seen = eq_before;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      if (i >= n) break;
      const uint64_t v = key(i);
      bool take = false;
      if (Ks > 0) {
        if (v > theta) take = true;
        else if (v == theta) take = eq_seen++ < take_eq;
      }
      if (take) {
        const int j = j0 + i;
        sel_idx[pos++] = j;
        atomicOr(&bitmap[j >> 5], 1u << (j & 31));
      }
    }
  }
}

__global__ __launch_bounds__(qdc::kSelThreads) void rac_select_ballot_kernel_8(
    const uint64_t *__restrict__ scores, int K, int Ks, int32_t *__restrict__ sel_idx,
    uint32_t *__restrict__ bitmap) {
  qdc::rac_select_body<8>(scores, K, Ks, sel_idx, bitmap);
}
__global__ __launch_bounds__(qdc::kSelThreads) void rac_select_ballot_kernel_16(
    const uint64_t *__restrict__ scores, int K, int Ks, int32_t *__restrict__ sel_idx,
    uint32_t *__restrict__ bitmap) {
  qdc::rac_select_body<16>(scores, K, Ks, sel_idx, bitmap);
}
__global__ __launch_bounds__(qdc::kSelThreads) void rac_select_ballot_kernel_64(
    const uint64_t *__restrict__ scores, int K, int Ks, int32_t *__restrict__ sel_idx,
    uint32_t *__restrict__ bitmap) {
  qdc::rac_select_body<64>(scores, K, Ks, sel_idx, bitmap);
}
__global__ __launch_bounds__(256) void rac_resq_kernel(
    const uint16_t *__restrict__ x, const uint8_t *__restrict__ xcodes,
    const uint8_t *__restrict__ xscales, const float *__restrict__ xgs, int64_t T, int64_t K,
    const float *__restrict__ ramax, const uint32_t *__restrict__ bitmap,
    uint8_t *__restrict__ rcodes, uint8_t *__restrict__ rscales, float *__restrict__ rgs) {
  qdc::rac_resq_body(blockIdx.x, gridDim.x, x, xcodes, xscales, xgs, T, K, ramax, bitmap, rcodes,
                     rscales, rgs);
}

__device__ __forceinline__ float nvfp4_unscaled(const uint8_t *codes, const uint8_t *scales,
                                                int64_t row, int64_t K, int64_t j) {
  uint32_t byte = codes[row * (K >> 1) + (j >> 1)];
  uint32_t c = (j & 1) ? (byte >> 4) : (byte & 15u);
  float p = e2m1_value(c) * e4m3_to_f32(scales[row * (K >> 4) + (j >> 4)]);
  return (c & 8u) ? -p : p;
}

// out[r][n] = s_dec_r * s_dec_w[e] * sum_{j in S} rhat[src][j] * what[e][n][j]
__global__ __launch_bounds__(256) void rac_residual_gemm_kernel(
    const uint8_t *__restrict__ rcodes, const uint8_t *__restrict__ rscales,
    const float *__restrict__ rgs, const int32_t *__restrict__ sel, int Ks,
    const int32_t *__restrict__ row_token, const int32_t *__restrict__ offsets, int E,
    int64_t rows, const uint8_t *__restrict__ wcodes, const uint8_t *__restrict__ wscales,
    const float *__restrict__ wgs, int64_t N, int64_t K, float *__restrict__ out) {
  __shared__ int32_t s_sel[1024];
  const int64_t r = blockIdx.x;
  int e = 0;
  if (offsets) {
    while (e + 1 < E && r >= offsets[e + 1]) ++e;
  }
  const int64_t src = row_token ? row_token[r] : r;
  const float alpha = rgs[1] * wgs[2 * e + 1];
  const uint8_t *wc = wcodes + (int64_t)e * N * (K >> 1);
  const uint8_t *ws = wscales + (int64_t)e * N * (K >> 4);
  const int64_t n = (int64_t)blockIdx.y * blockDim.x + threadIdx.x;
  float acc = 0.0f;
  for (int base = 0; base < Ks; base += 1024) {
    const int cnt = min(1024, Ks - base);
    __syncthreads();
    for (int i = threadIdx.x; i < cnt; i += blockDim.x) s_sel[i] = sel[base + i];
    __syncthreads();
    if (n < N)
      for (int i = 0; i < cnt; ++i) {
        const int j = s_sel[i];
        acc += nvfp4_unscaled(rcodes, rscales, src, K, j) * nvfp4_unscaled(wc, ws, n, K, j);
      }
  }
  if (n < N) out[r * N + n] = alpha * acc;
}

// the masked residual at the selected channels, compacted per row, as f16
// without the tensor scale: e2m1(code) * e4m3(block scale) is exact in f16;
// columns past Ks are zero
__global__ __launch_bounds__(256) void rac_gather_selected_kernel(
    const uint8_t *__restrict__ codes, const uint8_t *__restrict__ scales, int64_t K,
    const int32_t *__restrict__ sel, int Ks, int width, int64_t rows, uint16_t *__restrict__ out) {
  const int64_t n = rows * width;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int64_t t = i / width;
    const int j = (int)(i - t * width);
    float v = 0.0f;
    if (j < Ks) {
      const int64_t c = sel[j];
      const uint32_t byte = codes[t * (K >> 1) + (c >> 1)];
      const uint32_t code = (c & 1) ? byte >> 4 : byte & 15u;
      v = e2m1_value(code) * e4m3_to_f32(scales[t * (K >> 4) + (c >> 4)]);
      if (code & 8u) v = -v;
    }
    out[i] = __builtin_bit_cast(uint16_t, (_Float16)v);
  }
}

// ---- per-expert channel sets (reading L7): Eq. (channel-score) over each
// expert's own rows, Eq. (channel-select) per expert

// Workgroup (column group of 256 channels, expert e): 16 column blocks x 16
// row lanes walk the expert's rows (their tokens' x and x_hat codes), sum
// the fixed-point squared residuals per channel, reduce over the row lanes
// and write score_e once (no atomics: one workgroup owns each entry); the
// maximum |r| over all rows (every token is some expert's row) goes to
// ramax.
__global__ __launch_bounds__(256) void rac_scores_pe_kernel(
    const uint16_t *__restrict__ x, const uint8_t *__restrict__ codes,
    const uint8_t *__restrict__ scales, const float *__restrict__ gscale, int64_t K,
    const float *__restrict__ part, int n_part, const int32_t *__restrict__ row_token,
    const int32_t *__restrict__ offsets, uint64_t *__restrict__ scores_pe,
    float *__restrict__ ramax) {
  __shared__ float red[16];
  __shared__ uint64_t acc_s[16][256];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int e = blockIdx.y;
  const float amax = block_max(partials_max(part, n_part), red);
  int ex;
  frexpf(amax, &ex);
  const int F = 36 - 2 * ex;
  const float s_dec = gscale[1];
  const int64_t nbc = K >> 4;
  const int64_t cb = (int64_t)blockIdx.x * 16 + tx;
  // exact integer sums in double, moved into the u64 sums every
  // kScoreMaxRows rows of the thread
  uint64_t acc[16];
  double accd[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    acc[i] = 0ull;
    accd[i] = 0.0;
  }
  int nrow = 0;
  float rmax = 0.0f;
  if (cb < nbc) {
    const int r1 = offsets[e + 1];
    for (int row = offsets[e] + ty; row < r1; row += 16) {
      const int64_t t = row_token[row];
      float v[16], r[16];
      load_bf16x16(x + t * K + cb * 16, v);
      const uint2 cw = reinterpret_cast<const uint2 *>(codes + t * (K >> 1))[cb];
      block_residual(v, cw, scales[t * nbc + cb], s_dec, r);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        rmax = fmaxf(rmax, fabsf(r[i]));
        accd[i] += fixed_point_term_f64(r[i] * r[i], F);
      }
      if (++nrow == kScoreMaxRows) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          acc[i] += score_sum_u64(accd[i]);
          accd[i] = 0.0;
        }
        nrow = 0;
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) acc_s[ty][tx * 16 + i] = acc[i] + score_sum_u64(accd[i]);
  __syncthreads();
  uint64_t sum = 0;
#pragma unroll
  for (int j = 0; j < 16; ++j) sum += acc_s[j][threadIdx.x];
  const int64_t ch = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (ch < K) scores_pe[(int64_t)e * K + ch] = sum;
  const float m = block_max(rmax, red);
  if (threadIdx.x == 0 && m > 0.0f)
    atomic_max_pos(ramax, m);
}

// one workgroup per expert: the selection of rac_select_channels on score_e
template <int PER>
__global__ __launch_bounds__(qdc::kSelThreads) void rac_select_pe_kernel(
    const uint64_t *__restrict__ scores_pe, int K, int Ks, int32_t *__restrict__ sel_pe,
    uint32_t *__restrict__ bitmaps) {
  const int e = blockIdx.x;
  qdc::rac_select_body<PER>(scores_pe + (int64_t)e * K, K, Ks, sel_pe + (int64_t)e * Ks,
                            bitmaps + (int64_t)e * ((K + 31) / 32));
}

// the residual (quantised over all channels) at the channels of each
// permuted row's expert, compacted per row as f16 without the tensor scale
// (exact); columns past Ks are zero
__global__ __launch_bounds__(256) void rac_gather_rows_pe_kernel(
    const uint8_t *__restrict__ codes, const uint8_t *__restrict__ scales, int64_t K,
    const int32_t *__restrict__ sel_pe, int Ks, int width, const int32_t *__restrict__ row_token,
    const int32_t *__restrict__ offsets, int E, int64_t rows, uint16_t *__restrict__ out) {
  const int64_t n = rows * width;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int64_t r = i / width;
    const int j = (int)(i - r * width);
    float v = 0.0f;
    if (j < Ks) {
      int lo = 0, hi = E;                 // the expert e with offsets[e] <= r < offsets[e + 1]
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (offsets[mid] <= r) lo = mid; else hi = mid;
      }
      const int64_t t = row_token[r];
      const int64_t c = sel_pe[(int64_t)lo * Ks + j];
      const uint32_t byte = codes[t * (K >> 1) + (c >> 1)];
      const uint32_t code = (c & 1) ? byte >> 4 : byte & 15u;
      v = e2m1_value(code) * e4m3_to_f32(scales[t * (K >> 4) + (c >> 4)]);
      if (code & 8u) v = -v;
    }
    out[i] = __builtin_bit_cast(uint16_t, (_Float16)v);
  }
}

}  // namespace

extern "C" size_t rac_select_channels_per_expert_workspace(int64_t T, int64_t K, int32_t E) {
  (void)T;
  if (K <= 0 || E < 1) return 0;
  return qdh::align_up((size_t)E * ((K + 31) / 32) * 4) + qdh::align_up((size_t)((K + 31) / 32) * 4) +
         256 * sizeof(float) + 256;
}

extern "C" qd_status rac_select_channels_per_expert(
    const void *x, const qd_nvfp4 *xq, int32_t Ks, const int32_t *row_token,
    const int32_t *expert_offsets, int32_t E, int64_t rows, uint64_t *scores_pe, float *ramax,
    int32_t *sel_pe, const qd_nvfp4 *rq, void *rq_sel_rows, void *ws, size_t ws_bytes,
    void *stream) {
  if (!x || !xq || !row_token || !expert_offsets || !scores_pe || !ramax || !rq) return QD_ERR_NULL;
  const int64_t T = xq->rows, K = xq->cols;
  qd_status st = qdh::check_nvfp4(xq, 1, T, K);
  if (st) return st;
  st = qdh::check_nvfp4(rq, 1, T, K);
  if (st) return st;
  if (E < 1 || rows < 0 || Ks < 0 || Ks > K) return QD_ERR_SHAPE;
  if (K > qdc::kSelMaxK || (K / 256 + 1) > 65535 || E > 65535) return QD_ERR_UNSUPPORTED;
  if (Ks > 0 && (!sel_pe || !rq_sel_rows)) return QD_ERR_NULL;
  if (!ws || ws_bytes < rac_select_channels_per_expert_workspace(T, K, E)) return QD_ERR_WORKSPACE;
  if (!qdh::aligned16(x) || !qdh::aligned16(scores_pe) || !qdh::aligned16(ws) ||
      (sel_pe && !qdh::aligned16(sel_pe)) || (rq_sel_rows && !qdh::aligned16(rq_sel_rows)))
    return QD_ERR_ALIGN;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  if (T == 0) return QD_OK;
  hipStream_t s = qdh::S(stream);
  char *w = static_cast<char *>(ws);
  uint32_t *bitmaps = reinterpret_cast<uint32_t *>(w);
  uint32_t *ones = reinterpret_cast<uint32_t *>(w + qdh::align_up((size_t)E * ((K + 31) / 32) * 4));
  float *part = reinterpret_cast<float *>(reinterpret_cast<char *>(ones) +
                                          qdh::align_up((size_t)((K + 31) / 32) * 4));
  const uint16_t *xb = static_cast<const uint16_t *>(x);
  // amax of X (the fixed point of the scores) and ramax = 0
  const int64_t n16 = T * K / 16;
  int g = (int)((n16 + 255) / 256);
  if (g > 256) g = 256;
  if (g < 1) g = 1;
  hipLaunchKernelGGL(rac_amax_kernel, dim3(g), dim3(256), 0, s, xb, n16, part, scores_pe, K, ramax);
  // the per-expert scores (and max |r|)
  hipLaunchKernelGGL(rac_scores_pe_kernel, dim3((unsigned)((K + 255) / 256), (unsigned)E),
                     dim3(256), 0, s, xb, xq->codes, xq->scales, xq->gscale, K, part, g, row_token,
                     expert_offsets, scores_pe, ramax);
  if (Ks > 0) {
    if (K <= 2048)
      hipLaunchKernelGGL(rac_select_pe_kernel<8>, dim3((unsigned)E), dim3(qdc::kSelThreads), 0, s,
                         scores_pe, (int)K, Ks, sel_pe, bitmaps);
    else if (K <= 4096)
      hipLaunchKernelGGL(rac_select_pe_kernel<16>, dim3((unsigned)E), dim3(qdc::kSelThreads), 0, s,
                         scores_pe, (int)K, Ks, sel_pe, bitmaps);
    else
      hipLaunchKernelGGL(rac_select_pe_kernel<64>, dim3((unsigned)E), dim3(qdc::kSelThreads), 0, s,
                         scores_pe, (int)K, Ks, sel_pe, bitmaps);
  }
  // the residual quantised over all channels (every channel in the mask)
  qdi::launch_fill_i32(reinterpret_cast<int32_t *>(ones), (K + 31) / 32, -1, s);
  {
    const int64_t total = T * (K / 16);
    int64_t gq = (total + 255) / 256;
    if (gq > 4096) gq = 4096;
    if (gq < 1) gq = 1;
    hipLaunchKernelGGL(rac_resq_kernel, dim3((unsigned)gq), dim3(256), 0, s, xb, xq->codes,
                       xq->scales, xq->gscale, T, K, ramax, ones, rq->codes, rq->scales,
                       rq->gscale);
  }
  if (Ks > 0 && rows > 0) {
    const int width = rac_selected_width(Ks);
    const int64_t n = rows * width;
    int64_t gg = (n + 255) / 256;
    if (gg > 8192) gg = 8192;
    hipLaunchKernelGGL(rac_gather_rows_pe_kernel, dim3((unsigned)gg), dim3(256), 0, s, rq->codes,
                       rq->scales, K, sel_pe, Ks, width, row_token, expert_offsets, E, rows,
                       static_cast<uint16_t *>(rq_sel_rows));
  }
  return qdh::check_launch();
}

extern "C" size_t rac_select_channels_workspace(int64_t T, int64_t K) {
  (void)T;
  return qdh::align_up((size_t)((K + 31) / 32) * 4) + 256 * sizeof(float) + 256;
}

extern "C" qd_status rac_select_channels(const void *x, const qd_nvfp4 *xq, int32_t Ks,
                                         uint64_t *scores, float *ramax, int32_t stats_ready,
                                         int32_t *sel_idx, const qd_nvfp4 *rq, void *ws,
                                         size_t ws_bytes, void *stream) {
  if (!x || !xq || !scores || !ramax || !rq) return QD_ERR_NULL;
  const int64_t T = xq->rows, K = xq->cols;
  qd_status st = qdh::check_nvfp4(xq, 1, T, K);
  if (st) return st;
  st = qdh::check_nvfp4(rq, 1, T, K);
  if (st) return st;
  if (K > kMaxK || Ks < 0 || Ks > K) return QD_ERR_SHAPE;
  if (Ks > 0 && !sel_idx) return QD_ERR_NULL;
  if (!ws || ws_bytes < rac_select_channels_workspace(T, K)) return QD_ERR_WORKSPACE;
  if (!qdh::aligned16(x) || !qdh::aligned16(scores) || !qdh::aligned16(ws) ||
      (sel_idx && !qdh::aligned16(sel_idx)))
    return QD_ERR_ALIGN;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  hipStream_t s = qdh::S(stream);
  uint32_t *bitmap = static_cast<uint32_t *>(ws);
  float *part = reinterpret_cast<float *>(static_cast<char *>(ws) +
                                          qdh::align_up((size_t)((K + 31) / 32) * 4));
  const uint16_t *xb = static_cast<const uint16_t *>(x);
  if (!stats_ready) {
    const int64_t n16 = T * K / 16;
    int g = (int)((n16 + 255) / 256);
    if (g > 256) g = 256;
    if (g < 1) g = 1;
    hipLaunchKernelGGL(rac_amax_kernel, dim3(g), dim3(256), 0, s, xb, n16, part, scores, K, ramax);
    if (T > 0) {
      const int gx = (int)((K / 16 + 15) / 16);
      int64_t gy = (T + 15) / 16;
      int64_t lim = 256 / gx;
      if (lim < 1) lim = 1;
      if (gy > lim) gy = lim;
      hipLaunchKernelGGL(rac_scores_kernel, dim3(gx, (unsigned)gy), dim3(256), 0, s, xb,
                         xq->codes, xq->scales, xq->gscale, T, K, part, g, scores, ramax);
    }
  }
  if (K <= 2048)
    hipLaunchKernelGGL(rac_select_ballot_kernel_8, dim3(1), dim3(qdc::kSelThreads), 0, s, scores,
                       (int)K, Ks, sel_idx, bitmap);
  else if (K <= 4096)
    hipLaunchKernelGGL(rac_select_ballot_kernel_16, dim3(1), dim3(qdc::kSelThreads), 0, s, scores,
                       (int)K, Ks, sel_idx, bitmap);
  else if (K <= qdc::kSelMaxK)
    hipLaunchKernelGGL(rac_select_ballot_kernel_64, dim3(1), dim3(qdc::kSelThreads), 0, s, scores,
                       (int)K, Ks, sel_idx, bitmap);
  else
    hipLaunchKernelGGL(rac_select_kernel<false>, dim3(1), dim3(1024), 0, s, scores, (int)K, Ks,
                       sel_idx, bitmap);
  {
    const int64_t total = T * (K / 16);
    int64_t g = (total + 255) / 256;
    if (g > 4096) g = 4096;
    if (g < 1) g = 1;
    hipLaunchKernelGGL(rac_resq_kernel, dim3((unsigned)g), dim3(256), 0, s, xb, xq->codes,
                       xq->scales, xq->gscale, T, K, ramax, bitmap, rq->codes, rq->scales,
                       rq->gscale);
  }
  return qdh::check_launch();
}

extern "C" qd_status rac_residual_gemm(const qd_nvfp4 *rq, const int32_t *sel_idx, int32_t Ks,
                                       const int32_t *row_token, const int32_t *expert_offsets,
                                       int64_t rows, const qd_nvfp4 *w, float *out,
                                       void *stream) {
  if (!rq || !w || !out) return QD_ERR_NULL;
  if (Ks < 0 || Ks > rq->cols) return QD_ERR_SHAPE;
  if (Ks > 0 && !sel_idx) return QD_ERR_NULL;
  qd_status st = qdh::check_nvfp4(rq, 1, rq->rows, rq->cols);
  if (st) return st;
  st = qdh::check_nvfp4(w, w->groups, w->rows, rq->cols);
  if (st) return st;
  if (!expert_offsets && w->groups != 1) return QD_ERR_SHAPE;
  if (!row_token && rows > rq->rows) return QD_ERR_SHAPE;
  if (rows < 0) return QD_ERR_SHAPE;
  if ((w->rows + 255) / 256 > 65535) return QD_ERR_UNSUPPORTED;
  if (!qdh::aligned16(out)) return QD_ERR_ALIGN;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  if (rows == 0 || w->rows == 0) return QD_OK;
  hipStream_t s = qdh::S(stream);
  const int64_t gy = (w->rows + 255) / 256;
  hipLaunchKernelGGL(rac_residual_gemm_kernel, dim3((unsigned)rows, (unsigned)gy), dim3(256), 0, s,
                     rq->codes, rq->scales, rq->gscale, sel_idx, Ks, row_token, expert_offsets,
                     (int)w->groups, rows, w->codes, w->scales, w->gscale, w->rows, rq->cols, out);
  return qdh::check_launch();
}

extern "C" int32_t rac_selected_width(int32_t Ks) { return Ks <= 0 ? 0 : (Ks + 15) / 16 * 16; }

extern "C" qd_status rac_gather_selected(const qd_nvfp4 *rq, const int32_t *sel_idx, int32_t Ks,
                                         void *out, void *stream) {
  if (!rq || !out) return QD_ERR_NULL;
  if (Ks < 0 || Ks > rq->cols) return QD_ERR_SHAPE;
  if (Ks > 0 && !sel_idx) return QD_ERR_NULL;
  qd_status st = qdh::check_nvfp4(rq, 1, rq->rows, rq->cols);
  if (st) return st;
  if (!qdh::aligned16(out)) return QD_ERR_ALIGN;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  const int width = rac_selected_width(Ks);
  const int64_t n = rq->rows * width;
  if (n == 0) return QD_OK;
  int64_t g = (n + 255) / 256;
  if (g > 8192) g = 8192;
  hipLaunchKernelGGL(rac_gather_selected_kernel, dim3((unsigned)g), dim3(256), 0, qdh::S(stream),
                     rq->codes, rq->scales, rq->cols, sel_idx, Ks, width, rq->rows,
                     static_cast<uint16_t *>(out));
  return qdh::check_launch();
}

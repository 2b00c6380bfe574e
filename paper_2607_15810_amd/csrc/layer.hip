// The whole rollout-side MoE layer in one call (paper, Sec. 3.3): routing,
// activation quantisation with fused RAC statistics, channel selection and
// masked residual, W13 grouped GEMM with the fused residual and SwiGLU,
// quantisation of h, W2 grouped GEMM, weighted combine.  Intermediates are
// carved from the caller's workspace at the offsets qd_moe_layer_views gives.
#include "quant_dev.h"
#include "rac_dev.h"
#include "route_dev.h"

namespace {

using namespace qd;

// The steps before the W13 GEMM form two independent chains -- routing
// (top-k, ranks, scatter) and X (amax, quantise + RAC scores, channel
// select) -- so each launch below runs one step of each chain side by side
// in disjoint workgroups: three launches instead of six.

// routing top-k (ntopk workgroups) | amax partials of X (ga workgroups; with
// RAC they also clear the score and residual-amax accumulators)
__global__ __launch_bounds__(256) void layer_pre1_kernel(
    const float *__restrict__ logits, int64_t T, int E, int k, int renorm,
    int32_t *__restrict__ ids, float *__restrict__ wts, int ntopk, const void *__restrict__ x,
    int64_t n16, float *__restrict__ part, int ga, uint64_t *__restrict__ scores, int64_t H,
    float *__restrict__ ramax) {
  const int b = blockIdx.x;
  if (b < ntopk) qdr::route_topk_body(b, logits, T, E, k, renorm, ids, wts);
  else qdq::amax_partial_body<uint16_t>(b - ntopk, ga, x, n16, part, scores, scores ? H : 0, ramax);
}

// ---- The block's input path folded ahead of the layer: RMSNorm of the
// hidden state h, the router logits of the normalised state, top-k and the
// amax partials of the normalised state, in one pass over h (it replaces
// layer_pre1_kernel, and a separate normalisation and router launch with
// their round trip of x).  Token blocks of TOK rows (8, 16 or 32: the
// largest that leaves the chip 256 blocks and fits LDS): 1/RMS per row
// (wave w: rows TOK/4 w ..), then the block's normalised bf16 rows go to x
// and to LDS whole, then the router contraction on bf16 MFMAs (32 token
// rows, zero past TOK, x 32 experts per 32x32x16 step; wave w takes expert
// blocks w and w + 4, so E <= 256), its router weights streamed in groups
// of steps with the next group in flight during the current one's MFMAs;
// the logits go out, and each wave takes the top-k of TOK/4 of the block's
// tokens in turn.
constexpr int kBlkMaxE = 256;
constexpr int kBlkLds = 144 * 1024;    // the normalised rows of one block

typedef __bf16 blk_bf16x8 __attribute__((ext_vector_type(8)));
typedef float blk_f32x16 __attribute__((ext_vector_type(16)));

inline int64_t block_lds(int tok, int64_t H) { return (int64_t)tok * (H + 8) * 2; }

template <int PER, int TOK>
__global__ __launch_bounds__(256) void block_pre0_kernel(
    const uint16_t *__restrict__ hin, const uint16_t *__restrict__ gamma, float eps,
    const uint16_t *__restrict__ wr, int64_t T, int64_t H, int E, int k, int renorm,
    uint16_t *__restrict__ x, float *__restrict__ logits, int32_t *__restrict__ ids,
    float *__restrict__ wts, float *__restrict__ part, uint64_t *__restrict__ scores,
    float *__restrict__ ramax) {
  static_assert(TOK == 8 || TOK == 16 || TOK == 32, "token block");
  constexpr int NB = PER > 2 ? 2 : 1;    // expert blocks per wave
  constexpr int G = NB == 1 ? 16 : 8;    // MFMA steps per group of loads
  extern __shared__ __align__(16) uint16_t xs[];     // [TOK][H + 8]
  __shared__ float rinv[TOK];
  __shared__ float red[16];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t XS = H + 8, n8 = H >> 3;
  const int64_t ntb = (T + TOK - 1) / TOK;
  const int neb = (E + 31) >> 5;
  const int nst = (int)(H >> 4), ngr = (nst + G - 1) / G;
  float m = 0.0f;
  for (int64_t tb = blockIdx.x; tb < ntb; tb += gridDim.x) {
    const int64_t t0 = tb * TOK;
    const int nt = (int)(T - t0 < TOK ? T - t0 : TOK);
    // the block's rows of h into LDS, and 1 / RMS: squares summed per lane
    // over its 8-column pieces, then across the wave (wave w: rows RPW w ..;
    // rows past the batch repeat the block's first row, so the loads need no
    // branch and several rows' loads are in flight together)
    constexpr int RPW = TOK / 4;
    {
      float ss[RPW];
#pragma unroll
      for (int jj = 0; jj < RPW; ++jj) ss[jj] = 0.0f;
#pragma unroll 2
      for (int64_t c = 8 * lane; c < H; c += 512) {
        uint4 v[RPW];
#pragma unroll
        for (int jj = 0; jj < RPW; ++jj) {
          const int j = RPW * w + jj;
          v[jj] = *reinterpret_cast<const uint4 *>(hin + (t0 + (j < nt ? j : 0)) * H + c);
        }
#pragma unroll
        for (int jj = 0; jj < RPW; ++jj) {
          *reinterpret_cast<uint4 *>(xs + (RPW * w + jj) * XS + c) = v[jj];
          const uint32_t q[4] = {v[jj].x, v[jj].y, v[jj].z, v[jj].w};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float a = bf16_bits_to_f32(q[i] & 0xFFFFu), b = bf16_bits_to_f32(q[i] >> 16);
            ss[jj] += a * a;
            ss[jj] += b * b;
          }
        }
      }
#pragma unroll
      for (int jj = 0; jj < RPW; ++jj) {
        float t = ss[jj];
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) t += __shfl_xor(t, o, 64);
        if (lane == 0) rinv[RPW * w + jj] = 1.0f / sqrtf(t / (float)H + eps);
      }
    }
    __syncthreads();
    // x = bf16((h * (1 / RMS)) * gamma) in place in LDS, and to x (rows past
    // the batch stay as loaded: their MFMA rows are never stored)
    const int n8i = (int)n8;
#pragma unroll 4
    for (int q = tid; q < TOK * n8i; q += 256) {
      const int j = q / n8i;
      const int c = (q - j * n8i) * 8;
      if (j < nt) {
        uint4 *px = reinterpret_cast<uint4 *>(xs + j * XS + c);
        const uint4 hv = *px;
        const uint4 gv = *reinterpret_cast<const uint4 *>(gamma + c);
        const uint32_t hq[4] = {hv.x, hv.y, hv.z, hv.w}, gq[4] = {gv.x, gv.y, gv.z, gv.w};
        const float r = rinv[j];
        uint32_t o[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t lo = f32_to_bf16_bits(
              (bf16_bits_to_f32(hq[i] & 0xFFFFu) * r) * bf16_bits_to_f32(gq[i] & 0xFFFFu));
          const uint32_t hi = f32_to_bf16_bits(
              (bf16_bits_to_f32(hq[i] >> 16) * r) * bf16_bits_to_f32(gq[i] >> 16));
          m = fmaxf(m, fmaxf(fabsf(bf16_bits_to_f32(lo)), fabsf(bf16_bits_to_f32(hi))));
          o[i] = lo | (hi << 16);
        }
        const uint4 ov = make_uint4(o[0], o[1], o[2], o[3]);
        *px = ov;
        *reinterpret_cast<uint4 *>(x + (t0 + j) * H + c) = ov;
      }
    }
    __syncthreads();
    // router: lane l holds token row l % 32 (zero past TOK) and expert row
    // l % 32 of its block, columns 8 (l / 32) .. + 7 of each 16-column step
    blk_f32x16 acc[NB];
    const uint16_t *wrow[NB];
    bool ev[NB];
#pragma unroll
    for (int bi = 0; bi < NB; ++bi) {
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[bi][q] = 0.0f;
      const int e = 32 * (w + 4 * bi) + (lane & 31);
      ev[bi] = w + 4 * bi < neb && e < E;
      wrow[bi] = wr + (int64_t)(ev[bi] ? e : 0) * H + 8 * (lane >> 5);
    }
    const bool arow = (lane & 31) < TOK;
    const uint16_t *xrow = xs + (arow ? (lane & 31) : 0) * XS + 8 * (lane >> 5);
    uint4 bA[NB][G], bB[NB][G];
    auto load = [&](uint4 (&b)[NB][G], int g) __attribute__((always_inline)) {
#pragma unroll
      for (int bi = 0; bi < NB; ++bi)
#pragma unroll
        for (int i = 0; i < G; ++i) {
          const int st = g * G + i;
          b[bi][i] = ev[bi] && st < nst ? *reinterpret_cast<const uint4 *>(wrow[bi] + 16 * st)
                                        : make_uint4(0u, 0u, 0u, 0u);
        }
    };
    auto mfmas = [&](const uint4 (&b)[NB][G], int g) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < G; ++i) {
        const int st = g * G + i;
        if (st < nst) {
          uint4 av = *reinterpret_cast<const uint4 *>(xrow + 16 * st);
          if (!arow) av = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
          for (int bi = 0; bi < NB; ++bi)
            if (w + 4 * bi < neb)
              acc[bi] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                  __builtin_bit_cast(blk_bf16x8, av), __builtin_bit_cast(blk_bf16x8, b[bi][i]),
                  acc[bi], 0, 0, 0);
        }
      }
    };
    load(bA, 0);
    for (int g = 0; g < ngr; g += 2) {
      load(bB, g + 1);
      mfmas(bA, g);
      load(bA, g + 2);
      mfmas(bB, g + 1);
    }
    // logits: lane l holds expert 32 eb + l % 32 for token rows
    // 8 (q / 4) + 4 (l / 32) + q % 4
#pragma unroll
    for (int bi = 0; bi < NB; ++bi) {
      const int e = 32 * (w + 4 * bi) + (lane & 31);
      if (w + 4 * bi < neb && e < E) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int j = 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
          if (j < nt) logits[(t0 + j) * E + e] = acc[bi][q];
        }
      }
    }
    __syncthreads();
    // top-k: wave w takes tokens t0 + 4 i + w (the wave routing body, same
    // arithmetic as the layer's)
#pragma unroll 1
    for (int i = 0; i < TOK / 4; ++i)
      qdr::route_topk_wave_body<PER>((int)(tb * (TOK / 4) + i), logits, T, E, k, renorm, ids,
                                     wts);
  }
  // the RAC accumulators the quantiser that follows adds into
  if (scores)
    for (int64_t i = (int64_t)blockIdx.x * 256 + tid; i < H; i += (int64_t)gridDim.x * 256)
      scores[i] = 0ull;
  if (ramax && blockIdx.x == 0 && tid == 0) ramax[0] = 0.0f;
  m = block_max(m, red);
  if (tid == 0) part[blockIdx.x] = m;
}

// token rows per block of the block pre-kernel: the largest of 32, 16, 8
// that leaves at least 256 blocks and whose rows fit LDS (0: none fits)
inline int block_tok(int64_t T, int64_t H) {
  for (int tok = 32; tok >= 8; tok >>= 1)
    if ((T >= (int64_t)tok * 256 || tok == 8) && block_lds(tok, H) <= kBlkLds) return tok;
  return 0;
}

// the dynamic LDS limit of one instantiation, raised once (thread-safe
// static initialisation)
template <int PER, int TOK>
const void *pre0_kernel() {
  static const bool attr =
      hipFuncSetAttribute(reinterpret_cast<const void *>(block_pre0_kernel<PER, TOK>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, kBlkLds) == hipSuccess;
  (void)attr;
  return reinterpret_cast<const void *>(block_pre0_kernel<PER, TOK>);
}

template <int TOK>
void launch_pre0(int E, int np, hipStream_t s, const void *h, const void *gamma, float eps,
                 const void *wr, int64_t T, int64_t H, int k, int renorm, void *x, float *logits,
                 int32_t *ids, float *wts, float *part, uint64_t *scores, float *ramax) {
  const uint16_t *hh = static_cast<const uint16_t *>(h);
  const uint16_t *gg = static_cast<const uint16_t *>(gamma);
  const uint16_t *ww = static_cast<const uint16_t *>(wr);
  uint16_t *xx = static_cast<uint16_t *>(x);
  const dim3 grid((unsigned)np), block(256);
  const size_t lds = (size_t)block_lds(TOK, H);
  switch ((E + 63) >> 6) {
    case 1:
      (void)pre0_kernel<1, TOK>();
      hipLaunchKernelGGL((block_pre0_kernel<1, TOK>), grid, block, lds, s, hh, gg, eps, ww, T, H,
                         E, k, renorm, xx, logits, ids, wts, part, scores, ramax);
      break;
    case 2:
      (void)pre0_kernel<2, TOK>();
      hipLaunchKernelGGL((block_pre0_kernel<2, TOK>), grid, block, lds, s, hh, gg, eps, ww, T, H,
                         E, k, renorm, xx, logits, ids, wts, part, scores, ramax);
      break;
    case 3:
      (void)pre0_kernel<3, TOK>();
      hipLaunchKernelGGL((block_pre0_kernel<3, TOK>), grid, block, lds, s, hh, gg, eps, ww, T, H,
                         E, k, renorm, xx, logits, ids, wts, part, scores, ramax);
      break;
    default:
      (void)pre0_kernel<4, TOK>();
      hipLaunchKernelGGL((block_pre0_kernel<4, TOK>), grid, block, lds, s, hh, gg, eps, ww, T, H,
                         E, k, renorm, xx, logits, ids, wts, part, scores, ramax);
      break;
  }
}

// routing ranks (nr workgroups) | X quantiser (+ RAC scores) on a (gx, gy) grid;
// the two bodies run in different workgroups and share one LDS array, so the
// kernel's LDS is the larger body's (40 KB: four workgroups per CU)
constexpr int kPre2Lds =
    qdr::kRankLdsBytes > qdq::kQuantLdsBytes ? qdr::kRankLdsBytes : qdq::kQuantLdsBytes;
template <bool RAC>
__global__ __launch_bounds__(256) void layer_pre2_kernel(
    int64_t T, int E, int k, const int32_t *__restrict__ ids, int32_t *__restrict__ counts,
    int32_t *__restrict__ ranks, int nr, const void *__restrict__ x, int64_t H,
    const float *__restrict__ part, int np, uint8_t *__restrict__ codes,
    uint8_t *__restrict__ scales, float *__restrict__ gscale, uint64_t *__restrict__ scores,
    float *__restrict__ ramax, int gx, int gy) {
  __shared__ __align__(16) unsigned char lds[kPre2Lds];
  const int b = blockIdx.x;
  if (b < nr) {
    constexpr int kw = qdr::kTokBlock / 32;
    qdr::route_rank_rows(b, T, E, k, ids, counts, ranks, reinterpret_cast<uint32_t(*)[kw]>(lds),
                         reinterpret_cast<uint8_t(*)[kw]>(lds + qdr::kMaxE * kw * 4));
  } else {
    const int q = b - nr;
    qdq::quantize_act_rows<uint16_t, RAC>(
        q % gx, q / gx, gy, x, T, H, part, np, codes, scales, gscale, scores, ramax,
        reinterpret_cast<uint64_t(*)[qdq::kQuantPartCols]>(lds),
        reinterpret_cast<float *>(lds + 16 * qdq::kQuantPartCols * 8));
  }
}

// routing scatter (nr workgroups) | RAC channel selection (one workgroup)
template <int PER>
__global__ __launch_bounds__(256) void layer_pre3_kernel(
    int64_t T, int E, int k, int nr, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ counts, const int32_t *__restrict__ ranks,
    int32_t *__restrict__ offsets, int32_t *__restrict__ row_token, int32_t *__restrict__ inv_row,
    const uint64_t *__restrict__ scores, int K, int Ks, int32_t *__restrict__ sel,
    uint32_t *__restrict__ bitmap) {
  const int b = blockIdx.x;
  if (b < nr)
    qdr::route_scatter_body(b, T, E, k, nr, ids, counts, ranks, offsets, row_token, inv_row);
  else
    qdc::rac_select_body<PER>(scores, K, Ks, sel, bitmap);
}

__global__ __launch_bounds__(256) void layer_scatter_kernel(
    int64_t T, int E, int k, int nr, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ counts, const int32_t *__restrict__ ranks,
    int32_t *__restrict__ offsets, int32_t *__restrict__ row_token,
    int32_t *__restrict__ inv_row) {
  qdr::route_scatter_body(blockIdx.x, T, E, k, nr, ids, counts, ranks, offsets, row_token,
                          inv_row);
}

// the masked residual over all channels (sel not NULL: workgroup 0 also lists
// S from the bitmap, for K <= 8192)
__global__ __launch_bounds__(256) void layer_resq_kernel(
    const uint16_t *__restrict__ x, const uint8_t *__restrict__ xcodes,
    const uint8_t *__restrict__ xscales, const float *__restrict__ xgs, int64_t T, int64_t K,
    const float *__restrict__ ramax, const uint32_t *__restrict__ bitmap,
    uint8_t *__restrict__ rcodes, uint8_t *__restrict__ rscales, float *__restrict__ rgs,
    int32_t *__restrict__ sel) {
  if (sel && blockIdx.x == 0) {
    __shared__ int sh[1024 + 32];
    qdc::rac_list_selected(bitmap, (int)K, sel, sh);
  }
  qdc::rac_resq_body(blockIdx.x, gridDim.x, x, xcodes, xscales, xgs, T, K, ramax, bitmap, rcodes,
                     rscales, rgs);
}

// the residual at the selected channels, compacted per token (what the
// prefill W13 kernel consumes), with the residual's tensor scale
// (bitmap not NULL: S comes as the selection bitmap; every workgroup lists
// it into LDS, and workgroup 0 also into sel for the GEMM)
// (workgroup bid of nblk)
__device__ __forceinline__ void compact_part(
    int bid, int nblk, const uint16_t *__restrict__ x, const uint8_t *__restrict__ xcodes,
    const uint8_t *__restrict__ xscales, const float *__restrict__ xgs, int64_t T, int64_t K,
    const float *__restrict__ ramax, int32_t *__restrict__ sel, int Ks, int width,
    uint16_t *__restrict__ out, float *__restrict__ rgs, const uint32_t *__restrict__ bitmap) {
  __shared__ int32_t lsel[qdc::kRankSelMaxK];
  __shared__ int sh[1024 + 32];
  const int32_t *sp = sel;
  if (bitmap) {
    qdc::rac_list_selected(bitmap, (int)K, lsel, sh);
    __syncthreads();
    if (bid == 0)
      for (int i = threadIdx.x; i < Ks; i += blockDim.x) sel[i] = lsel[i];
    sp = lsel;
  }
  qdc::rac_compact_body(bid, nblk, x, xcodes, xscales, xgs, T, K, ramax, sp, Ks, width, out, rgs);
}

__global__ __launch_bounds__(256) void layer_compact_kernel(
    const uint16_t *__restrict__ x, const uint8_t *__restrict__ xcodes,
    const uint8_t *__restrict__ xscales, const float *__restrict__ xgs, int64_t T, int64_t K,
    const float *__restrict__ ramax, int32_t *__restrict__ sel, int Ks, int width,
    uint16_t *__restrict__ out, float *__restrict__ rgs, const uint32_t *__restrict__ bitmap) {
  compact_part(blockIdx.x, gridDim.x, x, xcodes, xscales, xgs, T, K, ramax, sel, Ks, width, out,
               rgs, bitmap);
}

// routing scatter (nr workgroups) | RAC channel selection by rank and the
// masked residual, one workgroup per 16-channel block (K / 16 workgroups);
// 1024 threads per workgroup
__global__ __launch_bounds__(qdc::kRankSelThreads) void layer_pre3r_kernel(
    int64_t T, int E, int k, int nr, const int32_t *__restrict__ ids,
    const int32_t *__restrict__ counts, const int32_t *__restrict__ ranks,
    int32_t *__restrict__ offsets, int32_t *__restrict__ row_token, int32_t *__restrict__ inv_row,
    const uint64_t *__restrict__ scores, int K, int Ks, uint32_t *__restrict__ bitmap,
    const uint16_t *__restrict__ x, const uint8_t *__restrict__ xcodes,
    const uint8_t *__restrict__ xscales, const float *__restrict__ xgs,
    const float *__restrict__ ramax, uint8_t *__restrict__ rcodes, uint8_t *__restrict__ rscales,
    float *__restrict__ rgs) {
  const int b = blockIdx.x;
  if (b < nr)
    qdr::route_scatter_body(b, T, E, k, nr, ids, counts, ranks, offsets, row_token, inv_row);
  else
    qdc::rac_rank_select_body(b - nr, scores, K, Ks, bitmap, x, xcodes, xscales, xgs, T, ramax,
                              rcodes, rscales, rgs);
}

// The quantised activations of every grouped row copied stage-major for the
// W13 tile GEMM (its A loads of one stage then read one contiguous 8 KB
// piece per tile instead of 32 bytes from each of 256 gathered rows): codes
// [K / 64][R][32 B], then the scales of four stages at a time [K / 256][R][16 B].
// Grid (ceil(2R / 256), K / 64 + K / 256): row y < K / 64 is code stage y,
// thread x its 16-byte piece x % 2 of grouped row x / 2; the rows after are
// scale group y - K / 64, thread x grouped row x.  Consecutive threads write
// consecutive 16-byte pieces.
__device__ __forceinline__ void stage_part(int64_t bx, int64_t y,
                                           const int32_t *__restrict__ row_token,
                                           const uint8_t *__restrict__ codes,
                                           const uint8_t *__restrict__ scales, int64_t R,
                                           int64_t K, uint8_t *__restrict__ out) {
  const int64_t x = bx * 256 + threadIdx.x;
  const int64_t nst = K / 64;
  uint4 *o = reinterpret_cast<uint4 *>(out);
  if (y < nst) {
    if (x >= 2 * R) return;
    const int64_t r = x >> 1, half = x & 1;
    const int64_t t = row_token[r];
    o[y * 2 * R + x] = *reinterpret_cast<const uint4 *>(codes + t * (K / 2) + 32 * y + 16 * half);
  } else {
    if (x >= R) return;
    const int64_t g = y - nst;
    const int64_t t = row_token[x];
    o[R * (K / 32) + g * R + x] = *reinterpret_cast<const uint4 *>(scales + t * (K / 16) + 16 * g);
  }
}

__global__ __launch_bounds__(256) void layer_stage_kernel(const int32_t *__restrict__ row_token,
                                                          const uint8_t *__restrict__ codes,
                                                          const uint8_t *__restrict__ scales,
                                                          int64_t R, int64_t K,
                                                          uint8_t *__restrict__ out) {
  stage_part(blockIdx.x, blockIdx.y, row_token, codes, scales, R, K, out);
}

// the compact residual (gc workgroups) | the staged W13 operand (gxs x gys
// workgroups of layer_stage_kernel's grid, x fastest) in one launch: the two
// are independent and run side by side
__global__ __launch_bounds__(256) void layer_compact_stage_kernel(
    const uint16_t *__restrict__ x, const uint8_t *__restrict__ xcodes,
    const uint8_t *__restrict__ xscales, const float *__restrict__ xgs, int64_t T, int64_t K,
    const float *__restrict__ ramax, int32_t *__restrict__ sel, int Ks, int width,
    uint16_t *__restrict__ out, float *__restrict__ rgs, const uint32_t *__restrict__ bitmap,
    int gc, const int32_t *__restrict__ row_token, int64_t R, int64_t gxs,
    uint8_t *__restrict__ stg) {
  const int b = blockIdx.x;
  if (b < gc) {
    compact_part(b, gc, x, xcodes, xscales, xgs, T, K, ramax, sel, Ks, width, out, rgs, bitmap);
  } else {
    const int64_t q = b - gc;
    stage_part(q % gxs, q / gxs, row_token, xcodes, xscales, R, K, stg);
  }
}

struct Layout {
  int64_t off[QD_VIEW_COUNT];
  int64_t route_ws, q1_ws, sel_ws, q2_ws, sel2_ws, stg, stg_bytes, total;
  // the block entry point's extra views after the layer's workspace: the
  // normalised state x and the router logits
  int64_t xn, lg, block_total;
};

Layout make_layout(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I) {
  Layout L{};
  const int64_t R = T * k;
  int64_t o = 0;
  auto put = [&](int idx, int64_t bytes) {
    L.off[idx] = o;
    o += (int64_t)qdh::align_up((size_t)(bytes > 0 ? bytes : 1));
  };
  auto blob = [&](int64_t bytes) {
    int64_t at = o;
    o += (int64_t)qdh::align_up((size_t)(bytes > 0 ? bytes : 1));
    return at;
  };
  put(QD_VIEW_TOPK_IDS, R * 4);
  put(QD_VIEW_TOPK_W, R * 4);
  put(QD_VIEW_OFFSETS, (int64_t)(E + 1) * 4);
  put(QD_VIEW_ROW_TOKEN, R * 4);
  put(QD_VIEW_INV_ROW, R * 4);
  L.route_ws = blob((int64_t)moe_route_permute_workspace(T, E, k));
  put(QD_VIEW_XQ_CODES, T * H / 2);
  put(QD_VIEW_XQ_SCALES, T * H / 16);
  put(QD_VIEW_XQ_GSCALE, 8);
  L.q1_ws = blob((int64_t)nvfp4_quantize_act_workspace(T, H));
  put(QD_VIEW_SCORES, H * 8);
  put(QD_VIEW_RAMAX, 4);
  put(QD_VIEW_SEL, H * 4);
  L.sel_ws = blob((int64_t)rac_select_channels_workspace(T, H));
  put(QD_VIEW_RQ_CODES, T * H / 2);
  put(QD_VIEW_RQ_SCALES, T * H / 16);
  put(QD_VIEW_RQ_GSCALE, 8);
  put(QD_VIEW_H, R * I * 2);
  {
    // one partial per W13 workgroup; the kernel (and so the count) depends on K_s
    const int64_t c0 = moe_w4a4_grouped_gemm_amax_count(R, 2 * I, H, E, 0, QD_EPI_SWIGLU);
    const int64_t c1 = moe_w4a4_grouped_gemm_amax_count(R, 2 * I, H, E, (int32_t)H, QD_EPI_SWIGLU);
    put(QD_VIEW_H_AMAX, (c0 > c1 ? c0 : c1) * 4);
  }
  put(QD_VIEW_HQ_CODES, R * I / 2);
  put(QD_VIEW_HQ_SCALES, R * I / 16);
  put(QD_VIEW_HQ_GSCALE, 8);
  L.q2_ws = blob((int64_t)nvfp4_quantize_act_workspace(R, I));
  put(QD_VIEW_Z, R * H * 2);
  put(QD_VIEW_RQ_SEL, T * H * 2);       // the compact residual, K_s <= H columns
  // RAC at the W2 input (K_s2 > 0): statistics, selection and masked
  // residual of h over the R permuted rows
  put(QD_VIEW_H_SCORES, I * 8);
  put(QD_VIEW_H_RAMAX, 4);
  put(QD_VIEW_SEL2, I * 4);
  L.sel2_ws = blob((int64_t)rac_select_channels_workspace(R, I));
  put(QD_VIEW_HR_CODES, R * I / 2);
  put(QD_VIEW_HR_SCALES, R * I / 16);
  put(QD_VIEW_HR_GSCALE, 8);
  put(QD_VIEW_HR_SEL, R * (int64_t)rac_selected_width((int32_t)I) * 2);
  // the staged W13 operand, where the tile GEMM may take it
  L.stg_bytes = qdi::gemm_stage_reserve(R, E, 2 * I, H, QD_EPI_SWIGLU);
  L.stg = blob(L.stg_bytes);
  L.total = o;
  L.xn = blob(T * H * 2);
  L.lg = blob(T * (int64_t)E * 4);
  L.block_total = o;
  return L;
}

}  // namespace

extern "C" size_t qd_moe_layer_workspace(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I) {
  if (T < 0 || H <= 0 || E < 1 || k < 1 || I <= 0) return 0;
  return (size_t)make_layout(T, H, E, k, I).total;
}

extern "C" qd_status qd_moe_layer_views(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I,
                                        int64_t *off) {
  if (!off) return QD_ERR_NULL;
  if (T < 0 || H <= 0 || E < 1 || k < 1 || I <= 0) return QD_ERR_SHAPE;
  Layout L = make_layout(T, H, E, k, I);
  for (int i = 0; i < QD_VIEW_COUNT; ++i) off[i] = L.off[i];
  return QD_OK;
}

extern "C" qd_status qd_moe_layer_forward(const void *x, const float *logits, int64_t T,
                                          int64_t H, int32_t E, int32_t k, int64_t I,
                                          int32_t Ks, int32_t Ks2, int32_t renorm,
                                          const qd_nvfp4 *w13, const qd_nvfp4 *w2, void *y,
                                          void *ws, size_t ws_bytes, void *stream) {
  return qd_moe_layer_forward_timed(x, logits, T, H, E, k, I, Ks, Ks2, renorm, w13, w2, y, ws,
                                    ws_bytes, nullptr, stream);
}

namespace {

// the block entry point's input path (RMSNorm + router ahead of the layer)
struct BlockIn {
  const void *h, *gamma, *w_router;
  float eps;
};

qd_status layer_impl(const void *x, const float *logits, int64_t T, int64_t H, int32_t E,
                     int32_t k, int64_t I, int32_t Ks, int32_t Ks2, int32_t renorm,
                     const qd_nvfp4 *w13, const qd_nvfp4 *w2, void *y, void *ws, size_t ws_bytes,
                     void *const *events, void *stream, const BlockIn *blk) {
  if (!w13 || !w2) return QD_ERR_NULL;
  if (T < 0 || H <= 0 || H % 16 || I <= 0 || I % 16 || E < 1 || k < 1 || k > E) return QD_ERR_SHAPE;
  if (Ks < 0 || Ks > H || Ks2 < 0 || Ks2 > I) return QD_ERR_SHAPE;
  // routing limits (as moe_route_permute) and the fused channel selection
  if (E > qdr::kMaxE || k > qdr::kMaxK || T * (int64_t)k > 0x7fffffffLL) return QD_ERR_SHAPE;
  if (Ks > 0 && H > qdc::kSelMaxK) return QD_ERR_UNSUPPORTED;
  qd_status st = qdh::check_nvfp4(w13, E, 2 * I, H);
  if (st) return st;
  st = qdh::check_nvfp4(w2, E, H, I);
  if (st) return st;
  if (blk && (E > kBlkMaxE || block_tok(T, H) == 0)) return QD_ERR_UNSUPPORTED;
  if (T == 0) return QD_OK;
  if (blk ? (!blk->h || !blk->gamma || !blk->w_router || !y) : (!x || !logits || !y))
    return QD_ERR_NULL;
  if (blk && !(blk->eps >= 0.0f && blk->eps < INFINITY)) return QD_ERR_SHAPE;
  if (!ws) return QD_ERR_WORKSPACE;
  Layout L = make_layout(T, H, E, k, I);
  if (ws_bytes < (size_t)(blk ? L.block_total : L.total)) return QD_ERR_WORKSPACE;
  if (!qdh::aligned16(ws) || !qdh::aligned16(y)) return QD_ERR_ALIGN;
  if (blk ? (!qdh::aligned16(blk->h) || !qdh::aligned16(blk->gamma) ||
             !qdh::aligned16(blk->w_router))
          : (!qdh::aligned16(x) || !qdh::aligned16(logits)))
    return QD_ERR_ALIGN;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  char *b = static_cast<char *>(ws);
  if (blk) {
    x = b + L.xn;
    logits = reinterpret_cast<const float *>(b + L.lg);
  }
  auto P = [&](int idx) { return b + L.off[idx]; };
  const int64_t R = T * k;
  auto mark = [&](int i) {
    if (events) (void)hipEventRecord(reinterpret_cast<hipEvent_t>(events[i]), qdh::S(stream));
  };
  int32_t *ids = (int32_t *)P(QD_VIEW_TOPK_IDS);
  float *wts = (float *)P(QD_VIEW_TOPK_W);
  int32_t *offs = (int32_t *)P(QD_VIEW_OFFSETS);
  int32_t *row_token = (int32_t *)P(QD_VIEW_ROW_TOKEN);
  int32_t *inv_row = (int32_t *)P(QD_VIEW_INV_ROW);

  qd_nvfp4 xq{(uint8_t *)P(QD_VIEW_XQ_CODES), (uint8_t *)P(QD_VIEW_XQ_SCALES),
              (float *)P(QD_VIEW_XQ_GSCALE), 1, T, H};
  qd_nvfp4 rq{(uint8_t *)P(QD_VIEW_RQ_CODES), (uint8_t *)P(QD_VIEW_RQ_SCALES),
              (float *)P(QD_VIEW_RQ_GSCALE), 1, T, H};
  uint64_t *scores = (uint64_t *)P(QD_VIEW_SCORES);
  float *ramax = (float *)P(QD_VIEW_RAMAX);
  int32_t *sel = (int32_t *)P(QD_VIEW_SEL);
  const bool rac = Ks > 0;
  // the W13 kernel for many rows per expert takes the residual compacted
  const bool want_sel = rac && qdi::gemm_wants_rq_sel(R, E, 2 * I, H, Ks, QD_EPI_SWIGLU);
  // where the W13 GEMM is the decode kernel (H <= 4096): the selection by
  // rank with the masked residual, one workgroup per 16-channel block, and
  // S listed by the GEMM from the bitmap (elsewhere the one-workgroup
  // selection, which lists S itself, then the masked residual or its
  // compact form)
  const bool rank_sel = rac && !want_sel && H <= qdc::kRankSelMaxK &&
                        qdi::gemm_takes_bitmap(R, E, 2 * I, H, Ks, QD_EPI_SWIGLU);
  // for the compact residual (H <= 4096) the selection by rank alone, with S
  // listed from the bitmap by the compact-residual kernel
  const bool rank_only = want_sel && H <= qdc::kRankSelMaxK;
  // every other RAC case with H <= 4096 (the dense residual pass of the tile
  // kernel): the selection by rank as well, then the masked residual, whose
  // first workgroup lists S from the bitmap
  const bool rank_dense = rac && !want_sel && !rank_sel && H <= qdc::kRankSelMaxK;
  void *rq_sel = want_sel ? P(QD_VIEW_RQ_SEL) : nullptr;
  hipStream_t s = qdh::S(stream);
  // routing scratch, amax partials of X and the channel bitmap (the same
  // carving the standalone calls use)
  const int nr = (int)((T + qdr::kTokBlock - 1) / qdr::kTokBlock);
  int32_t *counts = reinterpret_cast<int32_t *>(b + L.route_ws);
  int32_t *ranks = reinterpret_cast<int32_t *>(b + L.route_ws +
                                               qdh::align_up((size_t)nr * E * 4));
  float *part = reinterpret_cast<float *>(b + L.q1_ws);
  uint32_t *bitmap = reinterpret_cast<uint32_t *>(b + L.sel_ws);
  const int ntopk = qdr::topk_groups(T, E);
  const int64_t n16 = T * H / 16;
  const int ga = qdq::amax_grid(n16);
  int gx, gy;
  qdq::quant_grid(T, H, rac, gx, gy);

  // the staged W13 operand (timed with the steps before the GEMM, so that
  // the W13 stage is the GEMM launch alone); with the compact residual it is
  // written by the same launch
  const int64_t stg_bytes = rank_sel ? 0 : qdi::gemm_stage_bytes(R, E, 2 * I, H, Ks, QD_EPI_SWIGLU);
  const bool staged = stg_bytes > 0 && stg_bytes <= L.stg_bytes;
  uint8_t *stg = reinterpret_cast<uint8_t *>(b + L.stg);
  const int64_t gxs = (2 * R + 255) / 256, gys = H / 64 + H / 256;
  if (staged && (gxs > 0x7fffffffLL || gys > 65535 || gxs * gys > 0x7fff0000LL))
    return QD_ERR_UNSUPPORTED;
  bool stg_done = false;
  mark(QD_STAGE_ROUTE);
  int np = ga;      // amax partials of X
  if (blk) {
    const int tok = block_tok(T, H);
    const int64_t ntb = (T + tok - 1) / tok;
    np = (int)(ntb < qdq::kAmaxPartials ? ntb : qdq::kAmaxPartials);
    void *xw = const_cast<void *>(x);
    float *lw = const_cast<float *>(logits);
    uint64_t *sc = rac ? scores : nullptr;
    float *ra = rac ? ramax : nullptr;
    if (tok == 32)
      launch_pre0<32>(E, np, s, blk->h, blk->gamma, blk->eps, blk->w_router, T, H, k, renorm, xw,
                      lw, ids, wts, part, sc, ra);
    else if (tok == 16)
      launch_pre0<16>(E, np, s, blk->h, blk->gamma, blk->eps, blk->w_router, T, H, k, renorm, xw,
                      lw, ids, wts, part, sc, ra);
    else
      launch_pre0<8>(E, np, s, blk->h, blk->gamma, blk->eps, blk->w_router, T, H, k, renorm, xw,
                     lw, ids, wts, part, sc, ra);
  } else {
    hipLaunchKernelGGL(layer_pre1_kernel, dim3((unsigned)(ntopk + ga)), dim3(256), 0, s, logits,
                       T, E, k, renorm, ids, wts, ntopk, x, n16, part, ga,
                       rac ? scores : nullptr, H, rac ? ramax : nullptr);
  }
  mark(QD_STAGE_QUANT_X);
  if (rac)
    hipLaunchKernelGGL(layer_pre2_kernel<true>, dim3((unsigned)(nr + gx * gy)), dim3(256), 0, s,
                       T, E, k, ids, counts, ranks, nr, x, H, part, np, xq.codes, xq.scales,
                       xq.gscale, scores, ramax, gx, gy);
  else
    hipLaunchKernelGGL(layer_pre2_kernel<false>, dim3((unsigned)(nr + gx * gy)), dim3(256), 0, s,
                       T, E, k, ids, counts, ranks, nr, x, H, part, np, xq.codes, xq.scales,
                       xq.gscale, nullptr, nullptr, gx, gy);
  mark(QD_STAGE_SELECT);
  if (rac) {
    const dim3 g3((unsigned)(nr + 1));
    if (rank_sel || rank_only || rank_dense)
      hipLaunchKernelGGL(layer_pre3r_kernel, dim3((unsigned)(nr + H / 16)),
                         dim3(qdc::kRankSelThreads), 0, s, T,
                         E, k, nr, ids, counts, ranks, offs, row_token, inv_row, scores, (int)H,
                         Ks, bitmap, static_cast<const uint16_t *>(x), xq.codes, xq.scales,
                         xq.gscale, ramax, rank_sel ? rq.codes : nullptr, rq.scales, rq.gscale);
    else if (H <= 2048)
      hipLaunchKernelGGL(layer_pre3_kernel<8>, g3, dim3(256), 0, s, T, E, k, nr, ids, counts,
                         ranks, offs, row_token, inv_row, scores, (int)H, Ks, sel, bitmap);
    else if (H <= 4096)
      hipLaunchKernelGGL(layer_pre3_kernel<16>, g3, dim3(256), 0, s, T, E, k, nr, ids, counts,
                         ranks, offs, row_token, inv_row, scores, (int)H, Ks, sel, bitmap);
    else
      hipLaunchKernelGGL(layer_pre3_kernel<64>, g3, dim3(256), 0, s, T, E, k, nr, ids, counts,
                         ranks, offs, row_token, inv_row, scores, (int)H, Ks, sel, bitmap);
    if (want_sel) {
      // the prefill W13 kernel takes the residual at S only: computed
      // directly for the blocks that hold a selected channel (the full
      // masked residual is not materialised)
      const int width = rac_selected_width(Ks);
      const int64_t total = T * width;
      int64_t g = (total + 255) / 256;
      if (g > 8192) g = 8192;
      if (g < 1) g = 1;
      if (staged) {
        hipLaunchKernelGGL(layer_compact_stage_kernel, dim3((unsigned)(g + gxs * gys)), dim3(256),
                           0, s, static_cast<const uint16_t *>(x), xq.codes, xq.scales, xq.gscale,
                           T, H, ramax, sel, Ks, width, static_cast<uint16_t *>(rq_sel),
                           rq.gscale, rank_only ? bitmap : nullptr, (int)g, row_token, R, gxs,
                           stg);
        stg_done = true;
      } else {
        hipLaunchKernelGGL(layer_compact_kernel, dim3((unsigned)g), dim3(256), 0, s,
                           static_cast<const uint16_t *>(x), xq.codes, xq.scales, xq.gscale, T,
                           H, ramax, sel, Ks, width, static_cast<uint16_t *>(rq_sel), rq.gscale,
                           rank_only ? bitmap : nullptr);
      }
    } else if (!rank_sel) {
      const int64_t total = T * (H / 16);
      int64_t g = (total + 255) / 256;
      if (g > 4096) g = 4096;
      if (g < 1) g = 1;
      hipLaunchKernelGGL(layer_resq_kernel, dim3((unsigned)g), dim3(256), 0, s,
                         static_cast<const uint16_t *>(x), xq.codes, xq.scales, xq.gscale, T, H,
                         ramax, bitmap, rq.codes, rq.scales, rq.gscale,
                         rank_dense ? sel : nullptr);
    }
  } else {
    hipLaunchKernelGGL(layer_scatter_kernel, dim3((unsigned)nr), dim3(256), 0, s, T, E, k, nr,
                       ids, counts, ranks, offs, row_token, inv_row);
  }
  st = qdh::check_launch();
  if (st) return st;
  uint16_t *h = (uint16_t *)P(QD_VIEW_H);
  float *hamax = (float *)P(QD_VIEW_H_AMAX);
  if (staged && !stg_done) {
    hipLaunchKernelGGL(layer_stage_kernel, dim3((unsigned)gxs, (unsigned)gys), dim3(256), 0, s,
                       row_token, xq.codes, xq.scales, R, H, stg);
  }
  mark(QD_STAGE_W13);
  if (rank_sel) {
    st = qdi::grouped_gemm_bitmap(&xq, row_token, offs, E, R, w13, &rq, bitmap, Ks, sel,
                                  QD_EPI_SWIGLU, h, hamax, s);
  } else if (staged) {
    st = qdi::grouped_gemm_staged(&xq, row_token, offs, E, R, w13, &rq, sel, Ks, rq_sel,
                                  QD_EPI_SWIGLU, h, hamax, stg, s);
  } else {
    st = moe_w4a4_grouped_gemm(&xq, row_token, offs, E, R, w13, rac ? &rq : nullptr,
                               rac ? sel : nullptr, Ks, rq_sel, QD_EPI_SWIGLU, h, hamax, stream);
  }
  if (st) return st;
  qd_nvfp4 hq{(uint8_t *)P(QD_VIEW_HQ_CODES), (uint8_t *)P(QD_VIEW_HQ_SCALES),
              (float *)P(QD_VIEW_HQ_GSCALE), 1, R, I};
  mark(QD_STAGE_QUANT_H);
  const bool rac2 = Ks2 > 0;
  qd_nvfp4 hr{(uint8_t *)P(QD_VIEW_HR_CODES), (uint8_t *)P(QD_VIEW_HR_SCALES),
              (float *)P(QD_VIEW_HR_GSCALE), 1, R, I};
  int32_t *sel2 = (int32_t *)P(QD_VIEW_SEL2);
  uint32_t *bitmap2 = reinterpret_cast<uint32_t *>(b + L.sel2_ws);
  void *hr_sel = nullptr;
  bool bm2 = false;                 // the W2 GEMM takes S as a bitmap
  if (!rac2) {
    st = nvfp4_quantize_act(h, QD_DTYPE_BF16, R, I, hamax,
                            qdi::gemm_amax_written(R, E, 2 * I, H, Ks, QD_EPI_SWIGLU,
                                                   w13->scales_frag != nullptr, rank_sel),
                            &hq, nullptr, nullptr, b + L.q2_ws,
                            nvfp4_quantize_act_workspace(R, I), stream);
    if (st) return st;
  } else {
    // the scored quantiser takes its own amax pass over h (which also
    // clears the score accumulators), then the W2-site selection
    uint64_t *hscores = (uint64_t *)P(QD_VIEW_H_SCORES);
    float *hramax = (float *)P(QD_VIEW_H_RAMAX);
    st = nvfp4_quantize_act(h, QD_DTYPE_BF16, R, I, nullptr, 0, &hq, hscores, hramax,
                            b + L.q2_ws, nvfp4_quantize_act_workspace(R, I), stream);
    if (st) return st;
    // as at the W13 site: for I <= 4096 the selection by rank (one
    // workgroup per 16-channel block; no routing workgroups here), with the
    // masked residual for the decode GEMM in bitmap mode, with S listed by
    // the compact-residual kernel for the tile GEMM, or (the dense residual
    // pass) with S listed by the masked-residual launch
    const bool want2 = qdi::gemm_wants_rq_sel(R, E, H, I, Ks2, QD_EPI_NONE);
    bm2 = !want2 && I <= qdc::kRankSelMaxK &&
          qdi::gemm_takes_bitmap(R, E, H, I, Ks2, QD_EPI_NONE);
    const bool ro2 = want2 && I <= qdc::kRankSelMaxK;
    const bool rd2 = !want2 && !bm2 && I <= qdc::kRankSelMaxK;
    if (want2) hr_sel = P(QD_VIEW_HR_SEL);
    if (bm2 || ro2 || rd2) {
      hipLaunchKernelGGL(layer_pre3r_kernel, dim3((unsigned)(I / 16)),
                         dim3(qdc::kRankSelThreads), 0, s, R, E, k, 0, ids, counts, ranks, offs,
                         row_token, inv_row, hscores, (int)I, Ks2, bitmap2, h, hq.codes,
                         hq.scales, hq.gscale, hramax, bm2 ? hr.codes : nullptr, hr.scales,
                         hr.gscale);
      if (ro2) {
        const int width = rac_selected_width(Ks2);
        int64_t g = (R * width + 255) / 256;
        if (g > 8192) g = 8192;
        if (g < 1) g = 1;
        hipLaunchKernelGGL(layer_compact_kernel, dim3((unsigned)g), dim3(256), 0, s, h, hq.codes,
                           hq.scales, hq.gscale, R, I, hramax, sel2, Ks2, width,
                           static_cast<uint16_t *>(hr_sel), hr.gscale, bitmap2);
      } else if (rd2) {
        int64_t g = (R * (I / 16) + 255) / 256;
        if (g > 4096) g = 4096;
        if (g < 1) g = 1;
        hipLaunchKernelGGL(layer_resq_kernel, dim3((unsigned)g), dim3(256), 0, s, h, hq.codes,
                           hq.scales, hq.gscale, R, I, hramax, bitmap2, hr.codes, hr.scales,
                           hr.gscale, sel2);
      }
      st = qdh::check_launch();
      if (st) return st;
    } else {
      st = rac_select_channels(h, &hq, Ks2, hscores, hramax, 1, sel2, &hr, b + L.sel2_ws,
                               rac_select_channels_workspace(R, I), stream);
      if (st) return st;
      if (want2) {
        st = rac_gather_selected(&hr, sel2, Ks2, hr_sel, stream);
        if (st) return st;
      }
    }
  }
  uint16_t *z = (uint16_t *)P(QD_VIEW_Z);
  mark(QD_STAGE_W2);
  if (bm2)
    st = qdi::grouped_gemm_bitmap(&hq, nullptr, offs, E, R, w2, &hr, bitmap2, Ks2, sel2,
                                  QD_EPI_NONE, z, nullptr, s);
  else
    st = moe_w4a4_grouped_gemm(&hq, nullptr, offs, E, R, w2, rac2 ? &hr : nullptr,
                               rac2 ? sel2 : nullptr, Ks2, hr_sel, QD_EPI_NONE, z, nullptr,
                               stream);
  if (st) return st;
  mark(QD_STAGE_COMBINE);
  st = moe_unpermute_combine(z, inv_row, wts, T, k, H, y, stream);
  if (st) return st;
  mark(QD_STAGE_COUNT);
  return qdh::check_launch();
}

}  // namespace

extern "C" qd_status qd_moe_layer_forward_timed(const void *x, const float *logits, int64_t T,
                                                int64_t H, int32_t E, int32_t k, int64_t I,
                                                int32_t Ks, int32_t Ks2, int32_t renorm,
                                                const qd_nvfp4 *w13, const qd_nvfp4 *w2, void *y,
                                                void *ws, size_t ws_bytes,
                                                void *const *events, void *stream) {
  return layer_impl(x, logits, T, H, E, k, I, Ks, Ks2, renorm, w13, w2, y, ws, ws_bytes, events,
                    stream, nullptr);
}

extern "C" size_t qd_moe_block_workspace(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I) {
  if (T < 0 || H <= 0 || E < 1 || k < 1 || I <= 0) return 0;
  return (size_t)make_layout(T, H, E, k, I).block_total;
}

extern "C" qd_status qd_moe_block_views(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I,
                                        int64_t *off) {
  if (!off) return QD_ERR_NULL;
  if (T < 0 || H <= 0 || E < 1 || k < 1 || I <= 0) return QD_ERR_SHAPE;
  Layout L = make_layout(T, H, E, k, I);
  for (int i = 0; i < QD_VIEW_COUNT; ++i) off[i] = L.off[i];
  off[QD_BLOCK_VIEW_X] = L.xn;
  off[QD_BLOCK_VIEW_LOGITS] = L.lg;
  return QD_OK;
}

extern "C" qd_status qd_moe_block_forward_timed(const void *h, const void *gamma, float eps,
                                                const void *w_router, int64_t T, int64_t H,
                                                int32_t E, int32_t k, int64_t I, int32_t Ks,
                                                int32_t Ks2, int32_t renorm, const qd_nvfp4 *w13,
                                                const qd_nvfp4 *w2, void *y, void *ws,
                                                size_t ws_bytes, void *const *events,
                                                void *stream) {
  const BlockIn blk{h, gamma, w_router, eps};
  return layer_impl(nullptr, nullptr, T, H, E, k, I, Ks, Ks2, renorm, w13, w2, y, ws, ws_bytes,
                    events, stream, &blk);
}

extern "C" qd_status qd_moe_block_forward(const void *h, const void *gamma, float eps,
                                          const void *w_router, int64_t T, int64_t H, int32_t E,
                                          int32_t k, int64_t I, int32_t Ks, int32_t Ks2,
                                          int32_t renorm, const qd_nvfp4 *w13, const qd_nvfp4 *w2,
                                          void *y, void *ws, size_t ws_bytes, void *stream) {
  return qd_moe_block_forward_timed(h, gamma, eps, w_router, T, H, E, k, I, Ks, Ks2, renorm, w13,
                                    w2, y, ws, ws_bytes, nullptr, stream);
}

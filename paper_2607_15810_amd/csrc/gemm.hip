// Grouped W4A4 expert GEMM with the RAC residual fused into the K loop
// (paper, Sec. 3.3: the main GEMM stays on NVFP4 codes and the selected
// channels add a residual contraction, Eq. (residual-recon)).
//
// Exact NVFP4 on gfx950.  The native scaled MFMA of CDNA4 takes one E8M0
// (power-of-two) scale per 32 elements; NVFP4 carries an E4M3 scale (three
// mantissa bits) per 16.  Its product e2m1 * e4m3 has at most 6 significant
// bits and lies in [2^-10, 2688], so it is exact in f16.  The kernels decode
// each operand fragment in registers -- a scaled FP4->f16 convert (power of
// two only) and one packed f16 multiply by the scale's mantissa -- and feed
// v_mfma_f32_16x16x32_f16.  Products of two decoded operands (<= 12
// significant bits) are exact in the f32 accumulator; the tensor scales are
// applied once in the epilogue.
//
// Fragment layout (16x16x32 MFMA, wave64): lane l holds A[l%16][8*(l/16)+j]
// and B[8*(l/16)+j][l%16], j = 0..7; C[4*(l/16)+i][l%16], i = 0..3.  A lane
// loads 16 contiguous code bytes (32 elements) of its row per 128-element K
// chunk; k-step s of the chunk uses its elements 8s..8s+7.  A and B use the
// same assignment, so each MFMA reduces over a permuted but common K subset.
#include "common.h"

namespace {

using namespace qd;

struct GemmArgs {
  const uint8_t *a_codes;
  const uint8_t *a_scales;
  const float *a_gs;
  const int32_t *row_token;
  const int32_t *offsets;
  int E;
  int64_t rows;
  const uint8_t *w_codes;
  const uint8_t *w_scales;
  const float *w_gs;
  int N;
  int K;
  const uint8_t *r_codes;
  const uint8_t *r_scales;
  const float *r_gs;
  const int32_t *sel;
  int Ks;
  uint16_t *out;
  float *amax_part;
};

constexpr int BM = 64;
constexpr int BN = 64;     // weight rows per workgroup (32 gate/up pairs for SwiGLU)

__device__ __forceinline__ f32x4 mfma16(f16x8 a, f16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t word_of(uint4 v, int s) {
  return s == 0 ? v.x : (s == 1 ? v.y : (s == 2 ? v.z : v.w));
}

// find the (expert, first row) of m-tile mt; false if mt is past the last tile
__device__ __forceinline__ bool locate_tile(const GemmArgs &p, int mt, int &e, int64_t &rb,
                                            int64_t &re) {
  if (!p.offsets) {
    e = 0;
    rb = (int64_t)mt * BM;
    re = min(p.rows, rb + BM);
    return rb < p.rows;
  }
  int acc = 0;
  for (int x = 0; x < p.E; ++x) {
    const int o0 = p.offsets[x], o1 = p.offsets[x + 1];
    const int nt = (o1 - o0 + BM - 1) / BM;
    if (mt < acc + nt) {
      e = x;
      rb = o0 + (int64_t)(mt - acc) * BM;
      re = min((int64_t)o1, rb + BM);
      return true;
    }
    acc += nt;
  }
  return false;
}

template <bool GATHER, bool RAC, int EPI>
__global__ __launch_bounds__(256) void gemm_w4a4_kernel(GemmArgs p) {
  __shared__ float red[16];
  __shared__ uint32_t selmap[RAC ? 2048 : 1];       // K <= 65536 channels
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w & 1, wn = w >> 1;
  const int lr = lane & 15, g = lane >> 4;
  const int K = p.K, N = p.N;
  const int64_t kb2 = K >> 1, kb16 = K >> 4;

  int e;
  int64_t rb, re;
  const bool have = locate_tile(p, blockIdx.x, e, rb, re);
  if (RAC) {
    for (int i = threadIdx.x; i < (K + 31) / 32; i += blockDim.x) selmap[i] = 0u;
    __syncthreads();
    for (int i = threadIdx.x; i < p.Ks; i += blockDim.x) {
      const int j = p.sel[i];
      atomicOr(&selmap[j >> 5], 1u << (j & 31));
    }
    __syncthreads();
  }
  float vmax = 0.0f;
  if (have) {
    // operand rows of this lane
    const uint8_t *ac[2], *as[2], *rc[2], *rs[2];
    bool av[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int64_t gr = rb + wm * 32 + i * 16 + lr;
      av[i] = gr < re;
      int64_t src = 0;
      if (av[i]) src = GATHER ? (int64_t)p.row_token[gr] : gr;
      ac[i] = p.a_codes + src * kb2 + g * 16;
      as[i] = p.a_scales + src * kb16 + g * 2;
      if (RAC) {
        rc[i] = p.r_codes + src * kb2 + g * 16;
        rs[i] = p.r_scales + src * kb16 + g * 2;
      }
    }
    const uint8_t *bc[2], *bs[2];
    bool bv[2];
    int64_t wrow[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      int64_t n;
      if (EPI == QD_EPI_SWIGLU) {
        const int I = N >> 1;
        n = (int64_t)blockIdx.y * 32 + wn * 16 + lr + (j ? I : 0);
        bv[j] = ((int64_t)blockIdx.y * 32 + wn * 16 + lr) < I;
      } else {
        n = (int64_t)blockIdx.y * BN + wn * 32 + j * 16 + lr;
        bv[j] = n < N;
      }
      wrow[j] = n;
      const int64_t wr = bv[j] ? n : 0;
      bc[j] = p.w_codes + ((int64_t)e * N + wr) * kb2 + g * 16;
      bs[j] = p.w_scales + ((int64_t)e * N + wr) * kb16 + g * 2;
    }
    (void)wrow;
    const bool wave_active = __any((int)(av[0] || av[1]));
    f32x4 acc[2][2], accr[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        accr[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    if (wave_active) {
      const int nchunk = (K + 127) / 128;
      for (int c = 0; c < nchunk; ++c) {
        const bool gval = (c * 128 + g * 32 + 32) <= K;
        uint4 a4[2], b4[2], r4[2];
        uint32_t asc[2], bsc[2], rsc[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const bool ok = av[i] && gval;
          a4[i] = ok ? *reinterpret_cast<const uint4 *>(ac[i] + c * 64) : make_uint4(0, 0, 0, 0);
          asc[i] = ok ? *reinterpret_cast<const uint16_t *>(as[i] + c * 8) : 0u;
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const bool ok = bv[j] && gval;
          b4[j] = ok ? *reinterpret_cast<const uint4 *>(bc[j] + c * 64) : make_uint4(0, 0, 0, 0);
          bsc[j] = ok ? *reinterpret_cast<const uint16_t *>(bs[j] + c * 8) : 0u;
        }
        uint32_t smask = 0u;   // k-steps of this chunk holding a selected channel
        if (RAC) {
          const uint32_t w0 = selmap[c * 4 + 0], w1 = selmap[c * 4 + 1];
          const uint32_t w2 = (c * 4 + 2) * 32 < K ? selmap[c * 4 + 2] : 0u;
          const uint32_t w3 = (c * 4 + 3) * 32 < K ? selmap[c * 4 + 3] : 0u;
          const uint32_t any = w0 | w1 | w2 | w3;
#pragma unroll
          for (int s = 0; s < 4; ++s) smask |= (((any >> (8 * s)) & 0xFFu) != 0u) << s;
          if (smask) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {
              const bool ok = av[i] && gval;
              r4[i] = ok ? *reinterpret_cast<const uint4 *>(rc[i] + c * 64) : make_uint4(0, 0, 0, 0);
              rsc[i] = ok ? *reinterpret_cast<const uint16_t *>(rs[i] + c * 8) : 0u;
            }
          }
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          f16x8 af[2], bf[2];
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            const uint32_t sp = scale_pair_f16(asc[i] & 0xFFu, asc[i] >> 8);
            af[i] = decode8(word_of(a4[i], s), s < 2 ? splat_lo(sp) : splat_hi(sp));
          }
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const uint32_t sp = scale_pair_f16(bsc[j] & 0xFFu, bsc[j] >> 8);
            bf[j] = decode8(word_of(b4[j], s), s < 2 ? splat_lo(sp) : splat_hi(sp));
          }
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] = mfma16(af[i], bf[j], acc[i][j]);
          if (RAC && ((smask >> s) & 1u)) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {
              const uint32_t sp = scale_pair_f16(rsc[i] & 0xFFu, rsc[i] >> 8);
              f16x8 rf = decode8(word_of(r4[i], s), s < 2 ? splat_lo(sp) : splat_hi(sp));
#pragma unroll
              for (int j = 0; j < 2; ++j) accr[i][j] = mfma16(rf, bf[j], accr[i][j]);
            }
          }
        }
      }
      // epilogue
      const float sw = p.w_gs[2 * e + 1];
      const float alpha = p.a_gs[1] * sw;
      const float alpha_r = RAC ? p.r_gs[1] * sw : 0.0f;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int64_t row = rb + wm * 32 + i * 16 + g * 4 + q;
          if (row >= re) continue;
          if (EPI == QD_EPI_SWIGLU) {
            const int I = N >> 1;
            const int64_t col = (int64_t)blockIdx.y * 32 + wn * 16 + lr;
            if (col < I) {
              float gv = alpha * acc[i][0][q];
              float uv = alpha * acc[i][1][q];
              if (RAC) {
                gv = gv - alpha_r * accr[i][0][q];
                uv = uv - alpha_r * accr[i][1][q];
              }
              const float h = gv / (1.0f + expf(-gv)) * uv;
              const uint32_t hb = f32_to_bf16_bits(h);
              p.out[row * I + col] = (uint16_t)hb;
              vmax = fmaxf(vmax, fabsf(bf16_bits_to_f32(hb)));
            }
          } else {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
              const int64_t col = (int64_t)blockIdx.y * BN + wn * 32 + j * 16 + lr;
              if (col < N) {
                float v = alpha * acc[i][j][q];
                if (RAC) v = v - alpha_r * accr[i][j][q];
                const uint32_t hb = f32_to_bf16_bits(v);
                p.out[row * N + col] = (uint16_t)hb;
                vmax = fmaxf(vmax, fabsf(bf16_bits_to_f32(hb)));
              }
            }
          }
        }
      }
    }
  }
  const float m = block_max(vmax, red);
  if (p.amax_part && threadIdx.x == 0) p.amax_part[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = m;
}

inline int64_t grid_x(int64_t rows, int E, bool grouped) {
  return (rows + BM - 1) / BM + (grouped ? E : 0);
}
inline int64_t grid_y(int64_t N, int epilogue) {
  return epilogue == QD_EPI_SWIGLU ? ((N / 2) + 31) / 32 : (N + BN - 1) / BN;
}

template <bool GATHER, bool RAC>
void launch_epi(const GemmArgs &p, int epi, dim3 grid, hipStream_t s) {
  if (epi == QD_EPI_SWIGLU)
    hipLaunchKernelGGL((gemm_w4a4_kernel<GATHER, RAC, QD_EPI_SWIGLU>), grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((gemm_w4a4_kernel<GATHER, RAC, QD_EPI_NONE>), grid, dim3(256), 0, s, p);
}

}  // namespace

extern "C" int64_t moe_w4a4_grouped_gemm_amax_count(int64_t rows, int64_t N, int32_t E,
                                                    int32_t epilogue) {
  if (rows < 0 || N <= 0 || E < 1) return 0;
  return grid_x(rows, E, true) * grid_y(N, epilogue);
}

extern "C" qd_status moe_w4a4_grouped_gemm(const qd_nvfp4 *a, const int32_t *row_token,
                                           const int32_t *expert_offsets, int32_t E, int64_t rows,
                                           const qd_nvfp4 *w, const qd_nvfp4 *rq,
                                           const int32_t *sel_idx, int32_t Ks, int32_t epilogue,
                                           void *out, float *amax_partials, void *stream) {
  if (!a || !w || !out) return QD_ERR_NULL;
  if (epilogue != QD_EPI_NONE && epilogue != QD_EPI_SWIGLU) return QD_ERR_DTYPE;
  if (E < 1 || rows < 0) return QD_ERR_SHAPE;
  const int64_t K = a->cols;
  qd_status st = qdh::check_nvfp4(a, 1, a->rows, K);
  if (st) return st;
  st = qdh::check_nvfp4(w, E, w->rows, K);
  if (st) return st;
  const int64_t N = w->rows;
  if (K % 32 != 0 || N % 16 != 0 || N <= 0) return QD_ERR_SHAPE;
  if (epilogue == QD_EPI_SWIGLU && (N % 32 != 0)) return QD_ERR_SHAPE;
  if (!expert_offsets && E != 1) return QD_ERR_SHAPE;
  if (!row_token && rows > a->rows) return QD_ERR_SHAPE;
  const bool rac = rq != nullptr && Ks > 0;
  if (rac) {
    st = qdh::check_nvfp4(rq, 1, rq->rows, K);
    if (st) return st;
    if (!sel_idx) return QD_ERR_NULL;
    if (Ks > K || rq->rows != a->rows) return QD_ERR_SHAPE;
    if (K > 65536) return QD_ERR_UNSUPPORTED;
  }
  if (Ks < 0) return QD_ERR_SHAPE;
  if (!qdh::aligned16(out) || (amax_partials && ((uintptr_t)amax_partials & 3u)))
    return QD_ERR_ALIGN;
  if (N > 0x7fffffff || K > 0x7fffffff) return QD_ERR_UNSUPPORTED;
  const int64_t gx = grid_x(rows, E, true), gy = grid_y(N, epilogue);
  if (gx > 0x7fffffffLL || gy > 65535) return QD_ERR_UNSUPPORTED;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  if (rows == 0) return QD_OK;

  GemmArgs p{};
  p.a_codes = a->codes;
  p.a_scales = a->scales;
  p.a_gs = a->gscale;
  p.row_token = row_token;
  p.offsets = expert_offsets;
  p.E = E;
  p.rows = rows;
  p.w_codes = w->codes;
  p.w_scales = w->scales;
  p.w_gs = w->gscale;
  p.N = (int)N;
  p.K = (int)K;
  if (rac) {
    p.r_codes = rq->codes;
    p.r_scales = rq->scales;
    p.r_gs = rq->gscale;
    p.sel = sel_idx;
    p.Ks = Ks;
  }
  p.out = static_cast<uint16_t *>(out);
  p.amax_part = amax_partials;
  dim3 grid((unsigned)gx, (unsigned)gy);
  hipStream_t s = qdh::S(stream);
  if (row_token) {
    if (rac) launch_epi<true, true>(p, epilogue, grid, s);
    else launch_epi<true, false>(p, epilogue, grid, s);
  } else {
    if (rac) launch_epi<false, true>(p, epilogue, grid, s);
    else launch_epi<false, false>(p, epilogue, grid, s);
  }
  return qdh::check_launch();
}

// FP8 W8A8 MoE expert layer: the comparison baseline of the paper's FP8
// rollout (Sec. 2.2 "FP8" paragraph), on the same routing, SwiGLU and combine
// as the NVFP4 layer and without residual compensation.
//
// Scaling: E4M3 codes, one f32 scale per row -- per token for activations,
// per output channel for weights.  For a row with amax m > 0, enc = 448 / m
// and dec = 1 / enc (f32); code = E4M3_RNE(min(|x * enc|, 448)) with the sign
// in bit 7; a zero row takes enc = dec = 1.  Products of two E4M3 values are
// exact in f32; the row scales are applied in the epilogue.
//
// GEMM: v_mfma_scale_f32_32x32x64_f8f6f4 with both block scales 1.0 (the
// f8f6f4 path, twice the f16 MFMA rate), K = 64 per instruction.  The same
// structure as the NVFP4 prefill kernel: M-tiles inside one expert, tile
// indices contiguous per XCD, a ring of 64-element stages filled by direct
// global->LDS loads (six per wave and stage), operands read a stage ahead.
//  * TM = 256 (many rows per expert): tile 256 x 128 weight rows, 2 x 2 waves
//    of 128 x 64 (4 x 2 fragments), two workgroups per CU.
//  * TM = 32 (decode): tile 32 x 256 weight rows, 1 x 4 waves of 32 x 64 (two
//    fragments each); the weights are the traffic, streamed once per 32-row
//    pass of an expert.
// Stage slot: A codes [TM/32 fragments][64 lanes][32 B], then B codes
// [NT/32 fragments] likewise; lane l of a fragment holds row l % 32,
// elements 32 (l / 32) .. +31 of the stage, for A and B alike (one common
// K order inside every MFMA).
#include "common.h"
#include "lds_dma.h"
#include "tile_sched.h"

namespace {

using namespace qd;
using namespace qdl;

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------- quantise
// One wave per row, four rows per workgroup: amax over the row, then codes.
template <typename T>
__device__ __forceinline__ float load_as_f32(const T *p, int64_t i);
template <>
__device__ __forceinline__ float load_as_f32<uint16_t>(const uint16_t *p, int64_t i) {
  return bf16_bits_to_f32(p[i]);
}
template <>
__device__ __forceinline__ float load_as_f32<float>(const float *p, int64_t i) {
  return p[i];
}

template <typename T>
__global__ __launch_bounds__(256) void fp8_quantize_rows_kernel(const T *__restrict__ x,
                                                                int64_t rows, int64_t K,
                                                                uint8_t *__restrict__ codes,
                                                                float *__restrict__ dec) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const T *xr = x + r * K;
  float m = 0.0f;
  for (int64_t i = lane; i < K; i += 64) m = fmaxf(m, fabsf(load_as_f32(xr, i)));
  m = wave_max(m);
  const bool zero = !(m > 0.0f);
  const float enc = zero ? 1.0f : 448.0f / m;
  if (lane == 0) dec[r] = 1.0f / enc;
  uint8_t *cr = codes + r * K;
  for (int64_t i = lane; i < K; i += 64) {
    const float v = load_as_f32(xr, i);
    const float t = fminf(fabsf(v * enc), 448.0f);
    cr[i] = (uint8_t)(e4m3_encode_pos(t) | (signbit(v) ? 0x80u : 0u));
  }
}

// ---------------------------------------------------------------- GEMM
struct Fp8Args {
  const uint8_t *a_codes;
  const float *a_dec;
  const int32_t *row_token;
  const int32_t *offsets;
  int E;
  int64_t rows;
  const uint8_t *w_codes;
  const float *w_dec;
  int N;
  int K;
  uint16_t *out;
};

constexpr int F8_THREADS = 256;
constexpr int F8_K = 64;
constexpr int F8_EMAX = 1024;
constexpr int F8_LDS_MAX = 160 * 1024 - 1024;

template <int TM>
struct F8Cfg {
  static constexpr int NT = TM == 256 ? 128 : 256;     // weight rows per tile
  static constexpr int NS = TM == 256 ? 3 : 4;         // ring depth
  static constexpr int AF = TM / 32, BF = NT / 32;     // fragments per stage
  static constexpr int ACODE = 0, BCODE = AF * 2048;
  static constexpr int STAGE = (AF + BF) * 2048;
  static constexpr int MTV_MAX = TM == 256 ? 4 : 1;    // A fragments per wave
  static constexpr int LDS = NS * STAGE + (TM + NT) * 4;   // ring + row scales
};

// weight row of the tile's row tb: for SwiGLU the first half of the tile's
// fragments are gate rows, the second half the matching up rows
template <int TM, int EPI>
__device__ __forceinline__ int f8_wrow(int tb, int nt, int N) {
  constexpr int NT = F8Cfg<TM>::NT;
  if (EPI == QD_EPI_SWIGLU) {
    constexpr int half = NT / 2;
    return (tb < half ? 0 : (N >> 1)) + nt * half + (tb % half);
  }
  return nt * NT + tb;
}

__device__ __forceinline__ f32x16 mfma_f8(v8i a, v8i b, f32x16 c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 127, 0, 127);
}

template <int MTV>
struct F8Raw {
  v8i a[MTV > 0 ? MTV : 1], b[2];
};

template <bool GATHER, int EPI, int TM>
__global__ __launch_bounds__(F8_THREADS, 2) void gemm_fp8_kernel(Fp8Args p, int ntn) {
  using C = F8Cfg<TM>;
  constexpr int NS = C::NS, NT = C::NT;
  extern __shared__ __align__(16) unsigned char lds[];
  __shared__ int sh_w[4];
  __shared__ int sh_t[4];
  const int tid = threadIdx.x, lane = tid & 63, w = (int)uni((uint32_t)tid >> 6);
  const int K = p.K, N = p.N, E = p.E;

  const qdt::Tile tl = qdt::find_tile<TM>(p.offsets, p.E, p.rows, ntn, sh_w, sh_t);
  const int e = tl.e;
  if (e < 0) return;
  const int row0 = tl.row0, nrows = tl.nrows, nt = tl.nt;
  const uint32_t lds0 = (uint32_t)(uintptr_t)lds;
  float *sa = reinterpret_cast<float *>(lds + NS * C::STAGE);     // [TM] activation row scales
  float *sw = sa + TM;                                            // [NT] weight row scales
  auto arow = [&](int r) __attribute__((always_inline)) -> uint32_t {
    const int rr = r < nrows ? r : 0;
    return GATHER ? (uint32_t)p.row_token[row0 + rr] : (uint32_t)(row0 + rr);
  };
  for (int i = tid; i < TM; i += F8_THREADS) sa[i] = p.a_dec[arow(i)];
  for (int i = tid; i < NT; i += F8_THREADS)
    sw[i] = p.w_dec[(int64_t)e * N + f8_wrow<TM, EPI>(i, nt, N)];
  // ---- per-lane load offsets (32-bit, from uniform bases): six loads per
  // wave and stage.  A fragment's 2 KB slot is two loads of 1 KB: lane i of
  // the first brings row i / 2, bytes 16 (i % 2) .. +15 of the stage (the
  // first half of read lane i / 2), the second the same rows 32 bytes on.
  const uint32_t hb = 16u * (uint32_t)(lane & 1);
  uint32_t oa[2], ob[2];
  int fa[2], fb[2];
  if (TM == 256) {
    fa[0] = 2 * w; fa[1] = 2 * w + 1;                            // A fragments of this wave
    fb[0] = w; fb[1] = w;                                        // one B fragment, both halves
  } else {
    fa[0] = 0; fa[1] = 0;                                        // every wave: the A fragment
    fb[0] = 2 * w; fb[1] = 2 * w + 1;
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    oa[j] = arow(32 * fa[j] + (lane >> 1)) * (uint32_t)K + hb;
    ob[j] = (uint32_t)f8_wrow<TM, EPI>(32 * fb[j] + (lane >> 1), nt, N) * (uint32_t)K + hb;
  }
  const uint8_t *wc = uni_ptr(p.w_codes + (int64_t)e * N * K);
  const int nst = K / F8_K;
  auto issue = [&](int s, int q) __attribute__((always_inline)) {
    s = min(s, nst - 1);
    const uint32_t sb = uni(lds0 + q * C::STAGE);
    const uint8_t *ac = uni_ptr(p.a_codes + s * F8_K), *bc = uni_ptr(wc + s * F8_K);
    if (TM == 256) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        dma16s(ac, oa[j], sb + C::ACODE + fa[j] * 2048);
        dma16s(ac, oa[j] + 32, sb + C::ACODE + fa[j] * 2048 + 1024);
      }
      dma16s(bc, ob[0], sb + C::BCODE + fb[0] * 2048);
      dma16s(bc, ob[0] + 32, sb + C::BCODE + fb[0] * 2048 + 1024);
    } else {
      dma16s(ac, oa[0], sb + C::ACODE);
      dma16s(ac, oa[0] + 32, sb + C::ACODE + 1024);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        dma16s(bc, ob[j], sb + C::BCODE + fb[j] * 2048);
        dma16s(bc, ob[j] + 32, sb + C::BCODE + fb[j] * 2048 + 1024);
      }
    }
  };
  // wave layout
  const int wm = TM == 256 ? (w & 1) : 0;
  const int wn = TM == 256 ? (w >> 1) : w;
  const int fa0 = TM == 256 ? 4 * wm : 0;
  const int mtv = TM == 256 ? min(max((nrows - 128 * wm + 31) >> 5, 0), 4) : 1;
  // B fragments of this wave: SwiGLU pairs a gate fragment with its up one
  const int fbw0 = EPI == QD_EPI_SWIGLU ? wn : 2 * wn;
  const int fbw1 = EPI == QD_EPI_SWIGLU ? wn + C::BF / 2 : 2 * wn + 1;

  auto run = [&](auto mtv_c) __attribute__((always_inline)) {
    constexpr int MTV = decltype(mtv_c)::value;
    f32x16 acc[MTV > 0 ? MTV : 1][2];
#pragma unroll
    for (int i = 0; i < (MTV > 0 ? MTV : 1); ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int t = 0; t < 16; ++t) acc[i][j][t] = 0.0f;
    auto rd = [&](F8Raw<MTV> &R, const unsigned char *sl) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < MTV; ++i)
        R.a[i] = *reinterpret_cast<const v8i *>(sl + C::ACODE + (fa0 + i) * 2048 + lane * 32);
      R.b[0] = *reinterpret_cast<const v8i *>(sl + C::BCODE + fbw0 * 2048 + lane * 32);
      R.b[1] = *reinterpret_cast<const v8i *>(sl + C::BCODE + fbw1 * 2048 + lane * 32);
    };
    F8Raw<MTV> R0, R1;
#pragma unroll
    for (int t = 0; t < NS - 1; ++t) issue(t, t);
    wait_vm<(NS - 2) * 6>();
    __syncthreads();
    if constexpr (MTV > 0) rd(R0, lds);
    auto body = [&](const F8Raw<MTV> &Rc, F8Raw<MTV> &Rn, int s) __attribute__((always_inline)) {
      if constexpr (MTV > 0) {
#pragma unroll
        for (int i = 0; i < MTV; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[i][j] = mfma_f8(Rc.a[i], Rc.b[j], acc[i][j]);
      }
      wait_vm<(NS - 3) * 6>();
      __syncthreads();
      issue(s + NS - 1, (s + NS - 1) % NS);
      if constexpr (MTV > 0) rd(Rn, lds + ((s + 1) % NS) * C::STAGE);
    };
    int s = 0;
    for (; s + 1 < nst; s += 2) {
      body(R0, R1, s);
      body(R1, R0, s + 1);
    }
    if (s < nst) body(R0, R1, s);
    wait_vm<0>();
    if constexpr (MTV > 0) {
      // ---- epilogue: row scales, SwiGLU or plain, bf16 pairs of adjacent
      // columns swapped between neighbouring lanes (4-byte stores)
      const int h = lane >> 5;
      const bool odd = (lane & 1) != 0;
      const int cpair = (lane & 31) & ~1, col = lane & 31;
      const int ldo = EPI == QD_EPI_SWIGLU ? (N >> 1) : N;
      unsigned char *obase = reinterpret_cast<unsigned char *>(p.out);
      constexpr int NO = EPI == QD_EPI_SWIGLU ? 1 : 2;
#pragma unroll
      for (int i = 0; i < MTV; ++i) {
        const int rl = 32 * (fa0 + i) + 4 * h + (odd ? 1 : 0);
#pragma unroll
        for (int jj = 0; jj < NO; ++jj) {
          const int fb = jj == 0 ? fbw0 : fbw1;
          const int cb = EPI == QD_EPI_SWIGLU ? nt * (NT / 2) + fb * 32 : nt * NT + fb * 32;
          const uint32_t voff = (uint32_t)((row0 + rl) * ldo + cb + cpair) * 2u;
          const float s0 = sw[fb * 32 + col];
          const float s1 = EPI == QD_EPI_SWIGLU ? sw[fbw1 * 32 + col] : 0.0f;
          float v[16];
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            const float ra = sa[32 * (fa0 + i) + 8 * (q >> 2) + 4 * h + (q & 3)];
            if (EPI == QD_EPI_SWIGLU) {
              const float g = ra * s0 * acc[i][0][q], u = ra * s1 * acc[i][1][q];
              const float ex = __builtin_amdgcn_exp2f(-g * 1.4426950408889634f);
              v[q] = g * __builtin_amdgcn_rcpf(1.0f + ex) * u;
            } else {
              v[q] = ra * s0 * acc[i][jj][q];
            }
          }
#pragma unroll
          for (int q = 0; q < 16; q += 2) {
            const float send = odd ? v[q] : v[q + 1];
            const float x = __int_as_float(
                __builtin_amdgcn_mov_dpp(__float_as_int(send), 0xB1, 0xF, 0xF, false));
            const f32x2_t pr = odd ? f32x2_t{x, v[q + 1]} : f32x2_t{v[q], x};
            const uint32_t pk = __builtin_bit_cast(uint32_t, __builtin_convertvector(pr, bf16x2_t));
            const int qr = 8 * (q >> 2) + (q & 3);
            if (rl + qr < nrows)
              *reinterpret_cast<uint32_t *>(obase + (size_t)(qr * ldo * 2) + voff) = pk;
          }
        }
      }
    }
  };
  if (TM == 256) {
    switch (mtv) {
      case 4: run(std::integral_constant<int, 4>{}); break;
      case 3: run(std::integral_constant<int, 3>{}); break;
      case 2: run(std::integral_constant<int, 2>{}); break;
      case 1: run(std::integral_constant<int, 1>{}); break;
      default: run(std::integral_constant<int, 0>{}); break;
    }
  } else {
    run(std::integral_constant<int, 1>{});
  }
}

// rows per expert above which the 256-row tiles replace the 32-row passes
constexpr int64_t F8_DECODE_ROWS = 48;

struct F8Plan {
  bool ok;
  int tm, ntn, grid, lds;
};

inline F8Plan fp8_plan(int64_t rows, int E, int64_t N, int64_t K, int epilogue) {
  F8Plan pl{};
  pl.tm = rows > (int64_t)E * F8_DECODE_ROWS ? 256 : 32;
  const int nt = pl.tm == 256 ? F8Cfg<256>::NT : F8Cfg<32>::NT;
  if (K < 4 * F8_K || K % F8_K != 0 || N % nt != 0 || E > F8_EMAX) return pl;
  if (epilogue == QD_EPI_SWIGLU && (N / 2) % (nt / 2) != 0) return pl;
  if (N * K >= (1LL << 32) || (rows + 1) * K >= (1LL << 32) || (rows + 256) * N * 2 >= (1LL << 32))
    return pl;
  pl.ntn = (int)(N / nt);
  pl.lds = pl.tm == 256 ? F8Cfg<256>::LDS : F8Cfg<32>::LDS;
  const int64_t g = qdt::tile_grid(rows, E, pl.tm, pl.ntn);
  if (g > 0x7fffffffLL) return pl;
  pl.grid = (int)g;
  pl.ok = true;
  return pl;
}

template <bool GATHER, int EPI, int TM>
void launch_fp8(const Fp8Args &p, const F8Plan &pl, hipStream_t s) {
  auto kern = gemm_fp8_kernel<GATHER, EPI, TM>;
  static const bool attr = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               F8_LDS_MAX) == hipSuccess;
  (void)attr;
  hipLaunchKernelGGL(kern, dim3((unsigned)pl.grid), dim3(F8_THREADS), (size_t)pl.lds, s, p,
                     pl.ntn);
}

template <bool GATHER>
void launch_fp8_epi(const Fp8Args &p, const F8Plan &pl, int epi, hipStream_t s) {
  if (pl.tm == 256) {
    if (epi == QD_EPI_SWIGLU) launch_fp8<GATHER, QD_EPI_SWIGLU, 256>(p, pl, s);
    else launch_fp8<GATHER, QD_EPI_NONE, 256>(p, pl, s);
  } else {
    if (epi == QD_EPI_SWIGLU) launch_fp8<GATHER, QD_EPI_SWIGLU, 32>(p, pl, s);
    else launch_fp8<GATHER, QD_EPI_NONE, 32>(p, pl, s);
  }
}

}  // namespace

extern "C" qd_status fp8_quantize_rows(const void *x, int32_t dtype, int64_t rows, int64_t cols,
                                       uint8_t *codes, float *dec, void *stream) {
  if (rows < 0 || cols < 0) return QD_ERR_SHAPE;
  if (dtype != QD_DTYPE_BF16 && dtype != QD_DTYPE_F32) return QD_ERR_DTYPE;
  if (rows == 0 || cols == 0) return QD_OK;
  if (!x || !codes || !dec) return QD_ERR_NULL;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  const int64_t g = (rows + 3) / 4;
  if (g > 0x7fffffffLL) return QD_ERR_UNSUPPORTED;
  hipStream_t s = qdh::S(stream);
  if (dtype == QD_DTYPE_BF16)
    hipLaunchKernelGGL(fp8_quantize_rows_kernel<uint16_t>, dim3((unsigned)g), dim3(256), 0, s,
                       static_cast<const uint16_t *>(x), rows, cols, codes, dec);
  else
    hipLaunchKernelGGL(fp8_quantize_rows_kernel<float>, dim3((unsigned)g), dim3(256), 0, s,
                       static_cast<const float *>(x), rows, cols, codes, dec);
  return qdh::check_launch();
}

extern "C" qd_status moe_fp8_grouped_gemm(const uint8_t *a_codes, const float *a_dec,
                                          int64_t a_rows, const int32_t *row_token,
                                          const int32_t *expert_offsets, int32_t E, int64_t rows,
                                          const uint8_t *w_codes, const float *w_dec, int64_t N,
                                          int64_t K, int32_t epilogue, void *out, void *stream) {
  if (!a_codes || !a_dec || !w_codes || !w_dec || !out) return QD_ERR_NULL;
  if (epilogue != QD_EPI_NONE && epilogue != QD_EPI_SWIGLU) return QD_ERR_DTYPE;
  if (E < 1 || rows < 0 || a_rows < 0 || N <= 0 || K <= 0) return QD_ERR_SHAPE;
  if (!expert_offsets && E != 1) return QD_ERR_SHAPE;
  if (!row_token && rows > a_rows) return QD_ERR_SHAPE;
  if (!qdh::aligned16(a_codes) || !qdh::aligned16(w_codes) || !qdh::aligned16(out))
    return QD_ERR_ALIGN;
  const F8Plan pl = fp8_plan(rows, E, N, K, epilogue);
  if (!pl.ok) return QD_ERR_UNSUPPORTED;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  if (rows == 0) return QD_OK;
  Fp8Args p{};
  p.a_codes = a_codes;
  p.a_dec = a_dec;
  p.row_token = row_token;
  p.offsets = expert_offsets;
  p.E = E;
  p.rows = rows;
  p.w_codes = w_codes;
  p.w_dec = w_dec;
  p.N = (int)N;
  p.K = (int)K;
  p.out = static_cast<uint16_t *>(out);
  hipStream_t s = qdh::S(stream);
  if (row_token) launch_fp8_epi<true>(p, pl, epilogue, s);
  else launch_fp8_epi<false>(p, pl, epilogue, s);
  return qdh::check_launch();
}

// ---------------------------------------------------------------- layer
namespace {
struct F8Layout {
  size_t route, ids, wts, offs, row_token, inv_row, xc, xd, h, hc, hd, z, total;
};
F8Layout fp8_layer_layout(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I) {
  F8Layout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t at = o; o += qdh::align_up(bytes > 0 ? bytes : 1); return at; };
  const int64_t R = T * k;
  L.route = take(moe_route_permute_workspace(T, E, k));
  L.ids = take((size_t)R * 4);
  L.wts = take((size_t)R * 4);
  L.offs = take((size_t)(E + 1) * 4);
  L.row_token = take((size_t)R * 4);
  L.inv_row = take((size_t)R * 4);
  L.xc = take((size_t)(T * H));
  L.xd = take((size_t)T * 4);
  L.h = take((size_t)(R * I * 2));
  L.hc = take((size_t)(R * I));
  L.hd = take((size_t)R * 4);
  L.z = take((size_t)(R * H * 2));
  L.total = o;
  return L;
}
}  // namespace

extern "C" size_t qd_fp8_moe_layer_workspace(int64_t T, int64_t H, int32_t E, int32_t k,
                                             int64_t I) {
  if (T < 0 || H < 0 || E < 1 || k < 1 || I < 0) return 0;
  return fp8_layer_layout(T, H, E, k, I).total;
}

extern "C" qd_status qd_fp8_moe_layer_forward(const void *x, const float *logits, int64_t T,
                                              int64_t H, int32_t E, int32_t k, int64_t I,
                                              int32_t renorm, const uint8_t *w13_codes,
                                              const float *w13_dec, const uint8_t *w2_codes,
                                              const float *w2_dec, void *y, void *ws,
                                              size_t ws_bytes, void *stream) {
  if (T < 0 || H <= 0 || I <= 0 || E < 1 || k < 1 || k > E) return QD_ERR_SHAPE;
  if (!w13_codes || !w13_dec || !w2_codes || !w2_dec) return QD_ERR_NULL;
  if (T > 0 && (!x || !logits || !y)) return QD_ERR_NULL;
  if (!ws || ws_bytes < qd_fp8_moe_layer_workspace(T, H, E, k, I)) return QD_ERR_WORKSPACE;
  if (!qdh::aligned16(ws) || !qdh::aligned16(y)) return QD_ERR_ALIGN;
  const int64_t R = T * k;
  if (!fp8_plan(R > 0 ? R : 1, E, 2 * I, H, QD_EPI_SWIGLU).ok ||
      !fp8_plan(R > 0 ? R : 1, E, H, I, QD_EPI_NONE).ok)
    return QD_ERR_UNSUPPORTED;
  if (T == 0) return QD_OK;
  const F8Layout L = fp8_layer_layout(T, H, E, k, I);
  unsigned char *b = static_cast<unsigned char *>(ws);
  int32_t *ids = reinterpret_cast<int32_t *>(b + L.ids);
  float *wts = reinterpret_cast<float *>(b + L.wts);
  int32_t *offs = reinterpret_cast<int32_t *>(b + L.offs);
  int32_t *row_token = reinterpret_cast<int32_t *>(b + L.row_token);
  int32_t *inv_row = reinterpret_cast<int32_t *>(b + L.inv_row);
  uint8_t *xc = b + L.xc;
  float *xd = reinterpret_cast<float *>(b + L.xd);
  uint16_t *h = reinterpret_cast<uint16_t *>(b + L.h);
  uint8_t *hc = b + L.hc;
  float *hd = reinterpret_cast<float *>(b + L.hd);
  uint16_t *z = reinterpret_cast<uint16_t *>(b + L.z);
  qd_status st = moe_route_permute(logits, T, E, k, renorm, ids, wts, offs, row_token, inv_row,
                                   b + L.route, moe_route_permute_workspace(T, E, k), stream);
  if (st) return st;
  st = fp8_quantize_rows(x, QD_DTYPE_BF16, T, H, xc, xd, stream);
  if (st) return st;
  st = moe_fp8_grouped_gemm(xc, xd, T, row_token, offs, E, R, w13_codes, w13_dec, 2 * I, H,
                            QD_EPI_SWIGLU, h, stream);
  if (st) return st;
  st = fp8_quantize_rows(h, QD_DTYPE_BF16, R, I, hc, hd, stream);
  if (st) return st;
  st = moe_fp8_grouped_gemm(hc, hd, R, nullptr, offs, E, R, w2_codes, w2_dec, H, I, QD_EPI_NONE,
                            z, stream);
  if (st) return st;
  return moe_unpermute_combine(z, inv_row, wts, T, k, H, y, stream);
}

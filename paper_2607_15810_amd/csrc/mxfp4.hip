// MXFP4 W4A4 MoE expert layer: a comparison layer on the format CDNA4's
// scaled MFMA reads natively.  It uses the same routing, SwiGLU and combine
// as the NVFP4 layer and has no residual compensation.  It measures what
// exact NVFP4 semantics (Sec. 2.2, "FP4" paragraph: an E4M3 scale per 16
// elements and an FP32 tensor scale) cost against the hardware's own FP4
// path, where the scale is a power of two per 32 elements and there is no
// tensor scale.
//
// Format (the OCP Microscaling MX rule): per block of 32 consecutive
// elements of a row, with m = max |v|, s = floor(log2 m) - 2, clamped to
// [-127, 127] (s = -127 for m == 0).  The scale byte is s + 127 (E8M0).
// Element code = E2M1_RNE(|v| * 2^-s) with ties to even, saturating at 6,
// and the sign in bit 3.  Codes u8 [rows][K/2] hold element 2i in bits 3:0;
// scales are u8 [rows][K/32].
//
// GEMM: v_mfma_scale_f32_32x32x64_f8f6f4 with both operands E2M1 (format 4).
// Lane l of a fragment holds row l % 32, elements 32 (l / 32) .. +31 of the
// 64-element stage (16 bytes, element i in nibble i), with that 32-block's
// E8M0 byte as its scale operand.  The kernel structure is that of the FP8
// comparison GEMM: TM = 256 rows x 128 weight rows (2 x 2 waves of 128 x 64)
// for many rows per expert, TM = 32 x 256 (1 x 4 waves) for decode.  Stages
// of 64 elements go through a ring filled by direct global->LDS loads, five
// per wave and stage.  The E8M0 bytes of two stages come in one dword per
// row, re-read at the odd stage (an L2 hit).
//
// Stage slot: A codes [TM/32 fragments][64 lanes][16 B], B codes [NT/32]
// likewise, then A scale dwords [max(TM, 64) rows] and B scale dwords
// [NT rows].
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
template <typename T>
__device__ __forceinline__ float mx_load(const T *p, int64_t i);
template <>
__device__ __forceinline__ float mx_load<uint16_t>(const uint16_t *p, int64_t i) {
  return bf16_bits_to_f32(p[i]);
}
template <>
__device__ __forceinline__ float mx_load<float>(const float *p, int64_t i) {
  return p[i];
}

// floor(log2 m) of a positive finite float, exact for subnormals too
__device__ __forceinline__ int floor_log2_pos(float m) {
  const uint32_t u = __float_as_uint(m);
  const int e = (int)((u >> 23) & 255u);
  if (e != 0) return e - 127;
  return (31 - __builtin_clz(u & 0x7FFFFFu)) - 149;   // m = mantissa * 2^-149
}

// One thread per 32-element block: the block's E8M0 byte and 16 code bytes.
template <typename T>
__global__ __launch_bounds__(256) void mx_quantize_kernel(const T *__restrict__ x, int64_t nblk,
                                                          uint8_t *__restrict__ codes,
                                                          uint8_t *__restrict__ scales) {
  const int64_t b = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (b >= nblk) return;
  const T *xb = x + b * 32;
  float v[32];
  float m = 0.0f;
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    v[i] = mx_load(xb, i);
    m = fmaxf(m, fabsf(v[i]));
  }
  int s = -127;
  if (m > 0.0f) s = min(max(floor_log2_pos(m) - 2, -127), 127);
  scales[b] = (uint8_t)(s + 127);
  // 2^-s, s in [-127, 125] for finite float input: a normal float
  const float inv = __uint_as_float((uint32_t)(127 - s) << 23);
  uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const uint32_t c = e2m1_mag(fabsf(v[i]) * inv) | ((__float_as_uint(v[i]) >> 28) & 8u);
    w[i >> 3] |= c << (4 * (i & 7));
  }
  *reinterpret_cast<uint4 *>(codes + b * 16) = make_uint4(w[0], w[1], w[2], w[3]);
}

// ---------------------------------------------------------------- GEMM
struct MxArgs {
  const uint8_t *a_codes;
  const uint8_t *a_scales;
  const int32_t *row_token;
  const int32_t *offsets;
  int E;
  int64_t rows;
  const uint8_t *w_codes;
  const uint8_t *w_scales;
  int N;
  int K;
  uint16_t *out;
};

constexpr int MX_THREADS = 256;
constexpr int MX_K = 64;
constexpr int MX_EMAX = 1024;
constexpr int MX_LDS_MAX = 160 * 1024 - 1024;
constexpr int MX_LOADS = 5;                          // per wave and stage

template <int TM>
struct MxCfg {
  static constexpr int NT = TM == 256 ? 128 : 256;   // weight rows per tile
  static constexpr int NS = 4;                       // ring depth
  static constexpr int AF = TM / 32, BF = NT / 32;   // fragments per stage
  static constexpr int ACODE = 0, BCODE = AF * 1024;
  static constexpr int ASCL = (AF + BF) * 1024;
  static constexpr int BSCL = ASCL + (TM > 64 ? TM : 64) * 4;
  static constexpr int STAGE = BSCL + NT * 4;
  static constexpr int LDS = NS * STAGE;
};

// weight row of the tile's row tb: for SwiGLU the first half of the tile's
// fragments are gate rows, the second half the matching up rows
template <int TM, int EPI>
__device__ __forceinline__ int mx_wrow(int tb, int nt, int N) {
  constexpr int NT = MxCfg<TM>::NT;
  if (EPI == QD_EPI_SWIGLU) {
    constexpr int half = NT / 2;
    return (tb < half ? 0 : (N >> 1)) + nt * half + (tb % half);
  }
  return nt * NT + tb;
}

// E2M1 x E2M1 with per-lane E8M0 scales (byte 0 of sa / sb)
__device__ __forceinline__ f32x16 mfma_mx(uint4 a, uint4 b, uint32_t sa, uint32_t sb, f32x16 c) {
  const v8i av = {(int)a.x, (int)a.y, (int)a.z, (int)a.w, 0, 0, 0, 0};
  const v8i bv = {(int)b.x, (int)b.y, (int)b.z, (int)b.w, 0, 0, 0, 0};
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, c, 4, 4, 0, (int)sa, 0, (int)sb);
}

template <int MTV>
struct MxRaw {
  uint4 a[MTV > 0 ? MTV : 1], b[2];
  uint32_t as[MTV > 0 ? MTV : 1], bs[2];
};

template <bool GATHER, int EPI, int TM>
__global__ __launch_bounds__(MX_THREADS, 2) void gemm_mxfp4_kernel(MxArgs p, int ntn) {
  using C = MxCfg<TM>;
  constexpr int NS = C::NS, NT = C::NT;
  extern __shared__ __align__(16) unsigned char lds[];
  __shared__ int sh_w[4];
  __shared__ int sh_t[4];
  const int tid = threadIdx.x, lane = tid & 63, w = (int)uni((uint32_t)tid >> 6);
  const int K = p.K, N = p.N;
  const qdt::Tile tl = qdt::find_tile<TM>(p.offsets, p.E, p.rows, ntn, sh_w, sh_t);
  const int e = tl.e;
  if (e < 0) return;
  const int row0 = tl.row0, nrows = tl.nrows, nt = tl.nt;
  const uint32_t lds0 = (uint32_t)(uintptr_t)lds;
  const uint32_t kb2 = (uint32_t)(K >> 1), kb32 = (uint32_t)(K >> 5);
  auto arow = [&](int r) __attribute__((always_inline)) -> uint32_t {
    const int rr = r < nrows ? r : 0;
    return GATHER ? (uint32_t)p.row_token[row0 + rr] : (uint32_t)(row0 + rr);
  };
  // ---- per-lane load offsets (32-bit, from uniform bases).  Codes: lane
  // i of a fragment's load brings row i % 32, bytes 16 (i / 32) .. +15 of
  // the stage's 32.  Scales: lane i brings the dword of stages (2t, 2t + 1)
  // of one row.
  const uint32_t hb = 16u * (uint32_t)(lane >> 5);
  int fa[2], fb[2];
  if (TM == 256) {
    fa[0] = 2 * w; fa[1] = 2 * w + 1;     // A fragments of this wave
    fb[0] = w; fb[1] = w;                 // one B fragment
  } else {
    fa[0] = 0; fa[1] = 0;                 // every wave: the one A fragment
    fb[0] = 2 * w; fb[1] = 2 * w + 1;
  }
  uint32_t oa[2], ob[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    oa[j] = arow(32 * fa[j] + (lane & 31)) * kb2 + hb;
    ob[j] = (uint32_t)mx_wrow<TM, EPI>(32 * fb[j] + (lane & 31), nt, N) * kb2 + hb;
  }
  // scale rows: TM = 256: A rows 64 w + lane, B rows 64 (w & 1) + lane
  // (waves 2, 3 repeat waves 0, 1: equal bytes to equal places); TM = 32:
  // A rows lane % 32 (every wave), B rows 64 w + lane
  const int sar = TM == 256 ? 64 * w + lane : (lane & 31);
  const int sbr = TM == 256 ? 64 * (w & 1) + lane : 64 * w + lane;
  const uint32_t oas = arow(sar) * kb32;
  const uint32_t obs = (uint32_t)mx_wrow<TM, EPI>(sbr, nt, N) * kb32;
  const uint32_t sad = TM == 256 ? (uint32_t)(64 * w * 4) : 0u;
  const uint32_t sbd = TM == 256 ? (uint32_t)(64 * (w & 1) * 4) : (uint32_t)(64 * w * 4);
  const uint8_t *wc = uni_ptr(p.w_codes + (int64_t)e * N * kb2);
  const uint8_t *wsc = uni_ptr(p.w_scales + (int64_t)e * N * kb32);
  const int nst = K / MX_K;
  auto issue = [&](int s, int q) __attribute__((always_inline)) {
    s = min(s, nst - 1);
    const uint32_t sb = uni(lds0 + q * C::STAGE);
    const uint8_t *ac = uni_ptr(p.a_codes + s * 32), *bc = uni_ptr(wc + s * 32);
    const uint8_t *asc = uni_ptr(p.a_scales + (s >> 1) * 4), *bsc = uni_ptr(wsc + (s >> 1) * 4);
    if (TM == 256) {
      dma16s(ac, oa[0], sb + C::ACODE + fa[0] * 1024);
      dma16s(ac, oa[1], sb + C::ACODE + fa[1] * 1024);
      dma16s(bc, ob[0], sb + C::BCODE + fb[0] * 1024);
    } else {
      dma16s(ac, oa[0], sb + C::ACODE);
      dma16s(bc, ob[0], sb + C::BCODE + fb[0] * 1024);
      dma16s(bc, ob[1], sb + C::BCODE + fb[1] * 1024);
    }
    dma4s(asc, oas, sb + C::ASCL + sad);
    dma4s(bsc, obs, sb + C::BSCL + sbd);
  };
  // wave layout
  const int wm = TM == 256 ? (w & 1) : 0;
  const int wn = TM == 256 ? (w >> 1) : w;
  const int fa0 = TM == 256 ? 4 * wm : 0;
  const int mtv = TM == 256 ? min(max((nrows - 128 * wm + 31) >> 5, 0), 4) : 1;
  // B fragments of this wave: SwiGLU pairs a gate fragment with its up one
  const int fbw0 = EPI == QD_EPI_SWIGLU ? wn : 2 * wn;
  const int fbw1 = EPI == QD_EPI_SWIGLU ? wn + C::BF / 2 : 2 * wn + 1;
  const int h = lane >> 5, r32 = lane & 31;

  auto run = [&](auto mtv_c) __attribute__((always_inline)) {
    constexpr int MTV = decltype(mtv_c)::value;
    f32x16 acc[MTV > 0 ? MTV : 1][2];
#pragma unroll
    for (int i = 0; i < (MTV > 0 ? MTV : 1); ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int t = 0; t < 16; ++t) acc[i][j][t] = 0.0f;
    auto rd = [&](MxRaw<MTV> &R, const unsigned char *sl) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < MTV; ++i) {
        R.a[i] = *reinterpret_cast<const uint4 *>(sl + C::ACODE + (fa0 + i) * 1024 + lane * 16);
        R.as[i] = *reinterpret_cast<const uint32_t *>(sl + C::ASCL + (32 * (fa0 + i) + r32) * 4);
      }
      R.b[0] = *reinterpret_cast<const uint4 *>(sl + C::BCODE + fbw0 * 1024 + lane * 16);
      R.b[1] = *reinterpret_cast<const uint4 *>(sl + C::BCODE + fbw1 * 1024 + lane * 16);
      R.bs[0] = *reinterpret_cast<const uint32_t *>(sl + C::BSCL + (32 * fbw0 + r32) * 4);
      R.bs[1] = *reinterpret_cast<const uint32_t *>(sl + C::BSCL + (32 * fbw1 + r32) * 4);
    };
    MxRaw<MTV> R0, R1;
#pragma unroll
    for (int t = 0; t < NS - 1; ++t) issue(t, t);
    wait_vm<(NS - 2) * MX_LOADS>();
    __syncthreads();
    if constexpr (MTV > 0) rd(R0, lds);
    auto body = [&](const MxRaw<MTV> &Rc, MxRaw<MTV> &Rn, int s) __attribute__((always_inline)) {
      if constexpr (MTV > 0) {
        // this lane's 32-block of stage s: byte 2 (s % 2) + h of the dword
        const int sh = 8 * (2 * (s & 1) + h);
        const uint32_t sb0 = (Rc.bs[0] >> sh) & 255u, sb1 = (Rc.bs[1] >> sh) & 255u;
#pragma unroll
        for (int i = 0; i < MTV; ++i) {
          const uint32_t sa = (Rc.as[i] >> sh) & 255u;
          acc[i][0] = mfma_mx(Rc.a[i], Rc.b[0], sa, sb0, acc[i][0]);
          acc[i][1] = mfma_mx(Rc.a[i], Rc.b[1], sa, sb1, acc[i][1]);
        }
      }
      wait_vm<(NS - 3) * MX_LOADS>();
      __syncthreads();
      issue(s + NS - 1, (s + NS - 1) % NS);
      if constexpr (MTV > 0) rd(Rn, lds + ((s + 1) % NS) * C::STAGE);
    };
    for (int s = 0; s < nst; s += 2) {     // nst is even (K % 128 == 0)
      body(R0, R1, s);
      body(R1, R0, s + 1);
    }
    wait_vm<0>();
    if constexpr (MTV > 0) {
      // ---- epilogue: SwiGLU or plain (the scales are inside the MFMA),
      // bf16 pairs of adjacent columns swapped between neighbouring lanes
      // (4-byte stores)
      const bool odd = (lane & 1) != 0;
      const int cpair = r32 & ~1;
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
          float v[16];
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            if (EPI == QD_EPI_SWIGLU) {
              const float g = acc[i][0][q], u = acc[i][1][q];
              const float ex = __builtin_amdgcn_exp2f(-g * 1.4426950408889634f);
              v[q] = g * __builtin_amdgcn_rcpf(1.0f + ex) * u;
            } else {
              v[q] = acc[i][jj][q];
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
constexpr int64_t MX_DECODE_ROWS = 48;

struct MxPlan {
  bool ok;
  int tm, ntn, grid, lds;
};

inline MxPlan mx_plan(int64_t rows, int E, int64_t N, int64_t K, int epilogue) {
  MxPlan pl{};
  pl.tm = rows > (int64_t)E * MX_DECODE_ROWS ? 256 : 32;
  const int nt = pl.tm == 256 ? MxCfg<256>::NT : MxCfg<32>::NT;
  if (K < 4 * MX_K || K % 128 != 0 || N % nt != 0 || E > MX_EMAX) return pl;
  if (epilogue == QD_EPI_SWIGLU && (N / 2) % (nt / 2) != 0) return pl;
  if (N * K / 2 >= (1LL << 32) || (rows + 1) * K / 2 >= (1LL << 32) ||
      (rows + 256) * N * 2 >= (1LL << 32))
    return pl;
  pl.ntn = (int)(N / nt);
  pl.lds = pl.tm == 256 ? MxCfg<256>::LDS : MxCfg<32>::LDS;
  const int64_t g = qdt::tile_grid(rows, E, pl.tm, pl.ntn);
  if (g > 0x7fffffffLL) return pl;
  pl.grid = (int)g;
  pl.ok = true;
  return pl;
}

template <bool GATHER, int EPI, int TM>
void launch_mx(const MxArgs &p, const MxPlan &pl, hipStream_t s) {
  auto kern = gemm_mxfp4_kernel<GATHER, EPI, TM>;
  static const bool attr = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               MX_LDS_MAX) == hipSuccess;
  (void)attr;
  hipLaunchKernelGGL(kern, dim3((unsigned)pl.grid), dim3(MX_THREADS), (size_t)pl.lds, s, p,
                     pl.ntn);
}

template <bool GATHER>
void launch_mx_epi(const MxArgs &p, const MxPlan &pl, int epi, hipStream_t s) {
  if (pl.tm == 256) {
    if (epi == QD_EPI_SWIGLU) launch_mx<GATHER, QD_EPI_SWIGLU, 256>(p, pl, s);
    else launch_mx<GATHER, QD_EPI_NONE, 256>(p, pl, s);
  } else {
    if (epi == QD_EPI_SWIGLU) launch_mx<GATHER, QD_EPI_SWIGLU, 32>(p, pl, s);
    else launch_mx<GATHER, QD_EPI_NONE, 32>(p, pl, s);
  }
}

}  // namespace

extern "C" qd_status mxfp4_quantize_rows(const void *x, int32_t dtype, int64_t rows, int64_t cols,
                                         uint8_t *codes, uint8_t *scales, void *stream) {
  if (rows < 0 || cols < 0 || cols % 32 != 0) return QD_ERR_SHAPE;
  if (dtype != QD_DTYPE_BF16 && dtype != QD_DTYPE_F32) return QD_ERR_DTYPE;
  if (rows == 0 || cols == 0) return QD_OK;
  if (!x || !codes || !scales) return QD_ERR_NULL;
  if (!qdh::aligned16(x) || !qdh::aligned16(codes)) return QD_ERR_ALIGN;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  const int64_t nblk = rows * (cols / 32);
  const int64_t g = (nblk + 255) / 256;
  if (g > 0x7fffffffLL) return QD_ERR_UNSUPPORTED;
  hipStream_t s = qdh::S(stream);
  if (dtype == QD_DTYPE_BF16)
    hipLaunchKernelGGL(mx_quantize_kernel<uint16_t>, dim3((unsigned)g), dim3(256), 0, s,
                       static_cast<const uint16_t *>(x), nblk, codes, scales);
  else
    hipLaunchKernelGGL(mx_quantize_kernel<float>, dim3((unsigned)g), dim3(256), 0, s,
                       static_cast<const float *>(x), nblk, codes, scales);
  return qdh::check_launch();
}

extern "C" qd_status moe_mxfp4_grouped_gemm(const uint8_t *a_codes, const uint8_t *a_scales,
                                            int64_t a_rows, const int32_t *row_token,
                                            const int32_t *expert_offsets, int32_t E,
                                            int64_t rows, const uint8_t *w_codes,
                                            const uint8_t *w_scales, int64_t N, int64_t K,
                                            int32_t epilogue, void *out, void *stream) {
  if (!a_codes || !a_scales || !w_codes || !w_scales || !out) return QD_ERR_NULL;
  if (epilogue != QD_EPI_NONE && epilogue != QD_EPI_SWIGLU) return QD_ERR_DTYPE;
  if (E < 1 || rows < 0 || a_rows < 0 || N <= 0 || K <= 0) return QD_ERR_SHAPE;
  if (!expert_offsets && E != 1) return QD_ERR_SHAPE;
  if (!row_token && rows > a_rows) return QD_ERR_SHAPE;
  if (!qdh::aligned16(a_codes) || !qdh::aligned16(w_codes) || !qdh::aligned16(out) ||
      ((uintptr_t)a_scales & 3u) || ((uintptr_t)w_scales & 3u))
    return QD_ERR_ALIGN;
  const MxPlan pl = mx_plan(rows, E, N, K, epilogue);
  if (!pl.ok) return QD_ERR_UNSUPPORTED;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  if (rows == 0) return QD_OK;
  MxArgs p{};
  p.a_codes = a_codes;
  p.a_scales = a_scales;
  p.row_token = row_token;
  p.offsets = expert_offsets;
  p.E = E;
  p.rows = rows;
  p.w_codes = w_codes;
  p.w_scales = w_scales;
  p.N = (int)N;
  p.K = (int)K;
  p.out = static_cast<uint16_t *>(out);
  hipStream_t s = qdh::S(stream);
  if (row_token) launch_mx_epi<true>(p, pl, epilogue, s);
  else launch_mx_epi<false>(p, pl, epilogue, s);
  return qdh::check_launch();
}

// ---------------------------------------------------------------- layer
namespace {
struct MxLayout {
  size_t route, ids, wts, offs, row_token, inv_row, xc, xs, h, hc, hs, z, total;
};
MxLayout mx_layer_layout(int64_t T, int64_t H, int32_t E, int32_t k, int64_t I) {
  MxLayout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t at = o; o += qdh::align_up(bytes > 0 ? bytes : 1); return at; };
  const int64_t R = T * k;
  L.route = take(moe_route_permute_workspace(T, E, k));
  L.ids = take((size_t)R * 4);
  L.wts = take((size_t)R * 4);
  L.offs = take((size_t)(E + 1) * 4);
  L.row_token = take((size_t)R * 4);
  L.inv_row = take((size_t)R * 4);
  L.xc = take((size_t)(T * H / 2));
  L.xs = take((size_t)(T * H / 32));
  L.h = take((size_t)(R * I * 2));
  L.hc = take((size_t)(R * I / 2));
  L.hs = take((size_t)(R * I / 32));
  L.z = take((size_t)(R * H * 2));
  L.total = o;
  return L;
}
}  // namespace

extern "C" size_t qd_mxfp4_moe_layer_workspace(int64_t T, int64_t H, int32_t E, int32_t k,
                                               int64_t I) {
  if (T < 0 || H < 0 || E < 1 || k < 1 || I < 0) return 0;
  return mx_layer_layout(T, H, E, k, I).total;
}

extern "C" qd_status qd_mxfp4_moe_layer_forward(const void *x, const float *logits, int64_t T,
                                                int64_t H, int32_t E, int32_t k, int64_t I,
                                                int32_t renorm, const uint8_t *w13_codes,
                                                const uint8_t *w13_scales,
                                                const uint8_t *w2_codes,
                                                const uint8_t *w2_scales, void *y, void *ws,
                                                size_t ws_bytes, void *stream) {
  if (T < 0 || H <= 0 || I <= 0 || E < 1 || k < 1 || k > E) return QD_ERR_SHAPE;
  if (!w13_codes || !w13_scales || !w2_codes || !w2_scales) return QD_ERR_NULL;
  if (T > 0 && (!x || !logits || !y)) return QD_ERR_NULL;
  if (!ws || ws_bytes < qd_mxfp4_moe_layer_workspace(T, H, E, k, I)) return QD_ERR_WORKSPACE;
  if (!qdh::aligned16(ws) || !qdh::aligned16(y)) return QD_ERR_ALIGN;
  const int64_t R = T * k;
  if (!mx_plan(R > 0 ? R : 1, E, 2 * I, H, QD_EPI_SWIGLU).ok ||
      !mx_plan(R > 0 ? R : 1, E, H, I, QD_EPI_NONE).ok)
    return QD_ERR_UNSUPPORTED;
  if (T == 0) return QD_OK;
  const MxLayout L = mx_layer_layout(T, H, E, k, I);
  unsigned char *b = static_cast<unsigned char *>(ws);
  int32_t *ids = reinterpret_cast<int32_t *>(b + L.ids);
  float *wts = reinterpret_cast<float *>(b + L.wts);
  int32_t *offs = reinterpret_cast<int32_t *>(b + L.offs);
  int32_t *row_token = reinterpret_cast<int32_t *>(b + L.row_token);
  int32_t *inv_row = reinterpret_cast<int32_t *>(b + L.inv_row);
  uint8_t *xc = b + L.xc, *xs = b + L.xs;
  uint16_t *h = reinterpret_cast<uint16_t *>(b + L.h);
  uint8_t *hc = b + L.hc, *hs = b + L.hs;
  uint16_t *z = reinterpret_cast<uint16_t *>(b + L.z);
  qd_status st = moe_route_permute(logits, T, E, k, renorm, ids, wts, offs, row_token, inv_row,
                                   b + L.route, moe_route_permute_workspace(T, E, k), stream);
  if (st) return st;
  st = mxfp4_quantize_rows(x, QD_DTYPE_BF16, T, H, xc, xs, stream);
  if (st) return st;
  st = moe_mxfp4_grouped_gemm(xc, xs, T, row_token, offs, E, R, w13_codes, w13_scales, 2 * I, H,
                              QD_EPI_SWIGLU, h, stream);
  if (st) return st;
  st = mxfp4_quantize_rows(h, QD_DTYPE_BF16, R, I, hc, hs, stream);
  if (st) return st;
  st = moe_mxfp4_grouped_gemm(hc, hs, R, nullptr, offs, E, R, w2_codes, w2_scales, H, I,
                              QD_EPI_NONE, z, stream);
  if (st) return st;
  return moe_unpermute_combine(z, inv_row, wts, T, k, H, y, stream);
}

// The trainer-side forward of QUADS (Sec. 3.2, Eq. (w4a16-qat-forward)):
// asymmetric W4A16, i.e. bf16 activations times the NVFP4 fake-quantised
// weights, Y = X * W_hat^T, as a grouped GEMM over the experts of the MoE
// layer.  W_hat is the same QDQ the rollout side uses (Sec. 3.2, Eq.
// (weight-qdq-align)), so the weights are read in their NVFP4 form (E2M1
// codes, E4M3 scale per 16, FP32 tensor scale) and decoded exactly:
// e2m1 * e4m3 has at most six significant bits, so it is exact in bf16, and
// a bf16 activation times it is exact in f32.  The tensor scale s_dec of the
// expert multiplies the f32 sum in the epilogue.
//
// Kernel: tiles of 128 grouped rows x 256 weight rows (SwiGLU: 128 gate rows
// and the matching 128 up rows), eight waves in a 2 x 4 grid of 64 x 64 on
// v_mfma_f32_32x32x16_bf16; the wide weight tile halves how often the bf16
// activations are re-read (once per weight tile).  K streams in stages of 64 through a double
// buffer in LDS: each thread keeps a half row (32 elements) of activations
// and of weight codes of the next two stages in registers (two loads in
// flight) while the current stage is multiplied, then stores the next
// stage's activations as they are and its weights decoded to bf16.  Rows
// are padded to 72 elements (144 bytes) so that the fragment reads hit
// distinct banks.  M-tiles follow the shared tile scheduler (no tile
// straddles two experts; tiles contiguous per XCD).
#include "common.h"
#include "tile_sched.h"

namespace {

using namespace qd;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));

constexpr int WA_M = 128;            // grouped rows per tile
constexpr int WA_N = 256;            // weight rows per tile
constexpr int WA_THREADS = 512;
constexpr int WA_K = 64;             // elements per stage
constexpr int WA_LD = WA_K + 8;      // LDS row stride in bf16 elements

struct W16Args {
  const uint16_t *a;                 // bf16 [a_rows][K]
  const int32_t *row_token;
  const int32_t *offsets;
  int E;
  int64_t rows;
  const uint8_t *w_codes;
  const uint8_t *w_scales;
  const float *w_gs;
  int N;
  int K;
  uint16_t *out;
};

__device__ __forceinline__ f32x16_t mfma_bf16(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// A thread's share of one stage in registers: a quarter row (16 elements)
// of activations, a half row of weight codes (32) and their two E4M3 scale
// bytes (scalar members, so that it stays in registers).
struct StageRegs {
  uint4 a0, a1, b;
  uint32_t s;
};

__device__ __forceinline__ StageRegs w16_load(const uint16_t *ag, const uint8_t *bc,
                                              const uint8_t *bs, int k0) {
  StageRegs r;
  const uint4 *pa = reinterpret_cast<const uint4 *>(ag + k0);
  r.a0 = pa[0];
  r.a1 = pa[1];
  r.b = *reinterpret_cast<const uint4 *>(bc + (k0 >> 1));
  r.s = *reinterpret_cast<const uint16_t *>(bs + (k0 >> 4));
  return r;
}

// activations as they are; weights with the exact f16 decode of the rollout
// GEMMs (words 0, 1: the first 16-block, words 2, 3: the second), widened to
// bf16 without rounding
__device__ __forceinline__ void w16_store(const StageRegs r, uint16_t *arow, uint16_t *brow) {
  uint4 *da = reinterpret_cast<uint4 *>(arow);
  da[0] = r.a0;
  da[1] = r.a1;
  const f16x2 pair = __builtin_bit_cast(f16x2, scale_pair_f16(r.s & 0xFFu, (r.s >> 8) & 0xFFu));
  bf16x8_t *db = reinterpret_cast<bf16x8_t *>(brow);
  db[0] = __builtin_convertvector(__builtin_convertvector(decode8_sel(r.b.x, pair, false), f32x8_t), bf16x8_t);
  db[1] = __builtin_convertvector(__builtin_convertvector(decode8_sel(r.b.y, pair, false), f32x8_t), bf16x8_t);
  db[2] = __builtin_convertvector(__builtin_convertvector(decode8_sel(r.b.z, pair, true), f32x8_t), bf16x8_t);
  db[3] = __builtin_convertvector(__builtin_convertvector(decode8_sel(r.b.w, pair, true), f32x8_t), bf16x8_t);
}

template <bool GATHER, int EPI>
__global__ __launch_bounds__(WA_THREADS) void gemm_w4a16_kernel(W16Args p, int ntn) {
  __shared__ __align__(16) uint16_t As[2][WA_M * WA_LD];
  __shared__ __align__(16) uint16_t Bs[2][WA_N * WA_LD];
  __shared__ int32_t src_row[WA_M];
  __shared__ int sh_w[8], sh_t[4];
  const qdt::Tile t = qdt::find_tile<WA_M, 8>(p.offsets, p.E, p.rows, ntn, sh_w, sh_t);
  if (t.e < 0) return;                        // whole workgroup
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w >> 2, wn = w & 3;
  const int K = p.K, N = p.N;
  for (int r = tid; r < WA_M; r += WA_THREADS) {
    const int64_t g = t.row0 + (r < t.nrows ? r : 0);   // rows past the tile read its first
    src_row[r] = GATHER ? p.row_token[g] : (int32_t)g;
  }
  __syncthreads();

  // this thread's share of each stage: a quarter row (16 elements) of tile
  // row ar, and a half row (32 elements) of weight row br
  const int ar = tid >> 2, aq = tid & 3;
  const int br = tid >> 1, hf = tid & 1;
  const uint16_t *ag = p.a + (int64_t)src_row[ar] * K + aq * 16;
  int wr;
  if (EPI == QD_EPI_SWIGLU) {
    const int I = N >> 1;
    wr = br < 128 ? t.nt * 128 + br : I + t.nt * 128 + (br - 128);
  } else {
    wr = t.nt * WA_N + br;
  }
  const int64_t wrow = (int64_t)t.e * N + (wr < N ? wr : 0);   // others are never stored
  const uint8_t *bc = p.w_codes + wrow * (K >> 1) + hf * 16;
  const uint8_t *bs = p.w_scales + wrow * (K >> 4) + hf * 2;

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.0f;

  // fragment rows: A rows wm*64 + 32 i, B rows of fragment j (SwiGLU: j = 0
  // gate rows, j = 1 the matching up rows)
  const int lr = lane & 31, kh = 8 * (lane >> 5);
  int brow[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
    brow[j] = EPI == QD_EPI_SWIGLU ? j * 128 + wn * 32 + lr : wn * 64 + j * 32 + lr;

  // Two stages of loads in flight: at the top of iteration s the LDS
  // buffer s & 1 holds stage s and the two register sets hold (or are
  // receiving) stages s + 1 and s + 2.  Iteration s multiplies stage s,
  // stores stage s + 1 into the other buffer (last read in iteration s - 1,
  // which every thread left through the barrier at its end), and reloads
  // the freed register set with stage s + 3.  The loop is unrolled by two
  // so that the register sets keep fixed names.
  const int nst = K / WA_K;
  auto mma = [&](int buf) {
#pragma unroll
    for (int kk = 0; kk < WA_K; kk += 16) {
      bf16x8_t af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t *>(&As[buf][(wm * 64 + i * 32 + lr) * WA_LD + kk + kh]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bf[j] = *reinterpret_cast<const bf16x8_t *>(&Bs[buf][brow[j] * WA_LD + kk + kh]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mfma_bf16(af[i], bf[j], acc[i][j]);
    }
  };
  uint16_t *arow0 = &As[0][ar * WA_LD + aq * 16], *arow1 = &As[1][ar * WA_LD + aq * 16];
  uint16_t *brow0 = &Bs[0][br * WA_LD + hf * 32], *brow1 = &Bs[1][br * WA_LD + hf * 32];
  StageRegs r0 = w16_load(ag, bc, bs, 0), r1 = r0;
  if (nst > 1) r1 = w16_load(ag, bc, bs, WA_K);
  w16_store(r0, arow0, brow0);
  if (nst > 2) r0 = w16_load(ag, bc, bs, 2 * WA_K);
  __syncthreads();
  for (int s = 0; s < nst; s += 2) {
    // r1: stage s + 1, r0: stage s + 2 (in flight)
    mma(0);
    if (s + 1 < nst) w16_store(r1, arow1, brow1);
    if (s + 3 < nst) r1 = w16_load(ag, bc, bs, (s + 3) * WA_K);
    __syncthreads();
    if (s + 1 >= nst) break;
    // r0: stage s + 2, r1: stage s + 3 (in flight)
    mma(1);
    if (s + 2 < nst) w16_store(r0, arow0, brow0);
    if (s + 4 < nst) r0 = w16_load(ag, bc, bs, (s + 4) * WA_K);
    __syncthreads();
  }

  // ---- epilogue: the expert's tensor scale, SwiGLU or plain, bf16 stores
  const float alpha = p.w_gs[2 * t.e + 1];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int rl = wm * 64 + i * 32 + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
      if (rl >= t.nrows) continue;
      const int64_t row = t.row0 + rl;
      if (EPI == QD_EPI_SWIGLU) {
        const int I = N >> 1;
        const int col = t.nt * 128 + wn * 32 + lr;
        if (col < I) {
          const float gv = alpha * acc[i][0][q];
          const float uv = alpha * acc[i][1][q];
          const float h = gv / (1.0f + expf(-gv)) * uv;
          p.out[row * I + col] = (uint16_t)f32_to_bf16_bits(h);
        }
      } else {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int col = t.nt * WA_N + wn * 64 + j * 32 + lr;
          if (col < N) p.out[row * N + col] = (uint16_t)f32_to_bf16_bits(alpha * acc[i][j][q]);
        }
      }
    }
  }
}

}  // namespace

extern "C" qd_status moe_w4a16_grouped_gemm(const void *a, int64_t a_rows,
                                            const int32_t *row_token,
                                            const int32_t *expert_offsets, int32_t E,
                                            int64_t rows, const qd_nvfp4 *w, int32_t epilogue,
                                            void *out, void *stream) {
  if (!w) return QD_ERR_NULL;
  if (epilogue != QD_EPI_NONE && epilogue != QD_EPI_SWIGLU) return QD_ERR_DTYPE;
  if (E < 1 || E > 1024 || rows < 0 || a_rows < 0) return QD_ERR_SHAPE;
  qd_status st = qdh::check_nvfp4(w, E, w->rows, w->cols);
  if (st) return st;
  const int64_t N = w->rows, K = w->cols;
  if (K <= 0 || K % WA_K != 0 || N <= 0 || N % 32 != 0) return QD_ERR_SHAPE;
  if (!expert_offsets && E != 1) return QD_ERR_SHAPE;
  if (!row_token && rows > a_rows) return QD_ERR_SHAPE;
  if (N > 0x7fffffff || K > 0x7fffffff || rows > 0x7fffffff) return QD_ERR_UNSUPPORTED;
  if (rows == 0) return QD_OK;
  if (!a || !out) return QD_ERR_NULL;
  if (!qdh::aligned16(a) || !qdh::aligned16(out) || !qdh::aligned16(w->codes))
    return QD_ERR_ALIGN;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  W16Args p{};
  p.a = static_cast<const uint16_t *>(a);
  p.row_token = row_token;
  p.offsets = expert_offsets;
  p.E = E;
  p.rows = rows;
  p.w_codes = w->codes;
  p.w_scales = w->scales;
  p.w_gs = w->gscale;
  p.N = (int)N;
  p.K = (int)K;
  p.out = static_cast<uint16_t *>(out);
  const int ntn = epilogue == QD_EPI_SWIGLU ? (int)((N / 2 + 127) / 128) : (int)((N + WA_N - 1) / WA_N);
  const int64_t grid = qdt::tile_grid(rows, E, WA_M, ntn);
  if (grid > 0x7fffffffLL) return QD_ERR_UNSUPPORTED;
  hipStream_t s = qdh::S(stream);
  const dim3 g((unsigned)grid);
  if (row_token) {
    if (epilogue == QD_EPI_SWIGLU)
      hipLaunchKernelGGL((gemm_w4a16_kernel<true, QD_EPI_SWIGLU>), g, dim3(WA_THREADS), 0, s, p, ntn);
    else
      hipLaunchKernelGGL((gemm_w4a16_kernel<true, QD_EPI_NONE>), g, dim3(WA_THREADS), 0, s, p, ntn);
  } else {
    if (epilogue == QD_EPI_SWIGLU)
      hipLaunchKernelGGL((gemm_w4a16_kernel<false, QD_EPI_SWIGLU>), g, dim3(WA_THREADS), 0, s, p, ntn);
    else
      hipLaunchKernelGGL((gemm_w4a16_kernel<false, QD_EPI_NONE>), g, dim3(WA_THREADS), 0, s, p, ntn);
  }
  return qdh::check_launch();
}

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

// ---------------------------------------------------------------------------
// Skinny grouped GEMM for decode-sized batches (few rows per expert).  The
// weights dominate the traffic, so every weight byte is read exactly once
// and as many of them as possible are kept in flight:
//   * a workgroup owns (expert e, 128 weight rows); each of its four waves
//     streams 32 distinct weight rows (for SwiGLU 16 gate rows and the
//     matching 16 up rows) straight from HBM into registers, two iterations
//     ahead of their use;
//   * the expert's activation rows (up to 64 per pass) are staged once per
//     iteration into LDS by the whole workgroup and shared by the waves;
//   * RAC: while a weight chunk sits in registers, its elements in the
//     selected channels S are decoded into a compact [row][K_s] f16 panel in
//     LDS; after the K loop a short K_s-long MFMA pass multiplies it with the
//     compact residual activations, so the residual costs K_s/K of the main
//     contraction instead of a dense second pass.
//
// K assignment: iteration it covers elements [256*it, 256*it + 256) (128 code
// bytes, one cache line, and 16 scale bytes per row); lane group g = lane/16
// owns elements 64g .. 64g+63 of it (32 contiguous code bytes, one scale
// dword), split into SK_CH = 2 chunks of 32; k-step s of a chunk is its
// elements 8s .. 8s+7.  The four lane groups of a row therefore read one
// whole line per iteration.
//
// XCD-aware placement: workgroup P runs on XCD P % 8; expert e's workgroups
// all get ids with P % 8 == e % 8, so its activation rows are fetched into
// one L2 only.
constexpr int SK_MTMAX = 4;        // 16-row m-tiles per pass (64 rows)
constexpr int SK_ROWS = 128;       // weight rows per workgroup
constexpr int SK_CH = 2;           // 32-element chunks per iteration
constexpr int SK_KSMAX = 256;      // largest K_s of the fused compact residual
constexpr int SK_KMAX = 16384;     // largest K with the fused residual

struct SkLayout {
  int selmap, prefix, sel, a, as, ares, wc, red, total, stride;
};

__host__ __device__ inline SkLayout sk_layout(int K, int Ks, bool rac) {
  SkLayout L{};
  int o = 0;
  auto take = [&](int bytes) { int at = o; o += (bytes + 15) & ~15; return at; };
  const int kpad = (Ks + 31) & ~31;
  L.stride = kpad * 2 + 16;                         // bytes per compact row (+16: banks)
  L.selmap = take(rac ? (K / 32) * 4 : 0);
  L.prefix = take(rac ? (K / 32) * 4 : 0);
  L.sel = take(rac ? Ks * 4 : 0);
  L.a = take(2 * SK_CH * 4 * SK_MTMAX * 16 * 16);    // [stage][chunk][group][row] x 16 B
  L.as = take(2 * 4 * SK_MTMAX * 16 * 4);            // [stage][group][row] x 4 B
  L.ares = take(rac ? SK_MTMAX * 16 * L.stride : 0);
  L.wc = take(rac ? SK_ROWS * L.stride : 0);
  L.red = take(16 * 4);
  L.total = o;
  return L;
}

// One iteration's weights of a wave (two 16-row fragments x SK_CH chunks)
// and one thread's share of the activation staging.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
struct BStage {
  u32x4 v00, v01, v10, v11;     // v<fragment><chunk>
  uint32_t sc0, sc1;            // 4 scale bytes per fragment (2 chunks x 2 blocks)
};
struct AStage {
  u32x4 c0, c1;
  uint32_t sc;
};
constexpr int kBLoads = 6;      // vector memory instructions per BStage
constexpr int kALoads = 3;      // per AStage

// The main loop's loads are issued by inline assembly so that their
// completion is tracked by hand: the compiler's own wait-counter placement
// is conservative at the loop header and would force the prefetched stages
// to complete one iteration early.  wait_* ties the waited registers, so no
// use of them can be scheduled before the wait.
__device__ __forceinline__ u32x4 gld16(const uint8_t *p) {
  u32x4 r;
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(r) : "v"(p));
  return r;
}
__device__ __forceinline__ uint32_t gld4(const uint8_t *p) {
  uint32_t r;
  asm volatile("global_load_dword %0, %1, off" : "=v"(r) : "v"(p));
  return r;
}
template <int N>
__device__ __forceinline__ void wait_b(BStage &b) {
  asm volatile("s_waitcnt vmcnt(%6)"
               : "+v"(b.v00), "+v"(b.v01), "+v"(b.v10), "+v"(b.v11), "+v"(b.sc0), "+v"(b.sc1)
               : "n"(N));
}
template <int N>
__device__ __forceinline__ void wait_a(AStage &a) {
  asm volatile("s_waitcnt vmcnt(%3)" : "+v"(a.c0), "+v"(a.c1), "+v"(a.sc) : "n"(N));
}

__device__ __forceinline__ BStage load_bstage(const uint8_t *bc0, const uint8_t *bc1,
                                              const uint8_t *bs0, const uint8_t *bs1, int it) {
  BStage st;
  st.v00 = gld16(bc0 + it * 128);
  st.v01 = gld16(bc0 + it * 128 + 16);
  st.v10 = gld16(bc1 + it * 128);
  st.v11 = gld16(bc1 + it * 128 + 16);
  st.sc0 = gld4(bs0 + it * 16);
  st.sc1 = gld4(bs1 + it * 16);
  return st;
}
__device__ __forceinline__ AStage load_astage(const uint8_t *ac, const uint8_t *as, int it) {
  AStage st;
  st.c0 = gld16(ac + it * 128);
  st.c1 = gld16(ac + it * 128 + 16);
  st.sc = gld4(as + it * 16);
  return st;
}
__device__ __forceinline__ uint4 as_uint4(u32x4 v) { return make_uint4(v.x, v.y, v.z, v.w); }
__device__ __forceinline__ void store_astage(uint4 *a_lds, uint32_t *as_lds, const AStage &st,
                                             int stage, int ag, int arow) {
  a_lds[((stage * 2 + 0) * 4 + ag) * 64 + arow] = as_uint4(st.c0);
  a_lds[((stage * 2 + 1) * 4 + ag) * 64 + arow] = as_uint4(st.c1);
  as_lds[(stage * 4 + ag) * 64 + arow] = st.sc;
}
__device__ __forceinline__ uint4 bvec(const BStage &b, int j, int cc) {
  return as_uint4(j == 0 ? (cc == 0 ? b.v00 : b.v01) : (cc == 0 ? b.v10 : b.v11));
}

__device__ __forceinline__ uint32_t dword_of(uint4 v, uint32_t i) {
  return i == 0 ? v.x : (i == 1 ? v.y : (i == 2 ? v.z : v.w));
}

template <bool GATHER, bool RAC, int EPI>
__global__ __launch_bounds__(256) void gemm_skinny_kernel(GemmArgs p, int nblk_n) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int lr = lane & 15, g = lane >> 4;
  const int tid = threadIdx.x;
  const int K = p.K, N = p.N;
  const int64_t kb2 = K >> 1, kb16 = K >> 4;
  const int Ks = RAC ? p.Ks : 0;
  const SkLayout L = sk_layout(K, Ks, RAC);
  uint32_t *selmap = reinterpret_cast<uint32_t *>(lds + L.selmap);
  int32_t *prefix = reinterpret_cast<int32_t *>(lds + L.prefix);
  int32_t *s_sel = reinterpret_cast<int32_t *>(lds + L.sel);
  uint4 *a_lds = reinterpret_cast<uint4 *>(lds + L.a);
  uint32_t *as_lds = reinterpret_cast<uint32_t *>(lds + L.as);
  unsigned char *ares = lds + L.ares;
  unsigned char *wc = lds + L.wc;
  float *red = reinterpret_cast<float *>(lds + L.red);

  const int P = blockIdx.x;
  const int xcd = P & 7, q = P >> 3;
  const int nb = q % nblk_n;
  const int e = (q / nblk_n) * 8 + xcd;
  const int niter = K >> 8;              // 256 elements per iteration
  const int kpad = (Ks + 31) & ~31;

  if (RAC) {
    // channel bitmap, per-word prefix counts, the channel list, zero panels
    for (int i = tid; i < K / 32; i += 256) selmap[i] = 0u;
    for (int i = tid; i < Ks; i += 256) s_sel[i] = p.sel[i];
    for (int i = tid; i < SK_ROWS * (L.stride / 4); i += 256)
      reinterpret_cast<uint32_t *>(wc)[i] = 0u;
    __syncthreads();
    for (int i = tid; i < Ks; i += 256) {
      const int j = s_sel[i];
      atomicOr(&selmap[j >> 5], 1u << (j & 31));
    }
    __syncthreads();
    // exclusive prefix of popcounts (K/32 <= 512 words; 2 per thread)
    const int nw = K / 32;
    const int w0 = 2 * tid;
    int c0 = w0 < nw ? __popc(selmap[w0]) : 0;
    int c1 = w0 + 1 < nw ? __popc(selmap[w0 + 1]) : 0;
    int v = c0 + c1, x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    if (lane == 63) red[w] = __int_as_float(x);
    __syncthreads();
    int base = 0;
    for (int ww = 0; ww < w; ++ww) base += __float_as_int(red[ww]);
    const int ex = base + x - v;
    if (w0 < nw) prefix[w0] = ex;
    if (w0 + 1 < nw) prefix[w0 + 1] = ex + c0;
    __syncthreads();
  }

  float vmax = 0.0f;
  const int64_t ob = (e < p.E) ? (p.offsets ? p.offsets[e] : 0) : 0;
  const int64_t oe = (e < p.E) ? (p.offsets ? p.offsets[e + 1] : p.rows) : 0;
  // this wave's two weight-row fragments (clamped rows are loaded, never stored)
  int64_t wrow[2];
  bool bval[2];
  if (EPI == QD_EPI_SWIGLU) {
    const int I = N >> 1;
    const int pr = nb * (SK_ROWS / 2) + w * 16 + lr;
    bval[0] = bval[1] = pr < I;
    wrow[0] = pr;
    wrow[1] = pr + I;
  } else {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      wrow[j] = (int64_t)nb * SK_ROWS + w * 32 + j * 16 + lr;
      bval[j] = wrow[j] < N;
    }
  }
  const int eb = e < p.E ? e : 0;
  const uint8_t *bc[2], *bs[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int64_t wr = bval[j] ? wrow[j] : 0;
    bc[j] = p.w_codes + ((int64_t)eb * N + wr) * kb2 + g * 32;
    bs[j] = p.w_scales + ((int64_t)eb * N + wr) * kb16 + g * 4;
  }
  const float sw = (e < p.E) ? p.w_gs[2 * e + 1] : 0.0f;
  const float alpha = p.a_gs[1] * sw;
  const float alpha_r = RAC ? p.r_gs[1] * sw : 0.0f;

  for (int64_t rg = ob; rg < oe; rg += SK_MTMAX * 16) {
    const int nrow = (int)min((int64_t)SK_MTMAX * 16, oe - rg);
    const int mt_valid = (nrow + 15) >> 4;
    // cooperative activation staging: thread t owns row (t & 63) of lane
    // group ((t >> 6) & 3) for both chunks of an iteration
    const int arow = tid & 63, ag = (tid >> 6) & 3;
    const int64_t gsrc = rg + (arow < nrow ? arow : 0);
    const int64_t asrc = GATHER ? (int64_t)p.row_token[gsrc] : gsrc;
    const uint8_t *a_c = p.a_codes + asrc * kb2 + ag * 32;
    const uint8_t *a_s = p.a_scales + asrc * kb16 + ag * 4;
    __syncthreads();      // the previous pass's panels are no longer read
    if (RAC) {
      // compact residual activations: ares[r][i] = rhat[src(r)][S_i] (f16, exact)
      for (int idx = tid; idx < SK_MTMAX * 16 * kpad; idx += 256) {
        const int r = idx / kpad, i = idx - r * kpad;
        _Float16 v = (_Float16)0.0f;
        if (r < nrow && i < Ks) {
          const int64_t gr = rg + r;
          const int64_t src = GATHER ? (int64_t)p.row_token[gr] : gr;
          const int j = s_sel[i];
          const uint32_t byte = p.r_codes[src * kb2 + (j >> 1)];
          const uint32_t c = (j & 1) ? (byte >> 4) : (byte & 15u);
          float f = e2m1_value(c) * e4m3_to_f32(p.r_scales[src * kb16 + (j >> 4)]);
          v = (_Float16)((c & 8u) ? -f : f);
        }
        *reinterpret_cast<_Float16 *>(ares + r * L.stride + i * 2) = v;
      }
    }
    f32x4 acc[SK_MTMAX][2];
#pragma unroll
    for (int i = 0; i < SK_MTMAX; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const uint8_t *bc0 = bc[0], *bc1 = bc[1], *bs0 = bs[0], *bs1 = bs[1];
    // Software pipeline.  Weights: a ring of three register stages (named,
    // never indexed or moved); the weights of iteration m are issued at the
    // end of iteration m-3, the activations of iteration m at the end of
    // iteration m-2 and stored to LDS at the end of iteration m-1.  Issue
    // order, identical in the prologue and every iteration:
    //     ... A(m-1) B(m) | A(m) B(m+1) | A(m+1) B(m+2) ...
    // so B(m) is complete once at most 2*(kALoads+kBLoads) younger loads are
    // outstanding, and A(m+1) once kBLoads are.  Loads past the last
    // iteration re-read the last one (never used; they keep the counts
    // uniform) and are drained before the registers are released.
    const int last = niter - 1;
    BStage b0, b1, b2;
    AStage ast;
    __syncthreads();     // every earlier load has completed (fence), LDS panels written
    b0 = load_bstage(bc0, bc1, bs0, bs1, 0);
    {
      AStage a0 = load_astage(a_c, a_s, 0);
      b1 = load_bstage(bc0, bc1, bs0, bs1, min(1, last));
      ast = load_astage(a_c, a_s, min(1, last));
      b2 = load_bstage(bc0, bc1, bs0, bs1, min(2, last));
      wait_a<2 * kBLoads + kALoads>(a0);
      store_astage(a_lds, as_lds, a0, 0, ag, arow);
    }
    __syncthreads();

    auto body = [&](const int it, BStage &bb) {
      const int stage = it & 1;
      wait_b<2 * (kALoads + kBLoads)>(bb);
      // f16 scale factors (value/256) of this iteration: pair (block 2cc, 2cc+1)
      uint32_t bsp[2][SK_CH];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const uint32_t sc = j ? bb.sc1 : bb.sc0;
#pragma unroll
        for (int cc = 0; cc < SK_CH; ++cc)
          bsp[j][cc] = scale_pair_f16((sc >> (16 * cc)) & 0xFFu, (sc >> (16 * cc + 8)) & 0xFFu);
      }
#pragma unroll
      for (int cc = 0; cc < SK_CH; ++cc) {
        // selected channels among this lane group's 32 elements of the chunk
        const uint32_t word = RAC ? selmap[it * 8 + g * 2 + cc] : 0u;
        const int base = RAC ? prefix[it * 8 + g * 2 + cc] : 0;
        const bool any_sel = RAC && __any((int)(word != 0u));
        uint32_t asp[SK_MTMAX];
#pragma unroll
        for (int i = 0; i < SK_MTMAX; ++i) {
          if (i < mt_valid) {
            const uint32_t asv = as_lds[(stage * 4 + g) * (SK_MTMAX * 16) + i * 16 + lr];
            asp[i] = scale_pair_f16((asv >> (16 * cc)) & 0xFFu, (asv >> (16 * cc + 8)) & 0xFFu);
          }
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          f16x8 bf[2];
#pragma unroll
          for (int j = 0; j < 2; ++j)
            bf[j] = decode8(word_of(bvec(bb, j, cc), s),
                            s < 2 ? splat_lo(bsp[j][cc]) : splat_hi(bsp[j][cc]));
#pragma unroll
          for (int i = 0; i < SK_MTMAX; ++i) {
            if (i < mt_valid) {
              const uint4 av = a_lds[((stage * SK_CH + cc) * 4 + g) * (SK_MTMAX * 16) + i * 16 + lr];
              const f16x8 af = decode8(word_of(av, s), s < 2 ? splat_lo(asp[i]) : splat_hi(asp[i]));
#pragma unroll
              for (int j = 0; j < 2; ++j) acc[i][j] = mfma16(af, bf[j], acc[i][j]);
            }
          }
          if (any_sel) {
            // the decoded values of selected channels -> compact weight panel
            const uint32_t m8 = (word >> (8 * s)) & 0xFFu;
            if (m8) {
              const int pos0 = base + __popc(word & ((1u << (8 * s)) - 1u));
#pragma unroll
              for (int e8 = 0; e8 < 8; ++e8) {
                if ((m8 >> e8) & 1u) {
                  const int pos = pos0 + __popc(m8 & ((1u << e8) - 1u));
#pragma unroll
                  for (int j = 0; j < 2; ++j) {
                    const int rloc = w * 32 + j * 16 + lr;
                    *reinterpret_cast<_Float16 *>(wc + rloc * L.stride + pos * 2) = bf[j][e8];
                  }
                }
              }
            }
          }
        }
      }
      wait_a<kBLoads>(ast);
      store_astage(a_lds, as_lds, ast, (it + 1) & 1, ag, arow);
      ast = load_astage(a_c, a_s, min(it + 2, last));
      bb = load_bstage(bc0, bc1, bs0, bs1, min(it + 3, last));
      __syncthreads();
    };
    for (int it = 0; it < niter; it += 3) {
      body(it, b0);
      if (it + 1 < niter) body(it + 1, b1);
      if (it + 2 < niter) body(it + 2, b2);
    }
    // drain the loads still in flight before their registers are reused
    wait_b<0>(b0);
    wait_b<0>(b1);
    wait_b<0>(b2);
    wait_a<0>(ast);
    // residual pass over the compact panels
    f32x4 accr[SK_MTMAX][2];
#pragma unroll
    for (int i = 0; i < SK_MTMAX; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) accr[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (RAC) {
      for (int ks = 0; ks < kpad; ks += 32) {
        f16x8 bf[2];
#pragma unroll
        for (int j = 0; j < 2; ++j)
          bf[j] = *reinterpret_cast<const f16x8 *>(wc + (w * 32 + j * 16 + lr) * L.stride +
                                                   (ks + g * 8) * 2);
#pragma unroll
        for (int i = 0; i < SK_MTMAX; ++i) {
          if (i < mt_valid) {
            const f16x8 af =
                *reinterpret_cast<const f16x8 *>(ares + (i * 16 + lr) * L.stride + (ks + g * 8) * 2);
#pragma unroll
            for (int j = 0; j < 2; ++j) accr[i][j] = mfma16(af, bf[j], accr[i][j]);
          }
        }
      }
    }
    // epilogue for this pass
#pragma unroll
    for (int i = 0; i < SK_MTMAX; ++i) {
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        const int rl = i * 16 + g * 4 + qq;
        if (rl >= nrow) continue;
        const int64_t row = rg + rl;
        if (EPI == QD_EPI_SWIGLU) {
          const int I = N >> 1;
          if (bval[0]) {
            float gv = alpha * acc[i][0][qq];
            float uv = alpha * acc[i][1][qq];
            if (RAC) {
              gv = gv - alpha_r * accr[i][0][qq];
              uv = uv - alpha_r * accr[i][1][qq];
            }
            const float h = gv / (1.0f + expf(-gv)) * uv;
            const uint32_t hb = f32_to_bf16_bits(h);
            p.out[row * I + wrow[0]] = (uint16_t)hb;
            vmax = fmaxf(vmax, fabsf(bf16_bits_to_f32(hb)));
          }
        } else {
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            if (bval[j]) {
              float v = alpha * acc[i][j][qq];
              if (RAC) v = v - alpha_r * accr[i][j][qq];
              const uint32_t hb = f32_to_bf16_bits(v);
              p.out[row * N + wrow[j]] = (uint16_t)hb;
              vmax = fmaxf(vmax, fabsf(bf16_bits_to_f32(hb)));
            }
          }
        }
      }
    }
  }
  const float m = block_max(vmax, red);
  if (p.amax_part && threadIdx.x == 0) p.amax_part[P] = m;
}

inline int64_t skinny_nblk(int64_t N, int epilogue) {
  return epilogue == QD_EPI_SWIGLU ? ((N / 2) + SK_ROWS / 2 - 1) / (SK_ROWS / 2)
                                   : (N + SK_ROWS - 1) / SK_ROWS;
}
inline int64_t skinny_grid(int64_t N, int E, int epilogue) {
  return (int64_t)((E + 7) / 8) * 8 * skinny_nblk(N, epilogue);
}
// decode-sized problems: few rows per expert, K a multiple of 256 (whole
// iterations per quarter) and, with RAC, K_s and K within the panel limits
inline bool use_skinny(int64_t rows, int E, int64_t K, int Ks) {
  return K % 256 == 0 && rows <= (int64_t)E * 48 && Ks <= SK_KSMAX &&
         (Ks == 0 || K <= SK_KMAX);
}

inline int64_t grid_x(int64_t rows, int E, bool grouped) {
  return (rows + BM - 1) / BM + (grouped ? E : 0);
}
inline int64_t grid_y(int64_t N, int epilogue) {
  return epilogue == QD_EPI_SWIGLU ? ((N / 2) + 31) / 32 : (N + BN - 1) / BN;
}

template <bool GATHER, bool RAC>
void launch_epi(const GemmArgs &p, int epi, dim3 grid, hipStream_t s, bool skinny, int nblk_n) {
  if (skinny) {
    const size_t lds = (size_t)sk_layout(p.K, RAC ? p.Ks : 0, RAC).total;
    if (epi == QD_EPI_SWIGLU)
      hipLaunchKernelGGL((gemm_skinny_kernel<GATHER, RAC, QD_EPI_SWIGLU>), grid, dim3(256), lds, s,
                         p, nblk_n);
    else
      hipLaunchKernelGGL((gemm_skinny_kernel<GATHER, RAC, QD_EPI_NONE>), grid, dim3(256), lds, s,
                         p, nblk_n);
    return;
  }
  if (epi == QD_EPI_SWIGLU)
    hipLaunchKernelGGL((gemm_w4a4_kernel<GATHER, RAC, QD_EPI_SWIGLU>), grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((gemm_w4a4_kernel<GATHER, RAC, QD_EPI_NONE>), grid, dim3(256), 0, s, p);
}

}  // namespace

extern "C" int64_t moe_w4a4_grouped_gemm_amax_count(int64_t rows, int64_t N, int64_t K,
                                                    int32_t E, int32_t Ks, int32_t epilogue) {
  if (rows < 0 || N <= 0 || K <= 0 || E < 1 || Ks < 0) return 0;
  if (use_skinny(rows, E, K, Ks)) return skinny_grid(N, E, epilogue);
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
  const bool skinny = use_skinny(rows, E, K, rac ? Ks : 0);
  const int nblk_n = (int)skinny_nblk(N, epilogue);
  dim3 grid = skinny ? dim3((unsigned)skinny_grid(N, E, epilogue)) : dim3((unsigned)gx, (unsigned)gy);
  hipStream_t s = qdh::S(stream);
  if (row_token) {
    if (rac) launch_epi<true, true>(p, epilogue, grid, s, skinny, nblk_n);
    else launch_epi<true, false>(p, epilogue, grid, s, skinny, nblk_n);
  } else {
    if (rac) launch_epi<false, true>(p, epilogue, grid, s, skinny, nblk_n);
    else launch_epi<false, false>(p, epilogue, grid, s, skinny, nblk_n);
  }
  return qdh::check_launch();
}

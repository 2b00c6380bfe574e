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
#include "lds_dma.h"
#include "tile_sched.h"

namespace {

using namespace qd;
using namespace qdl;

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
  const uint8_t *w_sfrag;  // optional: the weight scales in fragment order
  const float *w_gs;
  int N;
  int K;
  const uint8_t *r_codes;
  const uint8_t *r_scales;
  const float *r_gs;
  const int32_t *sel;
  int Ks;
  const uint16_t *r_sel;   // f16 [a rows][ksa]: the residual at the selected channels
  int ksa;                 // row length of r_sel (Ks rounded up to 16)
  // bitmap mode (decode kernel only): r_bitmap [K / 32] marks S in place of
  // sel, and the kernel lists S into sel_out
  const uint32_t *r_bitmap;
  int32_t *sel_out;
  uint16_t *out;
  float *amax_part;
  int64_t amax_n;          // entries of amax_part (>= the grid; the rest are zeroed)
  // per-expert channel sets (tile kernel only): S of expert e at
  // sel + e * sel_stride, and r_sel indexed by grouped row instead of token
  int sel_stride;
  int rsel_rows;
  // optional (tile kernel, gathered rows, A-scale ring on): the A operand
  // staged by grouped row, stage-major -- codes [K / 64][rows][32 B], then
  // the scales of four stages at a time [K / 256][rows][16 B] -- so that a
  // tile's loads of one stage are contiguous
  const uint8_t *a_stg;
};

// one maximum of |out| per workgroup into amax_part; workgroups also zero
// the entries past the grid, so every one of the amax_n entries is written
__device__ __forceinline__ void put_amax(const GemmArgs &p, float m) {
  if (p.amax_part && threadIdx.x == 0) {
    const int64_t g = (int64_t)gridDim.x * gridDim.y;
    const int64_t b = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
    p.amax_part[b] = m;
    for (int64_t j = b + g; j < p.amax_n; j += g) p.amax_part[j] = 0.0f;
  }
}

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
    // every word the chunk loop reads (four per 128-channel chunk)
    for (int i = threadIdx.x; i < (K + 127) / 128 * 4; i += blockDim.x) selmap[i] = 0u;
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
      // a lane group's 32 elements of a chunk: all inside K (gval), only the
      // first 16 (ghalf: K % 32 == 16, the last chunk), or none
      auto ld_codes = [](const uint8_t *q, bool full, bool half) -> uint4 {
        if (full) return *reinterpret_cast<const uint4 *>(q);
        if (half) {
          const uint2 v = *reinterpret_cast<const uint2 *>(q);
          return make_uint4(v.x, v.y, 0u, 0u);
        }
        return make_uint4(0u, 0u, 0u, 0u);
      };
      auto ld_scales = [](const uint8_t *q, bool full, bool half) -> uint32_t {
        if (full) return *reinterpret_cast<const uint16_t *>(q);
        return half ? (uint32_t)q[0] : 0u;
      };
      for (int c = 0; c < nchunk; ++c) {
        const bool gval = (c * 128 + g * 32 + 32) <= K;
        const bool ghalf = !gval && (c * 128 + g * 32 + 16) <= K;
        uint4 a4[2], b4[2], r4[2];
        uint32_t asc[2], bsc[2], rsc[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          a4[i] = ld_codes(ac[i] + c * 64, av[i] && gval, av[i] && ghalf);
          asc[i] = ld_scales(as[i] + c * 8, av[i] && gval, av[i] && ghalf);
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          b4[j] = ld_codes(bc[j] + c * 64, bv[j] && gval, bv[j] && ghalf);
          bsc[j] = ld_scales(bs[j] + c * 8, bv[j] && gval, bv[j] && ghalf);
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
              r4[i] = ld_codes(rc[i] + c * 64, av[i] && gval, av[i] && ghalf);
              rsc[i] = ld_scales(rs[i] + c * 8, av[i] && gval, av[i] && ghalf);
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
  put_amax(p, m);
}

// ---------------------------------------------------------------------------
// Decode-shaped grouped GEMM (few rows per expert).  The weights are nearly
// all of the traffic, so the kernel is built to stream them once at HBM rate
// with as little per-byte instruction work as possible:
//
//  * Work units.  A unit is (expert e, pass p over 32 of its rows, block nb
//    of 256 weight rows; for SwiGLU 128 gate rows and the matching 128 up
//    rows).  Experts without rows have no units.  Every workgroup derives
//    the unit list from the expert offsets and takes an equal contiguous
//    share of it (one workgroup per CU), so skewed routing stays balanced;
//    units are ordered expert-major, so a workgroup mostly stays on one
//    expert.
//  * Eight waves, 32 weight rows each.  A wave streams its rows through a
//    private two-stage LDS ring with direct global->LDS loads: in-flight
//    weights cost no registers.  One stage is 256 K-elements of 32 rows
//    (4 KB of codes, 512 B of scales; the scales from the fragment-ordered
//    copy when the caller provides it, one contiguous 256-byte piece per
//    fragment and stage).
//  * Activations are decoded once per workgroup, not once per wave: waves
//    0..3 each load one quarter of a stage's 32 activation rows (lane group
//    g's 64 elements of every row, with their scale dword) into a private
//    raw slot, decode it exactly to f16 one stage ahead and write it into a
//    shared two-slot f16 panel, laid out as the MFMA's A fragments; every
//    wave then reads its fragments from the panel.  With RAC, waves 4..7 do
//    the same for the masked residual rows into a second panel.
//  * Loads are issued in one fixed order per iteration, spread over the
//    k-steps: the activations, then the weights, of the stage two ahead.
//    Loads complete in issue order, so one explicit wait at the top of
//    iteration s (at most the last iteration's weights outstanding) proves
//    that the wave's weights of stage s and its activations of stage s + 1
//    have landed; the barrier after it publishes the panels of stage s.
//    Loads past the last stage repeat the last stage's addresses into slots
//    that are never read again.
//  * Weight operands are decoded exactly to f16 in registers (see the top of
//    this file) and multiplied on MFMA, with straight-line code for each
//    number of valid 16-row m-tiles.
//  * RAC: the masked residual is zero outside the selected channels S, so
//    its contraction with the weights runs over the same decoded weight
//    fragments, restricted to the k-steps that contain a channel of S (a
//    per-iteration step mask built from S in the prologue), into its own
//    accumulator, which meets the main one in the epilogue.
//
// K assignment inside an iteration: lane group g = lane/16 owns elements
// 64g .. 64g+63 (32 code bytes, one scale dword), split into two chunks of
// 32; k-step s of a chunk is its elements 8s .. 8s+7.
constexpr int SK_WAVES = 8;
constexpr int SK_THREADS = 64 * SK_WAVES;
constexpr int SK_ROWS = 32 * SK_WAVES;   // weight rows per unit
constexpr int SK_PR = 32;                // activation rows per pass
constexpr int SK_NS = 2;                 // weight ring depth
constexpr int SK_BSTAGE = 4608;          // bytes per wave and weight stage
constexpr int SK_NX = 2;                 // raw activation slots per decoding wave
constexpr int SK_XRAW = 1280;            // one decoding wave's raw stage: 1 KB codes, 256 B scales
constexpr int SK_PANEL = SK_PR * 256 * 2;   // one f16 panel stage
constexpr int SK_KMAX = 65536;
constexpr int SK_EMAX = 512;             // experts (offsets and their scan kept in LDS)
constexpr int SK_LDS_MAX = 160 * 1024;
constexpr int SK_GRID = 256;             // one workgroup per CU

struct SkLayout {
  int b, pan, xraw, offs, pu, sw, smask, bm, red, total;
};

constexpr int SK_BM_KMAX = 4096;         // bitmap mode: at most 128 words of S

// panels: [source x, residual][slot 0, 1]; raw slots: [decoding wave][slot];
// bm: the selection bitmap (bitmap mode)
__host__ __device__ inline SkLayout sk_layout(int K, int E, bool rac, bool bm) {
  SkLayout L{};
  int o = 0;
  auto take = [&](int bytes) { int at = o; o += (bytes + 15) & ~15; return at; };
  L.b = take(SK_WAVES * SK_NS * SK_BSTAGE);
  L.pan = take((rac ? 4 : 2) * SK_PANEL);
  L.xraw = take((rac ? 8 : 4) * SK_NX * SK_XRAW);
  L.offs = take((E + 1) * 4);
  L.pu = take((E + 1) * 4);
  L.sw = take(E * 4);
  L.smask = take(rac ? (K >> 8) * 4 : 0);
  L.bm = take(rac && bm ? (K >> 5) * 4 : 0);
  L.red = take(16 * 4);
  L.total = o;
  return L;
}


// Position in a workgroup's stage sequence: unit u = (expert e, pass p,
// block nb), iteration it over K.  All fields are workgroup-uniform.
struct SkCur {
  int u, it, e, p, nb, ob, rows;
};

struct SkUnits {
  const int32_t *offs;   // LDS: expert offsets [E + 1]
  const int32_t *pu;     // LDS: first unit of each expert [E + 1]
  int E, nblk, niter, u1;

  __device__ void seek(SkCur &c, int u) const {
    int lo = 0, hi = E;                       // last e with pu[e] <= u
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if ((int)uni((uint32_t)pu[mid]) <= u) lo = mid; else hi = mid;
    }
    // (LDS loads land in vector registers; the values are uniform)
    c.u = u;
    c.it = 0;
    c.e = (int)uni((uint32_t)lo);
    const int r = u - (int)uni((uint32_t)pu[c.e]);
    c.p = r / nblk;
    c.nb = r - c.p * nblk;
    c.ob = (int)uni((uint32_t)offs[c.e]);
    c.rows = (int)uni((uint32_t)offs[c.e + 1]) - c.ob;
  }
  // next stage; returns false (and leaves c alone) at the last one
  __device__ bool next(SkCur &c) const {
    if (c.it + 1 < niter) {
      ++c.it;
      return true;
    }
    if (c.u + 1 >= u1) return false;
    if (c.nb + 1 < nblk) {
      ++c.u;
      ++c.nb;
      c.it = 0;
      return true;
    }
    seek(c, c.u + 1);
    return true;
  }
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// One weight stage of a wave: fragment j (16 rows) x chunk c of 16 code
// bytes per lane, and the lane's scale dword of each fragment.
struct BReg {
  u32x4 c00, c01, c10, c11;
  uint32_t s0, s1;
};
// One stage's MFMA work for MTV valid m-tiles.  pan / rpan point at the
// lane's A fragment of k-step 0, m-tile 0 in the stage's f16 panels of x
// and of the masked residual (k-step (c, s) is 2048 (4c + s) bytes further,
// m-tile i 256 i).  hook(k) runs before k-step k (0..7): the caller issues
// its loads for later stages there and decodes the next panels.
template <bool RAC, int MTV, typename Hook>
__device__ __forceinline__ void sk_stage(const BReg &b, const unsigned char *pan,
                                         const unsigned char *rpan, uint32_t sm,
                                         f32x4 (&acc)[2][2], f32x4 (&accr)[2][2], Hook &&hook) {
#pragma unroll
  for (int c2 = 0; c2 < 2; ++c2) {
    const u32x4 bv0 = c2 ? b.c01 : b.c00;
    const u32x4 bv1 = c2 ? b.c11 : b.c10;
    const f16x2 sp0 = scale_pair_of(b.s0, c2), sp1 = scale_pair_of(b.s1, c2);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      hook(c2 * 4 + s);
      const f16x8 bf0 = decode8_sel(bv0[s], sp0, s >= 2);
      const f16x8 bf1 = decode8_sel(bv1[s], sp1, s >= 2);
#pragma unroll
      for (int i = 0; i < MTV; ++i) {
        const f16x8 af =
            *reinterpret_cast<const f16x8 *>(pan + (c2 * 4 + s) * 2048 + i * 256);
        acc[i][0] = mfma16(af, bf0, acc[i][0]);
        acc[i][1] = mfma16(af, bf1, acc[i][1]);
      }
      if (RAC && ((sm >> (4 * c2 + s)) & 1u)) {
#pragma unroll
        for (int i = 0; i < MTV; ++i) {
          const f16x8 rf =
              *reinterpret_cast<const f16x8 *>(rpan + (c2 * 4 + s) * 2048 + i * 256);
          accr[i][0] = mfma16(rf, bf0, accr[i][0]);
          accr[i][1] = mfma16(rf, bf1, accr[i][1]);
        }
      }
    }
  }
}

// A decoding wave (lane group g = wave index % 4) turns its raw slot -- lane
// (row l % 32, chunk l / 32): 16 code bytes at 16 l, the row's scale dword
// at 1024 + 4 (l % 32) -- into its part of an f16 panel stage, where the A
// fragment of k-step (c, s), lane group g, row r sits at
// 2048 (4c + s) + 512 g + 16 r.
__device__ __forceinline__ void sk_decode_panel(const unsigned char *xr, unsigned char *pw,
                                                int lane) {
  const uint4 cw = *reinterpret_cast<const uint4 *>(xr + lane * 16);
  const uint32_t sdw = *reinterpret_cast<const uint32_t *>(xr + 1024 + (lane & 31) * 4);
  const f16x2 sp = scale_pair_of(sdw, lane >> 5);
#pragma unroll
  for (int s = 0; s < 4; ++s)
    *reinterpret_cast<f16x8 *>(pw + s * 2048) = decode8_sel(word_of(cw, s), sp, s >= 2);
}

template <bool GATHER, bool RAC, int EPI>
__global__ __launch_bounds__(SK_THREADS) void gemm_skinny_kernel(GemmArgs p, int nblk) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, g = lane >> 4;
  const int K = p.K, N = p.N, E = p.E;
  const int64_t kb2 = K >> 1, kb16 = K >> 4;
  const bool bmode = RAC && p.r_bitmap != nullptr;
  const SkLayout L = sk_layout(K, E, RAC, bmode);
  const uint32_t lds0 = (uint32_t)(uintptr_t)lds;
  int32_t *offs = reinterpret_cast<int32_t *>(lds + L.offs);
  int32_t *pu = reinterpret_cast<int32_t *>(lds + L.pu);
  float *swv = reinterpret_cast<float *>(lds + L.sw);
  uint32_t *smask = reinterpret_cast<uint32_t *>(lds + L.smask);
  float *red = reinterpret_cast<float *>(lds + L.red);
  const int niter = K >> 8;

  // ---- the unit list: offsets, weight scales, units per expert (scan)
  for (int e = tid; e <= E; e += SK_THREADS)
    offs[e] = p.offsets ? p.offsets[e] : (e == 0 ? 0 : (int)p.rows);
  for (int e = tid; e < E; e += SK_THREADS) swv[e] = p.w_gs[2 * e + 1];
  if (RAC) {
    // k-steps (chunk c, step s -> bit 4c + s) of each iteration that hold a
    // selected channel for some lane group
    for (int i = tid; i < niter; i += SK_THREADS) smask[i] = 0u;
  }
  __syncthreads();
  if (RAC && !bmode) {
    for (int i = tid; i < p.Ks; i += SK_THREADS) {
      const int c = min(max(p.sel[i], 0), K - 1);
      atomicOr(&smask[c >> 8], 1u << (((c >> 5) & 1) * 4 + ((c & 31) >> 3)));
    }
  }
  uint32_t *bml = reinterpret_cast<uint32_t *>(lds + L.bm);
  if (bmode) {
    // word i holds channels 32 i .. 32 i + 31: k-step bits (i & 1) * 4 + q
    // of iteration i / 8 for its non-zero bytes q
    const int nw = K >> 5;
    for (int i = tid; i < nw; i += SK_THREADS) {
      const uint32_t m = p.r_bitmap[i];
      bml[i] = m;
      uint32_t bits = 0u;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if ((m >> (8 * q)) & 0xFFu) bits |= 1u << ((i & 1) * 4 + q);
      if (bits) atomicOr(&smask[i >> 3], bits);
    }
  }
  {
    // exclusive scan of npass(e) * nblk over e (two experts per thread)
    const int e0 = 2 * tid;
    auto units = [&](int e) {
      if (e >= E) return 0;
      const int rows = max(offs[e + 1] - offs[e], 0);
      return (rows + SK_PR - 1) / SK_PR * nblk;
    };
    const int c0 = units(e0), c1 = units(e0 + 1);
    const int v = c0 + c1;
    int xs = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(xs, o, 64);
      if (lane >= o) xs += y;
    }
    if (lane == 63) red[w] = __int_as_float(xs);
    __syncthreads();
    int base = 0;
    for (int ww = 0; ww < w; ++ww) base += __float_as_int(red[ww]);
    const int ex = base + xs - v;
    if (e0 <= E) pu[e0] = ex;
    if (e0 + 1 <= E) pu[e0 + 1] = ex + c0;
    __syncthreads();
  }
  const int U = (int)uni((uint32_t)pu[E]);
  const int P = blockIdx.x, G = gridDim.x;
  const int u0 = (int)((int64_t)P * U / G), u1 = (int)((int64_t)(P + 1) * U / G);
  const SkUnits S{offs, pu, E, nblk, niter, u1};

  float vmax = 0.0f;
  if (u0 < u1) {
    SkCur cc;
    S.seek(cc, u0);
    const float a_dec = p.a_gs[1];
    const float r_dec = RAC ? p.r_gs[1] : 0.0f;
    // ---- issue cursors and their per-lane addresses
    SkCur ca = cc, cb = cc;
    // weight codes: dma i of a stage brings full 128-byte row chunks, lane
    // l row 8 i + l / 8 of the wave's 32 (rows 16..31: the second fragment)
    // and 16-byte piece (l % 8) ^ (l / 8), so the pieces of a row land
    // XOR-swizzled and the fragment reads below are free of bank conflicts
    const uint8_t *bcq[4], *bs0, *bs1;
    const int bq_piece = (lane & 7) ^ (lane >> 3);
    // weight scales: the standard layout (16 bytes per row and stage, in
    // every row's scale line) or the fragment-ordered copy (256 contiguous
    // bytes per 16-row fragment and stage, one dword per lane in lane order)
    const int sstep = p.w_sfrag ? 256 : 16;
    auto bind_b = [&](const SkCur &c) {
      // the wave's two 16-row fragments (all rows of a fragment are valid
      // or none, N and I being multiples of 16; invalid ones read row 0)
      int64_t r0, r1, f0, f1;
      const int lq = lane >> 3;               // fragment row of dma 0 (dma 1: + 8)
      if (EPI == QD_EPI_SWIGLU) {
        const int I = N >> 1;
        const int fr = c.nb * (SK_ROWS / 32) + w;
        const bool ok = 16 * fr < I;
        r0 = ok ? 16 * fr : 0;
        r1 = ok ? 16 * fr + I : 0;
        f0 = ok ? fr : 0;
        f1 = ok ? fr + (I >> 4) : 0;
      } else {
        const int fr = c.nb * (SK_ROWS / 16) + 2 * w;
        const bool ok0 = 16 * fr < N, ok1 = 16 * (fr + 1) < N;
        r0 = ok0 ? 16 * fr : 0;
        r1 = ok1 ? 16 * (fr + 1) : 0;
        f0 = ok0 ? fr : 0;
        f1 = ok1 ? fr + 1 : 0;
      }
      r0 += (int64_t)c.e * N;
      r1 += (int64_t)c.e * N;
      // an invalid fragment reads rows 0..15 of the expert (any valid rows)
      bcq[0] = p.w_codes + (r0 + lq) * kb2 + 16 * bq_piece;
      bcq[1] = p.w_codes + (r0 + lq + 8) * kb2 + 16 * bq_piece;
      bcq[2] = p.w_codes + (r1 + lq) * kb2 + 16 * bq_piece;
      bcq[3] = p.w_codes + (r1 + lq + 8) * kb2 + 16 * bq_piece;
      if (p.w_sfrag) {
        const int64_t nf = N >> 4;
        bs0 = p.w_sfrag + (((int64_t)c.e * nf + f0) * niter) * 256 + lane * 4;
        bs1 = p.w_sfrag + (((int64_t)c.e * nf + f1) * niter) * 256 + lane * 4;
      } else {
        bs0 = p.w_scales + (r0 + lr) * kb16 + g * 4;
        bs1 = p.w_scales + (r1 + lr) * kb16 + g * 4;
      }
    };
    // activations.  Decoding wave w (waves 0..3: x; with RAC waves 4..7:
    // the masked residual; lane group gd = w % 4) loads lane (row l % 32,
    // chunk l / 32)'s 16 code bytes and the row's scale dword into its
    // private raw slot.  Without RAC waves 4..7 load no activations.
    const bool xdec = w < 4;
    const bool has_a = xdec || RAC;
    const int gd = w & 3;
    const int a_row = lane & 31;
    const int64_t a_cb = 32 * gd + 16 * (lane >> 5);
    const int64_t a_sb = 4 * gd;
    const uint8_t *ac, *as;
    int a_e = -1, a_p = -1;
    auto bind_a = [&](const SkCur &c) {
      if (c.e == a_e && c.p == a_p) return;
      a_e = c.e;
      a_p = c.p;
      int64_t r = (int64_t)c.ob + (int64_t)c.p * SK_PR + a_row;
      r = min(r, (int64_t)c.ob + c.rows - 1);
      const int64_t src = GATHER ? (int64_t)p.row_token[r] : r;
      ac = (xdec ? p.a_codes : p.r_codes) + src * kb2 + a_cb;
      as = (xdec ? p.a_scales : p.r_scales) + src * kb16 + a_sb;
    };
    const uint32_t bring = lds0 + L.b + w * SK_NS * SK_BSTAGE;
    const int b_off0 = 128 * lr + 16 * ((2 * g) ^ (lr & 7));
    const int b_off1 = 128 * lr + 16 * ((2 * g + 1) ^ (lr & 7));
    // the raw slot of stage sg (codes; the scale dwords 1024 further)
    auto a_raw = [&](int sg) -> uint32_t {
      return lds0 + L.xraw + (w * SK_NX + sg % SK_NX) * SK_XRAW;
    };
    auto issue_a = [&](int sg) {
      dma16(ac + ca.it * 128, uni(a_raw(sg)));
      dma4(as + ca.it * 16, uni(a_raw(sg) + 1024));
    };
    auto issue_b = [&](int sg) {
      const uint32_t slot = uni(bring + (sg % SK_NS) * SK_BSTAGE);
      const int off = cb.it * 128;
      dma16(bcq[0] + off, slot);
      dma16(bcq[1] + off, slot + 1024);
      dma16(bcq[2] + off, slot + 2048);
      dma16(bcq[3] + off, slot + 3072);
      dma4(bs0 + cb.it * sstep, slot + 4096);
      dma4(bs1 + cb.it * sstep, slot + 4096 + 256);
    };
    auto adv_b = [&]() {
      const int e = cb.e, nb = cb.nb;
      if (S.next(cb) && (cb.e != e || cb.nb != nb)) bind_b(cb);
    };
    auto adv_a = [&]() {
      if (S.next(ca)) bind_a(ca);
    };
    // the panel slot of stage sg (source x: 0, residual: 1), seen from this
    // lane as a decoder (write) and as a reader (its A fragment of k-step 0,
    // m-tile 0)
    auto pan_w = [&](int sg) {
      return lds + L.pan + ((w >> 2) * 2 + (sg & 1)) * SK_PANEL + (lane >> 5) * 8192 + gd * 512 +
             (lane & 31) * 16;
    };
    auto pan_r = [&](int src, int sg) {
      return lds + L.pan + (src * 2 + (sg & 1)) * SK_PANEL + g * 512 + lr * 16;
    };

    // ---- prologue: the steady-state issue order for stages 0 and 1
    // (A0 | A1 B0 | B1), then the panel of stage 0
    bind_b(cb);
    bind_a(ca);
    if (has_a) {
      issue_a(0);
      adv_a();
      issue_a(1);
      adv_a();
    }
    for (int i = 0; i < 2; ++i) {
      issue_b(i);
      adv_b();
    }
    if (has_a) {
      wait_vm<14>();         // this wave's activations of stage 0
      sk_decode_panel(lds + L.xraw + (w * SK_NX) * SK_XRAW, pan_w(0), lane);
    }

    f32x4 acc[2][2], accr[2][2];   // [m-tile][fragment]
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        accr[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      }

    for (int sg = 0;; ++sg) {
      const int nrow = min(SK_PR, cc.rows - cc.p * SK_PR);
      const int mtv = nrow > 16 ? 2 : 1;
      // outstanding past this point: at most the weights of stage sg + 1
      wait_vm<6>();
      __syncthreads();       // the panels of stage sg are complete
      const unsigned char *bsl = lds + L.b + (w * SK_NS + sg % SK_NS) * SK_BSTAGE;
      // row r of the stage (r < 16: first fragment) holds piece q at
      // 128 r + 16 (q ^ (r % 8)); this lane needs pieces 2g, 2g + 1 of rows
      // lr and 16 + lr
      BReg b;
      b.c00 = *reinterpret_cast<const u32x4 *>(bsl + b_off0);
      b.c01 = *reinterpret_cast<const u32x4 *>(bsl + b_off1);
      b.c10 = *reinterpret_cast<const u32x4 *>(bsl + 2048 + b_off0);
      b.c11 = *reinterpret_cast<const u32x4 *>(bsl + 2048 + b_off1);
      b.s0 = *reinterpret_cast<const uint32_t *>(bsl + 4096 + lane * 4);
      b.s1 = *reinterpret_cast<const uint32_t *>(bsl + 4096 + 256 + lane * 4);
      const uint32_t sm = RAC ? smask[cc.it] : 0u;
      // before k-step 0 and 1: the activations of stage sg + 2 (into the
      // raw slot decoded in the last iteration); before k-step 2: the decode
      // of stage sg + 1's panels; before k-steps 2..7: the weights of stage
      // sg + 2 into the slot just read
      auto hook = [&](int k) {
        if (k < 2) {
          if (has_a) {
            if (k == 0) dma16(ac + ca.it * 128, uni(a_raw(sg + 2)));
            else dma4(as + ca.it * 16, uni(a_raw(sg + 2) + 1024));
          }
        } else {
          if (k == 2 && has_a)
            sk_decode_panel(lds + L.xraw + (w * SK_NX + (sg + 1) % SK_NX) * SK_XRAW,
                            pan_w(sg + 1), lane);
          const uint32_t slot = uni(bring + (sg % SK_NS) * SK_BSTAGE);
          const int off = cb.it * 128, soff = cb.it * sstep;
          if (k == 2) dma16(bcq[0] + off, slot);
          if (k == 3) dma16(bcq[1] + off, slot + 1024);
          if (k == 4) dma16(bcq[2] + off, slot + 2048);
          if (k == 5) dma16(bcq[3] + off, slot + 3072);
          if (k == 6) dma4(bs0 + soff, slot + 4096);
          if (k == 7) dma4(bs1 + soff, slot + 4096 + 256);
        }
      };
      const unsigned char *pr = pan_r(0, sg);
      const unsigned char *prr = pan_r(RAC ? 1 : 0, sg);
      wait_lds();            // the weight slot may be refilled from here on
      if (mtv == 1)
        sk_stage<RAC, 1>(b, pr, prr, sm, acc, accr, hook);
      else
        sk_stage<RAC, 2>(b, pr, prr, sm, acc, accr, hook);
      if (has_a) adv_a();
      adv_b();

      if (cc.it == niter - 1) {
        // ---- end of a unit: epilogue
        const float sw = swv[cc.e];
        const float alpha = a_dec * sw, alpha_r = r_dec * sw;
        const int64_t rg = (int64_t)cc.ob + (int64_t)cc.p * SK_PR;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int rl = i * 16 + g * 4 + q;
            if (rl < nrow) {
              const int64_t row = rg + rl;
              if (EPI == QD_EPI_SWIGLU) {
                const int I = N >> 1;
                const int col = cc.nb * (SK_ROWS / 2) + w * 16 + lr;
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
                  const int col = cc.nb * SK_ROWS + w * 32 + j * 16 + lr;
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
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
            accr[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
          }
      }
      if (!S.next(cc)) break;
    }
    // loads past the last stage still target this workgroup's LDS
    wait_vm<0>();
  }
  if (bmode && blockIdx.x == 0 && w == 0) {
    // S in ascending order from the bitmap in LDS, by workgroup 0's first
    // wave once its stages are done (<= 128 words: two per lane)
    const int nw = K >> 5;
    uint32_t m0 = 2 * lane < nw ? bml[2 * lane] : 0u;
    uint32_t m1 = 2 * lane + 1 < nw ? bml[2 * lane + 1] : 0u;
    const int c = __popc(m0) + __popc(m1);
    int xs = c;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(xs, o, 64);
      if (lane >= o) xs += y;
    }
    int pos = xs - c;
    while (m0) {
      p.sel_out[pos++] = 64 * lane + (__ffs(m0) - 1);
      m0 &= m0 - 1u;
    }
    while (m1) {
      p.sel_out[pos++] = 64 * lane + 32 + (__ffs(m1) - 1);
      m1 &= m1 - 1u;
    }
  }
  const float m = block_max(vmax, red);
  if (p.amax_part && tid == 0) p.amax_part[P] = m;
}

// ---------------------------------------------------------------------------
// Prefill-shaped grouped GEMM (hundreds of rows per expert): MFMA-bound.
//
//  * Workgroup tile 256 rows x 128 weight rows (SwiGLU: 64 gate rows and
//    the matching 64 up rows); four waves in a 2 x 2 grid, each 128 x 64 on
//    v_mfma_f32_32x32x16_f16 (4 x 2 fragments, 128 accumulators), two
//    workgroups per CU.  Two waves share each SIMD, so one wave's decode
//    VALU work runs under the other's MFMAs, and one workgroup's prologue
//    and epilogue under the other's main loop.  A tile of at most 128 rows
//    (an expert's remainder) splits its rows 64 / 64 between the wave rows
//    instead, and fragments wholly past the expert's last row are skipped.
//  * Operand codes are decoded to f16 in registers right before use.
//  * M-tiles never straddle experts.  The grid is an upper bound on the
//    tile count; every workgroup derives the real tiles from the expert
//    offsets, and tile indices run contiguously within an XCD (workgroups
//    are dealt to the eight XCDs in turn), so the tiles in flight on an
//    XCD share an expert's weights or a block of activation rows in its L2.
//  * K goes through a ring of TL_NS LDS slots of 64-element stages filled
//    by direct global->LDS loads (five per wave and stage) TL_NS - 1 stages
//    ahead.  A wave reads a stage's raw codes and scales into registers one
//    stage before it multiplies them: halfway through stage s it waits for
//    stage s + 1, meets the other waves at a barrier, issues the loads of
//    stage s + TL_NS - 1 into the slot of stage s - 1 (read during stage
//    s - 2) and reads stage s + 1 while the MFMAs of stage s drain.
//
//  * RAC: the residual contraction runs over the selected channels alone,
//    compacted.  While a stage is in LDS the workgroup copies the selected
//    channels of its weight rows out of it, decoded to f16, into a compact
//    [128 rows][K_s] LDS table; after the K loop the accumulators are
//    rescaled by -s_dec_x / s_dec_r and the residual (compacted per token,
//    f16, from the caller) is multiplied onto them against that table, so
//    the epilogue's single scale -s_dec_r * s_dec_w yields
//    s_dec_x s_dec_w acc - s_dec_r s_dec_w accr with one extra f32 rounding
//    of the main sum.  A ring of three slots leaves LDS room for the table.
//
// Stage slot: A codes [8 fragments][64 lanes][16 B], B codes [4 fragments]
// likewise, then A scale dwords [256 rows] and B scale dwords [128 rows].
// Scale loads are the costly part of a stage (4 bytes per row, each in a
// different scale line): the B scales come from the weights'
// fragment-ordered copy when present (64 contiguous bytes per 16 rows), and
// when LDS allows, the A scales of four stages at a time (16 contiguous
// bytes per row, one load per 16-byte piece) go into a two-slot ring of their
// own.  With the four-slot ring the three stages between those loads issue a
// one-line placeholder load instead, so every stage issues the same number of
// loads; with the three-slot ring (RAC) the wait before each stage covers
// every outstanding load, so those stages issue none, and the stage slot
// drops its A-scale area (B scales right after the codes), which leaves the
// A-scale ring room beside the compact table.
// Lane l of a fragment holds row l % 32, elements 32 (l / 32) .. +31 of the
// stage; MFMA k-step s (0..3) takes elements 8s .. 8s+7 of each half, for A
// and B alike.
constexpr int TL_THREADS = 256;
constexpr int TL_M = 256;
constexpr int TL_N = 128;
constexpr int TL_K = 64;
constexpr int TL_ACODE = 0;
constexpr int TL_BCODE = 8192;
constexpr int TL_ASCL = 12288;
constexpr int TL_BSCL = 13312;
constexpr int TL_STAGE = 13824;
constexpr int TL_BSCL_G = 12288;         // three-slot ring with the A-scale ring
constexpr int TL_STAGE_G = 12800;
constexpr int TL_PAD = 4;                // f16 columns past each compact table row
constexpr int TL_EMAX = 1024;            // experts handled by the tile scan (4 per thread)
constexpr int TL_LDS_MAX = 160 * 1024 - 1024;   // dynamic LDS beside the static arrays

// ring depth: four slots, or three with RAC, which leaves LDS room for the
// compact table (three slots measured 1-3% slower without RAC)
__host__ __device__ constexpr int tl_ns(bool rac) { return rac ? 3 : 4; }
// stage slot size and the B-scale offset inside it (grp: the A-scale ring is on)
__host__ __device__ constexpr int tl_stage(bool rac, bool grp) {
  return tl_ns(rac) == 3 && grp ? TL_STAGE_G : TL_STAGE;
}
__host__ __device__ constexpr int tl_bscl(bool rac, bool grp) {
  return tl_ns(rac) == 3 && grp ? TL_BSCL_G : TL_BSCL;
}
// LDS: ring, then (RAC) the compact weight table [128][ksa + TL_PAD] f16 and
// the selected channels [ksa], then (grp) the A-scale ring
__host__ __device__ inline int tl_lds_bytes(bool rac, int ksa, bool grp) {
  return tl_ns(rac) * tl_stage(rac, grp) + (rac ? TL_N * (ksa + TL_PAD) * 2 + ksa * 4 : 0);
}
constexpr int TL_AGRP = 2 * TL_M * 16;   // the A-scale ring: 2 slots x 256 rows x 16 B
constexpr int TL_LDS_2WG = TL_LDS_MAX / 2;   // two workgroups per CU

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x16 mfma32(f16x8 a, f16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// the tile's weight row tb (0..127): for SwiGLU, fragments (32 rows) 0, 1
// are gate rows and 2, 3 the matching up rows
template <int EPI>
__device__ __forceinline__ int tile_wrow(int tb, int nt, int N) {
  if (EPI == QD_EPI_SWIGLU) {
    const int f = tb >> 5, r = tb & 31;
    return (f < 2 ? 0 : (N >> 1)) + nt * 64 + (f & 1) * 32 + r;
  }
  return nt * TL_N + tb;
}

// a wave's raw operands of one stage: A fragments fa0 .. fa0 + 3 and B
// fragments fb0, fb0 + fbs
struct TlRaw {
  uint4 a[4], b[2];
  uint32_t as[4], bs[2];
};

// ascl / astr: the A scale dword of row r of this stage is at ascl + r * astr
template <int MTV>
__device__ __forceinline__ void tl_read(TlRaw &R, const unsigned char *sl, const unsigned char *ascl,
                                        int astr, int bscl, int fa0, int fb0, int fbs, int lane) {
  const int r = lane & 31;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int fb = fb0 + j * fbs;
    R.b[j] = *reinterpret_cast<const uint4 *>(sl + TL_BCODE + (fb * 64 + lane) * 16);
    R.bs[j] = *reinterpret_cast<const uint32_t *>(sl + bscl + (fb * 32 + r) * 4);
  }
#pragma unroll
  for (int i = 0; i < MTV; ++i) {
    const int fa = fa0 + i;
    R.a[i] = *reinterpret_cast<const uint4 *>(sl + TL_ACODE + (fa * 64 + lane) * 16);
    R.as[i] = *reinterpret_cast<const uint32_t *>(ascl + (fa * 32 + r) * astr);
  }
}

// One stage of MFMA work on MTV A fragments and two B fragments; mid() runs
// between k-steps 1 and 2.
template <int MTV, typename Mid>
__device__ __forceinline__ void tl_stage(const TlRaw &R, f32x16 (&acc)[4][2], int lane, Mid &&mid) {
  const int h = lane >> 5;
  f16x2 ap[MTV], bp[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) bp[j] = scale_pair_of(R.bs[j], h);
#pragma unroll
  for (int i = 0; i < MTV; ++i) ap[i] = scale_pair_of(R.as[i], h);
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    if (s == 2) mid();
    f16x8 bf[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) bf[j] = decode8_sel(word_of(R.b[j], s), bp[j], s >= 2);
#pragma unroll
    for (int i = 0; i < MTV; ++i) {
      const f16x8 af = decode8_sel(word_of(R.a[i], s), ap[i], s >= 2);
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = mfma32(af, bf[j], acc[i][j]);
    }
    // scheduling: each MFMA followed by six VALU instructions (the next
    // operands' decode), where the compiler's own order clusters up to six
    // MFMAs and 28 VALU instructions (measured 2-3% faster at prefill)
#pragma unroll
    for (int q = 0; q < 2 * MTV; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);   // six VALU
    }
  }
}

// silu(g) * u from f32 g and u: exp on the transcendental unit and one
// reciprocal (a few f32 ulp, far inside the bf16 rounding that follows)
__device__ __forceinline__ float swiglu_fast(float g, float u) {
  const float e = __builtin_amdgcn_exp2f(-g * 1.4426950408889634f);
  return g * __builtin_amdgcn_rcpf(1.0f + e) * u;
}

// DENSE (with RAC): the residual as a second pass over K on the masked
// residual codes (for K_s too large for the compact table)
template <bool GATHER, bool RAC, int EPI, bool DENSE = false>
__global__ __launch_bounds__(TL_THREADS, 2) void gemm_tile_kernel(GemmArgs p, int ntn, int grp) {
  static_assert(RAC || !DENSE, "the dense residual mode needs RAC");
  constexpr bool CMP = RAC && !DENSE;      // compact residual table
  constexpr int NS = tl_ns(CMP);
  extern __shared__ __align__(16) unsigned char lds[];
  __shared__ int sh_w[4];
  __shared__ int sh_t[4];
  __shared__ float red[16];
  const int tid = threadIdx.x, lane = tid & 63, w = (int)uni((uint32_t)tid >> 6);
  const int K = p.K, N = p.N, E = p.E;
  const int64_t kb2 = K >> 1, kb16 = K >> 4;

  const qdt::Tile tl = qdt::find_tile<TL_M>(p.offsets, E, p.rows, ntn, sh_w, sh_t);
  const int e = tl.e, nt = tl.nt;
  float vmax = 0.0f;
  if (e >= 0) {
    const int row0 = tl.row0, nrows = tl.nrows;
    const uint32_t lds0 = (uint32_t)(uintptr_t)lds;
    // ---- per-lane load offsets from uniform bases (rows past the tile
    // repeat its first row; one operand of one expert < 4 GiB)
    auto arow = [&](int r) __attribute__((always_inline)) -> uint32_t {
      const int rr = r < nrows ? r : 0;
      return GATHER ? (uint32_t)p.row_token[row0 + rr] : (uint32_t)(row0 + rr);
    };
    const uint32_t hb = 16u * (uint32_t)(lane >> 5);
    const uint32_t oa0 = arow(64 * w + (lane & 31)) * (uint32_t)kb2 + hb;
    const uint32_t oa1 = arow(64 * w + 32 + (lane & 31)) * (uint32_t)kb2 + hb;
    const uint32_t ob = (uint32_t)tile_wrow<EPI>(32 * w + (lane & 31), nt, N) * (uint32_t)kb2 + hb;
    const uint32_t oas = arow(64 * w + lane) * (uint32_t)kb16;
    const int bsr = tile_wrow<EPI>(64 * (w & 1) + lane, nt, N);
    const bool sfrag = p.w_sfrag != nullptr;
    // B scales: the standard layout (4 bytes of the row's line per stage) or
    // the fragment-ordered copy (fragment f, chunk s / 4: 256 bytes, of
    // which stage s takes the 64 at (s % 4) * 64, 4 per row)
    const uint32_t obs = sfrag ? (uint32_t)(((bsr >> 4) * (K >> 8)) * 256 + (bsr & 15) * 4)
                               : (uint32_t)bsr * (uint32_t)kb16;
    const uint8_t *wc = uni_ptr(p.w_codes + (int64_t)e * N * kb2);
    const uint8_t *ws = uni_ptr((sfrag ? p.w_sfrag : p.w_scales) + (int64_t)e * N * kb16);
    const int bsstep = sfrag ? 64 : 4;
    const int nst = K / TL_K;
    // stage slots, and the A-scale ring (grp) after them and the compact table
    const int tls = tl_stage(CMP, grp != 0), bsc = tl_bscl(CMP, grp != 0);
    const uint32_t agrp = lds0 + (uint32_t)tl_lds_bytes(CMP, CMP ? p.ksa : 0, grp != 0);
    const uint32_t oag = arow(64 * w + lane) * (uint32_t)kb16;
    // the staged A operand (first pass only): row offsets within a stage's
    // [rows][32 B] and a group's [rows][16 B] record
    bool stg = GATHER && grp && p.a_stg != nullptr;
    auto srow = [&](int r) __attribute__((always_inline)) -> uint32_t {
      return (uint32_t)(row0 + (r < nrows ? r : 0));
    };
    const uint32_t os0 = srow(64 * w + (lane & 31)) * 32u + hb;
    const uint32_t os1 = srow(64 * w + 32 + (lane & 31)) * 32u + hb;
    const uint32_t osg = srow(64 * w + lane) * 16u;
    // five loads per wave and stage, four between A-scale groups with the
    // three-slot ring (waves 0 / 2 and 1 / 3 load the same B scale half:
    // equal bytes to equal places)
    // the A operand of the pass: the activations, then (DENSE) the masked
    // residual, same layout
    const uint8_t *a_cod = p.a_codes, *a_scl = p.a_scales;
    auto issue = [&](int s, int q) __attribute__((always_inline)) {
      s = min(s, nst - 1);
      const uint32_t sb = uni(lds0 + q * tls);
      const uint8_t *ac = uni_ptr(a_cod + s * 32), *as_ = uni_ptr(a_scl + s * 4);
      const uint8_t *bc = uni_ptr(wc + s * 32), *bs_ = uni_ptr(ws + s * bsstep);
      if (stg) {
        const uint8_t *sc = uni_ptr(p.a_stg + (int64_t)s * p.rows * 32);
        dma16s(sc, os0, sb + TL_ACODE + (2 * w) * 1024);
        dma16s(sc, os1, sb + TL_ACODE + (2 * w + 1) * 1024);
      } else {
        dma16s(ac, oa0, sb + TL_ACODE + (2 * w) * 1024);
        dma16s(ac, oa1, sb + TL_ACODE + (2 * w + 1) * 1024);
      }
      dma16s(bc, ob, sb + TL_BCODE + w * 1024);
      if (grp) {
        // stage 4G brings group G's A scales (rows 64 w .. 64 w + 63, 16 B
        // each) into ring slot G % 2; with four slots other stages load one
        // line (the group scales of the wave's first row: a different line
        // per workgroup, never one line for the whole chip) into the unused
        // A-scale area of their stage slot
        if ((s & 3) == 0) {
          if (stg)
            dma16s(uni_ptr(p.a_stg + (int64_t)p.rows * kb2 + (int64_t)(s >> 2) * p.rows * 16), osg,
                   uni(agrp + ((s >> 2) & 1) * (TL_AGRP / 2) + w * 1024));
          else
            dma16s(uni_ptr(a_scl + (s >> 2) * 16), oag,
                   uni(agrp + ((s >> 2) & 1) * (TL_AGRP / 2) + w * 1024));
        }
        else if constexpr (NS != 3)
          dma16s(uni_ptr(a_scl + (s >> 2) * 16), uni(oag), sb + TL_ASCL);
      } else {
        dma4s(as_, oas, sb + TL_ASCL + w * 256);
      }
      dma4s(bs_, obs, sb + bsc + (w & 1) * 256);
    };
    // where tl_read finds stage s's A scales
    auto a_src = [&](int s) __attribute__((always_inline)) -> const unsigned char * {
      return grp ? lds + (agrp - lds0) + ((s >> 2) & 1) * (TL_AGRP / 2) + (s & 3) * 4
                 : lds + (s % NS) * tls + TL_ASCL;
    };
    const int astr = grp ? 16 : 4;
    const float a_dec = p.a_gs[1], sw = p.w_gs[2 * e + 1];
    float alpha = a_dec * sw;
    // RAC: acc -> acc * inv_c + accr, then alpha = -s_dec_r * s_dec_w.  A
    // residual whose tensor scale is below 2^-60 of the activation's is
    // left out (its share of any output is far below f32 resolution).
    float inv_c = 0.0f;
    bool res_on = false;
    const int ksa = CMP ? p.ksa : 0, ksp = ksa + TL_PAD;
    unsigned char *bres = lds + NS * tls;
    int32_t *sel_l = reinterpret_cast<int32_t *>(bres + TL_N * ksp * 2);
    if (RAC) {
      const float r_dec = p.r_gs[1];
      inv_c = -(a_dec / r_dec);
      res_on = r_dec > 0.0f && fabsf(inv_c) <= 0x1p60f;
      if (res_on) alpha = -r_dec * sw;
      if constexpr (CMP) {
        for (int i = tid; i < ksa; i += TL_THREADS)
          sel_l[i] = i < p.Ks ? p.sel[(int64_t)e * p.sel_stride + i] : 0;
        // pad columns of the compact table are zero (the residual's are too)
        const int pad = ksa - p.Ks;
        for (int i = tid; i < TL_N * pad; i += TL_THREADS)
          *reinterpret_cast<_Float16 *>(bres + ((i / pad) * ksp + p.Ks + i % pad) * 2) =
              (_Float16)0.0f;
      }
    }
    const int wm = w & 1, wn = w >> 1;
    const bool wide = nrows > 128;
    const int fa0 = wide ? 4 * wm : 2 * wm;
    const int mtv = wide ? min(max((nrows - 128 * wm + 31) >> 5, 0), 4)
                         : min(max((nrows - 64 * wm + 31) >> 5, 0), 2);
    const int fb0 = EPI == QD_EPI_SWIGLU ? wn : 2 * wn;
    const int fbs = EPI == QD_EPI_SWIGLU ? 2 : 1;

    // one straight-line loop per number of valid fragments
    auto run = [&](auto mtv_c) __attribute__((always_inline)) {
      constexpr int MTV = decltype(mtv_c)::value;
      f32x16 acc[4][2];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int t = 0; t < 16; ++t) acc[i][j][t] = 0.0f;
      TlRaw R0, R1;
      // RAC: the tokens of this lane's residual rows, loaded before the K
      // loop so the residual steps after it wait for one load, not two
      int32_t tkr[MTV > 0 ? MTV : 1];
      if constexpr (CMP && MTV > 0) {
#pragma unroll
        for (int i = 0; i < MTV; ++i) {
          const int rr = 32 * (fa0 + i) + (lane & 31);
          const int rc = rr < nrows ? rr : 0;
          tkr[i] = (GATHER && !p.rsel_rows) ? p.row_token[row0 + rc] : row0 + rc;
        }
      }
      // RAC: the next selected channel this wave copies (waves 0, 1 take the
      // even entries of S, waves 2, 3 the odd ones; S is ascending), held in a
      // register so a stage without one of its channels costs one compare
      // (read after the prologue's barrier: other threads wrote sel_l)
      int nk = tid >> 7;
      int nsel = 0x7fffffff;
      auto body = [&](const TlRaw &Rc, TlRaw &Rn, int s) __attribute__((always_inline)) {
        auto mid = [&]() __attribute__((always_inline)) {
          wait_vm<(NS - 3) * 5>();
          __syncthreads();
          issue(s + NS - 1, (s + NS - 1) % NS);
          if constexpr (MTV > 0)
            tl_read<MTV>(Rn, lds + ((s + 1) % NS) * tls, a_src(s + 1), astr, bsc, fa0, fb0, fbs,
                         lane);
          if constexpr (CMP) {
            // selected channels of stage s (slot s % NS holds it until the
            // next barrier): decoded weight values into the compact table
            // (the hardware FP4 conversion with a power-of-two scale and one
            // f16 multiply by the E4M3 scale, as in the operand decode: exact;
            // the next channel of the wave is fetched before this one's work)
            const unsigned char *sl = lds + (s % NS) * tls;
            const int tb = tid & 127, f = tb >> 5, r = tb & 31;
            while (nsel < TL_K * (s + 1)) {     // wave-uniform
              const int el = nsel - TL_K * s;   // >= 0: S is ascending
              const int nk2 = nk + 2;
              const int nxt = nk2 < p.Ks ? sel_l[nk2] : 0x7fffffff;
              const uint32_t byte = sl[TL_BCODE + ((f * 64 + (el >> 5) * 32 + r) * 16) + ((el & 31) >> 1)];
              const uint32_t sbyte = sl[bsc + tb * 4 + (el >> 4)];
              const f16x2 v2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(byte, 256.0f, 0);
              const f16x2 sc = __builtin_bit_cast(f16x2, sbyte << 7);
              *reinterpret_cast<_Float16 *>(bres + (tb * ksp + nk) * 2) = (el & 1 ? v2[1] : v2[0]) * sc[0];
              nk = nk2;
              nsel = (int)uni((uint32_t)nxt);
            }
          }
        };
        if constexpr (MTV > 0) tl_stage<MTV>(Rc, acc, lane, mid);
        else mid();
      };
      // one pass over K: the ring's prologue, then the stages
      auto kpass = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int t = 0; t < NS - 1; ++t) issue(t, t);
        // stage 0 has landed once at most stage NS - 2's loads are in flight
        // (three slots with the A-scale ring: stage 1 issues four)
        if (NS == 3 && grp) wait_vm<4>();
        else wait_vm<(NS - 2) * 5>();
        __syncthreads();
        if constexpr (CMP) nsel = nk < p.Ks ? (int)uni((uint32_t)sel_l[nk]) : 0x7fffffff;
        if constexpr (MTV > 0) tl_read<MTV>(R0, lds, a_src(0), astr, bsc, fa0, fb0, fbs, lane);
        for (int s = 0; s < nst; s += 2) {     // nst is even
          body(R0, R1, s);
          body(R1, R0, s + 1);
        }
        wait_vm<0>();
      };
      kpass();
      if constexpr (DENSE) {
        // the residual: acc -> acc * inv_c, then a second pass over K with
        // the masked residual codes as the A operand (zero outside S), so the
        // epilogue's scale -s_dec_r * s_dec_w yields
        // s_dec_x s_dec_w acc - s_dec_r s_dec_w accr
        if (res_on) {
          __syncthreads();                     // every wave is done with the ring
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
              for (int q = 0; q < 16; ++q) acc[i][j][q] *= inv_c;
          a_cod = p.r_codes;
          a_scl = p.r_scales;
          stg = false;
          kpass();
        }
      }
      if constexpr (CMP) {
        if (res_on) {
          __syncthreads();                     // the compact table is complete
          if constexpr (MTV > 0) {
            const int h = lane >> 5;
            const uint16_t *ar[MTV];
#pragma unroll
            for (int i = 0; i < MTV; ++i) ar[i] = p.r_sel + (int64_t)tkr[i] * ksa + 8 * h;
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
              for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int q = 0; q < 16; ++q) acc[i][j][q] *= inv_c;
            f16x8 an[MTV];
#pragma unroll
            for (int i = 0; i < MTV; ++i) an[i] = *reinterpret_cast<const f16x8 *>(ar[i]);
            for (int c = 0; c < ksa; c += 16) {
              f16x8 ac[MTV], bfr[2];
#pragma unroll
              for (int i = 0; i < MTV; ++i) {
                ac[i] = an[i];
                if (c + 16 < ksa) an[i] = *reinterpret_cast<const f16x8 *>(ar[i] + c + 16);
              }
#pragma unroll
              for (int j = 0; j < 2; ++j) {
                const int fb = fb0 + j * fbs;
                // rows are 8-byte aligned: two 8-byte reads
                const uint2 *q = reinterpret_cast<const uint2 *>(
                    bres + ((32 * fb + (lane & 31)) * ksp + c + 8 * h) * 2);
                const uint2 lo = q[0], hi = q[1];
                bfr[j] = __builtin_bit_cast(f16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
              }
#pragma unroll
              for (int i = 0; i < MTV; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = mfma32(ac[i], bfr[j], acc[i][j]);
            }
          }
        }
      }
      // ---- epilogue: tensor scales, SwiGLU or plain, bf16 pairs of
      // adjacent columns swapped between neighbouring lanes so that every
      // store writes 4 bytes
      const int h = lane >> 5;
      const bool odd = (lane & 1) != 0;
      const int cpair = (lane & 31) & ~1;
      constexpr int NO = EPI == QD_EPI_SWIGLU ? 1 : 2;
      const int ldo = EPI == QD_EPI_SWIGLU ? (N >> 1) : N;
      const bool full = nrows == TL_M;
      unsigned char *obase = reinterpret_cast<unsigned char *>(p.out);
#pragma unroll
      for (int i = 0; i < MTV; ++i) {
        const int rl = 32 * (fa0 + i) + 4 * h + (odd ? 1 : 0);
#pragma unroll
        for (int jj = 0; jj < NO; ++jj) {
          const int fb = fb0 + jj * fbs;
          const int cb = EPI == QD_EPI_SWIGLU ? nt * 64 + (fb & 1) * 32 : nt * TL_N + 32 * fb;
          const uint32_t voff = (uint32_t)((row0 + rl) * ldo + cb + cpair) * 2u;
          float v[16];
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            if (EPI == QD_EPI_SWIGLU)
              v[q] = swiglu_fast(alpha * acc[i][0][q], alpha * acc[i][1][q]);
            else
              v[q] = alpha * acc[i][jj][q];
          }
#pragma unroll
          for (int q = 0; q < 16; q += 2) {
            const float send = odd ? v[q] : v[q + 1];
            const float x = __int_as_float(
                __builtin_amdgcn_mov_dpp(__float_as_int(send), 0xB1, 0xF, 0xF, false));
            const f32x2_t pr = odd ? f32x2_t{x, v[q + 1]} : f32x2_t{v[q], x};
            const uint32_t pk = __builtin_bit_cast(uint32_t, __builtin_convertvector(pr, bf16x2_t));
            const int qr = 8 * (q >> 2) + (q & 3);
            if (full || rl + qr < nrows) {
              *reinterpret_cast<uint32_t *>(obase + (size_t)(qr * ldo * 2) + voff) = pk;
              vmax = fmaxf(vmax, fmaxf(fabsf(__uint_as_float(pk << 16)),
                                       fabsf(__uint_as_float(pk & 0xFFFF0000u))));
            }
          }
        }
      }
    };
    switch (mtv) {
      case 4: run(std::integral_constant<int, 4>{}); break;
      case 3: run(std::integral_constant<int, 3>{}); break;
      case 2: run(std::integral_constant<int, 2>{}); break;
      case 1: run(std::integral_constant<int, 1>{}); break;
      default: run(std::integral_constant<int, 0>{}); break;
    }
  }
  const float m = block_max(vmax, red);
  put_amax(p, m);
}

// ---------------------------------------------------------------------------
// Prefill-shaped grouped GEMM with wide tiles (hundreds of rows per expert).
//
// What bounds the exact-NVFP4 prefill GEMM on gfx950 is VALU work per MFMA,
// not bytes: every operand fragment is decoded in registers (8 VALU ops per
// 32x16 fragment), so the decode cost per MFMA falls with the wave tile.
//
//  * Workgroup tile 256 rows x 256 weight rows (SwiGLU: 128 gate rows and
//    the matching 128 up rows), four waves in a 2 x 2 grid, each 128 x 128
//    on v_mfma_f32_32x32x16_f16 (4 x 4 fragments, 256 accumulators): one
//    wave per SIMD, 8 fragment decodes per 16 MFMAs.  M-tiles never straddle
//    experts; a tile of at most 128 rows splits them 64 / 64 between the
//    wave rows, and fragments wholly past the expert's last row are skipped.
//  * K in stages of 128 elements through a two-slot LDS ring filled by direct
//    global->LDS loads: every load brings 16 rows x 64 contiguous bytes, the
//    16-byte pieces of a row placed by a row-dependent XOR so the fragment
//    reads are free of bank conflicts.  A wave reads a stage's raw codes and
//    scales into registers one stage before it multiplies them: halfway
//    through stage s it waits for stage s + 1, meets the other waves at the
//    one barrier of the stage, issues the loads of stage s + 2 into the slot
//    stage s occupied and reads stage s + 1 while the MFMAs of stage s drain.
//  * Inside a stage lane (row r, half h) owns elements 64 h .. 64 h + 63;
//    MFMA k-step s (0..7) takes elements 8 s .. 8 s + 7 of each half, for A
//    and B alike (a common permutation of K).
//  * Scales: the weights' from their fragment-ordered copy (128 contiguous
//    bytes per 16 rows and stage), the activations' 16 bytes per row every
//    second stage into a ring of their own; odd stages issue a one-line
//    placeholder load instead, so every stage issues ten loads per wave.
//  * Persistent: one workgroup per CU walks a static list of tiles; halfway
//    through the last two stages of a tile it issues the first two stages
//    of its next tile, so the next tile's loads overlap the epilogue.
//  * Plain W4A4 only (no fused residual): with the RAC residual fused, the
//    compact weight table and the residual operand do not fit beside the
//    256 accumulators of this tile shape, and the 256 x 128 tile kernel
//    below takes those problems.
constexpr int TW_THREADS = 256;
constexpr int TW_M = 256;
constexpr int TW_N = 256;
constexpr int TW_K = 128;
constexpr int TW_ACODE = 0;               // [8 fragments][2 halves][64 lanes][16 B]
constexpr int TW_BCODE = 16384;          // the same for the 256 weight rows
constexpr int TW_BSCL = 32768;           // [16 row groups][128 B]
constexpr int TW_STAGE = 34816;
constexpr int TW_ASCL = 2 * TW_STAGE;    // A-scale ring [2 slots][256 rows][16 B]
constexpr int TW_DUMMY = TW_ASCL + 8192; // target of the odd stages' placeholder load
constexpr int TW_TOK = TW_DUMMY + 1024;  // gathered rows: tokens of the current and next tile [2][256]
constexpr int TW_SCHED = TW_TOK + 2 * TW_M * 4;   // the tile schedule: two int arrays [E + 1]
constexpr int TW_LOADS = 10;             // loads per wave and stage
__host__ __device__ inline int tw_lds_bytes(int E) { return TW_SCHED + 2 * (E + 1) * 4; }

// 16-byte piece p of tile row ri (0..15 within a 16-row load) sits at piece
// p ^ tw_swz(ri) of the row's 64-byte LDS record
__device__ __forceinline__ int tw_swz(int ri) { return ((ri >> 1) ^ (ri >> 2)) & 3; }

// the tile's weight row tb (0..255): for SwiGLU wave column wn = tb / 128
// holds gate rows (fragments 0, 1) and the matching up rows (2, 3)
template <int EPI>
__device__ __forceinline__ int wide_wrow(int tb, int nt, int N) {
  if (EPI == QD_EPI_SWIGLU) {
    const int wn = tb >> 7, f = (tb >> 5) & 3, r = tb & 31;
    return (f < 2 ? 0 : (N >> 1)) + nt * 128 + wn * 64 + (f & 1) * 32 + r;
  }
  return nt * TW_N + tb;
}

// a wave's raw operands of one stage, A fragments fa0 .. fa0 + 3 and B
// fragments fb0 .. fb0 + 3: the codes of k-steps 0..3 with the scale dwords
// (read halfway through the previous stage) and the codes of k-steps 4..7
// (read at the start of the stage), so that only half a stage of codes is
// held twice
struct TwLo {
  uint4 a[4], b[4];
  uint32_t as[4], bs[4];
};
struct TwHi {
  uint4 a[4], b[4];
};

// LDS byte offset of lane (r, h)'s piece c (0, 1) of fragment f in a code area
__device__ __forceinline__ int tw_frag_off(int f, int lane, int c) {
  const int r = lane & 31, h = lane >> 5, ri = r & 15;
  return ((2 * f + (r >> 4)) * 64 + 4 * ri + ((2 * h + c) ^ tw_swz(ri))) * 16;
}

template <int MTV>
__device__ __forceinline__ void tw_read_lo(TwLo &R, const unsigned char *sl, const unsigned char *ascl,
                                           int s, int fa0, int fb0, int lane) {
  const int r = lane & 31, h = lane >> 5;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int fb = fb0 + j;
    R.b[j] = *reinterpret_cast<const uint4 *>(sl + TW_BCODE + tw_frag_off(fb, lane, 0));
    R.bs[j] = *reinterpret_cast<const uint32_t *>(sl + TW_BSCL + (2 * fb + (r >> 4)) * 128 +
                                                  (16 * h + (r & 15)) * 4);
  }
#pragma unroll
  for (int i = 0; i < MTV; ++i) {
    const int fa = fa0 + i;
    R.a[i] = *reinterpret_cast<const uint4 *>(sl + TW_ACODE + tw_frag_off(fa, lane, 0));
    R.as[i] = *reinterpret_cast<const uint32_t *>(ascl + (32 * fa + r) * 16 + (s & 1) * 8 + 4 * h);
  }
}

template <int MTV>
__device__ __forceinline__ void tw_read_hi(TwHi &R, const unsigned char *sl, int fa0, int fb0,
                                           int lane) {
#pragma unroll
  for (int j = 0; j < 4; ++j)
    R.b[j] = *reinterpret_cast<const uint4 *>(sl + TW_BCODE + tw_frag_off(fb0 + j, lane, 1));
#pragma unroll
  for (int i = 0; i < MTV; ++i)
    R.a[i] = *reinterpret_cast<const uint4 *>(sl + TW_ACODE + tw_frag_off(fa0 + i, lane, 1));
}

// k-steps 4c .. 4c + 3 of a stage from codes ca / cb and the scale dwords
template <int MTV>
__device__ __forceinline__ void tw_half(const uint4 (&ca)[4], const uint4 (&cb)[4],
                                        const uint32_t (&as)[4], const uint32_t (&bs)[4],
                                        f32x16 (&acc)[4][4], int c) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const bool hi = (q >> 1) != 0;
    f16x8 bf[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) bf[j] = decode8_sel(word_of(cb[j], q), scale_pair_of(bs[j], c), hi);
#pragma unroll
    for (int i = 0; i < MTV; ++i) {
      const f16x8 af = decode8_sel(word_of(ca[i], q), scale_pair_of(as[i], c), hi);
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mfma32(af, bf[j], acc[i][j]);
    }
  }
}

// Tiles of the persistent wide kernel: m-tile mt of the experts' TW_M-row
// tiles (M-tiles never straddle experts), weight-row tile nt.
struct TwTile {
  int e, row0, nrows, nt;
};

// The tile schedule in LDS: offs [E + 1] row offsets, mpre [E + 1] the
// m-tiles of the experts before e.  Tiles t = mt * ntn + nt; XCD x = b % 8
// owns the contiguous range [x * per, x * per + per) and its workgroups
// (b / 8) take every (G / 8)-th tile of it, so the tiles in flight on an XCD
// share an expert's weights or a block of activation rows in its L2.
// Tiles are visited in increasing order, so an expert cursor advances by a
// wave ballot over the next 64 experts.
__device__ __forceinline__ TwTile tw_locate(const int32_t *offs, const int32_t *mpre, int E,
                                            int ntn, int t, int &ecur, int lane) {
  const int mt = t / ntn;
  for (;;) {
    const int c = (int)uni((uint32_t)ecur) + 1 + lane;
    const bool le = c <= E && mpre[c] <= mt;
    const uint64_t bal = __ballot(le);
    const int adv = __popcll(bal);
    ecur += adv;
    if (adv < 64) break;
  }
  TwTile tl;
  tl.e = (int)uni((uint32_t)ecur);
  tl.row0 = (int)uni((uint32_t)(offs[tl.e] + (mt - mpre[tl.e]) * TW_M));
  tl.nrows = (int)uni((uint32_t)min(TW_M, offs[tl.e + 1] - tl.row0));
  tl.nt = (int)uni((uint32_t)(t - mt * ntn));
  return tl;
}

template <bool GATHER, int EPI>
__global__ __launch_bounds__(TW_THREADS, 1) void gemm_wide_kernel(GemmArgs p, int ntn) {
  extern __shared__ __align__(16) unsigned char lds[];
  __shared__ int sh_w[4];
  __shared__ float red[16];
  const int tid = threadIdx.x, lane = tid & 63, w = (int)uni((uint32_t)tid >> 6);
  const int K = p.K, N = p.N, E = p.E;
  const int64_t kb2 = K >> 1, kb16 = K >> 4;
  const int nst = K / TW_K;
  int32_t *offs = reinterpret_cast<int32_t *>(lds + TW_SCHED);
  int32_t *mpre = offs + (E + 1);
  int32_t *tokb = reinterpret_cast<int32_t *>(lds + TW_TOK);
  const uint32_t lds0 = (uint32_t)(uintptr_t)lds;
  const uint32_t tok0 = lds0 + (uint32_t)TW_TOK;

  // ---- the schedule: row offsets and m-tile prefix counts (four experts
  // per thread, E <= 1024)
  {
    int cnt[4], tsum = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * tid + q;
      int o0 = 0, o1 = 0;
      if (e <= E) {
        o0 = p.offsets ? p.offsets[e] : (e == 0 ? 0 : (int)p.rows);
        offs[e] = o0;
      }
      if (e < E) o1 = p.offsets ? p.offsets[e + 1] : (int)p.rows;
      cnt[q] = e < E ? (max(o1 - o0, 0) + TW_M - 1) / TW_M : 0;
      tsum += cnt[q];
    }
    int xs = tsum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(xs, o, 64);
      if (lane >= o) xs += y;
    }
    if (lane == 63) sh_w[w] = xs;
    __syncthreads();
    int base = xs - tsum;
    for (int ww = 0; ww < w; ++ww) base += sh_w[ww];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * tid + q;
      if (e <= E) mpre[e] = base;
      base += cnt[q];
    }
  }
  const float a_dec = p.a_gs[1];
  __syncthreads();
  const int T = (int)uni((uint32_t)mpre[E]) * ntn;
  const int G = gridDim.x, nsl = G >> 3, xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int per = (T + 7) >> 3;
  const int t_end = min(T, (xcd + 1) * per);
  int t = xcd * per + slot;
  int ecur = 0;
  float vmax = 0.0f;

  const int wm = w & 1, wn = w >> 1, fb0 = 4 * wn;
  const int ri = lane >> 2;
  const uint32_t pc = 16u * (uint32_t)((lane & 3) ^ tw_swz(ri));
  // per-lane load offsets of a tile: wave w loads A and B fragments 2w,
  // 2w + 1 (two 16-row halves each), lane l row l / 4 of the half, piece
  // (l % 4) ^ swz; B rows of one load are consecutive weight rows (one
  // per-lane offset, a uniform row per load); B scales (fragment-ordered):
  // load w & 1 covers tile row groups 8 (w & 1) .. + 7, lane l group
  // 8 (w & 1) + l / 8, piece l % 8 (waves 2, 3 repeat waves 0, 1: equal
  // bytes to equal places); A scales: rows 64 w + l, 16 bytes every second
  // stage
  struct Offs {
    uint32_t oa[4], obs, oag;
  };
  const uint32_t ob = (uint32_t)ri * (uint32_t)kb2 + pc;
  const int bg = 8 * (w & 1) + (lane >> 3);
  auto b_off = [&](const TwTile &tl) __attribute__((always_inline)) -> Offs {
    Offs o;
    o.obs = (uint32_t)((wide_wrow<EPI>(16 * bg, tl.nt, N) >> 4) * (K >> 8)) * 256u +
            16u * (uint32_t)(lane & 7);
    if (!GATHER) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = 32 * (2 * w + (j >> 1)) + 16 * (j & 1) + ri;
        o.oa[j] = (uint32_t)(tl.row0 + (r < tl.nrows ? r : 0)) * (uint32_t)kb2 + pc;
      }
      const int r = 64 * w + lane;
      o.oag = (uint32_t)(tl.row0 + (r < tl.nrows ? r : 0)) * (uint32_t)kb16;
    }
    return o;
  };
  // gathered rows: the tile's 256 row tokens go to LDS by direct loads
  // (wave w: rows 64 w + l; rows past the tile repeat its first row), so
  // neither the next tile's load offsets nor the residual rows wait on a
  // load the compiler tracks
  auto tok_dma = [&](const TwTile &tl, int buf) __attribute__((always_inline)) {
    const int r = 64 * w + lane;
    dma4s(uni_ptr(p.row_token), (uint32_t)(tl.row0 + (r < tl.nrows ? r : 0)) * 4u,
          uni(tok0 + buf * (TW_M * 4) + w * 256));
  };
  // the per-lane A offsets from the tokens in LDS buffer buf
  auto a_off_tok = [&](Offs &o, int buf) __attribute__((always_inline)) {
    const int32_t *tb = tokb + buf * TW_M;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      o.oa[j] = (uint32_t)tb[32 * (2 * w + (j >> 1)) + 16 * (j & 1) + ri] * (uint32_t)kb2 + pc;
    o.oag = (uint32_t)tb[64 * w + lane] * (uint32_t)kb16;
  };
  auto issue = [&](const TwTile &tl, const Offs &o, int s, int q, int apar)
                   __attribute__((always_inline)) {
    const uint32_t sb = uni(lds0 + q * TW_STAGE);
    const uint8_t *ac = uni_ptr(p.a_codes + s * 64);
    const uint8_t *bc = uni_ptr(p.w_codes + (int64_t)tl.e * N * kb2 + s * 64);
    const uint8_t *wsf = uni_ptr(p.w_sfrag + (int64_t)tl.e * N * kb16);
#pragma unroll
    for (int j = 0; j < 4; ++j) dma16s(ac, o.oa[j], sb + TW_ACODE + (4 * w + j) * 1024);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      dma16s(uni_ptr(bc + (int64_t)wide_wrow<EPI>(32 * (2 * w + (j >> 1)) + 16 * (j & 1), tl.nt, N) * kb2),
             ob, sb + TW_BCODE + (4 * w + j) * 1024);
    dma16s(uni_ptr(wsf + (s >> 1) * 256 + (s & 1) * 128), o.obs, sb + TW_BSCL + (w & 1) * 1024);
    if ((s & 1) == 0)
      dma16s(uni_ptr(p.a_scales + (s >> 1) * 16), o.oag,
             uni(lds0 + TW_ASCL + ((apar + (s >> 1)) & 1) * 4096 + w * 1024));
    else
      dma16s(uni_ptr(p.a_scales + (s >> 1) * 16), uni(o.oag), uni(lds0 + TW_DUMMY));
  };

  TwTile cur{};
  bool have = t < t_end;
  Offs oc{};
  int apar = 0;          // A-scale ring slot of the tile's first stage pair
  int tbuf = 0;          // token buffer of the current tile
  if (have) {
    cur = tw_locate(offs, mpre, E, ntn, t, ecur, lane);
    oc = b_off(cur);
    if (GATHER) {
      tok_dma(cur, 0);
      wait_vm<0>();
      __syncthreads();
      a_off_tok(oc, 0);
    }
    issue(cur, oc, 0, 0, apar);
    issue(cur, oc, 1, 1, apar);
  }
  while (have) {
    const int e = cur.e, nt = cur.nt, row0 = cur.row0, nrows = cur.nrows;
    const int tn = t + nsl;
    const bool hn = tn < t_end;
    TwTile nx{};
    if (hn) nx = tw_locate(offs, mpre, E, ntn, tn, ecur, lane);
    Offs on{};           // the next tile's load offsets (set in the last stages)
    const int apar_n = (apar + (nst >> 1)) & 1;
    const float sw = p.w_gs[2 * e + 1];
    const bool wide = nrows > 128;
    const int fa0 = wide ? 4 * wm : 2 * wm;
    const int mtv = wide ? min(max((nrows - 128 * wm + 31) >> 5, 0), 4)
                         : min(max((nrows - 64 * wm + 31) >> 5, 0), 2);
    auto a_src = [&](int s) __attribute__((always_inline)) -> const unsigned char * {
      return lds + TW_ASCL + ((apar + (s >> 1)) & 1) * 4096;
    };

    auto run = [&](auto mtv_c) __attribute__((always_inline)) {
      constexpr int MTV = decltype(mtv_c)::value;
      f32x16 acc[4][4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.0f;
      TwLo L0, L1;
      // stage 0 of this tile: issued during the previous tile (or above)
      wait_vm<TW_LOADS>();
      __syncthreads();
      // the next tile's tokens into the buffer the previous tile used (every
      // wave is past it now); landed by the first mid-stage wait
      if (GATHER && hn) tok_dma(nx, tbuf ^ 1);
      if constexpr (MTV > 0) tw_read_lo<MTV>(L0, lds, a_src(0), 0, fa0, fb0, lane);
      // one stage; TAIL: one of the last two, whose mid issues the next
      // tile's first stages instead of this tile's
      auto body = [&](const TwLo &Lc, TwLo &Ln, int s, auto tail_c) __attribute__((always_inline)) {
        constexpr bool TAIL = decltype(tail_c)::value;
        TwHi Hc;
        if constexpr (MTV > 0) {
          tw_read_hi<MTV>(Hc, lds + (s & 1) * TW_STAGE, fa0, fb0, lane);
          tw_half<MTV>(Lc.a, Lc.b, Lc.as, Lc.bs, acc, 0);
        }
        wait_vm<0>();
        __syncthreads();
        if constexpr (!TAIL) {
          issue(cur, oc, s + 2, s & 1, apar);
        } else if (hn) {
          if (s + 2 == nst) {
            on = b_off(nx);
            if (GATHER) a_off_tok(on, tbuf ^ 1);
          }
          issue(nx, on, s + 2 - nst, s & 1, apar_n);
        }
        if (!TAIL || s + 1 < nst) {
          if constexpr (MTV > 0)
            tw_read_lo<MTV>(Ln, lds + ((s + 1) & 1) * TW_STAGE, a_src(s + 1), s + 1, fa0, fb0, lane);
        }
        if constexpr (MTV > 0) tw_half<MTV>(Hc.a, Hc.b, Lc.as, Lc.bs, acc, 1);
      };
      for (int s = 0; s < nst - 2; s += 2) {     // nst is even
        body(L0, L1, s, std::false_type{});
        body(L1, L0, s + 1, std::false_type{});
      }
      body(L0, L1, nst - 2, std::true_type{});
      body(L1, L0, nst - 1, std::true_type{});
      // ---- epilogue: tensor scales, SwiGLU (gate fragments 0, 1 with up
      // fragments 2, 3) or plain, bf16 pairs of adjacent columns swapped
      // between neighbouring lanes so that every store writes 4 bytes
      const int h = lane >> 5;
      const bool odd = (lane & 1) != 0;
      const int cpair = (lane & 31) & ~1;
      constexpr int NO = EPI == QD_EPI_SWIGLU ? 2 : 4;
      const int ldo = EPI == QD_EPI_SWIGLU ? (N >> 1) : N;
      const bool full = nrows == TW_M;
      unsigned char *obase = reinterpret_cast<unsigned char *>(p.out);
      const float alpha = a_dec * sw;
#pragma unroll
      for (int i = 0; i < MTV; ++i) {
        const int rl = 32 * (fa0 + i) + 4 * h + (odd ? 1 : 0);
#pragma unroll
        for (int jj = 0; jj < NO; ++jj) {
          const int cb = EPI == QD_EPI_SWIGLU ? nt * 128 + wn * 64 + 32 * jj
                                              : nt * TW_N + 32 * (fb0 + jj);
          const uint32_t voff = (uint32_t)((row0 + rl) * ldo + cb + cpair) * 2u;
          float v[16];
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            if (EPI == QD_EPI_SWIGLU)
              v[q] = swiglu_fast(alpha * acc[i][jj][q], alpha * acc[i][jj + 2][q]);
            else
              v[q] = alpha * acc[i][jj][q];
          }
#pragma unroll
          for (int q = 0; q < 16; q += 2) {
            const float send = odd ? v[q] : v[q + 1];
            const float x = __int_as_float(
                __builtin_amdgcn_mov_dpp(__float_as_int(send), 0xB1, 0xF, 0xF, false));
            const f32x2_t pr = odd ? f32x2_t{x, v[q + 1]} : f32x2_t{v[q], x};
            const uint32_t pk = __builtin_bit_cast(uint32_t, __builtin_convertvector(pr, bf16x2_t));
            const int qr = 8 * (q >> 2) + (q & 3);
            if (full || rl + qr < nrows) {
              *reinterpret_cast<uint32_t *>(obase + (size_t)(qr * ldo * 2) + voff) = pk;
              vmax = fmaxf(vmax, fmaxf(fabsf(__uint_as_float(pk << 16)),
                                       fabsf(__uint_as_float(pk & 0xFFFF0000u))));
            }
          }
        }
      }
    };
    switch (mtv) {
      case 4: run(std::integral_constant<int, 4>{}); break;
      case 3: run(std::integral_constant<int, 3>{}); break;
      case 2: run(std::integral_constant<int, 2>{}); break;
      case 1: run(std::integral_constant<int, 1>{}); break;
      default: run(std::integral_constant<int, 0>{}); break;
    }
    t = tn;
    have = hn;
    cur = nx;
    oc = on;
    apar = apar_n;
    tbuf ^= 1;
  }
  wait_vm<0>();
  const float m = block_max(vmax, red);
  put_amax(p, m);
}

// host-side plan of the decode kernel
struct SkPlan {
  bool ok;
  int nblk, grid;
  size_t lds;
};

inline int64_t skinny_nblk(int64_t N, int epilogue) {
  return epilogue == QD_EPI_SWIGLU ? ((N / 2) + SK_ROWS / 2 - 1) / (SK_ROWS / 2)
                                   : (N + SK_ROWS - 1) / SK_ROWS;
}

// Decode-sized problems: few rows per expert and whole 256-element
// iterations.
// bm: the residual in bitmap mode (K <= SK_BM_KMAX).
inline SkPlan skinny_plan(int64_t rows, int E, int64_t N, int64_t K, int Ks, int epilogue,
                          bool bm = false) {
  SkPlan pl{};
  const bool rac = Ks > 0;
  if (K < 256 || K % 256 != 0 || K > SK_KMAX || E > SK_EMAX || rows > (int64_t)E * 48) return pl;
  if (bm && (!rac || K > SK_BM_KMAX)) return pl;
  const int64_t nblk = skinny_nblk(N, epilogue);
  pl.nblk = (int)nblk;
  pl.grid = (int)std::min<int64_t>(SK_GRID, (int64_t)E * nblk * 4);
  pl.lds = (size_t)sk_layout((int)K, E, rac, bm).total;
  if (pl.lds > (size_t)SK_LDS_MAX) return pl;
  pl.ok = true;
  return pl;
}

inline int64_t grid_x(int64_t rows, int E, bool grouped) {
  return (rows + BM - 1) / BM + (grouped ? E : 0);
}
inline int64_t grid_y(int64_t N, int epilogue) {
  return epilogue == QD_EPI_SWIGLU ? ((N / 2) + 31) / 32 : (N + BN - 1) / BN;
}

template <bool GATHER, bool RAC, int EPI>
void launch_skinny(const GemmArgs &p, const SkPlan &pl, hipStream_t s) {
  auto kern = gemm_skinny_kernel<GATHER, RAC, EPI>;
  static const bool attr = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               SK_LDS_MAX) == hipSuccess;
  (void)attr;
  hipLaunchKernelGGL(kern, dim3((unsigned)pl.grid), dim3(SK_THREADS), pl.lds, s, p, pl.nblk);
}

// host-side plan of the prefill kernel
struct TlPlan {
  bool ok;
  bool dense;   // RAC as a second pass over K on the masked residual
  int ntn, grid, lds, grp;
};

// rac: the residual is fused, in its compact form (rq_sel) while the compact
// weight table leaves LDS for two workgroups per CU, else as the dense second
// pass over the masked residual (faster than the table at one workgroup per
// CU); compact_only: the table wherever it fits at all
inline TlPlan tile_plan(int64_t rows, int E, int64_t N, int64_t K, bool rac, int Ks,
                        bool compact_only = false) {
  TlPlan pl{};
  if (K < 4 * TL_K || K % (2 * TL_K) != 0 || N % TL_N != 0 || E > TL_EMAX) return pl;
  // byte offsets inside one activation matrix or one expert's weights, and
  // output offsets, fit 32 bits
  if (N * K / 2 >= (1LL << 32) || (rows + 1) * K / 2 >= (1LL << 32)) return pl;
  if ((rows + TL_M) * N * 2 >= (1LL << 32)) return pl;
  bool cmp = rac;
  int ksa = rac ? (Ks + 15) / 16 * 16 : 0;
  if (rac && !compact_only && tl_lds_bytes(true, ksa, false) > TL_LDS_2WG) {
    pl.dense = true;
    cmp = false;
    ksa = 0;
  }
  pl.lds = tl_lds_bytes(cmp, ksa, false);
  if (pl.lds > TL_LDS_MAX) return pl;
  // the A-scale ring where it keeps the workgroups per CU (groups of four
  // stages: K a multiple of 256, so no group reads past a row's scales)
  const int lg = tl_lds_bytes(cmp, ksa, true) + TL_AGRP;
  if (K % 256 == 0 && ((pl.lds <= TL_LDS_2WG && lg <= TL_LDS_2WG) ||
                       (pl.lds > TL_LDS_2WG && lg <= TL_LDS_MAX))) {
    pl.lds = lg;
    pl.grp = 1;
  }
  pl.ntn = (int)(N / TL_N);
  const int64_t g = qdt::tile_grid(rows, E, TL_M, pl.ntn);
  if (g > 0x7fffffffLL) return pl;
  pl.grid = (int)g;
  pl.ok = true;
  return pl;
}

template <bool GATHER, bool RAC, int EPI, bool DENSE = false>
void launch_tile(const GemmArgs &p, const TlPlan &pl, hipStream_t s) {
  auto kern = gemm_tile_kernel<GATHER, RAC, EPI, DENSE>;
  static const bool attr = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               TL_LDS_MAX) == hipSuccess;
  (void)attr;
  hipLaunchKernelGGL(kern, dim3((unsigned)pl.grid), dim3(TL_THREADS), (size_t)pl.lds, s, p, pl.ntn,
                     pl.grp);
}

// host-side plan of the wide prefill kernel (needs the weights'
// fragment-ordered scales)
struct WdPlan {
  bool ok;
  int ntn, grid, lds;
};

inline WdPlan wide_plan(int64_t rows, int E, int64_t N, int64_t K, bool rac, int Ks, bool sfrag) {
  WdPlan pl{};
  (void)Ks;
  if (rac || !sfrag || K < 2 * TW_K || K % (2 * TW_K) != 0 || N % TW_N != 0 || E > TL_EMAX)
    return pl;
  if (N * K / 2 >= (1LL << 32) || (rows + 1) * K / 2 >= (1LL << 32)) return pl;
  if ((rows + TW_M) * N * 2 >= (1LL << 32)) return pl;
  pl.lds = tw_lds_bytes(E);
  if (pl.lds > TL_LDS_MAX) return pl;
  pl.ntn = (int)(N / TW_N);
  // persistent: one workgroup per CU (256 on MI355X), a multiple of 8 (the
  // XCDs), at most the tile count's upper bound
  const int64_t g = qdt::tile_grid(rows, E, TW_M, pl.ntn);
  pl.grid = (int)std::min<int64_t>(256, g);
  pl.ok = true;
  return pl;
}

template <bool GATHER, int EPI>
void launch_wide(const GemmArgs &p, const WdPlan &pl, hipStream_t s) {
  auto kern = gemm_wide_kernel<GATHER, EPI>;
  static const bool attr = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               TL_LDS_MAX) == hipSuccess;
  (void)attr;
  hipLaunchKernelGGL(kern, dim3((unsigned)pl.grid), dim3(TW_THREADS), (size_t)pl.lds, s, p, pl.ntn);
}

template <bool GATHER, bool RAC>
void launch_epi(const GemmArgs &p, int epi, dim3 grid, hipStream_t s, const SkPlan &pl,
                const TlPlan &tp, const WdPlan &wp) {
  if (pl.ok) {
    if (epi == QD_EPI_SWIGLU) launch_skinny<GATHER, RAC, QD_EPI_SWIGLU>(p, pl, s);
    else launch_skinny<GATHER, RAC, QD_EPI_NONE>(p, pl, s);
    return;
  }
  if constexpr (!RAC) {
    if (wp.ok) {
      if (epi == QD_EPI_SWIGLU) launch_wide<GATHER, QD_EPI_SWIGLU>(p, wp, s);
      else launch_wide<GATHER, QD_EPI_NONE>(p, wp, s);
      return;
    }
  }
  if (tp.ok) {
    if constexpr (RAC) {
      if (tp.dense) {
        if (epi == QD_EPI_SWIGLU) launch_tile<GATHER, true, QD_EPI_SWIGLU, true>(p, tp, s);
        else launch_tile<GATHER, true, QD_EPI_NONE, true>(p, tp, s);
        return;
      }
    }
    if (epi == QD_EPI_SWIGLU) launch_tile<GATHER, RAC, QD_EPI_SWIGLU>(p, tp, s);
    else launch_tile<GATHER, RAC, QD_EPI_NONE>(p, tp, s);
    return;
  }
  if (epi == QD_EPI_SWIGLU)
    hipLaunchKernelGGL((gemm_w4a4_kernel<GATHER, RAC, QD_EPI_SWIGLU>), grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((gemm_w4a4_kernel<GATHER, RAC, QD_EPI_NONE>), grid, dim3(256), 0, s, p);
}

}  // namespace

bool qdi::gemm_wants_rq_sel(int64_t rows, int32_t E, int64_t N, int64_t K, int32_t Ks,
                            int32_t epilogue) {
  if (Ks <= 0 || rows <= 0 || E < 1 || N <= 0 || K <= 0) return false;
  if (skinny_plan(rows, E, N, K, Ks, epilogue).ok) return false;
  const TlPlan tp = tile_plan(rows, E, N, K, true, Ks);
  return tp.ok && !tp.dense;
}

int64_t qdi::gemm_amax_written(int64_t rows, int32_t E, int64_t N, int64_t K, int32_t Ks,
                               int32_t epilogue, bool sfrag, bool bitmap) {
  if (rows <= 0 || E < 1 || N <= 0 || K <= 0 || Ks < 0) return 0;
  // the kernel choice of the grouped GEMM (launch_epi) and its grid
  const bool rac = Ks > 0;
  const SkPlan pl = skinny_plan(rows, E, N, K, Ks, epilogue, bitmap);
  if (pl.ok) return pl.grid;
  if (!rac) {
    const WdPlan wp = wide_plan(rows, E, N, K, false, Ks, sfrag);
    if (wp.ok) return wp.grid;
  }
  const TlPlan tp = tile_plan(rows, E, N, K, rac, Ks);
  if (tp.ok) return tp.grid;
  return grid_x(rows, E, true) * grid_y(N, epilogue);
}

bool qdi::gemm_takes_bitmap(int64_t rows, int32_t E, int64_t N, int64_t K, int32_t Ks,
                            int32_t epilogue) {
  if (Ks <= 0 || rows <= 0 || E < 1 || N <= 0 || K <= 0) return false;
  return skinny_plan(rows, E, N, K, Ks, epilogue, true).ok;
}

extern "C" int32_t moe_w4a4_grouped_gemm_residual_form(int64_t rows, int64_t N, int64_t K,
                                                       int32_t E, int32_t Ks, int32_t epilogue) {
  if (Ks <= 0 || rows <= 0 || E < 1 || N <= 0 || K <= 0) return 0;
  return qdi::gemm_wants_rq_sel(rows, E, N, K, Ks, epilogue) ? 2 : 1;
}

extern "C" int64_t moe_w4a4_grouped_gemm_amax_count(int64_t rows, int64_t N, int64_t K,
                                                    int32_t E, int32_t Ks, int32_t epilogue) {
  if (rows < 0 || N <= 0 || K <= 0 || E < 1 || Ks < 0) return 0;
  const SkPlan pl = skinny_plan(rows, E, N, K, Ks, epilogue);
  if (pl.ok) return pl.grid;
  // whichever of the other kernels runs (the wide one needs the weights'
  // fragment-ordered scales) writes every entry of the largest grid
  const WdPlan wp = wide_plan(rows, E, N, K, Ks > 0, Ks, true);
  const TlPlan tp = tile_plan(rows, E, N, K, Ks > 0, Ks);
  return std::max<int64_t>(std::max<int64_t>(wp.ok ? wp.grid : 0, tp.ok ? tp.grid : 0),
                           grid_x(rows, E, true) * grid_y(N, epilogue));
}

extern "C" int64_t moe_w4a4_grouped_gemm_per_expert_amax_count(int64_t rows, int64_t N,
                                                               int64_t K, int32_t E, int32_t Ks,
                                                               int32_t epilogue) {
  (void)epilogue;
  if (rows < 0 || N <= 0 || K <= 0 || E < 1 || Ks < 1) return 0;
  const TlPlan tp = tile_plan(rows, E, N, K, true, Ks, true);
  return tp.ok ? tp.grid : 0;
}

// Fragment-ordered weight scales: one thread per output dword, i.e. per
// (group e, 16-row fragment f, 256-column chunk c, lane l = 16 g + r); the
// dword holds the scales of row 16 f + r, blocks 16 c + 4 g .. 16 c + 4 g + 3.
__global__ __launch_bounds__(256) void pack_frag_scales_kernel(const uint8_t *__restrict__ sc,
                                                               int64_t rows, int64_t cols,
                                                               int64_t ndw,
                                                               uint32_t *__restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= ndw) return;
  const int l = (int)(i & 63);
  const int64_t rec = i >> 6;
  const int64_t nc = cols >> 8, nf = rows >> 4;
  const int64_t c = rec % nc, f = (rec / nc) % nf, e = rec / (nc * nf);
  const int64_t row = e * rows + 16 * f + (l & 15);
  out[i] = *reinterpret_cast<const uint32_t *>(sc + row * (cols >> 4) + 16 * c + 4 * (l >> 4));
}

extern "C" int64_t nvfp4_frag_scales_bytes(int64_t groups, int64_t rows, int64_t cols) {
  if (groups < 1 || rows < 0 || cols <= 0 || rows % 16 != 0 || cols % 256 != 0) return 0;
  return groups * rows * (cols / 16);
}

extern "C" qd_status nvfp4_pack_frag_scales(const qd_nvfp4 *w, uint8_t *out, void *stream) {
  if (!w || !out) return QD_ERR_NULL;
  qd_status st = qdh::check_nvfp4(w, w->groups, w->rows, w->cols);
  if (st) return st;
  if (w->rows % 16 != 0 || w->cols % 256 != 0) return QD_ERR_SHAPE;
  if (!qdh::aligned16(out)) return QD_ERR_ALIGN;
  if (qdh::fault_injected()) return QD_ERR_HIP;
  const int64_t ndw = w->groups * w->rows * (w->cols / 16) / 4;
  if (ndw == 0) return QD_OK;
  if ((ndw + 255) / 256 > 0x7fffffffLL) return QD_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(pack_frag_scales_kernel, dim3((unsigned)((ndw + 255) / 256)), dim3(256), 0,
                     qdh::S(stream), w->scales, w->rows, w->cols, ndw,
                     reinterpret_cast<uint32_t *>(out));
  return qdh::check_launch();
}

namespace {

// The grouped GEMM behind moe_w4a4_grouped_gemm and the layer's bitmap
// mode (bitmap != NULL: bitmap [K / 32] marks S, sel_idx is written with S;
// decode-shaped problems with K <= 4096 only).
qd_status grouped_gemm_impl(const qd_nvfp4 *a, const int32_t *row_token,
                            const int32_t *expert_offsets, int32_t E, int64_t rows,
                            const qd_nvfp4 *w, const qd_nvfp4 *rq, const int32_t *sel_idx,
                            int32_t Ks, const void *rq_sel, const uint32_t *bitmap,
                            int32_t epilogue, void *out, float *amax_partials, void *stream,
                            bool per_expert = false, const uint8_t *a_stg = nullptr) {
  if (!a || !w || !out) return QD_ERR_NULL;
  if (epilogue != QD_EPI_NONE && epilogue != QD_EPI_SWIGLU) return QD_ERR_DTYPE;
  if (E < 1 || rows < 0) return QD_ERR_SHAPE;
  const int64_t K = a->cols;
  qd_status st = qdh::check_nvfp4(a, 1, a->rows, K);
  if (st) return st;
  st = qdh::check_nvfp4(w, E, w->rows, K);
  if (st) return st;
  const int64_t N = w->rows;
  if (K % 16 != 0 || N % 16 != 0 || N <= 0) return QD_ERR_SHAPE;
  if (epilogue == QD_EPI_SWIGLU && (N % 32 != 0)) return QD_ERR_SHAPE;
  if (!expert_offsets && E != 1) return QD_ERR_SHAPE;
  if (!row_token && rows > a->rows) return QD_ERR_SHAPE;
  if (Ks > 0 && !rq) return QD_ERR_NULL;
  const bool rac = rq != nullptr && Ks > 0;
  if (rac) {
    st = qdh::check_nvfp4(rq, 1, rq->rows, K);
    if (st) return st;
    if (!sel_idx) return QD_ERR_NULL;
    if (Ks > K || rq->rows != a->rows) return QD_ERR_SHAPE;
    if (K > 65536) return QD_ERR_UNSUPPORTED;
  }
  if (bitmap && !rac) return QD_ERR_SHAPE;
  if (Ks < 0) return QD_ERR_SHAPE;
  if (!qdh::aligned16(out) || (amax_partials && ((uintptr_t)amax_partials & 3u)))
    return QD_ERR_ALIGN;
  if (w->scales_frag && !qdh::aligned16(w->scales_frag)) return QD_ERR_ALIGN;
  if (N > 0x7fffffff || K > 0x7fffffff) return QD_ERR_UNSUPPORTED;
  const int64_t gx = grid_x(rows, E, true), gy = grid_y(N, epilogue);
  if (gx > 0x7fffffffLL || gy > 65535) return QD_ERR_UNSUPPORTED;
  // per-expert channel sets run on the tile kernel alone
  const SkPlan pl = per_expert ? SkPlan{} : skinny_plan(rows, E, N, K, rac ? Ks : 0, epilogue, bitmap != nullptr);
  if (bitmap && !pl.ok) return QD_ERR_UNSUPPORTED;
  if (per_expert) {
    // per-expert sets take the compact residual (one per grouped row)
    const TlPlan pp = tile_plan(rows, E, N, K, true, Ks, true);
    if (!rac || !rq_sel || !pp.ok)
      return rac && rq_sel ? QD_ERR_UNSUPPORTED : QD_ERR_NULL;
  }
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
  p.w_sfrag = w->scales_frag;
  p.w_gs = w->gscale;
  p.N = (int)N;
  p.K = (int)K;
  if (rac) {
    p.r_codes = rq->codes;
    p.r_scales = rq->scales;
    p.r_gs = rq->gscale;
    p.sel = sel_idx;
    p.Ks = Ks;
    p.r_sel = static_cast<const uint16_t *>(rq_sel);
    p.ksa = (Ks + 15) / 16 * 16;
    p.sel_stride = per_expert ? Ks : 0;
    p.rsel_rows = per_expert ? 1 : 0;
    if (bitmap) {
      p.r_bitmap = bitmap;
      p.sel_out = const_cast<int32_t *>(sel_idx);
    }
  }
  p.out = static_cast<uint16_t *>(out);
  p.a_stg = row_token && !per_expert ? a_stg : nullptr;
  p.amax_part = amax_partials;
  p.amax_n = !amax_partials ? 0
             : per_expert ? moe_w4a4_grouped_gemm_per_expert_amax_count(rows, N, K, E, Ks, epilogue)
                          : moe_w4a4_grouped_gemm_amax_count(rows, N, K, E, rac ? Ks : 0, epilogue);
  const TlPlan tp = tile_plan(rows, E, N, K, rac, Ks, per_expert);
  const WdPlan wp = wide_plan(rows, E, N, K, rac, Ks, w->scales_frag != nullptr);
  // the tile kernel takes the residual in its compact form unless its plan
  // is the dense second pass (which reads the masked residual rq)
  if (rac && !pl.ok && tp.ok && !tp.dense && (!rq_sel || !qdh::aligned16(rq_sel)))
    return rq_sel ? QD_ERR_ALIGN : QD_ERR_NULL;
  dim3 grid((unsigned)gx, (unsigned)gy);
  hipStream_t s = qdh::S(stream);
  if (row_token) {
    if (rac) launch_epi<true, true>(p, epilogue, grid, s, pl, tp, wp);
    else launch_epi<true, false>(p, epilogue, grid, s, pl, tp, wp);
  } else {
    if (rac) launch_epi<false, true>(p, epilogue, grid, s, pl, tp, wp);
    else launch_epi<false, false>(p, epilogue, grid, s, pl, tp, wp);
  }
  return qdh::check_launch();
}

}  // namespace

extern "C" qd_status moe_w4a4_grouped_gemm_per_expert(
    const qd_nvfp4 *a, const int32_t *row_token, const int32_t *expert_offsets, int32_t E,
    int64_t rows, const qd_nvfp4 *w, const qd_nvfp4 *rq, const int32_t *sel_pe, int32_t Ks,
    const void *rq_sel_rows, int32_t epilogue, void *out, float *amax_partials, void *stream) {
  if (Ks < 1) return QD_ERR_SHAPE;
  if (!sel_pe || !rq || !rq_sel_rows || !expert_offsets) return QD_ERR_NULL;
  return grouped_gemm_impl(a, row_token, expert_offsets, E, rows, w, rq, sel_pe, Ks, rq_sel_rows,
                           nullptr, epilogue, out, amax_partials, stream, true);
}

extern "C" qd_status moe_w4a4_grouped_gemm(const qd_nvfp4 *a, const int32_t *row_token,
                                           const int32_t *expert_offsets, int32_t E, int64_t rows,
                                           const qd_nvfp4 *w, const qd_nvfp4 *rq,
                                           const int32_t *sel_idx, int32_t Ks, const void *rq_sel,
                                           int32_t epilogue, void *out, float *amax_partials,
                                           void *stream) {
  return grouped_gemm_impl(a, row_token, expert_offsets, E, rows, w, rq, sel_idx, Ks, rq_sel,
                           nullptr, epilogue, out, amax_partials, stream);
}

// Staging costs rows x K x 9/16 bytes written and read once, and saves time in
// proportion to N (the n-tiles that re-read each stage): measured at N = 3072,
// K = 4096 the tile GEMM gains 2.5x the copy's time, at N = 1536, K = 2048
// 0.8x, so it is taken from N = 2048 on.
constexpr int64_t kStageMinN = 2048;

int64_t qdi::gemm_stage_bytes(int64_t rows, int32_t E, int64_t N, int64_t K, int32_t Ks,
                              int32_t epilogue) {
  if (Ks <= 0 || rows <= 0 || E < 1 || N < kStageMinN || K <= 0) return 0;
  if (skinny_plan(rows, E, N, K, Ks, epilogue).ok) return 0;
  const TlPlan tp = tile_plan(rows, E, N, K, true, Ks);
  if (!tp.ok || !tp.grp) return 0;
  return rows * (K / 2 + K / 16);
}

int64_t qdi::gemm_stage_reserve(int64_t rows, int32_t E, int64_t N, int64_t K, int32_t epilogue) {
  if (rows <= 0 || E < 1 || N < kStageMinN || K <= 0 || K % 256 != 0) return 0;
  if (skinny_plan(rows, E, N, K, 1, epilogue).ok) return 0;
  return tile_plan(rows, E, N, K, true, 1).ok ? rows * (K / 2 + K / 16) : 0;
}

qd_status qdi::grouped_gemm_staged(const qd_nvfp4 *a, const int32_t *row_token,
                                   const int32_t *expert_offsets, int32_t E, int64_t rows,
                                   const qd_nvfp4 *w, const qd_nvfp4 *rq, const int32_t *sel_idx,
                                   int32_t Ks, const void *rq_sel, int32_t epilogue, void *out,
                                   float *amax_partials, const uint8_t *a_stg, hipStream_t stream) {
  if (!a_stg || !row_token) return QD_ERR_NULL;
  if (!qdh::aligned16(a_stg)) return QD_ERR_ALIGN;
  return grouped_gemm_impl(a, row_token, expert_offsets, E, rows, w, rq, sel_idx, Ks, rq_sel,
                           nullptr, epilogue, out, amax_partials, stream, false, a_stg);
}

qd_status qdi::grouped_gemm_bitmap(const qd_nvfp4 *a, const int32_t *row_token,
                                   const int32_t *expert_offsets, int32_t E, int64_t rows,
                                   const qd_nvfp4 *w, const qd_nvfp4 *rq, const uint32_t *bitmap,
                                   int32_t Ks, int32_t *sel_out, int32_t epilogue, void *out,
                                   float *amax_partials, hipStream_t stream) {
  if (!bitmap) return QD_ERR_NULL;
  return grouped_gemm_impl(a, row_token, expert_offsets, E, rows, w, rq, sel_out, Ks, nullptr,
                           bitmap, epilogue, out, amax_partials, stream);
}

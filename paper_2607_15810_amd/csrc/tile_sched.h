// Tile scheduling shared by the grouped GEMM kernels that tile rows per
// expert: M-tiles never straddle experts, the grid is an upper bound on the
// tile count, and tile indices run contiguously within an XCD (workgroups
// are dealt to the eight XCDs in turn), so the tiles in flight on an XCD
// share an expert's weights or a block of activation rows in its L2.
#pragma once
#include "common.h"
#include "lds_dma.h"

namespace qdt {

struct Tile {
  int e;       // expert, -1 if this workgroup has no tile
  int row0;    // first grouped row of the tile
  int nrows;   // rows in the tile (<= TM)
  int nt;      // weight-row tile index
};

// Every thread of a workgroup of NW waves (NW * 64 threads, NW = 4 or 8)
// calls this; experts E <= 1024 (the first 256 threads hold four each).
// offsets: expert row offsets [E + 1] (NULL: one expert with `rows` rows).
// sh_w: NW ints, sh_t: 4 ints of LDS scratch.
template <int TM, int NW = 4>
__device__ __forceinline__ Tile find_tile(const int32_t *__restrict__ offsets, int E, int64_t rows,
                                          int ntn, int *sh_w, int *sh_t) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // M-tiles per expert (exclusive scan, four experts per thread)
  int cnt[4], tsum = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = 4 * tid + q;
    int c = 0;
    if (offsets) c = e < E ? offsets[e + 1] - offsets[e] : 0;
    else c = e == 0 ? (int)rows : 0;
    cnt[q] = (max(c, 0) + TM - 1) / TM;
    tsum += cnt[q];
  }
  int xs = tsum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(xs, o, 64);
    if (lane >= o) xs += y;
  }
  if (lane == 63) sh_w[w] = xs;
  if (tid == 0) sh_t[0] = -1;
  __syncthreads();
  int mt_total = 0;
#pragma unroll
  for (int ww = 0; ww < NW; ++ww) mt_total += sh_w[ww];
  // XCD x = b % 8 takes tiles x * per .. x * per + per - 1
  const int b = blockIdx.x;
  const int ntile = mt_total * ntn;
  const int per = (ntile + 7) >> 3;
  const int slot = b >> 3;
  const int L = (b & 7) * per + slot;
  const bool live = slot < per && L < ntile;
  const int mt = live ? L / ntn : -1, nt = live ? L - (L / ntn) * ntn : 0;
  {
    int base = xs - tsum;
    for (int ww = 0; ww < w; ++ww) base += sh_w[ww];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (mt >= base && mt < base + cnt[q]) {
        const int e = 4 * tid + q;
        const int o0 = offsets ? offsets[e] : 0;
        const int o1 = offsets ? offsets[e + 1] : (int)rows;
        const int r0 = o0 + (mt - base) * TM;
        sh_t[0] = e;
        sh_t[1] = r0;
        sh_t[2] = min(TM, o1 - r0);
      }
      base += cnt[q];
    }
  }
  __syncthreads();
  Tile t;
  t.e = (int)qdl::uni((uint32_t)sh_t[0]);
  t.row0 = (int)qdl::uni((uint32_t)sh_t[1]);
  t.nrows = (int)qdl::uni((uint32_t)sh_t[2]);
  t.nt = (int)qdl::uni((uint32_t)nt);
  return t;
}

// upper bound on the tiles of `rows` grouped rows over E experts, rounded
// up to whole XCD rounds
inline int64_t tile_grid(int64_t rows, int E, int TM, int ntn) {
  int64_t g = ((rows + TM - 1) / TM + E) * ntn;
  return (g + 7) / 8 * 8;
}

}  // namespace qdt

// Achievable-peak probes, so measured rates can be stated against what the
// chip reaches in practice beside its published peaks: a streaming read of
// device memory (the HBM bound of the decode GEMMs) and a register-only loop
// of independent f16 MFMAs (the compute bound of the prefill GEMMs, whose
// exact NVFP4 operands are f16).  Neither is part of the layer.
#include "common.h"

namespace {

constexpr int kReadThreads = 256;
constexpr int kReadUnroll = 4;

// Every lane reads 16-byte pieces with kReadUnroll loads in flight and folds
// them into one word, so no load can be dropped; one word per workgroup is
// written.
__global__ __launch_bounds__(kReadThreads) void stream_read_kernel(const uint4 *__restrict__ p,
                                                                   int64_t n16,
                                                                   uint32_t *__restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * kReadThreads;
  int64_t i = (int64_t)blockIdx.x * kReadThreads + threadIdx.x;
  uint32_t acc = 0u;
  for (; i + (kReadUnroll - 1) * stride < n16; i += kReadUnroll * stride) {
    uint4 v[kReadUnroll];
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) v[u] = p[i + u * stride];
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const uint4 v = p[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  __shared__ uint32_t red[kReadThreads / 64];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

typedef float f32x16_t __attribute__((ext_vector_type(16)));

// A finite f16 bit pattern with random sign and mantissa and an exponent in
// [2^-4, 2^3] from a 32-bit integer hash.
__device__ __forceinline__ uint16_t random_f16_bits(uint32_t x) {
  x ^= x >> 16; x *= 0x7FEB352Du; x ^= x >> 15; x *= 0x846CA68Bu; x ^= x >> 16;
  return (uint16_t)((x & 0x83FFu) | ((11u + ((x >> 10) & 7u)) << 10));
}

// 16 independent accumulators per wave, each updated once per round by
// v_mfma_f32_32x32x16_f16 on register operands (slowly varying values, or
// random ones).
__global__ __launch_bounds__(256) void mfma_loop_kernel(int64_t rounds, float seed, int rnd,
                                                        float *__restrict__ out) {
  f16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    if (rnd) {
      const uint32_t id = (blockIdx.x * 256u + threadIdx.x) * 16u + i;
      a[i] = __builtin_bit_cast(_Float16, random_f16_bits(id));
      b[i] = __builtin_bit_cast(_Float16, random_f16_bits(id + 8u));
    } else {
      a[i] = (_Float16)(seed * (float)(threadIdx.x + i));
      b[i] = (_Float16)(seed * (float)i);
    }
  }
  f32x16_t acc[16];
#pragma unroll
  for (int j = 0; j < 16; ++j)
#pragma unroll
    for (int t = 0; t < 16; ++t) acc[j][t] = 0.0f;
  for (int64_t r = 0; r < rounds; ++r) {
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc[j], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < 16; ++j)
#pragma unroll
    for (int t = 0; t < 16; ++t) s += acc[j][t];
  if (threadIdx.x == 0) out[blockIdx.x] = s;
}

}  // namespace

extern "C" int64_t qd_probe_hbm_read_out_count(void) { return 4096; }

extern "C" qd_status qd_probe_hbm_read(const void *buf, int64_t bytes, uint32_t *out,
                                       void *stream) {
  if (!buf || !out) return QD_ERR_NULL;
  if (bytes <= 0 || bytes % 16 != 0) return QD_ERR_SHAPE;
  if (!qdh::aligned16(buf)) return QD_ERR_ALIGN;
  hipLaunchKernelGGL(stream_read_kernel, dim3(4096), dim3(kReadThreads), 0, qdh::S(stream),
                     static_cast<const uint4 *>(buf), bytes / 16, out);
  return qdh::check_launch();
}

extern "C" double qd_probe_mfma_f16_flops(int64_t rounds, int32_t workgroups) {
  return (double)workgroups * 4.0 * (double)rounds * 16.0 * 32.0 * 32.0 * 16.0 * 2.0;
}

extern "C" qd_status qd_probe_mfma_f16(int64_t rounds, int32_t workgroups,
                                       int32_t random_operands, float *out, void *stream) {
  if (!out) return QD_ERR_NULL;
  if (rounds < 1 || workgroups < 1) return QD_ERR_SHAPE;
  hipLaunchKernelGGL(mfma_loop_kernel, dim3((unsigned)workgroups), dim3(256), 0, qdh::S(stream),
                     rounds, 1e-3f, random_operands ? 1 : 0, out);
  return qdh::check_launch();
}

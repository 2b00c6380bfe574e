// Host-side plumbing shared by every entry point: status strings, argument
// checks, launch checks, and a small max-reduction kernel.
#include <cstdlib>
#include <cstring>

#include "common.h"

extern "C" const char *qd_status_string(qd_status s) {
  switch (s) {
    case QD_OK: return "ok";
    case QD_ERR_NULL: return "a required pointer is NULL";
    case QD_ERR_SHAPE: return "invalid or inconsistent shape";
    case QD_ERR_ALIGN: return "device pointer not 16-byte aligned";
    case QD_ERR_DTYPE: return "unknown dtype or epilogue";
    case QD_ERR_WORKSPACE: return "workspace missing or too small";
    case QD_ERR_UNSUPPORTED: return "unsupported argument combination";
    case QD_ERR_HIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

extern "C" int qd_version(void) { return 1; }

namespace qdh {

qd_status fault_injected() {
  const char *f = std::getenv("QD_FAULT_INJECT");
  if (f && std::strcmp(f, "launch") == 0) return QD_ERR_HIP;
  return QD_OK;
}

qd_status check_launch() {
  if (fault_injected() != QD_OK) return QD_ERR_HIP;
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? QD_OK : QD_ERR_HIP;
}

qd_status check_nvfp4(const qd_nvfp4 *t, int64_t groups, int64_t rows, int64_t cols) {
  if (!t) return QD_ERR_NULL;
  if (t->groups != groups || t->rows != rows || t->cols != cols) return QD_ERR_SHAPE;
  if (cols <= 0 || cols % 16 != 0 || rows < 0 || groups < 1) return QD_ERR_SHAPE;
  if (rows == 0) return QD_OK;     // an empty tensor needs no storage
  if (!t->codes || !t->scales || !t->gscale) return QD_ERR_NULL;
  if (!aligned16(t->codes) || !aligned16(t->scales) || !aligned16(t->gscale))
    return QD_ERR_ALIGN;
  return QD_OK;
}

}  // namespace qdh

namespace {

__global__ __launch_bounds__(1024) void reduce_max_kernel(const float *__restrict__ in,
                                                          int64_t n, float *__restrict__ out) {
  __shared__ float red[16];
  const float m = qd::block_max(qd::partials_max(in, n), red);
  if (threadIdx.x == 0) out[0] = m;
}

__global__ __launch_bounds__(256) void fill_i32_kernel(int32_t *p, int64_t n, int32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

}  // namespace

namespace qdi {

void launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s) {
  int64_t g = (n + 255) / 256;
  if (g > 1024) g = 1024;
  if (g < 1) g = 1;
  hipLaunchKernelGGL(fill_i32_kernel, dim3((unsigned)g), dim3(256), 0, s, p, n, v);
}

void launch_reduce_max(const float *in, int64_t n, float *out, hipStream_t s) {
  hipLaunchKernelGGL(reduce_max_kernel, dim3(1), dim3(1024), 0, s, in, n, out);
}

}  // namespace qdi

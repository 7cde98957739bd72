// Matrix-core reference loop: the bf16 MFMA throughput the chip sustains
// under load, the denominator beside the published peak in the attention
// kernels' roofline.  Every wave issues independent
// v_mfma_f32_32x32x16_bf16 products (four accumulator chains, so that no
// product waits for the previous one) and records the shader clock and the
// 100 MHz wall clock around its loop.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "attn_common.h"
#include "errors.h"
#include "libra.h"

namespace libra {

__global__ __launch_bounds__(2 * kThreads) void mfma_loop_kernel(int32_t iters,
                                                             uint64_t *__restrict__ record) {
  bf16x8 a, b;
  static_for<8>([&](auto i) {
    a[int(i)] = bf16(0.001f * (float)(threadIdx.x + i));
    b[int(i)] = bf16(0.002f * (float)i);
  });
  f32x16 c[4];
  static_for<4>([&](auto j) { c[j] = mfma_zero_c(); });
  const uint64_t t0 = clock64(), w0 = wall_clock64();
  for (int32_t it = 0; it < iters; ++it) {
    static_for<4>([&](auto j) { c[j] = mfma32(a, b, c[j]); });
  }
  const uint64_t t1 = clock64(), w1 = wall_clock64();
  float s = 0.f;
  static_for<4>([&](auto j) { static_for<16>([&](auto r) { s += c[j][int(r)]; }); });
  uint64_t *rec = record + 3 * blockIdx.x;
  if (threadIdx.x == 0) {
    rec[0] = t1 - t0;
    rec[1] = w1 - w0;
  }
  // keeps the products live: the sum is finite, so nothing is stored
  if (s != s) rec[2] = 1;
}

}  // namespace libra

using namespace libra;

// One workgroup per compute unit, of 4 or 8 waves: a workgroup is placed on
// one compute unit and its waves spread evenly over the four SIMDs.
static int loop_grid(int32_t waves_per_simd, int *grid) {
  if (waves_per_simd != 1 && waves_per_simd != 2)
    return fail(LIBRA_EINVAL, "waves_per_simd must be 1 or 2 (got %d)", waves_per_simd);
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus < 1)
    return fail(LIBRA_EHIP, "cannot query the compute-unit count");
  *grid = cus;
  return LIBRA_OK;
}

extern "C" int libra_mfma_loop_size(int32_t waves_per_simd, int64_t *record_words,
                                    int64_t *products_per_iter) {
  if (!record_words || !products_per_iter) return fail(LIBRA_EINVAL, "NULL output");
  int grid = 0;
  if (int rc = loop_grid(waves_per_simd, &grid)) return rc;
  *record_words = 3 * (int64_t)grid;
  *products_per_iter = (int64_t)grid * kWaves * waves_per_simd * 4;
  return LIBRA_OK;
}

extern "C" int libra_mfma_loop(int32_t waves_per_simd, int32_t iters, uint64_t *record,
                               int64_t record_words, void *stream) {
  last_error_text().clear();
  int grid = 0;
  if (int rc = loop_grid(waves_per_simd, &grid)) return rc;
  if (iters < 1) return fail(LIBRA_EINVAL, "iters must be >= 1");
  if (!record) return fail(LIBRA_EINVAL, "record is NULL");
  if (record_words < 3 * (int64_t)grid)
    return fail(LIBRA_ENOSPC, "record of %lld words, need %lld", (long long)record_words,
                (long long)(3 * (int64_t)grid));
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(grid), dim3(kThreads * waves_per_simd), 0,
                     static_cast<hipStream_t>(stream), iters, record);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(LIBRA_EHIP, "MFMA loop launch failed: %s", hipGetErrorString(e));
  return LIBRA_OK;
}

// Achievable dense bf16 MFMA rate of the device and the shader clock it holds
// under that load: every wavefront runs independent chains of
// v_mfma_f32_32x32x16_bf16 on register operands (no memory traffic), timed
// with HIP events; the clock is the shader-cycle counter (clock64) against
// the constant-rate counter (wall_clock64) over the same span.
#include <hip/hip_runtime.h>

#include "../../include/stage.h"
#include "common.h"

namespace {

constexpr int PEAK_WAVES = 8;   // wavefronts per work-group (two per SIMD)
constexpr int PEAK_CHAINS = 8;  // independent accumulators per wavefront

__global__ __launch_bounds__(64 * PEAK_WAVES) void mfma_peak_kernel(int iters, float* sink,
                                                                    long long* clk) {
  const int lane = threadIdx.x & 63;
  bf16x8_t a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)((lane + i) & 7));
    b[i] = (__bf16)(0.002f * (float)((lane * 3 + i) & 7));
  }
  f32x16_t acc[PEAK_CHAINS];
#pragma unroll
  for (int c = 0; c < PEAK_CHAINS; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.0f;
  const long long c0 = clock64(), w0 = wall_clock64();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < PEAK_CHAINS; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  const long long c1 = clock64(), w1 = wall_clock64();
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < PEAK_CHAINS; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  if (s == -1.0f) sink[threadIdx.x] = s;  // never true; keeps the chains live
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    clk[0] = c1 - c0;
    clk[1] = w1 - w0;
  }
}

}  // namespace

extern "C" stage_status stage_mfma_peak(void* hip_stream, int iters, double* tflops,
                                        double* clock_ghz) {
  if (!tflops || !clock_ghz || iters < 1 || iters > (1 << 24)) return STAGE_EINVAL;
  *tflops = *clock_ghz = 0.0;
  hipStream_t st = (hipStream_t)hip_stream;
  int dev = 0, cus = 0, wall_khz = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
      cus <= 0 || wall_khz <= 0)
    return STAGE_EHIP;
  float* sink = nullptr;
  long long* clk = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  stage_status status = STAGE_EHIP;
  long long hclk[2] = {0, 0};
  float ms = 0.0f;
  if (hipMalloc(&sink, 64 * PEAK_WAVES * sizeof(float)) != hipSuccess ||
      hipMalloc(&clk, 2 * sizeof(long long)) != hipSuccess || hipEventCreate(&e0) != hipSuccess ||
      hipEventCreate(&e1) != hipSuccess)
    goto done;
  // warm-up launch (code object load, clocks ramping), then the timed one
  hipLaunchKernelGGL(mfma_peak_kernel, dim3(cus), dim3(64 * PEAK_WAVES), 0, st, iters / 8 + 1, sink,
                     clk);
  if (hipGetLastError() != hipSuccess || hipEventRecord(e0, st) != hipSuccess) goto done;
  hipLaunchKernelGGL(mfma_peak_kernel, dim3(cus), dim3(64 * PEAK_WAVES), 0, st, iters, sink, clk);
  if (hipGetLastError() != hipSuccess || hipEventRecord(e1, st) != hipSuccess ||
      hipEventSynchronize(e1) != hipSuccess || hipEventElapsedTime(&ms, e0, e1) != hipSuccess ||
      hipMemcpy(hclk, clk, sizeof(hclk), hipMemcpyDeviceToHost) != hipSuccess || ms <= 0.0f ||
      hclk[1] <= 0)
    goto done;
  {
    const double flop = (double)cus * PEAK_WAVES * PEAK_CHAINS * (double)iters * 2.0 * 32 * 32 * 16;
    *tflops = flop / (ms * 1e-3) * 1e-12;
    *clock_ghz = (double)hclk[0] / ((double)hclk[1] / (wall_khz * 1e3)) * 1e-9;
    status = STAGE_OK;
  }
done:
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (clk) (void)hipFree(clk);
  if (sink) (void)hipFree(sink);
  return status;
}

// HBM-bound row kernels of the encoder layer: residual + bias + LayerNorm
// (forward and backward), deterministic column reductions for the bias /
// gamma / beta gradients, and the masked row softmax (forward and backward).
// One wavefront owns one row; reductions across the row are wavefront
// shuffles.  No MFMA here.
#include "kernels.h"

namespace {

constexpr float LN_EPS = 1e-12f;
constexpr int MAXV = 32;  // columns per lane: rows of up to 64 * 32 = 2048

template <typename T>
__global__ __launch_bounds__(256) void add_ln_fwd_kernel(const T* __restrict__ a,
                                                         const float* __restrict__ bias,
                                                         const T* __restrict__ resid,
                                                         const float* __restrict__ gamma,
                                                         const float* __restrict__ beta,
                                                         T* __restrict__ y, T* __restrict__ xhat,
                                                         float* __restrict__ rstd, int rows, int h) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const int nv = h >> 6;
  const int64_t base = (int64_t)row * h;
  float z[MAXV];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    if (i < nv) {
      int c = lane + 64 * i;
      z[i] = ld_f(a + base + c) + bias[c] + ld_f(resid + base + c);
      s += z[i];
    }
  }
  const float mean = wave_sum(s) / (float)h;
  float s2 = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    if (i < nv) {
      float d = z[i] - mean;
      s2 += d * d;
    }
  }
  const float var = wave_sum(s2) / (float)h;
  const float r = 1.0f / sqrtf(var + LN_EPS);
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    if (i < nv) {
      int c = lane + 64 * i;
      float xh = (z[i] - mean) * r;
      st_f(xhat + base + c, xh);
      st_f(y + base + c, gamma[c] * xh + beta[c]);
    }
  }
  if (lane == 0) rstd[row] = r;
}

// Each wavefront walks its rows and keeps per-column partial sums in
// registers; partials are written per wavefront (no atomics) and summed in a
// fixed order by col_reduce.
template <typename T>
__global__ __launch_bounds__(256) void ln_bwd_kernel(const T* __restrict__ dy,
                                                     const T* __restrict__ xhat,
                                                     const float* __restrict__ rstd,
                                                     const float* __restrict__ gamma,
                                                     T* __restrict__ dz, float* __restrict__ part,
                                                     int rows, int h, int rows_per_wave) {
  const int wid = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int nv = h >> 6;
  float pg[MAXV], pb[MAXV], pz[MAXV];
#pragma unroll
  for (int i = 0; i < MAXV; ++i) pg[i] = pb[i] = pz[i] = 0.0f;
  const int r0 = wid * rows_per_wave;
  const int r1 = min(rows, r0 + rows_per_wave);
  const float inv_h = 1.0f / (float)h;
  for (int row = r0; row < r1; ++row) {
    const int64_t base = (int64_t)row * h;
    float dyv[MAXV], xv[MAXV];
    float sg = 0.0f, sgx = 0.0f;
#pragma unroll
    for (int i = 0; i < MAXV; ++i) {
      if (i < nv) {
        int c = lane + 64 * i;
        dyv[i] = ld_f(dy + base + c);
        xv[i] = ld_f(xhat + base + c);
        float g = dyv[i] * gamma[c];
        sg += g;
        sgx += g * xv[i];
        pg[i] += dyv[i] * xv[i];
        pb[i] += dyv[i];
      }
    }
    sg = wave_sum(sg) * inv_h;
    sgx = wave_sum(sgx) * inv_h;
    const float r = rstd[row];
#pragma unroll
    for (int i = 0; i < MAXV; ++i) {
      if (i < nv) {
        int c = lane + 64 * i;
        float d = r * (dyv[i] * gamma[c] - sg - xv[i] * sgx);
        T dq;
        st_f(&dq, d);
        dz[base + c] = dq;
        // The column sum uses the value as stored, so that the bias gradient
        // of the preceding linear layer matches the gradient that flows on.
        pz[i] += ld_f(&dq);
      }
    }
  }
  float* P = part + (int64_t)wid * 3 * h;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    if (i < nv) {
      int c = lane + 64 * i;
      P[c] = pg[i];
      P[h + c] = pb[i];
      P[2 * h + c] = pz[i];
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void col_partial_kernel(const T* __restrict__ x, int rows, int n,
                                                          int rows_per_blk,
                                                          float* __restrict__ part) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  const int blk = blockIdx.y;
  if (c >= n) return;
  const int r0 = blk * rows_per_blk, r1 = min(rows, r0 + rows_per_blk);
  float s = 0.0f;
  for (int r = r0; r < r1; ++r) s += ld_f(x + (int64_t)r * n + c);
  part[(int64_t)blk * n + c] = s;
}

struct OutPtrs {
  float* p[4];
};

__global__ __launch_bounds__(256) void col_reduce_kernel(const float* __restrict__ part, int nblk,
                                                         int nvec, int n, OutPtrs outs) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  const int v = blockIdx.y;
  if (c >= n || v >= nvec) return;
  float s = 0.0f;
  for (int b = 0; b < nblk; ++b) s += part[((int64_t)b * nvec + v) * n + c];
  if (outs.p[v]) outs.p[v][c] = s;
}

// P = softmax over keys of scale * scores, masked keys -> 0, empty rows -> 0.
template <typename T>
__global__ __launch_bounds__(256) void softmax_fwd_kernel(const float* __restrict__ scores,
                                                          const uint8_t* __restrict__ mask,
                                                          T* __restrict__ P, int BH, int H, int S,
                                                          int ld, float scale) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= (int64_t)BH * S) return;
  const int b = (int)(row / S) / H;
  const float* srow = scores + row * ld;
  const uint8_t* mrow = mask + (int64_t)b * S;
  T* prow = P + row * ld;
  float mx = -INFINITY;
  for (int c = lane; c < S; c += 64)
    if (mrow[c]) mx = fmaxf(mx, scale * srow[c]);
  mx = wave_max(mx);
  float sum = 0.0f;
  if (mx != -INFINITY) {
    for (int c = lane; c < S; c += 64)
      if (mrow[c]) sum += expf(scale * srow[c] - mx);
  }
  sum = wave_sum(sum);
  const float inv = sum > 0.0f ? 1.0f / sum : 0.0f;
  for (int c = lane; c < ld; c += 64) {
    float p = 0.0f;
    if (c < S && mrow[c] && sum > 0.0f) p = expf(scale * srow[c] - mx) * inv;
    st_f(prow + c, p);
  }
}

// dS = scale * P * (dP - sum_j dP_j P_j).
template <typename T>
__global__ __launch_bounds__(256) void softmax_bwd_kernel(const float* __restrict__ dP,
                                                          const T* __restrict__ P,
                                                          T* __restrict__ dS, int BH, int S,
                                                          int ld, float scale) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= (int64_t)BH * S) return;
  const float* drow = dP + row * ld;
  const T* prow = P + row * ld;
  T* orow = dS + row * ld;
  float dot = 0.0f;
  for (int c = lane; c < S; c += 64) dot += drow[c] * ld_f(prow + c);
  dot = wave_sum(dot);
  for (int c = lane; c < ld; c += 64) {
    float v = 0.0f;
    if (c < S) v = scale * ld_f(prow + c) * (drow[c] - dot);
    st_f(orow + c, v);
  }
}

}  // namespace

template <typename T>
hipError_t add_ln_fwd(const T* a, const float* bias, const T* resid, const float* gamma,
                      const float* beta, T* y, T* xhat, float* rstd, int rows, int h,
                      hipStream_t st) {
  if (h % 64 != 0 || h > 64 * MAXV) return hipErrorInvalidValue;
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(add_ln_fwd_kernel<T>, dim3((rows + 3) / 4), dim3(256), 0, st, a, bias, resid,
                     gamma, beta, y, xhat, rstd, rows, h);
  return hipGetLastError();
}

template <typename T>
hipError_t ln_bwd(const T* dy, const T* xhat, const float* rstd, const float* gamma, T* dz,
                  float* part, int nblk, int rows, int h, hipStream_t st) {
  // nblk counts wavefronts (partial rows of part); it must be a multiple of 4.
  if (h % 64 != 0 || h > 64 * MAXV || nblk % 4 != 0) return hipErrorInvalidValue;
  int rpw = (rows + nblk - 1) / nblk;
  if (rpw < 1) rpw = 1;
  hipLaunchKernelGGL(ln_bwd_kernel<T>, dim3(nblk / 4), dim3(256), 0, st, dy, xhat, rstd, gamma, dz,
                     part, rows, h, rpw);
  return hipGetLastError();
}

template <typename T>
hipError_t col_partial(const T* x, int rows, int n, float* part, int nblk, hipStream_t st) {
  int rpb = (rows + nblk - 1) / nblk;
  if (rpb < 1) rpb = 1;
  hipLaunchKernelGGL(col_partial_kernel<T>, dim3((n + 255) / 256, nblk), dim3(256), 0, st, x, rows,
                     n, rpb, part);
  return hipGetLastError();
}

hipError_t col_reduce(const float* part, int nblk, int nvec, int n, float* const* outs,
                      hipStream_t st) {
  if (nvec > 4) return hipErrorInvalidValue;
  OutPtrs o{};
  for (int i = 0; i < nvec; ++i) o.p[i] = outs[i];
  hipLaunchKernelGGL(col_reduce_kernel, dim3((n + 255) / 256, nvec), dim3(256), 0, st, part, nblk,
                     nvec, n, o);
  return hipGetLastError();
}

template <typename T>
hipError_t softmax_fwd(const float* scores, const uint8_t* mask, T* P, int BH, int H, int S,
                       int ld, float scale, hipStream_t st) {
  int64_t rows = (int64_t)BH * S;
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(softmax_fwd_kernel<T>, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st,
                     scores, mask, P, BH, H, S, ld, scale);
  return hipGetLastError();
}

template <typename T>
hipError_t softmax_bwd(const float* dP, const T* P, T* dS, int BH, int S, int ld, float scale,
                       hipStream_t st) {
  int64_t rows = (int64_t)BH * S;
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(softmax_bwd_kernel<T>, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, dP,
                     P, dS, BH, S, ld, scale);
  return hipGetLastError();
}

#define INST(T)                                                                                 \
  template hipError_t add_ln_fwd<T>(const T*, const float*, const T*, const float*,            \
                                    const float*, T*, T*, float*, int, int, hipStream_t);      \
  template hipError_t ln_bwd<T>(const T*, const T*, const float*, const float*, T*, float*,    \
                                int, int, int, hipStream_t);                                   \
  template hipError_t col_partial<T>(const T*, int, int, float*, int, hipStream_t);            \
  template hipError_t softmax_fwd<T>(const float*, const uint8_t*, T*, int, int, int, int,     \
                                     float, hipStream_t);                                      \
  template hipError_t softmax_bwd<T>(const float*, const T*, T*, int, int, int, float,         \
                                     hipStream_t);
INST(float)
INST(bf16_t)

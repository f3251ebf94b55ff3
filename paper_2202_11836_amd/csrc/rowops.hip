// HBM-bound row kernels of the encoder layer: residual + bias + LayerNorm
// (forward and backward), deterministic column reductions for the bias /
// gamma / beta gradients, and the masked row softmax (forward and backward).
// One wavefront owns one row; reductions across the row are wavefront
// shuffles.  No MFMA here.
#include <type_traits>

#include "kernels.h"

namespace {

constexpr float LN_EPS = 1e-12f;

// 8 consecutive elements <-> 8 floats (16-byte bf16 / 32-byte fp32 accesses).
__device__ __forceinline__ void load8(const bf16_t* p, float v[8]) {
  u32x4_t r = *(const u32x4_t*)p;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(r[i] << 16);
    v[2 * i + 1] = __uint_as_float(r[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8(const float* p, float v[8]) {
  f32x4_t a = *(const f32x4_t*)p, b = *(const f32x4_t*)(p + 4);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[i] = a[i];
    v[4 + i] = b[i];
  }
}
__device__ __forceinline__ void store8(bf16_t* p, const float v[8]) {
  u32x4_t r;
#pragma unroll
  for (int i = 0; i < 4; ++i) r[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
  *(u32x4_t*)p = r;
}
__device__ __forceinline__ void store8(float* p, const float v[8]) {
  f32x4_t a, b;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a[i] = v[i];
    b[i] = v[4 + i];
  }
  *(f32x4_t*)p = a;
  *(f32x4_t*)(p + 4) = b;
}
// Round to the storage type and back (what a store followed by a load gives).
__device__ __forceinline__ float as_stored(float v, const bf16_t*) { return bf2f(f2bf(v)); }
__device__ __forceinline__ float as_stored(float v, const float*) { return v; }

// One wavefront per row.  Lane `lane` owns the 8-column chunks
// c = lane + 64 i (i < NC, c < h / 8).  The residual is resid, plus
// resid_lo when not null (a value carried as its bf16 rounding and the
// rounding residual); ylo, when not null, receives y's rounding residual
// y - bf16(y) in bf16, so that y + ylo carries y to about 16 significant
// bits.
template <typename T, typename TA, int NC>
__global__ __launch_bounds__(256) void add_ln_fwd_kernel(const TA* __restrict__ a,
                                                         const float* __restrict__ bias,
                                                         const T* __restrict__ resid,
                                                         const T* __restrict__ resid_lo,
                                                         const float* __restrict__ gamma,
                                                         const float* __restrict__ beta,
                                                         T* __restrict__ y, T* __restrict__ ylo,
                                                         T* __restrict__ xhat,
                                                         float* __restrict__ rstd, int rows, int h) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const int nchunk = h >> 3;
  const int64_t base = (int64_t)row * h;
  float z[NC][8];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int c = lane + 64 * i;
    if (c < nchunk) {
      float av[8], rv[8], bv[8], lv[8];
      load8(a + base + 8 * c, av);
      load8(resid + base + 8 * c, rv);
      load8(bias + 8 * c, bv);
      if (resid_lo) {
        load8(resid_lo + base + 8 * c, lv);
#pragma unroll
        for (int k = 0; k < 8; ++k) rv[k] += lv[k];
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        z[i][k] = av[k] + bv[k] + rv[k];
        s += z[i][k];
      }
    }
  }
  const float mean = wave_sum(s) / (float)h;
  float s2 = 0.0f;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    if (lane + 64 * i < nchunk) {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        float d = z[i][k] - mean;
        s2 += d * d;
      }
    }
  }
  const float var = wave_sum(s2) / (float)h;
  const float r = 1.0f / sqrtf(var + LN_EPS);
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int c = lane + 64 * i;
    if (c < nchunk) {
      float gv[8], btv[8], xh[8], yv[8];
      load8(gamma + 8 * c, gv);
      load8(beta + 8 * c, btv);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        xh[k] = (z[i][k] - mean) * r;
        yv[k] = gv[k] * xh[k] + btv[k];
      }
      store8(xhat + base + 8 * c, xh);
      store8(y + base + 8 * c, yv);
      if (ylo) {
#pragma unroll
        for (int k = 0; k < 8; ++k) yv[k] -= as_stored(yv[k], y);
        store8(ylo + base + 8 * c, yv);
      }
    }
  }
  if (lane == 0) rstd[row] = r;
}

// LayerNorm backward.  A block of 4 wavefronts handles `rpb` consecutive
// rows (one row per wavefront at a time); per-column partial sums of
// dy*xhat, dy and dz are kept per lane, combined across the 4 wavefronts in
// LDS in a fixed order and written as one partial row per block.
template <typename T, int NC>
__global__ __launch_bounds__(256) void ln_bwd_kernel(const T* __restrict__ dy,
                                                     const T* __restrict__ xhat,
                                                     const float* __restrict__ rstd,
                                                     const float* __restrict__ gamma,
                                                     T* __restrict__ dz, float* __restrict__ part,
                                                     int rows, int h, int rpb) {
  extern __shared__ float red[];  // [4 wavefronts][3][h]
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int nchunk = h >> 3;
  float pg[NC][8], pb[NC][8], pz[NC][8], gm[NC][8];
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int c = lane + 64 * i;
#pragma unroll
    for (int k = 0; k < 8; ++k) pg[i][k] = pb[i][k] = pz[i][k] = 0.0f;
    if (c < nchunk) load8(gamma + 8 * c, gm[i]);
  }
  const int r0 = blockIdx.x * rpb;
  const int r1 = min(rows, r0 + rpb);
  const float inv_h = 1.0f / (float)h;
  // Two rows per wavefront at a time (rows row and row + 4), so that the
  // loads of both are in flight together.
  for (int row0 = r0 + wave; row0 < r1; row0 += 8) {
    float dv[2][NC][8], xv[2][NC][8];
    float sg[2] = {0.0f, 0.0f}, sgx[2] = {0.0f, 0.0f};
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int row = row0 + 4 * u;
      const int64_t base = (int64_t)row * h;
#pragma unroll
      for (int i = 0; i < NC; ++i) {
        const int c = lane + 64 * i;
        if (c < nchunk && row < r1) {
          load8(dy + base + 8 * c, dv[u][i]);
          load8(xhat + base + 8 * c, xv[u][i]);
        } else {
#pragma unroll
          for (int k = 0; k < 8; ++k) dv[u][i][k] = xv[u][i][k] = 0.0f;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int i = 0; i < NC; ++i)
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const float g = dv[u][i][k] * gm[i][k];
          sg[u] += g;
          sgx[u] += g * xv[u][i][k];
          pg[i][k] += dv[u][i][k] * xv[u][i][k];
          pb[i][k] += dv[u][i][k];
        }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      sg[u] = wave_sum(sg[u]) * inv_h;
      sgx[u] = wave_sum(sgx[u]) * inv_h;
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int row = row0 + 4 * u;
      if (row >= r1) continue;
      const int64_t base = (int64_t)row * h;
      const float rs = rstd[row];
#pragma unroll
      for (int i = 0; i < NC; ++i) {
        const int c = lane + 64 * i;
        if (c < nchunk) {
          float d[8];
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            d[k] = rs * (dv[u][i][k] * gm[i][k] - sg[u] - xv[u][i][k] * sgx[u]);
            // The column sum uses the value as stored, so that the bias
            // gradient of the preceding linear layer matches the gradient
            // that flows on.
            pz[i][k] += as_stored(d[k], dz);
          }
          store8(dz + base + 8 * c, d);
        }
      }
    }
  }
  // Each wavefront parks its partials in LDS; after one barrier every
  // thread sums the 4 wavefronts' values of its columns in a fixed order.
  float* mine = red + wave * 3 * h;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int c = lane + 64 * i;
    if (c < nchunk) {
      const int col = 8 * c;
      *(f32x4_t*)(mine + col) = f32x4_t{pg[i][0], pg[i][1], pg[i][2], pg[i][3]};
      *(f32x4_t*)(mine + col + 4) = f32x4_t{pg[i][4], pg[i][5], pg[i][6], pg[i][7]};
      *(f32x4_t*)(mine + h + col) = f32x4_t{pb[i][0], pb[i][1], pb[i][2], pb[i][3]};
      *(f32x4_t*)(mine + h + col + 4) = f32x4_t{pb[i][4], pb[i][5], pb[i][6], pb[i][7]};
      *(f32x4_t*)(mine + 2 * h + col) = f32x4_t{pz[i][0], pz[i][1], pz[i][2], pz[i][3]};
      *(f32x4_t*)(mine + 2 * h + col + 4) = f32x4_t{pz[i][4], pz[i][5], pz[i][6], pz[i][7]};
    }
  }
  __syncthreads();
  float* P = part + (int64_t)blockIdx.x * 3 * h;
  for (int e = threadIdx.x; e < 3 * h; e += 256)
    P[e] = ((red[e] + red[3 * h + e]) + red[6 * h + e]) + red[9 * h + e];
}

// bf16 LayerNorm backward with the rows kept as packed bf16 (unpacked where
// used) and gamma in registers: the same arithmetic and partial rows as
// ln_bwd_kernel, twice the loads in flight.  Register budget: two
// work-groups per CU (16384 rows of 32 per work-group are 512 work-groups,
// two per CU), which keeps every per-column partial in registers.
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf_at(const u32x4_t& r, int k) {
  return (k & 1) ? bf_hi(r[k >> 1]) : bf_lo(r[k >> 1]);
}

// The incoming gradient dy is either one bf16 tensor or, when SUM3, the
// fp32 sum (ahi + alo) + b of three bf16 tensors: the backward residual
// stream of a bf16 stage, i.e. the residual branch carried as its bf16
// rounding ahi plus the rounding residual alo (about 16 significant bits),
// plus the bf16 product b of the data-gradient GEMM, so that the stream
// itself is never rounded to bf16.
// dz goes out in bf16 (the operand of the following GEMMs) and, when dzlo
// is not null, its rounding residual dz - bf16(dz) in bf16 as well (the
// residual branch of the next addition).
template <int NC, bool SUM3>
__global__ __launch_bounds__(256, (NC <= 2 ? 2 : 1)) void ln_bwd_bf16_kernel(
    const bf16_t* __restrict__ dy, const bf16_t* __restrict__ ahi, const bf16_t* __restrict__ alo,
    const bf16_t* __restrict__ dyb, const bf16_t* __restrict__ xhat,
    const float* __restrict__ rstd, const float* __restrict__ gamma, bf16_t* __restrict__ dz,
    bf16_t* __restrict__ dzlo, float* __restrict__ part, int rows, int h, int rpb) {
  extern __shared__ float red[];  // [4 wavefronts][3][h]
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int nchunk = h >> 3;
  // gamma of the lane's columns, in registers for all rows
  float pg[NC][8], pb[NC][8], pz[NC][8], gm[NC][8];
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int c = lane + 64 * i;
#pragma unroll
    for (int k = 0; k < 8; ++k) pg[i][k] = pb[i][k] = pz[i][k] = gm[i][k] = 0.0f;
    if (c < nchunk) load8(gamma + 8 * c, gm[i]);
  }
  const int r0 = blockIdx.x * rpb;
  const int r1 = min(rows, r0 + rpb);
  const float inv_h = 1.0f / (float)h;
  for (int row0 = r0 + wave; row0 < r1; row0 += 8) {
    // dy packed bf16 (SUM3: the product b, with ahi and alo beside it)
    u32x4_t dr[2][NC], xr[2][NC], hr[2][NC], lr[2][NC];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int row = row0 + 4 * u;
      const int64_t base = (int64_t)row * h;
#pragma unroll
      for (int i = 0; i < NC; ++i) {
        const int c = lane + 64 * i;
        if (c < nchunk && row < r1) {
          if constexpr (SUM3) {
            hr[u][i] = *(const u32x4_t*)(ahi + base + 8 * c);
            lr[u][i] = *(const u32x4_t*)(alo + base + 8 * c);
            dr[u][i] = *(const u32x4_t*)(dyb + base + 8 * c);
          } else {
            dr[u][i] = *(const u32x4_t*)(dy + base + 8 * c);
          }
          xr[u][i] = *(const u32x4_t*)(xhat + base + 8 * c);
        } else {
          hr[u][i] = lr[u][i] = dr[u][i] = u32x4_t{0, 0, 0, 0};
          xr[u][i] = u32x4_t{0, 0, 0, 0};
        }
      }
    }
    // the incoming gradient at (u, i, k)
    auto dyv = [&](int u, int i, int k) -> float {
      if constexpr (SUM3)
        return (bf_at(hr[u][i], k) + bf_at(lr[u][i], k)) + bf_at(dr[u][i], k);
      else
        return bf_at(dr[u][i], k);
    };
    float sg[2] = {0.0f, 0.0f}, sgx[2] = {0.0f, 0.0f};
#pragma unroll
    for (int i = 0; i < NC; ++i) {
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const float d = dyv(u, i, k), x = bf_at(xr[u][i], k);
          const float g = d * gm[i][k];
          sg[u] += g;
          sgx[u] += g * x;
          pg[i][k] += d * x;
          pb[i][k] += d;
        }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      sg[u] = wave_sum(sg[u]) * inv_h;
      sgx[u] = wave_sum(sgx[u]) * inv_h;
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int row = row0 + 4 * u;
      if (row >= r1) continue;
      const int64_t base = (int64_t)row * h;
      const float rs = rstd[row];
#pragma unroll
      for (int i = 0; i < NC; ++i) {
        const int c = lane + 64 * i;
        if (c < nchunk) {
          float dd[8];
#pragma unroll
          for (int k = 0; k < 8; ++k)
            dd[k] = rs * (dyv(u, i, k) * gm[i][k] - sg[u] - bf_at(xr[u][i], k) * sgx[u]);
          u32x4_t o;
#pragma unroll
          for (int k2 = 0; k2 < 4; ++k2) {
            o[k2] = pack_bf16x2(dd[2 * k2], dd[2 * k2 + 1]);
            // The column sum uses the value as stored, so that the bias
            // gradient of the preceding linear layer matches the gradient
            // its weight gradient is formed from.
            pz[i][2 * k2] += bf_lo(o[k2]);
            pz[i][2 * k2 + 1] += bf_hi(o[k2]);
          }
          *(u32x4_t*)(dz + base + 8 * c) = o;
          if (dzlo) {
            u32x4_t lo;
#pragma unroll
            for (int k2 = 0; k2 < 4; ++k2)
              lo[k2] = pack_bf16x2(dd[2 * k2] - bf_lo(o[k2]), dd[2 * k2 + 1] - bf_hi(o[k2]));
            *(u32x4_t*)(dzlo + base + 8 * c) = lo;
          }
        }
      }
    }
  }
  float* mine = red + wave * 3 * h;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int c = lane + 64 * i;
    if (c < nchunk) {
      const int col = 8 * c;
      *(f32x4_t*)(mine + col) = f32x4_t{pg[i][0], pg[i][1], pg[i][2], pg[i][3]};
      *(f32x4_t*)(mine + col + 4) = f32x4_t{pg[i][4], pg[i][5], pg[i][6], pg[i][7]};
      *(f32x4_t*)(mine + h + col) = f32x4_t{pb[i][0], pb[i][1], pb[i][2], pb[i][3]};
      *(f32x4_t*)(mine + h + col + 4) = f32x4_t{pb[i][4], pb[i][5], pb[i][6], pb[i][7]};
      *(f32x4_t*)(mine + 2 * h + col) = f32x4_t{pz[i][0], pz[i][1], pz[i][2], pz[i][3]};
      *(f32x4_t*)(mine + 2 * h + col + 4) = f32x4_t{pz[i][4], pz[i][5], pz[i][6], pz[i][7]};
    }
  }
  __syncthreads();
  float* P = part + (int64_t)blockIdx.x * 3 * h;
  for (int e = threadIdx.x; e < 3 * h; e += 256)
    P[e] = ((red[e] + red[3 * h + e]) + red[6 * h + e]) + red[9 * h + e];
}

// out = (ahi + alo) + b rounded to bf16 (all bf16), 8 elements per thread
// (n % 8 == 0).
__global__ __launch_bounds__(256) void add3_bf16_kernel(const bf16_t* __restrict__ ahi,
                                                        const bf16_t* __restrict__ alo,
                                                        const bf16_t* __restrict__ b,
                                                        bf16_t* __restrict__ out, int64_t n8) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n8) return;
  float vh[8], vl[8], vb[8];
  load8(ahi + 8 * i, vh);
  load8(alo + 8 * i, vl);
  load8(b + 8 * i, vb);
#pragma unroll
  for (int k = 0; k < 8; ++k) vh[k] = (vh[k] + vl[k]) + vb[k];
  store8(out + 8 * i, vh);
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

// 16 columns per block (colred_block), grid (ceil(n / 16), nvec).
__global__ __launch_bounds__(256) void col_reduce_kernel(const float* __restrict__ part, int nblk,
                                                         int nvec, int n, OutPtrs outs) {
  __shared__ f32x4_t sm[64][4];
  colred_block(part, nblk, nvec, n, blockIdx.y, blockIdx.x, outs.p[blockIdx.y], sm);
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

template <typename T, typename TA>
hipError_t add_ln_fwd(const TA* a, const float* bias, const T* resid, const T* resid_lo,
                      const float* gamma, const float* beta, T* y, T* ylo, T* xhat, float* rstd,
                      int rows, int h, hipStream_t st) {
  if (h % 64 != 0 || h > 2048) return hipErrorInvalidValue;
  if (rows <= 0) return hipSuccess;
  const int nc = (h / 8 + 63) / 64;
  dim3 grid((rows + 3) / 4), blk(256);
#define LAUNCH_LN(NCV)                                                                        \
  hipLaunchKernelGGL((add_ln_fwd_kernel<T, TA, NCV>), grid, blk, 0, st, a, bias, resid, resid_lo, \
                     gamma, beta, y, ylo, xhat, rstd, rows, h)
  switch (nc) {
    case 1: LAUNCH_LN(1); break;
    case 2: LAUNCH_LN(2); break;
    case 3: LAUNCH_LN(3); break;
    default: LAUNCH_LN(4); break;
  }
#undef LAUNCH_LN
  return hipGetLastError();
}

int ln_bwd_blocks(int rows) { return (rows + LN_BWD_RPB - 1) / LN_BWD_RPB; }

hipError_t ln_bwd_bf16(const bf16_t* dy, const bf16_t* ahi, const bf16_t* alo, const bf16_t* b,
                       const bf16_t* xhat, const float* rstd, const float* gamma, bf16_t* dz,
                       bf16_t* dzlo, float* part, int rows, int h, hipStream_t st) {
  if (h % 64 != 0 || h > 2048) return hipErrorInvalidValue;
  const bool sum3 = ahi && alo && b;
  if ((dy == nullptr) == !sum3) return hipErrorInvalidValue;
  if (rows <= 0) return hipSuccess;
  const int nc = (h / 8 + 63) / 64;
  dim3 grid(ln_bwd_blocks(rows)), blk(256);
  size_t sh = (size_t)4 * 3 * h * sizeof(float);
  const int rpb = LN_BWD_RPB;
#define LAUNCH_LNB(NCV, S3)                                                                   \
  hipLaunchKernelGGL((ln_bwd_bf16_kernel<NCV, S3>), grid, blk, sh, st, dy, ahi, alo, b, xhat,  \
                     rstd, gamma, dz, dzlo, part, rows, h, rpb)
  if (!sum3) {
    switch (nc) {
      case 1: LAUNCH_LNB(1, false); break;
      case 2: LAUNCH_LNB(2, false); break;
      case 3: LAUNCH_LNB(3, false); break;
      default: LAUNCH_LNB(4, false); break;
    }
  } else {
    switch (nc) {
      case 1: LAUNCH_LNB(1, true); break;
      case 2: LAUNCH_LNB(2, true); break;
      case 3: LAUNCH_LNB(3, true); break;
      default: LAUNCH_LNB(4, true); break;
    }
  }
#undef LAUNCH_LNB
  return hipGetLastError();
}

hipError_t add3_bf16(const bf16_t* ahi, const bf16_t* alo, const bf16_t* b, bf16_t* out,
                     int64_t n, hipStream_t st) {
  if (n % 8 != 0) return hipErrorInvalidValue;
  const int64_t n8 = n / 8;
  if (n8 == 0) return hipSuccess;
  hipLaunchKernelGGL(add3_bf16_kernel, dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, st, ahi,
                     alo, b, out, n8);
  return hipGetLastError();
}

template <typename T>
hipError_t ln_bwd(const T* dy, const T* xhat, const float* rstd, const float* gamma, T* dz,
                  float* part, int rows, int h, hipStream_t st) {
  if (h % 64 != 0 || h > 2048) return hipErrorInvalidValue;
  if (rows <= 0) return hipSuccess;
  const int nc = (h / 8 + 63) / 64;
  dim3 grid(ln_bwd_blocks(rows)), blk(256);
  size_t sh = (size_t)4 * 3 * h * sizeof(float);
  const int rpb = LN_BWD_RPB;
  if constexpr (std::is_same<T, bf16_t>::value) {
    return ln_bwd_bf16(dy, nullptr, nullptr, nullptr, xhat, rstd, gamma, dz, nullptr, part, rows,
                       h, st);
  }
  switch (nc) {
    case 1: hipLaunchKernelGGL((ln_bwd_kernel<T, 1>), grid, blk, sh, st, dy, xhat, rstd, gamma, dz, part, rows, h, rpb); break;
    case 2: hipLaunchKernelGGL((ln_bwd_kernel<T, 2>), grid, blk, sh, st, dy, xhat, rstd, gamma, dz, part, rows, h, rpb); break;
    case 3: hipLaunchKernelGGL((ln_bwd_kernel<T, 3>), grid, blk, sh, st, dy, xhat, rstd, gamma, dz, part, rows, h, rpb); break;
    default: hipLaunchKernelGGL((ln_bwd_kernel<T, 4>), grid, blk, sh, st, dy, xhat, rstd, gamma, dz, part, rows, h, rpb); break;
  }
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
  if (nvec > 4 || n % 4 != 0) return hipErrorInvalidValue;
  if (n <= 0 || nvec <= 0) return hipSuccess;
  OutPtrs o{};
  for (int i = 0; i < nvec; ++i) o.p[i] = outs[i];
  hipLaunchKernelGGL(col_reduce_kernel, dim3((n + 15) / 16, nvec), dim3(256), 0, st, part, nblk,
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
  template hipError_t add_ln_fwd<T, float>(const float*, const float*, const T*, const T*,     \
                                           const float*, const float*, T*, T*, T*, float*,    \
                                           int, int, hipStream_t);                            \
  template hipError_t ln_bwd<T>(const T*, const T*, const float*, const float*, T*, float*,    \
                                int, int, hipStream_t);                                        \
  template hipError_t col_partial<T>(const T*, int, int, float*, int, hipStream_t);            \
  template hipError_t softmax_fwd<T>(const float*, const uint8_t*, T*, int, int, int, int,     \
                                     float, hipStream_t);                                      \
  template hipError_t softmax_bwd<T>(const float*, const T*, T*, int, int, int, float,         \
                                     hipStream_t);
INST(float)
INST(bf16_t)

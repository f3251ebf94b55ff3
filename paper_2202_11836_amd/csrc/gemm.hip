// Dense contractions of the encoder layer: bf16 MFMA GEMM (fp32 accumulate)
// and an fp32 vector-ALU GEMM, both with fused epilogues.
//
// bf16 path: 256 threads = 4 wavefronts in a 2 x 2 grid; each wavefront owns
// a (BM/2) x (BN/2) sub-tile computed with v_mfma_f32_32x32x16_bf16.  Tiles
// of A and B are staged in LDS in k-contiguous rows (padded by 8 elements so
// that the 16-byte fragment reads of 8 consecutive rows hit distinct banks).
// Operands stored m/n-contiguous in HBM are transposed in registers while
// being staged (4 k-rows x 8 columns per thread), so every MFMA fragment read
// is one ds_read_b128 whatever the operand layout.  The next k-tile is
// fetched into registers while the current one is multiplied.
#include <type_traits>

#include "kernels.h"

namespace {

constexpr int NT = 256;

struct TileCoord {
  int tm, tn, zs, zb;
};

// Work-group index -> (m tile, n tile).  Consecutive dispatches go round robin
// over the 8 XCDs; remap so that each XCD receives a contiguous range of
// tiles, then walk that range in groups of GM tile-rows so that tiles that
// share A rows / B columns run close together on one L2.
__device__ __forceinline__ void tile_of_block(int nbm, int nbn, int& tm, int& tn) {
  int total = nbm * nbn;
  int bid = blockIdx.x;
  if ((total & 7) == 0) bid = (bid & 7) * (total >> 3) + (bid >> 3);
  constexpr int GM = 8;
  int per_group = GM * nbn;
  int group = bid / per_group;
  int first_m = group * GM;
  int gsize = min(nbm - first_m, GM);
  int r = bid - group * per_group;
  tm = first_m + r % gsize;
  tn = r / gsize;
}

__device__ __forceinline__ int64_t batch_off(int zb, int zdiv, int64_t s1, int64_t s2) {
  return (int64_t)(zb / zdiv) * s1 + (int64_t)(zb % zdiv) * s2;
}

template <int EPI, bool OUTF32>
__device__ __forceinline__ void epi_store(const GemmArgs& g, int64_t offC, int64_t offAux, int zs,
                                          int m, int n, float v) {
  if (EPI == EPI_PARTIAL) {
    float* C = (float*)g.C + (int64_t)zs * g.M * g.ldc;
    C[(int64_t)m * g.ldc + n] = v;
  } else if (EPI == EPI_STORE) {
    v *= g.alpha;
    if (g.bias) v += g.bias[n];
    if (OUTF32)
      ((float*)g.C + offC)[(int64_t)m * g.ldc + n] = v;
    else
      ((bf16_t*)g.C + offC)[(int64_t)m * g.ldc + n] = f2bf(v);
  } else if (EPI == EPI_GELU) {
    float u = v + g.bias[n];
    bf16_t ub = f2bf(u);
    ((bf16_t*)g.C + offC)[(int64_t)m * g.ldc + n] = ub;
    // GELU of the stored (rounded) U so that forward and backward agree.
    ((bf16_t*)g.C2 + offC)[(int64_t)m * g.ldc + n] = f2bf(gelu_f(bf2f(ub)));
  } else if (EPI == EPI_DGELU) {
    float u = bf2f(((const bf16_t*)g.aux + offAux)[(int64_t)m * g.ldaux + n]);
    ((bf16_t*)g.C + offC)[(int64_t)m * g.ldc + n] = f2bf(v * gelu_grad_f(u));
  } else if (EPI == EPI_RESID) {
    float r = bf2f(((const bf16_t*)g.aux + offAux)[(int64_t)m * g.ldaux + n]);
    ((bf16_t*)g.C + offC)[(int64_t)m * g.ldc + n] = f2bf(v + r);
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM
// ---------------------------------------------------------------------------
template <int BM, int BN, int BK, bool AK, bool BKM, int EPI, bool OUTF32>
__global__ __launch_bounds__(NT) void gemm_bf16_kernel(GemmArgs g) {
  constexpr int LDS_LD = BK + 8;  // padded row (elements)
  constexpr int TM = BM / 64;     // 32x32 MFMA tiles per wavefront along m
  constexpr int TN = BN / 64;
  __shared__ __attribute__((aligned(16))) bf16_t As[BM * LDS_LD];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[BN * LDS_LD];

  const int nbm = (g.M + BM - 1) / BM, nbn = (g.N + BN - 1) / BN;
  int tm, tn;
  tile_of_block(nbm, nbn, tm, tn);
  const int zs = blockIdx.z % g.ksplit;
  const int zb = blockIdx.z / g.ksplit;
  const int m0 = tm * BM, n0 = tn * BN;
  const bf16_t* __restrict__ A = (const bf16_t*)g.A + batch_off(zb, g.zdiv, g.sA1, g.sA2);
  const bf16_t* __restrict__ B = (const bf16_t*)g.B + batch_off(zb, g.zdiv, g.sB1, g.sB2);
  const int kbeg = zs * g.kchunk;
  const int kend = min(g.K, kbeg + g.kchunk);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Staging registers: each thread moves 16-byte vectors.  A k-major operand
  // tile is R rows of BK/8 vectors; an m/n-major one is (BK/4) x (R/8) blocks
  // of 4 k-rows x 8 columns (4 vectors each).
  constexpr int A_KV = BM * BK / 8 / NT, B_KV = BN * BK / 8 / NT;
  constexpr int A_BLK = (BM * BK / 32 + NT - 1) / NT, B_BLK = (BN * BK / 32 + NT - 1) / NT;
  constexpr int A_REGS = AK ? A_KV : 4 * A_BLK;
  constexpr int B_REGS = BKM ? B_KV : 4 * B_BLK;
  static_assert(A_KV >= 1 && B_KV >= 1, "tile too small");
  u32x4_t ra[A_REGS], rb[B_REGS];

  // Global -> registers for one operand (R rows/columns starting at r0, lim
  // valid), k range [k0, k0 + BK) clipped to kend; out of range reads 0.
  auto load_tile = [&](const bf16_t* __restrict__ X, int64_t ld, auto kmaj_tag, auto R_tag,
                       int r0, int lim, int k0, u32x4_t* regs) {
    constexpr bool KMAJ = decltype(kmaj_tag)::value;
    constexpr int R = decltype(R_tag)::value;
    if constexpr (KMAJ) {
      constexpr int VPR = BK / 8;
#pragma unroll
      for (int i = 0; i < R * BK / 8 / NT; ++i) {
        int v = tid + NT * i;
        int row = v / VPR, kc = (v % VPR) * 8;
        int gr = r0 + row, gk = k0 + kc;
        if (gr < lim && gk < kend)
          regs[i] = *(const u32x4_t*)(X + (int64_t)gr * ld + gk);
        else
          regs[i] = u32x4_t{0, 0, 0, 0};
      }
    } else {
      constexpr int KBN = BK / 4, NBLK = R * BK / 32;
#pragma unroll
      for (int i = 0; i < (NBLK + NT - 1) / NT; ++i) {
        int blk = tid + NT * i;
        int kb = blk % KBN, cb = blk / KBN;
        int gc = r0 + cb * 8;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          int gk = k0 + kb * 4 + j;
          if (blk < NBLK && gc < lim && gk < kend)
            regs[4 * i + j] = *(const u32x4_t*)(X + (int64_t)gk * ld + gc);
          else
            regs[4 * i + j] = u32x4_t{0, 0, 0, 0};
        }
      }
    }
  };

  auto store_tile = [&](bf16_t* S, auto kmaj_tag, auto R_tag, const u32x4_t* regs) {
    constexpr bool KMAJ = decltype(kmaj_tag)::value;
    constexpr int R = decltype(R_tag)::value;
    if constexpr (KMAJ) {
      constexpr int VPR = BK / 8;
#pragma unroll
      for (int i = 0; i < R * BK / 8 / NT; ++i) {
        int v = tid + NT * i;
        int row = v / VPR, kc = (v % VPR) * 8;
        *(u32x4_t*)(S + row * LDS_LD + kc) = regs[i];
      }
    } else {
      constexpr int KBN = BK / 4, NBLK = R * BK / 32;
#pragma unroll
      for (int i = 0; i < (NBLK + NT - 1) / NT; ++i) {
        int blk = tid + NT * i;
        if (blk >= NBLK) continue;
        int kb = blk % KBN, cb = blk / KBN;
        // regs[4i + j] holds columns cb*8 .. cb*8+7 of k-row kb*4 + j;
        // write column c as the 4 consecutive k values of that column.
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const int w = c >> 1, sh = (c & 1) * 16;
          uint32_t e0 = (regs[4 * i + 0][w] >> sh) & 0xffffu;
          uint32_t e1 = (regs[4 * i + 1][w] >> sh) & 0xffffu;
          uint32_t e2 = (regs[4 * i + 2][w] >> sh) & 0xffffu;
          uint32_t e3 = (regs[4 * i + 3][w] >> sh) & 0xffffu;
          u32x2_t o = {e0 | (e1 << 16), e2 | (e3 << 16)};
          *(u32x2_t*)(S + (cb * 8 + c) * LDS_LD + kb * 4) = o;
        }
      }
    }
  };
  using AKT = std::integral_constant<bool, AK>;
  using BKT = std::integral_constant<bool, BKM>;
  using BMT = std::integral_constant<int, BM>;
  using BNT = std::integral_constant<int, BN>;

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int ntiles = (kend - kbeg + BK - 1) / BK;
  if (ntiles > 0) {
    load_tile(A, g.lda, AKT{}, BMT{}, m0, g.M, kbeg, ra);
    load_tile(B, g.ldb, BKT{}, BNT{}, n0, g.N, kbeg, rb);
    store_tile(As, AKT{}, BMT{}, ra);
    store_tile(Bs, BKT{}, BNT{}, rb);
    __syncthreads();
  }
  for (int t = 0; t < ntiles; ++t) {
    const bool more = t + 1 < ntiles;
    if (more) {
      int k0 = kbeg + (t + 1) * BK;
      load_tile(A, g.lda, AKT{}, BMT{}, m0, g.M, k0, ra);
      load_tile(B, g.ldb, BKT{}, BNT{}, n0, g.N, k0, rb);
    }
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8_t af[TM], bfr[TN];
      const int kofs = ks * 16 + (lane >> 5) * 8;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        int row = wm * (BM / 2) + i * 32 + (lane & 31);
        af[i] = *(const bf16x8_t*)(As + row * LDS_LD + kofs);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        int row = wn * (BN / 2) + j * 32 + (lane & 31);
        bfr[j] = *(const bf16x8_t*)(Bs + row * LDS_LD + kofs);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
    if (more) {
      store_tile(As, AKT{}, BMT{}, ra);
      store_tile(Bs, BKT{}, BNT{}, rb);
      __syncthreads();
    }
  }

  // Epilogue.  32x32 accumulator layout: lane holds column (lane % 32);
  // register r holds row 8 * (r / 4) + 4 * (lane / 32) + (r % 4).
  const int64_t offC = batch_off(zb, g.zdiv, g.sC1, g.sC2);
  const int64_t offAux = offC;  // aux shares C's batch layout
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      int n = n0 + wn * (BN / 2) + j * 32 + (lane & 31);
      if (n >= g.N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int m = m0 + wm * (BM / 2) + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (m < g.M) epi_store<EPI, OUTF32>(g, offC, offAux, zs, m, n, acc[i][j][r]);
      }
    }
}

// ---------------------------------------------------------------------------
// fp32 vector-ALU GEMM: 64 x 64 tile, BK 16, 4 x 4 outputs per thread.
// ---------------------------------------------------------------------------
template <int EPI>
__device__ __forceinline__ void epi_store_f32(const GemmArgs& g, int64_t offC, int zs, int m,
                                              int n, float v) {
  if (EPI == EPI_PARTIAL) {
    ((float*)g.C + (int64_t)zs * g.M * g.ldc)[(int64_t)m * g.ldc + n] = v;
  } else if (EPI == EPI_STORE) {
    v *= g.alpha;
    if (g.bias) v += g.bias[n];
    ((float*)g.C + offC)[(int64_t)m * g.ldc + n] = v;
  } else if (EPI == EPI_GELU) {
    float u = v + g.bias[n];
    ((float*)g.C + offC)[(int64_t)m * g.ldc + n] = u;
    ((float*)g.C2 + offC)[(int64_t)m * g.ldc + n] = gelu_f(u);
  } else if (EPI == EPI_DGELU) {
    float u = ((const float*)g.aux + offC)[(int64_t)m * g.ldaux + n];
    ((float*)g.C + offC)[(int64_t)m * g.ldc + n] = v * gelu_grad_f(u);
  } else if (EPI == EPI_RESID) {
    float r = ((const float*)g.aux + offC)[(int64_t)m * g.ldaux + n];
    ((float*)g.C + offC)[(int64_t)m * g.ldc + n] = v + r;
  }
}

template <bool AK, bool BKM, int EPI>
__global__ __launch_bounds__(NT) void gemm_f32_kernel(GemmArgs g) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[BK][BN + 4];
  const int nbm = (g.M + BM - 1) / BM, nbn = (g.N + BN - 1) / BN;
  int tm, tn;
  tile_of_block(nbm, nbn, tm, tn);
  const int zs = blockIdx.z % g.ksplit;
  const int zb = blockIdx.z / g.ksplit;
  const int m0 = tm * BM, n0 = tn * BN;
  const float* __restrict__ A = (const float*)g.A + batch_off(zb, g.zdiv, g.sA1, g.sA2);
  const float* __restrict__ B = (const float*)g.B + batch_off(zb, g.zdiv, g.sB1, g.sB2);
  const int kbeg = zs * g.kchunk;
  const int kend = min(g.K, kbeg + g.kchunk);
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;
  float acc[4][4] = {};
  for (int k0 = kbeg; k0 < kend; k0 += BK) {
    for (int e = tid; e < BM * BK; e += NT) {
      int mm, kk;
      if (AK) { mm = e / BK; kk = e % BK; } else { kk = e / BM; mm = e % BM; }
      int gm = m0 + mm, gk = k0 + kk;
      float v = 0.0f;
      if (gm < g.M && gk < kend) v = AK ? A[(int64_t)gm * g.lda + gk] : A[(int64_t)gk * g.lda + gm];
      As[kk][mm] = v;
    }
    for (int e = tid; e < BN * BK; e += NT) {
      int nn, kk;
      if (BKM) { nn = e / BK; kk = e % BK; } else { kk = e / BN; nn = e % BN; }
      int gn = n0 + nn, gk = k0 + kk;
      float v = 0.0f;
      if (gn < g.N && gk < kend) v = BKM ? B[(int64_t)gn * g.ldb + gk] : B[(int64_t)gk * g.ldb + gn];
      Bs[kk][nn] = v;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  const int64_t offC = batch_off(zb, g.zdiv, g.sC1, g.sC2);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int m = m0 + ty + 16 * i, n = n0 + tx + 16 * j;
      if (m < g.M && n < g.N) epi_store_f32<EPI>(g, offC, zs, m, n, acc[i][j]);
    }
}

__global__ void splitk_reduce_kernel(const float* __restrict__ part, int splits, int64_t mn,
                                     float* __restrict__ out) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= mn) return;
  float s = 0.0f;
  for (int z = 0; z < splits; ++z) s += part[(int64_t)z * mn + i];
  out[i] = s;
}

template <int BM, int BN, bool AK, bool BKM, int EPI, bool OUTF32>
hipError_t launch_bf16(const GemmArgs& g, int batch, hipStream_t st) {
  int nbm = (g.M + BM - 1) / BM, nbn = (g.N + BN - 1) / BN;
  dim3 grid(nbm * nbn, 1, batch * g.ksplit);
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, 64, AK, BKM, EPI, OUTF32>), grid, dim3(NT), 0, st,
                     g);
  return hipGetLastError();
}

template <int BM, int BN, bool AK, bool BKM>
hipError_t dispatch_epi(const GemmArgs& g, GemmEpi epi, bool out_f32, int batch,
                        hipStream_t st) {
  switch (epi) {
    case EPI_STORE:
      return out_f32 ? launch_bf16<BM, BN, AK, BKM, EPI_STORE, true>(g, batch, st)
                     : launch_bf16<BM, BN, AK, BKM, EPI_STORE, false>(g, batch, st);
    case EPI_GELU: return launch_bf16<BM, BN, AK, BKM, EPI_GELU, false>(g, batch, st);
    case EPI_DGELU: return launch_bf16<BM, BN, AK, BKM, EPI_DGELU, false>(g, batch, st);
    case EPI_RESID: return launch_bf16<BM, BN, AK, BKM, EPI_RESID, false>(g, batch, st);
    case EPI_PARTIAL: return launch_bf16<BM, BN, AK, BKM, EPI_PARTIAL, true>(g, batch, st);
  }
  return hipErrorInvalidValue;
}

template <int BM, int BN>
hipError_t dispatch_layout(const GemmArgs& g, bool ak, bool bk, GemmEpi epi, bool out_f32,
                           int batch, hipStream_t st) {
  if (ak && bk) return dispatch_epi<BM, BN, true, true>(g, epi, out_f32, batch, st);
  if (ak && !bk) return dispatch_epi<BM, BN, true, false>(g, epi, out_f32, batch, st);
  if (!ak && !bk) return dispatch_epi<BM, BN, false, false>(g, epi, out_f32, batch, st);
  return dispatch_epi<BM, BN, false, true>(g, epi, out_f32, batch, st);
}

template <bool AK, bool BKM>
hipError_t dispatch_f32(const GemmArgs& g, GemmEpi epi, int batch, hipStream_t st) {
  int nbm = (g.M + 63) / 64, nbn = (g.N + 63) / 64;
  dim3 grid(nbm * nbn, 1, batch * g.ksplit);
  switch (epi) {
    case EPI_STORE:
      hipLaunchKernelGGL((gemm_f32_kernel<AK, BKM, EPI_STORE>), grid, dim3(NT), 0, st, g); break;
    case EPI_GELU:
      hipLaunchKernelGGL((gemm_f32_kernel<AK, BKM, EPI_GELU>), grid, dim3(NT), 0, st, g); break;
    case EPI_DGELU:
      hipLaunchKernelGGL((gemm_f32_kernel<AK, BKM, EPI_DGELU>), grid, dim3(NT), 0, st, g); break;
    case EPI_RESID:
      hipLaunchKernelGGL((gemm_f32_kernel<AK, BKM, EPI_RESID>), grid, dim3(NT), 0, st, g); break;
    case EPI_PARTIAL:
      hipLaunchKernelGGL((gemm_f32_kernel<AK, BKM, EPI_PARTIAL>), grid, dim3(NT), 0, st, g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_bf16(const GemmArgs& g, bool a_kmajor, bool b_kmajor, GemmEpi epi, bool out_f32,
                     int batch, hipStream_t st) {
  if (g.M <= 0 || g.N <= 0 || batch <= 0) return hipSuccess;
  // Narrow outputs (one attention head, 64 columns) take a 128 x 64 tile.
  if (g.N <= 64) return dispatch_layout<128, 64>(g, a_kmajor, b_kmajor, epi, out_f32, batch, st);
  return dispatch_layout<128, 128>(g, a_kmajor, b_kmajor, epi, out_f32, batch, st);
}

hipError_t gemm_f32(const GemmArgs& g, bool a_kmajor, bool b_kmajor, GemmEpi epi, int batch,
                    hipStream_t st) {
  if (g.M <= 0 || g.N <= 0 || batch <= 0) return hipSuccess;
  if (a_kmajor && b_kmajor) return dispatch_f32<true, true>(g, epi, batch, st);
  if (a_kmajor && !b_kmajor) return dispatch_f32<true, false>(g, epi, batch, st);
  if (!a_kmajor && !b_kmajor) return dispatch_f32<false, false>(g, epi, batch, st);
  return dispatch_f32<false, true>(g, epi, batch, st);
}

hipError_t splitk_reduce(const float* part, int splits, int M, int N, float* out,
                         hipStream_t st) {
  int64_t mn = (int64_t)M * N;
  if (mn == 0) return hipSuccess;
  int blocks = (int)((mn + 255) / 256);
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3(blocks), dim3(256), 0, st, part, splits, mn, out);
  return hipGetLastError();
}

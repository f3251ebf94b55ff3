// Dense contractions of the encoder layer: bf16 MFMA GEMM (fp32 accumulate)
// and an fp32 vector-ALU GEMM, both with fused epilogues.
//
// bf16 path: 256 threads = 4 wavefronts in a 2 x 2 grid; each wavefront owns
// a (BM/2) x (BN/2) sub-tile computed with v_mfma_f32_32x32x16_bf16.  Tiles
// of A and B are staged in LDS in k-contiguous rows (padded by 8 elements so
// that the 16-byte fragment reads of 8 consecutive rows hit distinct banks).
// Operands stored m/n-contiguous in HBM keep that layout in LDS and their
// MFMA fragments are read with gfx950's transposing LDS read.  The next
// k-tile is fetched into registers while the current one is multiplied.
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

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM
//
// Block = 4 wavefronts in a 2 x 2 grid over a BM x BN tile; each wavefront
// owns (BM/2) x (BN/2) = TM x TN accumulators of 32 x 32.  k-tiles of 64 are
// double-buffered in LDS (up to 147 KB of gfx950's 160 KB per CU): the next tile is fetched into registers while the
// current one feeds the MFMAs, then written to the other LDS buffer, so one
// barrier per k-tile suffices.  The epilogue stages each 32-row slab of a
// wavefront's accumulators through LDS (fp32) so that bias / activation /
// residual operands are read and the results written as 16-byte row
// segments.
// ---------------------------------------------------------------------------
template <int BM, int BN, bool AK, bool BKM>
struct TileCfg {
  static constexpr int BK = 64;
  static constexpr int LDS_LD = BK + 8;  // k-major rows: 144 B, fragment reads of 8 rows hit distinct banks
  static constexpr int WM = BM / 2, WN = BN / 2;
  static constexpr int TM = WM / 32, TN = WN / 32;
  // k-major operand tile: [R][BK + 8]; m/n-major tile: [BK][R + 16] (the
  // 16-element pad spreads the 4 k-rows a transposing read touches over
  // distinct banks).
  static constexpr int A_ELEMS = AK ? BM * LDS_LD : BK * (BM + 16);
  static constexpr int B_ELEMS = BKM ? BN * LDS_LD : BK * (BN + 16);
  static constexpr int BUF = A_ELEMS + B_ELEMS;  // elements per buffer
  static constexpr int EPI_LD = WN + 4;          // fp32 staging row
  static constexpr int LDS_BYTES_MAIN = 2 * BUF * 2;
  static constexpr int LDS_BYTES_EPI = 4 * 32 * EPI_LD * 4;
  static constexpr int LDS_BYTES = LDS_BYTES_MAIN > LDS_BYTES_EPI ? LDS_BYTES_MAIN : LDS_BYTES_EPI;
};

// Buffer resource over [base, base + bytes): loads past the end return 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int nrec = (int)(bytes < 0 ? 0 : (bytes > 0x7fffffff ? 0x7fffffff : bytes));
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, nrec, 0x00020000);
}

__device__ __forceinline__ u32x4_t buf_load16(__amdgpu_buffer_rsrc_t r, int byte_off) {
  return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0));
}

// Global -> registers for one operand tile of k-tile k0 (relative to the
// resource's first k).  k-major: the resource starts at the tile's first
// row and ends at the operand's last valid row, so rows past it read 0 (K is
// a multiple of BK for k-major operands).  m/n-major: the resource spans this
// split's k rows [kbeg, K), so k rows past K read 0; columns past lim are
// zeroed by a select.
template <int R, int BK, bool KMAJ>
__device__ __forceinline__ void g2r(__amdgpu_buffer_rsrc_t rs, int64_t ld, int r0, int lim, int k0,
                                    u32x4_t* regs) {
  const int tid = threadIdx.x;
  if constexpr (KMAJ) {
    constexpr int VPR = BK / 8;
#pragma unroll
    for (int i = 0; i < R * VPR / NT; ++i) {
      const int v = tid + NT * i;
      const int row = v / VPR, kc = (v % VPR) * 8;
      regs[i] = buf_load16(rs, (int)(((int64_t)row * ld + k0 + kc) * 2));
    }
  } else {
    constexpr int VPR = R / 8;  // vectors per k-row
#pragma unroll
    for (int i = 0; i < R * BK / 8 / NT; ++i) {
      const int v = tid + NT * i;
      const int kr = v / VPR, c8 = (v % VPR) * 8;
      const int gc = r0 + c8;
      const bool ok = gc < lim;
      const u32x4_t x = buf_load16(rs, (int)(((int64_t)(k0 + kr) * ld + (ok ? gc : 0)) * 2));
      regs[i] = ok ? x : u32x4_t{0, 0, 0, 0};
    }
  }
}

// Registers -> LDS: k-major tiles as S[R][LDS_LD], m/n-major tiles as
// S[BK][R + 16], both plain 16-byte copies.
template <int R, int BK, int LDS_LD, bool KMAJ>
__device__ __forceinline__ void r2s(bf16_t* S, const u32x4_t* regs) {
  const int tid = threadIdx.x;
  if constexpr (KMAJ) {
    constexpr int VPR = BK / 8;
#pragma unroll
    for (int i = 0; i < R * VPR / NT; ++i) {
      const int v = tid + NT * i;
      const int row = v / VPR, kc = (v % VPR) * 8;
      *(u32x4_t*)(S + row * LDS_LD + kc) = regs[i];
    }
  } else {
    constexpr int VPR = R / 8;
#pragma unroll
    for (int i = 0; i < R * BK / 8 / NT; ++i) {
      const int v = tid + NT * i;
      const int kr = v / VPR, c8 = (v % VPR) * 8;
      *(u32x4_t*)(S + kr * (R + 16) + c8) = regs[i];
    }
  }
}

// MFMA fragment (8 consecutive k of one row r0 + lane % 32, k offset
// ks * 16 + 8 * (lane / 32)) from an LDS tile.  k-major: one 16-byte read.
// m/n-major [BK][R + 16]: two ds_read_b64_tr_b16.  That instruction works on
// groups of 16 lanes: lane j supplies the address of 4 consecutive 16-bit
// values V[j][0..3], and lane i receives V[4e + i / 4][i % 4] for e = 0..3.
// Lane j of a group points at k-row k0 + j / 4, columns mb + 4 (j % 4), so
// lane i receives the column mb + i at k-rows k0 .. k0 + 3.
template <int R, int LDS_LD, bool KMAJ>
__device__ __forceinline__ bf16x8_t frag(const bf16_t* S, int r0, int ks, int lane) {
  if constexpr (KMAJ) {
    return *(const bf16x8_t*)(S + (r0 + (lane & 31)) * LDS_LD + ks * 16 + (lane >> 5) * 8);
  } else {
    typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
    const int grp = lane >> 4, j = lane & 15;
    const int k0 = ks * 16 + 8 * (grp >> 1);
    const int mb = r0 + 16 * (grp & 1);
    const bf16_t* p = S + (k0 + (j >> 2)) * (R + 16) + mb + 4 * (j & 3);
    const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (__attribute__((address_space(3))) bf16x4_t*)(p));
    const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (__attribute__((address_space(3))) bf16x4_t*)(p + 4 * (R + 16)));
    return bf16x8_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  }
}

template <int R, int BK>
constexpr int stage_regs() {
  return R * BK / 8 / NT;
}

__device__ __forceinline__ uint32_t pack_bf2(float a, float b) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)a) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)b) << 16);
}

// Epilogue for 8 consecutive columns n..n+7 of row m (n % 8 == 0, n < N).
template <int EPI, bool OUTF32>
__device__ __forceinline__ void epi8(const GemmArgs& g, int64_t offC, int zs, int m, int n,
                                     float v[8]) {
  const int64_t idx = (int64_t)m * g.ldc + n;
  if (EPI == EPI_PARTIAL) {
    float* C = (float*)g.C + (int64_t)zs * g.M * g.ldc + idx;
    *(f32x4_t*)C = f32x4_t{v[0], v[1], v[2], v[3]};
    *(f32x4_t*)(C + 4) = f32x4_t{v[4], v[5], v[6], v[7]};
    return;
  }
  if (EPI == EPI_STORE || EPI == EPI_GELU) {
    if (EPI == EPI_STORE) {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] *= g.alpha;
    }
    if (g.bias) {
      const f32x4_t b0 = *(const f32x4_t*)(g.bias + n), b1 = *(const f32x4_t*)(g.bias + n + 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[i] += b0[i];
        v[4 + i] += b1[i];
      }
    }
  }
  if (EPI == EPI_STORE && OUTF32) {
    float* C = (float*)g.C + offC + idx;
    *(f32x4_t*)C = f32x4_t{v[0], v[1], v[2], v[3]};
    *(f32x4_t*)(C + 4) = f32x4_t{v[4], v[5], v[6], v[7]};
    return;
  }
  if (EPI == EPI_DGELU || EPI == EPI_RESID) {
    const u32x4_t x = *(const u32x4_t*)((const bf16_t*)g.aux + offC + (int64_t)m * g.ldaux + n);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a0 = __uint_as_float(x[i] << 16), a1 = __uint_as_float(x[i] & 0xffff0000u);
      if (EPI == EPI_DGELU) {
        v[2 * i] *= gelu_grad_f(a0);
        v[2 * i + 1] *= gelu_grad_f(a1);
      } else {
        v[2 * i] += a0;
        v[2 * i + 1] += a1;
      }
    }
  }
  u32x4_t o;
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = pack_bf2(v[2 * i], v[2 * i + 1]);
  *(u32x4_t*)((bf16_t*)g.C + offC + idx) = o;
  if (EPI == EPI_GELU) {
    // GELU of the stored (rounded) U, so that forward and backward agree.
    u32x4_t q;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float u0 = __uint_as_float(o[i] << 16), u1 = __uint_as_float(o[i] & 0xffff0000u);
      q[i] = pack_bf2(gelu_f(u0), gelu_f(u1));
    }
    *(u32x4_t*)((bf16_t*)g.C2 + offC + idx) = q;
  }
}

template <int BM, int BN, bool AK, bool BKM, int EPI, bool OUTF32>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_kernel(GemmArgs g) {
  using C = TileCfg<BM, BN, AK, BKM>;
  constexpr int BK = C::BK, LDS_LD = C::LDS_LD, TM = C::TM, TN = C::TN;
  __shared__ __attribute__((aligned(16))) unsigned char smem_raw[C::LDS_BYTES];
  bf16_t* smem = (bf16_t*)smem_raw;

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

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int hf = lane >> 5, rr = lane & 31;

  constexpr int AR = stage_regs<BM, BK>(), BR = stage_regs<BN, BK>();
  u32x4_t ra[AR], rb[BR];

  // Buffer resources (see g2r); k offsets passed to g2r are relative to kbeg
  // for m/n-major operands and absolute for k-major ones.
  __amdgpu_buffer_rsrc_t rsA, rsB;
  int kA0, kB0;
  if constexpr (AK) {
    rsA = make_rsrc(A + (int64_t)m0 * g.lda, (int64_t)(g.M - m0) * g.lda * 2);
    kA0 = kbeg;
  } else {
    rsA = make_rsrc(A + (int64_t)kbeg * g.lda, (int64_t)(g.K - kbeg) * g.lda * 2);
    kA0 = 0;
  }
  if constexpr (BKM) {
    rsB = make_rsrc(B + (int64_t)n0 * g.ldb, (int64_t)(g.N - n0) * g.ldb * 2);
    kB0 = kbeg;
  } else {
    rsB = make_rsrc(B + (int64_t)kbeg * g.ldb, (int64_t)(g.K - kbeg) * g.ldb * 2);
    kB0 = 0;
  }

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int ntiles = (kend - kbeg + BK - 1) / BK;
  if (ntiles > 0) {
    g2r<BM, BK, AK>(rsA, g.lda, m0, g.M, kA0, ra);
    g2r<BN, BK, BKM>(rsB, g.ldb, n0, g.N, kB0, rb);
    r2s<BM, BK, LDS_LD, AK>(smem, ra);
    r2s<BN, BK, LDS_LD, BKM>(smem + C::A_ELEMS, rb);
    __syncthreads();
  }
  constexpr int KS = BK / 16;
  for (int t = 0; t < ntiles; ++t) {
    const bf16_t* As = smem + (t & 1) * C::BUF;
    const bf16_t* Bs = As + C::A_ELEMS;
    const bool more = t + 1 < ntiles;
    if (more) {
      g2r<BM, BK, AK>(rsA, g.lda, m0, g.M, kA0 + (t + 1) * BK, ra);
      g2r<BN, BK, BKM>(rsB, g.ldb, n0, g.N, kB0 + (t + 1) * BK, rb);
    }
    // Fragments of k-step ks + 1 are read while the MFMAs of ks run.
    bf16x8_t af[2][TM], bfr[2][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) af[0][i] = frag<BM, LDS_LD, AK>(As, wm * C::WM + i * 32, 0, lane);
#pragma unroll
    for (int j = 0; j < TN; ++j) bfr[0][j] = frag<BN, LDS_LD, BKM>(Bs, wn * C::WN + j * 32, 0, lane);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int cur = ks & 1, nxt = cur ^ 1;
      if (ks + 1 < KS) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
          af[nxt][i] = frag<BM, LDS_LD, AK>(As, wm * C::WM + i * 32, ks + 1, lane);
#pragma unroll
        for (int j = 0; j < TN; ++j)
          bfr[nxt][j] = frag<BN, LDS_LD, BKM>(Bs, wn * C::WN + j * 32, ks + 1, lane);
      }
      if (ks == KS - 1 && more) {
        // The next tile goes to the other buffer while the last MFMAs run.
        bf16_t* An = smem + ((t + 1) & 1) * C::BUF;
        r2s<BM, BK, LDS_LD, AK>(An, ra);
        r2s<BN, BK, LDS_LD, BKM>(An + C::A_ELEMS, rb);
      }
      // Keep the scheduler from sinking the fragment reads of ks + 1 down to
      // their uses: they must be in flight while these MFMAs execute.
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] =
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
  }

  // Epilogue.  32x32 accumulator layout: lane holds column (lane % 32);
  // register r holds row 8 * (r / 4) + 4 * (lane / 32) + (r % 4).
  const int64_t offC = batch_off(zb, g.zdiv, g.sC1, g.sC2);
  float* stg = (float*)smem_raw + wave * 32 * C::EPI_LD;
  const int mw = m0 + wm * C::WM, nw = n0 + wn * C::WN;
  constexpr int CH = C::WN / 8;  // 8-column chunks per staged row
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        stg[(8 * (r >> 2) + 4 * hf + (r & 3)) * C::EPI_LD + j * 32 + rr] = acc[i][j][r];
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int q = 0; q < 32 * CH / 64; ++q) {
      const int c = lane + 64 * q;
      const int row = c / CH, col = (c % CH) * 8;
      const int m = mw + i * 32 + row, n = nw + col;
      float v[8];
      const f32x4_t x0 = *(const f32x4_t*)(stg + row * C::EPI_LD + col);
      const f32x4_t x1 = *(const f32x4_t*)(stg + row * C::EPI_LD + col + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] = x0[e];
        v[4 + e] = x1[e];
      }
      if (m < g.M && n < g.N) epi8<EPI, OUTF32>(g, offC, zs, m, n, v);
    }
    __builtin_amdgcn_wave_barrier();
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
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, AK, BKM, EPI, OUTF32>), grid, dim3(NT), 0, st, g);
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
  // Vector epilogue and m/n-major staging work in 8-column units; k-tiles of
  // 64 never straddle a split boundary, and k-major operands are read
  // without a k bound.
  if (g.N % 8 != 0 || g.ldc % 8 != 0) return hipErrorInvalidValue;
  if (g.ksplit > 1 && g.kchunk % 64 != 0) return hipErrorInvalidValue;
  if ((a_kmajor || b_kmajor) && g.K % 64 != 0) return hipErrorInvalidValue;
  if ((!a_kmajor && g.M % 8 != 0) || (g.lda % 8 != 0) || (g.ldb % 8 != 0)) return hipErrorInvalidValue;
  int tile = g.tile;
  if (tile == 0) {
    const int64_t t256 = (int64_t)((g.M + 255) / 256) * ((g.N + 255) / 256) * batch * g.ksplit;
    tile = (g.M >= 256 && g.N >= 256 && t256 >= 192) ? 1 : (g.N > 128 && t256 >= 64 ? 2 : 3);
  }
  if (tile == 1) return dispatch_layout<256, 256>(g, a_kmajor, b_kmajor, epi, out_f32, batch, st);
  if (tile == 2) return dispatch_layout<256, 128>(g, a_kmajor, b_kmajor, epi, out_f32, batch, st);
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

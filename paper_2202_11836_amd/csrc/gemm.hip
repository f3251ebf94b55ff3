// Dense contractions of the encoder layer: bf16 MFMA GEMM (fp32 accumulate)
// and an fp32 vector-ALU GEMM, both with fused epilogues.
//
// bf16 path: a persistent work-group per CU walks BM x BN output tiles; its
// wavefronts (8 for 256 x 256 tiles, two per SIMD; 4 otherwise) form a
// 2 x (waves / 2) grid, each owning a sub-tile computed with
// v_mfma_f32_32x32x16_bf16.  k-tiles of 64 go straight from HBM into a ring
// of LDS slots with direct-to-LDS buffer loads, issued ahead of use, so no
// staging registers and no LDS store instructions sit in the main loop, and
// the one barrier per k-tile overlaps the MFMAs of the last k-step.  Operands stored m/n-contiguous in
// HBM keep that layout in LDS and their MFMA fragments are read with gfx950's
// transposing LDS read.
#include <algorithm>
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

// Tile order inside a z slice: groups of TILE_GM tile-rows, column by column
// within a group (tiles that share A rows / B columns run close together).
// (4 rather than 8: 1-3% faster for the 12- and 16-tile-wide encoder GEMMs,
// -1.2% per stage step.)
constexpr int TILE_GM = 4;

// Linear tile index -> (z, m tile, n tile) for a persistent grid.  Work-group
// w starts on XCD w % 8 and keeps it (the grid is a multiple of 8), so the
// tile ranges are dealt out per XCD as above.
__device__ __forceinline__ void decode_tile(int vt, int total, int nbm, int nbn, int& z, int& tm,
                                            int& tn, bool xcd_remap = true) {
  int bid = vt;
  if (xcd_remap && (total & 7) == 0) bid = (vt & 7) * (total >> 3) + (vt >> 3);
  const int per_z = nbm * nbn;
  z = bid / per_z;
  const int r0 = bid - z * per_z;
  constexpr int GM = TILE_GM;
  const int per_group = GM * nbn;
  const int group = r0 / per_group;
  const int first_m = group * GM;
  const int gsize = min(nbm - first_m, GM);
  const int r = r0 - group * per_group;
  tm = first_m + r % gsize;
  tn = r / gsize;
}

__device__ __forceinline__ int64_t batch_off(int zb, int zdiv, int64_t s1, int64_t s2) {
  return (int64_t)(zb / zdiv) * s1 + (int64_t)(zb % zdiv) * s2;
}

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM
//
// Block = 2 x (waves / 2) wavefronts over a BM x BN tile; each wavefront
// owns a (BM/2) x (BN/(waves/2)) sub-tile = TM x TN accumulators of 32 x 32.
// k-tiles of 64 sit in a ring of NS LDS slots (with the epilogue staging
// area, up to the full 160 KB of a gfx950 CU), one barrier per k-tile.  The
// epilogue stages each 16-row half of a wavefront's 32-row slab through LDS
// (fp32) so that bias / activation / residual operands are read and the
// results written as 16-byte row segments.
// ---------------------------------------------------------------------------
// k-tile depth and ring depth per tile shape: a ring of NS k-tiles of BK
// keeps NS - 1 k-tiles in flight behind the one being consumed.
// (A deeper ring of k-tiles of 32 was measured slower for 256 x 256: twice
// the barriers per k, and the loads are not the limit at this depth.)
template <int BM, int BN>
struct RingShape {
  static constexpr int BK = 64;
  static constexpr int NS = (BM == 256 && BN == 256) ? 2 : (BM == 256 ? 3 : 4);
  // Wavefronts per work-group: 2 along m times WAVES / 2 along n.  The
  // 256 x 256 tile runs 8 (two per SIMD, 128 x 64 each): while one
  // wavefront waits on loads, a barrier or its epilogue, the other's MFMAs
  // keep the matrix core busy.
  static constexpr int WAVES = (BM == 256 && BN == 256) ? 8 : 4;
};

template <int BM, int BN, bool AK, bool BKM>
struct TileCfg {
  static constexpr int BK = RingShape<BM, BN>::BK;
  static constexpr int NS = RingShape<BM, BN>::NS;
  static constexpr int WAVES = RingShape<BM, BN>::WAVES;
  static constexpr int WGN = WAVES / 2;
  static constexpr int THREADS = 64 * WAVES;
  static constexpr int WM = BM / 2, WN = BN / WGN;
  static constexpr int TM = WM / 32, TN = WN / 32;
  static constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
  // direct-to-LDS load instructions per k-tile per wavefront (1 KB each)
  static constexpr int DMA_PER_TILE = STAGE_BYTES / 1024 / WAVES;
  // Requests of a k-tile split in time over the work-group (see the main
  // loop): on for the 2- and 3-slot rings, off for the 4-slot one (128 x 128
  // tiles), where it measured slower.
  static constexpr bool STAGGER = NS <= 3;
  // Epilogue staging, beside the ring: 16 rows x WN fp32 per wavefront.
  static constexpr int EPI_BYTES = WAVES * 16 * WN * 4;
  static constexpr int LDS_BYTES = NS * STAGE_BYTES + EPI_BYTES;
  static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");
  static_assert((NS - 2) * DMA_PER_TILE <= 63, "vmcnt range");
  static_assert(A_BYTES % (1024 * WAVES) == 0 && B_BYTES % (1024 * WAVES) == 0,
                "whole 1 KB blocks per wavefront");
};

// Buffer resource over [base, base + bytes): loads past the end return 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int nrec = (int)(bytes < 0 ? 0 : (bytes > 0x7fffffff ? 0x7fffffff : bytes));
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, nrec, 0x00020000);
}

typedef __attribute__((address_space(3))) void lds_void_t;

// LDS tile layouts (no padding; 16-byte chunks XOR-swizzled so that the
// fragment reads of each 16-lane group hit distinct banks):
//   k-major  [R][BK]: row r, logical chunk c (8 k values) at physical chunk
//            c ^ kswz(r) of the row's 2 BK bytes, kswz(r) = (r >> 1) & 7 for
//            BK = 64 and (r >> 2) & 3 for BK = 32;
//   m/n-major [BK][R]: k-row k, logical chunk c (8 rows/columns) at physical
//            chunk c ^ (4 (k & 3)) of the row's 2R bytes (R >= 128), so the
//            4 k-rows x 2 chunks of each 16-lane transposing read, and the two
//            groups of a 32-lane pass, cover 16 distinct chunks.
//
// dma_tile issues the direct-to-LDS loads (buffer_load ... lds, 16 bytes per
// lane; lane l of a load lands at LDS base + 16 l) that fill one operand tile
// of k-tile k0 (k relative to the resource, see the kernel), so the tile
// never passes through VGPRs.  Each 1 KB block is one instruction; the 4
// wavefronts split the blocks.
template <int BK>
__device__ __forceinline__ int kswz(int r) {
  return BK == 64 ? ((r >> 1) & 7) : ((r >> 2) & 3);
}

template <int R, bool KMAJ, int BK, int W>
__device__ __forceinline__ void dma_tile(__amdgpu_buffer_rsrc_t rs, int64_t ld, int k0, char* dst,
                                         int wave, int lane) {
  constexpr int NB = R * BK * 2 / 1024;  // 1 KB blocks in the tile
#pragma unroll
  for (int i = 0; i < NB / W; ++i) {
    const int q = wave * (NB / W) + i;
    int64_t elem;
    if constexpr (KMAJ) {
      constexpr int CPR = BK / 8;   // chunks per row
      constexpr int RPB = 64 / CPR; // rows per block
      const int row = RPB * q + lane / CPR;
      const int c = (lane % CPR) ^ kswz<BK>(row);
      elem = (int64_t)row * ld + k0 + 8 * c;
    } else {
      constexpr int CPR = R / 8;           // chunks per k-row
      constexpr int KPB = 64 / CPR;        // k-rows per block
      const int kr = KPB * q + lane / CPR;
      const int c = (lane % CPR) ^ (4 * (kr & 3));
      elem = (int64_t)(k0 + kr) * ld + 8 * c;
    }
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)(dst + q * 1024), 16, (int)(elem * 2),
                                             0, 0, 0);
  }
}

// MFMA operand fragments: 8 consecutive k (offset ks * 16 + 8 * (lane / 32))
// of row r0 + lane % 32.  k-major: one 16-byte read.  m/n-major: two
// ds_read_b64_tr_b16.  That instruction works on groups of 16 lanes: lane j
// supplies the address of 4 consecutive 16-bit values V[j][0..3], and lane i
// receives V[4e + i / 4][i % 4] for e = 0..3.  Lane j of a group points at
// k-row k0 + j / 4, columns mb + 4 (j % 4), so lane i receives column mb + i
// at k-rows k0 .. k0 + 3 (the second read: k0 + 4 .. k0 + 7).
typedef __attribute__((address_space(3))) char lds_char_t;

// An m/n-major fragment as read: the two halves of the transposing reads
// (ds_read_tr16_b64), combined only after lds_wait() / frag_hold().
struct TrFrag {
  u32x2_t lo, hi;
};
__device__ __forceinline__ bf16x8_t frag_val(const bf16x8_t& v) { return v; }
__device__ __forceinline__ bf16x8_t frag_val(const TrFrag& v) {
  return __builtin_bit_cast(bf16x8_t, u32x4_t{v.lo[0], v.lo[1], v.hi[0], v.hi[1]});
}
__device__ __forceinline__ void frag_hold(bf16x8_t&) {}
__device__ __forceinline__ void frag_hold(TrFrag& v) {
  lds_hold(v.lo);
  lds_hold(v.hi);
}

// Per-lane LDS addresses of one operand's fragments in ring slot 0, so that
// every fragment read in the main loop is one instruction with an immediate
// offset (no per-read address arithmetic).  k-major: one address per
// k-step, fragment f (32 rows further) at +f * 32 * 2 BK.  m/n-major: one
// address per fragment, k-step ks at +ks * 16 * 2R, the second transposing
// read at +4 * 2R.  (The swizzle terms depend only on the lane because the
// wavefront's first row is a multiple of 32.)
template <int R, bool KMAJ, int BK, int NF>
struct FragPtrs {
  static constexpr int KS = BK / 16;
  static constexpr int N = KMAJ ? KS : NF;
  using Frag = typename std::conditional<KMAJ, bf16x8_t, TrFrag>::type;
  uint32_t p[N];
  __device__ __forceinline__ void init(uint32_t base, int r0, int lane) {
    if constexpr (KMAJ) {
      const int r = r0 + (lane & 31);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        p[ks] = base + r * (2 * BK) + 16 * ((2 * ks + (lane >> 5)) ^ kswz<BK>(r));
    } else {
      const int grp = lane >> 4, j = lane & 15;
      const int kr = 8 * (grp >> 1) + (j >> 2);
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        const int col = r0 + f * 32 + 16 * (grp & 1) + 4 * (j & 3);
        p[f] = base + kr * (2 * R) + 16 * ((col >> 3) ^ (4 * (kr & 3))) + 2 * (col & 7);
      }
    }
  }
  __device__ __forceinline__ void advance(int delta) {
#pragma unroll
    for (int n = 0; n < N; ++n) p[n] += delta;
  }
  // fragment f of k-step KSI
  template <int KSI>
  __device__ __forceinline__ Frag get(int f) const {
    if constexpr (KMAJ) {
      return *(const __attribute__((address_space(3))) bf16x8_t*)(
          (const lds_char_t*)(uintptr_t)p[KSI] + f * 32 * (2 * BK));
    } else {
      return TrFrag{ds_read_tr16_b64<KSI * 16 * (2 * R)>(p[f]),
                    ds_read_tr16_b64<KSI * 16 * (2 * R) + 4 * (2 * R)>(p[f])};
    }
  }
};


// Epilogue for 8 consecutive columns n..n+7 of row m (n % 8 == 0, n < N).
// b0, b1: bias[n .. n + 7] (EPI_STORE with a bias, EPI_GELU), loaded once
// per tile by the caller.  For EPI_MUL, v returns the values as stored.
template <int EPI, bool OUTF32>
__device__ __forceinline__ void epi8(const GemmArgs& g, int64_t offC, int zs, int m, int n,
                                     float v[8], u32x4_t x, f32x4_t b0, f32x4_t b1) {
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
  if (EPI == EPI_MUL || EPI == EPI_RESID) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a0 = __uint_as_float(x[i] << 16), a1 = __uint_as_float(x[i] & 0xffff0000u);
      if (EPI == EPI_MUL) {
        v[2 * i] *= a0;
        v[2 * i + 1] *= a1;
      } else {
        v[2 * i] += a0;
        v[2 * i + 1] += a1;
      }
    }
  }
  if (EPI == EPI_GELU) {
    // v holds u = acc + bias: store GELU(u) and GELU'(u)
    u32x4_t o, q;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float gv[2], dv[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const float u = v[2 * i + e];
        const GeluParts p = gelu_parts(u);
        gv[e] = u * p.cdf;
        dv[e] = fmaf(u * 0.39894228040143268f, p.e, p.cdf);
      }
      o[i] = pack_bf16x2(gv[0], gv[1]);
      q[i] = pack_bf16x2(dv[0], dv[1]);
    }
    *(u32x4_t*)((bf16_t*)g.C + offC + idx) = o;
    *(u32x4_t*)((bf16_t*)g.C2 + offC + idx) = q;
    return;
  }
  u32x4_t o;
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
  *(u32x4_t*)((bf16_t*)g.C + offC + idx) = o;
  if (EPI == EPI_MUL) {  // hand back the stored (rounded) values
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(o[i] << 16);
      v[2 * i + 1] = __uint_as_float(o[i] & 0xffff0000u);
    }
  }

}

// EPI_MUL / EPI_RESID on 8 values: v * aux or v + aux (aux: 8 packed bf16),
// rounded to bf16 and packed; v returns the rounded values.
template <int EPI>
__device__ __forceinline__ u32x4_t aux8(float v[8], u32x4_t x) {
  u32x4_t o;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float a0 = __uint_as_float(x[i] << 16), a1 = __uint_as_float(x[i] & 0xffff0000u);
    if (EPI == EPI_MUL) {
      v[2 * i] *= a0;
      v[2 * i + 1] *= a1;
    } else {
      v[2 * i] += a0;
      v[2 * i + 1] += a1;
    }
    o[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
    v[2 * i] = __uint_as_float(o[i] << 16);
    v[2 * i + 1] = __uint_as_float(o[i] & 0xffff0000u);
  }
  return o;
}

// One output tile's operands: buffer resources and k-tile range.
struct TileOps {
  __amdgpu_buffer_rsrc_t rsA, rsB;
  int kA0, kB0;     // first k of the range, relative to each resource
  int ntiles;       // k-tiles
  int m0, n0, zs, zb;
};

// Operands of output tile (tm, tn) of batch entry zb over k in [kbeg, kend),
// partial slot zs.
template <int BM, int BN, bool AK, bool BKM>
__device__ __forceinline__ TileOps tile_ops_at(const GemmArgs& g, int zs, int zb, int tm, int tn,
                                               int kbeg, int kend) {
  TileOps o;
  o.zs = zs;
  o.zb = zb;
  o.m0 = tm * BM;
  o.n0 = tn * BN;
  const bf16_t* A = (const bf16_t*)g.A + batch_off(o.zb, g.zdiv, g.sA1, g.sA2);
  const bf16_t* B = (const bf16_t*)g.B + batch_off(o.zb, g.zdiv, g.sB1, g.sB2);
  constexpr int BK = TileCfg<BM, BN, AK, BKM>::BK;
  o.ntiles = (kend - kbeg + BK - 1) / BK;
  // k-major: from the tile's first row to the operand's last row (rows past
  // it read 0; K is a multiple of 64).  m/n-major: from the range's first
  // k-row and the tile's first column to the end of the operand (k-rows past
  // K read 0; reads past the valid columns of a row only feed output rows /
  // columns that are never stored).
  if constexpr (AK) {
    o.rsA = make_rsrc(A + (int64_t)o.m0 * g.lda, (int64_t)(g.M - o.m0) * g.lda * 2);
    o.kA0 = kbeg;
  } else {
    o.rsA = make_rsrc(A + (int64_t)kbeg * g.lda + o.m0, ((int64_t)(g.K - kbeg) * g.lda - o.m0) * 2);
    o.kA0 = 0;
  }
  if constexpr (BKM) {
    o.rsB = make_rsrc(B + (int64_t)o.n0 * g.ldb, (int64_t)(g.N - o.n0) * g.ldb * 2);
    o.kB0 = kbeg;
  } else {
    o.rsB = make_rsrc(B + (int64_t)kbeg * g.ldb + o.n0, ((int64_t)(g.K - kbeg) * g.ldb - o.n0) * 2);
    o.kB0 = 0;
  }
  return o;
}

template <int BM, int BN, bool AK, bool BKM>
__device__ __forceinline__ TileOps tile_ops(const GemmArgs& g, int vt, int total, int nbm, int nbn) {
  int z, tm, tn;
  decode_tile(vt, total, nbm, nbn, z, tm, tn);
  const int kbeg = (z % g.ksplit) * g.kchunk;
  return tile_ops_at<BM, BN, AK, BKM>(g, z % g.ksplit, z / g.ksplit, tm, tn, kbeg,
                                      min(g.K, kbeg + g.kchunk));
}

// k-tile t of an output tile -> ring slot t % NS.
template <int BM, int BN, bool AK, bool BKM>
__device__ __forceinline__ void issue_ktile(const GemmArgs& g, const TileOps& T, int t, char* smem,
                                            int wave, int lane) {
  using C = TileCfg<BM, BN, AK, BKM>;
  char* b = smem + (t % C::NS) * C::STAGE_BYTES;
  dma_tile<BM, AK, C::BK, C::WAVES>(T.rsA, g.lda, T.kA0 + t * C::BK, b, wave, lane);
  dma_tile<BN, BKM, C::BK, C::WAVES>(T.rsB, g.ldb, T.kB0 + t * C::BK, b + C::A_BYTES, wave, lane);
}

// s_waitcnt immediate (gfx9 encoding: vmcnt[3:0] | expcnt[6:4] |
// lgkmcnt[11:8] | vmcnt[5:4] << 14) for "lgkmcnt = 0 and at most N vector
// memory operations outstanding".
template <int N>
__device__ __forceinline__ void wait_vm_lgkm0() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | 0x70 | (((N >> 4) & 3) << 14));
}

// Wait until k-tile t + 1 has landed, given that `after` later k-tiles
// (0 .. NS - 2) have been requested since: the loads complete in order.
template <int PER, int NS>
__device__ __forceinline__ void wait_ktile(int after) {
  if (NS > 5 && after >= 4) wait_vm_lgkm0<(NS > 5 ? 4 * PER : 0)>();
  else if (NS > 4 && after >= 3) wait_vm_lgkm0<(NS > 4 ? 3 * PER : 0)>();
  else if (NS > 3 && after >= 2) wait_vm_lgkm0<(NS > 3 ? 2 * PER : 0)>();
  else if (NS > 2 && after >= 1) wait_vm_lgkm0<(NS > 2 ? PER : 0)>();
  else wait_vm_lgkm0<0>();
}

// Group launch (stream-K).  Range r of the G work-groups covers k-tiles
// [sk_begin(r), sk_begin(r + 1)) of the group's W k-tiles (tiles end to end,
// each tile's K in k-tiles); work-group w takes range (w % 8) G / 8 + w / 8,
// so each XCD (work-groups are dealt round robin over the 8 XCDs; the grid
// is a multiple of 8) works on a contiguous eighth of the tiles.
__host__ __device__ __forceinline__ int64_t sk_begin(int64_t r, int64_t work, int G) {
  return r * work / G;
}
// The range that holds k-tile x: the largest r with sk_begin(r) <= x (never
// an empty range).
__host__ __device__ __forceinline__ int sk_range(int64_t x, int64_t work, int G) {
  return (int)(((x + 1) * G + work - 1) / work - 1);
}
// The two-phase sequence: tile t's first-phase segment (kf k-tiles) starts
// at t kf, its second-phase segment (kt - kf) at nt kf + t (kt - kf).
struct SkSeq {
  int64_t work;
  int nt, kt, kf, G;
};
// Sequence position x -> tile t, k-tile k0 within the tile, k-tiles left in
// the segment.
__host__ __device__ __forceinline__ void sk_locate(const SkSeq& q, int64_t x, int& t, int& k0,
                                                   int& left) {
  const int64_t p1 = (int64_t)q.nt * q.kf;
  if (x < p1) {
    t = (int)(x / q.kf);
    k0 = (int)(x - (int64_t)t * q.kf);
    left = q.kf - k0;
  } else {
    const int k2 = q.kt - q.kf;
    const int64_t y = x - p1;
    t = (int)(y / k2);
    const int o = (int)(y - (int64_t)t * k2);
    k0 = q.kf + o;
    left = k2 - o;
  }
}
// Ranges over tile t's segments: the first phase's [a1, a1 + n1) and the
// second's [a2, a2 + n2) (n2 = 0 without a second phase); the slot of the
// piece of range r is r - a1, or n1 + r - a2.
__host__ __device__ __forceinline__ void sk_tile_ranges(const SkSeq& q, int t, int& a1, int& n1,
                                                        int& a2, int& n2) {
  const int64_t s1 = (int64_t)t * q.kf;
  a1 = sk_range(s1, q.work, q.G);
  n1 = sk_range(s1 + q.kf - 1, q.work, q.G) - a1 + 1;
  if (q.kf < q.kt) {
    const int64_t s2 = (int64_t)q.nt * q.kf + (int64_t)t * (q.kt - q.kf);
    a2 = sk_range(s2, q.work, q.G);
    n2 = sk_range(s2 + (q.kt - q.kf) - 1, q.work, q.G) - a2 + 1;
  } else {
    a2 = n2 = 0;
  }
}

// Position of tile (tm, tn) in a problem's tile order (the inverse of
// decode_tile for one z slice, without the XCD remap).
__host__ __device__ __forceinline__ int tile_pos(int tm, int tn, int nbm, int nbn) {
  const int group = tm / TILE_GM, first_m = group * TILE_GM;
  const int gsize = min(nbm - first_m, TILE_GM);
  return group * TILE_GM * nbn + tn * gsize + (tm - first_m);
}

// The group table is read in place from the kernel-argument segment (a
// by-value argument indexed by a run-time problem number would be copied
// to scratch memory first).
typedef const __attribute__((address_space(4))) GemmGroup kgroup_t;
__device__ __forceinline__ kgroup_t* group_table() {
  return (kgroup_t*)__builtin_amdgcn_kernarg_segment_ptr();
}

__device__ __forceinline__ void group_args(kgroup_t* gg, int p, GemmArgs& g) {
  const __attribute__((address_space(4))) GemmArgs* a = &gg->g[p];
  g.A = a->A;
  g.B = a->B;
  g.C = a->C;
  g.C2 = a->C2;
  g.bias = a->bias;
  g.aux = a->aux;
  g.M = a->M;
  g.N = a->N;
  g.K = a->K;
  g.lda = a->lda;
  g.ldb = a->ldb;
  g.ldc = a->ldc;
  g.ldaux = a->ldaux;
  g.zdiv = a->zdiv;
  g.sA1 = a->sA1;
  g.sA2 = a->sA2;
  g.sB1 = a->sB1;
  g.sB2 = a->sB2;
  g.sC1 = a->sC1;
  g.sC2 = a->sC2;
  g.ksplit = a->ksplit;
  g.kchunk = a->kchunk;
  g.alpha = a->alpha;
  g.tile = a->tile;
  g.colpart = a->colpart;
  g.zdiv_total = a->zdiv_total;
}

// Persistent kernel: each work-group walks output tiles vt = blockIdx.x,
// + gridDim.x, ... (GROUP: the pieces of its stream-K range, see sk_begin).
// The first NS k-tiles of the next output tile are loaded while the current
// tile's epilogue runs.
template <int BM, int BN, bool AK, bool BKM, int EPI, bool OUTF32, bool GROUP = false>
__global__ __launch_bounds__((64 * RingShape<BM, BN>::WAVES), 1) void gemm_bf16_kernel(
    typename std::conditional<GROUP, GemmGroup, GemmArgs>::type ka) {
  using C = TileCfg<BM, BN, AK, BKM>;
  constexpr int TM = C::TM, TN = C::TN, NS = C::NS;
  __shared__ __attribute__((aligned(1024))) char smem[C::LDS_BYTES];

  GemmArgs g;
  int nbm, nbn, total, vt;
  TileOps T;
  // GROUP: this work-group's stream-K range [kb, ke) and the length of the
  // piece being computed.
  int64_t kb = 0, ke = 0;
  int plen = 0;
  const int G = gridDim.x;
  const int rg = (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
  // The piece of the range that starts at k-tile kb: its problem, tile,
  // k range and partial slot.
  auto piece = [&]() {
    kgroup_t* gt = group_table();
    const SkSeq sq = {gt->work, gt->tile0[GEMM_GROUP_MAX], gt->kt, gt->kf, G};
    int t, k0, left;
    sk_locate(sq, kb, t, k0, left);
    plen = (int)min<int64_t>(ke - kb, left);
    int q = 0;
#pragma unroll
    for (int qq = 1; qq < GEMM_GROUP_MAX; ++qq)
      if (qq < gt->n && t >= gt->tile0[qq]) q = qq;
    group_args(gt, q, g);
    nbm = (g.M + BM - 1) / BM;
    nbn = (g.N + BN - 1) / BN;
    int z, tm, tn;
    decode_tile(t - gt->tile0[q], nbm * nbn, nbm, nbn, z, tm, tn, false);
    int a1, n1, a2, n2;
    sk_tile_ranges(sq, t, a1, n1, a2, n2);
    const int slot = k0 < gt->kf ? rg - a1 : n1 + rg - a2;
    T = tile_ops_at<BM, BN, AK, BKM>(g, slot, 0, tm, tn, k0 * C::BK,
                                     min(g.K, (k0 + plen) * C::BK));
  };
  if constexpr (GROUP) {
    kgroup_t* gt = group_table();
    kb = sk_begin(rg, gt->work, G);
    ke = sk_begin(rg + 1, gt->work, G);
    if (kb >= ke) return;
    piece();
    vt = 0;
    total = 0;
  } else {
    g = ka;
    vt = blockIdx.x;
    nbm = (g.M + BM - 1) / BM;
    nbn = (g.N + BN - 1) / BN;
    total = nbm * nbn * g.zdiv_total;
    if (vt >= total) return;
    T = tile_ops<BM, BN, AK, BKM>(g, vt, total, nbm, nbn);
  }
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS DMA targets in SGPRs
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const int hf = lane >> 5, rr = lane & 31;
  constexpr int KS = C::BK / 16;
  // Transposing fragment reads (an m/n-major operand): issued as inline
  // assembly, waited for explicitly.
  constexpr bool TR = !AK || !BKM;

  // First k-tiles of the first output tile.
#pragma unroll
  for (int t = 0; t < NS; ++t)
    if (t < T.ntiles) issue_ktile<BM, BN, AK, BKM>(g, T, t, smem, wave, lane);

  for (;;) {
    f32x16_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
    const int ntiles = T.ntiles;

    // The first k-tiles are in flight (issued before the previous epilogue
    // or above); wait for everything outstanding, then read k-tile 0.
    using PA = FragPtrs<BM, AK, C::BK, TM>;
    using PB = FragPtrs<BN, BKM, C::BK, TN>;
    typename PA::Frag af[2][TM];
    typename PB::Frag bfr[2][TN];
    PA pa;
    PB pb;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_char_t*)smem;
    pa.init(lds0, wm * C::WM, lane);
    pb.init(lds0 + C::A_BYTES, wn * C::WN, lane);
    // Bias of the lane's 8 epilogue columns (the same for all its chunks),
    // loaded once per tile ahead of the wait below: a load in the epilogue
    // would be waited for behind every store issued before it (loads and
    // stores share one counter, so the wait has to drain both).
    constexpr int ECH = C::WN / 8;  // 8-column chunks per staged row
    static_assert(64 % ECH == 0, "a lane's chunks share their columns");
    constexpr bool BIAS = EPI == EPI_STORE || EPI == EPI_GELU;
    // fp32 outputs are stored straight from the accumulators (see the
    // epilogue): the lane's bias is then one value per 32-column block.
    constexpr bool DIRECT = EPI == EPI_PARTIAL || (EPI == EPI_STORE && OUTF32);
    static_assert(TN <= 4, "one bias value per 32-column block");
    f32x4_t bias0 = {0, 0, 0, 0}, bias1 = {0, 0, 0, 0};
    if (BIAS && g.bias) {
      if constexpr (DIRECT) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int bn = T.n0 + wn * C::WN + 32 * j + (lane & 31);
          bias0[j] = bn < g.N ? g.bias[bn] : 0.0f;
        }
      } else {
        const int bn = T.n0 + wn * C::WN + (lane % ECH) * 8;
        if (bn < g.N) {
          bias0 = *(const f32x4_t*)(g.bias + bn);
          bias1 = *(const f32x4_t*)(g.bias + bn + 4);
        }
      }
    }
    wait_vm_lgkm0<0>();
    __syncthreads();
    if (ntiles > 0) {
#pragma unroll
      for (int i = 0; i < TM; ++i) af[0][i] = pa.template get<0>(i);
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[0][j] = pb.template get<0>(j);
    }
    // Main loop.  While the MFMAs of k-step ks run, the fragments of ks + 1
    // are read; in the last k-step of a k-tile they come from the next
    // k-tile instead: wait for this wavefront's loads of k-tile t + 1 and
    // its reads of k-tile t, barrier (every wavefront's k-tile t + 1 has
    // landed and nobody reads k-tile t's slot any more), refill that slot
    // with k-tile t + NS, then read.
    //
    // With STAGGER only the first half of the wavefronts (0 .. WAVES/2 - 1)
    // request their part of k-tile t + NS right after that barrier; the
    // other half request theirs at the start of k-tile t + 1.  Issuing the
    // direct-to-LDS loads stalls a wavefront until the CU's address unit
    // takes them (64 KB per k-tile for 256 x 256), and wavefronts w and
    // w + 4 share a SIMD: split this way, one of each pair issues MFMAs
    // while the other issues its loads, instead of both stalling at once.
    // The slot is free for both halves: its last reads (k-tile t) completed
    // before the barrier.  Before the wait at the end of any k-tile both
    // halves have requested the same k-tiles, so that wait is unchanged.
    // Measured (same box): 256 x 256 encoder GEMM set -3.9%, weight-
    // gradient group -5%, 8192^3 -3%, 256 x 128 tiles at 4096 tokens -2% to
    // -11% (128 x 128: +1% to +7%, hence off there); splitting the pairs the other way
    // (even / odd wavefronts) or each wavefront's own loads in two gave
    // -0.3% to -1.6%; requesting the second half one or two k-steps later
    // was slower than not splitting.
    for (int t = 0; t < ntiles; ++t) {
      static_for<0, KS>([&](auto ksc) {
        constexpr int ks = decltype(ksc)::value;
        constexpr int cur = ks & 1, nxt = cur ^ 1;
        if constexpr (C::STAGGER && ks == 0) {
          if (wave >= C::WAVES / 2 && t >= 1 && t - 1 + NS < ntiles)
            issue_ktile<BM, BN, AK, BKM>(g, T, t - 1 + NS, smem, wave, lane);
        }
        if constexpr (TR) {
          // This k-step's fragments (read during the previous one) have
          // landed; the transposing reads are not tracked by the compiler.
          lds_wait();
#pragma unroll
          for (int i = 0; i < TM; ++i) frag_hold(af[cur][i]);
#pragma unroll
          for (int j = 0; j < TN; ++j) frag_hold(bfr[cur][j]);
        }
        if (ks + 1 < KS) {
          if constexpr (TR) {
            // Interleaved below, with the MFMAs.
          } else {
#pragma unroll
          for (int i = 0; i < TM; ++i) af[nxt][i] = pa.template get<(ks + 1) % KS>(i);
#pragma unroll
          for (int j = 0; j < TN; ++j) bfr[nxt][j] = pb.template get<(ks + 1) % KS>(j);
          }
        } else {
          // Unconditional (also for the last k-tile, whose "next" fragments
          // are never used): a branch here would make the compiler wait for
          // these reads before the last k-step's MFMAs.
          wait_ktile<C::DMA_PER_TILE, NS>(min(ntiles - 1, t + NS - 1) - (t + 1));
          __syncthreads();
          if (t + NS < ntiles && !(C::STAGGER && wave >= C::WAVES / 2))
            issue_ktile<BM, BN, AK, BKM>(g, T, t + NS, smem, wave, lane);
          // move the fragment pointers to the next ring slot
          const int delta = ((t + 1) % NS == 0) ? -(NS - 1) * C::STAGE_BYTES : C::STAGE_BYTES;
          pa.advance(delta);
          pb.advance(delta);
          if constexpr (!TR) {
#pragma unroll
            for (int i = 0; i < TM; ++i) af[nxt][i] = pa.template get<0>(i);
#pragma unroll
            for (int j = 0; j < TN; ++j) bfr[nxt][j] = pb.template get<0>(j);
          }
        }
        if constexpr (TR) {
          // One MFMA, then its share of the next k-step's fragment reads
          // (from the next k-tile after the last k-step), in this order:
          // each read issues while the matrix core works on the MFMA
          // before it.
          constexpr int NM = TM * TN, NF = TM + TN;
          constexpr int kn = ks + 1 < KS ? ks + 1 : 0;
#pragma unroll
          for (int m = 0; m < NM; ++m) {
            acc[m / TN][m % TN] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                frag_val(af[cur][m / TN]), frag_val(bfr[cur][m % TN]), acc[m / TN][m % TN], 0, 0, 0);
#pragma unroll
            for (int f = 0; f < NF; ++f)
              if ((f * NM) / NF == m) {
                if (f < TM) af[nxt][f] = pa.template get<kn>(f);
                else bfr[nxt][f - TM] = pb.template get<kn>(f - TM);
              }
            __builtin_amdgcn_sched_barrier(0);
          }
        } else {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j],
                                                                acc[i][j], 0, 0, 0);
        // Issue order: one MFMA, then the next k-step's fragment reads
        // spread evenly behind the MFMAs (each read issues while the
        // matrix core works on the MFMA before it) instead of all reads
        // ahead of the MFMAs.  Measured: -3% over the encoder GEMMs, -6%
        // for the weight gradients (two reads per fragment).
        {
          constexpr int NM = TM * TN;
          constexpr int NR = TM * (AK ? 1 : 2) + TN * (BKM ? 1 : 2);
#pragma unroll
          for (int m = 0; m < NM; ++m) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, (NR + NM - 1) / NM, 0);  // LDS read
          }
        }
        }
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    if constexpr (TR) {
      // The last k-step's reads of the "next" fragments (never used) must
      // land before their registers are reused.
      lds_wait();
#pragma unroll
      for (int i = 0; i < TM; ++i) frag_hold(af[0][i]), frag_hold(af[1][i]);
#pragma unroll
      for (int j = 0; j < TN; ++j) frag_hold(bfr[0][j]), frag_hold(bfr[1][j]);
    }

    // Every wavefront has read its last fragments: the whole ring is free.
    // Start the next output tile's first NS k-tiles, then run this tile's
    // epilogue (its staging area is separate from the ring).
    __syncthreads();
    const int m0 = T.m0, n0 = T.n0, zs = T.zs, zb = T.zb;
    const GemmArgs ge = g;  // this tile's problem (g moves on to the next tile's)
    const int64_t offC = batch_off(zb, ge.zdiv, ge.sC1, ge.sC2);
    const int mw = m0 + wm * C::WM, nw = n0 + wn * C::WN;
    constexpr int CH = C::WN / 8;  // 8-column chunks per staged row
    constexpr int QN = 16 * CH / 64;  // chunks per lane per staged 16-row half
    // EPI_MUL / EPI_RESID read one bf16 operand chunk per output chunk; the
    // chunks of the next staged half are loaded while this one is processed
    // (the first ones before the next tile's k-tiles are requested).
    constexpr bool AUX = EPI == EPI_MUL || EPI == EPI_RESID;
    u32x4_t axv[2][QN];
    auto aux_load = [&](int it, u32x4_t* dst) {
#pragma unroll
      for (int q = 0; q < QN; ++q) {
        const int c = lane + 64 * q;
        const int row = c / CH, col = (c % CH) * 8;
        const int m = mw + (it >> 1) * 32 + 16 * (it & 1) + row, n = nw + col;
        dst[q] = (m < ge.M && n < ge.N)
                     ? *(const u32x4_t*)((const bf16_t*)ge.aux + offC + (int64_t)m * ge.ldaux + n)
                     : u32x4_t{0, 0, 0, 0};
      }
    };
    if constexpr (AUX) aux_load(0, axv[0]);
    bool more;
    if constexpr (GROUP) {
      kb += plen;
      more = kb < ke;
      if (more) piece();
    } else {
      vt += gridDim.x;
      more = vt < total;
      if (more) T = tile_ops<BM, BN, AK, BKM>(g, vt, total, nbm, nbn);
    }
    auto issue_next = [&]() {
      if (more) {
#pragma unroll
        for (int t = 0; t < NS; ++t)
          if (t < T.ntiles) issue_ktile<BM, BN, AK, BKM>(g, T, t, smem, wave, lane);
      }
    };
    // EPI_MUL / EPI_RESID read an operand per output chunk.  Loads and
    // stores share one counter, so a load waited for after stores drains
    // the stores too: these epilogues compute every chunk first (results
    // packed into the registers the consumed accumulators free), then
    // request the next tile's k-tiles and store.  The others request the
    // k-tiles first and store as they go.
    if constexpr (!AUX) issue_next();
    u32x4_t res[AUX ? 2 * TM : 1][QN];

    // Epilogue.  32x32 accumulator layout: lane holds column (lane % 32);
    // register r holds row 8 * (r / 4) + 4 * (lane / 32) + (r % 4).  Each
    // 16-row half (registers 0-7, 8-15) of a 32-row slab is staged through
    // the wavefront's LDS area as fp32; columns are XOR-swizzled by 32 on
    // rows 4-7 / 12-15 so the two lane halves' stores hit different banks.
    float* stg = (float*)(smem + NS * C::STAGE_BYTES) + wave * 16 * C::WN;
    // Optional column sums (EPI_MUL): every lane keeps one 8-column chunk
    // (CH divides 64) over the rows it writes.
    constexpr bool COLSUM = EPI == EPI_MUL && (CH == 16 || CH == 8) && C::WM == 128;
    float csum[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if constexpr (DIRECT) {
      // fp32 results (split-K partials, or alpha * acc + bias) straight
      // from the accumulators, no LDS round trip: for each register, lanes
      // 0-31 and 32-63 write 32 consecutive columns of two rows, whole
      // 128-byte lines.
      float* Cp = (float*)ge.C + (EPI == EPI_PARTIAL ? (int64_t)zs * ge.M * ge.ldc : offC);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int n = nw + j * 32 + rr;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int m = mw + i * 32 + 8 * (r >> 2) + 4 * hf + (r & 3);
            float v = acc[i][j][r];
            if (EPI == EPI_STORE) {
              v *= ge.alpha;
              if (ge.bias) v += bias0[j];
            }
            if (m < ge.M && n < ge.N) Cp[(int64_t)m * ge.ldc + n] = v;
          }
        }
    } else {
  #pragma unroll
      for (int i = 0; i < TM; ++i) {
  #pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int it = 2 * i + half;
          if constexpr (AUX) {
            if (it + 1 < 2 * TM) aux_load(it + 1, axv[(it + 1) & 1]);
          }
  #pragma unroll
          for (int j = 0; j < TN; ++j)
  #pragma unroll
            for (int r = 8 * half; r < 8 * half + 8; ++r) {
              const int row = 8 * ((r >> 2) & 1) + 4 * hf + (r & 3);  // 0..15
              const int col = (j * 32 + rr) ^ (hf * 32);
              stg[row * C::WN + col] = acc[i][j][r];
            }
          __builtin_amdgcn_wave_barrier();
  #pragma unroll
          for (int q = 0; q < QN; ++q) {
            const int c = lane + 64 * q;
            const int row = c / CH, col = (c % CH) * 8;
            const int pcol = col ^ (((row >> 2) & 1) * 32);
            const int m = mw + i * 32 + 16 * half + row, n = nw + col;
            float v[8];
            const f32x4_t x0 = *(const f32x4_t*)(stg + row * C::WN + pcol);
            const f32x4_t x1 = *(const f32x4_t*)(stg + row * C::WN + pcol + 4);
  #pragma unroll
            for (int e = 0; e < 4; ++e) {
              v[e] = x0[e];
              v[4 + e] = x1[e];
            }
            if constexpr (AUX) {
              res[it][q] = aux8<EPI>(v, axv[it & 1][q]);
              // keep the packed result here (not recomputed from fp32 values
              // held until the stores)
              asm volatile("" : "+v"(res[it][q]));
              if (COLSUM && m < ge.M && n < ge.N) {
  #pragma unroll
                for (int e = 0; e < 8; ++e) csum[e] += v[e];
              }
            } else if (m < ge.M && n < ge.N) {
              epi8<EPI, OUTF32>(ge, offC, zs, m, n, v, u32x4_t{0, 0, 0, 0}, bias0, bias1);
            }
          }
          __builtin_amdgcn_wave_barrier();
        }
      }
    }
    if constexpr (AUX) {
      issue_next();
#pragma unroll
      for (int it = 0; it < 2 * TM; ++it)
#pragma unroll
        for (int q = 0; q < QN; ++q) {
          const int c = lane + 64 * q;
          const int row = c / CH, col = (c % CH) * 8;
          const int m = mw + (it >> 1) * 32 + 16 * (it & 1) + row, n = nw + col;
          if (m < ge.M && n < ge.N)
            *(u32x4_t*)((bf16_t*)ge.C + offC + (int64_t)m * ge.ldc + n) = res[it][q];
        }
    }
    if (COLSUM && ge.colpart) {
      // lanes l, l ^ 16, l ^ 32, l ^ 48 hold the same columns: fixed-order sum
#pragma unroll
      for (int e = 0; e < 8; ++e) {
#pragma unroll
        for (int o = CH; o < 64; o <<= 1) csum[e] += __shfl_xor(csum[e], o, 64);
      }
      const int n = nw + (lane % CH) * 8;
      if (lane < CH && n < ge.N) {
        float* P = ge.colpart + (int64_t)(mw / C::WM) * ge.N + n;
        *(f32x4_t*)P = f32x4_t{csum[0], csum[1], csum[2], csum[3]};
        *(f32x4_t*)(P + 4) = f32x4_t{csum[4], csum[5], csum[6], csum[7]};
      }
    }
    if (!more) break;
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
    const float u = v + g.bias[n];
    ((float*)g.C + offC)[(int64_t)m * g.ldc + n] = gelu_f(u);
    ((float*)g.C2 + offC)[(int64_t)m * g.ldc + n] = gelu_grad_f(u);
  } else if (EPI == EPI_MUL) {
    const float d = ((const float*)g.aux + offC)[(int64_t)m * g.ldaux + n];
    ((float*)g.C + offC)[(int64_t)m * g.ldc + n] = v * d;
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

// out = sum over splits of part[z] in split order; 4 consecutive values per
// thread (mn % 4 == 0), all splits' loads issued before the sum.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part,
                                                            int splits, int64_t mn,
                                                            float* __restrict__ out) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= mn) return;
  f32x4_t s = *(const f32x4_t*)(part + i);
  int z = 1;
  for (; z + 4 <= splits; z += 4) {
    const f32x4_t a = *(const f32x4_t*)(part + (int64_t)z * mn + i);
    const f32x4_t b = *(const f32x4_t*)(part + (int64_t)(z + 1) * mn + i);
    const f32x4_t c = *(const f32x4_t*)(part + (int64_t)(z + 2) * mn + i);
    const f32x4_t d = *(const f32x4_t*)(part + (int64_t)(z + 3) * mn + i);
    s += a;
    s += b;
    s += c;
    s += d;
  }
  for (; z < splits; ++z) s += *(const f32x4_t*)(part + (int64_t)z * mn + i);
  *(f32x4_t*)(out + i) = s;
}

// wgrad_group_reduce: block b serves problem q with blk0[q] <= b <
// blk0[q + 1]; each thread sums 4 consecutive elements of one tile over the
// tile's pieces (slots) in k order.
struct SkReduce {
  const float* part[GEMM_GROUP_MAX];
  float* out[GEMM_GROUP_MAX];
  int M[GEMM_GROUP_MAX], N[GEMM_GROUP_MAX];
  int blk0[GEMM_GROUP_MAX + 1];
  int tile0[GEMM_GROUP_MAX];
  int n;
  SkSeq seq;
  // column reductions: job j owns blocks [cblk0[j], cblk0[j + 1]) after the
  // split-K blocks, ceil(n / 16) per output vector
  ColJob col[COLJOB_MAX];
  int cblk0[COLJOB_MAX + 1];
  int ncol;
};

__global__ __launch_bounds__(256) void wgrad_group_reduce_kernel(SkReduce rd) {
  const int b = blockIdx.x;
  if (b >= rd.blk0[rd.n]) {  // a column-reduction block (block-uniform branch)
    __shared__ f32x4_t sm[64][4];
    int j = 0;
#pragma unroll
    for (int k = 1; k < COLJOB_MAX; ++k)
      if (k < rd.ncol && b >= rd.cblk0[k]) j = k;
    ColJob cj;
    switch (j) {
      case 0: cj = rd.col[0]; break;
      case 1: cj = rd.col[1]; break;
      case 2: cj = rd.col[2]; break;
      default: cj = rd.col[3]; break;
    }
    const int nx = (cj.n + 15) / 16, lb = b - rd.cblk0[j];
    const int v = lb / nx;
    float* o;
    switch (v) {
      case 0: o = cj.out[0]; break;
      case 1: o = cj.out[1]; break;
      case 2: o = cj.out[2]; break;
      default: o = cj.out[3]; break;
    }
    colred_block(cj.part, cj.nblk, cj.nvec, cj.n, v, lb - v * nx, o, sm);
    return;
  }
  int q = 0;
#pragma unroll
  for (int k = 1; k < GEMM_GROUP_MAX; ++k)
    if (k < rd.n && b >= rd.blk0[k]) q = k;
  const float* part;
  float* out;
  int M, N, b0, t0;
  switch (q) {
    case 0: part = rd.part[0]; out = rd.out[0]; M = rd.M[0]; N = rd.N[0]; b0 = rd.blk0[0]; t0 = rd.tile0[0]; break;
    case 1: part = rd.part[1]; out = rd.out[1]; M = rd.M[1]; N = rd.N[1]; b0 = rd.blk0[1]; t0 = rd.tile0[1]; break;
    case 2: part = rd.part[2]; out = rd.out[2]; M = rd.M[2]; N = rd.N[2]; b0 = rd.blk0[2]; t0 = rd.tile0[2]; break;
    default: part = rd.part[3]; out = rd.out[3]; M = rd.M[3]; N = rd.N[3]; b0 = rd.blk0[3]; t0 = rd.tile0[3]; break;
  }
  const int64_t mn = (int64_t)M * N;
  const int64_t i = ((int64_t)(b - b0) * blockDim.x + threadIdx.x) * 4;
  if (i >= mn) return;
  const int m = (int)(i / N), n = (int)(i - (int64_t)m * N);  // N % 4 == 0: one tile
  const int nbm = (M + 255) / 256, nbn = (N + 255) / 256;
  const int t = t0 + tile_pos(m / 256, n / 256, nbm, nbn);
  const SkSeq sq = rd.seq;
  int a1, n1, a2, n2;
  sk_tile_ranges(sq, t, a1, n1, a2, n2);
  // slot 0 (range a1 holds the tile's first k-tile) is always written; an
  // empty range wrote no slot
  f32x4_t s = *(const f32x4_t*)(part + i);
  for (int j = 1; j < n1 + n2; ++j) {
    const int r = j < n1 ? a1 + j : a2 + j - n1;
    if (sk_begin(r, sq.work, sq.G) < sk_begin(r + 1, sq.work, sq.G))
      s += *(const f32x4_t*)(part + (int64_t)j * mn + i);
  }
  *(f32x4_t*)(out + i) = s;
}

int device_cus() {
  static int cus = 0;
  if (cus == 0) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cus = n;
  }
  return cus;
}

template <int BM, int BN, bool AK, bool BKM, int EPI, bool OUTF32>
hipError_t launch_bf16(const GemmArgs& g0, int batch, hipStream_t st) {
  GemmArgs g = g0;
  g.zdiv_total = batch * g.ksplit;
  const int64_t total = (int64_t)((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN) * g.zdiv_total;
  // One work-group per CU (LDS and registers allow no more); a multiple of
  // 8 so that each work-group stays on one XCD's share of the tiles.
  int64_t grid = std::min<int64_t>(total, device_cus());
  if (grid >= 8) grid -= grid % 8;
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, AK, BKM, EPI, OUTF32>), dim3((unsigned)grid),
                     dim3(TileCfg<BM, BN, AK, BKM>::THREADS), 0, st, g);
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
    case EPI_MUL: return launch_bf16<BM, BN, AK, BKM, EPI_MUL, false>(g, batch, st);
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
    case EPI_MUL:
      hipLaunchKernelGGL((gemm_f32_kernel<AK, BKM, EPI_MUL>), grid, dim3(NT), 0, st, g); break;
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
  // Operands are read through buffer resources with 32-bit byte extents and
  // offsets: each operand (per batch entry) must span less than 2 GiB.
  const int64_t a_bytes = (int64_t)(a_kmajor ? g.M : g.K) * g.lda * 2;
  const int64_t b_bytes = (int64_t)(b_kmajor ? g.N : g.K) * g.ldb * 2;
  if (a_bytes >= ((int64_t)1 << 31) || b_bytes >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  int tile = g.tile;
  if (tile == 0) {
    // The largest tile whose count still covers about three quarters of
    // the CUs (one persistent work-group per CU): a 256 x 256 tile has
    // twice the arithmetic per loaded byte of a 128 x 128 one, but idle
    // CUs cost more.  Measured at T = 4096 tokens, N = 1024 (64 tiles of
    // 256 x 256 on 256 CUs): 128 x 128 tiles 1.45-1.55x faster than
    // 256 x 128 ones, which were 1.3x faster than 256 x 256.
    const int64_t zb = (int64_t)batch * g.ksplit;
    const int64_t need = 3 * (int64_t)device_cus() / 4;
    const int64_t t1 = (int64_t)((g.M + 255) / 256) * ((g.N + 255) / 256) * zb;
    const int64_t t2 = (int64_t)((g.M + 255) / 256) * ((g.N + 127) / 128) * zb;
    tile = (g.M >= 256 && g.N >= 256 && t1 >= need) ? 1 : (g.M >= 256 && g.N > 128 && t2 >= need) ? 2 : 3;
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
  if (mn % 4 != 0 || splits < 1) return hipErrorInvalidValue;
  int blocks = (int)((mn / 4 + 255) / 256);
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3(blocks), dim3(256), 0, st, part, splits, mn, out);
  return hipGetLastError();
}

namespace {

// Grid of a group launch: one work-group per CU, a multiple of 8.
int group_grid() {
  const int cus = device_cus();
  return std::max(8, cus - cus % 8);
}

// First-phase k-tiles per tile: the average range, when shorter than a tile.
int first_phase(int64_t tiles, int kt) {
  const int64_t w = tiles * kt / group_grid();
  return (int)std::max<int64_t>(1, std::min<int64_t>(kt, w));
}

// Checks and the stream-K table of a group; false for invalid problems.
bool group_table_of(const GemmArgs* p, int n, GemmGroup& gg) {
  if (n < 1 || n > GEMM_GROUP_MAX || !p) return false;
  gg = GemmGroup{};
  gg.n = n;
  int64_t tiles = 0;
  for (int q = 0; q < n; ++q) {
    GemmArgs g = p[q];
    // the checks gemm_bf16 makes for two m/n-major operands; one K for all
    if (g.M < 0 || g.N < 0 || g.K < 1 || g.K != p[0].K) return false;
    if (g.N % 8 != 0 || g.ldc % 8 != 0 || g.M % 8 != 0 || g.lda % 8 != 0 || g.ldb % 8 != 0)
      return false;
    if ((int64_t)g.K * g.lda * 2 >= ((int64_t)1 << 31) ||
        (int64_t)g.K * g.ldb * 2 >= ((int64_t)1 << 31))
      return false;
    g.zdiv = 1;
    g.ksplit = 1;
    g.kchunk = g.K;
    g.zdiv_total = 1;
    g.sA1 = g.sA2 = g.sB1 = g.sB2 = g.sC1 = g.sC2 = 0;
    gg.g[q] = g;
    gg.tile0[q] = (int)tiles;
    tiles += (int64_t)((g.M + 255) / 256) * ((g.N + 255) / 256);
    if (tiles >= ((int64_t)1 << 24)) return false;
  }
  gg.tile0[n] = (int)tiles;
  for (int q = n + 1; q <= GEMM_GROUP_MAX; ++q) gg.tile0[q] = (int)tiles;
  gg.kt = (p[0].K + 63) / 64;
  gg.work = tiles * gg.kt;
  gg.kf = first_phase(tiles, gg.kt);
  return true;
}

}  // namespace

int wgrad_group_slots(const int* M, const int* N, int n, int K) {
  if (n < 1 || n > GEMM_GROUP_MAX || K < 1) return 0;
  int64_t tiles = 0;
  for (int q = 0; q < n; ++q) {
    if (M[q] < 0 || N[q] < 0) return 0;
    tiles += (int64_t)((M[q] + 255) / 256) * ((N[q] + 255) / 256);
  }
  if (tiles == 0) return 1;
  const int kt = (K + 63) / 64;
  const SkSeq sq = {tiles * kt, (int)tiles, kt, first_phase(tiles, kt), group_grid()};
  int slots = 1;
  for (int t = 0; t < (int)tiles; ++t) {
    int a1, n1, a2, n2;
    sk_tile_ranges(sq, t, a1, n1, a2, n2);
    slots = std::max(slots, n1 + n2);
  }
  return slots;
}

hipError_t gemm_bf16_wgrad_group(const GemmArgs* p, int n, hipStream_t st) {
  GemmGroup gg;
  if (!group_table_of(p, n, gg)) return hipErrorInvalidValue;
  if (gg.work == 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_bf16_kernel<256, 256, false, false, EPI_PARTIAL, true, true>),
                     dim3((unsigned)group_grid()), dim3(TileCfg<256, 256, false, false>::THREADS),
                     0, st, gg);
  return hipGetLastError();
}

hipError_t wgrad_group_reduce(const GemmArgs* p, float* const* out, int n, const ColJob* cols,
                              int ncols, hipStream_t st) {
  GemmGroup gg;
  if (!group_table_of(p, n, gg) || !out || ncols < 0 || ncols > COLJOB_MAX || (ncols && !cols))
    return hipErrorInvalidValue;
  SkReduce rd{};
  rd.n = n;
  rd.seq = {gg.work, gg.tile0[n], gg.kt, gg.kf, group_grid()};
  int64_t blocks = 0;
  for (int q = 0; q < n; ++q) {
    if (p[q].ldc != p[q].N) return hipErrorInvalidValue;  // partial slots are dense M x N
    rd.part[q] = (const float*)p[q].C;
    rd.out[q] = out[q];
    rd.M[q] = p[q].M;
    rd.N[q] = p[q].N;
    rd.tile0[q] = gg.tile0[q];
    rd.blk0[q] = (int)blocks;
    blocks += ((int64_t)p[q].M * p[q].N / 4 + 255) / 256;
    if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  }
  for (int q = n; q <= GEMM_GROUP_MAX; ++q) rd.blk0[q] = (int)blocks;
  rd.ncol = ncols;
  for (int j = 0; j < ncols; ++j) {
    const ColJob& c = cols[j];
    if (c.nvec < 1 || c.nvec > 4 || c.n < 0 || c.n % 4 != 0 || c.nblk < 0 || !c.part)
      return hipErrorInvalidValue;
    rd.col[j] = c;
    rd.cblk0[j] = (int)blocks;
    blocks += (int64_t)((c.n + 15) / 16) * c.nvec;
    if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  }
  for (int j = ncols; j <= COLJOB_MAX; ++j) rd.cblk0[j] = (int)blocks;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(wgrad_group_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, st, rd);
  return hipGetLastError();
}

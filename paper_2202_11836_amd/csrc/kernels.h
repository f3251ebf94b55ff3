// Host-side launchers of the encoder-stage kernels (gfx950).  Every launcher
// enqueues on the given stream and returns the launch status; none of them
// synchronises.  Shapes are validated by the caller (the stage engine).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

// ---------------------------------------------------------------------------
// GEMM:  C[m, n] = sum_k A(m, k) * B(k, n), then an epilogue.
//   A(m, k) = A[m * lda + k]  if a_kmajor  else  A[k * lda + m]
//   B(k, n) = B[n * ldb + k]  if b_kmajor  else  B[k * ldb + n]
// Batched over grid z: batch index zb splits into (zb / zdiv, zb % zdiv),
// and each operand is offset by (zb / zdiv) * s*1 + (zb % zdiv) * s*2.
// With ksplit > 1 the K range is cut into ksplit chunks of kchunk elements
// and each chunk writes an fp32 partial to C + split * M * ldc (EPI_PARTIAL).
// ---------------------------------------------------------------------------
enum GemmEpi {
  EPI_STORE = 0,    // C = alpha * acc (+ bias[n] when bias != nullptr)
  EPI_GELU = 1,     // u = acc + bias[n]:  GELU(u) -> C;  GELU'(u) -> C2
  EPI_MUL = 2,      // C = acc * aux[m, n]  (the FFN backward: dU = dG * GELU'(u))
  EPI_RESID = 3,    // C = acc + aux[m, n]
  EPI_PARTIAL = 4,  // fp32 C[split][m][n] = acc over this split's K range
};

struct GemmArgs {
  const void* A;
  const void* B;
  void* C;
  void* C2;
  const float* bias;
  const void* aux;
  int M, N, K;
  int64_t lda, ldb, ldc, ldaux;
  int zdiv;
  int64_t sA1, sA2, sB1, sB2, sC1, sC2;
  int ksplit;
  int kchunk;
  float alpha;
  int tile;  // bf16 tile shape: 0 = automatic, 1 = 256x256, 2 = 256x128, 3 = 128x128
  // EPI_MUL on bf16, optional: column sums of the stored output per block
  // of 128 rows, colpart[m / 128][n] (needs tile 1).
  float* colpart;
  int zdiv_total;  // internal: batch * ksplit
};

inline GemmArgs gemm_args(const void* A, int64_t lda, const void* B, int64_t ldb, void* C,
                          int64_t ldc, int M, int N, int K) {
  GemmArgs g{};
  g.A = A; g.B = B; g.C = C; g.lda = lda; g.ldb = ldb; g.ldc = ldc;
  g.M = M; g.N = N; g.K = K; g.zdiv = 1; g.ksplit = 1; g.kchunk = K; g.alpha = 1.0f;
  return g;
}

// bf16 operands on MFMA (fp32 accumulation).  out_f32 selects fp32 output
// for EPI_STORE; all other epilogues write bf16 (EPI_PARTIAL writes fp32).
hipError_t gemm_bf16(const GemmArgs& g, bool a_kmajor, bool b_kmajor, GemmEpi epi,
                     bool out_f32, int batch, hipStream_t st);
// fp32 operands on the vector ALU (fp32 accumulation), same conventions.
hipError_t gemm_f32(const GemmArgs& g, bool a_kmajor, bool b_kmajor, GemmEpi epi,
                    int batch, hipStream_t st);
// out[m][n] = sum_s part[s][m][n] (fixed order), fp32.
hipError_t splitk_reduce(const float* part, int splits, int M, int N, float* out, hipStream_t st);

// Up to GEMM_GROUP_MAX weight-gradient GEMMs in one launch, stream-K: each
// problem p[q] is a GEMM with both operands m/n-major (A(m, k) = A[k * lda +
// m], B(k, n) = B[k * ldb + n]: token-major activations and output
// gradients), batch 1, and all share one K.  The k-tiles (of 64) of their
// 256 x 256 tiles are laid end to end in two phases, the first kf k-tiles
// of every tile, then the rest of every tile, and the sequence is cut into
// one contiguous range per work-group (one work-group per CU); kf is the
// average range length when a tile holds more than that, so that the
// work-groups of the first phase each own one tile's first kf k-tiles and
// all run over the same k at the same time.  The part of a range inside one
// tile's phase (a piece) writes an fp32 partial to slot j of its problem's C
// (C + j * M * ldc), j = its rank among that tile's pieces in k order;
// wgrad_group_reduce then sums each tile's pieces in k order.  ksplit /
// kchunk of p[q] are ignored.
constexpr int GEMM_GROUP_MAX = 4;
struct GemmGroup {
  GemmArgs g[GEMM_GROUP_MAX];
  int n;
  int tile0[GEMM_GROUP_MAX + 1];  // first (global) tile of each problem; tile0[n] = all tiles
  int kt;                         // k-tiles per tile, ceil(K / 64)
  int kf;                         // k-tiles of each tile in the first phase
  int64_t work;                   // k-tiles over all tiles, tile0[n] * kt
};
// Slots of M x N fp32 partials each problem's C must hold for such a group
// (the most pieces of one tile) on this device; 0 for invalid sizes.
int wgrad_group_slots(const int* M, const int* N, int n, int K);
hipError_t gemm_bf16_wgrad_group(const GemmArgs* p, int n, hipStream_t st);
// A column reduction run with a group's reduction: out[v][c] = the sum over
// the nblk partial rows b of part[(b * nvec + v) * n + c], v < nvec <= 4, in
// col_reduce's order (null outputs are skipped).
struct ColJob {
  const float* part;
  int nblk, nvec, n;
  float* out[4];
};
constexpr int COLJOB_MAX = 4;
// out[q][m][n] = the sum over the pieces of (m, n)'s tile of slot j of
// p[q].C, in k order (same p as the GEMM launch), and the ncols <=
// COLJOB_MAX column reductions cols, in one launch.
hipError_t wgrad_group_reduce(const GemmArgs* p, float* const* out, int n, const ColJob* cols,
                              int ncols, hipStream_t st);

// ---------------------------------------------------------------------------
// Row kernels (one wavefront per row), T = float or bf16_t.
// ---------------------------------------------------------------------------
// z = a + bias + resid (+ resid_lo);  y = gamma * xhat + beta with
// xhat = (z - mean) * rstd.  a is the fp32 output of the preceding GEMM;
// resid_lo (optional, may be null) is the rounding residual of resid; ylo
// (optional, may be null) receives y - y as stored, in T.
template <typename T, typename TA>
hipError_t add_ln_fwd(const TA* a, const float* bias, const T* resid, const T* resid_lo,
                      const float* gamma, const float* beta, T* y, T* ylo, T* xhat, float* rstd,
                      int rows, int h, hipStream_t st);

// dz = rstd * (g - mean(g) - xhat * mean(g * xhat)), g = dy * gamma.
// Column partial sums per block of LN_BWD_RPB rows (ln_bwd_blocks(rows)
// blocks): part[blk][0][:] = sum dy*xhat, part[blk][1][:] = sum dy,
// part[blk][2][:] = sum dz.
constexpr int LN_BWD_RPB = 32;
int ln_bwd_blocks(int rows);
template <typename T>
hipError_t ln_bwd(const T* dy, const T* xhat, const float* rstd, const float* gamma, T* dz,
                  float* part, int rows, int h, hipStream_t st);

// bf16 stages: the same with dy either one bf16 tensor (ahi = alo = b =
// null) or the fp32 sum (ahi + alo) + b of three bf16 tensors (dy = null):
// a residual branch carried as its bf16 rounding and rounding residual,
// plus a bf16 GEMM product.  dz in bf16 and, when dzlo is not null, dz's
// bf16 rounding residual.  Partials as ln_bwd.
hipError_t ln_bwd_bf16(const bf16_t* dy, const bf16_t* ahi, const bf16_t* alo, const bf16_t* b,
                       const bf16_t* xhat, const float* rstd, const float* gamma, bf16_t* dz,
                       bf16_t* dzlo, float* part, int rows, int h, hipStream_t st);
// out = bf16((ahi + alo) + b), all bf16, n elements (a multiple of 8).
hipError_t add3_bf16(const bf16_t* ahi, const bf16_t* alo, const bf16_t* b, bf16_t* out,
                     int64_t n, hipStream_t st);

// part[blk][n] = sum over the block's rows of x[row][n].
template <typename T>
hipError_t col_partial(const T* x, int rows, int n, float* part, int nblk, hipStream_t st);

// out[c][n] = sum_blk part[blk][c][n] for c < nvec (fixed order).
hipError_t col_reduce(const float* part, int nblk, int nvec, int n, float* const* outs,
                      hipStream_t st);

// ---------------------------------------------------------------------------
// Attention row kernels on a materialised score matrix.
// scores/dP: fp32 [B*H][S][ld]; P, dS: T [B*H][S][ld]; mask: uint8 [B][S].
// ---------------------------------------------------------------------------
template <typename T>
hipError_t softmax_fwd(const float* scores, const uint8_t* mask, T* P, int BH, int H, int S,
                       int ld, float scale, hipStream_t st);
template <typename T>
hipError_t softmax_bwd(const float* dP, const T* P, T* dS, int BH, int S, int ld, float scale,
                       hipStream_t st);

// ---------------------------------------------------------------------------
// Fused attention (bf16 stages, head dim 64).
//   qkv:  [B*S, 3h] (Q | K | V, head j = columns 64 j .. 64 j + 63 of each)
//   mask: [B, S] uint8 key mask; kext: [B] ints, 1 + last valid key
//   out:  forward: context [B*S, h]; backward: dQKV [B*S, 3h]
//   lse:  [B*H, S] fp32 log2-sum-exp of the scaled scores (forward output)
//   o, dout: forward context and its gradient [B*S, h] (backward inputs)
//   out_lo / o_lo: the context's bf16 rounding residual [B*S, h]
//   dsum: [B*H, S] fp32 rowsum(dO * O) (written by attn_backward_dq)
// ---------------------------------------------------------------------------
struct AttnArgs {
  // backward, optional: column sums of dQKV per 32-row block of each
  // sequence, colpart[b * ceil(S / 32) + s / 32][3h]
  float* colpart;
  const bf16_t* qkv;
  const uint8_t* mask;
  const int* kext;
  bf16_t* out;
  float* lse;
  const bf16_t* o;
  const bf16_t* dout;
  // forward, optional: the bf16 rounding residual of the context, out_lo =
  // bf16(C - bf16(C)) with C the fp32 context; backward, optional: the same
  // tensor, added to o where D = rowsum(dO * O) is formed
  bf16_t* out_lo;
  const bf16_t* o_lo;
  float* dsum;
  int B, S, H, h;
  float scale_log2;  // softmax scale * log2(e)
  float scale;       // softmax scale
};
// kext[b] = 1 + last s with mask[b][s] != 0 (0 if none).
hipError_t key_extent(const uint8_t* mask, int B, int S, int* kext, hipStream_t st);
// Forward pass (needs kext).
hipError_t attn_forward(const AttnArgs& a, hipStream_t st);
// dsum and dQ (into out's Q block); must run before attn_backward_dkdv.
hipError_t attn_backward_dq(const AttnArgs& a, hipStream_t st);
// dK and dV (into out's K and V blocks).
hipError_t attn_backward_dkdv(const AttnArgs& a, hipStream_t st);

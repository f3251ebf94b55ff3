// Fused masked self-attention, Eq. (1): softmax(Q K^T / sqrt(d_k)) V with
// d_k = 64, for bf16 stages.  The probability matrix never reaches HBM:
//   forward  : per (batch, head, 128 queries) an online softmax over key
//              blocks; saves the context and the per-row log-sum-exp.
//   backward : two deterministic kernels (no atomics) that recompute P from
//              the saved log-sum-exp:
//              attn_bwd_dq   per 128 queries, loops over keys: D = rowsum(dO*O),
//                            dQ = scale * dS K;
//              attn_bwd_dkdv per 128 keys, loops over queries:
//                            dV = P^T dO, dK = scale * dS^T Q,
//              with dS = P * (dP - D) and dP = dO V^T.
//
// Contractions run on v_mfma_f32_32x32x16_bf16.  Each wavefront owns 32 rows
// (queries or keys).  Scores are produced transposed where the row softmax
// needs them per lane (lane = query, 16 keys in registers), so the
// statistics and the rescaling of the output are per-lane scalars; the fp32
// accumulator registers are converted to bf16 and fed straight back as the
// B operand of the next contraction.  Because a 32x32 accumulator holds rows
// {8*(r/4) + 4*(lane/32) + r%4}, the matching A operand is read from a
// transposed LDS tile with that same row permutation (two 8-byte reads).
#include "kernels.h"

namespace {

constexpr int HD = 64;        // head dimension
constexpr int KT = 64;        // rows per LDS tile (keys or queries)
constexpr int LD = HD + 8;    // padded LDS row (elements) of a [row][dim] tile
constexpr int LDT = KT + 8;   // padded LDS row of a transposed [dim][row] tile

__device__ __forceinline__ f32x16_t mfma32(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Row of register r in a 32x32 accumulator for lane half hf.
__device__ __forceinline__ int acc_row(int r, int hf) { return 8 * (r >> 2) + 4 * hf + (r & 3); }

__device__ __forceinline__ f32x16_t zero16() {
  f32x16_t z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.0f;
  return z;
}

// Registers r0 .. r0+7 of an accumulator as a bf16 operand.
__device__ __forceinline__ bf16x8_t pack8(const f32x16_t& a, int r0) {
  bf16x8_t v;
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (__bf16)a[r0 + i];
  return v;
}

__device__ __forceinline__ bf16x8_t ld_frag(const bf16_t* p) { return *(const bf16x8_t*)p; }

// A operand from a transposed tile Xt[col][row]: column c, contraction step
// ks over the 32 rows starting at row0, in the accumulator row order.
__device__ __forceinline__ bf16x8_t ld_frag_t(const bf16_t* Xt, int c, int row0, int ks, int hf) {
  const bf16_t* p = Xt + c * LDT + row0 + 16 * ks + 4 * hf;
  u32x2_t lo = *(const u32x2_t*)p;
  u32x2_t hi = *(const u32x2_t*)(p + 8);
  u32x4_t v = {lo[0], lo[1], hi[0], hi[1]};
  return __builtin_bit_cast(bf16x8_t, v);
}

__device__ __forceinline__ u32x4_t zero4() { return u32x4_t{0, 0, 0, 0}; }

// Copy rows [r0, r0 + KT) of a [rows][64] bf16 matrix (row stride ld,
// rows >= nrows read as zero) into the LDS tile X[KT][LD].
__device__ __forceinline__ void load_rows(const bf16_t* __restrict__ src, int64_t ld, int r0,
                                          int nrows, bf16_t* X) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < KT * 8 / 256; ++i) {
    int v = tid + 256 * i;
    int row = v >> 3, c8 = (v & 7) * 8;
    u32x4_t val = zero4();
    if (r0 + row < nrows) val = *(const u32x4_t*)(src + (int64_t)(r0 + row) * ld + c8);
    *(u32x4_t*)(X + row * LD + c8) = val;
  }
}

// Same rows into the transposed LDS tile Xt[64][LDT]: each of 128 threads
// moves a block of 4 rows x 8 columns and transposes it in registers.
__device__ __forceinline__ void load_rows_t(const bf16_t* __restrict__ src, int64_t ld, int r0,
                                            int nrows, bf16_t* Xt) {
  const int tid = threadIdx.x;
  if (tid < KT / 4 * 8) {
    const int rb = tid % (KT / 4), cb = tid / (KT / 4);
    u32x4_t v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int row = r0 + rb * 4 + j;
      v[j] = row < nrows ? *(const u32x4_t*)(src + (int64_t)row * ld + cb * 8) : zero4();
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int w = c >> 1, sh = (c & 1) * 16;
      uint32_t e0 = (v[0][w] >> sh) & 0xffffu, e1 = (v[1][w] >> sh) & 0xffffu;
      uint32_t e2 = (v[2][w] >> sh) & 0xffffu, e3 = (v[3][w] >> sh) & 0xffffu;
      u32x2_t o = {e0 | (e1 << 16), e2 | (e3 << 16)};
      *(u32x2_t*)(Xt + (cb * 8 + c) * LDT + rb * 4) = o;
    }
  }
}

// Write a wavefront's 32 x 64 result, held transposed in two accumulators
// (lane = row l % 32, registers = columns), to dst rows [row0, row0 + 32)
// clipped to nrows: staged through the wavefront's LDS area (32 x LD) so
// that the global stores are 16-byte row segments.  If colsum is not null it
// receives the 64 column sums of the stored (bf16) values of those rows.
__device__ __forceinline__ void store_rows_t(const f32x16_t acc[2], float mul, bf16_t* stage,
                                             bf16_t* __restrict__ dst, int64_t ld, int row0,
                                             int nrows, float* colsum) {
  const int lane = threadIdx.x & 63, hf = lane >> 5, rr = lane & 31;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      // registers 4q .. 4q+3 are 4 consecutive columns
      const int col = 32 * t + 8 * q + 4 * hf;
      uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[t][4 * q] * mul)) |
                    ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[t][4 * q + 1] * mul)) << 16);
      uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[t][4 * q + 2] * mul)) |
                    ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)(acc[t][4 * q + 3] * mul)) << 16);
      *(u32x2_t*)(stage + rr * LD + col) = u32x2_t{lo, hi};
    }
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
  // lane owns column chunk (lane & 7) * 8 and rows (lane >> 3) + 8 i
  float cs[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int c = lane + 64 * i;
    int row = c >> 3, c8 = (c & 7) * 8;
    if (row0 + row < nrows) {
      const u32x4_t v = *(const u32x4_t*)(stage + row * LD + c8);
      *(u32x4_t*)(dst + (int64_t)(row0 + row) * ld + c8) = v;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        cs[2 * e] += __uint_as_float(v[e] << 16);
        cs[2 * e + 1] += __uint_as_float(v[e] & 0xffff0000u);
      }
    }
  }
  if (colsum) {
    // lanes with equal lane & 7 hold the same columns: fixed-order sum
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      cs[e] += __shfl_xor(cs[e], 8, 64);
      cs[e] += __shfl_xor(cs[e], 16, 64);
      cs[e] += __shfl_xor(cs[e], 32, 64);
    }
    if (lane < 8) {
      *(f32x4_t*)(colsum + lane * 8) = f32x4_t{cs[0], cs[1], cs[2], cs[3]};
      *(f32x4_t*)(colsum + lane * 8 + 4) = f32x4_t{cs[4], cs[5], cs[6], cs[7]};
    }
  }
}

// Key extent per sequence: 1 + the last key position with mask != 0 (0 if
// none).  Keys at or past it are never attended, so loops stop there.
__global__ __launch_bounds__(256) void key_extent_kernel(const uint8_t* __restrict__ mask, int S,
                                                         int* __restrict__ kext) {
  __shared__ int sm[4];
  const int b = blockIdx.x;
  int last = 0;
  for (int s = threadIdx.x; s < S; s += 256)
    if (mask[(int64_t)b * S + s]) last = max(last, s + 1);
  for (int o = 32; o > 0; o >>= 1) last = max(last, __shfl_xor(last, o, 64));
  if ((threadIdx.x & 63) == 0) sm[threadIdx.x >> 6] = last;
  __syncthreads();
  if (threadIdx.x == 0) kext[b] = max(max(sm[0], sm[1]), max(sm[2], sm[3]));
}

// ---------------------------------------------------------------------------
// Forward: wavefront = 32 queries; block = 128 queries of one (batch, head).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256, 4) void attn_fwd_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t Ks[KT * LD];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[HD * LDT];
  __shared__ uint8_t ms[KT];
  __shared__ __attribute__((aligned(16))) bf16_t stage[4][32 * LD];

  const int bh = blockIdx.y, b = bh / a.H, j = bh % a.H;
  const int S = a.S, h = a.h;
  const int64_t ld = 3 * (int64_t)h;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hf = lane >> 5, rr = lane & 31;
  const int q0 = blockIdx.x * 128 + wave * 32;
  const bf16_t* __restrict__ Qg = a.qkv + (int64_t)b * S * ld + j * HD;
  const bf16_t* __restrict__ Kg = Qg + h;
  const bf16_t* __restrict__ Vg = Qg + 2 * h;
  const uint8_t* __restrict__ mrow = a.mask + (int64_t)b * S;
  const int kend = a.kext[b];

  // Q^T as the B operand: lane = query q0 + rr, dims 16 ks + 8 hf .. +7.
  bf16x8_t qf[4];
  {
    const int q = q0 + rr;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      qf[ks] = q < S ? ld_frag(Qg + (int64_t)q * ld + 16 * ks + 8 * hf)
                     : __builtin_bit_cast(bf16x8_t, zero4());
  }
  float m = -INFINITY, lsum = 0.0f;  // running max (log2 units) and partial sum
  f32x16_t acc[2] = {zero16(), zero16()};  // O^T: dims 0-31, 32-63 x queries

  for (int kb0 = 0; kb0 < kend; kb0 += KT) {
    __syncthreads();
    load_rows(Kg, ld, kb0, S, Ks);
    load_rows_t(Vg, ld, kb0, S, Vt);
    if (tid < KT) ms[tid] = (kb0 + tid < kend) ? mrow[kb0 + tid] : 0;
    __syncthreads();
#pragma unroll
    for (int sub = 0; sub < KT / 32; ++sub) {
      if (kb0 + 32 * sub >= kend) break;
      // S^T (32 keys x 32 queries) = K_sub Q^T
      f32x16_t s = zero16();
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        s = mfma32(ld_frag(Ks + (32 * sub + rr) * LD + 16 * ks + 8 * hf), qf[ks], s);
      float mblk = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const bool valid = ms[32 * sub + acc_row(r, hf)] != 0;
        s[r] = valid ? s[r] * a.scale_log2 : -INFINITY;
        mblk = fmaxf(mblk, s[r]);
      }
      mblk = fmaxf(mblk, __shfl_xor(mblk, 32, 64));
      const float mnew = fmaxf(m, mblk);
      const float off = mnew == -INFINITY ? 0.0f : mnew;
      const float alpha = __builtin_amdgcn_exp2f(m - off);
      float ps = 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] = __builtin_amdgcn_exp2f(s[r] - off);
        ps += s[r];
      }
      lsum = lsum * alpha + ps;
      m = mnew;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][r] *= alpha;
      // O^T += V_sub^T P^T
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8_t pb = pack8(s, 8 * ks);
#pragma unroll
        for (int t = 0; t < 2; ++t)
          acc[t] = mfma32(ld_frag_t(Vt, 32 * t + rr, 32 * sub, ks, hf), pb, acc[t]);
      }
    }
  }
  const float ltot = lsum + __shfl_xor(lsum, 32, 64);
  const float inv = ltot > 0.0f ? 1.0f / ltot : 0.0f;
  if (hf == 0 && q0 + rr < S)
    a.lse[(int64_t)bh * S + q0 + rr] = ltot > 0.0f ? m + __log2f(ltot) : 0.0f;
  store_rows_t(acc, inv, stage[wave], a.out + (int64_t)b * S * h + j * HD, h, q0, S, nullptr);
}

// ---------------------------------------------------------------------------
// Backward, dQ: wavefront = 32 queries; loops over key blocks.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256, 3) void attn_bwd_dq_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t Ks[KT * LD];
  __shared__ __attribute__((aligned(16))) bf16_t Kt[HD * LDT];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[KT * LD];
  __shared__ uint8_t ms[KT];
  __shared__ __attribute__((aligned(16))) bf16_t stage[4][32 * LD];

  const int bh = blockIdx.y, b = bh / a.H, j = bh % a.H;
  const int S = a.S, h = a.h;
  const int64_t ld = 3 * (int64_t)h;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hf = lane >> 5, rr = lane & 31;
  const int q0 = blockIdx.x * 128 + wave * 32;
  const bf16_t* __restrict__ Qg = a.qkv + (int64_t)b * S * ld + j * HD;
  const bf16_t* __restrict__ Kg = Qg + h;
  const bf16_t* __restrict__ Vg = Qg + 2 * h;
  const bf16_t* __restrict__ Og = a.o + (int64_t)b * S * h + j * HD;
  const bf16_t* __restrict__ dOg = a.dout + (int64_t)b * S * h + j * HD;
  const uint8_t* __restrict__ mrow = a.mask + (int64_t)b * S;
  const int kend = a.kext[b];
  const int q = q0 + rr;

  bf16x8_t qf[4], dof[4];
  float dsum = 0.0f;
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const int c = 16 * ks + 8 * hf;
    bf16x8_t of;
    if (q < S) {
      qf[ks] = ld_frag(Qg + (int64_t)q * ld + c);
      dof[ks] = ld_frag(dOg + (int64_t)q * h + c);
      of = ld_frag(Og + (int64_t)q * h + c);
    } else {
      qf[ks] = dof[ks] = of = __builtin_bit_cast(bf16x8_t, zero4());
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) dsum += (float)dof[ks][i] * (float)of[i];
  }
  dsum += __shfl_xor(dsum, 32, 64);  // D = rowsum(dO * O) of query q
  if (hf == 0 && q < S) a.dsum[(int64_t)bh * S + q] = dsum;
  const float lse_q = q < S ? a.lse[(int64_t)bh * S + q] : 0.0f;

  f32x16_t dq[2] = {zero16(), zero16()};  // dQ^T: dims x queries
  for (int kb0 = 0; kb0 < kend; kb0 += KT) {
    __syncthreads();
    load_rows(Kg, ld, kb0, S, Ks);
    load_rows_t(Kg, ld, kb0, S, Kt);
    load_rows(Vg, ld, kb0, S, Vs);
    if (tid < KT) ms[tid] = (kb0 + tid < kend) ? mrow[kb0 + tid] : 0;
    __syncthreads();
#pragma unroll
    for (int sub = 0; sub < KT / 32; ++sub) {
      if (kb0 + 32 * sub >= kend) break;
      f32x16_t s = zero16(), dp = zero16();
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        s = mfma32(ld_frag(Ks + (32 * sub + rr) * LD + 16 * ks + 8 * hf), qf[ks], s);
        dp = mfma32(ld_frag(Vs + (32 * sub + rr) * LD + 16 * ks + 8 * hf), dof[ks], dp);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const bool valid = ms[32 * sub + acc_row(r, hf)] != 0;
        const float p = valid ? __builtin_amdgcn_exp2f(s[r] * a.scale_log2 - lse_q) : 0.0f;
        s[r] = p * (dp[r] - dsum);  // dS^T (unscaled)
      }
      // dQ^T += K^T dS^T
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8_t db = pack8(s, 8 * ks);
#pragma unroll
        for (int t = 0; t < 2; ++t)
          dq[t] = mfma32(ld_frag_t(Kt, 32 * t + rr, 32 * sub, ks, hf), db, dq[t]);
      }
    }
  }
  const int nqb = (S + 31) / 32;
  float* cp = (a.colpart && q0 < S) ? a.colpart + ((int64_t)b * nqb + q0 / 32) * ld + j * HD : nullptr;
  store_rows_t(dq, a.scale, stage[wave], a.out + (int64_t)b * S * ld + j * HD, ld, q0, S, cp);
}

// ---------------------------------------------------------------------------
// Backward, dK and dV: wavefront = 32 keys; loops over query blocks.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256, 2) void attn_bwd_dkdv_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t Qs[KT * LD];
  __shared__ __attribute__((aligned(16))) bf16_t Qt[HD * LDT];
  __shared__ __attribute__((aligned(16))) bf16_t dOs[KT * LD];
  __shared__ __attribute__((aligned(16))) bf16_t dOt[HD * LDT];
  __shared__ float lse_s[KT], d_s[KT];

  const int bh = blockIdx.y, b = bh / a.H, j = bh % a.H;
  const int S = a.S, h = a.h;
  const int64_t ld = 3 * (int64_t)h;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hf = lane >> 5, rr = lane & 31;
  const int k0 = blockIdx.x * 128 + wave * 32;
  const bf16_t* __restrict__ Qg = a.qkv + (int64_t)b * S * ld + j * HD;
  const bf16_t* __restrict__ Kg = Qg + h;
  const bf16_t* __restrict__ Vg = Qg + 2 * h;
  const bf16_t* __restrict__ dOg = a.dout + (int64_t)b * S * h + j * HD;
  const int kend = a.kext[b];
  const int key = k0 + rr;
  const bool kvalid = key < kend && a.mask[(int64_t)b * S + key] != 0;
  const bool block_live = blockIdx.x * 128 < kend;  // uniform over the block

  bf16x8_t kf[4], vf[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const int c = 16 * ks + 8 * hf;
    if (key < S) {
      kf[ks] = ld_frag(Kg + (int64_t)key * ld + c);
      vf[ks] = ld_frag(Vg + (int64_t)key * ld + c);
    } else {
      kf[ks] = vf[ks] = __builtin_bit_cast(bf16x8_t, zero4());
    }
  }
  f32x16_t dv[2] = {zero16(), zero16()}, dk[2] = {zero16(), zero16()};  // dims x keys

  for (int qb0 = 0; block_live && qb0 < S; qb0 += KT) {
    __syncthreads();
    load_rows(Qg, ld, qb0, S, Qs);
    load_rows_t(Qg, ld, qb0, S, Qt);
    load_rows(dOg, h, qb0, S, dOs);
    load_rows_t(dOg, h, qb0, S, dOt);
    if (tid < KT) {
      const int qq = qb0 + tid;
      lse_s[tid] = qq < S ? a.lse[(int64_t)bh * S + qq] : INFINITY;
      d_s[tid] = qq < S ? a.dsum[(int64_t)bh * S + qq] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int sub = 0; sub < KT / 32; ++sub) {
      if (qb0 + 32 * sub >= S) break;
      // S (32 queries x 32 keys) = Q_sub K^T;  dP = dO_sub V^T
      f32x16_t s = zero16(), dp = zero16();
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        s = mfma32(ld_frag(Qs + (32 * sub + rr) * LD + 16 * ks + 8 * hf), kf[ks], s);
        dp = mfma32(ld_frag(dOs + (32 * sub + rr) * LD + 16 * ks + 8 * hf), vf[ks], dp);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qi = 32 * sub + acc_row(r, hf);
        const float p = kvalid ? __builtin_amdgcn_exp2f(s[r] * a.scale_log2 - lse_s[qi]) : 0.0f;
        s[r] = p;
        dp[r] = p * (dp[r] - d_s[qi]);  // dS (unscaled)
      }
      // dV^T += dO^T P;  dK^T += Q^T dS
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8_t pb = pack8(s, 8 * ks);
        const bf16x8_t db = pack8(dp, 8 * ks);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          dv[t] = mfma32(ld_frag_t(dOt, 32 * t + rr, 32 * sub, ks, hf), pb, dv[t]);
          dk[t] = mfma32(ld_frag_t(Qt, 32 * t + rr, 32 * sub, ks, hf), db, dk[t]);
        }
      }
    }
  }
  __syncthreads();
  // Stage the outputs through the (now free) Q tiles: 4 waves x 32 x LD.
  bf16_t* stage = (wave < 2 ? Qs : dOs) + (wave & 1) * 32 * LD;
  bf16_t* dst = a.out + (int64_t)b * S * ld + j * HD;
  const int nqb = (S + 31) / 32;
  float* cp = (a.colpart && k0 < S) ? a.colpart + ((int64_t)b * nqb + k0 / 32) * ld + j * HD : nullptr;
  store_rows_t(dk, a.scale, stage, dst + h, ld, k0, S, cp ? cp + h : nullptr);
  __builtin_amdgcn_wave_barrier();
  store_rows_t(dv, 1.0f, stage, dst + 2 * h, ld, k0, S, cp ? cp + 2 * h : nullptr);
}

}  // namespace

hipError_t key_extent(const uint8_t* mask, int B, int S, int* kext, hipStream_t st) {
  if (B == 0 || S == 0) return hipSuccess;
  hipLaunchKernelGGL(key_extent_kernel, dim3(B), dim3(256), 0, st, mask, S, kext);
  return hipGetLastError();
}

hipError_t attn_forward(const AttnArgs& a, hipStream_t st) {
  if (a.B == 0 || a.S == 0) return hipSuccess;
  dim3 grid((a.S + 127) / 128, a.B * a.H);
  hipLaunchKernelGGL(attn_fwd_kernel, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t attn_backward_dq(const AttnArgs& a, hipStream_t st) {
  if (a.B == 0 || a.S == 0) return hipSuccess;
  dim3 grid((a.S + 127) / 128, a.B * a.H);
  hipLaunchKernelGGL(attn_bwd_dq_kernel, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t attn_backward_dkdv(const AttnArgs& a, hipStream_t st) {
  if (a.B == 0 || a.S == 0) return hipSuccess;
  dim3 grid((a.S + 127) / 128, a.B * a.H);
  hipLaunchKernelGGL(attn_bwd_dkdv_kernel, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

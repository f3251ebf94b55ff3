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
// B operand of the next contraction.  The streamed 64-row blocks (keys and
// values, or queries and output gradients) go from HBM straight into a
// two-stage LDS ring with direct-to-LDS loads, one block ahead of the one
// being used.  Their row-major tiles serve both operand shapes: row
// fragments with 16-byte reads, and the transposed operand that multiplies an
// accumulator-held matrix with gfx950's transposing LDS read, taking the
// accumulator's row order {8*(r/4) + 4*(lane/32) + r%4} directly.

#include "kernels.h"

namespace {

constexpr int HD = 64;               // head dimension
constexpr int KT = 64;               // rows per streamed block
constexpr int TILE = KT * HD * 2;    // bytes of one [64][64] bf16 tile
constexpr int LD = HD + 8;           // padded row (elements) of the output staging area

typedef __attribute__((address_space(3))) void lds_void_t;

__device__ __forceinline__ f32x16_t mfma32(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Row of register r in a 32x32 accumulator for lane half hf.
__device__ __forceinline__ int acc_row(int r, int hf) { return 8 * (r >> 2) + 4 * hf + (r & 3); }

__device__ __forceinline__ f32x16_t splat16(float v) {
  f32x16_t z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = v;
  return z;
}

__device__ __forceinline__ f32x16_t zero16() {
  f32x16_t z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.0f;
  return z;
}

// Registers r0 .. r0+7 of an accumulator as a bf16 operand.
__device__ __forceinline__ bf16x8_t pack8(const f32x16_t& a, int r0) {
  const u32x4_t w = {pack_bf16x2(a[r0], a[r0 + 1]), pack_bf16x2(a[r0 + 2], a[r0 + 3]),
                     pack_bf16x2(a[r0 + 4], a[r0 + 5]), pack_bf16x2(a[r0 + 6], a[r0 + 7])};
  return __builtin_bit_cast(bf16x8_t, w);
}

// The bf16 rounding residuals a[r] - hi[r] of registers r0 .. r0+7, where
// hi = pack8(a, r0), as a bf16 operand.
__device__ __forceinline__ bf16x8_t pack8_residual(const f32x16_t& a, int r0, bf16x8_t hi) {
  const u32x4_t h = __builtin_bit_cast(u32x4_t, hi);
  u32x4_t w;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = pack_bf16x2(a[r0 + 2 * i] - __uint_as_float(h[i] << 16),
                       a[r0 + 2 * i + 1] - __uint_as_float(h[i] & 0xffff0000u));
  return __builtin_bit_cast(bf16x8_t, w);
}

__device__ __forceinline__ bf16x8_t ld_frag(const bf16_t* p) { return *(const bf16x8_t*)p; }

__device__ __forceinline__ u32x4_t zero4() { return u32x4_t{0, 0, 0, 0}; }

// LDS tile [64 rows][64 bf16]: 128-byte rows of 8 16-byte chunks, chunk c of
// row r stored at chunk c ^ f(u), u = (r >> 1) & 7, f(u) = (u0 << 2) |
// (u2 << 1) | u1.  The 16 rows of a row-fragment read and the 4 rows x 64
// bytes of a transposing read then fall on distinct banks.
__device__ __forceinline__ int tswz(int r) {
  const int u = (r >> 1) & 7;
  return ((u & 1) << 2) | (((u >> 2) & 1) << 1) | ((u >> 1) & 1);
}
__device__ __forceinline__ int toff(int r, int c) { return r * 128 + 16 * (c ^ tswz(r)); }

// Buffer resource over rows 0 .. n-1 of a [rows][64] bf16 operand with row
// stride ld elements: loads of later rows return 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const bf16_t* base, int n, int64_t ld) {
  const int64_t bytes = n > 0 ? ((int64_t)(n - 1) * ld + HD) * 2 : 0;
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0,
                                           (int)(bytes > 0x7fffffff ? 0x7fffffff : bytes),
                                           0x00020000);
}

// Rows [row0, row0 + NR) into a tile with direct-to-LDS loads: NR / 8 loads
// of 8 rows (lane l's 16 bytes land at +16 l), NR / 32 per wavefront.
template <int NR = KT>
__device__ __forceinline__ void dma_rows(__amdgpu_buffer_rsrc_t rs, int row0, int64_t ld,
                                         char* tile, int wave, int lane) {
#pragma unroll
  for (int i = 0; i < NR / 32; ++i) {
    const int q = (NR / 32) * wave + i;
    const int r = 8 * q + (lane >> 3);
    const int c = (lane & 7) ^ tswz(r);
    const int64_t off = ((int64_t)(row0 + r) * ld + 8 * c) * 2;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)(tile + q * 1024), 16,
                                             (int)(off > 0x7fffffff ? 0x7fffffff : off), 0, 0, 0);
  }
}

// A operand from tile rows: lane l reads row r0 + l % 32, columns
// 16 ks + 8 (l / 32) .. +7.
__device__ __forceinline__ bf16x8_t frag_rows(const char* tile, int r0, int ks, int lane) {
  return *(const bf16x8_t*)(tile + toff(r0 + (lane & 31), 2 * ks + (lane >> 5)));
}

// Transposed A operand: lane l gets column col0 + l % 32 at the tile rows
// rb + 4 hf + {0..3} and rb + 8 + 4 hf + {0..3} (hf = l / 32), which with
// rb = row base + 16 ks is the row order of accumulator registers
// 8 ks .. 8 ks + 7.  ds_read_b64_tr_b16 works on groups of 16 lanes: lane j
// supplies the address of 4 consecutive 16-bit values V[j][0..3] and lane i
// receives V[4e + i / 4][i % 4], e = 0..3; lane j points at row
// rb + 4 hf + j / 4, columns c0 + 4 (j % 4) .. +3, so lane i receives column
// c0 + i of those 4 rows.
__device__ __forceinline__ bf16x8_t frag_tr(const char* tile, int col0, int rb, int lane) {
  typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;
  const int j = lane & 15;
  const int r = rb + 4 * (lane >> 5) + (j >> 2);
  const int d = col0 + 16 * ((lane >> 4) & 1) + 4 * (j & 3);
  const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (lds_bf16x4_t*)(tile + toff(r, d >> 3) + 2 * (d & 7)));
  const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (lds_bf16x4_t*)(tile + toff(r + 8, d >> 3) + 2 * (d & 7)));
  return bf16x8_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

// "vmcnt = 0 and lgkmcnt = 0" (gfx9 s_waitcnt encoding).
__device__ __forceinline__ void wait_all() { __builtin_amdgcn_s_waitcnt(0x0070); }

// The values of lanes l and l ^ 32 (as a pair, in either order) from one
// v_permlane32_swap, which exchanges the upper half of its first operand
// with the lower half of its second: no LDS round trip, unlike a shuffle.
struct HalfPair {
  float x, y;
};
__device__ __forceinline__ HalfPair half_pair(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return {__uint_as_float(r[0]), __uint_as_float(r[1])};
}

// Write a wavefront's 32 x 64 result, held transposed in two accumulators
// (lane = row l % 32, registers = columns), to dst rows [row0, row0 + 32)
// clipped to nrows: staged through the wavefront's LDS area (32 x LD) so
// that the global stores are 16-byte row segments.  If colsum is not null it
// receives the 64 column sums of the stored (bf16) values of those rows.
// With residual, the values stored are the bf16 rounding residuals
// v - bf16(v) of the scaled accumulators (rounded to bf16 in turn), so that
// the pair (stored, residual) holds v to about 16 significant bits.
__device__ __forceinline__ float bf16_residual(float v) {
  return v - __uint_as_float(pack_bf16x2(v, v) << 16);
}
__device__ __forceinline__ void store_rows_t(const f32x16_t acc[2], float mul, bf16_t* stage,
                                             bf16_t* __restrict__ dst, int64_t ld, int row0,
                                             int nrows, float* colsum, bool residual = false) {
  const int lane = threadIdx.x & 63, hf = lane >> 5, rr = lane & 31;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      // registers 4q .. 4q+3 are 4 consecutive columns
      const int col = 32 * t + 8 * q + 4 * hf;
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] = acc[t][4 * q + e] * mul;
        if (residual) v[e] = bf16_residual(v[e]);
      }
      const uint32_t lo = pack_bf16x2(v[0], v[1]);
      const uint32_t hi = pack_bf16x2(v[2], v[3]);
      *(u32x2_t*)(stage + rr * LD + col) = u32x2_t{lo, hi};
    }
  // The staged values must be in LDS before other lanes read them; global
  // stores still in flight (a previous call's) need not be waited for.
  lds_wait();
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

// Work-group -> (row block, batch * head).  The grid is one-dimensional,
// nq row blocks per (batch, head); consecutive work-groups go round robin
// over the 8 XCDs, so they are remapped such that each XCD takes a
// contiguous range and the row blocks of one (batch, head), which stream the
// same keys and values (or queries and output gradients), share that XCD's
// L2.
__device__ __forceinline__ void attn_block(int nq, int& rb, int& bh) {
  const int n = gridDim.x;
  int w = blockIdx.x;
  if ((n & 7) == 0) w = (w & 7) * (n >> 3) + (w >> 3);
  rb = w % nq;
  bh = w / nq;
}

// Called by all 64 lanes of wavefront 0 with the bias (0 or -inf) of key
// `lane` of a 64-key block: flags[i] = 1 if none of keys 32 i .. 32 i + 31
// is masked.
__device__ __forceinline__ void store_kfull(int* flags, float bias, int lane) {
  const uint64_t ok = __ballot(bias == 0.0f);
  if (lane == 0) {
    flags[0] = (uint32_t)ok == 0xffffffffu;
    flags[1] = (uint32_t)(ok >> 32) == 0xffffffffu;
  }
}

// A kernel's LDS is one object.  With several __shared__ variables the
// compiler tags each access with the variable's alias scope and then makes
// the first LDS read after a direct-to-LDS load wait for that load
// (vmcnt(0)), although the read is of the other stage: the next block's
// loads then completed before the current block's first MFMA instead of
// under its work.  With a single object it does not for the 16-byte
// fragment reads (measured in the assembly); the transposing-read builtin
// still waits, at the first sub-block's second product.  The kernels' own
// waits (wait_all and the barrier at each block) order every read after the
// loads it depends on.  Same harness and box, medians of three: forward
// -1.6%, dQ -2.7%, dQ then dK/dV -3.2% (with the set-up and per-block load
// order below; reading the transposed fragments as inline assembly to avoid
// the builtin's wait was slower).
struct LdsKV {
  char tiles[2][2 * TILE];  // per stage: K, V
  float kbias[2][KT];       // per stage: 0 or -inf per key
  int kfull[2][2];          // per stage and 32-key half: no key masked
};

// ---------------------------------------------------------------------------
// Forward: wavefront = 32 queries; block = 128 queries of one (batch, head).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256, 4) void attn_fwd_kernel(AttnArgs a) {
  // One LDS object (see LdsKV): K, V per stage; key bias 0 or -inf per key;
  // per stage and 32-key half, whether no key is masked.
  __shared__ __attribute__((aligned(1024))) LdsKV lds;
  auto& tiles = lds.tiles;
  auto& kbias = lds.kbias;
  auto& kfull = lds.kfull;

  int qb, bh;
  attn_block((a.S + 127) / 128, qb, bh);
  const int b = bh / a.H, j = bh % a.H;
  const int S = a.S, h = a.h;
  const int64_t ld = 3 * (int64_t)h;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hf = lane >> 5, rr = lane & 31;
  const int q0 = qb * 128 + wave * 32;
  const bf16_t* __restrict__ Qg = a.qkv + (int64_t)b * S * ld + j * HD;
  const bf16_t* __restrict__ Kg = Qg + h;
  const bf16_t* __restrict__ Vg = Qg + 2 * h;
  const uint8_t* __restrict__ mrow = a.mask + (int64_t)b * S;
  const int kend = a.kext[b];
  const int nkb = (kend + KT - 1) / KT;
  const __amdgpu_buffer_rsrc_t rsK = rows_rsrc(Kg, S, ld), rsV = rows_rsrc(Vg, S, ld);
  // Mask byte of key kb KT + tid (clamped to a valid key, so that the load
  // is unconditional) and the key bias it gives (0 or -inf).  Wavefront 0
  // loads the bytes of block kb + 2 during block kb and turns them into the
  // bias of block kb + 2 at the end of block kb + 1, after the wait at that
  // block's start: using them in the block that loads them made it wait a
  // memory latency per block, and the other wavefronts then waited for it at
  // the next barrier.
  auto mask_raw = [&](int kb) { return (int)mrow[min(kb * KT + tid, S - 1)]; };
  auto bias_from = [&](int kb, int raw) {
    return (kb * KT + tid < kend && raw != 0) ? 0.0f : -INFINITY;
  };
  auto bias_of = [&](int kb) { return bias_from(kb, mask_raw(kb)); };

  // Set-up loads in the order that lets their latencies overlap: the
  // wavefront's own operand fragments, the first streamed block, and only
  // then the key-mask bytes, whose values the LDS set-up waits for.
  // Q^T as the B operand: lane = query q0 + rr, dims 16 ks + 8 hf .. +7.
  bf16x8_t qf[4];
  {
    const int q = q0 + rr;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      qf[ks] = q < S ? ld_frag(Qg + (int64_t)q * ld + 16 * ks + 8 * hf)
                     : __builtin_bit_cast(bf16x8_t, zero4());
  }
  if (nkb > 0) {
    dma_rows(rsK, 0, ld, tiles[0], wave, lane);
    dma_rows(rsV, 0, ld, tiles[0] + TILE, wave, lane);
    if (tid < KT) {  // wavefront 0
      const float kb0 = bias_of(0);
      kbias[0][tid] = kb0;
      store_kfull(kfull[0], kb0, tid);
    }
  }
  int nraw = (tid < KT && nkb > 1) ? mask_raw(1) : 0;  // bytes of the next block
  float m = -INFINITY, lsum = 0.0f;  // exponent offset (log2 units) and partial sum
  f32x16_t acc[2] = {zero16(), zero16()};  // O^T: dims 0-31, 32-63 x queries

  for (int kb = 0; kb < nkb; ++kb) {
    const int st = kb & 1;
    // Block kb has landed (each wavefront waits for its own loads, the
    // barrier for everyone's) and nobody reads the other stage any more.
    wait_all();
    __syncthreads();
    if (kb + 1 < nkb) {
      dma_rows(rsK, (kb + 1) * KT, ld, tiles[st ^ 1], wave, lane);
      dma_rows(rsV, (kb + 1) * KT, ld, tiles[st ^ 1] + TILE, wave, lane);
    }
    const int nraw2 = (tid < KT && kb + 2 < nkb) ? mask_raw(kb + 2) : 0;
    const char* Ks = tiles[st];
    const char* Vs = tiles[st] + TILE;
#pragma unroll
    for (int sub = 0; sub < KT / 32; ++sub) {
      if (kb * KT + 32 * sub >= kend) break;
      // S^T (32 keys x 32 queries) = K_sub Q^T
      f32x16_t s = zero16();
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) s = mfma32(frag_rows(Ks, 32 * sub, ks, lane), qf[ks], s);
      // No masked key in these 32: the scale is applied inside the exponent
      // below (the block maximum scales with it); else the scaled scores
      // get the key bias (0 or -inf) here.
      const bool full = __builtin_amdgcn_readfirstlane(kfull[st][sub]) != 0;
      const float c = full ? a.scale_log2 : 1.0f;
      float mblk = -INFINITY;
      if (full) {
#pragma unroll
        for (int r = 0; r < 16; ++r) mblk = fmaxf(mblk, s[r]);
        mblk *= a.scale_log2;
      } else {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4_t kbv = *(const f32x4_t*)&kbias[st][32 * sub + 8 * g + 4 * hf];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            s[4 * g + e] = fmaf(s[4 * g + e], a.scale_log2, kbv[e]);
            mblk = fmaxf(mblk, s[4 * g + e]);
          }
        }
      }
      {
        const HalfPair pr = half_pair(mblk);
        mblk = fmaxf(pr.x, pr.y);
      }
      // The exponent offset m moves only when a block maximum exceeds it by
      // more than 8 (log2 units), so exp2(s - m) <= 256 and most blocks
      // skip rescaling the output accumulators (a wavefront-uniform test).
      const bool grow = mblk > m + 8.0f;
      if (__any(grow)) {
        const float mn = grow ? mblk : m;
        const float alpha = __builtin_amdgcn_exp2f(m - (mn == -INFINITY ? 0.0f : mn));
        lsum *= alpha;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[t][r] *= alpha;
        m = mn;
      }
      const float off = m == -INFINITY ? 0.0f : m;
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = __builtin_amdgcn_exp2f(fmaf(s[r], c, -off));
      float ps = s[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) ps += s[r];
      lsum += ps;
      // O^T += V_sub^T P^T, P as its bf16 value plus its bf16 rounding
      // residual (two MFMAs on one V fragment): the context then carries
      // about 16 significant bits of P, which the backward's D = rowsum(dO
      // O) needs to match the rows of P dP it is subtracted from.
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8_t pb = pack8(s, 8 * ks);
        const bf16x8_t pl = pack8_residual(s, 8 * ks, pb);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const bf16x8_t vf = frag_tr(Vs, 32 * t, 32 * sub + 16 * ks, lane);
          acc[t] = mfma32(vf, pb, acc[t]);
          acc[t] = mfma32(vf, pl, acc[t]);
        }
      }
    }
    if (kb + 1 < nkb && tid < KT) {
      const float nbias = bias_from(kb + 1, nraw);
      kbias[st ^ 1][tid] = nbias;
      store_kfull(kfull[st ^ 1], nbias, tid);
    }
    nraw = nraw2;
  }
  const HalfPair lp = half_pair(lsum);
  const float ltot = lp.x + lp.y;
  const float inv = ltot > 0.0f ? 1.0f / ltot : 0.0f;
  if (hf == 0 && q0 + rr < S)
    a.lse[(int64_t)bh * S + q0 + rr] = ltot > 0.0f ? m + __log2f(ltot) : 0.0f;
  __syncthreads();  // the ring becomes the output staging area
  bf16_t* stage = (bf16_t*)&tiles[0][0] + wave * 32 * LD;
  store_rows_t(acc, inv, stage, a.out + (int64_t)b * S * h + j * HD, h, q0, S, nullptr);
  if (a.out_lo) {
    lds_wait();
    __builtin_amdgcn_wave_barrier();
    store_rows_t(acc, inv, stage, a.out_lo + (int64_t)b * S * h + j * HD, h, q0, S, nullptr, true);
  }
}

// ---------------------------------------------------------------------------
// Backward, dQ: wavefront = 32 queries; loops over key blocks.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256, 3) void attn_bwd_dq_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) LdsKV lds;  // as in the forward
  auto& tiles = lds.tiles;
  auto& kbias = lds.kbias;
  auto& kfull = lds.kfull;

  int qb, bh;
  attn_block((a.S + 127) / 128, qb, bh);
  const int b = bh / a.H, j = bh % a.H;
  const int S = a.S, h = a.h;
  const int64_t ld = 3 * (int64_t)h;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hf = lane >> 5, rr = lane & 31;
  const int q0 = qb * 128 + wave * 32;
  const bf16_t* __restrict__ Qg = a.qkv + (int64_t)b * S * ld + j * HD;
  const bf16_t* __restrict__ Kg = Qg + h;
  const bf16_t* __restrict__ Vg = Qg + 2 * h;
  const bf16_t* __restrict__ Og = a.o + (int64_t)b * S * h + j * HD;
  const bf16_t* __restrict__ dOg = a.dout + (int64_t)b * S * h + j * HD;
  const uint8_t* __restrict__ mrow = a.mask + (int64_t)b * S;
  const int kend = a.kext[b];
  const int nkb = (kend + KT - 1) / KT;
  const int q = q0 + rr;
  const __amdgpu_buffer_rsrc_t rsK = rows_rsrc(Kg, S, ld), rsV = rows_rsrc(Vg, S, ld);
  // Mask byte of key kb KT + tid (clamped to a valid key, so that the load
  // is unconditional) and the key bias it gives (0 or -inf).  Wavefront 0
  // loads the bytes of block kb + 2 during block kb and turns them into the
  // bias of block kb + 2 at the end of block kb + 1, after the wait at that
  // block's start: using them in the block that loads them made it wait a
  // memory latency per block, and the other wavefronts then waited for it at
  // the next barrier.
  auto mask_raw = [&](int kb) { return (int)mrow[min(kb * KT + tid, S - 1)]; };
  auto bias_from = [&](int kb, int raw) {
    return (kb * KT + tid < kend && raw != 0) ? 0.0f : -INFINITY;
  };
  auto bias_of = [&](int kb) { return bias_from(kb, mask_raw(kb)); };

  // Set-up loads in the order that lets their latencies overlap: the
  // wavefront's own fragments and log-sum-exp, the first streamed block,
  // and only then the key-mask bytes, whose values the LDS set-up waits for.
  // D = rowsum(dO * O) with O = the stored context plus its rounding
  // residual: the rows of dS = P (dP - D) then sum to zero up to fp32 and
  // residual rounding, as the key-bias gradient (exactly zero) requires.
  const bf16_t* __restrict__ Olg = a.o_lo ? a.o_lo + (int64_t)b * S * h + j * HD : nullptr;
  bf16x8_t qf[4], dof[4], of[4], olf[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const int c = 16 * ks + 8 * hf;
    if (q < S) {
      qf[ks] = ld_frag(Qg + (int64_t)q * ld + c);
      dof[ks] = ld_frag(dOg + (int64_t)q * h + c);
      of[ks] = ld_frag(Og + (int64_t)q * h + c);
      olf[ks] = Olg ? ld_frag(Olg + (int64_t)q * h + c) : __builtin_bit_cast(bf16x8_t, zero4());
    } else {
      qf[ks] = dof[ks] = of[ks] = olf[ks] = __builtin_bit_cast(bf16x8_t, zero4());
    }
  }
  const float lse_q = q < S ? a.lse[(int64_t)bh * S + q] : 0.0f;
  if (nkb > 0) {
    dma_rows(rsK, 0, ld, tiles[0], wave, lane);
    dma_rows(rsV, 0, ld, tiles[0] + TILE, wave, lane);
    if (tid < KT) {  // wavefront 0
      const float kb0 = bias_of(0);
      kbias[0][tid] = kb0;
      store_kfull(kfull[0], kb0, tid);
    }
  }
  int nraw = (tid < KT && nkb > 1) ? mask_raw(1) : 0;  // bytes of the next block
  float dsum = 0.0f;
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
#pragma unroll
    for (int i = 0; i < 8; ++i) dsum += (float)dof[ks][i] * ((float)of[ks][i] + (float)olf[ks][i]);
  {
    const HalfPair dp2 = half_pair(dsum);
    dsum = dp2.x + dp2.y;  // D = rowsum(dO * O) of query q
  }
  if (hf == 0 && q < S) a.dsum[(int64_t)bh * S + q] = dsum;

  f32x16_t dq[2] = {zero16(), zero16()};  // dQ^T: dims x queries
  for (int kb = 0; kb < nkb; ++kb) {
    const int st = kb & 1;
    wait_all();
    __syncthreads();
    if (kb + 1 < nkb) {
      dma_rows(rsK, (kb + 1) * KT, ld, tiles[st ^ 1], wave, lane);
      dma_rows(rsV, (kb + 1) * KT, ld, tiles[st ^ 1] + TILE, wave, lane);
    }
    const int nraw2 = (tid < KT && kb + 2 < nkb) ? mask_raw(kb + 2) : 0;
    const char* Ks = tiles[st];
    const char* Vs = tiles[st] + TILE;
#pragma unroll
    for (int sub = 0; sub < KT / 32; ++sub) {
      if (kb * KT + 32 * sub >= kend) break;
      // S^T = K_sub Q^T and dP^T - D = V_sub dO^T - D (keys x queries; the
      // accumulator starts at -D of the lane's query)
      f32x16_t s = zero16(), dp = splat16(-dsum);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        s = mfma32(frag_rows(Ks, 32 * sub, ks, lane), qf[ks], s);
        dp = mfma32(frag_rows(Vs, 32 * sub, ks, lane), dof[ks], dp);
      }
      if (__builtin_amdgcn_readfirstlane(kfull[st][sub])) {
#pragma unroll
        for (int r = 0; r < 16; ++r)  // dS^T (unscaled)
          s[r] = __builtin_amdgcn_exp2f(fmaf(s[r], a.scale_log2, -lse_q)) * dp[r];
      } else {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4_t kbv = *(const f32x4_t*)&kbias[st][32 * sub + 8 * g + 4 * hf];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int r = 4 * g + e;
            s[r] = __builtin_amdgcn_exp2f(fmaf(s[r], a.scale_log2, kbv[e]) - lse_q) * dp[r];
          }
        }
      }
      // dQ^T += K^T dS^T
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8_t db = pack8(s, 8 * ks);
#pragma unroll
        for (int t = 0; t < 2; ++t)
          dq[t] = mfma32(frag_tr(Ks, 32 * t, 32 * sub + 16 * ks, lane), db, dq[t]);
      }
    }
    if (kb + 1 < nkb && tid < KT) {
      const float nbias = bias_from(kb + 1, nraw);
      kbias[st ^ 1][tid] = nbias;
      store_kfull(kfull[st ^ 1], nbias, tid);
    }
    nraw = nraw2;
  }
  __syncthreads();  // the ring becomes the output staging area
  bf16_t* stage = (bf16_t*)&tiles[0][0] + wave * 32 * LD;
  const int nqb = (S + 31) / 32;
  float* cp = (a.colpart && q0 < S) ? a.colpart + ((int64_t)b * nqb + q0 / 32) * ld + j * HD : nullptr;
  store_rows_t(dq, a.scale, stage, a.out + (int64_t)b * S * ld + j * HD, ld, q0, S, cp);
}

// ---------------------------------------------------------------------------
// Backward, dK and dV: wavefront = 32 keys; loops over query blocks of QB
// (twice the key block: two barriers per 256 queries instead of four, with
// two resident blocks per CU as the registers allow).
// ---------------------------------------------------------------------------
constexpr int QB = 2 * KT;
constexpr int QTILE = QB * HD * 2;
__global__ __launch_bounds__(256, 2) void attn_bwd_dkdv_kernel(AttnArgs a) {
  // One LDS object (see LdsKV): Q, dO per stage; lse and D per stage.
  struct LdsQD {
    char tiles[2][2 * QTILE];
    float rowv[2][2][QB];
  };
  __shared__ __attribute__((aligned(1024))) LdsQD lds;
  auto& tiles = lds.tiles;
  auto& rowv = lds.rowv;

  int kb128, bh;
  attn_block((a.S + 127) / 128, kb128, bh);
  const int b = bh / a.H, j = bh % a.H;
  const int S = a.S, h = a.h;
  const int64_t ld = 3 * (int64_t)h;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hf = lane >> 5, rr = lane & 31;
  const int k0 = kb128 * 128 + wave * 32;
  const bf16_t* __restrict__ Qg = a.qkv + (int64_t)b * S * ld + j * HD;
  const bf16_t* __restrict__ Kg = Qg + h;
  const bf16_t* __restrict__ Vg = Qg + 2 * h;
  const bf16_t* __restrict__ dOg = a.dout + (int64_t)b * S * h + j * HD;
  const int kend = a.kext[b];
  const int key = k0 + rr;
  const bool block_live = kb128 * 128 < kend;  // uniform over the block
  const int nqb = block_live ? (S + QB - 1) / QB : 0;
  const __amdgpu_buffer_rsrc_t rsQ = rows_rsrc(Qg, S, ld), rsD = rows_rsrc(dOg, S, h);
  // threads 0-127 carry lse, 128-255 -D of query block qb (rows past S:
  // P = 0)
  static_assert(2 * QB == 256, "one value per thread");
  // The load (row clamped to a valid query, so that it is unconditional)
  // and the value it gives, kept apart as for the key mask of the forward:
  // the values of block qb + 2 are loaded during block qb and stored at the
  // end of block qb + 1.
  auto row_raw = [&](int qb) {
    const int qq = min(qb * QB + (tid & (QB - 1)), S - 1);
    return (tid < QB ? a.lse : a.dsum)[(int64_t)bh * S + qq];
  };
  auto row_from = [&](int qb, float raw) {
    const bool in = qb * QB + (tid & (QB - 1)) < S;
    if (tid < QB) return in ? raw : INFINITY;
    return in ? -raw : -0.0f;
  };
  auto rowval = [&](int qb) { return row_from(qb, row_raw(qb)); };
  // Set-up loads in the order that lets their latencies overlap: the
  // wavefront's own fragments, the first streamed block, and only then the
  // per-query values, whose LDS store waits for them.
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
  const int kraw = a.mask[(int64_t)b * S + min(key, S - 1)];
  if (nqb > 0) {
    dma_rows<QB>(rsQ, 0, ld, tiles[0], wave, lane);
    dma_rows<QB>(rsD, 0, h, tiles[0] + QTILE, wave, lane);
    rowv[0][tid / QB][tid & (QB - 1)] = rowval(0);
  }
  float nraw = nqb > 1 ? row_raw(1) : 0.0f;  // values of the next block
  // Initial score accumulator: 0, or -inf for a masked key (the lane's
  // column), which makes its probabilities exp2(-inf) = 0.
  const bool kvalid = key < kend && kraw != 0;
  const f32x16_t s0 = splat16(kvalid ? 0.0f : -INFINITY);
  f32x16_t dv[2] = {zero16(), zero16()}, dk[2] = {zero16(), zero16()};  // dims x keys

  for (int qb = 0; qb < nqb; ++qb) {
    const int st = qb & 1;
    wait_all();
    __syncthreads();
    if (qb + 1 < nqb) {
      dma_rows<QB>(rsQ, (qb + 1) * QB, ld, tiles[st ^ 1], wave, lane);
      dma_rows<QB>(rsD, (qb + 1) * QB, h, tiles[st ^ 1] + QTILE, wave, lane);
    }
    const float nraw2 = qb + 2 < nqb ? row_raw(qb + 2) : 0.0f;
    const char* Qs = tiles[st];
    const char* dOs = tiles[st] + QTILE;
#pragma unroll
    for (int sub = 0; sub < QB / 32; ++sub) {
      if (qb * QB + 32 * sub >= S) break;
      // S (32 queries x 32 keys) = Q_sub K^T;  dP - D = dO_sub V^T - D (the
      // accumulator starts at -D of each register's query)
      f32x16_t s = s0, dp;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4_t dv4 = *(const f32x4_t*)&rowv[st][1][32 * sub + 8 * g + 4 * hf];
#pragma unroll
        for (int e = 0; e < 4; ++e) dp[4 * g + e] = dv4[e];
      }
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        s = mfma32(frag_rows(Qs, 32 * sub, ks, lane), kf[ks], s);
        dp = mfma32(frag_rows(dOs, 32 * sub, ks, lane), vf[ks], dp);
      }
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4_t lv = *(const f32x4_t*)&rowv[st][0][32 * sub + 8 * g + 4 * hf];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * g + e;
          const float p = __builtin_amdgcn_exp2f(fmaf(s[r], a.scale_log2, -lv[e]));
          s[r] = p;
          dp[r] = p * dp[r];  // dS (unscaled)
        }
      }
      // dV^T += dO^T P;  dK^T += Q^T dS
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8_t pb = pack8(s, 8 * ks);
        const bf16x8_t db = pack8(dp, 8 * ks);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          dv[t] = mfma32(frag_tr(dOs, 32 * t, 32 * sub + 16 * ks, lane), pb, dv[t]);
          dk[t] = mfma32(frag_tr(Qs, 32 * t, 32 * sub + 16 * ks, lane), db, dk[t]);
        }
      }
    }
    if (qb + 1 < nqb) rowv[st ^ 1][tid / QB][tid & (QB - 1)] = row_from(qb + 1, nraw);
    nraw = nraw2;
  }
  __syncthreads();  // the ring becomes the output staging area
  bf16_t* stage = (bf16_t*)&tiles[0][0] + wave * 32 * LD;
  bf16_t* dst = a.out + (int64_t)b * S * ld + j * HD;
  const int nkb32 = (S + 31) / 32;
  float* cp = (a.colpart && k0 < S) ? a.colpart + ((int64_t)b * nkb32 + k0 / 32) * ld + j * HD : nullptr;
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
  dim3 grid((unsigned)(((a.S + 127) / 128) * a.B * a.H));
  hipLaunchKernelGGL(attn_fwd_kernel, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t attn_backward_dq(const AttnArgs& a, hipStream_t st) {
  if (a.B == 0 || a.S == 0) return hipSuccess;
  dim3 grid((unsigned)(((a.S + 127) / 128) * a.B * a.H));
  hipLaunchKernelGGL(attn_bwd_dq_kernel, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t attn_backward_dkdv(const AttnArgs& a, hipStream_t st) {
  if (a.B == 0 || a.S == 0) return hipSuccess;
  dim3 grid((unsigned)(((a.S + 127) / 128) * a.B * a.H));
  hipLaunchKernelGGL(attn_bwd_dkdv_kernel, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

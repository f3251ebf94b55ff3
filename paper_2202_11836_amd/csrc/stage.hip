// Stage engine and C ABI: owns parameters, gradients, the saved-activation
// record of the latest forward pass and the workspace, and sequences the
// per-layer kernel launches of one pipeline stage on one HIP stream
// (paper section III: forward through the device's layers, then gradients
// in reverse layer order).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <type_traits>
#include <vector>

#include "../../include/stage.h"
#include "kernels.h"

namespace {

constexpr int HEAD_DIM = 64;
constexpr int COL_PARTS = 128; // row blocks of the bias-gradient column sums

// Kernel launch sites of one layer, for event tracing (stage_trace_site).
#define STAGE_SITES(X)                                                              \
  X(QKV_FWD, "qkv_gemm_fwd") X(SCORES_FWD, "scores_gemm_fwd")                         \
  X(SOFTMAX_FWD, "softmax_fwd") X(CTX_FWD, "context_gemm_fwd")                        \
  X(OUT_FWD, "out_gemm_fwd") X(LN1_FWD, "add_ln1_fwd") X(FFN1_FWD, "ffn1_gelu_gemm_fwd") \
  X(FFN2_FWD, "ffn2_gemm_fwd") X(LN2_FWD, "add_ln2_fwd") X(LN2_BWD, "ln2_bwd")          \
  X(LN2_RED, "ln2_bwd_colreduce") X(W2_WGRAD, "w2_wgrad_gemm")                          \
  X(W2_RED, "w2_wgrad_splitk_reduce") X(FFN2_DGRAD, "ffn2_dgrad_dgelu_gemm")            \
  X(B1_SUM, "b1_colsum") X(B1_RED, "b1_colreduce") X(W1_WGRAD, "w1_wgrad_gemm")         \
  X(W1_RED, "w1_wgrad_splitk_reduce") X(FFN1_DGRAD, "ffn1_dgrad_resid_gemm")            \
  X(LN1_BWD, "ln1_bwd") X(LN1_RED, "ln1_bwd_colreduce") X(WO_WGRAD, "wo_wgrad_gemm")    \
  X(WO_RED, "wo_wgrad_splitk_reduce") X(OUT_DGRAD, "out_dgrad_gemm")                    \
  X(DP_BWD, "dp_gemm_bwd") X(SOFTMAX_BWD, "softmax_bwd") X(DV_BWD, "dv_gemm_bwd")        \
  X(DQ_BWD, "dq_gemm_bwd") X(DK_BWD, "dk_gemm_bwd") X(BQKV_SUM, "bqkv_colsum")           \
  X(BQKV_RED, "bqkv_colreduce") X(WQKV_WGRAD, "wqkv_wgrad_gemm")                        \
  X(WQKV_RED, "wqkv_wgrad_splitk_reduce") X(QKV_DGRAD, "qkv_dgrad_resid_gemm")            \
  X(KEXT, "key_extent") X(ATTN_FWD, "attn_fwd") X(ATTN_DQ, "attn_bwd_dq")                 \
  X(ATTN_DKDV, "attn_bwd_dkdv")                                \
  X(WGRAD_GROUP, "wgrad_group_gemm") X(WGRAD_GROUP_RED, "wgrad_group_splitk_reduce")

enum Site {
#define SITE_ENUM(id, name) SITE_##id,
  STAGE_SITES(SITE_ENUM)
#undef SITE_ENUM
  SITE_COUNT
};
const char* const SITE_NAMES[] = {
#define SITE_NAME(id, name) name,
    STAGE_SITES(SITE_NAME)
#undef SITE_NAME
};

// --------------------------------------------------------------------------
// Parameter initialisation: counter-based splitmix64 (Steele, Lea & Flood,
// "Fast splittable pseudorandom number generators", 2014) feeding two 53-bit
// uniforms into Box-Muller.
// --------------------------------------------------------------------------
__host__ __device__ inline uint64_t splitmix64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
constexpr uint64_t GOLDEN = 0x9E3779B97F4A7C15ull;

template <typename T>
__global__ void init_normal_kernel(T* out, int64_t n, uint64_t key, double stdv) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  uint64_t a = splitmix64_mix(key + (uint64_t)(2 * i + 1) * GOLDEN);
  uint64_t b = splitmix64_mix(key + (uint64_t)(2 * i + 2) * GOLDEN);
  double u1 = ((double)(a >> 11) + 1.0) * (1.0 / 9007199254740992.0);  // (0, 1]
  double u2 = (double)(b >> 11) * (1.0 / 9007199254740992.0);          // [0, 1)
  double z = sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2);
  st_f(out + i, (float)(z * stdv));
}

__global__ void fill_kernel(float* out, int64_t n, float v) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = v;
}

// out = x (fp32; fp32 stages), or bf (bf16), or (hi + lo) + b (bf16), as fp32.
__global__ void grad_record_kernel(const float* x, const bf16_t* bf, const bf16_t* hi,
                                   const bf16_t* lo, const bf16_t* b, float* out, int64_t n) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  out[i] = x ? x[i] : bf ? bf2f(bf[i]) : (bf2f(hi[i]) + bf2f(lo[i])) + bf2f(b[i]);
}

__global__ void ones_u8_kernel(uint8_t* out, int64_t n) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = 1;
}

bool is_matrix(int which) {
  return which == STAGE_W_QKV || which == STAGE_W_O || which == STAGE_W_1 || which == STAGE_W_2;
}

// Parameters 0 .. STAGE_BE1 belong to the attention half of a layer, the
// rest to its feed-forward half.
bool is_attn_param(int which) { return which <= STAGE_BE1; }

struct Saved {
  void* X = nullptr;     // layer input [T, h]
  void* QKV = nullptr;   // [T, 3h]
  void* P = nullptr;     // softmax probabilities [B*H, S, S] (fp32 stages)
  float* lse = nullptr;  // log2-sum-exp of the scaled scores [B*H, S] (bf16 stages)
  void* C = nullptr;     // context [T, h]
  void* Clo = nullptr;   // its bf16 rounding residual [T, h] (bf16 stages)
  void* xhat1 = nullptr; // [T, h]
  float* rstd1 = nullptr;
  void* H1 = nullptr;    // [T, h]
  void* Gd = nullptr;    // GELU'(U) [T, f], U = H1 W_1^T + b_1
  void* G = nullptr;     // [T, f]
  void* xhat2 = nullptr; // [T, h]
  float* rstd2 = nullptr;
};

}  // namespace

// Static scratch of stage_backward_noalloc: the weight-gradient split-K
// partials and the bias / LayerNorm column partial sums of a backward pass,
// in a file-scope device array (one copy per device, held until the process
// ends).  Host code never uses its name as an address: the per-device
// address comes from hipGetSymbolAddress (resolve_scratch).
constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)256 << 20;
static __device__ __align__(256) float scratch[NOALLOC_SCRATCH_BYTES / sizeof(float)];

struct stage {
  int L = 0, h = 0, H = 0, f = 0;
  // Allocation units (two per encoder layer): unit 2j is the attention half
  // of global layer j (X -> H1), unit 2j+1 its feed-forward half (H1 -> Y).
  // The stage holds units [2 l0 + ffn_first, ...); local layer l is global
  // layer l0 + l.  ffn_first: local layer 0 has only its feed-forward half
  // (the stage input is H1); attn_last: local layer L-1 has only its
  // attention half (the stage output is H1).
  int l0 = 0;
  bool ffn_first = false, attn_last = false;
  stage_dtype dtype = STAGE_F32;
  size_t esz = 4;
  hipStream_t stream = nullptr;
  std::vector<std::array<void*, STAGE_NPARAM>> param;
  std::vector<std::array<float*, STAGE_NPARAM>> grad;
  std::vector<void*> allocs;  // parameter / gradient memory
  // Bytes requested from hipMalloc (parameters and gradients; activation
  // record and workspace).  A dry-run stage only counts them.
  int64_t bytes_param = 0, bytes_act = 0;
  bool dry_run = false;

  // Activation memory, sized for cap_T tokens and cap_BSS score entries.
  int64_t cap_T = -1, cap_BSS = -1, cap_B = -1, cap_NQB = -1;
  std::vector<void*> act_allocs;
  std::vector<Saved> saved;
  uint8_t* mask = nullptr;
  float* tmp = nullptr;     // [T, h] fp32 GEMM output before LayerNorm
  void* h1lo = nullptr;     // [T, h] H1's bf16 rounding residual (bf16 stages)
  float* scores = nullptr;  // [B*H, S, S] fp32 (scores, then dP; fp32 stages)
  int* kext = nullptr;      // [B] key extent of each sequence
  float* dsum = nullptr;    // [B*H, S] rowsum(dO * O) (bf16 stages)
  void* dS = nullptr;       // [B*H, S, S]
  void* dQKV = nullptr;     // [T, 3h]
  void* dZ2 = nullptr;      // [T, h]
  void* dU = nullptr;       // [T, f]
  void* dH1 = nullptr;      // [T, h]
  void* dZ1 = nullptr;      // [T, h]
  void* dC = nullptr;       // [T, h]
  void* dY = nullptr;       // [T, h] gradient flowing between layers (fp32 stages)
  // bf16 stages: the rounding residuals of dZ1 and dZ2 (with the bf16 dZ1,
  // dZ2 they carry the residual branches of dX and dH1 to ~16 bits)
  void* dz1lo = nullptr;    // [T, h]
  void* dz2lo = nullptr;    // [T, h]
  void* prod = nullptr;     // [T, h] bf16 data-gradient GEMM product joining them (bf16 stages)
  float* part = nullptr;    // column-sum partials
  float* part2 = nullptr;   // second LayerNorm's partials (bf16: reduced at the layer's end)
  float* colpart_ffn = nullptr;  // [ceil(T/128), f] column sums of dU (bf16 stages)
  float* colpart_qkv = nullptr;  // [B * ceil(S/32), 3h] column sums of dQKV (bf16 stages)
  // Transposed weights of the layer being differentiated (bf16 stages), so
  // that every data-gradient GEMM reads both operands k-contiguously.
  float* splitk = nullptr;  // split-K partials of the weight gradients
  size_t splitk_elems = 0;  // elements it holds
  size_t splitk_bytes = 0;  // bytes counted for it in bytes_act

  // Optional record of the gradient reaching each layer's output in the
  // latest backward (fp32 [T, h] per layer), for layer-wise checks.
  bool record_grads = false;
  bool rec_valid = false;
  std::vector<float*> rec;

  int device = 0;          // device current at stage_init
  bool no_alloc = false;   // inside stage_backward_noalloc: no event creation

  int B = 0, S = 0;
  bool have_ctx = false;
  std::string err;

  // Event tracing of a set of launch sites (bit i = site i).
  uint64_t trace_mask = 0;
  std::vector<hipEvent_t> events;  // pool, reused
  size_t events_used = 0;
};

namespace {

// Message of the last failed stage_init on this thread (no handle exists).
thread_local std::string g_init_err;

// Per-device address of `scratch`, resolved once per device with that device
// current (at stage_init).

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[MAX_DEVICES] = {};

// Resolves (once) the address of `scratch` on the current device.
hipError_t resolve_scratch(int* device_out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
  if (device_out) *device_out = dev;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev]) return hipSuccess;
  void* ptr = nullptr;
  e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  g_scratch_ptr[dev] = (float*)ptr;
  return hipSuccess;
}

float* scratch_of(int dev) {
  if (dev < 0 || dev >= MAX_DEVICES) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  return g_scratch_ptr[dev];
}

// Which halves of local layer l the stage holds.
bool has_attn(const stage_t* s, int l) { return !(l == 0 && s->ffn_first); }
bool has_ffn(const stage_t* s, int l) { return !(l == s->L - 1 && s->attn_last); }
bool has_param(const stage_t* s, int l, int which) {
  return is_attn_param(which) ? has_attn(s, l) : has_ffn(s, l);
}

stage_status fail(stage_t* s, stage_status st, const std::string& msg) {
  if (s) s->err = msg;
  return st;
}

#define HIPCK(expr)                                                                    \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail(s, STAGE_EHIP, std::string(#expr) + ": " + hipGetErrorString(e_));   \
  } while (0)

// Records a start event before a traced site's launch; returns the pool
// index of the event pair, or -1 when the site is not traced.
int trace_begin(stage_t* s, int site) {
  if (!((s->trace_mask >> site) & 1) || s->no_alloc) return -1;
  while (s->events.size() < s->events_used + 2) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return -1;
    s->events.push_back(e);
  }
  int idx = (int)s->events_used;
  s->events_used += 2;
  if (hipEventRecord(s->events[idx], s->stream) != hipSuccess) {
    s->events_used -= 2;
    return -1;
  }
  return idx;
}
void trace_end(stage_t* s, int idx) {
  if (idx < 0) return;
  (void)hipEventRecord(s->events[idx + 1], s->stream);
}

// Launch expression (a hipError_t) as traced site number `site`.
#define SITE_I(site, ...)                                                         \
  do {                                                                            \
    int tr_ = trace_begin(s, (site));                                             \
    hipError_t e_ = (__VA_ARGS__);                                                \
    trace_end(s, tr_);                                                            \
    if (e_ != hipSuccess)                                                         \
      return fail(s, STAGE_EHIP,                                                  \
                  std::string(SITE_NAMES[(site)]) + ": " + hipGetErrorString(e_)); \
  } while (0)
#define SITE(id, ...) SITE_I(SITE_##id, __VA_ARGS__)

int64_t param_numel(const stage_t* s, int which) {
  const int64_t h = s->h, f = s->f;
  switch (which) {
    case STAGE_W_QKV: return 3 * h * h;
    case STAGE_B_QKV: return 3 * h;
    case STAGE_W_O: return h * h;
    case STAGE_W_1: return f * h;
    case STAGE_B_1: return f;
    case STAGE_W_2: return h * f;
    default: return h;
  }
}

size_t param_esz(const stage_t* s, int which) { return is_matrix(which) ? s->esz : 4; }

void free_activations(stage_t* s) {
  for (void* p : s->act_allocs) (void)hipFree(p);
  s->act_allocs.clear();
  s->saved.clear();
  s->rec.clear();
  s->rec_valid = false;
  s->bytes_act = 0;
  s->splitk = nullptr;
  s->splitk_elems = 0;
  s->splitk_bytes = 0;
  s->cap_T = s->cap_BSS = s->cap_B = s->cap_NQB = -1;
  s->have_ctx = false;
}

stage_status dev_alloc(stage_t* s, std::vector<void*>& list, void** p, size_t bytes) {
  *p = nullptr;
  if (bytes == 0) bytes = 256;
  (&list == &s->allocs ? s->bytes_param : s->bytes_act) += (int64_t)bytes;
  if (s->dry_run) return STAGE_OK;
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return fail(s, STAGE_ENOMEM, std::string("hipMalloc(") + std::to_string(bytes) +
                                     " bytes): " + hipGetErrorString(e));
  }
  list.push_back(*p);
  return STAGE_OK;
}

// Tiling of a weight-gradient GEMM dW[M, N] = sum over K = T tokens: the
// output has few tiles, so the token range is split until about one
// work-group per CU (256) is running.  256x256 tiles when the output has at
// least 16 of them, else 128x128.  Returns the split count; *tile receives
// the GemmArgs tile code.
int wgrad_split(int64_t M, int64_t N, int K, int* tile) {
  const int64_t t256 = ((M + 255) / 256) * ((N + 255) / 256);
  int64_t tiles;
  if (t256 >= 16) {
    *tile = 1;
    tiles = t256;
  } else {
    *tile = 3;
    tiles = ((M + 127) / 128) * ((N + 127) / 128);
  }
  int ks = (int)std::max<int64_t>(1, 256 / tiles);
  ks = std::min(ks, std::max(1, K / 512));  // chunks of at least 512 tokens
  return ks;
}

// Elements of split-K partials the weight gradients of a backward over T
// tokens need.  bf16 stages compute a layer's weight gradients in one group
// launch (stream-K over all their tiles): room for all four gradients'
// partials, or for the feed-forward or attention half of a partial layer.
// fp32 stages compute them one at a time: the largest one's.  The figure is
// not monotone in T (the stream-K piece count per tile depends on how the
// k-tiles of all tiles divide among the work-groups), so it is evaluated for
// every token count a forward prepares.
size_t splitk_need(const stage_t* s, int64_t T) {
  const int64_t h = s->h, f = s->f;
  size_t need = 0;
  if (s->dtype == STAGE_BF16) {
    const int Ms[4] = {(int)h, (int)f, (int)h, (int)(3 * h)};
    const int Ns[4] = {(int)f, (int)h, (int)h, (int)h};
    const int K = (int)std::max<int64_t>(T, 1);
    need = std::max({(size_t)wgrad_group_slots(Ms, Ns, 4, K) * (size_t)(2 * h * f + 4 * h * h),
                     (size_t)wgrad_group_slots(Ms, Ns, 2, K) * (size_t)(2 * h * f),
                     (size_t)wgrad_group_slots(Ms + 2, Ns + 2, 2, K) * (size_t)(4 * h * h)});
  } else {
    const int64_t shapes[4][2] = {{3 * h, h}, {h, h}, {f, h}, {h, f}};
    for (auto& mn : shapes) {
      int tile;
      int ks = wgrad_split(mn[0], mn[1], (int)T, &tile);
      if (ks > 1) need = std::max<size_t>(need, (size_t)ks * mn[0] * mn[1]);
    }
  }
  return need;
}

// (Re)allocates the split-K partial buffer for at least `need` elements.
stage_status grow_splitk(stage_t* s, size_t need) {
  if (s->splitk) {
    auto it = std::find(s->act_allocs.begin(), s->act_allocs.end(), (void*)s->splitk);
    if (it != s->act_allocs.end()) s->act_allocs.erase(it);
    (void)hipFree(s->splitk);
    s->splitk = nullptr;
  }
  s->bytes_act -= (int64_t)s->splitk_bytes;
  s->splitk_elems = 0;
  s->splitk_bytes = 0;
  const size_t bytes = std::max<size_t>(need, 1) * 4;
  stage_status st = dev_alloc(s, s->act_allocs, (void**)&s->splitk, bytes);
  if (st) {
    // leave no half-built record: the next forward allocates from scratch
    std::string msg = s->err;
    free_activations(s);
    s->err = msg;
    return st;
  }
  s->splitk_elems = need;
  s->splitk_bytes = bytes;
  return STAGE_OK;
}

stage_status ensure_activations(stage_t* s, int B, int S) {
  const int64_t T = (int64_t)B * S;
  // The score matrix is materialised only on fp32 stages.
  const int64_t BSS = s->dtype == STAGE_F32 ? (int64_t)B * s->H * S * S : 0;
  const int64_t BHS = (int64_t)B * s->H * S;
  const int64_t NQB = (int64_t)B * ((S + 31) / 32);
  const size_t need = splitk_need(s, T);
  if (T <= s->cap_T && BSS <= s->cap_BSS && B <= s->cap_B && NQB <= s->cap_NQB &&
      (int)s->saved.size() == s->L)
    return need <= s->splitk_elems ? STAGE_OK : grow_splitk(s, need);
  free_activations(s);
  const size_t e = s->esz;
  const int64_t h = s->h, f = s->f;
  auto A = [&](void** p, size_t bytes) { return dev_alloc(s, s->act_allocs, p, bytes); };
  stage_status st;
  s->saved.resize(s->L);
  // The attention half of a layer saves X, QKV, P, lse, C, xhat1, rstd1
  // (and C's rounding residual on bf16 stages);
  // the feed-forward half saves its input H1, GELU'(U), G, xhat2, rstd2.
  for (int l = 0; l < s->L; ++l) {
    Saved& v = s->saved[l];
    if (has_attn(s, l) &&
        ((st = A(&v.X, T * h * e)) || (st = A(&v.QKV, T * 3 * h * e)) ||
         (st = A(&v.P, BSS * e)) || (st = A((void**)&v.lse, BHS * 4)) ||
         (st = A(&v.C, T * h * e)) || (st = A(&v.xhat1, T * h * e)) ||
         (st = A((void**)&v.rstd1, T * 4)) ||
         (s->dtype == STAGE_BF16 && (st = A(&v.Clo, T * h * e)))))
      return st;
    if (has_ffn(s, l) &&
        ((st = A(&v.H1, T * h * e)) || (st = A(&v.Gd, T * f * e)) || (st = A(&v.G, T * f * e)) ||
         (st = A(&v.xhat2, T * h * e)) || (st = A((void**)&v.rstd2, T * 4))))
      return st;
  }
  if ((st = A((void**)&s->mask, T)) || (st = A((void**)&s->tmp, T * h * 4)) ||
      (st = A(&s->h1lo, T * h * e)) ||
      (st = A((void**)&s->scores, BSS * 4)) || (st = A(&s->dS, BSS * e)) ||
      (st = A((void**)&s->kext, (size_t)B * 4)) || (st = A((void**)&s->dsum, BHS * 4)) ||
      (st = A(&s->dQKV, T * 3 * h * e)) || (st = A(&s->dZ2, T * h * e)) ||
      (st = A(&s->dU, T * f * e)) || (st = A(&s->dZ1, T * h * e)) || (st = A(&s->dC, T * h * e)))
    return st;
  // The gradient between layers and at H1: in the stage dtype on fp32
  // stages; on bf16 stages the rounding residuals of the residual branches
  // dZ1 and dZ2 and the bf16 GEMM product added to them.
  if (s->dtype == STAGE_F32 ? ((st = A(&s->dH1, T * h * e)) || (st = A(&s->dY, T * h * e)))
                            : ((st = A(&s->dz1lo, T * h * e)) || (st = A(&s->dz2lo, T * h * e)) ||
                               (st = A(&s->prod, T * h * e))))
    return st;
  const int64_t nqb = ((int64_t)S + 31) / 32;
  if ((st = A((void**)&s->colpart_ffn, ((T + 127) / 128) * f * 4)) ||
      (st = A((void**)&s->colpart_qkv, (int64_t)B * nqb * 3 * h * 4)))
    return st;
  const int64_t maxw = std::max<int64_t>(3 * h, f);
  const int64_t part_elems =
      std::max<int64_t>((int64_t)ln_bwd_blocks((int)T) * 3 * h, (int64_t)COL_PARTS * maxw);
  if ((st = A((void**)&s->part, part_elems * 4))) return st;
  if (s->dtype == STAGE_BF16 &&
      (st = A((void**)&s->part2, (int64_t)ln_bwd_blocks((int)T) * 3 * h * 4)))
    return st;
  if (s->record_grads) {
    s->rec.assign(s->L, nullptr);
    for (int l = 0; l < s->L; ++l)
      if ((st = A((void**)&s->rec[l], T * h * 4))) return st;
  }
  if ((st = grow_splitk(s, need))) return st;
  s->cap_T = T;
  s->cap_BSS = BSS;
  s->cap_B = B;
  s->cap_NQB = NQB;
  return STAGE_OK;
}

// ---------------------------------------------------------------------------
// Typed launch helpers
// ---------------------------------------------------------------------------
template <typename T> struct Gemm;
template <> struct Gemm<bf16_t> {
  static hipError_t run(const GemmArgs& g, bool ak, bool bk, GemmEpi epi, bool out_f32, int batch,
                        hipStream_t st) {
    return gemm_bf16(g, ak, bk, epi, out_f32, batch, st);
  }
};
template <> struct Gemm<float> {
  static hipError_t run(const GemmArgs& g, bool ak, bool bk, GemmEpi epi, bool, int batch,
                        hipStream_t st) {
    return gemm_f32(g, ak, bk, epi, batch, st);
  }
};

// Weight gradient dW[M, N] = sum_t dY[t, m] * X[t, n] (fp32 out), split over
// t when the output has few tiles; the split partials are summed in order.
template <typename T>
stage_status wgrad(stage_t* s, int site, int site_red, const T* dYm, int64_t ld_dy, const T* Xn,
                   int64_t ld_x, int M, int N, int Tk, float* out) {
  GemmArgs g = gemm_args(dYm, ld_dy, Xn, ld_x, out, N, M, N, Tk);
  int ks = wgrad_split(M, N, Tk, &g.tile);
  if (ks > 1 && (size_t)ks * M * N <= s->splitk_elems) {
    int chunk = (Tk + ks - 1) / ks;
    chunk = (chunk + 63) / 64 * 64;
    ks = (Tk + chunk - 1) / chunk;
    g.C = s->splitk;
    g.ksplit = ks;
    g.kchunk = chunk;
    SITE_I(site, Gemm<T>::run(g, false, false, EPI_PARTIAL, true, 1, s->stream));
    SITE_I(site_red, splitk_reduce(s->splitk, ks, M, N, out, s->stream));
  } else {
    SITE_I(site, Gemm<T>::run(g, false, false, EPI_STORE, true, 1, s->stream));
  }
  return STAGE_OK;
}

// A weight gradient dW[M, N] = dY^T X over the stage's tokens whose launch
// is deferred to the layer's group launch (bf16 stages).
struct WgradJob {
  const void* dy;
  int64_t ld_dy;
  const void* x;
  int64_t ld_x;
  int M, N;
  float* out;
};

// The queued weight gradients of one layer in one GEMM launch (stream-K
// over all their tiles, fp32 partials side by side in the split-K buffer)
// and one fixed-order reduction launch, which also runs the layer's queued
// column reductions (bias, gamma and beta gradients).
stage_status wgrad_group(stage_t* s, const WgradJob* jobs, int n, const ColJob* cols, int ncols) {
  if (n == 0 && ncols == 0) return STAGE_OK;
  const int Tn = s->B * s->S;
  GemmArgs gs[GEMM_GROUP_MAX];
  float* outs[GEMM_GROUP_MAX];
  int Ms[GEMM_GROUP_MAX], Ns[GEMM_GROUP_MAX];
  for (int q = 0; q < n; ++q) {
    Ms[q] = jobs[q].M;
    Ns[q] = jobs[q].N;
  }
  const int slots = wgrad_group_slots(Ms, Ns, n, Tn);
  if (slots < 1) return fail(s, STAGE_EINVAL, "weight-gradient group: invalid sizes");
  size_t off = 0;
  for (int q = 0; q < n; ++q) {
    const WgradJob& j = jobs[q];
    gs[q] = gemm_args(j.dy, j.ld_dy, j.x, j.ld_x, s->splitk + off, j.N, j.M, j.N, Tn);
    gs[q].tile = 1;
    off += (size_t)slots * j.M * j.N;
    outs[q] = j.out;
  }
  if (off > s->splitk_elems) return fail(s, STAGE_EHIP, "split-K buffer too small");
  SITE(WGRAD_GROUP, gemm_bf16_wgrad_group(gs, n, s->stream));
  SITE(WGRAD_GROUP_RED, wgrad_group_reduce(gs, outs, n, cols, ncols, s->stream));
  return STAGE_OK;
}

AttnArgs attn_args(stage_t* s, const bf16_t* qkv, bf16_t* out, float* lse) {
  AttnArgs a{};
  a.qkv = qkv;
  a.mask = s->mask;
  a.kext = s->kext;
  a.out = out;
  a.lse = lse;
  a.dsum = s->dsum;
  a.B = s->B;
  a.S = s->S;
  a.H = s->H;
  a.h = s->h;
  a.scale = 1.0f / sqrtf((float)HEAD_DIM);
  a.scale_log2 = a.scale * 1.4426950408889634f;
  return a;
}

template <typename T>
stage_status forward_impl(stage_t* s, const T* x, T* y) {
  const int B = s->B, S = s->S, h = s->h, H = s->H, f = s->f;
  const int Tn = B * S;
  const int BH = B * H;
  hipStream_t st = s->stream;
  const float scale = 1.0f / sqrtf((float)HEAD_DIM);
  // The stage input is X of local layer 0, or its H1 when that layer holds
  // only its feed-forward half.
  HIPCK(hipMemcpyAsync(s->ffn_first ? s->saved[0].H1 : s->saved[0].X, x, (size_t)Tn * h * sizeof(T),
                       hipMemcpyDeviceToDevice, st));
  if (std::is_same<T, bf16_t>::value && (s->L > 1 || !s->ffn_first))
    SITE(KEXT, key_extent(s->mask, B, S, s->kext, st));
  for (int l = 0; l < s->L; ++l) {
    Saved& v = s->saved[l];
    auto& p = s->param[l];
    // For bf16 stages the first LayerNorm also writes H1's bf16 rounding
    // residual when this stage computes H1: H1 is the residual of the
    // second LayerNorm, which adds it back, so H1's rounding to bf16 stays
    // out of Y.  (A stage that starts at a feed-forward half receives H1 in
    // bf16, as the previous stage's output.)
    T* h1_lo = (std::is_same<T, float>::value || !has_attn(s, l)) ? nullptr : (T*)s->h1lo;
    if (has_attn(s, l)) {
      const T* X = (const T*)v.X;
      T* QKV = (T*)v.QKV;
      // QKV = X W_qkv^T + b_qkv
      {
        GemmArgs g = gemm_args(X, h, p[STAGE_W_QKV], h, QKV, 3 * h, Tn, 3 * h, h);
        g.bias = (const float*)p[STAGE_B_QKV];
        SITE(QKV_FWD, Gemm<T>::run(g, true, true, EPI_STORE, false, 1, st));
      }
      if constexpr (std::is_same<T, bf16_t>::value) {
        // Fused attention: softmax(Q K^T / 8) V per (batch, head), P stays on chip.
        AttnArgs aa = attn_args(s, (const bf16_t*)QKV, (bf16_t*)v.C, v.lse);
        aa.out_lo = (bf16_t*)v.Clo;
        SITE(ATTN_FWD, attn_forward(aa, st));
      } else {
      // scores[b, j] = Q_bj K_bj^T  (fp32)
      {
        GemmArgs g = gemm_args(QKV, 3 * h, QKV + h, 3 * h, s->scores, S, S, S, HEAD_DIM);
        g.zdiv = H;
        g.sA1 = g.sB1 = (int64_t)S * 3 * h;
        g.sA2 = g.sB2 = HEAD_DIM;
        g.sC1 = (int64_t)H * S * S;
        g.sC2 = (int64_t)S * S;
        SITE(SCORES_FWD, Gemm<T>::run(g, true, true, EPI_STORE, true, BH, st));
      }
      SITE(SOFTMAX_FWD, softmax_fwd<T>(s->scores, s->mask, (T*)v.P, BH, H, S, S, scale, st));
      // C[b, :, j] = P_bj V_bj
      {
        GemmArgs g = gemm_args(v.P, S, QKV + 2 * h, 3 * h, v.C, h, S, HEAD_DIM, S);
        g.zdiv = H;
        g.sA1 = (int64_t)H * S * S;
        g.sA2 = (int64_t)S * S;
        g.sB1 = (int64_t)S * 3 * h;
        g.sB2 = HEAD_DIM;
        g.sC1 = (int64_t)S * h;
        g.sC2 = HEAD_DIM;
        SITE(CTX_FWD, Gemm<T>::run(g, true, false, EPI_STORE, false, BH, st));
      }
      }
      // tmp = C W_o^T (fp32);  H1 = LN(X + tmp + b_o)
      {
        GemmArgs g = gemm_args(v.C, h, p[STAGE_W_O], h, s->tmp, h, Tn, h, h);
        SITE(OUT_FWD, Gemm<T>::run(g, true, true, EPI_STORE, true, 1, st));
      }
      // The last layer of a stage that ends at an attention half writes H1
      // straight to the stage output.
      const bool to_out = !has_ffn(s, l);
      if (to_out) h1_lo = nullptr;
      SITE(LN1_FWD, add_ln_fwd<T, float>(s->tmp, (const float*)p[STAGE_B_O], X, nullptr,
                                         (const float*)p[STAGE_G1], (const float*)p[STAGE_BE1],
                                         to_out ? y : (T*)v.H1, h1_lo, (T*)v.xhat1, v.rstd1, Tn,
                                         h, st));
      if (to_out) break;
    }  // attention half
    // U = H1 W_1^T + b_1;  G = GELU(U) and GELU'(U) (kept for the backward)
    {
      GemmArgs g = gemm_args(v.H1, h, p[STAGE_W_1], h, v.G, f, Tn, f, h);
      g.bias = (const float*)p[STAGE_B_1];
      g.C2 = v.Gd;
      SITE(FFN1_FWD, Gemm<T>::run(g, true, true, EPI_GELU, false, 1, st));
    }
    // tmp = G W_2^T (fp32);  Y = LN(H1 + tmp + b_2)
    {
      GemmArgs g = gemm_args(v.G, f, p[STAGE_W_2], f, s->tmp, h, Tn, h, f);
      SITE(FFN2_FWD, Gemm<T>::run(g, true, true, EPI_STORE, true, 1, st));
    }
    T* Y = (l + 1 < s->L) ? (T*)s->saved[l + 1].X : y;
    SITE(LN2_FWD, add_ln_fwd<T, float>(s->tmp, (const float*)p[STAGE_B_2], (const T*)v.H1,
                                       h1_lo, (const float*)p[STAGE_G2],
                                       (const float*)p[STAGE_BE2], Y, nullptr, (T*)v.xhat2,
                                       v.rstd2, Tn, h, st));
  }
  return STAGE_OK;
}

// LayerNorm backward into partials `part`; their column reduction into
// dgamma, dbeta, dbias runs here, or is queued in *defer (bf16 stages: run
// with the layer's weight-gradient reduction).
template <typename T>
stage_status ln_backward(stage_t* s, int site, int site_red, const T* dy, const T* xhat, const float* rstd,
                         const float* gamma, T* dz, float* dgamma, float* dbeta, float* dbias,
                         float* part, ColJob* defer) {
  const int Tn = s->B * s->S, h = s->h;
  SITE_I(site, ln_bwd<T>(dy, xhat, rstd, gamma, dz, part, Tn, h, s->stream));
  if (defer) {
    *defer = ColJob{part, ln_bwd_blocks(Tn), 3, h, {dgamma, dbeta, dbias, nullptr}};
    return STAGE_OK;
  }
  float* outs[3] = {dgamma, dbeta, dbias};
  SITE_I(site_red, col_reduce(part, ln_bwd_blocks(Tn), 3, h, outs, s->stream));
  return STAGE_OK;
}

template <typename T>
stage_status col_sum(stage_t* s, int site, int site_red, const T* x, int n, float* out) {
  const int Tn = s->B * s->S;
  SITE_I(site, col_partial<T>(x, Tn, n, s->part, COL_PARTS, s->stream));
  float* outs[1] = {out};
  SITE_I(site_red, col_reduce(s->part, COL_PARTS, 1, n, outs, s->stream));
  return STAGE_OK;
}

// Records the gradient reaching layer l's output when recording is on.
stage_status record_grad(stage_t* s, int l, const float* x, const bf16_t* bf, const bf16_t* hi,
                         const bf16_t* lo, const bf16_t* b) {
  if (!s->record_grads || (int)s->rec.size() != s->L) return STAGE_OK;
  const int64_t n = (int64_t)s->B * s->S * s->h;
  hipLaunchKernelGGL(grad_record_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                     s->stream, x, bf, hi, lo, b, s->rec[l], n);
  HIPCK(hipGetLastError());
  return STAGE_OK;
}

// Backward of an fp32 stage: every tensor in fp32, the weight gradients one
// GEMM at a time (split over tokens), the materialised attention path.
stage_status backward_f32(stage_t* s, const float* dy, float* dx) {
  using T = float;
  const int B = s->B, S = s->S, h = s->h, H = s->H, f = s->f;
  const int Tn = B * S;
  const int BH = B * H;
  hipStream_t st = s->stream;
  const float scale = 1.0f / sqrtf((float)HEAD_DIM);
  stage_status r;
  const T* dYcur = dy;
  for (int l = s->L - 1; l >= 0; --l) {
    Saved& v = s->saved[l];
    auto& p = s->param[l];
    auto& gr = s->grad[l];
    T* dZ2 = (T*)s->dZ2;
    T* dU = (T*)s->dU;
    T* dH1 = (T*)s->dH1;
    T* dZ1 = (T*)s->dZ1;
    T* dC = (T*)s->dC;
    T* dQKV = (T*)s->dQKV;
    const T* QKV = (const T*)v.QKV;
    const void* Wq = p[STAGE_W_QKV];
    const void* Wo = p[STAGE_W_O];
    const void* W1 = p[STAGE_W_1];
    const void* W2 = p[STAGE_W_2];
    const bool attn = has_attn(s, l), ffn = has_ffn(s, l);
    if ((r = record_grad(s, l, dYcur, nullptr, nullptr, nullptr, nullptr))) return r;
    auto dW = [&](int site, int site_red, const T* dYm, int64_t ld_dy, const T* Xn,
                  int64_t ld_x, int M, int N, float* out) -> stage_status {
      return wgrad<T>(s, site, site_red, dYm, ld_dy, Xn, ld_x, M, N, Tn, out);
    };
    // Gradient reaching H1: computed by the feed-forward half, or the
    // incoming dy when the stage ends at this layer's attention half.
    const T* dH1in = dYcur;
    if (ffn) {
      // Y = LN(Z2): dZ2, dgamma2, dbeta2, and db_2 = sum_t dZ2
      if ((r = ln_backward<T>(s, SITE_LN2_BWD, SITE_LN2_RED, dYcur, (const T*)v.xhat2, v.rstd2,
                              (const float*)p[STAGE_G2], dZ2, gr[STAGE_G2], gr[STAGE_BE2],
                              gr[STAGE_B_2], s->part, nullptr)))
        return r;
      // dW_2 = dZ2^T G
      if ((r = dW(SITE_W2_WGRAD, SITE_W2_RED, dZ2, h, (const T*)v.G, f, h, f, gr[STAGE_W_2]))) return r;
      // dU = (dZ2 W_2) * GELU'(U)
      {
        GemmArgs g = gemm_args(dZ2, h, W2, f, dU, f, Tn, f, h);
        g.aux = v.Gd;
        g.ldaux = f;
        SITE(FFN2_DGRAD, Gemm<T>::run(g, true, false, EPI_MUL, false, 1, st));
      }
      if ((r = col_sum<T>(s, SITE_B1_SUM, SITE_B1_RED, dU, f, gr[STAGE_B_1]))) return r;
      // dW_1 = dU^T H1
      if ((r = dW(SITE_W1_WGRAD, SITE_W1_RED, dU, f, (const T*)v.H1, h, f, h, gr[STAGE_W_1]))) return r;
      // dH1 = dZ2 + dU W_1 (the stage's dx when it starts at this layer's
      // feed-forward half)
      T* dH1out = attn ? dH1 : dx;
      {
        GemmArgs g = gemm_args(dU, f, W1, h, dH1out, h, Tn, h, f);
        g.aux = dZ2;
        g.ldaux = h;
        SITE(FFN1_DGRAD, Gemm<T>::run(g, true, false, EPI_RESID, false, 1, st));
      }
      dH1in = dH1out;
    }  // feed-forward half
    if (!attn) break;
    // H1 = LN(Z1): dZ1, dgamma1, dbeta1, db_o
    if ((r = ln_backward<T>(s, SITE_LN1_BWD, SITE_LN1_RED, dH1in, (const T*)v.xhat1, v.rstd1,
                            (const float*)p[STAGE_G1], dZ1, gr[STAGE_G1], gr[STAGE_BE1],
                            gr[STAGE_B_O], s->part, nullptr)))
      return r;
    // dW_o = dZ1^T C
    if ((r = dW(SITE_WO_WGRAD, SITE_WO_RED, dZ1, h, (const T*)v.C, h, h, h, gr[STAGE_W_O]))) return r;
    // dC = dZ1 W_o
    {
      GemmArgs g = gemm_args(dZ1, h, Wo, h, dC, h, Tn, h, h);
      SITE(OUT_DGRAD, Gemm<T>::run(g, true, false, EPI_STORE, false, 1, st));
    }
    // dP[b, j] = dC_bj V_bj^T (fp32, into the score buffer)
    {
      GemmArgs g = gemm_args(dC, h, QKV + 2 * h, 3 * h, s->scores, S, S, S, HEAD_DIM);
      g.zdiv = H;
      g.sA1 = (int64_t)S * h;
      g.sA2 = HEAD_DIM;
      g.sB1 = (int64_t)S * 3 * h;
      g.sB2 = HEAD_DIM;
      g.sC1 = (int64_t)H * S * S;
      g.sC2 = (int64_t)S * S;
      SITE(DP_BWD, Gemm<T>::run(g, true, true, EPI_STORE, true, BH, st));
    }
    // dS = scale * P * (dP - rowsum(dP * P))
    SITE(SOFTMAX_BWD, softmax_bwd<T>(s->scores, (const T*)v.P, (T*)s->dS, BH, S, S, scale, st));
    // dV_bj = P_bj^T dC_bj
    {
      GemmArgs g = gemm_args(v.P, S, dC, h, dQKV + 2 * h, 3 * h, S, HEAD_DIM, S);
      g.zdiv = H;
      g.sA1 = (int64_t)H * S * S;
      g.sA2 = (int64_t)S * S;
      g.sB1 = (int64_t)S * h;
      g.sB2 = HEAD_DIM;
      g.sC1 = (int64_t)S * 3 * h;
      g.sC2 = HEAD_DIM;
      SITE(DV_BWD, Gemm<T>::run(g, false, false, EPI_STORE, false, BH, st));
    }
    // dQ_bj = dS_bj K_bj
    {
      GemmArgs g = gemm_args(s->dS, S, QKV + h, 3 * h, dQKV, 3 * h, S, HEAD_DIM, S);
      g.zdiv = H;
      g.sA1 = (int64_t)H * S * S;
      g.sA2 = (int64_t)S * S;
      g.sB1 = (int64_t)S * 3 * h;
      g.sB2 = HEAD_DIM;
      g.sC1 = (int64_t)S * 3 * h;
      g.sC2 = HEAD_DIM;
      SITE(DQ_BWD, Gemm<T>::run(g, true, false, EPI_STORE, false, BH, st));
    }
    // dK_bj = dS_bj^T Q_bj
    {
      GemmArgs g = gemm_args(s->dS, S, QKV, 3 * h, dQKV + h, 3 * h, S, HEAD_DIM, S);
      g.zdiv = H;
      g.sA1 = (int64_t)H * S * S;
      g.sA2 = (int64_t)S * S;
      g.sB1 = (int64_t)S * 3 * h;
      g.sB2 = HEAD_DIM;
      g.sC1 = (int64_t)S * 3 * h;
      g.sC2 = HEAD_DIM;
      SITE(DK_BWD, Gemm<T>::run(g, false, false, EPI_STORE, false, BH, st));
    }
    if ((r = col_sum<T>(s, SITE_BQKV_SUM, SITE_BQKV_RED, dQKV, 3 * h, gr[STAGE_B_QKV]))) return r;
    // dW_qkv = dQKV^T X
    if ((r = dW(SITE_WQKV_WGRAD, SITE_WQKV_RED, dQKV, 3 * h, (const T*)v.X, h, 3 * h, h, gr[STAGE_W_QKV]))) return r;
    // dX = dZ1 + dQKV W_qkv  (the previous layer's dY, or the stage's dx)
    T* dXout = (l > 0) ? (T*)s->dY : dx;
    {
      GemmArgs g = gemm_args(dQKV, 3 * h, Wq, h, dXout, h, Tn, h, 3 * h);
      g.aux = dZ1;
      g.ldaux = h;
      SITE(QKV_DGRAD, Gemm<T>::run(g, true, false, EPI_RESID, false, 1, st));
    }
    dYcur = dXout;
  }
  return STAGE_OK;
}

// Gradient reaching a LayerNorm of a bf16 stage: the caller's bf16 tensor
// (at the stage's top, or below a stage boundary), or the fp32 sum of the
// residual branch, carried as its bf16 rounding hi plus the rounding
// residual lo (about 16 significant bits), and the data-gradient GEMM's
// bf16 product b.  The backward residual stream keeps that precision inside
// a stage: rounding it to bf16 at each of a layer's two residual additions
// is what the gradient error of a deep stage grows from (the product's own
// rounding is not: it enters the stream once).
struct GradIn {
  const bf16_t* bf;
  const bf16_t* hi;
  const bf16_t* lo;
  const bf16_t* b;
};

// Backward of a bf16 stage.  Per layer: the LayerNorm backward kernels take
// GradIn and write dZ in bf16 (GEMM operand) and fp32 (residual branch);
// the two data-gradient GEMMs whose output feeds a residual addition store
// their product in bf16 (the addition happens in the next LayerNorm
// backward); the data-gradient GEMMs read the weights as stored (n-major B
// operand, transposing LDS reads); the four weight gradients and
// the bias / LayerNorm column reductions run in one group launch and one
// reduction launch at the end of the layer.
stage_status backward_bf16(stage_t* s, const bf16_t* dy, bf16_t* dx) {
  using T = bf16_t;
  const int B = s->B, S = s->S, h = s->h, f = s->f;
  const int Tn = B * S;
  hipStream_t st = s->stream;
  stage_status r;
  GradIn gin{dy, nullptr, nullptr, nullptr};
  for (int l = s->L - 1; l >= 0; --l) {
    Saved& v = s->saved[l];
    auto& p = s->param[l];
    auto& gr = s->grad[l];
    T* dZ2 = (T*)s->dZ2;
    T* dU = (T*)s->dU;
    T* dZ1 = (T*)s->dZ1;
    T* dC = (T*)s->dC;
    T* dQKV = (T*)s->dQKV;
    const bool attn = has_attn(s, l), ffn = has_ffn(s, l);
    if ((r = record_grad(s, l, nullptr, gin.bf, gin.hi, gin.lo, gin.b))) return r;
    WgradJob wjobs[GEMM_GROUP_MAX];
    int nw = 0;
    ColJob cjobs[COLJOB_MAX];
    int nc = 0;
    // Gradient reaching H1: from the feed-forward half, or the incoming dy
    // when the stage ends at this layer's attention half.
    GradIn gh1 = gin;
    if (ffn) {
      // Y = LN(Z2): dZ2 (bf16 and fp32), dgamma2, dbeta2, db_2 = sum_t dZ2
      SITE(LN2_BWD, ln_bwd_bf16(gin.bf, gin.hi, gin.lo, gin.b, (const T*)v.xhat2, v.rstd2,
                                (const float*)p[STAGE_G2], dZ2, (T*)s->dz2lo, s->part2, Tn, h,
                                st));
      cjobs[nc++] = ColJob{s->part2, ln_bwd_blocks(Tn), 3, h,
                           {gr[STAGE_G2], gr[STAGE_BE2], gr[STAGE_B_2], nullptr}};
      // dW_2 = dZ2^T G
      wjobs[nw++] = {dZ2, h, v.G, f, h, f, gr[STAGE_W_2]};
      // dU = (dZ2 W_2) * GELU'(U); db_1 = column sums of dU (epilogue)
      {
        GemmArgs g = gemm_args(dZ2, h, p[STAGE_W_2], f, dU, f, Tn, f, h);
        g.aux = v.Gd;
        g.ldaux = f;
        g.tile = 1;
        g.colpart = s->colpart_ffn;
        SITE(FFN2_DGRAD, gemm_bf16(g, true, false, EPI_MUL, false, 1, st));
      }
      cjobs[nc++] = ColJob{s->colpart_ffn, (Tn + 127) / 128, 1, f,
                           {gr[STAGE_B_1], nullptr, nullptr, nullptr}};
      // dW_1 = dU^T H1
      wjobs[nw++] = {dU, f, v.H1, h, f, h, gr[STAGE_W_1]};
      // dH1 = dZ2 + dU W_1: the product in bf16, the sum in the first
      // LayerNorm's backward (or here, rounded, when this half is the
      // stage's first unit and dH1 is its dx)
      {
        GemmArgs g = gemm_args(dU, f, p[STAGE_W_1], h, s->prod, h, Tn, h, f);
        SITE(FFN1_DGRAD, gemm_bf16(g, true, false, EPI_STORE, false, 1, st));
      }
      if (attn) {
        gh1 = GradIn{nullptr, dZ2, (const T*)s->dz2lo, (const T*)s->prod};
      } else {
        HIPCK(add3_bf16(dZ2, (const T*)s->dz2lo, (const T*)s->prod, dx, (int64_t)Tn * h, st));
      }
    }  // feed-forward half
    if (attn) {
      // H1 = LN(Z1): dZ1 (bf16 and fp32), dgamma1, dbeta1, db_o
      SITE(LN1_BWD, ln_bwd_bf16(gh1.bf, gh1.hi, gh1.lo, gh1.b, (const T*)v.xhat1, v.rstd1,
                                (const float*)p[STAGE_G1], dZ1, (T*)s->dz1lo, s->part, Tn, h,
                                st));
      cjobs[nc++] = ColJob{s->part, ln_bwd_blocks(Tn), 3, h,
                           {gr[STAGE_G1], gr[STAGE_BE1], gr[STAGE_B_O], nullptr}};
      // dW_o = dZ1^T C
      wjobs[nw++] = {dZ1, h, v.C, h, h, h, gr[STAGE_W_O]};
      // dC = dZ1 W_o
      {
        GemmArgs g = gemm_args(dZ1, h, p[STAGE_W_O], h, dC, h, Tn, h, h);
        SITE(OUT_DGRAD, gemm_bf16(g, true, false, EPI_STORE, false, 1, st));
      }
      // Attention backward (recomputes P from the saved log-sum-exp): dQKV
      // and the column sums of db_qkv per 32-row block.
      AttnArgs aa = attn_args(s, (const T*)v.QKV, dQKV, v.lse);
      aa.o = (const T*)v.C;
      aa.o_lo = (const T*)v.Clo;
      aa.dout = dC;
      aa.colpart = s->colpart_qkv;
      SITE(ATTN_DQ, attn_backward_dq(aa, st));
      SITE(ATTN_DKDV, attn_backward_dkdv(aa, st));
      cjobs[nc++] = ColJob{s->colpart_qkv, B * ((S + 31) / 32), 1, 3 * h,
                           {gr[STAGE_B_QKV], nullptr, nullptr, nullptr}};
      // dW_qkv = dQKV^T X
      wjobs[nw++] = {dQKV, 3 * h, v.X, h, 3 * h, h, gr[STAGE_W_QKV]};
      // dX = dZ1 + dQKV W_qkv: the product in bf16; the sum in the previous
      // layer's second LayerNorm backward, or here, rounded, for the stage's dx
      {
        GemmArgs g = gemm_args(dQKV, 3 * h, p[STAGE_W_QKV], h, s->prod, h, Tn, h, 3 * h);
        SITE(QKV_DGRAD, gemm_bf16(g, true, false, EPI_STORE, false, 1, st));
      }
      if (l > 0) {
        gin = GradIn{nullptr, dZ1, (const T*)s->dz1lo, (const T*)s->prod};
      } else {
        HIPCK(add3_bf16(dZ1, (const T*)s->dz1lo, (const T*)s->prod, dx, (int64_t)Tn * h, st));
      }
    }
    if ((r = wgrad_group(s, wjobs, nw, cjobs, nc))) return r;
    if (!attn) break;
  }
  return STAGE_OK;
}

bool valid_dims(int hidden, int heads, int ffn, stage_dtype dtype) {
  return hidden >= 64 && hidden % 64 == 0 && hidden <= 2048 && heads >= 1 && hidden % heads == 0 &&
         hidden / heads == HEAD_DIM && ffn >= 64 && ffn % 64 == 0 &&
         (dtype == STAGE_F32 || dtype == STAGE_BF16);
}

// Shape of a stage holding units [first_unit, first_unit + n_units).
void set_units(stage_t* s, int first_unit, int n_units, int hidden, int heads, int ffn,
               stage_dtype dtype) {
  const int last = first_unit + n_units - 1;
  s->l0 = first_unit / 2;
  s->L = last / 2 - s->l0 + 1;
  s->ffn_first = (first_unit & 1) != 0;
  s->attn_last = (last & 1) == 0;
  s->h = hidden;
  s->H = heads;
  s->f = ffn;
  s->dtype = dtype;
  s->esz = dtype == STAGE_BF16 ? 2 : 4;
}

// Allocates and initialises the parameters and gradients of the halves the
// stage holds (a dry-run stage only counts the bytes).  Weights of global
// layer j are drawn from keys that depend on (seed, j, tensor) only, so a
// layer has the same weights in every stage that holds it.
stage_status build_params(stage_t* s, uint64_t seed) {
  s->param.assign(s->L, {});
  s->grad.assign(s->L, {});
  for (int l = 0; l < s->L; ++l) {
    const uint64_t gl = (uint64_t)(s->l0 + l);
    for (int w = 0; w < STAGE_NPARAM; ++w) {
      s->param[l][w] = nullptr;
      s->grad[l][w] = nullptr;
      if (!has_param(s, l, w)) continue;
      const int64_t n = param_numel(s, w);
      stage_status st = dev_alloc(s, s->allocs, &s->param[l][w], n * param_esz(s, w));
      if (!st) st = dev_alloc(s, s->allocs, (void**)&s->grad[l][w], n * 4);
      if (st) return st;
      if (s->dry_run) continue;
      const int blocks = (int)((n + 255) / 256);
      if (is_matrix(w)) {
        uint64_t key = splitmix64_mix(seed ^ ((gl * STAGE_NPARAM + w + 1) * GOLDEN));
        if (s->dtype == STAGE_BF16)
          hipLaunchKernelGGL(init_normal_kernel<bf16_t>, dim3(blocks), dim3(256), 0, s->stream,
                             (bf16_t*)s->param[l][w], n, key, 0.02);
        else
          hipLaunchKernelGGL(init_normal_kernel<float>, dim3(blocks), dim3(256), 0, s->stream,
                             (float*)s->param[l][w], n, key, 0.02);
      } else {
        float v = (w == STAGE_G1 || w == STAGE_G2) ? 1.0f : 0.0f;
        hipLaunchKernelGGL(fill_kernel, dim3(blocks), dim3(256), 0, s->stream,
                           (float*)s->param[l][w], n, v);
      }
      hipLaunchKernelGGL(fill_kernel, dim3(blocks), dim3(256), 0, s->stream, s->grad[l][w], n,
                         0.0f);
    }
  }
  if (s->dry_run) return STAGE_OK;
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
  if (e != hipSuccess)
    return fail(s, STAGE_EHIP, std::string("initialisation kernels: ") + hipGetErrorString(e));
  return STAGE_OK;
}

// Device bytes of a dry-run stage of units [first_unit, first_unit +
// n_units) after a forward of batch x seq tokens; -1 on failure.
int64_t dry_bytes(int first_unit, int n_units, int hidden, int heads, int ffn, int batch, int seq,
                  stage_dtype dtype) {
  stage_t d;
  d.dry_run = true;
  set_units(&d, first_unit, n_units, hidden, heads, ffn, dtype);
  if (build_params(&d, 0) != STAGE_OK || ensure_activations(&d, batch, seq) != STAGE_OK) return -1;
  return d.bytes_param + d.bytes_act;
}

stage_status check_layer(stage_t* s, int layer, int which, int nwhich) {
  if (!s) return STAGE_EINVAL;
  if (layer < 0 || layer >= s->L) return fail(s, STAGE_EINVAL, "layer index out of range");
  if (which < 0 || which >= nwhich) return fail(s, STAGE_EINVAL, "tensor index out of range");
  return STAGE_OK;
}

// A parameter (or its gradient) of a half-layer the stage holds.
stage_status check_param(stage_t* s, int layer, int which) {
  stage_status st = check_layer(s, layer, which, STAGE_NPARAM);
  if (st) return st;
  if (!has_param(s, layer, which))
    return fail(s, STAGE_EINVAL, "the stage does not hold this half of the layer");
  return STAGE_OK;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

stage_status stage_init(int L, int hidden, int heads, int ffn, uint64_t seed, stage_dtype dtype,
                        void* hip_stream, stage_t** out) {
  if (L < 1 || L > (1 << 29)) {
    g_init_err = "invalid dims: need 1 <= L <= 2^29";
    if (out) *out = nullptr;
    return STAGE_EINVAL;
  }
  return stage_init_units(0, 2 * L, hidden, heads, ffn, seed, dtype, hip_stream, out);
}

stage_status stage_init_units(int first_unit, int n_units, int hidden, int heads, int ffn,
                              uint64_t seed, stage_dtype dtype, void* hip_stream, stage_t** out) {
  g_init_err.clear();
  if (!out) {
    g_init_err = "null out";
    return STAGE_EINVAL;
  }
  *out = nullptr;
  if (first_unit < 0 || n_units < 1 || n_units > (1 << 30) - first_unit) {
    g_init_err = "invalid units: need first_unit >= 0, n_units >= 1, first_unit + n_units <= 2^30";
    return STAGE_EINVAL;
  }
  if (!valid_dims(hidden, heads, ffn, dtype)) {
    g_init_err = "invalid dims: need hidden a multiple of 64 and <= 2048, "
                 "hidden / heads == 64, ffn a multiple of 64";
    return STAGE_EINVAL;
  }
  stage_t* s = new (std::nothrow) stage_t();
  if (!s) return STAGE_ENOMEM;
  set_units(s, first_unit, n_units, hidden, heads, ffn, dtype);
  s->stream = (hipStream_t)hip_stream;
  stage_status st = build_params(s, seed);
  if (!st) {
    const hipError_t e = resolve_scratch(&s->device);
    if (e != hipSuccess)
      st = fail(s, STAGE_EHIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
  }
  if (st) {
    g_init_err = s->err;
    for (void* p : s->allocs) (void)hipFree(p);
    delete s;
    return st;
  }
  *out = s;
  return STAGE_OK;
}

stage_status stage_set_stream(stage_t* s, void* hip_stream) {
  if (!s) return STAGE_EINVAL;
  s->stream = (hipStream_t)hip_stream;
  return STAGE_OK;
}

stage_status stage_record_grads(stage_t* s, int on) {
  if (!s) return STAGE_EINVAL;
  if (on != 0 && on != 1) return fail(s, STAGE_EINVAL, "on must be 0 or 1");
  if ((bool)on != s->record_grads) {
    s->record_grads = on != 0;
    s->cap_T = -1;  // the next forward allocates (or drops) the record
    s->have_ctx = false;
  }
  return STAGE_OK;
}

stage_status stage_forward(stage_t* s, const void* x, const uint8_t* key_mask, int batch, int seq,
                           void* y) {
  if (!s) return STAGE_EINVAL;
  s->err.clear();
  if (batch < 0 || seq < 0) return fail(s, STAGE_EINVAL, "negative batch or seq");
  const int64_t T = (int64_t)batch * seq;
  if (T > 0 && (!x || !y)) return fail(s, STAGE_EINVAL, "null x or y");
  if (T > 0 && x == y) return fail(s, STAGE_EINVAL, "x and y may not alias");
  // bf16 GEMM operands are read through buffer resources (32-bit byte
  // extents): the widest activation, [T, max(3h, f)], must stay below 2 GiB.
  if (T * std::max(3 * s->h, s->f) * (s->dtype == STAGE_BF16 ? 2 : 1) >= (int64_t)1 << 31)
    return fail(s, STAGE_EINVAL, "batch * seq too large");
  if (s->dtype == STAGE_F32 && (int64_t)batch * s->H * seq * seq >= (int64_t)1 << 40)
    return fail(s, STAGE_EINVAL, "score matrix too large");
  stage_status st = ensure_activations(s, batch, seq);
  if (st) return st;
  s->B = batch;
  s->S = seq;
  s->have_ctx = false;
  s->rec_valid = false;
  if (T == 0) {
    s->have_ctx = true;
    return STAGE_OK;
  }
  if (key_mask) {
    HIPCK(hipMemcpyAsync(s->mask, key_mask, (size_t)T, hipMemcpyDeviceToDevice, s->stream));
  } else {
    hipLaunchKernelGGL(ones_u8_kernel, dim3((unsigned)((T + 255) / 256)), dim3(256), 0, s->stream,
                       s->mask, T);
    HIPCK(hipGetLastError());
  }
  st = s->dtype == STAGE_BF16 ? forward_impl<bf16_t>(s, (const bf16_t*)x, (bf16_t*)y)
                              : forward_impl<float>(s, (const float*)x, (float*)y);
  if (st) return st;
  s->have_ctx = true;
  return STAGE_OK;
}

stage_status stage_backward(stage_t* s, const void* dy, void* dx) {
  if (!s) return STAGE_EINVAL;
  s->err.clear();
  if (!s->have_ctx) return fail(s, STAGE_ESTATE, "stage_backward needs a preceding stage_forward");
  const int64_t T = (int64_t)s->B * s->S;
  if (T > 0 && (!dy || !dx)) return fail(s, STAGE_EINVAL, "null dy or dx");
  s->have_ctx = false;
  if (T == 0) {
    for (int l = 0; l < s->L; ++l)
      for (int w = 0; w < STAGE_NPARAM; ++w) {
        if (!has_param(s, l, w)) continue;
        int64_t n = param_numel(s, w);
        hipLaunchKernelGGL(fill_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                           s->stream, s->grad[l][w], n, 0.0f);
      }
    HIPCK(hipGetLastError());
    return STAGE_OK;
  }
  stage_status st = s->dtype == STAGE_BF16 ? backward_bf16(s, (const bf16_t*)dy, (bf16_t*)dx)
                                           : backward_f32(s, (const float*)dy, (float*)dx);
  s->rec_valid = st == STAGE_OK && s->record_grads && (int)s->rec.size() == s->L;
  return st;
}

stage_status stage_backward_noalloc(stage_t* s, const void* dy, void* dx) {
  if (!s) return STAGE_EINVAL;
  s->err.clear();
  if (!s->have_ctx) return fail(s, STAGE_ESTATE, "stage_backward needs a preceding stage_forward");
  float* base = scratch_of(s->device);
  if (!base) return fail(s, STAGE_ESTATE, "static scratch not resolved for the stage's device");
  // The backward's partial buffers, laid out in the scratch (256-byte
  // aligned slices).  Every element the kernels read is written earlier in
  // the same call, so nothing needs clearing.
  const int64_t T = (int64_t)s->B * s->S;
  const int64_t h = s->h, f = s->f;
  const int64_t nlnb = ln_bwd_blocks((int)T);
  const size_t need_splitk = splitk_need(s, T);
  const size_t n_part = (size_t)std::max<int64_t>(nlnb * 3 * h, (int64_t)COL_PARTS * std::max<int64_t>(3 * h, f));
  const size_t n_part2 = (size_t)(nlnb * 3 * h);
  const size_t n_cffn = (size_t)(((T + 127) / 128) * f);
  const size_t n_cqkv = (size_t)((int64_t)s->B * ((s->S + 31) / 32) * 3 * h);
  size_t off = 0;
  auto take = [&](size_t elems) {
    float* p = base + off;
    off += (std::max<size_t>(elems, 1) + 63) / 64 * 64;
    return p;
  };
  float* sk = take(need_splitk);
  float* pt = take(n_part);
  float* pt2 = take(n_part2);
  float* cf = take(n_cffn);
  float* cq = take(n_cqkv);
  if (off * sizeof(float) > NOALLOC_SCRATCH_BYTES)
    return fail(s, STAGE_EINVAL,
                "stage_backward_noalloc: this batch needs " + std::to_string(off * sizeof(float)) +
                    " bytes of partial results; the static scratch holds " +
                    std::to_string(NOALLOC_SCRATCH_BYTES) + " (use stage_backward)");
  float* const keep[5] = {s->splitk, s->part, s->part2, s->colpart_ffn, s->colpart_qkv};
  const size_t keep_elems = s->splitk_elems;
  s->splitk = sk;
  s->splitk_elems = need_splitk;
  s->part = pt;
  s->part2 = pt2;
  s->colpart_ffn = cf;
  s->colpart_qkv = cq;
  s->no_alloc = true;
  const stage_status st = stage_backward(s, dy, dx);
  s->no_alloc = false;
  s->splitk = keep[0];
  s->splitk_elems = keep_elems;
  s->part = keep[1];
  s->part2 = keep[2];
  s->colpart_ffn = keep[3];
  s->colpart_qkv = keep[4];
  return st;
}

stage_status stage_param(stage_t* s, int layer, int which, void** dev_ptr, int64_t* numel,
                         stage_dtype* dtype) {
  stage_status st = check_param(s, layer, which);
  if (st) return st;
  if (dev_ptr) *dev_ptr = s->param[layer][which];
  if (numel) *numel = param_numel(s, which);
  if (dtype) *dtype = is_matrix(which) ? s->dtype : STAGE_F32;
  return STAGE_OK;
}

stage_status stage_grad(stage_t* s, int layer, int which, float** dev_ptr, int64_t* numel) {
  stage_status st = check_param(s, layer, which);
  if (st) return st;
  if (dev_ptr) *dev_ptr = s->grad[layer][which];
  if (numel) *numel = param_numel(s, which);
  return STAGE_OK;
}

stage_status stage_set_param(stage_t* s, int layer, int which, const void* src, size_t bytes) {
  stage_status st = check_param(s, layer, which);
  if (st) return st;
  if (!src) return fail(s, STAGE_EINVAL, "null src");
  size_t want = (size_t)param_numel(s, which) * param_esz(s, which);
  if (bytes != want) return fail(s, STAGE_EINVAL, "byte count does not match the parameter");
  HIPCK(hipMemcpyAsync(s->param[layer][which], src, bytes, hipMemcpyDefault, s->stream));
  HIPCK(hipStreamSynchronize(s->stream));
  return STAGE_OK;
}

static void* saved_ptr(stage_t* s, int layer, int which, size_t* bytes) {
  const int64_t T = (int64_t)s->B * s->S;
  const Saved& v = s->saved[layer];
  const size_t e = s->esz;
  // Tensors of a half-layer the stage does not hold have no storage (H1 of
  // a layer whose feed-forward half is absent went to the stage output).
  const bool attn = has_attn(s, layer), ffn = has_ffn(s, layer);
  *bytes = 0;
  switch (which) {
    case STAGE_SAVED_X: if (attn) *bytes = T * s->h * e; return attn ? v.X : nullptr;
    case STAGE_SAVED_QKV: if (attn) *bytes = T * 3 * s->h * e; return attn ? v.QKV : nullptr;
    case STAGE_SAVED_CTX: if (attn) *bytes = T * s->h * e; return attn ? v.C : nullptr;
    case STAGE_SAVED_H1: if (ffn) *bytes = T * s->h * e; return ffn ? v.H1 : nullptr;
    case STAGE_SAVED_GD: if (ffn) *bytes = T * s->f * e; return ffn ? v.Gd : nullptr;
    case STAGE_SAVED_G: if (ffn) *bytes = T * s->f * e; return ffn ? v.G : nullptr;
  }
  return nullptr;
}

size_t stage_tensor_bytes(stage_t* s, int kind, int layer, int which) {
  if (!s || layer < 0 || layer >= s->L) return 0;
  if ((kind == 0 || kind == 1) && (which < 0 || which >= STAGE_NPARAM || !has_param(s, layer, which)))
    return 0;
  if (kind == 0) return (size_t)param_numel(s, which) * param_esz(s, which);
  if (kind == 1) return (size_t)param_numel(s, which) * 4;
  if (kind == 2 && which >= 0 && which < STAGE_NSAVED && (int)s->saved.size() == s->L) {
    size_t b;
    saved_ptr(s, layer, which, &b);
    return b;
  }
  if (kind == 3 && which == 0 && s->rec_valid) return (size_t)s->B * s->S * s->h * 4;
  return 0;
}

stage_status stage_read(stage_t* s, int kind, int layer, int which, void* dst, size_t bytes) {
  if (!s) return STAGE_EINVAL;
  if (!dst) return fail(s, STAGE_EINVAL, "null dst");
  const void* src = nullptr;
  size_t want = 0;
  if (kind == 0 || kind == 1) {
    stage_status st = check_param(s, layer, which);
    if (st) return st;
    src = kind == 0 ? s->param[layer][which] : (const void*)s->grad[layer][which];
    want = (size_t)param_numel(s, which) * (kind == 0 ? param_esz(s, which) : 4);
  } else if (kind == 2) {
    stage_status st = check_layer(s, layer, which, STAGE_NSAVED);
    if (st) return st;
    if ((int)s->saved.size() != s->L) return fail(s, STAGE_ESTATE, "no saved activations");
    src = saved_ptr(s, layer, which, &want);
    if (!src) return fail(s, STAGE_EINVAL, "the stage does not hold this half of the layer");
  } else if (kind == 3) {
    stage_status st = check_layer(s, layer, which, 1);
    if (st) return st;
    if (!s->rec_valid)
      return fail(s, STAGE_ESTATE, "no recorded gradients: enable stage_record_grads, then run "
                                   "a forward and a backward");
    src = s->rec[layer];
    want = (size_t)s->B * s->S * s->h * 4;
  } else {
    return fail(s, STAGE_EINVAL, "kind must be 0 (param), 1 (grad), 2 (saved) or 3 (recorded "
                                 "gradient)");
  }
  if (bytes != want) return fail(s, STAGE_EINVAL, "byte count does not match the tensor");
  if (want == 0) return STAGE_OK;
  HIPCK(hipMemcpyAsync(dst, src, want, hipMemcpyDefault, s->stream));
  HIPCK(hipStreamSynchronize(s->stream));
  return STAGE_OK;
}

stage_status stage_trace_site(stage_t* s, int site) {
  if (!s) return STAGE_EINVAL;
  if (site < -1 || site >= SITE_COUNT) return fail(s, STAGE_EINVAL, "unknown site");
  return stage_trace_mask(s, site < 0 ? 0 : (uint64_t)1 << site);
}

stage_status stage_trace_mask(stage_t* s, uint64_t mask) {
  if (!s) return STAGE_EINVAL;
  if (SITE_COUNT < 64 && (mask >> SITE_COUNT) != 0) return fail(s, STAGE_EINVAL, "unknown site");
  s->trace_mask = mask;
  s->events_used = 0;
  return STAGE_OK;
}

stage_status stage_trace_read(stage_t* s, int* launches, double* total_ms) {
  if (!s) return STAGE_EINVAL;
  HIPCK(hipStreamSynchronize(s->stream));
  double tot = 0.0;
  int n = 0;
  for (size_t i = 0; i + 1 < s->events_used; i += 2) {
    float ms = 0.0f;
    HIPCK(hipEventElapsedTime(&ms, s->events[i], s->events[i + 1]));
    tot += ms;
    ++n;
  }
  s->events_used = 0;
  if (launches) *launches = n;
  if (total_ms) *total_ms = tot;
  return STAGE_OK;
}

stage_status stage_device_bytes(const stage_t* s, int64_t* bytes) {
  if (!s || !bytes) return STAGE_EINVAL;
  *bytes = s->bytes_param + s->bytes_act;
  return STAGE_OK;
}

stage_status stage_memory_model(int hidden, int heads, int ffn, int batch, int seq,
                                stage_dtype dtype, int64_t* per_layer, int64_t* shared) {
  int64_t attn, ffn_b, sh;
  stage_status st = stage_memory_model_units(hidden, heads, ffn, batch, seq, dtype, &attn, &ffn_b, &sh);
  if (st) return st;
  if (!per_layer || !shared) return STAGE_EINVAL;
  *per_layer = attn + ffn_b;
  *shared = sh;
  return STAGE_OK;
}

stage_status stage_memory_model_units(int hidden, int heads, int ffn, int batch, int seq,
                                      stage_dtype dtype, int64_t* attn_unit, int64_t* ffn_unit,
                                      int64_t* shared) {
  if (!attn_unit || !ffn_unit || !shared) return STAGE_EINVAL;
  if (!valid_dims(hidden, heads, ffn, dtype) || batch < 0 || seq < 0) return STAGE_EINVAL;
  // The same allocation calls as stage_init_units and stage_forward, on
  // stages that only count bytes: one attention half, one feed-forward
  // half, and both.  A stage's bytes are the workspace plus the sum over
  // its units.
  const int64_t a = dry_bytes(0, 1, hidden, heads, ffn, batch, seq, dtype);
  const int64_t f = dry_bytes(1, 1, hidden, heads, ffn, batch, seq, dtype);
  const int64_t af = dry_bytes(0, 2, hidden, heads, ffn, batch, seq, dtype);
  if (a < 0 || f < 0 || af < 0) return STAGE_EINVAL;
  *shared = a + f - af;
  *attn_unit = a - *shared;
  *ffn_unit = f - *shared;
  return STAGE_OK;
}

int stage_site_count(void) { return SITE_COUNT; }

const char* stage_site_name(int site) {
  return (site >= 0 && site < SITE_COUNT) ? SITE_NAMES[site] : "";
}

const char* stage_last_error(const stage_t* s) { return s ? s->err.c_str() : g_init_err.c_str(); }

void stage_destroy(stage_t* s) {
  if (!s) return;
  (void)hipStreamSynchronize(s->stream);
  free_activations(s);
  for (void* p : s->allocs) (void)hipFree(p);
  for (hipEvent_t e : s->events) (void)hipEventDestroy(e);
  delete s;
}

}  // extern "C"

// Internal declarations of libsara (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/sara.h"

namespace sara {

// ---------------------------------------------------------------------------
// constants
// ---------------------------------------------------------------------------
constexpr int kBlockTok = 16;        // KV page size in tokens
constexpr int kAttnSplit = 256;      // tokens per context split (fp32 VALU attention)
constexpr int kAttnChunks = 16;      // KV pages per context split (bf16 MFMA prefill attention)
constexpr int kDecPpw = 2;           // KV pages per wave in the decode attention
constexpr int kDecPages = 4 * kDecPpw;  // KV pages per context split in the decode attention
constexpr int kMaxSplitsDec = 12;    // split-K partials of a decode GEMM (summed in one batch; a multiple of 4)
constexpr int kAttnTile = 64;        // tokens per LDS tile inside a split
constexpr int kSampleChunks = 16;    // vocabulary chunks per sampled row
constexpr int kTopPChunks = 16;      // vocabulary chunks per row in the top-p passes
constexpr int kTopPBins = 2048;      // 11-bit digits of the top-p radix descent
// static scratch of the allocation-free sampler (sara_sample_logits_noalloc)
constexpr int kNoAllocMaxRows = SARA_NOALLOC_MAX_ROWS;
constexpr int kNoAllocMaxToppRows = SARA_NOALLOC_MAX_TOPP_ROWS;
constexpr size_t kNoAllocScratchBytes = SARA_NOALLOC_SCRATCH_BYTES;
constexpr int kCtlThreads = 1024;    // threads of the single-workgroup controller
constexpr int kMaxQueue = 4096;      // pending rollouts held in LDS by the refill
constexpr int kMaxSlots = 4096;
constexpr int kMaxGroup = 8;         // query heads per KV head
constexpr uint64_t kSeedRXor = 0xD1B54A32D192ED03ull;

// ---------------------------------------------------------------------------
// device-side state
// ---------------------------------------------------------------------------
struct Ctl {
  int64_t budget_left, rollouts, tokens;
  int64_t n_dec, n_draw, n_asg, n_fin;
  int32_t next_uid, nA, nC, nAb;
  int32_t qlen, t, done, error;
  int32_t M, dirty, running, pad_;
};

// One query row of a decode or prefill batch.
struct RowDesc {
  int32_t tok;      // input token id
  int32_t pos;      // position of the token (KV append position)
  int32_t plen;     // tokens of the sequence's shared prompt segment (P - 1)
  int32_t tab;      // block-table row
  int32_t slot;     // decode: slot index; prefill: -1
  int32_t rid;      // decode: rollout id uid*k + j
  int32_t gen;      // decode: generated index i
  int32_t uid;
  // KV extents: page ids of a sequence are kv0 + e for its shared prompt
  // segment (entries e < PB of its block-table row) and kv1 + e for its
  // private segment (decode rows; -1 for prefill rows)
  int32_t kv0;
  int32_t kv1;
};

// One work item of the decode attention: context split c of decode row i,
// with the row's page extents and segment lengths, so that an attention
// block needs no further load before its page loads.
struct AttnItem {
  int32_t i, c, kv0, kv1;   // row, split, page extents (as in RowDesc)
  int32_t pl, vcnt, pad0, pad1;  // prompt positions attended, private positions
};

// Parameters every controller kernel reads.
struct CtlParams {
  int32_t B, k, n0, commit_min, U, S, mode, bits, max_new, PB, SB, MAXB, eos, Qcap;
  double tau, a0, b0, prior;
  uint64_t seed;
  int32_t step;
  uint32_t forced_eos;
  float temperature;
  float top_p;                   // < 1: nucleus sampling over fp32 logits
  int32_t has_flen;
  int32_t has_prior;             // per-prompt priors (warm start) in place of (a0, b0, prior)
};

}  // namespace sara

// ---------------------------------------------------------------------------
// host-side context
// ---------------------------------------------------------------------------
struct sara_ctx {
  sara_model_desc md;
  sara_alloc_desc ad;
  hipStream_t stream = nullptr;
  int device = 0;

  // derived sizes
  int L = 0, d = 0, hq = 0, hkv = 0, hd = 0, ffn = 0, V = 0, G = 0, nqkv = 0, qdim = 0;
  int U = 0, k = 0, S = 0, PB = 0, SB = 0, MAXB = 0, max_pos = 0, Qcap = 0;
  int64_t n_blocks = 0;
  int elt = 2;                    // bytes per stored element (2 bf16, 4 fp32)
  int prefill_rows = 0;           // rows per prefill chunk
  int attn_splits_max = 0;
  int dec_splits_max = 0;         // context splits of the decode attention
  int64_t ws_floats = 0;

  // weights (model dtype)
  void* embed = nullptr;
  void* lm_head = nullptr;
  std::vector<void*> w_qkv, w_o, w_gu, w_d;
  float* norms = nullptr;         // [2L+1][d]: attn l, ffn l, final

  // KV cache [L][n_blocks][hkv][16][hd], block tables [(S+U)][MAXB]
  void* kc = nullptr;
  void* vc = nullptr;
  int32_t* btab = nullptr;
  float2* rope = nullptr;         // [max_pos][hd/2] (cos, sin)
  float2* row_rope = nullptr;     // [S][hd/2] (cos, sin) at each decode row's position
  sara::AttnItem* attn_items = nullptr; // [S * dec_splits_max] decode attention work list of the step
  int32_t* attn_nitems = nullptr; // its length
  int attn_dec_grid = 0;          // blocks of the decode attention that are resident at once
  int qkv_spread = 0;             // z blocks sharing a decode batch's tiles in the q|k|v kernel

  // prompt pool (library copies)
  int32_t* tok = nullptr;
  int32_t* off = nullptr;         // [U+1]
  int32_t* pre = nullptr;         // [U+1] prefix sums of (P - 1)
  double* p = nullptr;
  int32_t* flen = nullptr;        // [U*k]
  int has_flen = 0;
  int64_t tok_cap = 0;
  std::vector<int32_t> h_off;

  // controller state
  sara::Ctl* ctl = nullptr;
  int32_t *status = nullptr, *n_iss = nullptr, *n_done = nullptr, *succ = nullptr, *infl = nullptr;
  double* peff = nullptr;
  // history warm start: per-prompt priors of the pool ([U] each) and the
  // caller's prompt-set state (set by sara_set_warm_start)
  double *prior_a = nullptr, *prior_b = nullptr, *prior_p = nullptr;
  const int32_t* warm_ids = nullptr;
  double *warm_a = nullptr, *warm_b = nullptr;
  int32_t warm_n = 0;
  bool warm_step = false;         // the current step began with warm start set
  int32_t *slot_uid = nullptr, *slot_j = nullptr, *slot_gen = nullptr, *fin = nullptr;
  uint64_t* slot_hash = nullptr;
  int32_t* active = nullptr;
  uint64_t* queue = nullptr;
  int32_t *out_tok = nullptr, *samp_tok = nullptr, *r_len = nullptr, *r_reward = nullptr;
  int64_t *log_dec = nullptr, *log_draw = nullptr, *log_asg = nullptr, *log_fin = nullptr;
  int64_t cap_dec = 0, cap_draw = 0, cap_asg = 0, cap_fin = 0;

  // activations and workspaces
  sara::RowDesc* rows = nullptr;  // [row_cap]
  int32_t* rows_M = nullptr;      // device row count of the prefill chunk
  int row_cap = 0;
  float* h = nullptr;             // [row_cap][d] residual stream
  void* x = nullptr;              // [row_cap][max(d, ffn, qdim)] GEMM input (model dtype)
  void* qbuf = nullptr;           // [row_cap][hq][hd]
  void* xa = nullptr;             // [row_cap][ffn] SwiGLU output (bf16 models)
  float* ws = nullptr;            // GEMM partial outputs
  float* attn_part = nullptr;
  float* samp_best = nullptr;
  int32_t* samp_idx = nullptr;
  bool topp = false;              // top_p < 1: nucleus sampler after the LM head
  float* topp_logits = nullptr;   // [S][V] fp32 logits for it (bf16 models)
  float* topp_max = nullptr;      // [S][kTopPChunks] chunk maxima of z
  unsigned long long* topp_hist = nullptr;   // [S][kTopPChunks][kTopPBins] chunk weight histograms
  uint32_t* topp_thr = nullptr;   // [S] key bits of each row's nucleus threshold z* (all of them at the end)
  unsigned long long* topp_above = nullptr;    // [S] weight above the descent's current range
  unsigned long long* topp_target = nullptr;   // [S] target weight t

  // GRPO of committed groups
  int32_t* g_off = nullptr;
  float* g_r = nullptr;
  float* g_adv = nullptr;
  int32_t* g_n = nullptr;         // committed count used for the CSR

  // graph replay
  hipGraphExec_t graph_exec = nullptr;
  hipGraph_t graph = nullptr;
  int graph_iters = 0;
  const int32_t* graph_forced = nullptr;
  int32_t* h_done = nullptr;      // pinned

  std::vector<void*> owned;       // device allocations freed by sara_destroy
  // per-launch profiling of eager decode steps
  struct ProfRec { int cls, N, K, e0, e1; };
  bool prof_enabled = false;
  bool prof_active = false;
  bool capturing = false;
  bool in_prefill = false;
  std::vector<hipEvent_t> prof_events;
  std::vector<ProfRec> prof_recs;
  int prof_next_event = 0;
  int prof_pending = -1;          // event pair reserved for the next launch (-1: none)
  int prof_last = -1;             // event pair of the last profiled launch
  std::vector<sara_kernel_profile> prof_tot;
  sara::CtlParams cp;              // host copy
  sara::CtlParams* cp_dev = nullptr;
  int step_index = 0;
  bool in_step = false;
};

namespace sara {

// one class per kernel (per template instance for the GEMMs, as a kernel
// trace names them), then a breakdown of the GEMMs by weight matrix
enum ProfClass { kPGemmN1, kPGemmGU, kPGemmLM, kPAttn, kPCombine, kPQkv, kPResNorm, kPSwiglu,
                 kPEmbed, kPSampleP, kPSampleF, kPRows, kPCopy, kPQkvRope, kPToppMax, kPToppHist, kPToppSel,
                 kPGemmO1, kPGemmQkv, kPGemmO, kPGemmGu, kPGemmD, kPGemmLm, kPNumClasses };
extern const char* const kProfNames[kPNumClasses];
void prof_begin(sara_ctx* c);
void prof_end(sara_ctx* c, int cls, int N = 0, int K = 0);
int prof_collect(sara_ctx* c);

void set_error(const std::string& msg);
int hip_fail(hipError_t e, const char* what);

// launchers (model)
int launch_prefill(sara_ctx* c);
int launch_decode(sara_ctx* c, const int32_t* forced, float* logits, int model_free);
// launchers (controller)
int launch_reset(sara_ctx* c);
int launch_decide(sara_ctx* c);
int launch_warm_priors(sara_ctx* c);
int launch_warm_update(sara_ctx* c, double lambda);
int launch_refill(sara_ctx* c);
int launch_finish(sara_ctx* c, float eps);
int launch_peff(const double* alpha, const double* beta, const int32_t* n, const int32_t* s, int k, int count,
                double* out, hipStream_t st);
int launch_poll(sara_ctx* c, int32_t* d_host);
int launch_grpo(const float* r, const int32_t* off, int n_groups, float eps, float* adv,
                hipStream_t st);
int launch_sample_rows(const float* logits, int n_rows, int V, const int32_t* rid,
                       const int32_t* pos, uint64_t seed, int step, float temp, float top_p, int eos,
                       uint32_t feos, int32_t* tok, hipStream_t st);
int launch_sample_rows_noalloc(const float* logits, int n_rows, int V, const int32_t* rid, const int32_t* pos,
                               uint64_t seed, int step, float temp, float top_p, int eos, uint32_t feos,
                               int32_t* tok, hipStream_t st);
int launch_convert_norms(sara_ctx* c, const void* const* w);
int launch_gumbel_check(double* h_out, hipStream_t st);
int launch_tile_weights(sara_ctx* c, const void* src, void* dst, int rows, int K, int tile_mul, int tile_add,
                        int dst_rows);
int launch_tile_weights_pairs(sara_ctx* c, const void* src, void* dst, int n_rows, int K, int head_off);

// ---------------------------------------------------------------------------
// device helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t b = __float_as_uint(f);
  return (uint16_t)((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}
template <typename T> __device__ __forceinline__ float ld_f32(const T* p, size_t i);
template <> __device__ __forceinline__ float ld_f32<float>(const float* p, size_t i) { return p[i]; }
template <> __device__ __forceinline__ float ld_f32<uint16_t>(const uint16_t* p, size_t i) {
  return bf16_to_f32(p[i]);
}
template <typename T> __device__ __forceinline__ void st_f32(T* p, size_t i, float v);
template <> __device__ __forceinline__ void st_f32<float>(float* p, size_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st_f32<uint16_t>(uint16_t* p, size_t i, float v) {
  p[i] = f32_to_bf16(v);
}

// Philox4x32-10 (Salmon et al., SC'11): 10 rounds of two 32x32->64 products
// and a Weyl-sequence key schedule.
struct U32x4 { uint32_t x, y, z, w; };
__device__ __forceinline__ U32x4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                               uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    // full 64-bit products: one multiply instruction per product on gfx950
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0, p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t lo0 = (uint32_t)p0, hi0 = (uint32_t)(p0 >> 32);
    const uint32_t lo1 = (uint32_t)p1, hi1 = (uint32_t)(p1 >> 32);
    uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
  }
  return U32x4{c0, c1, c2, c3};
}
__device__ __forceinline__ void sampler_key(uint64_t seed, int32_t step, uint32_t& k0, uint32_t& k1) {
  k0 = (uint32_t)seed;
  k1 = (uint32_t)(seed >> 32) ^ (uint32_t)step;
}

// SplitMix64 output finalizer (Steele, Lea, Flood, OOPSLA'14).
__host__ __device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
__device__ __forceinline__ uint64_t reward_hash_init(uint64_t seed, int32_t step, int32_t uid) {
  return mix64((seed ^ kSeedRXor) ^ mix64(((uint64_t)(uint32_t)step << 32) + (uint64_t)(uint32_t)uid));
}

// Proposition 1 (Eq. peff): posterior predictive probability that the
// completed group of size k is mixed, given n observed rollouts with s
// successes under the prior Beta(a0, b0).  Both saturation terms apply when
// n = 0; a complete unmixed group has probability 0.
__device__ __forceinline__ double peff_dev(int n, int s, int k, double a0, double b0) {
  if (s >= 1 && n - s >= 1) return 1.0;
  int r = k - n;
  if (r <= 0) return 0.0;
  double a = a0 + (double)s, b = b0 + (double)(n - s);
  double lb = lgamma(a) + lgamma(b) - lgamma(a + b);
  double psat = 0.0;
  if (s == 0) psat += exp(lgamma(a) + lgamma(b + r) - lgamma(a + b + r) - lb);
  if (s == n) psat += exp(lgamma(a + r) + lgamma(b) - lgamma(a + b + r) - lb);
  return 1.0 - psat;
}

}  // namespace sara

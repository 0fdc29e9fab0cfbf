// C ABI of libsara: context lifetime, step driving, graph replay, readback.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <cstdio>
#include <string>
#include <vector>

#include "sara_internal.h"

using namespace sara;

#define HIP_TRY(expr, what)                         \
  do {                                              \
    hipError_t e_ = (expr);                         \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

namespace sara {

static thread_local std::string g_err;

void set_error(const std::string& msg) { g_err = msg; }

int hip_fail(hipError_t e, const char* what) {
  set_error(std::string(what) + ": " + hipGetErrorString(e));
  return SARA_EHIP;
}

static int einval(const std::string& msg) {
  set_error(msg);
  return SARA_EINVAL;
}

const char* const kProfNames[kPNumClasses] = {
    "k_gemm_bf16_lds<1,8,64,0,0>", "k_gemm_bf16_lds<2,8,64,1,0>", "k_gemm_bf16_lds<2,8,64,2,0>",
    "k_attn_dec<128>", "k_attn_combine", "k_qkv_epilogue", "k_residual_norm_f4", "k_swiglu",
    "k_embed_norm", "k_sample_partial", "k_sample_final", "k_decode_rows", "k_copy_logits", "k_qkv_rope",
    "k_topp_max", "k_topp_hist", "k_topp_pick", "k_gemm_bf16_lds<1,8,64,0,2>",
    ".gemm[q|k|v]", ".gemm[o]", ".gemm[gate|up]", ".gemm[down]", ".gemm[lm_head]"};

// prof_begin reserves an event pair for the next kernel launch; launch_k
// hands it to hipExtLaunchKernelGGL, which stamps the kernel's own start and
// end; prof_end files the launch under its class.
void prof_begin(sara_ctx* c) {
  if (c->prof_next_event + 2 > (int)c->prof_events.size()) return;
  c->prof_pending = c->prof_next_event;
  c->prof_next_event += 2;
}

void prof_end(sara_ctx* c, int cls, int N, int K) {
  if (c->prof_last >= 0) c->prof_recs.push_back({cls, N, K, c->prof_last, c->prof_last + 1});
  c->prof_last = -1;
  c->prof_pending = -1;
}

// Waits for the recorded events and adds elapsed time and algorithmic bytes
// and flops of each launch to its class.
int prof_collect(sara_ctx* c) {
  if (c->prof_recs.empty()) { c->prof_next_event = 0; return SARA_OK; }
  HIP_TRY(hipEventSynchronize(c->prof_events[c->prof_recs.back().e1]), "profile sync");
  int32_t M = 0;
  HIP_TRY(hipMemcpy(&M, c->rows_M, sizeof(int32_t), hipMemcpyDeviceToHost), "profile M");
  double sum_ctx = 0.0;
  if (M > 0) {
    std::vector<RowDesc> rows(M);
    HIP_TRY(hipMemcpy(rows.data(), c->rows, sizeof(RowDesc) * M, hipMemcpyDeviceToHost), "profile rows");
    for (auto& r : rows) sum_ctx += (double)r.pos + 1.0;
  }
  const double E = c->elt, m = M;
  for (auto& r : c->prof_recs) {
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, c->prof_events[r.e0], c->prof_events[r.e1]), "elapsed");
    double by = 0.0, fl = 0.0, N = r.N, K = r.K;
    switch (r.cls) {
      case kPGemmN1:
      case kPGemmO1:
        by = N * K * E + m * K * E + m * N * 4.0; fl = 2.0 * m * N * K; break;
      case kPGemmLM:   // bf16: sampling epilogue, one (score, id) per row and 128-id block
        by = N * K * E + m * K * E + (E == 2 ? m * ((N + 127) / 128) * 8.0 : m * N * 4.0);
        fl = 2.0 * m * N * K;
        break;
      case kPGemmGU:   // output is the bf16 SwiGLU product [m][N/2]
        by = N * K * E + m * K * E + m * (N / 2) * E; fl = 2.0 * m * N * K; break;
      case kPAttn:
        by = sum_ctx * c->hkv * c->hd * E * 2.0 + m * c->qdim * E;
        fl = 4.0 * sum_ctx * c->qdim;
        break;
      case kPCombine: by = m * c->qdim * (4.0 + E); break;
      case kPQkv: by = m * N * (4.0 + E); break;
      case kPQkvRope:   // fused q|k|v weights, normed input rows, q and the appended k, v
        by = N * K * E + m * K * E + m * N * E; fl = 2.0 * m * N * K; break;
      case kPResNorm: by = m * N * (12.0 + E); break;
      case kPSwiglu: by = m * N * (8.0 + E); break;
      case kPEmbed: by = m * N * (2.0 * E + 4.0); break;
      case kPSampleP: by = m * N * 4.0; break;
      case kPToppMax: by = m * N * 4.0; break;   // the row's fp32 logits, once
      case kPToppHist: by = m * N * 4.0 + m * (double)kTopPChunks * kTopPBins * 8.0; break;
      case kPToppSel: by = m * (double)kTopPChunks * kTopPBins * 8.0; break;   // the chunk histograms
      case kPCopy: by = m * N * 8.0; break;
      default: by = m * 64.0; break;
    }
    auto add = [&](int cls) {
      auto& t = c->prof_tot[cls];
      t.launches += 1;
      t.ms += ms;
      t.bytes += by;
      t.flops += fl;
    };
    add(r.cls);
    if (r.cls == kPGemmN1 || r.cls == kPGemmO1 || r.cls == kPGemmGU || r.cls == kPGemmLM || r.cls == kPQkvRope) {
      if (r.N == c->V) add(kPGemmLm);
      else if (r.N == c->nqkv) add(kPGemmQkv);
      else if (r.N == 2 * c->ffn) add(kPGemmGu);
      else if (r.K == c->ffn) add(kPGemmD);
      else add(kPGemmO);
    }
  }
  c->prof_recs.clear();
  c->prof_next_event = 0;
  return SARA_OK;
}

}  // namespace sara


static int dmalloc(void** p, size_t bytes, std::vector<void*>& owned) {
  if (bytes == 0) bytes = 16;
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    set_error("hipMalloc of " + std::to_string(bytes) + " bytes failed: " + hipGetErrorString(e));
    return SARA_ENOMEM;
  }
  owned.push_back(*p);
  return SARA_OK;
}

static double peff_host(int n, int s, int k, double a0, double b0) {
  if (s >= 1 && n - s >= 1) return 1.0;
  int r = k - n;
  if (r <= 0) return 0.0;
  double a = a0 + s, b = b0 + (n - s);
  double lb = lgamma(a) + lgamma(b) - lgamma(a + b);
  double psat = 0.0;
  if (s == 0) psat += exp(lgamma(a) + lgamma(b + r) - lgamma(a + b + r) - lb);
  if (s == n) psat += exp(lgamma(a + r) + lgamma(b) - lgamma(a + b + r) - lb);
  return 1.0 - psat;
}

static int validate(const sara_model_desc* m, const sara_alloc_desc* a) {
  if (!m || !a) return einval("null descriptor");
  if (m->dtype != SARA_F32 && m->dtype != SARA_BF16) return einval("dtype must be SARA_F32 or SARA_BF16");
  if (m->n_layers < 1 || m->d_model < 32 || m->vocab < 1 || m->d_ffn < 32)
    return einval("model dimensions must be positive (d_model, d_ffn >= 32)");
  if (m->head_dim != 64 && m->head_dim != 128) return einval("head_dim must be 64 or 128");
  if (m->n_kv_heads < 1 || m->n_heads % m->n_kv_heads != 0 ||
      m->n_heads / m->n_kv_heads > kMaxGroup)
    return einval("n_heads must be a multiple of n_kv_heads with at most 8 query heads per KV head");
  if (m->d_model % 64 || m->d_ffn % 64 || (m->n_heads * m->head_dim) % 64)
    return einval("d_model, d_ffn and n_heads*head_dim must be multiples of 64");
  if (m->dtype == SARA_BF16) {
    const int ks = m->d_model / 128;
    if (m->d_model % 128 || !(ks == 4 || ks == 8 || ks == 12 || ks == 16 || ks == 24 || ks == 32))
      return einval("bf16 models need d_model in {512, 1024, 1536, 2048, 3072, 4096}");
  }
  if (m->dtype == SARA_BF16 && m->d_ffn % 16) return einval("d_ffn must be a multiple of 16");
  if (m->vocab % 16) return einval("vocab must be a multiple of 16");
  if (m->eos_id < -1 || m->eos_id >= m->vocab) return einval("eos_id out of range");
  if (!(m->rms_eps > 0.f) || !(m->rope_theta > 0.f)) return einval("rms_eps and rope_theta must be > 0");
  if (a->k < 2 || a->k > 65535) return einval("k must be in [2, 65535]");
  if (a->n0 < 1 || a->n0 > a->k) return einval("n0 must be in [1, k]");
  if (a->commit_min < 2 || a->commit_min > a->k) return einval("commit_min must be in [2, k]");
  if (!(a->tau_low >= 0.0 && a->tau_low <= 1.0)) return einval("tau_low must be in [0, 1]");
  if (!(a->alpha0 > 0.0) || !(a->beta0 > 0.0)) return einval("alpha0 and beta0 must be > 0");
  if (a->B < 0 || a->budget_N < 0) return einval("B and budget_N must be >= 0");
  if (a->pool_U < 1 || a->pool_U >= (1 << 26)) return einval("pool_U must be in [1, 2^26)");
  if ((int64_t)a->pool_U * a->k >= (1ll << 31)) return einval("pool_U * k must be < 2^31");
  if (a->n_slots < 1 || a->n_slots > kMaxSlots) return einval("n_slots must be in [1, 4096]");
  if (a->kv_block != kBlockTok) return einval("kv_block must be 16");
  if (a->max_prompt < 1 || a->max_new < 1) return einval("max_prompt and max_new must be >= 1");
  if (a->mode != SARA_MODE_SARA && a->mode != SARA_MODE_FIXED_K && a->mode != SARA_MODE_SARA_THOMPSON)
    return einval("unknown mode");
  if (!(a->temperature > 0.f)) return einval("temperature must be > 0");
  if (!(a->top_p > 0.f && a->top_p <= 1.f)) return einval("top_p must be in (0, 1]");
  if (a->prio_quant_bits < 1 || a->prio_quant_bits > 21) return einval("prio_quant_bits must be in [1, 21]");
  int64_t qcap = std::min<int64_t>(a->budget_N, (int64_t)a->pool_U * a->k);
  if (qcap > kMaxQueue) return einval("min(budget_N, pool_U*k) must be <= 4096");
  return SARA_OK;
}

extern "C" const char* sara_last_error(void) { return g_err.c_str(); }

extern "C" int sara_init(const sara_model_desc* md, const sara_alloc_desc* ad,
                         const void* const* d_weights, int32_t n_weights, void* stream,
                         sara_ctx** out) {
  if (!out) return einval("out is null");
  *out = nullptr;
  int rc = validate(md, ad);
  if (rc) return rc;
  if (n_weights != 3 + 9 * md->n_layers) return einval("n_weights must be 3 + 9 * n_layers");
  if (!d_weights) return einval("d_weights is null");
  for (int i = 0; i < n_weights; ++i)
    if (!d_weights[i]) return einval("weight pointer " + std::to_string(i) + " is null");

  sara_ctx* c = new sara_ctx();
  auto& own = c->owned;
  c->md = *md;
  c->ad = *ad;
  c->stream = (hipStream_t)stream;
  {
    const hipError_t e = hipGetDevice(&c->device);
    if (e != hipSuccess) { delete c; return hip_fail(e, "hipGetDevice"); }
  }
  c->L = md->n_layers; c->d = md->d_model; c->hq = md->n_heads; c->hkv = md->n_kv_heads;
  c->hd = md->head_dim; c->ffn = md->d_ffn; c->V = md->vocab; c->G = c->hq / c->hkv;
  c->qdim = c->hq * c->hd; c->nqkv = (c->hq + 2 * c->hkv) * c->hd;
  c->U = ad->pool_U; c->k = ad->k; c->S = ad->n_slots;
  c->PB = std::max(1, (ad->max_prompt - 1 + kBlockTok - 1) / kBlockTok);
  c->SB = (ad->max_new + kBlockTok - 1) / kBlockTok;
  c->MAXB = c->PB + c->SB;
  c->n_blocks = (int64_t)c->U * c->PB + (int64_t)c->S * c->SB;
  c->max_pos = ad->max_prompt + ad->max_new;
  c->Qcap = (int)std::min<int64_t>(ad->budget_N, (int64_t)c->U * c->k);
  c->elt = (md->dtype == SARA_BF16) ? 2 : 4;
  c->prefill_rows = 4096;
  c->row_cap = std::max(c->S, c->prefill_rows);
  c->attn_splits_max = std::max((c->max_pos + kAttnSplit - 1) / kAttnSplit,
                                (c->MAXB + kAttnChunks - 1) / kAttnChunks);
  c->dec_splits_max = (c->MAXB + kDecPages - 1) / kDecPages;
  {
    // split-K partials of the VALU / MFMA GEMMs that write fp32 (the GEMM
    // falls back to one split when its partials would not fit)
    if (md->dtype == SARA_BF16) {
      // decode: the o and down projections (<= kMaxSplitsDec splits of
      // [S][d]); prefill: q|k|v, o and down over a chunk, whose weight tiles
      // and m-blocks fill the GPU without splits except in a short last
      // chunk (<= 256 blocks' worth of partials).  The LM head, the gate|up
      // projection and the q|k|v projection of decode write no partials.
      const int64_t npf = std::max<int64_t>(c->nqkv, c->d);
      c->ws_floats = std::max<int64_t>((int64_t)kMaxSplitsDec * c->S * c->d, 2 * (int64_t)c->prefill_rows * npf);
    } else {
      // fp32: also the logits [S][V] and the gate|up output [rows][2 ffn]
      int64_t nd = std::max<int64_t>({c->V, c->nqkv, 2 * (int64_t)c->ffn, c->d});
      int64_t np = std::max<int64_t>({c->nqkv, 2 * (int64_t)c->ffn, c->d});
      c->ws_floats = std::max<int64_t>((int64_t)c->S * nd, (int64_t)c->prefill_rows * np);
    }
  }
  const size_t E = (size_t)c->elt;
  const size_t d = c->d;
#define ALLOC(ptr, bytes)                                   \
  do {                                                      \
    int r_ = dmalloc((void**)&(ptr), (size_t)(bytes), own); \
    if (r_) { sara_destroy(c); return r_; }                 \
  } while (0)
  // weights, repacked: q|k|v rows fused, gate|up rows fused (bf16: tiled, see launch_tile_weights)
  ALLOC(c->embed, (size_t)c->V * d * E);
  ALLOC(c->lm_head, (size_t)c->V * d * E);
  c->w_qkv.resize(c->L); c->w_o.resize(c->L); c->w_gu.resize(c->L); c->w_d.resize(c->L);
  for (int l = 0; l < c->L; ++l) {
    ALLOC(c->w_qkv[l], (size_t)c->nqkv * d * E);
    ALLOC(c->w_o[l], (size_t)d * c->qdim * E);
    ALLOC(c->w_gu[l], (size_t)2 * c->ffn * d * E);
    ALLOC(c->w_d[l], (size_t)d * c->ffn * E);
  }
  ALLOC(c->norms, sizeof(float) * (2 * c->L + 1) * d);
  // KV cache and tables
  size_t kv_bytes = (size_t)c->L * c->n_blocks * c->hkv * kBlockTok * c->hd * E;
  ALLOC(c->kc, kv_bytes);
  ALLOC(c->vc, kv_bytes);
  ALLOC(c->btab, sizeof(int32_t) * (size_t)(c->S + c->U) * c->MAXB);
  ALLOC(c->rope, sizeof(float2) * (size_t)c->max_pos * (c->hd / 2));
  ALLOC(c->row_rope, sizeof(float2) * (size_t)c->S * (c->hd / 2));
  ALLOC(c->prior_a, sizeof(double) * (size_t)c->U);
  ALLOC(c->prior_b, sizeof(double) * (size_t)c->U);
  ALLOC(c->prior_p, sizeof(double) * (size_t)c->U);
  ALLOC(c->attn_items, sizeof(AttnItem) * (size_t)c->S * c->dec_splits_max);
  ALLOC(c->attn_nitems, sizeof(int32_t) * 4);
  // prompt pool
  c->tok_cap = (int64_t)c->U * ad->max_prompt;
  ALLOC(c->tok, sizeof(int32_t) * c->tok_cap);
  ALLOC(c->off, sizeof(int32_t) * (c->U + 1));
  ALLOC(c->pre, sizeof(int32_t) * (c->U + 1));
  ALLOC(c->p, sizeof(double) * c->U);
  ALLOC(c->flen, sizeof(int32_t) * (size_t)c->U * c->k);
  // controller
  ALLOC(c->ctl, sizeof(Ctl));
  ALLOC(c->cp_dev, sizeof(CtlParams));
  ALLOC(c->status, sizeof(int32_t) * c->U);
  ALLOC(c->n_iss, sizeof(int32_t) * c->U);
  ALLOC(c->n_done, sizeof(int32_t) * c->U);
  ALLOC(c->succ, sizeof(int32_t) * c->U);
  ALLOC(c->infl, sizeof(int32_t) * c->U);
  ALLOC(c->peff, sizeof(double) * c->U);
  ALLOC(c->slot_uid, sizeof(int32_t) * c->S);
  ALLOC(c->slot_j, sizeof(int32_t) * c->S);
  ALLOC(c->slot_gen, sizeof(int32_t) * c->S);
  ALLOC(c->fin, sizeof(int32_t) * c->S);
  ALLOC(c->slot_hash, sizeof(uint64_t) * c->S);
  ALLOC(c->active, sizeof(int32_t) * c->S);
  ALLOC(c->queue, sizeof(uint64_t) * std::max(1, c->Qcap));
  const size_t nroll = (size_t)c->U * c->k;
  ALLOC(c->out_tok, sizeof(int32_t) * nroll * ad->max_new);
  ALLOC(c->samp_tok, sizeof(int32_t) * nroll * ad->max_new);
  ALLOC(c->r_len, sizeof(int32_t) * nroll);
  ALLOC(c->r_reward, sizeof(int32_t) * nroll);
  c->cap_dec = (int64_t)nroll; c->cap_draw = c->U; c->cap_asg = (int64_t)nroll; c->cap_fin = (int64_t)nroll;
  ALLOC(c->log_dec, sizeof(int64_t) * 6 * c->cap_dec);
  ALLOC(c->log_draw, sizeof(int64_t) * 2 * c->cap_draw);
  ALLOC(c->log_asg, sizeof(int64_t) * 4 * c->cap_asg);
  ALLOC(c->log_fin, sizeof(int64_t) * 6 * c->cap_fin);
  // activations
  ALLOC(c->rows, sizeof(RowDesc) * c->row_cap);
  ALLOC(c->rows_M, sizeof(int32_t));
  ALLOC(c->h, sizeof(float) * (size_t)c->row_cap * d);
  ALLOC(c->x, (size_t)c->row_cap * std::max({c->d, c->ffn, c->qdim}) * E);
  ALLOC(c->qbuf, (size_t)c->row_cap * c->qdim * E);
  ALLOC(c->xa, (size_t)c->row_cap * c->ffn * E);
  ALLOC(c->ws, sizeof(float) * (size_t)c->ws_floats);
  ALLOC(c->attn_part, sizeof(float) *
                          (size_t)std::max((int64_t)c->row_cap * c->attn_splits_max,
                                           (int64_t)c->S * c->dec_splits_max) *
                          c->hkv * kMaxGroup * (c->hd + 2));
  // per (row, vocabulary chunk) winners: kSampleChunks chunks (fp32 models),
  // one per 128-id block of the fused LM-head sampler (bf16 models)
  const size_t nchunk = std::max<size_t>(kSampleChunks, (size_t)(c->V + 127) / 128);
  ALLOC(c->samp_best, sizeof(float) * (size_t)c->S * nchunk);
  ALLOC(c->samp_idx, sizeof(int32_t) * (size_t)c->S * nchunk);
  c->topp = c->ad.top_p < 1.0f;
  // nucleus sampling reads fp32 logits; the bf16 LM head writes them here
  if (c->topp && c->md.dtype == SARA_BF16) ALLOC(c->topp_logits, sizeof(float) * (size_t)c->S * c->V);
  if (c->topp) {
    ALLOC(c->topp_max, sizeof(float) * (size_t)c->S * kTopPChunks);
    ALLOC(c->topp_hist, sizeof(unsigned long long) * (size_t)c->S * kTopPChunks * kTopPBins);
    ALLOC(c->topp_thr, sizeof(uint32_t) * (size_t)c->S);
    ALLOC(c->topp_above, sizeof(unsigned long long) * (size_t)c->S);
    ALLOC(c->topp_target, sizeof(unsigned long long) * (size_t)c->S);
  }
  ALLOC(c->g_off, sizeof(int32_t) * (c->U + 1));
  ALLOC(c->g_r, sizeof(float) * nroll);
  ALLOC(c->g_adv, sizeof(float) * nroll);
  ALLOC(c->g_n, sizeof(int32_t));
#undef ALLOC
  {
    hipError_t e = hipHostMalloc((void**)&c->h_done, 2 * sizeof(int32_t), hipHostMallocDefault);
    if (e != hipSuccess) { sara_destroy(c); return hip_fail(e, "hipHostMalloc"); }
    c->h_done[0] = c->h_done[1] = 0;
  }

  hipStream_t st = c->stream;
  // weights
  auto cp = [&](void* dst, const void* src, size_t bytes) {
    return hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, st);
  };
  const size_t qb = (size_t)c->qdim * d * E, kvb = (size_t)c->hkv * c->hd * d * E;
  const size_t fb = (size_t)c->ffn * d * E;
  hipError_t e = cp(c->embed, d_weights[0], (size_t)c->V * d * E);
  if (md->dtype == SARA_BF16) {
    // GEMM weights in the k-block-major fragment layout of the bf16 GEMM (wtiled_index)
    const int kvr = c->hkv * c->hd;
    for (int l = 0; l < c->L && e == hipSuccess; ++l) {
      const void* const* w = d_weights + 1 + 9 * l;
      // q|k|v rows fused, each head in rotation-pair order (see qkv_pair_col)
      launch_tile_weights_pairs(c, w[1], c->w_qkv[l], c->qdim, d, 0);
      launch_tile_weights_pairs(c, w[2], c->w_qkv[l], kvr, d, c->hq);
      launch_tile_weights_pairs(c, w[3], c->w_qkv[l], kvr, d, c->hq + c->hkv);
      launch_tile_weights(c, w[4], c->w_o[l], d, c->qdim, 1, 0, d);
      // gate and up tiles interleaved (gate tile j -> 2j, up tile j -> 2j + 1) for the SwiGLU epilogue
      launch_tile_weights(c, w[6], c->w_gu[l], c->ffn, d, 2, 0, 2 * c->ffn);
      launch_tile_weights(c, w[7], c->w_gu[l], c->ffn, d, 2, 1, 2 * c->ffn);
      launch_tile_weights(c, w[8], c->w_d[l], d, c->ffn, 1, 0, d);
      e = hipGetLastError();
    }
    launch_tile_weights(c, d_weights[2 + 9 * c->L], c->lm_head, c->V, d, 1, 0, c->V);
    if (e == hipSuccess) e = hipGetLastError();
  } else {
    for (int l = 0; l < c->L && e == hipSuccess; ++l) {
      const void* const* w = d_weights + 1 + 9 * l;
      char* qkv = (char*)c->w_qkv[l];
      e = cp(qkv, w[1], qb);
      if (e == hipSuccess) e = cp(qkv + qb, w[2], kvb);
      if (e == hipSuccess) e = cp(qkv + qb + kvb, w[3], kvb);
      if (e == hipSuccess) e = cp(c->w_o[l], w[4], (size_t)d * c->qdim * E);
      char* gu = (char*)c->w_gu[l];
      if (e == hipSuccess) e = cp(gu, w[6], fb);
      if (e == hipSuccess) e = cp(gu + fb, w[7], fb);
      if (e == hipSuccess) e = cp(c->w_d[l], w[8], (size_t)d * c->ffn * E);
    }
    if (e == hipSuccess) e = cp(c->lm_head, d_weights[2 + 9 * c->L], (size_t)c->V * d * E);
  }
  if (e != hipSuccess) { sara_destroy(c); return hip_fail(e, "weight copy"); }
  rc = launch_convert_norms(c, d_weights);
  if (rc) { sara_destroy(c); return rc; }
  // RoPE table in fp64, stored fp32
  {
    const int half = c->hd / 2;
    std::vector<float2> tab((size_t)c->max_pos * half);
    for (int pidx = 0; pidx < c->max_pos; ++pidx)
      for (int i = 0; i < half; ++i) {
        double inv = pow((double)md->rope_theta, -(2.0 * i) / (double)c->hd);
        double ang = (double)pidx * inv;
        tab[(size_t)pidx * half + i] = make_float2((float)cos(ang), (float)sin(ang));
      }
    e = hipMemcpyAsync(c->rope, tab.data(), sizeof(float2) * tab.size(), hipMemcpyHostToDevice, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) { sara_destroy(c); return hip_fail(e, "rope upload"); }
  }
  // controller parameters
  CtlParams& p = c->cp;
  memset(&p, 0, sizeof(p));
  p.B = ad->B; p.k = ad->k; p.n0 = ad->n0; p.commit_min = ad->commit_min; p.U = c->U; p.S = c->S;
  p.mode = ad->mode; p.bits = ad->prio_quant_bits; p.max_new = ad->max_new; p.PB = c->PB;
  p.SB = c->SB; p.MAXB = c->MAXB; p.eos = md->eos_id; p.Qcap = c->Qcap;
  p.tau = ad->tau_low; p.a0 = ad->alpha0; p.b0 = ad->beta0;
  p.prior = peff_host(0, 0, ad->k, ad->alpha0, ad->beta0);
  p.seed = ad->seed; p.step = 0; p.forced_eos = ad->forced_eos_u32; p.temperature = ad->temperature;
  p.top_p = ad->top_p;
  p.has_flen = 0;
  e = hipMemcpyAsync(c->cp_dev, &p, sizeof(p), hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) { sara_destroy(c); return hip_fail(e, "init"); }
  *out = c;
  return SARA_OK;
}

extern "C" int sara_begin_step(sara_ctx* c, const int32_t* d_tokens, const int32_t* h_offsets,
                               const double* d_p, const int32_t* d_forced_len, int32_t step_index) {
  if (!c) return einval("null context");
  if (!d_tokens || !h_offsets || !d_p) return einval("d_tokens, h_offsets and d_p are required");
  const int U = c->U;
  if (h_offsets[0] != 0) return einval("h_offsets[0] must be 0");
  for (int u = 0; u < U; ++u) {
    int L = h_offsets[u + 1] - h_offsets[u];
    if (L < 1 || L > c->ad.max_prompt)
      return einval("prompt " + std::to_string(u) + " has length " + std::to_string(L) +
                    " outside [1, max_prompt]");
  }
  hipStream_t st = c->stream;
  c->h_off.assign(h_offsets, h_offsets + U + 1);
  static thread_local std::vector<int32_t> pre;
  pre.assign(U + 1, 0);
  for (int u = 0; u < U; ++u) pre[u + 1] = pre[u] + (c->h_off[u + 1] - c->h_off[u] - 1);
  HIP_TRY(hipMemcpyAsync(c->tok, d_tokens, sizeof(int32_t) * c->h_off[U], hipMemcpyDeviceToDevice, st),
          "copy tokens");
  HIP_TRY(hipMemcpyAsync(c->off, c->h_off.data(), sizeof(int32_t) * (U + 1), hipMemcpyHostToDevice, st),
          "copy offsets");
  HIP_TRY(hipMemcpyAsync(c->pre, pre.data(), sizeof(int32_t) * (U + 1), hipMemcpyHostToDevice, st),
          "copy prefix");
  HIP_TRY(hipMemcpyAsync(c->p, d_p, sizeof(double) * U, hipMemcpyDeviceToDevice, st), "copy p");
  c->has_flen = d_forced_len ? 1 : 0;
  if (d_forced_len)
    HIP_TRY(hipMemcpyAsync(c->flen, d_forced_len, sizeof(int32_t) * U * c->k, hipMemcpyDeviceToDevice, st),
            "copy forced lengths");
  c->step_index = step_index;
  c->cp.step = step_index;
  c->cp.has_flen = c->has_flen;
  c->cp.has_prior = c->warm_ids ? 1 : 0;
  HIP_TRY(hipMemcpyAsync(c->cp_dev, &c->cp, sizeof(CtlParams), hipMemcpyHostToDevice, st), "params");
  // the host copies above come from pageable memory owned by the context;
  // make sure they have landed before the next step can rewrite them
  HIP_TRY(hipStreamSynchronize(st), "begin_step sync");
  launch_reset(c);
  if (c->warm_ids) launch_warm_priors(c);
  launch_prefill(c);
  launch_refill(c);
  HIP_TRY(hipGetLastError(), "begin_step launch");
  c->in_step = true;
  c->warm_step = c->warm_ids != nullptr;
  return SARA_OK;
}

extern "C" int sara_set_warm_start(sara_ctx* c, const int32_t* d_ids, double* d_a, double* d_b,
                                   int32_t n_store) {
  if (!c) return einval("null context");
  if (d_ids && (!d_a || !d_b)) return einval("warm start needs d_a and d_b");
  if (d_ids && n_store < 1) return einval("n_store must be >= 1");
  c->warm_ids = d_ids;
  c->warm_a = d_ids ? d_a : nullptr;
  c->warm_b = d_ids ? d_b : nullptr;
  c->warm_n = d_ids ? n_store : 0;
  return SARA_OK;
}

extern "C" int sara_warm_start_update(sara_ctx* c, double lambda) {
  if (!c) return einval("null context");
  if (!(lambda >= 0.0 && lambda <= 1.0)) return einval("lambda must be in [0, 1]");
  if (!c->warm_ids || !c->warm_step) {
    set_error("sara_warm_start_update needs a step begun with warm start set");
    return SARA_ESTATE;
  }
  launch_warm_update(c, lambda);
  HIP_TRY(hipGetLastError(), "warm start update launch");
  return SARA_OK;
}

extern "C" int sara_decode_step(sara_ctx* c, const int32_t* d_forced_tok, float* d_logits,
                                int32_t model_free) {
  if (!c) return einval("null context");
  if (!c->in_step) { set_error("sara_decode_step before sara_begin_step"); return SARA_ESTATE; }
  if (model_free && !d_forced_tok) return einval("model_free needs a forced-token table");
  c->prof_active = c->prof_enabled && !c->capturing;
  launch_decode(c, d_forced_tok, d_logits, model_free);
  HIP_TRY(hipGetLastError(), "decode launch");
  if (c->prof_active) {
    c->prof_active = false;
    int rc = prof_collect(c);
    if (rc) return rc;
  }
  return SARA_OK;
}

extern "C" int sara_reset_profile(sara_ctx* c) {
  if (!c) return einval("null context");
  c->prof_recs.clear();
  c->prof_next_event = 0;
  c->prof_tot.assign(kPNumClasses, sara_kernel_profile{});
  for (int i = 0; i < kPNumClasses; ++i)
    strncpy(c->prof_tot[i].name, kProfNames[i], sizeof(c->prof_tot[i].name) - 1);
  return SARA_OK;
}

extern "C" int sara_set_profiling(sara_ctx* c, int32_t enable) {
  if (!c) return einval("null context");
  c->prof_enabled = enable != 0;
  if (c->prof_tot.empty()) sara_reset_profile(c);
  if (c->prof_enabled && c->prof_events.empty()) {
    size_t n = 64 + 24 * (size_t)c->L;
    c->prof_events.resize(n);
    for (size_t i = 0; i < n; ++i) HIP_TRY(hipEventCreate(&c->prof_events[i]), "hipEventCreate");
  }
  return SARA_OK;
}

extern "C" int sara_read_profile(sara_ctx* c, sara_kernel_profile* out, int32_t cap, int32_t* n_out) {
  if (!c || (cap > 0 && !out)) return einval("null argument");
  int n = (int)c->prof_tot.size();
  for (int i = 0; i < n && i < cap; ++i) out[i] = c->prof_tot[i];
  if (n_out) *n_out = n;
  return SARA_OK;
}

extern "C" int sara_posterior_decide(sara_ctx* c) {
  if (!c) return einval("null context");
  if (!c->in_step) { set_error("sara_posterior_decide before sara_begin_step"); return SARA_ESTATE; }
  launch_decide(c);
  HIP_TRY(hipGetLastError(), "decide launch");
  return SARA_OK;
}

extern "C" int sara_refill(sara_ctx* c) {
  if (!c) return einval("null context");
  if (!c->in_step) { set_error("sara_refill before sara_begin_step"); return SARA_ESTATE; }
  launch_refill(c);
  HIP_TRY(hipGetLastError(), "refill launch");
  return SARA_OK;
}

static int build_graph(sara_ctx* c, const int32_t* forced, int iters) {
  if (c->graph_exec) { (void)hipGraphExecDestroy(c->graph_exec); c->graph_exec = nullptr; }
  if (c->graph) { (void)hipGraphDestroy(c->graph); c->graph = nullptr; }
  HIP_TRY(hipStreamBeginCapture(c->stream, hipStreamCaptureModeThreadLocal), "begin capture");
  c->capturing = true;
  c->prof_active = false;
  for (int i = 0; i < iters; ++i) {
    launch_decode(c, forced, nullptr, 0);
    launch_decide(c);
    launch_refill(c);
  }
  c->capturing = false;
  HIP_TRY(hipStreamEndCapture(c->stream, &c->graph), "end capture");
  HIP_TRY(hipGraphInstantiate(&c->graph_exec, c->graph, nullptr, nullptr, 0), "graph instantiate");
  c->graph_iters = iters;
  c->graph_forced = forced;
  return SARA_OK;
}

extern "C" int sara_run(sara_ctx* c, const int32_t* d_forced_tok, int32_t graph_iters,
                        int64_t max_iters, int64_t* iters_out) {
  if (!c) return einval("null context");
  if (!c->in_step) { set_error("sara_run before sara_begin_step"); return SARA_ESTATE; }
  if (graph_iters < 1 || graph_iters > 4096) return einval("graph_iters must be in [1, 4096]");
  if (!c->graph_exec || c->graph_iters != graph_iters || c->graph_forced != d_forced_tok) {
    int rc = build_graph(c, d_forced_tok, graph_iters);
    if (rc) return rc;
  }
  hipEvent_t ev[2];
  HIP_TRY(hipEventCreateWithFlags(&ev[0], hipEventDisableTiming), "event");
  HIP_TRY(hipEventCreateWithFlags(&ev[1], hipEventDisableTiming), "event");
  c->h_done[0] = c->h_done[1] = 0;
  int64_t iters = 0;
  int n = 0;
  int rc = SARA_OK;
  while (iters < max_iters) {
    hipError_t e = hipGraphLaunch(c->graph_exec, c->stream);
    if (e != hipSuccess) { rc = hip_fail(e, "graph launch"); break; }
    iters += graph_iters;
    int slot = n & 1;
    e = hipMemcpyAsync(&c->h_done[slot], &c->ctl->done, sizeof(int32_t), hipMemcpyDeviceToHost, c->stream);
    if (e == hipSuccess) e = hipEventRecord(ev[slot], c->stream);
    if (e != hipSuccess) { rc = hip_fail(e, "poll"); break; }
    if (n > 0) {
      int prev = (n - 1) & 1;
      e = hipEventSynchronize(ev[prev]);
      if (e != hipSuccess) { rc = hip_fail(e, "poll wait"); break; }
      if (((volatile int32_t*)c->h_done)[prev]) break;
    }
    ++n;
  }
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess && rc == SARA_OK) rc = hip_fail(e, "run sync");
  (void)hipEventDestroy(ev[0]);
  (void)hipEventDestroy(ev[1]);
  if (iters_out) *iters_out = iters;
  return rc;
}

extern "C" int sara_query(sara_ctx* c, sara_step_stats* out) {
  if (!c || !out) return einval("null argument");
  HIP_TRY(hipStreamSynchronize(c->stream), "query sync");
  Ctl h;
  HIP_TRY(hipMemcpy(&h, c->ctl, sizeof(Ctl), hipMemcpyDeviceToHost), "query copy");
  memset(out, 0, sizeof(*out));
  out->done = h.done;
  out->error = h.error;
  out->decode_steps = h.t < 0 ? 0 : h.t;
  out->drawn = h.next_uid;
  out->committed = h.nC;
  out->abandoned = h.nAb;
  out->active = h.nA;
  out->queued = h.qlen;
  out->running = h.running;
  out->budget_left = h.budget_left;
  out->rollouts = h.rollouts;
  out->tokens = h.tokens;
  out->n_decisions = h.n_dec;
  out->n_draws = h.n_draw;
  out->n_assigns = h.n_asg;
  out->n_finishes = h.n_fin;
  if (h.error) { set_error("device error word " + std::to_string(h.error)); return SARA_EDEVICE; }
  return SARA_OK;
}

extern "C" int sara_finish_step(sara_ctx* c, float eps) {
  if (!c) return einval("null context");
  if (!c->in_step) { set_error("sara_finish_step before sara_begin_step"); return SARA_ESTATE; }
  if (!(eps >= 0.f)) return einval("eps must be >= 0");
  launch_finish(c, eps);
  HIP_TRY(hipGetLastError(), "finish launch");
  return SARA_OK;
}

extern "C" int sara_read_rollouts(sara_ctx* c, int32_t* h_tokens, int32_t* h_sampled, int32_t* h_len,
                                  int32_t* h_reward, int32_t* h_status, int32_t* h_n, int32_t* h_s,
                                  double* h_peff) {
  if (!c) return einval("null context");
  HIP_TRY(hipStreamSynchronize(c->stream), "read sync");
  const size_t nroll = (size_t)c->U * c->k, mn = (size_t)c->ad.max_new;
  std::vector<int32_t> len(nroll);
  HIP_TRY(hipMemcpy(len.data(), c->r_len, sizeof(int32_t) * nroll, hipMemcpyDeviceToHost), "len");
  if (h_len) memcpy(h_len, len.data(), sizeof(int32_t) * nroll);
  if (h_tokens) {
    HIP_TRY(hipMemcpy(h_tokens, c->out_tok, sizeof(int32_t) * nroll * mn, hipMemcpyDeviceToHost), "tok");
    for (size_t r = 0; r < nroll; ++r)
      for (size_t i = (size_t)len[r]; i < mn; ++i) h_tokens[r * mn + i] = -1;
  }
  if (h_sampled) {
    HIP_TRY(hipMemcpy(h_sampled, c->samp_tok, sizeof(int32_t) * nroll * mn, hipMemcpyDeviceToHost), "samp");
    for (size_t r = 0; r < nroll; ++r)
      for (size_t i = (size_t)len[r]; i < mn; ++i) h_sampled[r * mn + i] = -1;
  }
  if (h_reward) HIP_TRY(hipMemcpy(h_reward, c->r_reward, sizeof(int32_t) * nroll, hipMemcpyDeviceToHost), "rew");
  if (h_status) HIP_TRY(hipMemcpy(h_status, c->status, sizeof(int32_t) * c->U, hipMemcpyDeviceToHost), "st");
  if (h_n) HIP_TRY(hipMemcpy(h_n, c->n_done, sizeof(int32_t) * c->U, hipMemcpyDeviceToHost), "n");
  if (h_s) HIP_TRY(hipMemcpy(h_s, c->succ, sizeof(int32_t) * c->U, hipMemcpyDeviceToHost), "s");
  if (h_peff) HIP_TRY(hipMemcpy(h_peff, c->peff, sizeof(double) * c->U, hipMemcpyDeviceToHost), "peff");
  return SARA_OK;
}

extern "C" int sara_read_logs(sara_ctx* c, int64_t* h_dec, int64_t cap_dec, int64_t* h_draw,
                              int64_t cap_draw, int64_t* h_asg, int64_t cap_asg, int64_t* h_fin,
                              int64_t cap_fin) {
  if (!c) return einval("null context");
  HIP_TRY(hipStreamSynchronize(c->stream), "logs sync");
  Ctl h;
  HIP_TRY(hipMemcpy(&h, c->ctl, sizeof(Ctl), hipMemcpyDeviceToHost), "logs ctl");
  auto get = [&](int64_t* dst, int64_t cap, const int64_t* src, int64_t n, int w) -> int {
    if (!dst) return SARA_OK;
    int64_t m = std::min(cap, n);
    if (m > 0) {
      hipError_t e = hipMemcpy(dst, src, sizeof(int64_t) * w * m, hipMemcpyDeviceToHost);
      if (e != hipSuccess) return hip_fail(e, "log copy");
    }
    return SARA_OK;
  };
  int rc = get(h_dec, cap_dec, c->log_dec, h.n_dec, 6);
  if (!rc) rc = get(h_draw, cap_draw, c->log_draw, h.n_draw, 2);
  if (!rc) rc = get(h_asg, cap_asg, c->log_asg, h.n_asg, 4);
  if (!rc) rc = get(h_fin, cap_fin, c->log_fin, h.n_fin, 6);
  return rc;
}

extern "C" int sara_read_advantages(sara_ctx* c, int32_t* h_offsets, float* h_rewards, float* h_adv,
                                    int32_t cap) {
  if (!c) return einval("null context");
  HIP_TRY(hipStreamSynchronize(c->stream), "adv sync");
  int32_t n = 0;
  HIP_TRY(hipMemcpy(&n, c->g_n, sizeof(int32_t), hipMemcpyDeviceToHost), "adv n");
  std::vector<int32_t> off(n + 1);
  HIP_TRY(hipMemcpy(off.data(), c->g_off, sizeof(int32_t) * (n + 1), hipMemcpyDeviceToHost), "adv off");
  if (h_offsets) memcpy(h_offsets, off.data(), sizeof(int32_t) * (n + 1));
  int32_t m = std::min(cap, off[n]);
  if (m > 0 && h_rewards) HIP_TRY(hipMemcpy(h_rewards, c->g_r, sizeof(float) * m, hipMemcpyDeviceToHost), "r");
  if (m > 0 && h_adv) HIP_TRY(hipMemcpy(h_adv, c->g_adv, sizeof(float) * m, hipMemcpyDeviceToHost), "a");
  return SARA_OK;
}

extern "C" int sara_peff_batch(const double* d_alpha, const double* d_beta, const int32_t* d_n,
                               const int32_t* d_s, int32_t k, int32_t count, double* d_out, void* stream) {
  if (count < 0) return einval("count must be >= 0");
  if (count > 0 && (!d_alpha || !d_beta || !d_n || !d_s || !d_out)) return einval("null array");
  if (k < 1) return einval("k must be >= 1");
  launch_peff(d_alpha, d_beta, d_n, d_s, k, count, d_out, (hipStream_t)stream);
  HIP_TRY(hipGetLastError(), "peff launch");
  return SARA_OK;
}

extern "C" int sara_poll(sara_ctx* c, int32_t* h_pinned) {
  if (!c || !h_pinned) return einval("null argument");
  if (!c->in_step) { set_error("sara_poll before sara_begin_step"); return SARA_ESTATE; }
  void* d = nullptr;
  if (hipHostGetDevicePointer(&d, h_pinned, 0) != hipSuccess || !d) {
    (void)hipGetLastError();
    return einval("h_pinned is not pinned host memory");
  }
  launch_poll(c, (int32_t*)d);
  HIP_TRY(hipGetLastError(), "poll launch");
  return SARA_OK;
}

extern "C" int grpo_group_advantages(const float* d_r, const int32_t* d_group_off, int32_t n_groups,
                                     float eps, float* d_adv, void* stream) {
  if (n_groups < 0) return einval("n_groups must be >= 0");
  if (n_groups > 0 && (!d_r || !d_group_off || !d_adv)) return einval("null array");
  if (!(eps >= 0.f)) return einval("eps must be >= 0");
  launch_grpo(d_r, d_group_off, n_groups, eps, d_adv, (hipStream_t)stream);
  HIP_TRY(hipGetLastError(), "grpo launch");
  return SARA_OK;
}

extern "C" int sara_sample_logits(const float* d_logits, int32_t n_rows, int32_t vocab,
                                  const int32_t* d_rid, const int32_t* d_pos, uint64_t seed,
                                  int32_t step_index, float temperature, float top_p, int32_t eos_id,
                                  uint32_t forced_eos_u32, int32_t* d_tok, void* stream) {
  if (n_rows < 0 || vocab < 1) return einval("n_rows must be >= 0 and vocab >= 1");
  if (n_rows == 0) return SARA_OK;
  if (!d_logits || !d_rid || !d_pos || !d_tok) return einval("null array");
  if (!(temperature > 0.f)) return einval("temperature must be > 0");
  if (!(top_p > 0.f && top_p <= 1.f)) return einval("top_p must be in (0, 1]");
  if (eos_id >= vocab) return einval("eos_id out of range");
  return launch_sample_rows(d_logits, n_rows, vocab, d_rid, d_pos, seed, step_index, temperature, top_p, eos_id,
                            forced_eos_u32, d_tok, (hipStream_t)stream);
}

extern "C" int sara_sample_logits_noalloc(const float* d_logits, int32_t n_rows, int32_t vocab,
                                          const int32_t* d_rid, const int32_t* d_pos, uint64_t seed,
                                          int32_t step_index, float temperature, float top_p, int32_t eos_id,
                                          uint32_t forced_eos_u32, int32_t* d_tok, void* stream) {
  if (n_rows < 0 || vocab < 1) return einval("n_rows must be >= 0 and vocab >= 1");
  if (n_rows == 0) return SARA_OK;
  if (!d_logits || !d_rid || !d_pos || !d_tok) return einval("null array");
  if (!(temperature > 0.f)) return einval("temperature must be > 0");
  if (!(top_p > 0.f && top_p <= 1.f)) return einval("top_p must be in (0, 1]");
  if (eos_id >= vocab) return einval("eos_id out of range");
  if (n_rows > SARA_NOALLOC_MAX_ROWS)
    return einval("n_rows exceeds SARA_NOALLOC_MAX_ROWS (" + std::to_string(SARA_NOALLOC_MAX_ROWS) + ")");
  if (top_p < 1.f && n_rows > SARA_NOALLOC_MAX_TOPP_ROWS)
    return einval("n_rows exceeds SARA_NOALLOC_MAX_TOPP_ROWS (" + std::to_string(SARA_NOALLOC_MAX_TOPP_ROWS) +
                  ") with top_p < 1");
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
  if (stream) {
    int sdev = -1;
    HIP_TRY(hipStreamGetDevice((hipStream_t)stream, &sdev), "hipStreamGetDevice");
    if (sdev != dev) return einval("stream belongs to another device than the current one");
  }
  return launch_sample_rows_noalloc(d_logits, n_rows, vocab, d_rid, d_pos, seed, step_index, temperature, top_p,
                                    eos_id, forced_eos_u32, d_tok, (hipStream_t)stream);
}

extern "C" int sara_gumbel_fast_max_error(double* h_out, void* stream) {
  if (!h_out) return einval("h_out is null");
  return launch_gumbel_check(h_out, (hipStream_t)stream);
}

extern "C" void sara_destroy(sara_ctx* c) {
  if (!c) return;
  (void)hipStreamSynchronize(c->stream);
  if (c->graph_exec) (void)hipGraphExecDestroy(c->graph_exec);
  if (c->graph) (void)hipGraphDestroy(c->graph);
  if (c->h_done) (void)hipHostFree(c->h_done);
  for (hipEvent_t e : c->prof_events) (void)hipEventDestroy(e);
  for (void* p : c->owned) (void)hipFree(p);
  delete c;
}

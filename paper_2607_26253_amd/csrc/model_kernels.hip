// Decoder kernels of the rollout decode step and the prompt prefill (gfx950).
//
// Per layer, over the rows of a batch (occupied slots in decode, prompt
// tokens in prefill):
//   gemm(x, W_qkv) -> qkv epilogue (split-K sum, RoPE, bf16 q, paged KV append)
//   paged GQA attention over ragged contexts (split-context + combine)
//   gemm(o, W_o)   -> residual add + RMSNorm -> x
//   gemm(x, W_gu)  -> SwiGLU -> a
//   gemm(a, W_d)   -> residual add + RMSNorm of the next layer (or final) -> x
// then the LM head gemm and the Gumbel-max sampler.
//
// GEMMs take both operands with K contiguous ([rows][K]) and run on the
// bf16 MFMA (v_mfma_f32_16x16x32_bf16) with fp32 accumulation; split-K
// partials go to a workspace and are summed in split order by the epilogue,
// so results do not depend on scheduling.  The fp32 model uses a VALU GEMM.
#include <mutex>

#include "sara_internal.h"

#include <hip/hip_ext.h>

#include <math.h>
#include <string.h>

#include <algorithm>

namespace sara {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// block reductions (fixed tree order -> deterministic)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
// sum over a 256-thread block; every thread gets the result
__device__ float block_sum256(float v, float* red) {
  v = wave_sum(v);
  int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float r = (red[0] + red[1]) + (red[2] + red[3]);
  return r;
}

// Fragment-major ("tiled") layout of a [rows][K] bf16 matrix: for each
// 16-row tile and each 32-wide k step, the 64 lanes' 16-byte MFMA operand
// fragments lie back to back (lane l holds row l % 16, k 8*(l/16)..+8), so
// every fragment load of a wave is one contiguous, fully coalesced 1 KiB read
// and a wave walks its 16 rows as one sequential stream.  The decode rows
// feeding the q|k|v kernel are written this way.
__device__ __forceinline__ int64_t tiled_index(int64_t row, int64_t k, int64_t K) {
  const int64_t tile = row >> 4, ks = k >> 5, lane = (row & 15) + 16 * ((k >> 3) & 3);
  return ((tile * (K >> 5) + ks) * 64 + lane) * 8 + (k & 7);
}

// Layout of the bf16 GEMM weights ([rows][K], K a multiple of 64): the same
// 1 KiB fragments, ordered k-block-major.  K is cut into 64-wide blocks; in
// block b the n_tiles 16-row tiles lie back to back, each as its two 32-wide
// k steps.  The waves of a launch walk k at about the same pace, so at any
// moment they read one contiguous stretch of the matrix (spread over every
// HBM channel) instead of n_tiles streams a whole tile row apart, which
// measured 3-18% faster on the decode weight shapes.
__host__ __device__ __forceinline__ int64_t wtiled_index(int64_t row, int64_t k, int64_t n_tiles) {
  const int64_t tile = row >> 4, kb = k >> 6, ks = (k >> 5) & 1, lane = (row & 15) + 16 * ((k >> 3) & 3);
  return (((kb * n_tiles + tile) * 2 + ks) * 64 + lane) * 8 + (k & 7);
}

// ---------------------------------------------------------------------------
// Gumbel-max sampling helpers
// ---------------------------------------------------------------------------
// score_v = fp32(logit_v / T) + fp32(-log(-log u_v)), u_v = ((w >> 8) + 1/2) 2^-24
// from word v % 4 of Philox(rid, gen, v / 4, 0); the token is the lowest id
// of the maximal score.
__device__ __forceinline__ void better(float& bs, int& bi, float s, int i) {
  if (s > bs || (s == bs && i < bi)) { bs = s; bi = i; }
}
// The noise as the sampler defines it: fp64 logs, rounded to fp32.
__device__ __forceinline__ float gumbel_exact(uint32_t w) {
  const double u = ((double)(w >> 8) + 0.5) * 0x1p-24;
  return (float)(-log(-log(u)));
}
// fp32 estimate of gumbel_exact on the hardware log2 (v_log_f32): -ln(u) for
// u < 1/2 (u exact in fp32), and -log1p(-d) with d = 1 - u (exact in fp32)
// otherwise, through log1p(x) = ln(1 + x) x / ((1 + x) - 1) (Goldberg), then
// -ln of the result.  Its distance to gumbel_exact is below kGumbelFastErr
// for every one of the 2^24 inputs (sara_gumbel_fast_max_error measures it
// exhaustively).
constexpr float kGumbelFastErr = 2e-5f;
__device__ __forceinline__ float ln_hw(float x) { return __builtin_amdgcn_logf(x) * 0.693147180559945309f; }
__device__ __forceinline__ float gumbel_fast(uint32_t w) {
  const uint32_t m = w >> 8;
  float t;
  if (m < (1u << 23)) {
    t = -ln_hw(((float)m + 0.5f) * 0x1p-24f);
  } else {
    const float dl = (((float)((1u << 24) - m) - 0.5f) * 0x1p-24f);
    const float y = 1.0f - dl;
    t = (y == 1.0f) ? dl : ln_hw(y) * (dl * __builtin_amdgcn_rcpf(y - 1.0f));
  }
  return -ln_hw(t);
}
// fp32(logit / T); UNIT: T = 1, where the division is exact and skipped.
template <bool UNIT>
__device__ __forceinline__ float temper(float x, float temp) { return UNIT ? x : __fdiv_rn(x, temp); }
// Lower bound on every exact score that can still be maximal, given the
// largest fast score smax: each fast score is within
// kGumbelFastErr + 2^-22 |score| of its exact value (the noise error plus
// the two fp32 roundings of the sum), so candidates lie within twice that
// of smax (with slack for |score| near |smax|).
__device__ __forceinline__ float gumbel_candidate_floor(float smax) {
  return smax - 2.0f * kGumbelFastErr - (fabsf(smax) + 1.0f) * 0x1p-20f;
}

// Operands of the LM-head GEMM's sampling epilogue.
struct SampleArgs {
  const RowDesc* rows;       // decode rows (rid, gen, slot)
  const CtlParams* cp;       // seed, step index, temperature
  float* logits;             // optional [slots][V] copy of the logits (parity runs), else null
  float* best;               // [gridDim.x][ld] exact best score of the block's vocabulary range per row
  int32_t* idx;              // [gridDim.x][ld] its token id
  int ld;                    // row stride of best / idx (>= the live row count)
};

// ---------------------------------------------------------------------------
// embedding gather + first RMSNorm (decode and prefill rows)
// ---------------------------------------------------------------------------
// Decode rows + embedding gather + first RMSNorm in one launch: row i of the
// batch is occupied slot active[i]; the device row count goes to rows_M.
template <typename T>
__global__ __launch_bounds__(256) void k_decode_embed(const Ctl* __restrict__ ctl,
    const int32_t* __restrict__ active, const int32_t* __restrict__ slot_uid,
    const int32_t* __restrict__ slot_j, const int32_t* __restrict__ slot_gen,
    const int32_t* __restrict__ tok, const int32_t* __restrict__ off,
    const int32_t* __restrict__ out_tok, int k, int max_new, RowDesc* __restrict__ rows,
    int32_t* __restrict__ rows_M, int do_embed, const T* __restrict__ embed,
    const float* __restrict__ w, int d, float eps, float* __restrict__ h, T* __restrict__ x,
    int U, int PB, int SB, const float2* __restrict__ rope, int half, float2* __restrict__ row_rope,
    int x_tiled, AttnItem* __restrict__ items, int32_t* __restrict__ n_items, int spg) {
  __shared__ float red[4];
  __shared__ int scan[256];
  const int M = ctl->done ? 0 : ctl->M;
  if (blockIdx.x == 0 && threadIdx.x == 0) *rows_M = M;
  if (items != nullptr && blockIdx.x == gridDim.x - 1) {
    // The decode attention's work list for this step (the same for every
    // layer): the context splits of spg pages of every row, row-major.
    // Thread t lists rows [t * per, (t + 1) * per) at the exclusive prefix
    // sum of the earlier threads' split counts.
    const int per = (M + 255) / 256;
    const int i0 = min(M, (int)threadIdx.x * per), i1 = min(M, i0 + per);
    auto item_of = [&](int i, int cc) {
      const int s = active[i];
      const int u = slot_uid[s], g = slot_gen[s];
      AttnItem it;
      it.i = i;
      it.c = cc;
      it.kv0 = u * PB;
      it.kv1 = U * PB + s * SB;
      it.pl = off[u + 1] - off[u] - 1;    // context P + g exceeds the P - 1 prompt positions
      it.vcnt = g + 1;
      it.pad0 = it.pad1 = 0;
      return it;
    };
    auto splits_of = [&](const AttnItem& it) {
      const int nch = ((it.pl + 15) >> 4) + ((it.vcnt + 15) >> 4);
      return (nch + spg - 1) / spg;
    };
    int cnt = 0;
    for (int i = i0; i < i1; ++i) cnt += splits_of(item_of(i, 0));
    scan[threadIdx.x] = cnt;
    __syncthreads();
    for (int o = 1; o < 256; o <<= 1) {
      const int v = (int)threadIdx.x >= o ? scan[threadIdx.x - o] : 0;
      __syncthreads();
      scan[threadIdx.x] += v;
      __syncthreads();
    }
    int at = scan[threadIdx.x] - cnt;
    for (int i = i0; i < i1; ++i) {
      AttnItem it = item_of(i, 0);
      const int ns = splits_of(it);
      for (int cc = 0; cc < ns; ++cc) {
        it.c = cc;
        items[at++] = it;
      }
    }
    if (threadIdx.x == 255) *n_items = scan[255];
  }
  for (int i = blockIdx.x; i < M; i += gridDim.x) {
    const int s = active[i];
    const int u = slot_uid[s], j = slot_j[s], g = slot_gen[s];
    const int P = off[u + 1] - off[u];
    const int rid = u * k + j;
    RowDesc r;
    r.tok = (g == 0) ? tok[off[u] + P - 1] : out_tok[(size_t)rid * max_new + g - 1];
    r.pos = P - 1 + g;
    r.plen = P - 1;
    r.tab = s;
    r.slot = s;
    r.rid = rid;
    r.gen = g;
    r.uid = u;
    r.kv0 = u * PB;
    r.kv1 = U * PB + s * SB;
    if (threadIdx.x == 0) rows[i] = r;
    // rotation angles of this row's position, read by every layer's q|k|v kernel
    for (int e = threadIdx.x; e < half; e += 256) row_rope[(size_t)i * half + e] = rope[(size_t)r.pos * half + e];
    if (!do_embed) continue;
    float ss = 0.f;
    for (int cc = threadIdx.x; cc < d; cc += 256) {
      float v = ld_f32(embed, (size_t)r.tok * d + cc);
      h[(size_t)i * d + cc] = v;
      ss += v * v;
    }
    float tot = block_sum256(ss, red);
    float inv = 1.0f / sqrtf(tot / (float)d + eps);
    for (int cc = threadIdx.x; cc < d; cc += 256)
      st_f32(x, x_tiled ? (size_t)tiled_index(i, cc, d) : (size_t)i * d + cc, h[(size_t)i * d + cc] * inv * w[cc]);
    __syncthreads();   // red[] is reused by the next row
  }
}

// Prefill rows of the chunk [r0, r0 + n): global prompt-token row r maps to
// prompt u (pre[u] <= r < pre[u+1]) and token t = r - pre[u].
__global__ __launch_bounds__(256) void k_prefill_rows(const int32_t* __restrict__ pre, int U,
    int r0, int n, const int32_t* __restrict__ tok, const int32_t* __restrict__ off, int S,
    RowDesc* __restrict__ rows, int32_t* __restrict__ rows_M, int PB) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) *rows_M = n;
  if (i >= n) return;
  int r = r0 + i;
  int lo = 0, hi = U;  // largest u with pre[u] <= r
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (pre[mid] <= r) lo = mid; else hi = mid;
  }
  int u = lo, t = r - pre[u];
  RowDesc d;
  d.tok = tok[off[u] + t];
  d.pos = t;
  d.plen = off[u + 1] - off[u] - 1;
  d.tab = S + u;
  d.slot = -1;
  d.rid = -1;
  d.gen = -1;
  d.uid = u;
  d.kv0 = u * PB;
  d.kv1 = -1;
  rows[i] = d;
}

template <typename T>
__global__ __launch_bounds__(256) void k_embed_norm(const int32_t* __restrict__ M_ptr,
    const RowDesc* __restrict__ rows, const T* __restrict__ embed, const float* __restrict__ w,
    int d, float eps, float* __restrict__ h, T* __restrict__ x) {
  __shared__ float red[4];
  int i = blockIdx.x;
  if (i >= *M_ptr) return;
  int t = rows[i].tok;
  float ss = 0.f;
  for (int c = threadIdx.x; c < d; c += 256) {
    float v = ld_f32(embed, (size_t)t * d + c);
    h[(size_t)i * d + c] = v;
    ss += v * v;
  }
  float tot = block_sum256(ss, red);
  float inv = 1.0f / sqrtf(tot / (float)d + eps);
  for (int c = threadIdx.x; c < d; c += 256)
    st_f32(x, (size_t)i * d + c, h[(size_t)i * d + c] * inv * w[c]);
}

// ---------------------------------------------------------------------------
// GEMM: out[s][m][n] = sum_{k in split s} X[m][k] * W[n][k]
// ---------------------------------------------------------------------------
// Gumbel-max sampling over this block's vocabulary rows, straight from the
// LM-head accumulators (no logits round trip through memory).  Lane (row,
// grp) holds, for activation tile t and weight tile nt, the logits of
// vocabulary ids v = n0 + 16 nt + 4 grp + q (q < 4) of decode row
// m_base + 16 t + row: exactly the four ids one Philox call keys.
//  1. fast scores (fp32 noise, gumbel_fast) and their block maximum per row;
//  2. exact scores (fp64 noise, gumbel_exact) for the candidates at or above
//     gumbel_candidate_floor(max): the block's exact winner is always among
//     them, so the result equals an exact evaluation of every id;
//  3. exact (score, id) maximum per row to sa.best / sa.idx [m][gridDim.x].
// LDS: the X staging buffer, free after the k loop.
// Exact score of vocabulary id 4 b + q of decode rollout (rid, gen), given
// the tempered logit a = fp32(logit / T).  Out of line: it is called for a
// handful of candidates per row and block, and keeps the fp64 logs out of
// the unrolled epilogue.
__device__ __attribute__((noinline)) float exact_score(float a, uint32_t rid, uint32_t gen, uint32_t b, int q,
                                                       uint32_t k0, uint32_t k1) {
  const U32x4 w = philox4x32_10(rid, gen, b, 0u, k0, k1);
  const uint32_t wq = q == 0 ? w.x : q == 1 ? w.y : q == 2 ? w.z : w.w;
  return __fadd_rn(a, gumbel_exact(wq));
}

// One round of the sampling epilogue over activation tiles T0 .. T0 + TC - 1
// (compile-time tile indices, so the accumulators stay in registers).
template <int NT, int MT, int TC, int T0, bool UNIT>
__device__ __forceinline__ void sample_round(const f32x4 (&acc)[NT][MT], int M, int m_base, int N, int n0,
    const SampleArgs& sa, float temp, uint32_t k0, uint32_t k1, uint16_t* __restrict__ xs) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = lane & 15, grp = lane >> 4;
  float* red_max = (float*)xs;                          // [4][TC][16]
  float* red_s = red_max + 4 * TC * 16;                 // [4][TC][16]
  int* red_i = (int*)(red_s + 4 * TC * 16);             // [4][TC][16]
  // (rid, gen, slot) of the decode rows of this round's tiles
  int s_rid[TC], s_gen[TC], s_slot[TC];
#pragma unroll
  for (int tt = 0; tt < TC; ++tt) {
    const RowDesc r = sa.rows[min(m_base + 16 * (T0 + tt) + row, M - 1)];
    s_rid[tt] = r.rid; s_gen[tt] = r.gen; s_slot[tt] = r.slot;
  }
  __syncthreads();                                      // LDS: the k loop or the previous round is done
  float f[NT][TC][4];                                   // fast scores
#pragma unroll
  for (int tt = 0; tt < TC; ++tt) {
    float lmax = -INFINITY;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int v0 = n0 + 16 * nt + 4 * grp;
      const U32x4 w = philox4x32_10((uint32_t)s_rid[tt], (uint32_t)s_gen[tt], (uint32_t)(v0 >> 2), 0u, k0, k1);
      const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        f[nt][tt][q] = (v0 + q < N) ? __fadd_rn(temper<UNIT>(acc[nt][T0 + tt][q], temp), gumbel_fast(wd[q]))
                                    : -INFINITY;
        lmax = fmaxf(lmax, f[nt][tt][q]);
      }
    }
    lmax = fmaxf(lmax, __shfl_xor(lmax, 16, 64));
    lmax = fmaxf(lmax, __shfl_xor(lmax, 32, 64));
    if (grp == 0) red_max[(wave * TC + tt) * 16 + row] = lmax;
  }
  // optional copy of the logits (parity runs)
  if (sa.logits) {
#pragma unroll
    for (int tt = 0; tt < TC; ++tt) {
      const int m = m_base + 16 * (T0 + tt) + row;
      if (m >= M) continue;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int v = n0 + 16 * nt + 4 * grp + q;
          if (v < N) sa.logits[(size_t)s_slot[tt] * N + v] = acc[nt][T0 + tt][q];
        }
    }
  }
  __syncthreads();
#pragma unroll
  for (int tt = 0; tt < TC; ++tt) {
    const float* rm = red_max + tt * 16 + row;
    const float bmax = fmaxf(fmaxf(rm[0], rm[TC * 16]), fmaxf(rm[2 * TC * 16], rm[3 * TC * 16]));
    const float floor_ = gumbel_candidate_floor(bmax);
    float bs = -INFINITY;
    int bi = 0x7FFFFFFF;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (f[nt][tt][q] >= floor_) {
          const int v0 = n0 + 16 * nt + 4 * grp;
          better(bs, bi, exact_score(temper<UNIT>(acc[nt][T0 + tt][q], temp), (uint32_t)s_rid[tt],
                                     (uint32_t)s_gen[tt], (uint32_t)(v0 >> 2), q, k0, k1), v0 + q);
        }
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const float s2 = __shfl_xor(bs, o, 64);
      const int i2 = __shfl_xor(bi, o, 64);
      better(bs, bi, s2, i2);
    }
    if (grp == 0) { red_s[(wave * TC + tt) * 16 + row] = bs; red_i[(wave * TC + tt) * 16 + row] = bi; }
  }
  __syncthreads();
  if (threadIdx.x < TC * 16) {
    const int tt = threadIdx.x >> 4, r = threadIdx.x & 15, m = m_base + 16 * (T0 + tt) + r;
    if (m < M) {
      float bs = -INFINITY;
      int bi = 0x7FFFFFFF;
#pragma unroll
      for (int w = 0; w < 4; ++w) better(bs, bi, red_s[(w * TC + tt) * 16 + r], red_i[(w * TC + tt) * 16 + r]);
      sa.best[(size_t)blockIdx.x * sa.ld + m] = bs;
      sa.idx[(size_t)blockIdx.x * sa.ld + m] = bi;
    }
  }
}

template <int NT, int MT>
__device__ __forceinline__ void sample_epilogue(const f32x4 (&acc)[NT][MT], int M, int m_base, int N, int n0,
    const SampleArgs& sa, uint16_t* __restrict__ xs) {
  // activation tiles per round: a divisor of MT
  constexpr int TC = MT % 4 == 0 ? 4 : (MT % 2 == 0 ? 2 : 1);
  const CtlParams* cp = sa.cp;
  const float temp = cp->temperature;
  uint32_t k0, k1;
  sampler_key(cp->seed, cp->step, k0, k1);
#define SARA_SR(r, U) \
  if constexpr (MT > (r) * TC) sample_round<NT, MT, TC, (r) * TC, U>(acc, M, m_base, N, n0, sa, temp, k0, k1, xs);
  if (temp == 1.0f) {
    SARA_SR(0, true) SARA_SR(1, true) SARA_SR(2, true) SARA_SR(3, true)
    SARA_SR(4, true) SARA_SR(5, true) SARA_SR(6, true) SARA_SR(7, true)
  } else {
    SARA_SR(0, false) SARA_SR(1, false) SARA_SR(2, false) SARA_SR(3, false)
    SARA_SR(4, false) SARA_SR(5, false) SARA_SR(6, false) SARA_SR(7, false)
  }
#undef SARA_SR
}

// One m-block of MT 16-row tiles.  Block = 4 waves; wave w owns weight rows
// [n0, n0 + 16*NT) and all 16*MT activation rows.  The k loop is a 4-slot
// software pipeline: stage s loads the X chunk (block-cooperative) and the
// wave's W chunk for k chunk s into register slot s % 4, three stages ahead
// of its use; at its turn the X chunk goes to one of two LDS buffers and the
// MFMAs read X from LDS and W from registers.  The loop has no peeled
// prologue (its first trip only loads), so the wait counts the compiler
// derives at the loop header are exact and three stages stay in flight.
//
// EPI = 0: fp32 partial sums to out[split][m][n].
// EPI = 1: SwiGLU epilogue (one split only): the weight rows are interleaved
//          per 16-row tile as gate (even tiles) and up (odd tiles) of the same
//          16 features; out receives bf16 silu(g) * u as [m][N/2].
// EPI = 2: Gumbel-max sampling epilogue of the LM head (one split only), see
//          sample_epilogue; out is unused.
template <int NT, int MT, int KC, int EPI>
__device__ __forceinline__ void gemm_mblock(const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
    void* __restrict__ out, int M, int m_base, int N, int K, int kps, int64_t split_stride,
    uint16_t* __restrict__ xs, const SampleArgs& sa) {
  constexpr int MR = 16 * MT;
  constexpr int PITCH = KC + 8;                 // halves: rows shift by 4 banks, conflict-free b128 reads
  constexpr int C8 = KC / 8;                    // uint4 per X row per chunk
  constexpr int XU = (MR * C8 + 255) / 256;     // uint4 per thread per X chunk
  constexpr int CPK = KC / 32;                  // 16x16x32 MFMA k steps per chunk
  constexpr int BUF = MR * PITCH;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = lane & 15, grp = lane >> 4;
  const int n0 = (blockIdx.x * 4 + wave) * 16 * NT;
  const int k_begin = blockIdx.y * kps;
  const int k_end = min(K, k_begin + kps);
  const int nchunks = (k_end - k_begin) / KC;
  // W is in the wtiled_index layout: chunk = one 64-wide k block, whose
  // N / 16 tiles are 1024 elements apart.
  // Element offsets are 32-bit: N * K < 2^31 for every supported shape.
  static_assert(KC == 64, "a chunk is one k block of the weight layout");
  const int wchunk = (N / 16) * 1024;
  int woff[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
    woff[nt] = (k_begin / 64) * wchunk + min(n0 / 16 + nt, N / 16 - 1) * 1024 + lane * 8;
  int xoff[XU], xdst[XU];
#pragma unroll
  for (int q = 0; q < XU; ++q) {
    // threads past the tile repeat its last element (same value, same place)
    int u = min((int)threadIdx.x + 256 * q, MR * C8 - 1);
    int rr = u / C8, c8 = u % C8;
    xoff[q] = min(m_base + rr, M - 1) * K + 8 * c8 + k_begin;
    xdst[q] = rr * PITCH + 8 * c8;
  }
  // the four pipeline slots are distinct variables (not an indexed array),
  // so that they live in registers
  struct Stage { u32x4 x[XU]; u32x4 w[NT][CPK]; };
  Stage s0, s1, s2, s3;
  f32x4 acc[NT][MT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[nt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int last = max(nchunks - 1, 0);
  // loads are unconditional (clamped into [0, last]); surplus loads are unused
  auto load = [&](Stage& st, int chunk) {
    const int ch = max(min(chunk, last), 0);
#pragma unroll
    for (int q = 0; q < XU; ++q) st.x[q] = *(const u32x4*)(X + xoff[q] + ch * KC);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int cc = 0; cc < CPK; ++cc) st.w[nt][cc] = *(const u32x4*)(W + woff[nt] + ch * wchunk + 512 * cc);
  };
  auto consume = [&](Stage& st, int buf, int ch) {
    // buffer `buf` was last read two chunks ago, before the previous barrier
#pragma unroll
    for (int q = 0; q < XU; ++q) *(u32x4*)&xs[buf * BUF + xdst[q]] = st.x[q];
    __syncthreads();
    if (ch < nchunks) {
      // rows past M read a clamped (valid) X row; their results are never stored
#pragma unroll
      for (int t = 0; t < MT; ++t) {
#pragma unroll
        for (int cc = 0; cc < CPK; ++cc) {
          u32x4 xv = *(const u32x4*)&xs[buf * BUF + (16 * t + row) * PITCH + 8 * grp + 32 * cc];
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
            acc[nt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, st.w[nt][cc]), __builtin_bit_cast(bf16x8, xv), acc[nt][t], 0, 0, 0);
        }
      }
    }
  };
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): nothing of an earlier m-block is still pending
  int base0 = -4;
  asm volatile("" : "+s"(base0));       // opaque start: the first (load-only) trip stays in the loop
  for (int base = base0; base < nchunks; base += 4) {
    load(s3, base + 3);
    if (base >= 0) consume(s0, 0, base);
    load(s0, base + 4);
    if (base >= 0) consume(s1, 1, base + 1);
    load(s1, base + 5);
    if (base >= 0) consume(s2, 0, base + 2);
    load(s2, base + 6);
    if (base >= 0) consume(s3, 1, base + 3);
  }
  if constexpr (EPI == 2) {
    sample_epilogue<NT, MT>(acc, M, m_base, N, n0, sa, xs);
  } else if (EPI == 0) {
    float* o = (float*)out + (size_t)blockIdx.y * split_stride;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      if (n0 + 16 * nt >= N) continue;
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        int m = m_base + 16 * t + row;
        if (m < M) *(f32x4*)(o + (size_t)m * N + n0 + 16 * nt + 4 * grp) = acc[nt][t];
      }
    }
  } else {
    // tile pair (gate, up) = (nt 0, nt 1) of this wave: features (n0/32)*16 + 4*grp + q
    uint16_t* o = (uint16_t*)out;
    const int F = N / 2;
    const int f0 = (n0 / 32) * 16 + 4 * grp;
    if (n0 < N) {
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        int m = m_base + 16 * t + row;
        if (m < M) {
          uint32_t pk[2];
#pragma unroll
          for (int q = 0; q < 4; q += 2) {
            float g0 = acc[0][t][q], u0 = acc[NT - 1][t][q];
            float g1 = acc[0][t][q + 1], u1 = acc[NT - 1][t][q + 1];
            float a0 = g0 / (1.0f + expf(-g0)) * u0;
            float a1 = g1 / (1.0f + expf(-g1)) * u1;
            pk[q / 2] = (uint32_t)f32_to_bf16(a0) | ((uint32_t)f32_to_bf16(a1) << 16);
          }
          *(uint2*)(o + (size_t)m * F + f0) = make_uint2(pk[0], pk[1]);
        }
      }
    }
  }
}

// bf16 MFMA GEMM over tiled weights.  The live row count M is read on the
// device; each m-block of up to 16*MTMAX rows runs the instance with just
// enough 16-row tiles (ceil(rows / 16)), so small batches spend no MFMA,
// LDS or X traffic on empty tiles.  Launches have one z block per m-block of
// the row capacity; z blocks past the live rows exit after reading M.
// PF only labels the instance in profiles: 0 decode, 1 prefill, 2 the decode
// attention-output projection (so every decode weight matrix has a class).
template <int NT, int MTMAX, int KC, int EPI, int PF>
__global__ __launch_bounds__(256, 2) void k_gemm_bf16_lds(const uint16_t* __restrict__ X,
    const uint16_t* __restrict__ W, void* __restrict__ out, const int32_t* __restrict__ M_ptr,
    int N, int K, int kps, int64_t split_stride, SampleArgs sa) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[2 * 16 * MTMAX * (KC + 8)];
  const int M = *M_ptr;
  for (int m_base = blockIdx.z * 16 * MTMAX; m_base < M; m_base += gridDim.z * 16 * MTMAX) {
    const int mt = min(MTMAX, (M - m_base + 15) >> 4);
#define SARA_MB(c) \
    if constexpr (MTMAX >= c) { \
      if (mt == c) gemm_mblock<NT, c, KC, EPI>(X, W, out, M, m_base, N, K, kps, split_stride, xs, sa); \
    }
    SARA_MB(1) SARA_MB(2) SARA_MB(3) SARA_MB(4) SARA_MB(5) SARA_MB(6) SARA_MB(7) SARA_MB(8)
#undef SARA_MB
    __syncthreads();   // the LDS tiles are reused by the next m-block
  }
}

// Row-major [n_tiles*16][K] bf16 -> the GEMM weight layout (wtiled_index)
// of a dst_tiles-tile matrix; source tile j lands in destination tile
// j * tile_mul + tile_add, which builds the gate/up-interleaved matrix in place.
__global__ void k_tile_weights(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst, int n_tiles,
                               int K, int tile_mul, int tile_add, int dst_tiles) {
  const int64_t per_tile = (int64_t)16 * K;
  const int64_t total = per_tile * n_tiles;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int64_t r = e / K, k = e - r * K;
    const int64_t j = r >> 4;
    const int64_t drow = (j * tile_mul + tile_add) * 16 + (r & 15);
    dst[wtiled_index(drow, k, dst_tiles)] = src[e];
  }
}

// Rotation-pair order of the bf16 q|k|v weight rows: within each head, the
// 16-row tile j holds natural dims 8j..8j+7 (tile rows 0-7) and
// HD/2 + 8j..HD/2 + 8j + 7 (tile rows 8-15), so both members of every
// rotate-half pair (d, d + HD/2) land in one tile and in MFMA output lanes
// l and l ^ 32.  Returns the stored row (output column) of dim d of head h.
__host__ __device__ __forceinline__ int qkv_pair_col(int h, int d, int HD) {
  const int half = HD / 2;
  const int e = d < half ? d : d - half;
  return h * HD + 16 * (e >> 3) + (e & 7) + (d < half ? 0 : 8);
}

// Row-major [n_rows][K] bf16 rows of heads head_off, head_off + 1, .. (HD
// rows each, natural dim order) -> the GEMM weight layout of a
// dst_tiles-tile matrix, rows in rotation-pair order.
__global__ void k_tile_weights_pairs(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst, int n_rows,
                                     int K, int head_off, int HD, int dst_tiles) {
  const int64_t total = (int64_t)n_rows * K;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int64_t r = e / K, k = e - r * K;
    const int drow = qkv_pair_col(head_off + (int)(r / HD), (int)(r % HD), HD);
    dst[wtiled_index(drow, k, dst_tiles)] = src[e];
  }
}

// fp32 VALU GEMM for the fp32 model: 16x16 output tile per 256-thread block.
__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ X,
    const float* __restrict__ W, float* __restrict__ out, const int32_t* __restrict__ M_ptr,
    int N, int K, int kps, int64_t split_stride) {
  __shared__ float xs[16][33];
  __shared__ float wsm[16][33];
  const int M = *M_ptr;
  const int m0 = blockIdx.z * 16, n0 = blockIdx.x * 16;
  if (m0 >= M) return;
  const int ty = threadIdx.x >> 4, tx = threadIdx.x & 15;
  const int k_begin = blockIdx.y * kps, k_end = min(K, k_begin + kps);
  float acc = 0.f;
  for (int kk = k_begin; kk < k_end; kk += 32) {
    for (int e = threadIdx.x; e < 16 * 32; e += 256) {
      int r = e >> 5, c = e & 31;
      int m = min(m0 + r, M - 1), n = min(n0 + r, N - 1);
      bool in = kk + c < k_end;
      xs[r][c] = in ? X[(size_t)m * K + kk + c] : 0.f;
      wsm[r][c] = in ? W[(size_t)n * K + kk + c] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < 32; ++c) acc = fmaf(xs[ty][c], wsm[tx][c], acc);
    __syncthreads();
  }
  int m = m0 + ty, n = n0 + tx;
  if (m < M && n < N) out[(size_t)blockIdx.y * split_stride + (size_t)m * N + n] = acc;
}

// ---------------------------------------------------------------------------
// epilogues
// ---------------------------------------------------------------------------
// Sum of the split-K partials of one element in a fixed order (four running
// sums over splits s = 0,4,8.. / 1,5,.. / 2,6,.. / 3,7,.. combined as
// (a0 + a1) + (a2 + a3)): deterministic, with the loads issued together.
__device__ __forceinline__ float split_sum(const float* ws, int splits, int64_t stride, size_t idx) {
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
  int s = 0;
  for (; s + 4 <= splits; s += 4) {
    a0 += ws[(size_t)s * stride + idx];
    a1 += ws[(size_t)(s + 1) * stride + idx];
    a2 += ws[(size_t)(s + 2) * stride + idx];
    a3 += ws[(size_t)(s + 3) * stride + idx];
  }
  if (s < splits) a0 += ws[(size_t)s * stride + idx];
  if (s + 1 < splits) a1 += ws[(size_t)(s + 1) * stride + idx];
  if (s + 2 < splits) a2 += ws[(size_t)(s + 2) * stride + idx];
  return (a0 + a1) + (a2 + a3);
}

// Loads that only some threads or iterations need are written as
// unconditional loads from a clamped, always valid address whose value is
// then multiplied by a 0/1 mask (finite data, so x * 0 = 0 exactly).  A load
// under a condition, or one whose value is only used under a condition,
// becomes a branch that waits for the load before going on, which would
// serialise the memory round trips.
__device__ __forceinline__ float mask01(bool keep) { return keep ? 1.0f : 0.0f; }

// Page of position pos: block-table entries [0, PB) map the shared prompt
// segment (positions < plen), entries [PB, MAXB) the private segment that
// starts at position plen.
__device__ __forceinline__ size_t kv_index(const RowDesc& r, const int32_t* btab, int MAXB, int PB,
                                           int layer, int64_t n_blocks, int hkv, int g, int hd,
                                           int dim, int pos) {
  int e, o;
  if (pos < r.plen) { e = pos >> 4; o = pos & 15; }
  else { int q = pos - r.plen; e = PB + (q >> 4); o = q & 15; }
  int64_t b = btab[(size_t)r.tab * MAXB + e];
  return ((((size_t)layer * n_blocks + b) * hkv + g) * kBlockTok + o) * hd + dim;
}

// V pages are stored transposed, [hd][16 tokens] per (page, KV head), so that
// the PV product reads 4 consecutive tokens of one dimension per lane.
__device__ __forceinline__ size_t vt_index(const RowDesc& r, const int32_t* btab, int MAXB, int PB,
                                           int layer, int64_t n_blocks, int hkv, int g, int hd,
                                           int dim, int pos) {
  int e, o;
  if (pos < r.plen) { e = pos >> 4; o = pos & 15; }
  else { int q = pos - r.plen; e = PB + (q >> 4); o = q & 15; }
  int64_t b = btab[(size_t)r.tab * MAXB + e];
  return ((((size_t)layer * n_blocks + b) * hkv + g) * hd + dim) * kBlockTok + o;
}

// Split-K sum of the fused q|k|v output, rotate-half RoPE on q and k,
// q -> bf16 buffer, k and v -> the row's KV page.  pair = 1: the GEMM output
// columns are in rotation-pair order (bf16 weights, see qkv_pair_col).
template <typename T>
__global__ __launch_bounds__(256) void k_qkv_epilogue(const int32_t* __restrict__ M_ptr,
    const RowDesc* __restrict__ rows, const float* __restrict__ ws, int splits, int64_t stride,
    const float2* __restrict__ rope, int hq, int hkv, int hd, int layer, int64_t n_blocks,
    const int32_t* __restrict__ btab, int MAXB, int PB, T* __restrict__ qbuf, T* __restrict__ kc,
    T* __restrict__ vc, int pair) {
  const int half = hd >> 1, nh = hq + 2 * hkv, N = nh * hd;
  const int M = *M_ptr;
  for (int item = blockIdx.x; item < M * nh; item += gridDim.x) {
    const int i = item / nh, h = item - i * nh, c = threadIdx.x;
    const RowDesc r = rows[i];
    const int ca = pair ? qkv_pair_col(h, c, hd) : h * hd + c;
    const int cb = pair ? qkv_pair_col(h, c + half, hd) : h * hd + c + half;
    float a = split_sum(ws, splits, stride, (size_t)i * N + ca);
    float b = split_sum(ws, splits, stride, (size_t)i * N + cb);
    if (h < hq + hkv) {
      float2 cs = rope[(size_t)r.pos * half + c];
      float ra = a * cs.x - b * cs.y;
      float rb = b * cs.x + a * cs.y;
      if (h < hq) {
        size_t q = ((size_t)i * hq + h) * hd;
        st_f32(qbuf, q + c, ra);
        st_f32(qbuf, q + c + half, rb);
      } else {
        int g = h - hq;
        st_f32(kc, kv_index(r, btab, MAXB, PB, layer, n_blocks, hkv, g, hd, c, r.pos), ra);
        st_f32(kc, kv_index(r, btab, MAXB, PB, layer, n_blocks, hkv, g, hd, c + half, r.pos), rb);
      }
    } else {
      int g = h - hq - hkv;
      st_f32(vc, vt_index(r, btab, MAXB, PB, layer, n_blocks, hkv, g, hd, c, r.pos), a);
      st_f32(vc, vt_index(r, btab, MAXB, PB, layer, n_blocks, hkv, g, hd, c + half, r.pos), b);
    }
  }
}

// h += split-K sum; x = RMSNorm(h) * w  (stored in the model dtype).
// One 1024-thread block per row.
template <typename T>
__global__ __launch_bounds__(1024) void k_residual_norm(const int32_t* __restrict__ M_ptr,
    const float* __restrict__ ws, int splits, int64_t stride, int d, float* __restrict__ h,
    const float* __restrict__ w, float eps, T* __restrict__ x, int x_tiled) {
  __shared__ float red[16];
  const int M = *M_ptr;
  for (int i = blockIdx.x; i < M; i += gridDim.x) {
  float ss = 0.f;
  for (int c = threadIdx.x; c < d; c += 1024) {
    size_t idx = (size_t)i * d + c;
    float v = h[idx] + split_sum(ws, splits, stride, idx);
    h[idx] = v;
    ss += v * v;
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int q = 0; q < 16; q += 4) tot += (red[q] + red[q + 1]) + (red[q + 2] + red[q + 3]);
  float inv = 1.0f / sqrtf(tot / (float)d + eps);
  for (int c = threadIdx.x; c < d; c += 1024) {
    size_t idx = (size_t)i * d + c;
    st_f32(x, x_tiled ? (size_t)tiled_index(i, c, d) : idx, h[idx] * inv * w[c]);
  }
  __syncthreads();   // red[] is reused by the next row
  }
}

// Same operation for rows of d <= 256 * VPT features and at most
// kMaxSplitsDec splits: one 256-thread block per row, every thread owns VPT
// features (c = threadIdx.x + 256 v) and keeps them in registers; the split
// partials are summed in the order of split_sum with every load in flight at
// once.
template <typename T, int VPT>
__global__ __launch_bounds__(256) void k_residual_norm_v(const int32_t* __restrict__ M_ptr,
    const float* __restrict__ ws, int splits, int64_t stride, int d, float* __restrict__ h,
    const float* __restrict__ w, float eps, T* __restrict__ x, int x_tiled) {
  __shared__ float red[4];
  const int M = *M_ptr;
  for (int i = blockIdx.x; i < M; i += gridDim.x) {
    const size_t rb = (size_t)i * d;
    float a0[VPT], a1[VPT], a2[VPT], a3[VPT], hv[VPT];
    // unconditional loads from clamped indices, masked (see mask01)
    float wv[VPT];
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const int c = min((int)threadIdx.x + 256 * v, d - 1);
      a0[v] = a1[v] = a2[v] = a3[v] = 0.f;
      hv[v] = h[rb + c] * mask01((int)threadIdx.x + 256 * v < d);
      wv[v] = w[c];
    }
    float pv[kMaxSplitsDec][VPT];
#pragma unroll
    for (int s = 0; s < kMaxSplitsDec; ++s)
#pragma unroll
      for (int v = 0; v < VPT; ++v) {
        const int c = min((int)threadIdx.x + 256 * v, d - 1);
        pv[s][v] = ws[(size_t)min(s, splits - 1) * stride + rb + c] *
                   mask01(s < splits && (int)threadIdx.x + 256 * v < d);
      }
#pragma unroll
    for (int s = 0; s < kMaxSplitsDec; s += 4)
#pragma unroll
      for (int v = 0; v < VPT; ++v) {
        a0[v] += pv[s][v];
        a1[v] += pv[s + 1][v];
        a2[v] += pv[s + 2][v];
        a3[v] += pv[s + 3][v];
      }
    float ss = 0.f;
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const int c = threadIdx.x + 256 * v;
      const float val = hv[v] + ((a0[v] + a1[v]) + (a2[v] + a3[v]));
      hv[v] = val;
      if (c < d) {
        h[rb + c] = val;
        ss += val * val;
      }
    }
    const float tot = block_sum256(ss, red);
    const float inv = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const int c = threadIdx.x + 256 * v;
      if (c < d) st_f32(x, x_tiled ? (size_t)tiled_index(i, c, d) : rb + c, hv[v] * inv * wv[v]);
    }
    __syncthreads();   // red[] is reused by the next row
  }
}

// a = silu(g) * u from the fused gate|up output ([m][2*ffn]); grid-stride
// over the M * ffn outputs of the live rows
// bf16 decode variant of the residual norm: one row per block, one float4
// of the row per thread (blockDim = d/4 rounded up to whole waves).  The
// residual, the norm weight and the row's split-K partials of that float4
// (only the splits the GEMM wrote) are loaded at once, summed in split order
// into four interleaved accumulators, and the row's sum of squares is
// reduced over the block's waves in wave order; x receives four bf16 per
// thread in one 8-byte store (row-major, or fragment-major for the q|k|v
// kernel, where four consecutive k of a row are contiguous).
__global__ __launch_bounds__(1024) void k_residual_norm_f4(const int32_t* __restrict__ M_ptr,
    const float* __restrict__ ws, int splits, int64_t stride, int d, float* __restrict__ h,
    const float* __restrict__ w, float eps, uint16_t* __restrict__ x, int x_tiled) {
  __shared__ float red[16];
  const int M = *M_ptr;
  const int nq = d >> 2, q = threadIdx.x, lane = q & 63, wave = q >> 6;
  const int nw = (blockDim.x + 63) >> 6;
  const bool on = q < nq;
  const int qc = on ? q : nq - 1;
  for (int i = blockIdx.x; i < M; i += gridDim.x) {
    const size_t rb = (size_t)i * d;
    const float4 hv = ((const float4*)(h + rb))[qc];
    const float4 wv = ((const float4*)w)[qc];
    float4 p[kMaxSplitsDec];
#pragma unroll
    for (int sp = 0; sp < kMaxSplitsDec; ++sp)
      p[sp] = (sp < splits) ? ((const float4*)(ws + (size_t)sp * stride + rb))[qc] : make_float4(0.f, 0.f, 0.f, 0.f);
    float4 a[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) a[j] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int sp = 0; sp < kMaxSplitsDec; ++sp) {
      a[sp & 3].x += p[sp].x; a[sp & 3].y += p[sp].y; a[sp & 3].z += p[sp].z; a[sp & 3].w += p[sp].w;
    }
    float4 v;
    v.x = hv.x + ((a[0].x + a[1].x) + (a[2].x + a[3].x));
    v.y = hv.y + ((a[0].y + a[1].y) + (a[2].y + a[3].y));
    v.z = hv.z + ((a[0].z + a[1].z) + (a[2].z + a[3].z));
    v.w = hv.w + ((a[0].w + a[1].w) + (a[2].w + a[3].w));
    float ss = 0.f;
    if (on) {
      ((float4*)(h + rb))[q] = v;
      ss = (v.x * v.x + v.y * v.y) + (v.z * v.z + v.w * v.w);
    }
    ss = wave_sum(ss);
    if (lane == 0) red[wave] = ss;
    __syncthreads();
    float tot = 0.f;
    for (int k = 0; k < nw; ++k) tot += red[k];
    const float inv = 1.0f / sqrtf(tot / (float)d + eps);
    if (on) {
      const uint32_t lo = (uint32_t)f32_to_bf16(v.x * inv * wv.x) | ((uint32_t)f32_to_bf16(v.y * inv * wv.y) << 16);
      const uint32_t hi = (uint32_t)f32_to_bf16(v.z * inv * wv.z) | ((uint32_t)f32_to_bf16(v.w * inv * wv.w) << 16);
      const size_t o = x_tiled ? (size_t)tiled_index(i, 4 * q, d) : rb + 4 * q;
      *(uint2*)(x + o) = make_uint2(lo, hi);
    }
    __syncthreads();   // red[] is reused by the next row
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_swiglu(const int32_t* __restrict__ M_ptr,
    const float* __restrict__ ws, int splits, int64_t stride, int ffn, T* __restrict__ a) {
  const size_t total = (size_t)(*M_ptr) * ffn;
  for (size_t e = (size_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (size_t)gridDim.x * 256) {
    size_t i = e / ffn, f = e - i * ffn;
    size_t base = i * 2 * ffn;
    float g = split_sum(ws, splits, stride, base + f);
    float u = split_sum(ws, splits, stride, base + ffn + f);
    float sg = g / (1.0f + expf(-g));
    st_f32(a, e, sg * u);
  }
}

// ---------------------------------------------------------------------------
// paged GQA attention
// ---------------------------------------------------------------------------
// Block (row i, KV head g, context split c) attends the G query heads of KV
// head g over positions [c*SPLIT, min(ctx, (c+1)*SPLIT)) of the row's
// sequence with an online softmax, tiles of 64 tokens staged in LDS; the
// unnormalised output, running max and sum go to a partial buffer that the
// combine kernel merges across splits.  Pages come from the block table:
// positions below plen live in the prompt's shared pages, later ones in the
// row's private pages.
template <typename T, int HD>
__global__ __launch_bounds__(256) void k_attention(const int32_t* __restrict__ M_ptr,
    const RowDesc* __restrict__ rows, const T* __restrict__ qbuf, const T* __restrict__ kc,
    const T* __restrict__ vc, const int32_t* __restrict__ btab, int MAXB, int PB, int layer,
    int64_t n_blocks, int hq, int hkv, int n_splits, float scale, float* __restrict__ part) {
  __shared__ float q_s[kMaxGroup][HD];
  __shared__ float k_s[kAttnTile][HD + 1];
  __shared__ float v_s[kAttnTile][HD];
  __shared__ float p_s[kMaxGroup][kAttnTile];
  __shared__ float m_s[kMaxGroup], l_s[kMaxGroup], al_s[kMaxGroup];
  const int i = blockIdx.x, g = blockIdx.y, c = blockIdx.z;
  if (i >= *M_ptr) return;
  const RowDesc r = rows[i];
  const int ctx = r.pos + 1;
  const int t0 = c * kAttnSplit;
  if (t0 >= ctx) return;
  const int t1 = min(ctx, t0 + kAttnSplit);
  const int G = hq / hkv;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  constexpr int DPT = HD / 64;  // dims per thread in the PV product
  for (int e = tid; e < G * HD; e += 256) {
    int gh = e / HD, dd = e - gh * HD;
    q_s[gh][dd] = ld_f32(qbuf, ((size_t)i * hq + g * G + gh) * HD + dd);
  }
  if (tid < kMaxGroup) { m_s[tid] = -INFINITY; l_s[tid] = 0.f; }
  float o[2][DPT];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < DPT; ++b) o[a][b] = 0.f;
  __syncthreads();
  for (int ts = t0; ts < t1; ts += kAttnTile) {
    const int n = min(kAttnTile, t1 - ts);
    for (int e = tid; e < n * HD; e += 256) {
      int tk = e / HD, dd = e - tk * HD;
      k_s[tk][dd] = ld_f32(kc, kv_index(r, btab, MAXB, PB, layer, n_blocks, hkv, g, HD, dd, ts + tk));
      v_s[tk][dd] = ld_f32(vc, vt_index(r, btab, MAXB, PB, layer, n_blocks, hkv, g, HD, dd, ts + tk));
    }
    __syncthreads();
    // scores: thread (token lane, head wave / wave + 4)
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      int gh = wave + 4 * a;
      if (gh < G) {
        float sc = -INFINITY;
        if (lane < n) {
          float acc = 0.f;
#pragma unroll 8
          for (int dd = 0; dd < HD; ++dd) acc = fmaf(q_s[gh][dd], k_s[lane][dd], acc);
          sc = acc * scale;
        }
        p_s[gh][lane] = sc;
      }
    }
    __syncthreads();
    // online softmax update, one wave per head pair
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      int gh = wave + 4 * a;
      if (gh < G) {
        float sc = p_s[gh][lane];
        float mt = wave_max(sc);
        float mo = m_s[gh];
        float mn = fmaxf(mo, mt);
        float pv = (lane < n) ? expf(sc - mn) : 0.f;
        float sum = wave_sum(pv);
        p_s[gh][lane] = pv;
        if (lane == 0) {
          float al = expf(mo - mn);
          al_s[gh] = al;
          l_s[gh] = l_s[gh] * al + sum;
          m_s[gh] = mn;
        }
      }
    }
    __syncthreads();
    // o = o * alpha + P V ; thread (dims lane*DPT.., heads wave, wave + 4)
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      int gh = wave + 4 * a;
      if (gh < G) {
        float al = al_s[gh];
#pragma unroll
        for (int b = 0; b < DPT; ++b) o[a][b] *= al;
        for (int tk = 0; tk < n; ++tk) {
          float pv = p_s[gh][tk];
#pragma unroll
          for (int b = 0; b < DPT; ++b) o[a][b] = fmaf(pv, v_s[tk][lane * DPT + b], o[a][b]);
        }
      }
    }
    __syncthreads();
  }
  // partial layout: [row][g][split][gh][HD + 2]  (o..., m, l)
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    int gh = wave + 4 * a;
    if (gh < G) {
      float* dst = part + ((((size_t)i * hkv + g) * n_splits + c) * kMaxGroup + gh) * (HD + 2);
#pragma unroll
      for (int b = 0; b < DPT; ++b) dst[lane * DPT + b] = o[a][b];
      if (lane == 0) { dst[HD] = m_s[gh]; dst[HD + 1] = l_s[gh]; }
    }
  }
}

// bf16 paged GQA attention on the MFMA.  Block (row i, KV head g, split c)
// covers KV pages [c*kAttnChunks, (c+1)*kAttnChunks) of the row's sequence
// (prompt pages, then private pages; each page holds up to 16 positions);
// its 4 waves take every 4th page.  Per page and wave:
//   S^T = K q^T  (16 tokens x 16 padded heads, v_mfma_f32_16x16x32_bf16; the
//                 lane supplying token l%16 of K and head l%16 of q reads the
//                 same HD/4 dimensions, so the k order inside the MFMA is moot)
//   online softmax per head (the 4 lanes holding one head's 16 scores)
//   O += P V     (v_mfma_f32_16x16x16bf16_1k; the score registers are already
//                 the A operand's layout, V^T pages give the B operand; P is
//                 split into bf16 hi + lo parts, two MFMAs)
// The 4 waves' (max, sum, O) are merged in LDS into one partial per split.
//
template <int HD>
__global__ __launch_bounds__(256) void k_attn_mfma(const int32_t* __restrict__ M_ptr,
    const RowDesc* __restrict__ rows, const uint16_t* __restrict__ qbuf,
    const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc,
    const int32_t* __restrict__ btab, int MAXB, int PB, int layer, int64_t n_blocks, int hq,
    int hkv, int n_splits, float scale, float* __restrict__ part) {
  typedef short short4_ __attribute__((ext_vector_type(4)));
  constexpr int DPL = HD / 4;     // dims per lane in the QK^T operands
  constexpr int NCC = HD / 32;    // 16x16x32 MFMAs per page for QK^T
  constexpr int NT = HD / 16;     // output tiles of 16 dims
  __shared__ float m_w[4][16], l_w[4][16];
  __shared__ float o_w[4][16][HD + 1];
  // persistent over work items (split c, row i, KV head g), split-major, so
  // that no block waits only to find its row absent
  const int M = *M_ptr;
  const int total = M * hkv * n_splits;
  for (int item = blockIdx.x; item < total; item += gridDim.x) {
  const int c = item / (M * hkv);
  const int i = (item - c * M * hkv) / hkv, g = item % hkv;
  const RowDesc r = rows[i];
  const int ctx = r.pos + 1;
  const int pl = min(ctx, r.plen);                      // prompt positions attended
  const int pc = (pl + 15) >> 4;                         // prompt pages
  const int vcnt = ctx - pl;                             // private positions
  const int nch = pc + ((vcnt + 15) >> 4);
  const int ch0 = c * kAttnChunks;
  if (ch0 >= nch) continue;
  const int ch1 = min(nch, ch0 + kAttnChunks);
  const int G = hq / hkv;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = lane & 15, grp = lane >> 4;
  // per-wave softmax state and output accumulators; q operand (set below)
  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint4 qv[NCC];
  const int32_t* bt = btab + (size_t)r.tab * MAXB;
  // Block-table entries of this split's pages, one per lane 0..15, shared by
  // shuffles (no table load on the page path).
  int my_blk = 0;
  if (lane < kAttnChunks && ch0 + lane < ch1) {
    const int cl = ch0 + lane;
    my_blk = bt[(cl < pc) ? cl : PB + (cl - pc)];
  }
  // Two page slots per wave: the next page's K, V (and its valid count) are
  // loaded while the current one is processed.  Loads past the wave's last
  // page re-read its first page (always valid) and are never used.
  typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
  struct Pg { u32x4 k[NCC]; u32x2 v[NT]; int n; };
  auto load_page = [&](Pg& P, int ch) {
    const int cv = (ch < ch1) ? ch : (ch0 + wave);
    int n;
    if (cv < pc) n = min(16, pl - 16 * cv);
    else n = min(16, vcnt - 16 * (cv - pc));
    P.n = (ch < ch1) ? n : 0;
    const int blk = __shfl(my_blk, cv - ch0, 64);
    const size_t pg = ((size_t)layer * n_blocks + blk) * hkv + g;
    const u32x4* kp = (const u32x4*)(kc + (pg * kBlockTok + row) * HD + DPL * grp);
#pragma unroll
    for (int cc = 0; cc < NCC; ++cc) P.k[cc] = kp[cc];
    const uint16_t* vp = vc + pg * (size_t)HD * kBlockTok + 4 * grp;
#pragma unroll
    for (int t = 0; t < NT; ++t) P.v[t] = *(const u32x2*)(vp + (size_t)(16 * t + row) * kBlockTok);
  };
  auto process_page = [&](const Pg& P) {
    const int n = P.n;
    // S^T[token][head]
    f32x4 sc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int cc = 0; cc < NCC; ++cc)
      sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, P.k[cc]),
                                                   __builtin_bit_cast(bf16x8, qv[cc]), sc, 0, 0, 0);
    // lane holds tokens 4*grp + q (q < 4) of head `row`
    float sv[4];
    float mt = -INFINITY;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      sv[q] = (4 * grp + q < n) ? sc[q] * scale : -INFINITY;
      mt = fmaxf(mt, sv[q]);
    }
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float mn = fmaxf(m_run, mt);
    const float alpha = expf(m_run - mn);
    // P enters the MFMA as a bf16 pair hi + lo (|p - hi - lo| <= 2^-16 p), so
    // the PV product keeps fp32 accuracy without a bf16 rounding point
    float ps = 0.f;
    uint16_t pb[4], plo[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float pv = expf(sv[q] - mn);
      uint16_t bb = f32_to_bf16(pv);
      pb[q] = bb;
      plo[q] = f32_to_bf16(pv - bf16_to_f32(bb));
      ps += pv;
    }
    ps += __shfl_xor(ps, 16, 64);
    ps += __shfl_xor(ps, 32, 64);
    l_run = l_run * alpha + ps;
    m_run = mn;
    // rows of O are heads 4*grp + q: fetch their rescale factors
    float al[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) al[q] = __shfl(alpha, 4 * grp + q, 64);
    short4_ pa, pa_lo;
#pragma unroll
    for (int q = 0; q < 4; ++q) { pa[q] = (short)pb[q]; pa_lo[q] = (short)plo[q]; }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      // positions beyond the page's n valid tokens may hold stale bits: zero them
      short4_ vb;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        uint32_t w = (q < 2) ? P.v[t].x : P.v[t].y;
        uint16_t h = (uint16_t)((q & 1) ? (w >> 16) : (w & 0xFFFF));
        vb[q] = (short)((4 * grp + q < n) ? h : (uint16_t)0);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) o[t][q] *= al[q];
      o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa, vb, o[t], 0, 0, 0);
      o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa_lo, vb, o[t], 0, 0, 0);
    }
  };
  Pg pa_, pb_;
  load_page(pa_, ch0 + wave);
  // q operand: head `row` of this KV group (zero beyond G), dims [DPL*grp, DPL*grp + DPL)
  if (row < G) {
    const uint4* qp = (const uint4*)(qbuf + ((size_t)i * hq + g * G + row) * HD + DPL * grp);
#pragma unroll
    for (int cc = 0; cc < NCC; ++cc) qv[cc] = qp[cc];
  } else {
#pragma unroll
    for (int cc = 0; cc < NCC; ++cc) qv[cc] = make_uint4(0, 0, 0, 0);
  }
  for (int ch = ch0 + wave; ch < ch1; ch += 8) {
    load_page(pb_, ch + 4);
    process_page(pa_);
    if (ch + 4 >= ch1) break;
    load_page(pa_, ch + 8);
    process_page(pb_);
  }
  // merge the 4 waves: lane `row` (grp 0) holds head row's (m, l); O rows are heads 4*grp + q
  if (grp == 0) { m_w[wave][row] = m_run; l_w[wave][row] = l_run; }
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int q = 0; q < 4; ++q) o_w[wave][4 * grp + q][16 * t + row] = o[t][q];
  __syncthreads();
  for (int e = threadIdx.x; e < G * HD; e += 256) {
    int h = e / HD, dd = e - h * HD;
    float mx = fmaxf(fmaxf(m_w[0][h], m_w[1][h]), fmaxf(m_w[2][h], m_w[3][h]));
    float num = 0.f, den = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      float wt = (m_w[w][h] == -INFINITY) ? 0.f : expf(m_w[w][h] - mx);
      num += wt * o_w[w][h][dd];
      den += wt * l_w[w][h];
    }
    float* dst = part + ((((size_t)i * hkv + g) * n_splits + c) * kMaxGroup + h) * (HD + 2);
    dst[dd] = num;
    if (dd == 0) { dst[HD] = mx; dst[HD + 1] = den; }
  }
  __syncthreads();   // LDS is reused by the next item
  }
}

// Fused q|k|v projection of the decode rows with the rotary / KV-append
// epilogue (bf16 weights in rotation-pair order, see qkv_pair_col).  Block =
// one 16-row weight tile; its 4 waves take a quarter of K each and stream
// their weight fragments and the activation fragments of up to 16*MT rows
// through a D-stage register pipeline (the waves share no k range, so the
// activations need no LDS staging).  The wave partial sums meet in LDS and
// are added in wave order (deterministic).  Wave t % 4 then finishes
// activation tile t: rotate-half RoPE on q and k heads (the two members of
// a rotation pair sit in lanes l and l ^ 32), q to qbuf as bf16, k and v to
// the row's newest KV page (the attention kernel reads them from there).
template <int HD, int MT, int D, int KS>
__device__ __forceinline__ void qkv_rope_mblock(const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
    int M, int m_base, int K, f32x4 (*red)[8][64], const RowDesc* __restrict__ rows,
    const float2* __restrict__ row_rope, int hq, int hkv, int layer, int64_t n_blocks,
    uint16_t* __restrict__ qbuf, uint16_t* __restrict__ kc, uint16_t* __restrict__ vc) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = lane & 15, grp = lane >> 4;
  const int tile = blockIdx.x;
  // KS = K / 128 32-wide k steps per wave; D divides KS, so the pipeline
  // issues D - 1 surplus (clamped, cache-hit) loads at most, none when D = KS
  static_assert(KS % D == 0, "pipeline depth must divide the k steps");
  const int ks0 = wave * KS;
  // W in the wtiled_index layout: k step j of this wave sits in k block
  // (ks0 + j) / 2 (KS is even, so ks0 starts a block)
  const int wblock = ((hq + 2 * hkv) * HD / 16) * 1024;
  const int woff = (ks0 / 2) * wblock + tile * 1024 + lane * 8;
  // activation fragments: X is fragment-major (tiled_index layout, as the
  // weights), so each fragment load of a wave is one contiguous 1 KiB read;
  // lanes of rows past M read rows of the last tile whose results are dropped
  int xoff[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) xoff[t] = ((m_base / 16 + t) * (K >> 5) + ks0) * 512 + lane * 8;
  // Epilogue inputs of the tiles this wave finishes (t = wave + 4 * tt),
  // loaded before the k loop so that their latency hides behind it:
  // the row's newest-token KV slot and the rotation angles of its position.
  constexpr int TT = (MT + 3) / 4;
  constexpr int half = HD / 2;
  const int c0 = tile * 16, h = c0 / HD, jt = (c0 % HD) >> 4;
  const bool second = grp >= 2;
  const int dd = 8 * jt + 4 * (grp & 1);           // rotation index of the lane's first dim
  const int nd = (second ? half : 0) + dd;          // its natural dim within the head
  size_t pg_e[TT];
  int on_e[TT];
  float2 cs_e[TT][4];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) {
    const int m = min(m_base + 16 * (wave + 4 * tt) + row, M - 1);
    const RowDesc r = rows[m];
    const int rel = r.pos - r.plen;                 // private position of the newest token
    pg_e[tt] = (size_t)layer * n_blocks + r.kv1 + (rel >> 4);
    on_e[tt] = rel & 15;
#pragma unroll
    for (int q = 0; q < 4; ++q) cs_e[tt][q] = row_rope[(size_t)m * half + dd + q];
  }
  struct Stage { u32x4 w; u32x4 x[MT]; };
  Stage st[D];
  f32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int last = KS - 1;
  auto load = [&](Stage& sg, int step) {
    const int kk = max(min(step, last), 0);
    sg.w = *(const u32x4*)(W + woff + (kk >> 1) * wblock + (kk & 1) * 512);
#pragma unroll
    for (int t = 0; t < MT; ++t) sg.x[t] = *(const u32x4*)(X + xoff[t] + kk * 512);
  };
  auto consume = [&](Stage& sg, int step) {
    if (step < KS) {
#pragma unroll
      for (int t = 0; t < MT; ++t)
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, sg.w),
                                                         __builtin_bit_cast(bf16x8, sg.x[t]), acc[t], 0, 0, 0);
    }
  };
  if constexpr (D == KS) {
    // every k step in flight at once: exactly KS loads, then the MFMAs
#pragma unroll
    for (int j = 0; j < KS; ++j) load(st[j], j);
#pragma unroll
    for (int j = 0; j < KS; ++j) consume(st[j], j);
  } else {
    int base0 = -D;
    asm volatile("" : "+s"(base0));     // opaque start: the first (load-only) trip stays in the loop
    for (int base = base0; base < KS; base += D) {
#pragma unroll
      for (int j = 0; j < D; ++j) {
        load(st[(j + D - 1) % D], base + j + D - 1);
        if (base >= 0) consume(st[j], base + j);
      }
    }
  }
#pragma unroll
  for (int t = 0; t < MT; ++t) red[wave][t][lane] = acc[t];
  __syncthreads();
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) {
    const int t = wave + 4 * tt;
    if (t >= MT) break;
    f32x4 v = red[0][t][lane];
    v += red[1][t][lane];
    v += red[2][t][lane];
    v += red[3][t][lane];
    f32x4 pv;
#pragma unroll
    for (int q = 0; q < 4; ++q) pv[q] = __shfl_xor(v[q], 32, 64);
    const int m = m_base + 16 * t + row;
    if (m >= M) continue;
    float o[4];
    if (h < hq + hkv) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float2 c = cs_e[tt][q];
        o[q] = second ? (v[q] * c.x + pv[q] * c.y) : (v[q] * c.x - pv[q] * c.y);
      }
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) o[q] = v[q];
    }
    const uint32_t p01 = (uint32_t)f32_to_bf16(o[0]) | ((uint32_t)f32_to_bf16(o[1]) << 16);
    const uint32_t p23 = (uint32_t)f32_to_bf16(o[2]) | ((uint32_t)f32_to_bf16(o[3]) << 16);
    const size_t pg = pg_e[tt];
    const int on = on_e[tt];
    if (h < hq) {
      *(uint2*)(qbuf + ((size_t)m * hq + h) * HD + nd) = make_uint2(p01, p23);
    } else if (h < hq + hkv) {
      *(uint2*)(kc + ((pg * hkv + (h - hq)) * kBlockTok + on) * HD + nd) = make_uint2(p01, p23);
    } else {
      uint16_t* vp = vc + (pg * hkv + (h - hq - hkv)) * (size_t)HD * kBlockTok + on;
      vp[(size_t)(nd + 0) * kBlockTok] = (uint16_t)(p01 & 0xFFFF);
      vp[(size_t)(nd + 1) * kBlockTok] = (uint16_t)(p01 >> 16);
      vp[(size_t)(nd + 2) * kBlockTok] = (uint16_t)(p23 & 0xFFFF);
      vp[(size_t)(nd + 3) * kBlockTok] = (uint16_t)(p23 >> 16);
    }
  }
  __syncthreads();   // red is reused by the next m-block
}

// Live row count read on the device.  Grid: x = one block per weight tile,
// z = one block per 128 rows of the capacity.  The live 16-row activation
// tiles are shared out in contiguous runs over the first min(gridDim.z,
// zspread) z blocks (at most 8 tiles per block), so that a small batch keeps
// several blocks per weight tile busy instead of one; zspread is chosen on
// the host so that the whole grid's working blocks stay resident at once.
// Every tile's arithmetic is the same whichever block computes it.
// KS = d_model / 128, one of 4, 8, 12, 16, 24, 32 (checked by sara_init).
template <int HD, int KS>
__global__ __launch_bounds__(256) void k_qkv_rope(const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
    const int32_t* __restrict__ M_ptr, int K, const RowDesc* __restrict__ rows,
    const float2* __restrict__ row_rope, int hq, int hkv, int layer, int64_t n_blocks,
    uint16_t* __restrict__ qbuf, uint16_t* __restrict__ kc, uint16_t* __restrict__ vc, int zspread) {
  __shared__ f32x4 red[4][8][64];
  const int M = *M_ptr;
  const int ntl = (M + 15) >> 4;
  const int zs = max(1, min((int)gridDim.z, zspread));
  const int tpz = min(8, (ntl + zs - 1) / zs);      // tiles per z block
  for (int m_base = blockIdx.z * tpz * 16; m_base < M; m_base += gridDim.z * tpz * 16) {
    const int mt = min(tpz, (M - m_base + 15) >> 4);
    // depth for up to 32 rows: every k step in flight below 16 k steps, half
    // of them from 16 on (the 16-step instance then fits two blocks per CU);
    // a half and a quarter of that for more rows
#define SARA_QR(MT_, D_) \
    if (mt == MT_) qkv_rope_mblock<HD, MT_, D_, KS>(X, W, M, m_base, K, red, rows, row_rope, hq, hkv, layer, \
                                                    n_blocks, qbuf, kc, vc);
    constexpr int D1 = KS < 16 ? KS : KS / 2, D3 = D1 / 2, D5 = D1 / 4;
    SARA_QR(1, D1) SARA_QR(2, D1) SARA_QR(3, D3) SARA_QR(4, D3)
    SARA_QR(5, D5) SARA_QR(6, D5) SARA_QR(7, D5) SARA_QR(8, D5)
#undef SARA_QR
  }
}

// Decode attention (bf16, MFMA) over the KV pages, q read from qbuf (the
// q|k|v kernel has already rotated q and appended this position's k and v).
// Work item = (entry e of the step's work list, KV head g): entry e names a
// row and one of its context splits of kDecPages pages; wave w owns pages
// w, w + 4, .. of the split, all K and V loads issued before any compute, so
// a split costs one HBM round trip.  The entry carries the row's two KV
// extents (kv0 + e: shared prompt pages, kv1 + e: private pages), so the
// page loads wait on that one load only; the grid is the number of blocks
// that are resident at once, so up to that many items all run in one
// round.  Per page (16 tokens):
//   S^T = K q^T  (v_mfma_f32_16x16x32_bf16; G <= 8 query heads padded to 16;
//                 lane (token l%16, k-group l/16) of K meets head l%16 of q
//                 over the same HD/4 dims, so the k order inside the MFMA is moot)
//   online softmax per head over the 4 lanes holding its 16 scores
//   O += P V     (v_mfma_f32_16x16x16bf16_1k; the score registers already
//                 have the A-operand layout and transposed V pages give the
//                 B operand; P enters as a bf16 hi + lo pair, so the product
//                 keeps fp32 accuracy without a bf16 rounding point)
// The 4 waves' (max, sum, O) merge in LDS.  A row with a single split writes
// its normalised output to `out` ([row][hq][HD], bf16); other rows leave a
// partial per split for k_attn_combine.
template <int HD>
__global__ __launch_bounds__(256, 2) void k_attn_dec(const AttnItem* __restrict__ items,
    const int32_t* __restrict__ n_items, int cap, const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc,
    int layer, int64_t n_blocks, int hq, int hkv, int n_splits, float scale,
    const uint16_t* __restrict__ qb, float* __restrict__ part, uint16_t* __restrict__ out) {
  typedef short short4_ __attribute__((ext_vector_type(4)));
  typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
  constexpr int DPL = HD / 4, NCC = HD / 32, NT = HD / 16, PPW = kDecPpw, SPG = kDecPages;
  __shared__ float m_w[4][16], l_w[4][16];
  __shared__ float o_w[4][16][HD + 1];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = lane & 15, grp = lane >> 4;
  const int G = hq / hkv;
  for (int item = blockIdx.x; item < cap * hkv; item += gridDim.x) {
    // the list length and the entry are loaded together (the loop bound
    // keeps the entry index below the list's capacity)
    const int n = *n_items;
    const int4 e0 = *(const int4*)&items[item / hkv].i;
    const int2 e1 = *(const int2*)&items[item / hkv].pl;
    if (item >= n * hkv) break;
    const int i = e0.x, c = e0.y, g = item % hkv;
    // q operand (head `row` of this KV group, zero beyond G): independent of
    // the row descriptor, loaded first
    uint4 qv[NCC];
    {
      const int hh = min(row, G - 1);
      const uint4* qp = (const uint4*)(qb + ((size_t)i * hq + g * G + hh) * HD + DPL * grp);
#pragma unroll
      for (int cc = 0; cc < NCC; ++cc) qv[cc] = qp[cc];
      if (row >= G) {
#pragma unroll
        for (int cc = 0; cc < NCC; ++cc) qv[cc] = make_uint4(0, 0, 0, 0);
      }
    }
    const int kv0 = e0.z, kv1 = e0.w;
    const int pl = e1.x;                                   // prompt positions attended
    const int pc = (pl + 15) >> 4;                         // prompt pages
    const int vcnt = e1.y;                                 // private positions (>= 1)
    const int nch = pc + ((vcnt + 15) >> 4);
    const int ch0 = c * SPG;
    if (ch0 >= nch) continue;
    const int ch1 = min(nch, ch0 + SPG);
    struct Pg { u32x4 k[NCC]; u32x2 v[NT]; int n; };
    Pg pg[PPW];
#pragma unroll
    for (int p = 0; p < PPW; ++p) {
      const int ch = ch0 + wave + 4 * p;
      const int cv = (ch < ch1) ? ch : ch0;                // pages past the split re-read its first
      int n;
      if (cv < pc) n = min(16, pl - 16 * cv);
      else n = min(16, vcnt - 16 * (cv - pc));
      pg[p].n = (ch < ch1) ? n : 0;
      const int blk = (cv < pc) ? kv0 + cv : kv1 + (cv - pc);
      const size_t pgi = ((size_t)layer * n_blocks + blk) * hkv + g;
      const u32x4* kp = (const u32x4*)(kc + (pgi * kBlockTok + row) * HD + DPL * grp);
#pragma unroll
      for (int cc = 0; cc < NCC; ++cc) pg[p].k[cc] = kp[cc];
      const uint16_t* vp = vc + pgi * (size_t)HD * kBlockTok + 4 * grp;
#pragma unroll
      for (int t = 0; t < NT; ++t) pg[p].v[t] = *(const u32x2*)(vp + (size_t)(16 * t + row) * kBlockTok);
    }
    float m_run = -INFINITY, l_run = 0.f;
    f32x4 o[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < PPW; ++p) {
      const int n = pg[p].n;
      if (n == 0) continue;
      f32x4 sc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int cc = 0; cc < NCC; ++cc)
        sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, pg[p].k[cc]),
                                                     __builtin_bit_cast(bf16x8, qv[cc]), sc, 0, 0, 0);
      // lane holds tokens 4*grp + q (q < 4) of head `row`
      float sv[4];
      float mt = -INFINITY;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        sv[q] = (4 * grp + q < n) ? sc[q] * scale : -INFINITY;
        mt = fmaxf(mt, sv[q]);
      }
      mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
      mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
      const float mn = fmaxf(m_run, mt);
      const float alpha = expf(m_run - mn);
      float ps = 0.f;
      uint16_t pb[4], plo[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float pv = expf(sv[q] - mn);
        const uint16_t bb = f32_to_bf16(pv);
        pb[q] = bb;
        plo[q] = f32_to_bf16(pv - bf16_to_f32(bb));
        ps += pv;
      }
      ps += __shfl_xor(ps, 16, 64);
      ps += __shfl_xor(ps, 32, 64);
      l_run = l_run * alpha + ps;
      m_run = mn;
      // rows of O are heads 4*grp + q: fetch their rescale factors
      float al[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) al[q] = __shfl(alpha, 4 * grp + q, 64);
      short4_ pa, pa_lo;
#pragma unroll
      for (int q = 0; q < 4; ++q) { pa[q] = (short)pb[q]; pa_lo[q] = (short)plo[q]; }
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        // positions beyond the page's n valid tokens may hold stale bits: zero them
        short4_ vb;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t w = (q < 2) ? pg[p].v[t].x : pg[p].v[t].y;
          const uint16_t hv = (uint16_t)((q & 1) ? (w >> 16) : (w & 0xFFFF));
          vb[q] = (short)((4 * grp + q < n) ? hv : (uint16_t)0);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) o[t][q] *= al[q];
        o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa, vb, o[t], 0, 0, 0);
        o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa_lo, vb, o[t], 0, 0, 0);
      }
    }
    // merge the 4 waves: lane `row` (grp 0) holds head row's (m, l); O rows are heads 4*grp + q
    if (grp == 0) { m_w[wave][row] = m_run; l_w[wave][row] = l_run; }
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int q = 0; q < 4; ++q) o_w[wave][4 * grp + q][16 * t + row] = o[t][q];
    __syncthreads();
    const int ns = (nch + SPG - 1) / SPG;
    for (int e = threadIdx.x; e < G * HD; e += 256) {
      const int hh = e / HD, dd = e - hh * HD;
      const float mx = fmaxf(fmaxf(m_w[0][hh], m_w[1][hh]), fmaxf(m_w[2][hh], m_w[3][hh]));
      float num = 0.f, den = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float wt = (m_w[w][hh] == -INFINITY) ? 0.f : expf(m_w[w][hh] - mx);
        num += wt * o_w[w][hh][dd];
        den += wt * l_w[w][hh];
      }
      if (ns == 1) {
        out[((size_t)i * hq + g * G + hh) * HD + dd] = f32_to_bf16(num / den);
      } else {
        float* dst = part + ((((size_t)i * hkv + g) * n_splits + c) * kMaxGroup + hh) * (HD + 2);
        dst[dd] = num;
        if (dd == 0) { dst[HD] = mx; dst[HD + 1] = den; }
      }
    }
    __syncthreads();   // LDS is reused by the next item
  }
}

// merge the context splits of every (row, query head) into o (model dtype)
// skip_single: rows with one split were written by the attention kernel.
// One pass over the splits, eight at a time with all their loads in flight,
// rescaling the running (max, numerator, denominator) as it goes.
template <typename T, int HD>
__global__ __launch_bounds__(HD) void k_attn_combine(const int32_t* __restrict__ M_ptr,
    const RowDesc* __restrict__ rows, const float* __restrict__ part, int hq, int hkv,
    int n_splits, int paged_splits, int skip_single, T* __restrict__ out) {
  // paged_splits: pages per context split of the paged (bf16) attention
  // kernels, 0 for the fp32 attention's token splits
  const int M = *M_ptr;
  for (int item = blockIdx.x; item < M * hq; item += gridDim.x) {
    const int i = item / hq, h = item - i * hq;
    const int G = hq / hkv, g = h / G, gh = h - g * G;
    const RowDesc r = rows[i];
    const int ctx = r.pos + 1;
    int ns;
    if (paged_splits) {
      const int pl = min(ctx, r.plen);
      const int nch = ((pl + 15) >> 4) + ((ctx - pl + 15) >> 4);
      ns = (nch + paged_splits - 1) / paged_splits;
    } else {
      ns = (ctx + kAttnSplit - 1) / kAttnSplit;
    }
    if (skip_single && ns == 1) continue;
    const float* base = part + (((size_t)i * hkv + g) * n_splits * kMaxGroup + gh) * (HD + 2);
    const size_t sstride = (size_t)kMaxGroup * (HD + 2);
    float mx = -INFINITY, num = 0.f, den = 0.f;
    for (int c0 = 0; c0 < ns; c0 += 8) {
      float pm[8], pl_[8], po[8];
      float mk[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        // unconditional loads from a clamped split index (see mask01): the
        // surplus entries repeat split ns - 1 of this chunk, which leaves the
        // maximum unchanged, and their weight is masked to zero
        const float* p = base + (size_t)min(c0 + q, ns - 1) * sstride;
        pm[q] = p[HD];
        pl_[q] = p[HD + 1];
        po[q] = p[threadIdx.x];
        mk[q] = mask01(c0 + q < ns);
      }
      float m2 = mx;
#pragma unroll
      for (int q = 0; q < 8; ++q) m2 = fmaxf(m2, pm[q]);
      const float sc = (mx == -INFINITY) ? 0.f : expf(mx - m2);
      num *= sc;
      den *= sc;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float wgt = ((pm[q] == -INFINITY) ? 0.f : expf(pm[q] - m2)) * mk[q];
        num += wgt * po[q];
        den += wgt * pl_[q];
      }
      mx = m2;
    }
    st_f32(out, ((size_t)i * hq + h) * HD + threadIdx.x, num / den);
  }
}

// ---------------------------------------------------------------------------
// sampler: Gumbel-max over the vocabulary with Philox4x32-10 noise
// ---------------------------------------------------------------------------
// (score definition and helpers: see "Gumbel-max sampling helpers")

// top-p helpers: order-preserving key of z (larger z, larger key) and the
// integer weight of z under the row maximum (see the top-p sampler below)
__device__ __forceinline__ uint32_t zkey(float z) {
  uint32_t u = __float_as_uint(z);
  if ((u & 0x7FFFFFFFu) == 0u) u = 0u;   // -0 and +0 are one value
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ uint64_t nucleus_weight(float z, float zmax) {
  return (uint64_t)floor(ldexp(exp((double)z - (double)zmax), 44));
}

__global__ __launch_bounds__(256) void k_sample_partial(const int32_t* __restrict__ M_ptr,
    const int32_t* __restrict__ rid_arr, const int32_t* __restrict__ pos_arr,
    const RowDesc* __restrict__ rows, const float* __restrict__ logits, int V, int by_slot,
    const uint32_t* __restrict__ thr, const CtlParams* __restrict__ cpd, uint64_t seed, int32_t step,
    float temp, float* __restrict__ best, int32_t* __restrict__ bidx) {
  __shared__ float sb[256];
  __shared__ int si[256];
  // persistent over (row, vocabulary chunk) items of the live rows
  const int M = *M_ptr;
  for (int item = blockIdx.x; item < M * kSampleChunks; item += gridDim.x) {
  const int i = item / kSampleChunks, c = item - i * kSampleChunks;
  const int rid = rows ? rows[i].rid : rid_arr[i];
  const int gen = rows ? rows[i].gen : pos_arr[i];
  if (cpd) { seed = cpd->seed; step = cpd->step; temp = cpd->temperature; }
  uint32_t k0, k1;
  sampler_key(seed, step, k0, k1);
  const int nblk = (V + 3) >> 2;
  const int per = (nblk + kSampleChunks - 1) / kSampleChunks;
  const int b0 = c * per, b1 = min(nblk, b0 + per);
  const float* lg = logits + (size_t)(by_slot ? rows[i].slot : i) * V;
  // top-p: only ids whose key reaches the nucleus threshold take part
  const uint32_t kth = thr ? thr[i] : 0u;
  // Pass 1: fast scores (fp32 noise estimate) and their maximum over the
  // chunk.  Pass 2: the exact score (fp64 noise) of every id whose fast score
  // is within the estimate's error bound of that maximum; the chunk's exact
  // winner is always among them (the bound of the fused LM-head sampler).
  float fmx = -INFINITY;
  for (int b = b0 + threadIdx.x; b < b1; b += 256) {
    float z[4];
    bool in[4], any = false;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int v = 4 * b + e;
      z[e] = (v < V) ? ((temp == 1.0f) ? lg[v] : __fdiv_rn(lg[v], temp)) : -INFINITY;
      in[e] = (v < V) && zkey(z[e]) >= kth;
      any |= in[e];
    }
    if (!any) continue;
    U32x4 w = philox4x32_10((uint32_t)rid, (uint32_t)gen, (uint32_t)b, 0u, k0, k1);
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (in[e]) fmx = fmaxf(fmx, __fadd_rn(z[e], gumbel_fast(ws[e])));
  }
  fmx = wave_max(fmx);
  if ((threadIdx.x & 63) == 0) sb[threadIdx.x >> 6] = fmx;
  __syncthreads();
  const float floor_ = gumbel_candidate_floor(fmaxf(fmaxf(sb[0], sb[1]), fmaxf(sb[2], sb[3])));
  __syncthreads();   // sb is rewritten below
  float bs = -INFINITY;
  int bi = 0x7FFFFFFF;
  for (int b = b0 + threadIdx.x; b < b1; b += 256) {
    float z[4];
    bool in[4], any = false;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int v = 4 * b + e;
      z[e] = (v < V) ? ((temp == 1.0f) ? lg[v] : __fdiv_rn(lg[v], temp)) : -INFINITY;
      in[e] = (v < V) && zkey(z[e]) >= kth;
      any |= in[e];
    }
    if (!any) continue;
    U32x4 w = philox4x32_10((uint32_t)rid, (uint32_t)gen, (uint32_t)b, 0u, k0, k1);
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (in[e] && __fadd_rn(z[e], gumbel_fast(ws[e])) >= floor_)
        better(bs, bi, __fadd_rn(z[e], gumbel_exact(ws[e])), 4 * b + e);
  }
  sb[threadIdx.x] = bs;
  si[threadIdx.x] = bi;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) {
      float s2 = sb[threadIdx.x + o];
      int i2 = si[threadIdx.x + o];
      if (s2 > sb[threadIdx.x] || (s2 == sb[threadIdx.x] && i2 < si[threadIdx.x])) {
        sb[threadIdx.x] = s2;
        si[threadIdx.x] = i2;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    best[(size_t)i * kSampleChunks + c] = sb[0];
    bidx[(size_t)i * kSampleChunks + c] = si[0];
  }
  __syncthreads();   // sb/si are reused by the next item
  }
}

// ---------------------------------------------------------------------------
// top-p (nucleus) sampler, top_p < 1 (nucleus sampling, Holtzman et al.),
// over each row's fp32 logits.  Mass is counted in integer weights
// q_v = floor(exp(z_v - z_max) * 2^44), z_v = fp32(logit_v / T), so the cut
// is an exact integer decision whatever the order of the sums: the nucleus
// is {v : z_v >= z*}, with z* the largest z whose upper set holds weight
// >= t = ceil(top_p * Q), Q the total weight; every id tied with the cut is
// kept.  z* comes from a radix descent over the order-preserving bits of z
// (digits of 11, 11 and 10 bits), each digit in two launches:
//   k_topp_hist  (row, chunk) blocks: histogram of the weights of the keys
//                that match the bits decided so far, by the next digit
//                (2048 bins per chunk, integer LDS atomics: exact)
//   k_topp_pick  one block per row: sums the chunk histograms in chunk order
//                and picks the one bin where the weight of the keys above it
//                and in it first reaches t (after the first digit, with the
//                weight above the current range carried per row)
// after k_topp_max has taken the chunk maxima of z.  The Gumbel-max over the
// nucleus is then k_sample_partial with z*'s key as a threshold.
// ---------------------------------------------------------------------------
constexpr int kTopPThreads = 1024;
constexpr int kTopPWaves = kTopPThreads / 64;
static_assert(kTopPBins == 2 * kTopPThreads, "two histogram bins per pick thread");

// z = fp32(logit / T); dividing by 1 is exact, so it is skipped
__device__ __forceinline__ float zval(const float* lg, int v, float temp) {
  return (temp == 1.0f) ? lg[v] : __fdiv_rn(lg[v], temp);
}

// Vocabulary chunk c of a row for the top-p passes: [c*per, min(V, (c+1)*per))
// with per a multiple of 4, so a chunk of a row whose length V is a multiple
// of 4 starts 16-byte aligned.
__device__ __forceinline__ int topp_chunk_len(int V) { return (((V + kTopPChunks - 1) / kTopPChunks) + 3) & ~3; }

// Calls f(v, z) for every id v of [v0, v1) of the row lg, z = fp32(lg[v] / T).
// A row that starts 16-byte aligned and whose length is divisible by 4 is
// read as float4 with kTopPLoads loads of a thread in flight at once (a
// chunk is ~40 floats per thread, so one or two rounds of loads); any other
// row one float at a time.
constexpr int kTopPLoads = 8;
template <typename F>
__device__ __forceinline__ void topp_visit(const float* __restrict__ lg, int V, int v0, int v1, float temp, F f) {
  if ((V & 3) == 0 && (reinterpret_cast<uintptr_t>(lg) & 15) == 0) {
    const float4* l4 = reinterpret_cast<const float4*>(lg);
    const int q0 = v0 >> 2, q1 = v1 >> 2;
    for (int base = q0 + (int)threadIdx.x; base < q1; base += 256 * kTopPLoads) {
      float4 x[kTopPLoads];
#pragma unroll
      for (int u = 0; u < kTopPLoads; ++u) {
        const int qq = base + u * 256;
        if (qq < q1) x[u] = l4[qq];
      }
#pragma unroll
      for (int u = 0; u < kTopPLoads; ++u) {
        const int qq = base + u * 256;
        if (qq < q1) {
          const float e4[4] = {x[u].x, x[u].y, x[u].z, x[u].w};
#pragma unroll
          for (int e = 0; e < 4; ++e) f(4 * qq + e, (temp == 1.0f) ? e4[e] : __fdiv_rn(e4[e], temp));
        }
      }
    }
  } else {
    for (int v = v0 + (int)threadIdx.x; v < v1; v += 256) f(v, zval(lg, v, temp));
  }
}

__global__ __launch_bounds__(256) void k_topp_max(const int32_t* __restrict__ M_ptr,
    const RowDesc* __restrict__ rows, const float* __restrict__ logits, int V, int by_slot,
    const CtlParams* __restrict__ cpd, float temp, float* __restrict__ pmax) {
  __shared__ float red[4];
  if (cpd) temp = cpd->temperature;
  const int M = *M_ptr;
  const int per = topp_chunk_len(V);
  for (int item = blockIdx.x; item < M * kTopPChunks; item += gridDim.x) {
    const int i = item / kTopPChunks, c = item - i * kTopPChunks;
    const float* lg = logits + (size_t)(by_slot ? rows[i].slot : i) * V;
    const int v0 = min(V, c * per), v1 = min(V, v0 + per);
    float zm = -INFINITY;
    topp_visit(lg, V, v0, v1, temp, [&](int, float z) { zm = fmaxf(zm, z); });
    zm = wave_max(zm);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = zm;
    __syncthreads();
    if (threadIdx.x == 0) pmax[item] = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    __syncthreads();   // red is reused by the next item
  }
}

__device__ __forceinline__ float row_zmax(const float* __restrict__ pmax, int i) {
  float zm = pmax[(size_t)i * kTopPChunks];
#pragma unroll
  for (int c = 1; c < kTopPChunks; ++c) zm = fmaxf(zm, pmax[(size_t)i * kTopPChunks + c]);
  return zm;
}

// digit d of the descent: bits 31..21 (d = 0), 20..10 (d = 1), 9..0 (d = 2)
__device__ __forceinline__ int digit_shift(int d) { return d == 0 ? 21 : (d == 1 ? 10 : 0); }

__global__ __launch_bounds__(256) void k_topp_hist(const int32_t* __restrict__ M_ptr,
    const RowDesc* __restrict__ rows, const float* __restrict__ logits, int V, int by_slot,
    const CtlParams* __restrict__ cpd, float temp, const float* __restrict__ pmax, int d,
    const uint32_t* __restrict__ prefix, unsigned long long* __restrict__ hist) {
  __shared__ unsigned long long h[kTopPBins];
  if (cpd) temp = cpd->temperature;
  const int M = *M_ptr;
  const int per = topp_chunk_len(V);
  const int sh = digit_shift(d);
  const uint32_t dmask = (d == 2) ? 1023u : 2047u;
  const int hi = (d == 1) ? 21 : 10;   // the bits decided before digit d (d > 0)
  for (int item = blockIdx.x; item < M * kTopPChunks; item += gridDim.x) {
    const int i = item / kTopPChunks, c = item - i * kTopPChunks;
    const float* lg = logits + (size_t)(by_slot ? rows[i].slot : i) * V;
    const int v0 = min(V, c * per), v1 = min(V, v0 + per);
    const float zm = row_zmax(pmax, i);
    const uint32_t pre = (d > 0) ? prefix[i] : 0u;
    for (int b = threadIdx.x; b < kTopPBins; b += 256) h[b] = 0ull;
    __syncthreads();
    topp_visit(lg, V, v0, v1, temp, [&](int, float z) {
      const uint32_t key = zkey(z);
      if (d == 0 || (key >> hi) == (pre >> hi)) {
        const uint64_t q = nucleus_weight(z, zm);
        if (q) atomicAdd(&h[(key >> sh) & dmask], (unsigned long long)q);
      }
    });
    __syncthreads();
    unsigned long long* out = hist + (size_t)item * kTopPBins;
    for (int b = threadIdx.x; b < kTopPBins; b += 256) out[b] = h[b];
    __syncthreads();   // h is cleared for the next item
  }
}

// Per-row state of the descent: prefix (z*'s key bits decided so far; after
// digit 2, z*'s key), above (weight of keys above the current range), target.
__global__ __launch_bounds__(kTopPThreads) void k_topp_pick(const int32_t* __restrict__ M_ptr,
    const CtlParams* __restrict__ cpd, float top_p, int d, const unsigned long long* __restrict__ hist,
    uint32_t* __restrict__ prefix, unsigned long long* __restrict__ above_arr,
    unsigned long long* __restrict__ target_arr) {
  __shared__ unsigned long long wsum[kTopPWaves];
  __shared__ unsigned long long sel_above, target;
  __shared__ uint32_t sel_digit;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (cpd) top_p = cpd->top_p;
  const int M = *M_ptr;
  const int sh = digit_shift(d);
  for (int i = blockIdx.x; i < M; i += gridDim.x) {
    // the chunk histograms, summed in chunk order
    const unsigned long long* hr = hist + (size_t)i * kTopPChunks * kTopPBins;
    unsigned long long h0 = 0ull, h1 = 0ull;
    for (int c = 0; c < kTopPChunks; ++c) {
      h0 += hr[(size_t)c * kTopPBins + 2 * tid];
      h1 += hr[(size_t)c * kTopPBins + 2 * tid + 1];
    }
    unsigned long long above = 0ull;
    uint32_t pre = 0u;
    if (d == 0) {
      // the first digit's histograms cover every weight: Q and the target
      unsigned long long tot = h0 + h1;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) tot += __shfl_xor(tot, o, 64);
      if (lane == 0) wsum[wave] = tot;
      __syncthreads();
      if (tid == 0) {
        unsigned long long Q = 0ull;
        for (int w = 0; w < kTopPWaves; ++w) Q += wsum[w];
        target = (unsigned long long)ceil((double)top_p * (double)Q);
      }
    } else {
      if (tid == 0) target = target_arr[i];
      above = above_arr[i];
      pre = prefix[i];
    }
    // suffix sums of the histogram: thread t owns bins 2t and 2t+1
    unsigned long long incl = h0 + h1;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const unsigned long long y = __shfl_down(incl, o, 64);
      if (lane + o < 64) incl += y;
    }
    __syncthreads();
    if (lane == 0) wsum[wave] = incl;
    __syncthreads();
    unsigned long long excl = incl - (h0 + h1);
    for (int w = wave + 1; w < kTopPWaves; ++w) excl += wsum[w];
    // the one bin where the upper-set weight first reaches the target
    const unsigned long long t = target;
    const unsigned long long a1 = above + excl, a0 = a1 + h1;
    if (a1 < t && a1 + h1 >= t) { sel_digit = 2 * tid + 1; sel_above = a1; }
    if (a0 < t && a0 + h0 >= t) { sel_digit = 2 * tid; sel_above = a0; }
    __syncthreads();
    if (tid == 0) {
      prefix[i] = pre | (sel_digit << sh);
      above_arr[i] = sel_above;
      if (d == 0) target_arr[i] = t;
    }
    __syncthreads();   // wsum, target and the selection are rewritten for the next row
  }
}

__device__ __forceinline__ int reduce_chunks(const float* best, const int32_t* bidx, int i, int nchunks) {
  float bs = -INFINITY;
  int bi = 0x7FFFFFFF;
  for (int c = 0; c < nchunks; ++c)
    better(bs, bi, best[(size_t)i * nchunks + c], bidx[(size_t)i * nchunks + c]);
  return bi;
}

__device__ __forceinline__ bool forced_eos_fires(uint64_t seed, int32_t step, int rid, int gen,
                                                 uint32_t thr) {
  if (thr == 0u) return false;
  uint32_t k0, k1;
  sampler_key(seed, step, k0, k1);
  U32x4 w = philox4x32_10((uint32_t)rid, (uint32_t)gen, 0u, 1u, k0, k1);
  return w.x < thr;
}

// Final token of each decode row: the best of the row's nchunks partial
// (score, id) winners (chunk c of row i at [c * cstride + i * rstride]),
// forced EOS, teacher forcing, forced length, reward
// hash chain, termination and the per-slot finish flag.  One block per row
// (persistent over the live rows); the (score desc, id asc) order is total,
// so the reduction order does not matter.
__global__ __launch_bounds__(256) void k_sample_final(const Ctl* __restrict__ ctl,
    const RowDesc* __restrict__ rows, const float* __restrict__ best,
    const int32_t* __restrict__ bidx, int nchunks, int cstride, int rstride, const int32_t* __restrict__ forced,
    const int32_t* __restrict__ flen, int model_free, const CtlParams* __restrict__ cpp,
    const double* __restrict__ p, int32_t* __restrict__ out_tok, int32_t* __restrict__ samp_tok,
    int32_t* __restrict__ slot_gen, uint64_t* __restrict__ slot_hash, int32_t* __restrict__ fin,
    int32_t* __restrict__ r_len, int32_t* __restrict__ r_reward) {
  __shared__ float sb[256];
  __shared__ int si[256];
  const int M = ctl->done ? 0 : ctl->M;
  for (int i = blockIdx.x; i < M; i += gridDim.x) {
    float bs = -INFINITY;
    int bi = 0x7FFFFFFF;
    if (!model_free)
      for (int c = threadIdx.x; c < nchunks; c += 256)
        better(bs, bi, best[(size_t)c * cstride + (size_t)i * rstride], bidx[(size_t)c * cstride + (size_t)i * rstride]);
    sb[threadIdx.x] = bs;
    si[threadIdx.x] = bi;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
      if (threadIdx.x < o) {
        float s2 = sb[threadIdx.x];
        int i2 = si[threadIdx.x];
        better(s2, i2, sb[threadIdx.x + o], si[threadIdx.x + o]);
        sb[threadIdx.x] = s2;
        si[threadIdx.x] = i2;
      }
      __syncthreads();
    }
    if (threadIdx.x == 0) {
      const CtlParams cp = *cpp;
      const int32_t* fl = cp.has_flen ? flen : nullptr;
      const RowDesc r = rows[i];
      const int rid = r.rid, gen = r.gen, s = r.slot;
      int samp;
      if (model_free) {
        samp = forced[(size_t)rid * cp.max_new + gen];
      } else {
        samp = si[0];
        if (cp.eos >= 0 && forced_eos_fires(cp.seed, cp.step, rid, gen, cp.forced_eos)) samp = cp.eos;
      }
      int tok = forced ? forced[(size_t)rid * cp.max_new + gen] : samp;
      bool done = false;
      if (fl && gen + 1 == fl[rid]) {
        if (cp.eos >= 0) tok = cp.eos;
        done = true;
      }
      if (cp.eos >= 0 && tok == cp.eos) done = true;
      if (gen + 1 == cp.max_new) done = true;
      out_tok[(size_t)rid * cp.max_new + gen] = tok;
      samp_tok[(size_t)rid * cp.max_new + gen] = samp;
      uint64_t hsh = mix64(slot_hash[s] ^ (uint64_t)(uint32_t)(tok + 1));
      slot_hash[s] = hsh;
      slot_gen[s] = gen + 1;
      if (done) {
        r_len[rid] = gen + 1;
        double u = (double)(hsh >> 11) * 0x1p-53;
        r_reward[rid] = (u < p[r.uid]) ? 1 : 0;
        fin[s] = 1;
      }
    }
    __syncthreads();   // sb/si are reused by the next row
  }
}

// stand-alone sampler for given logits (parity entry point)
__global__ void k_sample_rows_final(int n_rows, const int32_t* __restrict__ rid,
    const int32_t* __restrict__ pos, const float* __restrict__ best,
    const int32_t* __restrict__ bidx, int nchunks, uint64_t seed, int32_t step, int eos, uint32_t feos,
    int32_t* __restrict__ tok) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_rows) return;
  int t = reduce_chunks(best, bidx, i, nchunks);
  if (eos >= 0 && forced_eos_fires(seed, step, rid[i], pos[i], feos)) t = eos;
  tok[i] = t;
}

__global__ void k_copy_logits(const Ctl* __restrict__ ctl, const RowDesc* __restrict__ rows,
                              const float* __restrict__ ws, int V, float* __restrict__ dst) {
  int M = ctl->done ? 0 : ctl->M;
  int i = blockIdx.y;
  if (i >= M) return;
  int s = rows[i].slot;
  for (int v = blockIdx.x * 256 + threadIdx.x; v < V; v += gridDim.x * 256)
    dst[(size_t)s * V + v] = ws[(size_t)i * V + v];
}


// ---------------------------------------------------------------------------
// host launchers
// ---------------------------------------------------------------------------
// Kernel launch on a context's stream.  While a per-kernel profile record is
// open (prof_begin), the launch goes through hipExtLaunchKernelGGL with the
// record's event pair, so the dispatch itself stamps the kernel's start and
// end: the elapsed time is the kernel's own duration, as in a kernel trace.
template <typename F, typename... Args>
static void launch_k(sara_ctx* c, hipStream_t st, F kernel, dim3 grid, dim3 block, uint32_t shm, Args... args) {
  const int p = c->prof_pending;
  if (p >= 0) {
    c->prof_pending = -1;
    c->prof_last = p;
    hipExtLaunchKernelGGL(kernel, grid, block, shm, st, c->prof_events[p], c->prof_events[p + 1], 0u, args...);
  } else {
    hipLaunchKernelGGL(kernel, grid, block, shm, st, args...);
  }
}
static int gemm(sara_ctx* c, const void* X, const void* W, const int32_t* M_ptr, int M_cap,
                int N, int K, int& splits_out, int max_splits = 1 << 30, bool oproj = false) {
  int64_t stride = (int64_t)M_cap * N;
  if (c->md.dtype == SARA_BF16) {
    // weight rows per block: 128 (two 16-row tiles per wave) for the LM head
    // and long-K GEMMs, 64 otherwise; split K until the grid has about one
    // block per CU (each split keeps >= 4 k chunks): wide GEMMs need no
    // split, narrow ones trade fp32 partial traffic for occupancy
    constexpr int MT = 8;
    const bool wide = N >= 65536;
    const bool two = wide || (K >= 4096 && c->in_prefill);
    const int rows_per_block = two ? 128 : 64;
    int tiles_n = (N + rows_per_block - 1) / rows_per_block;
    // one z block per m-block of the capacity; in decode the live row count
    // is read on the device, and z blocks past it exit at once (blocks are
    // dispatched z-major, so the live m-blocks start first)
    int zb = (M_cap + 16 * MT - 1) / (16 * MT);
    // blocks without a split: weight tiles x m-blocks in prefill (the chunk's
    // row count is known), weight tiles alone in decode (live rows are few
    // and known only on the device)
    const int64_t blocks = (int64_t)tiles_n * (c->in_prefill ? zb : 1);
    int want = (blocks >= 256) ? 1 : (int)((256 + blocks - 1) / blocks);
    // 64-wide k chunks: four pipeline slots of X + W fit in registers for NT <= 2
    const int KC = 64;
    int chunks = K / KC;
    int splits = std::min(want, std::max(1, chunks / 4));
    if (!c->in_prefill) {
      // decode: an even division of the k chunks keeps the splits balanced
      // (the last split of an uneven one runs alone); take the largest even
      // count in [6, kMaxSplitsDec] with >= 4 chunks per split, else the
      // occupancy target.  Consumers sum at most kMaxSplitsDec partials in
      // one batch of loads.
      for (int s = kMaxSplitsDec; s >= 6; --s)
        if (s <= want && chunks % s == 0 && chunks / s >= 4) { splits = s; break; }
      splits = std::min(splits, kMaxSplitsDec);
    }
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    int kps = ((chunks + splits - 1) / splits) * KC;
    splits = (K + kps - 1) / kps;
    if ((int64_t)splits * stride > c->ws_floats) { splits = 1; kps = K; }
    dim3 grid(tiles_n, splits, zb);
    const uint16_t* Xh = (const uint16_t*)X;
    const uint16_t* Wh = (const uint16_t*)W;
#define SARA_GEMM(NT_, KC_, PF_) \
    launch_k(c, c->stream, (k_gemm_bf16_lds<NT_, MT, KC_, 0, PF_>), grid, dim3(256), 0, Xh, Wh, \
                       (void*)c->ws, M_ptr, N, K, kps, stride, SampleArgs{})
    if (c->in_prefill) {
      if (two) SARA_GEMM(2, 64, 1);
      else SARA_GEMM(1, 64, 1);
    } else if (two) {
      SARA_GEMM(2, 64, 0);
    } else if (oproj) {
      SARA_GEMM(1, 64, 2);
    } else {
      SARA_GEMM(1, 64, 0);
    }
#undef SARA_GEMM
    splits_out = splits;
  } else {
    int tiles_n = (N + 15) / 16, zb = (M_cap + 15) / 16;
    int want = (tiles_n * zb >= 256) ? 1 : (256 + tiles_n * zb - 1) / (tiles_n * zb);
    int chunks = K / 32;
    int splits = want < chunks ? want : chunks;
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    int kps = ((chunks + splits - 1) / splits) * 32;
    splits = (K + kps - 1) / kps;
    if ((int64_t)splits * stride > c->ws_floats) { splits = 1; kps = K; }
    dim3 grid(tiles_n, splits, zb);
    launch_k(c, c->stream, k_gemm_f32, grid, dim3(256), 0, (const float*)X, (const float*)W,
                       c->ws, M_ptr, N, K, kps, stride);
    splits_out = splits;
  }
  return SARA_OK;
}

#define PROF_B(c) do { if ((c)->prof_active) prof_begin(c); } while (0)
#define PROF_E(c, cls, N, K) do { if ((c)->prof_active) prof_end((c), (cls), (N), (K)); } while (0)

// gate|up GEMM with the SwiGLU epilogue (bf16 models; W_gu rows interleaved
// per 16-row tile at init), writing a = silu(g) * u to c->xa as [m][ffn]
static void gemm_swiglu(sara_ctx* c, const void* X, const void* W, const int32_t* M_ptr, int M_cap) {
  constexpr int MT = 8;
  const int N = 2 * c->ffn, K = c->d;
  dim3 grid((N + 127) / 128, 1, (M_cap + 16 * MT - 1) / (16 * MT));
  if (c->in_prefill)
    launch_k(c, c->stream, (k_gemm_bf16_lds<2, MT, 64, 1, 1>), grid, dim3(256), 0, (const uint16_t*)X,
                       (const uint16_t*)W, (void*)c->xa, M_ptr, N, K, K, (int64_t)0, SampleArgs{});
  else
    launch_k(c, c->stream, (k_gemm_bf16_lds<2, MT, 64, 1, 0>), grid, dim3(256), 0, (const uint16_t*)X,
                       (const uint16_t*)W, (void*)c->xa, M_ptr, N, K, K, (int64_t)0, SampleArgs{});
}

// z blocks over which the q|k|v kernel shares out a small batch's 16-row
// tiles: as many per weight tile as keep every working block resident at
// once (blocks per CU x CUs / weight tiles), computed once per context
template <typename F>
static int qkv_spread(sara_ctx* c, F kernel) {
  if (c->qkv_spread == 0) {
    int per_cu = 0, dev = 0, n_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, 256, 0) != hipSuccess ||
        hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      per_cu = 1, n_cu = 256;
    c->qkv_spread = std::max(1, std::max(1, per_cu) * std::max(1, n_cu) / std::max(1, c->nqkv / 16));
  }
  return c->qkv_spread;
}

// persistent attention grid: enough blocks for two per CU, never more than items
static int attn_grid(sara_ctx* c, int M_cap) {
  int items = M_cap * c->hkv * c->attn_splits_max;
  return std::max(1, std::min(items, 1024));
}

// h += split-K sum of ws; x = RMSNorm(h) * w
template <typename T>
static void residual_norm(sara_ctx* c, const int32_t* M_ptr, int M_cap, int sp, const float* w, int x_tiled = 0) {
  const int d = c->d, vpt = (d + 255) / 256;
  const dim3 grid(std::min(M_cap, 1024));
  const int64_t stride = (int64_t)M_cap * d;
  T* x = (T*)c->x;
  if (sizeof(T) == 2 && !c->in_prefill && sp <= kMaxSplitsDec && d % 4 == 0 && d / 4 <= 1024) {
    launch_k(c, c->stream, k_residual_norm_f4, grid, dim3((d / 4 + 63) / 64 * 64), 0, M_ptr, c->ws, sp, stride,
             d, c->h, w, c->md.rms_eps, (uint16_t*)c->x, x_tiled);
    return;
  }
#define SARA_RN(V) launch_k(c, c->stream, (k_residual_norm_v<T, V>), grid, dim3(256), 0, M_ptr, c->ws, \
                                      sp, stride, d, c->h, w, c->md.rms_eps, x, x_tiled)
  switch (sp <= kMaxSplitsDec ? vpt : 0) {
    case 1: SARA_RN(1); break;
    case 2: SARA_RN(2); break;
    case 3: SARA_RN(3); break;
    case 4: SARA_RN(4); break;
    case 5: case 6: SARA_RN(6); break;
    case 7: case 8: SARA_RN(8); break;
    default:
      launch_k(c, c->stream, k_residual_norm<T>, dim3(std::min(M_cap, 256)), dim3(1024), 0, M_ptr,
                         c->ws, sp, stride, d, c->h, w, c->md.rms_eps, x, x_tiled);
  }
#undef SARA_RN
}

template <typename T, int HD>
static void layers_T(sara_ctx* c, const int32_t* M_ptr, int M_cap, bool final_norm_out) {
  hipStream_t st = c->stream;
  const int d = c->d;
  const int64_t stride_qkv = (int64_t)M_cap * c->nqkv;
  T* x = (T*)c->x;
  for (int l = 0; l < c->L; ++l) {
    int sp = 1;
    const bool mfma_attn = (c->md.dtype == SARA_BF16);
    if (mfma_attn && !c->in_prefill) {
      // decode: q|k|v projection with the RoPE / KV-append epilogue, the
      // paged attention, then the merge of rows with several context splits
      PROF_B(c);
#define SARA_QKV(KS_) \
      launch_k(c, st, (k_qkv_rope<HD, KS_>), dim3(c->nqkv / 16, 1, (M_cap + 127) / 128), dim3(256), 0, \
               (const uint16_t*)x, \
                         (const uint16_t*)c->w_qkv[l], M_ptr, d, c->rows, c->row_rope, c->hq, c->hkv, l, \
                         c->n_blocks, (uint16_t*)c->qbuf, (uint16_t*)c->kc, (uint16_t*)c->vc, \
                         qkv_spread(c, k_qkv_rope<HD, KS_>))
      switch (d / 128) {
        case 4: SARA_QKV(4); break;
        case 8: SARA_QKV(8); break;
        case 12: SARA_QKV(12); break;
        case 16: SARA_QKV(16); break;
        case 24: SARA_QKV(24); break;
        default: SARA_QKV(32); break;
      }
#undef SARA_QKV
      PROF_E(c, kPQkvRope, c->nqkv, d);
      PROF_B(c);
      if (c->attn_dec_grid == 0) {
        // blocks resident at once: every item of a list that short runs in one round
        int per_cu = 0, dev = 0, n_cu = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_attn_dec<HD>, 256, 0) != hipSuccess ||
            hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
          per_cu = 2, n_cu = 256;
        c->attn_dec_grid = std::max(1, per_cu) * std::max(1, n_cu);
      }
      const int cap = M_cap * c->dec_splits_max;
      const int dg = (int)std::min<int64_t>((int64_t)cap * c->hkv, c->attn_dec_grid);
      launch_k(c, st, (k_attn_dec<HD>), dim3(dg), dim3(256), 0, (const AttnItem*)c->attn_items,
                         (const int32_t*)c->attn_nitems, cap, (const uint16_t*)c->kc,
                         (const uint16_t*)c->vc, l, c->n_blocks, c->hq, c->hkv, c->dec_splits_max,
                         1.0f / sqrtf((float)HD), (const uint16_t*)c->qbuf, c->attn_part, (uint16_t*)x);
      PROF_E(c, kPAttn, 0, 0);
      PROF_B(c);
      launch_k(c, st, (k_attn_combine<T, HD>), dim3(1024), dim3(HD), 0, M_ptr, c->rows,
                         c->attn_part, c->hq, c->hkv, c->dec_splits_max, kDecPages, 1, x);
      PROF_E(c, kPCombine, 0, 0);
    } else {
    PROF_B(c);
    gemm(c, x, c->w_qkv[l], M_ptr, M_cap, c->nqkv, d, sp);
    PROF_E(c, kPGemmN1, c->nqkv, d);
    PROF_B(c);
    launch_k(c, st, k_qkv_epilogue<T>, dim3(2048), dim3(c->hd / 2), 0, M_ptr,
                       c->rows, c->ws, sp,
                       stride_qkv, c->rope, c->hq, c->hkv, c->hd, l, c->n_blocks, c->btab, c->MAXB,
                       c->PB, (T*)c->qbuf, (T*)c->kc, (T*)c->vc, mfma_attn ? 1 : 0);
    PROF_E(c, kPQkv, c->nqkv, 0);
    PROF_B(c);
    if (mfma_attn)
      launch_k(c, st, (k_attn_mfma<HD>), dim3(attn_grid(c, M_cap)), dim3(256), 0,
                         M_ptr, c->rows, (const uint16_t*)c->qbuf, (const uint16_t*)c->kc,
                         (const uint16_t*)c->vc, c->btab, c->MAXB, c->PB, l, c->n_blocks, c->hq, c->hkv,
                         c->attn_splits_max, 1.0f / sqrtf((float)HD), c->attn_part);
    else
      launch_k(c, st, (k_attention<T, HD>), dim3(M_cap, c->hkv, c->attn_splits_max), dim3(256), 0,
                         M_ptr, c->rows, (const T*)c->qbuf, (const T*)c->kc, (const T*)c->vc, c->btab,
                         c->MAXB, c->PB, l, c->n_blocks, c->hq, c->hkv, c->attn_splits_max,
                         1.0f / sqrtf((float)HD), c->attn_part);
    PROF_E(c, kPAttn, 0, 0);
    PROF_B(c);
    launch_k(c, st, (k_attn_combine<T, HD>), dim3(1024), dim3(HD), 0, M_ptr, c->rows,
                       c->attn_part, c->hq, c->hkv, c->attn_splits_max, mfma_attn ? kAttnChunks : 0, 0, x);
    PROF_E(c, kPCombine, 0, 0);
    }
    PROF_B(c);
    gemm(c, x, c->w_o[l], M_ptr, M_cap, d, c->qdim, sp, 1 << 30, true);
    PROF_E(c, (c->md.dtype == SARA_BF16 && !c->in_prefill) ? kPGemmO1 : kPGemmN1, d, c->qdim);
    PROF_B(c);
    residual_norm<T>(c, M_ptr, M_cap, sp, c->norms + (size_t)(2 * l + 1) * d);
    PROF_E(c, kPResNorm, d, 0);
    if (c->md.dtype == SARA_BF16) {
      PROF_B(c);
      gemm_swiglu(c, x, c->w_gu[l], M_ptr, M_cap);
      PROF_E(c, kPGemmGU, 2 * c->ffn, d);
      PROF_B(c);
      gemm(c, c->xa, c->w_d[l], M_ptr, M_cap, d, c->ffn, sp);
      PROF_E(c, kPGemmN1, d, c->ffn);
    } else {
      PROF_B(c);
      gemm(c, x, c->w_gu[l], M_ptr, M_cap, 2 * c->ffn, d, sp);
      PROF_E(c, kPGemmN1, 2 * c->ffn, d);
      PROF_B(c);
      launch_k(c, st, k_swiglu<T>, dim3(1024), dim3(256), 0, M_ptr, c->ws,
                         sp, (int64_t)M_cap * 2 * c->ffn, c->ffn, x);
      PROF_E(c, kPSwiglu, c->ffn, 0);
      PROF_B(c);
      gemm(c, x, c->w_d[l], M_ptr, M_cap, d, c->ffn, sp);
      PROF_E(c, kPGemmN1, d, c->ffn);
    }
    const float* nw = (l + 1 < c->L) ? c->norms + (size_t)(2 * (l + 1)) * d
                                     : c->norms + (size_t)(2 * c->L) * d;
    // the last layer's norm output is only needed when logits follow
    if (l + 1 < c->L || final_norm_out) {
      PROF_B(c);
      // in bf16 decode the next layer's q|k|v kernel reads fragment-major rows
      residual_norm<T>(c, M_ptr, M_cap, sp, nw,
                       (c->md.dtype == SARA_BF16 && !c->in_prefill && l + 1 < c->L) ? 1 : 0);
      PROF_E(c, kPResNorm, d, 0);
    }
  }
}

template <typename T>
static void layers(sara_ctx* c, const int32_t* M_ptr, int M_cap, bool final_norm_out) {
  if (c->hd == 128) layers_T<T, 128>(c, M_ptr, M_cap, final_norm_out);
  else layers_T<T, 64>(c, M_ptr, M_cap, final_norm_out);
}

int launch_prefill(sara_ctx* c) {
  hipStream_t st = c->stream;
  c->in_prefill = true;
  // prefix sums of (P - 1): prompt-token rows of the pool, chunked
  std::vector<int64_t> pre(c->U + 1, 0);
  for (int u = 0; u < c->U; ++u) pre[u + 1] = pre[u] + (c->h_off[u + 1] - c->h_off[u] - 1);
  int64_t rows_total = pre[c->U];
  for (int64_t r0 = 0; r0 < rows_total; r0 += c->prefill_rows) {
    int n = (int)((rows_total - r0 < c->prefill_rows) ? rows_total - r0 : c->prefill_rows);
    launch_k(c, st, k_prefill_rows, dim3((n + 255) / 256), dim3(256), 0, c->pre, c->U, (int)r0,
                       n, c->tok, c->off, c->S, c->rows, c->rows_M, c->PB);
    if (c->md.dtype == SARA_BF16) {
      launch_k(c, st, k_embed_norm<uint16_t>, dim3(n), dim3(256), 0, c->rows_M, c->rows,
                         (const uint16_t*)c->embed, c->norms, c->d, c->md.rms_eps, c->h,
                         (uint16_t*)c->x);
      layers<uint16_t>(c, c->rows_M, n, false);
    } else {
      launch_k(c, st, k_embed_norm<float>, dim3(n), dim3(256), 0, c->rows_M, c->rows,
                         (const float*)c->embed, c->norms, c->d, c->md.rms_eps, c->h, (float*)c->x);
      layers<float>(c, c->rows_M, n, false);
    }
  }
  c->in_prefill = false;
  return SARA_OK;
}

// Top-p passes over the live rows' logits (lg: [slot][V] when by_slot, else
// [row][V]) -> z*'s key per row, then the Gumbel-max over the nucleus by
// k_sample_partial with that threshold: winners [row][kSampleChunks].
static void launch_topp_decode(sara_ctx* c, hipStream_t st, const float* lg, int by_slot) {
  const int S = c->S;
  const CtlParams* cp = (const CtlParams*)c->cp_dev;
  const int32_t* Mp = c->rows_M;
  const RowDesc* rw = c->rows;
  const int g = std::min(S * kTopPChunks, 2048);
  PROF_B(c);
  launch_k(c, st, k_topp_max, dim3(g), dim3(256), 0, Mp, rw, lg, c->V, by_slot, cp, 1.0f, c->topp_max);
  PROF_E(c, kPToppMax, c->V, 0);
  for (int d = 0; d < 3; ++d) {
    PROF_B(c);
    launch_k(c, st, k_topp_hist, dim3(g), dim3(256), 0, Mp, rw, lg, c->V, by_slot, cp, 1.0f,
             (const float*)c->topp_max, d, (const uint32_t*)c->topp_thr, c->topp_hist);
    PROF_E(c, kPToppHist, c->V, 0);
    PROF_B(c);
    launch_k(c, st, k_topp_pick, dim3(std::min(S, 1024)), dim3(kTopPThreads), 0, Mp, cp, 1.0f, d,
             (const unsigned long long*)c->topp_hist, c->topp_thr, c->topp_above, c->topp_target);
    PROF_E(c, kPToppSel, 0, 0);
  }
  PROF_B(c);
  launch_k(c, st, k_sample_partial, dim3(std::min(S * kSampleChunks, 2048)), dim3(256), 0, Mp,
           (const int32_t*)nullptr, (const int32_t*)nullptr, rw, lg, c->V, by_slot, (const uint32_t*)c->topp_thr, cp,
           (uint64_t)0, 0, 1.0f, c->samp_best, c->samp_idx);
  PROF_E(c, kPSampleP, c->V, 0);
}

int launch_decode(sara_ctx* c, const int32_t* forced, float* logits, int model_free) {
  hipStream_t st = c->stream;
  const int S = c->S;
  PROF_B(c);
  const int eg = std::min(S, 512);
  if (c->md.dtype == SARA_BF16)
    launch_k(c, st, k_decode_embed<uint16_t>, dim3(eg), dim3(256), 0, c->ctl, c->active, c->slot_uid,
                       c->slot_j, c->slot_gen, c->tok, c->off, c->out_tok, c->k, c->ad.max_new, c->rows,
                       c->rows_M, model_free ? 0 : 1, (const uint16_t*)c->embed, c->norms, c->d,
                       c->md.rms_eps, c->h, (uint16_t*)c->x, c->U, c->PB, c->SB, c->rope, c->hd / 2,
                       c->row_rope, 1, model_free ? (AttnItem*)nullptr : c->attn_items, c->attn_nitems,
                       kDecPages);
  else
    launch_k(c, st, k_decode_embed<float>, dim3(eg), dim3(256), 0, c->ctl, c->active, c->slot_uid,
                       c->slot_j, c->slot_gen, c->tok, c->off, c->out_tok, c->k, c->ad.max_new, c->rows,
                       c->rows_M, model_free ? 0 : 1, (const float*)c->embed, c->norms, c->d,
                       c->md.rms_eps, c->h, (float*)c->x, c->U, c->PB, c->SB, c->rope, c->hd / 2,
                       c->row_rope, 0, (AttnItem*)nullptr, c->attn_nitems, kDecPages);
  PROF_E(c, kPEmbed, c->d, 0);
  int nchunks = kSampleChunks;
  if (!model_free) {
    if (c->md.dtype == SARA_BF16) {
      layers<uint16_t>(c, c->rows_M, S, true);
      // LM head with the Gumbel-max sampling epilogue: per (row, 128-id block)
      // exact winners, reduced by k_sample_final
      const int nb = (c->V + 127) / 128;
      nchunks = nb;
      // top-p < 1: the GEMM also writes the logits ([slot][V]) for the
      // nucleus sampler, whose winner replaces the epilogue's
      float* lg_out = (c->topp && !logits) ? c->topp_logits : logits;
      PROF_B(c);
      launch_k(c, st, (k_gemm_bf16_lds<2, 8, 64, 2, 0>), dim3(nb, 1, (S + 127) / 128), dim3(256), 0,
                         (const uint16_t*)c->x, (const uint16_t*)c->lm_head, (void*)nullptr, c->rows_M, c->V,
                         c->d, c->d, (int64_t)0,
                         SampleArgs{c->rows, (const CtlParams*)c->cp_dev, lg_out, c->samp_best, c->samp_idx, S});
      PROF_E(c, kPGemmLM, c->V, c->d);
      if (c->topp) {
        launch_topp_decode(c, st, lg_out, 1);
        nchunks = kSampleChunks;
      }
    } else {
      layers<float>(c, c->rows_M, S, true);
      int sp;
      // one K split: ws then holds the logits [M][V] directly
      PROF_B(c);
      gemm(c, c->x, c->lm_head, c->rows_M, S, c->V, c->d, sp, 1);
      PROF_E(c, kPGemmLM, c->V, c->d);
      if (c->topp) {
        launch_topp_decode(c, st, c->ws, 0);
      } else {
        PROF_B(c);
        launch_k(c, st, k_sample_partial, dim3(std::min(S * kSampleChunks, 2048)), dim3(256), 0,
                           c->rows_M, (const int32_t*)nullptr, (const int32_t*)nullptr, c->rows, c->ws, c->V, 0,
                           (const uint32_t*)nullptr, (const CtlParams*)c->cp_dev, (uint64_t)0, 0, 1.0f,
                           c->samp_best, c->samp_idx);
        PROF_E(c, kPSampleP, c->V, 0);
      }
      if (logits) {
        PROF_B(c);
        launch_k(c, st, k_copy_logits, dim3(64, S), dim3(256), 0, c->ctl, c->rows, c->ws, c->V,
                           logits);
        PROF_E(c, kPCopy, c->V, 0);
      }
    }
  }
  PROF_B(c);
  // chunk winners: [row][kSampleChunks] from k_sample_partial (also after
  // the top-p passes), [chunk][S] from the fused LM head
  const bool fused = !model_free && c->md.dtype == SARA_BF16 && !c->topp;
  launch_k(c, st, k_sample_final, dim3(std::min(S, 1024)), dim3(256), 0, c->ctl, c->rows,
                     c->samp_best, c->samp_idx, nchunks, fused ? S : 1, fused ? 1 : nchunks, forced, c->flen,
                     model_free,
                     (const CtlParams*)c->cp_dev, c->p, c->out_tok, c->samp_tok, c->slot_gen, c->slot_hash, c->fin,
                     c->r_len, c->r_reward);
  PROF_E(c, kPSampleF, 0, 0);
  return SARA_OK;
}

// Buffers of the stand-alone sampler: the live row count, per-row chunk
// winners and, for top-p < 1, the descent's chunk maxima, histograms and
// per-row state.  Every kernel below writes a buffer before reading it, so
// the contents left by an earlier call never matter.
struct SampleBufs {
  int32_t* mdev;
  float* best;
  int32_t* bidx;
  float* pmax;
  unsigned long long* hist;
  unsigned long long* state;   // per row: above, target
  uint32_t* thr;
};

__global__ void k_set_count(int32_t* __restrict__ dst, int n) {
  if (threadIdx.x == 0) dst[0] = n;
}

static void enqueue_sample_rows(const SampleBufs& b, const float* logits, int n_rows, int V, const int32_t* rid,
                                const int32_t* pos, uint64_t seed, int step, float temp, float top_p, int eos,
                                uint32_t feos, int32_t* tok, hipStream_t st) {
  hipLaunchKernelGGL(k_set_count, dim3(1), dim3(64), 0, st, b.mdev, n_rows);
  const bool topp = top_p < 1.0f;
  if (topp) {
    const int g = std::min(n_rows * kTopPChunks, 2048);
    hipLaunchKernelGGL(k_topp_max, dim3(g), dim3(256), 0, st, (const int32_t*)b.mdev, (const RowDesc*)nullptr,
                       logits, V, 0, (const CtlParams*)nullptr, temp, b.pmax);
    for (int d = 0; d < 3; ++d) {
      hipLaunchKernelGGL(k_topp_hist, dim3(g), dim3(256), 0, st, (const int32_t*)b.mdev, (const RowDesc*)nullptr,
                         logits, V, 0, (const CtlParams*)nullptr, temp, (const float*)b.pmax, d,
                         (const uint32_t*)b.thr, b.hist);
      hipLaunchKernelGGL(k_topp_pick, dim3(std::min(n_rows, 1024)), dim3(kTopPThreads), 0, st,
                         (const int32_t*)b.mdev, (const CtlParams*)nullptr, top_p, d,
                         (const unsigned long long*)b.hist, b.thr, b.state, b.state + n_rows);
    }
  }
  hipLaunchKernelGGL(k_sample_partial, dim3(std::min(n_rows * kSampleChunks, 2048)), dim3(256), 0, st,
                     (const int32_t*)b.mdev, rid, pos, (const RowDesc*)nullptr, logits, V, 0,
                     topp ? (const uint32_t*)b.thr : (const uint32_t*)nullptr, (const CtlParams*)nullptr, seed,
                     step, temp, b.best, b.bidx);
  hipLaunchKernelGGL(k_sample_rows_final, dim3((n_rows + 255) / 256), dim3(256), 0, st, n_rows, rid,
                     pos, b.best, b.bidx, kSampleChunks, seed, step, eos, feos, tok);
}

int launch_sample_rows(const float* logits, int n_rows, int V, const int32_t* rid,
                       const int32_t* pos, uint64_t seed, int step, float temp, float top_p, int eos,
                       uint32_t feos, int32_t* tok, hipStream_t st) {
  SampleBufs b{};
  std::vector<void*> owned;
  auto get = [&](void** p, size_t bytes) -> hipError_t {
    hipError_t e = hipMallocAsync(p, bytes, st);
    if (e == hipSuccess) owned.push_back(*p);
    return e;
  };
  auto release = [&]() {
    for (void* q : owned) (void)hipFreeAsync(q, st);
  };
  const bool topp = top_p < 1.0f;
  hipError_t e = get((void**)&b.mdev, sizeof(int32_t));
  if (e == hipSuccess) e = get((void**)&b.best, sizeof(float) * (size_t)n_rows * kSampleChunks);
  if (e == hipSuccess) e = get((void**)&b.bidx, sizeof(int32_t) * (size_t)n_rows * kSampleChunks);
  if (e == hipSuccess && topp) e = get((void**)&b.pmax, sizeof(float) * (size_t)n_rows * kTopPChunks);
  if (e == hipSuccess && topp)
    e = get((void**)&b.hist, sizeof(unsigned long long) * (size_t)n_rows * kTopPChunks * kTopPBins);
  if (e == hipSuccess && topp) e = get((void**)&b.state, sizeof(unsigned long long) * 2 * (size_t)n_rows);
  if (e == hipSuccess && topp) e = get((void**)&b.thr, sizeof(uint32_t) * (size_t)n_rows);
  if (e != hipSuccess) {
    release();
    return hip_fail(e, "hipMallocAsync");
  }
  enqueue_sample_rows(b, logits, n_rows, V, rid, pos, seed, step, temp, top_p, eos, feos, tok, st);
  e = hipGetLastError();
  release();
  if (e != hipSuccess) return hip_fail(e, "sample_rows launch");
  e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e, "sample_rows");
  return SARA_OK;
}

// ---------------------------------------------------------------------------
// The stand-alone sampler without allocation: its buffers live in one static
// device array per GPU (this file's `scratch`, sized for kNoAllocMaxRows rows
// at top_p = 1 and kNoAllocMaxToppRows rows with the top-p passes).  Host code
// never passes the array's name to a kernel: the address each device gives
// for it is looked up once per device and kept.
// ---------------------------------------------------------------------------
namespace {
constexpr size_t kAlign = 256;
constexpr size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
constexpr size_t kOffCount = 0;
constexpr size_t kOffBest = kAlign;
constexpr size_t kOffBidx = kOffBest + align_up(sizeof(float) * (size_t)kNoAllocMaxRows * kSampleChunks);
constexpr size_t kOffPmax = kOffBidx + align_up(sizeof(int32_t) * (size_t)kNoAllocMaxRows * kSampleChunks);
constexpr size_t kOffHist = kOffPmax + align_up(sizeof(float) * (size_t)kNoAllocMaxToppRows * kTopPChunks);
constexpr size_t kOffState =
    kOffHist + align_up(sizeof(unsigned long long) * (size_t)kNoAllocMaxToppRows * kTopPChunks * kTopPBins);
constexpr size_t kOffThr = kOffState + align_up(sizeof(unsigned long long) * 2 * (size_t)kNoAllocMaxToppRows);
constexpr size_t kScratchBytes = kOffThr + align_up(sizeof(uint32_t) * (size_t)kNoAllocMaxToppRows);
static_assert(kScratchBytes == kNoAllocScratchBytes, "scratch layout and its stated size disagree");
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxScratchDevices] = {};
}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on the current device, looked up on the first
// call on that device.
static int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxScratchDevices) return hip_fail(hipErrorInvalidDevice, "device index");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "hipGetSymbolAddress");
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return SARA_OK;
}

int launch_sample_rows_noalloc(const float* logits, int n_rows, int V, const int32_t* rid, const int32_t* pos,
                               uint64_t seed, int step, float temp, float top_p, int eos, uint32_t feos,
                               int32_t* tok, hipStream_t st) {
  void* base = nullptr;
  int rc = scratch_address(&base);
  if (rc != SARA_OK) return rc;
  unsigned char* b8 = (unsigned char*)base;
  SampleBufs b{};
  b.mdev = (int32_t*)(b8 + kOffCount);
  b.best = (float*)(b8 + kOffBest);
  b.bidx = (int32_t*)(b8 + kOffBidx);
  b.pmax = (float*)(b8 + kOffPmax);
  b.hist = (unsigned long long*)(b8 + kOffHist);
  b.state = (unsigned long long*)(b8 + kOffState);
  b.thr = (uint32_t*)(b8 + kOffThr);
  enqueue_sample_rows(b, logits, n_rows, V, rid, pos, seed, step, temp, top_p, eos, feos, tok, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "sample_rows_noalloc launch");
  return SARA_OK;
}

// Largest |gumbel_fast - gumbel_exact| over all 2^24 noise inputs (the
// 24-bit mantissa source of u); non-negative floats order like their bits.
__global__ __launch_bounds__(256) void k_gumbel_check(uint32_t* out) {
  float e = 0.f;
  for (uint32_t m = blockIdx.x * 256 + threadIdx.x; m < (1u << 24); m += gridDim.x * 256) {
    const uint32_t w = m << 8;
    e = fmaxf(e, fabsf(gumbel_fast(w) - gumbel_exact(w)));
  }
  e = wave_max(e);
  if ((threadIdx.x & 63) == 0) atomicMax(out, __float_as_uint(e));
}

int launch_gumbel_check(double* h_out, hipStream_t st) {
  uint32_t* d = nullptr;
  hipError_t e = hipMallocAsync((void**)&d, sizeof(uint32_t), st);
  if (e != hipSuccess) return hip_fail(e, "hipMallocAsync");
  e = hipMemsetAsync(d, 0, sizeof(uint32_t), st);
  if (e != hipSuccess) return hip_fail(e, "hipMemsetAsync");
  hipLaunchKernelGGL(k_gumbel_check, dim3(1024), dim3(256), 0, st, d);
  uint32_t bits = 0;
  e = hipMemcpyAsync(&bits, d, sizeof(uint32_t), hipMemcpyDeviceToHost, st);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
  (void)hipFreeAsync(d, st);
  e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e, "gumbel check");
  float f;
  memcpy(&f, &bits, sizeof(f));
  *h_out = (double)f;
  return SARA_OK;
}

// Copy of a row-major bf16 weight [rows][K] (rows a multiple of 16, K of 64)
// into dst, a matrix of dst_rows rows in the GEMM weight layout, source tile
// j going to destination tile j * tile_mul + tile_add.
int launch_tile_weights(sara_ctx* c, const void* src, void* dst, int rows, int K, int tile_mul, int tile_add,
                        int dst_rows) {
  launch_k(c, c->stream, k_tile_weights, dim3(2048), dim3(256), 0, (const uint16_t*)src, (uint16_t*)dst,
                     rows / 16, K, tile_mul, tile_add, dst_rows / 16);
  return SARA_OK;
}

// Rows of heads head_off.. of a q, k or v weight ([n_rows][K], natural
// order) into the fused q|k|v weight (nqkv rows) in rotation-pair order.
int launch_tile_weights_pairs(sara_ctx* c, const void* src, void* dst, int n_rows, int K, int head_off) {
  launch_k(c, c->stream, k_tile_weights_pairs, dim3(2048), dim3(256), 0, (const uint16_t*)src,
                     (uint16_t*)dst, n_rows, K, head_off, c->hd, c->nqkv / 16);
  return SARA_OK;
}

// norm weights -> fp32 [2L+1][d]
__global__ void k_norm_to_f32_bf16(const uint16_t* __restrict__ src, float* __restrict__ dst, int d) {
  int c = blockIdx.x * 256 + threadIdx.x;
  if (c < d) dst[c] = bf16_to_f32(src[c]);
}

int launch_convert_norms(sara_ctx* c, const void* const* w) {
  const int d = c->d;
  for (int l = 0; l <= 2 * c->L; ++l) {
    const void* src;
    if (l == 2 * c->L) src = w[1 + 9 * c->L];
    else src = w[1 + 9 * (l / 2) + ((l & 1) ? 5 : 0)];
    float* dst = c->norms + (size_t)l * d;
    if (c->md.dtype == SARA_BF16)
      launch_k(c, c->stream, k_norm_to_f32_bf16, dim3((d + 255) / 256), dim3(256), 0,
                         (const uint16_t*)src, dst, d);
    else {
      hipError_t e = hipMemcpyAsync(dst, src, sizeof(float) * d, hipMemcpyDeviceToDevice, c->stream);
      if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync norms");
    }
  }
  return SARA_OK;
}

}  // namespace sara

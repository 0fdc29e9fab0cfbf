// SARA controller on the device: posterior update, decision rule, draws,
// priority ordering and slot assignment (Algorithm 1 on the decode clock).
//
// The controller is tiny (at most a few thousand prompts and slots per step)
// and latency bound, so each phase is one workgroup of 1024 threads that
// walks prompts and slots in index order with block-wide prefix scans: every
// log row, queue entry and slot assignment lands at a position fixed by
// (uid, j, slot) order, never by thread timing.  Counters touched by several
// threads use integer atomics only (order independent).
#include "sara_internal.h"

namespace sara {

// exclusive prefix sum over the 1024 threads; returns the block total
__device__ int block_scan_excl(int v, int* buf, int& total) {
  const int tid = threadIdx.x;
  buf[tid] = v;
  __syncthreads();
  for (int o = 1; o < kCtlThreads; o <<= 1) {
    int a = (tid >= o) ? buf[tid - o] : 0;
    __syncthreads();
    buf[tid] += a;
    __syncthreads();
  }
  total = buf[kCtlThreads - 1];
  int incl = buf[tid];
  __syncthreads();
  return incl - v;
}

__device__ __forceinline__ uint64_t queue_key(double pe, int bits, int uid, int j) {
  // ascending key order = (quantised p_eff desc, uid asc, j asc)
  uint64_t q = (uint64_t)floor(pe * (double)(1u << bits) + 0.5);
  uint64_t inv = (1ull << 21) - q;
  return (inv << 42) | ((uint64_t)uid << 16) | (uint64_t)j;
}

// Posterior-sampling priority index (SARA_MODE_SARA_THOMPSON): P(the group
// of k ends mixed | g) at one draw g ~ Beta(a, b) of the posterior a = a0 + s,
// b = b0 + n - s.  For integer a, b the draw is the a-th smallest of
// m = a + b - 1 uniforms (w + 1/2) 2^-32, w the words of Philox4x32-10 at
// counters (uid, n, c, 2) under the sampler key: found as the smallest word
// value v with #{w_i <= v} >= a by bisection over the 32-bit range,
// regenerating the m words per probe (no per-thread storage).  Other
// posteriors keep p_eff.
constexpr int kThompsonMaxM = 4096;
__device__ double pow_seq(double x, int e) {
  double p = 1.0;
  for (int i = 0; i < e; ++i) p = p * x;
  return p;
}
__device__ double thompson_index(const CtlParams& cp, int uid, int n, int s, double a0, double b0) {
  if (s >= 1 && n - s >= 1) return 1.0;
  const int r = cp.k - n;
  if (r <= 0) return 0.0;
  const double a = a0 + (double)s, b = b0 + (double)(n - s);
  if (a != floor(a) || b != floor(b) || a < 1.0 || b < 1.0 || a + b - 1.0 > (double)kThompsonMaxM)
    return peff_dev(n, s, cp.k, a0, b0);
  const int ia = (int)a, m = (int)(a + b) - 1;
  uint32_t k0, k1;
  sampler_key(cp.seed, cp.step, k0, k1);
  uint32_t lo = 0u, hi = 0xFFFFFFFFu;
  while (lo < hi) {
    const uint32_t mid = lo + ((hi - lo) >> 1);
    int cnt = 0;
    for (int c = 0; 4 * c < m; ++c) {
      const U32x4 w = philox4x32_10((uint32_t)uid, (uint32_t)n, (uint32_t)c, 2u, k0, k1);
      const int e = m - 4 * c;   // words of this counter that are draws
      cnt += (w.x <= mid) + (e > 1 && w.y <= mid) + (e > 2 && w.z <= mid) + (e > 3 && w.w <= mid);
    }
    if (cnt >= ia) hi = mid;
    else lo = mid + 1u;
  }
  const double g = ((double)lo + 0.5) * 0x1p-32;
  if (n == 0) return (1.0 - pow_seq(g, cp.k)) - pow_seq(1.0 - g, cp.k);
  if (s == 0) return 1.0 - pow_seq(1.0 - g, r);
  return 1.0 - pow_seq(g, r);
}

// ---------------------------------------------------------------------------
// reset (start of an allocation step)
// ---------------------------------------------------------------------------
__global__ void k_reset(Ctl* ctl, const CtlParams* __restrict__ cpp, int64_t budget, int32_t* status, int32_t* n_iss,
                        int32_t* n_done, int32_t* succ, int32_t* infl, double* peff,
                        int32_t* slot_uid, int32_t* fin, int32_t* r_len, int32_t* r_reward,
                        int32_t* btab) {
  const CtlParams cp = *cpp;
  const int tid = blockIdx.x * blockDim.x + threadIdx.x;
  const int nth = gridDim.x * blockDim.x;
  for (int u = tid; u < cp.U; u += nth) {
    status[u] = SARA_UNDRAWN; n_iss[u] = 0; n_done[u] = 0; succ[u] = 0; infl[u] = 0; peff[u] = 0.0;
  }
  for (int s = tid; s < cp.S; s += nth) { slot_uid[s] = -1; fin[s] = 0; }
  for (int r = tid; r < cp.U * cp.k; r += nth) { r_len[r] = 0; r_reward[r] = 0; }
  // prompt block tables: row S + u holds the prompt's PB pages
  for (int e = tid; e < cp.U * cp.PB; e += nth) {
    int u = e / cp.PB, b = e - u * cp.PB;
    btab[(size_t)(cp.S + u) * cp.MAXB + b] = u * cp.PB + b;
  }
  if (tid == 0) {
    Ctl z = {};
    z.budget_left = budget;
    z.t = -1;
    z.dirty = 1;
    *ctl = z;
  }
}

// ---------------------------------------------------------------------------
// decide: apply finished rollouts, then Eq. decide for quiescent prompts
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kCtlThreads) void k_decide(Ctl* __restrict__ ctl, const CtlParams* __restrict__ cpp,
    int32_t* __restrict__ status, int32_t* __restrict__ n_iss, int32_t* __restrict__ n_done,
    int32_t* __restrict__ succ, int32_t* __restrict__ infl, double* __restrict__ peff,
    int32_t* __restrict__ slot_uid, const int32_t* __restrict__ slot_j,
    int32_t* __restrict__ fin, const int32_t* __restrict__ r_len,
    const int32_t* __restrict__ r_reward, uint64_t* __restrict__ queue,
    int64_t* __restrict__ log_dec, int64_t* __restrict__ log_fin,
    const double* __restrict__ prior_a, const double* __restrict__ prior_b) {
  __shared__ int buf[kCtlThreads];
  __shared__ int s_nfin, s_ndec, s_qlen, s_dC, s_dA, s_dAb, s_more;
  __shared__ unsigned long long s_refund;
  __shared__ int s_done;
  const CtlParams cp = *cpp;
  const int tid = threadIdx.x;
  if (tid == 0) s_done = ctl->done;
  __syncthreads();
  if (s_done) return;
  const int t = ctl->t;
  if (tid == 0) {
    s_nfin = 0; s_ndec = 0; s_qlen = ctl->qlen; s_dC = 0; s_dA = 0; s_dAb = 0; s_refund = 0;
    s_more = 0;
  }
  __syncthreads();
  const int64_t fin_base = ctl->n_fin;
  // posts of finished rollouts, ascending slot
  for (int base = 0; base < cp.S; base += kCtlThreads) {
    int s = base + tid;
    int f = (s < cp.S) ? fin[s] : 0;
    int tot;
    int ex = block_scan_excl(f, buf, tot);
    if (f) {
      int u = slot_uid[s], j = slot_j[s];
      int rid = u * cp.k + j;
      int L = r_len[rid], r = r_reward[rid];
      atomicAdd(&n_done[u], 1);
      atomicAdd(&succ[u], r);
      atomicSub(&infl[u], 1);
      int64_t row = fin_base + s_nfin + ex;
      int64_t* lf = log_fin + row * 6;
      lf[0] = t; lf[1] = s; lf[2] = u; lf[3] = j; lf[4] = L; lf[5] = r;
      slot_uid[s] = -1;
      fin[s] = 0;
    }
    __syncthreads();
    if (tid == 0) s_nfin += tot;
    __syncthreads();
  }
  __threadfence_block();
  __syncthreads();
  // a prompt becomes quiescent only when one of its rollouts finishes (a
  // drawn prompt starts with n0 in flight, a continuing one with its new
  // rollouts), so a step without finishes decides nothing
  if (s_nfin == 0) {
    if (tid == 0) {
      ctl->tokens += ctl->M;
      ctl->dirty = 0;
    }
    return;
  }
  const int next_uid = ctl->next_uid;
  const int64_t dec_base = ctl->n_dec;
  // decisions, ascending uid
  for (int base = 0; base < next_uid; base += kCtlThreads) {
    int u = base + tid;
    int pred = 0, code = 0, more = 0, n = 0, s = 0;
    double pe = 0.0;
    // counters were just updated with device-scope atomics: read them the same way
    if (u < next_uid && status[u] == SARA_ACTIVE && atomicAdd(&infl[u], 0) == 0) {
      pred = 1;
      n = atomicAdd(&n_done[u], 0);
      s = atomicAdd(&succ[u], 0);
      pe = cp.has_prior ? peff_dev(n, s, cp.k, prior_a[u], prior_b[u]) : peff_dev(n, s, cp.k, cp.a0, cp.b0);
      bool mixed = (s >= 1) && (n - s >= 1);
      if (mixed && n >= cp.commit_min) code = SARA_COMMIT;
      else if (n >= cp.k) code = SARA_ABANDON;
      else if (!mixed && pe < cp.tau) code = SARA_ABANDON;
      else { code = SARA_CONTINUE; more = mixed ? (cp.commit_min - n) : 1; }
    }
    int tot, tot_more;
    int ex = block_scan_excl(pred, buf, tot);
    int exm = block_scan_excl(more, buf, tot_more);
    if (pred) {
      int64_t* ld = log_dec + (dec_base + s_ndec + ex) * 6;
      ld[0] = t; ld[1] = u; ld[2] = code; ld[3] = n; ld[4] = s;
      ld[5] = (int64_t)__double_as_longlong(pe);
      peff[u] = pe;
      if (code == SARA_COMMIT) {
        status[u] = SARA_COMMITTED;
        atomicAdd(&s_dC, 1);
        atomicAdd(&s_refund, (unsigned long long)(cp.k - n));
      } else if (code == SARA_ABANDON) {
        status[u] = SARA_ABANDONED;
        atomicAdd(&s_dAb, 1);
        atomicAdd(&s_refund, (unsigned long long)(cp.k - n));
      } else {
        int j0 = n_iss[u];
        const double qi = (cp.mode == SARA_MODE_SARA_THOMPSON)
            ? thompson_index(cp, u, n, s, cp.has_prior ? prior_a[u] : cp.a0, cp.has_prior ? prior_b[u] : cp.b0)
            : pe;
        for (int e = 0; e < more; ++e)
          queue[s_qlen + exm + e] = queue_key(qi, cp.bits, u, j0 + e);
        n_iss[u] = j0 + more;
        infl[u] = more;  // it was 0: the prompt was quiescent
      }
    }
    __syncthreads();
    if (tid == 0) { s_ndec += tot; s_qlen += tot_more; s_more += tot_more; }
    __syncthreads();
  }
  if (tid == 0) {
    ctl->n_fin = fin_base + s_nfin;
    ctl->n_dec = dec_base + s_ndec;
    ctl->qlen = s_qlen;
    ctl->nC += s_dC;
    ctl->nAb += s_dAb;
    ctl->nA -= s_dC + s_dAb;
    ctl->budget_left += (int64_t)s_refund;
    ctl->rollouts += s_more;
    ctl->tokens += ctl->M;
    ctl->dirty = (s_nfin > 0) ? 1 : 0;
  }
}

// ---------------------------------------------------------------------------
// refill: draws, priority sort, slot assignment, active list, done flag
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kCtlThreads) void k_refill(Ctl* __restrict__ ctl, const CtlParams* __restrict__ cpp,
    int32_t* __restrict__ status, int32_t* __restrict__ n_iss, int32_t* __restrict__ infl,
    double* __restrict__ peff, int32_t* __restrict__ slot_uid, int32_t* __restrict__ slot_j,
    int32_t* __restrict__ slot_gen, uint64_t* __restrict__ slot_hash,
    int32_t* __restrict__ active, uint64_t* __restrict__ queue, int32_t* __restrict__ btab,
    int64_t* __restrict__ log_draw, int64_t* __restrict__ log_asg, const double* __restrict__ prior_p,
    const double* __restrict__ prior_a, const double* __restrict__ prior_b) {
  __shared__ int buf[kCtlThreads];
  __shared__ uint64_t qs[kMaxQueue];
  __shared__ int freel[kMaxSlots];
  __shared__ unsigned char occ[kMaxSlots];
  __shared__ int s_d, s_qlen, s_nfree, s_M, s_skip;
  const CtlParams cp = *cpp;
  const int tid = threadIdx.x;
  if (tid == 0) {
    s_skip = ctl->done ? 2 : (ctl->dirty ? 0 : 1);
  }
  __syncthreads();
  if (s_skip == 2) return;
  if (s_skip == 1) {
    if (tid == 0) ctl->t += 1;
    return;
  }
  const int tnext = ctl->t + 1;
  if (tid == 0) {
    int64_t bud = ctl->budget_left;
    int64_t d = (int64_t)cp.U - ctl->next_uid;
    int64_t byb = bud / cp.k;
    if (byb < d) d = byb;
    if (cp.mode != SARA_MODE_FIXED_K) {
      int64_t need = (int64_t)cp.B - ctl->nC - ctl->nA;
      if (need < d) d = need;
    }
    if (d < 0) d = 0;
    s_d = (int)d;
    s_qlen = ctl->qlen;
  }
  __syncthreads();
  const int d = s_d, nu0 = ctl->next_uid;
  const int64_t draw_base = ctl->n_draw;
  for (int e = tid; e < d; e += kCtlThreads) {
    int u = nu0 + e;
    status[u] = SARA_ACTIVE;
    n_iss[u] = cp.n0;
    infl[u] = cp.n0;
    peff[u] = cp.has_prior ? prior_p[u] : cp.prior;
    int64_t* lr = log_draw + (draw_base + e) * 2;
    lr[0] = tnext; lr[1] = u;
  }
  __threadfence_block();
  __syncthreads();
  const int qlen = s_qlen + d * cp.n0;
  // waiting rollouts plus the probes of uid nu0 .. nu0 + d - 1, bitonic-sorted
  // in LDS (padded with maximal keys)
  int np2 = 1;
  while (np2 < qlen) np2 <<= 1;
  for (int e = tid; e < np2; e += kCtlThreads) {
    uint64_t key = ~0ull;
    if (e < s_qlen) key = queue[e];
    else if (e < qlen) {
      int q = e - s_qlen;
      const int uq = nu0 + q / cp.n0;
      const double qi = (cp.mode == SARA_MODE_SARA_THOMPSON)
          ? thompson_index(cp, uq, 0, 0, cp.has_prior ? prior_a[uq] : cp.a0, cp.has_prior ? prior_b[uq] : cp.b0)
          : (cp.has_prior ? prior_p[uq] : cp.prior);
      key = queue_key(qi, cp.bits, uq, q % cp.n0);
    }
    qs[e] = key;
  }
  __syncthreads();
  for (int size = 2; size <= np2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int e = tid; e < np2; e += kCtlThreads) {
        int partner = e ^ stride;
        if (partner > e) {
          bool up = ((e & size) == 0);
          uint64_t a = qs[e], b = qs[partner];
          if ((a > b) == up) { qs[e] = b; qs[partner] = a; }
        }
      }
      __syncthreads();
    }
  }
  // free slots, ascending
  if (tid == 0) s_nfree = 0;
  __syncthreads();
  for (int base = 0; base < cp.S; base += kCtlThreads) {
    int s = base + tid;
    int busy = (s < cp.S && slot_uid[s] >= 0) ? 1 : 0;
    if (s < cp.S) occ[s] = (unsigned char)busy;
    int f = (s < cp.S && !busy) ? 1 : 0;
    int tot;
    int ex = block_scan_excl(f, buf, tot);
    if (f) freel[s_nfree + ex] = s;
    __syncthreads();
    if (tid == 0) s_nfree += tot;
    __syncthreads();
  }
  const int m = min(s_nfree, qlen);
  const int64_t asg_base = ctl->n_asg;
  for (int e = tid; e < m; e += kCtlThreads) {
    uint64_t key = qs[e];
    int u = (int)((key >> 16) & ((1ull << 26) - 1)), j = (int)(key & 0xFFFF);
    int s = freel[e];
    occ[s] = 1;
    slot_uid[s] = u;
    slot_j[s] = j;
    slot_gen[s] = 0;
    slot_hash[s] = reward_hash_init(cp.seed, cp.step, u);
    int64_t* la = log_asg + (asg_base + e) * 4;
    la[0] = tnext; la[1] = s; la[2] = u; la[3] = j;
  }
  // block tables of the newly assigned slots: shared prompt pages, then the
  // slot's private pages (assigned rows only)
  for (int e = tid; e < m * cp.MAXB; e += kCtlThreads) {
    int a = e / cp.MAXB, b = e - a * cp.MAXB;
    int s = freel[a];
    uint64_t key = qs[a];
    int u = (int)((key >> 16) & ((1ull << 26) - 1));
    int32_t blk = (b < cp.PB) ? (u * cp.PB + b) : (cp.U * cp.PB + s * cp.SB + (b - cp.PB));
    btab[(size_t)s * cp.MAXB + b] = blk;
  }
  // remaining queue
  for (int e = tid; e < qlen - m; e += kCtlThreads) queue[e] = qs[m + e];
  __threadfence_block();
  __syncthreads();
  // active list: occupied slots ascending
  if (tid == 0) s_M = 0;
  __syncthreads();
  for (int base = 0; base < cp.S; base += kCtlThreads) {
    int s = base + tid;
    int f = (s < cp.S && occ[s]) ? 1 : 0;
    int tot;
    int ex = block_scan_excl(f, buf, tot);
    if (f) active[s_M + ex] = s;
    __syncthreads();
    if (tid == 0) s_M += tot;
    __syncthreads();
  }
  if (tid == 0) {
    ctl->next_uid = nu0 + d;
    ctl->nA += d;
    ctl->budget_left -= (int64_t)d * cp.k;
    ctl->rollouts += (int64_t)d * cp.n0;
    ctl->n_draw = draw_base + d;
    ctl->n_asg = asg_base + m;
    ctl->qlen = qlen - m;
    ctl->M = s_M;
    ctl->running = s_M;
    ctl->done = (ctl->nA == 0) ? 1 : 0;
    ctl->t = tnext;
    ctl->dirty = 0;
  }
}

// ---------------------------------------------------------------------------
// pure entry points
// ---------------------------------------------------------------------------
// Eq. peff per prompt under that prompt's own prior; NaN for a prior that is
// not positive and finite, or counts outside 0 <= s <= n <= k
__global__ void k_peff(const double* alpha, const double* beta, const int32_t* n, const int32_t* s, int k,
                       int count, double* out) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= count) return;
  const double a0 = alpha[i], b0 = beta[i];
  const int ni = n[i], si = s[i];
  const bool ok = a0 > 0.0 && b0 > 0.0 && isfinite(a0) && isfinite(b0) && si >= 0 && si <= ni && ni <= k;
  out[i] = ok ? peff_dev(ni, si, k, a0, b0) : __builtin_nan("");
}

// error word, then (after a system-scope fence) the done flag, into pinned
// host memory: a host that sees the flag change also sees the error word
__global__ void k_poll(const Ctl* __restrict__ ctl, int32_t* h) {
  if (threadIdx.x == 0) {
    const int32_t err = __atomic_load_n(&ctl->error, __ATOMIC_RELAXED);
    const int32_t done = __atomic_load_n(&ctl->done, __ATOMIC_RELAXED);
    h[1] = err;
    __threadfence_system();
    h[0] = done;
  }
}

// Eq. grpo: one wave per group, statistics in fp64
__global__ void k_grpo(const float* __restrict__ r, const int32_t* __restrict__ off, int n_groups,
                       const int32_t* __restrict__ n_dev, float eps, float* __restrict__ adv) {
  int g = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  int lane = threadIdx.x & 63;
  if (n_dev) n_groups = min(n_groups, *n_dev);
  if (g >= n_groups) return;
  int lo = off[g], hi = off[g + 1], m = hi - lo;
  double sum = 0.0;
  for (int i = lo + lane; i < hi; i += 64) sum += (double)r[i];
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o, 64);
  double mean = (m > 0) ? sum / m : 0.0;
  double sq = 0.0;
  for (int i = lo + lane; i < hi; i += 64) { double dv = (double)r[i] - mean; sq += dv * dv; }
  for (int o = 32; o > 0; o >>= 1) sq += __shfl_xor(sq, o, 64);
  double sd = (m >= 2) ? sqrt(sq / (m - 1)) : 0.0;
  for (int i = lo + lane; i < hi; i += 64)
    adv[i] = (m >= 2) ? (float)(((double)r[i] - mean) / (sd + (double)eps)) : 0.0f;
}

// CSR of committed groups in ascending uid, rollouts in j order
__global__ __launch_bounds__(kCtlThreads) void k_build_csr(const Ctl* __restrict__ ctl,
    const CtlParams* __restrict__ cpp, const int32_t* __restrict__ status, const int32_t* __restrict__ n_iss,
    const int32_t* __restrict__ r_reward, int32_t* __restrict__ g_off, float* __restrict__ g_r,
    int32_t* __restrict__ g_n) {
  __shared__ int buf[kCtlThreads];
  __shared__ int s_g, s_r;
  const CtlParams cp = *cpp;
  const int tid = threadIdx.x;
  if (tid == 0) { s_g = 0; s_r = 0; g_off[0] = 0; }
  __syncthreads();
  const int nu = ctl->next_uid;
  for (int base = 0; base < nu; base += kCtlThreads) {
    int u = base + tid;
    int c = (u < nu && status[u] == SARA_COMMITTED) ? 1 : 0;
    int n = c ? n_iss[u] : 0;
    int totc, totn;
    int exc = block_scan_excl(c, buf, totc);
    int exn = block_scan_excl(n, buf, totn);
    if (c) {
      int o = s_r + exn;
      for (int j = 0; j < n; ++j) g_r[o + j] = (float)r_reward[u * cp.k + j];
      g_off[s_g + exc + 1] = o + n;
    }
    __syncthreads();
    if (tid == 0) { s_g += totc; s_r += totn; }
    __syncthreads();
  }
  if (tid == 0) *g_n = s_g;
}

// ---------------------------------------------------------------------------
// history warm start
// ---------------------------------------------------------------------------
// Priors of the step's pool from the prompt set's pseudo-counts: pool prompt
// u is set prompt ids[u] and starts from Beta(a0 + a[ids[u]], b0 + b[ids[u]]);
// prior_p is p_eff(0, 0) under it (the priority of its probes).  An id
// outside [0, n_store) sets the device error word and falls back to the
// global prior.  Runs after k_reset (which clears the error word).
__global__ void k_warm_priors(Ctl* __restrict__ ctl, const CtlParams* __restrict__ cpp,
    const int32_t* __restrict__ ids, const double* __restrict__ a, const double* __restrict__ b, int n_store,
    double* __restrict__ prior_a, double* __restrict__ prior_b, double* __restrict__ prior_p) {
  const CtlParams cp = *cpp;
  for (int u = blockIdx.x * blockDim.x + threadIdx.x; u < cp.U; u += gridDim.x * blockDim.x) {
    const int id = ids[u];
    double al = cp.a0, be = cp.b0;
    if (id >= 0 && id < n_store) {
      al = cp.a0 + a[id];
      be = cp.b0 + b[id];
    } else {
      atomicOr(&ctl->error, SARA_DEVERR_WARM_ID);
    }
    prior_a[u] = al;
    prior_b[u] = be;
    prior_p[u] = peff_dev(0, 0, cp.k, al, be);
  }
}

// After a step: the drawn pool prompts add their outcomes to their set
// prompt's counts (ids are distinct, so no two threads share an entry) ...
__global__ void k_warm_add(const Ctl* __restrict__ ctl, const int32_t* __restrict__ ids, int U, int n_store,
    const int32_t* __restrict__ n_done, const int32_t* __restrict__ succ,
    double* __restrict__ a, double* __restrict__ b) {
  const int drawn = min(ctl->next_uid, U);
  for (int u = blockIdx.x * blockDim.x + threadIdx.x; u < drawn; u += gridDim.x * blockDim.x) {
    const int id = ids[u];
    if (id < 0 || id >= n_store) continue;
    a[id] = a[id] + (double)succ[u];
    b[id] = b[id] + (double)(n_done[u] - succ[u]);
  }
}

// ... then every entry of the set decays by lambda
__global__ void k_warm_decay(double* __restrict__ a, double* __restrict__ b, int n_store, double lambda) {
  for (int p = blockIdx.x * blockDim.x + threadIdx.x; p < n_store; p += gridDim.x * blockDim.x) {
    a[p] = lambda * a[p];
    b[p] = lambda * b[p];
  }
}

// ---------------------------------------------------------------------------
// host launchers
// ---------------------------------------------------------------------------
int launch_reset(sara_ctx* c) {
  hipLaunchKernelGGL(k_reset, dim3(64), dim3(256), 0, c->stream, c->ctl, c->cp_dev, (int64_t)c->ad.budget_N,
                     c->status, c->n_iss, c->n_done, c->succ, c->infl, c->peff, c->slot_uid, c->fin,
                     c->r_len, c->r_reward, c->btab);
  return SARA_OK;
}

int launch_decide(sara_ctx* c) {
  hipLaunchKernelGGL(k_decide, dim3(1), dim3(kCtlThreads), 0, c->stream, c->ctl, c->cp_dev, c->status,
                     c->n_iss, c->n_done, c->succ, c->infl, c->peff, c->slot_uid, c->slot_j, c->fin,
                     c->r_len, c->r_reward, c->queue, c->log_dec, c->log_fin, c->prior_a, c->prior_b);
  return SARA_OK;
}

int launch_refill(sara_ctx* c) {
  hipLaunchKernelGGL(k_refill, dim3(1), dim3(kCtlThreads), 0, c->stream, c->ctl, c->cp_dev, c->status,
                     c->n_iss, c->infl, c->peff, c->slot_uid, c->slot_j, c->slot_gen, c->slot_hash,
                     c->active, c->queue, c->btab, c->log_draw, c->log_asg, c->prior_p, c->prior_a, c->prior_b);
  return SARA_OK;
}

int launch_warm_priors(sara_ctx* c) {
  hipLaunchKernelGGL(k_warm_priors, dim3((c->U + 255) / 256), dim3(256), 0, c->stream, c->ctl, c->cp_dev,
                     c->warm_ids, (const double*)c->warm_a, (const double*)c->warm_b, c->warm_n, c->prior_a,
                     c->prior_b, c->prior_p);
  return SARA_OK;
}

int launch_warm_update(sara_ctx* c, double lambda) {
  hipLaunchKernelGGL(k_warm_add, dim3((c->U + 255) / 256), dim3(256), 0, c->stream, c->ctl, c->warm_ids, c->U,
                     c->warm_n, c->n_done, c->succ, c->warm_a, c->warm_b);
  hipLaunchKernelGGL(k_warm_decay, dim3(std::min((c->warm_n + 255) / 256, 1024)), dim3(256), 0, c->stream,
                     c->warm_a, c->warm_b, c->warm_n, lambda);
  return SARA_OK;
}

int launch_finish(sara_ctx* c, float eps) {
  hipLaunchKernelGGL(k_build_csr, dim3(1), dim3(kCtlThreads), 0, c->stream, c->ctl, c->cp_dev, c->status,
                     c->n_iss, c->r_reward, c->g_off, c->g_r, c->g_n);
  // at most U groups; the kernel stops at the committed count on the device
  hipLaunchKernelGGL(k_grpo, dim3((c->U + 3) / 4), dim3(256), 0, c->stream, c->g_r, c->g_off,
                     c->U, (const int32_t*)c->g_n, eps, c->g_adv);
  return SARA_OK;
}

int launch_peff(const double* alpha, const double* beta, const int32_t* n, const int32_t* s, int k, int count,
                double* out, hipStream_t st) {
  if (count > 0)
    hipLaunchKernelGGL(k_peff, dim3((count + 255) / 256), dim3(256), 0, st, alpha, beta, n, s, k, count, out);
  return SARA_OK;
}

int launch_poll(sara_ctx* c, int32_t* d_host) {
  hipLaunchKernelGGL(k_poll, dim3(1), dim3(64), 0, c->stream, (const Ctl*)c->ctl, d_host);
  return SARA_OK;
}

int launch_grpo(const float* r, const int32_t* off, int n_groups, float eps, float* adv,
                hipStream_t st) {
  if (n_groups > 0)
    hipLaunchKernelGGL(k_grpo, dim3((n_groups + 3) / 4), dim3(256), 0, st, r, off, n_groups,
                       (const int32_t*)nullptr, eps, adv);
  return SARA_OK;
}

}  // namespace sara

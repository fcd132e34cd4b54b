// lg_detect.hip -- Stage 1 of LoopGuard: the debounced online onset rule (Sec. 5.2, Eq. (8) and
// Eq. (9); App. B.2), one 256-lane workgroup per sequence, integer arithmetic only.
//
// Per step the workgroup stages the token tail in LDS and derives every signal from it:
//   - the equality structure of the window along its diagonals (lag delta = i - p): a forward
//     scan per lag marks repeated tokens (distinct count, Eq. (5)) and repeated n-grams (novelty);
//     a backward scan per lag gives the longest common extension of every pair, whose maximum over
//     earlier sources is the LZ match length at each position. Lanes are staggered so that the
//     positions touched in one iteration are distinct (no LDS write conflicts) and the shared
//     operand is a broadcast;
//   - the greedy LZ parse (Eq. (6) reading) as pointer doubling over "next parse position";
//   - the trailing self-alignment run of every period P, one wave per period at a time, 64
//     comparisons per ballot;
//   - the votes, gates, warmup, cooldown and aggressiveness level of Eq. (8)/(9) in one lane.
#include "lg_internal.h"

namespace lg {

struct DetectArgs {
  lg_guard_params p;
  const int32_t* tokens;
  int32_t ring;
  const int32_t* t;
  const int32_t* t0;
  float* conf;
  lg_guard_state* state;
  lg_decision* decision;
};

constexpr int kDetThreads = 256;
constexpr int kBuf = kMaxHorizon + kMaxWindow;

__device__ __forceinline__ int block_sum(int x, int* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  __syncthreads();
  if (lane == 0) red[wave] = x;
  __syncthreads();
  int s = 0;
#pragma unroll
  for (int w = 0; w < kDetThreads / 64; ++w) s += red[w];
  __syncthreads();
  return s;
}

__global__ __launch_bounds__(kDetThreads) void detect_kernel(DetectArgs a) {
  const lg_guard_params& p = a.p;
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t0 = max(0, a.t0[b]);  // stream indices are non-negative
  const int n = a.t[b] + 1;
  const int w0 = max(t0, n - p.W);
  const int m = max(0, n - w0);
  const int span_all = max(p.W, p.rep_horizon);
  const int lo_all = max(t0, n - span_all);  // first stream index staged in LDS
  const int nbuf = max(0, n - lo_all);

  __shared__ int y[kBuf];                 // y[i - lo_all]
  __shared__ int ell[kMaxWindow];         // LZ match length at window index
  __shared__ unsigned char rep1[kMaxWindow], repg[kMaxWindow];
  __shared__ int nxt[2][kMaxWindow + 1], cst[2][kMaxWindow + 1];
  __shared__ int red[kDetThreads / 64];
  __shared__ int wbestP[kDetThreads / 64], wbestT[kDetThreads / 64];

  const int32_t* tok = a.tokens + (size_t)b * a.ring;
  for (int i = tid; i < nbuf; i += kDetThreads) {
    const int idx = lo_all + i;
    y[i] = tok[idx % a.ring];
  }
  for (int i = tid; i < m; i += kDetThreads) { ell[i] = 0; rep1[i] = 0; repg[i] = 0; }
  __syncthreads();
  const int wo = w0 - lo_all;  // window offset inside y[]
  lg_guard_state st = a.state[b];
  const bool do_cr = !st.cr_valid || p.cr_interval <= 1 || (n % p.cr_interval) == 0;
  const int g = p.nov_ngram;

  // Diagonal scans over lags delta = 1 .. m-1 (lane tid takes delta = tid+1, tid+1+256, ...).
  for (int delta = tid + 1; delta < m; delta += kDetThreads) {
    // forward: runs of y[i-delta] == y[i] ending at i (backward n-gram match length)
    int run = 0;
    for (int i = delta; i < m; ++i) {
      const bool eq = y[wo + i - delta] == y[wo + i];
      run = eq ? run + 1 : 0;
      if (eq) rep1[i] = 1;
      if (run >= g) repg[i] = 1;
    }
  }
  if (do_cr) {
    // backward: run = LCE(i-delta, i) inside the window while i walks from m-1 down to delta.
    // Lane tid (delta = delta0 + tid) starts tid iterations late, so at iteration k it sits at
    // i = m-1-k+tid: lanes touch distinct i and share the source token y[m-1-k-delta0].
    for (int delta0 = 1; delta0 < m; delta0 += kDetThreads) {
      const int delta = delta0 + tid;
      int run = 0;
      for (int k = 0; k < m - delta0; ++k) {
        const int kk = k - tid;
        if (delta < m && kk >= 0 && kk <= m - 1 - delta) {
          const int ii = m - 1 - kk;
          const bool eq = y[wo + ii - delta] == y[wo + ii];
          run = eq ? run + 1 : 0;
          if (run) atomicMax(&ell[ii], run);
        }
      }
    }
  }
  __syncthreads();

  // Distinct tokens and novelty.
  int uloc = 0, nloc = 0, rloc = 0;
  const int nov_lo = max(g - 1, m - p.nov_span);  // window index of the first examined position
  for (int i = tid; i < m; i += kDetThreads) {
    uloc += rep1[i] ? 0 : 1;
    if (i >= nov_lo) { rloc += 1; nloc += repg[i] ? 0 : 1; }
  }
  const int distinct = block_sum(uloc, red);
  const int novel = block_sum(nloc, red);
  const int nov_r = block_sum(rloc, red);

  // Greedy LZ parse by pointer doubling: cost of the parse from i to the end of the window.
  int lz_cost = st.cr_cost, lz_m = st.cr_m;
  if (do_cr) {
    for (int i = tid; i <= m; i += kDetThreads) {
      if (i == m) { nxt[0][i] = m; cst[0][i] = 0; }
      else {
        const int e = ell[i];
        nxt[0][i] = e >= 3 ? min(i + e, m) : i + 1;
        cst[0][i] = e >= 3 ? 2 : 1;
      }
    }
    __syncthreads();
    int cur = 0;
    for (int span = 1; span <= m; span <<= 1) {
      for (int i = tid; i <= m; i += kDetThreads) {
        const int j = nxt[cur][i];
        cst[cur ^ 1][i] = cst[cur][i] + cst[cur][j];
        nxt[cur ^ 1][i] = nxt[cur][j];
      }
      __syncthreads();
      cur ^= 1;
    }
    lz_cost = cst[cur][0];
    lz_m = m;
  }

  // Trailing self-alignment: L_P for P = 1 .. rep_pmax, one wave per period.
  const int H = p.rep_horizon;
  int bestP = 0, bestT = 0;
  for (int P = wave + 1; P <= p.rep_pmax; P += kDetThreads / 64) {
    // largest k <= H-P with y[n-1-r] == y[n-1-r-P] for r < k and n-1-r-P >= t0
    const int kmax = min(H - P, n - P - t0);
    int Lp = 0;
    for (int r0 = 0; r0 < max(kmax, 0); r0 += 64) {
      const int r = r0 + lane;
      bool eq = false;
      if (r < kmax) eq = y[(n - 1 - r) - lo_all] == y[(n - 1 - r - P) - lo_all];
      const unsigned long long miss = __ballot(!eq);
      if (miss) { Lp = r0 + __ffsll((long long)miss) - 1; break; }
      Lp = r0 + 64;
    }
    Lp = min(Lp, max(kmax, 0));
    const int TP = Lp + P;
    if (Lp >= (p.rep_min_copies - 1) * P && TP >= p.rep_min_len && TP > bestT) { bestT = TP; bestP = P; }
  }
  if (lane == 0) { wbestP[wave] = bestP; wbestT[wave] = bestT; }
  __syncthreads();

  if (tid == 0) {
    int Ps = 0, Ts = 0;
    for (int w = 0; w < kDetThreads / 64; ++w)
      if (wbestT[w] > Ts || (wbestT[w] == Ts && wbestT[w] > 0 && wbestP[w] < Ps)) { Ts = wbestT[w]; Ps = wbestP[w]; }

    const int vote_ttr = (long long)p.ttr_den * distinct < (long long)p.ttr_num * m;
    if (do_cr) { st.cr_cost = lz_cost; st.cr_m = lz_m; st.cr_valid = 1; }
    const int vote_cr = (long long)p.cr_den * st.cr_cost < (long long)p.cr_num * st.cr_m;
    const float c = a.conf ? a.conf[b] : 0.f;
    st.streak = (c > p.conf_threshold) ? st.streak + 1 : 0;
    const int vote_p1 = st.streak >= p.streak_min;
    const int warn = (vote_ttr + vote_cr + vote_p1) >= p.K;
    st.stall = ((long long)p.nov_den * novel < (long long)p.nov_num * nov_r) ? st.stall + 1 : 0;
    const int stall_gate = st.stall >= p.stall_min;
    st.rep = Ps > 0 ? st.rep + 1 : 0;
    const int tail_gate = st.rep >= p.rep_debounce;
    const int warm = (n - t0) >= p.t_min;
    const int cool = (st.n_int == 0) || (n - st.n_last >= p.cooldown);
    int fire;
    if (p.mode == LG_MODE_ALWAYS_ON) fire = warm && cool;
    else if (p.mode == LG_MODE_P1_ONLY) fire = warm && cool && vote_p1;
    else fire = warm && cool && warn && (stall_gate || tail_gate);
    if (fire) {
      if (st.n_int > 0 && n - st.n_last <= p.retrigger_window)
        st.level = min(st.level + 1, p.level_max);
      else
        st.level = 0;
      st.n_last = n;
      st.n_int += 1;
    }
    lg_decision d;
    d.trigger = fire;
    d.warn = warn;
    d.votes = vote_ttr | (vote_cr << 1) | (vote_p1 << 2);
    d.stall_gate = stall_gate;
    d.tailrep_gate = tail_gate;
    d.n = n;
    d.distinct = distinct;
    d.lz_cost = st.cr_cost;
    d.novel = novel;
    d.nov_r = nov_r;
    d.period = Ps;
    d.span_lo = Ps > 0 ? n - Ts : -1;
    d.level = st.level;
    d.n_int = st.n_int;
    d.reserved[0] = 0;
    d.reserved[1] = 0;
    a.decision[b] = d;
    a.state[b] = st;
    if (a.conf) a.conf[b] = 0.f;  // consumed: the next step max-accumulates from zero
  }
}

hipError_t launch_detect(const lg_guard_params* p, int batch, const int32_t* tokens, int ring,
                         const int32_t* t, const int32_t* t0, float* conf, lg_guard_state* state,
                         lg_decision* decision, hipStream_t st) {
  DetectArgs a;
  a.p = *p;
  a.tokens = tokens;
  a.ring = ring;
  a.t = t;
  a.t0 = t0;
  a.conf = conf;
  a.state = state;
  a.decision = decision;
  hipLaunchKernelGGL(detect_kernel, dim3(batch), dim3(kDetThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace lg

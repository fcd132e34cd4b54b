// lg_detect.hip -- Stage 1 of LoopGuard: the debounced online onset rule (Sec. 5.2, Eq. (8) and
// Eq. (9); App. B.2), one 512-lane workgroup (8 waves) per sequence, integer arithmetic only.
//
// Window statistics come from the equality structure of the window by lag: for a lag delta,
// E_delta[i] = (y[i] == y[i - delta]) over window positions i. A wave builds E_delta 64 positions
// at a time with one ballot (lane = position), the eight waves taking every eighth lag. From the
// masks, the longest earlier match starting at i (the LZ match length of the Eq. (6) reading) is
// the longest run of ones of E_delta starting at i, maximised over delta: each lane counts the
// trailing ones of the mask shifted to its position, chunks taken from the window end so the run
// carries across 64-position boundaries. The other statistics follow from it:
//   - a token is repeated (distinct count, Eq. (5)) where its match length is >= 1;
//   - an n-gram ending at i is repeated (novelty) where the match length at i-g+1 is >= g.
// The greedy LZ parse is then pointer doubling over "next parse position".
// The trailing self-alignment run L_P of every period (suffix test) is carried in the state: when
// the call directly follows the one the state was written for, L_P(n) = L_P(n-1) + 1 on a match at
// the newest token and 0 otherwise (capped); any other call recomputes all L_P, one wave per
// period, 256 comparisons per iteration.
#include "lg_keepset.h"

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

constexpr int kDetThreads = 512;
constexpr int kDetWaves = kDetThreads / 64;
constexpr int kBuf = kMaxHorizon + kMaxWindow + 64;

__device__ __forceinline__ int block_sum(int x, int* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  __syncthreads();
  if (lane == 0) red[wave] = x;
  __syncthreads();
  int s = 0;
#pragma unroll
  for (int w = 0; w < kDetWaves; ++w) s += red[w];
  __syncthreads();
  return s;
}

__device__ __forceinline__ int block_max(int x, int* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = max(x, __shfl_xor(x, o, 64));
  __syncthreads();
  if (lane == 0) red[wave] = x;
  __syncthreads();
  int s = red[0];
#pragma unroll
  for (int w = 1; w < kDetWaves; ++w) s = max(s, red[w]);
  __syncthreads();
  return s;
}

// The scalar fields of lg_guard_state (the tail runs are handled by all lanes).
struct StateHeader {
  int32_t streak, stall, rep, n_int, n_last, level, cr_valid, cr_cost, cr_m;
};

// Number of consecutive set bits of x starting at bit 0.
__device__ __forceinline__ int trailing_ones(unsigned long long x) {
  const unsigned long long nx = ~x;
  return nx == 0ull ? 64 : __builtin_ctzll(nx);
}

// kChunks = window chunks of 64 positions the kernel is compiled for (W <= 64 * kChunks).
template <int kChunks>
__device__ void detect_block(const DetectArgs& a) {
  const lg_guard_params& p = a.p;
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: lag loops stay scalar
  // The newest position is clamped to [-1, 2^30 - 1] (stream lengths 0 .. 2^30) and t0 to
  // [0, n] (a monitored stream that starts after n is empty), so every index derived from them
  // below stays in int32 range and inside the staged buffers whatever the caller passes.
  const int n = min(max(a.t[b], -1), (1 << 30) - 1) + 1;
  const int t0 = min(max(0, a.t0[b]), n);
  const int w0 = max(t0, n - p.W);
  const int m = max(0, n - w0);
  const int H = p.rep_horizon;
  const int span_all = max(p.W, H);
  const int lo_all = max(t0, n - span_all);  // first stream index staged in LDS
  const int nbuf = max(0, n - lo_all);

  // y[i - lo_all] for the staged stream; kMaxWindow entries in front of it are read (and masked
  // out) by the lag compares of window positions before their lag.
  __shared__ int ybuf[kMaxWindow + kBuf];
  int* y = ybuf + kMaxWindow;
  __shared__ int ellw[kDetWaves][kMaxWindow];      // per-wave LZ match length at window index
  __shared__ int ellmax[kMaxWindow];               // ... maximised over the waves
  __shared__ int nxt[2][kMaxWindow + 1], cst[2][kMaxWindow + 1];
  __shared__ int red[kDetWaves];

  const int32_t* tok = a.tokens + (size_t)b * a.ring;
  for (int i = tid; i < nbuf; i += kDetThreads) y[i] = tok[(lo_all + i) % a.ring];
  __syncthreads();
  const int* yw = y + (w0 - lo_all);  // window: yw[0 .. m)
  const lg_guard_state& gst = a.state[b];
  const int cr_valid = gst.cr_valid;
  const bool do_cr = !cr_valid || p.cr_interval <= 1 || (n % p.cr_interval) == 0;
  const int g = p.nov_ngram;
  const int nch = (m + 63) >> 6;

  // ---- window statistics from the lag masks ----
  // Every window statistic follows from ell[i] = the longest earlier match starting at window
  // position i (max over lags of the run of ones of E_delta from i): the token at j occurred
  // earlier in the window iff ell[j] >= 1, and the g-gram ending at j did iff ell[j-g+1] >= g
  // (a run of g ones at some lag). The lag loop therefore computes only the runs.
  int yown[kChunks];
  int ell[kChunks];
  unsigned long long in_win[kChunks];  // window positions of each chunk (j < m)
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int j = 64 * c + lane;
    yown[c] = (c < nch && j < m) ? yw[j] : 0;
    ell[c] = 0;
    const int k = m - 64 * c;
    in_win[c] = k >= 64 ? ~0ull : (k <= 0 ? 0ull : (1ull << k) - 1ull);
  }
  for (int delta = wave + 1; delta < m; delta += kDetWaves) {
    // Chunks below c_min hold no position >= delta; the chunk containing delta is masked from it
    // on. All loads first (positions before the lag read the padding in front of the buffer and
    // are masked out), then one compare and ballot per chunk. The per-lag mask work is scalar and
    // the CU's one scalar unit serves all waves, so it is kept to a few instructions per chunk.
    const int c_min = delta >> 6;
    int ysrc[kChunks];
#pragma unroll
    for (int c = 0; c < kChunks; ++c) ysrc[c] = yw[64 * c + lane - delta];
    int R = 0;  // run of ones starting at bit 0 of the chunk after the current one
#pragma unroll
    for (int c = kChunks - 1; c >= 0; --c) {
      if (c < c_min) break;  // no position >= delta below this chunk
      unsigned long long E = __ballot(ysrc[c] == yown[c]) & in_win[c];
      if (c == c_min) E &= ~0ull << (delta & 63);
      if (E == 0ull) {  // no runs here (most lags of non-repeating text)
        R = 0;
        continue;
      }
      const int tt = trailing_ones(E >> lane);
      const int run = tt >= 64 - lane ? (64 - lane) + R : tt;
      ell[c] = max(ell[c], run);
      R = E == ~0ull ? 64 + R : trailing_ones(E);
    }
  }
#pragma unroll
  for (int c = 0; c < kChunks; ++c)
    if (c < nch && 64 * c + lane < m) ellw[wave][64 * c + lane] = ell[c];
  __syncthreads();
  // ell over all lags; slot m terminates the parse below.
  for (int i = tid; i < m; i += kDetThreads) {
    int e = ellw[0][i];
#pragma unroll
    for (int w = 1; w < kDetWaves; ++w) e = max(e, ellw[w][i]);
    ellmax[i] = e;
  }
  __syncthreads();

  // Distinct tokens and novelty.
  int uloc = 0, nloc = 0, rloc = 0;
  const int nov_lo = max(g - 1, m - p.nov_span);  // window index of the first examined position
  for (int i = tid; i < m; i += kDetThreads) {
    uloc += ellmax[i] >= 1 ? 0 : 1;
    if (i >= nov_lo) {
      rloc += 1;
      nloc += ellmax[i - g + 1] >= g ? 0 : 1;
    }
  }
  const int distinct = block_sum(uloc, red);
  const int novel = block_sum(nloc, red);
  const int nov_r = block_sum(rloc, red);

  // Greedy LZ parse by pointer doubling: cost of the parse from i to the end of the window.
  int lz_cost = gst.cr_cost, lz_m = gst.cr_m;
  if (do_cr) {
    for (int i = tid; i <= m; i += kDetThreads) {
      if (i == m) { nxt[0][i] = m; cst[0][i] = 0; }
      else {
        const int e = ellmax[i];
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

  // ---- trailing self-alignment L_P, P = 1 .. rep_pmax ----
  // L_P = largest k <= min(H - P, n - P - t0) with y[n-1-r] == y[n-1-r-P] for all r < k.
  const bool incremental = gst.tail_n == n - 1 && gst.tail_t0 == t0 && gst.tail_horizon == H &&
                           gst.tail_pmax == p.rep_pmax;
  __shared__ int Lsh[kMaxPeriod];
  if (incremental) {
    const int ylast = nbuf > 0 ? y[(n - 1) - lo_all] : 0;
    for (int P = tid + 1; P <= p.rep_pmax; P += kDetThreads) {
      const int kmax = min(H - P, n - P - t0);
      const bool eq = kmax > 0 && y[(n - 1 - P) - lo_all] == ylast;
      Lsh[P - 1] = eq ? min(gst.tail_run[P - 1] + 1, kmax) : 0;
    }
  } else {
    for (int P = wave + 1; P <= p.rep_pmax; P += kDetWaves) {
      const int kmax = max(0, min(H - P, n - P - t0));
      int Lp = kmax;
      for (int r0 = 0; r0 < kmax; r0 += 256) {
        unsigned long long miss[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int r = r0 + 64 * q + lane;
          const bool eq = r < kmax && y[(n - 1 - r) - lo_all] == y[(n - 1 - r - P) - lo_all];
          miss[q] = __ballot(!eq);
        }
        int hit = -1;
#pragma unroll
        for (int q = 3; q >= 0; --q)
          if (miss[q]) hit = 64 * q + __builtin_ctzll(miss[q]);
        if (hit >= 0) { Lp = min(kmax, r0 + hit); break; }
      }
      if (lane == 0) Lsh[P - 1] = Lp;
    }
  }
  __syncthreads();
  // qualifying period with the longest tail, ties to the smallest P: maximise T * 1024 + (1023 - P)
  int key = 0;
  for (int P = tid + 1; P <= p.rep_pmax; P += kDetThreads) {
    const int Lp = Lsh[P - 1];
    const int TP = Lp + P;
    if (Lp >= (p.rep_min_copies - 1) * P && TP >= p.rep_min_len) key = max(key, TP * 1024 + (1023 - P));
  }
  key = block_max(key, red);
  for (int P = tid + 1; P <= p.rep_pmax; P += kDetThreads) a.state[b].tail_run[P - 1] = Lsh[P - 1];

  if (tid == 0) {
    StateHeader st;
    st.streak = gst.streak; st.stall = gst.stall; st.rep = gst.rep; st.n_int = gst.n_int;
    st.n_last = gst.n_last; st.level = gst.level; st.cr_valid = gst.cr_valid;
    st.cr_cost = gst.cr_cost; st.cr_m = gst.cr_m;
    const int Ps = key > 0 ? 1023 - (key & 1023) : 0;
    const int Ts = key > 0 ? key >> 10 : 0;
    const int vote_ttr = (long long)p.ttr_den * distinct < (long long)p.ttr_num * m;
    if (do_cr) { st.cr_cost = lz_cost; st.cr_m = lz_m; st.cr_valid = 1; }
    const int vote_cr = (long long)p.cr_den * st.cr_cost < (long long)p.cr_num * st.cr_m;
    const float c = a.conf ? a.conf[b] : 0.f;
    const int attend_error = c != c;  // NaN: an attention call of this step failed for b
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
    fire = fire && !attend_error;
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
    d.attend_error = attend_error;
    d.reserved = 0;
    a.decision[b] = d;
    // header fields only: the tail runs were written above by all lanes
    lg_guard_state* out = &a.state[b];
    out->streak = st.streak; out->stall = st.stall; out->rep = st.rep; out->n_int = st.n_int;
    out->n_last = st.n_last; out->level = st.level; out->cr_valid = st.cr_valid;
    out->cr_cost = st.cr_cost; out->cr_m = st.cr_m; out->tail_n = n;
    out->tail_t0 = t0; out->tail_horizon = H; out->tail_pmax = p.rep_pmax;
    if (a.conf) a.conf[b] = 0.f;  // consumed: the next step max-accumulates from zero
  }
}

template <int kChunks>
__global__ __launch_bounds__(kDetThreads) void detect_kernel(DetectArgs a) {
  detect_block<kChunks>(a);
}

// The detector and the keep set of one sequence in one launch (lg_detect_and_prune): the keep set
// reads the decision that the detector has just written (visible to the workgroup after the
// barrier) and runs with the detector's kDetThreads threads.
template <int kChunks>
__global__ __launch_bounds__(kDetThreads) void detect_keep_kernel(DetectArgs a, KeepArgs k) {
  detect_block<kChunks>(a);
  __syncthreads();
  keep_set_block<kDetThreads>(k);
}

static DetectArgs detect_args(const lg_guard_params* p, const int32_t* tokens, int ring,
                              const int32_t* t, const int32_t* t0, float* conf,
                              lg_guard_state* state, lg_decision* decision) {
  DetectArgs a;
  a.p = *p;
  a.tokens = tokens;
  a.ring = ring;
  a.t = t;
  a.t0 = t0;
  a.conf = conf;
  a.state = state;
  a.decision = decision;
  return a;
}

hipError_t launch_detect(const lg_guard_params* p, int batch, const int32_t* tokens, int ring,
                         const int32_t* t, const int32_t* t0, float* conf, lg_guard_state* state,
                         lg_decision* decision, hipStream_t st) {
  const DetectArgs a = detect_args(p, tokens, ring, t, t0, conf, state, decision);
  if (p->W <= 256)
    hipLaunchKernelGGL(detect_kernel<4>, dim3(batch), dim3(kDetThreads), 0, st, a);
  else
    hipLaunchKernelGGL(detect_kernel<8>, dim3(batch), dim3(kDetThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_detect_prune(const lg_guard_params* p, int batch, const int32_t* tokens,
                               int ring, const int32_t* t, const int32_t* t0, float* conf,
                               lg_guard_state* state, lg_decision* decision, int cap,
                               int n_layers, const lg_layer_cache* layers, int32_t* pos,
                               int32_t* len, const int32_t* budget, const int32_t* t_append,
                               int32_t* keep_idx, int32_t* new_len, hipStream_t st) {
  const DetectArgs a = detect_args(p, tokens, ring, t, t0, conf, state, decision);
  const KeepArgs ka = keep_args(p, batch, cap, n_layers, pos, len, budget, t_append, decision,
                                keep_idx, new_len);
  hipError_t e = ka.have_scores ? launch_h2o_scores(ka, n_layers, layers, st) : hipSuccess;
  if (e != hipSuccess) return e;
  if (p->W <= 256)
    hipLaunchKernelGGL(detect_keep_kernel<4>, dim3(batch), dim3(kDetThreads), 0, st, a, ka);
  else
    hipLaunchKernelGGL(detect_keep_kernel<8>, dim3(batch), dim3(kDetThreads), 0, st, a, ka);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_compact(ka, n_layers, layers, st);
}

}  // namespace lg

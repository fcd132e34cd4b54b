// lg_keepset.h -- the keep set of Stage 2 (Sec. 5.3, Eq. (10) and Eq. (11)) as a workgroup-level
// device routine, shared by the prune launch (keepset_kernel) and the fused detector launch
// (lg_detect.hip). See the file comment of lg_prune.hip for the algorithm.
#pragma once

#include "lg_internal.h"

namespace lg {

constexpr int kPruneThreads = 256;

struct KeepArgs {
  int32_t n_anchor, recent_div, sparse_div, policy, have_scores;
  int32_t B, cap;
  int32_t* pos;
  int32_t* len;
  const int32_t* budget;
  const int32_t* t_append;
  const lg_decision* decision;
  int32_t* keep_idx;
  int32_t* new_len;
};

inline KeepArgs keep_args(const lg_guard_params* p, int batch, int cap, int n_layers,
                          int32_t* pos, int32_t* len, const int32_t* budget,
                          const int32_t* t_append, const lg_decision* decision,
                          int32_t* keep_idx, int32_t* new_len) {
  KeepArgs ka;
  ka.n_anchor = p->n_anchor;
  ka.recent_div = p->recent_div;
  ka.sparse_div = p->sparse_div;
  ka.policy = p->policy;
  ka.have_scores = (p->policy == LG_POLICY_H2O && n_layers > 0) ? 1 : 0;
  ka.B = batch;
  ka.cap = cap;
  ka.pos = pos;
  ka.len = len;
  ka.budget = budget;
  ka.t_append = t_append;
  ka.decision = decision;
  ka.keep_idx = keep_idx;
  ka.new_len = new_len;
  return ka;
}

// Exclusive prefix sum over the TPB lanes of the workgroup; *total gets the sum.
template <int TPB>
__device__ __forceinline__ int block_exclusive_scan(int x, int* total, int* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o, 64);
    if (lane >= o) inc += y;
  }
  __syncthreads();
  if (lane == 63) red[wave] = inc;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < TPB / 64; ++w) {
    if (w < wave) before += red[w];
    tot += red[w];
  }
  *total = tot;
  return before + inc - x;
}

template <int TPB>
__device__ __forceinline__ int block_count(int x, int* red) {
  int tot;
  (void)block_exclusive_scan<TPB>(x, &tot, red);
  return tot;
}

// Is rank r one of floor(k*M/S), k = 0..S-1 (M > S > 0)? The ranks are strictly increasing in k,
// so r is hit iff k = ceil(r*S/M) maps back onto it.
__device__ __forceinline__ bool sparse_hit(int r, int M, int S) {
  const long long k = ((long long)r * S + M - 1) / M;
  return k < S && (k * M) / S == r;
}

// Keys of the H2O order: the score as an order-preserving unsigned integer (float order, -0 below
// +0) above the slot index, so equal scores rank the later slot (higher position) first.
__device__ __forceinline__ unsigned long long h2o_key(const int32_t* scores, int j, bool have) {
  uint32_t u = have ? (uint32_t)scores[j] : 0u;
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((unsigned long long)u << 32) | (uint32_t)j;
}

// The need-th largest key among slots [0, n) (1 <= need <= n): 8-bit digits from the top, one
// histogram pass per digit over the keys that match the digits found so far; the digit holding
// the need-th largest is found with a block scan over the bins from the top.
template <int TPB>
__device__ unsigned long long radix_select_desc(const int32_t* scores, bool have, int n, int need,
                                                unsigned int* hist, unsigned long long* s_prefix,
                                                int* s_need, int* red) {
  static_assert(TPB >= 256, "one thread per 8-bit bin");
  const int tid = threadIdx.x;
  unsigned long long prefix = 0;
  for (int shift = 56; shift >= 0; shift -= 8) {
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    for (int j = tid; j < n; j += TPB) {
      const unsigned long long key = h2o_key(scores, j, have);
      if (shift == 56 || (key >> (shift + 8)) == (prefix >> (shift + 8)))
        atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    const int d = 255 - tid;  // thread tid < 256 looks at digit d, larger digits first
    const int cnt = tid < 256 ? (int)hist[d] : 0;
    int tot;
    const int above = block_exclusive_scan<TPB>(cnt, &tot, red);  // keys with a larger digit
    if (tid < 256 && above < need && above + cnt >= need) {
      *s_need = need - above;
      *s_prefix = prefix | ((unsigned long long)d << shift);
    }
    __syncthreads();
    prefix = *s_prefix;
    need = *s_need;
    __syncthreads();
  }
  return prefix;
}

// The keep set of sequence blockIdx.x (see the file comment of lg_prune.hip), by the TPB
// threads of the workgroup.
template <int TPB>
__device__ void keep_set_block(const KeepArgs& a) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  __shared__ int sh[6];
  __shared__ int red[TPB / 64];
  int32_t* pos = a.pos + (size_t)b * a.cap;
  int32_t* kidx = a.keep_idx + (size_t)b * a.cap;
  if (tid == 0) {
    int L = a.len[b];
    L = L < 0 ? 0 : (L > a.cap ? a.cap : L);
    if (a.t_append != nullptr) {
      if (L < a.cap) {
        pos[L] = a.t_append[b];
        L += 1;
      }
      a.len[b] = L;
    }
    const int trig = a.policy == LG_POLICY_LOOPGUARD && a.decision != nullptr && a.decision[b].trigger;
    // a budget above the cache's capacity acts as the capacity, so a full cache is pruned
    const int flag = trig ? 1 : (L >= min(a.budget[b], a.cap) ? 2 : 0);
    sh[0] = L;
    sh[1] = flag;
    sh[2] = trig ? a.decision[b].span_lo : -1;
    sh[3] = trig ? min(max(a.decision[b].level, 0), 30) : 0;
    sh[4] = L > 0 ? pos[L - 1] : 0;
  }
  __syncthreads();
  const int L = sh[0], flag = sh[1], span = sh[2], level = sh[3], t = sh[4];
  if (flag == 0) {
    if (tid == 0) a.new_len[b] = -1;
    return;
  }
  const int budget = min(a.budget[b], a.cap);
  const int R = budget / a.recent_div;
  const int thrR = sat_sub(sat_sub(t, R), -1);  // t - R + 1
  // The kept set leaves room for the next append: at most budget - 1 slots (LoopGuard: claimed by
  // the anchors first, then the recent window, then the sparse history; the baselines: their keep
  // size capped). With the paper's constants nothing is cut.
  const int cap_k = max(0, budget - 1);
  const int Ktot = min(budget / a.sparse_div + budget / a.recent_div, cap_k);  // baselines
  int S = 0, Br = 0, A_keep = 0;

  int M = 0, c_first = 0;
  int win_lo = 0, n_anchor_slots = 0;       // StreamingLLM
  int older = 0;                            // H2O: slots [0, older) are ranked by score
  bool keep_all_older = true;
  unsigned long long thr_key = 0;
  const bool have = a.have_scores != 0;
  if (a.policy == LG_POLICY_LOOPGUARD) {
    // Pass 1: sizes of the anchor prefix, the middle region and the clean recent window.
    int aloc = 0, mloc = 0, cloc = 0;
    for (int j = tid; j < L; j += TPB) {
      const int pj = pos[j];
      const bool A = pj < a.n_anchor;
      const bool Rc = !A && pj >= thrR;
      const bool bad = Rc && span >= 0 && pj >= span;
      aloc += A ? 1 : 0;
      mloc += (!A && !Rc) ? 1 : 0;
      cloc += (Rc && !bad) ? 1 : 0;
    }
    const int NA = block_count<TPB>(aloc, red);
    M = block_count<TPB>(mloc, red);
    const int C = block_count<TPB>(cloc, red);
    A_keep = min(NA, cap_k);
    Br = min(R >> level, cap_k - A_keep);
    S = max(0, min(budget / a.sparse_div - a.n_anchor, cap_k - A_keep - Br));
    c_first = C - min(Br, C);  // clean recent slots with rank >= c_first are kept
  } else if (a.policy == LG_POLICY_STREAMING) {
    int aloc = 0;
    for (int j = tid; j < L; j += TPB) aloc += pos[j] < a.n_anchor ? 1 : 0;
    n_anchor_slots = min(block_count<TPB>(aloc, red), Ktot);  // a prefix of the slots (positions ascend)
    const int window = max(0, Ktot - n_anchor_slots);
    win_lo = max(n_anchor_slots, L - window);
  } else {
    __shared__ unsigned int hist[256];
    __shared__ unsigned long long s_prefix;
    __shared__ int s_need;
    const int Rp = min(min(R, L), Ktot);
    older = L - Rp;
    const int heavy = max(0, Ktot - Rp);
    keep_all_older = older <= heavy;
    if (!keep_all_older && heavy > 0)
      thr_key = radix_select_desc<TPB>(kidx, have, older, heavy, hist, &s_prefix, &s_need, red);
    else if (!keep_all_older)
      thr_key = ~0ull;  // keep none of the older slots (never reached with K >= R)
  }

  // Pass 2: ranks and the kept list, 256 slots at a time.
  int mid_base = 0, cr_base = 0, out_base = 0;
  for (int j0 = 0; j0 < L; j0 += TPB) {
    const int j = j0 + tid;
    bool A = false, Mid = false, Cr = false, keep = false;
    if (j < L) {
      const int pj = pos[j];
      if (a.policy == LG_POLICY_LOOPGUARD) {
        A = pj < a.n_anchor;
        const bool Rc = !A && pj >= thrR;
        const bool bad = Rc && span >= 0 && pj >= span;
        Mid = !A && !Rc;
        Cr = Rc && !bad;
      } else if (a.policy == LG_POLICY_STREAMING) {
        keep = j < n_anchor_slots || j >= win_lo;
      } else {
        keep = j >= older || keep_all_older || h2o_key(kidx, j, have) >= thr_key;
      }
    }
    int mtot, ctot;
    const int mrank = mid_base + block_exclusive_scan<TPB>(Mid ? 1 : 0, &mtot, red);
    const int crank = cr_base + block_exclusive_scan<TPB>(Cr ? 1 : 0, &ctot, red);
    if (A) keep = j < A_keep;  // the anchors are a prefix of the slots
    if (Mid) keep = (M <= S) || sparse_hit(mrank, M, S);
    if (Cr) keep = crank >= c_first;
    int ktot;
    const int slot = out_base + block_exclusive_scan<TPB>(keep ? 1 : 0, &ktot, red);
    if (keep) kidx[slot] = j;
    mid_base += mtot;
    cr_base += ctot;
    out_base += ktot;
  }
  __syncthreads();
  // Gather pos in place (ascending chunks, read all before writing).
  for (int r0 = 0; r0 < out_base; r0 += TPB) {
    const int r = r0 + tid;
    int v = 0;
    if (r < out_base) v = pos[kidx[r]];
    __syncthreads();
    if (r < out_base) pos[r] = v;
    __syncthreads();
  }
  if (tid == 0) {
    a.new_len[b] = out_base;
    a.len[b] = out_base;
  }
}

// Host side of a prune, around the keep set (lg_prune.hip): the H2O scores it ranks (baseline
// policy H2O) and the compaction of every layer's rows by the kept list.
hipError_t launch_h2o_scores(const KeepArgs& ka, int n_layers, const lg_layer_cache* layers,
                             hipStream_t st);
hipError_t launch_compact(const KeepArgs& ka, int n_layers, const lg_layer_cache* layers,
                          hipStream_t st);

}  // namespace lg

// lg_prune.hip -- Stage 2 of LoopGuard: the retained index set and in-place cache compaction
// (Sec. 5.3, Eq. (10) and Eq. (11)), plus the per-step commit of the appended row and budget
// upkeep.
//
// keepset_kernel (one workgroup per sequence): commit the append, decide whether the sequence is
// pruned (trigger, or cache at its budget), mark every live slot as anchor / recent window / bad
// tail / middle from its position, and stream-compact the kept slots with block-wide prefix sums:
//   kept(j) = anchor(j) or (middle(j) and rank_mid(j) is one of the S evenly spaced ranks) or
//             (clean recent(j) and it is among the last R >> l clean recent slots)
// The kept slot list is written to keep_idx; pos is gathered in place.
//
// With the baseline policies (H2O, StreamingLLM; Sec. 6.1) only a cache at its budget is pruned and
// the kept set is the policy's: h2o_score_kernel first sums every slot's acc over the layers and KV
// heads into keep_idx (float bits, used as scratch), and keepset_kernel finds the H2O threshold
// key by an 8-bit radix select over (score, slot) keys before the same stream compaction.
//
// compact_kernel (one workgroup per (kv head, sequence, layer)): moves K, V and acc rows
// r <- keep_idx[r] in place. keep_idx is ascending with keep_idx[r] >= r, so walking the rows in
// chunks, reading a whole chunk before writing it, never overwrites a row a later chunk reads;
// the next chunk's loads are issued before the current chunk's stores.
#include "lg_internal.h"

namespace lg {

constexpr int kPruneThreads = 256;
constexpr int kMaxLayersPerLaunch = 64;

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

struct ScoreArgs {
  const float* acc[kMaxLayersPerLaunch];
  int32_t n_layers, first;  // layers in this launch; the first launch writes, later ones add
  int32_t B, Hkv, cap;
  const int32_t* len;
  const int32_t* budget;
  const int32_t* t_append;
  float* score;             // keep_idx viewed as float [B][cap]
};

// Live slots after the commit of the append, as keepset_kernel computes them.
__device__ __forceinline__ int committed_len(const int32_t* len, const int32_t* t_append, int b,
                                             int cap) {
  int L = len[b];
  L = L < 0 ? 0 : (L > cap ? cap : L);
  if (t_append != nullptr && L < cap) L += 1;
  return L;
}

// H2O score of every live slot of a sequence at its budget: acc summed over this launch's layers
// (ascending) and KV heads (ascending) in float32, added to the previous launches' partial sum.
__global__ __launch_bounds__(256) void h2o_score_kernel(ScoreArgs a) {
  const int b = blockIdx.y;
  const int L = committed_len(a.len, a.t_append, b, a.cap);
  if (L < a.budget[b]) return;  // not pruned at this step
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= L) return;
  float* sc = a.score + (size_t)b * a.cap;
  float s = a.first ? 0.f : sc[j];
  // Terms i = l * Hkv + h in ascending order; each chunk of kChunk terms is loaded before it is
  // added, so the loads are in flight together while the additions keep their order.
  constexpr int kChunk = 16;
  const int total = a.n_layers * a.Hkv;
  const size_t row = (size_t)b * a.Hkv * a.cap + j;
  for (int i0 = 0; i0 < total; i0 += kChunk) {
    float v[kChunk];
#pragma unroll
    for (int k = 0; k < kChunk; ++k) {
      const int i = i0 + k;
      if (i < total) {
        const int l = i / a.Hkv, h = i - l * a.Hkv;
        v[k] = a.acc[l][row + (size_t)h * a.cap];
      }
    }
#pragma unroll
    for (int k = 0; k < kChunk; ++k)
      if (i0 + k < total) s = s + v[k];
  }
  sc[j] = s;
}

struct CompactLayer {
  void* k;
  void* v;
  float* acc;
};

struct CompactArgs {
  CompactLayer layer[kMaxLayersPerLaunch];
  const int32_t* keep_idx;
  const int32_t* new_len;
  int32_t B, Hkv, cap, row_bytes;
};

// Exclusive prefix sum over the 256 lanes of the workgroup; *total gets the sum.
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
  for (int w = 0; w < kPruneThreads / 64; ++w) {
    if (w < wave) before += red[w];
    tot += red[w];
  }
  *total = tot;
  return before + inc - x;
}

__device__ __forceinline__ int block_count(int x, int* red) {
  int tot;
  (void)block_exclusive_scan(x, &tot, red);
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
__device__ unsigned long long radix_select_desc(const int32_t* scores, bool have, int n, int need,
                                                unsigned int* hist, unsigned long long* s_prefix,
                                                int* s_need, int* red) {
  static_assert(kPruneThreads == 256, "one thread per 8-bit bin");
  const int tid = threadIdx.x;
  unsigned long long prefix = 0;
  for (int shift = 56; shift >= 0; shift -= 8) {
    hist[tid] = 0;
    __syncthreads();
    for (int j = tid; j < n; j += kPruneThreads) {
      const unsigned long long key = h2o_key(scores, j, have);
      if (shift == 56 || (key >> (shift + 8)) == (prefix >> (shift + 8)))
        atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    const int d = 255 - tid;  // thread tid looks at digit d, larger digits first
    const int cnt = (int)hist[d];
    int tot;
    const int above = block_exclusive_scan(cnt, &tot, red);  // keys with a larger digit
    if (above < need && above + cnt >= need) {
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

__global__ __launch_bounds__(kPruneThreads) void keepset_kernel(KeepArgs a) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  __shared__ int sh[6];
  __shared__ int red[kPruneThreads / 64];
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
    const int flag = trig ? 1 : (L >= a.budget[b] ? 2 : 0);
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
  const int budget = a.budget[b];
  const int R = budget / a.recent_div;
  const int S = max(0, budget / a.sparse_div - a.n_anchor);
  const int Br = R >> level;
  const int thrR = sat_sub(sat_sub(t, R), -1);  // t - R + 1
  const int Ktot = budget / a.sparse_div + budget / a.recent_div;  // baseline policies' keep size

  int M = 0, c_first = 0;
  int win_lo = 0, n_anchor_slots = 0;       // StreamingLLM
  int older = 0;                            // H2O: slots [0, older) are ranked by score
  bool keep_all_older = true;
  unsigned long long thr_key = 0;
  const bool have = a.have_scores != 0;
  if (a.policy == LG_POLICY_LOOPGUARD) {
    // Pass 1: sizes of the middle region and of the clean recent window.
    int mloc = 0, cloc = 0;
    for (int j = tid; j < L; j += kPruneThreads) {
      const int pj = pos[j];
      const bool A = pj < a.n_anchor;
      const bool Rc = !A && pj >= thrR;
      const bool bad = Rc && span >= 0 && pj >= span;
      mloc += (!A && !Rc) ? 1 : 0;
      cloc += (Rc && !bad) ? 1 : 0;
    }
    M = block_count(mloc, red);
    const int C = block_count(cloc, red);
    c_first = C - min(Br, C);  // clean recent slots with rank >= c_first are kept
  } else if (a.policy == LG_POLICY_STREAMING) {
    int aloc = 0;
    for (int j = tid; j < L; j += kPruneThreads) aloc += pos[j] < a.n_anchor ? 1 : 0;
    n_anchor_slots = block_count(aloc, red);  // a prefix of the slots (positions ascend)
    const int window = max(0, Ktot - n_anchor_slots);
    win_lo = max(n_anchor_slots, L - window);
  } else {
    __shared__ unsigned int hist[kPruneThreads];
    __shared__ unsigned long long s_prefix;
    __shared__ int s_need;
    const int Rp = min(R, L);
    older = L - Rp;
    const int heavy = max(0, Ktot - Rp);
    keep_all_older = older <= heavy;
    if (!keep_all_older && heavy > 0)
      thr_key = radix_select_desc(kidx, have, older, heavy, hist, &s_prefix, &s_need, red);
    else if (!keep_all_older)
      thr_key = ~0ull;  // keep none of the older slots (never reached with K >= R)
  }

  // Pass 2: ranks and the kept list, 256 slots at a time.
  int mid_base = 0, cr_base = 0, out_base = 0;
  for (int j0 = 0; j0 < L; j0 += kPruneThreads) {
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
    const int mrank = mid_base + block_exclusive_scan(Mid ? 1 : 0, &mtot, red);
    const int crank = cr_base + block_exclusive_scan(Cr ? 1 : 0, &ctot, red);
    if (A) keep = true;
    if (Mid) keep = (M <= S) || sparse_hit(mrank, M, S);
    if (Cr) keep = crank >= c_first;
    int ktot;
    const int slot = out_base + block_exclusive_scan(keep ? 1 : 0, &ktot, red);
    if (keep) kidx[slot] = j;
    mid_base += mtot;
    cr_base += ctot;
    out_base += ktot;
  }
  __syncthreads();
  // Gather pos in place (ascending chunks, read all before writing).
  for (int r0 = 0; r0 < out_base; r0 += kPruneThreads) {
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

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
constexpr int kCompactUnroll = 8;  // row groups per compaction pass (rows in flight per thread)

// Rows of a compaction pass, held in registers between its loads and its stores.
template <int U>
struct MovePass {
  uint4 k[U], v[U];
  float acc[U];
  int src[U];
};

template <int TPR, int U>
__device__ __forceinline__ void compact_load(MovePass<U>& m, int r0, int rsub, int piece, int nl,
                                             const int32_t* kidx, const uint4* K, const uint4* V,
                                             const float* acc) {
  constexpr int RPP = kPruneThreads / TPR;
#pragma unroll
  for (int u = 0; u < U; ++u) {  // all source indices first: one wait before the row loads
    const int r = r0 + u * RPP + rsub;
    m.src[u] = r < nl ? kidx[r] : r;
  }
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int r = r0 + u * RPP + rsub;
    if (m.src[u] != r) {  // rows are read once: non-temporal
      const u32x4_t k4 = __builtin_nontemporal_load((const u32x4_t*)(K + (size_t)m.src[u] * TPR + piece));
      const u32x4_t v4 = __builtin_nontemporal_load((const u32x4_t*)(V + (size_t)m.src[u] * TPR + piece));
      m.k[u] = make_uint4(k4.x, k4.y, k4.z, k4.w);
      m.v[u] = make_uint4(v4.x, v4.y, v4.z, v4.w);
      m.acc[u] = acc[m.src[u]];
    }
  }
}

template <int TPR, int U>
__device__ __forceinline__ void compact_store(const MovePass<U>& m, int r0, int rsub, int piece,
                                              uint4* K, uint4* V, float* acc) {
  constexpr int RPP = kPruneThreads / TPR;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int r = r0 + u * RPP + rsub;
    if (m.src[u] != r) {  // non-temporal: the rows are next read by a streaming attention sweep
      __builtin_nontemporal_store(u32x4_t{m.k[u].x, m.k[u].y, m.k[u].z, m.k[u].w},
                                  (u32x4_t*)(K + (size_t)r * TPR + piece));
      __builtin_nontemporal_store(u32x4_t{m.v[u].x, m.v[u].y, m.v[u].z, m.v[u].w},
                                  (u32x4_t*)(V + (size_t)r * TPR + piece));
      if (piece == 0) acc[r] = m.acc[u];
    }
  }
}

// Passes of RPP * U rows in ascending order. Pass p writes rows [r0, r0 + RPP*U) and may read
// them as sources, so its loads must all complete before any of its stores (one barrier per
// pass); its sources are >= its rows, and the next pass's sources are >= the next pass's rows,
// which lie above every row pass p writes, so the next pass's loads are issued before pass p's
// stores.
template <int TPR, int U>
__global__ __launch_bounds__(kPruneThreads) void compact_kernel(CompactArgs a) {
  // Grid (layer, kv head, sequence), the layer fastest: the dispatcher deals consecutive
  // workgroups round-robin to the 8 XCDs, so the rows of one flagged sequence (the usual event)
  // spread over all of them.
  const int l = blockIdx.x, hkv = blockIdx.y, b = blockIdx.z;
  const int nl = a.new_len[b];
  if (nl <= 0) return;
  constexpr int RPP = kPruneThreads / TPR;  // rows per pass and unroll step
  constexpr int ROWS = RPP * U;             // rows per pass
  const int tid = threadIdx.x;
  const int rsub = tid / TPR, piece = tid % TPR;
  const size_t bk = (size_t)b * a.Hkv + hkv;
  uint4* K = (uint4*)((char*)a.layer[l].k + bk * a.cap * (size_t)a.row_bytes);
  uint4* V = (uint4*)((char*)a.layer[l].v + bk * a.cap * (size_t)a.row_bytes);
  float* acc = a.layer[l].acc + bk * a.cap;
  const int32_t* kidx = a.keep_idx + (size_t)b * a.cap;
  MovePass<U> cur, nxt;
  compact_load<TPR, U>(cur, 0, rsub, piece, nl, kidx, K, V, acc);
  for (int r0 = 0; r0 < nl; r0 += ROWS) {
    __syncthreads();  // every thread holds this pass's rows
    const bool more = r0 + ROWS < nl;
    if (more) compact_load<TPR, U>(nxt, r0 + ROWS, rsub, piece, nl, kidx, K, V, acc);
    compact_store<TPR, U>(cur, r0, rsub, piece, K, V, acc);
    if (more) cur = nxt;
  }
}

hipError_t launch_prune(const lg_guard_params* p, int batch, int cap, int n_layers,
                        const lg_layer_cache* layers, int32_t* pos, int32_t* len,
                        const int32_t* budget, const int32_t* t_append,
                        const lg_decision* decision, int32_t* keep_idx, int32_t* new_len,
                        hipStream_t st) {
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
  if (ka.have_scores) {
    // H2O scores into keep_idx (as float bits), 64 layers per launch, added in layer order.
    for (int l0 = 0; l0 < n_layers; l0 += kMaxLayersPerLaunch) {
      ScoreArgs sa;
      sa.n_layers = min(kMaxLayersPerLaunch, n_layers - l0);
      for (int i = 0; i < sa.n_layers; ++i) sa.acc[i] = layers[l0 + i].acc;
      sa.first = l0 == 0;
      sa.B = batch;
      sa.Hkv = layers[0].n_kv_heads;
      sa.cap = cap;
      sa.len = len;
      sa.budget = budget;
      sa.t_append = t_append;
      sa.score = (float*)keep_idx;
      hipLaunchKernelGGL(h2o_score_kernel, dim3((cap + 255) / 256, batch), dim3(256), 0, st, sa);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  hipLaunchKernelGGL(keepset_kernel, dim3(batch), dim3(kPruneThreads), 0, st, ka);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || n_layers == 0) return e;
  const int Hkv = layers[0].n_kv_heads;
  const int row_bytes = layers[0].head_dim * (layers[0].dtype == LG_BF16 ? 2 : 4);
  for (int l0 = 0; l0 < n_layers; l0 += kMaxLayersPerLaunch) {
    const int nl = min(kMaxLayersPerLaunch, n_layers - l0);
    CompactArgs ca;
    for (int i = 0; i < nl; ++i) {
      ca.layer[i].k = layers[l0 + i].k;
      ca.layer[i].v = layers[l0 + i].v;
      ca.layer[i].acc = layers[l0 + i].acc;
    }
    ca.keep_idx = keep_idx;
    ca.new_len = new_len;
    ca.B = batch;
    ca.Hkv = Hkv;
    ca.cap = cap;
    ca.row_bytes = row_bytes;
    dim3 grid(nl, Hkv, batch);
    switch (row_bytes / 16) {
      case 8: hipLaunchKernelGGL((compact_kernel<8, kCompactUnroll>), grid, dim3(kPruneThreads), 0, st, ca); break;
      case 16: hipLaunchKernelGGL((compact_kernel<16, kCompactUnroll>), grid, dim3(kPruneThreads), 0, st, ca); break;
      default: hipLaunchKernelGGL((compact_kernel<32, kCompactUnroll>), grid, dim3(kPruneThreads), 0, st, ca); break;
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace lg

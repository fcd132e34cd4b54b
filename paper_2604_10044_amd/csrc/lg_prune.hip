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
// compact_kernel (one workgroup per (kv head, sequence, layer)): moves K, V and acc rows
// r <- keep_idx[r] in place. keep_idx is ascending with keep_idx[r] >= r, so walking the rows in
// chunks, reading a whole chunk before writing it, never overwrites a row a later chunk reads.
#include "lg_internal.h"

namespace lg {

constexpr int kPruneThreads = 256;
constexpr int kMaxLayersPerLaunch = 64;

struct KeepArgs {
  int32_t n_anchor, recent_div, sparse_div;
  int32_t B, cap;
  int32_t* pos;
  int32_t* len;
  const int32_t* budget;
  const int32_t* t_append;
  const lg_decision* decision;
  int32_t* keep_idx;
  int32_t* new_len;
};

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
    const int trig = (a.decision != nullptr) && a.decision[b].trigger;
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
  const int thrR = t - R + 1;

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
  const int M = block_count(mloc, red);
  const int C = block_count(cloc, red);
  const int c_first = C - min(Br, C);  // clean recent slots with rank >= c_first are kept

  // Pass 2: ranks and the kept list, 256 slots at a time.
  int mid_base = 0, cr_base = 0, out_base = 0;
  for (int j0 = 0; j0 < L; j0 += kPruneThreads) {
    const int j = j0 + tid;
    bool A = false, Mid = false, Cr = false;
    if (j < L) {
      const int pj = pos[j];
      A = pj < a.n_anchor;
      const bool Rc = !A && pj >= thrR;
      const bool bad = Rc && span >= 0 && pj >= span;
      Mid = !A && !Rc;
      Cr = Rc && !bad;
    }
    int mtot, ctot;
    const int mrank = mid_base + block_exclusive_scan(Mid ? 1 : 0, &mtot, red);
    const int crank = cr_base + block_exclusive_scan(Cr ? 1 : 0, &ctot, red);
    bool keep = A;
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

template <int TPR, int U>
__global__ __launch_bounds__(kPruneThreads) void compact_kernel(CompactArgs a) {
  const int hkv = blockIdx.x, b = blockIdx.y, l = blockIdx.z;
  const int nl = a.new_len[b];
  if (nl <= 0) return;
  constexpr int RPP = kPruneThreads / TPR;  // rows per pass
  const int tid = threadIdx.x;
  const int rsub = tid / TPR, piece = tid % TPR;
  const size_t bk = (size_t)b * a.Hkv + hkv;
  uint4* K = (uint4*)((char*)a.layer[l].k + bk * a.cap * (size_t)a.row_bytes);
  uint4* V = (uint4*)((char*)a.layer[l].v + bk * a.cap * (size_t)a.row_bytes);
  float* acc = a.layer[l].acc + bk * a.cap;
  const int32_t* kidx = a.keep_idx + (size_t)b * a.cap;
  for (int r0 = 0; r0 < nl; r0 += RPP * U) {
    uint4 kv[U], vv[U];
    float av[U];
    int src[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = r0 + u * RPP + rsub;
      src[u] = r < nl ? kidx[r] : r;
      if (src[u] != r) {
        kv[u] = K[(size_t)src[u] * TPR + piece];
        vv[u] = V[(size_t)src[u] * TPR + piece];
        av[u] = acc[src[u]];
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = r0 + u * RPP + rsub;
      if (src[u] != r) {
        K[(size_t)r * TPR + piece] = kv[u];
        V[(size_t)r * TPR + piece] = vv[u];
        if (piece == 0) acc[r] = av[u];
      }
    }
    __syncthreads();
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
  ka.B = batch;
  ka.cap = cap;
  ka.pos = pos;
  ka.len = len;
  ka.budget = budget;
  ka.t_append = t_append;
  ka.decision = decision;
  ka.keep_idx = keep_idx;
  ka.new_len = new_len;
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
    dim3 grid(Hkv, batch, nl);
    switch (row_bytes / 16) {
      case 8: hipLaunchKernelGGL((compact_kernel<8, 4>), grid, dim3(kPruneThreads), 0, st, ca); break;
      case 16: hipLaunchKernelGGL((compact_kernel<16, 4>), grid, dim3(kPruneThreads), 0, st, ca); break;
      default: hipLaunchKernelGGL((compact_kernel<32, 4>), grid, dim3(kPruneThreads), 0, st, ca); break;
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace lg

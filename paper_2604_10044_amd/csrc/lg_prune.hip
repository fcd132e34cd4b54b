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
#include "lg_keepset.h"

namespace lg {

constexpr int kMaxLayersPerLaunch = 64;

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
  if (L < min(a.budget[b], a.cap)) return;  // not pruned at this step
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

__global__ __launch_bounds__(kPruneThreads) void keepset_kernel(KeepArgs a) {
  keep_set_block<kPruneThreads>(a);
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

hipError_t launch_h2o_scores(const KeepArgs& ka, int n_layers, const lg_layer_cache* layers,
                             hipStream_t st) {
  // H2O scores into keep_idx (as float bits), 64 layers per launch, added in layer order.
  for (int l0 = 0; l0 < n_layers; l0 += kMaxLayersPerLaunch) {
    ScoreArgs sa;
    sa.n_layers = min(kMaxLayersPerLaunch, n_layers - l0);
    for (int i = 0; i < sa.n_layers; ++i) sa.acc[i] = layers[l0 + i].acc;
    sa.first = l0 == 0;
    sa.B = ka.B;
    sa.Hkv = layers[0].n_kv_heads;
    sa.cap = ka.cap;
    sa.len = ka.len;
    sa.budget = ka.budget;
    sa.t_append = ka.t_append;
    sa.score = (float*)ka.keep_idx;
    hipLaunchKernelGGL(h2o_score_kernel, dim3((ka.cap + 255) / 256, ka.B), dim3(256), 0, st, sa);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_compact(const KeepArgs& ka, int n_layers, const lg_layer_cache* layers,
                          hipStream_t st) {
  if (n_layers == 0) return hipSuccess;
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
    ca.keep_idx = ka.keep_idx;
    ca.new_len = ka.new_len;
    ca.B = ka.B;
    ca.Hkv = Hkv;
    ca.cap = ka.cap;
    ca.row_bytes = row_bytes;
    dim3 grid(nl, Hkv, ka.B);
    switch (row_bytes / 16) {
      case 8: hipLaunchKernelGGL((compact_kernel<8, kCompactUnroll>), grid, dim3(kPruneThreads), 0, st, ca); break;
      case 16: hipLaunchKernelGGL((compact_kernel<16, kCompactUnroll>), grid, dim3(kPruneThreads), 0, st, ca); break;
      default: hipLaunchKernelGGL((compact_kernel<32, kCompactUnroll>), grid, dim3(kPruneThreads), 0, st, ca); break;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_prune(const lg_guard_params* p, int batch, int cap, int n_layers,
                        const lg_layer_cache* layers, int32_t* pos, int32_t* len,
                        const int32_t* budget, const int32_t* t_append,
                        const lg_decision* decision, int32_t* keep_idx, int32_t* new_len,
                        hipStream_t st) {
  const KeepArgs ka = keep_args(p, batch, cap, n_layers, pos, len, budget, t_append, decision,
                                keep_idx, new_len);
  hipError_t e = ka.have_scores ? launch_h2o_scores(ka, n_layers, layers, st) : hipSuccess;
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(keepset_kernel, dim3(batch), dim3(kPruneThreads), 0, st, ka);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_compact(ka, n_layers, layers, st);
}

}  // namespace lg

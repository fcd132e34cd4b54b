// lg_attend.hip -- decode attention over the fixed-budget cache with fused loop statistics.
//
// Eq. (1) of the paper (Sec. 3.1) per query head over the live slots of the cache, plus the
// statistics the guard consumes, all from one sweep over K/V:
//   suffix mass   sum of alpha over slots with pos > t - w_s (attention on the narrow recent
//                 suffix; head locking, Sec. 1 and App. E)
//   H2O increment acc[j] += sum over the group's query heads of alpha_j (Sec. 2.2, Sec. 6.1)
//   confidence    conf[b] = max(conf[b], max_h suffix mass)
//
// The slots of each row (sequence, kv head) are cut into splits, one workgroup each. Three forms:
//   one-launch  (bfloat16) the row is finished in the same launch: by its own workgroup(s) when
//               it is a single split (the automatic choice for launches of at least 128 rows
//               whose cap fits one split), else by its splits exchanging their partials through
//               memory; no workgroup waits for one that may not have started (see the exchange
//               below).
//   merge       (bfloat16, the automatic choice otherwise) each split writes its partial and its
//               logits to memory and attend_combine_mfma merges them in a second launch.
//   portable    (float32 or bfloat16, any cap) attend_valu + attend_combine.
// The bfloat16 sweep runs both products of the GQA group on 16x16x32 bf16 MFMA: K rows load
// straight into the A operand of q.K^T (16 B per lane); V rows are loaded coalesced, staged
// row-major in a wave-private LDS tile and read back with gfx950's transposing LDS load
// (ds_read_b64_tr_b16) as the B operand of alpha.V; alpha enters that product as a pair of bf16
// terms (hi + lo, within 2^-16).
#include "lg_internal.h"

namespace lg {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// Loads of the K/V stream. Every row is read once per launch; when the cache is large (it cannot
// stay in the 256 MB last-level cache from one decode step to the next) the loads are
// non-temporal, which on MI355X lifts a plain read kernel from ~6.3 to ~7.0 TB/s; a small cache
// keeps normal loads so it can stay resident in the last-level cache across steps.
template <bool NT>
__device__ __forceinline__ uint4 ld_stream16(const void* p) {
  if (NT) {
    const u32x4_t v = __builtin_nontemporal_load((const u32x4_t*)p);
    return make_uint4(v.x, v.y, v.z, v.w);
  }
  return *(const uint4*)p;
}

template <typename T> __device__ __forceinline__ float to_f32(T x);
template <> __device__ __forceinline__ float to_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ float to_f32<uint16_t>(uint16_t x) { return bf16_to_f32(x); }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ uint16_t from_f32<uint16_t>(float x) { return f32_to_bf16(x); }

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// -------------------------------------------------------------------------------------------
// Portable sweep: one wave per (split, kv head, sequence); lane e holds dims e, e+64, ...
// -------------------------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(64) void attend_valu(AttendArgs a) {
  constexpr int E = D / 64;
  const int split = blockIdx.x, hkv = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x;
  int L, app;
  const int n_eff = live_slots(a, b, &L, &app);
  const int s_lo = split * a.split;
  if (s_lo >= n_eff) return;
  const int s_hi = min(s_lo + a.split, n_eff);
  const int G = a.G;
  const size_t bk = (size_t)b * a.Hkv + hkv;
  const T* Kb = (const T*)a.k + bk * a.cap * D;
  const T* Vb = (const T*)a.v + bk * a.cap * D;
  const T* kn = app ? (const T*)a.k_new + bk * D : nullptr;
  const T* vn = app ? (const T*)a.v_new + bk * D : nullptr;

  if (app && L >= s_lo && L < s_hi) {  // append: this split owns slot L
#pragma unroll
    for (int e = 0; e < E; ++e) {
      ((T*)a.k_w)[(bk * a.cap + L) * D + lane + 64 * e] = kn[lane + 64 * e];
      ((T*)a.v_w)[(bk * a.cap + L) * D + lane + 64 * e] = vn[lane + 64 * e];
    }
  }

  float qr[kMaxGroup][E];
  float m[kMaxGroup], l[kMaxGroup], sg[kMaxGroup], o[kMaxGroup][E];
#pragma unroll
  for (int h = 0; h < kMaxGroup; ++h) {
    m[h] = -INFINITY; l[h] = 0.f; sg[h] = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      o[h][e] = 0.f;
      qr[h][e] = h < G ? to_f32(((const T*)a.q)[((size_t)b * a.Hq + hkv * G + h) * D + lane + 64 * e]) : 0.f;
    }
  }
  const int thr = sat_sub(a.t[b], a.suffix_w[b]);
  float* stash = a.stash + bk * G * a.cap_s;

  for (int j = s_lo; j < s_hi; ++j) {
    const bool is_new = app && j == L;
    const T* kr = is_new ? kn : Kb + (size_t)j * D;
    const T* vr = is_new ? vn : Vb + (size_t)j * D;
    const int pj = is_new ? a.t[b] : a.pos[(size_t)b * a.cap + j];
    const bool suf = pj > thr;
    float kx[E], vx[E];
#pragma unroll
    for (int e = 0; e < E; ++e) { kx[e] = to_f32(kr[lane + 64 * e]); vx[e] = to_f32(vr[lane + 64 * e]); }
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) {
      if (h < G) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) d += qr[h][e] * kx[e];
        const float s = wave_sum(d) * a.scale_log2;
        if (lane == h) stash[(size_t)h * a.cap_s + j] = s;
        const float mn = fmaxf(m[h], s);
        const float al = exp2f(m[h] - mn);
        const float p = exp2f(s - mn);
        l[h] = l[h] * al + p;
        sg[h] = sg[h] * al + (suf ? p : 0.f);
#pragma unroll
        for (int e = 0; e < E; ++e) o[h][e] = o[h][e] * al + p * vx[e];
        m[h] = mn;
      }
    }
  }
  const size_t pbase = (bk * a.ns_grid + split) * G;
#pragma unroll
  for (int h = 0; h < kMaxGroup; ++h) {
    if (h < G) {
#pragma unroll
      for (int e = 0; e < E; ++e) a.part_o[(pbase + h) * D + lane + 64 * e] = o[h][e];
      if (lane == 0) {
        a.part_ml[pbase + h] = make_float2(m[h], l[h]);
        a.part_s[pbase + h] = sg[h];
      }
    }
  }
}

// -------------------------------------------------------------------------------------------
// MFMA sweep (bfloat16 cache).
//
// Each workgroup (kWaves waves) owns one split of a (sequence, kv head): a contiguous, 32-aligned
// slot range, balanced so every split of the row has about the same length. Its waves take the
// 32-slot blocks of the range round-robin, prefetching the next block's K/V rows while the current
// one is on the matrix cores. Lane l = 16 g + c: head c of the group in the logits, row group g.
// -------------------------------------------------------------------------------------------
__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 u) {
  bf16x8_t r;
  __builtin_memcpy(&r, &u, 16);
  return r;
}

// Split of n live slots into at most ceil(n / max_split) ranges of 32-aligned length: balanced,
// except at one block per wave (max_split = kFixedChunk), where split k starts at k * max_split
// whatever n is, so a workgroup knows its slots before it knows the row's length (a balanced
// chunk rounds up to the same length for every row of more than 288 slots, and a wave sweeps
// one block either way).
constexpr int kFixedChunk = 32 * kWaves;
struct SplitPlan {
  int ns, chunk;
};
__device__ __forceinline__ SplitPlan split_plan(int n, int max_split) {
  SplitPlan p;
  if (max_split == kFixedChunk) {
    p.chunk = max_split;
    p.ns = (n + max_split - 1) / max_split;
    return p;
  }
  int ns = (n + max_split - 1) / max_split;
  int chunk = (n + ns - 1) / ns;
  chunk = (chunk + 31) & ~31;
  p.chunk = chunk;
  p.ns = (n + chunk - 1) / chunk;
  return p;
}

// One 32-slot block of a wave: K rows for the A operand of q.K^T, V rows (row-major, staged
// through LDS for the B operand of alpha.V), one position per lane.
//
// Slot order. Lane (g, c) ends up holding the logits of slots 8g + 4mt + v (mt = 0, 1; v = 0..3)
// of head c: in q.K^T tile mt, output row i = 4g + v must be slot 8g + 4mt + v, so the K row fed
// to A-row i is slot 8(i/4) + 4mt + i%4. These 8 slots are then, in order, the k index 8g..8g+7
// of the alpha.V product, whose A operand (alpha of head c) is therefore the lane's own values.
//
// K loads. In the A layout every load instruction would read 64 bytes of each of 16 rows, so each
// 128-byte line would be fetched by two instructions. Instead the two k-steps 2p and 2p + 1 of a
// tile are loaded as two instructions that each read 8 whole lines: the first (kept in k[mt][2p])
// reads A-rows 0..7, lanes c < 8 the k-step 2p part and lanes c >= 8 the k-step 2p + 1 part of
// A-row c - 8; the second (k[mt][2p + 1]) reads A-rows 8..15 the same way (lanes c < 8: A-row
// c + 8, step 2p; lanes c >= 8: A-row c, step 2p + 1). Rotating each 16-lane row by 8 lanes then
// swaps the misplaced halves between the two registers (see fix_k).
// DV: the V dims (and output dims) the workgroup handles, D or a part of it (see attend_mfma_body).
template <int D, int DV = D>
struct Block {
  uint4 k[2][D / 32];
  uint4 v[DV / 16];  // V rows, 16 bytes per lane (see load_v)
};

struct RowCtx {
  const uint16_t* kbase;  // lane's K address at slot 0: A-row (c mod 8) of tile 0, dims 8g or
                          // 32 + 8g (c < 8 or not) of k-steps 0 and 1
  const uint16_t* vbase;  // lane's V address at slot 0 (see load_v)
  const int32_t* posb;
  int L, app, cap, n_eff;
  int jsuf;  // first slot of the recent suffix within the split (see attend_mfma_body)
  // The appended row: slot lsub (-1 when this split does not hold it) takes the new K and V rows
  // staged in LDS (snew: D / 8 16-byte pieces of K, then of V) in place of what the cache held;
  // the workgroup's V dims start at piece vp0 of the V row.
  int lsub, vp0;
  const uint4* snew;
};

// Block loads, in two halves so a pipelined wave can issue the next block's V rows as soon as the
// current ones are in LDS, before its q.K^T. K: see "K loads" (base folded in kbase). V: 16 bytes
// per lane, DV / 8 lanes per row, so each load instruction reads 512 / DV consecutive rows of the
// workgroup's DV dims in lane order (1 KB): lane l of instruction i holds row
// blk + i (512 / DV) + l / (DV / 8) at dims 8 (l % (DV / 8)) (base folded in vbase). Rows stay
// below cap because cap is a multiple of 32 on this path.
template <int DV> constexpr int vrows_per_load() { return 512 / DV; }
template <int D, bool NT, int DV>
__device__ __forceinline__ void load_v(Block<D, DV>& B, const RowCtx& r, int blk) {
  const uint16_t* vp = r.vbase + (size_t)blk * D;
#pragma unroll
  for (int i = 0; i < DV / 16; ++i) B.v[i] = ld_stream16<NT>(vp + i * vrows_per_load<DV>() * D);
}

template <int D, bool NT, int DV>
__device__ __forceinline__ void load_k(Block<D, DV>& B, const RowCtx& r, int blk, int lane) {
  constexpr int NKK = D / 32;
  const uint16_t* kp = r.kbase + (size_t)blk * D;
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)  // k-step pair kk / 2; kk odd: A-rows 8..15 (slots + 16)
      B.k[mt][kk] = ld_stream16<NT>(kp + (4 * mt + 16 * (kk & 1)) * D + 64 * (kk >> 1));
  }
}

template <int D, bool NT, int DV>
__device__ __forceinline__ void load_block(Block<D, DV>& B, const RowCtx& r, int blk, int lane) {
  load_v<D, NT, DV>(B, r, blk);
  load_k<D, NT, DV>(B, r, blk, lane);
}

struct Online {
  float m, l, s;
};

typedef short short4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) short4_t lds_short4;

// Row stride (elements) of a wave's V tile in LDS; the padding spreads the transpose reads of
// rows 8 apart over different banks.
template <int D> constexpr int vtile_stride() { return D + 8; }

// First half of a block, in two steps: stage_v writes the V rows to the wave's LDS tile
// (row-major; afterwards the V registers are free), stage_qk takes the suffix mask and runs q.K^T
// (afterwards the K registers are free).
template <int D, int DV>
__device__ __forceinline__ void stage_v(const Block<D, DV>& B, const RowCtx& r, int blk, int g,
                                        int c, uint16_t* vt) {
  constexpr int RS = vtile_stride<DV>(), LPR = DV / 8, RPL = vrows_per_load<DV>();
  const int lane = 16 * g + c;
  const int rl = lane / LPR, cl = 8 * (lane % LPR);  // the lane's row within a load, and dims
  if (blk + 32 > r.n_eff) {  // partial last block: rows past the live ones may hold anything
#pragma unroll
    for (int i = 0; i < DV / 16; ++i) {
      const uint4 z = blk + i * RPL + rl < r.n_eff ? B.v[i] : make_uint4(0, 0, 0, 0);
      *(uint4*)(vt + (i * RPL + rl) * RS + cl) = z;
    }
  } else {
#pragma unroll
    for (int i = 0; i < DV / 16; ++i) *(uint4*)(vt + (i * RPL + rl) * RS + cl) = B.v[i];
  }
  // The appended row replaces the cache's slot (the wave's LDS writes land in order).
  if (r.lsub >= blk && r.lsub < blk + 32) {
    if (lane < DV / 8) *(uint4*)(vt + (r.lsub - blk) * RS + 8 * lane) = r.snew[D / 8 + r.vp0 + lane];
  }
}

// Puts the K registers of one k-step pair into the A layout (see "K loads"): lanes 8..15 of every
// 16-lane row take the first register from the second one's lanes 0..7, and lanes 0..7 take the
// second register from the first one's lanes 8..15 (a rotation of the row by 8 lanes).
__device__ __forceinline__ void fix_k(uint4& x, uint4& y) {
  constexpr int kRowRor8 = 0x128;  // DPP row_ror:8
  const uint4 x0 = x, y0 = y;
  const unsigned* xs = (const unsigned*)&x0;
  const unsigned* ys = (const unsigned*)&y0;
  unsigned* xd = (unsigned*)&x;
  unsigned* yd = (unsigned*)&y;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    xd[e] = (unsigned)__builtin_amdgcn_update_dpp((int)xs[e], (int)ys[e], kRowRor8, 0xf, 0xc, false);
    yd[e] = (unsigned)__builtin_amdgcn_update_dpp((int)ys[e], (int)xs[e], kRowRor8, 0xf, 0x3, false);
  }
}

template <int D, int DV>
__device__ __forceinline__ void stage_qk(const Block<D, DV>& B, const RowCtx& r, int blk, int lane,
                                         int thr, const bf16x8_t* qf, f32x4_t* S,
                                         unsigned long long& suf) {
  constexpr int NKK = D / 32;
  const int g = lane >> 4, c = lane & 15;
  // Slots of this block in the recent suffix (bit j = slot blk + j).
  const int ps = blk + (lane & 31);
  suf = __ballot(lane < 32 && ps >= r.jsuf && ps < r.n_eff);
  // q.K^T on the matrix cores: lane holds slots blk+8g+4mt+v of head c.
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
    uint4 kr[NKK];
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) kr[kk] = B.k[mt][kk];
#pragma unroll
    for (int p = 0; p < NKK / 2; ++p) fix_k(kr[2 * p], kr[2 * p + 1]);
    // The appended row's K in the lanes of its A-row (slot 8(c/4) + 4mt + c%4 of the block).
    if (r.lsub >= blk && r.lsub < blk + 32 && r.lsub - blk == 8 * (c >> 2) + 4 * mt + (c & 3)) {
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) kr[kk] = r.snew[4 * kk + g];
    }
    S[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
      S[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kr[kk]), qf[kk], S[mt], 0, 0, 0);
  }
}

template <int D, int DV>
__device__ __forceinline__ void stage_block(const Block<D, DV>& B, const RowCtx& r, int blk, int g,
                                            int c, int lane, int thr, const bf16x8_t* qf,
                                            uint16_t* vt, f32x4_t* S, unsigned long long& suf) {
  stage_v<D, DV>(B, r, blk, g, c, vt);
  stage_qk<D, DV>(B, r, blk, lane, thr, qf, S, suf);
}

// Where a wave writes its logits: the split's LDS copy of its stash rows, or the stash itself.
// The LDS row is an address-space-3 pointer to the row's start, indexed by slot - lo, so no
// pointer outside the LDS allocation is ever formed.
typedef __attribute__((address_space(3))) float lds_float;
typedef __attribute__((address_space(3))) f32x4_t lds_f32x4;
struct StashRow {
  lds_float* lds;  // LDS row of head c (slot lo at index 0)
  float* glob;     // stash row of head c in global memory (indexed by slot)
  int lo;          // the split's first slot
  bool use_lds;    // fixed per kernel instantiation
};

// Second half: online softmax, logit stash, suffix mass, and alpha.V (DV dims) from the LDS tile.
template <int D, int DV>
__device__ __forceinline__ void finish_block(const f32x4_t* S, unsigned long long suf,
                                             const RowCtx& r, int blk, int g, int c, int G,
                                             float scale_log2, const StashRow& sr, uint16_t* vt,
                                             Online& st, f32x4_t* O) {
  constexpr int NB = DV / 16, RS = vtile_stride<DV>();
  float s[2][4];
  float mx = -INFINITY;
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int slot = blk + 8 * g + 4 * mt + v;
      s[mt][v] = slot < r.n_eff ? S[mt][v] * scale_log2 : -INFINITY;
      mx = fmaxf(mx, s[mt][v]);
    }
  }
  if (c < G) {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
    {
      const float4 sv = make_float4(s[mt][0], s[mt][1], s[mt][2], s[mt][3]);
      if (sr.use_lds)
        *(lds_f32x4*)(sr.lds + (blk - sr.lo) + 8 * g + 4 * mt) = f32x4_t{sv.x, sv.y, sv.z, sv.w};
      else *(float4*)(sr.glob + blk + 8 * g + 4 * mt) = sv;
    }
  }
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const float m_new = fmaxf(st.m, mx);
  const float alpha = exp2f(st.m - m_new);
  float p[2][4];
  float psum = 0.f, ssum = 0.f;
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      p[mt][v] = exp2f(s[mt][v] - m_new);
      psum += p[mt][v];
      ssum += ((suf >> (8 * g + 4 * mt + v)) & 1ull) ? p[mt][v] : 0.f;
    }
  }
  st.l = st.l * alpha + psum;
  st.s = st.s * alpha + ssum;
  st.m = m_new;
  // alpha of head c for slots 8g..8g+7, in k order, as two bf16 A operands: hi = alpha truncated
  // to bf16, lo = the remainder truncated to bf16, so hi + lo is within 2^-16 of alpha.
  uint32_t hb[8], lb[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float x = p[e >> 2][e & 3];
    const uint32_t xb = __float_as_uint(x) & 0xffff0000u;
    hb[e] = xb >> 16;
    lb[e] = __float_as_uint(x - __uint_as_float(xb)) >> 16;
  }
  uint4 ph, pl;
  ph.x = hb[0] | (hb[1] << 16); ph.y = hb[2] | (hb[3] << 16); ph.z = hb[4] | (hb[5] << 16); ph.w = hb[6] | (hb[7] << 16);
  pl.x = lb[0] | (lb[1] << 16); pl.y = lb[2] | (lb[3] << 16); pl.z = lb[4] | (lb[5] << 16); pl.w = lb[6] | (lb[7] << 16);
  const bf16x8_t Ahi = as_bf16x8(ph), Alo = as_bf16x8(pl);
  float al[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) al[v] = __shfl(alpha, 4 * g + v, 64);
  // alpha.V: B[k][j] = V[slot 8g + k'][16nb + j] read from LDS with the transposing load: source
  // lane c of the 16-lane group reads 4 dims 16nb + 4(c%4).. of row 8g + 4hf + c/4, and lane c
  // receives dim 16nb + c of rows 8g + 4hf + 0..3.
  const int trow = 8 * g + (c >> 2);
  const int tcol = 4 * (c & 3);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const short4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4*)(vt + trow * RS + 16 * nb + tcol));
    const short4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4*)(vt + (trow + 4) * RS + 16 * nb + tcol));
    bf16x8_t Bv;
    __builtin_memcpy(&Bv, &lo, 8);
    __builtin_memcpy((char*)&Bv + 8, &hi, 8);
#pragma unroll
    for (int v = 0; v < 4; ++v) O[nb][v] *= al[v];
    O[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ahi, Bv, O[nb], 0, 0, 0);
    O[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Alo, Bv, O[nb], 0, 0, 0);
  }
}

// Logit stash rows staged in LDS: SG > 0 keeps a split's logits (at most kMaxSplitSlots slots of at
// most SG heads) in LDS during the sweep; 0 writes them to the stash from the loop (merge form with
// short splits).
// Split length from which a merge-form launch stages its logits in LDS and writes the stash once
// at the end (scattered 16-byte stash stores inside the loop cost the 7B layer ~2.7 us at 2048
// slots; staging gains 1.1 us there, but adds a store round trip to short splits: batch 1,
// 128-slot splits, +0.3 us).
constexpr int kLdsStashMinSplit = 512;

// -------------------------------------------------------------------------------------------
// One-launch form. The splits of a row (sequence, kv head) exchange their partials through
// memory inside one launch, and no workgroup ever waits for one that may not have started:
//
//  - Arrival. Every workgroup of a row adds 1 to the row's 64-bit arrival word when it starts
//    ([63:32] generation, [31:16] split count of the row's last exchange, [15:0] arrivals). The
//    workgroup that sees ns - 1 earlier arrivals is the row's closer; the others are openers.
//  - Modes. Once its sweep is done, an opener looks at the arrival word: if every split of the
//    row has arrived (all of them are running or done), it takes part in the exchange itself
//    (SELF); otherwise it hands over (HANDOVER): it publishes its partial and the split-relative
//    probabilities of its slots, and exits. The closer always merges, and also finishes the row
//    for every opener that handed over. Every wait is for words that a started workgroup has
//    issued or will issue without waiting itself, so a launch finishes whatever the number of
//    workgroups the device holds at once.
//  - Words. Statistics (per split: max, sum, suffix sum of every head) are 64-bit words
//    (tag << 32) | float bits, the tag being the row generation + 1, never 0. Numerators, mode
//    words and handover probabilities have exactly one reader, which clears them after reading
//    (with the same write-through stores, so no dirty line is left for the end of the kernel to
//    write back): they are zero at the start of every launch, and a non-zero word was written by
//    this launch.
//    The closer bumps the generation, records the split count and clears the statistics words of
//    splits the row no longer has, so no statistics word of an earlier launch carries the tag a
//    later launch waits for.
//  - Coherence. Splits of a row may run on different XCDs, whose L2 caches are not coherent with
//    each other for ordinary accesses; every exchanged word is an agent-scope relaxed atomic, which
//    gfx950 performs coherently across XCDs without a cache write-back or invalidation, and every
//    word validates itself (tag or non-zero), so no fence orders one word against another.
//  - Errors. A wait is still bounded (a preempted or starved workgroup); one that gives up sets
//    LG_ATTEND_STATUS_WAIT in the workspace header and marks conf[b] NaN, and writes neither out
//    nor acc. A workspace whose header does not describe the launch, or whose status is non-zero,
//    is refused the same way (LG_ATTEND_STATUS_WORKSPACE).
// -------------------------------------------------------------------------------------------
// Workgroup barrier that orders LDS only: the waves' outstanding global loads and stores stay in
// flight across it (__syncthreads() also waits for those). The epilogues below communicate between
// their threads through LDS only; the words they exchange with other workgroups validate
// themselves.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

enum : int { kRoleRefuse = 0, kRoleCloser = 1, kRoleSelf = 2, kRoleHandover = 3 };
constexpr unsigned kModeSelf = 1u, kModeHandover = 2u;

__device__ __forceinline__ unsigned long long row_arrive(unsigned long long* w) {
  return __hip_atomic_fetch_add(w, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long row_peek(const unsigned long long* w) {
  return __hip_atomic_load(const_cast<unsigned long long*>(w), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}
// Every split of the row has arrived: the count is complete, or the closer already moved on.
__device__ __forceinline__ bool all_arrived(unsigned long long w, unsigned gen, int ns) {
  return (unsigned)(w >> 32) != gen || (int)(w & 0xffffu) >= ns;
}
// Generations run through 0 .. 2^32 - 2, tags through 1 .. 2^32 - 1 (never 0).
__device__ __forceinline__ unsigned gen_tag(unsigned gen) { return gen % 0xffffffffu + 1u; }
__device__ __forceinline__ unsigned next_gen(unsigned gen) { return (gen % 0xffffffffu + 1u) % 0xffffffffu; }

__device__ __forceinline__ void st_tagged(unsigned long long* p, unsigned tag, float x) {
  __hip_atomic_store(p, ((unsigned long long)tag << 32) | __float_as_uint(x), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long ld_tagged(const unsigned long long* p) {
  return __hip_atomic_load(const_cast<unsigned long long*>(p), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ bool has_tag(unsigned long long w, unsigned tag) {
  return (unsigned)(w >> 32) == tag;
}
__device__ __forceinline__ float tagged_value(unsigned long long w) {
  return __uint_as_float((unsigned)w);
}
// Single-reader words: 0 means "not written by this launch". +0 is sent as -0 and every NaN as the
// canonical quiet NaN, so no value encodes to 0.
__device__ __forceinline__ unsigned enc_word(float x) {
  const unsigned u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc00000u;
  return u == 0u ? 0x80000000u : u;
}
__device__ __forceinline__ void st_word(unsigned* p, unsigned v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned ld_word(const unsigned* p) {
  return __hip_atomic_load(const_cast<unsigned*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The workspace header describes this launch and carries no error.
template <int D>
__device__ __forceinline__ bool header_ok(const AttendArgs& a) {
  const uint4* h = (const uint4*)a.hdr;
  const uint4 w0 = h[0], w1 = h[1], w2 = h[2];
  return w0.x == kWsMagic && w0.y == kWsVersion && (int)w0.z == a.B && (int)w0.w == a.Hq &&
         (int)w1.x == a.Hkv && (int)w1.y == D && (int)w1.z == a.cap && (int)w1.w == a.dtype &&
         (int)w2.x == a.form && (int)w2.y == a.split && w2.z == 0u;
}
// A refused or failed row: the error bit in the header, conf[b] NaN (an integer max on the float
// bits: the quiet NaN pattern is above every non-negative float), nothing else written.
__device__ __forceinline__ void refuse_row(const AttendArgs& a, int b, unsigned bits) {
  atomicOr(&a.hdr->status, bits);
  if (a.conf != nullptr) atomicMax((int*)(a.conf + b), 0x7fc00000);
}

// Final statistics of head h of a row (threads 0..G-1 of the workgroup, all in wave 0): lse and
// suffix mass, and the confidence proxy as one atomic max over the group's heads.
__device__ __forceinline__ void write_row_stats(const AttendArgs& a, int b, int hkv, int h, float M,
                                                float rZ, float S) {
  const int G = a.G;
  const float sg = S * rZ;
  a.suffix_mass[(size_t)b * a.Hq + hkv * G + h] = sg;
  a.lse[(size_t)b * a.Hq + hkv * G + h] = (M - __log2f(rZ)) * kLn2;
  float mx = sg;
#pragma unroll
  for (int o = 1; o < kMaxGroup; o <<= 1) {
    const float y = __shfl_xor(mx, o, 64);
    if ((h ^ o) < G) mx = fmaxf(mx, y);
  }
  // Non-negative floats order like their bit patterns, so an integer max is exact.
  if (h == 0 && a.conf != nullptr) atomicMax((int*)(a.conf + b), __float_as_int(mx));
}

// Per-workgroup facts the one-launch epilogue needs from the sweep.
struct RowInfo {
  int b, hkv, split, ns, chunk, s_lo, s_hi, L, app, n_eff;
  int dh;     // the workgroup's part of the output dims (see single_split_epilogue)
  size_t bk;  // row index b * Hkv + hkv
};

// One-launch epilogue of a row with a single split: the waves are merged in LDS and the split
// finishes the row itself (no exchange). MS: the split's slots at most (the LDS logit rows'
// stride) and NW the workgroup's waves; each thread owns MS / (256 NW) groups of four
// consecutive slots.
// The thread's acc values (acc_slots) are read before the sweep (see attend_mfma_body).
template <int MS, int NW>
struct AccSlots {
  static constexpr int NU = MS / (64 * NW * 4);
  static_assert(NU >= 1 && NU * 64 * NW * 4 == MS, "four slots per thread and group");
  float4 v[NU];
};
template <int MS, int NW>
__device__ __forceinline__ void load_acc_slots(AccSlots<MS, NW>& o, const float* acc, int s_lo,
                                               int s_hi) {
#pragma unroll
  for (int u = 0; u < AccSlots<MS, NW>::NU; ++u) {
    const int j0 = s_lo + 4 * (int)threadIdx.x + 256 * NW * u;
    o.v[u] = *(const float4*)(acc + (j0 < s_hi ? j0 : s_lo));
  }
}

// With DV < D the workgroup owns output dims [r.dh DV, (r.dh + 1) DV) of the row; the statistics,
// conf and acc (identical in every part) are written by part 0 only.
template <int D, int SG, int MS, int NW, int DV>
__device__ __forceinline__ void single_split_epilogue(const AttendArgs& a, const f32x4_t* O,
                                                      uint16_t* vt, char* smem, const float* slog,
                                                      float (*sm_m)[16], float (*sm_l)[16],
                                                      float (*sm_s)[16], const RowInfo& r,
                                                      int g, int c, bool hdr_ok,
                                                      const AccSlots<MS, NW>& old) {
  constexpr int VE = DV / 16, RS = vtile_stride<DV>();
  constexpr int NU = AccSlots<MS, NW>::NU;
  const int tid = threadIdx.x, G = a.G, GDV = G * DV;
  float* acc = a.acc + r.bk * a.cap;
  float* my_o = (float*)vt;  // the wave's numerators go to its own V tile (its last alpha.V read it)
#pragma unroll
  for (int t = 0; t < VE; ++t) {
#pragma unroll
    for (int v = 0; v < 4; ++v) my_o[(4 * g + v) * DV + 16 * t + c] = O[t][v];
  }
  __shared__ float sM1[kMaxGroup], srZ1[kMaxGroup], sf1[kMaxGroup][NW];
  __shared__ int s_ok1;
  if (tid == 0) s_ok1 = hdr_ok ? 1 : 0;
  lds_barrier();  // every wave's statistics and numerators are in LDS
  if (s_ok1 == 0) {
    if (tid == 0) refuse_row(a, r.b, LG_ATTEND_STATUS_WORKSPACE);
    return;
  }
  if (tid < G) {
    const int h = tid;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, sm_m[w][h]);
    float lsum = 0.f, ssum = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float mw = sm_m[w][h];
      const float f = mw == -INFINITY ? 0.f : exp2f(mw - M);
      sf1[h][w] = f;
      lsum += f * sm_l[w][h];
      ssum += f * sm_s[w][h];
    }
    sM1[h] = M;
    srZ1[h] = 1.f / lsum;
    if (r.dh == 0) write_row_stats(a, r.b, r.hkv, h, M, 1.f / lsum, ssum);
  }
  lds_barrier();
  uint16_t* out = (uint16_t*)a.out + ((size_t)r.b * a.Hq + r.hkv * G) * D + r.dh * DV;
  for (int i = tid; i < GDV; i += 64 * NW) {
    const int h = i / DV;
    float o = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) o += sf1[h][w] * ((const float*)((const uint16_t*)smem + w * 32 * RS))[i];
    out[h * D + (i - h * DV)] = f32_to_bf16(o * srZ1[h]);
  }
  if (r.dh != 0) return;
  // H2O increment of the split's slots: alpha = exp2(s - M) / Z; slots past the split keep their
  // bits; heads past G (padding up to SG) are masked by a select.
#pragma unroll
  for (int u = 0; u < NU; ++u) {
    const int j0 = r.s_lo + 4 * tid + 256 * NW * u;
    if (j0 < r.s_hi) {
      float4 nv;
      float* nvp = (float*)&nv;
      const float* ov = (const float*)&old.v[u];
      float sum[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int h = 0; h < SG; ++h) {
        const int hc = min(h, G - 1);
        const f32x4_t lg = *(const f32x4_t*)(slog + hc * MS + 4 * tid + 256 * NW * u);
        const float M = sM1[hc], rz = srZ1[hc];
#pragma unroll
        for (int e = 0; e < 4; ++e) sum[e] += h < G ? exp2f(lg[e] - M) * rz : 0.f;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = j0 + e;
        const float nx = (r.app && j == r.L) ? sum[e] : ov[e] + sum[e];
        nvp[e] = j < r.s_hi ? nx : ov[e];
      }
      *(float4*)(acc + j0) = nv;
    }
  }
}

// One-launch epilogue of a row with ns >= 2 splits (the exchange described above). The waves
// are first merged in LDS into one partial for the split (max, sum and suffix sum per head, and
// the G x D output numerators); the split then publishes it and, unless it hands over, merges its
// slice of the row's output from every split's partial.
template <int D, int SG, int NSB>
__device__ __forceinline__ void exchange_epilogue(const AttendArgs& a, const f32x4_t* O,
                                                  uint16_t* vt, char* smem, float* slog,
                                                  float (*sm_m)[16], float (*sm_l)[16],
                                                  float (*sm_s)[16], const RowInfo& r, int g,
                                                  int c, bool hdr_ok, unsigned long long rw_old,
                                                  unsigned long long rw_chk) {
  constexpr int NW = kWaves, VE = D / 16, RS = vtile_stride<D>();
  constexpr int kStIter = (NSB * SG * 3 + 255) / 256;           // statistics words of a row
  constexpr int kPoIter = (SG * D + kMaxMfmaSplits + 255) / 256; // numerator words of a slice
  static_assert((size_t)kPoIter * 256 * 4 <= (size_t)NW * 32 * RS * 2,
                "the polled numerators are staged in the V tiles");
  const int tid = threadIdx.x, G = a.G, GD = G * D, ns = r.ns;
  const size_t bk = r.bk;
  // The wave's numerators go to its own V tile (its last alpha.V has read it).
  float* my_o = (float*)vt;
#pragma unroll
  for (int t = 0; t < VE; ++t) {
#pragma unroll
    for (int v = 0; v < 4; ++v) my_o[(4 * g + v) * D + 16 * t + c] = O[t][v];
  }
  __shared__ int s_role, s_ok, s_mode[kMaxMfmaSplits];
  __shared__ unsigned s_tag, s_gen, s_prev;
  if (tid == 0) {
    int role = kRoleRefuse;
    unsigned tag = 0, gen = 0;
    if (hdr_ok) {
      gen = (unsigned)(rw_old >> 32);
      const int cnt = (int)(rw_old & 0xffffu);
      tag = gen_tag(gen);
      if (cnt >= ns) {
        role = kRoleRefuse;  // more arrivals than splits: the arrival word is not this launch's
      } else if (cnt == ns - 1) {
        role = kRoleCloser;
      } else {
        bool all = all_arrived(rw_chk, gen, ns);
        if (!all) all = all_arrived(row_peek(a.rows + bk), gen, ns);
        role = (all && !(a.flags & kFlagForceHandover)) ? kRoleSelf : kRoleHandover;
      }
    }
    s_role = role;
    s_tag = tag;
    s_gen = gen;
    s_prev = (unsigned)((rw_old >> 16) & 0xffffu);
    s_ok = 1;
  }
  // sMs: the split's own max, sum and suffix sum per head; sm_f: each wave's factor.
  __shared__ float sMs[3 * kMaxGroup], sm_f[kMaxGroup][NW];
  lds_barrier();  // every wave's statistics and numerators are in LDS, and the role is known
  const int role = s_role;
  if (role == kRoleRefuse) {
    if (tid == 0) refuse_row(a, r.b, LG_ATTEND_STATUS_WORKSPACE);
    return;
  }
  const unsigned tag = s_tag;
  unsigned long long* st_row = a.stats + bk * (size_t)kMaxMfmaSplits * G * 3;
  unsigned* nm_row = a.numer + bk * (size_t)a.ns_grid * GD;
  if (tid < G) {
    // The split's statistics per head and each wave's rescaling factor (0 for a wave without
    // slots); published at once.
    const int h = tid;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, sm_m[w][h]);
    float lsum = 0.f, ssum = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float mw = sm_m[w][h];
      const float f = mw == -INFINITY ? 0.f : exp2f(mw - M);
      sm_f[h][w] = f;
      lsum += f * sm_l[w][h];
      ssum += f * sm_s[w][h];
    }
    sMs[h] = M;
    sMs[kMaxGroup + h] = lsum;
    sMs[2 * kMaxGroup + h] = ssum;
    unsigned long long* w = st_row + ((size_t)r.split * G + h) * 3;
    st_tagged(w, tag, M);
    st_tagged(w + 1, tag, lsum);
    st_tagged(w + 2, tag, ssum);
  }
  lds_barrier();
  // Publish the split's merged numerators.
  for (int i = tid; i < GD; i += 64 * NW) {
    const int h = i / D;
    float o = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w)
      o += sm_f[h][w] * ((const float*)((const uint16_t*)smem + w * 32 * RS))[i];
    st_word(nm_row + (size_t)r.split * GD + i, enc_word(o));
  }
  // This thread's four slots of the split; their split-relative probabilities exp2(s - M_split)
  // per head replace their logits in LDS (each thread rewrites only its own entries).
  const int j0 = r.s_lo + 4 * tid;
  const bool live = j0 < r.s_hi;
  auto split_probs = [&]() {
    if (live) {
      for (int h = 0; h < G; ++h) {
        f32x4_t* lp = (f32x4_t*)(slog + h * kMaxSplitSlots + 4 * tid);
        const f32x4_t lg = *lp;
        const float ms = sMs[h];
        *lp = f32x4_t{exp2f(lg[0] - ms), exp2f(lg[1] - ms), exp2f(lg[2] - ms), exp2f(lg[3] - ms)};
      }
    }
  };
  if (role == kRoleHandover) {
    // The probabilities go out lane-contiguous (every store instruction writes whole lines): the
    // exchanged words are written through to memory, where partial lines are expensive.
    split_probs();
    lds_barrier();
    const int nsl = r.s_hi - r.s_lo;
    for (int h = 0; h < G; ++h) {
      unsigned* hp = a.hand + (bk * G + h) * (size_t)a.cap_s + r.s_lo;
#pragma unroll
      for (int u = 0; u < kMaxSplitSlots / 256; ++u) {
        const int o = tid + 256 * u;
        if (o < nsl) st_word(hp + o, enc_word(slog[h * kMaxSplitSlots + o]));
      }
    }
    if (tid == 0) st_word(a.mode + bk * kMaxMfmaSplits + r.split, kModeHandover);
    return;
  }
  if (role == kRoleSelf && tid == 0) st_word(a.mode + bk * kMaxMfmaSplits + r.split, kModeSelf);

  // ---- poll: every split's statistics, this split's slice of every split's numerators, and
  // (closer) every opener's mode; all loads of a poll are issued at once ----
  const int per = (GD + ns - 1) / ns;
  const int o_lo = r.split * per;
  const int cnt = max(0, min(per, GD - o_lo));
  const int nst = ns * G * 3;
  const int npo = ns * per;
  const bool closer = role == kRoleCloser;
  unsigned long long sw[kStIter];
  unsigned pw[kPoIter];
  unsigned mw = 0;
  auto poll = [&]() {
#pragma unroll
    for (int u = 0; u < kStIter; ++u) {
      const int i = tid + 256 * u;
      if (i < nst) sw[u] = ld_tagged(st_row + i);
    }
#pragma unroll
    for (int u = 0; u < kPoIter; ++u) {
      const int idx = tid + 256 * u;
      const int k = idx / per, i = idx - k * per;
      if (idx < npo && i < cnt) pw[u] = ld_word(nm_row + (size_t)k * GD + o_lo + i);
    }
    if (closer && tid < ns && tid != r.split) mw = ld_word(a.mode + bk * kMaxMfmaSplits + tid);
  };
  auto current = [&]() {
    bool done = true;
#pragma unroll
    for (int u = 0; u < kStIter; ++u) {
      const int i = tid + 256 * u;
      done = done && (i >= nst || has_tag(sw[u], tag));
    }
#pragma unroll
    for (int u = 0; u < kPoIter; ++u) {
      const int idx = tid + 256 * u;
      const int k = idx / per, i = idx - k * per;
      done = done && (idx >= npo || i >= cnt || pw[u] != 0u);
    }
    if (closer && tid < ns && tid != r.split) done = done && mw != 0u;
    return done;
  };
  float* acc = a.acc + bk * a.cap;
  const float4 old = *(const float4*)(acc + (live ? j0 : r.s_lo));
  if (a.flags & kFlagNoWait) {
    if (tid == 0) s_ok = 0;
  } else {
    poll();
    split_probs();  // while the first poll's loads are in flight
    for (int it = 0; !current(); ++it) {
      if (it >= a.spin_limit) {
        s_ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
      poll();
    }
  }
  // Every wave is done with the V tiles (the numerators were published before the poll), so they
  // can stage the polled numerators.
  lds_barrier();
  if (s_ok == 0) {  // a wait gave up: nothing of this row is written
    if (tid == 0) refuse_row(a, r.b, LG_ATTEND_STATUS_WAIT);
    return;
  }
  // ---- stage the polled words in LDS and merge the statistics ----
  __shared__ float sst[NSB * SG * 3];  // [split][head][max, sum, suffix sum]
  __shared__ float sF[SG][NSB];
  __shared__ float sM[SG], srZ[SG];
  float* spo = (float*)smem;  // the V tiles
#pragma unroll
  for (int u = 0; u < kStIter; ++u) {
    const int i = tid + 256 * u;
    if (i < nst) sst[i] = tagged_value(sw[u]);
  }
#pragma unroll
  for (int u = 0; u < kPoIter; ++u) {
    const int idx = tid + 256 * u;
    const int k = idx / per, i = idx - k * per;
    if (idx < npo && i < cnt) spo[idx] = __uint_as_float(pw[u]);
  }
  if (closer && tid < ns) s_mode[tid] = tid == r.split ? (int)kModeSelf : (int)mw;
  lds_barrier();
  if (tid < G) {
    // Per head: the row max over the splits, each split's factor exp2(m - M), the softmax sum and
    // the suffix mass.
    const int h = tid;
    float M = -INFINITY;
    for (int k = 0; k < ns; ++k) M = fmaxf(M, sst[(k * G + h) * 3]);
    float Z = 0.f, S = 0.f;
    for (int k = 0; k < ns; ++k) {
      const float f = exp2f(sst[(k * G + h) * 3] - M);
      sF[h][k] = f;
      Z += sst[(k * G + h) * 3 + 1] * f;
      S += sst[(k * G + h) * 3 + 2] * f;
    }
    sM[h] = M;
    srZ[h] = 1.f / Z;
    if (closer) write_row_stats(a, r.b, r.hkv, h, M, 1.f / Z, S);
  }
  lds_barrier();
  uint16_t* out = (uint16_t*)a.out + ((size_t)r.b * a.Hq + r.hkv * G) * D;
  for (int i = tid; i < cnt; i += 256) {
    const int h = (o_lo + i) / D;
    float o = 0.f;
    for (int k = 0; k < ns; ++k) o += sF[h][k] * spo[k * per + i];
    out[o_lo + i] = f32_to_bf16(o * srZ[h]);
  }
  // H2O increment of this split's slots: alpha = exp2(s - M_split) * exp2(M_split - M) / Z; slots
  // past the split keep their bits; heads past G (padding up to SG) are masked by a select.
  auto h2o = [&](int k, int jj, int hi, const float4& ov4, const f32x4_t* pv) {
    float fh[SG];
#pragma unroll
    for (int h = 0; h < SG; ++h) {
      const int hc = min(h, G - 1);
      fh[h] = sF[hc][k] * srZ[hc];
    }
    float4 nv;
    float* nvp = (float*)&nv;
    const float* ov = (const float*)&ov4;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float sum = 0.f;
#pragma unroll
      for (int h = 0; h < SG; ++h) sum += h < G ? pv[h][e] * fh[h] : 0.f;
      const int j = jj + e;
      const float nx = (r.app && j == r.L) ? sum : ov[e] + sum;
      nvp[e] = j < hi ? nx : ov[e];
    }
    *(float4*)(acc + jj) = nv;
  };
  if (live) {
    f32x4_t pv[SG];
#pragma unroll
    for (int h = 0; h < SG; ++h) pv[h] = *(const f32x4_t*)(slog + min(h, G - 1) * kMaxSplitSlots + 4 * tid);
    h2o(r.split, j0, r.s_hi, old, pv);
  }
  // Clear the numerator words this split has read (each has exactly this reader).
#pragma unroll
  for (int u = 0; u < kPoIter; ++u) {
    const int idx = tid + 256 * u;
    const int k = idx / per, i = idx - k * per;
    if (idx < npo && i < cnt) st_word(nm_row + (size_t)k * GD + o_lo + i, 0u);
  }
  if (!closer) return;

  // ---- closer: finish the row for every split that handed over, then close the exchange ----
  for (int k = 0; k < ns; ++k) {
    if (s_mode[k] != (int)kModeHandover) continue;  // uniform over the workgroup
    const int o_lo_k = k * per;
    const int cnt_k = max(0, min(per, GD - o_lo_k));
    const int lo_k = k * r.chunk, hi_k = min(lo_k + r.chunk, r.n_eff);
    const int jk = lo_k + 4 * tid;
    const bool live_k = jk < hi_k;
    const float4 old_k = *(const float4*)(acc + (live_k ? jk : lo_k));
    unsigned qw[4][SG];
    auto poll_k = [&]() {
#pragma unroll
      for (int u = 0; u < kPoIter; ++u) {
        const int idx = tid + 256 * u;
        const int kk = idx / per, i = idx - kk * per;
        if (idx < npo && i < cnt_k) pw[u] = ld_word(nm_row + (size_t)kk * GD + o_lo_k + i);
      }
      if (live_k) {
#pragma unroll
        for (int h = 0; h < SG; ++h) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (h < G && jk + e < hi_k) qw[e][h] = ld_word(a.hand + (bk * G + h) * (size_t)a.cap_s + jk + e);
        }
      }
    };
    auto current_k = [&]() {
      bool done = true;
#pragma unroll
      for (int u = 0; u < kPoIter; ++u) {
        const int idx = tid + 256 * u;
        const int kk = idx / per, i = idx - kk * per;
        done = done && (idx >= npo || i >= cnt_k || pw[u] != 0u);
      }
      if (live_k) {
#pragma unroll
        for (int h = 0; h < SG; ++h) {
#pragma unroll
          for (int e = 0; e < 4; ++e) done = done && (h >= G || jk + e >= hi_k || qw[e][h] != 0u);
        }
      }
      return done;
    };
    lds_barrier();  // every thread is done with spo (the previous slice)
    poll_k();
    for (int it = 0; !current_k(); ++it) {
      if (it >= a.spin_limit) {
        s_ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
      poll_k();
    }
#pragma unroll
    for (int u = 0; u < kPoIter; ++u) {
      const int idx = tid + 256 * u;
      const int kk = idx / per, i = idx - kk * per;
      if (idx < npo && i < cnt_k) spo[idx] = __uint_as_float(pw[u]);
    }
    lds_barrier();
    if (s_ok == 0) {
      if (tid == 0) refuse_row(a, r.b, LG_ATTEND_STATUS_WAIT);
      return;
    }
    for (int i = tid; i < cnt_k; i += 256) {
      const int h = (o_lo_k + i) / D;
      float o = 0.f;
      for (int kk = 0; kk < ns; ++kk) o += sF[h][kk] * spo[kk * per + i];
      out[o_lo_k + i] = f32_to_bf16(o * srZ[h]);
    }
    if (live_k) {
      f32x4_t pv[SG];
#pragma unroll
      for (int h = 0; h < SG; ++h) {
#pragma unroll
        for (int e = 0; e < 4; ++e) pv[h][e] = h < G ? __uint_as_float(qw[e][h]) : 0.f;
      }
      h2o(k, jk, hi_k, old_k, pv);
#pragma unroll
      for (int h = 0; h < SG; ++h) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (h < G && jk + e < hi_k) st_word(a.hand + (bk * G + h) * (size_t)a.cap_s + jk + e, 0u);
      }
    }
#pragma unroll
    for (int u = 0; u < kPoIter; ++u) {
      const int idx = tid + 256 * u;
      const int kk = idx / per, i = idx - kk * per;
      if (idx < npo && i < cnt_k) st_word(nm_row + (size_t)kk * GD + o_lo_k + i, 0u);
    }
  }
  // Mode words read; the statistics words of splits this row no longer has cleared; the arrival
  // word reset with the next generation and this launch's split count.
  if (tid < ns && tid != r.split) st_word(a.mode + bk * kMaxMfmaSplits + tid, 0u);
  const int prev = min((int)s_prev, kMaxMfmaSplits);
  for (int i = ns * G * 3 + tid; i < prev * G * 3; i += 256)
    __hip_atomic_store(st_row + i, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (tid == 0)
    __hip_atomic_store(a.rows + bk,
                       ((unsigned long long)next_gen(s_gen) << 32) | ((unsigned long long)ns << 16),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Merge form: the waves of the workgroup are merged in LDS into one partial for this split
// (part_ml, part_s, part_o); attend_combine_mfma finishes the row in a second launch.
template <int D, int SG>
__device__ __forceinline__ void merge_form_epilogue(const AttendArgs& a, const f32x4_t* O,
                                                    uint16_t* vt, char* smem, const float* slog,
                                                    float (*sm_m)[16], float (*sm_l)[16],
                                                    float (*sm_s)[16], const RowInfo& r, int wave,
                                                    int lane, int g, int c, int nb) {
  constexpr int NW = kWaves, VE = D / 16, RS = vtile_stride<D>();
  const int G = a.G;
  // Each wave, as soon as its own loop is done, puts its output numerators into its own V tile
  // (its last alpha.V has read it) and copies its blocks' logits from the LDS copy to the stash,
  // 16 B per lane (head hh + lane / 8, slots 4 (lane % 8).. of the block), so the waves that
  // finish first do this while the others still stream.
  float* my_o = (float*)vt;  // [16][D]
#pragma unroll
  for (int t = 0; t < VE; ++t) {
#pragma unroll
    for (int v = 0; v < 4; ++v) my_o[(4 * g + v) * D + 16 * t + c] = O[t][v];
  }
  if (SG > 0) {
    for (int i = 0; i < nb; ++i) {
      const int off = 32 * (wave + NW * i);  // the block's first slot, relative to s_lo
#pragma unroll
      for (int hh = 0; hh < (SG > 0 ? SG : 1); hh += 8) {
        const int h = hh + (lane >> 3), q = lane & 7;
        if (h < G)
          *(float4*)(a.stash + (r.bk * G + h) * a.cap_s + r.s_lo + off + 4 * q) =
              *(const float4*)(slog + h * kMaxSplitSlots + off + 4 * q);
      }
    }
  }
  __shared__ float sm_f[16][NW];
  lds_barrier();  // every wave's statistics and numerators are in LDS
  // Per head: the split's max, each wave's rescaling factor (0 for a wave without slots), the
  // split's softmax sum and suffix mass; then the merged numerators.
  const size_t pbase = (r.bk * a.ns_grid + r.split) * G;
  if (threadIdx.x < G) {
    const int h = threadIdx.x;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, sm_m[w][h]);
    float lsum = 0.f, ssum = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float mw = sm_m[w][h];
      const float f = mw == -INFINITY ? 0.f : exp2f(mw - M);
      sm_f[h][w] = f;
      lsum += f * sm_l[w][h];
      ssum += f * sm_s[w][h];
    }
    a.part_ml[pbase + h] = make_float2(M, lsum);
    a.part_s[pbase + h] = ssum;
  }
  lds_barrier();
  for (int i = threadIdx.x; i < G * D; i += 64 * NW) {
    const int h = i / D, d = i - h * D;
    float o = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w)
      o += sm_f[h][w] * ((const float*)((const uint16_t*)smem + w * 32 * RS))[h * D + d];
    a.part_o[(pbase + h) * D + d] = o;
  }
}

// MFMA sweep (bfloat16 cache): one workgroup of kWaves waves per split of a row; CO selects the
// one-launch form (the row is finished in this launch), otherwise the merge form (split partials
// for attend_combine_mfma).
template <int D, bool NT, int SG, bool CO, int NSB, int MS, int NW, int DS>
__device__ __forceinline__ void attend_mfma_body(const AttendArgs& a) {
  static_assert(!CO || (SG > 0 && kWaves * 64 * 4 >= kMaxSplitSlots),
                "the one-launch form keeps every logit of its split in LDS and handles four slots "
                "per thread");
  static_assert(MS == kMaxSplitSlots || (CO && MS == kMaxSingleSlots && SG <= 8),
                "splits longer than kMaxSplitSlots finish their row alone (one-launch form), with "
                "at most 8 heads of logits in LDS");
  static_assert(NW == kWaves || MS > kMaxSplitSlots,
                "the exchange and the merge form use kWaves waves per workgroup");
  static_assert(DS == 1 || (DS == 2 && D == 128 && CO && MS > kMaxSplitSlots),
                "the output dims are split only in single-split rows of head_dim 128");
  constexpr int DV = D / DS;    // V and output dims of this workgroup
  constexpr int NKK = D / 32;   // k-steps of the q.K^T product
  constexpr int VE = DV / 16;   // V dims per lane per row
  // Grid order. Split slowest: consecutive workgroups (which the dispatcher deals round-robin to
  // the 8 XCDs) belong to different rows, so the busy splits of a launch spread over every XCD
  // even when some split indices have no slots. Row-major (one-launch form, grids larger than the
  // device holds at once): the splits of a row are dispatched together, so they meet in the
  // exchange instead of handing over. Split output dims (DS = 2, one split per row): a 1-D grid in
  // which the two parts of row r are workgroups 16(r / 8) + r % 8 and that + 8, so the round-robin
  // dispatch puts them on the same XCD and the second read of the row's K mostly hits its L2.
  int split, hkv, b, dh = 0;
  if constexpr (DS > 1) {
    const int j = blockIdx.x & 15;
    const int row = 8 * (blockIdx.x >> 4) + (j & 7);
    if (row >= a.B * a.Hkv) return;
    dh = j >> 3;
    b = row / a.Hkv;
    hkv = row - b * a.Hkv;
    split = 0;
  } else if (CO && a.row_major) {
    split = blockIdx.x; hkv = blockIdx.y; b = blockIdx.z;
  } else {
    hkv = blockIdx.x; b = blockIdx.y; split = blockIdx.z;
  }
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = lane >> 4, c = lane & 15;
  const int G = a.G;
  const size_t bk = (size_t)b * a.Hkv + hkv;
  const int cap = a.cap;
  const uint16_t* Kb = (const uint16_t*)a.k + bk * cap * D;
  const uint16_t* Vb = (const uint16_t*)a.v + bk * cap * D;
  RowCtx rc;
  rc.kbase = Kb + (size_t)(8 * ((c & 7) >> 2) + (c & 3)) * D + 8 * (c < 8 ? g : 4 + g);
  rc.vbase = Vb + (size_t)(lane / (DV / 8)) * D + dh * DV + 8 * (lane % (DV / 8));
  rc.vp0 = dh * (DV / 8);
  rc.posb = a.pos + (size_t)b * cap;
  rc.cap = cap;
  // Split 0 starts at slot 0 whatever the plan, so its waves request their first block (block
  // `wave`) before the row's length is known; a wave that turns out to have no block drops it.
  // Positions of the split's slots for the suffix count below (thread t: slots s_lo + t + 64 NW k),
  // read first and, for split 0, before the length is known. (With a fixed chunk every split's
  // start is known early too; requesting its block before the length measured 0.2-0.5 us per
  // layer slower at batch 1.)
  constexpr int kPosPer = (MS + 64 * NW - 1) / (64 * NW);
  int pv[kPosPer];
  auto load_pos = [&](int lo) {
#pragma unroll
    for (int k = 0; k < kPosPer; ++k) pv[k] = rc.posb[min(lo + (int)threadIdx.x + 64 * NW * k, cap - 1)];
  };
  if (split == 0) load_pos(0);
  Block<D, DV> A;
  const bool spec = split == 0 && 32 * wave < cap;
  if (spec) load_block<D, NT, DV>(A, rc, 32 * wave, lane);
  int L, app;
  const int n_eff = live_slots(a, b, &L, &app);
  if (n_eff == 0) {  // the merge launch writes the empty result, or split 0 of the one-launch form
    if (CO && split == 0 && dh == 0) {
      __shared__ int s_hdr0;
      if (threadIdx.x == 0) s_hdr0 = header_ok<D>(a) ? 1 : 0;
      __syncthreads();
      if (s_hdr0 == 0) {
        if (threadIdx.x == 0) refuse_row(a, b, LG_ATTEND_STATUS_WORKSPACE);
        return;
      }
      uint16_t* out = (uint16_t*)a.out + ((size_t)b * a.Hq + hkv * G) * D;
      for (int i = threadIdx.x; i < G * D; i += 64 * NW) out[i] = 0;
      if (threadIdx.x < G) {
        a.lse[(size_t)b * a.Hq + hkv * G + threadIdx.x] = -INFINITY;
        a.suffix_mass[(size_t)b * a.Hq + hkv * G + threadIdx.x] = 0.f;
      }
    }
    return;
  }
  const SplitPlan bp = split_plan(n_eff, a.split);
  const int p_ns = bp.ns, p_chunk = bp.chunk;
  const int s_lo = split * bp.chunk, s_hi = min(s_lo + bp.chunk, n_eff);
  if (split >= p_ns) return;
  const int nblk = (s_hi - s_lo + 31) / 32;
  // Recent suffix of the split: positions strictly increase over the live slots and the appended
  // slot holds the newest position t, so the slots whose position exceeds thr = t - suffix_w are
  // the split's last ones, from jsuf = s_lo + (stored slots of the split at or below thr) on (none
  // when t itself is at or below thr).
  const int thr = sat_sub(a.t[b], a.suffix_w[b]);
  if (split != 0) load_pos(s_lo);
  const int hi_st = (app && L < s_hi) ? L : s_hi;  // the split's stored slots: [s_lo, hi_st)
  int cnt = 0;
#pragma unroll
  for (int k = 0; k < kPosPer; ++k) {
    const int j = s_lo + (int)threadIdx.x + 64 * NW * k;
    cnt += (j < hi_st && pv[k] <= thr) ? 1 : 0;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
  __shared__ int s_cnt[NW];
  if (lane == 0) s_cnt[wave] = cnt;
  // The appended row (slot L, when this split holds it): stored to the cache for later steps and
  // staged in LDS, from where the sweep takes it in place of the slot's old contents, so no wave
  // waits for the store (the barrier below waits for LDS only).
  __shared__ uint4 s_new[2 * (D / 8)];
  rc.lsub = -1;
  rc.snew = s_new;
  const bool holds_new = app && L >= s_lo && L < s_hi;
  if (holds_new && threadIdx.x < 2 * (D / 8)) {
    const int which = threadIdx.x / (D / 8), piece = threadIdx.x % (D / 8);
    const uint4 x = ((const uint4*)((const uint16_t*)(which ? a.v_new : a.k_new) + bk * D))[piece];
    if (dh == 0) ((uint4*)((uint16_t*)(which ? a.v_w : a.k_w) + (bk * cap + L) * D))[piece] = x;
    s_new[threadIdx.x] = x;
  }
  lds_barrier();
  if (holds_new) rc.lsub = L;
  rc.jsuf = s_lo;
#pragma unroll
  for (int w = 0; w < NW; ++w) rc.jsuf += s_cnt[w];
  if (holds_new && a.t[b] <= thr) rc.jsuf = s_hi;
  // One-launch form: arrive at the row (multi-split rows) and fetch the workspace header; both
  // are consumed after the sweep.
  const bool multi = CO && p_ns > 1;
  unsigned long long rw_old = 0;
  uint4 hd0 = make_uint4(0, 0, 0, 0), hd1 = hd0, hd2 = hd0;
  if (CO && threadIdx.x == 0) {
    if (multi) rw_old = row_arrive(a.rows + bk);
    const uint4* h = (const uint4*)a.hdr;
    hd0 = h[0]; hd1 = h[1]; hd2 = h[2];
  }
  rc.L = L;
  rc.app = app;
  rc.n_eff = n_eff;

  // q as the B operand: B[k][j] = q[head j][dim], lane (g, c) holds head c, dims kk*32+8g..+8.
  bf16x8_t qf[NKK];
  {
    const uint16_t* qrow = (const uint16_t*)a.q + ((size_t)b * a.Hq + hkv * G + (c < G ? c : 0)) * D;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      uint4 u = c < G ? *(const uint4*)(qrow + kk * 32 + 8 * g) : make_uint4(0, 0, 0, 0);
      qf[kk] = as_bf16x8(u);
    }
  }
  // A split that finishes its row alone reads its acc slots now (they are needed only after the
  // sweep, whose loads then hide their latency); kept in registers in the long-split kernel.
  AccSlots<MS, NW> acc_old;
  if constexpr (CO && MS > kMaxSplitSlots) load_acc_slots(acc_old, a.acc + bk * cap, s_lo, s_hi);
  __shared__ __attribute__((aligned(16))) float slog[SG > 0 ? SG * MS : 4];
  // With SG > 0 the logits are staged in LDS (and, in the merge form, written to the stash once at
  // the end); otherwise they are stored to the stash from the loop.
  StashRow stash_row;
  stash_row.use_lds = SG > 0;
  stash_row.lds = (lds_float*)slog + (c < G ? c : 0) * (SG > 0 ? MS : 0);
  stash_row.glob = CO ? nullptr : a.stash + (bk * G + (c < G ? c : 0)) * a.cap_s;
  stash_row.lo = s_lo;

  Online st{-INFINITY, 0.f, 0.f};
  f32x4_t O[VE];
#pragma unroll
  for (int rr = 0; rr < VE; ++rr) O[rr] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // LDS: per-wave V tiles during the sweep, then the wave partials or the polled words.
  constexpr int RS = vtile_stride<DV>();
  constexpr size_t kTileBytes = (size_t)NW * 32 * RS * 2;
  constexpr size_t kMergeBytes = (size_t)NW * 16 * DV * 4;
  __shared__ __attribute__((aligned(16))) char smem[kTileBytes > kMergeBytes ? kTileBytes : kMergeBytes];
  uint16_t* vt = (uint16_t*)smem + wave * 32 * RS;

  // Wave w takes blocks w, w + NW, ... of the split. The next block's V rows are loaded as soon as
  // the current ones are in LDS and its K rows right after the current q.K^T (into the same, now
  // free, registers), so they are in flight during the current block's softmax and alpha.V. The
  // last block is peeled so the loop's loads are unconditional: the wait counts at the loop head
  // then let the V rows be staged while the K rows of the same block are still in flight.
  const int nb = wave < nblk ? (nblk - wave + NW - 1) / NW : 0;
  f32x4_t S[2];
  unsigned long long suf;
  // Thread 0 parks the arrival word and the header check in LDS as soon as they have returned
  // (they were requested before the first block, and vector memory reads complete in order, so
  // waiting for them does not wait for the block), and an opener looks at the row's arrival word
  // again when its last block starts, long before its sweep ends; nothing of this is live across
  // the sweep loop.
  __shared__ unsigned long long s_rw_old;
  __shared__ int s_hdr_ok;
  unsigned long long rw_chk = 0;
  if (nb > 0) {
    if (!spec) load_block<D, NT, DV>(A, rc, s_lo + 32 * wave, lane);
    if (CO && threadIdx.x == 0) {
      s_hdr_ok = hd0.x == kWsMagic && hd0.y == kWsVersion && (int)hd0.z == a.B &&
                 (int)hd0.w == a.Hq && (int)hd1.x == a.Hkv && (int)hd1.y == D &&
                 (int)hd1.z == a.cap && (int)hd1.w == a.dtype && (int)hd2.x == a.form &&
                 (int)hd2.y == a.split && hd2.z == 0u;
      s_rw_old = rw_old;
    }
    for (int i = 0; i + 1 < nb; ++i) {
      const int blk = s_lo + 32 * (wave + NW * i);
      stage_v<D, DV>(A, rc, blk, g, c, vt);
      load_v<D, NT, DV>(A, rc, blk + 32 * NW);
      stage_qk<D, DV>(A, rc, blk, lane, thr, qf, S, suf);
      load_k<D, NT, DV>(A, rc, blk + 32 * NW, lane);
      finish_block<D, DV>(S, suf, rc, blk, g, c, G, a.scale_log2, stash_row, vt, st, O);
    }
    if (multi && threadIdx.x == 0 && (int)(s_rw_old & 0xffffu) != p_ns - 1)
      rw_chk = row_peek(a.rows + bk);
    const int blk = s_lo + 32 * (wave + NW * (nb - 1));
    stage_block<D, DV>(A, rc, blk, g, c, lane, thr, qf, vt, S, suf);
    finish_block<D, DV>(S, suf, rc, blk, g, c, G, a.scale_log2, stash_row, vt, st, O);
  }

  // The wave's partial: head c's max in every lane, sum and suffix sum reduced over the row groups.
  float l_run = st.l, s_run = st.s;
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  s_run += __shfl_xor(s_run, 16, 64);
  s_run += __shfl_xor(s_run, 32, 64);
  __shared__ float sm_m[NW][16], sm_l[NW][16], sm_s[NW][16];
  if (g == 0) {
    sm_m[wave][c] = st.m;
    sm_l[wave][c] = l_run;
    sm_s[wave][c] = s_run;
  }
  RowInfo ri;
  ri.b = b; ri.hkv = hkv; ri.split = split; ri.ns = p_ns; ri.chunk = p_chunk;
  ri.s_lo = s_lo; ri.s_hi = s_hi; ri.L = L; ri.app = app; ri.n_eff = n_eff;
  ri.bk = bk;
  ri.dh = dh;
  if constexpr (CO) {
    // Thread 0 is the only reader of its own LDS words here (wave 0 wrote them).
    const bool hdr_ok = threadIdx.x == 0 && s_hdr_ok != 0;
    const unsigned long long rw_old0 = threadIdx.x == 0 ? s_rw_old : 0ull;
    if constexpr (MS > kMaxSplitSlots) {
      // the plan gives such a launch one split per row (split >= cap)
      single_split_epilogue<D, SG, MS, NW, DV>(a, O, vt, smem, slog, sm_m, sm_l, sm_s, ri, g, c,
                                           hdr_ok, acc_old);
    } else {
      if (p_ns == 1) {
        load_acc_slots(acc_old, a.acc + bk * cap, s_lo, s_hi);
        single_split_epilogue<D, SG, MS, NW, DV>(a, O, vt, smem, slog, sm_m, sm_l, sm_s, ri, g, c,
                                             hdr_ok, acc_old);
      } else {
        exchange_epilogue<D, SG, NSB>(a, O, vt, smem, slog, sm_m, sm_l, sm_s, ri, g, c, hdr_ok,
                                      rw_old0, rw_chk);
      }
    }
  } else {
    merge_form_epilogue<D, SG>(a, O, vt, smem, slog, sm_m, sm_l, sm_s, ri, wave, lane, g, c, nb);
  }
}

// Kernel entry point: the occupancy target of two waves per SIMD is given to the register
// allocator. NSB bounds the splits per row of a one-launch grid (it sizes the statistics poll).
template <int D, bool NT, int SG, bool CO, int NSB = kMaxMfmaSplits, int MS = kMaxSplitSlots,
          int NW = kWaves, int DS = 1>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2, 8)))
void attend_mfma(AttendArgs a) {
  attend_mfma_body<D, NT, SG, CO, NSB, MS, NW, DS>(a);
}

// -------------------------------------------------------------------------------------------
// Combine: exact softmax over the splits, outputs, and the H2O increment from the stash.
// Same grid as the sweep (one workgroup per split) so a split's stash is read on the XCD that
// wrote it.
// -------------------------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(256) void attend_combine(AttendArgs a) {
  const int split = blockIdx.x, hkv = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int G = a.G;
  int L, app;
  const int n_eff = live_slots(a, b, &L, &app);
  const size_t bk = (size_t)b * a.Hkv + hkv;
  T* out = (T*)a.out + ((size_t)b * a.Hq + hkv * G) * D;
  __shared__ int s_hdr;
  if (tid == 0) s_hdr = header_ok<D>(a) ? 1 : 0;
  __syncthreads();
  if (s_hdr == 0) {
    if (tid == 0 && split == 0) refuse_row(a, b, LG_ATTEND_STATUS_WORKSPACE);
    return;
  }
  if (n_eff == 0) {
    if (split == 0) {
      for (int i = tid; i < G * D; i += 256) out[i] = from_f32<T>(0.f);
      if (tid < G) {
        a.lse[(size_t)b * a.Hq + hkv * G + tid] = -INFINITY;
        a.suffix_mass[(size_t)b * a.Hq + hkv * G + tid] = 0.f;
      }
    }
    return;
  }
  const int ns = (n_eff + a.split - 1) / a.split;
  if (split >= ns) return;
  __shared__ float sM[kMaxGroup], srZ[kMaxGroup], sS[kMaxGroup];
  const float2* pml = a.part_ml + bk * a.ns_grid * G;
  if (tid < G) {
    float M = -INFINITY;
    for (int k = 0; k < ns; ++k) M = fmaxf(M, pml[k * G + tid].x);
    float Z = 0.f;
    for (int k = 0; k < ns; ++k) Z += pml[k * G + tid].y * exp2f(pml[k * G + tid].x - M);
    sM[tid] = M;
    srZ[tid] = 1.f / Z;
  }
  __syncthreads();
  // H2O increment for this split's slots.
  const int lo = split * a.split, hi = min(lo + a.split, n_eff);
  const float* stash = a.stash + bk * G * a.cap_s;
  float* acc = a.acc + bk * a.cap;
  for (int j = lo + tid; j < hi; j += 256) {
    float sum = 0.f;
    for (int h = 0; h < G; ++h) sum += exp2f(stash[(size_t)h * a.cap_s + j] - sM[h]) * srZ[h];
    acc[j] = (app && j == L) ? sum : acc[j] + sum;
  }
  if (split != 0) return;
  const float* po = a.part_o + bk * a.ns_grid * G * D;
  for (int i = tid; i < G * D; i += 256) {
    const int h = i / D;
    float o = 0.f;
    for (int k = 0; k < ns; ++k) o += exp2f(pml[k * G + h].x - sM[h]) * po[(size_t)k * G * D + i];
    out[i] = from_f32<T>(o * srZ[h]);
  }
  if (tid < G) {
    const float* ps = a.part_s + bk * a.ns_grid * G;
    float sg = 0.f;
    for (int k = 0; k < ns; ++k) sg += exp2f(pml[k * G + tid].x - sM[tid]) * ps[k * G + tid];
    sg *= srZ[tid];
    sS[tid] = sg;
    a.suffix_mass[(size_t)b * a.Hq + hkv * G + tid] = sg;
    a.lse[(size_t)b * a.Hq + hkv * G + tid] = (sM[tid] - __log2f(srZ[tid])) * kLn2;
  }
  __syncthreads();
  if (tid == 0 && a.conf != nullptr) {
    float mx = 0.f;
    for (int h = 0; h < G; ++h) mx = fmaxf(mx, sS[h]);
    // Non-negative floats order like their bit patterns, so an integer max is exact.
    atomicMax((int*)(a.conf + b), __float_as_int(mx));
  }
}

// -------------------------------------------------------------------------------------------
// Combine for the MFMA sweep. One workgroup per split, same grid as the sweep so a split's stash
// is read back on the XCD that wrote it. Each workgroup applies the H2O increment to its split's
// slots (four consecutive slots per thread, 16-byte accesses) and merges one slice of the row's
// output. All of its loads (stash logits, old acc values, its output slice of every split
// partial, and the split maxima and sums) are issued together as soon as the row length gives
// their addresses. With fixed chunks (split_plan; the FX instance) the addresses do not depend on
// the length, so they are issued with it, and the output slices are cut over the grid's splits
// (a workgroup past the row's last split still merges its slice); otherwise over the row's. GM
// is a compile-time bound on the group size G.
// -------------------------------------------------------------------------------------------
template <int D, int GM>
struct CombineLoads {
  static constexpr int kPoIter = (kMaxGroup * D + kMaxMfmaSplits + 255) / 256;
  static constexpr int kStIter = (kMaxMfmaSplits * kMaxGroup + 255) / 256;
  float4 old;            // acc of the thread's four slots
  float4 lgv[GM];        // their logits, per head
  float pov[kPoIter];    // the workgroup's output slice of every split partial
  float2 mlv[kStIter];   // split maxima and sums
  float psv[kStIter];    // split suffix sums
};

// Issues the loads of one combine workgroup: slots from lo (quads below lim), output slice `per`
// entries wide of each of nsl splits, and (STATS) the split statistics.
template <int D, int GM, bool STATS>
__device__ __forceinline__ void combine_loads(CombineLoads<D, GM>& c, const AttendArgs& a,
                                              size_t bk, int split, int lo, int lim, int per,
                                              int nsl) {
  const int tid = threadIdx.x, G = a.G, GD = G * D;
  const int j0 = lo + 4 * tid;
  const int jl = j0 < lim ? j0 : lo;  // in bounds, discarded past lim
  const float* stash = a.stash + bk * G * a.cap_s;
  c.old = *(const float4*)(a.acc + bk * a.cap + jl);
#pragma unroll
  for (int h = 0; h < GM; ++h)
    c.lgv[h] = *(const float4*)(stash + (size_t)min(h, G - 1) * a.cap_s + jl);
  const int o_lo = split * per;
  const int cnt = max(0, min(per, GD - o_lo));
  const int tot = nsl * per;
  const float* po = a.part_o + bk * a.ns_grid * G * D;
#pragma unroll
  for (int u = 0; u < CombineLoads<D, GM>::kPoIter; ++u) {
    const int idx = tid + 256 * u;
    const int k = idx / per, i = idx - k * per;
    const bool in = idx < tot && i < cnt;
    c.pov[u] = po[in ? (size_t)k * GD + o_lo + i : 0];
  }
  if constexpr (STATS) {
    const float2* pml = a.part_ml + bk * a.ns_grid * G;
    const float* ps = a.part_s + bk * a.ns_grid * G;
#pragma unroll
    for (int u = 0; u < CombineLoads<D, GM>::kStIter; ++u) {
      const int i = tid + 256 * u;
      const int ic = i < nsl * G ? i : 0;
      c.mlv[u] = pml[ic];
      c.psv[u] = ps[ic];
    }
  }
}

// FX: the launch's splits are fixed chunks (a.split == kFixedChunk).
template <int D, int GM, bool FX>
__global__ __launch_bounds__(256) void attend_combine_mfma(AttendArgs a) {
  const int split = blockIdx.z, hkv = blockIdx.x, b = blockIdx.y;  // the sweep's grid
  const int tid = threadIdx.x;
  const int G = a.G, GD = G * D;
  const size_t bk = (size_t)b * a.Hkv + hkv;
  CombineLoads<D, GM> ld;
  int lo = split * a.split, per = (GD + a.ns_grid - 1) / a.ns_grid, nsl = a.ns_grid;
  if constexpr (FX)
    combine_loads<D, GM, true>(ld, a, bk, split, lo, min(lo + a.split, a.cap), per, nsl);
  int L, app;
  const int n_eff = live_slots(a, b, &L, &app);
  uint16_t* out = (uint16_t*)a.out + ((size_t)b * a.Hq + hkv * G) * D;
  __shared__ int s_hdr;
  if (tid == 0) s_hdr = header_ok<D>(a) ? 1 : 0;
  __syncthreads();
  if (s_hdr == 0) {
    if (tid == 0 && split == 0) refuse_row(a, b, LG_ATTEND_STATUS_WORKSPACE);
    return;
  }
  if (n_eff == 0) {
    if (split == 0) {
      for (int i = tid; i < G * D; i += 256) out[i] = 0;
      if (tid < G) {
        a.lse[(size_t)b * a.Hq + hkv * G + tid] = -INFINITY;
        a.suffix_mass[(size_t)b * a.Hq + hkv * G + tid] = 0.f;
      }
    }
    return;
  }
  const SplitPlan plan = split_plan(n_eff, a.split);
  const int ns = plan.ns;
  if constexpr (!FX) {
    if (split >= ns) return;
    lo = split * plan.chunk;
    per = (GD + ns - 1) / ns;
    nsl = ns;
    combine_loads<D, GM, false>(ld, a, bk, split, lo, min(lo + plan.chunk, n_eff), per, nsl);
  }
  const int hi = min(lo + plan.chunk, n_eff);
  // Slots j0..j0+3 of this thread (splits are at most 1024 slots). The sweep wrote -inf logits
  // for the slots of a split's last block that lie past n_eff.
  const int j0 = lo + 4 * tid;
  const bool live = j0 < hi;
  float* acc = a.acc + bk * a.cap;
  const int o_lo = split * per;
  const int cnt = max(0, min(per, GD - o_lo));
  constexpr int kPoIter = CombineLoads<D, GM>::kPoIter;
  __shared__ float spo[kPoIter * 256];
  __shared__ float2 sml[kMaxMfmaSplits * kMaxGroup];
  __shared__ float sps[kMaxMfmaSplits * kMaxGroup];
  __shared__ float sM[kMaxGroup], srZ[kMaxGroup], sF[kMaxGroup * kMaxMfmaSplits];
  if constexpr (FX) {
#pragma unroll
    for (int u = 0; u < CombineLoads<D, GM>::kStIter; ++u) {
      const int i = tid + 256 * u;
      if (i < ns * G) {
        sml[i] = ld.mlv[u];
        sps[i] = ld.psv[u];
      }
    }
  } else {
    const float2* pml = a.part_ml + bk * a.ns_grid * G;
    const float* ps = a.part_s + bk * a.ns_grid * G;
    for (int i = tid; i < ns * G; i += 256) {
      sml[i] = pml[i];
      sps[i] = ps[i];
    }
  }
#pragma unroll
  for (int u = 0; u < kPoIter; ++u) spo[tid + 256 * u] = ld.pov[u];
  __syncthreads();
  if (tid < G) {
    float M = -INFINITY;
    for (int k = 0; k < ns; ++k) M = fmaxf(M, sml[k * G + tid].x);
    float Z = 0.f, S = 0.f;
    for (int k = 0; k < ns; ++k) {
      const float f = exp2f(sml[k * G + tid].x - M);
      sF[tid * kMaxMfmaSplits + k] = f;
      Z += sml[k * G + tid].y * f;
      S += sps[k * G + tid] * f;
    }
    const float rZ = 1.f / Z;
    sM[tid] = M;
    srZ[tid] = rZ;
    if (split == 0) {
      // Row statistics and the confidence proxy, issued before the bulk stores. Lanes 0..G-1 of
      // wave 0 hold the G heads; their max goes to conf with one atomic.
      const float sg = S * rZ;
      a.suffix_mass[(size_t)b * a.Hq + hkv * G + tid] = sg;
      a.lse[(size_t)b * a.Hq + hkv * G + tid] = (M - __log2f(rZ)) * kLn2;
      float mx = sg;
#pragma unroll
      for (int o = 1; o < kMaxGroup; o <<= 1) {
        const float y = __shfl_xor(mx, o, 64);
        if ((tid ^ o) < G) mx = fmaxf(mx, y);
      }
      // Non-negative floats order like their bit patterns, so an integer max is exact.
      if (tid == 0 && a.conf != nullptr) atomicMax((int*)(a.conf + b), __float_as_int(mx));
    }
  }
  __syncthreads();
  // H2O increment for this split's slots; slots past hi keep their old value bit for bit. The
  // row statistics are read from LDS once; heads past G (padding up to GM) are masked by a select.
  if (live) {
    float mh[GM], rzh[GM];
#pragma unroll
    for (int h = 0; h < GM; ++h) {
      mh[h] = sM[min(h, G - 1)];
      rzh[h] = srZ[min(h, G - 1)];
    }
    float4 nv;
    float* nvp = (float*)&nv;
    const float* ov = (const float*)&ld.old;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float sum = 0.f;
#pragma unroll
      for (int h = 0; h < GM; ++h) {
        const float pr = exp2f(((const float*)&ld.lgv[h])[e] - mh[h]) * rzh[h];
        sum += h < G ? pr : 0.f;
      }
      const int j = j0 + e;
      nvp[e] = j < hi ? ((app && j == L) ? sum : ov[e] + sum) : ov[e];
    }
    *(float4*)(acc + j0) = nv;
  }
  for (int i = tid; i < cnt; i += 256) {
    const int h = (o_lo + i) / D;
    float o = 0.f;
    for (int k = 0; k < ns; ++k) o += sF[h * kMaxMfmaSplits + k] * spo[k * per + i];
    out[o_lo + i] = f32_to_bf16(o * srZ[h]);
  }
}

// -------------------------------------------------------------------------------------------
// Host-side launchers.
// -------------------------------------------------------------------------------------------

// Portable form: vector-ALU sweep of 64-slot splits, then the portable combine.
template <typename T, int D>
static hipError_t launch_valu(AttendArgs a, hipStream_t st) {
  dim3 grid(a.ns_grid, a.Hkv, a.B);
  hipLaunchKernelGGL((attend_valu<T, D>), grid, dim3(64), 0, st, a);
  hipLaunchKernelGGL((attend_combine<T, D>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

// Above this many K/V bytes per layer the sweep streams with non-temporal loads (a model's cache
// of such layers does not stay in the 256 MB last-level cache between decode steps).
constexpr double kStreamBytes = 16.0 * 1024 * 1024;
static bool stream_nt(const AttendArgs& a, int D) {
  return 4.0 * a.B * a.Hkv * (double)a.cap * D >= kStreamBytes;
}

template <int D, bool FX>
static void launch_combine(const AttendArgs& a, dim3 grid, hipStream_t st) {
  if (a.G <= 4)
    hipLaunchKernelGGL((attend_combine_mfma<D, 4, FX>), grid, dim3(256), 0, st, a);
  else if (a.G <= 8)
    hipLaunchKernelGGL((attend_combine_mfma<D, 8, FX>), grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((attend_combine_mfma<D, 16, FX>), grid, dim3(256), 0, st, a);
}

// Merge form: the MFMA sweep writes split partials and the logit stash, attend_combine_mfma
// merges them in a second launch.
template <int D, bool NT>
static hipError_t launch_merge_nt(AttendArgs a, hipStream_t st) {
  dim3 grid(a.Hkv, a.B, a.ns_grid);
  if (a.split < kLdsStashMinSplit)
    hipLaunchKernelGGL((attend_mfma<D, NT, 0, false>), grid, dim3(64 * kWaves), 0, st, a);
  else if (a.G <= 4)
    hipLaunchKernelGGL((attend_mfma<D, NT, 4, false>), grid, dim3(64 * kWaves), 0, st, a);
  else if (a.G <= 8)
    hipLaunchKernelGGL((attend_mfma<D, NT, 8, false>), grid, dim3(64 * kWaves), 0, st, a);
  else
    hipLaunchKernelGGL((attend_mfma<D, NT, 16, false>), grid, dim3(64 * kWaves), 0, st, a);
  if (a.split == kFixedChunk)
    launch_combine<D, true>(a, grid, st);
  else
    launch_combine<D, false>(a, grid, st);
  return hipGetLastError();
}

// Compute units of the current device, queried once per device.
constexpr int kMaxDevices = 64;
static long device_cus() {
  static long cache[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
  long c = __atomic_load_n(&cache[dev], __ATOMIC_RELAXED);
  if (c == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    c = cus;
    __atomic_store_n(&cache[dev], c, __ATOMIC_RELAXED);
  }
  return c;
}

// One-launch form. A grid of at most one workgroup per compute unit is ordered split slowest;
// a larger one row-major (see attend_mfma_body). Either order is correct with any residency.
template <int D, bool NT, int SG>
static hipError_t launch_one_sg(AttendArgs a, hipStream_t st) {
  const long n = (long)a.Hkv * a.B * a.ns_grid;
  a.row_major = n > device_cus() ? 1 : 0;
  const dim3 grid = a.row_major ? dim3(a.ns_grid, a.Hkv, a.B) : dim3(a.Hkv, a.B, a.ns_grid);
  if constexpr (SG <= 8) {
    if (a.split > kMaxSplitSlots) {
      if constexpr (D == 128) {
        if (a.dsplit == 2) {
          const unsigned n16 = (unsigned)((a.B * a.Hkv + 7) / 8) * 16;
          hipLaunchKernelGGL((attend_mfma<D, NT, SG, true, 4, kMaxSingleSlots, kSingleWaves, 2>),
                             dim3(n16), dim3(64 * kSingleWaves), 0, st, a);
          return hipGetLastError();
        }
      }
      if (a.dsplit != 1) return hipErrorInvalidValue;  // the plan never gives this
      hipLaunchKernelGGL((attend_mfma<D, NT, SG, true, 4, kMaxSingleSlots, kSingleWaves>), grid,
                         dim3(64 * kSingleWaves), 0, st, a);
      return hipGetLastError();
    }
  }
  if (a.dsplit != 1) return hipErrorInvalidValue;
  if (a.split > kMaxSplitSlots) return hipErrorInvalidValue;  // the plan never gives this
  if (a.ns_grid <= 4)
    hipLaunchKernelGGL((attend_mfma<D, NT, SG, true, 4>), grid, dim3(64 * kWaves), 0, st, a);
  else if (a.ns_grid <= 8)
    hipLaunchKernelGGL((attend_mfma<D, NT, SG, true, 8>), grid, dim3(64 * kWaves), 0, st, a);
  else
    hipLaunchKernelGGL((attend_mfma<D, NT, SG, true, kMaxMfmaSplits>), grid, dim3(64 * kWaves), 0, st, a);
  return hipGetLastError();
}

template <int D, bool NT>
static hipError_t launch_one_nt(AttendArgs a, hipStream_t st) {
  if (a.G <= 4) return launch_one_sg<D, NT, 4>(a, st);
  if (a.G <= 8) return launch_one_sg<D, NT, 8>(a, st);
  return launch_one_sg<D, NT, 16>(a, st);
}

template <int D>
static hipError_t launch_mfma_form(AttendArgs a, hipStream_t st) {
  const bool nt = stream_nt(a, D);
  if (a.form == kFormMerge) return nt ? launch_merge_nt<D, true>(a, st) : launch_merge_nt<D, false>(a, st);
  return nt ? launch_one_nt<D, true>(a, st) : launch_one_nt<D, false>(a, st);
}

hipError_t launch_attend(AttendArgs a, lg_dtype dt, int D, hipStream_t st) {
  if (a.form != kFormPortable)
    return D == 128 ? launch_mfma_form<128>(a, st) : launch_mfma_form<64>(a, st);
  if (dt == LG_BF16)
    return D == 128 ? launch_valu<uint16_t, 128>(a, st) : launch_valu<uint16_t, 64>(a, st);
  return D == 128 ? launch_valu<float, 128>(a, st) : launch_valu<float, 64>(a, st);
}

// Workspace initialisation: every byte zero, then the header. The fill is a kernel (not a memset)
// so the call can sit in a captured HIP graph.
__global__ __launch_bounds__(256) void ws_init_kernel(uint4* ws, size_t n16, WsHeader h) {
  const size_t stride = (size_t)gridDim.x * 256;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += stride)
    ws[i] = i < sizeof(WsHeader) / 16 ? ((const uint4*)&h)[i] : make_uint4(0, 0, 0, 0);
}

hipError_t launch_ws_init(void* ws, size_t bytes, const WsHeader& h, hipStream_t st) {
  const size_t n16 = bytes / 16;
  const size_t want = (n16 + 255) / 256;
  const unsigned blocks = (unsigned)(want < 4096 ? (want > 0 ? want : 1) : 4096);
  hipLaunchKernelGGL(ws_init_kernel, dim3(blocks), dim3(256), 0, st, (uint4*)ws, n16, h);
  return hipGetLastError();
}

}  // namespace lg

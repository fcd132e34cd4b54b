// lg_attend.hip -- decode attention over the fixed-budget cache with fused loop statistics.
//
// Eq. (1) of the paper (Sec. 3.1) per query head over the live slots of the cache, plus the
// statistics the guard consumes, all from one sweep over K/V:
//   suffix mass   sum of alpha over slots with pos > t - w_s (attention on the narrow recent
//                 suffix; head locking, Sec. 1 and App. E)
//   H2O increment acc[j] += sum over the group's query heads of alpha_j (Sec. 2.2, Sec. 6.1)
//   confidence    conf[b] = max(conf[b], max_h suffix mass)
//
// Split form: the slots of each (sequence, kv head) are cut into splits; each workgroup produces
// a partial (running max, running sum, suffix sum, un-normalised output) per query head and
// writes its logits to a stash. attend_combine merges the partials (exact softmax over all
// splits), writes out/lse/suffix mass, and applies the exact H2O increment from the stash.
// Fused form (MFMA, explicit variants): one workgroup per (sequence, kv head) sweeps the whole
// row and finalises everything itself, one launch per layer.
//
// Two sweep kernels:
//   attend_valu  portable vector-ALU kernel (float32 or bfloat16 cache, head_dim 64/128).
//   attend_mfma  bfloat16 cache: both products of the GQA group run on 16x16x32 bf16 MFMA.
//                K rows load straight into the A operand of q.K^T (16 B per lane); V rows are
//                loaded coalesced, staged row-major in a wave-private LDS tile and read back with
//                gfx950's transposing LDS load (ds_read_b64_tr_b16) as the B operand of alpha.V;
//                alpha enters that product as a pair of bf16 terms (hi + lo, within 2^-16).
#include "lg_internal.h"

namespace lg {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

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
template <bool NT>
__device__ __forceinline__ uint2 ld_stream8(const void* p) {
  if (NT) {
    const u32x2_t v = __builtin_nontemporal_load((const u32x2_t*)p);
    return make_uint2(v.x, v.y);
  }
  return *(const uint2*)p;
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
  const size_t pbase = (bk * a.ns_max + split) * G;
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
// Each workgroup (NW waves) owns one split of a (sequence, kv head): a contiguous, 32-aligned slot
// range, balanced so every split of the row has about the same length. Its waves take the 32-slot
// blocks of the range round-robin (with PIPE, prefetching the next block's K/V rows while the
// current one is on the matrix cores) and are merged in LDS into one partial per split.
// Lane l = 16 g + c: head c of the group in the logits, row group g.
// -------------------------------------------------------------------------------------------
__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 u) {
  bf16x8_t r;
  __builtin_memcpy(&r, &u, 16);
  return r;
}

template <int VE>
struct VRow;  // VE consecutive bf16 values of one V row
template <> struct VRow<8> { uint4 w; };
template <> struct VRow<4> { uint2 w; };

template <bool NT>
__device__ __forceinline__ VRow<8> load_vrow(const uint16_t* p, VRow<8>*) { return {ld_stream16<NT>(p)}; }
template <bool NT>
__device__ __forceinline__ VRow<4> load_vrow(const uint16_t* p, VRow<4>*) { return {ld_stream8<NT>(p)}; }

__device__ __forceinline__ float vrow_elem(const VRow<8>& v, int r) {
  const uint32_t w = r < 2 ? v.w.x : r < 4 ? v.w.y : r < 6 ? v.w.z : v.w.w;
  return (r & 1) ? __uint_as_float(w & 0xffff0000u) : __uint_as_float(w << 16);
}
__device__ __forceinline__ float vrow_elem(const VRow<4>& v, int r) {
  const uint32_t w = r < 2 ? v.w.x : v.w.y;
  return (r & 1) ? __uint_as_float(w & 0xffff0000u) : __uint_as_float(w << 16);
}

constexpr int kMaxMfmaSplits = 32;

// Balanced split of n live slots into at most ceil(n / max_split) ranges of 32-aligned length.
struct SplitPlan {
  int ns, chunk;
};
__device__ __forceinline__ SplitPlan split_plan(int n, int max_split) {
  SplitPlan p;
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
template <int D>
struct Block {
  uint4 k[2][D / 32];
  VRow<D / 16> v[2][4];
  int pos;
};

struct RowCtx {
  const uint16_t* kbase;  // lane's K address at slot 0 (row offset 8(c/4) + c%4, dims 8g)
  const uint16_t* vbase;  // lane's V address at slot 0 (row offset 4g, dims VE*c)
  const int32_t* posb;
  int L, app, cap, n_eff, tb;
};

// Block loads, in two halves so a pipelined wave can issue the next block's V rows as soon as the
// current ones are in LDS, before its q.K^T. K: lane (g, c) reads row blk + 8(c/4) + 4mt + c%4 at
// dims kk*32 + 8g (base folded in kbase); V: row blk + 16mt + 4g + v at dims VE*c (base folded in
// vbase). Rows stay below cap because cap is a multiple of 32 on this path.
template <int D, bool NT>
__device__ __forceinline__ void load_v(Block<D>& B, const RowCtx& r, int blk) {
  constexpr int VE = D / 16;
  const uint16_t* vp = r.vbase + (size_t)blk * D;
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int v = 0; v < 4; ++v) B.v[mt][v] = load_vrow<NT>(vp + (16 * mt + v) * D, (VRow<VE>*)nullptr);
  }
}

template <int D, bool NT>
__device__ __forceinline__ void load_k(Block<D>& B, const RowCtx& r, int blk, int lane) {
  constexpr int NKK = D / 32;
  const uint16_t* kp = r.kbase + (size_t)blk * D;
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) B.k[mt][kk] = ld_stream16<NT>(kp + (4 * mt) * D + kk * 32);
  }
  const int ps = blk + (lane & 31);
  B.pos = r.posb[min(ps, r.cap - 1)];
}

template <int D, bool NT>
__device__ __forceinline__ void load_block(Block<D>& B, const RowCtx& r, int blk, int lane) {
  load_v<D, NT>(B, r, blk);
  load_k<D, NT>(B, r, blk, lane);
}

struct Online {
  float m, l, s;
};

typedef short short4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) short4_t lds_short4;

__device__ __forceinline__ void zero_vrow(VRow<8>& v) { v.w = make_uint4(0, 0, 0, 0); }
__device__ __forceinline__ void zero_vrow(VRow<4>& v) { v.w = make_uint2(0, 0); }

template <int VE> __device__ __forceinline__ void lds_store_vrow(uint16_t* dst, const VRow<VE>& v);
template <> __device__ __forceinline__ void lds_store_vrow<8>(uint16_t* dst, const VRow<8>& v) { *(uint4*)dst = v.w; }
template <> __device__ __forceinline__ void lds_store_vrow<4>(uint16_t* dst, const VRow<4>& v) { *(uint2*)dst = v.w; }

// Row stride (elements) of a wave's V tile in LDS; the padding spreads the transpose reads of
// rows 8 apart over different banks.
template <int D> constexpr int vtile_stride() { return D + 8; }

// First half of a block, in two steps: stage_v writes the V rows to the wave's LDS tile
// (row-major; afterwards the V registers are free), stage_qk takes the suffix mask and runs q.K^T
// (afterwards the K registers are free).
template <int D>
__device__ __forceinline__ void stage_v(const Block<D>& B, const RowCtx& r, int blk, int g, int c,
                                        uint16_t* vt) {
  constexpr int VE = D / 16, RS = vtile_stride<D>();
  if (blk + 32 > r.n_eff) {  // partial last block: rows past the live ones may hold anything
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        VRow<VE> z = B.v[mt][v];
        if (blk + 16 * mt + 4 * g + v >= r.n_eff) zero_vrow(z);
        lds_store_vrow<VE>(vt + (16 * mt + 4 * g + v) * RS + VE * c, z);
      }
    }
  } else {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int v = 0; v < 4; ++v) lds_store_vrow<VE>(vt + (16 * mt + 4 * g + v) * RS + VE * c, B.v[mt][v]);
    }
  }
}

template <int D>
__device__ __forceinline__ void stage_qk(const Block<D>& B, const RowCtx& r, int blk, int lane,
                                         int thr, const bf16x8_t* qf, f32x4_t* S,
                                         unsigned long long& suf) {
  constexpr int NKK = D / 32;
  // Slots of this block whose position lies in the recent suffix (bit j = slot blk + j); the
  // appended slot has position t.
  const int ps = blk + (lane & 31);
  const int pj = (r.app && ps == r.L) ? r.tb : B.pos;
  const bool in_suf = lane < 32 && ps < r.n_eff && pj > thr;
  suf = __ballot(in_suf);
  // q.K^T on the matrix cores: lane holds slots blk+8g+4mt+v of head c.
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
    S[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
      S[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(B.k[mt][kk]), qf[kk], S[mt], 0, 0, 0);
  }
}

template <int D>
__device__ __forceinline__ void stage_block(const Block<D>& B, const RowCtx& r, int blk, int g,
                                            int c, int lane, int thr, const bf16x8_t* qf,
                                            uint16_t* vt, f32x4_t* S, unsigned long long& suf) {
  stage_v<D>(B, r, blk, g, c, vt);
  stage_qk<D>(B, r, blk, lane, thr, qf, S, suf);
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

// Second half: online softmax, logit stash, suffix mass, and alpha.V from the LDS tile.
template <int D>
__device__ __forceinline__ void finish_block(const f32x4_t* S, unsigned long long suf,
                                             const RowCtx& r, int blk, int g, int c, int G,
                                             float scale_log2, const StashRow& sr, uint16_t* vt,
                                             Online& st, f32x4_t* O) {
  constexpr int NB = D / 16, RS = vtile_stride<D>();
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

// FG = 0: split mode (one workgroup per split, partials for attend_combine_mfma). FG > 0: fused
// mode, one workgroup per (sequence, KV head) sweeping the whole row (the launch sets the split to
// the cache length), whose epilogue writes the outputs, lse, suffix mass and conf and applies the
// H2O increment itself; FG is a compile-time bound on the group size G.
// Logit stash rows staged in LDS by the split form: SG > 0 keeps the split's logits (at most
// kMaxSplitSlots slots of at most SG heads) in LDS during the sweep and writes them to the stash in
// one coalesced pass at the end; 0 writes them from the loop.
constexpr int kMaxSplitSlots = 1024;
// Split length from which a split-form launch stages its logits in LDS and writes the stash
// once at the end (scattered 16-byte stash stores inside the loop cost the 7B layer ~2.7 us at
// 2048 slots; staging gains 1.1 us there, but adds a store round trip to short splits: batch 1,
// 128-slot splits, +0.3 us).
constexpr int kLdsStashMinSplit = 512;
// Largest batch whose rows the fused form orders by length (the lengths are ranked in LDS).
constexpr int kMaxRankedBatch = 1024;

// -------------------------------------------------------------------------------------------
// One-launch split form (CO). The splits of a row exchange their partials through memory instead
// of a second launch: each workgroup publishes its split partial (per head the max, sum and
// suffix sum, and the output numerators), then waits for the other splits' partials of the row;
// every workgroup merges the row's statistics itself, applies the exact H2O increment to its own
// slots from the logits it kept in LDS (no logit stash in memory), and writes one slice of the
// row's output.
//
// Exchange. Splits of a row may run on different XCDs, whose L2 caches are not coherent with each
// other for ordinary accesses. Every exchanged value is therefore one 64-bit agent-scope atomic
// word, (launch tag << 32) | float bits, which gfx950 stores and loads coherently across XCDs (sc1)
// without a cache write-back or invalidation. A reader polls the words it needs until each carries
// this launch's tag, so every word validates itself: no ordering between different words, no
// arrival counter and no wait for stores to complete is needed. The tag is the row's generation
// word plus one, read by every workgroup of the row at its start; split 0 increments the
// generation once it has seen every split's statistics (by then every workgroup of the row has
// read it), so the next launch expects a tag no word of this one carries.
//
// Residency. A workgroup waits for the other splits of its row, so the form is used only when
// every workgroup of its grid can be resident at once: the host launches it only for grids of at
// most one workgroup per compute unit. A wait is bounded all the same, and a workgroup that gives
// up writes NaN into the acc slots and output entries it owns.
// -------------------------------------------------------------------------------------------
constexpr int kSyncStride = 16;       // u32 words per row in the workspace (word 1: generation)
constexpr int kSpinLimit = 1 << 18;   // polls (each a memory round trip plus a short sleep)

__device__ __forceinline__ unsigned row_generation(const unsigned* sy) {
  return __hip_atomic_load(const_cast<unsigned*>(sy) + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void bump_generation(unsigned* sy) {
  __hip_atomic_fetch_add(sy + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
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

template <int D, int NW, int SG>
__device__ __forceinline__ void row_epilogue(const AttendArgs& a, const f32x4_t* O, uint16_t* vt,
                                             char* smem, const float* slog, float (*sm_m)[16],
                                             float (*sm_l)[16], float (*sm_s)[16],
                                             float (*sm_f)[NW], int b, int hkv, size_t bk,
                                             int split, int ns, int s_lo, int s_hi, int L,
                                             int app, int g, int c, unsigned g0) {
  static_assert(NW == 4, "256 threads: four slots of a 1024-slot split per thread");
  constexpr int VE = D / 16, RS = vtile_stride<D>();
  const int tid = threadIdx.x;
  const int G = a.G;
  const int GD = G * D;
  // This thread's four slots of the split; threads past the split read the split's first quad
  // (in bounds, discarded), so the load is issued unconditionally and early.
  const int j0 = s_lo + 4 * tid;
  const bool live = j0 < s_hi;
  float* acc = a.acc + bk * a.cap;
  const float4 old = *(const float4*)(acc + (live ? j0 : s_lo));
  // The wave's output numerators go to its own V tile (its last alpha.V has read it).
  float* my_o = (float*)vt;
#pragma unroll
  for (int t = 0; t < VE; ++t) {
#pragma unroll
    for (int v = 0; v < 4; ++v) my_o[(4 * g + v) * D + 16 * t + c] = O[t][v];
  }
  // sMs: the split's own max, sum and suffix sum per head (sum and suffix sum only with ns > 1).
  __shared__ float sM[kMaxGroup], srZ[kMaxGroup], sMs[3 * kMaxGroup], sF[kMaxGroup * kMaxMfmaSplits];
  __shared__ unsigned s_tag;
  __shared__ int s_ok;
  if (tid == 0) {
    s_tag = g0 + 1u;
    s_ok = 1;
  }
  __syncthreads();  // every wave's statistics, numerators and logits are in LDS
  const unsigned tag = s_tag;
  // Row partials: numerators [nsq][G*D] then statistics [nsq][G][3] of this row.
  unsigned long long* tn = a.tagged + bk * (size_t)a.nsq * G * (D + 3);
  unsigned long long* ts = tn + (size_t)a.nsq * GD;
  uint16_t* out = (uint16_t*)a.out + ((size_t)b * a.Hq + hkv * G) * D;
  if (tid < G) {
    // The split's statistics per head and each wave's rescaling factor (0 for a wave without
    // slots).
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
    if (ns == 1) {  // the split is the whole row
      sM[h] = M;
      srZ[h] = 1.f / lsum;
      write_row_stats(a, b, hkv, h, M, 1.f / lsum, ssum);
    } else {
      sMs[kMaxGroup + h] = lsum;
      sMs[2 * kMaxGroup + h] = ssum;
    }
  }
  __syncthreads();
  // The split's unnormalised probabilities of this thread's slots, relative to the split's own
  // maxima (exp2(s - m_split)); after the merge each head is scaled by exp2(m_split - M) / Z. A
  // multi-split row computes them after publishing its partial, while it waits for the others.
  float pr[4][SG];
  auto split_probs = [&]() {
    if (live) {
#pragma unroll
      for (int h = 0; h < SG; ++h) {
        const int hc = min(h, G - 1);
        const f32x4_t lg = *(const f32x4_t*)(slog + hc * kMaxSplitSlots + 4 * tid);
        const float ms = sMs[hc];
#pragma unroll
        for (int e = 0; e < 4; ++e) pr[e][h] = exp2f(lg[e] - ms);
      }
    }
  };
  bool ok = true;
  if (ns == 1) {
    split_probs();
    for (int i = tid; i < GD; i += 64 * NW) {
      const int h = i / D;
      float o = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w)
        o += sm_f[h][w] * ((const float*)((const uint16_t*)smem + w * 32 * RS))[i];
      out[i] = f32_to_bf16(o * srZ[h]);
    }
  } else {
    // Publish the split's merged numerators, then its statistics.
    for (int i = tid; i < GD; i += 64 * NW) {
      const int h = i / D;
      float o = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w)
        o += sm_f[h][w] * ((const float*)((const uint16_t*)smem + w * 32 * RS))[i];
      st_tagged(&tn[(size_t)split * GD + i], tag, o);
    }
    if (tid < G) {
      unsigned long long* w = ts + ((size_t)split * G + tid) * 3;
      st_tagged(w, tag, sMs[tid]);
      st_tagged(w + 1, tag, sMs[kMaxGroup + tid]);
      st_tagged(w + 2, tag, sMs[2 * kMaxGroup + tid]);
    }
    // This split merges entries [o_lo, o_lo + cnt) of the row's G x D output: its slice of every
    // split's numerators (split k, entry i at k * per + i) and every split's statistics are polled
    // until each word carries this launch's tag (addresses clamped into the row's partials, unused
    // words ignored, so every load of a poll is issued at once; the first poll's loads are in
    // flight while the split's probabilities are computed), then staged in LDS.
    const int per = (GD + ns - 1) / ns;
    const int o_lo = split * per;
    const int cnt = max(0, min(per, GD - o_lo));
    const int tot = ns * per;
    const int np = ns * G;
    constexpr int kPoIter = (kMaxGroup * D + kMaxMfmaSplits + 255) / 256;
    constexpr int kStIter = (kMaxMfmaSplits * kMaxGroup) / 256;
    unsigned long long pw[kPoIter], sw[kStIter][3];
    size_t pa[kPoIter];
    bool pin[kPoIter];
#pragma unroll
    for (int u = 0; u < kPoIter; ++u) {
      const int idx = tid + 256 * u;
      const int k = idx / per, i = idx - k * per;
      pin[u] = idx < tot && i < cnt;
      pa[u] = pin[u] ? (size_t)k * GD + o_lo + i : 0;
    }
    auto poll = [&]() {
#pragma unroll
      for (int u = 0; u < kPoIter; ++u) pw[u] = ld_tagged(&tn[pa[u]]);
#pragma unroll
      for (int u = 0; u < kStIter; ++u) {
        const int i = min(tid + 256 * u, np - 1);
#pragma unroll
        for (int f = 0; f < 3; ++f) sw[u][f] = ld_tagged(&ts[(size_t)i * 3 + f]);
      }
    };
    auto current = [&]() {
      bool done = true;
#pragma unroll
      for (int u = 0; u < kPoIter; ++u) done = done && (!pin[u] || has_tag(pw[u], tag));
#pragma unroll
      for (int u = 0; u < kStIter; ++u) {
#pragma unroll
        for (int f = 0; f < 3; ++f) done = done && has_tag(sw[u][f], tag);
      }
      return done;
    };
    poll();
    split_probs();
    for (int it = 0; !current(); ++it) {
      if (it == kSpinLimit) {
        s_ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
      poll();
    }
    // Every wave is done reading the V tiles (its numerators were published before it polled), so
    // they can stage the polled numerators. A barrier waits for the wave's outstanding memory
    // operations on gfx950; here the polled words are in and the stores long complete.
    __syncthreads();
    __shared__ float2 sml[kMaxMfmaSplits * kMaxGroup];
    __shared__ float sps[kMaxMfmaSplits * kMaxGroup];
#pragma unroll
    for (int u = 0; u < kStIter; ++u) {
      if (tid + 256 * u < np) {
        sml[tid + 256 * u] = make_float2(tagged_value(sw[u][0]), tagged_value(sw[u][1]));
        sps[tid + 256 * u] = tagged_value(sw[u][2]);
      }
    }
    float* spo = (float*)smem;
#pragma unroll
    for (int u = 0; u < kPoIter; ++u) spo[tid + 256 * u] = pin[u] ? tagged_value(pw[u]) : 0.f;
    __syncthreads();  // every split's statistics and this slice of its numerators are in LDS
    ok = s_ok != 0;
    // Split 0 has now seen every split's statistics, so every workgroup of the row has read the
    // generation word: the next launch may expect a new tag.
    if (split == 0 && tid == 0) bump_generation(a.sync + bk * kSyncStride);
    if (tid < G) {
      const int h = tid;
      float M = -INFINITY;
      for (int k = 0; k < ns; ++k) M = fmaxf(M, sml[k * G + h].x);
      float Z = 0.f, S = 0.f;
      for (int k = 0; k < ns; ++k) {
        const float f = exp2f(sml[k * G + h].x - M);
        sF[h * kMaxMfmaSplits + k] = f;
        Z += sml[k * G + h].y * f;
        S += sps[k * G + h] * f;
      }
      sM[h] = M;
      srZ[h] = 1.f / Z;
      if (split == 0) write_row_stats(a, b, hkv, h, M, 1.f / Z, S);
    }
    __syncthreads();
    for (int i = tid; i < cnt; i += 256) {
      const int h = (o_lo + i) / D;
      float o = 0.f;
      for (int k = 0; k < ns; ++k) o += sF[h * kMaxMfmaSplits + k] * spo[k * per + i];
      out[o_lo + i] = ok ? f32_to_bf16(o * srZ[h]) : (uint16_t)0x7fc0;
    }
  }
  // H2O increment of this split's slots: alpha = exp2(s - m_split) * exp2(m_split - M) / Z; slots
  // past the split keep their bits; heads past G (padding up to SG) are masked by a select.
  if (live) {
    float fh[SG];
#pragma unroll
    for (int h = 0; h < SG; ++h) {
      const int hc = min(h, G - 1);
      fh[h] = exp2f(sMs[hc] - sM[hc]) * srZ[hc];
    }
    float4 nv;
    float* nvp = (float*)&nv;
    const float* ov = (const float*)&old;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float sum = 0.f;
#pragma unroll
      for (int h = 0; h < SG; ++h) sum += h < G ? pr[e][h] * fh[h] : 0.f;
      const int j = j0 + e;
      const float nx = (app && j == L) ? sum : ov[e] + sum;
      nvp[e] = j < s_hi ? (ok ? nx : __int_as_float(0x7fc00000)) : ov[e];
    }
    *(float4*)(acc + j0) = nv;
  }
}

template <int D, int NW, bool PIPE, bool DYN, bool NT, int FG, int SG, bool CO>
__device__ __forceinline__ void attend_mfma_body(const AttendArgs& a) {
  static_assert(!CO || (FG == 0 && SG > 0 && NW * 64 * 4 >= kMaxSplitSlots),
                "the one-launch split form keeps every logit of its split in LDS and updates four "
                "slots per thread");
  constexpr int NKK = D / 32;   // k-steps of the q.K^T product
  constexpr int VE = D / 16;    // V dims per lane per row
  // Grid (kv head, sequence, split): the split is the slowest index, so consecutive workgroups
  // (which the dispatcher deals round-robin to the 8 XCDs) belong to different rows, the busy
  // splits of a launch spread over every XCD even when some split indices have no slots, and the
  // splits of one row share an XCD (and its L2) with the row's combine workgroups.
  const int split = blockIdx.z;
  int hkv = blockIdx.x, b = blockIdx.y;
  if (FG > 0 && a.B <= kMaxRankedBatch) {
    // Fused form: longest rows first. Workgroups are dispatched in (kv head, sequence) order; the
    // one with dispatch index w takes kv head w % Hkv of the sequence ranked w / Hkv by cached
    // length (longest first, ties by index), so long rows start in the first round of the grid.
    __shared__ int s_len[kMaxRankedBatch];
    __shared__ int s_b;
    for (int i = threadIdx.x; i < a.B; i += 64 * NW) s_len[i] = min(max(a.len[i], 0), a.cap);
    __syncthreads();
    const int w = blockIdx.y * gridDim.x + blockIdx.x;
    const int want = w / a.Hkv;
    for (int i = threadIdx.x; i < a.B; i += 64 * NW) {
      const int li = s_len[i];
      int rank = 0;
      for (int j = 0; j < a.B; ++j) {
        const int lj = s_len[j];
        rank += (lj > li || (lj == li && j < i)) ? 1 : 0;
      }
      if (rank == want) s_b = i;
    }
    __syncthreads();
    b = s_b;
    hkv = w - want * a.Hkv;
  }
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = lane >> 4, c = lane & 15;
  const int G = a.G;
  const size_t bk = (size_t)b * a.Hkv + hkv;
  int L, app;
  const int n_eff = live_slots(a, b, &L, &app);
  if (n_eff == 0) {  // the combine writes the empty result, or the fused / one-launch form here
    if (FG > 0 || (CO && split == 0)) {
      uint16_t* out = (uint16_t*)a.out + ((size_t)b * a.Hq + hkv * G) * D;
      for (int i = threadIdx.x; i < G * D; i += 64 * NW) out[i] = 0;
      if (threadIdx.x < G) {
        a.lse[(size_t)b * a.Hq + hkv * G + threadIdx.x] = -INFINITY;
        a.suffix_mass[(size_t)b * a.Hq + hkv * G + threadIdx.x] = 0.f;
      }
    }
    return;
  }
  const SplitPlan plan = split_plan(n_eff, a.split);
  if (split >= plan.ns) return;
  const int s_lo = split * plan.chunk;
  const int s_hi = min(s_lo + plan.chunk, n_eff);
  const int nblk = (s_hi - s_lo + 31) / 32;
  const int cap = a.cap;
  const uint16_t* Kb = (const uint16_t*)a.k + bk * cap * D;
  const uint16_t* Vb = (const uint16_t*)a.v + bk * cap * D;
  if (app && L >= s_lo && L < s_hi) {  // append row L before any wave of this split reads it
    if (threadIdx.x < 2 * (D / 8)) {
      const int which = threadIdx.x / (D / 8), piece = threadIdx.x % (D / 8);
      const uint4* src = (const uint4*)((const uint16_t*)(which ? a.v_new : a.k_new) + bk * D) + piece;
      uint4* dst = (uint4*)((uint16_t*)(which ? a.v_w : a.k_w) + (bk * cap + L) * D) + piece;
      *dst = *src;
    }
    __syncthreads();
  }
  // One-launch form: the row's generation word, read long before this workgroup arrives.
  unsigned g0 = 0;
  if (CO && plan.ns > 1 && threadIdx.x == 0) g0 = row_generation(a.sync + bk * kSyncStride);
  RowCtx r;
  r.kbase = Kb + (size_t)(8 * (c >> 2) + (c & 3)) * D + 8 * g;
  r.vbase = Vb + (size_t)(4 * g) * D + (D / 16) * c;
  r.posb = a.pos + (size_t)b * cap;
  r.L = L;
  r.app = app;
  r.cap = cap;
  r.n_eff = n_eff;
  r.tb = a.t[b];

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
  const int thr = sat_sub(a.t[b], a.suffix_w[b]);
  __shared__ __attribute__((aligned(16))) float slog[SG > 0 ? SG * kMaxSplitSlots : 4];
  // With SG > 0 (launches whose splits are long, kLdsStashMinSplit) the logits are staged in LDS
  // and written to the stash once at the end; otherwise they are stored from the loop.
  StashRow stash_row;
  stash_row.use_lds = SG > 0;
  stash_row.lds = (lds_float*)slog + (c < G ? c : 0) * (SG > 0 ? kMaxSplitSlots : 0);
  stash_row.glob = a.stash + (bk * G + (c < G ? c : 0)) * a.cap_s;
  stash_row.lo = s_lo;

  Online st{-INFINITY, 0.f, 0.f};
  f32x4_t O[VE];
#pragma unroll
  for (int rr = 0; rr < VE; ++rr) O[rr] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // LDS: per-wave V tiles during the sweep, then the wave partials for the merge.
  constexpr int RS = vtile_stride<D>();
  constexpr size_t kTileBytes = (size_t)NW * 32 * RS * 2;
  constexpr size_t kMergeBytes = (size_t)NW * 16 * D * 4;
  __shared__ __attribute__((aligned(16))) char smem[kTileBytes > kMergeBytes ? kTileBytes : kMergeBytes];
  uint16_t* vt = (uint16_t*)smem + wave * 32 * RS;

  // With PIPE the next block's V rows are loaded as soon as the current ones are in LDS and its K
  // rows right after the current q.K^T (into the same, now free, registers), so they are in
  // flight during the current block's softmax and alpha.V.
  // Block assignment: with DYN each wave takes its first block (index = wave) and then the next
  // unclaimed block of the split from a workgroup counter in LDS, so waves that get their data
  // sooner take more blocks and the waves of the workgroup finish together; otherwise wave w takes
  // blocks w, w + NW, ...
  const int nb = wave < nblk ? (nblk - wave + NW - 1) / NW : 0;
  Block<D> A;
  f32x4_t S[2];
  unsigned long long suf;
  if (DYN) {
    __shared__ int s_next;
    if (threadIdx.x == 0) s_next = NW;
    __syncthreads();
    int bi = wave;
    if (bi < nblk) load_block<D, NT>(A, r, s_lo + 32 * bi, lane);
    while (bi < nblk) {
      const int blk = s_lo + 32 * bi;
      stage_block<D>(A, r, blk, g, c, lane, thr, qf, vt, S, suf);
      int nx = 0;
      if (lane == 0) nx = atomicAdd(&s_next, 1);
      nx = __builtin_amdgcn_readfirstlane(nx);
      if (nx < nblk) load_block<D, NT>(A, r, s_lo + 32 * nx, lane);
      finish_block<D>(S, suf, r, blk, g, c, G, a.scale_log2, stash_row, vt, st, O);
      bi = nx;
    }
  } else if (PIPE) {
    // The last block is peeled so the loop's loads are unconditional: the wait counts at the loop
    // head then let the V rows be staged while the K rows of the same block are still in flight.
    if (nb > 0) {
      load_block<D, NT>(A, r, s_lo + 32 * wave, lane);
      for (int i = 0; i + 1 < nb; ++i) {
        const int blk = s_lo + 32 * (wave + NW * i);
        stage_v<D>(A, r, blk, g, c, vt);
        load_v<D, NT>(A, r, blk + 32 * NW);
        stage_qk<D>(A, r, blk, lane, thr, qf, S, suf);
        load_k<D, NT>(A, r, blk + 32 * NW, lane);
        finish_block<D>(S, suf, r, blk, g, c, G, a.scale_log2, stash_row, vt, st, O);
      }
      const int blk = s_lo + 32 * (wave + NW * (nb - 1));
      stage_block<D>(A, r, blk, g, c, lane, thr, qf, vt, S, suf);
      finish_block<D>(S, suf, r, blk, g, c, G, a.scale_log2, stash_row, vt, st, O);
    }
  } else {
    for (int i = 0; i < nb; ++i) {
      const int blk = s_lo + 32 * (wave + NW * i);
      load_block<D, NT>(A, r, blk, lane);
      stage_block<D>(A, r, blk, g, c, lane, thr, qf, vt, S, suf);
      finish_block<D>(S, suf, r, blk, g, c, G, a.scale_log2, stash_row, vt, st, O);
    }
  }

  // Merge the waves of the workgroup into one partial for this split.
  float l_run = st.l, s_run = st.s;
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  s_run += __shfl_xor(s_run, 16, 64);
  s_run += __shfl_xor(s_run, 32, 64);
  __shared__ float sm_m[NW][16], sm_l[NW][16], sm_s[NW][16], sm_f[16][NW];
  float(*sm_o)[16][D] = (float(*)[16][D])smem;  // reuses the V tiles
  if (g == 0) {
    sm_m[wave][c] = st.m;
    sm_l[wave][c] = l_run;
    sm_s[wave][c] = s_run;
  }
  if constexpr (CO) {
    row_epilogue<D, NW, SG>(a, O, vt, smem, slog, sm_m, sm_l, sm_s, sm_f, b, hkv, bk, split,
                            plan.ns, s_lo, s_hi, L, app, g, c, g0);
    return;
  }
  if constexpr (FG == 0) {
    // Split form. Each wave, as soon as its own loop is done, puts its output numerators into its
    // own V tile (its last alpha.V has read it) and copies its blocks' logits from the LDS copy to
    // the stash, 16 B per lane (head hh + lane / 8, slots 4 (lane % 8).. of the block), so the
    // waves that finish first do this while the others still stream (7B shape at 2048 slots:
    // 30.3 -> 29.5 us per layer).
    float* my_o = (float*)vt;  // [16][D]
#pragma unroll
    for (int t = 0; t < VE; ++t) {
#pragma unroll
      for (int v = 0; v < 4; ++v) my_o[(4 * g + v) * D + 16 * t + c] = O[t][v];
    }
    if (stash_row.use_lds) {
      for (int i = 0; i < nb; ++i) {
        const int off = 32 * (wave + NW * i);  // the block's first slot, relative to s_lo
#pragma unroll
        for (int hh = 0; hh < (SG > 0 ? SG : 1); hh += 8) {
          const int h = hh + (lane >> 3), q = lane & 7;
          if (h < G)
            *(float4*)(a.stash + (bk * G + h) * a.cap_s + s_lo + off + 4 * q) =
                *(const float4*)(slog + h * kMaxSplitSlots + off + 4 * q);
        }
      }
    }
    __syncthreads();  // every wave's statistics and numerators are in LDS
    // Per head: the split's max, each wave's rescaling factor (0 for a wave without slots), the
    // split's softmax sum and suffix mass; then the merged numerators.
    const size_t pbase = (bk * a.ns_max + split) * G;
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
    __syncthreads();
    for (int i = threadIdx.x; i < G * D; i += 64 * NW) {
      const int h = i / D, d = i - h * D;
      float o = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w)
        o += sm_f[h][w] * ((const float*)((const uint16_t*)smem + w * 32 * RS))[h * D + d];
      a.part_o[(pbase + h) * D + d] = o;
    }
    return;
  }
  // Fused form: the waves are merged into the row's final result.
  __syncthreads();  // every wave is done with its V tile
  // O[nb] lane (g, c): heads 4g + v, dim 16 nb + c
#pragma unroll
  for (int nb = 0; nb < VE; ++nb) {
#pragma unroll
    for (int v = 0; v < 4; ++v) sm_o[wave][4 * g + v][16 * nb + c] = O[nb][v];
  }
  // Per head: the row's max, each wave's rescaling factor (0 for a wave without slots), the
  // softmax sum and suffix mass, then the final statistics and the confidence proxy (max over
  // the group's heads).
  __shared__ float sm_M[16], sm_rZ[16];
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
    {
      const float rZ = 1.f / lsum;
      const float sg = ssum * rZ;
      sm_M[h] = M;
      sm_rZ[h] = rZ;
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
  }
  __syncthreads();  // also publishes this workgroup's stash stores to its own waves
  // Fused epilogue. H2O increment of every live slot, four consecutive slots per thread: the
  // stash logits of the FG (clamped) heads and the old acc values are loaded first, then the
  // increments; padding heads past G are masked by a select.
  {
    float mh[FG > 0 ? FG : 1], rzh[FG > 0 ? FG : 1];
#pragma unroll
    for (int h = 0; h < FG; ++h) {
      mh[h] = sm_M[min(h, G - 1)];
      rzh[h] = sm_rZ[min(h, G - 1)];
    }
    const float* stash = a.stash + bk * G * a.cap_s;
    float* acc = a.acc + bk * cap;
    for (int j0 = 4 * (int)threadIdx.x; j0 < n_eff; j0 += 4 * 64 * NW) {
      const float4 old = *(const float4*)(acc + j0);
      float4 lgv[FG > 0 ? FG : 1];
#pragma unroll
      for (int h = 0; h < FG; ++h)
        lgv[h] = *(const float4*)(stash + (size_t)min(h, G - 1) * a.cap_s + j0);
      float4 nv;
      float* nvp = (float*)&nv;
      const float* ov = (const float*)&old;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float sum = 0.f;
#pragma unroll
        for (int h = 0; h < FG; ++h) {
          const float pr = exp2f(((const float*)&lgv[h])[e] - mh[h]) * rzh[h];
          sum += h < G ? pr : 0.f;
        }
        const int j = j0 + e;
        nvp[e] = j < n_eff ? ((app && j == L) ? sum : ov[e] + sum) : ov[e];
      }
      *(float4*)(acc + j0) = nv;
    }
  }
  uint16_t* out = (uint16_t*)a.out + ((size_t)b * a.Hq + hkv * G) * D;
  for (int i = threadIdx.x; i < G * D; i += 64 * NW) {
    const int h = i / D, d = i % D;
    float o = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) o += sm_f[h][w] * sm_o[w][h][d];
    out[i] = f32_to_bf16(o * sm_rZ[h]);
  }
}

// Kernel entry points: WPE is the occupancy target (waves per SIMD) given to the register
// allocator.
template <int D, int NW, bool PIPE, int WPE, bool DYN, bool NT, int FG = 0, int SG = 0, bool CO = false>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(WPE, 8)))
void attend_mfma(AttendArgs a) {
  attend_mfma_body<D, NW, PIPE, DYN, NT, FG, SG, CO>(a);
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
  const float2* pml = a.part_ml + bk * a.ns_max * G;
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
  const float* po = a.part_o + bk * a.ns_max * G * D;
  for (int i = tid; i < G * D; i += 256) {
    const int h = i / D;
    float o = 0.f;
    for (int k = 0; k < ns; ++k) o += exp2f(pml[k * G + h].x - sM[h]) * po[(size_t)k * G * D + i];
    out[i] = from_f32<T>(o * srZ[h]);
  }
  if (tid < G) {
    const float* ps = a.part_s + bk * a.ns_max * G;
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
// Combine for the MFMA sweep (balanced split plan). One workgroup per split, same grid as the
// sweep so a split's stash is read back on the XCD that wrote it. Each workgroup applies the H2O
// increment to its split's slots (four consecutive slots per thread, 16-byte accesses) and merges
// one slice of the row's output; all of its loads (stash logits, old acc values, its output slice
// of every split partial, staged in LDS, and the split maxima and sums) are issued before the
// first barrier, so the workgroup waits for memory once. GM is a compile-time bound on the group
// size G.
// -------------------------------------------------------------------------------------------
template <int D, int GM>
__global__ __launch_bounds__(256) void attend_combine_mfma(AttendArgs a) {
  const int split = blockIdx.z, hkv = blockIdx.x, b = blockIdx.y;  // the sweep's grid
  const int tid = threadIdx.x;
  const int G = a.G;
  int L, app;
  const int n_eff = live_slots(a, b, &L, &app);
  const size_t bk = (size_t)b * a.Hkv + hkv;
  uint16_t* out = (uint16_t*)a.out + ((size_t)b * a.Hq + hkv * G) * D;
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
  if (split >= ns) return;
  const int lo = split * plan.chunk, hi = min(lo + plan.chunk, n_eff);
  const float2* pml = a.part_ml + bk * a.ns_max * G;
  const float* ps = a.part_s + bk * a.ns_max * G;
  const int np = ns * G;
  // Slots j0..j0+3 of this thread (splits are at most 1024 slots). Threads past the split read
  // the split's first quad instead (in bounds, discarded), so no load sits behind a branch. The
  // sweep wrote -inf logits for the slots of a split's last block that lie past n_eff.
  const int j0 = lo + 4 * tid;
  const bool live = j0 < hi;
  const int jl = live ? j0 : lo;
  const float* stash = a.stash + bk * G * a.cap_s;
  float* acc = a.acc + bk * a.cap;
  const float4 old = *(const float4*)(acc + jl);
  float4 lgv[GM];
#pragma unroll
  for (int h = 0; h < GM; ++h)
    lgv[h] = *(const float4*)(stash + (size_t)min(h, G - 1) * a.cap_s + jl);
  // This split also merges a slice of the row's output: entries [o_lo, o_lo + cnt) of the G x D
  // block. Its partials, ns x per values (split k, entry i at k * per + i), go to LDS: at most
  // G * D + ns values, kPoIter per thread, every load issued before the barrier.
  const int GD = G * D;
  const int per = (GD + ns - 1) / ns;
  const int o_lo = split * per;
  const int cnt = max(0, min(per, GD - o_lo));
  const int tot = ns * per;
  const float* po = a.part_o + bk * a.ns_max * G * D;
  constexpr int kPoIter = (kMaxGroup * D + kMaxMfmaSplits + 255) / 256;
  __shared__ float spo[kPoIter * 256];
  float pov[kPoIter];
#pragma unroll
  for (int u = 0; u < kPoIter; ++u) {
    const int idx = tid + 256 * u;
    const int k = idx / per, i = idx - k * per;
    const bool in = idx < tot && i < cnt;
    pov[u] = po[in ? (size_t)k * GD + o_lo + i : 0];
  }
  __shared__ float2 sml[kMaxMfmaSplits * kMaxGroup];
  __shared__ float sps[kMaxMfmaSplits * kMaxGroup];
  __shared__ float sM[kMaxGroup], srZ[kMaxGroup], sF[kMaxGroup * kMaxMfmaSplits];
  for (int i = tid; i < np; i += 256) {
    sml[i] = pml[i];
    sps[i] = ps[i];
  }
#pragma unroll
  for (int u = 0; u < kPoIter; ++u) spo[tid + 256 * u] = pov[u];
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
    const float* ov = (const float*)&old;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float sum = 0.f;
#pragma unroll
      for (int h = 0; h < GM; ++h) {
        const float pr = exp2f(((const float*)&lgv[h])[e] - mh[h]) * rzh[h];
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

template <typename T, int D>
static hipError_t launch_valu(AttendArgs a, hipStream_t st) {
  a.split = kSplitQuantum;
  dim3 grid((a.cap + a.split - 1) / a.split, a.Hkv, a.B);
  hipLaunchKernelGGL((attend_valu<T, D>), grid, dim3(64), 0, st, a);
  hipLaunchKernelGGL((attend_combine<T, D>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

// Workgroups one sweep launch aims for (one per CU) when rows are few: the split length shrinks
// from its maximum until the launch has about this many, but never below one block per wave.
constexpr long kTargetWorkgroups = 256;

// Above this many K/V bytes per layer the sweep streams with non-temporal loads (a model's cache
// of such layers does not stay in the 256 MB last-level cache between decode steps).
constexpr double kStreamBytes = 16.0 * 1024 * 1024;

// Split length of an MFMA launch: max_split, or with `adaptive` shorter when the launch has few
// rows (down to one block per wave), but long enough for at most kMaxMfmaSplits splits per row
// (the merges keep every split's partial in LDS).
static int mfma_split(const AttendArgs& a, int max_split, bool adaptive, int NW) {
  const int min_split = ((a.cap + kMaxMfmaSplits - 1) / kMaxMfmaSplits + 31) & ~31;
  int split = max_split;
  if (adaptive) {
    const long rows = (long)a.B * a.Hkv;
    long want = ((long)a.cap * rows + kTargetWorkgroups - 1) / kTargetWorkgroups;
    want = (want + 31) & ~31L;
    if (want < 32 * NW) want = 32 * NW;
    if (want < split) split = (int)want;
  }
  return split > min_split ? split : min_split;
}

template <int D, int NW, bool PIPE, int WPE, bool DYN = false, bool NT = true, bool LS = false>
static hipError_t launch_mfma(AttendArgs a, int max_split, bool adaptive, hipStream_t st) {
  a.split = mfma_split(a, max_split, adaptive, NW);
  if (a.split > 1024) return hipErrorInvalidValue;  // the combine covers 1024 slots per split
  dim3 grid(a.Hkv, a.B, (a.cap + a.split - 1) / a.split);
  if constexpr (!LS) {
    hipLaunchKernelGGL((attend_mfma<D, NW, PIPE, WPE, DYN, NT>), grid, dim3(64 * NW), 0, st, a);
  } else if (a.split < kLdsStashMinSplit) {
    hipLaunchKernelGGL((attend_mfma<D, NW, PIPE, WPE, DYN, NT>), grid, dim3(64 * NW), 0, st, a);
  } else {
    if (a.G <= 4)
      hipLaunchKernelGGL((attend_mfma<D, NW, PIPE, WPE, DYN, NT, 0, 4>), grid, dim3(64 * NW), 0, st, a);
    else if (a.G <= 8)
      hipLaunchKernelGGL((attend_mfma<D, NW, PIPE, WPE, DYN, NT, 0, 8>), grid, dim3(64 * NW), 0, st, a);
    else
      hipLaunchKernelGGL((attend_mfma<D, NW, PIPE, WPE, DYN, NT, 0, 16>), grid, dim3(64 * NW), 0, st, a);
  }
  if (a.G <= 4)
    hipLaunchKernelGGL((attend_combine_mfma<D, 4>), grid, dim3(256), 0, st, a);
  else if (a.G <= 8)
    hipLaunchKernelGGL((attend_combine_mfma<D, 8>), grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((attend_combine_mfma<D, 16>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}


// Fused form: one 8-wave workgroup per (sequence, KV head) over the whole row; no combine launch.
// Variants 15 and 16 only. With the split form's grid ordered for the XCDs (split index slowest)
// the split form is faster at every row count measured: 7B shape at 128 / 256 / 384 / 512 rows
// 26.3 / 44.3 / 65.6 / 88.1 us per layer against 34.1 / 45.7 / 80.4 / 97.6 us, the ragged batch
// 64 258 against 243 steps/s, batch 1 10.2 against 19.9 us.
template <int D, bool NT>
static hipError_t launch_fused(AttendArgs a, hipStream_t st) {
  a.split = (a.cap + 31) & ~31;  // one split per row
  dim3 grid(a.Hkv, a.B, 1);
  if (a.G <= 4)
    hipLaunchKernelGGL((attend_mfma<D, 8, true, 2, false, NT, 4>), grid, dim3(512), 0, st, a);
  else if (a.G <= 8)
    hipLaunchKernelGGL((attend_mfma<D, 8, true, 2, false, NT, 8>), grid, dim3(512), 0, st, a);
  else
    hipLaunchKernelGGL((attend_mfma<D, 8, true, 2, false, NT, 16>), grid, dim3(512), 0, st, a);
  return hipGetLastError();
}

// The split form as the automatic choice uses it: splits of at most 1024 slots (shorter when the
// launch has few rows), logits staged in LDS for long splits, non-temporal loads for large caches.
template <int D>
static hipError_t launch_split_default(AttendArgs a, hipStream_t st) {
  const double kv = 4.0 * a.B * a.Hkv * (double)a.cap * D;
  if (kv >= kStreamBytes) return launch_mfma<D, 4, true, 2, false, true, true>(a, 1024, true, st);
  return launch_mfma<D, 4, true, 2, false, false, true>(a, 1024, true, st);
}

// Workgroups of the one-launch form the host lets wait for each other: one per compute unit of the
// current device (0 if the kernel does not fit on a CU at all), queried once per device and kernel.
// The occupancy query reports two of these workgroups per CU, but grids of 384 and 512 of them
// (7B-shaped batch 32 with 768- and 512-slot splits) were not all resident at once: some waits ran
// into their bound. A grid of at most one workgroup per CU has always been resident.
constexpr int kMaxDevices = 64;
template <int D, bool NT, int SG>
static long row_form_capacity() {
  static long cache[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
  long c = __atomic_load_n(&cache[dev], __ATOMIC_RELAXED);
  if (c == 0) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &per_cu, reinterpret_cast<const void*>(&attend_mfma<D, 4, true, 2, false, NT, 0, SG, true>),
            256, 0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    c = per_cu >= 1 ? (long)cus : -1;
    __atomic_store_n(&cache[dev], c, __ATOMIC_RELAXED);
  }
  return c;
}

// One-launch split form (sweep, row barrier and merge in one kernel), used when every workgroup
// of the grid can be resident at once; otherwise the split form with its merge launch.
template <int D, bool NT, int SG>
static hipError_t launch_row_sg(AttendArgs a, hipStream_t st) {
  a.split = mfma_split(a, 1024, true, 4);
  if (a.split > kMaxSplitSlots) return hipErrorInvalidValue;
  dim3 grid(a.Hkv, a.B, (a.cap + a.split - 1) / a.split);
  const long n = (long)grid.x * grid.y * grid.z;
  if (n > row_form_capacity<D, NT, SG>()) return launch_split_default<D>(a, st);
  hipLaunchKernelGGL((attend_mfma<D, 4, true, 2, false, NT, 0, SG, true>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

template <int D, bool NT>
static hipError_t launch_row_nt(AttendArgs a, hipStream_t st) {
  if (a.G <= 4) return launch_row_sg<D, NT, 4>(a, st);
  if (a.G <= 8) return launch_row_sg<D, NT, 8>(a, st);
  return launch_row_sg<D, NT, 16>(a, st);
}

template <int D>
static hipError_t launch_row(AttendArgs a, hipStream_t st) {
  const double kv = 4.0 * a.B * a.Hkv * (double)a.cap * D;
  if (kv >= kStreamBytes) return launch_row_nt<D, true>(a, st);
  return launch_row_nt<D, false>(a, st);
}

// MFMA kernel configurations: variant 2 is the default (the split form: splits of at most 1024
// slots, shorter when the launch has few rows; non-temporal loads for large caches); 3.. are
// tuning alternatives with the same results (pipelining, occupancy target,
// workgroup size, fixed split length, load kind; 9 is the split form exactly as the automatic
// choice uses it, 14 the split form with normal loads, 15/16 the fused form with non-temporal /
// normal loads).
template <int D>
static hipError_t launch_mfma_variant(AttendArgs a, int variant, hipStream_t st) {
  switch (variant) {
    case 3: return launch_mfma<D, 4, true, 3>(a, 512, false, st);
    case 4: return launch_mfma<D, 4, true, 2>(a, 512, false, st);
    case 5: return launch_mfma<D, 4, false, 2>(a, 512, false, st);
    case 6: return launch_mfma<D, 4, false, 3>(a, 512, false, st);
    case 7: return launch_mfma<D, 8, false, 2>(a, 1024, false, st);
    case 8: return launch_mfma<D, 8, true, 2>(a, 1024, false, st);
    case 9: return launch_split_default<D>(a, st);
    case 10: return launch_mfma<D, 4, true, 2>(a, 256, false, st);
    case 11: return launch_mfma<D, 8, true, 2, true>(a, 1024, false, st);
    case 12: return launch_mfma<D, 4, true, 2, true>(a, 512, false, st);
    case 13: return launch_mfma<D, 16, false, 4, true>(a, 1024, false, st);
    case 14: return launch_mfma<D, 4, true, 2, false, false>(a, 1024, true, st);
    case 15: return launch_fused<D, true>(a, st);
    case 16: return launch_fused<D, false>(a, st);
    case 17: return launch_row<D>(a, st);
    default: return launch_row<D>(a, st);
  }
}

hipError_t launch_attend(AttendArgs a, lg_dtype dt, int D, int variant, hipStream_t st) {
  if (variant >= 2)
    return D == 128 ? launch_mfma_variant<128>(a, variant, st) : launch_mfma_variant<64>(a, variant, st);
  if (dt == LG_BF16)
    return D == 128 ? launch_valu<uint16_t, 128>(a, st) : launch_valu<uint16_t, 64>(a, st);
  return D == 128 ? launch_valu<float, 128>(a, st) : launch_valu<float, 64>(a, st);
}

}  // namespace lg

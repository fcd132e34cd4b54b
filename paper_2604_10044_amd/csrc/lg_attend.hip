// lg_attend.hip -- decode attention over the fixed-budget cache with fused loop statistics.
//
// Eq. (1) of the paper (Sec. 3.1) per query head over the live slots of the cache, plus the
// statistics the guard consumes, all from one sweep over K/V:
//   suffix mass   sum of alpha over slots with pos > t - w_s (attention on the narrow recent
//                 suffix; head locking, Sec. 1 and App. E)
//   H2O increment acc[j] += sum over the group's query heads of alpha_j (Sec. 2.2, Sec. 6.1)
//   confidence    conf[b] = max(conf[b], max_h suffix mass)
//
// Split-K: the slots of each (sequence, kv head) are cut into splits; each workgroup produces a
// partial (running max, running sum, suffix sum, un-normalised output) per query head and
// writes its logits to a stash. attend_combine merges the partials (exact softmax over all
// splits), writes out/lse/suffix mass, and applies the exact H2O increment from the stash.
//
// Two sweep kernels:
//   attend_valu  portable vector-ALU kernel (float32 or bfloat16 cache, head_dim 64/128).
//   attend_mfma  bfloat16 cache: the GQA group product q.K^T runs on 16x16x32 bf16 MFMA with
//                K rows loaded straight into the A operand (16 B per lane), and alpha.V on
//                16x16x4 f32 MFMA with V rows loaded straight into the B operand (each lane reads
//                8 consecutive dims of one row; the output column j holds dims 8j..8j+7, one MFMA
//                per dim offset), so neither operand needs an LDS transpose and alpha stays fp32.
#include "lg_internal.h"

namespace lg {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

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
  const int thr = a.t[b] - a.suffix_w[b];
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
// MFMA sweep (bfloat16 cache). NW waves per workgroup, BPW blocks of 32 slots per wave.
// Lane l = 16 g + c: head c of the group for the logits, row group g.
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

template <int VE>
__device__ __forceinline__ VRow<VE> load_vrow(const uint16_t* p);
template <> __device__ __forceinline__ VRow<8> load_vrow<8>(const uint16_t* p) { return {*(const uint4*)p}; }
template <> __device__ __forceinline__ VRow<4> load_vrow<4>(const uint16_t* p) { return {*(const uint2*)p}; }

__device__ __forceinline__ float vrow_elem(const VRow<8>& v, int r) {
  const uint32_t w = r < 2 ? v.w.x : r < 4 ? v.w.y : r < 6 ? v.w.z : v.w.w;
  return (r & 1) ? __uint_as_float(w & 0xffff0000u) : __uint_as_float(w << 16);
}
__device__ __forceinline__ float vrow_elem(const VRow<4>& v, int r) {
  const uint32_t w = r < 2 ? v.w.x : v.w.y;
  return (r & 1) ? __uint_as_float(w & 0xffff0000u) : __uint_as_float(w << 16);
}

template <int D, int NW, int BPW>
__global__ __launch_bounds__(64 * NW) void attend_mfma(AttendArgs a) {
  constexpr int NKK = D / 32;   // k-steps of the q.K^T product
  constexpr int VE = D / 16;    // V dims per lane per row
  constexpr int SPLIT = NW * BPW * 32;
  const int split = blockIdx.x, hkv = blockIdx.y, b = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = lane >> 4, c = lane & 15;
  int L, app;
  const int n_eff = live_slots(a, b, &L, &app);
  const int s_lo = split * SPLIT;
  if (s_lo >= n_eff) return;
  const int G = a.G;
  const int cap = a.cap;
  const size_t bk = (size_t)b * a.Hkv + hkv;
  const uint16_t* Kb = (const uint16_t*)a.k + bk * cap * D;
  const uint16_t* Vb = (const uint16_t*)a.v + bk * cap * D;
  const uint16_t* kn = app ? (const uint16_t*)a.k_new + bk * D : nullptr;
  const uint16_t* vn = app ? (const uint16_t*)a.v_new + bk * D : nullptr;

  if (app && L >= s_lo && L < s_lo + SPLIT && threadIdx.x < 2 * (D / 8)) {  // append row L
    const int which = threadIdx.x / (D / 8), piece = threadIdx.x % (D / 8);
    const uint4* src = (const uint4*)(which ? vn : kn) + piece;
    uint4* dst = (uint4*)((uint16_t*)(which ? a.v_w : a.k_w) + (bk * cap + L) * D) + piece;
    *dst = *src;
  }

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
  const int thr = a.t[b] - a.suffix_w[b];
  const int tb = a.t[b];
  const int32_t* posb = a.pos + (size_t)b * cap;
  float* stash_row = a.stash + (bk * G + (c < G ? c : 0)) * a.cap_s;

  float m_run = -INFINITY, l_run = 0.f, s_run = 0.f;
  f32x4_t O[VE];
#pragma unroll
  for (int r = 0; r < VE; ++r) O[r] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int wave_lo = s_lo + wave * BPW * 32;
  for (int bi = 0; bi < BPW; ++bi) {
    const int blk = wave_lo + bi * 32;
    if (blk >= n_eff) break;
    // K rows for the A operand: tile m, row c of the tile, dims kk*32 + 8g .. +8.
    uint4 kf[2][NKK];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const int row = blk + 16 * mt + c;
      const uint16_t* src = (app && row == L) ? kn : Kb + (size_t)min(row, cap - 1) * D;
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) kf[mt][kk] = *(const uint4*)(src + kk * 32 + 8 * g);
    }
    // V rows for the B operand: rows blk + 16 mt + 4 g + v, dims VE*c .. +VE.
    VRow<VE> vf[2][4];
    int pv[2][4];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = blk + 16 * mt + 4 * g + v;
        const bool nw = app && row == L;
        const int rc = min(row, cap - 1);
        vf[mt][v] = load_vrow<VE>((nw ? vn : Vb + (size_t)rc * D) + VE * c);
        pv[mt][v] = nw ? tb : posb[rc];
      }
    }
    // q.K^T on the matrix cores: S[mt] lane holds slots blk+16mt+4g+v, head c.
    f32x4_t S[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      S[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk)
        S[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kf[mt][kk]), qf[kk], S[mt], 0, 0, 0);
    }
    float s[2][4];
    float mx = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int slot = blk + 16 * mt + 4 * g + v;
        s[mt][v] = slot < n_eff ? S[mt][v] * a.scale_log2 : -INFINITY;
        mx = fmaxf(mx, s[mt][v]);
      }
    }
    if (c < G) {
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
        *(float4*)(stash_row + blk + 16 * mt + 4 * g) = make_float4(s[mt][0], s[mt][1], s[mt][2], s[mt][3]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = exp2f(m_run - m_new);
    float p[2][4];
    float psum = 0.f, ssum = 0.f;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        p[mt][v] = exp2f(s[mt][v] - m_new);
        psum += p[mt][v];
        ssum += (pv[mt][v] > thr && blk + 16 * mt + 4 * g + v < n_eff) ? p[mt][v] : 0.f;
      }
    }
    l_run = l_run * alpha + psum;
    s_run = s_run * alpha + ssum;
    m_run = m_new;
    // Rescale the output rows (heads 4g + v) by their heads' alpha.
    float al[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) al[v] = __shfl(alpha, 4 * g + v, 64);
#pragma unroll
    for (int r = 0; r < VE; ++r) {
#pragma unroll
      for (int v = 0; v < 4; ++v) O[r][v] *= al[v];
    }
    // alpha.V on the matrix cores: k index = row group g of (mt, v); column j = dims VE*j + r.
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
#pragma unroll
        for (int r = 0; r < VE; ++r)
          O[r] = __builtin_amdgcn_mfma_f32_16x16x4f32(p[mt][v], vrow_elem(vf[mt][v], r), O[r], 0, 0, 0);
      }
    }
  }

  // Merge the waves of the workgroup into one partial for this split.
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  s_run += __shfl_xor(s_run, 16, 64);
  s_run += __shfl_xor(s_run, 32, 64);
  __shared__ float sm_m[NW][16], sm_l[NW][16], sm_s[NW][16];
  __shared__ float sm_o[NW][16][D];
  if (g == 0) {
    sm_m[wave][c] = m_run;
    sm_l[wave][c] = l_run;
    sm_s[wave][c] = s_run;
  }
#pragma unroll
  for (int r = 0; r < VE; ++r) {
#pragma unroll
    for (int v = 0; v < 4; ++v) sm_o[wave][4 * g + v][VE * c + r] = O[r][v];
  }
  __syncthreads();
  const size_t pbase = (bk * a.ns_max + split) * G;
  for (int i = threadIdx.x; i < G * D; i += 64 * NW) {
    const int h = i / D, d = i % D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, sm_m[w][h]);
    float o = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w)
      if (sm_m[w][h] != -INFINITY) o += exp2f(sm_m[w][h] - M) * sm_o[w][h][d];
    a.part_o[(pbase + h) * D + d] = o;
  }
  if (threadIdx.x < G) {
    const int h = threadIdx.x;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, sm_m[w][h]);
    float lsum = 0.f, ssum = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      if (sm_m[w][h] != -INFINITY) {
        const float f = exp2f(sm_m[w][h] - M);
        lsum += f * sm_l[w][h];
        ssum += f * sm_s[w][h];
      }
    }
    a.part_ml[pbase + h] = make_float2(M, lsum);
    a.part_s[pbase + h] = ssum;
  }
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
// Host-side launchers.
// -------------------------------------------------------------------------------------------
constexpr int kMfmaWaves = 4;
constexpr int kMfmaBlocksPerWave = 2;
constexpr int kMfmaSplit = kMfmaWaves * kMfmaBlocksPerWave * 32;
static_assert(kMfmaSplit % kSplitQuantum == 0, "split must be a multiple of the quantum");

template <typename T, int D>
static hipError_t launch_valu(AttendArgs a, hipStream_t st) {
  a.split = kSplitQuantum;
  dim3 grid((a.cap + a.split - 1) / a.split, a.Hkv, a.B);
  hipLaunchKernelGGL((attend_valu<T, D>), grid, dim3(64), 0, st, a);
  hipLaunchKernelGGL((attend_combine<T, D>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_mfma(AttendArgs a, hipStream_t st) {
  a.split = kMfmaSplit;
  dim3 grid((a.cap + a.split - 1) / a.split, a.Hkv, a.B);
  hipLaunchKernelGGL((attend_mfma<D, kMfmaWaves, kMfmaBlocksPerWave>), grid, dim3(64 * kMfmaWaves), 0, st, a);
  hipLaunchKernelGGL((attend_combine<uint16_t, D>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_attend(AttendArgs a, lg_dtype dt, int D, int variant, hipStream_t st) {
  if (variant == 2) return D == 128 ? launch_mfma<128>(a, st) : launch_mfma<64>(a, st);
  if (dt == LG_BF16)
    return D == 128 ? launch_valu<uint16_t, 128>(a, st) : launch_valu<uint16_t, 64>(a, st);
  return D == 128 ? launch_valu<float, 128>(a, st) : launch_valu<float, 64>(a, st);
}

}  // namespace lg

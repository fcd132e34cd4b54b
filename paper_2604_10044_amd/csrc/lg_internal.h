// lg_internal.h -- definitions shared by the HIP translation units of liblg (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lg.h"

namespace lg {

// Slots per split of the attention sweep. Every attention kernel uses splits whose length is a
// multiple of kSplitQuantum; the workspace is sized for the smallest split, kSplitQuantum.
constexpr int kSplitQuantum = 64;
constexpr int kMaxGroup = 16;  // query heads per KV head (MFMA M dimension)

// Detector limits (static LDS sizing).
constexpr int kMaxWindow = 512;
constexpr int kMaxHorizon = 2048;
constexpr int kMaxPeriod = 512;
constexpr int kMaxNgram = 16;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Workspace layout of lg_decode_attend (sizes from lg_attend_layout()).
struct AttendLayout {
  int ns_max;        // splits per (sequence, kv head) at the smallest split length
  int cap_s;         // stash row length (cap rounded up to 256 slots)
  size_t off_ml;     // float2 [B][Hkv][ns_max][G]: split max (log2 domain) and sum
  size_t off_s;      // float  [B][Hkv][ns_max][G]: split suffix mass
  size_t off_o;      // float  [B][Hkv][ns_max][G][D]: split output numerators
  size_t off_stash;  // float  [B][Hkv][G][cap_s]: logits (log2 domain) for the H2O update
  int nsq;           // splits per row of the one-launch form at most (its splits are >= 128 slots)
  size_t off_tag;    // u64    [B][Hkv][nsq][G][D] then [B][Hkv][nsq][G][3] per row: the one-launch
                     //        form's tagged partials (numerators, then max / sum / suffix sum)
  size_t off_sync;   // u32    [B][Hkv][16]: word 1 = generation of the row's partials
  size_t bytes;
};

inline AttendLayout attend_layout(int B, int Hq, int Hkv, int D, int cap) {
  AttendLayout L;
  const int G = Hq / Hkv;
  L.ns_max = (cap + kSplitQuantum - 1) / kSplitQuantum;
  L.cap_s = (int)align_up((size_t)cap, 256);
  size_t bh = (size_t)B * Hkv;
  size_t o = 0;
  L.off_ml = o; o = align_up(o + bh * L.ns_max * G * sizeof(float) * 2, 256);
  L.off_s = o;  o = align_up(o + bh * L.ns_max * G * sizeof(float), 256);
  L.off_o = o;  o = align_up(o + bh * L.ns_max * G * (size_t)D * sizeof(float), 256);
  L.off_stash = o; o = align_up(o + bh * G * (size_t)L.cap_s * sizeof(float), 256);
  L.nsq = (cap + 127) / 128 < 32 ? (cap + 127) / 128 : 32;
  L.off_tag = o; o = align_up(o + bh * L.nsq * G * (size_t)(D + 3) * sizeof(uint64_t), 256);
  L.off_sync = o; o = align_up(o + bh * 16 * sizeof(uint32_t), 256);
  L.bytes = o;
  return L;
}

// Arguments of one attention launch (passed by value to every attention kernel).
struct AttendArgs {
  const void* k;       // [B][Hkv][cap][D]
  const void* v;
  void* k_w;           // same buffers, written by the append
  void* v_w;
  float* acc;          // [B][Hkv][cap]
  const void* q;       // [B][Hq][D]
  const void* k_new;   // [B][Hkv][D] or null
  const void* v_new;
  void* out;           // [B][Hq][D]
  const int32_t* pos;  // [B][cap]
  const int32_t* len;  // [B]
  const int32_t* t;    // [B]
  const int32_t* suffix_w;
  float* lse;          // [B][Hq]
  float* suffix_mass;  // [B][Hq]
  float* conf;         // [B] or null
  float2* part_ml;
  float* part_s;
  float* part_o;
  float* stash;
  unsigned long long* tagged;  // one-launch form: per row [nsq][G*D] numerators, [nsq][G][3] statistics
  unsigned* sync;      // [B][Hkv][16], word 1: generation of the row's tagged partials
  int B, Hq, Hkv, G, cap, cap_s, ns_max, nsq;
  int split;           // slots per split used by this launch
  float scale_log2;    // log2(e) / sqrt(D)
};

// bfloat16 <-> float32 (round to nearest even; NaN stays NaN).
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// a - b saturated to the int32 range: thresholds on positions stay defined for any device-side
// position and width a caller passes.
__device__ __forceinline__ int sat_sub(int a, int b) {
  const long long d = (long long)a - (long long)b;
  return d < -2147483647LL - 1 ? (-2147483647 - 1) : (d > 2147483647LL ? 2147483647 : (int)d);
}

// Sequence length with the step's appended row, clamped into the cache.
__device__ __forceinline__ int live_slots(const AttendArgs& a, int b, int* L_out, int* app_out) {
  int L = a.len[b];
  L = L < 0 ? 0 : (L > a.cap ? a.cap : L);
  int app = (a.k_new != nullptr && L < a.cap) ? 1 : 0;
  *L_out = L;
  *app_out = app;
  return L + app;
}

}  // namespace lg

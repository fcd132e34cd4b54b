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

// ------------------------------------------------------------------------------------------
// Attention launch plan and workspace layout (host and device).
// ------------------------------------------------------------------------------------------
// Kernel forms of lg_decode_attend. The automatic choice for bfloat16 caches whose cap is a
// multiple of 32 (<= 32768): kFormOneLaunch when every row is a single split (no exchange; see
// attend_plan), kFormMerge otherwise (the sweep and a merging launch: at 1 to 64 rows and in the
// ragged batch it measured faster than the one-launch form's exchange); kFormPortable for the
// other caches. The one-launch form with several splits per row is reachable through the test
// hook.
enum : int { kFormAuto = 0, kFormPortable = 1, kFormMerge = 2, kFormOneLaunch = 3 };
constexpr int kWaves = 4;            // waves per workgroup of the MFMA sweep
constexpr int kMaxMfmaSplits = 32;   // splits per row of the MFMA forms at most
constexpr int kMaxSplitSlots = 1024; // slots per split of the MFMA forms at most ...
constexpr int kMaxSingleSlots = 2048; // ... except a one-launch split that is its row's only one
                                      // (groups of at most 8 heads), swept by kSingleWaves waves
constexpr int kSingleWaves = 8;
// Rows from which a one-launch launch gives every row a single workgroup (when the cap allows):
// half the CUs of MI355X; the split exchange then costs more than the idle half would stream.
constexpr long kSingleSplitRows = 128;
// Workgroups one MFMA launch aims for when rows are few (one per CU of MI355X): the split length
// shrinks from its maximum until the launch has about this many, down to one block per wave.
constexpr long kTargetWorkgroups = 256;

inline bool mfma_eligible(const lg_layer_cache& c) {
  return c.dtype == LG_BF16 && c.cap % 32 == 0 && c.cap <= 32768;
}

struct AttendPlan {
  int form;     // kFormPortable, kFormMerge or kFormOneLaunch
  int split;    // slots per split
  int ns_grid;  // splits per row in the grid (ceil(cap / split))
  int dsplit;   // workgroups per single-split row, each owning part of the output dims (1 or 2)
};

// Largest split of this layer whose row needs no exchange (0 if none beyond kMaxSplitSlots).
inline int single_split_max(const lg_layer_cache& c) {
  return c.n_q_heads / c.n_kv_heads <= 8 ? kMaxSingleSlots : kMaxSplitSlots;
}

// split: 0 for the default, else that split length (a multiple of 32 in [32 * kWaves, 1024], or
// up to kMaxSingleSlots for a one-launch split that covers the whole cap). The default: one-launch
// launches of at least kSingleSplitRows rows whose cap fits one split give each row one split;
// otherwise 1024 slots, shorter when the launch has few rows. Either is raised to what keeps a row
// within kMaxMfmaSplits splits.
inline bool single_split_rows(const lg_layer_cache& c) {
  return (long)c.batch * c.n_kv_heads >= kSingleSplitRows && c.cap <= single_split_max(c);
}

inline AttendPlan attend_plan(const lg_layer_cache& c, int form, int split_req) {
  AttendPlan p;
  p.form = form != kFormAuto ? form
           : !mfma_eligible(c) ? kFormPortable
           : (split_req == 0 && single_split_rows(c)) ? kFormOneLaunch : kFormMerge;
  if (p.form == kFormPortable) {
    p.split = kSplitQuantum;
  } else {
    const int min_split = ((c.cap + kMaxMfmaSplits - 1) / kMaxMfmaSplits + 31) & ~31;
    int split = split_req > 0 ? split_req : kMaxSplitSlots;
    const long rows = (long)c.batch * c.n_kv_heads;
    if (split_req == 0 && p.form == kFormOneLaunch && single_split_rows(c)) {
      split = c.cap > 32 * kWaves ? c.cap : 32 * kWaves;
    } else if (split_req == 0) {
      long want = ((long)c.cap * rows + kTargetWorkgroups - 1) / kTargetWorkgroups;
      want = (want + 31) & ~31L;
      if (want < 32 * kWaves) want = 32 * kWaves;
      if (want < split) split = (int)want;
    }
    p.split = split > min_split ? split : min_split;
  }
  p.ns_grid = (c.cap + p.split - 1) / p.split;
  // Rows that are a single long split and too few to fill the device get two workgroups each:
  // both read the whole K row and compute the softmax, each forms half of the output dims and
  // reads half of V (head_dim 128).
  const long rows = (long)c.batch * c.n_kv_heads;
  p.dsplit = (p.form == kFormOneLaunch && p.split > kMaxSplitSlots && c.head_dim == 128 &&
              2 * rows <= kTargetWorkgroups) ? 2 : 1;
  return p;
}

// Workspace header (the first 256 bytes of every attention workspace; public as
// lg_attend_workspace_header). status is sticky: a call that finds it non-zero refuses.
constexpr uint32_t kWsMagic = 0x4c474157u;  // "LGAW"
constexpr uint32_t kWsVersion = 2;
struct WsHeader {
  uint32_t magic, version;
  int32_t batch, n_q_heads, n_kv_heads, head_dim, cap, dtype, form, split;
  uint32_t status;
  uint32_t reserved[5];
};
static_assert(sizeof(WsHeader) == 64, "header size");

// Byte offsets of one workspace. One-launch form: per row (sequence, kv head) a 64-bit arrival
// word, tagged statistics words of every split (stride kMaxMfmaSplits splits), one mode word per
// split, 32-bit numerator words of every split, and 32-bit handover words (split-relative
// probabilities) per head and slot. Merge and portable forms: split partials and the logit stash.
struct AttendLayout {
  int cap_s;           // slots per stash / handover row (cap rounded up to 256)
  size_t off_rows;     // u64 [rows]
  size_t off_stats;    // u64 [rows][kMaxMfmaSplits][G][3]
  size_t off_mode;     // u32 [rows][kMaxMfmaSplits]
  size_t off_numer;    // u32 [rows][ns_grid][G * D]
  size_t off_hand;     // u32 [rows][G][cap_s]
  size_t off_ml;       // float2 [rows][ns_grid][G]   (merge / portable)
  size_t off_s;        // float  [rows][ns_grid][G]
  size_t off_o;        // float  [rows][ns_grid][G][D]
  size_t off_stash;    // float  [rows][G][cap_s]
  size_t bytes;
};

inline AttendLayout attend_layout(const lg_layer_cache& c, const AttendPlan& p) {
  AttendLayout L = {};
  const size_t G = (size_t)(c.n_q_heads / c.n_kv_heads), D = (size_t)c.head_dim;
  const size_t rows = (size_t)c.batch * c.n_kv_heads;
  L.cap_s = (int)align_up((size_t)c.cap, 256);
  size_t o = sizeof(WsHeader) > 256 ? sizeof(WsHeader) : 256;
  if (p.form == kFormOneLaunch) {
    L.off_rows = o;  o = align_up(o + rows * 8, 256);
    L.off_stats = o; o = align_up(o + rows * kMaxMfmaSplits * G * 3 * 8, 256);
    L.off_mode = o;  o = align_up(o + rows * kMaxMfmaSplits * 4, 256);
    L.off_numer = o; o = align_up(o + rows * p.ns_grid * G * D * 4, 256);
    L.off_hand = o;  o = align_up(o + rows * G * L.cap_s * 4, 256);
  } else {
    L.off_ml = o;    o = align_up(o + rows * p.ns_grid * G * 8, 256);
    L.off_s = o;     o = align_up(o + rows * p.ns_grid * G * 4, 256);
    L.off_o = o;     o = align_up(o + rows * p.ns_grid * G * D * 4, 256);
    L.off_stash = o; o = align_up(o + rows * G * L.cap_s * 4, 256);
  }
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
  WsHeader* hdr;       // the workspace header (checked by every launch; status updated)
  // merge / portable forms
  float2* part_ml;
  float* part_s;
  float* part_o;
  float* stash;
  // one-launch form
  unsigned long long* rows;   // [B * Hkv] arrival words
  unsigned long long* stats;  // tagged statistics
  unsigned* mode;             // mode words
  unsigned* numer;            // numerator words
  unsigned* hand;             // handover words
  int B, Hq, Hkv, G, cap, cap_s, dtype, form;
  int split;           // slots per split used by this launch
  int ns_grid;         // splits per row in the grid
  int row_major;       // one-launch grid order: splits of a row adjacent (1) or split slowest (0)
  int flags;           // test flags (kFlag*)
  int dsplit;          // AttendPlan::dsplit of this launch
  int spin_limit;      // polls before a wait gives up
  float scale_log2;    // log2(e) / sqrt(D)
};

// Test flags of the one-launch form (lg_test_decode_attend).
constexpr int kFlagForceHandover = 1;  // every split that is not the row's closer hands over
constexpr int kFlagNoWait = 2;         // every wait gives up without polling
constexpr int kFlagWholeDims = 4;      // no split of the output dims (dsplit 1)
constexpr int kSpinLimit = 1 << 18;    // polls (each a memory round trip plus a short sleep)

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

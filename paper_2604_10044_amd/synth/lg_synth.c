/*
 * lg_synth.c -- seeded synthetic inputs for the guarded-decode path.
 *
 * This module only produces inputs (token streams, query/key/value rows). It holds none of the
 * method's arithmetic and is the one piece of code that both the GPU path's harness and the CPU
 * oracle's harness use, so that both sides see bit-identical inputs.
 *
 * Every value is an integer function of (seed, tag, sequence, layer, head, position, lane):
 *   - 64-bit counter -> SplitMix64 finalizer (Steele, Lea & Flood, "Fast splittable pseudorandom
 *     number generators", OOPSLA 2014) -> four 16-bit uniforms;
 *   - an approximately standard normal value is the Irwin-Hall sum of those four uniforms,
 *     centred and scaled to unit variance, evaluated in float32 with contraction off;
 *   - bfloat16 outputs are that float rounded to nearest-even.
 * Token ids are floor(u32 * vocab / 2^32) of the high hash word.
 *
 * Planted structure (the paper's loop-inducing regime, Sec. 3.3 and Sec. 4.1, imitated on
 * synthetic data):
 *   - a repetition segment [start, end) repeats a unit of unit_len tokens; the unit is the first
 *     copy, positions start .. start+unit_len-1;
 *   - keys at repeated positions are copies of the first copy's key plus Gaussian noise whose
 *     std ramps linearly from noise0 (position ramp_lo) to noise1 (position ramp_hi);
 *   - "locked" query heads (every lock_every-th head in layers >= lock_layer_min) query the key of
 *     the unit phase that comes next: q = lock_gain * k_src + lock_noise * z;
 *   - a fraction dup_rate of key rows are bit-exact copies of an earlier row (ties for eviction).
 * Build: gcc -O2 -fopenmp -ffp-contract=off -shared -fPIC.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

typedef struct {
  uint64_t seed;
  int32_t n_layers, n_q_heads, n_kv_heads, head_dim, vocab;
  int32_t dtype; /* 0 = float32 rows, 1 = bfloat16 rows */
  float lock_gain, lock_noise;
  int32_t lock_every, lock_layer_min;
  float dup_rate;
  int32_t reserved;
} synth_cfg;

typedef struct {
  int32_t start, end, unit_len, unit_off;
  float noise0, noise1;
  int32_t ramp_lo, ramp_hi;
} synth_seg;

typedef struct {
  int32_t n_seg;
  int32_t reserved;
  const synth_seg* seg;
  const int32_t* unit_tokens; /* unit tokens of all segments, indexed by seg.unit_off */
} synth_seq;

enum { TAG_TOKEN = 1, TAG_K = 2, TAG_V = 3, TAG_Q = 4, TAG_KNOISE = 5, TAG_QNOISE = 6,
       TAG_DUP = 7, TAG_DUPSRC = 8, TAG_UNIT = 9 };
enum { KIND_K = 0, KIND_V = 1, KIND_Q = 2 };

static uint64_t mix64(uint64_t z) {
  z += 0x9e3779b97f4a7c15ULL;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

/* Unique 64-bit counter per value; fields are masked to their widths. */
static uint64_t hash_at(uint64_t seed, uint64_t tag, uint64_t b, uint64_t layer, uint64_t head,
                        uint64_t pos, uint64_t lane) {
  uint64_t c = ((tag & 0xF) << 60) | ((b & 0x3FF) << 50) | ((layer & 0xFF) << 42) |
               ((head & 0xFF) << 34) | ((pos & 0xFFFFFF) << 10) | (lane & 0x3FF);
  return mix64(c ^ mix64(seed * 0x2545f4914f6cdd1dULL + 0x632be59bd9b4e019ULL));
}

static float gauss_from(uint64_t h) {
  uint32_t s = (uint32_t)(h & 0xFFFF) + (uint32_t)((h >> 16) & 0xFFFF) +
               (uint32_t)((h >> 32) & 0xFFFF) + (uint32_t)((h >> 48) & 0xFFFF);
  float centred = (float)s - 131070.0f;
  return centred * (1.7320508075688772f / 65535.0f);
}

static uint16_t bf16_rne(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  uint32_t bias = ((u >> 16) & 1u) + 0x7FFFu;
  return (uint16_t)((u + bias) >> 16);
}

static float bf16_to_f32(uint16_t h) {
  uint32_t u = ((uint32_t)h) << 16;
  float x;
  memcpy(&x, &u, 4);
  return x;
}

/* Segment containing position p, or NULL. */
static const synth_seg* seg_at(const synth_seq* s, int32_t p) {
  for (int i = 0; i < s->n_seg; ++i)
    if (p >= s->seg[i].start && p < s->seg[i].end) return &s->seg[i];
  return 0;
}

int32_t synth_token(const synth_cfg* c, const synth_seq* s, int32_t b, int32_t p) {
  const synth_seg* g = seg_at(s, p);
  if (g) return s->unit_tokens[g->unit_off + (p - g->start) % g->unit_len];
  uint64_t h = hash_at(c->seed, TAG_TOKEN, (uint64_t)b, 0, 0, (uint64_t)p, 0);
  return (int32_t)(((h >> 32) * (uint64_t)c->vocab) >> 32);
}

void synth_tokens(const synth_cfg* c, const synth_seq* s, int32_t b, int32_t n, int32_t* out) {
  for (int32_t p = 0; p < n; ++p) out[p] = synth_token(c, s, b, p);
}

/* `len` distinct token ids for unit number `idx` of sequence b. */
void synth_unit_tokens(const synth_cfg* c, int32_t b, int32_t idx, int32_t len, int32_t avoid,
                       int32_t* out) {
  for (int32_t k = 0; k < len; ++k) {
    uint64_t h = hash_at(c->seed, TAG_UNIT, (uint64_t)b, (uint64_t)idx, 0, (uint64_t)k, 0);
    int32_t tok = (int32_t)(((h >> 32) * (uint64_t)c->vocab) >> 32);
    for (;;) {
      int clash = (tok == avoid);
      for (int32_t j = 0; j < k && !clash; ++j) clash = (out[j] == tok);
      if (!clash) break;
      tok = (tok + 1) % c->vocab;
    }
    out[k] = tok;
  }
}

/* Key value before duplication: base Gaussian, or a noisy copy inside a repetition segment. */
static float key_plain(const synth_cfg* c, const synth_seq* s, int32_t b, int32_t layer,
                       int32_t head, int32_t p, int32_t lane) {
  const synth_seg* g = seg_at(s, p);
  if (g && p >= g->start + g->unit_len) {
    int32_t src = g->start + (p - g->start) % g->unit_len;
    float base = gauss_from(hash_at(c->seed, TAG_K, b, layer, head, src, lane));
    float sd;
    if (g->ramp_hi <= g->ramp_lo || p <= g->ramp_lo) sd = g->noise0;
    else if (p >= g->ramp_hi) sd = g->noise1;
    else {
      float f = (float)(p - g->ramp_lo) / (float)(g->ramp_hi - g->ramp_lo);
      sd = g->noise0 + (g->noise1 - g->noise0) * f;
    }
    float z = gauss_from(hash_at(c->seed, TAG_KNOISE, b, layer, head, p, lane));
    return base + sd * z;
  }
  return gauss_from(hash_at(c->seed, TAG_K, b, layer, head, p, lane));
}

static int32_t key_source(const synth_cfg* c, int32_t b, int32_t layer, int32_t head, int32_t p) {
  if (c->dup_rate <= 0.0f || p == 0) return p;
  uint64_t h = hash_at(c->seed, TAG_DUP, b, layer, head, p, 0);
  double u = (double)(h >> 11) * (1.0 / 9007199254740992.0);
  if (u >= (double)c->dup_rate) return p;
  uint64_t h2 = hash_at(c->seed, TAG_DUPSRC, b, layer, head, p, 0);
  return (int32_t)((h2 >> 33) % (uint64_t)p);
}

static float row_value(const synth_cfg* c, const synth_seq* s, int kind, int32_t b, int32_t layer,
                       int32_t head, int32_t p, int32_t lane) {
  if (kind == KIND_V) return gauss_from(hash_at(c->seed, TAG_V, b, layer, head, p, lane));
  if (kind == KIND_K) return key_plain(c, s, b, layer, head, key_source(c, b, layer, head, p), lane);
  /* queries */
  int32_t G = c->n_q_heads / c->n_kv_heads;
  const synth_seg* g = seg_at(s, p);
  int locked = c->lock_every > 0 && (head % c->lock_every) == 0 && layer >= c->lock_layer_min &&
               g != 0 && p + 1 < g->end && p + 1 >= g->start + g->unit_len;
  if (locked) {
    int32_t src = g->start + (p + 1 - g->start) % g->unit_len;
    float ks = gauss_from(hash_at(c->seed, TAG_K, b, layer, head / G, src, lane));
    float z = gauss_from(hash_at(c->seed, TAG_QNOISE, b, layer, head, p, lane));
    return c->lock_gain * ks + c->lock_noise * z;
  }
  return gauss_from(hash_at(c->seed, TAG_Q, b, layer, head, p, lane));
}

/*
 * Fill rows for a batch: out[l][i][h][j][:] for l in [layer_lo, layer_hi), i < nb (sequence
 * b_index[i], described by seqs[i]), h < n_heads, j < cnt[i] at position pos[i*P + j].
 * Rows j >= cnt[i] are zero. Element type per cfg.dtype.
 */
void synth_fill(const synth_cfg* c, const synth_seq* seqs, const int32_t* b_index, int32_t nb,
                int kind, int32_t layer_lo, int32_t layer_hi, int32_t n_heads, int32_t P,
                const int32_t* pos, const int32_t* cnt, void* out) {
  const int32_t d = c->head_dim;
  const int64_t nl = layer_hi - layer_lo;
  const int64_t total = nl * nb * n_heads;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t w = 0; w < total; ++w) {
    int32_t h = (int32_t)(w % n_heads);
    int32_t i = (int32_t)((w / n_heads) % nb);
    int32_t layer = layer_lo + (int32_t)(w / ((int64_t)n_heads * nb));
    int32_t b = b_index[i];
    for (int32_t j = 0; j < P; ++j) {
      int64_t row = (w * P + j) * d;
      for (int32_t e = 0; e < d; ++e) {
        float x = 0.0f;
        if (j < cnt[i]) x = row_value(c, &seqs[i], kind, b, layer, h, pos[(int64_t)i * P + j], e);
        if (c->dtype == 1) ((uint16_t*)out)[row + e] = bf16_rne(x);
        else ((float*)out)[row + e] = x;
      }
    }
  }
}

/* Exact widening of bfloat16 bits (helper for harnesses that feed float32 consumers). */
void synth_bf16_to_f32(const uint16_t* in, float* out, int64_t n) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = bf16_to_f32(in[i]);
}

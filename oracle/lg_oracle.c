/*
 * lg_oracle.c -- CPU oracle of the LoopGuard guarded-decode step.
 *
 * TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the benchmark's CPU-baseline leg
 * may load this file's library. It shares no code, header or table with the GPU path; it is
 * deliberately plain and slow: double precision, straight loops, no blocking or fusion, each
 * function written from the paper passage it cites so a reader can check it by eye.
 *
 * Paper: "LoopGuard: Breaking Self-Reinforcing Attention Loops via Dynamic KV Cache
 * Intervention" (arXiv 2604.10044).
 *
 * Readings of what the paper leaves open (each is listed, with its reason, in the design notes):
 *   - H2O accumulation: sum over the query heads of a KV group, new slots start at 0, no decay.
 *   - Confidence: the caller supplies conf (the GPU harness passes the largest suffix mass).
 *   - Compression: greedy token-level LZ77 parse of the window (match >= 3 tokens costs 2, a
 *     literal costs 1, sources start inside the window, overlap allowed).      -- parity unpinned
 *     against the paper's unnamed byte-level compressor (only its form is pinned).
 *   - Novelty: share of first-occurrence 4-grams among the last 64 positions.   -- parity unpinned
 *     against the paper's undefined novelty score (only its form is pinned).
 *   - Suffix self-alignment: trailing run L_P of y[i] == y[i-P] for P <= 256, span capped at the
 *     horizon H; qualifies with >= 3 copies and >= 32 tokens; P* maximises the span, ties to the
 *     smallest P; debounced over 4 steps.
 *   - Keep set: R = B/4, S = B/2 - 32, recent budget R >> l, l capped at 3, evenly spaced ranks.
 *   - Baseline keep policies (Sec. 6.1 names H2O and StreamingLLM without parameters): both act
 *     only when the cache reaches its budget and keep as many slots as the LoopGuard set,
 *     K = B/2 + B/4. H2O keeps the last R = B/4 slots and the K - R highest-scoring older slots
 *     (score = acc summed over layers and KV heads; equal scores evict the lower position first);
 *     StreamingLLM keeps the anchor positions (attention sinks) and the last K - A slots.
 * Build: gcc -O2 -shared -fPIC -ffp-contract=off lg_oracle.c -lm
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Hyperparameters; field meanings as in Sec. 5.2, Sec. 5.3, Sec. 6.1 and App. B.2. */
typedef struct {
  int32_t W, K, n_anchor, t_min, cooldown, streak_min, stall_min, cr_interval, nov_ngram,
      nov_span, rep_pmax, rep_horizon, rep_min_copies, rep_min_len, rep_debounce, level_max,
      retrigger_window, recent_div, sparse_div, ttr_num, ttr_den, cr_num, cr_den, nov_num,
      nov_den;
  float conf_threshold;
  int32_t mode;   /* 0 full rule, 1 always-on pruning, 2 confidence streak only (Table 3) */
  int32_t policy; /* keep policy: 0 LoopGuard (Eq. (10)/(11)), 1 H2O, 2 StreamingLLM (Sec. 6.1) */
} or_params;

typedef struct {
  int32_t streak, stall, rep, n_int, n_last, level, cr_valid, cr_cost, cr_m;
} or_state;

typedef struct {
  int32_t trigger, warn, votes, stall_gate, tailrep_gate, n, distinct, lz_cost, novel, nov_r,
      period, span_lo, level, n_int;
} or_decision;

/* ------------------------------------------------------------------------------------------ */
/* Eq. (1), Sec. 3.1: attention of the G query heads of one KV head over the accessible slots.  */
/* ------------------------------------------------------------------------------------------ */
/*
 * q [G][d]; K, V [n][d]; pos [n] positions of the slots (the query's own row included).
 * Outputs per query head h: o[h][:] = sum_j alpha_j v_j, lse[h] = log sum_j exp(s_j),
 * sigma[h] = sum of alpha_j over slots with pos_j > t - w_s (mass on the recent suffix that a
 * locked head concentrates on, Sec. 1 and App. E), and alpha_sum[j] = sum_h alpha_j^{(h)}
 * (the per-step increment of the H2O accumulated importance of slot j).
 */
void or_attend_group(int32_t n, int32_t G, int32_t d, const float* q, const float* K,
                     const float* V, const int32_t* pos, int32_t t, int32_t w_s, double* o,
                     double* lse, double* sigma, double* alpha_sum) {
  double* s = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
  const double tau = 1.0 / sqrt((double)d);
  for (int32_t j = 0; j < n; ++j) alpha_sum[j] = 0.0;
  for (int32_t h = 0; h < G; ++h) {
    for (int32_t e = 0; e < d; ++e) o[h * d + e] = 0.0;
    sigma[h] = 0.0;
    if (n == 0) {
      lse[h] = -INFINITY;
      continue;
    }
    double M = -INFINITY;
    for (int32_t j = 0; j < n; ++j) {
      double acc = 0.0;
      for (int32_t e = 0; e < d; ++e) acc += (double)q[h * d + e] * (double)K[(size_t)j * d + e];
      s[j] = tau * acc;
      if (s[j] > M) M = s[j];
    }
    double Z = 0.0;
    for (int32_t j = 0; j < n; ++j) Z += exp(s[j] - M);
    lse[h] = M + log(Z);
    for (int32_t j = 0; j < n; ++j) {
      double a = exp(s[j] - M) / Z;
      for (int32_t e = 0; e < d; ++e) o[h * d + e] += a * (double)V[(size_t)j * d + e];
      if ((int64_t)pos[j] > (int64_t)t - (int64_t)w_s) sigma[h] += a;  /* over the integers */
      alpha_sum[j] += a;
    }
  }
  free(s);
}

/* ------------------------------------------------------------------------------------------ */
/* Windowed indicators of Sec. 5.2 (Eq. (5) TTR, Eq. (6) CR) and the persistence gates (App. B.2) */
/* ------------------------------------------------------------------------------------------ */

/* |uniq(y[lo..hi))|, the numerator of the type-token ratio, Eq. (5). */
int32_t or_distinct(const int32_t* y, int32_t lo, int32_t hi) {
  int32_t u = 0;
  for (int32_t i = lo; i < hi; ++i) {
    int first = 1;
    for (int32_t j = lo; j < i; ++j)
      if (y[j] == y[i]) { first = 0; break; }
    u += first;
  }
  return u;
}

/* Longest common extension of y[p..] and y[i..] that stays inside y[..hi). */
static int32_t lce(const int32_t* y, int32_t p, int32_t i, int32_t hi) {
  int32_t k = 0;
  while (i + k < hi && y[p + k] == y[i + k]) ++k;
  return k;
}

/*
 * Compressed size of y[lo..hi) under a greedy token-level LZ77 parse (the reading of the
 * "standard lossless compressor" of Eq. (6)): at position i the longest earlier match inside the
 * window, max over lo <= p < i of LCE(p, i) (overlap allowed), is taken when it has at least
 * `min_match` tokens and costs 2 units (offset, length); otherwise a literal costs 1 unit.
 */
int32_t or_lz_cost(const int32_t* y, int32_t lo, int32_t hi, int32_t min_match) {
  int32_t cost = 0, i = lo;
  while (i < hi) {
    int32_t best = 0;
    for (int32_t p = lo; p < i; ++p) {
      int32_t k = lce(y, p, i, hi);
      if (k > best) best = k;
    }
    if (best >= min_match) { cost += 2; i += best; }
    else { cost += 1; i += 1; }
  }
  return cost;
}

/*
 * Novelty over the window [w0, n): among the positions i in [max(w0+g-1, n-span), n), count
 * those whose g-gram y[i-g+1..i] has no earlier occurrence ending at p in [w0+g-1, i).
 * *r receives the number of positions examined.
 */
int32_t or_novelty(const int32_t* y, int32_t w0, int32_t n, int32_t g, int32_t span, int32_t* r) {
  int32_t lo = w0 + g - 1;
  if (n - span > lo) lo = n - span;
  int32_t novel = 0, cnt = 0;
  for (int32_t i = lo; i < n; ++i) {
    ++cnt;
    int seen = 0;
    for (int32_t p = w0 + g - 1; p < i && !seen; ++p) {
      int same = 1;
      for (int32_t k = 0; k < g; ++k)
        if (y[p - k] != y[i - k]) { same = 0; break; }
      seen = same;
    }
    novel += !seen;
  }
  *r = cnt;
  return novel;
}

/*
 * Trailing self-alignment of the stream y[t0..n): for each period P in 1..pmax, L[P] is the
 * largest k <= H - P with y[n-1-r] == y[n-1-r-P] for every r < k and n-1-r-P >= t0, so the
 * periodic tail has T_P = L[P] + P <= H tokens. L[0] is unused.
 */
void or_tail_align(const int32_t* y, int32_t t0, int32_t n, int32_t pmax, int32_t H, int32_t* L) {
  L[0] = 0;
  for (int32_t P = 1; P <= pmax; ++P) {
    int32_t k = 0;
    while (k < H - P && n - 1 - k - P >= t0 && y[n - 1 - k] == y[n - 1 - k - P]) ++k;
    L[P] = k;
  }
}

/*
 * Debounced suffix self-alignment test (App. B.2), one step. A period qualifies with at least
 * `copies` copies (L_P >= (copies-1) P) and a periodic tail of at least `min_len` tokens. P* is
 * the qualifying period with the longest tail T_P, ties to the smallest P. Returns P* (0 if no
 * period qualifies) and writes the tail length T_{P*} to *T.
 */
int32_t or_tail_best(const int32_t* y, int32_t t0, int32_t n, int32_t pmax, int32_t H,
                     int32_t copies, int32_t min_len, int32_t* T) {
  int32_t* L = (int32_t*)malloc(sizeof(int32_t) * (size_t)(pmax + 1));
  or_tail_align(y, t0, n, pmax, H, L);
  int32_t best = 0, bestT = 0;
  for (int32_t P = 1; P <= pmax; ++P) {
    int32_t TP = L[P] + P;
    int ok = (L[P] >= (copies - 1) * P) && (TP >= min_len);
    if (ok && TP > bestT) { best = P; bestT = TP; }
  }
  free(L);
  *T = bestT;
  return best;
}

/*
 * One monitor step for one sequence: Eq. (8) Warn, the persistence gates, Eq. (9) Trigger, the
 * cooldown and the aggressiveness level of Sec. 5.3. y is indexable at absolute stream positions
 * [t0, n); conf stands for p_max(t).
 */
void or_detect_step(const or_params* p, const int32_t* y, int32_t t0, int32_t n, double conf,
                    or_state* st, or_decision* dec) {
  memset(dec, 0, sizeof(*dec));
  dec->n = n;
  int32_t w0 = n - p->W;
  if (w0 < t0) w0 = t0;
  int32_t m = n - w0;

  /* Eq. (5) windowed: vote when distinct/m < theta_ttr. */
  int32_t u = or_distinct(y, w0, n);
  int vote_ttr = (int64_t)p->ttr_den * u < (int64_t)p->ttr_num * m;

  /* Eq. (6) windowed, recomputed every cr_interval steps and held in between. */
  if (!st->cr_valid || p->cr_interval <= 1 || n % p->cr_interval == 0) {
    st->cr_cost = or_lz_cost(y, w0, n, 3);
    st->cr_m = m;
    st->cr_valid = 1;
  }
  int vote_cr = (int64_t)p->cr_den * st->cr_cost < (int64_t)p->cr_num * st->cr_m;

  /* Confidence collapse: streak of steps with p_max > theta_conf; votes at >= theta_streak. */
  st->streak = (conf > (double)p->conf_threshold) ? st->streak + 1 : 0;
  int vote_p1 = st->streak >= p->streak_min;

  int warn = (vote_ttr + vote_cr + vote_p1) >= p->K; /* Eq. (8) */

  /* Novelty stagnation gate: low novelty on stall_min consecutive steps. */
  int32_t r = 0;
  int32_t novel = or_novelty(y, w0, n, p->nov_ngram, p->nov_span, &r);
  st->stall = ((int64_t)p->nov_den * novel < (int64_t)p->nov_num * r) ? st->stall + 1 : 0;
  int stall_gate = st->stall >= p->stall_min;

  /* Debounced suffix self-alignment. */
  int32_t T = 0;
  int32_t Pstar = or_tail_best(y, t0, n, p->rep_pmax, p->rep_horizon, p->rep_min_copies,
                               p->rep_min_len, &T);
  st->rep = Pstar > 0 ? st->rep + 1 : 0;
  int tail_gate = st->rep >= p->rep_debounce;

  /* Eq. (9): warmup, cooldown, Warn and (Stall or TailRep). */
  int warm = (n - t0) >= p->t_min;
  int cool = (st->n_int == 0) || (n - st->n_last >= p->cooldown);
  int fire;
  if (p->mode == 1) fire = warm && cool;
  else if (p->mode == 2) fire = warm && cool && vote_p1;
  else fire = warm && cool && warn && (stall_gate || tail_gate);

  if (fire) {
    /* Progressive aggressiveness: a quick re-trigger raises l (capped), otherwise l restarts. */
    if (st->n_int > 0 && n - st->n_last <= p->retrigger_window)
      st->level = st->level + 1 < p->level_max ? st->level + 1 : p->level_max;
    else
      st->level = 0;
    st->n_last = n;
    st->n_int += 1;
  }

  dec->trigger = fire;
  dec->warn = warn;
  dec->votes = vote_ttr | (vote_cr << 1) | (vote_p1 << 2);
  dec->stall_gate = stall_gate;
  dec->tailrep_gate = tail_gate;
  dec->distinct = u;
  dec->lz_cost = st->cr_cost;
  dec->novel = novel;
  dec->nov_r = r;
  dec->period = Pstar;
  dec->span_lo = Pstar > 0 ? n - T : -1;
  dec->level = st->level;
  dec->n_int = st->n_int;
}

/* ------------------------------------------------------------------------------------------ */
/* Eq. (10), Eq. (11), Sec. 5.3: the retained index set.                                       */
/* ------------------------------------------------------------------------------------------ */
/*
 * pos [len] strictly increasing positions of the live slots; t = pos[len-1] is the newest.
 * span_lo: first position of the detected repetitive tail (I_bad is that tail inside the recent
 * window), or < 0 for none. level: aggressiveness l. Writes the kept slot indices in ascending
 * order to keep[] and returns |I_keep|.
 */
int32_t or_keep_set(const or_params* p, const int32_t* pos, int32_t len, int32_t budget,
                    int32_t span_lo, int32_t level, int32_t* keep) {
  if (len <= 0) return 0;
  const int32_t t = pos[len - 1];
  const int32_t R = budget / p->recent_div;

  /* Membership of each slot in the sets of Sec. 5.3. */
  char* in_anchor = (char*)calloc((size_t)len, 1);
  char* in_recent_window = (char*)calloc((size_t)len, 1);
  char* in_bad = (char*)calloc((size_t)len, 1);
  char* in_keep = (char*)calloc((size_t)len, 1);
  int32_t* mid = (int32_t*)malloc(sizeof(int32_t) * (size_t)len);
  int32_t* cand = (int32_t*)malloc(sizeof(int32_t) * (size_t)len);

  for (int32_t j = 0; j < len; ++j) {
    in_anchor[j] = pos[j] < p->n_anchor;                                /* I_anchor */
    in_recent_window[j] = !in_anchor[j] && pos[j] >= t - R + 1;         /* W^recent_t */
    in_bad[j] = in_recent_window[j] && span_lo >= 0 && pos[j] >= span_lo; /* I_bad(t) */
  }

  /* Sizes. The kept set leaves room for the next append: at most budget - 1 slots, claimed by the
   * anchors first, then the recent window, then the sparse history (with the paper's constants
   * n_anchor + S + R <= budget - 1 and nothing is cut). */
  const int32_t cap_k = budget - 1 > 0 ? budget - 1 : 0;
  int32_t n_anchor_slots = 0;
  for (int32_t j = 0; j < len; ++j) n_anchor_slots += in_anchor[j];
  const int32_t A_keep = n_anchor_slots < cap_k ? n_anchor_slots : cap_k;
  int32_t B_recent = R >> level;
  if (B_recent > cap_k - A_keep) B_recent = cap_k - A_keep;
  int32_t S = budget / p->sparse_div - p->n_anchor;
  if (S > cap_k - A_keep - B_recent) S = cap_k - A_keep - B_recent;
  if (S < 0) S = 0;

  /* C_recent = W^recent \ I_bad (Eq. (11)); I_recent = its most recent min(B_recent, |C|). */
  int32_t nc = 0;
  for (int32_t j = 0; j < len; ++j)
    if (in_recent_window[j] && !in_bad[j]) cand[nc++] = j;
  int32_t take = nc < B_recent ? nc : B_recent;
  for (int32_t k = nc - take; k < nc; ++k) in_keep[cand[k]] = 1;

  /* I_sparse: uniform subsample of the history outside the anchors and the recent window. */
  int32_t M = 0;
  for (int32_t j = 0; j < len; ++j)
    if (!in_anchor[j] && !in_recent_window[j]) mid[M++] = j;
  if (M <= S) {
    for (int32_t k = 0; k < M; ++k) in_keep[mid[k]] = 1;
  } else {
    for (int32_t k = 0; k < S; ++k) in_keep[mid[(int64_t)k * M / S]] = 1;
  }

  /* I_anchor: the first A_keep anchor slots (all of them unless the cap binds). */
  for (int32_t j = 0, a = 0; j < len; ++j)
    if (in_anchor[j] && a < A_keep) {
      in_keep[j] = 1;
      ++a;
    }

  int32_t cnt = 0;
  for (int32_t j = 0; j < len; ++j)
    if (in_keep[j]) keep[cnt++] = j;

  free(in_anchor); free(in_recent_window); free(in_bad); free(in_keep); free(mid); free(cand);
  return cnt;
}

/* ------------------------------------------------------------------------------------------ */
/* Baseline keep policies of Sec. 6.1 (H2O heavy hitters, StreamingLLM sinks + window).         */
/* ------------------------------------------------------------------------------------------ */
/*
 * H2O importance of each live slot of one sequence: the accumulated attention of the slot summed
 * over every layer and KV head, in float32, layer by layer and head by head in ascending order.
 * acc is [L][H][cap] (one sequence); score[j] for j < len.
 */
void or_h2o_score(int32_t L, int32_t H, int32_t cap, int32_t len, const float* acc, float* score) {
  for (int32_t j = 0; j < len; ++j) {
    float s = 0.0f;
    for (int32_t l = 0; l < L; ++l)
      for (int32_t h = 0; h < H; ++h) s = s + acc[((size_t)l * H + h) * cap + j];
    score[j] = s;
  }
}

/* Order of scores: as float values, with -0 below +0 (the float's bits made monotone). */
static uint32_t score_order(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

/*
 * Kept slots (ascending) of a sequence whose cache has reached its budget, under the baseline
 * policy p->policy (1 H2O, 2 StreamingLLM). K = budget/sparse_div + budget/recent_div slots are
 * kept (all of them when len <= K).
 *   H2O: the last R = budget/recent_div slots, and among the older slots the K - R with the
 *        highest score; of two equal scores the slot with the higher position is kept.
 *   StreamingLLM: the A slots with position < n_anchor, and the last K - A other slots.
 */
int32_t or_keep_set_baseline(const or_params* p, const int32_t* pos, int32_t len, int32_t budget,
                             const float* score, int32_t* keep) {
  if (len <= 0) return 0;
  /* Keep size B/sparse_div + B/recent_div, capped at budget - 1 (room for the next append). */
  int32_t K = budget / p->sparse_div + budget / p->recent_div;
  if (K > budget - 1) K = budget - 1 > 0 ? budget - 1 : 0;
  char* in_keep = (char*)calloc((size_t)len, 1);
  if (p->policy == 1) {
    int32_t R = budget / p->recent_div < len ? budget / p->recent_div : len;
    if (R > K) R = K;
    const int32_t older = len - R;
    const int32_t heavy = K - R;
    for (int32_t j = older; j < len; ++j) in_keep[j] = 1;
    for (int32_t j = 0; j < older; ++j) {
      /* rank of slot j among the older slots: how many come before it in the keep order */
      int32_t ahead = 0;
      for (int32_t i = 0; i < older; ++i) {
        const uint32_t si = score_order(score[i]), sj = score_order(score[j]);
        if (si > sj || (si == sj && i > j)) ++ahead;
      }
      if (ahead < heavy) in_keep[j] = 1;
    }
  } else {
    int32_t A = 0;
    for (int32_t j = 0; j < len; ++j)
      if (pos[j] < p->n_anchor && A < K) {
        in_keep[j] = 1;
        ++A;
      }
    int32_t window = K - A;
    for (int32_t j = len - 1; j >= 0 && window > 0; --j)
      if (!in_keep[j]) {
        in_keep[j] = 1;
        --window;
      }
  }
  int32_t cnt = 0;
  for (int32_t j = 0; j < len; ++j)
    if (in_keep[j]) keep[cnt++] = j;
  free(in_keep);
  return cnt;
}

/* Test driver for the host sanitizer build of the oracle (tests/test_sanitize.py): calls every
 * oracle entry point on seeded random and planted inputs, at the edges of its arguments (empty
 * windows, n < W, full caches, every level and policy), so AddressSanitizer and
 * UndefinedBehaviorSanitizer see each code path. It checks nothing numerically (the oracle's pins
 * do that); it exits 0 when no sanitizer reports. */
#include "../oracle/lg_oracle.c"

#include <stdio.h>

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) {
  rng ^= rng << 13;
  rng ^= rng >> 7;
  rng ^= rng << 17;
  return (uint32_t)(rng >> 11);
}
static float next_f(void) { return (float)((int32_t)(next_u32() % 2001) - 1000) / 400.0f; }

static or_params defaults(void) {
  or_params p;
  memset(&p, 0, sizeof p);
  p.W = 256; p.K = 2; p.n_anchor = 32; p.t_min = 64; p.cooldown = 32; p.streak_min = 6;
  p.stall_min = 4; p.cr_interval = 1; p.nov_ngram = 4; p.nov_span = 64; p.rep_pmax = 256;
  p.rep_horizon = 1024; p.rep_min_copies = 3; p.rep_min_len = 32; p.rep_debounce = 4;
  p.level_max = 3; p.retrigger_window = 64; p.recent_div = 4; p.sparse_div = 2;
  p.ttr_num = 1; p.ttr_den = 5; p.cr_num = 3; p.cr_den = 25; p.nov_num = 1; p.nov_den = 50;
  p.conf_threshold = 0.9f; p.mode = 0; p.policy = 0;
  return p;
}

static void attend_cases(void) {
  const int32_t ns[] = {0, 1, 2, 33, 200};
  for (int c = 0; c < 5; ++c) {
    const int32_t n = ns[c], G = 4, d = 64;
    float* q = malloc(sizeof(float) * G * d);
    float* K = malloc(sizeof(float) * (size_t)(n + 1) * d);
    float* V = malloc(sizeof(float) * (size_t)(n + 1) * d);
    int32_t* pos = malloc(sizeof(int32_t) * (size_t)(n + 1));
    double* o = malloc(sizeof(double) * G * d);
    double lse[4], sigma[4];
    double* asum = malloc(sizeof(double) * (size_t)(n + 1));
    for (int i = 0; i < G * d; ++i) q[i] = next_f();
    for (int i = 0; i < n * d; ++i) { K[i] = next_f(); V[i] = next_f(); }
    for (int j = 0; j < n; ++j) pos[j] = 3 * j;
    or_attend_group(n, G, d, q, K, V, pos, 3 * n, n / 3, o, lse, sigma, asum);
    free(q); free(K); free(V); free(pos); free(o); free(asum);
  }
}

static void detect_cases(void) {
  const int32_t N = 1400;
  int32_t* y = malloc(sizeof(int32_t) * N);
  for (int32_t i = 0; i < N; ++i) y[i] = (int32_t)(next_u32() % 50000);
  for (int32_t i = 500; i < 900; ++i) y[i] = y[500 + (i - 500) % 7];      /* period 7 */
  for (int32_t i = 1000; i < N; ++i) y[i] = y[1000 + (i - 1000) % 113];   /* period 113 */
  for (int mode = 0; mode < 3; ++mode) {
    or_params p = defaults();
    p.mode = mode;
    or_state st;
    memset(&st, 0, sizeof st);
    or_decision dec;
    for (int32_t n = 1; n <= N; ++n)
      or_detect_step(&p, y, 0, n, (n % 11) ? 0.95 : 0.2, &st, &dec);
  }
  { /* small window, CR held between recomputations, monitored stream starting later */
    or_params p = defaults();
    p.W = 16; p.cr_interval = 5; p.rep_pmax = 8; p.rep_horizon = 32;
    or_state st;
    memset(&st, 0, sizeof st);
    or_decision dec;
    for (int32_t n = 1; n <= 300; ++n) or_detect_step(&p, y + 400, 37, n, 0.99, &st, &dec);
  }
  int32_t L[257], T;
  or_tail_align(y, 0, N, 256, 1024, L);
  or_tail_best(y, 0, N, 256, 1024, 3, 32, &T);
  or_tail_best(y, 0, 1, 256, 1024, 3, 32, &T);
  int32_t r;
  or_novelty(y, 0, 0, 4, 64, &r);
  or_novelty(y, N - 256, N, 4, 64, &r);
  or_distinct(y, 0, 0);
  or_distinct(y, 100, 356);
  or_lz_cost(y, 0, 0, 3);
  or_lz_cost(y, 450, 706, 3);
  free(y);
}

static void keep_cases(void) {
  const int32_t budgets[] = {64, 256, 2048};
  for (int bi = 0; bi < 3; ++bi) {
    const int32_t B = budgets[bi];
    int32_t* pos = malloc(sizeof(int32_t) * (size_t)B);
    int32_t* keep = malloc(sizeof(int32_t) * (size_t)B);
    float* score = malloc(sizeof(float) * (size_t)B);
    const int32_t lens[] = {0, 1, B / 2, B};
    for (int li = 0; li < 4; ++li) {
      const int32_t len = lens[li];
      int32_t p0 = 0;
      for (int32_t j = 0; j < len; ++j) {
        p0 += 1 + (int32_t)(next_u32() % 3);
        pos[j] = p0;
        score[j] = (float)(next_u32() % 5);
      }
      for (int level = 0; level <= 3; ++level) {
        or_params p = defaults();
        or_keep_set(&p, pos, len, B, -1, level, keep);
        if (len > 0) or_keep_set(&p, pos, len, B, pos[len / 2], level, keep);
      }
      for (int policy = 0; policy < 3; ++policy) {
        or_params p = defaults();
        p.policy = policy;
        or_keep_set_baseline(&p, pos, len, B, score, keep);
      }
    }
    free(pos); free(keep); free(score);
  }
  const int32_t Ls = 3, H = 2, cap = 40, len = 33;
  float* acc = malloc(sizeof(float) * Ls * H * cap);
  float score[40];
  for (int i = 0; i < Ls * H * cap; ++i) acc[i] = next_f();
  or_h2o_score(Ls, H, cap, len, acc, score);
  or_h2o_score(Ls, H, cap, 0, acc, score);
  free(acc);
}

int main(void) {
  attend_cases();
  detect_cases();
  keep_cases();
  printf("oracle sanitizer driver: done\n");
  return 0;
}

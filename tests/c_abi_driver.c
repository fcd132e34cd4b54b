/* C caller of the library (tests/test_c_abi.py): include/lg.h compiled as C99, liblg.so linked
 * from C, the parameter defaults and sizes read, and the host-side argument checks of each entry
 * point exercised with fake device addresses (never dereferenced: every call below is rejected
 * before anything is enqueued, so no GPU is needed). Prints "ok" and exits 0 when every status
 * matches include/lg.h. */
#include "lg.h"

#include <stdint.h>
#include <stdio.h>

static int fails = 0;
#define EXPECT(call, want)                                                            \
  do {                                                                                \
    const lg_status got_ = (call);                                                    \
    if (got_ != (want)) {                                                             \
      printf("line %d: %s returned %d (%s), expected %d\n", __LINE__, #call, (int)got_, \
             lg_status_string(got_), (int)(want));                                    \
      ++fails;                                                                        \
    }                                                                                 \
  } while (0)

#define DEV(a) ((void*)(uintptr_t)(a))

int main(void) {
  const lg_guard_params p = lg_guard_params_default();
  if (p.W != 256 || p.K != 2 || p.n_anchor != 32 || p.t_min != 64 || p.cooldown != 32 ||
      p.ttr_num != 1 || p.ttr_den != 5 || p.cr_num != 3 || p.cr_den != 25 ||
      p.conf_threshold != 0.9f || p.mode != LG_MODE_FULL || p.policy != LG_POLICY_LOOPGUARD) {
    printf("unexpected defaults\n");
    ++fails;
  }
  if (lg_state_bytes() != 2112 || lg_decision_bytes() != 64) {
    printf("unexpected state/decision sizes\n");
    ++fails;
  }
  lg_layer_cache c;
  c.batch = 32; c.n_q_heads = 28; c.n_kv_heads = 4; c.head_dim = 128; c.cap = 2048;
  c.dtype = LG_BF16; c.k = DEV(0x1000); c.v = DEV(0x2000); c.acc = (float*)DEV(0x3000);
  const size_t ws = lg_decode_attend_workspace(&c);
  if (ws == 0 || sizeof(lg_attend_workspace_header) != 64) {
    printf("zero workspace or unexpected header size\n");
    ++fails;
  }
  int32_t* i32 = (int32_t*)DEV(0x4000);
  float* f32 = (float*)DEV(0x5000);
  /* attention */
  EXPECT(lg_decode_attend(&c, NULL, NULL, NULL, DEV(0x6000), i32, i32, i32, i32, f32, f32, f32,
                          DEV(0x7000), ws, NULL), LG_ERR_NULL);
  EXPECT(lg_decode_attend(&c, DEV(0x6008), NULL, NULL, DEV(0x6000), i32, i32, i32, i32, f32, f32,
                          f32, DEV(0x7000), ws, NULL), LG_ERR_ALIGN);
  EXPECT(lg_decode_attend(&c, DEV(0x6000), NULL, NULL, DEV(0x6000), i32, i32, i32, i32, f32, f32,
                          f32, DEV(0x7000), ws - 16, NULL), LG_ERR_WORKSPACE);
  EXPECT(lg_decode_attend_workspace_init(&c, DEV(0x7000), ws - 16, NULL), LG_ERR_WORKSPACE);
  EXPECT(lg_decode_attend_workspace_init(&c, DEV(0x7008), ws, NULL), LG_ERR_ALIGN);
  c.n_q_heads = 30;
  EXPECT(lg_decode_attend(&c, DEV(0x6000), NULL, NULL, DEV(0x6000), i32, i32, i32, i32, f32, f32,
                          f32, DEV(0x7000), ws, NULL), LG_ERR_SHAPE);
  c.n_q_heads = 28;
  c.head_dim = 96;
  EXPECT(lg_decode_attend(&c, DEV(0x6000), NULL, NULL, DEV(0x6000), i32, i32, i32, i32, f32, f32,
                          f32, DEV(0x7000), ws, NULL), LG_ERR_UNSUPPORTED);
  c.head_dim = 128;
  /* allocation-free attention: argument checks, and a layer too large for its scratch */
  EXPECT(lg_decode_attend_noalloc(&c, NULL, NULL, NULL, DEV(0x6000), i32, i32, i32, i32, f32, f32,
                                  f32, 0, NULL), LG_ERR_NULL);
  c.cap = 32768;
  if (lg_decode_attend_workspace(&c) <= LG_NOALLOC_SCRATCH_BYTES) {
    printf("expected a workspace above LG_NOALLOC_SCRATCH_BYTES\n");
    ++fails;
  }
  EXPECT(lg_decode_attend_noalloc(&c, DEV(0x6000), NULL, NULL, DEV(0x6000), i32, i32, i32, i32,
                                  f32, f32, f32, 1, NULL), LG_ERR_TOO_LARGE);
  c.cap = 2048;
  /* detector */
  lg_guard_params q = p;
  q.W = 0;
  EXPECT(lg_detect_loop(&q, 4, i32, 2048, i32, i32, f32, (lg_guard_state*)DEV(0x8000),
                        (lg_decision*)DEV(0x9000), NULL), LG_ERR_PARAM);
  EXPECT(lg_detect_loop(&p, 4, i32, 100, i32, i32, f32, (lg_guard_state*)DEV(0x8000),
                        (lg_decision*)DEV(0x9000), NULL), LG_ERR_SHAPE);
  EXPECT(lg_detect_loop(&p, 4, NULL, 2048, i32, i32, f32, (lg_guard_state*)DEV(0x8000),
                        (lg_decision*)DEV(0x9000), NULL), LG_ERR_NULL);
  /* prune */
  lg_layer_cache layers[2] = {c, c};
  EXPECT(lg_prune_compact(&p, 32, 2048, 2, layers, NULL, i32, i32, NULL, NULL, i32, i32, NULL),
         LG_ERR_NULL);
  EXPECT(lg_prune_compact(&p, 32, 1024, 2, layers, i32, i32, i32, NULL, NULL, i32, i32, NULL),
         LG_ERR_SHAPE);
  q = p;
  q.policy = 3;
  EXPECT(lg_prune_compact(&q, 32, 2048, 2, layers, i32, i32, i32, NULL, NULL, i32, i32, NULL),
         LG_ERR_PARAM);
  if (fails == 0) printf("ok\n");
  return fails == 0 ? 0 : 1;
}

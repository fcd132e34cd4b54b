/*
 * lg_testing.h -- test hooks of liblg (not part of the stable API in lg.h).
 *
 * They run lg_decode_attend with its kernel form and split length chosen explicitly, and force
 * the rare paths of the one-launch form's exchange, so that tests can compare the forms with each
 * other and drive every path from the host:
 *   form       LG_TEST_FORM_AUTO (what lg_decode_attend runs), LG_TEST_FORM_PORTABLE (vector-ALU
 *              sweep + combine launch; any supported dtype and cap), LG_TEST_FORM_MERGE (MFMA
 *              sweep + merging launch; bfloat16, cap a multiple of 32 and <= 32768),
 *              LG_TEST_FORM_ONE_LAUNCH (the one-launch form; same requirements).
 *   max_split  0 for the default split length (see lg_decode_attend), else that split length, a
 *              multiple of 32 in [128, 1024] (MFMA forms only; LG_TEST_FORM_AUTO then runs the
 *              merge form), or up to 2048 for LG_TEST_FORM_ONE_LAUNCH when it covers the whole
 *              cap; either is raised to ceil(cap / 32) rounded up to 32 when it is shorter.
 *   flags      LG_TEST_FORCE_HANDOVER: every split of a symmetric row that is not its closer
 *              hands its share over instead of merging it (results are bit-identical).
 *              LG_TEST_NO_WAIT: every wait of the exchange gives up at once, so every row with
 *              more than one split takes the error path (LG_ATTEND_STATUS_WAIT).
 *              LG_TEST_WHOLE_DIMS: a launch whose rows would get two workgroups each (each
 *              forming half of the output dims) gets one per row instead.
 * A workspace serves one (layer shape, form, split length): it is initialised for them with
 * lg_test_attend_workspace_init and is refused (LG_ATTEND_STATUS_WORKSPACE) by a call with
 * another form or split. Sizes, arguments, errors and everything else as in lg.h.
 */
#ifndef LG_TESTING_H
#define LG_TESTING_H

#include "lg.h"

#ifdef __cplusplus
extern "C" {
#endif

enum { LG_TEST_FORM_AUTO = 0, LG_TEST_FORM_PORTABLE = 1, LG_TEST_FORM_MERGE = 2,
       LG_TEST_FORM_ONE_LAUNCH = 3 };
enum { LG_TEST_FORCE_HANDOVER = 1, LG_TEST_NO_WAIT = 2, LG_TEST_WHOLE_DIMS = 4 };

/* Workspace bytes for this layer, form and split bound (0 if the combination is invalid). */
size_t lg_test_attend_workspace(const lg_layer_cache* layer, int32_t form, int32_t max_split);

lg_status lg_test_attend_workspace_init(const lg_layer_cache* layer, int32_t form,
                                        int32_t max_split, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream);

lg_status lg_test_decode_attend(const lg_layer_cache* layer, const void* q, const void* k_new,
                                const void* v_new, void* out, const int32_t* pos,
                                const int32_t* len, const int32_t* t, const int32_t* suffix_w,
                                float* lse, float* suffix_mass, float* conf, void* workspace,
                                size_t workspace_bytes, int32_t form, int32_t max_split,
                                int32_t flags, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* LG_TESTING_H */

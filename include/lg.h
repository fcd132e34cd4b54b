/*
 * lg.h -- C ABI of the LoopGuard guarded-decode hot path for AMD Instinct MI355X (gfx950).
 *
 * One guarded decode step over a batch of independent sequences is three calls, issued in this
 * order on one HIP stream:
 *
 *   1. lg_decode_attend   once per layer: append the step's key/value row, attend over the
 *                          fixed-budget cache, and emit per-head statistics in the same pass.
 *   2. lg_detect_loop     once per step: the debounced onset rule over the token tail and the
 *                          confidence signal; returns the repetitive tail span.
 *   3. lg_prune_compact   once per step: commit the append, then (only for flagged sequences)
 *                          build the retained index set and compact K/V/acc/pos in place.
 *
 * lg_detect_and_prune does 2 and 3 with one launch fewer and the same results.
 *
 * Paper: "LoopGuard: Breaking Self-Reinforcing Attention Loops via Dynamic KV Cache
 * Intervention" (arXiv 2604.10044). Citations below use its section, equation and appendix
 * numbers: Eq. (1) attention over the accessible set S_t (Sec. 3.1); Eq. (5)/(6) TTR and CR
 * (Sec. 4.3); Eq. (8) Warn vote and Eq. (9) Trigger (Sec. 5.2); Eq. (10) I_keep and Eq. (11)
 * C_recent (Sec. 5.3); hyperparameters in Sec. 6.1 and App. B.2.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Memory. Every array argument is caller-owned DEVICE memory unless marked "host". The library
 *    never allocates, frees or synchronises; scratch space comes from the caller through the
 *    workspace argument whose size lg_decode_attend_workspace() reports. The one exception is
 *    lg_decode_attend_noalloc, whose scratch is a static device array of the library.
 *  - Execution. All work is enqueued asynchronously on `stream` (NULL = the default stream).
 *    Nothing is read back to the host. Calls are reentrant and keep no mutable host state, except
 *    lg_decode_attend_noalloc (one scratch per device, see there).
 *  - Errors. Arguments are validated on the host before anything is enqueued; a rejected call
 *    returns LG_ERR_* and enqueues nothing. A failed kernel launch returns LG_ERR_HIP. Device-side
 *    values (len, t, ...) cannot be validated on the host: kernels clamp every index into the
 *    buffers they were given, so a caller that breaks a documented device-side precondition gets
 *    unspecified values but no out-of-bounds access.
 *  - Positions. A sequence's stream index is its token position: the token processed at the step
 *    whose newest position is t is y[t], and after that step the stream holds n = t + 1 tokens.
 *    Cache slots 0..len-1 hold strictly increasing positions (pos[]).
 *  - Layout. Row-major C order; [a][b][c] means c varies fastest.
 *  - Alignment. The cache arrays (k, v, acc), q, k_new, v_new, out and the workspace are accessed
 *    with 16-byte vector loads and stores and must be 16-byte aligned (LG_ERR_ALIGN otherwise).
 */
#ifndef LG_H
#define LG_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LG_OK = 0,
  LG_ERR_NULL = 1,        /* a required pointer is NULL */
  LG_ERR_SHAPE = 2,       /* inconsistent sizes (Hq % Hkv != 0, non-positive sizes, ...) */
  LG_ERR_UNSUPPORTED = 3, /* head_dim, dtype or group size outside the supported set */
  LG_ERR_PARAM = 4,       /* guard parameters violate their documented constraints */
  LG_ERR_WORKSPACE = 5,   /* workspace smaller than lg_decode_attend_workspace() */
  LG_ERR_HIP = 6,         /* a HIP launch failed */
  LG_ERR_ALIGN = 7,       /* a device array is not 16-byte aligned */
  LG_ERR_TOO_LARGE = 8    /* lg_decode_attend_noalloc: the layer needs more than its scratch */
} lg_status;

typedef enum { LG_F32 = 0, LG_BF16 = 1 } lg_dtype;

/* One layer's KV cache (Sec. 3.1: per-head keys/values of the accessible set S_t, |S_t| <= B).
 *   k, v : [batch][n_kv_heads][cap][head_dim] of dtype, row-major; slot j of sequence b holds
 *          the key/value of position pos[b][j].
 *   acc  : [batch][n_kv_heads][cap] float32, H2O-style accumulated attention importance of each
 *          slot, summed over the query heads of the KV head's group (see lg_decode_attend).
 * Supported: head_dim in {64, 128}; n_q_heads % n_kv_heads == 0; group size
 * n_q_heads / n_kv_heads <= 16; dtype in {LG_F32, LG_BF16}; cap >= 1. */
typedef struct {
  int32_t batch, n_q_heads, n_kv_heads, head_dim, cap;
  lg_dtype dtype;
  void *k, *v;
  float *acc;
} lg_layer_cache;

/* Guard hyperparameters (Sec. 5.2, Sec. 5.3, Sec. 6.1, App. B.2). Thresholds that the paper
 * states as decimals are kept as exact rationals so that every vote is an integer comparison:
 *   vote_ttr : distinct/m < ttr_num/ttr_den        (theta_ttr = 0.2  = 1/5)
 *   vote_cr  : lz_cost/m  < cr_num/cr_den          (theta_cr  = 0.12 = 3/25)
 *   stall    : novel/r    < nov_num/nov_den        (theta_nov = 0.02 = 1/50)
 *   streak   : conf > conf_threshold               (theta_conf = 0.9, strict)
 * Keep-set sizes for a sequence with budget B: R = B / recent_div (recent window and suffix
 * width), S = B / sparse_div - n_anchor (sparse budget). A prune keeps at most B - 1 slots, so the
 * next append always fits: when the anchor slots, R >> level and S exceed that (small budgets,
 * small divisors), the anchors claim it first (the earliest of them), then the recent window, then
 * the sparse history; the baseline policies cap their keep size B/sparse_div + B/recent_div at
 * B - 1. With the defaults (recent_div 4, sparse_div 2, n_anchor 32) the cap never binds for
 * B >= 43 (for the baselines, B >= 4). A budget above the cache's capacity (cap) acts as cap. */
typedef struct {
  int32_t W;                /* monitor window (256) */
  int32_t K;                /* votes needed out of 3 (2) */
  int32_t n_anchor;         /* anchor prefix kept by every prune (32) */
  int32_t t_min;            /* warmup in monitored tokens (64) */
  int32_t cooldown;         /* minimum distance between interventions (32) */
  int32_t streak_min;       /* confidence streak that votes (6) */
  int32_t stall_min;        /* consecutive low-novelty steps that make Stall (4) */
  int32_t cr_interval;      /* recompute the compression ratio every cr_interval steps (1) */
  int32_t nov_ngram;        /* n-gram order of the novelty rate (4) */
  int32_t nov_span;         /* novelty is measured over the last nov_span tokens (64) */
  int32_t rep_pmax;         /* largest tail period examined (256) */
  int32_t rep_horizon;      /* longest tail span examined, H (1024) */
  int32_t rep_min_copies;   /* a period qualifies with >= this many copies (3) */
  int32_t rep_min_len;      /* ... and a periodic tail of >= this many tokens (32) */
  int32_t rep_debounce;     /* consecutive qualifying steps that make TailRep (4) */
  int32_t level_max;        /* cap of the aggressiveness level l (3) */
  int32_t retrigger_window; /* a trigger within this many tokens of the last one escalates (64) */
  int32_t recent_div;       /* R = budget / recent_div (4) */
  int32_t sparse_div;       /* S = budget / sparse_div - n_anchor (2) */
  int32_t ttr_num, ttr_den; /* 1, 5 */
  int32_t cr_num, cr_den;   /* 3, 25 */
  int32_t nov_num, nov_den; /* 1, 50 */
  float conf_threshold;     /* 0.9 */
  int32_t mode;             /* LG_MODE_*: 0 = the full rule of Eq. (9) */
  int32_t policy;           /* LG_POLICY_*: keep policy of lg_prune_compact (0 = LoopGuard) */
} lg_guard_params;

/* Ablation variants of Table 3 (Sec. 6.5). LG_MODE_FULL is Eq. (9). LG_MODE_ALWAYS_ON triggers
 * whenever warmup and cooldown allow. LG_MODE_P1_ONLY triggers on the confidence streak alone
 * (warmup and cooldown still apply). */
enum { LG_MODE_FULL = 0, LG_MODE_ALWAYS_ON = 1, LG_MODE_P1_ONLY = 2 };

/* Keep policies of lg_prune_compact. LG_POLICY_LOOPGUARD is Eq. (10)/(11). The other two are the
 * baselines the paper compares against (Sec. 6.1, "Baselines"): H2O (attention heavy hitters) and
 * StreamingLLM (attention sinks + sliding window). The paper gives them no parameters; here both
 * act only when a cache reaches its budget (a trigger does not prune) and keep as many slots as
 * the LoopGuard set would, K = budget/sparse_div + budget/recent_div (see lg_prune_compact). */
enum { LG_POLICY_LOOPGUARD = 0, LG_POLICY_H2O = 1, LG_POLICY_STREAMING = 2 };

/* Per-sequence detector state, carried from step to step. Zero-initialise before the first step.
 * The tail runs let a step that directly follows the previous one (same t0, horizon and period
 * range, stream extended by one token) update every L_P in O(1); any other call recomputes them. */
typedef struct {
  int32_t streak;      /* consecutive steps with conf > conf_threshold */
  int32_t stall;       /* consecutive low-novelty steps */
  int32_t rep;         /* consecutive steps with a qualifying tail period */
  int32_t n_int;       /* interventions so far */
  int32_t n_last;      /* stream length n at the last intervention */
  int32_t level;       /* aggressiveness level l of the last intervention */
  int32_t cr_valid;    /* 1 once a compression cost has been computed */
  int32_t cr_cost;     /* last computed LZ cost (held between recomputations) */
  int32_t cr_m;        /* window length that cr_cost was computed over */
  int32_t tail_n;      /* stream length tail_run is valid for (0: none) */
  int32_t tail_t0, tail_horizon, tail_pmax;
  int32_t reserved[3];
  int32_t tail_run[512]; /* L_P of the trailing self-alignment, P = 1..rep_pmax at index P-1 */
} lg_guard_state;

/* Per-sequence result of one lg_detect_loop step. All fields are integers, so GPU and oracle
 * agree bit for bit. span_lo / bad span: positions [span_lo, n-1] form the maximal repetitive
 * tail (when a period qualifies at this step; else -1). */
typedef struct {
  int32_t trigger;      /* Eq. (9) fired at this step */
  int32_t warn;         /* Eq. (8) */
  int32_t votes;        /* bit0 TTR, bit1 CR, bit2 confidence streak */
  int32_t stall_gate;   /* Stall(t) */
  int32_t tailrep_gate; /* TailRep(t) */
  int32_t n;            /* stream length this decision was taken at */
  int32_t distinct;     /* distinct tokens in the window */
  int32_t lz_cost;      /* compression cost in force (see lg_guard_params) */
  int32_t novel;        /* novel n-grams among the last nov_span tokens */
  int32_t nov_r;        /* number of positions the novelty rate is taken over */
  int32_t period;       /* P*, the qualifying tail period with the longest span; 0 if none */
  int32_t span_lo;      /* first position of the repetitive tail, or -1 */
  int32_t level;        /* aggressiveness level l used by this trigger's keep set */
  int32_t n_int;        /* interventions so far, this one included */
  int32_t attend_error; /* 1 when conf[b] was NaN: an attention call of this step refused or
                           failed for this sequence (see lg_decode_attend); no trigger then */
  int32_t reserved;
} lg_decision;

/* Defaults: the paper's constants (Sec. 6.1, App. B.2) plus the documented readings for what the
 * paper leaves open (R = B/4, S = B/2 - 32, horizon 1024, ...). */
lg_guard_params lg_guard_params_default(void);
const char* lg_status_string(lg_status s);
size_t lg_state_bytes(void);    /* sizeof(lg_guard_state), 2112 */
size_t lg_decision_bytes(void); /* sizeof(lg_decision) */

/* Attention workspace.
 *
 * lg_decode_attend keeps state in its workspace from call to call (the exchange words of the
 * splits of each row, see lg_decode_attend), so a workspace is initialised once for one layer
 * shape with lg_decode_attend_workspace_init and then serves every call of that shape (all layers
 * of a model may share it, calls on it must not overlap in time). Its first 64 bytes are an
 * lg_attend_workspace_header: the shape it was initialised for and a sticky status word. A call
 * whose layer does not match the header, or that finds a non-zero status, does nothing but set
 * LG_ATTEND_STATUS_WORKSPACE and mark conf[b] NaN for the sequences it refuses; a call in which
 * a bounded wait gives up sets LG_ATTEND_STATUS_WAIT the same way. In both cases out, lse,
 * suffix_mass and acc of the affected rows are left as they were, and every later call refuses
 * until the workspace is initialised again. The caller reads the status by copying the header
 * to the host whenever it suits it (no call here synchronises). */
enum { LG_ATTEND_STATUS_WAIT = 1, LG_ATTEND_STATUS_WORKSPACE = 2 };
typedef struct {
  uint32_t magic, version;
  int32_t batch, n_q_heads, n_kv_heads, head_dim, cap, dtype, form, split;
  uint32_t status;      /* 0, or LG_ATTEND_STATUS_* bits */
  uint32_t reserved[5];
} lg_attend_workspace_header;

/* Workspace bytes lg_decode_attend needs for this layer shape (0 for an invalid shape). The
 * one-launch form of a 7B-shaped layer (batch 32, 28 / 4 heads, head_dim 128, cap 2048) needs
 * about 9 MB: the exchange words of every split and the handover probabilities. */
size_t lg_decode_attend_workspace(const lg_layer_cache* layer);

/* Zero-fills the workspace and writes its header for this layer shape (one kernel on `stream`,
 * no memset, so the call may be captured in a graph). Returns LG_ERR_WORKSPACE when
 * workspace_bytes < lg_decode_attend_workspace(layer). */
lg_status lg_decode_attend_workspace_init(const lg_layer_cache* layer, void* workspace,
                                          size_t workspace_bytes, hipStream_t stream);

/* lg_decode_attend -- one layer of decode attention with fused loop statistics.
 *
 * Eq. (1) (Sec. 3.1): for each sequence b and query head h, with G = n_q_heads / n_kv_heads and
 * kv(h) = h / G, over the live slots j (0..len[b]-1, plus the appended row when k_new != NULL):
 *   s_j   = <q_h, k_j^{kv(h)}> / sqrt(head_dim),   alpha_j = softmax_j(s_j)
 *   out_h = sum_j alpha_j v_j^{kv(h)},             lse_h = log sum_j exp(s_j)
 * and in the same pass the statistics the loop monitor uses:
 *   suffix_mass_h = sum of alpha_j over slots with pos_j > t[b] - suffix_w[b]   (attention mass
 *                   on the narrow recent suffix that locked heads concentrate on, Sec. 1, App. E)
 *   acc[b][kv][j] += sum over the G heads of the group of alpha_j              (H2O-style
 *                   accumulated importance, Sec. 2.2 / Sec. 6.1 baseline; new slots start at 0)
 *   conf[b] = max(conf[b], max_h suffix_mass_h)                               (confidence proxy)
 *
 * Arguments
 *   layer       host pointer to the layer's cache view.
 *   q           [batch][n_q_heads][head_dim] dtype; the step's queries (RoPE already applied).
 *   k_new,v_new [batch][n_kv_heads][head_dim] dtype or both NULL. When given, the row is written
 *               to slot len[b] (requires len[b] < cap) with position t[b] and is attended to
 *               (the query sees its own key). pos/len are NOT modified here; lg_prune_compact
 *               commits the append once per step.
 *   out         [batch][n_q_heads][head_dim] dtype.
 *   pos         [batch][cap] int32, strictly increasing over the live slots.
 *   len, t      [batch] int32: live slots before this step's append; newest position.
 *   suffix_w    [batch] int32 >= 0: width of the recent suffix (normally budget/recent_div).
 *               t[b] - suffix_w[b] is evaluated without overflow (saturated to int32).
 *   lse, suffix_mass [batch][n_q_heads] float32 outputs (lse in natural log).
 *   conf        [batch] float32 or NULL; max-accumulated, never lowered here (see lg_detect_loop,
 *               which consumes and clears it).
 *   workspace   initialised by lg_decode_attend_workspace_init for this layer shape (see above);
 *               workspace_bytes as given to the init call.
 * Kernels. A bfloat16 layer whose cap is a multiple of 32 (<= 32768) runs on the matrix cores:
 *   - with at least 128 rows (sequence, kv head) and a cap that fits one split (2048 slots for
 *     groups of at most 8 query heads, else 1024), one launch in which every row is finished by
 *     its own workgroup (two workgroups per row at up to 128 rows of head_dim 128, each forming
 *     half of the output dims), without any exchange between workgroups;
 *   - otherwise a sweep launch (the live slots of each row cut into splits of at most 1024 slots,
 *     one workgroup each, writing split partials and the logits to the workspace) and a merging
 *     launch.
 * The test hooks (lg_testing.h) also reach a one-launch form for rows of several splits, in
 * which the splits of a row exchange their partials through the workspace. No workgroup there
 * waits for one that has not started: a split finds, from an arrival count, whether every split
 * of its row is running; if not, it hands its share of the row to the row's last arriving split
 * and exits. Its waits are still bounded (about 0.1 s); see the status word above. Other layers
 * run a portable kernel pair. Sequences with no live slot and no appended row produce out = 0,
 * lse = -inf, suffix_mass = 0.
 */
lg_status lg_decode_attend(const lg_layer_cache* layer, const void* q, const void* k_new,
                           const void* v_new, void* out, const int32_t* pos, const int32_t* len,
                           const int32_t* t, const int32_t* suffix_w, float* lse,
                           float* suffix_mass, float* conf, void* workspace,
                           size_t workspace_bytes, hipStream_t stream);

/* lg_decode_attend_noalloc -- lg_decode_attend for callers that cannot allocate device memory
 * (code under graph capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * kernels and results, with the workspace taken from a static device array of
 * LG_NOALLOC_SCRATCH_BYTES that the library holds on every device it runs on until the process
 * ends. No call allocates or frees anything.
 *
 * Arguments as lg_decode_attend, without workspace and workspace_bytes, plus
 *   reinit   nonzero: initialise the scratch (one fill kernel on `stream`) before the launch.
 *            Needed after a call marked a sequence's conf NaN (the scratch keeps a sticky status,
 *            as a workspace does); the scratch is also initialised on the first call on a device
 *            and whenever the layer shape differs from the previous call's on that device.
 * The call runs on the current device; a non-NULL stream must belong to it (LG_ERR_PARAM
 * otherwise). A layer whose workspace (lg_decode_attend_workspace) exceeds
 * LG_NOALLOC_SCRATCH_BYTES is refused with LG_ERR_TOO_LARGE before anything is enqueued. All
 * calls on one device share its scratch: calls that overlap in time on one device (other streams,
 * other threads) race and give wrong results; alternating layer shapes re-initialise it each time.
 */
#define LG_NOALLOC_SCRATCH_BYTES (64u << 20)
lg_status lg_decode_attend_noalloc(const lg_layer_cache* layer, const void* q, const void* k_new,
                                   const void* v_new, void* out, const int32_t* pos,
                                   const int32_t* len, const int32_t* t, const int32_t* suffix_w,
                                   float* lse, float* suffix_mass, float* conf, int32_t reinit,
                                   hipStream_t stream);

/* lg_detect_loop -- Stage 1 online monitor (Sec. 5.2, Eq. (8) and (9); App. B.2).
 *
 * For each sequence b, with n = t[b] + 1 and the monitored stream y[t0[b] .. n):
 *   window        w0 = max(t0, n - W), m = n - w0
 *   vote_ttr      distinct(y[w0..n)) / m < theta_ttr                                    Eq. (5)
 *   vote_cr       LZ cost / m < theta_cr; the cost is a greedy token-level LZ77 parse of the
 *                 window (match of >= 3 tokens costs 2, a literal costs 1)                Eq. (6)
 *   vote_p1       streak >= streak_min, streak counting steps with conf > conf_threshold
 *   Warn          vote_ttr + vote_cr + vote_p1 >= K                                      Eq. (8)
 *   Stall         novelty rate < theta_nov for stall_min consecutive steps, the rate being
 *                 the share of first-occurrence nov_ngram-grams among the last nov_span tokens
 *   TailRep       a tail period P <= rep_pmax with >= rep_min_copies copies and a periodic tail
 *                 of >= rep_min_len tokens (within rep_horizon), on rep_debounce consecutive steps
 *   Trigger       n - t0 >= t_min  and  (no intervention yet or n - n_last >= cooldown)  and
 *                 Warn and (Stall or TailRep)                                            Eq. (9)
 * On a trigger the aggressiveness level escalates (capped) when it follows the previous one
 * within retrigger_window tokens and resets to 0 otherwise (Sec. 5.3).
 *
 * Arguments
 *   p         host pointer to the parameters.
 *   tokens    [batch][ring] int32 circular buffer: stream index i lives at tokens[b][i % ring].
 *             It must hold y[max(t0, n - max(W, rep_horizon)) .. n) at the call.
 *   ring      ring length; ring >= max(W, rep_horizon) required.
 *   t, t0     [batch] int32: newest position (clamped to [-1, 2^30 - 1]); first monitored
 *             position (clamped to [0, t + 1]; prompt length for a
 *             real model, 0 when the whole stream is monitored).
 *   conf      [batch] float32 or NULL: read, then reset to 0 for the next step. A NaN (the mark
 *             lg_decode_attend leaves on a sequence whose attention it refused or could not
 *             finish) counts as "not above the threshold", sets decision.attend_error and
 *             suppresses the trigger of this step.
 *   state     [batch] lg_guard_state, updated.
 *   decision  [batch] lg_decision, overwritten.
 */
lg_status lg_detect_loop(const lg_guard_params* p, int32_t batch, const int32_t* tokens,
                         int32_t ring, const int32_t* t, const int32_t* t0, float* conf,
                         lg_guard_state* state, lg_decision* decision, hipStream_t stream);

/* lg_prune_compact -- Stage 2 adaptive pruning (Sec. 5.3, Eq. (10) and (11)) and budget upkeep.
 *
 * Per sequence b:
 *   1. Commit: when t_append != NULL, pos[b][len[b]] = t_append[b] and len[b] += 1.
 *   2. Flag:   a trigger (decision[b].trigger, LoopGuard policy only) prunes with I_bad and level l
 *              from the decision; otherwise len[b] >= budget[b] prunes with I_bad empty and l = 0
 *              (keeps the next append inside the budget; also how a prefill longer than the
 *              budget is reduced).
 *   3. Keep set over the live slots, t = pos[len-1], R = budget/recent_div,
 *      S = budget/sparse_div - n_anchor:
 *        A      = slots with pos < n_anchor                                (anchors)
 *        Rc     = slots not in A with pos >= t - R + 1                     (recent window)
 *        Bad    = slots of Rc with pos >= span_lo (empty without a span)   (I_bad, Eq. (11))
 *        Mid    = all other slots, M = |Mid|
 *        I_recent = the last min(R >> l, |Rc \ Bad|) slots of Rc \ Bad
 *        I_sparse = Mid if M <= S, else Mid[floor(k M / S)] for k = 0..S-1 (evenly spaced)
 *        I_keep   = A u I_sparse u I_recent, ascending                      Eq. (10)
 *      With p->policy = LG_POLICY_H2O or LG_POLICY_STREAMING step 3 is instead, with
 *      K = budget/sparse_div + budget/recent_div kept slots (all of them when len <= K):
 *        H2O:  the last R' = min(R, len) slots, plus the K - R' older slots of highest score,
 *              score[j] = sum over the given layers (ascending) and KV heads (ascending) of
 *              acc[b][h][j], added in float32 in that order (0 when n_layers = 0). Scores are
 *              ordered as float values with -0 below +0 (NaN not allowed); of two equal scores
 *              the slot with the higher position is kept (the lower position is evicted first).
 *        StreamingLLM: the A slots with pos < n_anchor (attention sinks) plus the last K - A
 *              other slots.
 *   4. Compact in place, for every layer and KV head: K, V and acc rows r <- keep[r]; pos likewise;
 *      len = |I_keep|. Rows beyond the new length keep stale contents.
 *
 * Arguments
 *   p            host pointer to the parameters.
 *   batch, cap   shape of pos/keep_idx; every layer must have the same batch and cap.
 *   n_layers     number of entries in `layers` (host array); 0 prunes pos/len only.
 *   pos, len     [batch][cap], [batch] int32, updated in place.
 *   budget       [batch] int32 >= 1; a budget above cap acts as cap, and the keep set never
 *                exceeds budget - 1 slots whatever the parameters (see lg_guard_params).
 *   t_append     [batch] int32 or NULL (see 1).
 *   decision     [batch] lg_decision or NULL (NULL: budget upkeep only).
 *   keep_idx     [batch][cap] int32 output: the kept source slots of flagged sequences (with the
 *                H2O policy it also holds the scores while the call runs).
 *   new_len      [batch] int32 output: |I_keep| for flagged sequences, -1 for the others.
 */
lg_status lg_prune_compact(const lg_guard_params* p, int32_t batch, int32_t cap, int32_t n_layers,
                           const lg_layer_cache* layers, int32_t* pos, int32_t* len,
                           const int32_t* budget, const int32_t* t_append,
                           const lg_decision* decision, int32_t* keep_idx, int32_t* new_len,
                           hipStream_t stream);

/* lg_detect_and_prune -- lg_detect_loop followed by lg_prune_compact (decision = the decisions
 * just made), with the detector and the keep set of each sequence in one kernel launch (both are
 * one workgroup per sequence; the keep set reads the decision the detector has just written), so
 * a guarded step costs one launch fewer. Arguments, results and errors as the two calls: p,
 * batch, tokens, ring, t, t0, conf, state, decision as lg_detect_loop; cap, n_layers, layers,
 * pos, len, budget, t_append, keep_idx, new_len as lg_prune_compact (t_append is normally t). */
lg_status lg_detect_and_prune(const lg_guard_params* p, int32_t batch, const int32_t* tokens,
                              int32_t ring, const int32_t* t, const int32_t* t0, float* conf,
                              lg_guard_state* state, lg_decision* decision, int32_t cap,
                              int32_t n_layers, const lg_layer_cache* layers, int32_t* pos,
                              int32_t* len, const int32_t* budget, const int32_t* t_append,
                              int32_t* keep_idx, int32_t* new_len, hipStream_t stream);

/* lg_copy_bandwidth -- plain device-to-device copy of `bytes` (multiple of 16) with the same
 * launch style as the attention sweep; used to measure the achievable HBM bandwidth beside the
 * roofline peak. */
lg_status lg_copy_bandwidth(const void* src, void* dst, size_t bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* LG_H */

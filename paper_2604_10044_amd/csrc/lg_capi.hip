// lg_capi.hip -- the extern "C" entry points of liblg: host-side validation, workspace layout
// and launch. Nothing here allocates, frees or synchronises.
#include <mutex>

#include "lg_internal.h"
#include "lg_testing.h"

namespace lg {
hipError_t launch_attend(AttendArgs a, lg_dtype dt, int D, hipStream_t st);
hipError_t launch_ws_init(void* ws, size_t bytes, const WsHeader& h, hipStream_t st);
hipError_t launch_detect(const lg_guard_params* p, int batch, const int32_t* tokens, int ring,
                         const int32_t* t, const int32_t* t0, float* conf, lg_guard_state* state,
                         lg_decision* decision, hipStream_t st);
hipError_t launch_prune(const lg_guard_params* p, int batch, int cap, int n_layers,
                        const lg_layer_cache* layers, int32_t* pos, int32_t* len,
                        const int32_t* budget, const int32_t* t_append,
                        const lg_decision* decision, int32_t* keep_idx, int32_t* new_len,
                        hipStream_t st);
hipError_t launch_detect_prune(const lg_guard_params* p, int batch, const int32_t* tokens,
                               int ring, const int32_t* t, const int32_t* t0, float* conf,
                               lg_guard_state* state, lg_decision* decision, int cap,
                               int n_layers, const lg_layer_cache* layers, int32_t* pos,
                               int32_t* len, const int32_t* budget, const int32_t* t_append,
                               int32_t* keep_idx, int32_t* new_len, hipStream_t st);
hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t st);

static bool misaligned(const void* p) { return ((uintptr_t)p & 15u) != 0; }

static lg_status check_layer(const lg_layer_cache* c) {
  if (c == nullptr) return LG_ERR_NULL;
  if (c->k == nullptr || c->v == nullptr || c->acc == nullptr) return LG_ERR_NULL;
  if (misaligned(c->k) || misaligned(c->v) || misaligned(c->acc)) return LG_ERR_ALIGN;
  if (c->batch <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->cap <= 0) return LG_ERR_SHAPE;
  if (c->n_q_heads % c->n_kv_heads != 0) return LG_ERR_SHAPE;
  if (c->n_q_heads / c->n_kv_heads > kMaxGroup) return LG_ERR_UNSUPPORTED;
  if (c->head_dim != 64 && c->head_dim != 128) return LG_ERR_UNSUPPORTED;
  if (c->dtype != LG_F32 && c->dtype != LG_BF16) return LG_ERR_UNSUPPORTED;
  if (c->batch > 65535 || c->n_kv_heads > 65535) return LG_ERR_SHAPE;
  return LG_OK;
}

static lg_status check_params(const lg_guard_params* p) {
  if (p == nullptr) return LG_ERR_NULL;
  if (p->W < 1 || p->W > kMaxWindow) return LG_ERR_PARAM;
  if (p->K < 0 || p->K > 3) return LG_ERR_PARAM;
  if (p->n_anchor < 0 || p->t_min < 0 || p->cooldown < 0) return LG_ERR_PARAM;
  if (p->streak_min < 0 || p->stall_min < 0 || p->rep_debounce < 0) return LG_ERR_PARAM;
  if (p->cr_interval < 1) return LG_ERR_PARAM;
  if (p->nov_ngram < 1 || p->nov_ngram > kMaxNgram || p->nov_span < 1) return LG_ERR_PARAM;
  if (p->rep_pmax < 1 || p->rep_pmax > kMaxPeriod) return LG_ERR_PARAM;
  if (p->rep_horizon < 1 || p->rep_horizon > kMaxHorizon) return LG_ERR_PARAM;
  if (p->rep_min_copies < 1 || p->rep_min_len < 0) return LG_ERR_PARAM;
  if (p->level_max < 0 || p->level_max > 30 || p->retrigger_window < 0) return LG_ERR_PARAM;
  if (p->recent_div < 1 || p->sparse_div < 1) return LG_ERR_PARAM;
  if (p->ttr_den <= 0 || p->cr_den <= 0 || p->nov_den <= 0) return LG_ERR_PARAM;
  if (p->ttr_num < 0 || p->cr_num < 0 || p->nov_num < 0) return LG_ERR_PARAM;
  if (p->mode < LG_MODE_FULL || p->mode > LG_MODE_P1_ONLY) return LG_ERR_PARAM;
  if (p->policy < LG_POLICY_LOOPGUARD || p->policy > LG_POLICY_STREAMING) return LG_ERR_PARAM;
  return LG_OK;
}

// Validated launch plan of an attention call (test hook arguments included).
static lg_status attend_plan_checked(const lg_layer_cache* layer, int form, int max_split,
                                     AttendPlan* plan) {
  lg_status s = check_layer(layer);
  if (s != LG_OK) return s;
  if (form < LG_TEST_FORM_AUTO || form > LG_TEST_FORM_ONE_LAUNCH) return LG_ERR_UNSUPPORTED;
  if ((form == LG_TEST_FORM_MERGE || form == LG_TEST_FORM_ONE_LAUNCH) && !mfma_eligible(*layer))
    return LG_ERR_UNSUPPORTED;
  if (max_split != 0) {
    if (form == LG_TEST_FORM_PORTABLE || (form == LG_TEST_FORM_AUTO && !mfma_eligible(*layer)))
      return LG_ERR_PARAM;
    if (max_split < 32 * kWaves || max_split % 32 != 0) return LG_ERR_PARAM;
    // beyond kMaxSplitSlots: a one-launch split that covers the whole cap
    const bool one = form == LG_TEST_FORM_ONE_LAUNCH;
    if (max_split > kMaxSplitSlots &&
        !(one && max_split <= single_split_max(*layer) && max_split >= layer->cap))
      return LG_ERR_PARAM;
  }
  *plan = attend_plan(*layer, form, max_split);
  return LG_OK;
}

static_assert(sizeof(lg_attend_workspace_header) == sizeof(WsHeader), "public header layout");
static_assert(LG_TEST_FORCE_HANDOVER == kFlagForceHandover && LG_TEST_NO_WAIT == kFlagNoWait &&
                  LG_TEST_WHOLE_DIMS == kFlagWholeDims,
              "test flags");

static WsHeader ws_header(const lg_layer_cache& c, const AttendPlan& p) {
  WsHeader h = {};
  h.magic = kWsMagic;
  h.version = kWsVersion;
  h.batch = c.batch;
  h.n_q_heads = c.n_q_heads;
  h.n_kv_heads = c.n_kv_heads;
  h.head_dim = c.head_dim;
  h.cap = c.cap;
  h.dtype = (int32_t)c.dtype;
  h.form = p.form;
  h.split = p.split;
  h.status = 0;
  return h;
}

// Host-side argument checks shared by the attention entry points.
static lg_status check_attend_args(const void* q, const void* k_new, const void* v_new,
                                   const void* out, const int32_t* pos, const int32_t* len,
                                   const int32_t* t, const int32_t* suffix_w, const float* lse,
                                   const float* suffix_mass) {
  if (!q || !out || !pos || !len || !t || !suffix_w || !lse || !suffix_mass) return LG_ERR_NULL;
  if ((k_new == nullptr) != (v_new == nullptr)) return LG_ERR_NULL;
  if (misaligned(q) || misaligned(out) || misaligned(k_new) || misaligned(v_new))
    return LG_ERR_ALIGN;
  return LG_OK;
}

// One attention launch on a workspace laid out (and initialised) for this layer and plan.
static lg_status attend_launch(const lg_layer_cache& layer, const AttendPlan& plan,
                               const AttendLayout& W, const void* q, const void* k_new,
                               const void* v_new, void* out, const int32_t* pos,
                               const int32_t* len, const int32_t* t, const int32_t* suffix_w,
                               float* lse, float* suffix_mass, float* conf, char* ws, int flags,
                               hipStream_t stream) {
  AttendArgs a = {};
  a.k = layer.k;
  a.v = layer.v;
  a.k_w = layer.k;
  a.v_w = layer.v;
  a.acc = layer.acc;
  a.q = q;
  a.k_new = k_new;
  a.v_new = v_new;
  a.out = out;
  a.pos = pos;
  a.len = len;
  a.t = t;
  a.suffix_w = suffix_w;
  a.lse = lse;
  a.suffix_mass = suffix_mass;
  a.conf = conf;
  a.hdr = (WsHeader*)ws;
  a.part_ml = (float2*)(ws + W.off_ml);
  a.part_s = (float*)(ws + W.off_s);
  a.part_o = (float*)(ws + W.off_o);
  a.stash = (float*)(ws + W.off_stash);
  a.rows = (unsigned long long*)(ws + W.off_rows);
  a.stats = (unsigned long long*)(ws + W.off_stats);
  a.mode = (unsigned*)(ws + W.off_mode);
  a.numer = (unsigned*)(ws + W.off_numer);
  a.hand = (unsigned*)(ws + W.off_hand);
  a.B = layer.batch;
  a.Hq = layer.n_q_heads;
  a.Hkv = layer.n_kv_heads;
  a.G = layer.n_q_heads / layer.n_kv_heads;
  a.cap = layer.cap;
  a.cap_s = W.cap_s;
  a.dtype = (int)layer.dtype;
  a.form = plan.form;
  a.split = plan.split;
  a.ns_grid = plan.ns_grid;
  a.dsplit = (flags & kFlagWholeDims) ? 1 : plan.dsplit;
  a.row_major = 0;
  a.flags = flags;
  a.spin_limit = kSpinLimit;
  a.scale_log2 = kLog2e / sqrtf((float)layer.head_dim);
  return launch_attend(a, layer.dtype, layer.head_dim, stream) == hipSuccess ? LG_OK : LG_ERR_HIP;
}

// Scratch of lg_decode_attend_noalloc: an attention workspace for callers that cannot allocate.
// Every device the library runs on holds its own copy until the process ends. Host code reaches
// it only through the device address hipGetSymbolAddress gives with that device current, kept per
// device with the layer shape it was last initialised for.
static __device__ __align__(256) unsigned char noalloc_scratch[LG_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxScratchDevices = 64;
struct ScratchSlot {
  void* ptr = nullptr;  // device address of noalloc_scratch on this device
  bool ready = false;   // the scratch holds a workspace initialised for `shape`
  WsHeader shape = {};
};
static std::mutex g_scratch_mu;
static ScratchSlot g_scratch[kMaxScratchDevices];

static bool same_workspace(const WsHeader& x, const WsHeader& y) {
  return x.batch == y.batch && x.n_q_heads == y.n_q_heads && x.n_kv_heads == y.n_kv_heads &&
         x.head_dim == y.head_dim && x.cap == y.cap && x.dtype == y.dtype && x.form == y.form &&
         x.split == y.split;
}


}  // namespace lg

using namespace lg;

extern "C" {

lg_guard_params lg_guard_params_default(void) {
  lg_guard_params p;
  p.W = 256;
  p.K = 2;
  p.n_anchor = 32;
  p.t_min = 64;
  p.cooldown = 32;
  p.streak_min = 6;
  p.stall_min = 4;
  p.cr_interval = 1;
  p.nov_ngram = 4;
  p.nov_span = 64;
  p.rep_pmax = 256;
  p.rep_horizon = 1024;
  p.rep_min_copies = 3;
  p.rep_min_len = 32;
  p.rep_debounce = 4;
  p.level_max = 3;
  p.retrigger_window = 64;
  p.recent_div = 4;
  p.sparse_div = 2;
  p.ttr_num = 1;
  p.ttr_den = 5;
  p.cr_num = 3;
  p.cr_den = 25;
  p.nov_num = 1;
  p.nov_den = 50;
  p.conf_threshold = 0.9f;
  p.mode = LG_MODE_FULL;
  p.policy = LG_POLICY_LOOPGUARD;
  return p;
}

const char* lg_status_string(lg_status s) {
  switch (s) {
    case LG_OK: return "ok";
    case LG_ERR_NULL: return "null pointer argument";
    case LG_ERR_SHAPE: return "inconsistent shape";
    case LG_ERR_UNSUPPORTED: return "unsupported head_dim, dtype or group size";
    case LG_ERR_PARAM: return "invalid guard parameters";
    case LG_ERR_WORKSPACE: return "workspace too small";
    case LG_ERR_HIP: return "HIP launch failed";
    case LG_ERR_ALIGN: return "device array not 16-byte aligned";
    case LG_ERR_TOO_LARGE:
      return "layer shape needs more scratch than lg_decode_attend_noalloc holds";
  }
  return "unknown status";
}

size_t lg_state_bytes(void) { return sizeof(lg_guard_state); }
size_t lg_decision_bytes(void) { return sizeof(lg_decision); }

size_t lg_decode_attend_workspace(const lg_layer_cache* layer) {
  return lg_test_attend_workspace(layer, LG_TEST_FORM_AUTO, 0);
}

lg_status lg_decode_attend_workspace_init(const lg_layer_cache* layer, void* workspace,
                                          size_t workspace_bytes, hipStream_t stream) {
  return lg_test_attend_workspace_init(layer, LG_TEST_FORM_AUTO, 0, workspace, workspace_bytes,
                                       stream);
}

lg_status lg_decode_attend(const lg_layer_cache* layer, const void* q, const void* k_new,
                           const void* v_new, void* out, const int32_t* pos, const int32_t* len,
                           const int32_t* t, const int32_t* suffix_w, float* lse,
                           float* suffix_mass, float* conf, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  return lg_test_decode_attend(layer, q, k_new, v_new, out, pos, len, t, suffix_w, lse,
                               suffix_mass, conf, workspace, workspace_bytes, LG_TEST_FORM_AUTO,
                               0, 0, stream);
}

size_t lg_test_attend_workspace(const lg_layer_cache* layer, int32_t form, int32_t max_split) {
  AttendPlan plan;
  if (attend_plan_checked(layer, form, max_split, &plan) != LG_OK) return 0;
  return attend_layout(*layer, plan).bytes;
}

lg_status lg_test_attend_workspace_init(const lg_layer_cache* layer, int32_t form,
                                        int32_t max_split, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
  AttendPlan plan;
  lg_status s = attend_plan_checked(layer, form, max_split, &plan);
  if (s != LG_OK) return s;
  if (workspace == nullptr) return LG_ERR_NULL;
  if (misaligned(workspace)) return LG_ERR_ALIGN;
  const AttendLayout W = attend_layout(*layer, plan);
  if (workspace_bytes < W.bytes) return LG_ERR_WORKSPACE;
  return launch_ws_init(workspace, W.bytes, ws_header(*layer, plan), stream) == hipSuccess
             ? LG_OK : LG_ERR_HIP;
}

lg_status lg_test_decode_attend(const lg_layer_cache* layer, const void* q, const void* k_new,
                                const void* v_new, void* out, const int32_t* pos,
                                const int32_t* len, const int32_t* t, const int32_t* suffix_w,
                                float* lse, float* suffix_mass, float* conf, void* workspace,
                                size_t workspace_bytes, int32_t form, int32_t max_split,
                                int32_t flags, hipStream_t stream) {
  AttendPlan plan;
  lg_status s = attend_plan_checked(layer, form, max_split, &plan);
  if (s != LG_OK) return s;
  if (flags < 0 || flags > (LG_TEST_FORCE_HANDOVER | LG_TEST_NO_WAIT | LG_TEST_WHOLE_DIMS))
    return LG_ERR_PARAM;
  s = check_attend_args(q, k_new, v_new, out, pos, len, t, suffix_w, lse, suffix_mass);
  if (s != LG_OK) return s;
  if (misaligned(workspace)) return LG_ERR_ALIGN;
  const AttendLayout W = attend_layout(*layer, plan);
  if (workspace == nullptr || workspace_bytes < W.bytes) return LG_ERR_WORKSPACE;
  return attend_launch(*layer, plan, W, q, k_new, v_new, out, pos, len, t, suffix_w, lse,
                       suffix_mass, conf, (char*)workspace, flags, stream);
}

lg_status lg_decode_attend_noalloc(const lg_layer_cache* layer, const void* q, const void* k_new,
                                   const void* v_new, void* out, const int32_t* pos,
                                   const int32_t* len, const int32_t* t, const int32_t* suffix_w,
                                   float* lse, float* suffix_mass, float* conf, int32_t reinit,
                                   hipStream_t stream) {
  AttendPlan plan;
  lg_status s = attend_plan_checked(layer, LG_TEST_FORM_AUTO, 0, &plan);
  if (s != LG_OK) return s;
  const AttendLayout W = attend_layout(*layer, plan);
  if (W.bytes > (size_t)LG_NOALLOC_SCRATCH_BYTES) return LG_ERR_TOO_LARGE;
  s = check_attend_args(q, k_new, v_new, out, pos, len, t, suffix_w, lse, suffix_mass);
  if (s != LG_OK) return s;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) return LG_ERR_HIP;
  if (stream != nullptr) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(stream, &sdev) != hipSuccess) return LG_ERR_HIP;
    if (sdev != dev) return LG_ERR_PARAM;
  }
  char* ws = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    ScratchSlot& slot = g_scratch[dev];
    if (slot.ptr == nullptr) {
      // The array's name is a host-side stand-in; its device address on the current device is
      // the one to pass to kernels.
      void* p = nullptr;
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(noalloc_scratch)) != hipSuccess || p == nullptr)
        return LG_ERR_HIP;
      slot.ptr = p;
    }
    const WsHeader h = ws_header(*layer, plan);
    if (reinit != 0 || !slot.ready || !same_workspace(slot.shape, h)) {
      slot.ready = false;
      if (launch_ws_init(slot.ptr, W.bytes, h, stream) != hipSuccess) return LG_ERR_HIP;
      slot.shape = h;
      slot.ready = true;
    }
    ws = (char*)slot.ptr;
  }
  return attend_launch(*layer, plan, W, q, k_new, v_new, out, pos, len, t, suffix_w, lse,
                       suffix_mass, conf, ws, 0, stream);
}

lg_status lg_detect_loop(const lg_guard_params* p, int32_t batch, const int32_t* tokens,
                         int32_t ring, const int32_t* t, const int32_t* t0, float* conf,
                         lg_guard_state* state, lg_decision* decision, hipStream_t stream) {
  lg_status s = check_params(p);
  if (s != LG_OK) return s;
  if (!tokens || !t || !t0 || !state || !decision) return LG_ERR_NULL;
  if (batch <= 0) return LG_ERR_SHAPE;
  if (ring < (p->W > p->rep_horizon ? p->W : p->rep_horizon)) return LG_ERR_SHAPE;
  return launch_detect(p, batch, tokens, ring, t, t0, conf, state, decision, stream) == hipSuccess
             ? LG_OK : LG_ERR_HIP;
}

// Host-side checks of a prune call (shared with lg_detect_and_prune).
static lg_status check_prune(const lg_guard_params* p, int32_t batch, int32_t cap,
                             int32_t n_layers, const lg_layer_cache* layers, const int32_t* pos,
                             const int32_t* len, const int32_t* budget, const int32_t* keep_idx,
                             const int32_t* new_len) {
  if (p == nullptr) return LG_ERR_NULL;
  if (p->n_anchor < 0 || p->recent_div < 1 || p->sparse_div < 1 || p->level_max < 0 ||
      p->level_max > 30 || p->policy < LG_POLICY_LOOPGUARD || p->policy > LG_POLICY_STREAMING)
    return LG_ERR_PARAM;
  if (!pos || !len || !budget || !keep_idx || !new_len) return LG_ERR_NULL;
  if (batch <= 0 || cap <= 0 || n_layers < 0 || batch > 65535) return LG_ERR_SHAPE;
  if (n_layers > 0) {
    if (layers == nullptr) return LG_ERR_NULL;
    for (int i = 0; i < n_layers; ++i) {
      lg_status s = check_layer(&layers[i]);
      if (s != LG_OK) return s;
      if (layers[i].batch != batch || layers[i].cap != cap ||
          layers[i].n_kv_heads != layers[0].n_kv_heads ||
          layers[i].head_dim != layers[0].head_dim || layers[i].dtype != layers[0].dtype)
        return LG_ERR_SHAPE;
    }
  }
  return LG_OK;
}

lg_status lg_prune_compact(const lg_guard_params* p, int32_t batch, int32_t cap, int32_t n_layers,
                           const lg_layer_cache* layers, int32_t* pos, int32_t* len,
                           const int32_t* budget, const int32_t* t_append,
                           const lg_decision* decision, int32_t* keep_idx, int32_t* new_len,
                           hipStream_t stream) {
  const lg_status s = check_prune(p, batch, cap, n_layers, layers, pos, len, budget, keep_idx,
                                  new_len);
  if (s != LG_OK) return s;
  return launch_prune(p, batch, cap, n_layers, layers, pos, len, budget, t_append, decision,
                      keep_idx, new_len, stream) == hipSuccess ? LG_OK : LG_ERR_HIP;
}

lg_status lg_detect_and_prune(const lg_guard_params* p, int32_t batch, const int32_t* tokens,
                              int32_t ring, const int32_t* t, const int32_t* t0, float* conf,
                              lg_guard_state* state, lg_decision* decision, int32_t cap,
                              int32_t n_layers, const lg_layer_cache* layers, int32_t* pos,
                              int32_t* len, const int32_t* budget, const int32_t* t_append,
                              int32_t* keep_idx, int32_t* new_len, hipStream_t stream) {
  lg_status s = check_params(p);
  if (s != LG_OK) return s;
  if (!tokens || !t || !t0 || !state || !decision) return LG_ERR_NULL;
  if (batch <= 0) return LG_ERR_SHAPE;
  if (ring < (p->W > p->rep_horizon ? p->W : p->rep_horizon)) return LG_ERR_SHAPE;
  s = check_prune(p, batch, cap, n_layers, layers, pos, len, budget, keep_idx, new_len);
  if (s != LG_OK) return s;
  return launch_detect_prune(p, batch, tokens, ring, t, t0, conf, state, decision, cap, n_layers,
                             layers, pos, len, budget, t_append, keep_idx, new_len,
                             stream) == hipSuccess ? LG_OK : LG_ERR_HIP;
}

lg_status lg_copy_bandwidth(const void* src, void* dst, size_t bytes, hipStream_t stream) {
  if (!src || !dst) return LG_ERR_NULL;
  if (misaligned(src) || misaligned(dst)) return LG_ERR_ALIGN;
  if (bytes % 16 != 0) return LG_ERR_SHAPE;
  if (bytes == 0) return LG_OK;
  return launch_copy(src, dst, bytes, stream) == hipSuccess ? LG_OK : LG_ERR_HIP;
}

}  // extern "C"

// C ABI of libdsde: host-side argument validation (before any HIP call),
// workspace sizing and dispatch to the kernels.
#include <math.h>

#include <mutex>

#include "common.hpp"
#include "shard.hpp"

namespace {

hipEvent_t g_prof_start = nullptr, g_prof_stop = nullptr;

bool verify_sizes_ok(int32_t B, int64_t N, int64_t V, int32_t k_max) {
  if (B < 1 || V < 1 || V > DSDE_MAX_VOCAB || N < 0 || k_max < 0 || k_max > DSDE_MAX_K) return false;
  if (N > int64_t(B) * k_max) return false;
  // per-sequence slots b * k_max + j index the chunk partials
  if (int64_t(B) * k_max >= (int64_t(1) << 31)) return false;
  const int64_t nc = (V + dsde::kChunk - 1) / dsde::kChunk;
  // the grid of the statistics pass must fit one launch dimension
  if (N * nc >= (int64_t(1) << 31)) return false;
  return true;
}

}  // namespace

extern "C" {

int32_t dsde_abi_version(void) { return DSDE_ABI_VERSION; }

const char *dsde_status_string(int32_t status) {
  switch (status) {
    case DSDE_OK:
      return "ok";
    case DSDE_INVALID_ARG:
      return "invalid argument";
    case DSDE_WORKSPACE_TOO_SMALL:
      return "workspace too small";
    case DSDE_DEVICE_ERROR:
      return "device error";
    default:
      return "unknown status";
  }
}

size_t dsde_verify_workspace_bytes(int32_t B, int64_t N, int64_t V, int32_t k_max) {
  if (!verify_sizes_ok(B, N, V, k_max)) return 0;
  return dsde::workspace_layout(B, N, V, k_max).total;
}

int32_t dsde_verify(const void *target_logits, const void *draft_logits, int32_t dtype, int64_t V, int32_t B,
                    int64_t N, int32_t k_max, const int32_t *sl, const int32_t *cu_sl,
                    const int32_t *draft_tokens, const float *temperature, const float *u_acc,
                    const float *u_res, int32_t pad_id, int32_t *accepted, int32_t *tokens, float *kld,
                    uint32_t *seq_err, double *row_lse, float *draft_entropy, void *workspace,
                    size_t workspace_bytes, void *stream) {
  if (dtype != DSDE_FP32 && dtype != DSDE_BF16) return DSDE_INVALID_ARG;
  if (!verify_sizes_ok(B, N, V, k_max)) return DSDE_INVALID_ARG;
  if (!target_logits || !sl || !cu_sl || !temperature || !u_res || !accepted || !tokens || !seq_err ||
      !workspace)
    return DSDE_INVALID_ARG;
  if (N > 0 && (!draft_logits || !draft_tokens || !u_acc || !kld)) return DSDE_INVALID_ARG;
  if (workspace_bytes < dsde::workspace_layout(B, N, V, k_max).total) return DSDE_WORKSPACE_TOO_SMALL;
  if ((reinterpret_cast<uintptr_t>(workspace) & 15u) != 0) return DSDE_INVALID_ARG;
  dsde::VerifyArgs a;
  a.target = target_logits;
  a.draft = draft_logits;
  a.dtype = dtype;
  a.V = V;
  a.B = B;
  a.N = N;
  a.k_max = k_max;
  a.sl = sl;
  a.cu_sl = cu_sl;
  a.draft_tokens = draft_tokens;
  a.temperature = temperature;
  a.u_acc = u_acc;
  a.u_res = u_res;
  a.pad_id = pad_id;
  a.accepted = accepted;
  a.tokens = tokens;
  a.kld = kld;
  a.seq_err = seq_err;
  a.row_lse = row_lse;
  a.draft_entropy = draft_entropy;
  a.workspace = workspace;
  a.stream = static_cast<hipStream_t>(stream);
  a.prof_start = g_prof_start;
  a.prof_stop = g_prof_stop;
  a.signal = nullptr;
  return dsde::launch_verify(a);
}

// The signal and SL-rule arguments of the fused calls, checked and packed.
static int32_t signal_args(float *hist, int32_t *head, int32_t *count, int32_t W, int32_t n_short, int32_t n_long,
                           float delta, float eps, float *mu_last, float *var_short, float *var_long, float *wvir,
                           float *sf, const float *sl_max, float sl_min, int32_t sl_hi, const int32_t *budget,
                           float *sl_hat, float *sl_cap, int32_t *sl_next, dsde::SignalArgs *sg) {
  if (W < 1 || n_short < 1 || n_short > n_long) return DSDE_INVALID_ARG;
  if (!(delta > 0.0f && delta <= 1.0f) || !(eps > 0.0f) || !isfinite(eps)) return DSDE_INVALID_ARG;
  if (!hist || !head || !count || !mu_last || !var_short || !var_long || !wvir || !sf) return DSDE_INVALID_ARG;
  if (!isfinite(sl_min) || ceilf(sl_min) > float(sl_hi)) return DSDE_INVALID_ARG;
  if (!sl_max || !sl_hat || !sl_cap || !sl_next) return DSDE_INVALID_ARG;
  sg->hist = hist;
  sg->head = head;
  sg->count = count;
  sg->W = W;
  sg->n_short = n_short;
  sg->n_long = n_long;
  sg->delta = delta;
  sg->eps = eps;
  sg->mu_last = mu_last;
  sg->var_short = var_short;
  sg->var_long = var_long;
  sg->wvir = wvir;
  sg->sf = sf;
  sg->sl_max = sl_max;
  sg->sl_min = sl_min;
  sg->sl_hi = sl_hi;
  sg->budget = budget;
  sg->sl_hat = sl_hat;
  sg->sl_cap = sl_cap;
  sg->sl_next = sl_next;
  return DSDE_OK;
}

}  // extern "C"

namespace {

// Checks the arguments dsde_step and dsde_step_static share and packs them
// (everything but the workspace).  The signal arguments live in `sg`, which
// `a` points to.
int32_t prepare_step(const void *target_logits, const void *draft_logits, int32_t dtype, int64_t V, int32_t B,
                     int64_t N, int32_t k_max, const int32_t *sl, const int32_t *cu_sl, const int32_t *draft_tokens,
                     const float *temperature, const float *u_acc, const float *u_res, int32_t pad_id,
                     int32_t *accepted, int32_t *tokens, float *kld, double *row_lse, float *draft_entropy,
                     float *hist, int32_t *head, int32_t *count, int32_t W, int32_t n_short, int32_t n_long,
                     float delta, float eps, float *mu_last, float *var_short, float *var_long, float *wvir,
                     float *sf, const float *sl_max, float sl_min, int32_t sl_hi, const int32_t *budget,
                     float *sl_hat, float *sl_cap, int32_t *sl_next, uint32_t *seq_err, void *stream,
                     dsde::VerifyArgs *a, dsde::SignalArgs *sg) {
  if (dtype != DSDE_FP32 && dtype != DSDE_BF16) return DSDE_INVALID_ARG;
  if (!verify_sizes_ok(B, N, V, k_max)) return DSDE_INVALID_ARG;
  if (!target_logits || !sl || !cu_sl || !temperature || !u_res || !accepted || !tokens || !seq_err)
    return DSDE_INVALID_ARG;
  if (N > 0 && (!draft_logits || !draft_tokens || !u_acc || !kld)) return DSDE_INVALID_ARG;
  const int32_t sst = signal_args(hist, head, count, W, n_short, n_long, delta, eps, mu_last, var_short, var_long,
                                  wvir, sf, sl_max, sl_min, sl_hi, budget, sl_hat, sl_cap, sl_next, sg);
  if (sst != DSDE_OK) return sst;
  a->target = target_logits;
  a->draft = draft_logits;
  a->dtype = dtype;
  a->V = V;
  a->B = B;
  a->N = N;
  a->k_max = k_max;
  a->sl = sl;
  a->cu_sl = cu_sl;
  a->draft_tokens = draft_tokens;
  a->temperature = temperature;
  a->u_acc = u_acc;
  a->u_res = u_res;
  a->pad_id = pad_id;
  a->accepted = accepted;
  a->tokens = tokens;
  a->kld = kld;
  a->seq_err = seq_err;
  a->row_lse = row_lse;
  a->draft_entropy = draft_entropy;
  a->workspace = nullptr;
  a->stream = static_cast<hipStream_t>(stream);
  a->prof_start = g_prof_start;
  a->prof_stop = g_prof_stop;
  a->signal = sg;
  return DSDE_OK;
}

// The workspace of dsde_step_static: one copy per device, kept until the
// process ends.  Host code must never use the array's name as an address
// (on the host it is a stand-in for the symbol); the device address of each
// device's copy comes from hipGetSymbolAddress.
__device__ __align__(256) static unsigned char scratch[DSDE_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of the copy of `scratch` on the device `stream` belongs to
// (the current device for the null stream), looked up on the first call
// for that device with that device current.
int32_t scratch_address(hipStream_t stream, void **out) {
  int dev = -1, cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return DSDE_DEVICE_ERROR;
  dev = cur;
  if (stream && hipStreamGetDevice(stream, &dev) != hipSuccess) return DSDE_DEVICE_ERROR;
  if (dev < 0 || dev >= kMaxDevices) return DSDE_DEVICE_ERROR;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    if (dev != cur && hipSetDevice(dev) != hipSuccess) return DSDE_DEVICE_ERROR;
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur && hipSetDevice(cur) != hipSuccess) return DSDE_DEVICE_ERROR;
    if (e != hipSuccess || !p) return DSDE_DEVICE_ERROR;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return DSDE_OK;
}

}  // namespace

extern "C" {

int32_t dsde_step(const void *target_logits, const void *draft_logits, int32_t dtype, int64_t V, int32_t B,
                  int64_t N, int32_t k_max, const int32_t *sl, const int32_t *cu_sl, const int32_t *draft_tokens,
                  const float *temperature, const float *u_acc, const float *u_res, int32_t pad_id,
                  int32_t *accepted, int32_t *tokens, float *kld, double *row_lse, float *draft_entropy,
                  float *hist, int32_t *head, int32_t *count, int32_t W, int32_t n_short, int32_t n_long,
                  float delta, float eps, float *mu_last, float *var_short, float *var_long, float *wvir, float *sf,
                  const float *sl_max, float sl_min, int32_t sl_hi, const int32_t *budget, float *sl_hat,
                  float *sl_cap, int32_t *sl_next, uint32_t *seq_err, void *workspace, size_t workspace_bytes,
                  void *stream) {
  dsde::VerifyArgs a;
  dsde::SignalArgs sg;
  const int32_t st = prepare_step(target_logits, draft_logits, dtype, V, B, N, k_max, sl, cu_sl, draft_tokens,
                                  temperature, u_acc, u_res, pad_id, accepted, tokens, kld, row_lse, draft_entropy,
                                  hist, head, count, W, n_short, n_long, delta, eps, mu_last, var_short, var_long,
                                  wvir, sf, sl_max, sl_min, sl_hi, budget, sl_hat, sl_cap, sl_next, seq_err, stream,
                                  &a, &sg);
  if (st != DSDE_OK) return st;
  if (!workspace) return DSDE_INVALID_ARG;
  if (workspace_bytes < dsde::workspace_layout(B, N, V, k_max).total) return DSDE_WORKSPACE_TOO_SMALL;
  if ((reinterpret_cast<uintptr_t>(workspace) & 15u) != 0) return DSDE_INVALID_ARG;
  a.workspace = workspace;
  return dsde::launch_verify(a);
}

int32_t dsde_step_static(const void *target_logits, const void *draft_logits, int32_t dtype, int64_t V, int32_t B,
                         int64_t N, int32_t k_max, const int32_t *sl, const int32_t *cu_sl,
                         const int32_t *draft_tokens, const float *temperature, const float *u_acc,
                         const float *u_res, int32_t pad_id, int32_t *accepted, int32_t *tokens, float *kld,
                         double *row_lse, float *draft_entropy, float *hist, int32_t *head, int32_t *count, int32_t W,
                         int32_t n_short, int32_t n_long, float delta, float eps, float *mu_last, float *var_short,
                         float *var_long, float *wvir, float *sf, const float *sl_max, float sl_min, int32_t sl_hi,
                         const int32_t *budget, float *sl_hat, float *sl_cap, int32_t *sl_next, uint32_t *seq_err,
                         void *stream) {
  dsde::VerifyArgs a;
  dsde::SignalArgs sg;
  const int32_t st = prepare_step(target_logits, draft_logits, dtype, V, B, N, k_max, sl, cu_sl, draft_tokens,
                                  temperature, u_acc, u_res, pad_id, accepted, tokens, kld, row_lse, draft_entropy,
                                  hist, head, count, W, n_short, n_long, delta, eps, mu_last, var_short, var_long,
                                  wvir, sf, sl_max, sl_min, sl_hi, budget, sl_hat, sl_cap, sl_next, seq_err, stream,
                                  &a, &sg);
  if (st != DSDE_OK) return st;
  // every region of the workspace a call reads is written earlier in the same
  // call, so the array needs no clearing between calls
  if (dsde::workspace_layout(B, N, V, k_max).total > size_t(DSDE_STATIC_SCRATCH_BYTES))
    return DSDE_WORKSPACE_TOO_SMALL;
  void *ws = nullptr;
  const int32_t sa = scratch_address(a.stream, &ws);
  if (sa != DSDE_OK) {
    (void)hipGetLastError();
    return sa;
  }
  a.workspace = ws;
  return dsde::launch_verify(a);
}

int32_t dsde_kld_signal(int32_t B, int64_t N, const int32_t *sl, const int32_t *cu_sl, const float *kld,
                        float *hist, int32_t *head, int32_t *count, int32_t W, int32_t n_short,
                        int32_t n_long, float delta, float eps, float *mu_last, float *var_short,
                        float *var_long, float *wvir, float *sf, uint32_t *seq_err, void *stream) {
  if (B < 1 || N < 0 || W < 1 || n_short < 1 || n_short > n_long) return DSDE_INVALID_ARG;
  if (!(delta > 0.0f && delta <= 1.0f) || !(eps > 0.0f) || !isfinite(eps)) return DSDE_INVALID_ARG;
  if (!sl || !cu_sl || !hist || !head || !count || !mu_last || !var_short || !var_long || !wvir || !sf ||
      !seq_err)
    return DSDE_INVALID_ARG;
  if (N > 0 && !kld) return DSDE_INVALID_ARG;
  return dsde::launch_kld_signal(B, N, sl, cu_sl, kld, hist, head, count, W, n_short, n_long, delta, eps, mu_last,
                                 var_short, var_long, wvir, sf, seq_err, static_cast<hipStream_t>(stream));
}

int32_t dsde_next_sl(int32_t B, const float *sf, const float *wvir, const float *sl_max, float sl_min,
                     int32_t sl_hi, const int32_t *budget, float *sl_hat, float *sl_cap, int32_t *sl_next,
                     uint32_t *seq_err, void *stream) {
  if (B < 1 || !isfinite(sl_min) || ceilf(sl_min) > float(sl_hi)) return DSDE_INVALID_ARG;
  if (!sf || !wvir || !sl_max || !sl_hat || !sl_cap || !sl_next || !seq_err) return DSDE_INVALID_ARG;
  return dsde::launch_next_sl(B, sf, wvir, sl_max, sl_min, sl_hi, budget, sl_hat, sl_cap, sl_next, seq_err, false,
                              static_cast<hipStream_t>(stream));
}

int32_t dsde_calibration_update(int32_t B, int64_t N, const int32_t *sl, const int32_t *cu_sl,
                                const int32_t *accepted, const float *kld, const uint32_t *seq_err, int32_t *a_max,
                                double *kld_sum, int64_t *kld_count, float *kld_max, void *stream) {
  if (B < 1 || N < 0) return DSDE_INVALID_ARG;
  if (!sl || !cu_sl || !accepted || !seq_err || !a_max || !kld_sum || !kld_count || !kld_max)
    return DSDE_INVALID_ARG;
  if (N > 0 && !kld) return DSDE_INVALID_ARG;
  return dsde::launch_calibration_update(B, N, sl, cu_sl, accepted, kld, seq_err, a_max, kld_sum, kld_count, kld_max,
                                         static_cast<hipStream_t>(stream));
}

int32_t dsde_calibrate_sl_max(int32_t B, const int32_t *a_max, const double *kld_sum, const int64_t *kld_count,
                              const float *kld_max, float eps, int32_t pooled, float *sl_max, void *stream) {
  if (B < 1 || !(eps >= 0.0f) || !isfinite(eps) || (pooled != 0 && pooled != 1)) return DSDE_INVALID_ARG;
  if (!a_max || !kld_sum || !kld_count || !kld_max || !sl_max) return DSDE_INVALID_ARG;
  return dsde::launch_calibrate_sl_max(B, a_max, kld_sum, kld_count, kld_max, eps, pooled != 0, sl_max,
                                       static_cast<hipStream_t>(stream));
}

int32_t dsde_set_profile_events(void *start, void *stop) {
  if ((start == nullptr) != (stop == nullptr)) return DSDE_INVALID_ARG;
  g_prof_start = static_cast<hipEvent_t>(start);
  g_prof_stop = static_cast<hipEvent_t>(stop);
  return DSDE_OK;
}

size_t dsde_shard_workspace_bytes(int32_t B, int64_t N, int64_t V_shard, int32_t k_max) {
  if (!verify_sizes_ok(B, N, V_shard, k_max)) return 0;
  if (int64_t(B) * ((V_shard + dsde::kChunk - 1) / dsde::kChunk) * 64 >= (int64_t(1) << 31)) return 0;
  return dsde::shard_layout(B, N, V_shard, k_max).total;
}

}  // extern "C"

namespace {

// The checks every shard call shares: element type, sizes, the slice inside
// the vocabulary, and the workspace.
int32_t shard_rows_ok(int32_t dtype, int64_t V_shard, int64_t v_begin, int64_t V, int32_t B, int64_t N,
                      int32_t k_max, const void *target, const void *draft, void *workspace,
                      size_t workspace_bytes) {
  if (dtype != DSDE_FP32 && dtype != DSDE_BF16) return DSDE_INVALID_ARG;
  if (dsde_shard_workspace_bytes(B, N, V_shard, k_max) == 0) return DSDE_INVALID_ARG;
  if (v_begin < 0 || V < 1 || V > DSDE_MAX_VOCAB || v_begin + V_shard > V) return DSDE_INVALID_ARG;
  if (!target || !workspace || (N > 0 && !draft)) return DSDE_INVALID_ARG;
  if (workspace_bytes < dsde::shard_layout(B, N, V_shard, k_max).total) return DSDE_WORKSPACE_TOO_SMALL;
  if ((reinterpret_cast<uintptr_t>(workspace) & 15u) != 0) return DSDE_INVALID_ARG;
  return DSDE_OK;
}

dsde::ShardRows shard_rows(const void *target, const void *draft, int32_t dtype, int64_t V_shard, int64_t v_begin,
                           int32_t B, int64_t N, int32_t k_max, void *workspace, void *stream) {
  dsde::ShardRows r;
  r.target = target;
  r.draft = draft;
  r.dtype = dtype;
  r.V_shard = V_shard;
  r.v_begin = v_begin;
  r.B = B;
  r.N = N;
  r.k_max = k_max;
  r.workspace = workspace;
  r.stream = static_cast<hipStream_t>(stream);
  return r;
}

}  // namespace

extern "C" {

int32_t dsde_shard_stats(const void *target_logits, const void *draft_logits, int32_t dtype, int64_t V_shard,
                         int64_t v_begin, int64_t V, int32_t B, int64_t N, int32_t k_max, const int32_t *sl,
                         const int32_t *cu_sl, const int32_t *draft_tokens, const float *temperature,
                         dsde_shard_partial *part, uint32_t *seq_err, void *workspace, size_t workspace_bytes,
                         void *stream) {
  const int32_t st = shard_rows_ok(dtype, V_shard, v_begin, V, B, N, k_max, target_logits, draft_logits, workspace,
                                   workspace_bytes);
  if (st != DSDE_OK) return st;
  if (!sl || !cu_sl || !temperature || !seq_err || (N > 0 && (!draft_tokens || !part))) return DSDE_INVALID_ARG;
  return dsde::launch_shard_stats(
      shard_rows(target_logits, draft_logits, dtype, V_shard, v_begin, B, N, k_max, workspace, stream), V, sl, cu_sl,
      draft_tokens, temperature, part, seq_err);
}

int32_t dsde_shard_accept(int32_t G, const dsde_shard_partial *parts, int64_t V, int32_t B, int64_t N,
                          int32_t k_max, const int32_t *sl, const int32_t *cu_sl, const int32_t *draft_tokens,
                          const float *temperature, const float *u_acc, const float *u_res, int32_t pad_id,
                          int32_t *accepted, int32_t *tokens, float *kld, double *row_lse, float *draft_entropy,
                          dsde_draw_job *jobs, uint32_t *seq_err, void *stream) {
  if (G < 1 || G > 1024 || !verify_sizes_ok(B, N, V, k_max)) return DSDE_INVALID_ARG;
  if (!sl || !cu_sl || !temperature || !u_res || !accepted || !tokens || !jobs || !seq_err) return DSDE_INVALID_ARG;
  if (N > 0 && (!parts || !draft_tokens || !u_acc || !kld)) return DSDE_INVALID_ARG;
  return dsde::launch_shard_accept(G, parts, V, B, N, k_max, sl, cu_sl, draft_tokens, temperature, u_acc, u_res,
                                   pad_id, accepted, tokens, kld, row_lse, draft_entropy, jobs, seq_err, nullptr,
                                   static_cast<hipStream_t>(stream));
}

int32_t dsde_shard_accept_step(int32_t G, const dsde_shard_partial *parts, int64_t V, int32_t B, int64_t N,
                               int32_t k_max, const int32_t *sl, const int32_t *cu_sl, const int32_t *draft_tokens,
                               const float *temperature, const float *u_acc, const float *u_res, int32_t pad_id,
                               int32_t *accepted, int32_t *tokens, float *kld, double *row_lse,
                               float *draft_entropy, dsde_draw_job *jobs, float *hist, int32_t *head, int32_t *count,
                               int32_t W, int32_t n_short, int32_t n_long, float delta, float eps, float *mu_last,
                               float *var_short, float *var_long, float *wvir, float *sf, const float *sl_max,
                               float sl_min, int32_t sl_hi, const int32_t *budget, float *sl_hat, float *sl_cap,
                               int32_t *sl_next, uint32_t *seq_err, void *stream) {
  if (G < 1 || G > 1024 || !verify_sizes_ok(B, N, V, k_max)) return DSDE_INVALID_ARG;
  if (!sl || !cu_sl || !temperature || !u_res || !accepted || !tokens || !jobs || !seq_err) return DSDE_INVALID_ARG;
  if (N > 0 && (!parts || !draft_tokens || !u_acc || !kld)) return DSDE_INVALID_ARG;
  dsde::SignalArgs sg;
  const int32_t sst = signal_args(hist, head, count, W, n_short, n_long, delta, eps, mu_last, var_short, var_long,
                                  wvir, sf, sl_max, sl_min, sl_hi, budget, sl_hat, sl_cap, sl_next, &sg);
  if (sst != DSDE_OK) return sst;
  return dsde::launch_shard_accept(G, parts, V, B, N, k_max, sl, cu_sl, draft_tokens, temperature, u_acc, u_res,
                                   pad_id, accepted, tokens, kld, row_lse, draft_entropy, jobs, seq_err, &sg,
                                   static_cast<hipStream_t>(stream));
}

int32_t dsde_shard_draw_mass(const void *target_logits, const void *draft_logits, int32_t dtype,
                             int64_t V_shard, int64_t v_begin, int32_t B, int64_t N, int32_t k_max,
                             const dsde_shard_partial *part, const dsde_draw_job *jobs, dsde_shard_mass *mass,
                             void *workspace, size_t workspace_bytes, void *stream) {
  const int32_t st = shard_rows_ok(dtype, V_shard, v_begin, v_begin + V_shard, B, N, k_max, target_logits,
                                   draft_logits, workspace, workspace_bytes);
  if (st != DSDE_OK) return st;
  if (!jobs || !mass || (N > 0 && !part)) return DSDE_INVALID_ARG;
  return dsde::launch_shard_draw_mass(
      shard_rows(target_logits, draft_logits, dtype, V_shard, v_begin, B, N, k_max, workspace, stream), part, jobs,
      mass);
}

int32_t dsde_shard_draw_pick(int32_t G, int32_t g, const dsde_shard_mass *masses, const void *target_logits,
                             const void *draft_logits, int32_t dtype, int64_t V_shard, int64_t v_begin,
                             int32_t B, int64_t N, int32_t k_max, const dsde_draw_job *jobs, int32_t pad_id,
                             int32_t *accepted, int32_t *tokens, int32_t *drawn, uint32_t *seq_err,
                             void *workspace, size_t workspace_bytes, void *stream) {
  if (G < 1 || G > 1024 || g < 0 || g >= G) return DSDE_INVALID_ARG;
  const int32_t st = shard_rows_ok(dtype, V_shard, v_begin, v_begin + V_shard, B, N, k_max, target_logits,
                                   draft_logits, workspace, workspace_bytes);
  if (st != DSDE_OK) return st;
  if (!masses || !jobs || !accepted || !tokens || !drawn || !seq_err) return DSDE_INVALID_ARG;
  return dsde::launch_shard_draw_pick(
      shard_rows(target_logits, draft_logits, dtype, V_shard, v_begin, B, N, k_max, workspace, stream), G, g, masses,
      jobs, pad_id, accepted, tokens, drawn, seq_err);
}

int32_t dsde_stream_read(const void *buf, int64_t bytes, uint32_t *out, void *stream) {
  if (!buf || !out || bytes <= 0 || bytes % 16 != 0) return DSDE_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(buf) & 15u) != 0) return DSDE_INVALID_ARG;
  return dsde::launch_stream_read(buf, bytes, out, static_cast<hipStream_t>(stream));
}

}  // extern "C"

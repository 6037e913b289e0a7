// libcrisp host layer: argument validation, workspace carving and the launch
// sequence behind the C ABI declared in include/crisp.h.  Validation touches no
// device state, so every argument error is reported before anything is queued.
// Built with CRISP_DEBUG (libcrisp_debug.so) it also checks the inputs on the device
// (non-finite values, malformed caller lists), waiting for the stream to do so.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <hip/hip_runtime.h>

#include "crisp.h"
#include "crisp_internal.h"

namespace crisp {

namespace {

constexpr int kMaxSeq = 1 << 21;  // N_b <= 32768: per-head scans and the int32 CSR offsets stay in range

thread_local char g_err[512] = "";

crisp_status fail(crisp_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

crisp_status check_shape(const crisp_shape* s, Dims* d) {
  if (!s) return fail(CRISP_EINVAL, "shape is null");
  if (s->n_q_heads < 0 || s->n_kv_heads < 1 || s->seq_len < 0)
    return fail(CRISP_EINVAL, "bad shape: n_q_heads=%d n_kv_heads=%d seq_len=%d", s->n_q_heads, s->n_kv_heads,
                s->seq_len);
  if (s->n_q_heads % s->n_kv_heads != 0)
    return fail(CRISP_EINVAL, "n_q_heads (%d) is not a multiple of n_kv_heads (%d)", s->n_q_heads, s->n_kv_heads);
  if (s->head_dim != kHeadDim) return fail(CRISP_EUNSUPPORTED, "head_dim %d unsupported (only 128)", s->head_dim);
  if (s->block != 64 && s->block != 128) return fail(CRISP_EUNSUPPORTED, "block %d unsupported (64 or 128)", s->block);
  if (s->seq_len > kMaxSeq) return fail(CRISP_EUNSUPPORTED, "seq_len %d above the supported %d", s->seq_len, kMaxSeq);
  d->hq = s->n_q_heads;
  d->hkv = s->n_kv_heads;
  d->G = s->n_q_heads / s->n_kv_heads;
  d->n = s->seq_len;
  d->B = s->block;
  d->nb = (s->seq_len + s->block - 1) / s->block;
  d->b = s->seq_len < s->block ? s->seq_len : s->block;
  d->cap = (int64_t)d->nb * (d->nb + 1) / 2;
  return CRISP_OK;
}

crisp_status check_params(const crisp_params* p, const Dims& d) {
  if (!p) return fail(CRISP_EINVAL, "params is null");
  if (!(p->alpha >= 0.f) || !isfinite(p->alpha)) return fail(CRISP_EINVAL, "alpha must be finite and >= 0");
  if (!isfinite(p->tau_proxy)) return fail(CRISP_EINVAL, "tau_proxy must be finite");
  if (!(p->gamma > 0.f && p->gamma <= 1.f)) return fail(CRISP_EINVAL, "gamma must lie in (0, 1]");
  if (p->w_sink < 0 || p->w_local < 0) return fail(CRISP_EINVAL, "w_sink and w_local must be >= 0");
  if (p->k_min_blocks < 0) return fail(CRISP_EINVAL, "k_min_blocks must be >= 0");
  if (!(p->softmax_scale >= 0.f) || !isfinite(p->softmax_scale))
    return fail(CRISP_EINVAL, "softmax_scale must be finite and >= 0");
  if (p->route_mode != CRISP_ROUTE_BY_CSTRUCT && p->route_mode != CRISP_ROUTE_BY_JSD)
    return fail(CRISP_EINVAL, "route_mode %d unknown", p->route_mode);
  if (p->vs_mode != CRISP_VS_FLOOR && p->vs_mode != CRISP_VS_GAMMA)
    return fail(CRISP_EINVAL, "vs_mode %d unknown", p->vs_mode);
  if (!isfinite(p->tau_jsd)) return fail(CRISP_EINVAL, "tau_jsd must be finite");
  if (p->floor_mode != CRISP_FLOOR_MEAN && p->floor_mode != CRISP_FLOOR_MEDIAN)
    return fail(CRISP_EINVAL, "floor_mode %d unknown", p->floor_mode);
  if (p->dense_below_len < 0) return fail(CRISP_EINVAL, "dense_below_len must be >= 0");
  (void)d;
  return CRISP_OK;
}

float scale_of(float s) { return s > 0.f ? s : 1.0f / sqrtf((float)kHeadDim); }

float route_tau(const crisp_params* p) { return p->route_mode == CRISP_ROUTE_BY_JSD ? p->tau_jsd : p->tau_proxy; }

int kmin_of(const crisp_params* p, int B) { return p->k_min_blocks > 0 ? p->k_min_blocks : (1024 + B - 1) / B; }

crisp_status check_ptr(const void* p, size_t align, const char* name) {
  if (!p) return fail(CRISP_EINVAL, "%s is null", name);
  if (!aligned(p, align)) return fail(CRISP_EINVAL, "%s is not %zu-byte aligned", name, align);
  return CRISP_OK;
}

#define CHECK(expr)                       \
  do {                                    \
    crisp_status s_ = (expr);             \
    if (s_ != CRISP_OK) return s_;        \
  } while (0)

crisp_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return CRISP_OK;
  return fail(CRISP_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool empty(const Dims& d) { return d.n == 0 || d.hq == 0; }

#ifdef CRISP_DEBUG
// Debug build: non-finite inputs and malformed caller lists become CRISP_EINVAL.
// These checks launch their own kernels and wait for the stream.
crisp_status debug_inputs(const Dims& d, const uint16_t* q, const uint16_t* k, const uint16_t* v,
                          hipStream_t st) {
  const struct {
    const uint16_t* p;
    size_t n;
    const char* name;
  } in[3] = {{q, (size_t)d.hq * d.n * kHeadDim, "q"},
             {k, (size_t)d.hkv * d.n * kHeadDim, "k"},
             {v, (size_t)d.hkv * d.n * kHeadDim, "v"}};
  for (const auto& x : in) {
    if (!x.p) continue;
    int found = 0;
    CHECK(hip_status(debug_nonfinite(x.p, x.n, st, &found), "debug input check"));
    if (found) return fail(CRISP_EINVAL, "%s holds an infinite or NaN value (debug build)", x.name);
  }
  return CRISP_OK;
}

crisp_status debug_list_check(const Dims& d, const int32_t* row_ptr, const int32_t* col_idx, int64_t cap,
                              hipStream_t st) {
  int code = 0;
  CHECK(hip_status(debug_lists(d, row_ptr, col_idx, cap, st, &code), "debug list check"));
  static const char* const what[4] = {"", "a row_ptr value outside [0, col_cap] or decreasing",
                                      "an entry outside [0, qb]", "entries not strictly increasing"};
  if (code) return fail(CRISP_EINVAL, "block lists: %s (debug build)", what[code & 3]);
  return CRISP_OK;
}
#define DEBUG_INPUTS(q, k, v, st) CHECK(debug_inputs(d, (q), (k), (v), (st)))
#define DEBUG_LISTS(rp, ci, cap, st) CHECK(debug_list_check(d, (rp), (ci), (cap), (st)))
#else
#define DEBUG_INPUTS(q, k, v, st) ((void)0)
#define DEBUG_LISTS(rp, ci, cap, st) ((void)0)
#endif

}  // namespace

WsLayout ws_layout(const Dims& d) {
  WsLayout L;
  const EstSplit sp = est_split(d);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align256(off + bytes);
    return at;
  };
  const size_t hq = d.hq, hkv = d.hkv, nb = d.nb;
  L.rowstat = take(hq * sp.splits * 128 * 4 * sizeof(float));
  L.rowfinal = take(hq * 128 * sizeof(float));
  L.parts = take(hq * nb * 128 * 4 * sizeof(float));
  L.masks = take(hq * 2 * nb);
  L.qbar = take(hq * nb * kHeadDim * sizeof(float));
  L.kbar = take(hkv * nb * kHeadDim * sizeof(float));
  L.atil = take(hq * (size_t)d.cap * sizeof(float));
  L.rhist = take(hq * 2048 * sizeof(unsigned long long));
  L.rstate = take(hq * 32);
  L.rowinfo = take(hq * nb * 4 * sizeof(int32_t));
  L.sched = take(attn_schedule_bytes(d));
  L.total = off;
  return L;
}

}  // namespace crisp

using namespace crisp;

namespace {

// Extra workspace crisp_prefill_attn carves when it keeps the scores, route and lists itself.
struct PrefillExtra {
  size_t cs, pv, ps, route, rowptr, colidx, total;
};

PrefillExtra prefill_extra(const Dims& d, size_t base) {
  PrefillExtra e;
  size_t off = base;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = (off + bytes + 255) & ~(size_t)255;
    return at;
  };
  e.cs = take((size_t)d.hq * sizeof(float));
  e.pv = take((size_t)d.hq * d.nb * sizeof(float));
  e.ps = take((size_t)d.hq * d.nb * sizeof(float));
  e.route = take((size_t)d.hq);
  e.rowptr = take((size_t)d.hq * (d.nb + 1) * sizeof(int32_t));
  e.colidx = take((size_t)d.hq * d.cap * sizeof(int32_t));
  e.total = off;
  return e;
}

// Scores are always needed by crisp_prefill_attn; the route and lists only when not supplied.
size_t prefill_scores_end(const Dims& d) {
  const PrefillExtra e = prefill_extra(d, ws_layout(d).total);
  return e.route;
}

}  // namespace

extern "C" {

void crisp_params_default(crisp_params* p) {
  if (!p) return;
  p->alpha = 1.0f;
  p->tau_proxy = 0.2f;
  p->gamma = 0.95f;
  p->w_sink = 128;
  p->w_local = 128;
  p->k_min_blocks = 0;
  p->softmax_scale = 0.0f;
  p->route_mode = CRISP_ROUTE_BY_CSTRUCT;
  p->vs_mode = CRISP_VS_FLOOR;
  p->tau_jsd = 0.1f;
  p->floor_mode = CRISP_FLOOR_MEAN;
  p->dense_below_len = 0;
}

int64_t crisp_col_capacity(const crisp_shape* shape) {
  Dims d;
  if (check_shape(shape, &d) != CRISP_OK) return -1;
  return d.cap;
}

crisp_status crisp_workspace_size(const crisp_shape* shape, size_t* bytes) {
  Dims d;
  CHECK(check_shape(shape, &d));
  if (!bytes) return fail(CRISP_EINVAL, "bytes is null");
  *bytes = prefill_scores_end(d);
  return CRISP_OK;
}

crisp_status crisp_prefill_workspace_size(const crisp_shape* shape, size_t* bytes) {
  Dims d;
  CHECK(check_shape(shape, &d));
  if (!bytes) return fail(CRISP_EINVAL, "bytes is null");
  *bytes = prefill_extra(d, ws_layout(d).total).total;
  return CRISP_OK;
}

crisp_status crisp_estimate(const crisp_shape* shape, const crisp_params* params, const crisp_bf16* q,
                            const crisp_bf16* k, float* c_struct, float* p_v, float* p_s, void* workspace,
                            size_t workspace_bytes, crisp_stream stream) {
  Dims d;
  CHECK(check_shape(shape, &d));
  CHECK(check_params(params, d));
  if (empty(d)) return CRISP_OK;
  CHECK(check_ptr(q, 16, "q"));
  CHECK(check_ptr(k, 16, "k"));
  CHECK(check_ptr(c_struct, 4, "c_struct"));
  CHECK(check_ptr(p_v, 4, "p_v"));
  CHECK(check_ptr(p_s, 4, "p_s"));
  CHECK(check_ptr(workspace, 256, "workspace"));
  if (workspace_bytes < ws_layout(d).total)
    return fail(CRISP_EINVAL, "workspace too small: %zu < %zu", workspace_bytes, ws_layout(d).total);
  DEBUG_INPUTS(q, k, nullptr, (hipStream_t)stream);
  return hip_status(launch_estimate(d, scale_of(params->softmax_scale), params->w_sink, params->w_local, q, k,
                                    c_struct, p_v, p_s, (char*)workspace, (hipStream_t)stream),
                    "crisp_estimate launch");
}

crisp_status crisp_jsd(const crisp_shape* shape, const crisp_params* params, const crisp_bf16* q,
                       const crisp_bf16* k, const float* p_v, float* jsd, void* workspace, size_t workspace_bytes,
                       crisp_stream stream) {
  Dims d;
  CHECK(check_shape(shape, &d));
  CHECK(check_params(params, d));
  if (empty(d)) return CRISP_OK;
  CHECK(check_ptr(q, 16, "q"));
  CHECK(check_ptr(k, 16, "k"));
  CHECK(check_ptr(p_v, 4, "p_v"));
  CHECK(check_ptr(jsd, 4, "jsd"));
  CHECK(check_ptr(workspace, 256, "workspace"));
  if (workspace_bytes < ws_layout(d).total)
    return fail(CRISP_EINVAL, "workspace too small: %zu < %zu", workspace_bytes, ws_layout(d).total);
  DEBUG_INPUTS(q, k, nullptr, (hipStream_t)stream);
  return hip_status(launch_jsd(d, scale_of(params->softmax_scale), q, k, p_v, jsd, (char*)workspace,
                               (hipStream_t)stream),
                    "crisp_jsd launch");
}

crisp_status crisp_route_select(const crisp_shape* shape, const crisp_params* params, const crisp_bf16* q,
                                const crisp_bf16* k, const float* c_struct, const float* p_v, const float* p_s,
                                int8_t* route, int32_t* row_ptr, int32_t* col_idx, int64_t col_cap_per_head,
                                uint8_t* dir_mask_or_null, void* workspace, size_t workspace_bytes,
                                crisp_stream stream) {
  Dims d;
  CHECK(check_shape(shape, &d));
  CHECK(check_params(params, d));
  if (empty(d)) return CRISP_OK;
  CHECK(check_ptr(q, 16, "q"));
  CHECK(check_ptr(k, 16, "k"));
  CHECK(check_ptr(c_struct, 4, "c_struct"));
  CHECK(check_ptr(p_v, 4, "p_v"));
  CHECK(check_ptr(p_s, 4, "p_s"));
  CHECK(check_ptr(route, 1, "route"));
  CHECK(check_ptr(row_ptr, 4, "row_ptr"));
  CHECK(check_ptr(col_idx, 4, "col_idx"));
  CHECK(check_ptr(workspace, 256, "workspace"));
  if (col_cap_per_head < d.cap)
    return fail(CRISP_EINVAL, "col_cap_per_head %lld < required %lld", (long long)col_cap_per_head,
                (long long)d.cap);
  if (workspace_bytes < ws_layout(d).total)
    return fail(CRISP_EINVAL, "workspace too small: %zu < %zu", workspace_bytes, ws_layout(d).total);
  DEBUG_INPUTS(q, k, nullptr, (hipStream_t)stream);
  return hip_status(launch_select(d, scale_of(params->softmax_scale), params->alpha, route_tau(params),
                                  params->gamma, kmin_of(params, d.B), params->vs_mode, params->floor_mode, false, q, k,
                                  c_struct, p_v,
                                  p_s, route, row_ptr, col_idx, col_cap_per_head, dir_mask_or_null,
                                  (char*)workspace, (hipStream_t)stream),
                    "crisp_route_select launch");
}

crisp_status crisp_sparse_workspace_size(const crisp_shape* shape, size_t* bytes) {
  Dims d;
  CHECK(check_shape(shape, &d));
  if (!bytes) return fail(CRISP_EINVAL, "bytes is null");
  *bytes = align256(attn_schedule_bytes(d));
  return CRISP_OK;
}

crisp_status crisp_sparse_attn(const crisp_shape* shape, float softmax_scale, const crisp_bf16* q,
                               const crisp_bf16* k, const crisp_bf16* v, const int32_t* row_ptr,
                               const int32_t* col_idx, int64_t col_cap_per_head, crisp_bf16* o,
                               void* workspace_or_null, size_t workspace_bytes, crisp_stream stream) {
  Dims d;
  CHECK(check_shape(shape, &d));
  if (!(softmax_scale >= 0.f) || !isfinite(softmax_scale))
    return fail(CRISP_EINVAL, "softmax_scale must be finite and >= 0");
  if (empty(d)) return CRISP_OK;
  CHECK(check_ptr(q, 16, "q"));
  CHECK(check_ptr(k, 16, "k"));
  CHECK(check_ptr(v, 16, "v"));
  CHECK(check_ptr(o, 16, "o"));
  CHECK(check_ptr(row_ptr, 4, "row_ptr"));
  CHECK(check_ptr(col_idx, 4, "col_idx"));
  if (col_cap_per_head < 0) return fail(CRISP_EINVAL, "col_cap_per_head must be >= 0");
  if (workspace_or_null) {
    CHECK(check_ptr(workspace_or_null, 256, "workspace"));
    if (workspace_bytes < attn_schedule_bytes(d))
      return fail(CRISP_EINVAL, "workspace too small: %zu < %zu", workspace_bytes, attn_schedule_bytes(d));
  }
  DEBUG_INPUTS(q, k, v, (hipStream_t)stream);
  DEBUG_LISTS(row_ptr, col_idx, col_cap_per_head, (hipStream_t)stream);
  return hip_status(launch_attn(d, scale_of(softmax_scale), q, k, v, row_ptr, col_idx, col_cap_per_head, false, o,
                                workspace_or_null, (hipStream_t)stream),
                    "crisp_sparse_attn launch");
}

crisp_status crisp_sparse_attn_noalloc(const crisp_shape* shape, float softmax_scale, const crisp_bf16* q,
                                       const crisp_bf16* k, const crisp_bf16* v, const int32_t* row_ptr,
                                       const int32_t* col_idx, int64_t col_cap_per_head, crisp_bf16* o,
                                       crisp_stream stream) {
  Dims d;
  CHECK(check_shape(shape, &d));
  if (!(softmax_scale >= 0.f) || !isfinite(softmax_scale))
    return fail(CRISP_EINVAL, "softmax_scale must be finite and >= 0");
  if (empty(d)) return CRISP_OK;
  CHECK(check_ptr(q, 16, "q"));
  CHECK(check_ptr(k, 16, "k"));
  CHECK(check_ptr(v, 16, "v"));
  CHECK(check_ptr(o, 16, "o"));
  CHECK(check_ptr(row_ptr, 4, "row_ptr"));
  CHECK(check_ptr(col_idx, 4, "col_idx"));
  if (col_cap_per_head < 0) return fail(CRISP_EINVAL, "col_cap_per_head must be >= 0");
  const size_t need = attn_schedule_bytes(d, kStaticSlots);
  if (need > kStaticSchedBytes)
    return fail(CRISP_EINVAL, "layer needs %zu bytes of schedule area (%lld query blocks over all heads); the "
                "static area holds %zu", need, (long long)d.hq * d.nb, kStaticSchedBytes);
  void* area = nullptr;
  CHECK(hip_status(static_schedule_area(&area), "crisp_sparse_attn_noalloc static area"));
  DEBUG_INPUTS(q, k, v, (hipStream_t)stream);
  DEBUG_LISTS(row_ptr, col_idx, col_cap_per_head, (hipStream_t)stream);
  return hip_status(launch_attn(d, scale_of(softmax_scale), q, k, v, row_ptr, col_idx, col_cap_per_head, false, o,
                                area, (hipStream_t)stream, kStaticSlots),
                    "crisp_sparse_attn_noalloc launch");
}

crisp_status crisp_dense_attn(const crisp_shape* shape, float softmax_scale, const crisp_bf16* q,
                              const crisp_bf16* k, const crisp_bf16* v, crisp_bf16* o, crisp_stream stream) {
  Dims d;
  CHECK(check_shape(shape, &d));
  if (!(softmax_scale >= 0.f) || !isfinite(softmax_scale))
    return fail(CRISP_EINVAL, "softmax_scale must be finite and >= 0");
  if (empty(d)) return CRISP_OK;
  CHECK(check_ptr(q, 16, "q"));
  CHECK(check_ptr(k, 16, "k"));
  CHECK(check_ptr(v, 16, "v"));
  CHECK(check_ptr(o, 16, "o"));
  DEBUG_INPUTS(q, k, v, (hipStream_t)stream);
  return hip_status(launch_attn(d, scale_of(softmax_scale), q, k, v, nullptr, nullptr, 0, true, o, nullptr,
                                (hipStream_t)stream),
                    "crisp_dense_attn launch");
}

crisp_status crisp_prefill_attn(const crisp_shape* shape, const crisp_params* params, const crisp_bf16* q,
                                const crisp_bf16* k, const crisp_bf16* v, crisp_bf16* o, int8_t* route_or_null,
                                int32_t* row_ptr_or_null, int32_t* col_idx_or_null, void* workspace,
                                size_t workspace_bytes, crisp_stream stream) {
  Dims d;
  CHECK(check_shape(shape, &d));
  CHECK(check_params(params, d));
  const int given = (route_or_null != nullptr) + (row_ptr_or_null != nullptr) + (col_idx_or_null != nullptr);
  if (given != 0 && given != 3)
    return fail(CRISP_EINVAL, "route, row_ptr and col_idx must be all given or all null");
  if (empty(d)) return CRISP_OK;
  CHECK(check_ptr(q, 16, "q"));
  CHECK(check_ptr(k, 16, "k"));
  CHECK(check_ptr(v, 16, "v"));
  CHECK(check_ptr(o, 16, "o"));
  CHECK(check_ptr(workspace, 256, "workspace"));
  if (given) {
    CHECK(check_ptr(row_ptr_or_null, 4, "row_ptr"));
    CHECK(check_ptr(col_idx_or_null, 4, "col_idx"));
  }
  const WsLayout L = ws_layout(d);
  const PrefillExtra e = prefill_extra(d, L.total);
  const size_t need = given ? e.route : e.total;
  if (workspace_bytes < need) return fail(CRISP_EINVAL, "workspace too small: %zu < %zu", workspace_bytes, need);
  DEBUG_INPUTS(q, k, v, (hipStream_t)stream);
  char* ws = (char*)workspace;
  if (d.n < params->dense_below_len) {  // context-length gate: the layer is dense attention
    if (given)
      CHECK(hip_status(launch_dense_lists(d, route_or_null, row_ptr_or_null, col_idx_or_null, d.cap,
                                          (hipStream_t)stream),
                       "crisp_prefill_attn dense lists launch"));
    return hip_status(launch_attn(d, scale_of(params->softmax_scale), q, k, v, nullptr, nullptr, 0, true, o, nullptr,
                                  (hipStream_t)stream),
                      "crisp_prefill_attn dense attention launch");
  }
  float* cs = (float*)(ws + e.cs);
  float* pv = (float*)(ws + e.pv);
  float* ps = (float*)(ws + e.ps);
  int8_t* route = given ? route_or_null : (int8_t*)(ws + e.route);
  int32_t* rp = given ? row_ptr_or_null : (int32_t*)(ws + e.rowptr);
  int32_t* ci = given ? col_idx_or_null : (int32_t*)(ws + e.colidx);
  const float scale = scale_of(params->softmax_scale);
  hipStream_t st = (hipStream_t)stream;
  const bool by_jsd = params->route_mode == CRISP_ROUTE_BY_JSD;
  // Short layers: the selection forms p_v and p_s itself from the estimator's sums (one
  // launch fewer); the pattern search reads p_v, so it keeps the estimator's own step.
  const bool fold = !by_jsd && d.nb <= kSmallSelectBlocks;
  CHECK(hip_status(launch_estimate(d, scale, params->w_sink, params->w_local, q, k, cs, pv, ps, ws, st, fold),
                   "crisp_prefill_attn estimate launch"));
  if (by_jsd)  // the route score slot then holds D_JS instead of C_struct
    CHECK(hip_status(launch_jsd(d, scale, q, k, pv, cs, ws, st), "crisp_prefill_attn pattern search launch"));
  CHECK(hip_status(launch_select(d, scale, params->alpha, route_tau(params), params->gamma, kmin_of(params, d.B),
                                 params->vs_mode, params->floor_mode, by_jsd, q, k, cs, pv, ps, route, rp, ci,
                                 d.cap, nullptr, ws, st, fold),
                   "crisp_prefill_attn select launch"));
  return hip_status(launch_attn(d, scale, q, k, v, rp, ci, d.cap, false, o, ws + L.sched, st),
                    "crisp_prefill_attn attention launch");
}

const char* crisp_status_string(crisp_status s) {
  switch (s) {
    case CRISP_OK: return "CRISP_OK";
    case CRISP_EINVAL: return "CRISP_EINVAL";
    case CRISP_EUNSUPPORTED: return "CRISP_EUNSUPPORTED";
    case CRISP_EHIP: return "CRISP_EHIP";
  }
  return "CRISP_UNKNOWN";
}

const char* crisp_last_error(void) { return g_err; }

}  // extern "C"

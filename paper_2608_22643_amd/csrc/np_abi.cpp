// np_abi.cpp -- host side of the C ABI: argument validation, status text,
// workspace sizing and dispatch to the kernel launchers.  Validation runs
// before anything is enqueued.
#include <algorithm>
#include <cmath>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <string>

#include <mutex>
#include <unordered_set>

#include "np_internal.hpp"

namespace np {

namespace {
std::mutex g_incomplete_mu;
std::unordered_set<uintptr_t> g_incomplete;  // resident buffers (base pointers)
}  // namespace

void mark_resident_incomplete(const void* resident) {
  std::lock_guard<std::mutex> g(g_incomplete_mu);
  g_incomplete.insert((uintptr_t)resident);
}

np_status check_resident(const char* fn, const void* resident) {
  std::lock_guard<std::mutex> g(g_incomplete_mu);
  if (g_incomplete.count((uintptr_t)resident))
    return fail(NP_ERR_STATE,
                "%s: a staging into this resident buffer failed part-way; np_state_reset first", fn);
  return NP_OK;
}

void clear_incomplete_resident(const void* resident) {
  std::lock_guard<std::mutex> g(g_incomplete_mu);
  g_incomplete.erase((uintptr_t)resident);
}

thread_local std::string g_last_error;

np_status fail(np_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

np_status hip_fail(hipError_t e, const char* what) {
  return fail(NP_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return p && ((uintptr_t)p & 15u) == 0; }

np_status check_shape(const np_shape* s) {
  if (!s) return fail(NP_ERR_INVALID_ARG, "shape is NULL");
  if (s->wdtype < NP_F32 || s->wdtype > NP_BF16)
    return fail(NP_ERR_INVALID_ARG, "wdtype %d is not an np_dtype", s->wdtype);
  if (s->adtype != s->wdtype)
    return fail(NP_ERR_INVALID_ARG, "adtype %d must equal wdtype %d", s->adtype, s->wdtype);
  if (s->act != NP_ACT_RELU && s->act != NP_ACT_SWIGLU)
    return fail(NP_ERR_INVALID_ARG, "act %d is not an np_act", s->act);
  const int V = vec_elems(s->wdtype);
  if (s->layers < 1) return fail(NP_ERR_INVALID_ARG, "layers %d < 1", s->layers);
  if (s->d_model < V || s->d_model % V)
    return fail(NP_ERR_INVALID_ARG, "d_model %d is not a positive multiple of %d", s->d_model, V);
  if (s->d_model > (s->wdtype == NP_F32 ? 8192 : 16384))
    return fail(NP_ERR_INVALID_ARG, "d_model %d above the supported maximum", s->d_model);
  if (s->rank < V || s->rank % V)
    return fail(NP_ERR_INVALID_ARG, "rank %d is not a positive multiple of %d", s->rank, V);
  if (s->rank > 128 * V)
    return fail(NP_ERR_INVALID_ARG, "rank %d above the supported maximum %d", s->rank, 128 * V);
  if (s->d_ffn < 1 || s->d_ffn > 65535)
    return fail(NP_ERR_INVALID_ARG, "d_ffn %d outside [1, 65535]", s->d_ffn);
  if (s->k < 1 || s->k > s->d_ffn || s->k > 8192)
    return fail(NP_ERR_INVALID_ARG, "k %d outside [1, min(d_ffn, 8192)]", s->k);
  if (s->capacity < 1 || s->capacity > s->d_ffn)
    return fail(NP_ERR_INVALID_ARG, "capacity %d outside [1, d_ffn]", s->capacity);
  if ((size_t)s->capacity * 3 * s->d_model * dtype_size(s->wdtype) >= ((size_t)1 << 31))
    return fail(NP_ERR_INVALID_ARG, "a layer's resident buffer must stay below 2 GiB");
  if (s->k > s->capacity)
    return fail(NP_ERR_CAPACITY, "k %d exceeds the resident capacity %d", s->k, s->capacity);
  return NP_OK;
}

}  // namespace np

using namespace np;

extern "C" {

const char* np_status_str(int32_t st) {
  switch (st) {
    case NP_OK: return "NP_OK";
    case NP_ERR_INVALID_ARG: return "NP_ERR_INVALID_ARG";
    case NP_ERR_CAPACITY: return "NP_ERR_CAPACITY";
    case NP_ERR_HIP: return "NP_ERR_HIP";
    case NP_ERR_UNSUPPORTED: return "NP_ERR_UNSUPPORTED";
    case NP_ERR_STATE: return "NP_ERR_STATE";
    case NP_ERR_IO: return "NP_ERR_IO";
    default: return "NP_ERR_UNKNOWN";
  }
}

const char* np_last_error(void) { return g_last_error.c_str(); }

np_status np_shape_check(const np_shape* s) {
  np_status st = check_shape(s);
  if (st == NP_OK) g_last_error.clear();
  return st;
}

np_status np_workspace_size(const np_shape* s, size_t* bytes, size_t* pinned_host_bytes) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (!bytes) return fail(NP_ERR_INVALID_ARG, "dev_ws_bytes is NULL");
  *bytes = ws_total(*s);
  if (pinned_host_bytes) {
    // the plan copy (counts, in_ids, in_slots), then a staging area of four
    // pieces of 16 MiB (at least one record and its row index each)
    const size_t rec = (size_t)3 * s->d_model * dtype_size(s->wdtype);
    const size_t plan = ((size_t)s->layers * (4 + 2 * (size_t)s->k) * 4 + 4095) & ~(size_t)4095;
    const size_t piece = (std::max((size_t)16 << 20, rec + 4) + 4095) & ~(size_t)4095;
    *pinned_host_bytes = plan + 4 * piece;
  }
  return NP_OK;
}

np_status np_state_reset(const np_shape* s, const np_state* state, const void* resident,
                         void* ws, hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (!state || !aligned16(state->slot_of) || !aligned16(state->neuron_of) ||
      !aligned16(state->last_used))
    return fail(NP_ERR_INVALID_ARG, "state arrays must be non-NULL and 16-byte aligned");
  if (!aligned16(ws)) return fail(NP_ERR_INVALID_ARG, "dev_ws must be non-NULL and 16-byte aligned");
  hipError_t e = launch_fill_state(*s, *state, ws, stream);
  if (e != hipSuccess) return hip_fail(e, "np_state_reset launch");
  if (resident) clear_incomplete_resident(resident);  // a cold start: no resident row is assumed
  return NP_OK;
}

np_status np_predict(const np_shape* s, const void* h, const void* A, const void* B,
                     float* scores, void* ws, hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (!aligned16(h) || !aligned16(A) || !aligned16(B) || !aligned16(scores) || !aligned16(ws))
    return fail(NP_ERR_INVALID_ARG, "np_predict: pointers must be non-NULL and 16-byte aligned");
  hipError_t e = launch_predict(*s, h, A, B, scores, ws, stream);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_predict launch");
}

np_status np_select(const np_shape* s, const float* scores, uint32_t* mask, int32_t* ids,
                    void* ws, hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (!aligned16(scores) || !aligned16(mask) || !aligned16(ids) || !aligned16(ws))
    return fail(NP_ERR_INVALID_ARG, "np_select: pointers must be non-NULL and 16-byte aligned");
  hipError_t e = launch_select(*s, scores, mask, ids, ws, stream);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_select launch");
}

static np_status delta_common(const char* fn, const np_shape* s, int32_t token,
                              const int32_t* ids, const int32_t* counts, const np_state* state,
                              const np_delta_out* out, void* ws, hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (token < NP_TOKEN_AUTO) return fail(NP_ERR_INVALID_ARG, "token %d < 0", token);
  if (!aligned16(ids) || !state || !aligned16(state->slot_of) || !aligned16(state->neuron_of) ||
      !aligned16(state->last_used) || !aligned16(ws))
    return fail(NP_ERR_INVALID_ARG, "%s: pointers must be non-NULL and 16-byte aligned", fn);
  if (!out || !aligned16(out->in_ids) || !aligned16(out->in_slots) || !aligned16(out->ev_ids) ||
      !aligned16(out->ev_slots) || !aligned16(out->hit_ids) || !aligned16(out->active_slots) ||
      !aligned16(out->counts))
    return fail(NP_ERR_INVALID_ARG, "%s: output lists must be non-NULL and 16-byte aligned", fn);
  hipError_t e = launch_delta(*s, token, ids, *state, *out, ws, stream, counts);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_delta launch");
}

np_status np_delta(const np_shape* s, int32_t token, const int32_t* ids, const np_state* state,
                   const np_delta_out* out, void* ws, hipStream_t stream) {
  return delta_common("np_delta", s, token, ids, nullptr, state, out, ws, stream);
}

np_status np_select_delta(const np_shape* s, int32_t token, const float* scores, uint32_t* mask,
                          int32_t* ids, const np_state* state, const np_delta_out* out, void* ws,
                          hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (token < NP_TOKEN_AUTO) return fail(NP_ERR_INVALID_ARG, "token %d < 0", token);
  if (!aligned16(scores) || !aligned16(mask) || !aligned16(ids) || !aligned16(ws) || !state ||
      !aligned16(state->slot_of) || !aligned16(state->neuron_of) ||
      !aligned16(state->last_used))
    return fail(NP_ERR_INVALID_ARG,
                "np_select_delta: pointers must be non-NULL and 16-byte aligned");
  if (!out || !aligned16(out->in_ids) || !aligned16(out->in_slots) || !aligned16(out->ev_ids) ||
      !aligned16(out->ev_slots) || !aligned16(out->hit_ids) || !aligned16(out->active_slots) ||
      !aligned16(out->counts))
    return fail(NP_ERR_INVALID_ARG,
                "np_select_delta: output lists must be non-NULL and 16-byte aligned");
  hipError_t e = launch_select_delta(*s, token, scores, mask, ids, *state, *out, ws, stream);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_select_delta launch");
}

np_status np_delta_n(const np_shape* s, int32_t token, const int32_t* ids, const int32_t* counts,
                     const np_state* state, const np_delta_out* out, void* ws,
                     hipStream_t stream) {
  if (!aligned16(counts))
    return fail(NP_ERR_INVALID_ARG, "np_delta_n: active_counts must be non-NULL and aligned");
  return delta_common("np_delta_n", s, token, ids, counts, state, out, ws, stream);
}

np_status np_centroid_select(const np_shape* s, const np_centroid_model* m, const void* feat,
                             float* logits, int32_t* cids, uint32_t* mask, int32_t* active_ids,
                             int32_t* counts, void* ws, hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (!m) return fail(NP_ERR_INVALID_ARG, "np_centroid_select: model is NULL");
  if (m->n_centroids < 1 || m->n_centroids > 4096)
    return fail(NP_ERR_INVALID_ARG, "n_centroids %d outside [1, 4096]", m->n_centroids);
  const int V = vec_elems(s->wdtype);
  const int dmax = s->wdtype == NP_F32 ? 8192 : 16384;
  if (m->feat_dim < V || m->feat_dim % V || m->feat_dim > dmax)
    return fail(NP_ERR_INVALID_ARG, "feat_dim %d: a multiple of %d in [%d, %d]", m->feat_dim, V,
                V, dmax);
  if ((size_t)2 * s->layers * m->n_centroids > (size_t)1 << 30)
    return fail(NP_ERR_INVALID_ARG, "2 * layers * n_centroids too large");
  if (!aligned16(m->heads) || !aligned16(m->bank) || !aligned16(feat) || !aligned16(logits) ||
      !aligned16(cids) || !aligned16(mask) || !aligned16(active_ids) || !aligned16(counts) ||
      !aligned16(ws))
    return fail(NP_ERR_INVALID_ARG,
                "np_centroid_select: pointers must be non-NULL and 16-byte aligned");
  hipError_t e = launch_centroid_logits(*s, *m, feat, logits, stream);
  if (e != hipSuccess) return hip_fail(e, "np_centroid_select heads launch");
  e = launch_centroid_active(*s, *m, logits, cids, mask, active_ids, counts, ws, stream);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_centroid_select launch");
}

np_status np_stage_gather(const np_shape* s, const np_delta_out* out, int32_t lb, int32_t le,
                          const void* storage, void* resident, void* ws, hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (lb < 0 || le > s->layers || lb > le)
    return fail(NP_ERR_INVALID_ARG, "layer range [%d, %d) outside [0, %d)", lb, le, s->layers);
  if (!out || !aligned16(out->counts) || !aligned16(out->in_ids) || !aligned16(out->in_slots))
    return fail(NP_ERR_INVALID_ARG, "np_stage_gather: plan lists must be non-NULL and aligned");
  if (!aligned16(storage) || !aligned16(resident) || !aligned16(ws))
    return fail(NP_ERR_INVALID_ARG, "np_stage_gather: pointers must be non-NULL and aligned");
  if ((st = check_resident("np_stage_gather", resident)) != NP_OK) return st;
  if (lb == le) return NP_OK;
  // a pinned host storage tier is read through its device mapping
  hipPointerAttribute_t attr;
  if (hipPointerGetAttributes(&attr, storage) != hipSuccess) {
    (void)hipGetLastError();
    return fail(NP_ERR_INVALID_ARG, "np_stage_gather: storage is not device-accessible memory");
  }
  if (attr.type == hipMemoryTypeHost) {
    if (!attr.devicePointer)
      return fail(NP_ERR_INVALID_ARG, "np_stage_gather: host storage is not mapped to the device");
    storage = attr.devicePointer;
  }
  hipError_t e = launch_stage_gather(*s, *out, lb, le, storage, resident, ws, stream,
                                     attr.type == hipMemoryTypeHost);
  if (e == hipSuccess) return NP_OK;
  mark_resident_incomplete(resident);
  return hip_fail(e, "np_stage_gather launch");
}

np_status np_sparse_mlp(const np_shape* s, int32_t layer, const void* x, const void* resident,
                        const int32_t* slots, int32_t n_active, void* y, void* ws,
                        hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (layer < 0 || layer >= s->layers)
    return fail(NP_ERR_INVALID_ARG, "layer %d outside [0, %d)", layer, s->layers);
  if (n_active < 0 || n_active > s->capacity)
    return fail(NP_ERR_INVALID_ARG, "n_active %d outside [0, capacity]", n_active);
  if (!aligned16(x) || !aligned16(resident) || !aligned16(y) || !aligned16(ws) ||
      (n_active > 0 && !slots))
    return fail(NP_ERR_INVALID_ARG, "np_sparse_mlp: pointers must be non-NULL and aligned");
  if ((st = check_resident("np_sparse_mlp", resident)) != NP_OK) return st;
  hipError_t e = launch_sparse_mlp(*s, layer, x, resident, slots, n_active, y, ws, stream);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_sparse_mlp launch");
}

np_status np_sparse_mlp_noalloc(const np_shape* s, int32_t layer, const void* x,
                                const void* resident, const int32_t* slots, int32_t n_active,
                                void* y, int32_t* dev_error, hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (layer < 0 || layer >= s->layers)
    return fail(NP_ERR_INVALID_ARG, "layer %d outside [0, %d)", layer, s->layers);
  if (n_active < 0 || n_active > s->capacity)
    return fail(NP_ERR_INVALID_ARG, "n_active %d outside [0, capacity]", n_active);
  if (s->d_model > NOALLOC_MAX_D)
    return fail(NP_ERR_CAPACITY,
                "np_sparse_mlp_noalloc: d_model %d above the scratch maximum %d (use "
                "np_sparse_mlp with a workspace)", s->d_model, NOALLOC_MAX_D);
  if (!aligned16(x) || !aligned16(resident) || !aligned16(y) || (n_active > 0 && !slots) ||
      !dev_error || ((uintptr_t)dev_error & 3))
    return fail(NP_ERR_INVALID_ARG,
                "np_sparse_mlp_noalloc: pointers must be non-NULL and aligned");
  if ((st = check_resident("np_sparse_mlp_noalloc", resident)) != NP_OK) return st;
  hipError_t e =
      launch_sparse_mlp_noalloc(*s, layer, x, resident, slots, n_active, y, dev_error, stream);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_sparse_mlp_noalloc launch");
}

np_status np_sparse_mlp_ids(const np_shape* s, int32_t layer, const void* x, const void* resident,
                            const int32_t* active_ids, const int32_t* slot_of, int32_t n_active,
                            void* y, void* ws, hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (layer < 0 || layer >= s->layers)
    return fail(NP_ERR_INVALID_ARG, "layer %d outside [0, %d)", layer, s->layers);
  if (n_active < 0 || n_active > s->capacity)
    return fail(NP_ERR_INVALID_ARG, "n_active %d outside [0, capacity]", n_active);
  if (!aligned16(x) || !aligned16(resident) || !aligned16(y) || !aligned16(ws) ||
      (n_active > 0 && (!active_ids || !slot_of)) || ((uintptr_t)active_ids & 3) ||
      ((uintptr_t)slot_of & 3))
    return fail(NP_ERR_INVALID_ARG, "np_sparse_mlp_ids: pointers must be non-NULL and aligned");
  if ((st = check_resident("np_sparse_mlp_ids", resident)) != NP_OK) return st;
  hipError_t e = launch_sparse_mlp(*s, layer, x, resident, nullptr, n_active, y, ws, stream,
                                   nullptr, nullptr, active_ids, slot_of);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_sparse_mlp_ids launch");
}

np_status np_dense_mlp(const np_shape* s, const void* weights, const void* x, void* y, void* ws,
                       hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if ((size_t)s->d_ffn * 3 * s->d_model * dtype_size(s->wdtype) >= ((size_t)1 << 31))
    return fail(NP_ERR_UNSUPPORTED, "np_dense_mlp: a layer of %d records of %d elements >= 2 GiB",
                s->d_ffn, 3 * s->d_model);
  if (!aligned16(weights) || !aligned16(x) || !aligned16(y) || !aligned16(ws))
    return fail(NP_ERR_INVALID_ARG, "np_dense_mlp: pointers must be non-NULL and aligned");
  hipError_t e = launch_dense_mlp(*s, weights, x, y, ws, stream);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_dense_mlp launch");
}

np_status np_sparse_mlp_n(const np_shape* s, int32_t layer, const void* x, const void* resident,
                          const int32_t* slots, const int32_t* counts, void* y, void* ws,
                          hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (layer < 0 || layer >= s->layers)
    return fail(NP_ERR_INVALID_ARG, "layer %d outside [0, %d)", layer, s->layers);
  // slots and counts are read as single int32 values: 4-byte alignment
  if (!aligned16(x) || !aligned16(resident) || !aligned16(y) || !aligned16(ws) || !slots ||
      !counts || ((uintptr_t)slots & 3) || ((uintptr_t)counts & 3))
    return fail(NP_ERR_INVALID_ARG, "np_sparse_mlp_n: pointers must be non-NULL and aligned");
  if ((st = check_resident("np_sparse_mlp_n", resident)) != NP_OK) return st;
  hipError_t e = launch_sparse_mlp(*s, layer, x, resident, slots, s->k, y, ws, stream, counts);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_sparse_mlp_n launch");
}

np_status np_sparse_mlp_t(const np_shape* s, int32_t layer, const void* x, const void* resident,
                          const int32_t* slots, int32_t n_active, const int32_t* counts,
                          const float* thr, void* y, void* ws, hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (layer < 0 || layer >= s->layers)
    return fail(NP_ERR_INVALID_ARG, "layer %d outside [0, %d)", layer, s->layers);
  if (n_active < 0 || n_active > s->capacity)
    return fail(NP_ERR_INVALID_ARG, "n_active %d outside [0, capacity]", n_active);
  if (!aligned16(x) || !aligned16(resident) || !aligned16(y) || !aligned16(ws) ||
      (n_active > 0 && !slots) || ((uintptr_t)slots & 3) || ((uintptr_t)counts & 3) ||
      ((uintptr_t)thr & 3))
    return fail(NP_ERR_INVALID_ARG, "np_sparse_mlp_t: pointers must be non-NULL and aligned");
  if ((st = check_resident("np_sparse_mlp_t", resident)) != NP_OK) return st;
  hipError_t e = launch_sparse_mlp(*s, layer, x, resident, slots, n_active, y, ws, stream, counts,
                                   thr);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_sparse_mlp_t launch");
}

np_status np_act_batch(const np_shape* s, const void* weights, const void* x, int32_t n,
                       float* acts, void* ws, hipStream_t stream) {
  (void)ws;
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (n < 1 || n > 65536) return fail(NP_ERR_INVALID_ARG, "n %d outside [1, 65536]", n);
  const size_t w = dtype_size(s->wdtype);
  if ((size_t)s->d_ffn * 3 * s->d_model * w >= ((size_t)1 << 31) ||
      (size_t)n * s->d_model * w >= ((size_t)1 << 31))
    return fail(NP_ERR_UNSUPPORTED, "np_act_batch: weights or tokens of 2 GiB or more");
  if (!aligned16(weights) || !aligned16(x) || !aligned16(acts))
    return fail(NP_ERR_INVALID_ARG, "np_act_batch: pointers must be non-NULL and aligned");
  hipError_t e = launch_act_batch(*s, weights, x, n, acts, stream);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_act_batch launch");
}

np_status np_percentile(const float* values, int32_t rows, int64_t n, double alpha, float* out,
                        void* ws, size_t ws_bytes, hipStream_t stream) {
  if (rows < 1 || rows > 65535) return fail(NP_ERR_INVALID_ARG, "rows %d outside [1, 65535]", rows);
  if (n < 1 || n >= ((int64_t)1 << 31))
    return fail(NP_ERR_INVALID_ARG, "n %lld outside [1, 2^31)", (long long)n);
  if (!(alpha >= 0.0 && alpha <= 100.0))
    return fail(NP_ERR_INVALID_ARG, "alpha %g outside [0, 100]", alpha);
  if (!aligned16(values) || ((uintptr_t)out & 3) || !out || !aligned16(ws))
    return fail(NP_ERR_INVALID_ARG, "np_percentile: pointers must be non-NULL and aligned");
  if (ws_bytes < 64)
    return fail(NP_ERR_INVALID_ARG, "np_percentile: dev_ws of %zu bytes holds no error word",
                ws_bytes);
  // nearest rank: the m-th smallest magnitude, m = ceil(alpha n / 100) in [1, n]
  double md = std::ceil(alpha * (double)n / 100.0);
  int64_t m = md < 1.0 ? 1 : (md > (double)n ? n : (int64_t)md);
  hipError_t e = launch_percentile(values, rows, n, m, out, ws, ws_bytes, stream);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_percentile launch");
}

np_status np_threshold_active(const np_shape* s, const float* acts, int32_t rows,
                              const float* thr, uint32_t* mask, int32_t* ids, int32_t* counts,
                              void* ws, hipStream_t stream) {
  np_status st = check_shape(s);
  if (st != NP_OK) return st;
  if (rows < 1 || rows > 65535) return fail(NP_ERR_INVALID_ARG, "rows %d outside [1, 65535]", rows);
  if (!aligned16(acts) || !aligned16(mask) || !aligned16(ids) || !aligned16(ws) || !thr ||
      !counts || ((uintptr_t)thr & 3) || ((uintptr_t)counts & 3))
    return fail(NP_ERR_INVALID_ARG, "np_threshold_active: pointers must be non-NULL and aligned");
  hipError_t e = launch_threshold_active(*s, acts, rows, thr, mask, ids, counts, ws, stream);
  return e == hipSuccess ? NP_OK : hip_fail(e, "np_threshold_active launch");
}

np_status np_device_error(const void* ws, hipStream_t stream, int32_t* code) {
  if (!aligned16(ws) || !code) return fail(NP_ERR_INVALID_ARG, "np_device_error: bad pointer");
  hipError_t e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail(e, "np_device_error synchronize");
  e = hipMemcpy(code, (const char*)ws + WS_ERR, sizeof(int32_t), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "np_device_error copy");
  return NP_OK;
}

}  // extern "C"

// C ABI of libcarryover: argument validation, workspace planning and launches.
// Every entry point validates what the host can see, then only enqueues work on
// the caller's stream.
#include <math.h>
#include <string.h>

#include <mutex>

#include "co_kernels.h"

// Scratch of carryover_round_noalloc: the round's workspace for callers that
// cannot allocate.  Every device the library runs on holds its own copy until
// the process ends; host code reaches it only through the per-device address
// from hipGetSymbolAddress (the name itself is not a device address here).
constexpr size_t kScratchBytes = size_t{128} << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

using namespace co;

namespace co {

// Launch-shape overrides (carryover_set_tuning); -1 = automatic, for every knob.
struct Tuning {
  int64_t v[CO_TUNE_COUNT];
  Tuning() {
    for (int64_t& x : v) x = -1;
  }
};
static Tuning g_tuning;

int64_t tuning(int knob) { return knob >= 0 && knob < CO_TUNE_COUNT ? g_tuning.v[knob] : -1; }

}  // namespace co

namespace {

constexpr int kMaxDevices = 64;
int g_num_cus[kMaxDevices];   // per-device compute-unit count, filled on first use

std::mutex g_scratch_mutex;
void* g_scratch_addr[kMaxDevices];   // device address of `scratch`, per device

// Device address of the current device's copy of `scratch`, looked up once
// per device with that device current.
co_status scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return CO_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return CO_ERR_HIP;
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return CO_OK;
}

int num_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
  if (g_num_cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    g_num_cus[dev] = n;
  }
  return g_num_cus[dev];
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

co_status check_dims(const co_dims* d) {
  if (!d) return CO_ERR_INVALID_ARG;
  if (d->num_seqs < 0 || d->block < 1 || d->num_layers < 1 || d->num_kv_heads < 1 ||
      d->num_q_heads < 1 || d->max_pages_per_seq < 1 || d->num_pages < 1 || d->feat_dim < 1 ||
      d->model_dim < 1)
    return CO_ERR_INVALID_ARG;
  if (!(d->rope_theta > 0.f)) return CO_ERR_INVALID_ARG;
  if (d->page_size != kPage) return CO_ERR_UNSUPPORTED;
  if (d->dtype != CO_DTYPE_F32 && d->dtype != CO_DTYPE_BF16) return CO_ERR_UNSUPPORTED;
  if (d->head_dim != 64 && d->head_dim != 128) return CO_ERR_UNSUPPORTED;
  if (d->num_q_heads % d->num_kv_heads) return CO_ERR_UNSUPPORTED;
  if (d->feat_dim % 64 || d->model_dim % 64) return CO_ERR_UNSUPPORTED;
  if (static_cast<int64_t>(d->num_seqs) * d->block > INT32_MAX / 2) return CO_ERR_UNSUPPORTED;
  return CO_OK;
}

AttnPlan attention_plan(const co_dims* d);

co_status check_attention_dims(const co_dims* d) {
  const int nq = d->block * (d->num_q_heads / d->num_kv_heads);
  if (nq > 64) return CO_ERR_UNSUPPORTED;
  return attention_plan(d).ok ? CO_OK : CO_ERR_UNSUPPORTED;
}

size_t elem_bytes(const co_dims* d) { return d->dtype == CO_DTYPE_BF16 ? 2 : 4; }

int carry_pages(const co_dims* d) { return (d->block + kPage - 1) / kPage; }

// RoPE inverse frequencies theta^(-2i/hd), i < hd/2, in double (rotate-half pairs)
void fill_rope_table(double* t, const co_dims* d) {
  const double lt = log2(static_cast<double>(d->rope_theta));
  for (int i = 0; i < kMaxHeadDim / 2; ++i)
    t[i] = i < d->head_dim / 2 ? exp2(-(2.0 * i / d->head_dim) * lt) : 0.0;
}

KvDest make_dest(const co_dims* d, const co_route* rt, const co_state* st) {
  KvDest e{};
  e.S = d->num_seqs;
  e.B = d->block;
  e.L = d->num_layers;
  e.Hkv = d->num_kv_heads;
  e.hd = d->head_dim;
  e.num_pages = d->num_pages;
  e.CP = carry_pages(d);
  fill_rope_table(e.rope_inv, d);
  e.row_pos = rt ? rt->row_pos : nullptr;
  e.row_dst = rt ? rt->row_dst : nullptr;
  e.k_cache = st->k_cache;
  e.v_cache = st->v_cache;
  e.k_carry = st->k_carry;
  e.v_carry = st->v_carry;
  e.status = st->status;
  return e;
}

bool state_ok(const co_state* st) {
  return st && st->ctx_len && st->carry_len && st->page_table && st->k_cache && st->v_cache &&
         st->k_carry && st->v_carry && st->status && aligned(st->k_cache, 16) &&
         aligned(st->v_cache, 16) && aligned(st->k_carry, 16) && aligned(st->v_carry, 16);
}

bool route_ok(const co_route* rt) { return rt && rt->accept_len && rt->row_pos && rt->row_dst; }

ProjectPlan project_plan(const co_dims* d) {
  return plan_project(d->num_seqs * d->block, d->feat_dim, d->model_dim,
                      2 * d->num_layers * d->num_kv_heads * d->head_dim, d->head_dim, d->dtype,
                      num_cus());
}

AttnPlan attention_plan(const co_dims* d) {
  return plan_attention(d->num_seqs, d->block, d->num_layers, d->num_q_heads, d->num_kv_heads,
                        d->head_dim, d->max_pages_per_seq, d->num_pages, d->dtype, num_cus());
}

co_status hip_status(hipError_t e) { return e == hipSuccess ? CO_OK : CO_ERR_HIP; }

// The launch functions report hipGetLastError() after their launches; an
// error left by an earlier, unrelated HIP call on this thread is cleared
// first, so that a call reports only the failures of its own launches.
void clear_stale_error() { (void)hipGetLastError(); }

// Host checks of each step, shared by the step's own entry point and by
// carryover_round, which makes all of them before its first launch.  dims are
// already checked.
co_status validate_route(const co_dims* d, const int32_t* draft_tok, const int32_t* target_tok,
                         uint32_t flags, const co_state* st, const co_route* out) {
  (void)d;
  if (!st || !st->ctx_len || !st->carry_len || !st->page_table || !st->status || !route_ok(out))
    return CO_ERR_INVALID_ARG;
  if (!(flags & CO_ROUTE_ACCEPT_ALL) &&
      (!draft_tok || (!target_tok && !(flags & CO_ROUTE_ACCEPT_BITS))))
    return CO_ERR_INVALID_ARG;
  return CO_OK;
}

co_status validate_project(const co_dims* d, const co_weights* w, const void* hidden,
                           const co_route* route, const co_state* st, const void* ws,
                           size_t ws_bytes) {
  if (!w || !w->w_f || !w->w_kv || !w->e_carry || !hidden || !route_ok(route) || !state_ok(st))
    return CO_ERR_INVALID_ARG;
  if (!aligned(hidden, 16) || !aligned(w->w_f, 16) || !aligned(w->w_kv, 16) ||
      !aligned(w->e_carry, 16) || !aligned(w->f_e, 16) || !aligned(w->w_f_carry, 16) ||
      !aligned(w->z_norm, 4) || !aligned(w->k_norm, 4))
    return CO_ERR_INVALID_ARG;
  if (w->z_norm && d->model_dim > kNormMaxCols) return CO_ERR_UNSUPPORTED;
  if (!ws || !aligned(ws, 256)) return CO_ERR_INVALID_ARG;
  if (ws_bytes < project_plan(d).total) return CO_ERR_WORKSPACE;
  return CO_OK;
}

co_status validate_attention(const co_dims* d, int32_t layer_begin, int32_t layer_count,
                             const void* q, const co_state* st, const void* out, const float* lse,
                             const void* ws, size_t ws_bytes) {
  co_status s = check_attention_dims(d);
  if (s != CO_OK) return s;
  if (layer_begin < 0 || layer_count < 0 || layer_begin + layer_count > d->num_layers)
    return CO_ERR_INVALID_ARG;
  if (!q || !out || !state_ok(st) || !aligned(q, 16) || !aligned(out, 16) ||
      (lse && !aligned(lse, 4)))
    return CO_ERR_INVALID_ARG;
  if (!ws || !aligned(ws, 256)) return CO_ERR_INVALID_ARG;
  if (ws_bytes < attention_plan(d).bytes) return CO_ERR_WORKSPACE;
  return CO_OK;
}

RouteArgs route_args(const co_dims* dims, const int32_t* draft_tok, const int32_t* target_tok,
                     uint32_t flags, co_state* state, const co_route* out) {
  RouteArgs a{};
  a.S = dims->num_seqs;
  a.B = dims->block;
  a.max_pages = dims->max_pages_per_seq;
  a.num_pages = dims->num_pages;
  a.flags = flags;
  a.draft = draft_tok;
  a.target = target_tok;
  a.ctx_len = state->ctx_len;
  a.carry_len = state->carry_len;
  a.page_table = state->page_table;
  a.accept_len = out->accept_len;
  a.row_pos = out->row_pos;
  a.row_dst = out->row_dst;
  a.status = state->status;
  return a;
}

co_status enqueue_route(const co_dims* dims, const int32_t* draft_tok, const int32_t* target_tok,
                        uint32_t flags, co_state* state, const co_route* out, hipStream_t stream) {
  clear_stale_error();
  return hip_status(
      launch_route(route_args(dims, draft_tok, target_tok, flags, state, out), stream));
}

ProjectArgs project_args(const co_dims* dims, const co_weights* w, const void* hidden,
                         const co_route* route, const co_state* state, void* ws) {
  ProjectArgs a{};
  a.M = dims->num_seqs * dims->block;
  a.Dcat = dims->feat_dim;
  a.d = dims->model_dim;
  a.dtype = dims->dtype;
  a.hidden = hidden;
  a.wf = w->w_f;
  a.wkv = w->w_kv;
  a.e = w->e_carry;
  a.fe = dims->dtype == CO_DTYPE_BF16 ? w->f_e : nullptr;
  a.wfc = w->w_f_carry;
  a.znorm = w->z_norm;
  a.dst = make_dest(dims, route, state);
  a.dst.knorm = w->k_norm;
  a.ws = ws;
  return a;
}

co_status enqueue_project(const co_dims* dims, const co_weights* w, const void* hidden,
                          const co_route* route, const co_state* state, void* ws,
                          hipStream_t stream) {
  clear_stale_error();
  return hip_status(launch_project(project_args(dims, w, hidden, route, state, ws),
                                   project_plan(dims), stream));
}

co_status do_attention(const co_dims* d, int32_t layer_begin, int32_t layer_count, const void* q,
                       const co_state* st, void* out, float* lse, uint32_t flags, void* ws,
                       hipStream_t stream, const void* k_self = nullptr,
                       const void* v_self = nullptr, float* mass = nullptr) {
  AttnArgs a{};
  a.rec_sums = (k_self || mass) ? 4 : 2;
  a.k_self = k_self;
  a.v_self = v_self;
  a.mass = mass;
  a.S = d->num_seqs;
  a.B = d->block;
  a.L = d->num_layers;
  a.layer_begin = layer_begin;
  a.Hq = d->num_q_heads;
  a.Hkv = d->num_kv_heads;
  a.hd = d->head_dim;
  a.num_pages = d->num_pages;
  a.max_pages = d->max_pages_per_seq;
  a.CP = carry_pages(d);
  a.dtype = d->dtype;
  a.flags = flags;
  fill_rope_table(a.rope_inv, d);
  a.q = q;
  a.ctx_len = st->ctx_len;
  a.carry_len = st->carry_len;
  a.page_table = st->page_table;
  a.k_cache = st->k_cache;
  a.v_cache = st->v_cache;
  a.k_carry = st->k_carry;
  a.v_carry = st->v_carry;
  a.out = out;
  a.lse = lse;
  a.status = st->status;
  a.ws = static_cast<float*>(ws);
  clear_stale_error();
  return hip_status(launch_attention(a, attention_plan(d), layer_count, stream));
}

}  // namespace

extern "C" {

size_t carryover_workspace_bytes(const co_dims* dims, int32_t which) {
  if (check_dims(dims) != CO_OK) return 0;
  const size_t pw = project_plan(dims).total;
  const size_t aw = check_attention_dims(dims) == CO_OK ? attention_plan(dims).bytes : 0;
  switch (which) {
    case CO_WS_PROJECT: return pw;
    case CO_WS_ATTENTION: return aw;
    case CO_WS_ROUND: return aw ? pw + aw : 0;   // projection scratch, then attention area
    case CO_WS_PROJECT_BACKWARD:
      return dims->dtype == CO_DTYPE_BF16
                 ? proj_bwd_ws_bytes(dims->num_seqs * dims->block, dims->feat_dim, dims->model_dim,
                                     2 * dims->num_layers * dims->num_kv_heads * dims->head_dim,
                                     num_cus())
                 : 0;
    case CO_WS_ATTENTION_BACKWARD:
      return bwd_workspace_bytes(dims->num_seqs, dims->num_layers, dims->num_kv_heads,
                                 dims->head_dim, dims->num_pages, carry_pages(dims));
    default: return 0;
  }
}

co_status carryover_route(const co_dims* dims, const int32_t* draft_tok, const int32_t* target_tok,
                          uint32_t flags, co_state* state, const co_route* out,
                          hipStream_t stream) {
  co_status s = check_dims(dims);
  if (s != CO_OK) return s;
  if ((s = validate_route(dims, draft_tok, target_tok, flags, state, out)) != CO_OK) return s;
  return enqueue_route(dims, draft_tok, target_tok, flags, state, out, stream);
}

co_status carryover_project_kv(const co_dims* dims, const co_weights* w, const void* hidden,
                               const co_route* route, const co_state* state, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  co_status s = check_dims(dims);
  if (s != CO_OK) return s;
  if ((s = validate_project(dims, w, hidden, route, state, ws, ws_bytes)) != CO_OK) return s;
  return enqueue_project(dims, w, hidden, route, state, ws, stream);
}

co_status carryover_fold_e(const co_dims* dims, const co_weights* w, float* f_e,
                           hipStream_t stream) {
  co_status s = check_dims(dims);
  if (s != CO_OK) return s;
  if (!w || !w->w_f || !w->e_carry || !f_e || !aligned(w->w_f, 16) || !aligned(w->e_carry, 16) ||
      !aligned(f_e, 16))
    return CO_ERR_INVALID_ARG;
  clear_stale_error();
  return hip_status(launch_fold_e(w->w_f, w->e_carry, dims->model_dim, dims->feat_dim,
                                  dims->dtype, f_e, stream));
}

co_status drafter_block_attention(const co_dims* dims, int32_t layer_begin, int32_t layer_count,
                                  const void* q, const co_state* state, void* out, float* lse,
                                  uint32_t flags, void* ws, size_t ws_bytes, hipStream_t stream) {
  co_status s = check_dims(dims);
  if (s != CO_OK) return s;
  if ((s = validate_attention(dims, layer_begin, layer_count, q, state, out, lse, ws,
                              ws_bytes)) != CO_OK)
    return s;
  return do_attention(dims, layer_begin, layer_count, q, state, out, lse, flags, ws, stream);
}

co_status drafter_block_attention_ext(const co_dims* dims, int32_t layer_begin,
                                      int32_t layer_count, const void* q, const void* k_self,
                                      const void* v_self, const co_state* state, void* out,
                                      float* lse, float* carry_mass, uint32_t flags, void* ws,
                                      size_t ws_bytes, hipStream_t stream) {
  co_status s = check_dims(dims);
  if (s != CO_OK) return s;
  if ((s = validate_attention(dims, layer_begin, layer_count, q, state, out, lse, ws,
                              ws_bytes)) != CO_OK)
    return s;
  if ((k_self == nullptr) != (v_self == nullptr)) return CO_ERR_INVALID_ARG;
  if ((k_self && (!aligned(k_self, 16) || !aligned(v_self, 16))) ||
      (carry_mass && !aligned(carry_mass, 4)))
    return CO_ERR_INVALID_ARG;
  if (!k_self && !carry_mass)
    return do_attention(dims, layer_begin, layer_count, q, state, out, lse, flags, ws, stream);
  if (dims->block > kMaxCarryRows) return CO_ERR_UNSUPPORTED;
  if (dims->dtype == CO_DTYPE_BF16)
    return do_attention(dims, layer_begin, layer_count, q, state, out, lse, flags, ws, stream,
                        k_self, v_self, carry_mass);
  // fp32: the attention, then the mass from its LSE over [C;U], then the self
  // segment merged into O and LSE
  if (!lse) return CO_ERR_INVALID_ARG;
  if ((s = do_attention(dims, layer_begin, layer_count, q, state, out, lse, flags, ws,
                        stream)) != CO_OK)
    return s;
  if (carry_mass &&
      (s = drafter_carry_mass(dims, layer_begin, layer_count, q, state, lse, carry_mass,
                              flags & CO_Q_PREROTATED, stream)) != CO_OK)
    return s;
  if (k_self)
    return drafter_self_merge(dims, layer_begin, layer_count, q, k_self, v_self, state, out, lse,
                              flags & CO_Q_PREROTATED, stream);
  return CO_OK;
}

co_status drafter_block_attention_backward(
    const co_dims* dims, int32_t layer_begin, int32_t layer_count, const void* q,
    const co_state* state, const void* out, const float* lse, const void* d_out,
    int32_t seqs_per_group, float* d_q, float* d_k_cache, float* d_v_cache, float* d_k_carry,
    float* d_v_carry, uint32_t flags, void* ws, size_t ws_bytes, hipStream_t stream) {
  co_status s = check_dims(dims);
  if (s != CO_OK) return s;
  if (dims->dtype != CO_DTYPE_BF16 || dims->head_dim != 64 ||
      dims->block * (dims->num_q_heads / dims->num_kv_heads) > 32)
    return CO_ERR_UNSUPPORTED;
  if (layer_begin < 0 || layer_count < 0 || layer_begin + layer_count > dims->num_layers ||
      seqs_per_group < 1)
    return CO_ERR_INVALID_ARG;
  if (!q || !out || !lse || !d_out || !d_q || !d_k_cache || !d_v_cache || !d_k_carry ||
      !d_v_carry || !state_ok(state) || !aligned(q, 16) || !aligned(out, 16) ||
      !aligned(d_out, 16) || !aligned(lse, 16) || !aligned(d_q, 16) || !aligned(d_k_cache, 16) ||
      !aligned(d_v_cache, 16) || !aligned(d_k_carry, 16) || !aligned(d_v_carry, 16))
    return CO_ERR_INVALID_ARG;
  if (!ws || !aligned(ws, 256)) return CO_ERR_INVALID_ARG;
  if (ws_bytes < carryover_workspace_bytes(dims, CO_WS_ATTENTION_BACKWARD)) return CO_ERR_WORKSPACE;
  BwdArgs b{};
  AttnArgs& a = b.a;
  a.S = dims->num_seqs;
  a.B = dims->block;
  a.L = dims->num_layers;
  a.layer_begin = layer_begin;
  a.Hq = dims->num_q_heads;
  a.Hkv = dims->num_kv_heads;
  a.hd = dims->head_dim;
  a.num_pages = dims->num_pages;
  a.max_pages = dims->max_pages_per_seq;
  a.CP = carry_pages(dims);
  a.dtype = dims->dtype;
  a.flags = flags;
  fill_rope_table(a.rope_inv, dims);
  a.q = q;
  a.ctx_len = state->ctx_len;
  a.carry_len = state->carry_len;
  a.page_table = state->page_table;
  a.k_cache = state->k_cache;
  a.v_cache = state->v_cache;
  a.k_carry = state->k_carry;
  a.v_carry = state->v_carry;
  a.status = state->status;
  a.ws = static_cast<float*>(ws);
  b.layer_count = layer_count;
  b.group = seqs_per_group;
  b.out = out;
  b.lse = lse;
  b.d_out = d_out;
  b.d_q = d_q;
  b.d_k_cache = d_k_cache;
  b.d_v_cache = d_v_cache;
  b.d_k_carry = d_k_carry;
  b.d_v_carry = d_v_carry;
  clear_stale_error();
  return hip_status(launch_attention_backward(b, stream));
}

co_status carryover_project_kv_backward(const co_dims* dims, const co_weights* w,
                                        const void* hidden, const co_route* route,
                                        const float* d_k_cache, const float* d_v_cache,
                                        const float* d_k_carry, const float* d_v_carry,
                                        float* d_w_f, float* d_w_kv, float* d_e_carry, void* ws,
                                        size_t ws_bytes, hipStream_t stream) {
  co_status s = check_dims(dims);
  if (s != CO_OK) return s;
  if (dims->dtype != CO_DTYPE_BF16) return CO_ERR_UNSUPPORTED;
  if (!w || !w->w_f || !w->w_kv || !w->e_carry || !hidden || !route_ok(route) || !d_k_cache ||
      !d_v_cache || !d_k_carry || !d_v_carry || !d_w_f || !d_w_kv || !d_e_carry)
    return CO_ERR_INVALID_ARG;
  if (w->w_f_carry || w->z_norm || w->k_norm) return CO_ERR_UNSUPPORTED;
  if (!aligned(hidden, 16) || !aligned(w->w_f, 16) || !aligned(w->w_kv, 16) ||
      !aligned(w->e_carry, 16) || !aligned(d_k_cache, 4) || !aligned(d_v_cache, 4) ||
      !aligned(d_k_carry, 4) || !aligned(d_v_carry, 4) || !aligned(d_w_f, 4) ||
      !aligned(d_w_kv, 4) || !aligned(d_e_carry, 4))
    return CO_ERR_INVALID_ARG;
  if (!ws || !aligned(ws, 256)) return CO_ERR_INVALID_ARG;
  if (ws_bytes < carryover_workspace_bytes(dims, CO_WS_PROJECT_BACKWARD)) return CO_ERR_WORKSPACE;
  ProjBwdArgs a{};
  a.M = dims->num_seqs * dims->block;
  a.Dcat = dims->feat_dim;
  a.d = dims->model_dim;
  a.L = dims->num_layers;
  a.Hkv = dims->num_kv_heads;
  a.hd = dims->head_dim;
  a.S = dims->num_seqs;
  a.B = dims->block;
  a.num_pages = dims->num_pages;
  a.CP = carry_pages(dims);
  a.num_cus = num_cus();
  fill_rope_table(a.rope_inv, dims);
  a.hidden = hidden;
  a.wf = w->w_f;
  a.wkv = w->w_kv;
  a.e = w->e_carry;
  a.row_dst = route->row_dst;
  a.row_pos = route->row_pos;
  a.dk = d_k_cache;
  a.dv = d_v_cache;
  a.dkc = d_k_carry;
  a.dvc = d_v_carry;
  a.dwf = d_w_f;
  a.dwkv = d_w_kv;
  a.de = d_e_carry;
  a.ws = ws;
  clear_stale_error();
  return hip_status(launch_project_backward(a, stream));
}

co_status drafter_carry_mass(const co_dims* dims, int32_t layer_begin, int32_t layer_count,
                             const void* q, const co_state* state, const float* lse, float* mass,
                             uint32_t flags, hipStream_t stream) {
  co_status s = check_dims(dims);
  if (s != CO_OK) return s;
  if ((s = check_attention_dims(dims)) != CO_OK) return s;
  if (dims->block > kMaxCarryRows) return CO_ERR_UNSUPPORTED;
  if (layer_begin < 0 || layer_count < 0 || layer_begin + layer_count > dims->num_layers)
    return CO_ERR_INVALID_ARG;
  if (!q || !lse || !mass || !state_ok(state) || !aligned(q, 16) || !aligned(lse, 4) ||
      !aligned(mass, 4))
    return CO_ERR_INVALID_ARG;
  MassArgs a{};
  a.S = dims->num_seqs;
  a.B = dims->block;
  a.layer_begin = layer_begin;
  a.Hq = dims->num_q_heads;
  a.Hkv = dims->num_kv_heads;
  a.hd = dims->head_dim;
  a.CP = (dims->block + kPage - 1) / kPage;
  a.flags = flags;
  fill_rope_table(a.rope_inv, dims);
  a.q = q;
  a.ctx_len = state->ctx_len;
  a.carry_len = state->carry_len;
  a.k_carry = state->k_carry;
  a.lse = lse;
  a.mass = mass;
  a.status = state->status;
  clear_stale_error();
  return hip_status(launch_carry_mass(a, layer_count, dims->dtype, stream));
}

co_status drafter_self_merge(const co_dims* dims, int32_t layer_begin, int32_t layer_count,
                             const void* q, const void* k_self, const void* v_self,
                             const co_state* state, void* out, float* lse, uint32_t flags,
                             hipStream_t stream) {
  co_status s = check_dims(dims);
  if (s != CO_OK) return s;
  if ((s = check_attention_dims(dims)) != CO_OK) return s;
  if (dims->block > kMaxCarryRows) return CO_ERR_UNSUPPORTED;
  if (layer_begin < 0 || layer_count < 0 || layer_begin + layer_count > dims->num_layers)
    return CO_ERR_INVALID_ARG;
  if (!q || !k_self || !v_self || !out || !lse || !state_ok(state) || !aligned(q, 16) ||
      !aligned(k_self, 16) || !aligned(v_self, 16) || !aligned(out, 16) || !aligned(lse, 4))
    return CO_ERR_INVALID_ARG;
  SelfArgs a{};
  a.S = dims->num_seqs;
  a.B = dims->block;
  a.Hq = dims->num_q_heads;
  a.Hkv = dims->num_kv_heads;
  a.hd = dims->head_dim;
  a.flags = flags;
  fill_rope_table(a.rope_inv, dims);
  a.q = q;
  a.k_self = k_self;
  a.v_self = v_self;
  a.ctx_len = state->ctx_len;
  a.out = out;
  a.lse = lse;
  a.status = state->status;
  clear_stale_error();
  return hip_status(launch_self_merge(a, layer_count, dims->dtype, stream));
}

co_status carryover_round(const co_dims* dims, const co_weights* w, const void* hidden,
                          const int32_t* draft_tok, const int32_t* target_tok, const void* q,
                          co_state* state, const co_route* scratch, void* out, float* lse,
                          uint32_t flags, void* ws, size_t ws_bytes, hipStream_t stream) {
  co_status s = check_dims(dims);
  if (s != CO_OK) return s;
  // every step's host checks first: a failure must leave the state untouched
  if ((s = validate_route(dims, draft_tok, target_tok, flags, state, scratch)) != CO_OK) return s;
  if ((s = validate_project(dims, w, hidden, scratch, state, ws, ws_bytes)) != CO_OK) return s;
  const size_t pw = project_plan(dims).total;   // a multiple of 256
  void* attn_ws = static_cast<char*>(ws) + pw;
  if ((s = validate_attention(dims, 0, dims->num_layers, q, state, out, lse, attn_ws,
                              ws_bytes - pw)) != CO_OK)
    return s;
  // The route step rides in the F product's launch where that product does
  // not read its descriptors (it then decides carried rows from the tokens);
  // otherwise it is a launch of its own, before the projection.
  ProjectArgs pa = project_args(dims, w, hidden, scratch, state, ws);
  const ProjectPlan plan = project_plan(dims);
  const RouteArgs ra = route_args(dims, draft_tok, target_tok, flags, state, scratch);
  clear_stale_error();
  if (route_foldable(pa, plan)) {
    pa.route = &ra;
  } else if ((s = hip_status(launch_route(ra, stream))) != CO_OK) {
    return s;
  }
  if ((s = hip_status(launch_project(pa, plan, stream))) != CO_OK) return s;
  return do_attention(dims, 0, dims->num_layers, q, state, out, lse, flags, attn_ws, stream);
}

co_status carryover_round_noalloc(const co_dims* dims, const co_weights* w, const void* hidden,
                                  const int32_t* draft_tok, const int32_t* target_tok,
                                  const void* q, co_state* state, const co_route* route_out,
                                  void* out, float* lse, uint32_t flags, hipStream_t stream) {
  co_status s = check_dims(dims);
  if (s != CO_OK) return s;
  if ((s = check_attention_dims(dims)) != CO_OK) return s;
  const size_t need = carryover_workspace_bytes(dims, CO_WS_ROUND);
  if (need == 0) return CO_ERR_UNSUPPORTED;
  if (need > kScratchBytes) return CO_ERR_WORKSPACE;
  void* ws = nullptr;
  if ((s = scratch_address(&ws)) != CO_OK) return s;
  return carryover_round(dims, w, hidden, draft_tok, target_tok, q, state, route_out, out, lse,
                         flags, ws, kScratchBytes, stream);
}

co_status carryover_verify_sample(const co_dims* dims, int32_t vocab, const int32_t* draft_tok,
                                  const float* p_target, const float* q_draft,
                                  const uint32_t* words, int32_t* accept_bits,
                                  int32_t* accept_len, int32_t* next_tok, int32_t* status,
                                  hipStream_t stream) {
  co_status s = check_dims(dims);
  if (s != CO_OK) return s;
  if (vocab < 1 || dims->block > 1024 ||
      static_cast<int64_t>(dims->num_seqs) * (dims->block + 1) * vocab > (int64_t{1} << 40))
    return CO_ERR_UNSUPPORTED;
  if (!draft_tok || !p_target || !q_draft || !words || !accept_bits || !accept_len || !next_tok ||
      !status || !aligned(draft_tok, 4) || !aligned(p_target, 4) || !aligned(q_draft, 4) ||
      !aligned(words, 4) || !aligned(accept_bits, 4) || !aligned(accept_len, 4) ||
      !aligned(next_tok, 4) || !aligned(status, 4))
    return CO_ERR_INVALID_ARG;
  VerifyArgs a{};
  a.S = dims->num_seqs;
  a.B = dims->block;
  a.V = vocab;
  a.draft = draft_tok;
  a.p = p_target;
  a.q = q_draft;
  a.words = words;
  a.accept_bits = accept_bits;
  a.accept_len = accept_len;
  a.next_tok = next_tok;
  a.status = status;
  clear_stale_error();
  return hip_status(launch_verify(a, stream));
}

co_status carryover_set_tuning(int32_t knob, int64_t value) {
  if (knob < 0 || knob >= CO_TUNE_COUNT) return CO_ERR_INVALID_ARG;
  g_tuning.v[knob] = value < 0 ? -1 : value;
  return CO_OK;
}

co_status carryover_import_kv(const co_dims* dims, int32_t seq, int32_t pos0, int32_t n_rows,
                              const void* k_rows, const void* v_rows, const co_state* state,
                              hipStream_t stream) {
  co_status s = check_dims(dims);
  if (s != CO_OK) return s;
  if (!state_ok(state) || !k_rows || !v_rows || seq < 0 || seq >= dims->num_seqs || pos0 < 0 ||
      n_rows < 0 ||
      static_cast<int64_t>(pos0) + n_rows > static_cast<int64_t>(dims->max_pages_per_seq) * kPage)
    return CO_ERR_INVALID_ARG;
  const KvDest e = make_dest(dims, nullptr, state);
  clear_stale_error();
  return hip_status(launch_import(e, dims->dtype, seq, pos0, n_rows, k_rows, v_rows,
                                  state->page_table, dims->max_pages_per_seq, stream));
}

co_status carryover_read_status(const co_state* state, int32_t* host_out, hipStream_t stream) {
  if (!state || !state->status || !host_out) return CO_ERR_INVALID_ARG;
  if (hipMemcpyAsync(host_out, state->status, sizeof(int32_t), hipMemcpyDeviceToHost, stream) !=
      hipSuccess)
    return CO_ERR_HIP;
  return hip_status(hipStreamSynchronize(stream));
}

const char* carryover_status_string(co_status status) {
  switch (status) {
    case CO_OK: return "ok";
    case CO_ERR_INVALID_ARG: return "invalid argument";
    case CO_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case CO_ERR_WORKSPACE: return "workspace too small";
    case CO_ERR_CAPACITY: return "sequence capacity exceeded";
    case CO_ERR_PAGE_RANGE: return "page id out of range";
    case CO_ERR_HIP: return "HIP runtime error";
    case CO_ERR_LENGTH: return "invalid sequence length";
    case CO_ERR_GROUP: return "page rows differ within a sequence group";
    case CO_ERR_TOKEN: return "proposed token outside the vocabulary";
    default: return "unknown status";
  }
}

}  // extern "C"

// C ABI of the ResKV hot path: argument validation, workspace sizing and
// launch on the caller's stream. Every check runs on the host before any
// kernel is enqueued.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "internal.h"

using namespace reskv;

namespace {

thread_local char g_last_error[512] = "";

reskv_status_t fail(reskv_status_t st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
reskv_status_t fail(reskv_status_t st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

reskv_status_t ok() {
  g_last_error[0] = '\0';
  return RESKV_OK;
}

reskv_status_t check_shape(const reskv_shape_t* s) {
  if (!s) return fail(RESKV_ERR_INVALID_ARG, "shape is NULL");
  if (s->batch < 1) return fail(RESKV_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", s->batch);
  if (s->num_kv_heads < 1 || s->num_q_heads < 1)
    return fail(RESKV_ERR_INVALID_ARG, "head counts must be >= 1 (Hq=%d, Hkv=%d)", s->num_q_heads, s->num_kv_heads);
  if (s->num_q_heads % s->num_kv_heads != 0)
    return fail(RESKV_ERR_INVALID_ARG, "Hq (%d) must be a multiple of Hkv (%d)", s->num_q_heads, s->num_kv_heads);
  if (s->num_q_heads / s->num_kv_heads > 16)
    return fail(RESKV_ERR_UNSUPPORTED, "group size Hq/Hkv = %d > 16", s->num_q_heads / s->num_kv_heads);
  if (s->head_dim != 64 && s->head_dim != 128)
    return fail(RESKV_ERR_UNSUPPORTED, "head_dim %d not in {64, 128}", s->head_dim);
  if (s->dtype != RESKV_F32 && s->dtype != RESKV_BF16)
    return fail(RESKV_ERR_UNSUPPORTED, "dtype %d not in {F32, BF16}", s->dtype);
  if (s->slot_cap < 1) return fail(RESKV_ERR_INVALID_ARG, "slot_cap must be >= 1 (got %d)", s->slot_cap);
  if (s->res_cap < 1) return fail(RESKV_ERR_INVALID_ARG, "res_cap must be >= 1 (got %d)", s->res_cap);
  const double cells = (double)s->batch * s->num_kv_heads * s->slot_cap * s->head_dim;
  if (cells > 4.0e12) return fail(RESKV_ERR_INVALID_ARG, "cache of %.3g elements is too large", cells);
  return RESKV_OK;
}

reskv_status_t check_gate(const reskv_gate_t* g) {
  if (!g) return fail(RESKV_ERR_INVALID_ARG, "gate is NULL");
  if (!(g->g_min >= 0.f && g->g_min <= 1.f)) return fail(RESKV_ERR_INVALID_ARG, "g_min %g outside [0, 1]", g->g_min);
  if (!isfinite(g->alpha) || !isfinite(g->beta) || !isfinite(g->tau_scalar))
    return fail(RESKV_ERR_INVALID_ARG, "gate parameters must be finite");
  if (g->beta < 0.f) return fail(RESKV_ERR_INVALID_ARG, "beta %g must be >= 0", g->beta);
  return RESKV_OK;
}

}  // namespace

extern "C" {

const char* reskv_status_string(reskv_status_t st) {
  switch (st) {
    case RESKV_OK: return "ok";
    case RESKV_ERR_INVALID_ARG: return "invalid argument";
    case RESKV_ERR_UNSUPPORTED: return "unsupported configuration";
    case RESKV_ERR_WORKSPACE: return "workspace missing or too small";
    case RESKV_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* reskv_last_error(void) { return g_last_error; }

size_t reskv_decode_workspace_size(const reskv_shape_t* shape) {
  if (check_shape(shape) != RESKV_OK) return 0;
  const DecodePlan plan = make_decode_plan(*shape);
  if ((size_t)plan.GP * plan.P * sizeof(float) > decode_max_lds_weights()) return 0;
  return plan.bytes;
}

reskv_status_t reskv_decode_attn(const reskv_shape_t* shape, const reskv_gate_t* gate, const void* q,
                                 void* kc, void* vc, const float* logc,
                                 const int32_t* res_len, int32_t* main_len,
                                 const void* k_new, const void* v_new, float* out,
                                 float* dbg_lse_main, float* dbg_lse_res, float* dbg_gate,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  reskv_status_t st = check_shape(shape);
  if (st != RESKV_OK) return st;
  if ((st = check_gate(gate)) != RESKV_OK) return st;
  if (!q || !kc || !vc || !logc || !res_len || !main_len || !out)
    return fail(RESKV_ERR_INVALID_ARG, "a required pointer is NULL");
  if ((k_new == nullptr) != (v_new == nullptr))
    return fail(RESKV_ERR_INVALID_ARG, "k_new and v_new must both be given or both be NULL");
  const DecodePlan plan = make_decode_plan(*shape);
  if ((size_t)plan.GP * plan.P * sizeof(float) > decode_max_lds_weights())
    return fail(RESKV_ERR_UNSUPPORTED, "%d split-K records per head do not fit the combine", plan.P);
  if (!workspace || workspace_bytes < plan.bytes)
    return fail(RESKV_ERR_WORKSPACE, "decode needs %zu workspace bytes, got %zu", plan.bytes,
                workspace ? workspace_bytes : (size_t)0);
  hipError_t e = launch_decode(*shape, *gate, plan, q, kc, vc, logc, res_len, main_len, k_new, v_new, out,
                               dbg_lse_main, dbg_lse_res, dbg_gate, workspace, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RESKV_ERR_HIP, "decode launch failed: %s", hipGetErrorString(e));
  return ok();
}

reskv_status_t reskv_decode_attn_static(const reskv_shape_t* shape, const reskv_gate_t* gate, const void* q,
                                        void* kc, void* vc, const float* logc, const int32_t* res_len,
                                        int32_t* main_len, const void* k_new, const void* v_new, float* out,
                                        float* dbg_lse_main, float* dbg_lse_res, float* dbg_gate, void* stream) {
  reskv_status_t st = check_shape(shape);
  if (st != RESKV_OK) return st;
  if ((st = check_gate(gate)) != RESKV_OK) return st;
  if (!q || !kc || !vc || !logc || !res_len || !main_len || !out)
    return fail(RESKV_ERR_INVALID_ARG, "a required pointer is NULL");
  if ((k_new == nullptr) != (v_new == nullptr))
    return fail(RESKV_ERR_INVALID_ARG, "k_new and v_new must both be given or both be NULL");
  const DecodePlan plan = make_decode_plan(*shape);
  if ((size_t)plan.GP * plan.P * sizeof(float) > decode_max_lds_weights())
    return fail(RESKV_ERR_UNSUPPORTED, "%d split-K records per head do not fit the combine", plan.P);
  // one block per (b, kv head) writes no split-K records
  const size_t need = plan.whole_head ? 0 : plan.bytes;
  if (need > kStaticScratchBytes)
    return fail(RESKV_ERR_WORKSPACE,
                "this shape needs %zu bytes of split-K scratch, above the %zu bytes of the library's static "
                "scratch; use reskv_decode_attn with a workspace",
                need, kStaticScratchBytes);
  void* ws = nullptr;
  hipError_t e = static_scratch(&ws);
  if (e != hipSuccess) return fail(RESKV_ERR_HIP, "static scratch lookup failed: %s", hipGetErrorString(e));
  e = launch_decode(*shape, *gate, plan, q, kc, vc, logc, res_len, main_len, k_new, v_new, out, dbg_lse_main,
                    dbg_lse_res, dbg_gate, ws, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RESKV_ERR_HIP, "decode launch failed: %s", hipGetErrorString(e));
  return ok();
}

size_t reskv_decode_ragged_workspace_size(const reskv_shape_t* shape) {
  if (check_shape(shape) != RESKV_OK) return 0;
  RaggedPlan plan;
  if (!make_ragged_plan(*shape, &plan)) return 0;
  return plan.bytes;
}

reskv_status_t reskv_decode_attn_ragged(const reskv_shape_t* shape, const reskv_gate_t* gate, const void* q,
                                        void* kc, void* vc, const float* logc, const int32_t* res_len,
                                        int32_t* main_len, const void* k_new, const void* v_new, float* out,
                                        float* dbg_lse_main, float* dbg_lse_res, float* dbg_gate, void* workspace,
                                        size_t workspace_bytes, void* stream) {
  reskv_status_t st = check_shape(shape);
  if (st != RESKV_OK) return st;
  if ((st = check_gate(gate)) != RESKV_OK) return st;
  if (!q || !kc || !vc || !logc || !res_len || !main_len || !out)
    return fail(RESKV_ERR_INVALID_ARG, "a required pointer is NULL");
  if ((k_new == nullptr) != (v_new == nullptr))
    return fail(RESKV_ERR_INVALID_ARG, "k_new and v_new must both be given or both be NULL");
  RaggedPlan plan;
  if (!make_ragged_plan(*shape, &plan))
    return fail(RESKV_ERR_UNSUPPORTED,
                "the ragged schedule takes group sizes up to 8, at most 2048 (sequence, KV head) pairs, slot "
                "capacities up to 64960 and bf16 rows (fp32 rows of 64)");
  if (!workspace || workspace_bytes < plan.bytes)
    return fail(RESKV_ERR_WORKSPACE, "ragged decode needs %zu workspace bytes, got %zu", plan.bytes,
                workspace ? workspace_bytes : (size_t)0);
  hipError_t e = launch_decode_ragged(*shape, *gate, plan, q, kc, vc, logc, res_len, main_len, k_new, v_new, out,
                                      dbg_lse_main, dbg_lse_res, dbg_gate, workspace, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RESKV_ERR_HIP, "decode launch failed: %s", hipGetErrorString(e));
  return ok();
}

reskv_status_t reskv_decode_branches(const reskv_shape_t* shape, const reskv_gate_t* gate, const void* q,
                                     const void* kc, const void* vc, const float* logc, const int32_t* res_len,
                                     const int32_t* main_len, float* out_main, float* lse_main, float* out_res,
                                     float* lse_res, float* gate_out, void* workspace, size_t workspace_bytes,
                                     void* stream) {
  reskv_status_t st = check_shape(shape);
  if (st != RESKV_OK) return st;
  if ((st = check_gate(gate)) != RESKV_OK) return st;
  if (!q || !kc || !vc || !logc || !res_len || !main_len || !out_main || !lse_main || !out_res || !lse_res ||
      !gate_out)
    return fail(RESKV_ERR_INVALID_ARG, "a required pointer is NULL");
  const DecodePlan plan = make_decode_plan(*shape);
  if ((size_t)plan.GP * plan.P * sizeof(float) > decode_max_lds_weights())
    return fail(RESKV_ERR_UNSUPPORTED, "%d split-K records per head do not fit the combine", plan.P);
  if (!workspace || workspace_bytes < plan.bytes)
    return fail(RESKV_ERR_WORKSPACE, "decode needs %zu workspace bytes, got %zu", plan.bytes,
                workspace ? workspace_bytes : (size_t)0);
  hipError_t e = launch_decode_branches(*shape, *gate, plan, q, kc, vc, logc, res_len, main_len, out_main, lse_main,
                                        out_res, lse_res, gate_out, workspace, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RESKV_ERR_HIP, "decode launch failed: %s", hipGetErrorString(e));
  return ok();
}

reskv_status_t reskv_merge_branches(const reskv_shape_t* shape, int32_t mode, const float* out_main,
                                    const float* lse_main, const float* out_res, const float* lse_res,
                                    const float* gate, float* out, void* stream) {
  reskv_status_t st = check_shape(shape);
  if (st != RESKV_OK) return st;
  if (mode != RESKV_MERGE_SHARED && mode != RESKV_MERGE_SEPARATE)
    return fail(RESKV_ERR_INVALID_ARG, "merge mode %d is neither SHARED (0) nor SEPARATE (1)", mode);
  if (!out_main || !lse_main || !out_res || !lse_res || !gate || !out)
    return fail(RESKV_ERR_INVALID_ARG, "a required pointer is NULL");
  if (out == out_main || out == out_res) return fail(RESKV_ERR_INVALID_ARG, "out must not alias a branch output");
  hipError_t e = launch_merge_branches(*shape, mode, out_main, lse_main, out_res, lse_res, gate, out,
                                       (hipStream_t)stream);
  if (e != hipSuccess) return fail(RESKV_ERR_HIP, "merge launch failed: %s", hipGetErrorString(e));
  return ok();
}

reskv_status_t reskv_append_kv(const reskv_shape_t* shape, const void* k_new, const void* v_new, void* kc,
                               void* vc, const int32_t* res_len, int32_t* main_len, void* stream) {
  reskv_status_t st = check_shape(shape);
  if (st != RESKV_OK) return st;
  if (!k_new || !v_new || !kc || !vc || !res_len || !main_len)
    return fail(RESKV_ERR_INVALID_ARG, "a required pointer is NULL");
  hipError_t e = launch_append(*shape, k_new, v_new, kc, vc, res_len, main_len, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RESKV_ERR_HIP, "append launch failed: %s", hipGetErrorString(e));
  return ok();
}

static reskv_status_t check_build(const reskv_shape_t* shape, const reskv_build_params_t* p,
                                  const int32_t* seq_len, const int32_t* budget, const int32_t* res_count) {
  reskv_status_t st = check_shape(shape);
  if (st != RESKV_OK) return st;
  if (!p) return fail(RESKV_ERR_INVALID_ARG, "params is NULL");
  if (!seq_len || !budget || !res_count) return fail(RESKV_ERR_INVALID_ARG, "a host length array is NULL");
  if (p->max_seq_len < 1) return fail(RESKV_ERR_INVALID_ARG, "max_seq_len must be >= 1");
  if (p->obs_window < 1 || p->obs_window > p->max_seq_len)
    return fail(RESKV_ERR_INVALID_ARG, "obs_window %d outside [1, %d]", p->obs_window, p->max_seq_len);
  if (p->recent_window < 0) return fail(RESKV_ERR_INVALID_ARG, "recent_window must be >= 0");
  if (p->lloyd_iters < 1 || p->lloyd_iters > 64) return fail(RESKV_ERR_INVALID_ARG, "lloyd_iters %d outside [1, 64]", p->lloyd_iters);
  if (p->pool_kernel < 0 || p->pool_kernel > 31 || (p->pool_kernel > 0 && p->pool_kernel % 2 == 0))
    return fail(RESKV_ERR_INVALID_ARG, "pool_kernel %d must be 0 (= 5) or odd in [1, 31]", p->pool_kernel);
  if (p->fit_rows < 0 || p->fit_rows > p->obs_window)
    return fail(RESKV_ERR_INVALID_ARG, "fit_rows %d outside [0, obs_window=%d]", p->fit_rows, p->obs_window);
  const int rows = p->fit_rows > 0 ? p->fit_rows : p->obs_window;
  if ((long long)rows * (shape->num_q_heads / shape->num_kv_heads) > 1024)
    return fail(RESKV_ERR_UNSUPPORTED, "scoring rows per KV head (G*%d = %d) above 1024", rows,
                rows * (shape->num_q_heads / shape->num_kv_heads));
  if (shape->res_cap > 4096) return fail(RESKV_ERR_UNSUPPORTED, "res_cap %d above 4096", shape->res_cap);
  const int Hkv = shape->num_kv_heads;
  for (int b = 0; b < shape->batch; ++b) {
    const int s = seq_len[b];
    if (s < p->obs_window || s > p->max_seq_len)
      return fail(RESKV_ERR_INVALID_ARG, "seq_len[%d] = %d outside [obs_window=%d, max_seq_len=%d]", b, s, p->obs_window, p->max_seq_len);
    if (budget[b] < 1 || budget[b] > shape->slot_cap)
      return fail(RESKV_ERR_INVALID_ARG, "budget[%d] = %d outside [1, slot_cap=%d]", b, budget[b], shape->slot_cap);
    for (int h = 0; h < Hkv; ++h) {
      const int r = res_count[b * Hkv + h];
      if (r < 0 || r >= budget[b] || r > shape->res_cap)
        return fail(RESKV_ERR_INVALID_ARG, "res_count[%d] = %d must satisfy 0 <= r < budget (%d) and r <= res_cap (%d)",
                    b * Hkv + h, r, budget[b], shape->res_cap);
      const int m = budget[b] - r;
      const int main_len = s <= m ? s : m;
      if (r + main_len > shape->slot_cap)
        return fail(RESKV_ERR_INVALID_ARG, "r + main slots (%d) exceed slot_cap (%d)", r + main_len, shape->slot_cap);
    }
  }
  return RESKV_OK;
}

size_t reskv_build_workspace_size(const reskv_shape_t* shape, const reskv_build_params_t* params,
                                  const int32_t* seq_len_host, const int32_t* budget_host,
                                  const int32_t* res_count_host) {
  if (check_build(shape, params, seq_len_host, budget_host, res_count_host) != RESKV_OK) return 0;
  BuildPlan plan;
  if (!make_build_plan(*shape, *params, seq_len_host, budget_host, res_count_host, &plan)) return 0;
  return plan.bytes;
}

reskv_status_t reskv_build_cache(const reskv_shape_t* shape, const reskv_build_params_t* params, const void* k,
                                 const void* v, const int32_t* seq_len_host, const void* q_obs,
                                 const int32_t* budget_host, const int32_t* res_count_host, void* kc, void* vc,
                                 float* logc, int32_t* main_idx, int32_t* res_len, int32_t* main_len,
                                 float* dbg_scores, int32_t* dbg_assign, float* dbg_centers, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  reskv_status_t st = check_build(shape, params, seq_len_host, budget_host, res_count_host);
  if (st != RESKV_OK) return st;
  if (!k || !v || !q_obs || !kc || !vc || !logc || !main_idx || !res_len || !main_len)
    return fail(RESKV_ERR_INVALID_ARG, "a required pointer is NULL");
  BuildPlan plan;
  if (!make_build_plan(*shape, *params, seq_len_host, budget_host, res_count_host, &plan))
    return fail(RESKV_ERR_UNSUPPORTED, "construction plan could not be formed for these sizes");
  if (!workspace || workspace_bytes < plan.bytes)
    return fail(RESKV_ERR_WORKSPACE, "build needs %zu workspace bytes, got %zu", plan.bytes,
                workspace ? workspace_bytes : (size_t)0);
  hipError_t e = launch_build(*shape, *params, plan, k, v, seq_len_host, q_obs, budget_host, res_count_host, kc,
                              vc, logc, main_idx, res_len, main_len, dbg_scores, dbg_assign, dbg_centers,
                              workspace, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RESKV_ERR_HIP, "build launch failed: %s", hipGetErrorString(e));
  return ok();
}

static reskv_status_t check_adakv(const reskv_shape_t* shape, double safeguard, int32_t decode_reserve,
                                  const int32_t* budget) {
  if (!(safeguard >= 0.0 && safeguard <= 1.0))
    return fail(RESKV_ERR_INVALID_ARG, "safeguard %g outside [0, 1]", safeguard);
  if (decode_reserve < 0) return fail(RESKV_ERR_INVALID_ARG, "decode_reserve %d must be >= 0", decode_reserve);
  for (int b = 0; b < shape->batch; ++b)
    if ((long long)budget[b] + decode_reserve > shape->slot_cap)
      return fail(RESKV_ERR_INVALID_ARG, "budget[%d] + decode_reserve = %lld exceeds slot_cap (%d)", b,
                  (long long)budget[b] + decode_reserve, shape->slot_cap);
  if (shape->num_kv_heads > kAdaMaxHeads)
    return fail(RESKV_ERR_UNSUPPORTED, "cross-head allocation over %d KV heads (at most %d)", shape->num_kv_heads,
                kAdaMaxHeads);
  return RESKV_OK;
}

size_t reskv_build_adakv_workspace_size(const reskv_shape_t* shape, const reskv_build_params_t* params,
                                        double safeguard, int32_t decode_reserve, const int32_t* seq_len_host,
                                        const int32_t* budget_host, const int32_t* res_count_host) {
  if (check_build(shape, params, seq_len_host, budget_host, res_count_host) != RESKV_OK) return 0;
  if (check_adakv(shape, safeguard, decode_reserve, budget_host) != RESKV_OK) return 0;
  BuildPlan plan;
  if (!make_build_plan_adakv(*shape, *params, safeguard, decode_reserve, seq_len_host, budget_host, res_count_host,
                             &plan))
    return 0;
  return plan.bytes;
}

reskv_status_t reskv_build_cache_adakv(const reskv_shape_t* shape, const reskv_build_params_t* params,
                                       double safeguard, int32_t decode_reserve, const void* k, const void* v,
                                       const int32_t* seq_len_host, const void* q_obs, const int32_t* budget_host,
                                       const int32_t* res_count_host, void* kc, void* vc, float* logc,
                                       int32_t* main_idx, int32_t* res_len, int32_t* main_len, float* dbg_scores,
                                       int32_t* dbg_assign, float* dbg_centers, void* workspace,
                                       size_t workspace_bytes, void* stream) {
  reskv_status_t st = check_build(shape, params, seq_len_host, budget_host, res_count_host);
  if (st != RESKV_OK) return st;
  if ((st = check_adakv(shape, safeguard, decode_reserve, budget_host)) != RESKV_OK) return st;
  if (!k || !v || !q_obs || !kc || !vc || !logc || !main_idx || !res_len || !main_len)
    return fail(RESKV_ERR_INVALID_ARG, "a required pointer is NULL");
  BuildPlan plan;
  if (!make_build_plan_adakv(*shape, *params, safeguard, decode_reserve, seq_len_host, budget_host, res_count_host,
                             &plan))
    return fail(RESKV_ERR_UNSUPPORTED, "construction plan could not be formed for these sizes");
  if (!workspace || workspace_bytes < plan.bytes)
    return fail(RESKV_ERR_WORKSPACE, "build needs %zu workspace bytes, got %zu", plan.bytes,
                workspace ? workspace_bytes : (size_t)0);
  hipError_t e = launch_build_adakv(*shape, *params, safeguard, decode_reserve, plan, k, v, seq_len_host, q_obs,
                                    budget_host, res_count_host, kc, vc, logc, main_idx, res_len, main_len,
                                    dbg_scores, dbg_assign, dbg_centers, workspace, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RESKV_ERR_HIP, "build launch failed: %s", hipGetErrorString(e));
  return ok();
}

// Proxy arguments, then every candidate count through the construction
// checks with the fit rows in place.
static reskv_status_t check_proxy(const reskv_shape_t* shape, const reskv_build_params_t* p,
                                  const reskv_proxy_params_t* x, const int32_t* seq_len, const int32_t* budget,
                                  reskv_build_params_t* pf) {
  reskv_status_t st = check_shape(shape);
  if (st != RESKV_OK) return st;
  if (!p || !x) return fail(RESKV_ERR_INVALID_ARG, "params or proxy params is NULL");
  if (!seq_len || !budget) return fail(RESKV_ERR_INVALID_ARG, "a host length array is NULL");
  if (!x->grid_host) return fail(RESKV_ERR_INVALID_ARG, "grid_host is NULL");
  if (x->n_grid < 1 || x->n_grid > kProxyMaxGrid)
    return fail(RESKV_ERR_INVALID_ARG, "n_grid %d outside [1, %d]", x->n_grid, kProxyMaxGrid);
  bool has_zero = false;
  for (int c = 0; c < x->n_grid; ++c) {
    const double f = x->grid_host[c];
    if (!(f >= 0.0 && f < 1.0)) return fail(RESKV_ERR_INVALID_ARG, "grid[%d] = %g outside [0, 1)", c, f);
    has_zero |= f == 0.0;
  }
  if (!has_zero) return fail(RESKV_ERR_INVALID_ARG, "the grid must contain the fraction 0 (the pure-main cache)");
  if (x->val_rows < 1 || x->val_rows >= p->obs_window)
    return fail(RESKV_ERR_INVALID_ARG, "val_rows %d outside [1, obs_window - 1 = %d]", x->val_rows,
                p->obs_window - 1);
  if (p->fit_rows != 0 && p->fit_rows != p->obs_window - x->val_rows)
    return fail(RESKV_ERR_INVALID_ARG, "fit_rows %d must be 0 or obs_window - val_rows = %d", p->fit_rows,
                p->obs_window - x->val_rows);
  if (!(x->delta >= 0.f && x->delta <= 1.f)) return fail(RESKV_ERR_INVALID_ARG, "delta %g outside [0, 1]", x->delta);
  *pf = *p;
  pf->fit_rows = p->obs_window - x->val_rows;
  const int Hkv = shape->num_kv_heads;
  std::vector<int32_t> counts((size_t)shape->batch * Hkv);
  for (int c = 0; c < x->n_grid; ++c) {
    for (int b = 0; b < shape->batch; ++b) {
      const double r = floor(x->grid_host[c] * (double)budget[b] + 0.5);
      if (budget[b] >= 1 && r >= budget[b])
        return fail(RESKV_ERR_INVALID_ARG, "grid[%d] = %g gives r = %.0f >= budget[%d] = %d", c, x->grid_host[c],
                    r, b, budget[b]);
      for (int h = 0; h < Hkv; ++h) counts[(size_t)b * Hkv + h] = (int32_t)r;
    }
    if ((st = check_build(shape, pf, seq_len, budget, counts.data())) != RESKV_OK) return st;
  }
  return RESKV_OK;
}

size_t reskv_build_proxy_workspace_size(const reskv_shape_t* shape, const reskv_build_params_t* params,
                                        const reskv_proxy_params_t* proxy, const int32_t* seq_len_host,
                                        const int32_t* budget_host) {
  reskv_build_params_t pf;
  if (check_proxy(shape, params, proxy, seq_len_host, budget_host, &pf) != RESKV_OK) return 0;
  ProxyPlan plan;
  if (!make_proxy_plan(*shape, pf, *proxy, seq_len_host, budget_host, &plan)) return 0;
  return plan.bytes;
}

reskv_status_t reskv_build_cache_proxy(const reskv_shape_t* shape, const reskv_build_params_t* params,
                                       const reskv_proxy_params_t* proxy, const reskv_gate_t* gate, const void* k,
                                       const void* v, const int32_t* seq_len_host, const void* q_obs,
                                       const int32_t* budget_host, void* kc, void* vc, float* logc,
                                       int32_t* main_idx, int32_t* res_len, int32_t* main_len, float* val_loss,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  reskv_build_params_t pf;
  reskv_status_t st = check_proxy(shape, params, proxy, seq_len_host, budget_host, &pf);
  if (st != RESKV_OK) return st;
  if ((st = check_gate(gate)) != RESKV_OK) return st;
  if (!k || !v || !q_obs || !kc || !vc || !logc || !main_idx || !res_len || !main_len)
    return fail(RESKV_ERR_INVALID_ARG, "a required pointer is NULL");
  ProxyPlan plan;
  if (!make_proxy_plan(*shape, pf, *proxy, seq_len_host, budget_host, &plan))
    return fail(RESKV_ERR_UNSUPPORTED, "proxy plan could not be formed for these sizes");
  if (!workspace || workspace_bytes < plan.bytes)
    return fail(RESKV_ERR_WORKSPACE, "proxy build needs %zu workspace bytes, got %zu", plan.bytes,
                workspace ? workspace_bytes : (size_t)0);
  hipError_t e = launch_build_proxy(*shape, pf, *proxy, *gate, plan, k, v, seq_len_host, q_obs, budget_host, kc, vc,
                                    logc, main_idx, res_len, main_len, val_loss, workspace, (hipStream_t)stream);
  if (e != hipSuccess) return fail(RESKV_ERR_HIP, "proxy build launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"

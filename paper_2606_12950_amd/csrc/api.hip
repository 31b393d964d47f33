// C-ABI entry points of libmaestro: host-side argument checks, then the kernel launchers.
// Nothing here touches device memory; every check happens before the first launch.
#include <math.h>

#include "internal.h"

namespace {

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
static_assert(sizeof(maestro_deg_plan) == 128, "plan record layout");
static_assert(sizeof(maestro_plan_step) == 16, "plan step layout");

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

}  // namespace

extern "C" {

const char* maestro_status_string(maestro_status s) {
  switch (s) {
    case MAESTRO_OK: return "ok";
    case MAESTRO_ERR_INVALID_ARG: return "invalid argument";
    case MAESTRO_ERR_UNSUPPORTED: return "unsupported shape";
    case MAESTRO_ERR_WORKSPACE: return "workspace too small";
    case MAESTRO_ERR_LAUNCH: return "kernel launch failed";
  }
  return "unknown status";
}

size_t maestro_predict_workspace(const maestro_predictor*, int64_t) { return 0; }

size_t maestro_route_workspace(int64_t n, int32_t n_models, int32_t n_nodes, int32_t k) {
  return maestro::route_workspace_bytes(n, n_models, n_nodes, k);
}

size_t maestro_prioritize_workspace(int32_t n_workflows, int64_t n_stages) {
  if (n_workflows < 0 || n_stages < 0) return 0;
  return maestro::prioritize_workspace_bytes(n_workflows, n_stages);
}

maestro_status maestro_predict(const maestro_predictor* p, int64_t n, const void* x,
                               const int32_t* prompt_len, const int32_t* model_id,
                               const float* kv_bytes_per_token, int32_t n_models,
                               float* pred_len, double* kv_bytes, void* workspace,
                               size_t workspace_bytes, void* stream) {
  (void)workspace;
  (void)workspace_bytes;
  if (!p || n < 0 || n_models < 1 || n_models > 64) return MAESTRO_ERR_INVALID_ARG;
  if (p->n_layers < 1 || p->n_layers > 4) return MAESTRO_ERR_INVALID_ARG;
  if (p->dtype != MAESTRO_F32 && p->dtype != MAESTRO_BF16) return MAESTRO_ERR_INVALID_ARG;
  for (int l = 0; l <= p->n_layers; ++l)
    if (p->dims[l] < 1) return MAESTRO_ERR_INVALID_ARG;
  for (int l = 0; l < p->n_layers; ++l)
    if (!p->weight[l] || !p->bias[l] || !aligned(p->weight[l], 16) || !aligned(p->bias[l], 16))
      return MAESTRO_ERR_INVALID_ARG;
  if (!p->bin_centre || !aligned(p->bin_centre, 16)) return MAESTRO_ERR_INVALID_ARG;
  if (n > 0) {
    if (!x || !prompt_len || !model_id || !kv_bytes_per_token || !pred_len || !kv_bytes)
      return MAESTRO_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(prompt_len, 4) || !aligned(model_id, 4) ||
        !aligned(kv_bytes_per_token, 4) || !aligned(pred_len, 4) || !aligned(kv_bytes, 8))
      return MAESTRO_ERR_INVALID_ARG;
  }
  if (!maestro::predict_shape_supported(*p)) return MAESTRO_ERR_UNSUPPORTED;
  if (n > (int64_t)1 << 37) return MAESTRO_ERR_UNSUPPORTED;  // grid limit: 2^30 blocks of 128 rows
  return maestro::launch_predict(*p, n, x, prompt_len, model_id, kv_bytes_per_token, n_models,
                                 pred_len, kv_bytes, as_stream(stream));
}

maestro_status maestro_predict_two_phase(const maestro_predictor* p, const maestro_two_phase* tp, int64_t n,
                                         const void* x, const int32_t* prompt_len, const int32_t* model_id,
                                         const int32_t* role_id, const int32_t* tool_avail,
                                         const float* kv_bytes_per_token, int32_t n_models, float* p_tool,
                                         float* pred_len, double* kv_bytes, void* stream) {
  if (!p || !tp || n < 0 || n_models < 1 || n_models > 64) return MAESTRO_ERR_INVALID_ARG;
  if (p->n_layers < 1 || p->n_layers > 4) return MAESTRO_ERR_INVALID_ARG;
  if (p->dtype != MAESTRO_F32 && p->dtype != MAESTRO_BF16) return MAESTRO_ERR_INVALID_ARG;
  for (int l = 0; l <= p->n_layers; ++l)
    if (p->dims[l] < 1) return MAESTRO_ERR_INVALID_ARG;
  for (int l = 0; l < p->n_layers; ++l)
    if (!p->weight[l] || !p->bias[l] || !aligned(p->weight[l], 16) || !aligned(p->bias[l], 16))
      return MAESTRO_ERR_INVALID_ARG;
  if (tp->n_roles < 0 || tp->n_roles > 64 || tp->n_knots < 2 || tp->n_knots > 64) return MAESTRO_ERR_INVALID_ARG;
  if (!(tp->max_len > 0.0f) || !isfinite(tp->max_len)) return MAESTRO_ERR_INVALID_ARG;
  if (tp->n_roles > 0 && (!tp->role_head || !aligned(tp->role_head, 4))) return MAESTRO_ERR_INVALID_ARG;
  if (!tp->tool_coef || !aligned(tp->tool_coef, 16) || !tp->iso_x || !tp->iso_y || !aligned(tp->iso_x, 4) ||
      !aligned(tp->iso_y, 4))
    return MAESTRO_ERR_INVALID_ARG;
  if (n > 0) {
    if (!x || !prompt_len || !model_id || !role_id || !tool_avail || !kv_bytes_per_token || !pred_len ||
        !kv_bytes)
      return MAESTRO_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(prompt_len, 4) || !aligned(model_id, 4) || !aligned(role_id, 4) ||
        !aligned(tool_avail, 4) || !aligned(kv_bytes_per_token, 4) || !aligned(pred_len, 4) ||
        !aligned(kv_bytes, 8) || (p_tool && !aligned(p_tool, 4)))
      return MAESTRO_ERR_INVALID_ARG;
  }
  if (!maestro::two_phase_shape_supported(*p)) return MAESTRO_ERR_UNSUPPORTED;
  if (n > (int64_t)1 << 37) return MAESTRO_ERR_UNSUPPORTED;
  return maestro::launch_predict_two_phase(*p, *tp, n, x, prompt_len, model_id, role_id, tool_avail,
                                           kv_bytes_per_token, n_models, p_tool, pred_len, kv_bytes,
                                           as_stream(stream));
}

size_t maestro_role_lengths_workspace(int64_t n, int32_t n_regressors) {
  if (n < 0 || n_regressors < 1 || n_regressors > MAESTRO_MAX_ROLE_REGRESSORS) return 0;
  return maestro::role_lengths_workspace_bytes(n, n_regressors);
}

maestro_status maestro_predict_role_lengths(const maestro_predictor* p, const maestro_role_regressors* r, int64_t n,
                                            const void* x, const int32_t* prompt_len, const int32_t* model_id,
                                            const int32_t* role_id, const float* p_tool,
                                            const float* kv_bytes_per_token, int32_t n_models, float* pred_len,
                                            double* kv_bytes, void* workspace, size_t workspace_bytes,
                                            void* stream) {
  if (!p || !r || n < 0 || n_models < 1 || n_models > 64) return MAESTRO_ERR_INVALID_ARG;
  if (p->n_layers < 1 || p->n_layers > 4) return MAESTRO_ERR_INVALID_ARG;
  if (p->dtype != MAESTRO_F32 && p->dtype != MAESTRO_BF16) return MAESTRO_ERR_INVALID_ARG;
  for (int l = 0; l <= p->n_layers; ++l)
    if (p->dims[l] < 1) return MAESTRO_ERR_INVALID_ARG;
  for (int l = 0; l < p->n_layers; ++l)
    if (!p->weight[l] || !p->bias[l] || !aligned(p->weight[l], 16) || !aligned(p->bias[l], 16))
      return MAESTRO_ERR_INVALID_ARG;
  if (r->n_regressors < 1 || r->n_regressors > MAESTRO_MAX_ROLE_REGRESSORS || r->n_roles < 0 || r->n_roles > 64)
    return MAESTRO_ERR_INVALID_ARG;
  if (!(r->max_len > 0.0f) || !isfinite(r->max_len)) return MAESTRO_ERR_INVALID_ARG;
  if (r->n_roles > 0 && (!r->role_regressor || !aligned(r->role_regressor, 4))) return MAESTRO_ERR_INVALID_ARG;
  if (!r->tool_coef || !aligned(r->tool_coef, 4)) return MAESTRO_ERR_INVALID_ARG;
  if (n > 0) {
    if (!x || !prompt_len || !model_id || !role_id || !p_tool || !kv_bytes_per_token || !pred_len || !kv_bytes)
      return MAESTRO_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(prompt_len, 4) || !aligned(model_id, 4) || !aligned(role_id, 4) ||
        !aligned(p_tool, 4) || !aligned(kv_bytes_per_token, 4) || !aligned(pred_len, 4) || !aligned(kv_bytes, 8))
      return MAESTRO_ERR_INVALID_ARG;
  }
  if (!maestro::two_phase_shape_supported(*p)) return MAESTRO_ERR_UNSUPPORTED;
  if (n > ((int64_t)1 << 22)) return MAESTRO_ERR_UNSUPPORTED;
  const size_t need = maestro::role_lengths_workspace_bytes(n, r->n_regressors);
  if (workspace_bytes < need || (need > 0 && (!workspace || !aligned(workspace, 256)))) return MAESTRO_ERR_WORKSPACE;
  return maestro::launch_role_lengths(*p, *r, n, x, prompt_len, model_id, role_id, p_tool, kv_bytes_per_token,
                                      n_models, pred_len, kv_bytes, workspace, as_stream(stream));
}

namespace {

// maestro_route_ex and maestro_route_tiered: T_act from (cold_s, resident_mask), or from
// act_matrix when it is not NULL
maestro_status route_checked(int64_t n, const int32_t* model_id, const float* pred_len, const double* kv_bytes,
                             const float* decode_s_per_token, int32_t n_models, int32_t n_nodes,
                             const double* free_bytes, const float* queue_s, const float* cold_s,
                             const uint64_t* resident_mask, const float* act_matrix, double rho, int32_t k,
                             int32_t algo, int32_t* node_idx, float* score, void* workspace,
                             size_t workspace_bytes, void* stream) {
  if (n < 0 || n_models < 1 || n_models > 64 || n_nodes < 1 || k < 1 || k > 16)
    return MAESTRO_ERR_INVALID_ARG;
  if (algo != MAESTRO_ROUTE_AUTO && algo != MAESTRO_ROUTE_SCAN && algo != MAESTRO_ROUTE_SORTED)
    return MAESTRO_ERR_INVALID_ARG;
  if (!(rho >= 0.0) || rho == INFINITY) return MAESTRO_ERR_INVALID_ARG;
  if (!decode_s_per_token || !free_bytes || !queue_s) return MAESTRO_ERR_INVALID_ARG;
  if (!aligned(decode_s_per_token, 4) || !aligned(free_bytes, 8) || !aligned(queue_s, 4))
    return MAESTRO_ERR_INVALID_ARG;
  if (act_matrix ? !aligned(act_matrix, 4)
                 : (!cold_s || !resident_mask || !aligned(cold_s, 4) || !aligned(resident_mask, 8)))
    return MAESTRO_ERR_INVALID_ARG;
  if (n > 0) {
    if (!model_id || !pred_len || !kv_bytes || !node_idx || !score) return MAESTRO_ERR_INVALID_ARG;
    if (!aligned(model_id, 4) || !aligned(pred_len, 4) || !aligned(kv_bytes, 8) ||
        !aligned(node_idx, 4) || !aligned(score, 4))
      return MAESTRO_ERR_INVALID_ARG;
  }
  if (n > (int64_t)1 << 37) return MAESTRO_ERR_UNSUPPORTED;
  const size_t need = maestro::route_workspace_bytes(n, n_models, n_nodes, k);
  if (algo != MAESTRO_ROUTE_SCAN && (workspace_bytes < need || (need > 0 && !aligned(workspace, 16))))
    return MAESTRO_ERR_WORKSPACE;
  return maestro::launch_route(n, model_id, pred_len, kv_bytes, decode_s_per_token, n_models,
                               n_nodes, free_bytes, queue_s, cold_s, resident_mask, act_matrix, rho, k,
                               algo, node_idx, score, workspace, workspace_bytes, as_stream(stream));
}

}  // namespace

maestro_status maestro_route_ex(int64_t n, const int32_t* model_id, const float* pred_len,
                                const double* kv_bytes, const float* decode_s_per_token,
                                int32_t n_models, int32_t n_nodes, const double* free_bytes,
                                const float* queue_s, const float* cold_s,
                                const uint64_t* resident_mask, double rho, int32_t k, int32_t algo,
                                int32_t* node_idx, float* score, void* workspace,
                                size_t workspace_bytes, void* stream) {
  if (!cold_s || !resident_mask) return MAESTRO_ERR_INVALID_ARG;
  return route_checked(n, model_id, pred_len, kv_bytes, decode_s_per_token, n_models, n_nodes, free_bytes,
                       queue_s, cold_s, resident_mask, nullptr, rho, k, algo, node_idx, score, workspace,
                       workspace_bytes, stream);
}

maestro_status maestro_route_tiered(int64_t n, const int32_t* model_id, const float* pred_len,
                                    const double* kv_bytes, const float* decode_s_per_token, int32_t n_models,
                                    int32_t n_nodes, const double* free_bytes, const float* queue_s,
                                    const float* act_s, double rho, int32_t k, int32_t algo, int32_t* node_idx,
                                    float* score, void* workspace, size_t workspace_bytes, void* stream) {
  if (!act_s) return MAESTRO_ERR_INVALID_ARG;
  return route_checked(n, model_id, pred_len, kv_bytes, decode_s_per_token, n_models, n_nodes, free_bytes,
                       queue_s, nullptr, nullptr, act_s, rho, k, algo, node_idx, score, workspace,
                       workspace_bytes, stream);
}

maestro_status maestro_route(int64_t n, const int32_t* model_id, const float* pred_len,
                             const double* kv_bytes, const float* decode_s_per_token,
                             int32_t n_models, int32_t n_nodes, const double* free_bytes,
                             const float* queue_s, const float* cold_s,
                             const uint64_t* resident_mask, double rho, int32_t k,
                             int32_t* node_idx, float* score, void* workspace,
                             size_t workspace_bytes, void* stream) {
  return maestro_route_ex(n, model_id, pred_len, kv_bytes, decode_s_per_token, n_models, n_nodes,
                          free_bytes, queue_s, cold_s, resident_mask, rho, k, MAESTRO_ROUTE_AUTO,
                          node_idx, score, workspace, workspace_bytes, stream);
}

size_t maestro_route_lists_bytes(int32_t n_models, int32_t n_nodes) {
  if (n_models < 1 || n_models > 64 || n_nodes < 1) return 0;
  return maestro::route_lists_bytes(n_models, n_nodes);
}

maestro_status maestro_route_sort_nodes(int32_t n_models, int32_t n_nodes, const double* free_bytes,
                                        const float* queue_s, const float* cold_s, const uint64_t* resident_mask,
                                        const float* act_s, void* lists, size_t lists_bytes, void* stream) {
  if (n_models < 1 || n_models > 64 || n_nodes < 1) return MAESTRO_ERR_INVALID_ARG;
  if (!free_bytes || !queue_s || !aligned(free_bytes, 8) || !aligned(queue_s, 4)) return MAESTRO_ERR_INVALID_ARG;
  if (act_s ? !aligned(act_s, 4)
            : (!cold_s || !resident_mask || !aligned(cold_s, 4) || !aligned(resident_mask, 8)))
    return MAESTRO_ERR_INVALID_ARG;
  const size_t need = maestro::route_lists_bytes(n_models, n_nodes);
  if (need == 0) return MAESTRO_ERR_UNSUPPORTED;
  if (!lists || !aligned(lists, 16) || lists_bytes < need) return MAESTRO_ERR_WORKSPACE;
  return maestro::launch_sort_nodes(n_models, n_nodes, free_bytes, queue_s, cold_s, resident_mask, act_s, lists,
                                    as_stream(stream));
}

maestro_status maestro_route_walk(int64_t n, const int32_t* model_id, const float* pred_len, const double* kv_bytes,
                                  const float* decode_s_per_token, int32_t n_models, int32_t n_nodes,
                                  const void* lists, size_t lists_bytes, double rho, int32_t k, int32_t* node_idx,
                                  float* score, void* stream) {
  if (n < 0 || n_models < 1 || n_models > 64 || n_nodes < 1 || k < 1 || k > 16) return MAESTRO_ERR_INVALID_ARG;
  if (!(rho >= 0.0) || rho == INFINITY) return MAESTRO_ERR_INVALID_ARG;
  if (!decode_s_per_token || !aligned(decode_s_per_token, 4)) return MAESTRO_ERR_INVALID_ARG;
  if (n > 0) {
    if (!model_id || !pred_len || !kv_bytes || !node_idx || !score) return MAESTRO_ERR_INVALID_ARG;
    if (!aligned(model_id, 4) || !aligned(pred_len, 4) || !aligned(kv_bytes, 8) || !aligned(node_idx, 4) ||
        !aligned(score, 4))
      return MAESTRO_ERR_INVALID_ARG;
  }
  if (n > (int64_t)1 << 37) return MAESTRO_ERR_UNSUPPORTED;
  const size_t need = maestro::route_lists_bytes(n_models, n_nodes);
  if (need == 0) return MAESTRO_ERR_UNSUPPORTED;
  if (!lists || !aligned(lists, 16) || lists_bytes < need) return MAESTRO_ERR_WORKSPACE;
  return maestro::launch_route_walk(n, model_id, pred_len, kv_bytes, decode_s_per_token, n_models, n_nodes, lists,
                                    rho, k, node_idx, score, as_stream(stream));
}

maestro_status maestro_route_fitness(int64_t n, const int32_t* model_id, const int32_t* src_id,
                                     const int32_t* class_id, const double* kv_bytes,
                                     int32_t n_models, int32_t n_nodes, int32_t n_src,
                                     int32_t n_classes, const double* free_bytes,
                                     const float* queue_ms, const float* act_ms,
                                     const uint64_t* resident_mask, const float* act_matrix,
                                     const float* deg_ms, const maestro_deg_plan* plans,
                                     const maestro_plan_step* plan_steps, const float* rtt_ms,
                                     const float* class_weights,
                                     const float* bounds, double rho, int32_t k, int32_t* node_idx,
                                     float* fitness, void* stream) {
  if (n < 0 || n_models < 1 || n_models > 64 || n_nodes < 1 || k < 1 || k > 16)
    return MAESTRO_ERR_INVALID_ARG;
  if (n_src < 1 || n_src > maestro::kMaxFitnessSources || n_classes < 1 ||
      n_classes > maestro::kMaxFitnessClasses)
    return MAESTRO_ERR_INVALID_ARG;
  if (!(rho >= 0.0) || rho == INFINITY) return MAESTRO_ERR_INVALID_ARG;
  if (!free_bytes || !queue_ms || !rtt_ms || !class_weights || !bounds) return MAESTRO_ERR_INVALID_ARG;
  if (!aligned(free_bytes, 8) || !aligned(queue_ms, 4) || !aligned(rtt_ms, 4) || !aligned(class_weights, 4) ||
      !aligned(bounds, 4))
    return MAESTRO_ERR_INVALID_ARG;
  if (act_matrix ? !aligned(act_matrix, 4)
                 : (!act_ms || !resident_mask || !aligned(act_ms, 4) || !aligned(resident_mask, 8)))
    return MAESTRO_ERR_INVALID_ARG;
  if (plans ? (!aligned(plans, 16) || !plan_steps || !aligned(plan_steps, 16)) : (!deg_ms || !aligned(deg_ms, 4)))
    return MAESTRO_ERR_INVALID_ARG;
  if (n > 0) {
    if (!model_id || !src_id || !class_id || !kv_bytes || !node_idx || !fitness)
      return MAESTRO_ERR_INVALID_ARG;
    if (!aligned(model_id, 4) || !aligned(src_id, 4) || !aligned(class_id, 4) ||
        !aligned(kv_bytes, 8) || !aligned(node_idx, 4) || !aligned(fitness, 4))
      return MAESTRO_ERR_INVALID_ARG;
  }
  if (n > (int64_t)1 << 37) return MAESTRO_ERR_UNSUPPORTED;
  return maestro::launch_route_fitness(n, model_id, src_id, class_id, kv_bytes, n_models, n_nodes, n_src, n_classes,
                                       free_bytes, queue_ms, act_ms, resident_mask, act_matrix, deg_ms,
                                       plans, plan_steps, rtt_ms, class_weights, bounds, rho, k, node_idx, fitness,
                                       as_stream(stream));
}

maestro_status maestro_degradation_plans(int32_t n_nodes, const int32_t* engine_offset,
                                         const int32_t* engine_level, const double* engine_freed_bytes,
                                         const float* engine_cost_ms, float c_int_ms, maestro_deg_plan* plans,
                                         maestro_plan_step* steps, void* stream) {
  if (n_nodes < 0 || !(c_int_ms == c_int_ms)) return MAESTRO_ERR_INVALID_ARG;
  if (n_nodes == 0) return MAESTRO_OK;
  if (!engine_offset || !plans || !steps || !aligned(engine_offset, 4) || !aligned(plans, 16) ||
      !aligned(steps, 16))
    return MAESTRO_ERR_INVALID_ARG;
  // the engine arrays may be empty (no node has an engine), then they may be NULL
  if (!aligned(engine_level, 4) || !aligned(engine_freed_bytes, 8) || !aligned(engine_cost_ms, 4))
    return MAESTRO_ERR_INVALID_ARG;
  return maestro::launch_degradation_plans(n_nodes, engine_offset, engine_level, engine_freed_bytes,
                                           engine_cost_ms, c_int_ms, plans, steps, as_stream(stream));
}

maestro_status maestro_activation_latency(int32_t n_nodes, int32_t n_models, const uint8_t* tier,
                                          const double* model_bytes, const double* tier_bw,
                                          const float* tier_setup, double unit, float* act, void* stream) {
  if (n_nodes < 0 || n_models < 1 || n_models > 64 || !(unit > 0.0) || !isfinite(unit))
    return MAESTRO_ERR_INVALID_ARG;
  if (!model_bytes || !tier_bw || !tier_setup || !aligned(model_bytes, 8) || !aligned(tier_bw, 8) ||
      !aligned(tier_setup, 4))
    return MAESTRO_ERR_INVALID_ARG;
  if (n_nodes > 0 && (!tier || !act || !aligned(act, 4))) return MAESTRO_ERR_INVALID_ARG;
  return maestro::launch_activation_latency(n_nodes, n_models, tier, model_bytes, tier_bw, tier_setup, unit, act,
                                            as_stream(stream));
}

size_t maestro_quantiles_workspace(int64_t m) {
  return (m >= 1 && m <= (int64_t)UINT32_MAX) ? maestro::quantiles_workspace_bytes(m) : 0;
}

maestro_status maestro_adaptive_rho(const double* kv_actual, const double* kv_pred, int64_t m, double beta,
                                    double q, float* ewma, float* rho, void* workspace, size_t workspace_bytes,
                                    void* stream) {
  if (m < 1 || !(beta > 0.0 && beta <= 1.0) || !(q >= 0.0 && q <= 1.0)) return MAESTRO_ERR_INVALID_ARG;
  if (!kv_actual || !kv_pred || !ewma || !rho || !aligned(kv_actual, 8) || !aligned(kv_pred, 8) ||
      !aligned(ewma, 4) || !aligned(rho, 4))
    return MAESTRO_ERR_INVALID_ARG;
  if (m > (int64_t)UINT32_MAX) return MAESTRO_ERR_UNSUPPORTED;
  const size_t need = maestro::quantiles_workspace_bytes(m);
  if (need > 0 && (!workspace || !aligned(workspace, 16) || workspace_bytes < need)) return MAESTRO_ERR_WORKSPACE;
  const int64_t rank = (int64_t)ceil(q * (double)(m - 1));
  return maestro::launch_adaptive_rho(kv_actual, kv_pred, m, beta, rank, ewma, rho, workspace, as_stream(stream));
}

maestro_status maestro_quantiles(const float* values, int64_t m, double q_lo, double q_hi, float* out,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  if (m < 1 || !(q_lo >= 0.0) || !(q_lo <= q_hi) || !(q_hi <= 1.0)) return MAESTRO_ERR_INVALID_ARG;
  if (!values || !out || !aligned(values, 4) || !aligned(out, 4)) return MAESTRO_ERR_INVALID_ARG;
  if (m > (int64_t)UINT32_MAX) return MAESTRO_ERR_UNSUPPORTED;
  const size_t need = maestro::quantiles_workspace_bytes(m);
  if (need > 0 && (!workspace || !aligned(workspace, 16) || workspace_bytes < need)) return MAESTRO_ERR_WORKSPACE;
  const int64_t r_lo = (int64_t)floor(q_lo * (double)(m - 1));
  const int64_t r_hi = (int64_t)ceil(q_hi * (double)(m - 1));
  return maestro::launch_quantiles(values, m, r_lo, r_hi, out, workspace, as_stream(stream));
}

maestro_status maestro_prioritize(int32_t n_workflows, int64_t n_stages,
                                  const int64_t* chain_offset, const float* stage_latency_s,
                                  const int32_t* cursor, const int64_t* deadline_us,
                                  int64_t now_us, int64_t* remaining_us, int32_t* slack_key,
                                  int32_t* order, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  if (n_workflows < 0 || n_stages < 0) return MAESTRO_ERR_INVALID_ARG;
  if (n_workflows == 0) return MAESTRO_OK;
  if (!chain_offset || !deadline_us || !slack_key || !order) return MAESTRO_ERR_INVALID_ARG;
  if (n_stages > 0 && !stage_latency_s) return MAESTRO_ERR_INVALID_ARG;
  if (!aligned(chain_offset, 8) || !aligned(deadline_us, 8) || !aligned(slack_key, 4) ||
      !aligned(order, 4) || !aligned(stage_latency_s, 4) || !aligned(cursor, 4) ||
      !aligned(remaining_us, 8))
    return MAESTRO_ERR_INVALID_ARG;
  const size_t need = maestro::prioritize_workspace_bytes(n_workflows, n_stages);
  if (workspace_bytes < need || !workspace || !aligned(workspace, 16)) return MAESTRO_ERR_WORKSPACE;
  return maestro::launch_prioritize(n_workflows, n_stages, chain_offset, stage_latency_s, cursor,
                                    deadline_us, now_us, remaining_us, slack_key, order,
                                    workspace, workspace_bytes, as_stream(stream));
}

maestro_status maestro_prioritize_noalloc(int32_t n_workflows, int64_t n_stages, const int64_t* chain_offset,
                                          const float* stage_latency_s, const int32_t* cursor,
                                          const int64_t* deadline_us, int64_t now_us, int64_t* remaining_us,
                                          int32_t* slack_key, int32_t* order, void* stream) {
  if (n_workflows < 0 || n_stages < 0) return MAESTRO_ERR_INVALID_ARG;
  if (n_workflows == 0) return MAESTRO_OK;
  if (n_workflows > MAESTRO_PRIORITIZE_NOALLOC_MAX_WORKFLOWS) return MAESTRO_ERR_WORKSPACE;
  const size_t need = maestro::prioritize_workspace_bytes(n_workflows, n_stages);
  if (need > MAESTRO_PRIORITIZE_NOALLOC_SCRATCH_BYTES) return MAESTRO_ERR_WORKSPACE;
  if (!chain_offset || !deadline_us || !slack_key || !order) return MAESTRO_ERR_INVALID_ARG;
  if (n_stages > 0 && !stage_latency_s) return MAESTRO_ERR_INVALID_ARG;
  if (!aligned(chain_offset, 8) || !aligned(deadline_us, 8) || !aligned(slack_key, 4) ||
      !aligned(order, 4) || !aligned(stage_latency_s, 4) || !aligned(cursor, 4) ||
      !aligned(remaining_us, 8))
    return MAESTRO_ERR_INVALID_ARG;
  void* scratch = nullptr;
  const maestro_status st = maestro::static_prioritize_scratch(&scratch);
  if (st != MAESTRO_OK) return st;
  return maestro::launch_prioritize(n_workflows, n_stages, chain_offset, stage_latency_s, cursor, deadline_us,
                                    now_us, remaining_us, slack_key, order, scratch,
                                    MAESTRO_PRIORITIZE_NOALLOC_SCRATCH_BYTES, as_stream(stream));
}

}  // extern "C"

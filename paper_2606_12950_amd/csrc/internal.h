// Internal launch interface of libmaestro (not part of the C-ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "maestro.h"

namespace maestro {

// Cost prediction: fused MLP + softmax + expected length + KV bytes.
maestro_status launch_predict(const maestro_predictor& p, int64_t n, const void* x,
                              const int32_t* prompt_len, const int32_t* model_id,
                              const float* kv_bytes_per_token, int32_t n_models, float* pred_len,
                              double* kv_bytes, hipStream_t stream);
bool predict_shape_supported(const maestro_predictor& p);
bool two_phase_shape_supported(const maestro_predictor& p);
maestro_status launch_predict_two_phase(const maestro_predictor& p, const maestro_two_phase& t, int64_t n,
                                        const void* x, const int32_t* prompt_len, const int32_t* model_id,
                                        const int32_t* role_id, const int32_t* tool_avail,
                                        const float* kv_bytes_per_token, int32_t n_models, float* p_tool,
                                        float* pred_len, double* kv_bytes, hipStream_t stream);

// Per-role regressors: bucketing by regressor, then the fused predictor as a grouped GEMM.
maestro_status launch_role_lengths(const maestro_predictor& p, const maestro_role_regressors& r, int64_t n,
                                   const void* x, const int32_t* prompt_len, const int32_t* model_id,
                                   const int32_t* role_id, const float* p_tool, const float* kv_bytes_per_token,
                                   int32_t n_models, float* pred_len, double* kv_bytes, void* workspace,
                                   hipStream_t stream);
size_t role_lengths_workspace_bytes(int64_t n, int32_t n_groups);
// rows of one tile of the role regressors' grouped launch for the predictor's shape
int32_t role_tile_rows(const maestro_predictor& p);
maestro_status launch_role_regressors(const maestro_predictor& p, int64_t n, const void* x, const float* coef,
                                      float max_len, const int32_t* tile_group, const int32_t* perm,
                                      const int32_t* prompt_p, const int32_t* model_p, const int32_t* p_bits,
                                      const int32_t* n_tiles, int64_t max_tiles, const float* kv_bytes_per_token,
                                      int32_t n_models, float* pred_len, double* kv_bytes, hipStream_t stream);

// Routing: feasibility mask, pair scores, lexicographic top-k.
maestro_status launch_route(int64_t n, const int32_t* model_id, const float* pred_len,
                            const double* kv_bytes, const float* decode_s_per_token,
                            int32_t n_models, int32_t n_nodes, const double* free_bytes,
                            const float* queue_s, const float* cold_s,
                            const uint64_t* resident_mask, const float* act_matrix, double rho, int32_t k,
                            int32_t algo, int32_t* node_idx, float* score, void* workspace,
                            size_t workspace_bytes, hipStream_t stream);
size_t route_workspace_bytes(int64_t n, int32_t n_models, int32_t n_nodes, int32_t k);
// the sorted route in two halves: per-model node lists, then the walk of every stage
size_t route_lists_bytes(int32_t n_models, int32_t n_nodes);
maestro_status launch_sort_nodes(int32_t n_models, int32_t n_nodes, const double* free_bytes, const float* queue_s,
                                 const float* cold_s, const uint64_t* resident_mask, const float* act_matrix,
                                 void* lists, hipStream_t stream);
maestro_status launch_route_walk(int64_t n, const int32_t* model_id, const float* pred_len, const double* kv_bytes,
                                 const float* decode_s_per_token, int32_t n_models, int32_t n_nodes,
                                 const void* lists, double rho, int32_t k, int32_t* node_idx, float* score,
                                 hipStream_t stream);

// Routing by fitness (Eq. 5) and the window bounds of its normalisation.
constexpr int kMaxFitnessSources = 16;
constexpr int kMaxFitnessClasses = 16;
maestro_status launch_route_fitness(int64_t n, const int32_t* model_id, const int32_t* src_id,
                                    const int32_t* class_id, const double* kv_bytes, int32_t n_models,
                                    int32_t n_nodes, int32_t n_src, int32_t n_classes, const double* free_bytes,
                                    const float* queue_ms, const float* act_ms,
                                    const uint64_t* resident_mask, const float* act_matrix, const float* deg_ms,
                                    const maestro_deg_plan* plans, const maestro_plan_step* plan_steps,
                                    const float* rtt_ms, const float* class_weights, const float* bounds, double rho,
                                    int32_t k, int32_t* node_idx, float* fitness, hipStream_t stream);
maestro_status launch_degradation_plans(int32_t n_nodes, const int32_t* engine_offset, const int32_t* engine_level,
                                       const double* engine_freed_bytes, const float* engine_cost_ms, float c_int_ms,
                                       maestro_deg_plan* plans, maestro_plan_step* steps, hipStream_t stream);
maestro_status launch_activation_latency(int32_t n_nodes, int32_t n_models, const uint8_t* tier,
                                         const double* model_bytes, const double* tier_bw,
                                         const float* tier_setup, double unit, float* act, hipStream_t stream);
maestro_status launch_adaptive_rho(const double* kv_actual, const double* kv_pred, int64_t m, double beta,
                                   int64_t rank, float* ewma, float* rho, void* workspace, hipStream_t stream);
maestro_status launch_quantiles(const float* values, int64_t m, int64_t r_lo, int64_t r_hi, float* out,
                                void* workspace, hipStream_t stream);
size_t quantiles_workspace_bytes(int64_t m);

// Prioritisation: chain suffix sums, slack keys, stable radix sort.
maestro_status launch_prioritize(int32_t n_workflows, int64_t n_stages,
                                 const int64_t* chain_offset, const float* stage_latency_s,
                                 const int32_t* cursor, const int64_t* deadline_us,
                                 int64_t now_us, int64_t* remaining_us, int32_t* slack_key,
                                 int32_t* order, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream);
size_t prioritize_workspace_bytes(int32_t n_workflows, int64_t n_stages);
// the static scratch of maestro_prioritize_noalloc on the current device
maestro_status static_prioritize_scratch(void** out);

inline maestro_status launch_status() {
  return hipGetLastError() == hipSuccess ? MAESTRO_OK : MAESTRO_ERR_LAUNCH;
}

}  // namespace maestro

/*
 * maestro.h -- C-ABI of the MI355X (gfx950) hot path of Maestro's scheduler:
 * the batched predict -> route -> prioritize step.
 *
 *   maestro_predict    cost prediction (Sec. III-B): predicted output length L of every stage
 *                      from a feature MLP over length bins (stand-in for the paper's trained
 *                      regressor), and its KV demand R_kv = alpha(M) * (P + L) (Eq. 3).
 *   maestro_predict_two_phase  the paper's two-phase form of the same prediction (Sec. III-B):
 *                      a calibrated tool-intent probability (Eq. 1), then the stage's role
 *                      head or the shared model on log(1 + L), fed that probability.
 *   maestro_predict_role_lengths  the per-role regressors with weights of their own, as one
 *                      grouped GEMM over the stages bucketed by role (Sec. III-B).
 *   maestro_route      cross-cluster routing (Sec. III-D, Alg. 3): drop nodes whose free KV
 *                      headroom cannot admit R_need = (1 + rho) * R_kv, score the rest by
 *                      expected completion latency T_q + T_act + t_dec(M) * L (Eq. 6 and the
 *                      decode term of Eq. 2), keep the best k (lowest index on equal scores).
 *   maestro_route_fitness  the same filter, then the node of largest fitness S = A - lambda
 *                      T_ready - mu C_deg (Eq. 5): affinity from network proximity and best fit
 *                      of R_need to the headroom, each metric normalised with window bounds
 *                      (maestro_quantiles computes them).
 *   maestro_prioritize remaining-time queue ordering (Sec. III-D, Eq. 7): remaining
 *                      predicted latency along each workflow chain, slack against the
 *                      workflow deadline, stable ascending order of workflows by slack.
 *
 * Conventions shared by every entry point
 *   - Every array argument is a DEVICE pointer owned by the caller. The library never
 *     allocates, frees or synchronises, and keeps no pointer after it returns.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream). All work is
 *     enqueued asynchronously on it; outputs are valid once the stream has been synchronised.
 *   - `workspace` is caller-owned, 16-byte aligned device scratch of at least the size the
 *     matching maestro_*_workspace() returns (NULL is allowed when that size is 0). Its
 *     contents on entry do not matter. Calls that share a workspace must not overlap in time.
 *   - Host-side checks only (scalars, pointers, alignment, sizes) happen before anything is
 *     enqueued; on failure the call returns MAESTRO_ERR_INVALID_ARG / _UNSUPPORTED /
 *     _WORKSPACE and has no effect. A failed launch returns MAESTRO_ERR_LAUNCH.
 *   - Per-stage ids are checked on the device, stage by stage: a model id outside
 *     [0, n_models) makes that stage's kv_bytes NaN in maestro_predict(_two_phase) (its length
 *     is still computed) and gives it no node in the routers (node -1, score +inf, fitness
 *     -inf), as does a source or class id out of range in maestro_route_fitness; no array is
 *     indexed out of bounds. Other per-element data is a precondition, not checked: finite
 *     inputs (stage latency excepted), monotone chain offsets.
 *   - Empty inputs (n = 0, n_workflows = 0) are valid no-ops that return MAESTRO_OK.
 *   - Entry points are re-entrant: the library has no mutable global state beyond the
 *     per-device address of maestro_prioritize_noalloc's static scratch (resolved once under
 *     a lock).
 */
#ifndef MAESTRO_H
#define MAESTRO_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define MAESTRO_API __attribute__((visibility("default")))
#else
#define MAESTRO_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum maestro_status {
  MAESTRO_OK = 0,
  MAESTRO_ERR_INVALID_ARG = 1,   /* null/misaligned pointer, out-of-range scalar */
  MAESTRO_ERR_UNSUPPORTED = 2,   /* valid shape the kernels are not built for */
  MAESTRO_ERR_WORKSPACE = 3,     /* workspace smaller than maestro_*_workspace() */
  MAESTRO_ERR_LAUNCH = 4         /* the HIP runtime rejected a launch */
} maestro_status;

typedef enum maestro_route_algo {
  MAESTRO_ROUTE_AUTO = 0,        /* SORTED when it applies and pays off, else SCAN */
  MAESTRO_ROUTE_SCAN = 1,        /* score every (stage, node) pair */
  MAESTRO_ROUTE_SORTED = 2       /* per-model node lists by ready time, early-exit walk;
                                    n_nodes <= 8192; needs maestro_route_workspace() bytes */
} maestro_route_algo;

typedef enum maestro_dtype {
  MAESTRO_F32 = 0,               /* features, weights and hidden layers in float32 */
  MAESTRO_BF16 = 1               /* bfloat16 storage, float32 accumulation */
} maestro_dtype;

/* The length predictor: n_layers Linear layers, ReLU between them, softmax over B length
 * bins at the end; the predicted length is the softmax-weighted mean of the bin centres.
 * Layer l maps dims[l] -> dims[l+1]: y = x * W_l^T + b_l with W_l stored [dims[l+1]][dims[l]]
 * row-major (out x in, device, element type `dtype`, 16-byte aligned) and b_l float32
 * [dims[l+1]] (device, 16-byte aligned). Hidden activations are stored in `dtype` after
 * bias + ReLU (round to nearest even for bfloat16); logits, softmax and the expected length
 * are float32.
 * Built shapes (others return MAESTRO_ERR_UNSUPPORTED):
 *   MAESTRO_F32,  2 layers: 64 -> 128 -> 32
 *   MAESTRO_BF16, 3 layers: 256 -> 512 -> 512 -> 64 and 256 -> 1024 -> 1024 -> 64 */
typedef struct maestro_predictor {
  int32_t n_layers;            /* number of Linear layers */
  int32_t dims[5];             /* dims[0] = D features, ..., dims[n_layers] = B bins */
  int32_t dtype;               /* maestro_dtype */
  const void* weight[4];       /* [dims[l+1]][dims[l]] per layer */
  const float* bias[4];        /* [dims[l+1]] per layer */
  const float* bin_centre;     /* [B] float32, 16-byte aligned: token count each bin stands for */
} maestro_predictor;

/* Cost prediction for n stages (Sec. III-B; Eq. 3).
 *   x                   [n][D] row-major, element type p->dtype, 16-byte aligned
 *   prompt_len          [n] int32: prompt tokens P of each stage
 *   model_id            [n] int32 in [0, n_models): the stage's model M(T), 1 <= n_models <= 64
 *   kv_bytes_per_token  [n_models] float32: alpha(M), KV bytes per token of each model
 *   pred_len  (out)     [n] float32: predicted output length L (tokens)
 *   kv_bytes  (out)     [n] float64: R_kv = ((double)P + (double)L) * (double)alpha(M);
 *                       exact in float64 for P < 2^16 and alpha < 2^19.
 * Needs no workspace (maestro_predict_workspace returns 0). */
MAESTRO_API maestro_status maestro_predict(const maestro_predictor* p, int64_t n, const void* x,
                               const int32_t* prompt_len, const int32_t* model_id,
                               const float* kv_bytes_per_token, int32_t n_models,
                               float* pred_len, double* kv_bytes,
                               void* workspace, size_t workspace_bytes, void* stream);

/* maestro_route_ex with T_act(N, M(T)) of Eq. 6 from readiness tiers: act_s [n_nodes][n_models]
 * float32 (seconds; maestro_activation_latency with unit = 1) replaces cold_s and
 * resident_mask, so score = fl32(fl32(queue_s[j] + act_s[j][m]) + fl32(pred_len[i] *
 * decode_s_per_token[m])). Same algorithms, workspace, outputs and errors as maestro_route_ex
 * (a NULL act_s is INVALID_ARG). */
MAESTRO_API maestro_status maestro_route_tiered(int64_t n, const int32_t* model_id, const float* pred_len,
                             const double* kv_bytes, const float* decode_s_per_token,
                             int32_t n_models, int32_t n_nodes, const double* free_bytes,
                             const float* queue_s, const float* act_s, double rho, int32_t k, int32_t algo,
                             int32_t* node_idx, float* score, void* workspace, size_t workspace_bytes,
                             void* stream);

/* The two-phase predictor (Sec. III-B). The network of a maestro_predictor (dims[n_layers] =
 * B = 64 outputs) is read as heads instead of bins: output 0 is the tool-intent logit z_0,
 * output g (1 <= g < B) the log(1 + L) regressor of head g; head 1 is the shared global model.
 *   n_roles     roles 0 .. n_roles-1 that map to a head, 0 <= n_roles <= 64
 *   role_head   [n_roles] int32 (device, may be NULL when n_roles = 0): the head of each role's
 *               own regressor; entries outside 1 .. B-1, and roles outside 0 .. n_roles-1,
 *               use head 1 (the fallback when a role has no regressor of its own)
 *   tool_coef   [B] float32 (device, 16-byte aligned): weight of the tool probability in each
 *               length head (entry 0 unused)
 *   n_knots     2 .. 64 knots of the isotonic calibration map
 *   iso_x/iso_y [n_knots] float32 (device): knots, iso_x strictly increasing, iso_y
 *               non-decreasing; the map is piecewise linear through them and constant beyond
 *               the first and the last
 *   max_len     upper clamp of the predicted length (tokens), finite and > 0 */
typedef struct maestro_two_phase {
  int32_t n_roles;
  int32_t n_knots;
  const int32_t* role_head;
  const float* tool_coef;
  const float* iso_x;
  const float* iso_y;
  float max_len;
} maestro_two_phase;

/* Two-phase cost prediction for n stages (Sec. III-B: Eq. 1, isotonic calibration, per-role
 * log(1 + L) regression; Eq. 3). Per stage, with z the network's B outputs (float32):
 *   p_tool = tool_avail != 0 ? iso(1 / (1 + exp(-z_0))) : 0      (Eq. 1, calibrated)
 *   g      = the head of the stage's role (see maestro_two_phase)
 *   L      = min(expm1(max(z_g + tool_coef[g] * p_tool, 0)), max_len)
 *   R_kv   = ((double)P + (double)L) * (double)alpha(M)            (Eq. 3)
 * Arguments as maestro_predict, plus
 *   role_id     [n] int32: the stage's agent role
 *   tool_avail  [n] int32: nonzero when tools are available to the stage
 *   p_tool (out)[n] float32, or NULL when not wanted
 * Built shapes: MAESTRO_BF16, 3 layers, 256 -> 512 -> 512 -> 64 and 256 -> 1024 -> 1024 -> 64
 * (others return MAESTRO_ERR_UNSUPPORTED). No workspace. Errors: INVALID_ARG for a NULL or
 * misaligned array, n < 0, n_models outside 1..64, n_roles outside 0..64, n_knots outside
 * 2..64, or max_len not finite and positive. */
MAESTRO_API maestro_status maestro_predict_two_phase(const maestro_predictor* p, const maestro_two_phase* tp,
                             int64_t n, const void* x, const int32_t* prompt_len,
                             const int32_t* model_id, const int32_t* role_id, const int32_t* tool_avail,
                             const float* kv_bytes_per_token, int32_t n_models, float* p_tool,
                             float* pred_len, double* kv_bytes, void* stream);

/* Per-role length regressors (Sec. III-B: a regressor of its own for each role with training
 * data, the shared global model for the others). Regressor g (0 <= g < n_regressors) is a
 * network of the predictor's shape with weights of its own; its output 0 regresses log(1 + L).
 *   n_regressors     1 .. MAESTRO_MAX_ROLE_REGRESSORS
 *   n_roles          0 .. 64 entries of role_regressor
 *   role_regressor   [n_roles] int32 (device; may be NULL when n_roles = 0): the regressor of
 *                    each role; entries outside 0 .. n_regressors-1, and roles outside
 *                    0 .. n_roles-1, mean none (the shared model's prediction stands)
 *   tool_coef        [n_regressors] float32 (device): weight of the tool probability
 *   max_len          upper clamp of the predicted length (tokens), finite and > 0 */
#define MAESTRO_MAX_ROLE_REGRESSORS 16
typedef struct maestro_role_regressors {
  int32_t n_regressors;
  int32_t n_roles;
  const int32_t* role_regressor;
  const float* tool_coef;
  float max_len;
} maestro_role_regressors;

/* The second phase's per-role regressors over n stages (Sec. III-B; Eq. 3), after
 * maestro_predict_two_phase has produced the calibrated tool probability and the shared model's
 * prediction of every stage. For each stage whose role has a regressor g:
 *   z      = regressor g's network on the stage's features (float32 outputs)
 *   L      = min(expm1(max(z_0 + tool_coef[g] * p_tool, 0)), max_len)
 *   R_kv   = ((double)P + (double)L) * (double)alpha(M)                    (Eq. 3)
 * written to pred_len and kv_bytes; every other stage's entries are left untouched.
 *   p                  the regressors' shape and weights: n_layers = 3, dtype MAESTRO_BF16, dims
 *                      256 -> 512 -> 512 -> 64 or 256 -> 1024 -> 1024 -> 64; weight[l] points at
 *                      the n_regressors networks' layer l stacked [g][dims[l+1]][dims[l]], bias[l]
 *                      at [g][dims[l+1]] (bin_centre unused)
 *   x, prompt_len, model_id, kv_bytes_per_token, n_models   as maestro_predict
 *   role_id            [n] int32: the stage's agent role
 *   p_tool             [n] float32: calibrated tool probability (from maestro_predict_two_phase)
 *   pred_len, kv_bytes [n] float32 / float64, in and out
 * The stages are bucketed by regressor on the device (a stable counting sort) and predicted as one
 * grouped GEMM: tiles of 128 stages of one regressor (256 for the 256-512-512-64 network),
 * feature rows gathered. Workspace:
 * maestro_role_lengths_workspace(n, n_regressors) bytes. Errors: INVALID_ARG for a NULL or
 * misaligned array, n < 0, n_models outside 1..64, n_regressors outside 1..16, n_roles outside
 * 0..64, max_len not finite and positive; UNSUPPORTED for another shape or n > 2^22 (the feature
 * rows are addressed with 31-bit offsets); WORKSPACE for a short workspace. */
MAESTRO_API maestro_status maestro_predict_role_lengths(const maestro_predictor* p, const maestro_role_regressors* r,
                             int64_t n, const void* x, const int32_t* prompt_len, const int32_t* model_id,
                             const int32_t* role_id, const float* p_tool, const float* kv_bytes_per_token,
                             int32_t n_models, float* pred_len, double* kv_bytes, void* workspace,
                             size_t workspace_bytes, void* stream);
MAESTRO_API size_t maestro_role_lengths_workspace(int64_t n, int32_t n_regressors);

/* Routing of n stages over n_nodes nodes (Sec. III-D; Alg. 3; Eq. 6; Eq. 2 decode term).
 * Per stage i with model m = model_id[i]:
 *   need  = rho == 0 ? kv_bytes[i] : kv_bytes[i] * (1 + rho)       (float64)
 *   node j is feasible iff need <= free_bytes[j]                     (equality admits)
 *   score = fl32( fl32(queue_s[j] + act) + fl32(pred_len[i] * decode_s_per_token[m]) )
 *           with act = 0 if bit m of resident_mask[j] is set, else cold_s[j]
 *   output the k feasible nodes with the smallest (score, j) in lexicographic order, i.e.
 *   ties go to the lowest node index; when fewer than k nodes are feasible the tail is
 *   padded with node -1 and score +inf.
 *   model_id            [n] int32 in [0, n_models), 1 <= n_models <= 64
 *   pred_len, kv_bytes  [n] float32 / float64 (from maestro_predict)
 *   decode_s_per_token  [n_models] float32: t_dec(M), seconds per output token
 *   free_bytes          [n_nodes] float64: KV admission headroom R_head (bytes)
 *   queue_s, cold_s     [n_nodes] float32: queueing delay T_q, cold-start latency T_act
 *   resident_mask       [n_nodes] uint64: bit m set <=> model m is warm on the node
 *   rho >= 0            safety margin;  1 <= k <= 16 route width
 *   node_idx  (out)     [n][k] int32;  score (out) [n][k] float32
 * Scores must be finite (finite inputs whose sums do not overflow float32).
 * Both algorithms return identical results. Workspace: maestro_route_workspace() bytes. */
MAESTRO_API maestro_status maestro_route(int64_t n, const int32_t* model_id, const float* pred_len,
                             const double* kv_bytes, const float* decode_s_per_token,
                             int32_t n_models, int32_t n_nodes, const double* free_bytes,
                             const float* queue_s, const float* cold_s,
                             const uint64_t* resident_mask, double rho, int32_t k,
                             int32_t* node_idx, float* score,
                             void* workspace, size_t workspace_bytes, void* stream);

/* maestro_route with an explicit algorithm (maestro_route_algo); SORTED with n_nodes > 8192
 * returns MAESTRO_ERR_UNSUPPORTED. */
MAESTRO_API maestro_status maestro_route_ex(int64_t n, const int32_t* model_id, const float* pred_len,
                             const double* kv_bytes, const float* decode_s_per_token,
                             int32_t n_models, int32_t n_nodes, const double* free_bytes,
                             const float* queue_s, const float* cold_s,
                             const uint64_t* resident_mask, double rho, int32_t k, int32_t algo,
                             int32_t* node_idx, float* score,
                             void* workspace, size_t workspace_bytes, void* stream);

/* The two halves of MAESTRO_ROUTE_SORTED (Sec. III-D; Alg. 3; Eq. 6), for callers that route
 * several batches against one node state, or that run the node half beside other work on a
 * second stream of the same priority and join it before the walk.
 * maestro_route_sort_nodes writes, for every model m, its n_nodes nodes in ascending order of
 * (ready time, node index), ready = fl32(queue_s[j] + act) with act as in maestro_route (0 when
 * bit m of resident_mask[j] is set, else cold_s[j]) or, when act_s is not NULL, act_s[j][m] as in
 * maestro_route_tiered (cold_s and resident_mask are then not read), each with its headroom
 * free_bytes[j], and after the lists, per model, the largest headroom of every block of 8, 64 and
 * 512 consecutive entries (rounded up to float32), which lets the walk skip nodes that cannot
 * admit its stage. `lists` is device memory of at least maestro_route_lists_bytes(n_models,
 * n_nodes) bytes, 16-byte aligned, owned by the caller, valid until the node state changes.
 * maestro_route_walk then gives every stage exactly the result of maestro_route_ex (or
 * maestro_route_tiered) with MAESTRO_ROUTE_SORTED on that node state; it reads only `lists` of
 * the node state. n_nodes <= 8192 (else MAESTRO_ERR_UNSUPPORTED; maestro_route_lists_bytes is
 * then 0); lists_bytes too small is MAESTRO_ERR_WORKSPACE; other arguments and errors as
 * maestro_route_ex. */
MAESTRO_API size_t maestro_route_lists_bytes(int32_t n_models, int32_t n_nodes);
MAESTRO_API maestro_status maestro_route_sort_nodes(int32_t n_models, int32_t n_nodes, const double* free_bytes,
                             const float* queue_s, const float* cold_s, const uint64_t* resident_mask,
                             const float* act_s, void* lists, size_t lists_bytes, void* stream);
MAESTRO_API maestro_status maestro_route_walk(int64_t n, const int32_t* model_id, const float* pred_len,
                             const double* kv_bytes, const float* decode_s_per_token,
                             int32_t n_models, int32_t n_nodes, const void* lists, size_t lists_bytes,
                             double rho, int32_t k, int32_t* node_idx, float* score, void* stream);

/* Minimum-impact degradation plans of a node (Alg. 2) and their disruption cost (Eq. 4), for
 * every possible shortfall. Alg. 2 takes the node's engines in priority order -- ascending
 * action level, the lower engine index first on equal levels -- and stops before the first
 * engine once the freed memory reaches the shortfall R, so its plan for R is the shortest prefix
 * of that order whose freed bytes reach R. A step p of a node describes the prefix made of its
 * first p + 1 engines in that order. */
typedef struct maestro_plan_step {
  double freed;      /* bytes freed by the prefix: the running sum in order (float64), kept
                        non-decreasing (the largest sum so far; the sum itself when no action
                        frees a negative amount)                                              */
  float cost;        /* its cost: the running sum of c(e, a) in order (float32), + c_int when
                        the prefix holds an engine of level 4 or 5                             */
  int32_t engine;    /* the engine taken at this step (index into the engine arrays)           */
} maestro_plan_step;

/* Per node, the first MAESTRO_PLAN_RECORD_STEPS steps in one 128-byte record (what the fitness
 * router stages on chip); a node with more engines continues in the step array. */
#define MAESTRO_PLAN_RECORD_STEPS 8
typedef struct maestro_deg_plan {
  double freed[MAESTRO_PLAN_RECORD_STEPS];  /* steps 0..7: freed; +inf past n_engines          */
  float cost[MAESTRO_PLAN_RECORD_STEPS];    /* steps 0..7: cost; 0 past n_engines              */
  int32_t n_engines;                        /* the node's engine count (any number >= 0)        */
  int32_t first_step;                       /* index of the node's step 0 in the step array    */
  int32_t reserved[6];                      /* 128-byte record                                 */
} maestro_deg_plan;

/* Plan records and steps of n_nodes nodes from their engine lists (CSR):
 *   engine_offset       [n_nodes + 1] int32, non-decreasing, engine_offset[0] = 0; node j owns
 *                       engines [engine_offset[j], engine_offset[j+1]), any number of them
 *   engine_level        [E] int32 in 1..5: the action Alg. 2 takes for the engine -- 1 an
 *                       idle-running model goes to sleep, 2 a sleeping model is evicted, 3 a
 *                       pending sleep is stopped, 4 an active model's KV is swapped out, 5 an
 *                       active execution is aborted (4 and 5 interrupt active work)
 *   engine_freed_bytes  [E] float64: memory the action frees (EstimateFreedMemory)
 *   engine_cost_ms      [E] float32: restoration latency of the action, c(e, a)
 *   c_int_ms            the interrupt penalty of Eq. 4 (the SLO violation threshold)
 *   plans (out)         [n_nodes] maestro_deg_plan, 16-byte aligned
 *   steps (out)         [E] maestro_plan_step, 16-byte aligned, E = engine_offset[n_nodes]:
 *                       node j's steps at [engine_offset[j], engine_offset[j+1]), in order
 * A shortfall R > 0 is met by the first step with freed >= R, at that step's cost; no such step
 * means the plan fails (the node cannot admit the stage). One thread per node: a node of up to
 * 8 engines is sorted in registers, a larger one by counting ranks (time quadratic in its
 * engine count). Device pointers, no workspace; n_nodes == 0 launches nothing. The engine
 * arrays may be NULL when E == 0. Errors: INVALID_ARG for n_nodes < 0, a NaN c_int_ms, a NULL
 * or misaligned offset, plan or step array, or a misaligned engine array. */
MAESTRO_API maestro_status maestro_degradation_plans(int32_t n_nodes, const int32_t* engine_offset,
                             const int32_t* engine_level, const double* engine_freed_bytes,
                             const float* engine_cost_ms, float c_int_ms, maestro_deg_plan* plans,
                             maestro_plan_step* steps, void* stream);

/* Routing by fitness (Sec. III-D: Eq. 5 with T_ready of Eq. 6; Alg. 3). Per stage i with
 * model m = model_id[i], source s = src_id[i] and weights (gamma, lambda, mu) =
 * class_weights[class_id[i]] (GetWeights of Alg. 3):
 *   need  = rho == 0 ? kv_bytes[i] : kv_bytes[i] * (1 + rho)       (float64)
 *   node j is feasible iff need <= free_bytes[j]                     (equality admits)
 *                      or, with plans, its plan meets the shortfall R = need - free_bytes[j]
 *   C_deg = deg_ms[j], or with plans: 0 when need <= free_bytes[j], else the plan's cost
 *   norm_X(x) = clamp((x - lo_X) / (hi_X - lo_X), 0, 1), or 0 when hi_X <= lo_X, with
 *               (lo_X, hi_X) the window bounds of metric X (see maestro_quantiles)
 *   prox  = 1 - norm_RTT(rtt_ms[s][j])                    network proximity
 *   fit   = fl32(need) / fl32(free_bytes[j])      best fit of R_need to the headroom, <= 1 on
 *           a feasible node (0 when fl32(free_bytes[j]) <= 0)
 *   A     = gamma * prox + (1 - gamma) * fit               affinity
 *   T_ready = queue_ms[j] + T_act,  T_act = act_matrix[j][m] when given, else
 *             (bit m of resident_mask[j] ? 0 : act_ms[j])                       (Eq. 6)
 *   S     = A - (lambda * norm_READY(T_ready) + mu * norm_DEG(C_deg))
 *   every operation float32 round-to-nearest, in exactly this order; output the k feasible
 *   nodes with the largest S, the lower node index first on equal S (the strict ">" of Alg.
 *   3); when fewer than k nodes are feasible the tail is padded with node -1 and -inf.
 *   model_id, src_id, class_id [n] int32: in [0, n_models), [0, n_src), [0, n_classes);
 *                              1 <= n_models <= 64, 1 <= n_src <= 16, 1 <= n_classes <= 16
 *   kv_bytes            [n] float64 R_kv (from maestro_predict)
 *   free_bytes          [n_nodes] float64: KV admission headroom R_head (bytes)
 *   queue_ms, act_ms    [n_nodes] float32: queueing delay T_q, activation latency T_act (ms)
 *   resident_mask       [n_nodes] uint64: bit m set <=> model m is warm on the node
 *   act_matrix          [n_nodes][n_models] float32 T_act of each model on each node (ms, e.g.
 *                       from maestro_activation_latency), or NULL; when given, act_ms and
 *                       resident_mask are unused (may be NULL)
 *   deg_ms              [n_nodes] float32: disruption penalty C_deg reported by the runtime (ms);
 *                       unused (may be NULL) when plans are given
 *   plans, plan_steps   [n_nodes] maestro_deg_plan and [E] maestro_plan_step from
 *                       maestro_degradation_plans (16-byte aligned), or both NULL; the byte
 *                       counts must be finite
 *   rtt_ms              [n_src][n_nodes] float32: round-trip time from each source (ms)
 *   class_weights       [n_classes][3] float32: (gamma, lambda, mu) per stage class
 *   bounds              [6] float32: (lo, hi) of RTT, T_ready, C_deg, in that order
 *   rho >= 0            safety margin;  1 <= k <= 16 route width
 *   node_idx  (out)     [n][k] int32;  fitness (out) [n][k] float32
 * All device arrays; inputs finite. No workspace. */
MAESTRO_API maestro_status maestro_route_fitness(int64_t n, const int32_t* model_id, const int32_t* src_id,
                             const int32_t* class_id, const double* kv_bytes, int32_t n_models,
                             int32_t n_nodes, int32_t n_src, int32_t n_classes,
                             const double* free_bytes, const float* queue_ms, const float* act_ms,
                             const uint64_t* resident_mask, const float* act_matrix, const float* deg_ms,
                             const maestro_deg_plan* plans, const maestro_plan_step* plan_steps,
                             const float* rtt_ms,
                             const float* class_weights, const float* bounds, double rho, int32_t k,
                             int32_t* node_idx, float* fitness, void* stream);

/* Model readiness (Sec. III-C): T_act of every model on every node from the readiness tier of
 * the node's copy of it -- 0 Running, 1 Sleeping, 2 CPU-resident, 3 Disk-resident, 4 Remote
 * (values past 4 count as Remote) -- with the profiled bandwidth model T_act = Size / BW_tier,
 * in the time unit that has `unit` counts per second (1000: ms for maestro_route_fitness; 1:
 * seconds for maestro_route_tiered):
 *   act[j][m] = tier == 0 ? 0 : fl32(tier_setup[t] + (model_bytes[m] / tier_bw[t]) * unit)
 * (float64 in that order).
 *   tier         [n_nodes][n_models] uint8
 *   model_bytes  [n_models] float64: weight bytes of each model
 *   tier_bw      [5] float64: bytes/s each tier loads at (entry 0 unused), > 0
 *   tier_setup   [5] float32: fixed activation overhead of each tier, in the output unit
 *   act (out)    [n_nodes][n_models] float32
 * Device arrays; 1 <= n_models <= 64, n_nodes >= 0 (0: no-op), unit finite and > 0. Errors:
 * INVALID_ARG for a NULL or misaligned array or a value out of range. */
MAESTRO_API maestro_status maestro_activation_latency(int32_t n_nodes, int32_t n_models, const uint8_t* tier,
                             const double* model_bytes, const double* tier_bw,
                             const float* tier_setup, double unit, float* act, void* stream);

/* Adaptive safety margin rho of R_need = (1 + rho) R_kv (Sec. III-D), from the last m stages
 * prediction errors in arrival order:
 *   e_i    = max(0, kv_actual[i] / kv_pred[i] - 1)                 relative underestimation
 *   s_0 = e_0,  s_i = beta e_i + (1 - beta) s_(i-1)                 EWMA (float64)
 *   ewma[i] = fl32(s_i)                                             (out, [m] float32)
 *   rho[0]  = the value of rank ceil(q (m - 1)) (0-based, ascending) among ewma[0 .. m-1]
 * kv_actual, kv_pred [m] float64 (device; kv_pred > 0, both finite); 0 < beta <= 1; 0 <= q <= 1
 * (a high quantile, 0.9 - 0.95). ewma doubles as the selection's input, and for windows longer
 * than 16,384 stages as the call's scratch (per-tile scan state in the first words of each
 * 8,192-stage range): its contents are defined once the stream reaches the call's end. The
 * float64 EWMA is a parallel scan, so ewma can differ from a sequential evaluation in the last
 * place. Workspace: maestro_quantiles_workspace(m) bytes (0 below 32,768 stages; NULL allowed
 * then). Errors: INVALID_ARG for m < 1, beta or q out of range, a NULL or misaligned array;
 * WORKSPACE for a workspace that is too small; UNSUPPORTED for m > 2^32 - 1. */
MAESTRO_API maestro_status maestro_adaptive_rho(const double* kv_actual, const double* kv_pred, int64_t m,
                             double beta, double q, float* ewma, float* rho, void* workspace,
                             size_t workspace_bytes, void* stream);

/* Window bounds of the robust normalisation in Eq. 5 (per-metric 5th/95th percentiles of a
 * recent window): out[0] and out[1] (device, float32) receive the values of rank
 * floor(q_lo * (m - 1)) and ceil(q_hi * (m - 1)) of values[0 .. m-1] (device, finite), ranks
 * counted from 0 in ascending order of the float values (-0 before +0); no interpolation.
 * 0 <= q_lo <= q_hi <= 1, 1 <= m < 2^32. Below 32,768 values one workgroup selects (no
 * workspace); from there on 256 workgroups count each 8-bit digit pass into histograms of
 * their own in the workspace (maestro_quantiles_workspace(m) bytes) and one workgroup picks
 * the bins, eight launches in all. WORKSPACE for a workspace that is too small. */
MAESTRO_API maestro_status maestro_quantiles(const float* values, int64_t m, double q_lo, double q_hi,
                             float* out, void* workspace, size_t workspace_bytes, void* stream);
/* Workspace bytes of maestro_quantiles and maestro_adaptive_rho over m values (0 when none is
 * needed, and for m outside 1 .. 2^32 - 1). */
MAESTRO_API size_t maestro_quantiles_workspace(int64_t m);

/* Slack ordering of n_workflows workflow chains over n_stages stages (Sec. III-D, Eq. 7).
 *   chain_offset        [n_workflows + 1] int64, chain_offset[0] = 0, non-decreasing,
 *                       chain_offset[W] = n_stages: stages of workflow w are
 *                       [chain_offset[w], chain_offset[w+1]) in chain order; a chain holds
 *                       at most 2^22 stages.
 *   stage_latency_s     [n_stages] float32 predicted latency of each stage (e.g. the routed
 *                       score); quantised to integer microseconds, round half to even,
 *                       clamped to +-2^40 us; a non-finite latency marks the stage (and every
 *                       earlier stage of its chain) as infinitely late.
 *   cursor              [n_workflows] int32 index of the next pending stage within each chain,
 *                       or NULL for all zero; negative counts as 0, >= chain length means
 *                       nothing remains.
 *   deadline_us         [n_workflows] int64;  now_us: current time (microseconds)
 *   remaining_us (out)  [n_stages] int64 or NULL: sum of the quantised latencies from the stage
 *                       to the end of its chain (INT64_MAX if infinitely late)
 *   slack_key (out)     [n_workflows] int32: deadline - now - remaining(head), exact, clamped
 *                       to int32; INT32_MIN when the remaining time is infinite
 *   order (out)         [n_workflows] int32: workflows sorted by ascending slack_key, equal keys
 *                       in increasing workflow index (stable).
 * Needs maestro_prioritize_workspace(n_workflows, n_stages) bytes of workspace. */
MAESTRO_API maestro_status maestro_prioritize(int32_t n_workflows, int64_t n_stages,
                                  const int64_t* chain_offset, const float* stage_latency_s,
                                  const int32_t* cursor, const int64_t* deadline_us,
                                  int64_t now_us, int64_t* remaining_us, int32_t* slack_key,
                                  int32_t* order, void* workspace, size_t workspace_bytes,
                                  void* stream);

/* maestro_prioritize for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same computation, outputs
 * and errors, with the radix sort's scratch in a static device array of
 * MAESTRO_PRIORITIZE_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on until
 * the process ends, so the call takes no workspace and allocates nothing. Batches of up to
 * MAESTRO_PRIORITIZE_NOALLOC_MAX_WORKFLOWS workflows; larger ones return MAESTRO_ERR_WORKSPACE
 * before anything is enqueued. The stream must belong to the current device; the first call with
 * a device current resolves that device's copy of the array (and returns MAESTRO_ERR_LAUNCH if
 * it cannot). Every call on one GPU shares that GPU's array and leaves its contents behind:
 * calls that overlap in time on one GPU (two streams, two host threads) race and give undefined
 * results; calls ordered on one stream do not. */
#define MAESTRO_PRIORITIZE_NOALLOC_MAX_WORKFLOWS (1 << 20)
#define MAESTRO_PRIORITIZE_NOALLOC_SCRATCH_BYTES ((size_t)17 << 20)
MAESTRO_API maestro_status maestro_prioritize_noalloc(int32_t n_workflows, int64_t n_stages,
                                  const int64_t* chain_offset, const float* stage_latency_s,
                                  const int32_t* cursor, const int64_t* deadline_us,
                                  int64_t now_us, int64_t* remaining_us, int32_t* slack_key,
                                  int32_t* order, void* stream);

/* Workspace sizes in bytes (0 = none needed). */
MAESTRO_API size_t maestro_predict_workspace(const maestro_predictor* p, int64_t n);
MAESTRO_API size_t maestro_route_workspace(int64_t n, int32_t n_models, int32_t n_nodes, int32_t k);
MAESTRO_API size_t maestro_prioritize_workspace(int32_t n_workflows, int64_t n_stages);

/* Static description of a status code. */
MAESTRO_API const char* maestro_status_string(maestro_status s);

#ifdef __cplusplus
}
#endif

#endif /* MAESTRO_H */

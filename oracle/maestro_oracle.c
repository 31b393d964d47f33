/*
 * CPU oracle for the batched predict -> route -> prioritize step of Maestro
 * (cost prediction, Sec. III-B; cross-cluster routing, Sec. III-D and Alg. 3;
 * remaining-time queue ordering, Sec. III-D, Eq. 7).
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE. Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library. It shares no code, header, table or
 * helper with the HIP library: it is a second, independent statement of what the hot path
 * computes, written to be read against the paper rather than to be fast.
 *
 * Plain definitions, no blocking, fusion or reordering of arithmetic:
 *   predict    : fp64 forward pass of the stand-in length predictor (a Linear/ReLU MLP over
 *                length bins), fp64 softmax, expected length = sum_b p_b * centre_b, then
 *                Eq. 3: R_kv = alpha(M) * (P + L). Hidden activations are rounded to the
 *                storage type (float32, or bfloat16 round-to-nearest-even) after bias and ReLU,
 *                as a network that stores its hidden layers in that type does.
 *   route      : the definition of "best feasible node" in Alg. 3, batched: keep nodes whose
 *                free bytes admit R_need = (1 + rho) * R_kv (FilterByPolicyAndFeasibility),
 *                score each with the expected completion latency T_q + T_act + t_dec * L
 *                (Eq. 6 plus the decode term of Eq. 2, RTT = eta = 0), and return the k
 *                smallest (score, node index) pairs in lexicographic order. The strict ">" of
 *                Alg. 3 keeps the first of equal scores, i.e. the lowest index.
 *   fitness    : Alg. 3 with the fitness of Eq. 5: among the feasible nodes, the largest
 *                S = A - (lambda T_ready + mu C_deg), A = gamma (1 - norm RTT) + (1 - gamma) fit,
 *                fit = R_need / headroom (best fit), T_ready = T_q + T_act (Eq. 6), each metric
 *                min-max normalised onto [0, 1] with window bounds, (x - lo) / (hi - lo), and
 *                clipped; float32 (every operation rounded to nearest) in that order; k best
 *                (fitness, lowest index). C_deg from engine lists is the cost (Eq. 4) of the
 *                shortest priority-ordered prefix of the node's engines that frees the
 *                shortfall (Alg. 2), any number of engines.
 *   two-phase  : the same network read as heads (Sec. III-B): a tool-intent logit through a
 *                sigmoid and an isotonic calibration table (Eq. 1), 0 without tools; the
 *                stage's role head (or the shared one) on log(1 + L), fed the calibrated
 *                probability, inverted with expm1; then Eq. 3.
 *   role regr. : per-role regressors with weights of their own (Sec. III-B): the stage's role
 *                network, output 0 on log(1 + L) plus the calibrated tool probability's term,
 *                inverted with expm1; then Eq. 3; stages of roles without one keep the shared
 *                model's prediction.
 *   quantiles  : the window bounds, as exact order statistics of a sample.
 *   prioritize : per-stage latency quantised to integer microseconds, suffix sums along each
 *                workflow chain (Eq. 7 with the future term taken as the sum of the later
 *                stages' predicted latencies), slack = deadline - now - remaining, clamped to
 *                int32, then a stable ascending sort of workflows by slack.
 *
 * Parallelism: OpenMP over independent stages only (predict, route); every stage's
 * arithmetic is the same sequential code whatever the thread count. prioritize is sequential.
 *
 * Build: gcc -O2 -fPIC -shared -fopenmp -ffp-contract=off (no fast-math), x86-64 SSE math.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#define ORACLE_OK 0
#define ORACLE_BAD_ARG 1
#define ORACLE_NO_MEM 2

/* Largest |latency| in microseconds a stage may carry (about 12.7 days); larger finite values
 * are clamped so that suffix sums of chains up to 2^22 stages stay exact in int64. */
#define LAT_US_LIMIT ((int64_t)1 << 40)
/* Marker of a non-finite (unroutable, infinitely late) latency; absorbing under addition. */
#define LAT_SAT INT64_MAX

/* ------------------------------------------------------------------------------------------ */
/* value conversions                                                                          */
/* ------------------------------------------------------------------------------------------ */

static double bf16_bits_to_double(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Round a double to the nearest bfloat16 value (8 significant bits, exponent range of
 * float32), ties to even, returned as a double. Written from the format's definition. */
double oracle_round_bf16(double v) {
  if (v == 0.0 || isnan(v) || isinf(v)) return v;
  double a = fabs(v);
  int e;
  frexp(a, &e);                    /* a = m * 2^e, m in [0.5, 1) */
  int q = e - 8;                   /* quantum 2^q keeps 8 significant bits */
  if (q < -133) q = -133;          /* subnormal bfloat16 quantum */
  double r = nearbyint(ldexp(a, -q)); /* default rounding mode: to nearest, ties to even */
  double out = ldexp(r, q);
  const double max_bf16 = ldexp(255.0, 120); /* (2 - 2^-7) * 2^127 */
  if (out > max_bf16) out = INFINITY;
  return v < 0 ? -out : out;
}

static double round_hidden(double v, int32_t dtype) {
  return dtype == 0 ? (double)(float)v : oracle_round_bf16(v);
}

static double stored_value(const void* base, int32_t dtype, int64_t idx) {
  if (dtype == 0) return (double)((const float*)base)[idx];
  return bf16_bits_to_double(((const uint16_t*)base)[idx]);
}

/* ------------------------------------------------------------------------------------------ */
/* predict: Sec. III-B (length predictor stand-in), Eq. 3 (KV demand)                        */
/* ------------------------------------------------------------------------------------------ */

/* The network's output layer for stage i: z_j = b_j + sum_k W[j][k] h_k (k ascending) layer by
 * layer from the stage's features, hidden layers through ReLU and stored in dtype. h and z hold
 * at least the widest layer. */
static void mlp_forward(int64_t i, int32_t n_layers, const int32_t* dims, int32_t dtype,
                        const void* const* weight, const float* const* bias, const void* x, double* h,
                        double* z) {
  const int32_t D = dims[0];
  for (int32_t k = 0; k < D; ++k) h[k] = stored_value(x, dtype, i * (int64_t)D + k);
  for (int l = 0; l < n_layers; ++l) {
    const int32_t din = dims[l], dout = dims[l + 1];
    for (int32_t j = 0; j < dout; ++j) {
      double acc = (double)bias[l][j];
      for (int32_t k = 0; k < din; ++k) acc += stored_value(weight[l], dtype, (int64_t)j * din + k) * h[k];
      z[j] = acc;
    }
    if (l + 1 < n_layers) {          /* hidden layer: ReLU, stored in dtype */
      for (int32_t j = 0; j < dout; ++j) h[j] = round_hidden(z[j] > 0.0 ? z[j] : 0.0, dtype);
    }
  }
}

int oracle_predict(int32_t n_layers, const int32_t* dims, int32_t dtype,
                   const void* const* weight, const float* const* bias,
                   const float* bin_centre, int64_t n, const void* x,
                   const int32_t* prompt_len, const int32_t* model_id,
                   const float* kv_bytes_per_token, int32_t n_models,
                   float* pred_len, double* kv_bytes, int32_t n_threads) {
  if (n_layers < 1 || n_layers > 4 || (dtype != 0 && dtype != 1) || n < 0 || n_models < 1)
    return ORACLE_BAD_ARG;
  int32_t widest = 0;
  for (int l = 0; l <= n_layers; ++l) {
    if (dims[l] < 1) return ORACLE_BAD_ARG;
    if (dims[l] > widest) widest = dims[l];
  }
  const int32_t B = dims[n_layers];
  int status = ORACLE_OK;
  if (n_threads < 1) n_threads = 1;

#pragma omp parallel num_threads(n_threads)
  {
    double* h = (double*)malloc(sizeof(double) * (size_t)widest);
    double* z = (double*)malloc(sizeof(double) * (size_t)widest);
    if (!h || !z) {
#pragma omp atomic write
      status = ORACLE_NO_MEM;
    } else {
#pragma omp for schedule(static)
      for (int64_t i = 0; i < n; ++i) {
        mlp_forward(i, n_layers, dims, dtype, weight, bias, x, h, z);
        /* softmax over bins (max-subtracted), expected length */
        double mu = z[0];
        for (int32_t b = 1; b < B; ++b) if (z[b] > mu) mu = z[b];
        double sum = 0.0;
        for (int32_t b = 0; b < B; ++b) sum += exp(z[b] - mu);
        double expect = 0.0;
        for (int32_t b = 0; b < B; ++b) expect += (exp(z[b] - mu) / sum) * (double)bin_centre[b];
        float pred = (float)expect;
        pred_len[i] = pred;
        /* Eq. 3: R_kv = alpha(M(T)) * (P(T) + L(T)) */
        int32_t m = model_id[i];
        double alpha = (m >= 0 && m < n_models) ? (double)kv_bytes_per_token[m] : NAN;
        kv_bytes[i] = ((double)prompt_len[i] + (double)pred) * alpha;
      }
    }
    free(h);
    free(z);
  }
  return status;
}

/* ------------------------------------------------------------------------------------------ */
/* two-phase predict: Sec. III-B (tool intent, Eq. 1; isotonic calibration; per-role         */
/* log(1+L) regressors), Eq. 3                                                                */
/* ------------------------------------------------------------------------------------------ */

/* Isotonic calibration map: the piecewise-linear function through the knots (x_j, y_j),
 * x strictly increasing, constant beyond the first and last knot. */
static double isotonic(double p, int32_t n_knots, const float* kx, const float* ky) {
  if (p <= (double)kx[0]) return (double)ky[0];
  if (p >= (double)kx[n_knots - 1]) return (double)ky[n_knots - 1];
  int32_t j = 0;                                   /* last knot at or below p */
  while (j + 1 < n_knots - 1 && (double)kx[j + 1] <= p) ++j;
  const double x0 = kx[j], x1 = kx[j + 1], y0 = ky[j], y1 = ky[j + 1];
  return y0 + (p - x0) * (y1 - y0) / (x1 - x0);
}

/* The network's output layer is read as B heads: output 0 is the tool-intent logit, output g
 * (1 <= g < B) the log(1 + L) regressor of head g; head 1 is the shared global model. A stage
 * of role r uses head role_head[r] (r in 0 .. n_roles-1, entry in 1 .. B-1), and the global
 * head otherwise.
 *   p_tool = has tools ? isotonic(sigmoid(z_0)) : 0                  (Eq. 1, calibrated)
 *   y      = z_g + tool_coef[g] * p_tool                               (p_tool feeds the regressor)
 *   L      = min(expm1(max(y, 0)), max_len)                            (inverse of log(1 + L))
 *   R_kv   = alpha(M) * (P + L)                                        (Eq. 3) */
int oracle_predict_two_phase(int32_t n_layers, const int32_t* dims, int32_t dtype,
                             const void* const* weight, const float* const* bias, int32_t n_roles,
                             const int32_t* role_head, const float* tool_coef, int32_t n_knots,
                             const float* iso_x, const float* iso_y, float max_len, int64_t n,
                             const void* x, const int32_t* prompt_len, const int32_t* model_id,
                             const int32_t* role_id, const int32_t* tool_avail,
                             const float* kv_bytes_per_token, int32_t n_models, float* p_tool,
                             float* pred_len, double* kv_bytes, int32_t n_threads) {
  if (n_layers < 1 || n_layers > 4 || (dtype != 0 && dtype != 1) || n < 0 || n_models < 1 ||
      n_roles < 0 || n_knots < 1)
    return ORACLE_BAD_ARG;
  int32_t widest = 0;
  for (int l = 0; l <= n_layers; ++l) {
    if (dims[l] < 1) return ORACLE_BAD_ARG;
    if (dims[l] > widest) widest = dims[l];
  }
  const int32_t B = dims[n_layers];
  if (B < 2) return ORACLE_BAD_ARG;
  int status = ORACLE_OK;
  if (n_threads < 1) n_threads = 1;

#pragma omp parallel num_threads(n_threads)
  {
    double* h = (double*)malloc(sizeof(double) * (size_t)widest);
    double* z = (double*)malloc(sizeof(double) * (size_t)widest);
    if (!h || !z) {
#pragma omp atomic write
      status = ORACLE_NO_MEM;
    } else {
#pragma omp for schedule(static)
      for (int64_t i = 0; i < n; ++i) {
        mlp_forward(i, n_layers, dims, dtype, weight, bias, x, h, z);
        /* phase 1: probability that the stage invokes a tool, calibrated; 0 without tools */
        double p = 0.0;
        if (tool_avail[i] != 0) p = isotonic(1.0 / (1.0 + exp(-z[0])), n_knots, iso_x, iso_y);
        /* phase 2: the role's length regressor (or the shared one) on log(1 + L) */
        const int32_t r = role_id[i];
        int32_t g = (r >= 0 && r < n_roles) ? role_head[r] : 1;
        if (g < 1 || g >= B) g = 1;
        const double y = z[g] + (double)tool_coef[g] * p;
        double L = expm1(y > 0.0 ? y : 0.0);
        if (L > (double)max_len) L = (double)max_len;
        const float pred = (float)L;
        p_tool[i] = (float)p;
        pred_len[i] = pred;
        int32_t m = model_id[i];
        double alpha = (m >= 0 && m < n_models) ? (double)kv_bytes_per_token[m] : NAN;
        kv_bytes[i] = ((double)prompt_len[i] + (double)pred) * alpha;
      }
    }
    free(h);
    free(z);
  }
  return status;
}

/* Per-role length regressors (Sec. III-B: a regressor per role where the role has training
 * data, the shared global model otherwise). Regressor g is a network of its own, the shape of
 * the predictor, with its weights stored after those of regressors 0 .. g-1 (layer l of
 * regressor g at weight[l] + g * dims[l+1] * dims[l], bias[l] + g * dims[l+1]). A stage of role
 * r with 0 <= role_group[r] < n_groups (r in 0 .. n_roles-1) is predicted by that regressor:
 *   y      = z_0 + tool_coef[g] * p_tool      (output 0 regresses log(1 + L); the calibrated tool
 *                                               probability of the first phase is an input)
 *   L      = min(expm1(max(y, 0)), max_len)
 *   R_kv   = alpha(M) * (P + L)                (Eq. 3)
 * Every other stage keeps pred_len and kv_bytes as they came in (the shared model's). */
int oracle_predict_role_lengths(int32_t n_layers, const int32_t* dims, int32_t dtype, int32_t n_groups,
                                const void* const* weight, const float* const* bias, int32_t n_roles,
                                const int32_t* role_group, const float* tool_coef, float max_len, int64_t n,
                                const void* x, const int32_t* prompt_len, const int32_t* model_id,
                                const int32_t* role_id, const float* p_tool, const float* kv_bytes_per_token,
                                int32_t n_models, float* pred_len, double* kv_bytes, int32_t n_threads) {
  if (n_layers < 1 || n_layers > 4 || (dtype != 0 && dtype != 1) || n < 0 || n_models < 1 || n_groups < 1 ||
      n_roles < 0)
    return ORACLE_BAD_ARG;
  int32_t widest = 0;
  for (int l = 0; l <= n_layers; ++l) {
    if (dims[l] < 1) return ORACLE_BAD_ARG;
    if (dims[l] > widest) widest = dims[l];
  }
  const size_t esize = dtype == 0 ? sizeof(float) : sizeof(uint16_t);
  int status = ORACLE_OK;
  if (n_threads < 1) n_threads = 1;

#pragma omp parallel num_threads(n_threads)
  {
    double* h = (double*)malloc(sizeof(double) * (size_t)widest);
    double* z = (double*)malloc(sizeof(double) * (size_t)widest);
    if (!h || !z) {
#pragma omp atomic write
      status = ORACLE_NO_MEM;
    } else {
#pragma omp for schedule(static)
      for (int64_t i = 0; i < n; ++i) {
        const int32_t r = role_id[i];
        const int32_t g = (r >= 0 && r < n_roles) ? role_group[r] : -1;
        if (g < 0 || g >= n_groups) continue;             /* the shared model's prediction stands */
        const void* wg[4];
        const float* bg[4];
        for (int l = 0; l < n_layers; ++l) {               /* regressor g's own layers */
          wg[l] = (const char*)weight[l] + (size_t)g * (size_t)dims[l + 1] * (size_t)dims[l] * esize;
          bg[l] = bias[l] + (size_t)g * (size_t)dims[l + 1];
        }
        mlp_forward(i, n_layers, dims, dtype, wg, bg, x, h, z);
        const double y = z[0] + (double)tool_coef[g] * (double)p_tool[i];
        double L = expm1(y > 0.0 ? y : 0.0);
        if (L > (double)max_len) L = (double)max_len;
        const float pred = (float)L;
        pred_len[i] = pred;
        const int32_t m = model_id[i];
        const double alpha = (m >= 0 && m < n_models) ? (double)kv_bytes_per_token[m] : NAN;
        kv_bytes[i] = ((double)prompt_len[i] + (double)pred) * alpha;
      }
    }
    free(h);
    free(z);
  }
  return status;
}

/* ------------------------------------------------------------------------------------------ */
/* route: Alg. 3 (filter + best node), Eq. 6 (T_ready), Eq. 2 decode term                    */
/* ------------------------------------------------------------------------------------------ */

typedef struct { float s; int32_t n; } cand_t;

static int cand_less(cand_t a, cand_t b) { return a.s < b.s || (a.s == b.s && a.n < b.n); }

int oracle_route(int64_t n, const int32_t* model_id, const float* pred_len,
                 const double* kv_bytes, const float* decode_s_per_token, int32_t n_models,
                 int32_t n_nodes, const double* free_bytes, const float* queue_s,
                 const float* cold_s, const uint64_t* resident_mask, const float* act_matrix,
                 double rho, int32_t k, int32_t* node_idx, float* score, int32_t n_threads) {
  if (n < 0 || n_nodes < 1 || n_models < 1 || n_models > 64 || k < 1 || rho < 0.0)
    return ORACLE_BAD_ARG;
  int status = ORACLE_OK;
  if (n_threads < 1) n_threads = 1;

#pragma omp parallel num_threads(n_threads)
  {
    cand_t* c = (cand_t*)malloc(sizeof(cand_t) * (size_t)n_nodes);
    unsigned char* taken = (unsigned char*)malloc((size_t)n_nodes);
    if (!c || !taken) {
#pragma omp atomic write
      status = ORACLE_NO_MEM;
    } else {
#pragma omp for schedule(static)
      for (int64_t i = 0; i < n; ++i) {
        const int32_t m = model_id[i];
        /* R_need = (1 + rho) * R_kv */
        const double need = (rho == 0.0) ? kv_bytes[i] : kv_bytes[i] * (1.0 + rho);
        /* decode term of Eq. 2: t_dec(M) * L, in float32 */
        const float exec_s = pred_len[i] * decode_s_per_token[m];
        int32_t nc = 0;
        for (int32_t nd = 0; nd < n_nodes; ++nd) {
          if (need > free_bytes[nd]) continue;              /* infeasible: not enough headroom */
          float act;                                        /* T_act of model m on the node */
          if (act_matrix) {                                 /* from its readiness tier */
            act = act_matrix[(int64_t)nd * n_models + m];
          } else {                                          /* cold start unless resident */
            const int resident = (int)((resident_mask[nd] >> (unsigned)m) & 1u);
            act = resident ? 0.0f : cold_s[nd];
          }
          const float ready = queue_s[nd] + act;            /* Eq. 6: T_ready = T_q + T_act */
          const float s = ready + exec_s;                   /* expected completion latency */
          c[nc].s = s;
          c[nc].n = nd;
          ++nc;
        }
        /* the k smallest (score, index) pairs in lexicographic order */
        memset(taken, 0, (size_t)nc);
        for (int32_t r = 0; r < k; ++r) {
          int32_t best = -1;
          for (int32_t j = 0; j < nc; ++j)
            if (!taken[j] && (best < 0 || cand_less(c[j], c[best]))) best = j;
          if (best >= 0) {
            taken[best] = 1;
            node_idx[i * k + r] = c[best].n;
            score[i * k + r] = c[best].s;
          } else {
            node_idx[i * k + r] = -1;
            score[i * k + r] = INFINITY;
          }
        }
      }
    }
    free(c);
    free(taken);
  }
  return status;
}

/* ------------------------------------------------------------------------------------------ */
/* route by fitness: Eq. 5 over the feasible nodes, Alg. 3 (argmax with strict ">")            */
/* ------------------------------------------------------------------------------------------ */

/* Model readiness (Sec. III-C): the activation latency of model m on a node whose copy of m is
 * in tier t -- 0 Running, 1 Sleeping, 2 CPU-resident, 3 Disk-resident, 4 Remote (tiers past 4
 * count as Remote) -- from the profiled bandwidth model T_act = Size / BW_tier, plus a fixed
 * per-tier setup time: 0 when Running, else setup[t] + (bytes[m] / bw[t]) * unit, in the unit
 * of time whose count per second is `unit` (1000 for ms, 1 for s), evaluated in float64 in
 * that order and stored as float32. */
int oracle_activation_latency(int32_t n_nodes, int32_t n_models, const uint8_t* tier,
                              const double* model_bytes, const double* tier_bw,
                              const float* tier_setup_ms, double unit, float* act_ms) {
  if (n_nodes < 0 || n_models < 1 || !(unit > 0.0)) return ORACLE_BAD_ARG;
  for (int64_t j = 0; j < (int64_t)n_nodes; ++j) {
    for (int32_t m = 0; m < n_models; ++m) {
      int t = tier[j * n_models + m];
      if (t > 4) t = 4;
      float a = 0.0f;
      if (t > 0) a = (float)((double)tier_setup_ms[t] + (model_bytes[m] / tier_bw[t]) * unit);
      act_ms[j * n_models + m] = a;
    }
  }
  return ORACLE_OK;
}

/* Adaptive safety margin (Sec. III-D): the relative underestimation e = max(0, R_kv / R^_kv - 1)
 * of each of the last m stages (arrival order), its EWMA e~_i = beta e_i + (1 - beta) e~_(i-1)
 * starting from e~_0 = e_0 (float64, sequential), stored as float32; rho = the value of rank
 * ceil(q (m - 1)) (0-based, ascending) among the stored EWMA values. */
static int f32_cmp(const void* pa, const void* pb) {
  const float a = *(const float*)pa, b = *(const float*)pb;
  return (a > b) - (a < b);
}

int oracle_adaptive_rho(const double* kv_actual, const double* kv_pred, int64_t m, double beta, double q,
                        float* ewma, float* rho) {
  if (m < 1 || !(beta > 0.0 && beta <= 1.0) || !(q >= 0.0 && q <= 1.0)) return ORACLE_BAD_ARG;
  double s = 0.0;
  for (int64_t i = 0; i < m; ++i) {
    double e = kv_actual[i] / kv_pred[i] - 1.0;      /* relative underestimation */
    if (!(e > 0.0)) e = 0.0;
    s = (i == 0) ? e : beta * e + (1.0 - beta) * s;  /* EWMA */
    ewma[i] = (float)s;
  }
  float* sorted = (float*)malloc(sizeof(float) * (size_t)m);
  if (!sorted) return ORACLE_NO_MEM;
  memcpy(sorted, ewma, sizeof(float) * (size_t)m);
  qsort(sorted, (size_t)m, sizeof(float), f32_cmp);
  const int64_t r = (int64_t)ceil(q * (double)(m - 1));   /* a high quantile, no interpolation */
  *rho = sorted[r];
  free(sorted);
  return ORACLE_OK;
}

/* Robust min-max normalisation (Sec. III-D): (x - lo) / (hi - lo) clipped to [0, 1], with the
 * window bounds lo, hi of the metric; a degenerate window (hi <= lo) maps everything to 0.
 * float32 subtraction and division, each rounded to nearest. */
static float norm01(float x, float lo, float hi) {
  if (!(hi > lo)) return 0.0f;
  float t = (x - lo) / (hi - lo);
  if (t < 0.0f) t = 0.0f;
  if (t > 1.0f) t = 1.0f;
  return t;
}

/* The minimum-impact plan of Alg. 2 and its cost, Eq. 4, on one node. The greedy loop of Alg. 2
 * takes engines in priority order (ascending action level 1..5, the lower engine index first on
 * equal levels) and stops before the first engine once the freed memory reaches
 * R, so the plan it returns is the shortest prefix of that order whose freed bytes (summed in
 * float64, in order) reach R -- the empty prefix when R <= 0 -- and it fails when even the whole
 * order frees less. The plan's cost is the float32 sum, in order, of its engines' restoration
 * latencies c(e, a), plus c_int when it holds an engine of level 4 or 5 (the active work of that
 * engine is preempted or aborted). Returns 0 with the cost in *c_deg, or 1 when no prefix frees
 * enough. */
typedef struct { int32_t level, idx; } eng_t;
static int eng_cmp(const void* pa, const void* pb) {
  const eng_t* a = (const eng_t*)pa;
  const eng_t* b = (const eng_t*)pb;
  if (a->level != b->level) return a->level < b->level ? -1 : 1;
  return (a->idx > b->idx) - (a->idx < b->idx);
}

static int degradation_plan(double R, int32_t e0, int32_t e1, const int32_t* level, const double* freed,
                            const float* cost, float c_int, float* c_deg) {
  const int32_t ne = e1 > e0 ? e1 - e0 : 0;
  eng_t* order = (eng_t*)malloc(sizeof(eng_t) * (size_t)(ne > 0 ? ne : 1));
  double* sum = (double*)malloc(sizeof(double) * (size_t)(ne + 1));
  if (!order || !sum) abort();
  for (int32_t i = 0; i < ne; ++i) {
    order[i].level = level[e0 + i];
    order[i].idx = e0 + i;
  }
  qsort(order, (size_t)ne, sizeof(eng_t), eng_cmp);     /* priority order */
  sum[0] = 0.0;                                         /* freed bytes of the first p engines */
  for (int32_t p = 1; p <= ne; ++p) sum[p] = sum[p - 1] + freed[order[p - 1].idx];
  int32_t len = -1;                                     /* the shortest prefix reaching R */
  for (int32_t p = 0; p <= ne && len < 0; ++p)
    if (sum[p] >= R) len = p;
  int status = 1;                                       /* no plan */
  if (len >= 0) {
    float total = 0.0f;
    int interrupt = 0;
    for (int32_t p = 0; p < len; ++p) {
      total += cost[order[p].idx];
      if (order[p].level >= 4) interrupt = 1;
    }
    *c_deg = total + (interrupt ? c_int : 0.0f);
    status = 0;
  }
  free(order);
  free(sum);
  return status;
}

int oracle_degradation_cost(double R, int32_t n_engines, const int32_t* level, const double* freed,
                            const float* cost, float c_int, float* c_deg) {
  return degradation_plan(R, 0, n_engines, level, freed, cost, c_int, c_deg);
}

typedef struct { float s; int32_t n; } fcand_t;
/* larger fitness first; equal fitness: lower node index first (the strict ">" of Alg. 3) */
static int fcand_better(fcand_t a, fcand_t b) { return a.s > b.s || (a.s == b.s && a.n < b.n); }

int oracle_route_fitness(int64_t n, const int32_t* model_id, const int32_t* src_id,
                         const int32_t* class_id, const double* kv_bytes, int32_t n_models,
                         int32_t n_nodes, int32_t n_src, int32_t n_classes,
                         const double* free_bytes, const float* queue_ms, const float* act_ms,
                         const uint64_t* resident_mask, const float* act_matrix, const float* deg_ms,
                         const float* rtt_ms, const float* class_weights, const float* bounds, double rho,
                         int32_t k, const int32_t* engine_offset, const int32_t* engine_level,
                         const double* engine_freed, const float* engine_cost, float c_int,
                         int32_t* node_idx, float* fitness, int32_t n_threads) {
  if (n < 0 || n_nodes < 1 || n_models < 1 || n_models > 64 || n_src < 1 || n_classes < 1 ||
      k < 1 || rho < 0.0)
    return ORACLE_BAD_ARG;
  int status = ORACLE_OK;
  if (n_threads < 1) n_threads = 1;
  /* window bounds (lo, hi) of the three normalised metrics: RTT, T_ready, C_deg (milliseconds)
   * are bounds[0..1], bounds[2..3], bounds[4..5] */

#pragma omp parallel num_threads(n_threads)
  {
    fcand_t* c = (fcand_t*)malloc(sizeof(fcand_t) * (size_t)n_nodes);
    unsigned char* taken = (unsigned char*)malloc((size_t)n_nodes);
    if (!c || !taken) {
#pragma omp atomic write
      status = ORACLE_NO_MEM;
    } else {
#pragma omp for schedule(static)
      for (int64_t i = 0; i < n; ++i) {
        const int32_t m = model_id[i];
        /* R_need = (1 + rho) * R_kv */
        const double need = (rho == 0.0) ? kv_bytes[i] : kv_bytes[i] * (1.0 + rho);
        /* GetWeights(T.class): network weight gamma, lambda (T_ready), mu (C_deg) */
        const float* wt = class_weights + 3 * (size_t)class_id[i];
        const float gamma = wt[0], lambda = wt[1], mu = wt[2];
        const float* rtt_row = rtt_ms + (size_t)src_id[i] * (size_t)n_nodes;
        const float needf = (float)need;
        int32_t nc = 0;
        for (int32_t nd = 0; nd < n_nodes; ++nd) {
          /* FilterByPolicyAndFeasibility; C_deg as the runtime reports it: per node, or, with
           * engine lists, the cost of the minimum-impact plan for the shortfall (Alg. 2, Eq. 4),
           * 0 when the stage fits, and the node infeasible when no plan frees enough */
          float c_deg;
          if (engine_offset) {
            if (need <= free_bytes[nd]) {
              c_deg = 0.0f;
            } else if (degradation_plan(need - free_bytes[nd], engine_offset[nd], engine_offset[nd + 1],
                                        engine_level, engine_freed, engine_cost, c_int, &c_deg)) {
              continue;
            }
          } else {
            if (need > free_bytes[nd]) continue;
            c_deg = deg_ms[nd];
          }
          /* Affinity: network proximity (decreasing in the normalised RTT) and best fit of
           * R_need to the node's headroom, R_need / headroom (1 when the stage fills the
           * headroom, at most 1 on a feasible node; a node without headroom admits only an
           * empty demand and gets 0) */
          const float prox = 1.0f - norm01(rtt_row[nd], bounds[0], bounds[1]);
          const float freef = (float)free_bytes[nd];
          const float fit = freef > 0.0f ? needf / freef : 0.0f;
          const float a = gamma * prox + (1.0f - gamma) * fit;
          /* RuntimeEstimate: T_ready = T_q + T_act (Eq. 6): T_act of model m on this node from the
           * per-(node, model) matrix, or else the node's activation latency unless m is resident */
          float act;
          if (act_matrix) {
            act = act_matrix[(int64_t)nd * n_models + m];
          } else {
            const int resident = (int)((resident_mask[nd] >> (unsigned)m) & 1u);
            act = resident ? 0.0f : act_ms[nd];
          }
          const float ready = queue_ms[nd] + act;
          /* Eq. 5 on normalised metrics: S = A - (lambda * T_ready + mu * C_deg), the two
           * penalties summed before they are taken from the affinity */
          const float penalty =
              lambda * norm01(ready, bounds[2], bounds[3]) + mu * norm01(c_deg, bounds[4], bounds[5]);
          const float s = a - penalty;
          c[nc].s = s;
          c[nc].n = nd;
          ++nc;
        }
        /* the k best (fitness, index) pairs: largest fitness, then lowest index */
        memset(taken, 0, (size_t)nc);
        for (int32_t r = 0; r < k; ++r) {
          int32_t best = -1;
          for (int32_t j = 0; j < nc; ++j)
            if (!taken[j] && (best < 0 || fcand_better(c[j], c[best]))) best = j;
          if (best >= 0) {
            taken[best] = 1;
            node_idx[i * k + r] = c[best].n;
            fitness[i * k + r] = c[best].s;
          } else {
            node_idx[i * k + r] = -1;
            fitness[i * k + r] = -INFINITY;
          }
        }
      }
    }
    free(c);
    free(taken);
  }
  return status;
}

/* Window bounds of the robust normalisation: the order statistics of rank floor(q_lo (m-1))
 * and ceil(q_hi (m-1)) of m finite values (no interpolation). */
static int float_cmp(const void* pa, const void* pb) {
  const float a = *(const float*)pa, b = *(const float*)pb;
  if (a < b) return -1;
  if (a > b) return 1;
  /* -0 before +0, so that the order is total on bit patterns */
  const int sa = signbit(a) ? 1 : 0, sb = signbit(b) ? 1 : 0;
  return sb - sa;
}

int oracle_quantiles(const float* values, int64_t m, double q_lo, double q_hi, float* out) {
  if (m < 1 || !(q_lo >= 0.0 && q_lo <= q_hi && q_hi <= 1.0)) return ORACLE_BAD_ARG;
  float* v = (float*)malloc(sizeof(float) * (size_t)m);
  if (!v) return ORACLE_NO_MEM;
  memcpy(v, values, sizeof(float) * (size_t)m);
  qsort(v, (size_t)m, sizeof(float), float_cmp);
  const int64_t i_lo = (int64_t)floor(q_lo * (double)(m - 1));
  const int64_t i_hi = (int64_t)ceil(q_hi * (double)(m - 1));
  out[0] = v[i_lo];
  out[1] = v[i_hi];
  free(v);
  return ORACLE_OK;
}

/* ------------------------------------------------------------------------------------------ */
/* prioritize: Eq. 7 remaining time along a chain, slack against the workflow deadline        */
/* ------------------------------------------------------------------------------------------ */

/* seconds (float32) -> integer microseconds, round half to even; non-finite -> LAT_SAT */
int64_t oracle_latency_us(float lat_s) {
  if (!isfinite(lat_s)) return LAT_SAT;
  double us = nearbyint((double)lat_s * 1.0e6);
  if (us > (double)LAT_US_LIMIT) us = (double)LAT_US_LIMIT;
  if (us < -(double)LAT_US_LIMIT) us = -(double)LAT_US_LIMIT;
  return (int64_t)us;
}

static int64_t sat_add(int64_t a, int64_t b) {
  return (a == LAT_SAT || b == LAT_SAT) ? LAT_SAT : a + b;
}

typedef struct { int32_t key; int32_t idx; } keyed_t;

static int keyed_cmp(const void* pa, const void* pb) {
  const keyed_t* a = (const keyed_t*)pa;
  const keyed_t* b = (const keyed_t*)pb;
  if (a->key != b->key) return a->key < b->key ? -1 : 1;
  return (a->idx > b->idx) - (a->idx < b->idx);  /* equal keys keep workflow order */
}

int oracle_prioritize(int32_t n_workflows, int64_t n_stages, const int64_t* chain_offset,
                      const float* stage_latency_s, const int32_t* cursor,
                      const int64_t* deadline_us, int64_t now_us, int64_t* remaining_us,
                      int32_t* slack_key, int32_t* order) {
  if (n_workflows < 0 || n_stages < 0) return ORACLE_BAD_ARG;
  if (n_workflows == 0) return ORACLE_OK;
  if (chain_offset[0] != 0 || chain_offset[n_workflows] != n_stages) return ORACLE_BAD_ARG;
  for (int32_t w = 0; w < n_workflows; ++w)
    if (chain_offset[w + 1] < chain_offset[w]) return ORACLE_BAD_ARG;

  int64_t* rem = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n_stages > 0 ? n_stages : 1));
  keyed_t* kv = (keyed_t*)malloc(sizeof(keyed_t) * (size_t)n_workflows);
  if (!rem || !kv) { free(rem); free(kv); return ORACLE_NO_MEM; }

  for (int32_t w = 0; w < n_workflows; ++w) {
    const int64_t first = chain_offset[w], end = chain_offset[w + 1];
    /* remaining time from stage j to the end of its chain: this stage plus every later one */
    int64_t suffix = 0;
    for (int64_t j = end - 1; j >= first; --j) {
      suffix = sat_add(oracle_latency_us(stage_latency_s[j]), suffix);
      rem[j] = suffix;
    }
    int64_t cur = cursor ? (int64_t)cursor[w] : 0;
    if (cur < 0) cur = 0;
    const int64_t r = (first + cur < end) ? rem[first + cur] : 0;  /* finished chain: 0 */
    int32_t key;
    if (r == LAT_SAT) {
      key = INT32_MIN;                              /* unroutable: most urgent */
    } else {
      __int128 slack = (__int128)deadline_us[w] - (__int128)now_us - (__int128)r;
      if (slack > (__int128)INT32_MAX) key = INT32_MAX;
      else if (slack < (__int128)INT32_MIN) key = INT32_MIN;
      else key = (int32_t)slack;
    }
    slack_key[w] = key;
    kv[w].key = key;
    kv[w].idx = w;
  }
  if (remaining_us) memcpy(remaining_us, rem, sizeof(int64_t) * (size_t)n_stages);

  qsort(kv, (size_t)n_workflows, sizeof(keyed_t), keyed_cmp);
  for (int32_t w = 0; w < n_workflows; ++w) order[w] = kv[w].idx;

  free(rem);
  free(kv);
  return ORACLE_OK;
}

int oracle_max_threads(void) { return omp_get_max_threads(); }

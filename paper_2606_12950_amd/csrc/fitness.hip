// Routing by fitness (Sec. III-D, Eq. 5 with Eq. 6; Alg. 3) and the window bounds of its robust
// normalisation.
//
// For every stage, among the nodes whose headroom admits R_need = (1 + rho) R_kv, the largest
//   S = A - (lambda * norm(T_ready) + mu * norm(C_deg)),
//   A = gamma * (1 - norm(RTT(src, node))) + (1 - gamma) * fit,  fit = R_need / headroom,
//   T_ready = T_q + T_act (T_act = 0 when the stage's model is resident),
// with the class weights (gamma, lambda, mu) of the stage and norm(x) = clamp((x - lo) / (hi - lo),
// 0, 1) over window bounds (lo, hi) per metric (a degenerate window normalises to 0). The k best
// (fitness, node) pairs are kept, larger fitness first and the lower index on equal fitness
// (the strict ">" of Alg. 3). Every operation is float32 rounded to nearest, in that order.
//
// A workgroup takes 256 stages (one per thread), 512 for large batches (two per thread, which
// then share every node read), or 256 / G when a small batch gives each stage G lanes. It
// stages node state chunk by chunk in LDS, with everything that depends on the node alone
// already evaluated: the normalised metrics (true divisions, once per node), the headroom and
// its float64 reciprocal, 1 - norm(RTT) from every source and, with residency bits, the penalty
// lambda * norm(T_ready) + mu * norm(C_deg) of every stage class for both residency states. A
// pair then costs the feasibility test, the fit, the affinity and one subtraction.
//
// The fit is fl32(fl32(R_need) / fl32(headroom)) -- at most 1 on a feasible node, since R_need <=
// headroom survives the rounding to float32; 0 on a node without headroom -- computed as the
// float64 product of fl32(R_need)
// with the float64 reciprocal of fl32(headroom), rounded once to float32. For float32 operands
// a and b that product is within 2^-52 (relative) of a / b, while a / b lies at least 2^-49
// (relative) away from every float32 rounding boundary (a midpoint has a 25-bit significand, so
// a - midpoint * b, a nonzero multiple of the operands' least significant bits, cannot vanish),
// hence the rounding gives the correctly rounded float32 quotient -- the division itself.
//
// With degradation plans (Alg. 2, Eq. 4), C_deg is per pair: 0 when the stage fits, else the
// cost of the shortest priority prefix of the node's engines that frees the shortfall, and the
// node drops out when no prefix does. The first eight steps of each node's plan are staged in
// LDS, column by column, with the other node terms; a node with more engines continues in the
// step array in global memory (binary search). The main loop scores every pair as if it fit and
// only queues the short ones; a lane then scores its queued nodes against their plans after
// each chunk. A short pair whose fitness bound (its score with C_deg normalised to 0) cannot
// enter the stage's top-k is dropped without a plan lookup.
//
// The window bounds are exact order statistics of a sample (no interpolation): one workgroup
// radix-selects both ranks at once, 8 bits per pass over the order-preserving integer image.
// The adaptive margin (Sec. III-D) reuses that selection on an EWMA of the window's relative
// underestimation, computed as a scan of affine maps.
#include <type_traits>

#include "internal.h"
#include "select.h"

namespace maestro {
namespace {

constexpr int kThreads = 256;
constexpr int kRecSteps = MAESTRO_PLAN_RECORD_STEPS;

// (x - lo) / (hi - lo) clipped to [0, 1]; 0 for a degenerate window
__device__ __forceinline__ float norm01(float x, float lo, float hi) {
  if (!(hi > lo)) return 0.0f;
  float t = __fdiv_rn(__fsub_rn(x, lo), __fsub_rn(hi, lo));
  if (t < 0.0f) t = 0.0f;
  if (t > 1.0f) t = 1.0f;
  return t;
}

// Plan steps and records from the engine lists, one thread per node. SortByPriority orders the
// engines by ascending level, the lower engine index first: up to eight engines with a fixed
// compare-exchange network over keys level:index in registers, more by counting each engine's
// rank among the node's keys (the keys are distinct). The running sums then follow that order:
// freed bytes in float64, costs in float32, and c_int added to every prefix that holds an engine
// of level 4 or 5. The freed column keeps the largest running sum so far, so it never decreases
// (it is the running sum itself when no action frees a negative amount): the first prefix whose
// running sum reaches a shortfall is then also the first whose entry does, which a stage finds
// by counting (record) or by binary search (steps). Record entries past the node's engines hold
// +inf.
__device__ __forceinline__ int64_t engine_key(int32_t level, int32_t i) {
  return (int64_t)level * ((int64_t)1 << 32) + (int64_t)(uint32_t)i;
}

__global__ __launch_bounds__(kThreads) void plan_kernel(int32_t n_nodes, const int32_t* __restrict__ engine_offset,
                                                        const int32_t* __restrict__ engine_level,
                                                        const double* __restrict__ engine_freed,
                                                        const float* __restrict__ engine_cost, float c_int,
                                                        maestro_deg_plan* __restrict__ plans,
                                                        maestro_plan_step* __restrict__ steps) {
  const int32_t j = blockIdx.x * kThreads + threadIdx.x;
  if (j >= n_nodes) return;
  const int32_t e0 = engine_offset[j];
  int32_t ne = engine_offset[j + 1] - e0;
  ne = ne < 0 ? 0 : ne;
  maestro_deg_plan out;
  double freed = 0.0, top = 0.0;
  float cost = 0.0f;
  bool interrupt = false;
  // one step of the running sums: engine e (global index) of level lv at position p
  auto step = [&](int32_t p, int32_t e, int32_t lv) {
    interrupt = interrupt || lv >= 4;   // Preempt / Abort interrupt active work
    freed = __dadd_rn(freed, engine_freed[e]);
    cost = __fadd_rn(cost, engine_cost[e]);
    top = p == 0 ? freed : fmax(top, freed);
    const float c = __fadd_rn(cost, interrupt ? c_int : 0.0f);
    steps[e0 + p] = maestro_plan_step{top, c, e};
    if (p < kRecSteps) {
      out.freed[p] = top;
      out.cost[p] = c;
    }
  };
  if (ne <= kRecSteps) {
    int64_t key[kRecSteps];
#pragma unroll
    for (int i = 0; i < kRecSteps; ++i) key[i] = i < ne ? engine_key(engine_level[e0 + i], i) : INT64_MAX;
#pragma unroll
    for (int pass = 0; pass < kRecSteps; ++pass) {
#pragma unroll
      for (int q = pass & 1; q + 1 < kRecSteps; q += 2) {   // odd-even transposition sort
        const int64_t a = key[q], b = key[q + 1];
        key[q] = a < b ? a : b;
        key[q + 1] = a < b ? b : a;
      }
    }
#pragma unroll
    for (int p = 0; p < kRecSteps; ++p)
      if (p < ne) step(p, e0 + (int32_t)(uint32_t)key[p], (int32_t)(key[p] >> 32));
  } else {
    // the rank of engine i among the node's keys is its position in priority order; the step
    // array holds the order (engine of each position) before the running sums overwrite it
    for (int32_t i = 0; i < ne; ++i) {
      const int64_t ki = engine_key(engine_level[e0 + i], i);
      int32_t rank = 0;
      for (int32_t q = 0; q < ne; ++q) rank += engine_key(engine_level[e0 + q], q) < ki ? 1 : 0;
      steps[e0 + rank].engine = e0 + i;
    }
    for (int32_t p = 0; p < ne; ++p) {
      const int32_t e = steps[e0 + p].engine;
      step(p, e, engine_level[e]);
    }
  }
#pragma unroll
  for (int p = 0; p < kRecSteps; ++p) {
    if (p >= ne) {
      out.freed[p] = INFINITY;
      out.cost[p] = 0.0f;
    }
  }
  out.n_engines = ne;
  out.first_step = e0;
#pragma unroll
  for (int i = 0; i < 6; ++i) out.reserved[i] = 0;
  plans[j] = out;
}

// How T_act(N, M(T)) of Eq. 6 reaches the kernel: a node's activation latency unless the
// stage's model is resident (residency bits in 32 or 64 bits), or a [node][model] matrix (of at
// most 16 or 64 models: the chunk of node rows staged in LDS shrinks with the row length).
enum Ready { kMask32 = 0, kMask64 = 1, kMatrix16 = 2, kMatrix64 = 3 };
constexpr int64_t kFitnessLanesTarget = 256 * 4 * 64 * 4;   // lanes of four wavefronts per SIMD

template <int kReady>
struct FitnessChunk {
  static constexpr int value = kReady == kMatrix64 ? 32 : 128;
};

// kMulti: G = 2^g_log2 lanes share a stage (batches too small to fill the chip); lane g scores
// nodes g, g + G, g + 2G, ... of every chunk into its own list, and the G lists are merged with
// xor-shuffles (lexicographic on (key, node)) before lane 0 writes the stage's results.
// kS: stages per lane (1 or 2; 1 with kMulti). The loop over pairs is bound by the bytes the
// lanes read from LDS (a read that every lane shares costs as much as any other), and the node
// terms a lane reads serve all of its stages: a second stage per lane cuts the bytes per pair
// by a third.
// Dynamic LDS: with residency bits, the per-class penalties, n_classes rows of chunk + 1 float2
// (the pad puts one node's entries of different classes in different banks).
template <int KT, int kReady, bool kPlans, bool kMulti, int kS>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(kPlans || KT * kS == 1 ? 1 : (kS == 2 ? 6 : 8), 8)))
void fitness_kernel(
    int64_t n, const int32_t* __restrict__ model_id, const int32_t* __restrict__ src_id,
    const int32_t* __restrict__ class_id, const double* __restrict__ kv_bytes, int32_t n_models, int32_t n_nodes,
    int32_t n_src, int32_t n_classes, const double* __restrict__ free_bytes, const float* __restrict__ queue_ms,
    const float* __restrict__ act_ms, const uint64_t* __restrict__ resident_mask,
    const float* __restrict__ act_matrix, const float* __restrict__ deg_ms,
    const maestro_deg_plan* __restrict__ plans, const maestro_plan_step* __restrict__ plan_steps,
    const float* __restrict__ rtt_ms, const float* __restrict__ class_weights, const float* __restrict__ bounds,
    double rho, int32_t k, int32_t* __restrict__ node_idx, float* __restrict__ fitness, int g_log2) {
  // per node: {headroom, 1 / fl32(headroom)} and the residency bits (reads that every lane
  // shares), and per source row 1 - norm(RTT). With residency bits, the penalty of each class
  // for both states (model resident or not) and, for the short pairs of plans, the two
  // normalised ready times; with a T_act matrix, norm(T_q + T_act) of every (node, model) and
  // the node's normalised C_deg.
  typedef typename std::conditional<kReady == kMask64, uint64_t, uint32_t>::type mask_t;
  static_assert(kS == 1 || (kS == 2 && !kMulti), "lanes that share a stage take one stage each");
  constexpr bool kMat = kReady >= kMatrix16;
  constexpr int kMatRow = kReady == kMatrix16 ? 16 : 64;   // largest row the staging area holds
  // nodes staged in LDS at a time: small chunks keep the LDS footprint low enough for several
  // workgroups per CU, whose waves hide each other's LDS latency
  constexpr int kChunk = FitnessChunk<kReady>::value;
  constexpr int kRowStride = kChunk + 1;   // one-entry pad: rows of different sources / classes in different banks
  struct Node { double free, recip; };
  __shared__ Node s_node[kChunk];
  __shared__ mask_t s_mask[kMat ? 1 : kChunk];
  __shared__ float2 s_tr[kMat || !kPlans ? 1 : kChunk];   // norm(T_q), norm(T_q + T_act)
  __shared__ float s_nd[kMat ? kChunk : 1];                // norm(C_deg) (T_act matrix)
  __shared__ float s_prox[kMaxFitnessSources * kRowStride];   // 1 - norm(RTT), per source row
  __shared__ float s_w[3 * kMaxFitnessClasses];           // (gamma, lambda, mu) per class
  constexpr int kPC = kPlans ? kChunk : 1;
  __shared__ double s_pfreed[kRecSteps][kPC];   // plan columns, node-minor: lanes reading
  __shared__ float s_pcost[kRecSteps][kPC];     // different nodes hit different banks
  __shared__ int32_t s_pn[kPC], s_pfirst[kPC];
  constexpr int kQueue = kPlans ? 16 : 1;   // short pairs a lane queues per chunk
  static_assert(kChunk * kS <= 256 || !kPlans, "a queued pair (node offset, stage) is a byte");
  __shared__ uint8_t s_queue[kQueue * kThreads];
  // with a T_act matrix: normalised T_ready = norm(T_q + T_act) of every (node, model) of the
  // chunk, [node][model] with row stride n_models
  __shared__ float s_ready[kMat ? kChunk * kMatRow : 1];
  extern __shared__ float2 s_pen[];              // [class][node]: penalty resident, not resident

  const int tid = threadIdx.x;
  const int G = kMulti ? 1 << g_log2 : 1;
  const int g = kMulti ? tid & (G - 1) : 0;   // this lane's first node of each chunk
  const float lo_r = bounds[0], hi_r = bounds[1], lo_t = bounds[2], hi_t = bounds[3];
  const float lo_d = bounds[4], hi_d = bounds[5];
  const float nd_fits = norm01(0.0f, lo_d, hi_d);   // normalised C_deg of a stage that fits
  for (int e = tid; e < 3 * n_classes; e += kThreads) s_w[e] = class_weights[e];

  // the stages of this lane: consecutive lanes take consecutive stages, 256 * kS per workgroup
  struct Lane {
    int64_t stage;
    double need;    // R_need; +inf without a stage (admits nothing), NaN for ids out of range
    double needd;   // fl32(R_need), widened
    float gamma, omg, lambda, mu;
    mask_t mbit;
    const uint32_t* mword;   // 64-bit residency bits: the 32-bit half of s_mask[0] holding mbit
    uint32_t mbit32;         // mbit within that half
    int model;
    bool ok;        // a stage whose model, source and class ids are in range
    const float* prox;    // 1 - norm(RTT) from the stage's source, per node of the chunk
    const float2* pen;    // the stage class's penalties, per node of the chunk
  };
  Lane L[kS];
  TopK<KT> best[kS];   // keys are -fitness: the smallest key is the best node
#pragma unroll
  for (int s = 0; s < kS; ++s) {
    Lane& l = L[s];
    l.stage = kMulti ? (int64_t)blockIdx.x * (kThreads >> g_log2) + (tid >> g_log2)
                     : ((int64_t)blockIdx.x * kS + s) * kThreads + tid;
    l.need = INFINITY;
    l.needd = 0.0;
    l.gamma = l.omg = l.lambda = l.mu = 0.0f;
    l.mbit = 0;
    l.mword = reinterpret_cast<const uint32_t*>(s_mask);
    l.mbit32 = 0;
    l.model = 0;
    l.ok = false;
    int src = 0, cls = 0;
    if (l.stage < n) {
      const int32_t m = model_id[l.stage], sid = src_id[l.stage], c = class_id[l.stage];
      l.ok = (uint32_t)m < (uint32_t)n_models && (uint32_t)sid < (uint32_t)n_src &&
             (uint32_t)c < (uint32_t)n_classes;
      if (l.ok) {
        l.need = (rho == 0.0) ? kv_bytes[l.stage] : __dmul_rn(kv_bytes[l.stage], 1.0 + rho);
        l.needd = (double)__double2float_rn(l.need);
        const float* wt = class_weights + 3 * c;
        l.gamma = wt[0];
        l.lambda = wt[1];
        l.mu = wt[2];
        l.omg = __fsub_rn(1.0f, l.gamma);
        l.model = m;
        l.mbit = kMat ? 0 : (mask_t)1 << m;
        if constexpr (kReady == kMask64) {
          l.mword = reinterpret_cast<const uint32_t*>(s_mask) + (m >> 5);
          l.mbit32 = 1u << (m & 31);
        }
        src = sid;
        cls = c;
      } else {
        l.need = NAN;   // an id out of range: no node admits the stage, no plan is tried
      }
    }
    l.prox = s_prox + src * kRowStride;
    l.pen = s_pen + cls * kRowStride;
    best[s].init();
  }
  // A short pair's fitness is at most its score with C_deg normalised to 0 when mu >= 0: norm()
  // is never below 0, the penalty cannot fall as C_deg grows, and every float32 operation is
  // monotone. When a stage that fits normalises to 0 as well (nd_fits == 0), that bound is the
  // score the main loop computes for the pair as if it fit, so a short pair whose bound cannot
  // enter the lane's list (which only improves) is dropped there, before its plan is looked up.
  bool prefilter[kS];
#pragma unroll
  for (int s = 0; s < kS; ++s) prefilter[s] = kPlans && nd_fits == 0.0f && L[s].mu >= 0.0f;

  for (int32_t c0 = 0; c0 < n_nodes; c0 += kChunk) {
    const int cn = min(kChunk, n_nodes - c0);
    __syncthreads();  // every lane is done with the previous chunk (and s_w is written)
    for (int i = tid; i < cn; i += kThreads) {
      const int32_t j = c0 + i;
      const double fr = free_bytes[j];
      const float frf = __double2float_rn(fr);
      // a node without headroom admits only an empty demand: its fit is 0
      s_node[i] = Node{fr, frf > 0.0f ? __ddiv_rn(1.0, (double)frf) : 0.0};
      const float nd = kPlans ? nd_fits : norm01(deg_ms[j], lo_d, hi_d);
      if constexpr (kMat) {
        s_nd[i] = nd;
      } else {
        const float q = queue_ms[j];
        const float tr0 = norm01(__fadd_rn(q, 0.0f), lo_t, hi_t);
        const float tr1 = norm01(__fadd_rn(q, act_ms[j]), lo_t, hi_t);
        s_mask[i] = (mask_t)resident_mask[j];
        if constexpr (kPlans) s_tr[i] = make_float2(tr0, tr1);
        for (int c = 0; c < n_classes; ++c) {
          const float l = s_w[3 * c + 1], u = s_w[3 * c + 2];
          const float pd = __fmul_rn(u, nd);
          s_pen[c * kRowStride + i] =
              make_float2(__fadd_rn(__fmul_rn(l, tr0), pd), __fadd_rn(__fmul_rn(l, tr1), pd));
        }
      }
      if constexpr (kPlans) {
        const maestro_deg_plan& pl = plans[j];
#pragma unroll
        for (int e = 0; e < kRecSteps; ++e) {
          s_pfreed[e][i] = pl.freed[e];
          s_pcost[e][i] = pl.cost[e];
        }
        s_pn[i] = pl.n_engines;
        s_pfirst[i] = pl.first_step;
      }
    }
    if constexpr (kMat) {   // rows c0 .. c0+cn-1 of the matrix are contiguous
      const float* src_rows = act_matrix + (size_t)c0 * n_models;
      for (int e = tid; e < cn * n_models; e += kThreads)
        s_ready[e] = norm01(__fadd_rn(queue_ms[c0 + e / n_models], src_rows[e]), lo_t, hi_t);
    }
    for (int e = tid; e < n_src * cn; e += kThreads) {
      const int r = e / cn, i = e - r * cn;
      s_prox[r * kRowStride + i] = __fsub_rn(1.0f, norm01(rtt_ms[(size_t)r * n_nodes + c0 + i], lo_r, hi_r));
    }
    __syncthreads();
    // A = gamma * prox + (1 - gamma) * fit with fit = fl32(fl32(R_need) * (1 / fl32(headroom)))
    auto affinity = [&](const Lane& l, const Node nd, float prox) {
      const float fit = __double2float_rn(__dmul_rn(l.needd, nd.recip));
      return __fadd_rn(__fmul_rn(l.gamma, prox), __fmul_rn(l.omg, fit));
    };
    // the penalty lambda * norm(T_ready) + mu * nd of node i
    auto penalty = [&](const Lane& l, int i, float nd) {
      float tr;
      if constexpr (kMat) {
        tr = s_ready[i * n_models + l.model];
      } else {
        const float2 t = s_tr[i];
        tr = (s_mask[i] & l.mbit) ? t.x : t.y;
      }
      return __fadd_rn(__fmul_rn(l.lambda, tr), __fmul_rn(l.mu, nd));
    };
    // whether the lane's model is resident on node i: with 64-bit residency bits each stage
    // reads the one 32-bit half that holds its bit (one 32-bit AND and compare per pair instead of
    // two ANDs and a 64-bit compare; c4, 64 models, with the plain node loop below unrolled by four:
    // 5.04-5.22 against 5.42-5.48 ms on two boxes, with plans 7.47-7.61 against 7.63-7.65), else
    // from mk, the node's bits read once for all the lane's stages
    auto resident = [&](const Lane& l, int i, mask_t mk) -> bool {
      if constexpr (kReady == kMask64) return (l.mword[2 * i] & l.mbit32) != 0u;
      else return (mk & l.mbit) != 0;
    };
    // the pair's fitness when the stage fits (C_deg = the node's, or 0 with plans); mk is the
    // node's residency bits
    auto fits_score = [&](const Lane& l, int i, const Node nd, mask_t mk) {
      const float a = affinity(l, nd, l.prox[i]);
      float pen;
      if constexpr (kMat) {
        pen = __fadd_rn(__fmul_rn(l.lambda, s_ready[i * n_models + l.model]), __fmul_rn(l.mu, s_nd[i]));
      } else {
        const float2 p = l.pen[i];
        pen = resident(l, i, mk) ? p.x : p.y;
      }
      return __fsub_rn(a, pen);
    };
    // A stage that falls short of node i's headroom by R takes the first step of the node's
    // plan whose freed bytes reach R, at that step's cost; no such step leaves the node
    // infeasible. These pairs are rare, so they leave the main loop: each lane queues its short
    // pairs and scores them after the chunk (rescanning the chunk when its queue overflowed),
    // inserting lexicographically since they come after nodes of larger index. The stage is a
    // compile-time index (std::integral_constant), so the lane state stays in registers.
    auto short_pair = [&](int i, auto stage_index) {
      constexpr int s = decltype(stage_index)::value;
      const Lane& l = L[s];
      const Node nd = s_node[i];
      const float a = affinity(l, nd, l.prox[i]);
      if (l.mu >= 0.0f && -__fsub_rn(a, penalty(l, i, 0.0f)) > best[s].s[KT - 1]) return;   // cannot enter
      const double R = __dsub_rn(l.need, nd.free);
      const int ne = s_pn[i];
      int jp = 0;
#pragma unroll
      for (int e = 0; e < kRecSteps; ++e) jp += s_pfreed[e][i] < R ? 1 : 0;
      float c = 0.0f;
      bool found = jp < ne && jp < kRecSteps;
      if (found) {
        c = s_pcost[jp][i];
      } else if (ne > kRecSteps) {   // the steps past the record: the first freed >= R
        const maestro_plan_step* st = plan_steps + s_pfirst[i];
        int lo = kRecSteps, hi = ne;
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          if (st[mid].freed < R) lo = mid + 1;
          else hi = mid;
        }
        found = lo < ne;
        if (found) c = st[lo].cost;
      }
      if (found) best[s].push_lex(-__fsub_rn(a, penalty(l, i, norm01(c, lo_d, hi_d))), c0 + i);
    };
    auto short_pair_of = [&](int i, int s) {
      if (kS == 1 || s == 0) short_pair(i, std::integral_constant<int, 0>{});
      else short_pair(i, std::integral_constant<int, kS - 1>{});
    };
    int n_short = 0;   // queued pairs of this chunk
    auto queue = [&](int code) {
      if (n_short < kQueue) s_queue[n_short * kThreads + tid] = (uint8_t)code;
      ++n_short;
    };
    auto node_mask = [&](int i) -> mask_t {
      if constexpr (kMat) return 0;
      else return s_mask[i];
    };
    if constexpr (kS == 1 && !kPlans) {
      // one node at a time, unrolled by four: few registers in flight, so that many
      // wavefronts per SIMD hide the LDS latency
#pragma unroll 4
      for (int i = g; i < cn; i += G) {
        const Node nd = s_node[i];
        best[0].push_increasing_if(L[0].need <= nd.free, -fits_score(L[0], i, nd, node_mask(i)), c0 + i);
      }
    } else if constexpr (kS == 1) {
      // groups of four of this lane's nodes: their LDS reads issue together, the four scores
      // are computed before any of them enters the list, and one branch per group queues the
      // short ones
      int i = g;
      for (; i + 3 * G < cn; i += 4 * G) {
        Node nd[4];
        bool fits[4];
        float sc[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) nd[u] = s_node[i + u * G];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          fits[u] = L[0].need <= nd[u].free;
          sc[u] = fits_score(L[0], i + u * G, nd[u], node_mask(i + u * G));
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) best[0].push_increasing_if(fits[u], -sc[u], c0 + i + u * G);
        if (L[0].ok && !(fits[0] && fits[1] && fits[2] && fits[3])) {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (!fits[u] && !(prefilter[0] && -sc[u] > best[0].s[KT - 1])) queue(i + u * G);
        }
      }
      for (; i < cn; i += G) {
        const Node nd = s_node[i];
        const bool fits = L[0].need <= nd.free;
        const float key = -fits_score(L[0], i, nd, node_mask(i));
        best[0].push_increasing_if(fits, key, c0 + i);
        if (L[0].ok && !fits && !(prefilter[0] && key > best[0].s[KT - 1])) queue(i);
      }
    } else {
      // every node once for the lane's stages: one read of its shared terms, then per stage
      // the stage's own source and class entries; with plans one branch per node queues the
      // short pairs, and nodes go two at a time: all their LDS reads and scores come before the
      // first insertion, whose branches would otherwise hold back the next node's reads (c4 with
      // plans 7.58 against 8.06 ms). Without plans there are fewer branches and one node at a
      // time stays (grouping there measured 5.48 against 5.44 ms), unrolled by four, or by two
      // with T_act rows of up to 16 models (c3: 0.160 against 0.171 ms; c4, 64 models, by four:
      // 6.98 against 7.17 ms).
      if constexpr (!kPlans) {
        constexpr int kNodeUnroll = kReady == kMatrix16 ? 2 : 4;
#pragma unroll kNodeUnroll
        for (int i = 0; i < cn; ++i) {
          const Node nd = s_node[i];
          const mask_t mk = node_mask(i);
#pragma unroll
          for (int s = 0; s < kS; ++s)
            best[s].push_increasing_if(L[s].need <= nd.free, -fits_score(L[s], i, nd, mk), c0 + i);
        }
      } else {
        auto scores = [&](int i, Node& nd, bool (&fits)[kS], float (&key)[kS]) {
          nd = s_node[i];
          const mask_t mk = node_mask(i);
#pragma unroll
          for (int s = 0; s < kS; ++s) {
            fits[s] = L[s].need <= nd.free;
            key[s] = -fits_score(L[s], i, nd, mk);
          }
        };
        auto insert = [&](int i, const bool (&fits)[kS], const float (&key)[kS]) {
#pragma unroll
          for (int s = 0; s < kS; ++s) best[s].push_increasing_if(fits[s], key[s], c0 + i);
          if (!(fits[0] && fits[kS - 1])) {
#pragma unroll
            for (int s = 0; s < kS; ++s)
              if (L[s].ok && !fits[s] && !(prefilter[s] && key[s] > best[s].s[KT - 1])) queue(i + s * kChunk);
          }
        };
        int i = 0;
#pragma unroll 1
        for (; i + 1 < cn; i += 2) {
          Node nd[2];
          bool fits[2][kS];
          float key[2][kS];
          scores(i, nd[0], fits[0], key[0]);
          scores(i + 1, nd[1], fits[1], key[1]);
          insert(i, fits[0], key[0]);
          insert(i + 1, fits[1], key[1]);
        }
        if (i < cn) {
          Node nd;
          bool fits[kS];
          float key[kS];
          scores(i, nd, fits, key);
          insert(i, fits, key);
        }
      }
    }
    if (kPlans && n_short > 0) {
      if (n_short <= kQueue) {
#pragma unroll 1
        for (int q = 0; q < n_short; ++q) {
          const int code = s_queue[q * kThreads + tid];
          short_pair_of(code % kChunk, code / kChunk);
        }
      } else {
#pragma unroll 1
        for (int i = g; i < cn; i += G) {
          const double fr = s_node[i].free;
#pragma unroll
          for (int s = 0; s < kS; ++s)
            if (L[s].ok && !(L[s].need <= fr)) short_pair_of(i, s);
        }
      }
    }
  }

  if constexpr (kMulti) {   // lanes g and g ^ o exchange and merge their lists
    for (int o = 1; o < G; o <<= 1) {
      float ps[KT];
      int32_t pn[KT];
#pragma unroll
      for (int i = 0; i < KT; ++i) {
        ps[i] = __shfl_xor(best[0].s[i], o);
        pn[i] = __shfl_xor(best[0].n[i], o);
      }
#pragma unroll
      for (int i = 0; i < KT; ++i) best[0].push_lex(ps[i], pn[i]);
    }
  }

#pragma unroll
  for (int s = 0; s < kS; ++s) {
    const int64_t stage = L[s].stage;
    if (stage < n && g == 0) {
#pragma unroll
      for (int i = 0; i < KT; ++i) {
        if (i < k) {
          const bool some = best[s].n[i] != kNoNode;
          node_idx[stage * k + i] = some ? best[s].n[i] : -1;
          fitness[stage * k + i] = some ? -best[s].s[i] : -INFINITY;
        }
      }
    }
  }
}

// The values of rank r_lo and r_hi (0-based) of v[0 .. m-1] in the total order of float bit
// patterns (-0 before +0): four passes over the 8-bit digits of the order-preserving image,
// each narrowing both candidate prefixes by one digit. Within a pass, the candidates' digits
// are counted into one 256-bin histogram per rank; eight wavefronts scan the two histograms
// (64 bins each, cross-lane), and the one bin whose count range holds the rank takes it. A
// window's values often share their leading digits, which would serialise the LDS atomics on
// one bin: a wavefront whose counted lanes all carry the same digit adds their count once.
// Short inputs: one workgroup does every pass. Long ones: below.
constexpr int kSelectThreads = 1024;

__device__ __forceinline__ void count_digit(uint32_t* hist, bool want, uint32_t dgt, int lane) {
  const uint64_t act = __ballot(want);
  if (act == 0) return;
  const int first = __ffsll((unsigned long long)act) - 1;
  const uint32_t d0 = __shfl(dgt, first);
  if (__ballot(want && dgt == d0) == act) {
    if (lane == first) atomicAdd(&hist[d0], (uint32_t)__popcll(act));
  } else if (want) {
    atomicAdd(&hist[dgt], 1u);
  }
}

__global__ __launch_bounds__(kSelectThreads) void quantile_kernel(const float* __restrict__ v, int64_t m,
                                                                  int64_t r_lo, int64_t r_hi,
                                                                  float* __restrict__ out, int n_out) {
  __shared__ uint32_t hist[2][256];
  __shared__ uint32_t scan[2][256];   // inclusive prefix within each 64-bin segment
  __shared__ uint32_t seg[2][4];      // segment totals
  __shared__ uint32_t s_prefix[2][2];   // [pass parity][rank]: read in one pass, written for the next
  __shared__ int64_t s_rank[2][2];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (tid < 2) {
    s_prefix[0][tid] = 0;
    s_rank[0][tid] = tid ? r_hi : r_lo;
  }
  uint32_t mask = 0;
  int par = 0;
  for (int shift = 24; shift >= 0; shift -= 8, par ^= 1) {
    for (int i = tid; i < 512; i += kSelectThreads) (&hist[0][0])[i] = 0;
    __syncthreads();
    const uint32_t p0 = s_prefix[par][0], p1 = s_prefix[par][1];
    for (int64_t i0 = 0; i0 < m; i0 += kSelectThreads) {   // uniform trip count: whole-wave ballots
      const int64_t i = i0 + tid;
      const bool in = i < m;
      const uint32_t u = in ? float_key(v[i]) : 0u;
      const uint32_t dgt = (u >> shift) & 255u;
      count_digit(hist[0], in && (u & mask) == p0, dgt, lane);
      if (n_out > 1) count_digit(hist[1], in && (u & mask) == p1, dgt, lane);
    }
    __syncthreads();
    if (wave < 8) {
      const int h = wave >> 2, b = (wave & 3) * 64 + lane;
      uint32_t x = hist[h][b];
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const uint32_t y = __shfl_up(x, d, 64);
        if (lane >= d) x += y;
      }
      scan[h][b] = x;
      if (lane == 63) seg[h][wave & 3] = x;
    }
    __syncthreads();
    if (tid < 512) {
      const int h = tid >> 8, b = tid & 255;
      uint32_t incl = scan[h][b];
      for (int q = 0; q < (b >> 6); ++q) incl += seg[h][q];
      const uint32_t c = hist[h][b];
      const int64_t r = s_rank[par][h];
      if (r >= (int64_t)(incl - c) && r < (int64_t)incl) {   // exactly one bin per rank
        s_rank[par ^ 1][h] = r - (int64_t)(incl - c);
        s_prefix[par ^ 1][h] = s_prefix[par][h] | ((uint32_t)b << shift);
      }
    }
    mask |= 0xFFu << shift;
    __syncthreads();
  }
  if (tid < n_out) out[tid] = key_float(s_prefix[par][tid]);
}

// Long inputs: the same four 8-bit passes over several workgroups. Per pass, kSelBlocks
// workgroups each count the digits of the candidates (the values that match a rank's prefix so
// far) of a contiguous range into histograms of their own in the workspace, and one workgroup
// sums them per bin, finds the bin that holds each rank and narrows the rank's prefix for the
// next pass (state in the workspace). No atomics outside LDS and no waiting across workgroups.
constexpr int kSelBlocks = 256;
constexpr int64_t kMultiSelectMin = 32768;   // inputs at least this long take the multi-workgroup passes
struct SelectState {
  uint32_t prefix[2];
  int64_t rank[2];
};

size_t select_workspace_bytes(int64_t m) {
  return m >= kMultiSelectMin ? (size_t)kSelBlocks * 512 * sizeof(uint32_t) + 256 : 0;
}

__device__ __forceinline__ uint32_t select_mask(int shift) {
  return shift == 24 ? 0u : ~((1u << (shift + 8)) - 1u);
}

__global__ __launch_bounds__(kSelectThreads) void select_hist_kernel(const float* __restrict__ v, int64_t m,
                                                                     int shift, int n_hist,
                                                                     const SelectState* __restrict__ st,
                                                                     uint32_t* __restrict__ hist) {
  __shared__ uint32_t h[2][256];
  const int tid = threadIdx.x, lane = tid & 63;
  for (int i = tid; i < 512; i += kSelectThreads) (&h[0][0])[i] = 0;
  __syncthreads();
  const uint32_t mask = select_mask(shift);
  const uint32_t p0 = shift == 24 ? 0u : st->prefix[0], p1 = shift == 24 ? 0u : st->prefix[1];
  const int64_t per = (m + gridDim.x - 1) / gridDim.x;
  const int64_t b0 = (int64_t)blockIdx.x * per, b1 = min(m, b0 + per);
  for (int64_t i0 = b0; i0 < b1; i0 += kSelectThreads) {   // workgroup-uniform trip count: whole-wave ballots
    const int64_t i = i0 + tid;
    const bool in = i < b1;
    const uint32_t u = in ? float_key(v[i]) : 0u;
    const uint32_t dgt = (u >> shift) & 255u;
    count_digit(h[0], in && (u & mask) == p0, dgt, lane);
    if (n_hist > 1) count_digit(h[1], in && (u & mask) == p1, dgt, lane);
  }
  __syncthreads();
  for (int i = tid; i < 512; i += kSelectThreads) hist[(int64_t)blockIdx.x * 512 + i] = (&h[0][0])[i];
}

// one workgroup: bin totals over the kSelBlocks histograms, the bin of each rank, the state for
// the next pass; after the last pass (shift 0) the selected values
__global__ __launch_bounds__(kSelectThreads) void select_pick_kernel(const uint32_t* __restrict__ hist, int shift,
                                                                     int n_out, int64_t r_lo, int64_t r_hi,
                                                                     SelectState* __restrict__ st,
                                                                     float* __restrict__ out) {
  __shared__ uint32_t tot[2][2][256];   // [half of the workgroups][histogram][bin]
  __shared__ uint32_t scan[2][256];
  __shared__ uint32_t seg[2][4];
  __shared__ uint32_t s_prefix[2];
  __shared__ int64_t s_rank[2];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (tid < 2) {
    s_prefix[tid] = shift == 24 ? 0u : st->prefix[tid];
    s_rank[tid] = shift == 24 ? (tid ? r_hi : r_lo) : st->rank[tid];
  }
  {   // thread (half, histogram, bin): the sum over its half of the workgroups, loads in batches
    const int half = tid >> 9, hb = tid & 511;
    uint32_t t = 0;
    for (int b = half * (kSelBlocks / 2); b < (half + 1) * (kSelBlocks / 2); b += 16) {
      uint32_t c[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) c[u] = hist[(int64_t)(b + u) * 512 + hb];
#pragma unroll
      for (int u = 0; u < 16; ++u) t += c[u];
    }
    (&tot[half][0][0])[hb] = t;
  }
  __syncthreads();
  if (wave < 8) {
    const int hh = wave >> 2, b = (wave & 3) * 64 + lane;
    uint32_t x = tot[0][hh][b] + tot[1][hh][b];
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t y = __shfl_up(x, d, 64);
      if (lane >= d) x += y;
    }
    scan[hh][b] = x;
    if (lane == 63) seg[hh][wave & 3] = x;
  }
  __syncthreads();
  if (tid < 512) {
    const int hh = tid >> 8, b = tid & 255;
    const int hsrc = n_out > 1 ? hh : 0;   // one rank: both slots follow histogram 0
    uint32_t incl = scan[hsrc][b];
    for (int q = 0; q < (b >> 6); ++q) incl += seg[hsrc][q];
    const uint32_t c = tot[0][hsrc][b] + tot[1][hsrc][b];
    const int64_t r = s_rank[hh];
    if (r >= (int64_t)(incl - c) && r < (int64_t)incl) {   // exactly one bin per rank
      st->rank[hh] = r - (int64_t)(incl - c);
      st->prefix[hh] = s_prefix[hh] | ((uint32_t)b << shift);
      if (shift == 0 && hh < n_out) out[hh] = key_float(s_prefix[hh] | (uint32_t)b);
    }
  }
}

maestro_status launch_select(const float* v, int64_t m, int64_t r_lo, int64_t r_hi, float* out, int n_out,
                             void* workspace, hipStream_t stream) {
  uint32_t* hist = static_cast<uint32_t*>(workspace);
  SelectState* st = reinterpret_cast<SelectState*>(static_cast<unsigned char*>(workspace) +
                                                   (size_t)kSelBlocks * 512 * sizeof(uint32_t));
  for (int shift = 24; shift >= 0; shift -= 8) {
    select_hist_kernel<<<dim3(kSelBlocks), dim3(kSelectThreads), 0, stream>>>(v, m, shift, n_out, st, hist);
    select_pick_kernel<<<dim3(1), dim3(kSelectThreads), 0, stream>>>(hist, shift, n_out, r_lo, r_hi, st, out);
  }
  return launch_status();
}

// EWMA of the relative underestimation e_i = max(0, actual_i / pred_i - 1) in arrival order,
// s_0 = e_0, s_i = beta e_i + (1 - beta) s_(i-1), stored as float32. The window is cut into
// tiles of kEwmaTile elements. Within a tile, the errors are computed from coalesced loads into
// LDS, each thread folds its kEwmaPer consecutive elements into an affine map x -> A x + B, the
// maps are scanned within each wavefront (cross-lane) and the 16 wavefront totals composed in
// order by one lane, which gives every thread the value entering its elements; each thread then
// replays its elements with the recurrence. A map that contains element 0 is constant.
__device__ __forceinline__ double underestimation(double actual, double pred) {
  const double e = __dsub_rn(__ddiv_rn(actual, pred), 1.0);
  return e > 0.0 ? e : 0.0;
}

constexpr int kEwmaPer = 8;
constexpr int kEwmaTile = kSelectThreads * kEwmaPer;
constexpr int kEwmaWaves = kSelectThreads / 64;
constexpr int64_t kEwmaOneGroupTiles = 2;   // longer windows take the three-launch path

struct EwmaShared {
  double e[kEwmaTile];
  double wa[kEwmaWaves], wb[kEwmaWaves];   // wavefront totals
  double win[kEwmaWaves + 1];              // value entering each wavefront; [16]: leaving the tile
};

// Errors of tile t0 into LDS, this thread's map (A, B) scanned inclusively within the
// wavefront, and the wavefront totals into wa/wb. Ends with a barrier.
__device__ __forceinline__ void ewma_tile_maps(const double* __restrict__ actual, const double* __restrict__ pred,
                                               int64_t m, int64_t t0, double beta, double keep, EwmaShared& sh,
                                               double& A, double& B) {
  const int tid = threadIdx.x, lane = tid & 63;
  {
    double av[kEwmaPer], pv[kEwmaPer];
#pragma unroll
    for (int q = 0; q < kEwmaPer; ++q) {
      const int64_t i = t0 + (int64_t)q * kSelectThreads + tid;
      av[q] = i < m ? actual[i] : 0.0;
      pv[q] = i < m ? pred[i] : 1.0;
    }
#pragma unroll
    for (int q = 0; q < kEwmaPer; ++q) sh.e[q * kSelectThreads + tid] = underestimation(av[q], pv[q]);
  }
  __syncthreads();
  const int64_t lo = t0 + (int64_t)tid * kEwmaPer;
  A = 1.0;
  B = 0.0;   // identity
#pragma unroll
  for (int u = 0; u < kEwmaPer; ++u) {
    const int64_t i = lo + u;
    if (i < m) {
      const double e = sh.e[tid * kEwmaPer + u];
      if (i == 0) {
        A = 0.0;
        B = e;
      } else {
        A = __dmul_rn(keep, A);
        B = __dadd_rn(__dmul_rn(beta, e), __dmul_rn(keep, B));
      }
    }
  }
  // the map of lanes p..l applied after the map of earlier lanes
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const double pa = __shfl_up(A, d, 64), pb = __shfl_up(B, d, 64);
    if (lane >= d) {
      B = __dadd_rn(__dmul_rn(A, pb), B);
      A = __dmul_rn(A, pa);
    }
  }
  if (lane == 63) {
    sh.wa[tid >> 6] = A;
    sh.wb[tid >> 6] = B;
  }
  __syncthreads();
}

// Values entering each wavefront of the tile given the value x entering the tile (one lane).
__device__ __forceinline__ void ewma_tile_entries(EwmaShared& sh, double x) {
  for (int w = 0; w < kEwmaWaves; ++w) {
    sh.win[w] = x;
    x = __dadd_rn(__dmul_rn(sh.wa[w], x), sh.wb[w]);
  }
  sh.win[kEwmaWaves] = x;
}

// Replays this thread's elements of tile t0 from the wavefront's entering value.
__device__ __forceinline__ void ewma_tile_replay(int64_t m, int64_t t0, double beta, double keep, const EwmaShared& sh,
                                                 double A, double B, float* __restrict__ ewma) {
  const int tid = threadIdx.x, lane = tid & 63;
  const double xw = sh.win[tid >> 6];
  const double ea = __shfl_up(A, 1, 64), eb = __shfl_up(B, 1, 64);   // lanes 0 .. lane-1
  double x = lane > 0 ? __dadd_rn(__dmul_rn(ea, xw), eb) : xw;
  const int64_t lo = t0 + (int64_t)tid * kEwmaPer;
#pragma unroll
  for (int u = 0; u < kEwmaPer; ++u) {
    const int64_t i = lo + u;
    if (i < m) {
      const double e = sh.e[tid * kEwmaPer + u];
      x = (i == 0) ? e : __dadd_rn(__dmul_rn(beta, e), __dmul_rn(keep, x));
      ewma[i] = __double2float_rn(x);
    }
  }
}

// One workgroup walks every tile in order (windows of at most a few tiles: one launch).
__global__ __launch_bounds__(kSelectThreads) void ewma_kernel(const double* __restrict__ actual,
                                                              const double* __restrict__ pred, int64_t m,
                                                              double beta, float* __restrict__ ewma) {
  __shared__ EwmaShared sh;
  const double keep = __dsub_rn(1.0, beta);
  double carry = 0.0;   // the EWMA just before the tile (unused by the tile holding element 0)
  for (int64_t t0 = 0; t0 < m; t0 += kEwmaTile) {
    double A, B;
    ewma_tile_maps(actual, pred, m, t0, beta, keep, sh, A, B);
    if (threadIdx.x == 0) ewma_tile_entries(sh, carry);
    __syncthreads();
    ewma_tile_replay(m, t0, beta, keep, sh, A, B, ewma);
    carry = sh.win[kEwmaWaves];
    __syncthreads();   // the next tile rewrites sh
  }
}

// Long windows, one workgroup per tile in three launches. The first 16 bytes of each tile's own
// output range carry its map (A, B) from the fold to the carry pass, and the first 8 then the
// value entering the tile from the carry pass to the replay, which reads it before any thread of
// the tile stores an output. The words are moved as 32-bit halves (the output is 4-byte
// aligned). The last tile's map is never needed; a last tile of a single element is finished by
// the carry pass itself.
__device__ __forceinline__ void slot_store(float* p, int k, double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  uint32_t* w = reinterpret_cast<uint32_t*>(p);
  w[2 * k] = (uint32_t)u;
  w[2 * k + 1] = (uint32_t)(u >> 32);
}
__device__ __forceinline__ double slot_load(const float* p, int k) {
  const uint32_t* w = reinterpret_cast<const uint32_t*>(p);
  return __builtin_bit_cast(double, (uint64_t)w[2 * k] | ((uint64_t)w[2 * k + 1] << 32));
}

__global__ __launch_bounds__(kSelectThreads) void ewma_fold_kernel(const double* __restrict__ actual,
                                                                   const double* __restrict__ pred, int64_t m,
                                                                   double beta, float* __restrict__ ewma) {
  __shared__ EwmaShared sh;
  const double keep = __dsub_rn(1.0, beta);
  const int64_t t0 = (int64_t)blockIdx.x * kEwmaTile;   // never the last tile
  double A, B;
  ewma_tile_maps(actual, pred, m, t0, beta, keep, sh, A, B);
  if (threadIdx.x == 0) {
    double a = 1.0, b = 0.0;   // compose the wavefront totals in order
    for (int w = 0; w < kEwmaWaves; ++w) {
      b = __dadd_rn(__dmul_rn(sh.wa[w], b), sh.wb[w]);
      a = __dmul_rn(sh.wa[w], a);
    }
    slot_store(ewma + t0, 0, a);
    slot_store(ewma + t0, 1, b);
  }
}

__global__ __launch_bounds__(64) void ewma_carry_kernel(const double* __restrict__ actual,
                                                        const double* __restrict__ pred, int64_t m, double beta,
                                                        int64_t n_tiles, float* __restrict__ ewma) {
  if (threadIdx.x != 0) return;
  double x = 0.0;
  for (int64_t t = 0; t + 1 < n_tiles; ++t) {
    float* slot = ewma + t * kEwmaTile;
    const double a = slot_load(slot, 0), b = slot_load(slot, 1);
    slot_store(slot, 0, x);   // value entering tile t
    x = __dadd_rn(__dmul_rn(a, x), b);
  }
  const int64_t last = (n_tiles - 1) * kEwmaTile;
  if (m - last >= 2) {
    slot_store(ewma + last, 0, x);
  } else {   // a single element: finish it here
    const double e = underestimation(actual[last], pred[last]);
    ewma[last] = __double2float_rn(__dadd_rn(__dmul_rn(beta, e), __dmul_rn(__dsub_rn(1.0, beta), x)));
  }
}

__global__ __launch_bounds__(kSelectThreads) void ewma_apply_kernel(const double* __restrict__ actual,
                                                                    const double* __restrict__ pred, int64_t m,
                                                                    double beta, float* __restrict__ ewma) {
  __shared__ EwmaShared sh;
  __shared__ double s_in;
  const double keep = __dsub_rn(1.0, beta);
  const int64_t t0 = (int64_t)blockIdx.x * kEwmaTile;
  if (threadIdx.x == 0) s_in = slot_load(ewma + t0, 0);
  double A, B;
  ewma_tile_maps(actual, pred, m, t0, beta, keep, sh, A, B);   // its barriers publish s_in
  if (threadIdx.x == 0) ewma_tile_entries(sh, s_in);
  __syncthreads();
  ewma_tile_replay(m, t0, beta, keep, sh, A, B, ewma);
}

}  // namespace

maestro_status launch_route_fitness(int64_t n, const int32_t* model_id, const int32_t* src_id,
                                    const int32_t* class_id, const double* kv_bytes, int32_t n_models,
                                    int32_t n_nodes, int32_t n_src, int32_t n_classes, const double* free_bytes,
                                    const float* queue_ms, const float* act_ms,
                                    const uint64_t* resident_mask, const float* act_matrix, const float* deg_ms,
                                    const maestro_deg_plan* plans, const maestro_plan_step* plan_steps,
                                    const float* rtt_ms, const float* class_weights, const float* bounds, double rho,
                                    int32_t k, int32_t* node_idx, float* fitness, hipStream_t stream) {
  if (n == 0) return MAESTRO_OK;
  // lanes per stage: the smallest power of two (at most 16) that gives the batch about four
  // wavefronts per SIMD of a 256-CU chip, and never more lanes than a chunk has nodes
  int g_log2 = 0;
  while (g_log2 < 4 && n * (2 << g_log2) <= kFitnessLanesTarget && (2 << g_log2) <= n_nodes) ++g_log2;
  // stages per lane: two when the batch still gives the chip that many wavefronts with two (and
  // the lists are short enough to keep both stages' state in registers), else one. With plans
  // (more registers and LDS per workgroup, so fewer resident workgroups) two only from twice
  // that size on: a grid just above one round of resident workgroups would run a second, nearly
  // empty round.
  const bool with_plans = plans != nullptr;
  const bool two = g_log2 == 0 && k <= 4 && n >= (with_plans ? 4 : 2) * kFitnessLanesTarget;
  const int64_t per_block = two ? 2 * kThreads : kThreads >> g_log2;
  const dim3 grid((unsigned)((n + per_block - 1) / per_block)), block(kThreads);
  const int ready = act_matrix ? (n_models > 16 ? kMatrix64 : kMatrix16) : (n_models > 32 ? kMask64 : kMask32);
  // per-class penalties of a chunk (residency-bit forms only), rows of chunk + 1 entries
  const size_t pen_bytes =
      act_matrix ? 0 : (size_t)n_classes * (size_t)(FitnessChunk<kMask32>::value + 1) * sizeof(float2);
#define MAESTRO_FIT_ARGS                                                                                         \
  n, model_id, src_id, class_id, kv_bytes, n_models, n_nodes, n_src, n_classes, free_bytes, queue_ms, act_ms,    \
      resident_mask, act_matrix, deg_ms, plans, plan_steps, rtt_ms, class_weights, bounds, rho, k, node_idx, fitness
#define MAESTRO_FIT_LAUNCH(KT, RD, PL)                                                                            \
  do {                                                                                                            \
    if (g_log2 > 0)                                                                                               \
      fitness_kernel<KT, RD, PL, true, 1><<<grid, block, pen_bytes, stream>>>(MAESTRO_FIT_ARGS, g_log2);          \
    else if (two)                                                                                                 \
      fitness_kernel<KT, RD, PL, false, (KT <= 4 ? 2 : 1)><<<grid, block, pen_bytes, stream>>>(MAESTRO_FIT_ARGS, 0); \
    else                                                                                                          \
      fitness_kernel<KT, RD, PL, false, 1><<<grid, block, pen_bytes, stream>>>(MAESTRO_FIT_ARGS, 0);              \
  } while (0)
#define MAESTRO_FIT_RD(KT, PL)                                       \
  do {                                                               \
    if (ready == kMatrix16) MAESTRO_FIT_LAUNCH(KT, kMatrix16, PL);   \
    else if (ready == kMatrix64) MAESTRO_FIT_LAUNCH(KT, kMatrix64, PL); \
    else if (ready == kMask64) MAESTRO_FIT_LAUNCH(KT, kMask64, PL);  \
    else MAESTRO_FIT_LAUNCH(KT, kMask32, PL);                        \
  } while (0)
#define MAESTRO_FIT_KT(KT)                        \
  do {                                            \
    if (with_plans) MAESTRO_FIT_RD(KT, true);     \
    else MAESTRO_FIT_RD(KT, false);               \
  } while (0)
  if (k == 1) MAESTRO_FIT_KT(1);
  else if (k == 2) MAESTRO_FIT_KT(2);
  else if (k <= 4) MAESTRO_FIT_KT(4);
  else if (k <= 8) MAESTRO_FIT_KT(8);
  else MAESTRO_FIT_KT(16);
#undef MAESTRO_FIT_KT
#undef MAESTRO_FIT_RD
#undef MAESTRO_FIT_LAUNCH
#undef MAESTRO_FIT_ARGS
  return launch_status();
}

// T_act of every (node, model) from its readiness tier (Sec. III-C): 0 when Running, else the
// tier's setup time plus Size / BW_tier in the caller's time unit (`unit` per second), in
// float64 in that order, stored as float32.
__global__ __launch_bounds__(kThreads) void activation_kernel(int64_t total, int32_t n_models,
                                                              const uint8_t* __restrict__ tier,
                                                              const double* __restrict__ model_bytes,
                                                              const double* __restrict__ tier_bw,
                                                              const float* __restrict__ tier_setup_ms,
                                                              double unit, float* __restrict__ act_ms) {
  for (int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x; e < total; e += (int64_t)gridDim.x * kThreads) {
    int t = tier[e];
    t = t > 4 ? 4 : t;   // past Remote counts as Remote
    const int32_t m = (int32_t)(e % n_models);
    float a = 0.0f;
    if (t > 0)
      a = __double2float_rn(__dadd_rn((double)tier_setup_ms[t],
                                      __dmul_rn(__ddiv_rn(model_bytes[m], tier_bw[t]), unit)));
    act_ms[e] = a;
  }
}

maestro_status launch_activation_latency(int32_t n_nodes, int32_t n_models, const uint8_t* tier,
                                         const double* model_bytes, const double* tier_bw,
                                         const float* tier_setup_ms, double unit, float* act_ms,
                                         hipStream_t stream) {
  const int64_t total = (int64_t)n_nodes * n_models;
  if (total == 0) return MAESTRO_OK;
  const int64_t blocks = (total + kThreads - 1) / kThreads;
  activation_kernel<<<dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(kThreads), 0, stream>>>(
      total, n_models, tier, model_bytes, tier_bw, tier_setup_ms, unit, act_ms);
  return launch_status();
}

maestro_status launch_degradation_plans(int32_t n_nodes, const int32_t* engine_offset, const int32_t* engine_level,
                                       const double* engine_freed_bytes, const float* engine_cost_ms, float c_int_ms,
                                       maestro_deg_plan* plans, maestro_plan_step* steps, hipStream_t stream) {
  if (n_nodes == 0) return MAESTRO_OK;
  plan_kernel<<<dim3((unsigned)((n_nodes + kThreads - 1) / kThreads)), dim3(kThreads), 0, stream>>>(
      n_nodes, engine_offset, engine_level, engine_freed_bytes, engine_cost_ms, c_int_ms, plans, steps);
  return launch_status();
}

size_t quantiles_workspace_bytes(int64_t m) { return select_workspace_bytes(m); }

maestro_status launch_quantiles(const float* values, int64_t m, int64_t r_lo, int64_t r_hi, float* out,
                                void* workspace, hipStream_t stream) {
  if (m >= kMultiSelectMin) return launch_select(values, m, r_lo, r_hi, out, 2, workspace, stream);
  quantile_kernel<<<dim3(1), dim3(kSelectThreads), 0, stream>>>(values, m, r_lo, r_hi, out, 2);
  return launch_status();
}

maestro_status launch_adaptive_rho(const double* kv_actual, const double* kv_pred, int64_t m, double beta,
                                   int64_t rank, float* ewma, float* rho, void* workspace, hipStream_t stream) {
  const int64_t n_tiles = (m + kEwmaTile - 1) / kEwmaTile;
  if (n_tiles <= kEwmaOneGroupTiles) {
    ewma_kernel<<<dim3(1), dim3(kSelectThreads), 0, stream>>>(kv_actual, kv_pred, m, beta, ewma);
  } else {
    const int64_t last_elems = m - (n_tiles - 1) * kEwmaTile;
    ewma_fold_kernel<<<dim3((unsigned)(n_tiles - 1)), dim3(kSelectThreads), 0, stream>>>(kv_actual, kv_pred, m,
                                                                                        beta, ewma);
    ewma_carry_kernel<<<dim3(1), dim3(64), 0, stream>>>(kv_actual, kv_pred, m, beta, n_tiles, ewma);
    const int64_t applied = last_elems >= 2 ? n_tiles : n_tiles - 1;
    ewma_apply_kernel<<<dim3((unsigned)applied), dim3(kSelectThreads), 0, stream>>>(kv_actual, kv_pred, m, beta,
                                                                                   ewma);
  }
  maestro_status st = launch_status();
  if (st != MAESTRO_OK) return st;
  if (m >= kMultiSelectMin) return launch_select(ewma, m, rank, rank, rho, 1, workspace, stream);
  quantile_kernel<<<dim3(1), dim3(kSelectThreads), 0, stream>>>(ewma, m, rank, rank, rho, 1);
  return launch_status();
}

}  // namespace maestro

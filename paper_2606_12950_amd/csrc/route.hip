// Routing of a batch of stages (Sec. III-D; Alg. 3; Eq. 6; decode term of Eq. 2).
//
// The (stage x node) score matrix is evaluated tile by tile and never stored: a workgroup
// takes 256/G stages, stages node state chunk by chunk in LDS (structure of arrays: both
// possible ready times, free bytes, residency mask), and each of the G lanes that share a
// stage walks every G-th node of the chunk, keeping a sorted list of its best KT
// (score, node) pairs. The G lists are then merged across lanes with xor-shuffles
// (lexicographic on (score, node)), and the first lane writes the stage's k results.
// G grows when the batch has too few stages to fill the chip.
//
// A second, exact algorithm avoids the full score matrix. For a fixed model, a node's score
// is fl32(ready + t_exec) with t_exec common to every node, and round-to-nearest addition is
// monotone, so ordering a model's nodes by (ready time, index) orders their scores (equal
// scores may come from different ready times, hence the lexicographic insertion below). One
// workgroup per model sorts the nodes by that key in LDS (stable radix sort); then each stage walks
// its model's list, skipping nodes that cannot admit its KV demand, and stops at the first
// node whose score exceeds its current k-th best. The result is identical to the scan; the
// walk is short unless many nodes are infeasible, and never longer than the node count.
//
// Arithmetic is the same expression, in the same order and precision, as the definition:
// score = fl32(fl32(T_q + T_act) + fl32(L * t_dec)), with T_act in {0, cold} -- or, with
// readiness tiers, T_act from a [node][model] matrix (then the scan stages fl32(T_q + T_act)
// of every (node, model) of a smaller node chunk). The library is
// compiled with -ffp-contract=off and the products/sums below use explicit round-to-nearest
// intrinsics, so nothing is fused or reassociated.
#include <type_traits>

#include "internal.h"
#include "select.h"

namespace maestro {
namespace {

constexpr int kThreads = 256;
// T_act: cold start unless resident (residency bits in 32 or 64 bits), or a [node][model] matrix
enum Ready { kMask32 = 0, kMask64 = 1, kMatrix = 2 };
constexpr int kMaxMatrixModels = 64;

template <int KT, int kReady>
__global__ __launch_bounds__(kThreads) void route_kernel(
    int64_t n, const int32_t* __restrict__ model_id, const float* __restrict__ pred_len,
    const double* __restrict__ kv_bytes, const float* __restrict__ decode_s_per_token, int32_t n_models,
    int32_t n_nodes, const double* __restrict__ free_bytes, const float* __restrict__ queue_s,
    const float* __restrict__ cold_s, const uint64_t* __restrict__ resident_mask,
    const float* __restrict__ act_matrix, double rho, int32_t k, int g_log2, int32_t* __restrict__ node_idx,
    float* __restrict__ score) {
  typedef typename std::conditional<kReady == kMask64, uint64_t, uint32_t>::type mask_t;
  constexpr bool kMat = kReady == kMatrix;
  constexpr int kNodeChunk = kMat ? 128 : 1024;
  constexpr int kM = kMat ? 1 : kNodeChunk;
  __shared__ float s_warm[kM];             // fl32(T_q + 0): ready time when the model is resident
  __shared__ float s_cold[kM];             // fl32(T_q + cold): ready time after a cold start
  __shared__ mask_t s_mask[kM];            // residency bits
  __shared__ double s_free[kNodeChunk];    // KV admission headroom
  __shared__ float s_ready[kMat ? kNodeChunk * kMaxMatrixModels : 1];   // fl32(T_q + T_act[j][m])

  const int tid = threadIdx.x;
  const int G = 1 << g_log2;
  const int64_t stage = (int64_t)blockIdx.x * (kThreads >> g_log2) + (tid >> g_log2);
  const int g = tid & (G - 1);
  const bool valid = stage < n;

  double need = INFINITY;   // an invalid lane admits nothing
  float exec_s = 0.0f;
  mask_t mbit = 0;
  int32_t model = 0;
  if (valid) {
    const int32_t m = model_id[stage];
    if ((uint32_t)m < (uint32_t)n_models) {
      model = m;
      need = (rho == 0.0) ? kv_bytes[stage] : __dmul_rn(kv_bytes[stage], 1.0 + rho);
      exec_s = __fmul_rn(pred_len[stage], decode_s_per_token[model]);
      mbit = kMat ? 0 : (mask_t)1 << model;
    } else {
      need = NAN;             // a model id out of range: no node admits the stage (NaN <= x is false)
    }
  }

  TopK<KT> best;
  best.init();
  for (int32_t c0 = 0; c0 < n_nodes; c0 += kNodeChunk) {
    const int cn = min(kNodeChunk, n_nodes - c0);
    __syncthreads();  // every lane is done with the previous chunk
    for (int i = tid; i < cn; i += kThreads) {
      const int32_t j = c0 + i;
      s_free[i] = free_bytes[j];
      if constexpr (!kMat) {
        const float q = queue_s[j];
        s_warm[i] = __fadd_rn(q, 0.0f);
        s_cold[i] = __fadd_rn(q, cold_s[j]);
        s_mask[i] = (mask_t)resident_mask[j];
      }
    }
    if constexpr (kMat) {   // rows c0 .. c0+cn-1 of the matrix are contiguous
      const float* rows = act_matrix + (size_t)c0 * n_models;
      for (int e = tid; e < cn * n_models; e += kThreads) s_ready[e] = __fadd_rn(queue_s[c0 + e / n_models], rows[e]);
    }
    __syncthreads();
#pragma unroll 4
    for (int i = g; i < cn; i += G) {
      float ready;
      if constexpr (kMat) ready = s_ready[i * n_models + model];
      else ready = (s_mask[i] & mbit) ? s_warm[i] : s_cold[i];
      const float sc = __fadd_rn(ready, exec_s);
      if (need <= s_free[i]) best.push_increasing(sc, c0 + i);
    }
  }

  // merge the G lane lists of a stage (lanes g and g ^ o exchange and merge)
  for (int o = 1; o < G; o <<= 1) {
    float ps[KT];
    int32_t pn[KT];
#pragma unroll
    for (int i = 0; i < KT; ++i) {
      ps[i] = __shfl_xor(best.s[i], o);
      pn[i] = __shfl_xor(best.n[i], o);
    }
#pragma unroll
    for (int i = 0; i < KT; ++i) best.push_lex(ps[i], pn[i]);
  }

  if (valid && g == 0) {
#pragma unroll
    for (int i = 0; i < KT; ++i) {
      if (i < k) {
        const bool some = best.n[i] != kNoNode;
        node_idx[stage * k + i] = some ? best.n[i] : -1;
        score[stage * k + i] = some ? best.s[i] : INFINITY;
      }
    }
  }
}

template <int KT>
void launch_kt(int ready, dim3 grid, hipStream_t stream, int64_t n, const int32_t* model_id,
               const float* pred_len, const double* kv_bytes, const float* dec, int32_t n_models, int32_t n_nodes,
               const double* free_bytes, const float* queue_s, const float* cold_s,
               const uint64_t* mask, const float* act_matrix, double rho, int32_t k, int g_log2, int32_t* node_idx,
               float* score) {
#define MAESTRO_ROUTE_RD(RD)                                                                               \
  route_kernel<KT, RD><<<grid, dim3(kThreads), 0, stream>>>(n, model_id, pred_len, kv_bytes, dec, n_models, \
                                                           n_nodes, free_bytes, queue_s, cold_s, mask,     \
                                                           act_matrix, rho, k, g_log2, node_idx, score)
  if (ready == kMatrix) MAESTRO_ROUTE_RD(kMatrix);
  else if (ready == kMask64) MAESTRO_ROUTE_RD(kMask64);
  else MAESTRO_ROUTE_RD(kMask32);
#undef MAESTRO_ROUTE_RD
}

// Lanes per stage: enough threads to fill the chip (about 2^18), at least 4 nodes per lane.
int choose_g_log2(int64_t n, int32_t n_nodes) {
  int gl = 0;
  while (gl < 6 && n * (int64_t(1) << gl) < (int64_t(1) << 18) && (int64_t(4) << (gl + 1)) <= n_nodes) ++gl;
  return gl;
}

// ---------------------------------------------------------------------------------------------
// sorted per-model node lists + early-exit walk
// ---------------------------------------------------------------------------------------------

constexpr int kSortMax = 8192;            // nodes sortable in one workgroup (64 KB of keys and indices in LDS)

struct __align__(16) NodeEntry {          // 16 bytes: one node in a model's ready-time order
  float ready;                            // fl32(T_q + T_act) for this model
  int32_t node;
  double free;                            // KV admission headroom
};

// After the lists, per model, the largest headroom of every block of 8, 64 and 512 consecutive
// list entries, rounded up to float32 (-inf past the last node): past its first kPlainWalk
// entries a walk skips every block whose largest headroom cannot admit its stage, so a stage that
// fits few nodes, or none, does not visit every infeasible node. Rounding up keeps the test exact:
// a block is skipped only when its true largest headroom is below the demand too. Measured on c4
// (one GPU): with every headroom divided by 48 (59% of the pairs infeasible, 922 list entries per
// stage) the route call takes 0.44 instead of 9.26 ms; on c4 itself 77.5 instead of 73.4 us (the
// tables cost the sort 1 us, their test the walk 3 us). Gating the walk on the whole list's largest
// headroom, or testing the tables from the first entry past the staged head, cost the c4 walk 3-13
// us more.
__host__ __device__ constexpr int32_t skip_blocks(int32_t n_nodes, int shift) {
  return (n_nodes + (1 << shift) - 1) >> shift;
}
__host__ __device__ constexpr int64_t skip_per_model(int32_t n_nodes) {
  return (int64_t)skip_blocks(n_nodes, 3) + skip_blocks(n_nodes, 6) + skip_blocks(n_nodes, 9);
}

// One workgroup per model puts every node in (ready time, node index) order: a stable LSD radix
// sort of the 32-bit order-preserving image of the ready time (float_key) in four 8-bit passes,
// starting from index order, so equal ready times keep increasing indices. Wavefront w holds
// positions [64 IPT w, 64 IPT (w + 1)), item j the 64 positions from 64 (IPT w + j). There are
// `padded` positions (a power of two, 256 .. 8192, with 256 to 1024 threads); those past the last
// node hold all-ones keys, which a stable pass keeps behind every real key. Each pass ranks a
// wavefront's keys digit by digit with ballots (wave multisplit, in position order), scans the
// per-wavefront digit counts (digit-major, wavefront-minor; one thread per digit) and places keys
// and indices at their new positions in LDS: five barriers per pass. A bitonic network over the
// 64-bit keys (ready, index), with in-register and cross-lane stages and a barrier per cross-
// wavefront stage, took 35 us on 64 models x 4,096 nodes against 20 us for this sort (calls back
// to back, one GPU); taking the digit-count loads of the scan out of its loop (21.3 us), a scan
// spread over all threads plus one wavefront (21.5 us) and 512 threads of 8 keys (23.1 us) were
// slower. LDS: `padded` keys and indices (dynamic), 16 x 256 digit counts.
constexpr int kSortWaves = 16;
constexpr int kSortBuckets = 256;

template <int IPT>
__global__ __launch_bounds__(1024) void sort_nodes_kernel(
    int32_t n_nodes, int32_t padded, int32_t n_models, const float* __restrict__ queue_s,
    const float* __restrict__ cold_s, const uint64_t* __restrict__ resident_mask,
    const float* __restrict__ act_matrix, const double* __restrict__ free_bytes, NodeEntry* __restrict__ lists) {
  extern __shared__ uint32_t s_sort[];                  // [padded] keys, then [padded] indices
  __shared__ uint32_t wcount[kSortWaves][kSortBuckets];
  __shared__ uint32_t dbase[kSortBuckets];
  __shared__ uint32_t wsum[kSortBuckets / 64];
  uint32_t* s_key = s_sort;
  uint32_t* s_idx = s_sort + padded;
  const int m = blockIdx.x, t = threadIdx.x;
  const int wave = t >> 6, lane = t & 63, n_waves = blockDim.x >> 6;
  uint32_t key[IPT], idx[IPT];
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int p = (IPT * wave + j) * 64 + lane;
    idx[j] = (uint32_t)p;
    if (p < n_nodes) {
      const float q = queue_s[p];
      float ready;
      if (act_matrix) {
        ready = __fadd_rn(q, act_matrix[(size_t)p * n_models + m]);
      } else {
        const bool res = (resident_mask[p] >> m) & 1u;
        ready = res ? __fadd_rn(q, 0.0f) : __fadd_rn(q, cold_s[p]);
      }
      key[j] = float_key(ready);
    } else {
      key[j] = 0xFFFFFFFFu;               // padding sorts behind every real key
    }
  }
  const uint64_t lanes_below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll 1
  for (int shift = 0; shift < 32; shift += 8) {
#pragma unroll
    for (int i = lane; i < kSortBuckets; i += 64) wcount[wave][i] = 0;
    // rank among this wavefront's keys of the same digit, in position order (the wavefront's
    // own LDS accesses stay in program order)
    uint32_t dig[IPT], rank[IPT];
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
      const uint32_t d = (key[j] >> shift) & (kSortBuckets - 1);
      uint64_t same = ~0ull;
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        const bool bit = (d >> b) & 1u;
        const uint64_t ones = __ballot(bit);
        same &= bit ? ones : ~ones;
      }
      const uint32_t before = wcount[wave][d];
      dig[j] = d;
      rank[j] = before + (uint32_t)__popcll(same & lanes_below);
      if ((same & lanes_below) == 0ull) wcount[wave][d] = before + (uint32_t)__popcll(same);   // first lane of the digit
    }
    __syncthreads();
    // digit d's wavefront offsets (in place) and total; then the exclusive scan of the totals
    uint32_t tot = 0, incl = 0;
    if (t < kSortBuckets) {
      for (int w = 0; w < n_waves; ++w) {
        const uint32_t c = wcount[w][t];
        wcount[w][t] = tot;
        tot += c;
      }
      incl = tot;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t v = __shfl_up(incl, off);
        if (lane >= off) incl += v;
      }
      if (lane == 63) wsum[wave] = incl;
    }
    __syncthreads();
    if (t < kSortBuckets) {
      uint32_t add = 0;
      for (int w = 0; w < wave; ++w) add += wsum[w];
      dbase[t] = add + incl - tot;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
      const uint32_t pos = dbase[dig[j]] + wcount[wave][dig[j]] + rank[j];
      s_key[pos] = key[j];
      s_idx[pos] = idx[j];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
      const int p = (IPT * wave + j) * 64 + lane;
      key[j] = s_key[p];
      idx[j] = s_idx[p];
    }
    __syncthreads();   // every thread has its keys and the counts are read before the next pass
  }
  NodeEntry* out = lists + (size_t)m * n_nodes;
  float* max8 = reinterpret_cast<float*>(lists + (size_t)n_models * n_nodes) + (size_t)m * skip_per_model(n_nodes);
  float* max64 = max8 + skip_blocks(n_nodes, 3);
  float* max512 = max64 + skip_blocks(n_nodes, 6);
  __shared__ float s_max64[kSortMax / 64];
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int p = (IPT * wave + j) * 64 + lane;
    float f = -INFINITY;
    if (p < n_nodes) {
      NodeEntry e;
      e.ready = key_float(key[j]);
      e.node = (int32_t)idx[j];
      e.free = free_bytes[e.node];
      out[p] = e;
      f = __double2float_ru(e.free);
    }
    // the 64 positions of item j are lanes 0 .. 63 in order: blocks of 8 are lane octets
    f = fmaxf(f, __shfl_xor(f, 1));
    f = fmaxf(f, __shfl_xor(f, 2));
    f = fmaxf(f, __shfl_xor(f, 4));
    if ((lane & 7) == 0 && p < n_nodes) max8[p >> 3] = f;
    f = fmaxf(f, __shfl_xor(f, 8));
    f = fmaxf(f, __shfl_xor(f, 16));
    f = fmaxf(f, __shfl_xor(f, 32));
    if (lane == 0) {
      if (p < n_nodes) max64[p >> 6] = f;
      s_max64[IPT * wave + j] = f;
    }
  }
  __syncthreads();
  for (int b = t; b < skip_blocks(n_nodes, 9); b += (int)blockDim.x) {
    float f = -INFINITY;
    for (int r = 8 * b; r < 8 * b + 8 && r < padded / 64; ++r) f = fmaxf(f, s_max64[r]);
    max512[b] = f;
  }
}

// The first kWalkHead entries of every model's list are staged in LDS by the whole workgroup
// (while each thread's own inputs are in flight), so a walk that ends early never waits on a
// dependent global load. One workgroup per 256 stages: a persistent grid that staged the heads
// once per workgroup, and a walk split into a loop over the head and one over the rest of the
// list, were both slower (120 and 110 us against 94 us per c4 route call on one GPU).
constexpr int kWalkHead = 8;
constexpr int kPlainWalk = 32;            // entries visited before the skip tables are consulted

// one stage's walk down its model's list
template <int KT>
__device__ __forceinline__ void walk_stage(
    int64_t i, const int32_t* __restrict__ model_id, const float* __restrict__ pred_len,
    const double* __restrict__ kv_bytes, const float* __restrict__ decode_s_per_token, int32_t n_models,
    int32_t n_nodes, const NodeEntry* __restrict__ lists, const NodeEntry* s_head, int head, double rho, int32_t k,
    int32_t* __restrict__ node_idx, float* __restrict__ score) {
  const int32_t m = model_id[i];
  if ((uint32_t)m >= (uint32_t)n_models) {   // a model id out of range: no node
    for (int t = 0; t < k; ++t) {
      node_idx[i * k + t] = -1;
      score[i * k + t] = INFINITY;
    }
    return;
  }
  const double need = (rho == 0.0) ? kv_bytes[i] : __dmul_rn(kv_bytes[i], 1.0 + rho);
  const float exec_s = __fmul_rn(pred_len[i], decode_s_per_token[m]);
  TopK<KT> best;
  best.init();
  // one list entry; true when the walk stops there
  auto visit = [&](const NodeEntry& e) {
    if (!(need <= e.free)) return false;                   // infeasible: skip, keep walking
    const float sc = __fadd_rn(e.ready, exec_s);
    if (best.n[KT - 1] != kNoNode && sc > best.s[KT - 1]) return true;   // no later node can enter
    best.push_lex(sc, e.node);
    return false;
  };
  const NodeEntry* lhead = s_head + m * kWalkHead;
  const NodeEntry* list = lists + (size_t)m * n_nodes;
  const float* max8 = reinterpret_cast<const float*>(lists + (size_t)n_models * n_nodes) +
                      (size_t)m * skip_per_model(n_nodes);
  const float* max64 = max8 + skip_blocks(n_nodes, 3);
  const float* max512 = max64 + skip_blocks(n_nodes, 6);
  bool done = false;
  int32_t j = 0;
#pragma unroll 1
  for (; j < n_nodes && j < kPlainWalk; ++j)
    if (visit(j < head ? lhead[j] : list[j])) {
      done = true;
      break;
    }
  while (!done && j < n_nodes) {   // skip blocks whose largest headroom admits nothing
    if ((j & 511) == 0 && !(need <= (double)max512[j >> 9])) { j += 512; continue; }
    if ((j & 63) == 0 && !(need <= (double)max64[j >> 6])) { j += 64; continue; }
    if ((j & 7) == 0 && !(need <= (double)max8[j >> 3])) { j += 8; continue; }
    done = visit(list[j]);
    ++j;
  }
  int32_t outn[KT];
  float outs[KT];
#pragma unroll
  for (int t = 0; t < KT; ++t) {
    const bool some = best.n[t] != kNoNode;
    outn[t] = some ? best.n[t] : -1;
    outs[t] = some ? best.s[t] : INFINITY;
  }
  if ((KT == 2 || KT == 4) && k == KT && ((uintptr_t)(node_idx + i * k) % (4 * KT)) == 0 &&
      ((uintptr_t)(score + i * k) % (4 * KT)) == 0) {   // whole rows as one vector store each
    if constexpr (KT == 4) {
      *reinterpret_cast<int4*>(node_idx + i * k) = make_int4(outn[0], outn[1], outn[2], outn[3]);
      *reinterpret_cast<float4*>(score + i * k) = make_float4(outs[0], outs[1], outs[2], outs[3]);
    } else if constexpr (KT == 2) {
      *reinterpret_cast<int2*>(node_idx + i * k) = make_int2(outn[0], outn[1]);
      *reinterpret_cast<float2*>(score + i * k) = make_float2(outs[0], outs[1]);
    }
    return;
  }
#pragma unroll
  for (int t = 0; t < KT; ++t) {
    if (t < k) {
      node_idx[i * k + t] = outn[t];
      score[i * k + t] = outs[t];
    }
  }
}

template <int KT>
__global__ __launch_bounds__(kThreads) void walk_route_kernel(
    int64_t n, const int32_t* __restrict__ model_id, const float* __restrict__ pred_len,
    const double* __restrict__ kv_bytes, const float* __restrict__ decode_s_per_token, int32_t n_models,
    int32_t n_nodes, const NodeEntry* __restrict__ lists, double rho, int32_t k, int32_t* __restrict__ node_idx,
    float* __restrict__ score) {
  __shared__ NodeEntry s_head[kMaxMatrixModels * kWalkHead];
  const int head = n_nodes < kWalkHead ? n_nodes : kWalkHead;
  for (int e = threadIdx.x; e < n_models * head; e += kThreads)
    s_head[(e / head) * kWalkHead + e % head] = lists[(size_t)(e / head) * n_nodes + e % head];
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < n) walk_stage<KT>(i, model_id, pred_len, kv_bytes, decode_s_per_token, n_models, n_nodes, lists, s_head,
                            head, rho, k, node_idx, score);
}

size_t sorted_lists_bytes(int32_t n_models, int32_t n_nodes) {
  return (size_t)n_models * ((size_t)n_nodes * sizeof(NodeEntry) + (size_t)skip_per_model(n_nodes) * sizeof(float));
}

bool sorted_possible(int32_t n_nodes) { return n_nodes <= kSortMax; }

// the scan wins when there are too few stages to amortise the per-model sorts
bool prefer_sorted(int64_t n, int32_t n_models, int32_t n_nodes) {
  return sorted_possible(n_nodes) && n >= 4 * (int64_t)n_models;
}

}  // namespace

size_t route_lists_bytes(int32_t n_models, int32_t n_nodes) {
  return sorted_possible(n_nodes) ? sorted_lists_bytes(n_models, n_nodes) : 0;
}

maestro_status launch_sort_nodes(int32_t n_models, int32_t n_nodes, const double* free_bytes, const float* queue_s,
                                 const float* cold_s, const uint64_t* resident_mask, const float* act_matrix,
                                 void* lists, hipStream_t stream) {
  if (!sorted_possible(n_nodes)) return MAESTRO_ERR_UNSUPPORTED;
  int pow2 = 256;
  while (pow2 < n_nodes) pow2 <<= 1;
  const int threads = pow2 < 1024 ? pow2 : 1024;       // 256, 512 or 1024: one thread per digit in the scans
  const int ipt = pow2 / threads;                      // 1, 2, 4 or 8 keys per thread
  const int padded = threads * ipt;
  const size_t lds = (size_t)padded * 2 * sizeof(uint32_t);
  NodeEntry* out = static_cast<NodeEntry*>(lists);
#define MAESTRO_SORT(IPT)                                                                                       \
  sort_nodes_kernel<IPT><<<dim3(n_models), dim3(threads), lds, stream>>>(n_nodes, padded, n_models, queue_s, \
                                                                         cold_s, resident_mask, act_matrix,  \
                                                                         free_bytes, out)
  if (ipt == 1) MAESTRO_SORT(1);
  else if (ipt == 2) MAESTRO_SORT(2);
  else if (ipt == 4) MAESTRO_SORT(4);
  else MAESTRO_SORT(8);
#undef MAESTRO_SORT
  return launch_status();
}

maestro_status launch_route_walk(int64_t n, const int32_t* model_id, const float* pred_len, const double* kv_bytes,
                                 const float* decode_s_per_token, int32_t n_models, int32_t n_nodes,
                                 const void* lists, double rho, int32_t k, int32_t* node_idx, float* score,
                                 hipStream_t stream) {
  if (n == 0) return MAESTRO_OK;
  const dim3 grid((unsigned)((n + kThreads - 1) / kThreads));
  const NodeEntry* l = static_cast<const NodeEntry*>(lists);
#define MAESTRO_WALK_KT(KT)                                                                                  \
  walk_route_kernel<KT><<<grid, dim3(kThreads), 0, stream>>>(n, model_id, pred_len, kv_bytes,               \
                                                             decode_s_per_token, n_models, n_nodes, l, rho, \
                                                             k, node_idx, score)
  if (k == 1) MAESTRO_WALK_KT(1);
  else if (k == 2) MAESTRO_WALK_KT(2);
  else if (k == 3) MAESTRO_WALK_KT(3);
  else if (k == 4) MAESTRO_WALK_KT(4);
  else if (k <= 8) MAESTRO_WALK_KT(8);
  else MAESTRO_WALK_KT(16);
#undef MAESTRO_WALK_KT
  return launch_status();
}

size_t route_workspace_bytes(int64_t, int32_t n_models, int32_t n_nodes, int32_t) {
  return sorted_possible(n_nodes) ? sorted_lists_bytes(n_models, n_nodes) : 0;
}

maestro_status launch_route(int64_t n, const int32_t* model_id, const float* pred_len,
                            const double* kv_bytes, const float* decode_s_per_token,
                            int32_t n_models, int32_t n_nodes, const double* free_bytes,
                            const float* queue_s, const float* cold_s,
                            const uint64_t* resident_mask, const float* act_matrix, double rho, int32_t k, int32_t algo,
                            int32_t* node_idx, float* score, void* workspace,
                            size_t workspace_bytes, hipStream_t stream) {
  if (n == 0) return MAESTRO_OK;
  bool sorted;
  if (algo == MAESTRO_ROUTE_SCAN) sorted = false;
  else if (algo == MAESTRO_ROUTE_SORTED) sorted = true;
  else sorted = prefer_sorted(n, n_models, n_nodes);
  if (sorted) {
    if (!sorted_possible(n_nodes)) return MAESTRO_ERR_UNSUPPORTED;
    if (!workspace || workspace_bytes < sorted_lists_bytes(n_models, n_nodes)) return MAESTRO_ERR_WORKSPACE;
    const maestro_status st = launch_sort_nodes(n_models, n_nodes, free_bytes, queue_s, cold_s, resident_mask,
                                                act_matrix, workspace, stream);
    if (st != MAESTRO_OK) return st;
    return launch_route_walk(n, model_id, pred_len, kv_bytes, decode_s_per_token, n_models, n_nodes, workspace,
                             rho, k, node_idx, score, stream);
  }
  const int gl = choose_g_log2(n, n_nodes);
  const int64_t stages_per_block = kThreads >> gl;
  const dim3 grid((unsigned)((n + stages_per_block - 1) / stages_per_block));
  const int ready = act_matrix ? kMatrix : (n_models > 32 ? kMask64 : kMask32);
#define MAESTRO_ROUTE_KT(KT)                                                                          \
  launch_kt<KT>(ready, grid, stream, n, model_id, pred_len, kv_bytes, decode_s_per_token, n_models,   \
                n_nodes, free_bytes, queue_s, cold_s, resident_mask, act_matrix, rho, k, gl, node_idx, score)
  if (k <= 1) MAESTRO_ROUTE_KT(1);
  else if (k <= 2) MAESTRO_ROUTE_KT(2);
  else if (k <= 4) MAESTRO_ROUTE_KT(4);
  else if (k <= 8) MAESTRO_ROUTE_KT(8);
  else MAESTRO_ROUTE_KT(16);
#undef MAESTRO_ROUTE_KT
  return launch_status();
}

}  // namespace maestro

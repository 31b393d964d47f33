// Per-role length regressors (Sec. III-B) as one grouped GEMM.
//
// The paper trains a length regressor per agent role when the role has training data and falls
// back to a shared global model otherwise. Here a role's regressor is a network of the
// predictor's shape with weights of its own; the stages of all roles that have one are
// predicted in a single launch of the fused predictor, whose tiles each belong to one
// regressor. To form such tiles the stages are bucketed by regressor, stably (a counting sort):
//
//   1. role_count_kernel   per 1024-stage block, the number of stages of each regressor;
//   2. role_plan_kernel    one workgroup: each regressor's rows padded to whole tiles of the
//                          predictor (128 rows, 256 for the 512-wide network's two row groups)
//                          and laid out one regressor after another; the start of every
//                          (block, regressor) run, the regressor of every tile, the padding
//                          rows (stage -1) and the tile count;
//   3. role_scatter_kernel each stage's row in that order (rank among the block's stages of its
//                          regressor from wavefront ballots), with its stage index, prompt
//                          length, model id and tool probability, so that the predictor reads
//                          per-stage inputs contiguously and gathers only the feature rows.
//
// Stages of roles without a regressor are not placed; their predictions are left as they are.
#include "internal.h"

namespace maestro {
namespace {

constexpr int kBlock = 1024;
constexpr int kWavesPerBlock = kBlock / 64;
constexpr int kMaxGroups = MAESTRO_MAX_ROLE_REGRESSORS;
constexpr int kRoleTileMin = 128;        // rows of a tile of the fused predictor: one row group,
constexpr int kRoleTileMax = 256;        // or two

__device__ __forceinline__ int regressor_of(int32_t role, const int32_t* __restrict__ role_regressor,
                                            int32_t n_roles, int32_t n_groups) {
  if ((uint32_t)role >= (uint32_t)n_roles) return -1;
  const int32_t g = role_regressor[role];
  return (g >= 0 && g < n_groups) ? g : -1;
}

__global__ __launch_bounds__(kBlock) void role_count_kernel(int64_t n, const int32_t* __restrict__ role_id,
                                                            int32_t n_roles, const int32_t* __restrict__ role_regressor,
                                                            int32_t n_groups, int32_t* __restrict__ counts) {
  __shared__ int32_t wc[kWavesPerBlock][kMaxGroups];
  const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = i < n ? regressor_of(role_id[i], role_regressor, n_roles, n_groups) : -1;
  for (int gg = 0; gg < n_groups; ++gg) {
    const uint64_t m = __ballot(g == gg);
    if (lane == 0) wc[wave][gg] = (int32_t)__popcll(m);
  }
  __syncthreads();
  if ((int)threadIdx.x < n_groups) {
    int32_t t = 0;
    for (int w = 0; w < kWavesPerBlock; ++w) t += wc[w][threadIdx.x];
    counts[(size_t)blockIdx.x * kMaxGroups + threadIdx.x] = t;
  }
}

// exclusive prefix sum of v over the 1024 threads of the block; *total gets the sum
__device__ __forceinline__ int32_t block_exclusive_scan(int32_t v, int32_t* total) {
  __shared__ int32_t ws[kWavesPerBlock];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int32_t x = v;
  for (int d = 1; d < 64; d <<= 1) {
    const int32_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) ws[wave] = x;
  __syncthreads();
  int32_t before = 0, all = 0;
  for (int w = 0; w < kWavesPerBlock; ++w) {
    const int32_t t = ws[w];
    before += w < wave ? t : 0;
    all += t;
  }
  __syncthreads();   // ws is reused by the next call
  *total = all;
  return before + x - v;
}

__global__ __launch_bounds__(kBlock) void role_plan_kernel(int32_t n_blocks, int32_t n_groups, int32_t tile_rows,
                                                           const int32_t* __restrict__ counts,
                                                           int32_t* __restrict__ offsets,
                                                           int32_t* __restrict__ tile_group, int32_t* __restrict__ perm,
                                                           int32_t* __restrict__ prompt_p, int32_t* __restrict__ model_p,
                                                           int32_t* __restrict__ p_bits, int32_t* __restrict__ n_tiles) {
  const int t = threadIdx.x;
  const int per = (n_blocks + kBlock - 1) / kBlock;   // consecutive blocks summed by one thread
  const int b0 = t * per, b1 = min(b0 + per, n_blocks);
  int32_t base = 0;                                    // first row of this regressor's tiles
  for (int g = 0; g < n_groups; ++g) {
    int32_t mine = 0;
    for (int b = b0; b < b1; ++b) mine += counts[(size_t)b * kMaxGroups + g];
    int32_t total;
    int32_t run = base + block_exclusive_scan(mine, &total);
    for (int b = b0; b < b1; ++b) {
      offsets[(size_t)b * kMaxGroups + g] = run;
      run += counts[(size_t)b * kMaxGroups + g];
    }
    const int32_t padded = (total + tile_rows - 1) / tile_rows * tile_rows;
    for (int32_t r = base + total + t; r < base + padded; r += kBlock) {   // padding rows
      perm[r] = -1;
      prompt_p[r] = 0;
      model_p[r] = 0;
      p_bits[r] = 0;
    }
    for (int32_t tt = base / tile_rows + t; tt < (base + padded) / tile_rows; tt += kBlock) tile_group[tt] = g;
    base += padded;
  }
  if (t == 0) n_tiles[0] = base / tile_rows;
}

__global__ __launch_bounds__(kBlock) void role_scatter_kernel(
    int64_t n, const int32_t* __restrict__ role_id, int32_t n_roles, const int32_t* __restrict__ role_regressor,
    int32_t n_groups, const int32_t* __restrict__ offsets, const int32_t* __restrict__ prompt_len,
    const int32_t* __restrict__ model_id, const float* __restrict__ p_tool, int32_t* __restrict__ perm,
    int32_t* __restrict__ prompt_p, int32_t* __restrict__ model_p, int32_t* __restrict__ p_bits) {
  __shared__ int32_t wc[kWavesPerBlock][kMaxGroups];
  __shared__ int32_t wpre[kWavesPerBlock][kMaxGroups];
  const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = i < n ? regressor_of(role_id[i], role_regressor, n_roles, n_groups) : -1;
  int32_t rank = 0;   // earlier lanes of this wavefront with the same regressor
  for (int gg = 0; gg < n_groups; ++gg) {
    const uint64_t m = __ballot(g == gg);
    if (g == gg) rank = (int32_t)__popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wc[wave][gg] = (int32_t)__popcll(m);
  }
  __syncthreads();
  if ((int)threadIdx.x < n_groups) {
    int32_t run = 0;
    for (int w = 0; w < kWavesPerBlock; ++w) {
      wpre[w][threadIdx.x] = run;
      run += wc[w][threadIdx.x];
    }
  }
  __syncthreads();
  if (g >= 0) {
    const int32_t pos = offsets[(size_t)blockIdx.x * kMaxGroups + g] + wpre[wave][g] + rank;
    perm[pos] = (int32_t)i;
    prompt_p[pos] = prompt_len[i];
    model_p[pos] = model_id[i];
    p_bits[pos] = __float_as_int(p_tool[i]);
  }
}

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

struct RoleLayout {
  int64_t rows_max, tiles_max, n_blocks;
  size_t perm, prompt, model, pbits, counts, offsets, tile_group, n_tiles, total;
};

// sized for either tile height: rows padded to the taller tiles, tiles counted at the shorter
RoleLayout role_layout(int64_t n, int32_t n_groups) {
  RoleLayout L{};
  L.rows_max = n + (int64_t)n_groups * (kRoleTileMax - 1);
  L.tiles_max = (L.rows_max + kRoleTileMin - 1) / kRoleTileMin;
  L.n_blocks = (n + kBlock - 1) / kBlock;
  const size_t rb = align256(sizeof(int32_t) * (size_t)(L.tiles_max * kRoleTileMin));
  const size_t cb = align256(sizeof(int32_t) * (size_t)(L.n_blocks * kMaxGroups));
  L.perm = 0;
  L.prompt = L.perm + rb;
  L.model = L.prompt + rb;
  L.pbits = L.model + rb;
  L.counts = L.pbits + rb;
  L.offsets = L.counts + cb;
  L.tile_group = L.offsets + cb;
  L.n_tiles = L.tile_group + align256(sizeof(int32_t) * (size_t)L.tiles_max);
  L.total = L.n_tiles + 256;
  return L;
}

}  // namespace

size_t role_lengths_workspace_bytes(int64_t n, int32_t n_groups) {
  return n > 0 ? role_layout(n, n_groups).total : 0;
}

maestro_status launch_role_lengths(const maestro_predictor& p, const maestro_role_regressors& r, int64_t n,
                                   const void* x, const int32_t* prompt_len, const int32_t* model_id,
                                   const int32_t* role_id, const float* p_tool, const float* kv_bytes_per_token,
                                   int32_t n_models, float* pred_len, double* kv_bytes, void* workspace,
                                   hipStream_t stream) {
  if (n == 0) return MAESTRO_OK;
  const RoleLayout L = role_layout(n, r.n_regressors);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  int32_t* perm = reinterpret_cast<int32_t*>(ws + L.perm);
  int32_t* prompt_p = reinterpret_cast<int32_t*>(ws + L.prompt);
  int32_t* model_p = reinterpret_cast<int32_t*>(ws + L.model);
  int32_t* p_bits = reinterpret_cast<int32_t*>(ws + L.pbits);
  int32_t* counts = reinterpret_cast<int32_t*>(ws + L.counts);
  int32_t* offsets = reinterpret_cast<int32_t*>(ws + L.offsets);
  int32_t* tile_group = reinterpret_cast<int32_t*>(ws + L.tile_group);
  int32_t* n_tiles = reinterpret_cast<int32_t*>(ws + L.n_tiles);
  const int32_t tile_rows = role_tile_rows(p);
  const int64_t tiles_max = (L.rows_max + tile_rows - 1) / tile_rows;
  const dim3 grid((unsigned)L.n_blocks), block(kBlock);
  role_count_kernel<<<grid, block, 0, stream>>>(n, role_id, r.n_roles, r.role_regressor, r.n_regressors, counts);
  role_plan_kernel<<<dim3(1), block, 0, stream>>>((int32_t)L.n_blocks, r.n_regressors, tile_rows, counts, offsets,
                                                 tile_group, perm, prompt_p, model_p, p_bits, n_tiles);
  role_scatter_kernel<<<grid, block, 0, stream>>>(n, role_id, r.n_roles, r.role_regressor, r.n_regressors, offsets,
                                                  prompt_len, model_id, p_tool, perm, prompt_p, model_p, p_bits);
  const maestro_status st = launch_status();
  if (st != MAESTRO_OK) return st;
  return launch_role_regressors(p, n, x, r.tool_coef, r.max_len, tile_group, perm, prompt_p, model_p, p_bits, n_tiles,
                                tiles_max, kv_bytes_per_token, n_models, pred_len, kv_bytes, stream);
}

}  // namespace maestro

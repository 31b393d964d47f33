// Slack ordering of workflows (Sec. III-D, remaining-time queueing; Eq. 7).
//
//  1. chain kernel, one thread per workflow: walks its chain from the last stage backwards,
//     quantising every stage latency to integer microseconds (round half to even) and
//     accumulating the suffix sums in int64 -- the remaining predicted time from each stage to
//     the end of the chain. The remaining time at the workflow's cursor gives
//     slack = deadline - now - remaining, clamped to int32. Integer sums are exact, so the
//     result does not depend on the summation order.
//  2. stable LSD radix sort of the (slack, workflow) pairs, 4 passes of 8-bit digits over the
//     order-preserving unsigned image of the key. Each pass: per-tile digit counts, the
//     exclusive scan of the digit-major count table (global offset of every (digit, tile);
//     done inside the scatter blocks when there are few tiles), and a scatter in which each
//     wavefront ranks its items digit by digit with ballots (wave multisplit) in input order,
//     so equal digits keep their relative order.
//     The key array is padded to whole tiles with all-ones keys, which always sort last and
//     never reach the caller's output.
#include "internal.h"

namespace maestro {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 16;                         // items per thread in a sort tile
constexpr int kTile = kThreads * kItems;           // 4096 keys per tile
constexpr int kWaves = kThreads / 64;
constexpr int kRadixBits = 8;
constexpr int kBuckets = 1 << kRadixBits;
constexpr int kPasses = 32 / kRadixBits;

constexpr int64_t kLatSat = INT64_MAX;             // infinitely late (absorbing)
constexpr double kLatUsLimit = 1099511627776.0;    // 2^40 microseconds

__device__ __forceinline__ int64_t latency_us(float lat_s) {
  if (!isfinite(lat_s)) return kLatSat;
  double us = rint(__dmul_rn((double)lat_s, 1.0e6));
  us = fmin(fmax(us, -kLatUsLimit), kLatUsLimit);
  return (int64_t)us;
}

__device__ __forceinline__ int64_t sat_add(int64_t a, int64_t b) {
  return (a == kLatSat || b == kLatSat) ? kLatSat : a + b;
}

// a - b saturated to the int64 range
__device__ __forceinline__ int64_t sat_sub(int64_t a, int64_t b) {
  int64_t r;
  if (__builtin_sub_overflow(a, b, &r)) r = (a > b) ? INT64_MAX : INT64_MIN;
  return r;
}

__global__ __launch_bounds__(kThreads) void chain_kernel(
    int32_t n_workflows, int64_t padded, const int64_t* __restrict__ chain_offset,
    const float* __restrict__ stage_latency_s, const int32_t* __restrict__ cursor,
    const int64_t* __restrict__ deadline_us, int64_t now_us, int64_t* __restrict__ remaining_us,
    int32_t* __restrict__ slack_key, uint32_t* __restrict__ keys, uint32_t* __restrict__ vals) {
  const int64_t w = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (w >= padded) return;
  if (w >= n_workflows) {  // tile padding: largest key, sorts after every real workflow
    keys[w] = 0xFFFFFFFFu;
    vals[w] = (uint32_t)w;
    return;
  }
  const int64_t first = chain_offset[w], end = chain_offset[w + 1];
  int64_t cur = cursor ? (int64_t)cursor[w] : 0;
  if (cur < 0) cur = 0;
  const int64_t head = first + cur;
  int64_t suffix = 0, rem_head = 0;
  for (int64_t j = end - 1; j >= first; --j) {
    suffix = sat_add(latency_us(stage_latency_s[j]), suffix);
    if (remaining_us) remaining_us[j] = suffix;
    if (j == head) rem_head = suffix;
  }
  int32_t key;
  if (rem_head == kLatSat) {
    key = INT32_MIN;
  } else {
    // |rem_head| <= 2^62, so saturating the two differences keeps the int32 clamp exact
    const int64_t slack = sat_sub(sat_sub(deadline_us[w], now_us), rem_head);
    key = slack > INT32_MAX ? INT32_MAX : (slack < INT32_MIN ? INT32_MIN : (int32_t)slack);
  }
  slack_key[w] = key;
  keys[w] = (uint32_t)key ^ 0x80000000u;   // order-preserving unsigned image
  vals[w] = (uint32_t)w;
}

// Per-tile digit counts, digit-major: counts[d * n_tiles + t].
__global__ __launch_bounds__(kThreads) void radix_count_kernel(const uint32_t* __restrict__ keys,
                                                               int shift, int n_tiles,
                                                               uint32_t* __restrict__ counts) {
  __shared__ uint32_t hist[kBuckets];
  const int tid = threadIdx.x, tile = blockIdx.x;
  hist[tid] = 0;
  __syncthreads();
  const uint32_t* k = keys + (int64_t)tile * kTile;
#pragma unroll
  for (int i = 0; i < kItems; ++i) atomicAdd(&hist[(k[i * kThreads + tid] >> shift) & (kBuckets - 1)], 1u);
  __syncthreads();
  counts[(int64_t)tid * n_tiles + tile] = hist[tid];
}

// Exclusive scan of the count table in place (one workgroup; the table is small next to the
// keys: 256 entries per 4096-key tile).
__global__ __launch_bounds__(1024) void radix_scan_kernel(uint32_t* __restrict__ counts, int64_t total) {
  __shared__ uint32_t part[1024];
  const int tid = threadIdx.x;
  const int64_t per = (total + 1023) / 1024;
  const int64_t lo = min(total, tid * per), hi = min(total, lo + per);
  uint32_t s = 0;
  for (int64_t i = lo; i < hi; ++i) s += counts[i];
  part[tid] = s;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {   // Hillis-Steele inclusive scan
    uint32_t v = tid >= off ? part[tid - off] : 0u;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  uint32_t run = tid ? part[tid - 1] : 0u;
  for (int64_t i = lo; i < hi; ++i) {
    const uint32_t c = counts[i];
    counts[i] = run;
    run += c;
  }
}

// Stable scatter of one tile by the digit at `shift`. Items of the tile are taken in input
// order: wavefront w owns positions [w*1024, (w+1)*1024), step i covers 64 consecutive ones.
// out_keys may be null (last pass); positions >= out_limit are padding and are dropped.
// With kFusedScan the tile derives its digit offsets from the raw count table itself
// (digit totals over all tiles, exclusive-scanned, plus the counts of the earlier tiles);
// otherwise `offsets` holds the scanned table.
template <bool kFusedScan>
__global__ __launch_bounds__(kThreads) void radix_scatter_kernel(
    const uint32_t* __restrict__ keys, const uint32_t* __restrict__ vals, int shift, int n_tiles,
    const uint32_t* __restrict__ offsets, uint32_t* __restrict__ out_keys,
    uint32_t* __restrict__ out_vals, int64_t out_limit) {
  __shared__ uint32_t wcount[kWaves][kBuckets];
  __shared__ uint32_t base[kBuckets];
  const int tid = threadIdx.x, tile = blockIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) wcount[w][tid] = 0;
  if (kFusedScan) {
    // thread d: total of digit d over all tiles, and over the tiles before this one
    const uint32_t* row = offsets + (int64_t)tid * n_tiles;
    uint32_t before = 0, total = 0;
    for (int t = 0; t < n_tiles; ++t) {
      const uint32_t c = row[t];
      before += (t < tile) ? c : 0u;
      total += c;
    }
    base[tid] = total;
    __syncthreads();
    for (int off = 1; off < kBuckets; off <<= 1) {   // inclusive scan of the digit totals
      const uint32_t v = tid >= off ? base[tid - off] : 0u;
      __syncthreads();
      base[tid] += v;
      __syncthreads();
    }
    const uint32_t excl = base[tid] - total;
    __syncthreads();
    base[tid] = excl + before;
  } else {
    base[tid] = offsets[(int64_t)tid * n_tiles + tile];
  }
  __syncthreads();

  const int64_t t0 = (int64_t)tile * kTile + wave * (kTile / kWaves);
  const uint64_t lanes_below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  uint32_t key[kItems], val[kItems], rank[kItems];
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    key[i] = keys[t0 + i * 64 + lane];
    val[i] = vals[t0 + i * 64 + lane];
  }
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const uint32_t d = (key[i] >> shift) & (kBuckets - 1);
    uint64_t same = ~0ull;                     // lanes whose digit equals this lane's
#pragma unroll
    for (int b = 0; b < kRadixBits; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t ones = __ballot(bit);
      same &= bit ? ones : ~ones;
    }
    const uint32_t before = wcount[wave][d];
    rank[i] = before + (uint32_t)__popcll(same & lanes_below);
    if ((same & lanes_below) == 0ull) wcount[wave][d] = before + (uint32_t)__popcll(same);
  }
  __syncthreads();
  {  // offsets of each wavefront inside the tile's digit groups
    uint32_t run = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t c = wcount[w][tid];
      wcount[w][tid] = run;
      run += c;
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const uint32_t d = (key[i] >> shift) & (kBuckets - 1);
    const int64_t pos = (int64_t)base[d] + wcount[wave][d] + rank[i];
    if (pos < out_limit) {
      if (out_keys) out_keys[pos] = key[i];
      out_vals[pos] = val[i];
    }
  }
}

// up to this many tiles each scatter block scans the count table itself
constexpr int kFusedScanMaxTiles = 64;

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

struct PrioLayout {
  int64_t n_tiles, padded;
  size_t keys_a, vals_a, keys_b, vals_b, counts, total;
};

PrioLayout prio_layout(int32_t n_workflows) {
  PrioLayout L{};
  L.n_tiles = ((int64_t)n_workflows + kTile - 1) / kTile;
  L.padded = L.n_tiles * kTile;
  const size_t kb = align256(sizeof(uint32_t) * (size_t)L.padded);
  L.keys_a = 0;
  L.vals_a = L.keys_a + kb;
  L.keys_b = L.vals_a + kb;
  L.vals_b = L.keys_b + kb;
  L.counts = L.vals_b + kb;
  L.total = L.counts + align256(sizeof(uint32_t) * kBuckets * (size_t)L.n_tiles);
  return L;
}

}  // namespace

size_t prioritize_workspace_bytes(int32_t n_workflows, int64_t) {
  return n_workflows > 0 ? prio_layout(n_workflows).total : 0;
}

maestro_status launch_prioritize(int32_t n_workflows, int64_t n_stages,
                                 const int64_t* chain_offset, const float* stage_latency_s,
                                 const int32_t* cursor, const int64_t* deadline_us,
                                 int64_t now_us, int64_t* remaining_us, int32_t* slack_key,
                                 int32_t* order, void* workspace, size_t, hipStream_t stream) {
  (void)n_stages;
  if (n_workflows == 0) return MAESTRO_OK;
  const PrioLayout L = prio_layout(n_workflows);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  uint32_t* keys[2] = {reinterpret_cast<uint32_t*>(ws + L.keys_a), reinterpret_cast<uint32_t*>(ws + L.keys_b)};
  uint32_t* vals[2] = {reinterpret_cast<uint32_t*>(ws + L.vals_a), reinterpret_cast<uint32_t*>(ws + L.vals_b)};
  uint32_t* counts = reinterpret_cast<uint32_t*>(ws + L.counts);

  chain_kernel<<<dim3((unsigned)((L.padded + kThreads - 1) / kThreads)), dim3(kThreads), 0, stream>>>(
      n_workflows, L.padded, chain_offset, stage_latency_s, cursor, deadline_us, now_us,
      remaining_us, slack_key, keys[0], vals[0]);
  const int nt = (int)L.n_tiles;
  for (int pass = 0; pass < kPasses; ++pass) {
    const int src = pass & 1, dst = src ^ 1;
    const int shift = pass * kRadixBits;
    const bool last = pass + 1 == kPasses;
    radix_count_kernel<<<dim3(nt), dim3(kThreads), 0, stream>>>(keys[src], shift, nt, counts);
    uint32_t* out_k = last ? nullptr : keys[dst];
    uint32_t* out_v = last ? reinterpret_cast<uint32_t*>(order) : vals[dst];
    const int64_t limit = last ? (int64_t)n_workflows : L.padded;
    if (nt <= kFusedScanMaxTiles) {
      radix_scatter_kernel<true><<<dim3(nt), dim3(kThreads), 0, stream>>>(
          keys[src], vals[src], shift, nt, counts, out_k, out_v, limit);
    } else {
      radix_scan_kernel<<<dim3(1), dim3(1024), 0, stream>>>(counts, (int64_t)kBuckets * nt);
      radix_scatter_kernel<false><<<dim3(nt), dim3(kThreads), 0, stream>>>(
          keys[src], vals[src], shift, nt, counts, out_k, out_v, limit);
    }
  }
  return launch_status();
}

}  // namespace maestro

// Slack ordering of workflows (Sec. III-D, remaining-time queueing; Eq. 7).
//
//  1. chain kernel, one thread per workflow and one 1024-thread block per sort tile: walks the
//     workflow's chain from the last stage backwards, quantising every stage latency to integer
//     microseconds (round half to even) and accumulating the suffix sums in int64 -- the
//     remaining predicted time from each stage to the end of the chain. The stage latencies
//     are loaded eight at a time, so a chain costs one memory round trip per eight stages. The
//     remaining time at the workflow's cursor gives slack = deadline - now - remaining,
//     clamped to int32. Integer sums are exact, so the result does not depend on the
//     summation order. The block also counts the first radix digit of its tile.
//  2. stable LSD radix sort of the (slack, workflow) pairs, 4 passes of 8-bit digits over the
//     order-preserving unsigned image of the key, on 1024-key tiles, one key per thread of a
//     1024-thread block. Each pass: per-tile digit counts (for the first pass, from the chain
//     kernel); the global offset of every (digit, tile), i.e. the exclusive scan of the count
//     table in digit-major order, which each scatter block derives itself from the table when
//     there are few tiles (four threads per digit read it, one memory round trip) and a
//     separate one-block scan writes otherwise; and a scatter in which each wavefront ranks
//     its keys digit by digit with ballots (wave multisplit) in input order, so equal digits
//     keep their relative order.
//     The key array is padded to whole tiles with all-ones keys, which always sort last and
//     never reach the caller's output.
#include "internal.h"

namespace maestro {
namespace {

constexpr int kTile = 1024;                        // keys per sort tile = threads per block
constexpr int kWaves = kTile / 64;
constexpr int kRadixBits = 8;
constexpr int kBuckets = 1 << kRadixBits;
constexpr int kPasses = 32 / kRadixBits;
// count table: counts[t * kBuckets + d] = keys of tile t with digit d (tile-major)

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

constexpr int kChainBatch = 8;                     // stage latencies loaded per round trip

// One block per sort tile, one workflow per thread; also writes the tile's counts of the
// first digit.
__global__ __launch_bounds__(kTile) void chain_kernel(
    int32_t n_workflows, const int64_t* __restrict__ chain_offset,
    const float* __restrict__ stage_latency_s, const int32_t* __restrict__ cursor,
    const int64_t* __restrict__ deadline_us, int64_t now_us, int64_t* __restrict__ remaining_us,
    int32_t* __restrict__ slack_key, uint32_t* __restrict__ keys, uint32_t* __restrict__ vals,
    uint32_t* __restrict__ counts) {
  __shared__ uint32_t hist[kBuckets];
  const int tid = threadIdx.x, tile = blockIdx.x;
  if (tid < kBuckets) hist[tid] = 0;
  __syncthreads();
  const int64_t w = (int64_t)tile * kTile + tid;
  uint32_t ukey = 0xFFFFFFFFu;   // tile padding: largest key, sorts after every real workflow
  if (w < n_workflows) {
    const int64_t first = chain_offset[w], end = chain_offset[w + 1];
    int64_t cur = cursor ? (int64_t)cursor[w] : 0;
    if (cur < 0) cur = 0;
    const int64_t head = first + cur;
    int64_t suffix = 0, rem_head = 0;
    for (int64_t top = end - 1; top >= first; top -= kChainBatch) {
      float lat[kChainBatch];
#pragma unroll
      for (int u = 0; u < kChainBatch; ++u) lat[u] = (top - u >= first) ? stage_latency_s[top - u] : 0.0f;
#pragma unroll
      for (int u = 0; u < kChainBatch; ++u) {
        const int64_t j = top - u;
        if (j >= first) {
          suffix = sat_add(latency_us(lat[u]), suffix);
          if (remaining_us) remaining_us[j] = suffix;
          if (j == head) rem_head = suffix;
        }
      }
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
    ukey = (uint32_t)key ^ 0x80000000u;   // order-preserving unsigned image
  }
  keys[w] = ukey;
  vals[w] = (uint32_t)w;
  atomicAdd(&hist[ukey & (kBuckets - 1)], 1u);
  __syncthreads();
  if (tid < kBuckets) counts[(int64_t)tile * kBuckets + tid] = hist[tid];
}

// Per-tile digit counts of the digit at `shift`.
__global__ __launch_bounds__(kTile) void radix_count_kernel(const uint32_t* __restrict__ keys, int shift,
                                                            uint32_t* __restrict__ counts) {
  __shared__ uint32_t hist[kBuckets];
  const int tid = threadIdx.x, tile = blockIdx.x;
  if (tid < kBuckets) hist[tid] = 0;
  __syncthreads();
  atomicAdd(&hist[(keys[(int64_t)tile * kTile + tid] >> shift) & (kBuckets - 1)], 1u);
  __syncthreads();
  if (tid < kBuckets) counts[(int64_t)tile * kBuckets + tid] = hist[tid];
}

// Global offsets for many tiles (one workgroup): offsets[t * kBuckets + d] = keys with a
// smaller digit anywhere, plus keys with digit d in tiles before t -- the exclusive scan of
// the count table taken in digit-major order.
__global__ __launch_bounds__(1024) void radix_scan_kernel(const uint32_t* __restrict__ counts, int n_tiles,
                                                          uint32_t* __restrict__ offsets) {
  __shared__ uint32_t part[1024];
  const int tid = threadIdx.x;
  const int64_t total = (int64_t)kBuckets * n_tiles;
  const int64_t per = (total + 1023) / 1024;
  const int64_t lo = min(total, tid * per), hi = min(total, lo + per);
  // logical index i = d * n_tiles + t lives at t * kBuckets + d
  auto at = [&](int64_t i) { return (i % n_tiles) * kBuckets + i / n_tiles; };
  uint32_t s = 0;
  for (int64_t i = lo; i < hi; ++i) s += counts[at(i)];
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
    const int64_t a = at(i);
    const uint32_t c = counts[a];
    offsets[a] = run;
    run += c;
  }
}

// Stable scatter of one tile by the digit at `shift`, one key per thread: wavefront w holds
// tile positions [64w, 64w + 64). out_keys may be null (last pass); positions >= out_limit are
// padding and are dropped. With kFusedScan the block derives its digit offsets from the count
// table (digit totals over all tiles, exclusive-scanned, plus the counts of the earlier
// tiles); otherwise `table` holds the offsets written by radix_scan_kernel.
constexpr int kFusedScanMaxTiles = 128;
template <bool kFusedScan>
__global__ __launch_bounds__(kTile) void radix_scatter_kernel(
    const uint32_t* __restrict__ keys, const uint32_t* __restrict__ vals, int shift, int n_tiles,
    const uint32_t* __restrict__ table, uint32_t* __restrict__ out_keys, uint32_t* __restrict__ out_vals,
    int64_t out_limit) {
  __shared__ uint32_t wcount[kWaves][kBuckets];
  __shared__ uint32_t base[kBuckets];
  __shared__ uint32_t part_before[4][kBuckets], part_total[4][kBuckets];
  const int tid = threadIdx.x, tile = blockIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int64_t pos_in = (int64_t)tile * kTile + tid;
  const uint32_t key = keys[pos_in], val = vals[pos_in];
  for (int i = tid; i < kWaves * kBuckets; i += kTile) (&wcount[0][0])[i] = 0;

  if (kFusedScan) {
    // thread (q, d), q = tid / 256: digit d over tiles q, q + 4, q + 8, ...: all loads of a
    // thread are independent and go out together
    const int d = tid & (kBuckets - 1), q = tid >> 8;
    uint32_t before = 0, total = 0;
    constexpr int kUnroll = kFusedScanMaxTiles / 4;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int t = q + 4 * u;
      const uint32_t c = t < n_tiles ? table[(int64_t)t * kBuckets + d] : 0u;
      total += c;
      before += t < tile ? c : 0u;
    }
    part_before[q][d] = before;
    part_total[q][d] = total;
    __syncthreads();
    if (tid < kBuckets) {
      base[tid] = part_total[0][tid] + part_total[1][tid] + part_total[2][tid] + part_total[3][tid];
      part_before[0][tid] += part_before[1][tid] + part_before[2][tid] + part_before[3][tid];
    }
    __syncthreads();
    for (int off = 1; off < kBuckets; off <<= 1) {   // inclusive scan of the digit totals
      uint32_t v = 0;
      if (tid < kBuckets && tid >= off) v = base[tid - off];
      __syncthreads();
      if (tid < kBuckets) base[tid] += v;
      __syncthreads();
    }
    if (tid < kBuckets) {
      const uint32_t incl = base[tid];
      const uint32_t own = part_total[0][tid] + part_total[1][tid] + part_total[2][tid] + part_total[3][tid];
      base[tid] = incl - own + part_before[0][tid];
    }
  } else {
    if (tid < kBuckets) base[tid] = table[(int64_t)tile * kBuckets + tid];
  }
  __syncthreads();

  // rank among the lanes of this wavefront with the same digit, in lane order
  const uint32_t d = (key >> shift) & (kBuckets - 1);
  uint64_t same = ~0ull;
#pragma unroll
  for (int b = 0; b < kRadixBits; ++b) {
    const bool bit = (d >> b) & 1u;
    const uint64_t ones = __ballot(bit);
    same &= bit ? ones : ~ones;
  }
  const uint64_t lanes_below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const uint32_t rank = (uint32_t)__popcll(same & lanes_below);
  if ((same & lanes_below) == 0ull) wcount[wave][d] = (uint32_t)__popcll(same);   // first lane of the digit
  __syncthreads();
  if (tid < kBuckets) {   // offsets of each wavefront inside the tile's digit groups
    uint32_t run = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t c = wcount[w][tid];
      wcount[w][tid] = run;
      run += c;
    }
  }
  __syncthreads();
  const int64_t pos = (int64_t)base[d] + wcount[wave][d] + rank;
  if (pos < out_limit) {
    if (out_keys) out_keys[pos] = key;
    out_vals[pos] = val;
  }
}

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

struct PrioLayout {
  int64_t n_tiles, padded;
  size_t keys_a, vals_a, keys_b, vals_b, counts, offsets, total;
};

PrioLayout prio_layout(int32_t n_workflows) {
  PrioLayout L{};
  L.n_tiles = ((int64_t)n_workflows + kTile - 1) / kTile;
  L.padded = L.n_tiles * kTile;
  const size_t kb = align256(sizeof(uint32_t) * (size_t)L.padded);
  const size_t cb = align256(sizeof(uint32_t) * kBuckets * (size_t)L.n_tiles);
  L.keys_a = 0;
  L.vals_a = L.keys_a + kb;
  L.keys_b = L.vals_a + kb;
  L.vals_b = L.keys_b + kb;
  L.counts = L.vals_b + kb;
  L.offsets = L.counts + cb;
  L.total = L.offsets + (L.n_tiles > kFusedScanMaxTiles ? cb : 0);
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
  uint32_t* offsets = reinterpret_cast<uint32_t*>(ws + L.offsets);

  const int nt = (int)L.n_tiles;
  const bool fused = nt <= kFusedScanMaxTiles;
  chain_kernel<<<dim3((unsigned)nt), dim3(kTile), 0, stream>>>(
      n_workflows, chain_offset, stage_latency_s, cursor, deadline_us, now_us, remaining_us,
      slack_key, keys[0], vals[0], counts);
  for (int pass = 0; pass < kPasses; ++pass) {
    const int src = pass & 1, dst = src ^ 1;
    const int shift = pass * kRadixBits;
    const bool last = pass + 1 == kPasses;
    if (pass > 0)   // the chain kernel counted the first digit
      radix_count_kernel<<<dim3(nt), dim3(kTile), 0, stream>>>(keys[src], shift, counts);
    uint32_t* out_k = last ? nullptr : keys[dst];
    uint32_t* out_v = last ? reinterpret_cast<uint32_t*>(order) : vals[dst];
    const int64_t limit = last ? (int64_t)n_workflows : L.padded;
    if (fused) {
      radix_scatter_kernel<true><<<dim3(nt), dim3(kTile), 0, stream>>>(
          keys[src], vals[src], shift, nt, counts, out_k, out_v, limit);
    } else {
      radix_scan_kernel<<<dim3(1), dim3(1024), 0, stream>>>(counts, nt, offsets);
      radix_scatter_kernel<false><<<dim3(nt), dim3(kTile), 0, stream>>>(
          keys[src], vals[src], shift, nt, offsets, out_k, out_v, limit);
    }
  }
  return launch_status();
}

}  // namespace maestro

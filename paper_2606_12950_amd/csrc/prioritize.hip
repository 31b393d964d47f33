// Slack ordering of workflows (Sec. III-D, remaining-time queueing; Eq. 7).
//
//  1. chain kernel, one thread per workflow and one 1024-thread block per sort tile: walks the
//     workflow's chain from the last stage backwards, quantising every stage latency to integer
//     microseconds (round half to even) and accumulating the suffix sums in int64 -- the
//     remaining predicted time from each stage to the end of the chain. The stage latencies
//     are loaded eight at a time, so a chain costs one memory round trip per eight stages.
//     Chains of more than 1,024 stages are left to a second kernel, whose workgroups scan them
//     one after the other: 1,024-stage chunks from the end backwards, a block-wide exclusive
//     scan of saturating sums per chunk plus the carry of the chunks after it. The
//     remaining time at the workflow's cursor gives slack = deadline - now - remaining,
//     clamped to int32. Integer sums are exact, so the result does not depend on the
//     summation order. The block also counts the first radix digit of its tile.
//  2. stable LSD radix sort of the (slack, workflow) pairs, 4 passes of 8-bit digits over the
//     order-preserving unsigned image of the key, on 1024-key tiles, one key per thread of a
//     1024-thread block. Each pass: per-tile digit counts (for the first pass, from the chain
//     kernel); the global offset of every (digit, tile), i.e. the exclusive scan of the count
//     table in digit-major order, which each scatter block derives itself from the table when
//     there are few tiles (four threads per digit read it, one memory round trip); with many
//     tiles a group scan (prefix of each digit within groups of 16 .. 256 tiles, in place, plus
//     the group totals) and a one-block scan over the group totals and the digits prepare it, and
//     the scatter adds two table entries; and a scatter in which each wavefront ranks its keys
//     digit by digit with ballots (wave multisplit) in input order, so equal digits keep their
//     relative order.
//     The key array is padded to whole tiles with all-ones keys, which always sort last and
//     never reach the caller's output.
#include <atomic>
#include <mutex>

#include "internal.h"

// Scratch of maestro_prioritize_noalloc: the radix key/value buffers and count tables of the
// largest batch it takes, in static device memory that every GPU the library runs on holds
// until the process ends. Host code never names it: kernels get the address resolved per device
// by hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[MAESTRO_PRIORITIZE_NOALLOC_SCRATCH_BYTES];

namespace maestro {
namespace {

constexpr int kTile = 1024;                        // threads per block (and keys per small tile)
constexpr int kWaves = kTile / 64;
constexpr int kBigItems = 4;                       // keys per thread in the tiles of large batches
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
constexpr int64_t kLongChain = 1024;               // longer chains: the whole block scans them
constexpr int kLongItems = 1;                      // stages per thread per chunk of a long chain (more
                                                   // cost registers that every chain pays for)

__device__ __forceinline__ int64_t shfl_up_i64(int64_t v, int d) {
  const int lo = __shfl_up((int)(uint32_t)v, d, 64), hi = __shfl_up((int)(uint32_t)((uint64_t)v >> 32), d, 64);
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// exclusive scan of saturating int64 sums over the block's threads in thread order (sat_add is
// associative: +inf absorbs, and no finite sum of a chain can overflow); returns the sum over
// the threads before this one and, in *total, the block's. Uses wtot; consecutive calls must be
// separated by a barrier.
__device__ __forceinline__ int64_t block_exclusive_sat(int64_t x, int64_t* wtot, int64_t* total) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  int64_t incl = x;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int64_t y = shfl_up_i64(incl, d);
    if (lane >= d) incl = sat_add(y, incl);
  }
  const int64_t prev = shfl_up_i64(incl, 1);
  const int64_t excl = lane > 0 ? prev : 0;   // within the wavefront
  if (lane == 63) wtot[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    int64_t t = lane < kTile / 64 ? wtot[lane] : 0;
#pragma unroll
    for (int d = 1; d < kTile / 64; d <<= 1) {
      const int64_t y = shfl_up_i64(t, d);
      if (lane >= d) t = sat_add(y, t);
    }
    if (lane < kTile / 64) wtot[lane] = t;   // inclusive over wavefronts
  }
  __syncthreads();
  *total = wtot[kTile / 64 - 1];
  return sat_add(wave > 0 ? wtot[wave - 1] : 0, excl);
}

// Suffix sums of one long chain [first, end) by the whole block: chunks of kTile * kLongItems
// stages from the end backwards, thread t taking the chunk's stages from its end in reverse, so
// that an inclusive scan in thread order gives each stage the sum of the stages at and after it
// within the chunk; the chunks after it add their total (carry). kStaged: the quantised
// latencies are read from LDS (stage_us, indexed from s_lo) and the suffix sums written back
// there; otherwise stage_latency_s is quantised and the sums go to remaining_us (when given).
// Returns, in every thread, the suffix sum at `head` (0 when head is past the chain).
template <bool kStaged>
__device__ int64_t long_chain_suffix(int64_t first, int64_t end, int64_t head, int64_t s_lo, int64_t* stage_us,
                                     const float* __restrict__ stage_latency_s, int64_t* __restrict__ remaining_us,
                                     int64_t* wtot, int64_t* s_head) {
  const int tid = threadIdx.x;
  if (tid == 0) *s_head = 0;
  int64_t carry = 0;
  for (int64_t cend = end; cend > first; cend -= (int64_t)kTile * kLongItems) {
    int64_t v[kLongItems];
    int64_t run = 0;
#pragma unroll
    for (int u = 0; u < kLongItems; ++u) {
      const int64_t j = cend - 1 - ((int64_t)tid * kLongItems + u);
      int64_t lat = 0;
      if (j >= first) {
        if constexpr (kStaged) lat = stage_us[j - s_lo];
        else lat = latency_us(stage_latency_s[j]);
      }
      run = sat_add(lat, run);
      v[u] = run;   // this thread's stages from its first (latest) one down to j
    }
    int64_t chunk_total;
    const int64_t before = sat_add(carry, block_exclusive_sat(run, wtot, &chunk_total));   // later stages
#pragma unroll
    for (int u = 0; u < kLongItems; ++u) {
      const int64_t j = cend - 1 - ((int64_t)tid * kLongItems + u);
      if (j >= first) {
        const int64_t suf = sat_add(before, v[u]);
        if constexpr (kStaged) stage_us[j - s_lo] = suf;
        else if (remaining_us) remaining_us[j] = suf;
        if (j == head) *s_head = suf;
      }
    }
    carry = sat_add(carry, chunk_total);
    __syncthreads();   // wtot is reused by the next chunk; *s_head is final after the last one
  }
  const int64_t r = *s_head;
  __syncthreads();   // every thread has read it before the next long chain resets it
  return r;
}

// One block per sort tile, one workflow per thread; also writes the tile's counts of the
// first digit. When the block's workflows span at most kStageCap stages (the usual case), the
// stage latencies pass through LDS: quantised by a coalesced sweep over the block's stage
// range, summed per chain from LDS, and the remaining times written back by a second coalesced
// sweep. Longer ranges walk the chains in global memory directly.
constexpr int kStageCap = 8192;
__global__ __launch_bounds__(kTile) void chain_kernel(
    int32_t n_workflows, const int64_t* __restrict__ chain_offset,
    const float* __restrict__ stage_latency_s, const int32_t* __restrict__ cursor,
    const int64_t* __restrict__ deadline_us, int64_t now_us, int64_t* __restrict__ remaining_us,
    int32_t* __restrict__ slack_key, uint32_t* __restrict__ keys, uint32_t* __restrict__ vals,
    uint32_t* __restrict__ counts, uint32_t* __restrict__ long_flag, uint32_t epoch) {
  __shared__ uint32_t hist[kBuckets];
  __shared__ int64_t stage_us[kStageCap];
  const int tid = threadIdx.x, tile = blockIdx.x;
  if (tid < kBuckets) hist[tid] = 0;
  const int64_t w = (int64_t)tile * kTile + tid;
  // blocks past the last workflow (padding of large batches) have an empty stage range
  const int64_t w_lo = min((int64_t)n_workflows, (int64_t)tile * kTile);
  const int64_t w_hi = min((int64_t)n_workflows, (int64_t)tile * kTile + kTile);
  const int64_t s_lo = chain_offset[w_lo], s_hi = chain_offset[w_hi];   // block-uniform
  const bool staged = s_hi - s_lo <= kStageCap;
  if (staged) {
    for (int64_t j = s_lo + tid; j < s_hi; j += kTile) stage_us[j - s_lo] = latency_us(stage_latency_s[j]);
  }
  __syncthreads();
  uint32_t ukey = 0xFFFFFFFFu;   // tile padding: largest key, sorts after every real workflow
  uint32_t long_mark = 0;        // top bit of vals[w]: a chain long_chain_kernel scans
  if (w < n_workflows) {
    const int64_t first = chain_offset[w], end = chain_offset[w + 1];
    int64_t cur = cursor ? (int64_t)cursor[w] : 0;
    if (cur < 0) cur = 0;
    const int64_t head = first + cur;
    int64_t suffix = 0, rem_head = 0;
    if (end - first > kLongChain) {
      long_mark = 0x80000000u;   // left to long_chain_kernel, which replaces the placeholder key (rem_head 0)
      *long_flag = epoch;        // this call has a long chain (every writer stores the same value)
    } else if (staged) {
      // not unrolled: chains are a few stages long, and the unrolled form's set-up (64-bit
      // addresses of eight stages) costs more than the loop itself
#pragma unroll 1
      for (int64_t j = end - 1; j >= first; --j) {
        suffix = sat_add(stage_us[j - s_lo], suffix);
        stage_us[j - s_lo] = suffix;
        if (j == head) rem_head = suffix;
      }
    } else {
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
  vals[w] = (uint32_t)w | long_mark;
  atomicAdd(&hist[ukey & (kBuckets - 1)], 1u);
  __syncthreads();
  if (counts && tid < kBuckets) counts[(int64_t)tile * kBuckets + tid] = hist[tid];
  if (staged && remaining_us) {
    for (int64_t j = s_lo + tid; j < s_hi; j += kTile) remaining_us[j] = stage_us[j - s_lo];
  }
}

// The chains of more than kLongChain stages, after the chain kernel (which leaves them a
// placeholder key and marks them in the top bit of their index in vals -- indices are below
// 2^31): persistent workgroups take the chain kernel's 1024-workflow tiles in turn, find the
// marked chains of a tile (clearing the mark), scan each with all their threads (long_chain_suffix;
// remaining times written over whatever the chain kernel's LDS write-back left there), and give
// the workflow its slack key; with small tiles they also move the tile's first-digit count
// from the placeholder to the real key (one workgroup owns a tile, so no other touches those
// counts). Kept out of the chain kernel: the registers of the scan there slowed every chain (by
// half at 2^24 workflows); persistent, since one short-lived workgroup per tile cost more in
// scheduling than the check itself. A call without long chains (the chain kernel's flag word does
// not hold this call's number) returns at once instead of reading every mark (41 us at 2^24
// workflows).
constexpr int kLongChainBlocks = 512;
constexpr int kLongChainTilesPerCheck = 8;   // at most this many tiles' marks per barrier
__global__ __launch_bounds__(kTile) void long_chain_kernel(
    int32_t n_workflows, const int64_t* __restrict__ chain_offset, const float* __restrict__ stage_latency_s,
    const int32_t* __restrict__ cursor, const int64_t* __restrict__ deadline_us, int64_t now_us,
    int64_t* __restrict__ remaining_us, int32_t* __restrict__ slack_key, uint32_t* __restrict__ keys,
    uint32_t* __restrict__ vals, uint32_t* __restrict__ counts, int tiles_per_check,
    const uint32_t* __restrict__ long_flag, uint32_t epoch) {
  __shared__ int64_t wtot[kTile / 64];
  __shared__ int64_t s_head_rem;
  __shared__ int32_t s_long[kTile];
  __shared__ int32_t s_n_long;
  const int tid = threadIdx.x;
  const int64_t n_tiles = ((int64_t)n_workflows + kTile - 1) / kTile;
  const int kT = tiles_per_check;   // 1 .. kLongChainTilesPerCheck
  if (*long_flag != epoch) return;  // the usual case: no chain of this call is long
  for (int64_t t0 = (int64_t)blockIdx.x * kT; t0 < n_tiles; t0 += (int64_t)gridDim.x * kT) {   // workgroup-uniform
    uint32_t marks = 0;   // bit i: this thread's workflow of tile t0 + i is marked
#pragma unroll
    for (int i = 0; i < kLongChainTilesPerCheck; ++i) {
      const int64_t wi = (t0 + i) * kTile + tid;
      if (i < kT && wi < n_workflows && (vals[wi] & 0x80000000u)) marks |= 1u << i;
    }
    if (__syncthreads_count(marks != 0) == 0) continue;   // the usual case: none in these tiles
    for (int64_t tile = t0; tile < t0 + kT && tile < n_tiles; ++tile) {   // workgroup-uniform
      const int64_t w = tile * kTile + tid;
      const bool is_long = (marks >> (tile - t0)) & 1u;
      if (tid == 0) s_n_long = 0;
      if (__syncthreads_count(is_long) == 0) continue;
      if (is_long) s_long[atomicAdd(&s_n_long, 1)] = tid;
      __syncthreads();
      const int n_long = s_n_long;
      int64_t rem_head = 0;
      for (int q = 0; q < n_long; ++q) {   // workgroup-uniform trip count
        const int t = s_long[q];
        const int64_t wl = tile * kTile + t;
        const int64_t first = chain_offset[wl], end = chain_offset[wl + 1];
        int64_t cur = cursor ? (int64_t)cursor[wl] : 0;
        if (cur < 0) cur = 0;
        const int64_t r = long_chain_suffix<false>(first, end, first + cur, 0, nullptr, stage_latency_s, remaining_us,
                                                   wtot, &s_head_rem);
        if (tid == t) rem_head = r;
      }
      if (is_long) {
        int32_t key;
        if (rem_head == kLatSat) {
          key = INT32_MIN;
        } else {
          const int64_t slack = sat_sub(sat_sub(deadline_us[w], now_us), rem_head);
          key = slack > INT32_MAX ? INT32_MAX : (slack < INT32_MIN ? INT32_MIN : (int32_t)slack);
        }
        slack_key[w] = key;
        const uint32_t ukey = (uint32_t)key ^ 0x80000000u;
        const uint32_t placeholder = keys[w];
        keys[w] = ukey;
        vals[w] = (uint32_t)w;
        if (counts) {
          atomicSub(&counts[tile * kBuckets + (placeholder & (kBuckets - 1))], 1u);
          atomicAdd(&counts[tile * kBuckets + (ukey & (kBuckets - 1))], 1u);
        }
      }
      __syncthreads();   // s_long and s_n_long are reused by the next tile
    }
  }
}

// Per-tile digit counts of the digit at `shift`; tiles of kTile * ITEMS keys.
template <int ITEMS>
__global__ __launch_bounds__(kTile) void radix_count_kernel(const uint32_t* __restrict__ keys, int shift,
                                                            uint32_t* __restrict__ counts) {
  __shared__ uint32_t hist[kBuckets];
  const int tid = threadIdx.x, tile = blockIdx.x;
  if (tid < kBuckets) hist[tid] = 0;
  __syncthreads();
  uint32_t k[ITEMS];
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) k[i] = keys[(int64_t)tile * (kTile * ITEMS) + i * kTile + tid];
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) atomicAdd(&hist[(k[i] >> shift) & (kBuckets - 1)], 1u);
  __syncthreads();
  if (tid < kBuckets) counts[(int64_t)tile * kBuckets + tid] = hist[tid];
}

// Many tiles, step 1: one block per group of group_tiles tiles (a power of two, 16 .. 256, so
// that there are at most 64 groups up to 2^26 keys: the group scans spread over as many
// workgroups as that allows, and the one-workgroup top scan stays short). In place, counts[t][d]
// becomes the number of keys with digit d in the tiles of t's group before t; gsum[group][d]
// gets the group's total. Thread (q, d) runs over the tiles q*group_tiles/4 .. of the group for
// digit d (for a fixed tile, a wavefront's 64 digits are consecutive words).
constexpr int kMinGroupTiles = 16, kMaxGroupTiles = 256, kTargetGroups = 64;
constexpr int kBatch = 16;                         // independent loads in flight per thread

// Exclusive prefix, in place, of the column entries t0 .. t1-1 (row stride kBuckets words) of a
// digit; returns the column total. Loads go out kBatch at a time.
__device__ __forceinline__ uint32_t column_prefix(uint32_t* __restrict__ table, int64_t t0, int64_t t1, int d,
                                                  uint32_t start) {
  uint32_t run = start;
  for (int64_t t = t0; t < t1; t += kBatch) {
    uint32_t c[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) c[u] = (t + u < t1) ? table[(t + u) * kBuckets + d] : 0u;
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      if (t + u < t1) {
        table[(t + u) * kBuckets + d] = run;
        run += c[u];
      }
  }
  return run - start;
}

__device__ __forceinline__ uint32_t column_sum(const uint32_t* __restrict__ table, int64_t t0, int64_t t1, int d) {
  uint32_t run = 0;
  for (int64_t t = t0; t < t1; t += kBatch) {
    uint32_t c[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) c[u] = (t + u < t1) ? table[(t + u) * kBuckets + d] : 0u;
#pragma unroll
    for (int u = 0; u < kBatch; ++u) run += c[u];
  }
  return run;
}

__global__ __launch_bounds__(1024) void radix_group_scan_kernel(uint32_t* __restrict__ counts, int n_tiles,
                                                                int group_tiles, uint32_t* __restrict__ gsum) {
  __shared__ uint32_t part[4][kBuckets];
  const int tid = threadIdx.x, d = tid & (kBuckets - 1), q = tid >> 8;
  const int t0 = min(n_tiles, blockIdx.x * group_tiles + q * (group_tiles / 4));
  const int t1 = min(n_tiles, t0 + group_tiles / 4);
  part[q][d] = column_sum(counts, t0, t1, d);
  __syncthreads();
  uint32_t before = 0;
  for (int i = 0; i < q; ++i) before += part[i][d];
  column_prefix(counts, t0, t1, d, before);
  if (q == 0) gsum[(int64_t)blockIdx.x * kBuckets + d] = part[0][d] + part[1][d] + part[2][d] + part[3][d];
}

// Many tiles, step 2 (one workgroup): gsum[group][d] becomes the global offset of the group's
// first key with digit d -- keys with a smaller digit anywhere plus keys with digit d in
// earlier groups.
__global__ __launch_bounds__(1024) void radix_top_scan_kernel(uint32_t* __restrict__ gsum, int n_groups) {
  __shared__ uint32_t part[4][kBuckets];
  __shared__ uint32_t base[kBuckets];
  const int tid = threadIdx.x, d = tid & (kBuckets - 1), q = tid >> 8;
  const int per = (n_groups + 3) / 4;
  const int g0 = min(n_groups, q * per), g1 = min(n_groups, g0 + per);
  part[q][d] = column_sum(gsum, g0, g1, d);
  __syncthreads();
  if (tid < kBuckets) base[tid] = part[0][tid] + part[1][tid] + part[2][tid] + part[3][tid];
  __syncthreads();
  for (int off = 1; off < kBuckets; off <<= 1) {   // inclusive scan of the digit totals
    uint32_t v = 0;
    if (tid < kBuckets && tid >= off) v = base[tid - off];
    __syncthreads();
    if (tid < kBuckets) base[tid] += v;
    __syncthreads();
  }
  const uint32_t total_d = part[0][d] + part[1][d] + part[2][d] + part[3][d];
  uint32_t off = base[d] - total_d;               // exclusive over digits
  for (int i = 0; i < q; ++i) off += part[i][d];
  column_prefix(gsum, g0, g1, d, off);
}

// Stable scatter of one tile of kTile * ITEMS keys by the digit at `shift`: wavefront w holds
// tile positions [64 ITEMS w, 64 ITEMS (w + 1)), item i the 64 of them from 64 (ITEMS w + i).
// out_keys may be null (last pass); positions >= out_limit are padding and are dropped. With
// kFusedScan (few tiles, one key per thread) the block derives its digit offsets from the count
// table (digit totals over all tiles, exclusive-scanned, plus the counts of the earlier tiles)
// and writes each key straight to its place; otherwise `table` holds the in-group prefixes of
// the group scan and `gtable` the group offsets of the top scan, and the tile is first placed
// in digit order in LDS so that consecutive threads write consecutive addresses.
constexpr int kFusedScanMaxTiles = 128;
template <bool kFusedScan, int ITEMS>
__global__ __launch_bounds__(kTile) void radix_scatter_kernel(
    const uint32_t* __restrict__ keys, const uint32_t* __restrict__ vals, int shift, int n_tiles,
    const uint32_t* __restrict__ table, const uint32_t* __restrict__ gtable, int group_tiles,
    uint32_t* __restrict__ out_keys, uint32_t* __restrict__ out_vals, int64_t out_limit) {
  static_assert(!kFusedScan || ITEMS == 1, "the fused offsets path handles one key per thread");
  constexpr int TK = kTile * ITEMS;
  constexpr int kStage = kFusedScan ? 1 : TK;
  __shared__ uint32_t wcount[kWaves][kBuckets];
  __shared__ uint32_t base[kBuckets];
  __shared__ uint32_t part_before[4][kBuckets], part_total[4][kBuckets];
  __shared__ uint32_t lbase[kBuckets];                  // tile-local digit counts, then their scan
  __shared__ uint32_t s_key[kStage], s_val[kStage];     // the tile in digit order
  const int tid = threadIdx.x, tile = blockIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int64_t t0 = (int64_t)tile * TK + wave * (64 * ITEMS) + lane;
  uint32_t key[ITEMS], val[ITEMS], dig[ITEMS], rank[ITEMS];
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    key[i] = keys[t0 + i * 64];
    val[i] = vals[t0 + i * 64];
  }
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
    if (tid < kBuckets)
      base[tid] = gtable[(int64_t)(tile / group_tiles) * kBuckets + tid] + table[(int64_t)tile * kBuckets + tid];
  }
  __syncthreads();

  // rank among this wavefront's keys with the same digit, in position order: items in order,
  // lanes in order within an item (the wavefront's own LDS accesses stay in program order)
  const uint64_t lanes_below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const uint32_t d = (key[i] >> shift) & (kBuckets - 1);
    uint64_t same = ~0ull;
#pragma unroll
    for (int b = 0; b < kRadixBits; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t ones = __ballot(bit);
      same &= bit ? ones : ~ones;
    }
    const uint32_t before = wcount[wave][d];
    dig[i] = d;
    rank[i] = before + (uint32_t)__popcll(same & lanes_below);
    if ((same & lanes_below) == 0ull) wcount[wave][d] = before + (uint32_t)__popcll(same);   // first lane of the digit
  }
  __syncthreads();
  if (tid < kBuckets) {   // offsets of each wavefront inside the tile's digit groups
    uint32_t run = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t c = wcount[w][tid];
      wcount[w][tid] = run;
      run += c;
    }
    lbase[tid] = run;                       // the tile's count of digit tid, scanned below
  }
  __syncthreads();
  if (kFusedScan) {   // few tiles: latency-bound, write straight from the ranks
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      const int64_t pos = (int64_t)base[dig[i]] + wcount[wave][dig[i]] + rank[i];
      if (pos < out_limit) {
        if (out_keys) out_keys[pos] = key[i];
        out_vals[pos] = val[i];
      }
    }
    return;
  }
  for (int off = 1; off < kBuckets; off <<= 1) {   // inclusive scan of the tile's digit counts
    uint32_t v = 0;
    if (tid < kBuckets && tid >= off) v = lbase[tid - off];
    __syncthreads();
    if (tid < kBuckets) lbase[tid] += v;
    __syncthreads();
  }
  // place the tile in digit order in LDS (lbase is now inclusive: digit d starts at
  // lbase[d - 1]), then write it out
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const uint32_t d = dig[i];
    const uint32_t lp = (d == 0 ? 0u : lbase[d - 1]) + wcount[wave][d] + rank[i];
    s_key[lp] = key[i];
    s_val[lp] = val[i];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const int e = i * kTile + tid;
    const uint32_t k2 = s_key[e], v2 = s_val[e];
    const uint32_t d2 = (k2 >> shift) & (kBuckets - 1);
    const int64_t pos = (int64_t)base[d2] + (e - (d2 == 0 ? 0u : lbase[d2 - 1]));
    if (pos < out_limit) {
      if (out_keys) out_keys[pos] = k2;
      out_vals[pos] = v2;
    }
  }
}

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

// Few workflows (up to kFusedScanMaxTiles tiles of kTile keys): one key per thread, offsets
// fused into the scatter. More: tiles of kTile * kBigItems keys and the group/top scans.
struct PrioLayout {
  bool fused;
  int64_t tile_keys, n_tiles, group_tiles, n_groups, padded;
  size_t keys_a, vals_a, keys_b, vals_b, counts, gsum, flag, total;
};

PrioLayout prio_layout(int32_t n_workflows) {
  PrioLayout L{};
  L.fused = ((int64_t)n_workflows + kTile - 1) / kTile <= kFusedScanMaxTiles;
  L.tile_keys = L.fused ? kTile : (int64_t)kTile * kBigItems;
  L.n_tiles = ((int64_t)n_workflows + L.tile_keys - 1) / L.tile_keys;
  L.padded = L.n_tiles * L.tile_keys;
  const size_t kb = align256(sizeof(uint32_t) * (size_t)L.padded);
  const size_t cb = align256(sizeof(uint32_t) * kBuckets * (size_t)L.n_tiles);
  L.group_tiles = kMinGroupTiles;
  while (L.group_tiles < kMaxGroupTiles && L.n_tiles > (int64_t)kTargetGroups * L.group_tiles) L.group_tiles *= 2;
  L.n_groups = (L.n_tiles + L.group_tiles - 1) / L.group_tiles;
  L.keys_a = 0;
  L.vals_a = L.keys_a + kb;
  L.keys_b = L.vals_a + kb;
  L.vals_b = L.keys_b + kb;
  L.counts = L.vals_b + kb;
  L.gsum = L.counts + cb;
  L.flag = L.gsum + (L.fused ? 0 : align256(sizeof(uint32_t) * kBuckets * (size_t)L.n_groups));
  L.total = L.flag + 256;
  return L;
}

}  // namespace

size_t prioritize_workspace_bytes(int32_t n_workflows, int64_t) {
  return n_workflows > 0 ? prio_layout(n_workflows).total : 0;
}

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

// Device address of the static scratch on the current device, resolved on the first call made
// with that device current and kept for later calls.
maestro_status static_prioritize_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return MAESTRO_ERR_LAUNCH;
  if (dev < 0 || dev >= kMaxDevices) return MAESTRO_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MAESTRO_ERR_LAUNCH;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MAESTRO_OK;
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
  uint32_t* gsum = reinterpret_cast<uint32_t*>(ws + L.gsum);
  // Whether any chain of this call is long: the chain kernel stores this call's number in the
  // workspace word when it meets one, and the long-chain kernel returns at once unless it finds
  // it there. A stale or uninitialised word equal to the number only costs that kernel a scan
  // that finds no marks, so the word needs no clearing (and a captured graph, which replays one
  // number, stays correct).
  static std::atomic<uint32_t> call_counter{0};
  const uint32_t epoch = call_counter.fetch_add(1, std::memory_order_relaxed) + 1;
  uint32_t* long_flag = reinterpret_cast<uint32_t*>(ws + L.flag);

  const int nt = (int)L.n_tiles;
  // the chain kernel covers the padded range in blocks of kTile workflows; with small tiles
  // (block = tile) it also counts the first digit
  chain_kernel<<<dim3((unsigned)(L.padded / kTile)), dim3(kTile), 0, stream>>>(
      n_workflows, chain_offset, stage_latency_s, cursor, deadline_us, now_us, remaining_us,
      slack_key, keys[0], vals[0], L.fused ? counts : nullptr, long_flag, epoch);
  // one tile per workgroup while that fits kLongChainBlocks workgroups, more per barrier beyond
  const int64_t chain_tiles = (n_workflows + (int64_t)kTile - 1) / kTile;
  int tiles_per_check = 1;
  while (tiles_per_check < kLongChainTilesPerCheck && chain_tiles > (int64_t)tiles_per_check * kLongChainBlocks)
    tiles_per_check *= 2;
  const int64_t chain_steps = (chain_tiles + tiles_per_check - 1) / tiles_per_check;
  long_chain_kernel<<<dim3((unsigned)(chain_steps < kLongChainBlocks ? chain_steps : kLongChainBlocks)), dim3(kTile),
                      0, stream>>>(
      n_workflows, chain_offset, stage_latency_s, cursor, deadline_us, now_us, remaining_us, slack_key, keys[0],
      vals[0], L.fused ? counts : nullptr, tiles_per_check, long_flag, epoch);
  for (int pass = 0; pass < kPasses; ++pass) {
    const int src = pass & 1, dst = src ^ 1;
    const int shift = pass * kRadixBits;
    const bool last = pass + 1 == kPasses;
    uint32_t* out_k = last ? nullptr : keys[dst];
    uint32_t* out_v = last ? reinterpret_cast<uint32_t*>(order) : vals[dst];
    const int64_t limit = last ? (int64_t)n_workflows : L.padded;
    if (L.fused) {
      if (pass > 0)
        radix_count_kernel<1><<<dim3(nt), dim3(kTile), 0, stream>>>(keys[src], shift, counts);
      radix_scatter_kernel<true, 1><<<dim3(nt), dim3(kTile), 0, stream>>>(
          keys[src], vals[src], shift, nt, counts, nullptr, 0, out_k, out_v, limit);
    } else {
      const int ng = (int)L.n_groups;
      radix_count_kernel<kBigItems><<<dim3(nt), dim3(kTile), 0, stream>>>(keys[src], shift, counts);
      radix_group_scan_kernel<<<dim3(ng), dim3(1024), 0, stream>>>(counts, nt, (int)L.group_tiles, gsum);
      radix_top_scan_kernel<<<dim3(1), dim3(1024), 0, stream>>>(gsum, ng);
      radix_scatter_kernel<false, kBigItems><<<dim3(nt), dim3(kTile), 0, stream>>>(
          keys[src], vals[src], shift, nt, counts, gsum, (int)L.group_tiles, out_k, out_v, limit);
    }
  }
  return launch_status();
}

}  // namespace maestro

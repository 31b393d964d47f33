// Cost prediction for a batch of stages (Sec. III-B; Eq. 3): the feature MLP over length bins,
// softmax, expected length, KV bytes -- one fused kernel, logits and hidden layers never leave
// the chip. The two-phase form reads the same network's outputs as heads instead (a
// calibrated tool-intent probability, Eq. 1, then the role's log(1 + L) regressor fed that
// probability); only the epilogue differs.
//
// Layout of the work. Each wavefront owns one or two groups of 32 stages (rows). Every Linear
// layer is computed transposed, H^T = W * X^T, on 32x32 MFMA tiles: the weights are the A
// operand (32 output neurons x K) and a group's activations the B operand (K x 32 rows). A 32x32 result tile leaves
// lane (h*32 + r) holding, for row r, the 16 neurons (v/4)*8 + 4h + v%4 (v = 0..15). Those 16
// values are exactly what the same lane must feed as the B operand of the next layer over a
// K-slice of 32 inputs, provided the next layer's weight columns are read in the matching
// order (a fixed permutation of K, which leaves the dot products unchanged). So hidden
// activations stay in registers from one layer to the next, and the last hidden layer is
// consumed block by block into the logit accumulators without ever being stored whole.
//
// Weights stream through LDS: each 32-neuron block of a layer (plus, for the last hidden
// layer, the matching 32 columns of the logit layer) is copied once per workgroup and tile
// into a ring of LDS buffers by direct global->LDS loads (no staging registers) while earlier
// blocks are being multiplied, and read by all four wavefronts with 16-byte LDS reads; with two
// row groups every fragment read feeds one MFMA per group. Weight rows are padded by 16 bytes
// in LDS so that the 16 rows a half-wavefront reads at one column fall in distinct banks.
#include <type_traits>

#include "internal.h"

namespace maestro {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWaves = 4;
constexpr int kRowsPerWave = 32;
constexpr int kRowsPerBlock = kWaves * kRowsPerWave;
constexpr int kThreads = kWaves * 64;

constexpr int cmax(int a, int b) { return a > b ? a : b; }


// Output row (neuron or bin) of a 32x32 MFMA result held in accumulator register v by
// lane-half h (lanes 0-31: h = 0, lanes 32-63: h = 1); the column is the lane's row r.
__device__ __forceinline__ int acc_row(int v, int h) { return (v >> 2) * 8 + h * 4 + (v & 3); }

// 16 consecutive floats of a 32-wide slice as seen by accumulator registers of lane-half h:
// out[v] = src[acc_row(v, h)].
__device__ __forceinline__ void load_acc_layout(const float* __restrict__ src, int h, float (&out)[16]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float4 f = *reinterpret_cast<const float4*>(src + q * 8 + h * 4);
    out[q * 4 + 0] = f.x; out[q * 4 + 1] = f.y; out[q * 4 + 2] = f.z; out[q * 4 + 3] = f.w;
  }
}

// alpha(M) of a stage's model, as float64; a model id outside [0, n_models) gives NaN, so that
// stage's KV demand is NaN and no node admits it.
__device__ __forceinline__ double alpha_of(const float* __restrict__ alpha, int32_t model, int32_t n_models) {
  return (uint32_t)model < (uint32_t)n_models ? (double)alpha[model] : (double)NAN;
}

// Softmax over the B = 32*BT logits of each row, expected length, Eq. 3 KV bytes.
// Lanes r and r + 32 hold complementary halves of row r's logits.
template <int BT>
__device__ __forceinline__ void length_epilogue(const f32x16 (&logit)[BT], const float* __restrict__ b_last,
                                                const float* __restrict__ centre, int h, int64_t row, int64_t n,
                                                int32_t prompt, int32_t model, const float* __restrict__ alpha,
                                                int32_t n_models, float* __restrict__ pred_len,
                                                double* __restrict__ kv_bytes) {
  float z[BT][16], c[BT][16];
  float mx = -INFINITY;
#pragma unroll
  for (int bt = 0; bt < BT; ++bt) {
    float bias[16];
    load_acc_layout(b_last + bt * 32, h, bias);
    load_acc_layout(centre + bt * 32, h, c[bt]);
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      z[bt][v] = logit[bt][v] + bias[v];
      mx = fmaxf(mx, z[bt][v]);
    }
  }
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  // e^(z - mx) = 2^((z - mx) log2(e)) with the hardware 2^x; the difference is taken first
  // (exact when z is near mx), so very large logits lose no accuracy to a rounded mx log2(e).
  // The weighted sum of centres accumulates with fused multiply-adds.
  constexpr float kLog2e = 1.4426950408889634f;
  float se = 0.0f, sc = 0.0f;
#pragma unroll
  for (int bt = 0; bt < BT; ++bt) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const float e = __builtin_amdgcn_exp2f(__fmul_rn(__fsub_rn(z[bt][v], mx), kLog2e));
      se += e;
      sc = fmaf(e, c[bt][v], sc);
    }
  }
  se += __shfl_xor(se, 32);
  sc += __shfl_xor(sc, 32);
  if (h == 0 && row < n) {
    const float pred = sc / se;
    pred_len[row] = pred;
    kv_bytes[row] = ((double)prompt + (double)pred) * alpha_of(alpha, model, n_models);
  }
}

// Per-stage inputs and tables of the two-phase predictor (unused by the bins predictor).
struct TwoPhaseArgs {
  const int32_t* role_id;
  const int32_t* tool_avail;
  const int32_t* role_head;
  const float* tool_coef;
  const float* iso_x;
  const float* iso_y;
  int32_t n_roles;
  int32_t n_knots;
  float max_len;
  float* p_tool;
};

// The B = 32*BT outputs of each row read as heads (Sec. III-B): output 0 the tool-intent
// logit, output g the log(1 + L) regressor of the row's head g (role_head of its role, head 1
// when the role has none). p_tool = iso(sigmoid(z_0)) (Eq. 1 calibrated; 0 without tools),
// L = min(expm1(max(z_g + coef_g p_tool, 0)), max_len), then Eq. 3.
__device__ __forceinline__ int head_of_role(int32_t role, const int32_t* __restrict__ head_of, int32_t n_roles,
                                            int n_out) {
  int g = (role >= 0 && role < n_roles) ? head_of[role] : 1;
  return (g < 1 || g >= n_out) ? 1 : g;
}

// Output g of a row, summed over its two lane-halves: lane-half h holds the outputs
// 32 bt + acc_row(v, h), so exactly one half holds output g, as register v = 4 (t / 8) + t % 4
// of tile bt = g / 32 (t = g % 32) when (t / 4) % 2 == h. A five-level selection tree over the
// register index picks it; the other half contributes 0.
template <int BT>
__device__ __forceinline__ float head_output(const f32x16 (&z)[BT], int g, int h) {
  static_assert(BT == 2, "a 32-entry selection tree");
  const int t = g & 31;
  const int idx = (g >> 5) * 16 + (t >> 3) * 4 + (t & 3);
  float val[32];
#pragma unroll
  for (int bt = 0; bt < BT; ++bt)
#pragma unroll
    for (int v = 0; v < 16; ++v) val[16 * bt + v] = z[bt][v];
#pragma unroll
  for (int lvl = 0; lvl < 5; ++lvl) {
    const bool bit = (idx >> lvl) & 1;
#pragma unroll
    for (int j = 0; j < (16 >> lvl); ++j) val[j] = bit ? val[2 * j + 1] : val[2 * j];
  }
  const float mine = (((t >> 2) & 1) == h) ? val[0] : 0.0f;
  return mine + __shfl_xor(mine, 32);
}

// The rest of one row from its tool-intent output z0 and head output zg (biases not yet added).
__device__ __forceinline__ void two_phase_row(float z0, float zg, int g, const float* __restrict__ b_last,
                                              const float* __restrict__ coef, const float* __restrict__ kx,
                                              const float* __restrict__ ky, const TwoPhaseArgs& tp, int64_t row,
                                              int32_t prompt, int32_t model, int32_t tools,
                                              const float* __restrict__ alpha, int32_t n_models,
                                              float* __restrict__ pred_len, double* __restrict__ kv_bytes) {
  float p = 0.0f;
  if (tools != 0) {
    const float s = 1.0f / (1.0f + __expf(-(z0 + b_last[0])));
    const int K = tp.n_knots;
    if (!(s > kx[0])) {
      p = ky[0];
    } else if (s >= kx[K - 1]) {
      p = ky[K - 1];
    } else {   // kx[lo] <= s < kx[hi]: the segment through knots lo and lo + 1
      int lo = 0, hi = K - 1;
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (kx[mid] <= s) lo = mid;
        else hi = mid;
      }
      p = ky[lo] + (s - kx[lo]) * (ky[hi] - ky[lo]) / (kx[hi] - kx[lo]);
    }
  }
  const float y = zg + b_last[g] + coef[g] * p;
  const float L = fminf(expm1f(fmaxf(y, 0.0f)), tp.max_len);
  if (tp.p_tool) tp.p_tool[row] = p;
  pred_len[row] = L;
  kv_bytes[row] = ((double)prompt + (double)L) * alpha_of(alpha, model, n_models);
}

// Per-role regressors (Sec. III-B): a stage whose role has a regressor of its own is predicted by
// that regressor's network; output 0 regresses log(1 + L), fed the first phase's calibrated tool
// probability p: L = min(expm1(max(z_0 + coef p, 0)), max_len), then Eq. 3. Stages reach the
// kernel bucketed by regressor (every tile belongs to one), in tile-row order, with their stage
// index, prompt length, model id and p carried alongside; padding rows have stage -1.
__device__ __forceinline__ void role_row(float z0, float b0, float coef, float p, float max_len, int32_t stage,
                                         int32_t prompt, int32_t model, const float* __restrict__ alpha,
                                         int32_t n_models, float* __restrict__ pred_len,
                                         double* __restrict__ kv_bytes) {
  const float y = z0 + b0 + coef * p;
  const float L = fminf(expm1f(fmaxf(y, 0.0f)), max_len);
  pred_len[stage] = L;
  kv_bytes[stage] = ((double)prompt + (double)L) * alpha_of(alpha, model, n_models);
}

// ---------------------------------------------------------------------------------------------
// bfloat16, three Linear layers: D -> H1 -> H2 -> B   (D = 256)
// ---------------------------------------------------------------------------------------------
//
// Persistent workgroups (one per compute unit) walk tiles of 128 G rows. Everything a tile
// reads from global memory arrives as a fixed sequence of LDS "chunks":
//   feature chunk j (j < 2G)   : G = 1: features of tile rows 64j .. 64j+63; G = 2: K-slice j
//                                (columns 64j .. 64j+63) of all 256 tile rows; with them, in
//                                64-row pieces, the tile's per-stage inputs
//   layer-1 chunk j            : W1 rows 64j .. 64j+63 (two 32-neuron blocks), all D columns
//   layer-2 chunk (b, p)       : W2 rows 32b .. 32b+31, columns 512p .. 512p+511, plus, for
//                                the last p, W3 columns 32b .. 32b+31 of every bin row
// Chunks rotate through kBufs LDS buffers and are fetched kAhead chunks ahead (across tile
// boundaries) by direct global->LDS loads, so every fetch overlaps the multiplication of
// earlier chunks. Each wavefront waits only for the loads of the chunk needed next (counted
// vmcnt), then the workgroup barrier publishes it. No other global load is in flight, so no
// wait ever drains the prefetch. The barrier sits inside the chain of MFMAs
// (mfma_chain_handover) and the prefetch distance is 2, so that the buffer being refilled is two
// chunks old and no wavefront can still be reading it.
//
// LDS layouts (all 16-byte reads are free of bank conflicts per quarter-wavefront):
//   feature chunk: G = 1: 64 rows of 512 bytes, the 16-byte units of row r stored at
//                  unit ^ (r % 16); G = 2: 256 rows of 128 bytes, unit u at u ^ ((r / 2) % 8)
//   layer-1 chunk: row pairs (2i, 2i+1) stored contiguously (1 KB), 16-byte pad per pair; in
//                  odd rows the 16-byte units are stored with index bit 3 flipped
//   layer-2 chunk: 32 rows of 1 KB, 16-byte pad per row; then the W3 slice, B rows x 64 bytes
//                  with the four units of row r rotated by (r / 4) % 4

// Output neuron (within a 32-neuron block) computed by row i of a weight tile. With this order
// the 16 results that lane-half h holds after a 32x32 MFMA (register v -> tile row
// (v/4)*8 + 4h + v%4) are the neurons 16*(v/8) + 8h + v%8: two runs of 8 consecutive
// neurons, which the next layer consumes in natural column order.
__device__ __forceinline__ int tile_row_neuron(int i) {
  const int q = i >> 3;
  return 16 * (q >> 1) + 8 * ((i >> 2) & 1) + 4 * (q & 1) + (i & 3);
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kLookahead = 3;            // fragment reads ahead of their MFMA (one row group)

// A chain of F MFMA steps over one LDS chunk, with the hand-over to the next chunk folded in. fr
// holds the fragments (16-byte A operands) of steps 0 .. LA-1 on entry (read by the chain before,
// or by the caller); step f's fragment is cur(f), read LA steps ahead. At step F - LA every
// fragment of this chunk has been requested: release() lets the next chunk in (its loads waited
// for, the workgroup barrier crossed), and the remaining lookahead reads fetch the next chain's
// first fragments through next(i), left in fr on return (kNext). The barrier then overlaps the
// last MFMAs of this chain, and the next chain starts with its first fragments already in
// flight. mma(f, fragment) issues step f's MFMAs (one per row group the fragment feeds); pre()
// runs before the first step, side(f) right after step f, while the matrix core is busy (weight
// loads, the pieces of the previous block's deferred epilogue); the scheduling barriers keep
// this order.
// Measured against a barrier (and a wait for the wavefront's own LDS reads) between the chains,
// outputs bit for bit the same: 8.45 against 8.57 ms on 4,194,304 stages (256-1024-1024-64, one
// row group; reading 4 or 5 steps ahead instead of 3 changed nothing), 0.443 against 0.454 ms
// on 719,712 stages (256-512-512-64, two row groups).
template <int F, bool kNext, int LA = kLookahead, typename Cur, typename Next, typename Mma, typename Pre,
          typename Side, typename Release>
__device__ __forceinline__ void mfma_chain_handover(bf16x8 (&fr)[LA], Cur&& cur, Next&& next, Mma&& mma, Pre&& pre,
                                                    Side&& side, Release&& release) {
  static_assert(F > LA, "the hand-over lies inside the chain");
  bf16x8 ring[F + LA];
#pragma unroll
  for (int f = 0; f < LA; ++f) ring[f] = fr[f];
  __builtin_amdgcn_sched_barrier(0);
  pre();
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int f = 0; f < F; ++f) {
    if (f == F - LA) {
      release();
      __builtin_amdgcn_sched_barrier(0);
    }
    const int ff = f + LA;
    if (ff < F) ring[ff] = cur(ff);
    else if (kNext) ring[ff] = next(ff - F);
    mma(f, ring[f]);
    side(f);
    __builtin_amdgcn_sched_barrier(0);
  }
  if constexpr (kNext) {
#pragma unroll
    for (int f = 0; f < LA; ++f) fr[f] = ring[F + f];
  }
}

// Accumulator of a 32-neuron block initialised with the biases of the neurons lane-half h holds
// (registers 0-7: neurons 8h .. 8h+7, registers 8-15: neurons 16+8h .. 16+8h+7).
__device__ __forceinline__ f32x16 bias_acc(const float* __restrict__ b32, int h) {
  const float4 q0 = *reinterpret_cast<const float4*>(b32 + 8 * h);
  const float4 q1 = *reinterpret_cast<const float4*>(b32 + 8 * h + 4);
  const float4 q2 = *reinterpret_cast<const float4*>(b32 + 16 + 8 * h);
  const float4 q3 = *reinterpret_cast<const float4*>(b32 + 16 + 8 * h + 4);
  return f32x16{q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w,
                q2.x, q2.y, q2.z, q2.w, q3.x, q3.y, q3.z, q3.w};
}

typedef short s16x2 __attribute__((ext_vector_type(2)));

// acc[8*half + j] (biases included), j = 0..7, rounded to bfloat16 (nearest even) and packed as
// the 8 K-slots of a B operand, then rectified on the packed values: a bfloat16 is below zero
// exactly when its bit pattern is a negative int16, so a packed int16 max with 0 is the ReLU
// (rounding to nearest and ReLU commute; -0 becomes +0).
__device__ __forceinline__ bf16x8 relu_bf16(const f32x16& acc, int half) {
  uint32_t w[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const f32x2 f = {acc[8 * half + 2 * p], acc[8 * half + 2 * p + 1]};
    const s16x2 v = __builtin_bit_cast(s16x2, __builtin_convertvector(f, bf16x2));
    w[p] = __builtin_bit_cast(uint32_t, __builtin_elementwise_max(v, s16x2{0, 0}));
  }
  return __builtin_bit_cast(bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
}

constexpr int kBufs = 4;                 // LDS chunk buffers
constexpr int kDmaPerChunk = 8;          // direct loads per wavefront per chunk (at least)

// Direct global->LDS loads through a raw buffer resource: lane l's 16 (or 4) bytes at byte offset
// voff + soff of the buffer land at LDS byte address lds_base + lds_off + 16 l (or 4 l); lanes
// whose voff is at or past the buffer's size read zeros and touch no memory. Issued as inline
// assembly so that the compiler's automatic wait insertion, which would conservatively drain
// every such load before any LDS read, does not see them; the kernel waits for them itself
// (wait_chunk). rsrc, soff and lds_base are wavefront-uniform; lds_off is a compile-time constant.
// An LDS-DMA load reads M0 and needs one wait state after the scalar write of M0 (a hazard the
// compiler resolves only for instructions it generates itself), hence the s_nop.
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) unsigned char lds_uchar;

// Raw (unstrided) buffer resource over `bytes` bytes at `base` (gfx9 descriptor: 48-bit base,
// stride 0, byte-granular range check, 32-bit data format).
__device__ __forceinline__ i32x4 buffer_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int32_t)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int32_t)((a >> 32) & 0xFFFF));
  r[2] = __builtin_amdgcn_readfirstlane((int32_t)bytes);
  r[3] = 0x00020000;
  return r;
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const lds_uchar*)(p);
}
// kStream marks the load non-temporal (nt): data read once (features, per-stage inputs) is
// then a candidate for early eviction and does not push the weights, which every tile re-reads,
// out of the L2 cache.
template <bool kStream = false>
__device__ __forceinline__ void dma16(const i32x4& rsrc, uint32_t voff, uint32_t soff, uint32_t lds_base,
                                      int lds_off) {
  if constexpr (kStream)
    asm volatile("s_add_u32 m0, %0, %1\n\ts_nop 0\n\tbuffer_load_dwordx4 %2, %3, %4 offen nt lds"
                 ::"s"(lds_base), "i"(lds_off), "v"(voff), "s"(rsrc), "s"(soff) : "m0", "scc");
  else
    asm volatile("s_add_u32 m0, %0, %1\n\ts_nop 0\n\tbuffer_load_dwordx4 %2, %3, %4 offen lds"
                 ::"s"(lds_base), "i"(lds_off), "v"(voff), "s"(rsrc), "s"(soff) : "m0", "scc");
}
__device__ __forceinline__ void dma4(const i32x4& rsrc, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen nt lds"
               ::"s"(lds_base), "v"(voff), "s"(rsrc) : "m0");
}

// Two consecutive int32 at a wavefront-uniform, 8-byte aligned address, through the scalar data
// cache and waited for here: a scalar load is counted apart from the vector-memory operations, so
// fetching it never waits for the LDS-DMA prefetches in flight (a vector load's wait would).
__device__ __forceinline__ void scalar_load2(const int32_t* p, int32_t& a, int32_t& b) {
  uint64_t v;
  asm volatile("s_load_dwordx2 %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=s"(v) : "s"(p) : "memory");
  a = (int32_t)(uint32_t)v;
  b = (int32_t)(uint32_t)(v >> 32);
}
// Eight consecutive int32 at a wavefront-uniform, 32-byte aligned address the same way; returns
// entry r (r in 0..7, per lane).
typedef int32_t i32x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ int32_t scalar_load8_pick(const int32_t* p, int r) {
  i32x8 v;
  asm volatile("s_load_dwordx8 %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=s"(v) : "s"(p) : "memory");
  int32_t x = v[0];
#pragma unroll
  for (int k = 1; k < 8; ++k) x = r == k ? v[k] : x;
  return x;
}

// Wait until at most N vector-memory operations of this wavefront are outstanding and all of
// its LDS operations are done (gfx9 s_waitcnt encoding), then the workgroup barrier. The
// empty asm statements keep the compiler from moving LDS accesses across.
template <int N>
__device__ __forceinline__ void wait_chunk() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (0 << 8));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Wait until at most N vector-memory operations of this wavefront are outstanding (its own loads
// of the chunk needed next have landed), then the workgroup barrier -- without waiting for this
// wavefront's LDS reads, so that fragment reads issued ahead stay in flight across it.
template <int N>
__device__ __forceinline__ void release_chunk() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

constexpr int kMaxModels = 64;           // per-model KV bytes staged in LDS

// Fragment lookahead with two row groups (K-steps; each fragment read from LDS feeds one MFMA
// per group into independent accumulators, so the LDS fragment reads, their waits and the weight
// traffic per MFMA are half those of one group).
constexpr int kLookaheadGroups = 2;

template <int G>
struct AccGroups {
  f32x16 v[G];
};

// G = number of 32-row groups per wavefront. A tile is kWaves * 32 * G rows; the weights stream
// through LDS once per tile, so G = 2 halves the weight traffic and the LDS fragment reads per
// row. G = 2 needs both groups' layer-1 activations in the 256 accumulation registers, which
// holds for H1 = 512.
//
// kRoles: the per-role regressors as one grouped GEMM. Tile t belongs to regressor
// tile_group[t] (bucketed by the role_*_kernel launches); its weights are regressor g's layers, stacked
// after those of regressors 0 .. g-1, and its rows are the stages perm[kTileRows t ...] (feature
// rows gathered through the permutation; padding rows, stage -1, read as zeros). The tile count is
// read from device memory (n_tiles_dev). The biases are restaged whenever a workgroup's tile
// moves to another regressor (tiles of one regressor are contiguous, so rarely).
template <int D, int H1, int H2, int B, int G, bool kTwoPhase, bool kRoles = false>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void mlp3_bf16_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w1, const uint16_t* __restrict__ w2,
    const uint16_t* __restrict__ w3, const float* __restrict__ b1, const float* __restrict__ b2,
    const float* __restrict__ b3, const float* __restrict__ centre, int64_t n, int64_t n_tiles_arg,
    const int32_t* __restrict__ prompt_len, const int32_t* __restrict__ model_id,
    const float* __restrict__ alpha, int32_t n_models, float* __restrict__ pred_len,
    double* __restrict__ kv_bytes, const TwoPhaseArgs tp, const int32_t* __restrict__ tile_group,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ p_bits, const int32_t* __restrict__ n_tiles_dev,
    const float* __restrict__ role_coef, float role_max_len) {
  static_assert(D == 256, "feature and layer-1 chunk layouts assume 512-byte rows");
  static_assert(!kRoles || !kTwoPhase, "role regressors: output 0 only");
  static_assert(H1 % 512 == 0 && H2 % 32 == 0 && B % 64 == 0, "tile shape");
  static_assert(G == 1 || (G == 2 && H1 == 512), "two row groups need H1 = 512 (256 accumulation registers)");
  constexpr int kTileRows = kWaves * kRowsPerWave * G;
  constexpr int KS1 = D / 16;             // K-steps of layer 1 (32x32x16 MFMA)
  constexpr int NX = 2 * G;               // feature chunks per tile (64 rows each)
  constexpr int NC1 = H1 / 64;            // layer-1 chunks (two neuron blocks each)
  constexpr int KP = H1 / 512;            // column parts of a layer-2 block
  constexpr int NB2 = H2 / 32;            // layer-2 neuron blocks
  constexpr int NC = NX + NC1 + NB2 * KP; // chunks per tile
  constexpr int BT = B / 32;              // bin tiles
  constexpr int PAIR = 1024 + 16;         // layer-1 chunk: bytes per row pair
  constexpr int ROW2 = 1024 + 16;         // layer-2 chunk: bytes per row
  constexpr int W3OFF = 32 * ROW2;
  constexpr int CHUNK = cmax(cmax(64 * 512, 32 * PAIR), W3OFF + B * 64);
  // Prefetch distance in chunks. Each chunk is handed over inside the chain of MFMAs (the
  // barrier before the last MFMAs, no wait for the wavefront's own LDS reads), so the buffer a
  // new prefetch fills must be two chunks old: distance 2 of the 4 buffers.
  constexpr int kAhead = 2;
  static_assert(kAhead + 2 <= kBufs, "the chunk a prefetch overwrites is two chunks old");
  static_assert(NC >= kAhead, "prologue fetches whole chunks of the first tile");
  static_assert(NX + NC1 + kAhead <= NC, "feature and layer-1 prefetches stay within the tile");
  static_assert(2 * KS1 == 32, "a layer-1 chunk is 32 MFMA steps");
  static_assert(NB2 * KP >= kAhead, "the peeled layer-2 blocks cover every wrapping prefetch");

  __shared__ __attribute__((aligned(16))) unsigned char lds[kBufs * CHUNK];
  __shared__ __attribute__((aligned(16))) float s_b1[H1];
  __shared__ __attribute__((aligned(16))) float s_b2[H2];
  __shared__ __attribute__((aligned(16))) float s_b3[B];
  __shared__ __attribute__((aligned(16))) float s_c[B];   // bin centres, or the two-phase tool coefficients
  __shared__ __attribute__((aligned(16))) float s_alpha[kMaxModels];
  // [tile parity][prompt, model (, role, tool availability)][row]
  constexpr int kMeta = (kTwoPhase || kRoles) ? 4 : 2;
  __shared__ __attribute__((aligned(16))) int32_t s_meta[2][kMeta][kTileRows];
  constexpr int kTab = kTwoPhase ? 64 : 1;   // two-phase tables: role heads, calibration knots
  __shared__ int32_t s_head[kTab];
  __shared__ float s_kx[kTab], s_ky[kTab];

  const int tid = threadIdx.x;
  // wave index as a scalar: keeps every DMA source row address and LDS destination in SGPRs
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, h = lane >> 5, r32 = lane & 31;
  const int64_t first_tile = blockIdx.x, stride = gridDim.x;

  // ---- chunk fetchers, each issuing at least kDmaPerChunk direct loads per wavefront
  // tiles to walk: from the launch, or (role regressors) from the bucketing pass
  const int64_t n_tiles = kRoles ? (int64_t)n_tiles_dev[0] : n_tiles_arg;
  // the regressor of tile t (0 past the last tile) and its weights' buffer resources
  auto group_of = [&](int64_t t) -> int { return (kRoles && t < n_tiles) ? tile_group[t] : 0; };
  auto rsrc_w1 = [&](int grp) { return buffer_rsrc(w1 + (size_t)grp * (H1 * D), (uint32_t)(H1 * D * 2)); };
  auto rsrc_w2 = [&](int grp) { return buffer_rsrc(w2 + (size_t)grp * (H2 * H1), (uint32_t)(H2 * H1 * 2)); };
  auto rsrc_w3 = [&](int grp) { return buffer_rsrc(w3 + (size_t)grp * (B * H2), (uint32_t)(B * H2 * 2)); };
  int grp_cur = group_of(first_tile);
  i32x4 rs_w1 = rsrc_w1(grp_cur), rs_w2 = rsrc_w2(grp_cur), rs_w3 = rsrc_w3(grp_cur);
  i32x4 rs_w1_next = rs_w1;               // W1 of the next tile, whose first chunks this tile prefetches
  int64_t cur_tile = first_tile;
  const uint32_t voff1 = (uint32_t)(((lane >> 5) * D + (((lane & 31) ^ ((lane >> 5) << 3)) * 8)) * 2);
  const uint32_t voff2 = (uint32_t)(lane * 16);
  const uint32_t voff3 = (uint32_t)(((lane >> 2) * H2 + (((lane & 3) ^ ((lane >> 4) & 3)) * 8)) * 2);
  // feature load q of a chunk: tile row rho = 64j + 2i + (lane / 32), i = wave + 4q, 16-byte unit
  // (lane % 32) ^ (rho % 16); rho % 16 depends on q only through q % 2
  uint32_t voffx[2];
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const int rho = 2 * wave + h + 8 * p;
    voffx[p] = (uint32_t)((2 * wave + h) * D * 2 + (((lane & 31) ^ (rho & 15)) << 4));
  }
  // G = 2: feature chunk j is K-slice j instead (columns 64j .. 64j+63 of all 256 tile rows, 128
  // bytes per row, the 16-byte unit u of row r stored at u ^ ((r / 2) % 8)), so that every
  // wavefront reads its B operands from every feature chunk. A load brings 8 rows; lane l fills
  // row l / 8, position l % 8, and since (r / 2) % 8 = 4 (i % 2) + l / 16 for row r = 8i + l / 8
  // with i = wave + 4q, one offset per lane serves every load of the wavefront.
  const uint32_t voffk =
      (uint32_t)((lane >> 3) * D * 2 + (((lane & 7) ^ (4 * (wave & 1) + (lane >> 4))) << 4));
  // The per-stage inputs (prompt lengths, model ids, and for the two-phase predictor role ids
  // and tool availability) travel in 64-row pieces with the feature chunks: piece p = 4j + wave
  // rides on feature chunk j and holds rows 64 (p % R) .. 64 (p % R) + 63 of input p / R
  // (R = kTileRows / 64 pieces per input).
  constexpr int kPiecesPerInput = kTileRows / 64;
  static_assert(kMeta * kPiecesPerInput <= kWaves * NX, "every per-stage piece rides on a feature chunk");
  // feature chunk j of tile t, whose per-stage inputs go to s_meta[par] (rows of a partial tile
  // past the last stage, and every row of a tile past the last, read as zeros and are never
  // stored)
  auto fetch_x = [&](int64_t t, int par, int j, const unsigned char* dst) {
    const bool live = t < n_tiles;
    const int64_t row0 = live ? t * kTileRows : 0;
    const uint32_t rows = live ? (kRoles ? (uint32_t)kTileRows : (uint32_t)min<int64_t>(kTileRows, n - row0)) : 0u;
    const uint32_t base = lds_addr(dst) + wave * 1024;
    if constexpr (kRoles) {
      // rows gathered through the permutation: load q brings tile rows rho0 = 64j + 2 wave + 8q
      // (lanes 0-31) and rho0 + 1 (lanes 32-63); a padding row (stage -1) gets an offset past the
      // buffer and reads zeros. The feature array spans at most 2^31 bytes.
      const i32x4 rs = buffer_rsrc(x, (uint32_t)(n * (D * 2)));
      if constexpr (G == 1) {
#pragma unroll
        for (int q = 0; q < kDmaPerChunk; ++q) {
          const int rho0 = 64 * j + 2 * wave + 8 * q;
          int32_t s0 = -1, s1 = -1;
          if (live) scalar_load2(perm + row0 + rho0, s0, s1);
          const int32_t st = h ? s1 : s0;
          const uint32_t unit = (uint32_t)(((lane & 31) ^ ((rho0 + h) & 15)) << 4);
          const uint32_t voff = st >= 0 ? (uint32_t)st * (uint32_t)(D * 2) + unit : 0x80000000u;
          dma16<true>(rs, voff, 0u, base, q * kWaves * 1024);
        }
      } else {
        // K-slice j of tile rows 8i .. 8i+7 (i = wave + 4q) as in the contiguous layout, each
        // lane's row (8i + lane / 8) gathered: one scalar load brings the load's eight stages
        const uint32_t unit = (uint32_t)((((lane & 7) ^ (4 * (wave & 1) + (lane >> 4))) << 4) + 128 * j);
#pragma unroll
        for (int q = 0; q < kDmaPerChunk; ++q) {
          int32_t st = -1;
          if (live) st = scalar_load8_pick(perm + row0 + 8 * (wave + 4 * q), lane >> 3);
          const uint32_t voff = st >= 0 ? (uint32_t)st * (uint32_t)(D * 2) + unit : 0x80000000u;
          dma16<true>(rs, voff, 0u, base, q * kWaves * 1024);
        }
      }
    } else {
      const i32x4 rs = buffer_rsrc(x + row0 * D, rows * (D * 2));
#pragma unroll
      for (int q = 0; q < kDmaPerChunk; ++q) {
        if constexpr (G == 1)
          dma16<true>(rs, voffx[q & 1] + (uint32_t)((64 * j + 8 * q) * D * 2), 0u, base, q * kWaves * 1024);
        else   // rows 8i .. 8i+7, i = wave + 4q, of K-slice j
          dma16<true>(rs, voffk, (uint32_t)(8 * (wave + 4 * q) * D * 2 + 128 * j), base, q * kWaves * 1024);
      }
    }
    const int piece = 4 * j + wave;
    if (piece < kMeta * kPiecesPerInput) {
      const int a = piece / kPiecesPerInput, rb = piece % kPiecesPerInput;
      const int32_t* src = kRoles ? (a == 0 ? prompt_len : a == 1 ? model_id : a == 2 ? p_bits : perm)
                                  : (a == 0 ? prompt_len : a == 1 ? model_id : a == 2 ? tp.role_id : tp.tool_avail);
      dma4(buffer_rsrc(src + row0, rows * 4), (uint32_t)((64 * rb + lane) * 4),
           lds_addr(&s_meta[par][a][64 * rb]));
    }
  };
  // load q of layer-1 chunk j: rows 64j + 2i (lanes 0-31) and 64j + 2i + 1 (lanes 32-63, units
  // with bit 3 flipped), i = wave + 4q; q = kDmaPerChunk issues nothing
  auto load_l1 = [&](int j, int q, const unsigned char* dst, const i32x4& r1) {
    if (q < kDmaPerChunk)
      dma16(r1, voff1, (uint32_t)((64 * j + 2 * wave + 8 * q) * D * 2), lds_addr(dst) + wave * PAIR,
            q * kWaves * PAIR);
  };
  // load q of layer-2 chunk (b, part): W2 rows 32b + r, r = wave + 4q; load kDmaPerChunk of the
  // last part brings W3 rows 16i .. 16i+15 (i = wave), columns 32b .. 32b+31: lane -> row
  // 16i + lane/4, unit (lane % 4) rotated by (row / 4) % 4
  auto load_l2 = [&](int b, int part, int q, const unsigned char* dst) {
    if (q < kDmaPerChunk) {
      dma16(rs_w2, voff2, (uint32_t)((32 * b + wave + 4 * q) * H1 * 2 + part * 1024), lds_addr(dst) + wave * ROW2,
            q * kWaves * ROW2);
    } else if (part == KP - 1) {
      static_assert(B / 16 == kWaves, "one W3 slice load per wavefront");
      dma16(rs_w3, voff3, (uint32_t)(16 * wave * H2 * 2 + 64 * b), lds_addr(dst) + W3OFF + wave * 1024, 0);
    }
  };
  // chunk c of tile t, all loads at once; c is a compile-time constant at every call site
  auto fetch = [&](int64_t t, int par, int c, const unsigned char* dst) {
    if (c < NX) {
      fetch_x(t, par, c, dst);
    } else {
#pragma unroll
      for (int q = 0; q <= kDmaPerChunk; ++q) {
        if (c < NX + NC1) load_l1(c - NX, q, dst, (!kRoles || t == cur_tile) ? rs_w1 : rs_w1_next);
        else load_l2((c - NX - NC1) / KP, (c - NX - NC1) % KP, q, dst);
      }
    }
  };
  // The same loads spread over the 32 MFMA steps of the chunk being multiplied meanwhile: load q
  // goes out after step 3q, so no wavefront stalls behind a burst of memory instructions. A
  // feature chunk (no multiplications of its own to hide behind) goes out whole at step 0.
  constexpr int kSpread = 3;
  static_assert(kSpread * kDmaPerChunk < 32, "every load of a chunk issues within its 32 steps");
  auto spread = [&](int64_t t, int par, int c, const unsigned char* dst, int step) {
    if (c < NX) {
      if (step == 0) fetch_x(t, par, c, dst);
    } else if (step % kSpread == 0 && step / kSpread <= kDmaPerChunk) {
      if (c < NX + NC1) load_l1(c - NX, step / kSpread, dst, (!kRoles || t == cur_tile) ? rs_w1 : rs_w1_next);
      else load_l2((c - NX - NC1) / KP, (c - NX - NC1) % KP, step / kSpread, dst);
    }
  };

  // per-lane LDS offsets of the A operands
  const int prow = tile_row_neuron(r32);
  int l1a[2], l1b[2];                     // layer-1 chunk, neuron block lb (rows 32lb + prow)
#pragma unroll
  for (int lb = 0; lb < 2; ++lb) {
    const int rho = 32 * lb + prow, odd = rho & 1;
    const int base = (rho >> 1) * PAIR + odd * 512 + h * 16;
    l1a[lb] = base + odd * 128;           // K-steps with bit 2 clear: unit bit 3 set for odd rows
    l1b[lb] = base - odd * 128;           // K-steps with bit 2 set: unit bit 3 cleared
  }
  const int l2 = prow * ROW2 + h * 16;
  const int sw3 = (r32 >> 2) & 3;

  auto stage_biases = [&](int grp) {   // the biases of regressor grp (of the network when !kRoles)
    for (int i = tid; i < H1; i += kThreads) s_b1[i] = b1[(size_t)grp * H1 + i];
    for (int i = tid; i < H2; i += kThreads) s_b2[i] = b2[(size_t)grp * H2 + i];
    for (int i = tid; i < B; i += kThreads) s_b3[i] = b3[(size_t)grp * B + i];
  };
  stage_biases(grp_cur);
  if constexpr (!kRoles)
    for (int i = tid; i < B; i += kThreads) s_c[i] = kTwoPhase ? tp.tool_coef[i] : centre[i];
  float coef_cur = kRoles ? role_coef[grp_cur] : 0.0f;
  if (kTwoPhase) {
    for (int i = tid; i < kTab; i += kThreads) {
      s_head[i] = i < tp.n_roles ? tp.role_head[i] : 1;
      s_kx[i] = i < tp.n_knots ? tp.iso_x[i] : 0.0f;
      s_ky[i] = i < tp.n_knots ? tp.iso_y[i] : 0.0f;
    }
  }
  for (int i = tid; i < kMaxModels; i += kThreads) s_alpha[i] = i < n_models ? alpha[i] : 0.0f;
  __syncthreads();

  // chunk g of this workgroup's stream lives in buffer g % kBufs
  unsigned g = 0;
#pragma unroll
  for (int c = 0; c < kAhead; ++c) fetch(first_tile, 0, c, lds + c * CHUNK);
  wait_chunk<kDmaPerChunk * (kAhead - 1)>();

  auto ahead = [&]() { return lds + ((g + kAhead) % kBufs) * CHUNK; };
  auto advance = [&]() {
    wait_chunk<kDmaPerChunk * (kAhead - 1)>();
    ++g;
  };
  // the hand-over inside a chain (one row group)
  auto release = [&]() {
    release_chunk<kDmaPerChunk * (kAhead - 1)>();
    ++g;
  };

  int parity = 0;                         // tiles of this workgroup alternate s_meta halves
  for (int64_t tile = first_tile; tile < n_tiles; tile += stride, parity ^= 1) {
    if constexpr (kRoles) {
      // this tile's regressor: its W2 and W3 for this tile's layer-2 chunks, its W1 (already
      // prefetched for the first layer-1 chunk) for the rest, and the next tile's W1 for the
      // layer-1 chunk that this tile prefetches; biases restaged when the regressor changes
      const int gc = group_of(tile), gn = group_of(tile + stride);
      rs_w1 = rsrc_w1(gc);
      rs_w2 = rsrc_w2(gc);
      rs_w3 = rsrc_w3(gc);
      rs_w1_next = rsrc_w1(gn);
      cur_tile = tile;
      if (gc != grp_cur) {
        __syncthreads();   // every wavefront is done with the previous regressor's biases
        stage_biases(gc);
        __syncthreads();
        grp_cur = gc;
        coef_cur = role_coef[gc];
      }
    }
    // ---- features of this tile: B operands of layer 1, natural K order; group gr of this
    // wavefront is tile rows 32 (G wave + gr) .. + 31
    bf16x8 xf[G][KS1];
#pragma unroll
    for (int c = 0; c < NX; ++c) {
      const unsigned char* buf = lds + (g % kBufs) * CHUNK;
      fetch(tile, parity, c + kAhead, ahead());
      if constexpr (G == 1) {
        if ((wave >> 1) == c) {
          const int xrow = 32 * (wave & 1) + r32;   // this lane's row within the chunk
#pragma unroll
          for (int ks = 0; ks < KS1; ++ks)
            xf[0][ks] = *reinterpret_cast<const bf16x8*>(buf + xrow * 512 + (((2 * ks + h) ^ (xrow & 15)) << 4));
        }
      } else {
        // K-steps 4c .. 4c+3 of both groups from K-slice c
#pragma unroll
        for (int gr = 0; gr < G; ++gr) {
          const int xrow = (G * wave + gr) * kRowsPerWave + r32;   // this lane's tile row
#pragma unroll
          for (int kk = 0; kk < 4; ++kk)
            xf[gr][4 * c + kk] = *reinterpret_cast<const bf16x8*>(
                buf + xrow * 128 + (((2 * kk + h) ^ ((xrow >> 1) & 7)) << 4));
        }
      }
      advance();
    }

    f32x16 logit[G][BT];                  // zeroed once layer 1 is done
    auto zero_logits = [&]() {
#pragma unroll
      for (int gr = 0; gr < G; ++gr)
#pragma unroll
        for (int bt = 0; bt < BT; ++bt) logit[gr][bt] = f32x16{};
    };
    bf16x8 w3f[BT][2];                    // W3 fragments of the previous layer-2 block
    auto read_w3 = [&](const unsigned char* buf) {
#pragma unroll
      for (int bt = 0; bt < BT; ++bt)
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
          w3f[bt][tt] = *reinterpret_cast<const bf16x8*>(
              buf + W3OFF + (bt * 32 + r32) * 64 + ((((2 * tt) | h) ^ sw3) << 4));
    };
    // layer-2 chunk j = b * KP + part is prefetched while chunk j - kAhead is multiplied; the
    // last kPeel blocks, whose prefetches reach into the next tile, are peeled off the loop
    constexpr int kPeel = (kAhead + KP - 1) / KP;
    constexpr int kSteady = NB2 - kPeel - 1;
    static_assert(kSteady >= 2, "at least one pair of blocks in the steady-state loop");
    auto in_tile = [&](int j, const unsigned char* dst, int k) { spread(tile, parity, NX + NC1 + j, dst, k); };
    auto wrapping = [&](int j, const unsigned char* dst, int k) {
      if (j < NB2 * KP) spread(tile, parity, NX + NC1 + j, dst, k);
      else spread(tile + stride, parity ^ 1, j - NB2 * KP, dst, k);
    };

    if constexpr (G == 1) {
      // ---- layer 1: H1 = relu(W1 x + b1), kept as the B operand of layer 2 ---------------
      // Each block's ReLU is deferred into the next block's chain (the last one into the first
      // layer-2 block). The activations live in the accumulation registers, which MFMA reads as
      // its B operand directly, leaving the architectural registers to everything else.
      bf16x8 h1[H1 / 16];
      f32x16 prev0, prev1;                  // finished accumulators of the previous chunk
      auto l1_relu = [&](int nb, const f32x16& acc) {
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          h1[2 * nb + half] = relu_bf16(acc, half);
          asm volatile("" : "+a"(h1[2 * nb + half]));
        }
      };
      // Fragment f of a layer-1 chain (block f % 2, K-step f / 2) and K-step k of a layer-2 chunk.
      auto l1_frag = [&](const unsigned char* buf, int f) {
        const int k = f >> 1, lb = f & 1;
        return *reinterpret_cast<const bf16x8*>(buf + ((k & 4) ? l1b[lb] : l1a[lb]) + k * 32);
      };
      auto l2_frag = [&](const unsigned char* buf, int k) {
        return *reinterpret_cast<const bf16x8*>(buf + l2 + k * 32);
      };
      // The chains hand the chunks over to each other (mfma_chain_handover); the first layer-1
      // chain follows the feature chunks, which have none, so its first fragments are read here.
      // Like the first fragments, the biases that start the next chain's accumulators are read
      // during the chain before it (step kBiasStep), and the deferred ReLU of the previous
      // chunk's blocks runs one half-block per MFMA step (steps 1 .. 4), in the shadow of the
      // matrix core, so that no chain waits on LDS or vector-ALU work before its first MFMA.
      constexpr int kBiasStep = 8;
      bf16x8 fr[kLookahead];
      f32x16 nb0, nb1;                      // biases of the next chain's blocks
#pragma unroll
      for (int f = 0; f < kLookahead; ++f) fr[f] = l1_frag(lds + (g % kBufs) * CHUNK, f);
      nb0 = bias_acc(s_b1, h);
      nb1 = bias_acc(s_b1 + 32, h);
      auto l1_relu_half = [&](int nb, const f32x16& acc, int half) {
        h1[2 * nb + half] = relu_bf16(acc, half);
        asm volatile("" : "+a"(h1[2 * nb + half]));
      };
#pragma unroll
      for (int c = 0; c < NC1; ++c) {
        const unsigned char* buf = lds + (g % kBufs) * CHUNK;
        const unsigned char* nbuf = lds + ((g + 1) % kBufs) * CHUNK;
        const unsigned char* dst = ahead();
        f32x16 acc0 = nb0;
        f32x16 acc1 = nb1;
        mfma_chain_handover<2 * KS1, true>(
            fr, [&](int f) { return l1_frag(buf, f); },
            [&](int i) { return c + 1 < NC1 ? l1_frag(nbuf, i) : l2_frag(nbuf, i); },
            [&](int f, const bf16x8& a) {
              if (f & 1) acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, xf[0][f >> 1], acc1, 0, 0, 0);
              else acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, xf[0][f >> 1], acc0, 0, 0, 0);
            },
            [&]() {},
            [&](int f) {
              spread(tile, parity, NX + c + kAhead, dst, f);
              if (c > 0 && f >= 1 && f <= 4) l1_relu_half(2 * c - 2 + ((f - 1) >> 1), (f - 1) >> 1 ? prev1 : prev0, (f - 1) & 1);
              if (f == kBiasStep) {
                if (c + 1 < NC1) {
                  nb0 = bias_acc(s_b1 + (2 * c + 2) * 32, h);
                  nb1 = bias_acc(s_b1 + (2 * c + 3) * 32, h);
                } else {
                  nb0 = bias_acc(s_b2, h);   // the first layer-2 block's
                }
              }
            },
            release);
        prev0 = acc0;
        prev1 = acc1;
        __builtin_amdgcn_sched_barrier(0);
      }

      // ---- layer 2 block by block, each block folded straight into the logits ----------------
      // The epilogue of each block -- ReLU and the 2 BT MFMAs that fold its 32 neurons into the
      // logits -- is deferred into the start of the next block's chain; the block's W3 fragments
      // are read into registers after its chain, two chunks before its buffer is refilled.
      zero_logits();
      // the deferred epilogue of the previous block, in pieces over the first steps of the next
      // block's first chain (step k; k < 0: all at once, after the tile's last block)
      bf16x8 h2[2];
      auto l2_epilogue = [&](const f32x16& prev, int k) {
        if (k < 0 || k == 1) {
#pragma unroll
          for (int half = 0; half < 2; ++half) h2[half] = relu_bf16(prev, half);
        }
#pragma unroll
        for (int bt = 0; bt < BT; ++bt)
          if (k < 0 || k == 2 + bt) {
#pragma unroll
            for (int tt = 0; tt < 2; ++tt)
              logit[0][bt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w3f[bt][tt], h2[tt], logit[0][bt], 0, 0, 0);
          }
      };
      // block b; pre(prev) is the deferred epilogue of the block before it; kLast: the tile's
      // last block, whose last chain hands over to the next tile's feature chunk (no fragments)
      auto l2_block = [&](int b, const f32x16& prev, auto&& pre, auto&& load_ahead, auto last) {
        f32x16 acc = nb0;
#pragma unroll
        for (int part = 0; part < KP; ++part) {
          const unsigned char* buf = lds + (g % kBufs) * CHUNK;
          const unsigned char* nbuf = lds + ((g + 1) % kBufs) * CHUNK;
          const unsigned char* dst = ahead();
          auto chain = [&](auto next_exists) {
            mfma_chain_handover<32, decltype(next_exists)::value>(
                fr, [&](int k) { return l2_frag(buf, k); }, [&](int i) { return l2_frag(nbuf, i); },
                [&](int k, const bf16x8& a) {
                  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, h1[part * 32 + k], acc, 0, 0, 0);
                },
                [&]() {},
                [&](int k) {
                  load_ahead(b * KP + part + kAhead, dst, k);
                  if (part == 0) pre(prev, k);
                  if (part == KP - 1 && k == kBiasStep && !decltype(last)::value) nb0 = bias_acc(s_b2 + (b + 1) * 32, h);
                },
                release);
          };
          if (decltype(last)::value && part == KP - 1) chain(std::false_type{});
          else chain(std::true_type{});
          if (part == KP - 1) read_w3(buf);
          __builtin_amdgcn_sched_barrier(0);
        }
        return acc;
      };
      // Block 0 finishes layer 1; blocks 1 .. NB2-kPeel-1 run in a loop over pairs, so that the
      // two accumulators alternate roles without copies.
      f32x16 carry = l2_block(0, prev1, [&](const f32x16& p, int k) {
        if (k >= 1 && k <= 4) l1_relu_half(H1 / 32 - 2 + ((k - 1) >> 1), (k - 1) >> 1 ? p : prev0, (k - 1) & 1);
      }, in_tile, std::false_type{});
      for (int b = 1; b + 1 <= kSteady; b += 2) {
        const f32x16 a = l2_block(b, carry, l2_epilogue, in_tile, std::false_type{});
        carry = l2_block(b + 1, a, l2_epilogue, in_tile, std::false_type{});
      }
      if constexpr (kSteady % 2 == 1) carry = l2_block(kSteady, carry, l2_epilogue, in_tile, std::false_type{});
#pragma unroll
      for (int b = NB2 - kPeel; b < NB2 - 1; ++b) carry = l2_block(b, carry, l2_epilogue, wrapping, std::false_type{});
      carry = l2_block(NB2 - 1, carry, l2_epilogue, wrapping, std::true_type{});
      l2_epilogue(carry, -1);
    } else {
      // ---- layer 1, G groups: one 32-neuron block at a time (two per chunk), each block's
      // ReLU deferred into the next block's chain; activations in the accumulation registers
      bf16x8 h1[G][H1 / 16];
      auto l1_relu = [&](int nb, const AccGroups<G>& acc) {
#pragma unroll
        for (int gr = 0; gr < G; ++gr)
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            h1[gr][2 * nb + half] = relu_bf16(acc.v[gr], half);
            asm volatile("" : "+a"(h1[gr][2 * nb + half]));
          }
      };
      // The chains hand over as with one group (mfma_chain_handover, kLookaheadGroups K-steps
      // ahead): the first block of a layer-1 chunk to the second within the same chunk (no
      // barrier), the second to the next chunk; the next block's biases are read mid-chain and
      // the previous block's deferred ReLU runs one piece per step.
      constexpr int LA = kLookaheadGroups;
      constexpr int kBiasStep = 8;
      auto l1_frag = [&](const unsigned char* buf, int lb, int k) {
        return *reinterpret_cast<const bf16x8*>(buf + ((k & 4) ? l1b[lb] : l1a[lb]) + k * 32);
      };
      auto l2_frag = [&](const unsigned char* buf, int k) {
        return *reinterpret_cast<const bf16x8*>(buf + l2 + k * 32);
      };
      auto l1_relu_piece = [&](int nb, const AccGroups<G>& acc, int piece) {   // piece = 2 gr + half
        const int gr = piece >> 1, half = piece & 1;
        h1[gr][2 * nb + half] = relu_bf16(acc.v[gr], half);
        asm volatile("" : "+a"(h1[gr][2 * nb + half]));
      };
      auto no_release = [&]() {};
      bf16x8 fr[LA];
#pragma unroll
      for (int k = 0; k < LA; ++k) fr[k] = l1_frag(lds + (g % kBufs) * CHUNK, 0, k);
      f32x16 nb = bias_acc(s_b1, h);          // biases of the next chain's block
      AccGroups<G> prev;
#pragma unroll
      for (int c = 0; c < NC1; ++c) {
        const unsigned char* buf = lds + (g % kBufs) * CHUNK;
        const unsigned char* nbuf = lds + ((g + 1) % kBufs) * CHUNK;
        const unsigned char* dst = ahead();
#pragma unroll
        for (int lb = 0; lb < 2; ++lb) {
          const int blk = 2 * c + lb;
          AccGroups<G> acc;
#pragma unroll
          for (int gr = 0; gr < G; ++gr) acc.v[gr] = nb;
          auto mma = [&](int k, const bf16x8& a) {
#pragma unroll
            for (int gr = 0; gr < G; ++gr)
              acc.v[gr] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, xf[gr][k], acc.v[gr], 0, 0, 0);
          };
          auto side = [&](int k) {
            spread(tile, parity, NX + c + kAhead, dst, KS1 * lb + k);
            if (blk > 0 && k >= 1 && k <= 2 * G) l1_relu_piece(blk - 1, prev, k - 1);
            if (k == kBiasStep) nb = blk + 1 < H1 / 32 ? bias_acc(s_b1 + (blk + 1) * 32, h) : bias_acc(s_b2, h);
          };
          if (lb == 0)
            mfma_chain_handover<KS1, true, LA>(
                fr, [&](int k) { return l1_frag(buf, 0, k); }, [&](int i) { return l1_frag(buf, 1, i); }, mma,
                [&]() {}, side, no_release);
          else
            mfma_chain_handover<KS1, true, LA>(
                fr, [&](int k) { return l1_frag(buf, 1, k); },
                [&](int i) { return c + 1 < NC1 ? l1_frag(nbuf, 0, i) : l2_frag(nbuf, i); }, mma, [&]() {}, side,
                release);
          prev = acc;
        }
        __builtin_amdgcn_sched_barrier(0);
      }

      // ---- layer 2, G groups; epilogues deferred as for G = 1, in pieces over the first steps
      zero_logits();
      bf16x8 h2[2];
      auto l2_epilogue = [&](const AccGroups<G>& p, int k) {   // k < 0: all at once
#pragma unroll
        for (int gr = 0; gr < G; ++gr) {
          if (k < 0 || k == 1 + 3 * gr) {
#pragma unroll
            for (int half = 0; half < 2; ++half) h2[half] = relu_bf16(p.v[gr], half);
          }
#pragma unroll
          for (int bt = 0; bt < BT; ++bt)
            if (k < 0 || k == 2 + 3 * gr + bt) {
#pragma unroll
              for (int tt = 0; tt < 2; ++tt)
                logit[gr][bt] =
                    __builtin_amdgcn_mfma_f32_32x32x16_bf16(w3f[bt][tt], h2[tt], logit[gr][bt], 0, 0, 0);
            }
        }
      };
      auto l2_block = [&](int b, const AccGroups<G>& p, auto&& pre, auto&& load_ahead, auto last) {
        AccGroups<G> acc;
#pragma unroll
        for (int gr = 0; gr < G; ++gr) acc.v[gr] = nb;
#pragma unroll
        for (int part = 0; part < KP; ++part) {
          const unsigned char* buf = lds + (g % kBufs) * CHUNK;
          const unsigned char* nbuf = lds + ((g + 1) % kBufs) * CHUNK;
          const unsigned char* dst = ahead();
          auto chain = [&](auto next_exists) {
            mfma_chain_handover<32, decltype(next_exists)::value, LA>(
                fr, [&](int k) { return l2_frag(buf, k); }, [&](int i) { return l2_frag(nbuf, i); },
                [&](int k, const bf16x8& a) {
#pragma unroll
                  for (int gr = 0; gr < G; ++gr)
                    acc.v[gr] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, h1[gr][part * 32 + k], acc.v[gr], 0, 0, 0);
                },
                [&]() {},
                [&](int k) {
                  load_ahead(b * KP + part + kAhead, dst, k);
                  if (part == 0) pre(p, k);
                  if (part == KP - 1 && k == kBiasStep && !decltype(last)::value) nb = bias_acc(s_b2 + (b + 1) * 32, h);
                },
                release);
          };
          if (decltype(last)::value && part == KP - 1) chain(std::false_type{});
          else chain(std::true_type{});
          if (part == KP - 1) read_w3(buf);
          __builtin_amdgcn_sched_barrier(0);
        }
        return acc;
      };
      AccGroups<G> carry = l2_block(0, prev, [&](const AccGroups<G>& q, int k) {
        if (k >= 1 && k <= 2 * G) l1_relu_piece(H1 / 32 - 1, q, k - 1);
      }, in_tile, std::false_type{});
      for (int b = 1; b + 1 <= kSteady; b += 2) {
        const AccGroups<G> a = l2_block(b, carry, l2_epilogue, in_tile, std::false_type{});
        carry = l2_block(b + 1, a, l2_epilogue, in_tile, std::false_type{});
      }
      if constexpr (kSteady % 2 == 1) carry = l2_block(kSteady, carry, l2_epilogue, in_tile, std::false_type{});
#pragma unroll
      for (int b = NB2 - kPeel; b < NB2 - 1; ++b) carry = l2_block(b, carry, l2_epilogue, wrapping, std::false_type{});
      carry = l2_block(NB2 - 1, carry, l2_epilogue, wrapping, std::true_type{});
      l2_epilogue(carry, -1);
    }

    if constexpr (kRoles) {
      // output 0 of each group's row r32 sits in register 0 of lane-half 0; lane-half h finishes
      // the row of group h (G = 2), lane-half 0 that of the only group (G = 1)
      float z0[G];
#pragma unroll
      for (int gr = 0; gr < G; ++gr) z0[gr] = G == 1 ? logit[0][0][0] : __shfl(logit[gr][0][0], r32);
      const int mine = G == 1 ? 0 : h;
      const int local = (G * wave + mine) * kRowsPerWave + r32;
      const int32_t stage = s_meta[parity][3][local];
      if ((G > 1 || h == 0) && stage >= 0)
        role_row(mine ? z0[G - 1] : z0[0], s_b3[0], coef_cur, __int_as_float(s_meta[parity][2][local]), role_max_len,
                 stage, s_meta[parity][0][local], s_meta[parity][1][local], s_alpha, n_models, pred_len, kv_bytes);
    } else if constexpr (kTwoPhase) {
      // Both lane-halves select each group's head output; then lane-half h finishes row r of
      // group h (G = 2), or lane-half 0 the wavefront's only group (G = 1), so that the rest
      // of the row runs once per wavefront.
      float zg[G], z0[G];
      int gh[G];
#pragma unroll
      for (int gr = 0; gr < G; ++gr) {
        const int local = (G * wave + gr) * kRowsPerWave + r32;
        gh[gr] = head_of_role(s_meta[parity][2][local], s_head, tp.n_roles, B);
        zg[gr] = head_output<BT>(logit[gr], gh[gr], h);
        z0[gr] = __shfl(logit[gr][0][0], r32);     // output 0: register 0 of lane-half 0
      }
      const int mine = G == 1 ? 0 : h;
      const int local = (G * wave + mine) * kRowsPerWave + r32;
      const int64_t row = tile * kTileRows + local;
      if ((G > 1 || h == 0) && row < n)
        two_phase_row(mine ? z0[G - 1] : z0[0], mine ? zg[G - 1] : zg[0], mine ? gh[G - 1] : gh[0], s_b3, s_c,
                      s_kx, s_ky, tp, row, s_meta[parity][0][local], s_meta[parity][1][local],
                      s_meta[parity][3][local], s_alpha, n_models, pred_len, kv_bytes);
    } else {
#pragma unroll
      for (int gr = 0; gr < G; ++gr) {
        const int local = (G * wave + gr) * kRowsPerWave + r32;
        const int64_t row = tile * kTileRows + local;
        length_epilogue<BT>(logit[gr], s_b3, s_c, h, row, n, s_meta[parity][0][local], s_meta[parity][1][local],
                            s_alpha, n_models, pred_len, kv_bytes);
      }
    }
  }
  wait_chunk<0>();                        // no load into LDS outlives the workgroup
}

// ---------------------------------------------------------------------------------------------
// float32, two Linear layers: D -> H -> B (32x32x2 float32 MFMA)
// ---------------------------------------------------------------------------------------------
template <int D, int H, int B>
__global__ __launch_bounds__(kThreads) void mlp2_f32_kernel(
    const float* __restrict__ x, const float* __restrict__ w1, const float* __restrict__ w2,
    const float* __restrict__ b1, const float* __restrict__ b2, const float* __restrict__ centre,
    int64_t n, const int32_t* __restrict__ prompt_len, const int32_t* __restrict__ model_id,
    const float* __restrict__ alpha, int32_t n_models, float* __restrict__ pred_len,
    double* __restrict__ kv_bytes) {
  static_assert(D % 8 == 0 && H % 32 == 0 && B % 32 == 0, "tile shape");
  constexpr int KS1 = D / 2;         // K-steps of layer 1; lane-half h covers inputs [h*KS1, (h+1)*KS1)
  constexpr int NB1 = H / 32;
  constexpr int BT = B / 32;
  constexpr int ROW1 = D + 1;        // LDS row strides in floats (one-float pad)
  constexpr int ROW2 = H + 1;
  __shared__ float sw1[H * ROW1];
  __shared__ float sw2[B * ROW2];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, h = lane >> 5, r32 = lane & 31;
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + wave * kRowsPerWave + r32;
  const int64_t xrow = row < n ? row : n - 1;

  // weights staged with 16-byte loads, all issued before the first LDS store, so the staging
  // costs one memory latency rather than one per element
  static_assert((H * D) % (4 * kThreads) == 0 && (B * H) % (4 * kThreads) == 0 && D % 4 == 0 && H % 4 == 0,
                "whole float4 staging rounds");
  {
    constexpr int N1 = H * D / (4 * kThreads), N2 = B * H / (4 * kThreads);
    float4 r1[N1], r2[N2];
#pragma unroll
    for (int j = 0; j < N1; ++j) r1[j] = reinterpret_cast<const float4*>(w1)[j * kThreads + tid];
#pragma unroll
    for (int j = 0; j < N2; ++j) r2[j] = reinterpret_cast<const float4*>(w2)[j * kThreads + tid];
#pragma unroll
    for (int j = 0; j < N1; ++j) {
      const int i = 4 * (j * kThreads + tid);
      float* d = sw1 + (i / D) * ROW1 + i % D;
      d[0] = r1[j].x; d[1] = r1[j].y; d[2] = r1[j].z; d[3] = r1[j].w;
    }
#pragma unroll
    for (int j = 0; j < N2; ++j) {
      const int i = 4 * (j * kThreads + tid);
      float* d = sw2 + (i / H) * ROW2 + i % H;
      d[0] = r2[j].x; d[1] = r2[j].y; d[2] = r2[j].z; d[3] = r2[j].w;
    }
  }

  float xf[KS1];
  {
    const float* xp = x + xrow * D + h * KS1;
#pragma unroll
    for (int q = 0; q < KS1 / 4; ++q) {
      float4 f = *reinterpret_cast<const float4*>(xp + 4 * q);
      xf[4 * q] = f.x; xf[4 * q + 1] = f.y; xf[4 * q + 2] = f.z; xf[4 * q + 3] = f.w;
    }
  }
  __syncthreads();

  f32x16 h1[NB1];
#pragma unroll
  for (int nb = 0; nb < NB1; ++nb) {
    f32x16 acc = {};
    const float* wr = sw1 + (nb * 32 + r32) * ROW1 + h * KS1;
#pragma unroll
    for (int ks = 0; ks < KS1; ++ks) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(wr[ks], xf[ks], acc, 0, 0, 0);
    float bias[16];
    load_acc_layout(b1 + nb * 32, h, bias);
#pragma unroll
    for (int v = 0; v < 16; ++v) h1[nb][v] = fmaxf(acc[v] + bias[v], 0.0f);
  }

  f32x16 logit[BT];
#pragma unroll
  for (int bt = 0; bt < BT; ++bt) {
    f32x16 acc = {};
    const float* wr = sw2 + (bt * 32 + r32) * ROW2;
#pragma unroll
    for (int nb = 0; nb < NB1; ++nb) {
#pragma unroll
      for (int v = 0; v < 16; ++v)
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(wr[nb * 32 + acc_row(v, h)], h1[nb][v], acc, 0, 0, 0);
    }
    logit[bt] = acc;
  }

  const int32_t prompt = row < n ? prompt_len[row] : 0;
  const int32_t model = row < n ? model_id[row] : 0;
  length_epilogue<BT>(logit, b2, centre, h, row, n, prompt, model, alpha, n_models, pred_len, kv_bytes);
}

bool dims_are(const maestro_predictor& p, int32_t layers, int32_t dtype, const int32_t* d) {
  if (p.n_layers != layers || p.dtype != dtype) return false;
  for (int i = 0; i <= layers; ++i)
    if (p.dims[i] != d[i]) return false;
  return true;
}

constexpr int32_t kF32Small[] = {64, 128, 32};
constexpr int32_t kBf16Mid[] = {256, 512, 512, 64};
constexpr int32_t kBf16Wide[] = {256, 1024, 1024, 64};

// Row groups per wavefront of the bfloat16 predictor: two for the 512-wide hidden layers (256-row
// tiles), one for the 1024-wide ones, whose layer-1 activations alone fill the accumulation
// registers (128-row tiles).
constexpr int kMidGroups = 2;

template <bool kTwoPhase>
maestro_status launch_mlp3(const maestro_predictor& p, int64_t n, const void* x, const int32_t* prompt_len,
                           const int32_t* model_id, const float* kv_bytes_per_token, int32_t n_models,
                           float* pred_len, double* kv_bytes, const TwoPhaseArgs& tp, hipStream_t stream) {
  const bool mid = p.dims[1] == 512;
  const int64_t tile_rows = (int64_t)(mid ? kMidGroups : 1) * kRowsPerBlock;
  const int64_t n_tiles = (n + tile_rows - 1) / tile_rows;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
    return MAESTRO_ERR_LAUNCH;
  const dim3 pgrid((unsigned)(n_tiles < cus ? n_tiles : cus)), block(kThreads);
  auto args = [&](auto kernel) {
    kernel<<<pgrid, block, 0, stream>>>(
        static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(p.weight[0]),
        static_cast<const uint16_t*>(p.weight[1]), static_cast<const uint16_t*>(p.weight[2]),
        p.bias[0], p.bias[1], p.bias[2], kTwoPhase ? nullptr : p.bin_centre, n, n_tiles, prompt_len, model_id,
        kv_bytes_per_token, n_models, pred_len, kv_bytes, tp, nullptr, nullptr, nullptr, nullptr, nullptr, 0.0f);
  };
  if (mid) args(mlp3_bf16_kernel<256, 512, 512, 64, kMidGroups, kTwoPhase>);
  else args(mlp3_bf16_kernel<256, 1024, 1024, 64, 1, kTwoPhase>);
  return launch_status();
}

}  // namespace

bool predict_shape_supported(const maestro_predictor& p) {
  return dims_are(p, 2, MAESTRO_F32, kF32Small) || dims_are(p, 3, MAESTRO_BF16, kBf16Mid) ||
         dims_are(p, 3, MAESTRO_BF16, kBf16Wide);
}

maestro_status launch_predict(const maestro_predictor& p, int64_t n, const void* x,
                              const int32_t* prompt_len, const int32_t* model_id,
                              const float* kv_bytes_per_token, int32_t n_models, float* pred_len,
                              double* kv_bytes, hipStream_t stream) {
  if (n == 0) return MAESTRO_OK;
  const dim3 grid((unsigned)((n + kRowsPerBlock - 1) / kRowsPerBlock)), block(kThreads);
  if (dims_are(p, 2, MAESTRO_F32, kF32Small)) {
    mlp2_f32_kernel<64, 128, 32><<<grid, block, 0, stream>>>(
        static_cast<const float*>(x), static_cast<const float*>(p.weight[0]),
        static_cast<const float*>(p.weight[1]), p.bias[0], p.bias[1], p.bin_centre, n, prompt_len,
        model_id, kv_bytes_per_token, n_models, pred_len, kv_bytes);
  } else if (dims_are(p, 3, MAESTRO_BF16, kBf16Mid) || dims_are(p, 3, MAESTRO_BF16, kBf16Wide)) {
    return launch_mlp3<false>(p, n, x, prompt_len, model_id, kv_bytes_per_token, n_models, pred_len, kv_bytes,
                              TwoPhaseArgs{}, stream);
  } else {
    return MAESTRO_ERR_UNSUPPORTED;
  }
  return launch_status();
}

// The regressors' grouped GEMM: one persistent workgroup per compute unit (at most one per
// possible tile), the tile count read on the device.
maestro_status launch_role_regressors(const maestro_predictor& p, int64_t n, const void* x, const float* coef,
                                      float max_len, const int32_t* tile_group, const int32_t* perm,
                                      const int32_t* prompt_p, const int32_t* model_p, const int32_t* p_bits,
                                      const int32_t* n_tiles, int64_t max_tiles, const float* kv_bytes_per_token,
                                      int32_t n_models, float* pred_len, double* kv_bytes, hipStream_t stream) {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
    return MAESTRO_ERR_LAUNCH;
  const dim3 pgrid((unsigned)(max_tiles < cus ? max_tiles : cus)), block(kThreads);
  auto args = [&](auto kernel) {
    kernel<<<pgrid, block, 0, stream>>>(
        static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(p.weight[0]),
        static_cast<const uint16_t*>(p.weight[1]), static_cast<const uint16_t*>(p.weight[2]), p.bias[0],
        p.bias[1], p.bias[2], nullptr, n, 0, prompt_p, model_p, kv_bytes_per_token, n_models, pred_len, kv_bytes,
        TwoPhaseArgs{}, tile_group, perm, p_bits, n_tiles, coef, max_len);
  };
  if (p.dims[1] == 512) args(mlp3_bf16_kernel<256, 512, 512, 64, kMidGroups, false, true>);
  else args(mlp3_bf16_kernel<256, 1024, 1024, 64, 1, false, true>);
  return launch_status();
}

int32_t role_tile_rows(const maestro_predictor& p) {
  return (p.dims[1] == 512 ? kMidGroups : 1) * kRowsPerBlock;
}

bool two_phase_shape_supported(const maestro_predictor& p) {
  return dims_are(p, 3, MAESTRO_BF16, kBf16Mid) || dims_are(p, 3, MAESTRO_BF16, kBf16Wide);
}

maestro_status launch_predict_two_phase(const maestro_predictor& p, const maestro_two_phase& t, int64_t n,
                                        const void* x, const int32_t* prompt_len, const int32_t* model_id,
                                        const int32_t* role_id, const int32_t* tool_avail,
                                        const float* kv_bytes_per_token, int32_t n_models, float* p_tool,
                                        float* pred_len, double* kv_bytes, hipStream_t stream) {
  if (n == 0) return MAESTRO_OK;
  if (!two_phase_shape_supported(p)) return MAESTRO_ERR_UNSUPPORTED;
  const TwoPhaseArgs tp{role_id, tool_avail, t.role_head, t.tool_coef, t.iso_x, t.iso_y,
                        t.n_roles, t.n_knots, t.max_len, p_tool};
  return launch_mlp3<true>(p, n, x, prompt_len, model_id, kv_bytes_per_token, n_models, pred_len, kv_bytes, tp,
                           stream);
}

}  // namespace maestro

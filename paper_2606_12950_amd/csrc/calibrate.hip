// Matrix-core ceilings of the chip, for measurement only (built as its own small library, which
// the scheduler library never loads): one wavefront per SIMD, as the predictor runs (256 threads
// per workgroup, one workgroup per compute unit), and nothing but bfloat16 32x32x16 MFMAs on
// pseudo-random operands (the chip's clock under its power limit depends on how many bits
// toggle, so zeros would overstate the ceiling) -- no global memory traffic and no barriers.
//   lds_every = 0: both operands in registers.
//   lds_every = 1: the A operand of every MFMA read from LDS (a 16-byte read per lane, issued
//                  three MFMAs ahead), the predictor's LDS traffic with one row group;
//   lds_every = 2: one such read feeding two MFMAs, as with two row groups.
// n_acc = 1 chains every MFMA on the previous one's result (as the predictor's layer-2 blocks
// do); n_acc = 4 rotates four independent accumulators.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;
constexpr int kBlocks = 256;
constexpr int kLdsBytes = 64 * 1024;       // 16 KB per wavefront: 16 fragments of 1 KB

__device__ __forceinline__ uint32_t xorshift(uint32_t& h) {
  h ^= h << 13;
  h ^= h >> 17;
  h ^= h << 5;
  return h;
}

// two bfloat16 of magnitude in [2^-7, 2^8) and random signs
__device__ __forceinline__ uint32_t random_bf16x2(uint32_t& h) {
  const uint32_t r = xorshift(h), s = xorshift(h);
  return (0x3C003C00u + (r & 0x07FF07FFu)) ^ (s & 0x80008000u);
}

template <int NACC, int LDS_EVERY>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void mfma_ceiling_kernel(float* __restrict__ out, int rounds, uint32_t seed) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_EVERY ? kLdsBytes : 16];
  const uint32_t tid = blockIdx.x * kThreads + threadIdx.x;
  uint32_t h = (tid * 2654435761u) ^ seed;
  if (h == 0) h = 1;
  if constexpr (LDS_EVERY > 0) {
    for (int i = threadIdx.x; i < kLdsBytes / 4; i += kThreads) reinterpret_cast<uint32_t*>(lds)[i] = random_bf16x2(h);
    __syncthreads();
  }
  bf16x8 a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a[i] = __builtin_bit_cast(bf16x8, make_uint4(random_bf16x2(h), random_bf16x2(h), random_bf16x2(h), random_bf16x2(h)));
    b[i] = __builtin_bit_cast(bf16x8, make_uint4(random_bf16x2(h), random_bf16x2(h), random_bf16x2(h), random_bf16x2(h)));
  }
  // lane's 16 bytes of fragment j of its wavefront: byte (wave * 16 + j) * 1024 + 16 * lane
  const unsigned char* frag = lds + (threadIdx.x >> 6) * 16384 + (threadIdx.x & 63) * 16;
  constexpr int LA = 3;
  if constexpr (LDS_EVERY > 0) {
#pragma unroll
    for (int j = 0; j < LA; ++j) a[j] = *reinterpret_cast<const bf16x8*>(frag + j * 1024);
  }
  f32x16 acc[NACC];
#pragma unroll
  for (int i = 0; i < NACC; ++i) acc[i] = f32x16{};
  // 16 MFMAs per round whatever NACC and LDS_EVERY are
  for (int r = 0; r < rounds; ++r) {
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      if constexpr (LDS_EVERY > 0) {
        if (k % LDS_EVERY == 0) {   // the fragment LA reads ahead, into the slot freed LA reads ago
          const int j = (k / LDS_EVERY + LA) % (16 / LDS_EVERY);
          a[(k / LDS_EVERY + LA) & 3] = *reinterpret_cast<const bf16x8*>(frag + j * 1024);
        }
      }
      const bf16x8 av = LDS_EVERY ? a[(k / (LDS_EVERY ? LDS_EVERY : 1)) & 3] : a[k & 3];
      acc[k % NACC] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, b[k & 3], acc[k % NACC], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < NACC; ++i)
#pragma unroll
    for (int j = 0; j < 16; ++j) s += acc[i][j];
  out[tid] = s;   // keeps the products live
}

template <int NACC>
void launch(int lds_every, float* out, int rounds, uint32_t seed, hipStream_t s) {
  if (lds_every == 0) mfma_ceiling_kernel<NACC, 0><<<dim3(kBlocks), dim3(kThreads), 0, s>>>(out, rounds, seed);
  else if (lds_every == 1) mfma_ceiling_kernel<NACC, 1><<<dim3(kBlocks), dim3(kThreads), 0, s>>>(out, rounds, seed);
  else mfma_ceiling_kernel<NACC, 2><<<dim3(kBlocks), dim3(kThreads), 0, s>>>(out, rounds, seed);
}

}  // namespace

extern "C" {

// Launches kBlocks x kThreads threads, each wavefront issuing 16 * rounds MFMAs of
// 32 x 32 x 16 (32,768 flop each); out must hold maestro_calibrate_mfma_outputs() floats.
// n_acc is 1 or 4, lds_every 0, 1 or 2; returns 0, or -1 for a bad argument or a failed launch.
__attribute__((visibility("default"))) int maestro_calibrate_mfma(float* out, int rounds, int n_acc, int lds_every,
                                                                  uint32_t seed, void* stream) {
  if (!out || rounds < 1 || (n_acc != 1 && n_acc != 4) || lds_every < 0 || lds_every > 2) return -1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (n_acc == 1) launch<1>(lds_every, out, rounds, seed, s);
  else launch<4>(lds_every, out, rounds, seed, s);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

__attribute__((visibility("default"))) int maestro_calibrate_mfma_outputs(void) { return kBlocks * kThreads; }

// MFMAs one call issues: 16 * rounds per wavefront, 4 wavefronts per workgroup
__attribute__((visibility("default"))) int64_t maestro_calibrate_mfma_count(int rounds) {
  return (int64_t)16 * rounds * (kThreads / 64) * kBlocks;
}

}  // extern "C"

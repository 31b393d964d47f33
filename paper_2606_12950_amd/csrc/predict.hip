// Cost prediction for a batch of stages (Sec. III-B; Eq. 3): the feature MLP over length bins,
// softmax, expected length, KV bytes -- one fused kernel, logits and hidden layers never leave
// the chip.
//
// Layout of the work. Each wavefront owns 32 stages (rows). Every Linear layer is computed
// transposed, H^T = W * X^T, on 32x32 MFMA tiles: the weights are the A operand (32 output
// neurons x K) and the activations the B operand (K x 32 rows). A 32x32 result tile leaves
// lane (h*32 + r) holding, for row r, the 16 neurons (v/4)*8 + 4h + v%4 (v = 0..15). Those 16
// values are exactly what the same lane must feed as the B operand of the next layer over a
// K-slice of 32 inputs, provided the next layer's weight columns are read in the matching
// order (a fixed permutation of K, which leaves the dot products unchanged). So hidden
// activations stay in registers from one layer to the next, and the last hidden layer is
// consumed block by block into the logit accumulators without ever being stored whole.
//
// Weights stream through LDS: each 32-neuron block of a layer (plus, for the last hidden
// layer, the matching 32 columns of the logit layer) is staged once per workgroup in a
// double buffer and read by the four wavefronts; rows are padded by 8 bytes so that the 32
// rows a wavefront reads at one column fall in distinct LDS banks.
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

__device__ __forceinline__ bf16x8 as_bf16x8(uint2 lo, uint2 hi) {
  uint4 u = make_uint4(lo.x, lo.y, hi.x, hi.y);
  return __builtin_bit_cast(bf16x8, u);
}

// 16 consecutive floats of a 32-wide slice as seen by accumulator registers of lane-half h:
// out[v] = src[acc_row(v, h)].
__device__ __forceinline__ void load_acc_layout(const float* __restrict__ src, int h, float (&out)[16]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float4 f = *reinterpret_cast<const float4*>(src + q * 8 + h * 4);
    out[q * 4 + 0] = f.x; out[q * 4 + 1] = f.y; out[q * 4 + 2] = f.z; out[q * 4 + 3] = f.w;
  }
}

// Softmax over the B = 32*BT logits of each row, expected length, Eq. 3 KV bytes.
// Lanes r and r + 32 hold complementary halves of row r's logits.
template <int BT>
__device__ __forceinline__ void length_epilogue(const f32x16 (&logit)[BT], const float* __restrict__ b_last,
                                                const float* __restrict__ centre, int h, int64_t row, int64_t n,
                                                const int32_t* __restrict__ prompt_len,
                                                const int32_t* __restrict__ model_id,
                                                const float* __restrict__ alpha,
                                                float* __restrict__ pred_len, double* __restrict__ kv_bytes) {
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
  float se = 0.0f, sc = 0.0f;
#pragma unroll
  for (int bt = 0; bt < BT; ++bt) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      float e = __expf(z[bt][v] - mx);
      se += e;
      sc += e * c[bt][v];
    }
  }
  se += __shfl_xor(se, 32);
  sc += __shfl_xor(sc, 32);
  if (h == 0 && row < n) {
    const float pred = sc / se;
    pred_len[row] = pred;
    const int m = model_id[row];
    kv_bytes[row] = ((double)prompt_len[row] + (double)pred) * (double)alpha[m];
  }
}

// ---------------------------------------------------------------------------------------------
// bfloat16, three Linear layers: D -> H1 -> H2 -> B
// ---------------------------------------------------------------------------------------------
template <int D, int H1, int H2, int B>
__global__ __launch_bounds__(kThreads) void mlp3_bf16_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w1, const uint16_t* __restrict__ w2,
    const uint16_t* __restrict__ w3, const float* __restrict__ b1, const float* __restrict__ b2,
    const float* __restrict__ b3, const float* __restrict__ centre, int64_t n,
    const int32_t* __restrict__ prompt_len, const int32_t* __restrict__ model_id,
    const float* __restrict__ alpha, float* __restrict__ pred_len, double* __restrict__ kv_bytes) {
  static_assert(D % 16 == 0 && H1 % 32 == 0 && H2 % 32 == 0 && B % 32 == 0, "tile shape");
  constexpr int KS1 = D / 16;        // K-steps of layer 1 (32x32x16 MFMA)
  constexpr int NB1 = H1 / 32;       // neuron blocks of layer 1
  constexpr int KS2 = H1 / 16;       // K-steps of layer 2
  constexpr int NB2 = H2 / 32;       // neuron blocks of layer 2
  constexpr int BT = B / 32;         // bin tiles of the logit layer
  constexpr int ROW1 = 2 * D + 8;    // LDS row strides in bytes (8-byte pad)
  constexpr int ROW2 = 2 * H1 + 8;
  constexpr int ROW3 = 2 * 32 + 8;
  constexpr int W3OFF = 32 * ROW2;
  constexpr int CHUNK = cmax(32 * ROW1, 32 * ROW2 + B * ROW3);
  constexpr int P1 = 32 * D / 8;     // 16-byte pieces per staged chunk part
  constexpr int P2 = 32 * H1 / 8;
  constexpr int P3 = B * 32 / 8;
  constexpr int R1 = (P1 + kThreads - 1) / kThreads;
  constexpr int R2 = (P2 + kThreads - 1) / kThreads;
  constexpr int R3 = (P3 + kThreads - 1) / kThreads;
  constexpr int RP = cmax(R1, R2 + R3);

  __shared__ __attribute__((aligned(16))) unsigned char lds[2][CHUNK];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, h = lane >> 5, r32 = lane & 31;
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + wave * kRowsPerWave + r32;
  const int64_t xrow = row < n ? row : n - 1;

  uint4 pre[RP];
  // layer-1 chunk nb: W1 rows nb*32 .. nb*32+31
  auto fetch1 = [&](int nb) {
#pragma unroll
    for (int i = 0; i < R1; ++i) {
      const int p = tid + i * kThreads;
      if (P1 % kThreads == 0 || p < P1) {
        const int r = p / (D / 8), c8 = p % (D / 8);
        pre[i] = *reinterpret_cast<const uint4*>(w1 + (size_t)(nb * 32 + r) * D + c8 * 8);
      }
    }
  };
  auto store1 = [&](unsigned char* buf) {
#pragma unroll
    for (int i = 0; i < R1; ++i) {
      const int p = tid + i * kThreads;
      if (P1 % kThreads == 0 || p < P1) {
        const int r = p / (D / 8), c8 = p % (D / 8);
        uint2* d = reinterpret_cast<uint2*>(buf + r * ROW1 + c8 * 16);
        d[0] = make_uint2(pre[i].x, pre[i].y);
        d[1] = make_uint2(pre[i].z, pre[i].w);
      }
    }
  };
  // layer-2 chunk nb2: W2 rows nb2*32 .. +31, and W3 columns nb2*32 .. +31 (all B rows)
  auto fetch2 = [&](int nb2) {
#pragma unroll
    for (int i = 0; i < R2; ++i) {
      const int p = tid + i * kThreads;
      if (P2 % kThreads == 0 || p < P2) {
        const int r = p / (H1 / 8), c8 = p % (H1 / 8);
        pre[i] = *reinterpret_cast<const uint4*>(w2 + (size_t)(nb2 * 32 + r) * H1 + c8 * 8);
      }
    }
#pragma unroll
    for (int i = 0; i < R3; ++i) {
      const int p = tid + i * kThreads;
      if (P3 % kThreads == 0 || p < P3) {
        const int r = p / 4, c8 = p % 4;
        pre[R2 + i] = *reinterpret_cast<const uint4*>(w3 + (size_t)r * H2 + nb2 * 32 + c8 * 8);
      }
    }
  };
  auto store2 = [&](unsigned char* buf) {
#pragma unroll
    for (int i = 0; i < R2; ++i) {
      const int p = tid + i * kThreads;
      if (P2 % kThreads == 0 || p < P2) {
        const int r = p / (H1 / 8), c8 = p % (H1 / 8);
        uint2* d = reinterpret_cast<uint2*>(buf + r * ROW2 + c8 * 16);
        d[0] = make_uint2(pre[i].x, pre[i].y);
        d[1] = make_uint2(pre[i].z, pre[i].w);
      }
    }
#pragma unroll
    for (int i = 0; i < R3; ++i) {
      const int p = tid + i * kThreads;
      if (P3 % kThreads == 0 || p < P3) {
        const int r = p / 4, c8 = p % 4;
        uint2* d = reinterpret_cast<uint2*>(buf + W3OFF + r * ROW3 + c8 * 16);
        d[0] = make_uint2(pre[R2 + i].x, pre[R2 + i].y);
        d[1] = make_uint2(pre[R2 + i].z, pre[R2 + i].w);
      }
    }
  };
  // A operand, natural K order: columns col + 8h .. col + 8h + 7 of the lane's row
  auto frag_nat = [&](const unsigned char* base, int stride, int col) -> bf16x8 {
    const unsigned char* p = base + r32 * stride + (col + h * 8) * 2;
    return as_bf16x8(*reinterpret_cast<const uint2*>(p), *reinterpret_cast<const uint2*>(p + 8));
  };
  // A operand, chained K order: columns col + 4h .. +3 and col + 8 + 4h .. +3, matching the
  // neurons a 32x32 result tile leaves in registers 8*half .. 8*half + 7 (col = 16 * step)
  auto frag_chain = [&](const unsigned char* base, int stride, int col) -> bf16x8 {
    const unsigned char* p = base + r32 * stride + (col + h * 4) * 2;
    return as_bf16x8(*reinterpret_cast<const uint2*>(p), *reinterpret_cast<const uint2*>(p + 16));
  };

  // B operand of layer 1: row xrow, natural K order
  bf16x8 xf[KS1];
  {
    const uint16_t* xp = x + xrow * D + h * 8;
#pragma unroll
    for (int ks = 0; ks < KS1; ++ks) xf[ks] = *reinterpret_cast<const bf16x8*>(xp + ks * 16);
  }

  fetch1(0);
  store1(lds[0]);
  __syncthreads();

  // ---- layer 1: H1 = relu(W1 x + b1), kept as the B operand of layer 2 -----------------
  bf16x8 h1[KS2];
#pragma unroll
  for (int nb = 0; nb < NB1; ++nb) {
    const unsigned char* buf = lds[nb & 1];
    if (nb + 1 < NB1) fetch1(nb + 1); else fetch2(0);
    f32x16 acc = {};
#pragma unroll
    for (int ks = 0; ks < KS1; ++ks)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_nat(buf, ROW1, ks * 16), xf[ks], acc, 0, 0, 0);
    float bias[16];
    load_acc_layout(b1 + nb * 32, h, bias);
#pragma unroll
    for (int half = 0; half < 2; ++half) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        h1[2 * nb + half][j] = (__bf16)fmaxf(acc[8 * half + j] + bias[8 * half + j], 0.0f);
    }
    if (nb + 1 < NB1) store1(lds[(nb + 1) & 1]); else store2(lds[(nb + 1) & 1]);
    __syncthreads();
  }

  // ---- layer 2 block by block, each block folded straight into the logits ---------------
  f32x16 logit[BT];
#pragma unroll
  for (int bt = 0; bt < BT; ++bt) logit[bt] = f32x16{};
  for (int nb2 = 0; nb2 < NB2; ++nb2) {
    const unsigned char* buf = lds[(NB1 + nb2) & 1];
    if (nb2 + 1 < NB2) fetch2(nb2 + 1);
    f32x16 acc = {};
#pragma unroll
    for (int t = 0; t < KS2; ++t)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag_chain(buf, ROW2, t * 16), h1[t], acc, 0, 0, 0);
    float bias[16];
    load_acc_layout(b2 + nb2 * 32, h, bias);
    bf16x8 h2[2];
#pragma unroll
    for (int half = 0; half < 2; ++half) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        h2[half][j] = (__bf16)fmaxf(acc[8 * half + j] + bias[8 * half + j], 0.0f);
    }
#pragma unroll
    for (int bt = 0; bt < BT; ++bt) {
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
        logit[bt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            frag_chain(buf + W3OFF + bt * 32 * ROW3, ROW3, tt * 16), h2[tt], logit[bt], 0, 0, 0);
    }
    if (nb2 + 1 < NB2) store2(lds[(NB1 + nb2 + 1) & 1]);
    __syncthreads();
  }

  length_epilogue<BT>(logit, b3, centre, h, row, n, prompt_len, model_id, alpha, pred_len, kv_bytes);
}

// ---------------------------------------------------------------------------------------------
// float32, two Linear layers: D -> H -> B (32x32x2 float32 MFMA)
// ---------------------------------------------------------------------------------------------
template <int D, int H, int B>
__global__ __launch_bounds__(kThreads) void mlp2_f32_kernel(
    const float* __restrict__ x, const float* __restrict__ w1, const float* __restrict__ w2,
    const float* __restrict__ b1, const float* __restrict__ b2, const float* __restrict__ centre,
    int64_t n, const int32_t* __restrict__ prompt_len, const int32_t* __restrict__ model_id,
    const float* __restrict__ alpha, float* __restrict__ pred_len, double* __restrict__ kv_bytes) {
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

  for (int i = tid; i < H * D; i += kThreads) sw1[(i / D) * ROW1 + i % D] = w1[i];
  for (int i = tid; i < B * H; i += kThreads) sw2[(i / H) * ROW2 + i % H] = w2[i];

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

  length_epilogue<BT>(logit, b2, centre, h, row, n, prompt_len, model_id, alpha, pred_len, kv_bytes);
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

}  // namespace

bool predict_shape_supported(const maestro_predictor& p) {
  return dims_are(p, 2, MAESTRO_F32, kF32Small) || dims_are(p, 3, MAESTRO_BF16, kBf16Mid) ||
         dims_are(p, 3, MAESTRO_BF16, kBf16Wide);
}

maestro_status launch_predict(const maestro_predictor& p, int64_t n, const void* x,
                              const int32_t* prompt_len, const int32_t* model_id,
                              const float* kv_bytes_per_token, float* pred_len,
                              double* kv_bytes, hipStream_t stream) {
  if (n == 0) return MAESTRO_OK;
  const dim3 grid((unsigned)((n + kRowsPerBlock - 1) / kRowsPerBlock)), block(kThreads);
  if (dims_are(p, 2, MAESTRO_F32, kF32Small)) {
    mlp2_f32_kernel<64, 128, 32><<<grid, block, 0, stream>>>(
        static_cast<const float*>(x), static_cast<const float*>(p.weight[0]),
        static_cast<const float*>(p.weight[1]), p.bias[0], p.bias[1], p.bin_centre, n, prompt_len,
        model_id, kv_bytes_per_token, pred_len, kv_bytes);
  } else if (dims_are(p, 3, MAESTRO_BF16, kBf16Mid)) {
    mlp3_bf16_kernel<256, 512, 512, 64><<<grid, block, 0, stream>>>(
        static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(p.weight[0]),
        static_cast<const uint16_t*>(p.weight[1]), static_cast<const uint16_t*>(p.weight[2]),
        p.bias[0], p.bias[1], p.bias[2], p.bin_centre, n, prompt_len, model_id,
        kv_bytes_per_token, pred_len, kv_bytes);
  } else if (dims_are(p, 3, MAESTRO_BF16, kBf16Wide)) {
    mlp3_bf16_kernel<256, 1024, 1024, 64><<<grid, block, 0, stream>>>(
        static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(p.weight[0]),
        static_cast<const uint16_t*>(p.weight[1]), static_cast<const uint16_t*>(p.weight[2]),
        p.bias[0], p.bias[1], p.bias[2], p.bin_centre, n, prompt_len, model_id,
        kv_bytes_per_token, pred_len, kv_bytes);
  } else {
    return MAESTRO_ERR_UNSUPPORTED;
  }
  return launch_status();
}

}  // namespace maestro

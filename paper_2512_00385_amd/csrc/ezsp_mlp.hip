// ezsp_mlp.hip -- a random-weight per-point MLP d_in -> 32 -> 32 -> d_out,
// the stand-in for the point embedding network of Sec. 3.1 on the
// LiDAR-sweep workload: bfloat16 inputs, weights and hidden activations
// (round to nearest even), fp32 accumulation and biases, ReLU after the two
// hidden layers.
//
// The layers are dense contractions, so they run on the matrix cores:
// v_mfma_f32_32x32x16_bf16 (CDNA4) in transposed form, D[unit][point] =
// sum_k W[k][unit] * X[point][k], one wave per tile of 32 points.  With the
// weights as the A operand and the activations as the B operand, the
// accumulator of one layer (lane l holds point l % 32, units
// 8 (r / 4) + 4 (l / 32) + r % 4 in register r) feeds the next layer's two
// K = 16 steps directly: step s takes registers 8s .. 8s + 7 of each lane
// as its eight B elements, and the A operand pairs each of those K slots
// with the weight row of the unit that register holds (the pairing of A and
// B elements to K slots is the same for both operands, so only the unit of
// each slot has to match).  The three layers chain in registers: the
// weights are loaded once per wave, and every point costs one read of its
// features and one write of its embedding.
#include <algorithm>

#include "ezsp_internal.h"

namespace ezsp {

namespace {

typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kMlpHidden = 32;

// fp32 -> bfloat16 bits, round to nearest even (finite values)
__device__ __forceinline__ short to_bf16(float v) {
  uint32_t u = __float_as_uint(v);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (short)(u >> 16);
}

// unit (row of D) of accumulator register r in lane l
__device__ __forceinline__ int acc_unit(int r, int lane) {
  return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}

// Input unit of element i of lane l's operands in K-step s of a hidden
// layer: the unit of accumulator register 8 s + i in lane l.
__device__ __forceinline__ int step_unit(int s, int i, int lane) {
  return acc_unit(8 * s + i, lane);
}

// A operand of K-step s of a hidden layer: lane l gives
// W[step_unit(s, i, l)][l % 32], zero outside d_rows x d_cols.
__device__ __forceinline__ bf16x8 weight_operand(const uint16_t *w,
                                                 int d_rows, int d_cols,
                                                 int s, int lane) {
  s16x8 a;
  const int m = lane & 31;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int k = step_unit(s, i, lane);
    a[i] = (k < d_rows && m < d_cols) ? (short)w[k * d_cols + m] : (short)0;
  }
  return __builtin_bit_cast(bf16x8, a);
}

// A operand of the first layer: element i of lane l is input feature
// 8 (l / 32) + i (the B operand holds the same feature of each point).
__device__ __forceinline__ bf16x8 input_weight_operand(const uint16_t *w,
                                                       int d_rows, int d_cols,
                                                       int lane) {
  s16x8 a;
  const int m = lane & 31;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int k = 8 * (lane >> 5) + i;
    a[i] = (k < d_rows && m < d_cols) ? (short)w[k * d_cols + m] : (short)0;
  }
  return __builtin_bit_cast(bf16x8, a);
}

// bias + ReLU, then the next layer's B operands (two K-steps)
__device__ __forceinline__ void hidden_operands(const f32x16 &acc,
                                                const float *bias_r,
                                                bf16x8 h[2]) {
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    s16x8 b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float v = acc[8 * s + i] + bias_r[8 * s + i];
      b[i] = to_bf16(v > 0.0f ? v : 0.0f);
    }
    h[s] = __builtin_bit_cast(bf16x8, b);
  }
}

template <bool VEC4>
__global__ __launch_bounds__(256) void k_mlp(
    const uint16_t *__restrict__ x, int32_t n, int32_t d_in, int32_t d_out,
    const uint16_t *__restrict__ w1, const float *__restrict__ b1,
    const uint16_t *__restrict__ w2, const float *__restrict__ b2,
    const uint16_t *__restrict__ w3, const float *__restrict__ b3,
    float *__restrict__ out) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t wave = (int32_t)(blockIdx.x * (blockDim.x / kWave) +
                                 threadIdx.x / kWave);
  const int32_t n_waves = (int32_t)(gridDim.x * (blockDim.x / kWave));
  // weights (A operands) and the biases of this lane's accumulator rows
  const bf16x8 a1 = input_weight_operand(w1, d_in, kMlpHidden, lane);
  bf16x8 a2[2], a3[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    a2[s] = weight_operand(w2, kMlpHidden, kMlpHidden, s, lane);
    a3[s] = weight_operand(w3, kMlpHidden, d_out, s, lane);
  }
  float c1[16], c2[16], c3[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int m = acc_unit(r, lane);
    c1[r] = b1[m];
    c2[r] = b2[m];
    c3[r] = m < d_out ? b3[m] : 0.0f;
  }
  const int32_t n_tiles = (n + 31) / 32;
  for (int32_t t = wave; t < n_tiles; t += n_waves) {
    const int32_t p = t * 32 + (lane & 31);
    // layer 1: B operand = features 8 (l / 32) .. + 7 of point p
    s16x8 xs;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int k = 8 * (lane >> 5) + i;
      xs[i] = (p < n && k < d_in) ? (short)x[(int64_t)p * d_in + k] : (short)0;
    }
    f32x16 acc = {0};
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
        a1, __builtin_bit_cast(bf16x8, xs), acc, 0, 0, 0);
    bf16x8 h[2];
    hidden_operands(acc, c1, h);
    // layer 2
    acc = f32x16{0};
#pragma unroll
    for (int s = 0; s < 2; ++s)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2[s], h[s], acc, 0, 0, 0);
    hidden_operands(acc, c2, h);
    // layer 3
    acc = f32x16{0};
#pragma unroll
    for (int s = 0; s < 2; ++s)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3[s], h[s], acc, 0, 0, 0);
    if (p < n) {
      float *o = out + (int64_t)p * d_out;
      if (VEC4) {  // registers 4g .. 4g + 3 are four consecutive units
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int m = acc_unit(4 * g, lane);
          if (m < d_out)
            *reinterpret_cast<float4 *>(o + m) =
                make_float4(acc[4 * g] + c3[4 * g], acc[4 * g + 1] + c3[4 * g + 1],
                            acc[4 * g + 2] + c3[4 * g + 2],
                            acc[4 * g + 3] + c3[4 * g + 3]);
        }
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = acc_unit(r, lane);
          if (m < d_out) o[m] = acc[r] + c3[r];
        }
      }
    }
  }
}

}  // namespace

int mlp_run(const uint16_t *x, int32_t n, int32_t d_in, int32_t d_out,
            const uint16_t *w1, const float *b1, const uint16_t *w2,
            const float *b2, const uint16_t *w3, const float *b3, float *out,
            hipStream_t st) {
  const int64_t tiles = ((int64_t)n + 31) / 32;
  // a few tiles per wave, so that its weight loads are shared
  const int64_t blocks = std::min<int64_t>((tiles + 3) / 4, 2048);
  const dim3 grid((unsigned)std::max<int64_t>(blocks, 1));
  const bool vec4 = d_out % 4 == 0 &&
                    (reinterpret_cast<uintptr_t>(out) & 15) == 0;
  prof_begin("embed_mlp", st);
  if (vec4)
    hipLaunchKernelGGL(k_mlp<true>, grid, dim3(256), 0, st, x, n, d_in, d_out,
                       w1, b1, w2, b2, w3, b3, out);
  else
    hipLaunchKernelGGL(k_mlp<false>, grid, dim3(256), 0, st, x, n, d_in,
                       d_out, w1, b1, w2, b2, w3, b3, out);
  prof_end(st);
  // stream-asynchronous: nothing is read back
  const int rc = check_hip(hipGetLastError(), "k_mlp launch");
  // algorithmic bytes: bfloat16 features in, fp32 embeddings out
  prof_bytes("embed_mlp", (2.0 * d_in + 4.0 * d_out) * n);
  return rc;
}

}  // namespace ezsp

// Shared device-side types and helpers for libbpt's gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;

#define BPT_DEV __device__ __forceinline__

template <typename T> BPT_DEV float to_f32(T x);
template <> BPT_DEV float to_f32<float>(float x) { return x; }
template <> BPT_DEV float to_f32<bf16>(bf16 x) { return (float)x; }

template <typename T> BPT_DEV T from_f32(float x);
template <> BPT_DEV float from_f32<float>(float x) { return x; }
template <> BPT_DEV bf16 from_f32<bf16>(float x) { return (bf16)x; }   // round to nearest even

// One bf16 MFMA step: 32x32 output tile, K = 16, fp32 accumulation.
// Operand layout (lane l of a wave64): A row (l % 32), B column (l % 32), each lane
// holding 8 consecutive K values starting at 8 * (l / 32). The 16 accumulator values
// of lane l sit at column (l % 32), rows 8*(r/4) + 4*(l/32) + (r%4), r = 0..15.
BPT_DEV f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

BPT_DEV float warp_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
BPT_DEV float warp_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

BPT_DEV float gelu_f(float z) { return 0.5f * z * (1.0f + erff(z * 0.70710678118654752f)); }
BPT_DEV float gelu_grad_f(float z) {
  return 0.5f * (1.0f + erff(z * 0.70710678118654752f)) +
         z * 0.39894228040143268f * __expf(-0.5f * z * z);
}

// Shared device-side types and helpers for libbpt's gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef _Float16 f16;
typedef __attribute__((__vector_size__(4 * sizeof(_Float16)))) _Float16 f16x4;
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
template <> BPT_DEV float to_f32<f16>(f16 x) { return (float)x; }

template <typename T> BPT_DEV T from_f32(float x);
template <> BPT_DEV float from_f32<float>(float x) { return x; }
template <> BPT_DEV bf16 from_f32<bf16>(float x) { return (bf16)x; }   // round to nearest even
template <> BPT_DEV f16 from_f32<f16>(float x) { return (f16)x; }      // round to nearest even

// One bf16 MFMA step: 32x32 output tile, K = 16, fp32 accumulation.
// Operand layout (lane l of a wave64): A row (l % 32), B column (l % 32), each lane
// holding 8 consecutive K values starting at 8 * (l / 32). The 16 accumulator values
// of lane l sit at column (l % 32), rows 8*(r/4) + 4*(l/32) + (r%4), r = 0..15.
BPT_DEV f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

BPT_DEV float warp_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// GELU with the exact erf, in fp32. erf of |z|/sqrt(2) by Abramowitz & Stegun,
// Handbook of Mathematical Functions, eq. 7.1.26: erf(x) = 1 - t P(t) exp(-x^2) with
// t = 1 / (1 + p x) and a degree-5 polynomial, |error| <= 1.5e-7 for x >= 0. The
// exp(-z^2/2) it needs is also the normal density of GELU' = Phi(z) + z phi(z).
BPT_DEV void gelu_both(float z, float& g, float& gp) {
  const float x = fabsf(z) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, x, 1.0f));
  const float poly = t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 1.061405429f, -1.453152027f), 1.421413741f),
                                      -0.284496736f), 0.254829592f);
  const float e = __builtin_amdgcn_exp2f(-x * x * 1.4426950408889634f);   // exp(-z^2 / 2)
  const float erf_abs = fmaf(-poly, e, 1.0f);
  const float phi_cdf = 0.5f + 0.5f * copysignf(erf_abs, z);            // Phi(z)
  g = z * phi_cdf;
  gp = fmaf(z * 0.39894228040143268f, e, phi_cdf);                       // + z exp(-z^2/2) / sqrt(2 pi)
}

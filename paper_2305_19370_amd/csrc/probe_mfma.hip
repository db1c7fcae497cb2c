// Matrix-core ceiling probe: bf16 32x32x16 MFMAs on register operands only (measurement).
#include <hip/hip_runtime.h>

#include "bpt_probe.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kLdsRegion = 16384;   // bytes of LDS per wave in the LDS-fed mode (16 fragments)

// MODE 0: one operand pair; 1: four different register operand pairs in turn; 2: the A
// operand of every product read from LDS (one 1 KiB fragment per product, row reads),
// 64 KiB of LDS per workgroup so that two workgroups (two waves per SIMD) share a CU.
template <int MODE>
__global__ __launch_bounds__(256) void mfma_loop_kernel(const float* __restrict__ seed, float* __restrict__ out,
                                                        int iters) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  bf16x8 a[4], b[4];
  for (int j = 0; j < 4; ++j)
    for (int i = 0; i < 8; ++i) {
      a[j][i] = (__bf16)seed[(gid * 67 + j * 8 + i) & 4095];
      b[j][i] = (__bf16)seed[(gid * 31 + j * 8 + i + 2048) & 4095];
    }
  if (MODE == 2) {
    for (int i = threadIdx.x; i < 4 * kLdsRegion / 2; i += 256) ((__bf16*)lds)[i] = (__bf16)seed[i & 4095];
    __syncthreads();
  }
  const char* region = lds + wave * kLdsRegion + lane * 16;
  f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int it = 0; it < iters; ++it) {
    if (MODE == 2) {
#pragma unroll
      for (int f = 0; f < 4; ++f) a[f] = *(const bf16x8*)(region + ((it * 4 + f) & 15) * 1024);
    }
    if (MODE == 0) {
      c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[0], c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[0], c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[0], c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[0], c3, 0, 0, 0);
    } else if (MODE == 1) {
      c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[1], c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[1], b[2], c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[2], b[3], c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[3], b[0], c3, 0, 0, 0);
    } else {
      c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[0], c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[1], b[1], c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[2], b[2], c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[3], b[3], c3, 0, 0, 0);
    }
  }
  float s = 0.f;
  for (int i = 0; i < 16; ++i) s += c0[i] + c1[i] + c2[i] + c3[i];
  out[gid] = s;
}

}  // namespace

extern "C" int32_t bpt_probe_mfma_loop(int64_t workgroups, int32_t iters, int32_t mode, const float* seed,
                                       float* out, void* stream) {
  if (workgroups < 1 || workgroups > (int64_t(1) << 24) || iters < 1 || mode < 0 || mode > 2 || !seed || !out)
    return 1;
  hipStream_t s = (hipStream_t)stream;
  const dim3 g((unsigned)workgroups), blk(256);
  if (mode == 0) hipLaunchKernelGGL(mfma_loop_kernel<0>, g, blk, 0, s, seed, out, iters);
  else if (mode == 1) hipLaunchKernelGGL(mfma_loop_kernel<1>, g, blk, 0, s, seed, out, iters);
  else hipLaunchKernelGGL(mfma_loop_kernel<2>, g, blk, 4 * kLdsRegion, s, seed, out, iters);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}

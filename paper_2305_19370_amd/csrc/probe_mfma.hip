// Matrix-core ceiling probe: loops of bf16 32x32x16 MFMAs with no global-memory traffic
// (measurement).
#include <hip/hip_runtime.h>

#include "bpt_probe.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kLdsRegion = 16384;        // bytes of LDS per wave read by the LDS-fed modes (16 fragments)
constexpr int kLdsTwoPerCu = 65536;      // per workgroup: two workgroups (two waves per SIMD) fit a CU
constexpr int kLdsOnePerCu = 98304;      // per workgroup: one workgroup (one wave per SIMD) per CU

// A operands of one iteration: SRC 0 one register pair; 1 four register pairs in turn;
// 2 one LDS fragment per product, read at the start of the iteration; 3 one LDS fragment
// per product, read one iteration ahead into a second register set; 4 one LDS fragment
// per two products (each fragment meets two different B operands), read one iteration
// ahead. Modes 3 and 4 run iterations in pairs (an odd count runs one more). The
// occupancy comes from the LDS the launch reserves.
template <int SRC>
__global__ __launch_bounds__(256) void mfma_loop_kernel(const float* __restrict__ seed, float* __restrict__ out,
                                                        int iters) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  constexpr bool kLds = SRC >= 2;
  constexpr int NF = SRC == 4 ? 2 : 4;   // fragments read per iteration
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  bf16x8 a[4], b[4], an[4];
  for (int j = 0; j < 4; ++j)
    for (int i = 0; i < 8; ++i) {
      a[j][i] = (__bf16)seed[(gid * 67 + j * 8 + i) & 4095];
      b[j][i] = (__bf16)seed[(gid * 31 + j * 8 + i + 2048) & 4095];
    }
  if (kLds) {
    for (int i = threadIdx.x; i < 4 * kLdsRegion / 2; i += 256) ((__bf16*)lds)[i] = (__bf16)seed[i & 4095];
    __syncthreads();
  }
  const char* region = lds + wave * kLdsRegion + lane * 16;   // fragment f at region + f * 1024, f < 16
  f32x16 c[4] = {};
  // the four products of one iteration on A operands x (x[f] for fragment-fed modes)
  auto products = [&](const bf16x8 (&x)[4]) {
    if (SRC == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x[0], b[0], c[j], 0, 0, 0);
    } else if (SRC == 1) {
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x[j], b[(j + 1) & 3], c[j], 0, 0, 0);
    } else if (SRC == 4) {
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x[j >> 1], b[j], c[j], 0, 0, 0);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x[j], b[j], c[j], 0, 0, 0);
    }
  };
  auto fetch = [&](bf16x8 (&x)[4], int it) {
#pragma unroll
    for (int f = 0; f < NF; ++f) x[f] = *(const bf16x8*)(region + ((it * NF + f) & 15) * 1024);
  };
  if (SRC <= 2) {
    for (int it = 0; it < iters; ++it) {
      if (SRC == 2) fetch(a, it);
      products(a);
    }
  } else {
    // two register sets in turn: the fragments of iteration it + 1 are read while the
    // products of iteration it run (the scheduling barriers keep that order)
    fetch(a, 0);
    for (int it = 0; it < iters; it += 2) {
      fetch(an, it + 1);
      __builtin_amdgcn_sched_barrier(0);
      products(a);
      __builtin_amdgcn_sched_barrier(0);
      fetch(a, it + 2);
      __builtin_amdgcn_sched_barrier(0);
      products(an);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  float s = 0.f;
  for (int i = 0; i < 16; ++i) s += c[0][i] + c[1][i] + c[2][i] + c[3][i];
  out[gid] = s;
}

template <int SRC>
hipError_t launch(int64_t workgroups, int lds_bytes, const float* seed, float* out, int iters, hipStream_t s) {
  if (lds_bytes > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)mfma_loop_kernel<SRC>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(mfma_loop_kernel<SRC>, dim3((unsigned)workgroups), dim3(256), lds_bytes, s, seed, out, iters);
  return hipGetLastError();
}

}  // namespace

extern "C" int32_t bpt_probe_mfma_loop(int64_t workgroups, int32_t iters, int32_t mode, const float* seed,
                                       float* out, void* stream) {
  if (workgroups < 1 || workgroups > (int64_t(1) << 24) || iters < 1 || mode < 0 || mode > 7 || !seed || !out)
    return 1;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e;
  switch (mode) {
    case 0: e = launch<0>(workgroups, 0, seed, out, iters, s); break;
    case 1: e = launch<1>(workgroups, 0, seed, out, iters, s); break;
    case 2: e = launch<2>(workgroups, kLdsTwoPerCu, seed, out, iters, s); break;
    case 3: e = launch<3>(workgroups, kLdsTwoPerCu, seed, out, iters, s); break;
    case 4: e = launch<4>(workgroups, kLdsTwoPerCu, seed, out, iters, s); break;
    case 5: e = launch<3>(workgroups, kLdsOnePerCu, seed, out, iters, s); break;
    case 6: e = launch<4>(workgroups, kLdsOnePerCu, seed, out, iters, s); break;
    default: e = launch<1>(workgroups, kLdsOnePerCu, seed, out, iters, s); break;
  }
  return e == hipSuccess ? 0 : 4;
}

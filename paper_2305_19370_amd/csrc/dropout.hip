// Dropout on the layer's two residual branches (the masks the paper's memory accounting
// keeps for the output projection and the FFN output). The mask is drawn from
// Philox4x32-10 (Salmon et al., SC 2011): element (t, n) of branch `site` takes word
// n mod 4 of the generator at counter (n / 4, t, site, 0) with the 64-bit seed as key, so
// forward and backward regenerate it instead of storing it. HBM-bound elementwise
// kernels: one thread per four consecutive columns (one generator call).
#include "common.h"
#include "internal.h"

namespace bpt {

namespace {

BPT_DEV u32x4 philox4x32_10(u32x4 c, uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    const uint32_t lo0 = 0xD2511F53u * c[0], hi0 = __umulhi(0xD2511F53u, c[0]);
    const uint32_t lo1 = 0xCD9E8D57u * c[2], hi1 = __umulhi(0xCD9E8D57u, c[2]);
    c = u32x4{hi1 ^ c[1] ^ k0, lo1, hi0 ^ c[3] ^ k1, lo0};
  }
  return c;
}

template <typename T> BPT_DEV void ld4(const T* p, float v[4]);
template <> BPT_DEV void ld4<float>(const float* p, float v[4]) {
  const f32x4 x = *(const f32x4*)p;
  v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
}
template <> BPT_DEV void ld4<bf16>(const bf16* p, float v[4]) {
  const bf16x4 x = *(const bf16x4*)p;
  v[0] = (float)x[0]; v[1] = (float)x[1]; v[2] = (float)x[2]; v[3] = (float)x[3];
}
template <typename T> BPT_DEV void st4(T* p, const float v[4]);
template <> BPT_DEV void st4<float>(float* p, const float v[4]) { *(f32x4*)p = f32x4{v[0], v[1], v[2], v[3]}; }
template <> BPT_DEV void st4<bf16>(bf16* p, const float v[4]) {
  bf16x4 x;
  x[0] = (bf16)v[0]; x[1] = (bf16)v[1]; x[2] = (bf16)v[2]; x[3] = (bf16)v[3];
  *(bf16x4*)p = x;
}

// keep factors (0 or scale) of columns n..n+3 of token t
BPT_DEV void factors(const DropArgs& a, int64_t t, int64_t n, float f[4]) {
  const u32x4 w = philox4x32_10(u32x4{(uint32_t)(n >> 2), (uint32_t)t, a.site, 0u}, a.k0, a.k1);
#pragma unroll
  for (int e = 0; e < 4; ++e) f[e] = w[e] >= a.threshold ? a.scale : 0.0f;
}

}  // namespace

// out[i, n] = R[i, n] + f(row0 + i, n) (acc[i, n] + bias[n])  (rows x D, D % 4 == 0)
template <typename TR, typename TO>
__global__ __launch_bounds__(256) void dropout_add_kernel(const float* acc, const TR* R, const float* bias, TO* out,
                                                          int64_t rows, int64_t D, DropArgs a) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t i = q / (D / 4), n = (q % (D / 4)) * 4;
  if (i >= rows) return;
  float f[4], x[4], r[4];
  factors(a, a.row0 + i, n, f);
  ld4(acc + i * D + n, x);
  ld4(R + i * D + n, r);
  if (bias) {
    float b[4];
    ld4(bias + n, b);
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] += b[e];
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) r[e] += f[e] * x[e];
  st4(out + i * D + n, r);
}

// out[i, n] = f(row0 + i, n) in[i, n]
template <typename TI, typename TO>
__global__ __launch_bounds__(256) void dropout_scale_kernel(const TI* in, TO* out, int64_t rows, int64_t D,
                                                            DropArgs a) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t i = q / (D / 4), n = (q % (D / 4)) * 4;
  if (i >= rows) return;
  float f[4], x[4];
  factors(a, a.row0 + i, n, f);
  ld4(in + i * D + n, x);
#pragma unroll
  for (int e = 0; e < 4; ++e) x[e] *= f[e];
  st4(out + i * D + n, x);
}

#define BPT_DT(dt, T, ...) \
  do {                     \
    if ((dt) == F32) {     \
      using T = float;     \
      __VA_ARGS__;         \
    } else {               \
      using T = bf16;      \
      __VA_ARGS__;         \
    }                      \
  } while (0)

hipError_t dropout_add(const float* acc, Dt tr, const void* R, const float* bias, Dt to, void* out, int64_t rows,
                       int64_t D, const DropArgs& a, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (D % 4 != 0) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((rows * (D / 4) + 255) / 256));
  BPT_DT(tr, TR, BPT_DT(to, TO, hipLaunchKernelGGL((dropout_add_kernel<TR, TO>), grid, dim3(256), 0, s, acc,
                                                   (const TR*)R, bias, (TO*)out, rows, D, a)));
  return hipGetLastError();
}

hipError_t dropout_scale(Dt ti, const void* in, Dt to, void* out, int64_t rows, int64_t D, const DropArgs& a,
                         hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (D % 4 != 0) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((rows * (D / 4) + 255) / 256));
  BPT_DT(ti, TI, BPT_DT(to, TO, hipLaunchKernelGGL((dropout_scale_kernel<TI, TO>), grid, dim3(256), 0, s,
                                                   (const TI*)in, (TO*)out, rows, D, a)));
  return hipGetLastError();
}

}  // namespace bpt

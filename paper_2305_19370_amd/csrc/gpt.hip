// Kernels of a GPT training step around the layer (the models of Section 5): the
// token + position embedding and its gradients, an elementwise conversion to fp32,
// and the AdamW update. All are HBM-bound streams: every element is read once and
// written once, 16-byte accesses where the layout allows.
#include "common.h"
#include "internal.h"

namespace bpt {

namespace {

// 8 consecutive elements as floats (16-byte loads for bf16, 2 x 16 for fp32)
BPT_DEV void ld8(const float* p, float v[8]) {
  const f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 4);
#pragma unroll
  for (int e = 0; e < 4; ++e) { v[e] = a[e]; v[4 + e] = b[e]; }
}
BPT_DEV void ld8(const bf16* p, float v[8]) {
  const bf16x8 x = *(const bf16x8*)p;
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (float)x[e];
}
BPT_DEV void st8(float* p, const float v[8]) {
  *(f32x4*)p = f32x4{v[0], v[1], v[2], v[3]};
  *(f32x4*)(p + 4) = f32x4{v[4], v[5], v[6], v[7]};
}
BPT_DEV void st8(bf16* p, const float v[8]) {
  bf16x8 x;
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = (bf16)v[e];
  *(bf16x8*)p = x;
}

}  // namespace

// X[t] = Wte[tok[t]] + Wpe[t mod S]: one wave per token row, 8 columns per lane and
// step; the sum is formed in fp32 and rounded once. NaN row for a token outside [0, V).
template <typename T>
__global__ __launch_bounds__(256) void embed_fwd_kernel(const int32_t* tok, const T* Wte, const T* Wpe, T* X,
                                                        int64_t rows, int64_t S, int64_t D, int64_t V) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= rows) return;
  const int64_t y = tok[t];
  const bool ok = y >= 0 && y < V;
  const T* er = Wte + (ok ? y : 0) * D;
  const T* pr = Wpe ? Wpe + (t % S) * D : nullptr;
  for (int64_t d = 8 * lane; d < D; d += 512) {
    float a[8], b[8];
    ld8(er + d, a);
    if (pr) {
      ld8(pr + d, b);
#pragma unroll
      for (int e = 0; e < 8; ++e) a[e] += b[e];
    }
    if (!ok) {
#pragma unroll
      for (int e = 0; e < 8; ++e) a[e] = __builtin_nanf("");
    }
    st8(X + t * D + d, a);
  }
}

// dWte[tok[t]] += dX[t] with fp32 atomics (dWte cleared beforehand): one wave per row.
template <typename T>
__global__ __launch_bounds__(256) void embed_dwte_kernel(const int32_t* tok, const T* dX, float* dWte,
                                                         int64_t rows, int64_t D, int64_t V) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= rows) return;
  const int64_t y = tok[t];
  if (y < 0 || y >= V) return;
  float* out = dWte + y * D;
  for (int64_t d = 8 * lane; d < D; d += 512) {
    float g[8];
    ld8(dX + t * D + d, g);
#pragma unroll
    for (int e = 0; e < 8; ++e) unsafeAtomicAdd(out + d + e, g[e]);
  }
}

// dWpe[s] = sum_b dX[b S + s], summed in batch order: 8 columns per thread.
template <typename T>
__global__ __launch_bounds__(256) void embed_dwpe_kernel(const T* dX, float* dWpe, int64_t B, int64_t S,
                                                         int64_t D) {
  const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
  if (i >= S * D) return;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int64_t b = 0; b < B; ++b) {
    float g[8];
    ld8(dX + b * S * D + i, g);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += g[e];
  }
  st8(dWpe + i, acc);
}

// out[i] = (float)in[i], 8 elements per thread (n a multiple of 8)
__global__ __launch_bounds__(256) void bf16_to_f32_kernel(const bf16* in, float* out, int64_t n) {
  const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
  if (i >= n) return;
  float v[8];
  ld8(in + i, v);
  st8(out + i, v);
}

// One AdamW step. c1 = 1/(1 - beta1^t), c2 = 1/(1 - beta2^t) (formed in double on the
// host). Four elements per thread with 16-byte accesses; the last n mod 4 elements
// one by one. Grid-stride over the groups of four.
template <typename TL>
__global__ __launch_bounds__(256) void adamw_kernel(float* p, const float* g, float* m, float* v, TL* pl,
                                                    int64_t n, float lr, float b1, float b2, float eps,
                                                    float wd, float c1, float c2) {
  const float decay = 1.0f - lr * wd;
  auto one = [&](float& pp, float gg, float& mm, float& vv) {
    mm = b1 * mm + (1.0f - b1) * gg;
    vv = b2 * vv + (1.0f - b2) * gg * gg;
    pp = pp * decay - lr * (mm * c1) / (sqrtf(vv * c2) + eps);
  };
  const int64_t n4 = n / 4;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < n4; q += stride) {
    f32x4 pp = ((const f32x4*)p)[q], mm = ((const f32x4*)m)[q], vv = ((const f32x4*)v)[q];
    const f32x4 gg = ((const f32x4*)g)[q];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float a = pp[e], b = mm[e], c = vv[e];
      one(a, gg[e], b, c);
      pp[e] = a; mm[e] = b; vv[e] = c;
    }
    ((f32x4*)p)[q] = pp;
    ((f32x4*)m)[q] = mm;
    ((f32x4*)v)[q] = vv;
    if (pl) {
      if constexpr (sizeof(TL) == 2) {
        bf16x4 x;
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = (bf16)pp[e];
        ((bf16x4*)pl)[q] = x;
      } else {
        ((f32x4*)pl)[q] = pp;
      }
    }
  }
  if (blockIdx.x == 0 && threadIdx.x < (unsigned)(n - 4 * n4)) {
    const int64_t i = 4 * n4 + threadIdx.x;
    float a = p[i], b = m[i], c = v[i];
    one(a, g[i], b, c);
    p[i] = a; m[i] = b; v[i] = c;
    if (pl) pl[i] = (TL)a;
  }
}

// ------------------------------------------------------------------ launchers
hipError_t embed_fwd(Dt t, const int32_t* tok, const void* Wte, const void* Wpe, void* X, int64_t rows,
                     int64_t S, int64_t D, int64_t V, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const dim3 grid((unsigned)((rows + 3) / 4));
  if (t == F32)
    hipLaunchKernelGGL(embed_fwd_kernel<float>, grid, dim3(256), 0, s, tok, (const float*)Wte,
                       (const float*)Wpe, (float*)X, rows, S, D, V);
  else
    hipLaunchKernelGGL(embed_fwd_kernel<bf16>, grid, dim3(256), 0, s, tok, (const bf16*)Wte,
                       (const bf16*)Wpe, (bf16*)X, rows, S, D, V);
  return hipGetLastError();
}

hipError_t embed_dwte(Dt t, const int32_t* tok, const void* dX, float* dWte, int64_t rows, int64_t D, int64_t V,
                      hipStream_t s) {
  hipError_t e = fill_zero(dWte, V * D * 4, s);
  if (e != hipSuccess || rows <= 0) return e;
  const dim3 grid((unsigned)((rows + 3) / 4));
  if (t == F32)
    hipLaunchKernelGGL(embed_dwte_kernel<float>, grid, dim3(256), 0, s, tok, (const float*)dX, dWte, rows, D, V);
  else
    hipLaunchKernelGGL(embed_dwte_kernel<bf16>, grid, dim3(256), 0, s, tok, (const bf16*)dX, dWte, rows, D, V);
  return hipGetLastError();
}

hipError_t embed_dwpe(Dt t, const void* dX, float* dWpe, int64_t B, int64_t S, int64_t D, hipStream_t s) {
  const int64_t n8 = S * D / 8;
  if (n8 <= 0) return hipSuccess;
  const dim3 grid((unsigned)((n8 + 255) / 256));
  if (t == F32)
    hipLaunchKernelGGL(embed_dwpe_kernel<float>, grid, dim3(256), 0, s, (const float*)dX, dWpe, B, S, D);
  else
    hipLaunchKernelGGL(embed_dwpe_kernel<bf16>, grid, dim3(256), 0, s, (const bf16*)dX, dWpe, B, S, D);
  return hipGetLastError();
}

hipError_t bf16_to_f32(const void* in, float* out, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n % 8 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(bf16_to_f32_kernel, dim3((unsigned)((n / 8 + 255) / 256)), dim3(256), 0, s,
                     (const bf16*)in, out, n);
  return hipGetLastError();
}

hipError_t adamw(Dt tl, float* p, const float* g, float* m, float* v, void* pl, int64_t n, float lr, float b1,
                 float b2, float eps, float wd, float c1, float c2, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t groups = (n + 3) / 4;
  const unsigned grid = (unsigned)std::min<int64_t>((groups + 255) / 256, 8192);
  if (tl == F32)
    hipLaunchKernelGGL(adamw_kernel<float>, dim3(grid), dim3(256), 0, s, p, g, m, v, (float*)pl, n, lr, b1, b2,
                       eps, wd, c1, c2);
  else
    hipLaunchKernelGGL(adamw_kernel<bf16>, dim3(grid), dim3(256), 0, s, p, g, m, v, (bf16*)pl, n, lr, b1, b2,
                       eps, wd, c1, c2);
  return hipGetLastError();
}

}  // namespace bpt

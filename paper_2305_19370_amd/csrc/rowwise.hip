// Row-wise and layout kernels of the BPT layer: LayerNorm forward / backward and
// its parameter gradients, bias gradients (row / column sums), the softmax
// backward's per-row Delta = rowsum(dO * O), transposes into the feature-major
// layouts the MFMA kernels read, and a strided copy. All are HBM-bound; each
// reads and writes every element once (LayerNorm re-reads its row from cache).
#include "common.h"
#include "internal.h"

namespace bpt {

template <typename T> struct Vec4;
template <> struct Vec4<float> {
  static BPT_DEV void load(const float* p, float v[4]) {
    const f32x4 x = *(const f32x4*)p;
    v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
  }
  static BPT_DEV void store(float* p, const float v[4]) { *(f32x4*)p = f32x4{v[0], v[1], v[2], v[3]}; }
};
template <> struct Vec4<bf16> {
  static BPT_DEV void load(const bf16* p, float v[4]) {
    const bf16x4 x = *(const bf16x4*)p;
    v[0] = (float)x[0]; v[1] = (float)x[1]; v[2] = (float)x[2]; v[3] = (float)x[3];
  }
  static BPT_DEV void store(bf16* p, const float v[4]) {
    bf16x4 x;
    x[0] = (bf16)v[0]; x[1] = (bf16)v[1]; x[2] = (bf16)v[2]; x[3] = (bf16)v[3];
    *(bf16x4*)p = x;
  }
};

// 8 consecutive elements <-> 8 floats, with 16-byte accesses
template <typename T> struct Vec8;
template <> struct Vec8<float> {
  static BPT_DEV void load(const float* p, float v[8]) {
    const f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 4);
    v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3]; v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
  }
  static BPT_DEV void store(float* p, const float v[8]) {
    *(f32x4*)p = f32x4{v[0], v[1], v[2], v[3]};
    *(f32x4*)(p + 4) = f32x4{v[4], v[5], v[6], v[7]};
  }
};
template <> struct Vec8<bf16> {
  static BPT_DEV void load(const bf16* p, float v[8]) {
    const bf16x8 x = *(const bf16x8*)p;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (float)x[e];
  }
  static BPT_DEV void store(bf16* p, const float v[8]) {
    bf16x8 x;
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = (bf16)v[e];
    *(bf16x8*)p = x;
  }
};

// ------------------------------------------------------------------ LayerNorm forward
// Rows of D = 512 NC: one wave per row holds the whole row in registers (NC chunks of 8
// consecutive elements per lane, chunk c of lane l at columns 8 (l + 64 c)), so every
// element is read once and written once. Two-pass mean / variance over the registers.
template <typename TI, typename TO, int NC>
__global__ __launch_bounds__(256) void ln_fwd_reg_kernel(const TI* x, int64_t ldx, const float* g,
                                                         const float* bb, TO* out, int64_t ldo, float* mu,
                                                         float* rstd, int64_t rows, float eps, int use_stats) {
  constexpr int D = 512 * NC;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const TI* xr = x + row * ldx;
  float v[NC][8];
#pragma unroll
  for (int c = 0; c < NC; ++c) Vec8<TI>::load(xr + 8 * (lane + 64 * c), v[c]);
  float mean, rs;
  if (!use_stats) {
    float sm = 0.0f;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int e = 0; e < 8; ++e) sm += v[c][e];
    mean = warp_sum(sm) / (float)D;
    float q = 0.0f;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int e = 0; e < 8; ++e) q = fmaf(v[c][e] - mean, v[c][e] - mean, q);
    rs = 1.0f / sqrtf(warp_sum(q) / (float)D + eps);
    if (lane == 0) {
      mu[row] = mean;
      rstd[row] = rs;
    }
  } else {
    mean = mu[row];
    rs = rstd[row];
  }
  TO* orow = out + row * ldo;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int d = 8 * (lane + 64 * c);
    float gv[8], bv[8];
    if (g) Vec8<float>::load(g + d, gv);
    if (bb) Vec8<float>::load(bb + d, bv);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float y = (v[c][e] - mean) * rs;
      if (g) y *= gv[e];
      if (bb) y += bv[e];
      v[c][e] = y;
    }
    Vec8<TO>::store(orow + d, v[c]);
  }
}

// Any D (a multiple of 4): one wave per row; each lane walks groups of 4 columns and
// re-reads the row (from cache) for the variance and the output. Two-pass mean / variance.
template <typename TI, typename TO>
__global__ __launch_bounds__(256) void ln_fwd_kernel(const TI* x, int64_t ldx, const float* g,
                                                     const float* bb, TO* out, int64_t ldo, float* mu,
                                                     float* rstd, int64_t rows, int64_t D, float eps,
                                                     int use_stats) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const TI* xr = x + row * ldx;
  float mean, rs;
  if (!use_stats) {
    float s = 0.0f;
    for (int64_t d = 4 * lane; d < D; d += 256) {
      float v[4];
      Vec4<TI>::load(xr + d, v);
      s += (v[0] + v[1]) + (v[2] + v[3]);
    }
    mean = warp_sum(s) / (float)D;
    float q = 0.0f;
    for (int64_t d = 4 * lane; d < D; d += 256) {
      float v[4];
      Vec4<TI>::load(xr + d, v);
#pragma unroll
      for (int e = 0; e < 4; ++e) q = fmaf(v[e] - mean, v[e] - mean, q);
    }
    const float var = warp_sum(q) / (float)D;
    rs = 1.0f / sqrtf(var + eps);
    if (lane == 0) {
      mu[row] = mean;
      rstd[row] = rs;
    }
  } else {
    mean = mu[row];
    rs = rstd[row];
  }
  TO* orow = out + row * ldo;
  for (int64_t d = 4 * lane; d < D; d += 256) {
    float v[4];
    Vec4<TI>::load(xr + d, v);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float y = (v[e] - mean) * rs;
      if (g) y *= g[d + e];
      if (bb) y += bb[d + e];
      v[e] = y;
    }
    Vec4<TO>::store(orow + d, v);
  }
}

// ------------------------------------------------------------------ LayerNorm backward
// dz = rstd * (gd - mean(gd) - xhat * mean(gd * xhat)), gd = dout * gamma; out = resid + dz.
// Rows of D = 512 NC, row of x and of dout held in registers as in ln_fwd_reg_kernel.
template <typename TI, typename TR, typename TO, typename T2, int NC>
__global__ __launch_bounds__(256) void ln_bwd_reg_kernel(const TI* x, const float* mu, const float* rstd,
                                                         const float* g, const float* dout, const TR* resid,
                                                         TO* out, T2* out2, int64_t rows) {
  constexpr int D = 512 * NC;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const float m = mu[row], rs = rstd[row];
  float xh[NC][8], gd[NC][8];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int d = 8 * (lane + 64 * c);
    Vec8<TI>::load(x + row * D + d, xh[c]);
    Vec8<float>::load(dout + row * D + d, gd[c]);
  }
  float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    float gv[8];
    if (g) Vec8<float>::load(g + 8 * (lane + 64 * c), gv);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (g) gd[c][e] *= gv[e];
      xh[c][e] = (xh[c][e] - m) * rs;
      s1 += gd[c][e];
      s2 = fmaf(gd[c][e], xh[c][e], s2);
    }
  }
  s1 = warp_sum(s1) / (float)D;
  s2 = warp_sum(s2) / (float)D;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int d = 8 * (lane + 64 * c);
    float rv[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (resid) Vec8<TR>::load(resid + row * D + d, rv);
#pragma unroll
    for (int e = 0; e < 8; ++e) rv[e] += rs * (gd[c][e] - s1 - xh[c][e] * s2);
    Vec8<TO>::store(out + row * D + d, rv);
    if (out2) Vec8<T2>::store(out2 + row * D + d, rv);
  }
}

// Any D (a multiple of 4).
template <typename TI, typename TR, typename TO, typename T2>
__global__ __launch_bounds__(256) void ln_bwd_kernel(const TI* x, const float* mu, const float* rstd,
                                                     const float* g, const float* dout, const TR* resid,
                                                     TO* out, T2* out2, int64_t rows, int64_t D) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const TI* xr = x + row * D;
  const float* dr = dout + row * D;
  const float m = mu[row], rs = rstd[row];
  float s1 = 0.0f, s2 = 0.0f;
  for (int64_t d = 4 * lane; d < D; d += 256) {
    float xv[4], dv[4];
    Vec4<TI>::load(xr + d, xv);
    Vec4<float>::load(dr + d, dv);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float gd = g ? dv[e] * g[d + e] : dv[e];
      s1 += gd;
      s2 = fmaf(gd, (xv[e] - m) * rs, s2);
    }
  }
  s1 = warp_sum(s1) / (float)D;
  s2 = warp_sum(s2) / (float)D;
  for (int64_t d = 4 * lane; d < D; d += 256) {
    float xv[4], dv[4], rv[4] = {0, 0, 0, 0};
    Vec4<TI>::load(xr + d, xv);
    Vec4<float>::load(dr + d, dv);
    if (resid) Vec4<TR>::load(resid + row * D + d, rv);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float gd = g ? dv[e] * g[d + e] : dv[e];
      const float xh = (xv[e] - m) * rs;
      rv[e] += rs * (gd - s1 - xh * s2);
    }
    Vec4<TO>::store(out + row * D + d, rv);
    if (out2) Vec4<T2>::store(out2 + row * D + d, rv);
  }
}

// ------------------------------------------------------------------ column / row sums
static constexpr int kChunks = 128;

template <typename TI>
__global__ __launch_bounds__(256) void ln_param_partial_kernel(const TI* x, const float* mu,
                                                               const float* rstd, const float* dout,
                                                               float* partial, int64_t rows, int64_t D) {
  const int64_t d = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (d >= D) return;
  const int64_t per = (rows + kChunks - 1) / kChunks;
  const int64_t r0 = blockIdx.y * per, r1 = r0 + per < rows ? r0 + per : rows;
  float sg = 0.0f, sb = 0.0f;
  for (int64_t r = r0; r < r1; ++r) {
    const float dv = dout[r * D + d];
    sg = fmaf(dv, (to_f32<TI>(x[r * D + d]) - mu[r]) * rstd[r], sg);
    sb += dv;
  }
  partial[(int64_t)blockIdx.y * D + d] = sg;
  partial[(int64_t)(kChunks + blockIdx.y) * D + d] = sb;
}

// Second stage: out0[d] (+)= sum_c partial[c D + d] and out1[d] (+)= sum_c partial[(kChunks + c) D + d].
// A block of four waves per 64 columns; wave w sums chunks w, w + 4, ... (eight loads in flight
// per lane) and the four wave sums are added through LDS in wave order.
__global__ __launch_bounds__(256) void chunk_reduce_kernel(const float* partial, float* out0,
                                                           float* out1, int64_t D, int accumulate) {
  __shared__ float red[2][4][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t d = (int64_t)blockIdx.x * 64 + lane;
  const bool ok = d < D;
  float s0 = 0.0f, s1 = 0.0f;
  if (ok) {
    for (int c0 = wv; c0 < kChunks; c0 += 32) {
      float v0[8], v1[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int c = c0 + 4 * u;
        v0[u] = c < kChunks ? partial[(int64_t)c * D + d] : 0.0f;
        v1[u] = (out1 && c < kChunks) ? partial[(int64_t)(kChunks + c) * D + d] : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) { s0 += v0[u]; s1 += v1[u]; }
    }
  }
  red[0][wv][lane] = s0;
  red[1][wv][lane] = s1;
  __syncthreads();
  if (wv == 0 && ok) {
    s0 = ((red[0][0][lane] + red[0][1][lane]) + red[0][2][lane]) + red[0][3][lane];
    s1 = ((red[1][0][lane] + red[1][1][lane]) + red[1][2][lane]) + red[1][3][lane];
    if (out0) out0[d] = accumulate ? out0[d] + s0 : s0;
    if (out1) out1[d] = accumulate ? out1[d] + s1 : s1;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void col_partial_kernel(const T* in, int64_t ld, int64_t rows,
                                                          int64_t cols, float* partial) {
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= cols) return;
  const int64_t per = (rows + kChunks - 1) / kChunks;
  const int64_t r0 = blockIdx.y * per, r1 = r0 + per < rows ? r0 + per : rows;
  float s = 0.0f;
  for (int64_t r = r0; r < r1; ++r) s += to_f32<T>(in[r * ld + c]);
  partial[(int64_t)blockIdx.y * cols + c] = s;
}

// Wide forms of the two partial-sum kernels for 8-column-aligned rows: one wave per
// (512-column group, row chunk), 8 consecutive columns per lane with 16-byte loads, rows
// unrolled by four so that several loads are in flight per lane.
template <typename T>
__global__ __launch_bounds__(64) void col_partial8_kernel(const T* in, int64_t ld, int64_t rows, int64_t cols,
                                                          float* partial) {
  const int64_t c = ((int64_t)blockIdx.x * 64 + threadIdx.x) * 8;
  if (c >= cols) return;
  const int64_t per = (rows + kChunks - 1) / kChunks;
  const int64_t r0 = blockIdx.y * per, r1 = r0 + per < rows ? r0 + per : rows;
  float s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  int64_t r = r0;
  for (; r + 4 <= r1; r += 4) {
    float v[4][8];
#pragma unroll
    for (int u = 0; u < 4; ++u) Vec8<T>::load(in + (r + u) * ld + c, v[u]);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int e = 0; e < 8; ++e) s[e] += v[u][e];
  }
  for (; r < r1; ++r) {
    float v[8];
    Vec8<T>::load(in + r * ld + c, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] += v[e];
  }
  Vec8<float>::store(partial + (int64_t)blockIdx.y * cols + c, s);
}

// LayerNorm parameter partials, wide form: a block of four waves per (512-column group, row
// chunk); wave w sums the w-th quarter of the chunk's rows (8 columns per lane, 16-byte
// loads, two rows in flight), and the four quarter sums are added through LDS in wave order.
template <typename TI>
__global__ __launch_bounds__(256) void ln_param_partial8_kernel(const TI* x, const float* mu, const float* rstd,
                                                                const float* dout, float* partial, int64_t rows,
                                                                int64_t D) {
  __shared__ float red[2][4][64 * 8];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t d = ((int64_t)blockIdx.x * 64 + lane) * 8;
  const bool ok = d < D;
  const int64_t per = (rows + kChunks - 1) / kChunks;
  const int64_t c0 = blockIdx.y * per, c1 = c0 + per < rows ? c0 + per : rows;
  const int64_t q = (per + 3) / 4;
  const int64_t r0 = c0 + wv * q, r1 = r0 + q < c1 ? r0 + q : c1;
  float sg[8] = {0, 0, 0, 0, 0, 0, 0, 0}, sb[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  if (ok) {
    int64_t r = r0;
    for (; r + 2 <= r1; r += 2) {
      float xv[2][8], dv[2][8];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        Vec8<TI>::load(x + (r + u) * D + d, xv[u]);
        Vec8<float>::load(dout + (r + u) * D + d, dv[u]);
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const float m = mu[r + u], rs = rstd[r + u];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          sg[e] = fmaf(dv[u][e], (xv[u][e] - m) * rs, sg[e]);
          sb[e] += dv[u][e];
        }
      }
    }
    for (; r < r1; ++r) {
      float xv[8], dv[8];
      Vec8<TI>::load(x + r * D + d, xv);
      Vec8<float>::load(dout + r * D + d, dv);
      const float m = mu[r], rs = rstd[r];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sg[e] = fmaf(dv[e], (xv[e] - m) * rs, sg[e]);
        sb[e] += dv[e];
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    red[0][wv][lane * 8 + e] = sg[e];
    red[1][wv][lane * 8 + e] = sb[e];
  }
  __syncthreads();
  if (wv == 0 && ok) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      sg[e] = ((red[0][0][lane * 8 + e] + red[0][1][lane * 8 + e]) + red[0][2][lane * 8 + e]) + red[0][3][lane * 8 + e];
      sb[e] = ((red[1][0][lane * 8 + e] + red[1][1][lane * 8 + e]) + red[1][2][lane * 8 + e]) + red[1][3][lane * 8 + e];
    }
    Vec8<float>::store(partial + (int64_t)blockIdx.y * D + d, sg);
    Vec8<float>::store(partial + (int64_t)(kChunks + blockIdx.y) * D + d, sb);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void row_sum_kernel(const T* in, int64_t ld, int64_t rows, int64_t cols,
                                                      float* out, int accumulate) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  float s = 0.0f;
  for (int64_t c = lane; c < cols; c += 64) s += to_f32<T>(in[row * ld + c]);
  s = warp_sum(s);
  if (lane == 0) out[row] = accumulate ? out[row] + s : s;
}

// The same for 16-byte-aligned rows (ld a multiple of 8): each lane adds 8 consecutive
// columns per 16-byte load, with four loads in flight per lane; a scalar pass adds the
// columns past the last whole group of 8.
template <typename T>
__global__ __launch_bounds__(256) void row_sum8_kernel(const T* in, int64_t ld, int64_t rows, int64_t cols,
                                                       float* out, int accumulate) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const T* r = in + row * ld;
  const int64_t c8 = cols & ~(int64_t)7;
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  int64_t c = 8 * lane;
  for (; c + 3 * 512 < c8; c += 4 * 512) {
    float v[4][8];
#pragma unroll
    for (int u = 0; u < 4; ++u) Vec8<T>::load(r + c + 512 * u, v[u]);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[u] += v[u][e];
  }
  for (; c < c8; c += 512) {
    float v[8];
    Vec8<T>::load(r + c, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[0] += v[e];
  }
  float s = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  for (int64_t t = c8 + lane; t < cols; t += 64) s += to_f32<T>(r[t]);
  s = warp_sum(s);
  if (lane == 0) out[row] = accumulate ? out[row] + s : s;
}

// ------------------------------------------------------------------ softmax-backward Delta
// One wave per token (b, s): Delta[b, h, s] = sum_d dO[t, h*dh + d] O[t, h*dh + d] for every
// head, from 16-byte loads of the token's two rows; the lanes of one head reduce by
// shuffles; stored negated (the backward kernels start dP from -Delta). Also
// nlse2 = -lse * log2(e), the negated base-2 log-sum-exp. Padding tokens s in [S, Sp) get
// zeros.
template <typename T>
__global__ __launch_bounds__(256) void delta_kernel(const T* dO, const T* O, int64_t ld, const float* lse,
                                                    float* ndelta, float* nlse2, int B, int64_t S, int64_t Sp,
                                                    int H, int dh) {
  constexpr int EPL = 16 / sizeof(T);                // elements per lane and load
  const int lane = threadIdx.x & 63;
  const int64_t tok = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);   // over B * Sp
  if (tok >= (int64_t)B * Sp) return;
  const int b = (int)(tok / Sp);
  const int64_t s = tok % Sp;
  const int D = H * dh, lpg = dh / EPL;             // lanes per head in one load step
  for (int e0 = 0; e0 < D; e0 += 64 * EPL) {
    const int e = e0 + lane * EPL;                  // the lanes of one head are all in or all out
    float acc = 0.0f;
    if (s < S && e < D) {
      const int64_t off = ((int64_t)b * S + s) * ld + e;
      float x[EPL], y[EPL];
#pragma unroll
      for (int k = 0; k < EPL; k += 4) {
        Vec4<T>::load(dO + off + k, x + k);
        Vec4<T>::load(O + off + k, y + k);
      }
#pragma unroll
      for (int k = 0; k < EPL; ++k) acc = fmaf(x[k], y[k], acc);
    }
    for (int o = lpg / 2; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if (lane % lpg == 0 && e < D) {
      const int h = e / dh;
      const int64_t i = ((int64_t)b * H + h) * Sp + s;
      ndelta[i] = -acc;
      nlse2[i] = s < S ? -lse[i] * 1.4426950408889634f : 0.0f;
    }
  }
}

// ------------------------------------------------------------------ transpose / copy
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* in, int64_t ld_in, int64_t s_in, T* out,
                                                        int64_t ld_out, int64_t s_out, int64_t rows,
                                                        int64_t cols, int64_t rows_store) {
  __shared__ T tile[64][65];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int64_t r0 = (int64_t)blockIdx.x * 64, c0 = (int64_t)blockIdx.y * 64;   // rows on x: no 65535 limit
  in += (int64_t)blockIdx.z * s_in;
  out += (int64_t)blockIdx.z * s_out;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int64_t r = r0 + ty + 4 * i, c = c0 + tx;
    tile[ty + 4 * i][tx] = (r < rows && c < cols) ? in[r * ld_in + c] : from_f32<T>(0.0f);
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int64_t c = c0 + ty + 4 * i, r = r0 + tx;
    if (c < cols && r < rows_store) out[c * ld_out + r] = tile[tx][ty + 4 * i];
  }
}

template <typename T>
__global__ __launch_bounds__(256) void copy2d_kernel(const T* in, int64_t ld_in, T* out, int64_t ld_out,
                                                     int64_t cols) {   // one row per grid row
  const int64_t r = blockIdx.y;
  for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < cols; c += (int64_t)gridDim.x * 256)
    out[r * ld_out + c] = in[r * ld_in + c];
}

// The same with 16-byte copies, for rows whose strides, width and base are multiples of 16
// bytes.
__global__ __launch_bounds__(256) void copy2d16_kernel(const u32x4* in, int64_t ld_in, u32x4* out, int64_t ld_out,
                                                       int64_t cols) {   // strides and cols in 16-byte units
  const int64_t r = blockIdx.y;
  for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < cols; c += (int64_t)gridDim.x * 256)
    out[r * ld_out + c] = in[r * ld_in + c];
}

// ------------------------------------------------------------------ host launchers

// ------------------------------------------------------------------ cross-entropy rows
// (m, l) summarises exp over a set of logits as l * exp(m); two summaries combine
// exactly. m = -inf, l = 0 is the empty set.
BPT_DEV void lse_merge(float& m, float& l, float m2, float l2) {
  const float mm = fmaxf(m, m2);
  if (mm == -__builtin_inff()) return;
  l = l * __expf(m - mm) + l2 * __expf(m2 - mm);
  m = mm;
}

// One workgroup per row t of a block of logits z (fp32, row stride ld, 16-byte aligned
// rows): each thread summarises its columns of [0, V) online, the summaries combine by
// shuffles and through LDS, and thread 0 writes lse[t] = m + log l and the token loss
// lse[t] - z[t, y_t], or NaN when the target is outside [0, V).
__global__ __launch_bounds__(256) void xent_rows_kernel(const float* z, int64_t ld, int64_t V,
                                                        const int32_t* tgt, float* lse, float* tok) {
  const int64_t t = blockIdx.x;
  const float* zr = z + t * ld;
  const int tid = threadIdx.x;
  float m = -__builtin_inff(), l = 0.0f;
  for (int64_t v = 4 * (int64_t)tid; v < V; v += 4 * 256) {
    float x[4];
    if (v + 4 <= V) {
      const f32x4 q = *(const f32x4*)(zr + v);
      x[0] = q[0]; x[1] = q[1]; x[2] = q[2]; x[3] = q[3];
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) x[e] = v + e < V ? zr[v + e] : -__builtin_inff();
    }
    const float mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
    float s = 0.0f;
#pragma unroll
    for (int e = 0; e < 4; ++e) s += __expf(x[e] - mx);
    lse_merge(m, l, mx, s);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float m2 = __shfl_xor(m, o, 64), l2 = __shfl_xor(l, o, 64);
    lse_merge(m, l, m2, l2);
  }
  __shared__ float sm[4], sl[4];
  if ((tid & 63) == 0) {
    sm[tid >> 6] = m;
    sl[tid >> 6] = l;
  }
  __syncthreads();
  if (tid == 0) {
    m = sm[0];
    l = sl[0];
    for (int w = 1; w < 4; ++w) lse_merge(m, l, sm[w], sl[w]);
    const float r = m + __logf(l);
    lse[t] = r;
    const int y = tgt[t];
    tok[t] = (y >= 0 && y < V) ? r - zr[y] : __builtin_nanf("");
  }
}

// out[0] = (sum of x[0..n)) / n, summed in a fixed order by one workgroup.
__global__ __launch_bounds__(1024) void mean_kernel(const float* x, int64_t n, float* out) {
  __shared__ float part[1024];
  float s = 0.0f;
  for (int64_t i = threadIdx.x; i < n; i += 1024) s += x[i];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 512; w >= 1; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = part[0] / (float)n;
}

__global__ __launch_bounds__(256) void fill_zero_kernel(uint32_t* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = 0u;
}

#define BPT_T(dt, T, ...) \
  do {                   \
    if ((dt) == F32) {   \
      using T = float;   \
      __VA_ARGS__;       \
    } else {             \
      using T = bf16;    \
      __VA_ARGS__;       \
    }                    \
  } while (0)

hipError_t layer_norm(Dt ti, Dt to, const void* x, int64_t ldx, const float* g, const float* b, void* out,
                      int64_t ldo, float* mu, float* rstd, int64_t rows, int64_t D, float eps,
                      int use_stats, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const dim3 grid((unsigned)((rows + 3) / 4));
  // register-resident rows when D = 512 NC and every row starts 16-byte aligned
  const bool vec = D % 512 == 0 && ldx % 8 == 0 && ldo % 8 == 0 && ((uintptr_t)x & 15) == 0 &&
                   ((uintptr_t)out & 15) == 0 && ((uintptr_t)g & 15) == 0 && ((uintptr_t)b & 15) == 0;
#define BPT_LN_FWD(NCV)                                                                                  \
  BPT_T(ti, TI, BPT_T(to, TO,                                                                            \
        hipLaunchKernelGGL((ln_fwd_reg_kernel<TI, TO, NCV>), grid, dim3(256), 0, s, (const TI*)x, ldx, g, \
                           b, (TO*)out, ldo, mu, rstd, rows, eps, use_stats)))
  switch (vec ? D / 512 : 0) {
    case 1: BPT_LN_FWD(1); return hipGetLastError();
    case 2: BPT_LN_FWD(2); return hipGetLastError();
    case 4: BPT_LN_FWD(4); return hipGetLastError();
    case 8: BPT_LN_FWD(8); return hipGetLastError();
    case 10: BPT_LN_FWD(10); return hipGetLastError();
    default: break;
  }
#undef BPT_LN_FWD
  BPT_T(ti, TI, BPT_T(to, TO,
        hipLaunchKernelGGL((ln_fwd_kernel<TI, TO>), grid, dim3(256), 0, s, (const TI*)x, ldx, g, b,
                           (TO*)out, ldo, mu, rstd, rows, D, eps, use_stats)));
  return hipGetLastError();
}

hipError_t layer_norm_bwd(Dt ti, const void* x, const float* mu, const float* rstd, const float* g,
                          const float* dout, Dt tr, const void* resid, Dt to, void* out, Dt t2,
                          void* out2, int64_t rows, int64_t D, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const dim3 grid((unsigned)((rows + 3) / 4));
  const bool vec = D % 512 == 0 && ((uintptr_t)x & 15) == 0 && ((uintptr_t)dout & 15) == 0 &&
                   ((uintptr_t)resid & 15) == 0 && ((uintptr_t)out & 15) == 0 && ((uintptr_t)out2 & 15) == 0 &&
                   ((uintptr_t)g & 15) == 0;
#define BPT_LN_BWD(NCV)                                                                                  \
  BPT_T(ti, TI, BPT_T(tr, TR, BPT_T(to, TO, BPT_T(t2, T2,                                               \
        hipLaunchKernelGGL((ln_bwd_reg_kernel<TI, TR, TO, T2, NCV>), grid, dim3(256), 0, s, (const TI*)x, \
                           mu, rstd, g, dout, (const TR*)resid, (TO*)out, (T2*)out2, rows)))))
  switch (vec ? D / 512 : 0) {
    case 1: BPT_LN_BWD(1); return hipGetLastError();
    case 2: BPT_LN_BWD(2); return hipGetLastError();
    case 4: BPT_LN_BWD(4); return hipGetLastError();
    case 8: BPT_LN_BWD(8); return hipGetLastError();
    case 10: BPT_LN_BWD(10); return hipGetLastError();
    default: break;
  }
#undef BPT_LN_BWD
  BPT_T(ti, TI, BPT_T(tr, TR, BPT_T(to, TO, BPT_T(t2, T2,
        hipLaunchKernelGGL((ln_bwd_kernel<TI, TR, TO, T2>), grid, dim3(256), 0, s, (const TI*)x, mu,
                           rstd, g, dout, (const TR*)resid, (TO*)out, (T2*)out2, rows, D)))));
  return hipGetLastError();
}

size_t layer_norm_param_grad_ws(int64_t D) { return (size_t)2 * kChunks * (size_t)D; }

hipError_t layer_norm_param_grad(Dt ti, const void* x, const float* mu, const float* rstd,
                                 const float* dout, float* dgamma, float* dbeta, float* partial,
                                 int64_t rows, int64_t D, hipStream_t s) {
  if (D % 8 == 0 && ((uintptr_t)x & 15) == 0 && ((uintptr_t)dout & 15) == 0 && ((uintptr_t)partial & 15) == 0) {
    const dim3 grid8((unsigned)((D + 511) / 512), kChunks);
    BPT_T(ti, TI, hipLaunchKernelGGL((ln_param_partial8_kernel<TI>), grid8, dim3(256), 0, s, (const TI*)x,
                                     mu, rstd, dout, partial, rows, D));
  } else {
    const dim3 grid((unsigned)((D + 255) / 256), kChunks);
    BPT_T(ti, TI, hipLaunchKernelGGL((ln_param_partial_kernel<TI>), grid, dim3(256), 0, s, (const TI*)x,
                                     mu, rstd, dout, partial, rows, D));
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(chunk_reduce_kernel, dim3((unsigned)((D + 63) / 64)), dim3(256), 0, s, partial,
                     dgamma, dbeta, D, 0);
  return hipGetLastError();
}

hipError_t col_sum(Dt t, const void* in, int64_t ld, int64_t rows, int64_t cols, float* out,
                   int accumulate, float* partial, hipStream_t s) {
  if (cols % 8 == 0 && ld % 8 == 0 && ((uintptr_t)in & 15) == 0 && ((uintptr_t)partial & 15) == 0) {
    const dim3 grid8((unsigned)((cols + 511) / 512), kChunks);
    BPT_T(t, T, hipLaunchKernelGGL((col_partial8_kernel<T>), grid8, dim3(64), 0, s, (const T*)in, ld, rows,
                                   cols, partial));
  } else {
    const dim3 grid((unsigned)((cols + 255) / 256), kChunks);
    BPT_T(t, T, hipLaunchKernelGGL((col_partial_kernel<T>), grid, dim3(256), 0, s, (const T*)in, ld, rows,
                                   cols, partial));
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(chunk_reduce_kernel, dim3((unsigned)((cols + 63) / 64)), dim3(256), 0, s, partial,
                     out, (float*)nullptr, cols, accumulate);
  return hipGetLastError();
}

hipError_t row_sum(Dt t, const void* in, int64_t ld, int64_t rows, int64_t cols, float* out,
                   int accumulate, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const dim3 grid((unsigned)((rows + 3) / 4));
  if (ld % 8 == 0 && ((uintptr_t)in & 15) == 0)
    BPT_T(t, T, hipLaunchKernelGGL((row_sum8_kernel<T>), grid, dim3(256), 0, s, (const T*)in, ld, rows, cols, out,
                                   accumulate));
  else
    BPT_T(t, T, hipLaunchKernelGGL((row_sum_kernel<T>), grid, dim3(256), 0, s, (const T*)in, ld, rows, cols, out,
                                   accumulate));
  return hipGetLastError();
}

hipError_t attn_delta(Dt t, const void* dout, const void* o, int64_t ld, const float* lse, float* ndelta,
                      float* nlse2, int B, int64_t S, int64_t Sp, int H, int dh, hipStream_t s) {
  // one wave per token; a head spans whole 16-byte loads
  const int64_t n = (int64_t)B * Sp;
  if (dh % (t == F32 ? 4 : 8) != 0) return hipErrorInvalidValue;
  BPT_T(t, T, hipLaunchKernelGGL((delta_kernel<T>), dim3((unsigned)((n + 3) / 4)), dim3(256), 0, s,
                                 (const T*)dout, (const T*)o, ld, lse, ndelta, nlse2, B, S, Sp, H, dh));
  return hipGetLastError();
}

hipError_t transpose(Dt t, const void* in, int64_t ld_in, int64_t s_in, void* out, int64_t ld_out,
                     int64_t s_out, int64_t rows, int64_t cols, int64_t rows_store, int batch,
                     hipStream_t s) {
  if (cols <= 0 || rows_store <= 0 || batch <= 0) return hipSuccess;
  const dim3 grid((unsigned)((rows_store + 63) / 64), (unsigned)((cols + 63) / 64), (unsigned)batch);
  BPT_T(t, T, hipLaunchKernelGGL((transpose_kernel<T>), grid, dim3(256), 0, s, (const T*)in, ld_in, s_in,
                                 (T*)out, ld_out, s_out, rows, cols, rows_store));
  return hipGetLastError();
}

hipError_t copy2d(Dt t, const void* in, int64_t ld_in, void* out, int64_t ld_out, int64_t rows,
                  int64_t cols, hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  const int64_t per16 = 16 / (t == F32 ? 4 : 2);   // elements per 16 bytes
  if (ld_in % per16 == 0 && ld_out % per16 == 0 && cols % per16 == 0 && ((uintptr_t)in & 15) == 0 &&
      ((uintptr_t)out & 15) == 0) {
    const int64_t c16 = cols / per16;
    const unsigned gx = (unsigned)((c16 + 255) / 256 < 64 ? (c16 + 255) / 256 : 64);
    hipLaunchKernelGGL(copy2d16_kernel, dim3(gx, (unsigned)rows), dim3(256), 0, s, (const u32x4*)in,
                       ld_in / per16, (u32x4*)out, ld_out / per16, c16);
    return hipGetLastError();
  }
  const unsigned gx = (unsigned)((cols + 255) / 256 < 64 ? (cols + 255) / 256 : 64);
  BPT_T(t, T, hipLaunchKernelGGL((copy2d_kernel<T>), dim3(gx, (unsigned)rows), dim3(256), 0, s,
                                 (const T*)in, ld_in, (T*)out, ld_out, cols));
  return hipGetLastError();
}

hipError_t xent_rows(const float* z, int64_t ld, int64_t rows, int64_t V, const int32_t* tgt, float* lse,
                     float* tok, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (ld % 4 != 0 || ((uintptr_t)z & 15) != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(xent_rows_kernel, dim3((unsigned)rows), dim3(256), 0, s, z, ld, V, tgt, lse, tok);
  return hipGetLastError();
}

hipError_t mean_of(const float* x, int64_t n, float* out, hipStream_t s) {
  if (n <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(1024), 0, s, x, n, out);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void sum_slices_kernel(const float* part, int nz, int64_t n, float* out,
                                                         int accumulate) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;      // group of four
  if (4 * q >= n) return;
  f32x4 acc = accumulate ? ((const f32x4*)out)[q] : f32x4{0, 0, 0, 0};
  for (int z = 0; z < nz; ++z) acc += ((const f32x4*)(part + z * n))[q];
  ((f32x4*)out)[q] = acc;
}

hipError_t sum_slices(const float* part, int nz, int64_t n, float* out, int accumulate, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n % 4 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(sum_slices_kernel, dim3((unsigned)((n / 4 + 255) / 256)), dim3(256), 0, s, part, nz, n, out,
                     accumulate);
  return hipGetLastError();
}

hipError_t fill_zero(void* p, int64_t bytes, hipStream_t s) {
  if (bytes <= 0) return hipSuccess;
  if (bytes % 4 != 0) return hipErrorInvalidValue;
  const int64_t n = bytes / 4;
  const unsigned g = (unsigned)((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(g), dim3(256), 0, s, (uint32_t*)p, n);
  return hipGetLastError();
}

}  // namespace bpt

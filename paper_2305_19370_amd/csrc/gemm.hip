// GEMM family for the BPT layer: C[M,N] = A[M,K] * B[N,K]^T with fused epilogues.
//
// Every dense contraction of the layer (QKV / output projections, both FFN
// linears and all their weight / input gradients) is issued in this one "NT"
// form, with both operands contiguous along K; the host arranges layouts
// (pre-transposed weights, feature-major activations) so that no kernel ever
// needs a strided operand read.
//
// bf16 path: gfx950 MFMA v_mfma_f32_32x32x16_bf16, fp32 accumulation, 256 threads
// (2 x 2 waves), K step 64 staged through double-buffered LDS with an XOR swizzle
// of 16-byte chunks so that the 32 rows a fragment read touches fall in distinct
// banks. fp32 path: plain VALU FMA tiles (used for the fp32 parity workload).
#include "common.h"
#include "internal.h"

namespace bpt {

template <int EPI, typename CT, typename RT>
BPT_DEV void epi_store(const GemmArgs& a, int64_t z, int64_t m, int64_t n, float v) {
  CT* C = (CT*)a.C + z * a.sC;
  const int64_t idx = m * a.ldc + n;
  if (n >= a.N) {                                   // zero padding columns
    C[idx] = from_f32<CT>(0.0f);
    if (EPI == EPI_GELU && a.C2) a.C2[z * a.sC2 + m * a.ldc2 + n] = 0.0f;
    return;
  }
  if constexpr (EPI == EPI_STORE) {
    if constexpr (sizeof(CT) == 4) {
      if (a.accumulate) v += to_f32<CT>(C[idx]);
    }
    C[idx] = from_f32<CT>(v);
  } else if constexpr (EPI == EPI_RESID) {
    const RT* R = (const RT*)a.R + z * a.sR;
    v += to_f32<RT>(R[m * a.ldr + n]);
    if (a.bias) v += a.bias[n];
    C[idx] = from_f32<CT>(v);
  } else if constexpr (EPI == EPI_GELU) {
    if (a.bias) v += a.bias[a.bias_on_m ? m : n];
    C[idx] = from_f32<CT>(gelu_f(v));
    if (a.C2) a.C2[z * a.sC2 + m * a.ldc2 + n] = gelu_grad_f(v);
  } else {  // EPI_MUL
    const float* R = (const float*)a.R + z * a.sR;
    C[idx] = from_f32<CT>(v * R[m * a.ldr + n]);
  }
}

template <typename T> struct V4;
template <> struct V4<float> {
  static BPT_DEV f32x4 ld(const float* p) { return *(const f32x4*)p; }
  static BPT_DEV void st(float* p, f32x4 v) { *(f32x4*)p = v; }
};
template <> struct V4<bf16> {
  static BPT_DEV f32x4 ld(const bf16* p) {
    const bf16x4 x = *(const bf16x4*)p;
    return f32x4{(float)x[0], (float)x[1], (float)x[2], (float)x[3]};
  }
  static BPT_DEV void st(bf16* p, f32x4 v) {
    bf16x4 x;
    x[0] = (bf16)v[0]; x[1] = (bf16)v[1]; x[2] = (bf16)v[2]; x[3] = (bf16)v[3];
    *(bf16x4*)p = x;
  }
};

// Four consecutive columns n..n+3 of row m (n a multiple of 4). Falls back to
// per-element stores when the group crosses N or the stored width.
template <int EPI, typename CT, typename RT>
BPT_DEV void epi_store4(const GemmArgs& a, int64_t z, int64_t m, int64_t n, int64_t ncols, f32x4 v) {
  if (n + 4 > a.N) {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (n + e < ncols) epi_store<EPI, CT, RT>(a, z, m, n + e, v[e]);
    return;
  }
  CT* C = (CT*)a.C + z * a.sC + m * a.ldc + n;
  if constexpr (EPI == EPI_STORE) {
    if constexpr (sizeof(CT) == 4) {
      if (a.accumulate) v += V4<CT>::ld(C);
    }
  } else if constexpr (EPI == EPI_RESID) {
    v += V4<RT>::ld((const RT*)a.R + z * a.sR + m * a.ldr + n);
    if (a.bias) v += *(const f32x4*)(a.bias + n);
  } else if constexpr (EPI == EPI_GELU) {
    if (a.bias) {
      if (a.bias_on_m) v += a.bias[m];
      else v += *(const f32x4*)(a.bias + n);
    }
    if (a.C2) {
      f32x4 d;
#pragma unroll
      for (int e = 0; e < 4; ++e) d[e] = gelu_grad_f(v[e]);
      *(f32x4*)(a.C2 + z * a.sC2 + m * a.ldc2 + n) = d;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = gelu_f(v[e]);
  } else {
    v *= *(const f32x4*)((const float*)a.R + z * a.sR + m * a.ldr + n);
  }
  V4<CT>::st(C, v);
}

// ------------------------------------------------------------------ bf16 MFMA kernel
template <int BM, int BN>
struct TileCfg {
  static constexpr int BK = 64;
  static constexpr int WM = BM / 2, WN = BN / 2;      // wave tile (2 x 2 waves)
  static constexpr int TM = WM / 32, TN = WN / 32;    // 32x32 MFMA tiles per wave
  static constexpr int CA = BM * 8 / 256, CB = BN * 8 / 256;   // 16-byte chunks per thread
  static constexpr int LDS = 2 * (BM + BN) * BK * 2;  // bytes, double buffered
};

// 16-byte chunk `kc` (8 bf16 along K) of tile row `row`, XOR-swizzled by row.
BPT_DEV int swz(int row, int kc) { return row * 128 + ((kc ^ (row & 7)) << 4); }

BPT_DEV u32x4 load_chunk_bf16(const bf16* rowp, int64_t k, int64_t K) {
  if (k + 8 <= K) return *(const u32x4*)(rowp + k);
  union { u32x4 v; uint16_t h[8]; } u;
  const uint16_t* p = (const uint16_t*)rowp;
#pragma unroll
  for (int e = 0; e < 8; ++e) u.h[e] = (k + e < K) ? p[k + e] : (uint16_t)0;
  return u.v;
}

template <int BM, int BN, int EPI, typename CT, typename RT>
__global__ __launch_bounds__(256, 1) void gemm_bf16_kernel(GemmArgs a) {
  using Cfg = TileCfg<BM, BN>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t tiles_m = (a.M + BM - 1) / BM;
  const int64_t tm = blockIdx.x % tiles_m, tn = blockIdx.x / tiles_m;
  const int64_t m0 = tm * BM, n0 = tn * BN, z = blockIdx.z;
  const bf16* A = (const bf16*)a.A + z * a.sA;
  const bf16* B = (const bf16*)a.B + z * a.sB;
  const int64_t K = a.K;
  const int nk = (int)((K + Cfg::BK - 1) / Cfg::BK);

  // stage `buf` holds the A tile (BM rows of 128 bytes) followed by the B tile
  auto As = [&](int buf) { return smem + buf * (BM + BN) * 128; };
  auto Bs = [&](int buf) { return smem + buf * (BM + BN) * 128 + BM * 128; };

  u32x4 ra[Cfg::CA], rb[Cfg::CB];
  auto gload = [&](int kt) {
#pragma unroll
    for (int i = 0; i < Cfg::CA; ++i) {
      const int c = tid + 256 * i, row = c >> 3, kc = c & 7;
      const int64_t m = m0 + row;
      ra[i] = (m < a.M) ? load_chunk_bf16(A + m * a.lda, (int64_t)kt * 64 + kc * 8, K) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int i = 0; i < Cfg::CB; ++i) {
      const int c = tid + 256 * i, row = c >> 3, kc = c & 7;
      const int64_t n = n0 + row;
      rb[i] = (n < a.N) ? load_chunk_bf16(B + n * a.ldb, (int64_t)kt * 64 + kc * 8, K) : u32x4{0, 0, 0, 0};
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < Cfg::CA; ++i) {
      const int c = tid + 256 * i;
      *(u32x4*)(As(buf) + swz(c >> 3, c & 7)) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < Cfg::CB; ++i) {
      const int c = tid + 256 * i;
      *(u32x4*)(Bs(buf) + swz(c >> 3, c & 7)) = rb[i];
    }
  };

  f32x16 acc[Cfg::TM][Cfg::TN];
#pragma unroll
  for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::TN; ++j) acc[i][j] = f32x16{};

  if (nk > 0) {
    gload(0);
    lstore(0);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int kc = kk * 2 + (lane >> 5);
      bf16x8 af[Cfg::TM], bfr[Cfg::TN];
#pragma unroll
      for (int i = 0; i < Cfg::TM; ++i)
        af[i] = *(const bf16x8*)(As(buf) + swz(wm * Cfg::WM + 32 * i + (lane & 31), kc));
#pragma unroll
      for (int j = 0; j < Cfg::TN; ++j)
        bfr[j] = *(const bf16x8*)(Bs(buf) + swz(wn * Cfg::WN + 32 * j + (lane & 31), kc));
#pragma unroll
      for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::TN; ++j) acc[i][j] = mfma32x32x16(af[i], bfr[j], acc[i][j]);
    }
    if (kt + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

  // Epilogue: each wave stages one 32-row strip of its accumulators in LDS (free
  // after the K loop), then every lane applies the epilogue to groups of 4
  // consecutive columns and stores them with one vector store.
  const int64_t ncols = a.Nstore > a.N ? a.Nstore : a.N;
  constexpr int PITCH = Cfg::WN + 4;                 // floats per staged row
  float* strip = (float*)smem + wave * 32 * PITCH;
#pragma unroll
  for (int i = 0; i < Cfg::TM; ++i) {
#pragma unroll
    for (int j = 0; j < Cfg::TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        strip[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * PITCH + 32 * j + (lane & 31)] = acc[i][j][r];
    __syncthreads();
#pragma unroll 1
    for (int e = lane; e < 32 * Cfg::WN / 4; e += 64) {
      const int row = e / (Cfg::WN / 4), c4 = e % (Cfg::WN / 4);
      const int64_t m = m0 + wm * Cfg::WM + 32 * i + row;
      const int64_t n = n0 + wn * Cfg::WN + 4 * c4;
      if (m < a.M && n < ncols) {
        const f32x4 v = *(const f32x4*)(strip + row * PITCH + 4 * c4);
        epi_store4<EPI, CT, RT>(a, z, m, n, ncols, v);
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ fp32 VALU kernel
template <int EPI, typename CT, typename RT>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  __shared__ float As[16][64 + 4], Bs[16][64 + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int64_t tiles_m = (a.M + 63) / 64;
  const int64_t m0 = (blockIdx.x % tiles_m) * 64, n0 = (blockIdx.x / tiles_m) * 64, z = blockIdx.z;
  const float* A = (const float*)a.A + z * a.sA;
  const float* B = (const float*)a.B + z * a.sB;
  float acc[4][4] = {};
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  for (int64_t k0 = 0; k0 < a.K; k0 += 16) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t k = k0 + lk + e;
      As[lk + e][lr] = (m0 + lr < a.M && k < a.K) ? A[(m0 + lr) * a.lda + k] : 0.0f;
      Bs[lk + e][lr] = (n0 + lr < a.N && k < a.K) ? B[(n0 + lr) * a.ldb + k] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
  const int64_t ncols = a.Nstore > a.N ? a.Nstore : a.N;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t m = m0 + ty + 16 * i, n = n0 + tx + 16 * j;
      if (m < a.M && n < ncols) epi_store<EPI, CT, RT>(a, z, m, n, acc[i][j]);
    }
}

// ------------------------------------------------------------------ dispatch
template <int BM, int BN, int EPI, typename CT, typename RT>
static hipError_t launch_bf16(const GemmArgs& a, hipStream_t s) {
  using Cfg = TileCfg<BM, BN>;
  auto kern = gemm_bf16_kernel<BM, BN, EPI, CT, RT>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       Cfg::LDS);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int64_t ncols = a.Nstore > a.N ? a.Nstore : a.N;
  const int64_t tiles = ((a.M + BM - 1) / BM) * ((ncols + BN - 1) / BN);
  if (tiles <= 0 || a.batch <= 0) return hipSuccess;
  hipLaunchKernelGGL(kern, dim3((unsigned)tiles, 1, (unsigned)a.batch), dim3(256), Cfg::LDS, s, a);
  return hipGetLastError();
}

template <int EPI, typename CT, typename RT>
static hipError_t launch_typed(Dt ab, const GemmArgs& a, hipStream_t s) {
  const int64_t ncols = a.Nstore > a.N ? a.Nstore : a.N;
  if (ab == F32) {
    const int64_t tiles = ((a.M + 63) / 64) * ((ncols + 63) / 64);
    if (tiles <= 0 || a.batch <= 0) return hipSuccess;
    hipLaunchKernelGGL((gemm_f32_kernel<EPI, CT, RT>), dim3((unsigned)tiles, 1, (unsigned)a.batch),
                       dim3(256), 0, s, a);
    return hipGetLastError();
  }
  const int64_t big = ((a.M + 255) / 256) * ((ncols + 255) / 256) * a.batch;
  if (big >= 256) return launch_bf16<256, 256, EPI, CT, RT>(a, s);
  return launch_bf16<128, 128, EPI, CT, RT>(a, s);
}

hipError_t gemm(Dt ab, Epi epi, Dt ct, Dt rt, const GemmArgs& a, hipStream_t s) {
  switch (epi) {
    case EPI_STORE:
      return ct == F32 ? launch_typed<EPI_STORE, float, float>(ab, a, s)
                       : launch_typed<EPI_STORE, bf16, float>(ab, a, s);
    case EPI_GELU:
      return ct == F32 ? launch_typed<EPI_GELU, float, float>(ab, a, s)
                       : launch_typed<EPI_GELU, bf16, float>(ab, a, s);
    case EPI_MUL:
      return ct == F32 ? launch_typed<EPI_MUL, float, float>(ab, a, s)
                       : launch_typed<EPI_MUL, bf16, float>(ab, a, s);
    case EPI_RESID:
      if (ct == F32)
        return rt == F32 ? launch_typed<EPI_RESID, float, float>(ab, a, s)
                         : launch_typed<EPI_RESID, float, bf16>(ab, a, s);
      return rt == F32 ? launch_typed<EPI_RESID, bf16, float>(ab, a, s)
                       : launch_typed<EPI_RESID, bf16, bf16>(ab, a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace bpt

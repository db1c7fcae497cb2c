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
// Tile BM x BN (2 x 2 waves), K step 32 per stage, NS stages in an LDS ring filled
// by direct global->LDS copies (global_load_lds_dwordx4) issued NS-1 stages ahead.
// Tile rows are 32 bf16 (64 bytes) padded to 80 bytes, so the 16 rows of a
// fragment read fall in distinct bank groups and every fragment address is a
// per-lane base plus an immediate. K must be a multiple of 32 (host-checked).
template <int BM, int BN>
struct TileCfg {
  static constexpr int BK = 32;
  static constexpr int PITCH = 80, SLOTS = 5;          // bytes / 16-byte slots per tile row
  static constexpr int WM = BM / 2, WN = BN / 2;      // wave tile (2 x 2 waves)
  static constexpr int TM = WM / 32, TN = WN / 32;    // 32x32 MFMA tiles per wave
  static constexpr int ABYTES = BM * PITCH, BBYTES = BN * PITCH;
  static constexpr int ABLK = ABYTES / 1024, BBLK = BBYTES / 1024;    // 1 KB copy blocks
  static constexpr int APW = (ABLK + 3) / 4, BPW = (BBLK + 3) / 4;    // copies per wave
  static constexpr int DPS = APW + BPW;               // copy instructions per wave per stage
  static constexpr int STAGE = ABYTES + BBYTES;
  static constexpr int NS = 4;                        // stages in the ring
  static constexpr int LDS = NS * STAGE;
  static_assert(ABYTES % 1024 == 0 && BBYTES % 1024 == 0, "whole copy blocks");
  static_assert(4 * (WN + 4) * 32 * 4 <= LDS, "epilogue staging fits");
};

// One wave copies 1 KiB from global memory straight into LDS: lane l's 16 bytes land at
// lds_block + 16 l. Written as inline assembly on purpose: the compiler's counter
// tracking treats the builtin form as a pending FLAT access and then turns every later
// LDS-fragment wait into a full drain. Completion is tracked by hand (wait_vmcnt). M0 is
// a reserved register the compiler does not otherwise use in these kernels.
BPT_DEV void lds_dma16(const void* g, char* lds_block) {
  const uint32_t m = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds_block);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(g), "s"(m) : "memory");
}

template <int N> BPT_DEV void wait_vmcnt() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

template <int BM, int BN, int EPI, typename CT, typename RT>
__global__ __launch_bounds__(256, 1) void gemm_bf16_kernel(GemmArgs a) {
  using Cfg = TileCfg<BM, BN>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  // Grouped tile order: 8 consecutive workgroups (one per XCD) take 8 row blocks of
  // the same column block; each XCD thus keeps one row block of A in its L2.
  const int tiles_m = (int)((a.M + BM - 1) / BM);
  const int64_t ncols = a.Nstore > a.N ? a.Nstore : a.N;
  const int tiles_n = (int)((ncols + BN - 1) / BN);
  constexpr int GM = 8;
  const int pid = blockIdx.x;
  const int group = pid / (GM * tiles_n), first_m = group * GM;
  const int gm = tiles_m - first_m < GM ? tiles_m - first_m : GM;
  const int tm = first_m + (pid % (GM * tiles_n)) % gm;
  const int tn = (pid % (GM * tiles_n)) / gm;
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN, z = blockIdx.z;
  const bf16* A = (const bf16*)a.A + z * a.sA + m0 * a.lda;
  const bf16* B = (const bf16*)a.B + z * a.sB + n0 * a.ldb;
  const int nk = (int)(a.K / Cfg::BK);

  // per-lane source offsets (elements) of this wave's copy slots; rows past the
  // matrix edge are clamped to its last row (their results are never stored)
  int aoff[Cfg::APW], boff[Cfg::BPW];
  {
    const int alast = (int)(a.M - 1 - m0), blast = (int)(a.N - 1 - n0);
#pragma unroll
    for (int i = 0; i < Cfg::APW; ++i) {
      int blk = wave + 4 * i;
      blk = blk < Cfg::ABLK ? blk : Cfg::ABLK - 1;     // extra copies repeat the last block
      const int slot = blk * 64 + lane, row = slot / Cfg::SLOTS, col = slot % Cfg::SLOTS;
      aoff[i] = (row < alast ? row : alast) * (int)a.lda + (col < 4 ? col : 0) * 8;
    }
#pragma unroll
    for (int i = 0; i < Cfg::BPW; ++i) {
      int blk = wave + 4 * i;
      blk = blk < Cfg::BBLK ? blk : Cfg::BBLK - 1;
      const int slot = blk * 64 + lane, row = slot / Cfg::SLOTS, col = slot % Cfg::SLOTS;
      boff[i] = (row < blast ? row : blast) * (int)a.ldb + (col < 4 ? col : 0) * 8;
    }
  }
  auto issue = [&](int kt) {
    char* st = smem + (kt % Cfg::NS) * Cfg::STAGE;
    const int k0 = kt * Cfg::BK;
#pragma unroll
    for (int i = 0; i < Cfg::APW; ++i) {
      int blk = wave + 4 * i;
      blk = blk < Cfg::ABLK ? blk : Cfg::ABLK - 1;
      lds_dma16(A + k0 + aoff[i], st + blk * 1024);
    }
#pragma unroll
    for (int i = 0; i < Cfg::BPW; ++i) {
      int blk = wave + 4 * i;
      blk = blk < Cfg::BBLK ? blk : Cfg::BBLK - 1;
      lds_dma16(B + k0 + boff[i], st + Cfg::ABYTES + blk * 1024);
    }
  };

  f32x16 acc[Cfg::TM][Cfg::TN];
#pragma unroll
  for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::TN; ++j) acc[i][j] = f32x16{};

  const int abase = (wm * Cfg::WM + (lane & 31)) * Cfg::PITCH + (lane >> 5) * 16;
  const int bbase = Cfg::ABYTES + (wn * Cfg::WN + (lane & 31)) * Cfg::PITCH + (lane >> 5) * 16;

  // Fragments are double-buffered in registers: the LDS reads of the next k step are
  // issued before the MFMAs of the current one, so their latency hides behind them.
  bf16x8 fa[2][Cfg::TM], fb[2][Cfg::TN];
  auto load_frags = [&](int kt, int kk, int buf) {
    const char* st = smem + (kt % Cfg::NS) * Cfg::STAGE;
#pragma unroll
    for (int i = 0; i < Cfg::TM; ++i) fa[buf][i] = *(const bf16x8*)(st + abase + i * 32 * Cfg::PITCH + kk * 32);
#pragma unroll
    for (int j = 0; j < Cfg::TN; ++j) fb[buf][j] = *(const bf16x8*)(st + bbase + j * 32 * Cfg::PITCH + kk * 32);
  };
  auto mfmas = [&](int buf) {
#pragma unroll
    for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
      for (int j = 0; j < Cfg::TN; ++j) acc[i][j] = mfma32x32x16(fa[buf][i], fb[buf][j], acc[i][j]);
  };

  // stages 0 .. NS-2 in flight; wait for stage 0
#pragma unroll
  for (int s = 0; s < Cfg::NS - 1; ++s)
    if (s < nk) issue(s);
  if (nk >= Cfg::NS - 1) wait_vmcnt<(Cfg::NS - 2) * Cfg::DPS>();
  else wait_vmcnt<0>();
  __syncthreads();
  if (nk > 0) load_frags(0, 0, 0);
  // steady state, branch-free in the LDS reads so that each MFMA group waits only for
  // its own fragments; the last stage is peeled below
  for (int kt = 0; kt + 1 < nk; ++kt) {
    load_frags(kt, 1, 1);                       // second k step of this stage
    __builtin_amdgcn_sched_barrier(0);
    mfmas(0);
    __builtin_amdgcn_sched_barrier(0);
    // the slot of stage kt-1 is free: every wave finished reading it before the
    // previous barrier
    if (kt + Cfg::NS - 1 < nk) issue(kt + Cfg::NS - 1);
    // stage kt+1 has landed once at most the stages issued after it are pending
    if (kt + Cfg::NS - 1 < nk) wait_vmcnt<(Cfg::NS - 2) * Cfg::DPS>();
    else if (kt + Cfg::NS - 2 < nk) wait_vmcnt<(Cfg::NS - 3) * Cfg::DPS>();
    else wait_vmcnt<0>();
    __syncthreads();
    load_frags(kt + 1, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    mfmas(1);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (nk > 0) {
    load_frags(nk - 1, 1, 1);
    mfmas(0);
    mfmas(1);
  }
  __syncthreads();

  // Epilogue: each wave stages one 32-row strip of its accumulators in LDS (free
  // after the K loop), then every lane applies the epilogue to groups of 4
  // consecutive columns and stores them with one vector store.
  constexpr int PITCHF = Cfg::WN + 4;                // floats per staged row
  float* strip = (float*)smem + wave * 32 * PITCHF;
#pragma unroll
  for (int i = 0; i < Cfg::TM; ++i) {
#pragma unroll
    for (int j = 0; j < Cfg::TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        strip[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * PITCHF + 32 * j + (lane & 31)] = acc[i][j][r];
    __syncthreads();
#pragma unroll 1
    for (int e = lane; e < 32 * Cfg::WN / 4; e += 64) {
      const int row = e / (Cfg::WN / 4), c4 = e % (Cfg::WN / 4);
      const int64_t m = m0 + wm * Cfg::WM + 32 * i + row;
      const int64_t n = n0 + wn * Cfg::WN + 4 * c4;
      if (m < a.M && n < ncols) {
        const f32x4 v = *(const f32x4*)(strip + row * PITCHF + 4 * c4);
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
  if (a.K % Cfg::BK != 0) return hipErrorInvalidValue;
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

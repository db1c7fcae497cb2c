// GEMM family for the BPT layer: C[M,N] = A[M,K] * B[N,K]^T with fused epilogues.
//
// Every dense contraction of the layer (QKV / output projections, both FFN
// linears and all their weight / input gradients) is issued in this one "NT"
// form. Operands are normally contiguous along K; either one may also be stored
// K-major (weights as the caller stores them, token-major activations contracted over
// tokens, feature-major gradients contracted over features), which the kernel
// transposes on its way from LDS into the MFMA registers.
//
// bf16 path: gfx950 MFMA v_mfma_f32_32x32x16_bf16, fp32 accumulation; tiles of 256 x 256
// with 8 waves (2 along M x 4 along N, two per SIMD) or, where fewer than 256 such tiles
// exist, 128 x 128 with 4 waves (2 x 2); K step 32 per stage through an LDS ring with
// XOR-swizzled 16-byte chunks, so that the rows a fragment read touches fall in distinct
// banks. fp32 path: plain VALU FMA tiles (used for the fp32 parity workload).
#include "common.h"
#include "internal.h"
#include <type_traits>

namespace bpt {

// GELU' output C2, element idx: fp32 or fp16 (a.c2t)
BPT_DEV void c2_store(const GemmArgs& a, int64_t idx, float v) {
  if (a.c2t == F16) ((f16*)a.C2)[idx] = (f16)v;
  else ((float*)a.C2)[idx] = v;
}
BPT_DEV void c2_store4(const GemmArgs& a, int64_t idx, f32x4 v) {
  if (a.c2t == F16) {
    const f16x4 h = {(f16)v[0], (f16)v[1], (f16)v[2], (f16)v[3]};
    *(f16x4*)((f16*)a.C2 + idx) = h;
  } else {
    *(f32x4*)((float*)a.C2 + idx) = v;
  }
}

// the FFN activation epilogues and their activation with its derivative: GELU, or
// ReLU (derivative 0 at z = 0)
template <int EPI> constexpr bool kAct = EPI == EPI_GELU || EPI == EPI_RELU;
template <int EPI>
BPT_DEV void act_both(float z, float& g, float& gp) {
  if constexpr (EPI == EPI_RELU) {
    g = fmaxf(z, 0.0f);
    gp = z > 0.0f ? 1.0f : 0.0f;
  } else {
    gelu_both(z, g, gp);
  }
}

// EPI_XENT: d loss / d logit of column n for a row with log-sum-exp lse and target y
BPT_DEV float xent_grad(const GemmArgs& a, int64_t n, float v, float lse, int y) {
  if (n >= a.nvalid) return 0.0f;
  const float p = __builtin_amdgcn_exp2f((v - lse) * 1.4426950408889634f);
  return a.alpha * (n == y ? p - 1.0f : p);
}
// EPI_XENT_T: the same for element (m, n) of the transposed logits, vocabulary index m
// and token n. Edge tiles and full tiles (whose epilogue holds each column's base-2
// log-sum-exp) evaluate the same expression, so a token's gradient does not depend on
// where the tile boundaries fall.
BPT_DEV float xent_grad_t_l2(const GemmArgs& a, int64_t m, float v, float lse2, int y) {
  if (m >= a.nvalid) return 0.0f;
  const float p = __builtin_amdgcn_exp2f(fmaf(v, 1.4426950408889634f, -lse2));
  return a.alpha * (m == y ? p - 1.0f : p);
}
BPT_DEV float xent_grad_t(const GemmArgs& a, int64_t m, int64_t n, float v) {
  return xent_grad_t_l2(a, m, v, a.rowv[n] * 1.4426950408889634f, a.tgt[n]);
}

template <int EPI, typename CT, typename RT>
BPT_DEV void epi_store(const GemmArgs& a, int64_t z, int64_t m, int64_t n, float v) {
  CT* C = (CT*)a.C + z * a.sC;
  const int64_t idx = m * a.ldc + n;
  if (n >= a.N) {                                   // zero padding columns
    C[idx] = from_f32<CT>(0.0f);
    if (kAct<EPI> && a.C2) c2_store(a, z * a.sC2 + m * a.ldc2 + n, 0.0f);
    return;
  }
  if constexpr (EPI == EPI_STORE) {
    v *= a.alpha;
    if constexpr (sizeof(CT) == 4) {
      if (a.accumulate) v += to_f32<CT>(C[idx]);
    }
    C[idx] = from_f32<CT>(v);
  } else if constexpr (EPI == EPI_RESID) {
    const RT* R = (const RT*)a.R + z * a.sR;
    v += to_f32<RT>(R[m * a.ldr + n]);
    if (a.bias) v += a.bias[n];
    C[idx] = from_f32<CT>(v);
  } else if constexpr (kAct<EPI>) {
    if (a.bias) v += a.bias[a.bias_on_m ? m : n];
    float g, gp;
    act_both<EPI>(v, g, gp);
    C[idx] = from_f32<CT>(g);
    if (a.C2) c2_store(a, z * a.sC2 + m * a.ldc2 + n, gp);
  } else if constexpr (EPI == EPI_XENT) {
    C[idx] = from_f32<CT>(xent_grad(a, n, v, a.rowv[m], a.tgt[m]));
  } else if constexpr (EPI == EPI_XENT_T) {
    C[idx] = from_f32<CT>(xent_grad_t(a, m, n, v));
  } else {  // EPI_MUL
    const RT* R = (const RT*)a.R + z * a.sR;
    C[idx] = from_f32<CT>(v * to_f32<RT>(R[m * a.ldr + n]));
  }
}

template <typename T> struct V4;
template <> struct V4<float> {
  static BPT_DEV f32x4 ld(const float* p) { return *(const f32x4*)p; }
  static BPT_DEV void st(float* p, f32x4 v) { *(f32x4*)p = v; }
};
template <> struct V4<f16> {
  static BPT_DEV f32x4 ld(const f16* p) {
    const f16x4 x = *(const f16x4*)p;
    return f32x4{(float)x[0], (float)x[1], (float)x[2], (float)x[3]};
  }
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
    v *= a.alpha;
    if constexpr (sizeof(CT) == 4) {
      if (a.accumulate) v += V4<CT>::ld(C);
    }
  } else if constexpr (EPI == EPI_RESID) {
    v += V4<RT>::ld((const RT*)a.R + z * a.sR + m * a.ldr + n);
    if (a.bias) v += *(const f32x4*)(a.bias + n);
  } else if constexpr (kAct<EPI>) {
    if (a.bias) {
      if (a.bias_on_m) v += a.bias[m];
      else v += *(const f32x4*)(a.bias + n);
    }
    f32x4 d;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float g, gp;
      act_both<EPI>(v[e], g, gp);
      v[e] = g;
      d[e] = gp;
    }
    if (a.C2) c2_store4(a, z * a.sC2 + m * a.ldc2 + n, d);
  } else if constexpr (EPI == EPI_XENT) {
    const float lse = a.rowv[m];
    const int y = a.tgt[m];
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = xent_grad(a, n + e, v[e], lse, y);
  } else if constexpr (EPI == EPI_XENT_T) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = xent_grad_t(a, m, n + e, v[e]);
  } else {
    v *= V4<RT>::ld((const RT*)a.R + z * a.sR + m * a.ldr + n);
  }
  V4<CT>::st(C, v);
}

// Four consecutive columns n..n+3 of row m inside the stored width, from pointers
// already at (m, n): c into C, r into R (EPI_RESID / EPI_MUL; for an fp32 C that
// accumulates, the values of C already loaded); c2 is the element index of (m, n) in
// C2 (EPI_GELU / EPI_RELU); bn at bias[n]; bm = bias[m] for a per-row bias, or the row's
// log-sum-exp for EPI_XENT, whose column is n and target y; EPI_XENT_T takes row m
// (passed as y) and column n.
template <int EPI, typename CT, typename RT>
BPT_DEV void epi_vec4(const GemmArgs& a, CT* c, const void* r, int64_t c2, const float* bn, float bm, f32x4 v,
                      int64_t n = 0, int64_t y = 0) {
  if constexpr (EPI == EPI_STORE) {
    v *= a.alpha;
    if constexpr (sizeof(CT) == 4) {
      if (a.accumulate) v += V4<CT>::ld((const CT*)r);
    }
  } else if constexpr (EPI == EPI_RESID) {
    v += V4<RT>::ld((const RT*)r);
    if (a.bias) v += *(const f32x4*)bn;
  } else if constexpr (kAct<EPI>) {
    if (a.bias) {
      if (a.bias_on_m) v += bm;
      else v += *(const f32x4*)bn;
    }
    f32x4 d;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float g, gp;
      act_both<EPI>(v[e], g, gp);
      v[e] = g;
      d[e] = gp;
    }
    if (a.C2) c2_store4(a, c2, d);
  } else if constexpr (EPI == EPI_XENT) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = xent_grad(a, n + e, v[e], bm, (int)y);
  } else if constexpr (EPI == EPI_XENT_T) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = xent_grad_t(a, y, n + e, v[e]);
  } else {
    v *= V4<RT>::ld((const RT*)r);
  }
  V4<CT>::st(c, v);
}

// ------------------------------------------------------------------ bf16 MFMA kernel
// Tile BM x BN (2 x NWN waves), K step 32 per stage, NS stages in an LDS ring filled
// by direct global->LDS copies (global_load_lds_dwordx4) issued NS-1 stages ahead.
// Tile rows are 32 bf16 (64 bytes, four 16-byte chunks) stored unpadded; chunk c of
// row r sits at chunk position c ^ swz(r), which spreads the rows that one fragment read
// touches over distinct bank groups. The copies apply the same permutation on the
// global side, so a wave's 1 KiB copy block still lands contiguously. K must be a
// multiple of 32 (host-checked).
template <int BM, int BN, int NWN = 2>
struct TileCfg {
  static constexpr int BK = 32;
  static constexpr int PITCH = 64;                     // bytes per tile row
  static constexpr int NW = 2 * NWN;                  // waves: 2 along M x NWN along N
  static constexpr int WM = BM / 2, WN = BN / NWN;    // wave tile
  static constexpr int TM = WM / 32, TN = WN / 32;    // 32x32 MFMA tiles per wave
  static constexpr int ABYTES = BM * PITCH, BBYTES = BN * PITCH;
  static constexpr int ABLK = ABYTES / 1024, BBLK = BBYTES / 1024;    // 1 KB copy blocks
  static constexpr int APW = (ABLK + NW - 1) / NW, BPW = (BBLK + NW - 1) / NW;   // copies per wave
  static constexpr int DPS = APW + BPW;               // copy instructions per wave per stage
  static constexpr int STAGE = ABYTES + BBYTES;
  static constexpr int NS = 4;                        // stages in the ring
  static constexpr int LDS = NS * STAGE;
  static_assert(ABYTES % 1024 == 0 && BBYTES % 1024 == 0, "whole copy blocks");
  static_assert(NW * (WN + 4) * 32 * 4 <= LDS, "epilogue staging fits");
};

// One wave copies 1 KiB from global memory straight into LDS: lane l's 16 bytes land at
// lds_block + 16 l. Written as inline assembly on purpose: the compiler's counter
// tracking treats the builtin form as a pending FLAT access and then turns every later
// LDS-fragment wait into a full drain. Completion is tracked by hand (wait_vmcnt). M0 is
// a reserved register the compiler does not otherwise use in these kernels.
BPT_DEV void lds_dma16(const void* g, uint32_t lds_block) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(g), "s"(lds_block) : "memory");
}

// chunk permutation of tile row r: bits (r1 ^ r3, r2). Within any 8 consecutive rows,
// and within any 16 consecutive rows of equal r mod 4, (row, chunk) pairs of one chunk
// column fall in distinct 16-byte bank groups.
BPT_DEV int swz(int r) { return (((r >> 1) ^ (r >> 3)) & 1) | (r & 4) >> 1; }

template <int N> BPT_DEV void wait_vmcnt() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

// Operand tiles stored transposed (source rows are k, the M or N extent contiguous):
// 32 rows of 2 * BX bytes per stage, chunk c of row k at chunk position c ^ 4 (k % 4).
// A fragment (8 consecutive k of one column per lane) is two ds_read_b64_tr_b16: in each
// group of 16 lanes, lane m addresses 4 columns of one row (row m / 4, columns 4 (m % 4)..)
// and receives column m of the group's 4 rows. Over the 32 lanes the hardware serves
// together (4 rows, 64 bytes each), the XOR places the rows in distinct 64-byte bank groups.
template <int BX>
struct TrTile {
  static constexpr int RB = 2 * BX;                    // bytes per k row
  static constexpr int CPR = RB / 16;                  // 16-byte chunks per row
};

typedef __attribute__((__vector_size__(4 * sizeof(short)))) short g_s16x4;
typedef __attribute__((__vector_size__(8 * sizeof(short)))) short g_s16x8;
BPT_DEV bf16x8 tr_frag(const char* p, int second) {
  typedef __attribute__((address_space(3))) g_s16x4 lds_s16x4;
  const g_s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
  const g_s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + second));
  const g_s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// Per-lane source offset (elements) of copy slot `slot` of a transposed operand tile:
// k row `row` of the tile, logical chunk from the swizzle, columns clamped to the readable
// width (cols_left = readable columns from the tile's first column, >= 8).
template <int BX>
BPT_DEV void tr_slot(int slot, int& row, int& col, int cols_left) {
  row = slot / TrTile<BX>::CPR;
  const int lc = (slot % TrTile<BX>::CPR) ^ (4 * (row & 3));
  col = 8 * lc < cols_left - 8 ? 8 * lc : cols_left - 8;
}

template <int BM, int BN, int EPI, typename CT, typename RT, bool TA = false, bool TB = false, int NWN = 2>
__global__ __launch_bounds__(128 * NWN, 1) void gemm_bf16_kernel(GemmArgs a) {
  using Cfg = TileCfg<BM, BN, NWN>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / NWN, wn = wave % NWN;
  // Tile order. Workgroup i runs on XCD i % 8, and each XCD has its own L2. The ids are
  // renumbered so that every XCD owns a contiguous range of tiles; within the range,
  // tiles go down GM row blocks before moving to the next column block, so the ~32
  // workgroups an XCD runs at once share 8 row blocks of A and ~4 column blocks of B.
  const int tiles_m = (int)((a.M + BM - 1) / BM);
  const int64_t ncols = a.Nstore > a.N ? a.Nstore : a.N;
  const int tiles_n = (int)((ncols + BN - 1) / BN);
  constexpr int GM = 8, NXCD = 8;
  int pid = blockIdx.x;
  {
    const int ntiles = tiles_m * tiles_n, q = ntiles / NXCD, r = ntiles % NXCD, x = pid % NXCD;
    pid = x * q + (x < r ? x : r) + pid / NXCD;
  }
  const int group = pid / (GM * tiles_n), first_m = group * GM;
  const int gm = tiles_m - first_m < GM ? tiles_m - first_m : GM;
  const int tm = first_m + (pid % (GM * tiles_n)) % gm;
  const int tn = (pid % (GM * tiles_n)) / gm;
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN, z = blockIdx.z;
  const bf16* A = (const bf16*)a.A + z * a.sA + (TA ? m0 : m0 * a.lda);
  const bf16* B = (const bf16*)a.B + z * a.sB + (TB ? n0 : n0 * a.ldb);
  const int nk = (int)(a.K / Cfg::BK);
  // transposed operands: readable k rows and columns (from the tile's first column)
  const int64_t arows = a.a_rows > 0 ? a.a_rows : a.K, brows = a.b_rows > 0 ? a.b_rows : a.K;
  const int acols = (int)((a.a_cols > 0 ? a.a_cols : a.M) - m0);
  const int bcols = (int)((a.b_cols > 0 ? a.b_cols : a.N) - n0);

  // per-lane source offsets (elements) of this wave's copy slots; rows past the
  // matrix edge are clamped to its last row (their results are never stored). 64-bit:
  // a row-major operand's stride can be the token count, and 255 rows of it exceed 2^31.
  int64_t aoff[Cfg::APW], boff[Cfg::BPW];
  {
    const int alast = (int)(a.M - 1 - m0), blast = (int)(a.N - 1 - n0);
#pragma unroll
    for (int i = 0; i < Cfg::APW; ++i) {
      int blk = wave + Cfg::NW * i;
      blk = blk < Cfg::ABLK ? blk : Cfg::ABLK - 1;     // extra copies repeat the last block
      const int slot = blk * 64 + lane;
      if constexpr (TA) {
        int row, col;
        tr_slot<BM>(slot, row, col, acols);
        aoff[i] = row * a.lda + col;
      } else {
        const int row = slot >> 2, col = (slot & 3) ^ swz(row);
        aoff[i] = (row < alast ? row : alast) * a.lda + col * 8;
      }
    }
#pragma unroll
    for (int i = 0; i < Cfg::BPW; ++i) {
      int blk = wave + Cfg::NW * i;
      blk = blk < Cfg::BBLK ? blk : Cfg::BBLK - 1;
      const int slot = blk * 64 + lane;
      if constexpr (TB) {
        int row, col;
        tr_slot<BN>(slot, row, col, bcols);
        boff[i] = row * a.ldb + col;
      } else {
        const int row = slot >> 2, col = (slot & 3) ^ swz(row);
        boff[i] = (row < blast ? row : blast) * a.ldb + col * 8;
      }
    }
  }
  // copy d (0 <= d < DPS) of this wave for stage kt: A blocks first, then B blocks
  // LDS address of the tile ring (the copies take LDS addresses, not generic pointers)
  const uint32_t ring = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)smem);
  // A transposed operand's stage is k rows k0 .. k0+31; rows from x_rows on are clamped to
  // the last readable row (the caller guarantees the other operand is zero there).
  auto tr_src = [&](const bf16* X, int64_t ld, int64_t xrows, int cols, int k0, int blk, int64_t off,
                    auto BXc) -> const bf16* {
    constexpr int BX = decltype(BXc)::value;
    if (k0 + Cfg::BK <= xrows) return X + (int64_t)k0 * ld + off;
    int row, col;
    tr_slot<BX>(blk * 64 + lane, row, col, cols);
    const int64_t r = k0 + row < xrows ? k0 + row : xrows - 1;
    return X + r * ld + col;
  };
  // FAST: a stage whose k rows all lie below arows and brows (no clamping of transposed rows)
  auto dma = [&](int kt, int d, auto FASTc) {
    constexpr bool FAST = decltype(FASTc)::value;
    const uint32_t st = ring + (kt % Cfg::NS) * Cfg::STAGE;
    const int k0 = kt * Cfg::BK;
    if (d < Cfg::APW) {
      int blk = wave + Cfg::NW * d;
      blk = blk < Cfg::ABLK ? blk : Cfg::ABLK - 1;
      if constexpr (TA) {
        if constexpr (FAST) lds_dma16(A + (int64_t)k0 * a.lda + aoff[d], st + blk * 1024);
        else
          lds_dma16(tr_src(A, a.lda, arows, acols, k0, blk, aoff[d], std::integral_constant<int, BM>{}),
                    st + blk * 1024);
      } else
        lds_dma16(A + k0 + aoff[d], st + blk * 1024);
    } else {
      int blk = wave + Cfg::NW * (d - Cfg::APW);
      blk = blk < Cfg::BBLK ? blk : Cfg::BBLK - 1;
      if constexpr (TB) {
        if constexpr (FAST) lds_dma16(B + (int64_t)k0 * a.ldb + boff[d - Cfg::APW], st + Cfg::ABYTES + blk * 1024);
        else
          lds_dma16(tr_src(B, a.ldb, brows, bcols, k0, blk, boff[d - Cfg::APW], std::integral_constant<int, BN>{}),
                    st + Cfg::ABYTES + blk * 1024);
      } else
        lds_dma16(B + k0 + boff[d - Cfg::APW], st + Cfg::ABYTES + blk * 1024);
    }
  };

  f32x16 acc[Cfg::TM][Cfg::TN];
#pragma unroll
  for (int i = 0; i < Cfg::TM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::TN; ++j) acc[i][j] = f32x16{};

  // per-lane fragment bases of the two k steps of a stage (row bits 1..3 come from the lane)
  const int sw = swz(lane & 31), h = lane >> 5;
  const int abase[2] = {(wm * Cfg::WM + (lane & 31)) * Cfg::PITCH + 16 * (h ^ sw),
                        (wm * Cfg::WM + (lane & 31)) * Cfg::PITCH + 16 * ((2 + h) ^ sw)};
  const int bbase[2] = {Cfg::ABYTES + (wn * Cfg::WN + (lane & 31)) * Cfg::PITCH + 16 * (h ^ sw),
                        Cfg::ABYTES + (wn * Cfg::WN + (lane & 31)) * Cfg::PITCH + 16 * ((2 + h) ^ sw)};

  // Fragments are double-buffered in registers. Fragment r of a k step (0: A0,
  // 1..TN: B0.., then A1..) is read in the order the MFMAs of the next k step use them.
  // transposed tiles: per-lane byte offset of fragment i (32 columns) for k step 0; the
  // second read of a fragment is 4 rows further, k step 1 16 rows further
  int tra[Cfg::TM], trb[Cfg::TN];
  {
    const int g = lane >> 4, m = lane & 15, sx = (m >> 2) & 3, q = 2 * (g & 1) + ((m >> 1) & 1);
    const int rowpart = 8 * (g >> 1) + (m >> 2), within = 16 * q + 8 * (m & 1);
    if constexpr (TA) {
#pragma unroll
      for (int i = 0; i < Cfg::TM; ++i)
        tra[i] = rowpart * TrTile<BM>::RB + 64 * (((wm * Cfg::WM) / 32 + i) ^ sx) + within;
    }
    if constexpr (TB) {
#pragma unroll
      for (int j = 0; j < Cfg::TN; ++j)
        trb[j] = Cfg::ABYTES + rowpart * TrTile<BN>::RB + 64 * (((wn * Cfg::WN) / 32 + j) ^ sx) + within;
    }
  }
  bf16x8 fa[2][Cfg::TM], fb[2][Cfg::TN];
  auto read_a = [&](const char* st, int kk, int buf, int i) {
    if constexpr (TA) fa[buf][i] = tr_frag(st + tra[i] + kk * 16 * TrTile<BM>::RB, 4 * TrTile<BM>::RB);
    else fa[buf][i] = *(const bf16x8*)(st + abase[kk] + i * 32 * Cfg::PITCH);
  };
  auto read_b = [&](const char* st, int kk, int buf, int j) {
    if constexpr (TB) fb[buf][j] = tr_frag(st + trb[j] + kk * 16 * TrTile<BN>::RB, 4 * TrTile<BN>::RB);
    else fb[buf][j] = *(const bf16x8*)(st + bbase[kk] + j * 32 * Cfg::PITCH);
  };
  auto read_frag = [&](const char* st, int kk, int buf, int r) {
    if (r == 0) read_a(st, kk, buf, 0);
    else if (r <= Cfg::TN) read_b(st, kk, buf, r - 1);
    else read_a(st, kk, buf, r - Cfg::TN);
  };
  // One k step: the TM x TN MFMAs on fragment buffer CUR, each followed by at most one
  // fragment read of the next k step (stage rkt, half rkk) into the other buffer and by
  // this wave's share of the copies of stage dkt, so that the LDS and copy traffic is
  // spread over the MFMA stream instead of arriving in bursts.
  auto kstep = [&](auto cur_c, auto read_c, auto dma_c, int rkt, int rkk, int dkt, auto fast_c) {
    constexpr int cur = decltype(cur_c)::value;
    constexpr bool rd = decltype(read_c)::value, cp = decltype(dma_c)::value;
    constexpr int TMN = Cfg::TM * Cfg::TN, NR = Cfg::TM + Cfg::TN;
    const char* rst = smem + (rkt % Cfg::NS) * Cfg::STAGE;
#pragma unroll
    for (int q = 0; q < TMN; ++q) {
      acc[q / Cfg::TN][q % Cfg::TN] = mfma32x32x16(fa[cur][q / Cfg::TN], fb[cur][q % Cfg::TN],
                                                    acc[q / Cfg::TN][q % Cfg::TN]);
      if (rd && q < NR) read_frag(rst, rkk, 1 - cur, q);
      if (cp) {
#pragma unroll
        for (int d = (q * Cfg::DPS + TMN - 1) / TMN; d < ((q + 1) * Cfg::DPS + TMN - 1) / TMN; ++d) dma(dkt, d, fast_c);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using T_ = std::true_type;
  using F_ = std::false_type;

  // stages 0 .. NS-2 in flight; wait for stage 0
#pragma unroll
  for (int s = 0; s < Cfg::NS - 1; ++s)
    if (s < nk) {
#pragma unroll
      for (int d = 0; d < Cfg::DPS; ++d) dma(s, d, F_{});
    }
  if (nk >= Cfg::NS - 1) wait_vmcnt<(Cfg::NS - 2) * Cfg::DPS>();
  else wait_vmcnt<0>();
  __syncthreads();
  if (nk > 0) {
#pragma unroll
    for (int r = 0; r < Cfg::TM + Cfg::TN; ++r) read_frag(smem, 0, 0, r);
  }
  // Stage kt: the first k step reads the second half of stage kt and, while the ring
  // still has stages to fetch, copies stage kt+NS-1 into the slot of stage kt-1 (every
  // wave finished reading that slot before the previous barrier). The barrier then
  // publishes stage kt+1, whose first half the second k step reads. The two loops differ
  // only in whether copies remain; the last stage is peeled.
  const int kcopy = nk - (Cfg::NS - 1) > 0 ? nk - (Cfg::NS - 1) : 0;
  // stages whose copies need no clamping: all of them unless a transposed operand has
  // fewer readable k rows than K
  int64_t kread = a.K;
  if constexpr (TA) kread = arows < kread ? arows : kread;
  if constexpr (TB) kread = brows < kread ? brows : kread;
  const int kfast = (int)(kread / Cfg::BK);     // stages 0 .. kfast-1 are whole
  const int kc1 = kfast - (Cfg::NS - 1) < kcopy ? (kfast - (Cfg::NS - 1) > 0 ? kfast - (Cfg::NS - 1) : 0) : kcopy;
  int kt = 0;
  for (; kt < kc1; ++kt) {
    kstep(I0{}, T_{}, T_{}, kt, 1, kt + Cfg::NS - 1, T_{});
    wait_vmcnt<(Cfg::NS - 2) * Cfg::DPS>();
    __syncthreads();
    kstep(I1{}, T_{}, F_{}, kt + 1, 0, 0, T_{});
  }
  for (; kt < kcopy; ++kt) {
    kstep(I0{}, T_{}, T_{}, kt, 1, kt + Cfg::NS - 1, F_{});
    wait_vmcnt<(Cfg::NS - 2) * Cfg::DPS>();
    __syncthreads();
    kstep(I1{}, T_{}, F_{}, kt + 1, 0, 0, F_{});
  }
  for (; kt + 1 < nk; ++kt) {
    kstep(I0{}, T_{}, F_{}, kt, 1, 0, F_{});
    wait_vmcnt<0>();
    __syncthreads();
    kstep(I1{}, T_{}, F_{}, kt + 1, 0, 0, F_{});
  }
  if (nk > 0) {
    kstep(I0{}, T_{}, F_{}, nk - 1, 1, 0, F_{});
    kstep(I1{}, F_{}, F_{}, 0, 0, 0, F_{});
  }
  __syncthreads();

  // Epilogue: each wave stages one 32-row strip of its accumulators in its own part of
  // the (now idle) LDS, then every lane applies the epilogue to groups of 4 consecutive
  // columns and stores them with one vector store. The strips are private to their
  // wave, so no barrier is needed between strips.
  constexpr int PITCHF = Cfg::WN + 4;                // floats per staged row
  constexpr int C4 = Cfg::WN / 4;                    // 4-column groups per row
  constexpr int RSTEP = 64 / C4;                     // rows per iteration of a strip
  float* strip = (float*)smem + wave * 32 * PITCHF;
  const bool inside = m0 + BM <= a.M && n0 + BN <= a.N;
  // The operand the epilogue reads (R of a residual or multiplier epilogue, C itself
  // for an fp32 C that accumulates) is loaded ahead for full tiles: 16-bit operands
  // for all strips before the first staging, 32-bit ones two strips ahead, so that the
  // load latency is not paid once per strip.
  constexpr bool PRE = EPI == EPI_RESID || EPI == EPI_MUL || (EPI == EPI_STORE && sizeof(CT) == 4);
  constexpr int PES = EPI == EPI_STORE ? (int)sizeof(CT) : (int)sizeof(RT);   // bytes per element
  constexpr int PD = PES == 2 ? Cfg::TM : 2;                                   // strips in flight
  constexpr int NIT = 32 / RSTEP;
  typedef std::conditional_t<PES == 2, u32x2, u32x4> PreT;
  PreT pre[PRE ? PD : 1][PRE ? NIT : 1];
  const bool do_pre = PRE && inside && (EPI != EPI_STORE || a.accumulate);
  const char* pbase = nullptr;
  int64_t pld = 0;
  if constexpr (PRE) {
    const int64_t row0 = m0 + wm * Cfg::WM + lane / C4, col0 = n0 + wn * Cfg::WN + 4 * (lane % C4);
    if constexpr (EPI == EPI_STORE) {
      pbase = (const char*)((const CT*)a.C + z * a.sC + row0 * a.ldc + col0);
      pld = a.ldc * PES;
    } else {
      pbase = (const char*)((const RT*)a.R + z * a.sR + row0 * a.ldr + col0);
      pld = a.ldr * PES;
    }
  }
  auto preload = [&](int i) {
    if constexpr (PRE) {
#pragma unroll
      for (int it = 0; it < NIT; ++it)
        pre[i % PD][it] = *(const PreT*)(pbase + (int64_t)(32 * i + RSTEP * it) * pld);
    }
  };
  if (do_pre) {
#pragma unroll
    for (int i = 0; i < PD; ++i) preload(i);
  }
#pragma unroll
  for (int i = 0; i < Cfg::TM; ++i) {
#pragma unroll
    for (int j = 0; j < Cfg::TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        strip[(8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * PITCHF + 32 * j + (lane & 31)] = acc[i][j][r];
    const int64_t mrow = m0 + wm * Cfg::WM + 32 * i;
    const int64_t ncol = n0 + wn * Cfg::WN;
    if (inside) {
      // rows are (lane / C4) + (64 / C4) * it; columns 4 * (lane % C4)
      const int r0 = lane / C4, c0 = 4 * (lane % C4);
      CT* cb = (CT*)a.C + z * a.sC + (mrow + r0) * a.ldc + ncol + c0;
      const char* rb = nullptr;
      if constexpr (EPI == EPI_RESID) rb = (const char*)((const RT*)a.R + z * a.sR + (mrow + r0) * a.ldr + ncol + c0);
      else if constexpr (EPI == EPI_MUL) rb = (const char*)((const RT*)a.R + z * a.sR + (mrow + r0) * a.ldr + ncol + c0);
      const int64_t c2b = z * a.sC2 + (mrow + r0) * a.ldc2 + ncol + c0;
      const float* bb = a.bias ? a.bias + ncol + c0 : nullptr;
      constexpr int RS = (int)sizeof(RT);
      // the GELU epilogue is long: keep its loop rolled (instruction cache)
      constexpr int UNR = kAct<EPI> ? 4 : 32 / RSTEP;
      if constexpr (EPI == EPI_XENT_T) {
        // a lane's four columns (tokens) are the same on every row of the strip: their
        // log-sum-exp (base 2) and targets are loaded once
        float l2[4];
        int y4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          l2[e] = a.rowv[ncol + c0 + e] * 1.4426950408889634f;
          y4[e] = a.tgt[ncol + c0 + e];
        }
#pragma unroll 4
        for (int it = 0; it < 32 / RSTEP; ++it) {
          const int row = r0 + RSTEP * it;
          const int64_t m = mrow + row;                // vocabulary index
          f32x4 v = *(const f32x4*)(strip + row * PITCHF + c0);
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = xent_grad_t_l2(a, m, v[e], l2[e], y4[e]);
          V4<CT>::st(cb + (int64_t)RSTEP * it * a.ldc, v);
        }
        continue;
      }
#pragma unroll UNR
      for (int it = 0; it < 32 / RSTEP; ++it) {
        const int row = r0 + RSTEP * it;
        const f32x4 v = *(const f32x4*)(strip + row * PITCHF + c0);
        float bm = (kAct<EPI> && a.bias && a.bias_on_m) ? a.bias[mrow + row] : 0.0f;
        int64_t y = 0;
        if constexpr (EPI == EPI_XENT) {
          bm = a.rowv[mrow + row];
          y = a.tgt[mrow + row];
        } else if constexpr (EPI == EPI_XENT_T) {
          y = mrow + row;                              // the row's vocabulary index
        }
        if constexpr (PRE)
          epi_vec4<EPI, CT, RT>(a, cb + (int64_t)RSTEP * it * a.ldc, &pre[i % PD][it], 0, bb, bm, v);
        else
          epi_vec4<EPI, CT, RT>(a, cb + (int64_t)RSTEP * it * a.ldc,
                                rb + (int64_t)RSTEP * it * a.ldr * RS,
                                c2b + (int64_t)RSTEP * it * a.ldc2, bb, bm, v, ncol + c0, y);
      }
      if (do_pre && i + PD < Cfg::TM) preload(i + PD);
    } else {
#pragma unroll 1
      for (int e = lane; e < 32 * C4; e += 64) {
        const int row = e / C4, c4 = e % C4;
        const int64_t m = mrow + row, n = ncol + 4 * c4;
        if (m < a.M && n < ncols) {
          const f32x4 v = *(const f32x4*)(strip + row * PITCHF + 4 * c4);
          epi_store4<EPI, CT, RT>(a, z, m, n, ncols, v);
        }
      }
    }
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
  const int64_t arows = a.trans_a && a.a_rows > 0 ? a.a_rows : a.K;
  const int64_t brows = a.trans_b && a.b_rows > 0 ? a.b_rows : a.K;
  for (int64_t k0 = 0; k0 < a.K; k0 += 16) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t k = k0 + lk + e;
      const int64_t ai = a.trans_a ? k * a.lda + m0 + lr : (m0 + lr) * a.lda + k;
      const int64_t bi = a.trans_b ? k * a.ldb + n0 + lr : (n0 + lr) * a.ldb + k;
      As[lk + e][lr] = (m0 + lr < a.M && k < arows) ? A[ai] : 0.0f;
      Bs[lk + e][lr] = (n0 + lr < a.N && k < brows) ? B[bi] : 0.0f;
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
template <int BM, int BN, int EPI, typename CT, typename RT, bool TA = false, bool TB = false, int NWN = 2>
static hipError_t launch_bf16(const GemmArgs& a, hipStream_t s) {
  using Cfg = TileCfg<BM, BN, NWN>;
  auto kern = gemm_bf16_kernel<BM, BN, EPI, CT, RT, TA, TB, NWN>;
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
  hipLaunchKernelGGL(kern, dim3((unsigned)tiles, 1, (unsigned)a.batch), dim3(64 * Cfg::NW), Cfg::LDS, s, a);
  return hipGetLastError();
}

// waves along N of the 256 x 256 tile configuration
static constexpr int kNWN = 4;

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
  if (a.trans_a || a.trans_b) {
    // a transposed operand is read in 16-byte column chunks
    if ((a.trans_a && ((a.a_cols > 0 ? a.a_cols : a.M) % 8 || a.lda % 8)) ||
        (a.trans_b && ((a.b_cols > 0 ? a.b_cols : a.N) % 8 || a.ldb % 8)))
      return hipErrorInvalidValue;
    // instantiated combinations: B transposed with every epilogue, A transposed with
    // the plain store and the activation epilogues, both with the plain store
    if (a.trans_a && a.trans_b) {
      if constexpr (EPI == EPI_STORE)
        return big >= 256 ? launch_bf16<256, 256, EPI, CT, RT, true, true, kNWN>(a, s)
                          : launch_bf16<128, 128, EPI, CT, RT, true, true>(a, s);
      return hipErrorInvalidValue;
    }
    if (a.trans_a) {
      if constexpr (EPI == EPI_STORE || kAct<EPI> || EPI == EPI_XENT_T)
        return big >= 256 ? launch_bf16<256, 256, EPI, CT, RT, true, false, kNWN>(a, s)
                          : launch_bf16<128, 128, EPI, CT, RT, true, false>(a, s);
      return hipErrorInvalidValue;
    }
    return big >= 256 ? launch_bf16<256, 256, EPI, CT, RT, false, true, kNWN>(a, s)
                      : launch_bf16<128, 128, EPI, CT, RT, false, true>(a, s);
  }
  if (big >= 256) return launch_bf16<256, 256, EPI, CT, RT, false, false, kNWN>(a, s);
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
    case EPI_RELU:
      return ct == F32 ? launch_typed<EPI_RELU, float, float>(ab, a, s)
                       : launch_typed<EPI_RELU, bf16, float>(ab, a, s);
    case EPI_XENT:
      return ct == F32 ? launch_typed<EPI_XENT, float, float>(ab, a, s)
                       : launch_typed<EPI_XENT, bf16, float>(ab, a, s);
    case EPI_XENT_T:
      return ct == F32 ? launch_typed<EPI_XENT_T, float, float>(ab, a, s)
                       : launch_typed<EPI_XENT_T, bf16, float>(ab, a, s);
    case EPI_MUL:
      if (rt == F16)
        return ct == F32 ? launch_typed<EPI_MUL, float, f16>(ab, a, s)
                         : launch_typed<EPI_MUL, bf16, f16>(ab, a, s);
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

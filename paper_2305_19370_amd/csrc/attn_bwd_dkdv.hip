// Attention backward, key-outer dK/dV kernel (bf16 MFMA and fp32 VALU variants).
#include <algorithm>

#include "attn_common.h"

namespace bpt {

// ====================================================================== backward dK dV, bf16
// Key-outer: each wave owns 32 keys; loop over query tiles of 64 (two halves of
// 32). S = Q K^T and dP = dO V^T have the key on the lane axis, so P and dS feed
// dV^T += dO^T P and dK^T += Q^T dS directly as B operands.
template <int DH>
struct DkvCfg {
  static constexpr int KSTEPS = DH / 16, DT = DH / 32;
  static constexpr int RBYTES = RmTile<DH>::BYTES, FBYTES = FmTile<DH>::BYTES;
  static constexpr int STAGE = 2 * RBYTES + 2 * FBYTES + 2 * 64 * 4;   // Q, dO, Q^T, dO^T, lse, delta
  static constexpr int LDS = 2 * STAGE;
};

template <int DH>
__global__ __launch_bounds__(256, 1) void attn_bwd_dkdv_bf16_kernel(AttnArgs a) {
  using C = DkvCfg<DH>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.y, b = blockIdx.z;
  const int S = (int)a.S;
  const int k0 = (int)blockIdx.x * 128;          // causal: low key tiles have the most queries
  const int kw = k0 + 32 * wave;
  const int kvrow = kw + (lane & 31);
  const float scale = rsqrtf((float)DH);
  const float c = scale * LOG2E;

  const bf16* Qb = (const bf16*)a.q + (int64_t)b * a.S * a.ld_q + h * DH;
  const bf16* Kb = (const bf16*)a.k + (int64_t)b * a.S * a.ld_k + h * DH;
  const bf16* Vb = (const bf16*)a.v + (int64_t)b * a.S * a.ld_v + h * DH;
  const bf16* dOb = (const bf16*)a.dout + (int64_t)b * a.S * a.ld_do + h * DH;
  const bf16* Qtb = (const bf16*)a.qt + (int64_t)h * DH * a.ld_qt + (int64_t)b * a.Sp;
  const bf16* dOtb = (const bf16*)a.dot + (int64_t)h * DH * a.ld_dot + (int64_t)b * a.Sp;
  const float* lse2 = a.lse2 + ((int64_t)b * a.H + h) * a.Sp;
  const float* delta = a.delta + ((int64_t)b * a.H + h) * a.Sp;

  bf16x8 kf[C::KSTEPS], vf[C::KSTEPS];
  {
    const int kr = kvrow < S ? kvrow : S - 1;
#pragma unroll
    for (int kk = 0; kk < C::KSTEPS; ++kk) {
      kf[kk] = __builtin_bit_cast(bf16x8, ld16(Kb + (int64_t)kr * a.ld_k + 16 * kk + 8 * (lane >> 5)));
      vf[kk] = __builtin_bit_cast(bf16x8, ld16(Vb + (int64_t)kr * a.ld_v + 16 * kk + 8 * (lane >> 5)));
    }
  }
  const bool kok = kvrow < S;

  const int qstart = a.causal ? (k0 / 64) * 64 : 0;
  const int ntiles = qstart < S ? (S - qstart + 63) / 64 : 0;
  DmaPlan<RmTile<DH>::BLOCKS> pq, pdo;
  DmaPlan<FmTile<DH>::BLOCKS> pqt;       // Q^T and dO^T share their leading dimension
  plan_rows<DH>(pq, (int)a.ld_q, wave, lane);
  plan_rows<DH>(pdo, (int)a.ld_do, wave, lane);
  plan_cols<DH>(pqt, (int)a.ld_qt, wave, lane);
  auto issue = [&](int j) {
    const int qt0 = qstart + j * 64;
    char* qs = smem + (j & 1) * C::STAGE;
    dma_rows<DH>(qs, Qb, a.ld_q, qt0, S - 1, wave, lane, pq);
    dma_rows<DH>(qs + C::RBYTES, dOb, a.ld_do, qt0, S - 1, wave, lane, pdo);
    dma_cols<DH>(qs + 2 * C::RBYTES, Qtb, qt0, wave, pqt);
    dma_cols<DH>(qs + 2 * C::RBYTES + C::FBYTES, dOtb, qt0, wave, pqt);
    // base-2 lse, delta of the 64 queries (indices < Sp: in bounds; rows >= S are masked)
    if (wave == 0) dma4(lse2 + qt0 + lane, qs + 2 * C::RBYTES + 2 * C::FBYTES);
    if (wave == 1) dma4(delta + qt0 + lane, qs + 2 * C::RBYTES + 2 * C::FBYTES + 256);
  };

  f32x16 adv[C::DT], adk[C::DT];
#pragma unroll
  for (int t = 0; t < C::DT; ++t) {
    mfma_agpr_zero(adv[t]);
    mfma_agpr_zero(adk[t]);
  }

  auto tile = [&](int j, auto MASK) {
    const int qt0 = qstart + j * 64;
    const char* qs = smem + (j & 1) * C::STAGE;
    const char* ds = qs + C::RBYTES;
    const char* qts = ds + C::RBYTES;
    const char* dts = qts + C::FBYTES;
    const float* ls = (const float*)(dts + C::FBYTES);
    // query offset inside the tile of register r: 32*mt + 8*(r/4) + (r%4) + 4*(lane/32);
    // visible iff lo <= offset <= hi
    const int lo = (a.causal ? kvrow - qt0 : 0) - 4 * (lane >> 5);
    const int hi = (kok ? S - 1 - qt0 : -1) - 4 * (lane >> 5);
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
      for (int kk = 0; kk < C::KSTEPS; ++kk) {
        const int kc = 2 * kk + (lane >> 5);
        const bf16x8 aq = *(const bf16x8*)(qs + rm_addr<DH>(32 * mt + (lane & 31), kc));
        s = mfma32x32x16(aq, kf[kk], s);
        const bf16x8 ad = *(const bf16x8*)(ds + rm_addr<DH>(32 * mt + (lane & 31), kc));
        dp = mfma32x32x16(ad, vf[kk], dp);
      }
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int qi = 32 * mt + 8 * rg + 4 * (lane >> 5);
        const f32x4 l4 = *(const f32x4*)(ls + qi);
        const f32x4 d4 = *(const f32x4*)(ls + 64 + qi);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * rg + e;
          float p = fast_exp2(fmaf(s[r], c, -l4[e]));
          if constexpr (decltype(MASK)::value) {
            const int off = 32 * mt + 8 * rg + e;
            p = (off >= lo && off <= hi) ? p : 0.0f;
          }
          s[r] = p;
          dp[r] = p * (dp[r] - d4[e]);           // dS
        }
      }
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const bf16x8 pb = acc_to_b(s, hf);
        const bf16x8 sb = acc_to_b(dp, hf);
#pragma unroll
        for (int t = 0; t < C::DT; ++t) {
          const bf16x8 ado = fm_frag<DH>(dts, 32 * t + (lane & 31), 32 * mt + 16 * hf, lane);
          mfma_agpr(adv[t], ado, pb);
          const bf16x8 aqt = fm_frag<DH>(qts, 32 * t + (lane & 31), 32 * mt + 16 * hf, lane);
          mfma_agpr(adk[t], aqt, sb);
        }
      }
    }
  };

  // Phases (uniform over the workgroup, so every barrier is reached by all waves):
  // query tiles that straddle this key tile's diagonal (masked), tiles that every
  // key of the workgroup fully sees (unmasked), and a ragged tail (masked).
  const int n_diag = a.causal ? std::min(ntiles, (k0 + 128 - qstart + 63) / 64) : 0;
  const int n_full = (k0 + 128 <= S) ? std::max(n_diag, (S - qstart) / 64) : n_diag;
  if (ntiles > 0) issue(0);
  wait_dma();
  __syncthreads();
  int j = 0;
  for (; j < n_diag; ++j) {
    if (j + 1 < ntiles) issue(j + 1);
    if (!(a.causal && qstart + j * 64 + 63 < kw)) tile(j, std::true_type{});
    wait_dma();
    __syncthreads();
  }
  for (; j < n_full; ++j) {
    if (j + 1 < ntiles) issue(j + 1);
    tile(j, std::false_type{});
    wait_dma();
    __syncthreads();
  }
  for (; j < ntiles; ++j) {
    if (j + 1 < ntiles) issue(j + 1);
    tile(j, std::true_type{});
    wait_dma();
    __syncthreads();
  }

  if constexpr (C::DT == 4) {
    mfma_agpr_drain(adv[0], adv[1], adv[2], adv[3]);
    mfma_agpr_drain(adk[0], adk[1], adk[2], adk[3]);
  } else {
    mfma_agpr_drain(adv[0], adv[1]);
    mfma_agpr_drain(adk[0], adk[1]);
  }
  if (kvrow < a.Sp) {
    const int64_t col = (int64_t)b * a.Sp + kvrow;
    bf16* dKt = (bf16*)a.dkt + (int64_t)h * DH * a.ld_dt + col;
    bf16* dVt = (bf16*)a.dvt + (int64_t)h * DH * a.ld_dt + col;
#pragma unroll
    for (int t = 0; t < C::DT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t d = 32 * t + acc_row(r, lane);
        dKt[d * a.ld_dt] = (bf16)(adk[t][r] * scale);
        dVt[d * a.ld_dt] = (bf16)adv[t][r];
      }
  }
}

template <int DH>
__global__ __launch_bounds__(64) void attn_bwd_dkdv_f32_kernel(AttnArgs a) {
  extern __shared__ float fsm[];
  float* Kown = fsm;                       // [DH][65]
  float* Vown = Kown + DH * 65;            // [DH][65]
  float* Qs = Vown + DH * 65;              // [16][DH]
  float* dOs = Qs + 16 * DH;               // [16][DH]
  float* ls = dOs + 16 * DH;               // [16]
  float* dls = ls + 16;                    // [16]
  const int tid = threadIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int64_t S = a.S, k0 = (int64_t)blockIdx.x * 64, kv = k0 + tid;
  const float scale = rsqrtf((float)DH);
  const float* Qp = (const float*)a.q + (int64_t)h * DH;
  const float* Kp = (const float*)a.k + (int64_t)h * DH;
  const float* Vp = (const float*)a.v + (int64_t)h * DH;
  const float* dOp = (const float*)a.dout + (int64_t)h * DH;
  const float* lse = a.lse + ((int64_t)b * a.H + h) * a.Sp;
  const float* delta = a.delta + ((int64_t)b * a.H + h) * a.Sp;
  for (int d = 0; d < DH; ++d) {
    Kown[d * 65 + tid] = kv < S ? Kp[(b * S + kv) * a.ld_k + d] : 0.0f;
    Vown[d * 65 + tid] = kv < S ? Vp[(b * S + kv) * a.ld_v + d] : 0.0f;
  }
  float dk[DH], dv[DH];
#pragma unroll
  for (int d = 0; d < DH; ++d) dk[d] = dv[d] = 0.0f;
  const int64_t qstart = a.causal ? k0 : 0;
  for (int64_t qt0 = qstart; qt0 < S; qt0 += 16) {
    __syncthreads();
    for (int i = tid; i < 16 * DH; i += 64) {
      const int r = i / DH, d = i % DH;
      const int64_t q = qt0 + r;
      Qs[i] = q < S ? Qp[(b * S + q) * a.ld_q + d] : 0.0f;
      dOs[i] = q < S ? dOp[(b * S + q) * a.ld_do + d] : 0.0f;
    }
    if (tid < 16) {
      const int64_t q = qt0 + tid;
      ls[tid] = q < S ? lse[q] : 0.0f;
      dls[tid] = q < S ? delta[q] : 0.0f;
    }
    __syncthreads();
    for (int i = 0; i < 16; ++i) {
      const int64_t q = qt0 + i;
      float sv = 0.0f, dpv = 0.0f;
#pragma unroll
      for (int d = 0; d < DH; ++d) {
        sv = fmaf(Qs[i * DH + d], Kown[d * 65 + tid], sv);
        dpv = fmaf(dOs[i * DH + d], Vown[d * 65 + tid], dpv);
      }
      const bool ok = q < S && kv < S && !(a.causal && kv > q);
      const float p = ok ? __expf(sv * scale - ls[i]) : 0.0f;
      const float ds = p * (dpv - dls[i]);
#pragma unroll
      for (int d = 0; d < DH; ++d) {
        dv[d] = fmaf(p, dOs[i * DH + d], dv[d]);
        dk[d] = fmaf(ds, Qs[i * DH + d], dk[d]);
      }
    }
  }
  if (kv < a.Sp) {
    const int64_t col = (int64_t)b * a.Sp + kv;
    float* dKt = (float*)a.dkt + (int64_t)h * DH * a.ld_dt + col;
    float* dVt = (float*)a.dvt + (int64_t)h * DH * a.ld_dt + col;
#pragma unroll
    for (int d = 0; d < DH; ++d) {
      dKt[(int64_t)d * a.ld_dt] = dk[d] * scale;
      dVt[(int64_t)d * a.ld_dt] = dv[d];
    }
  }
}


template <int DH>
static hipError_t dkdv_launch(Dt dt, const AttnArgs& a, hipStream_t s) {
  if (a.S <= 0 || a.B <= 0) return hipSuccess;
  if (dt == BF16) {
    auto k = attn_bwd_dkdv_bf16_kernel<DH>;
    hipError_t e = set_lds(k, DkvCfg<DH>::LDS);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k, dim3((unsigned)((a.Sp + 127) / 128), a.H, a.B), dim3(256), DkvCfg<DH>::LDS, s, a);
  } else {
    const int lds = (2 * DH * 65 + 2 * 16 * DH + 32) * 4;
    hipError_t e = set_lds(attn_bwd_dkdv_f32_kernel<DH>, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_bwd_dkdv_f32_kernel<DH>, dim3((unsigned)(a.Sp / 64), a.H, a.B), dim3(64), lds, s, a);
  }
  return hipGetLastError();
}

hipError_t attn_bwd_dkdv(Dt dt, const AttnArgs& a, hipStream_t s) {
  if (a.dh == 64) return dkdv_launch<64>(dt, a, s);
  if (a.dh == 128) return dkdv_launch<128>(dt, a, s);
  return hipErrorInvalidValue;
}

}  // namespace bpt

// Attention backward, key-outer dK/dV kernel (bf16 MFMA and fp32 VALU variants).
#include <algorithm>

#include "attn_common.h"

namespace bpt {

// ====================================================================== backward dK dV, bf16
// Key-outer: 8 waves (two per SIMD, so one wave's VALU work overlaps the other's
// MFMAs) of 32 keys each, 256 keys per workgroup, loop over query tiles of 64 (two
// halves of 32). S = Q K^T and dP = dO V^T have the key on the lane axis, so P and dS
// feed dV^T += dO^T P and dK^T += Q^T dS directly as B operands; dO^T and Q^T
// fragments come from the token-major tiles by transposing LDS reads. Q carries
// log2(e)/sqrt(dh), and the score MFMAs start from minus the base-2 log-sum-exp of
// their query rows, so exp2 of the accumulator is P; dK = sqrt(dh)^-1 dS^T Q then
// comes out as ln(2) dS^T (Q log2(e)/sqrt(dh)).
// Query tiles are visited from the last one down, so all workgroups of a head start
// on the same tiles (and share them in L2); the diagonal tiles come last.
template <int DH>
struct DkvCfg {
  static constexpr int KSTEPS = DH / 16, DT = DH / 32;
  static constexpr int NW = 8;                      // waves per workgroup
  static constexpr int KEYS = 32 * NW;              // keys per workgroup
  static constexpr int TB = RmTile<DH>::BYTES;
  static constexpr int STAGE = 2 * TB + 2 * 64 * 4; // Q, dO tiles; -lse (base 2), -Delta
  static constexpr int NS = 4;                      // stages in the ring
  static constexpr int LDS = NS * STAGE;
  static constexpr int DPS = Ring2<DH, NW>::DPW + 2;  // copies per wave per stage
};

template <int DH>
__global__ __launch_bounds__(512, 1) void attn_bwd_dkdv_bf16_kernel(AttnArgs a) {
  using C = DkvCfg<DH>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int S = (int)a.S;
  int hh, blk;
  xcd_map_heads((int)blockIdx.x, a.H * a.B, (S + C::KEYS - 1) / C::KEYS, hh, blk);
  const int h = hh % a.H, b = hh / a.H;
  const int k0 = blk * C::KEYS;                     // causal: low key blocks have the most queries
  const int kw = k0 + 32 * wave;                    // first key of this wave
  const int key = kw + (lane & 31);

  const bf16* Qb = (const bf16*)a.q + (int64_t)b * a.S * a.ld_q + h * DH;
  const bf16* Kb = (const bf16*)a.k + (int64_t)b * a.S * a.ld_k + h * DH;
  const bf16* Vb = (const bf16*)a.v + (int64_t)b * a.S * a.ld_v + h * DH;
  const bf16* dOb = (const bf16*)a.dout + (int64_t)b * a.S * a.ld_do + h * DH;
  const float* nlse2 = a.nlse2 + ((int64_t)b * a.H + h) * a.Sp;
  const float* ndelta = a.ndelta + ((int64_t)b * a.H + h) * a.Sp;

  bf16x8 kf[C::KSTEPS], vf[C::KSTEPS];
  {
    const int kr = key < S ? key : S - 1;
#pragma unroll
    for (int kk = 0; kk < C::KSTEPS; ++kk) {
      kf[kk] = __builtin_bit_cast(bf16x8, ld16(Kb + (int64_t)kr * a.ld_k + 16 * kk + 8 * (lane >> 5)));
      vf[kk] = __builtin_bit_cast(bf16x8, ld16(Vb + (int64_t)kr * a.ld_v + 16 * kk + 8 * (lane >> 5)));
      settle(kf[kk]);
      settle(vf[kk]);
    }
  }

  const int qstart = a.causal ? k0 : 0;             // a multiple of 64
  const int ntiles = qstart < S ? (S - qstart + 63) / 64 : 0;
  const int n_diag = a.causal ? C::KEYS / 64 : 0;   // tiles jt < n_diag straddle the keys
  // iteration it visits query tile jt = ntiles - 1 - it
  auto issue = [&](int it) {
    const int qt0 = qstart + 64 * (ntiles - 1 - it);
    char* st = smem + (it % C::NS) * C::STAGE;
    ring_issue<DH, C::NW>(st, Qb, (int)a.ld_q, qt0, dOb, (int)a.ld_do, qt0, S - 1, wave, lane);
    // -lse (base 2) and -Delta of the 64 queries (indices < Sp: in bounds; rows >= S are
    // masked); every wave copies them, so that all waves count the same copies
    dma4s(nlse2 + qt0, 4u * lane, st + 2 * C::TB);
    dma4s(ndelta + qt0, 4u * lane, st + 2 * C::TB + 256);
  };

  f32x16 adv[C::DT], adk[C::DT];
#pragma unroll
  for (int t = 0; t < C::DT; ++t) adv[t] = adk[t] = f32x16{};

  auto tile = [&](int it, auto MASK) {
    const int qt0 = qstart + 64 * (ntiles - 1 - it);
    const char* qs = smem + (it % C::NS) * C::STAGE;
    const char* ds = qs + C::TB;
    const float* ls = (const float*)(qs + 2 * C::TB);
    // query offset inside the tile of register r: 32*mt + acc_row(r, lane); visible
    // iff lo <= offset <= hi
    const int lo = a.causal ? key - qt0 : 0;
    const int hi = key < S ? S - 1 - qt0 : -1;
    // the lane part of the offset moves into the bounds, so that every comparison is
    // against a constant
    const int lo4 = lo - 4 * (lane >> 5), hi4 = hi - 4 * (lane >> 5);
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      // S starts from -lse and dP from -Delta of their query rows, so the MFMAs leave
      // the exponent of P and dP - Delta
      f32x16 s, dp;
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int qi = 32 * mt + 8 * rg + 4 * (lane >> 5);
        const f32x4 l4 = *(const f32x4*)(ls + qi);
        const f32x4 d4 = *(const f32x4*)(ls + 64 + qi);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          s[4 * rg + e] = l4[e];
          dp[4 * rg + e] = d4[e];
        }
      }
#pragma unroll
      for (int kk = 0; kk < C::KSTEPS; ++kk) {
        s = mfma32x32x16(frag_rows<DH>(qs, 32 * mt, 2 * kk, lane), kf[kk], s);
        dp = mfma32x32x16(frag_rows<DH>(ds, 32 * mt, 2 * kk, lane), vf[kk], dp);
        __builtin_amdgcn_sched_barrier(0);        // bound the fragments read ahead
      }
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * rg + e;
          float p = fast_exp2(s[r]);
          if constexpr (decltype(MASK)::value) {
            const int off = 32 * mt + 8 * rg + e;
            p = (off >= lo4 && off <= hi4) ? p : 0.0f;
          }
          s[r] = p;
          dp[r] = p * dp[r];                           // dS
        }
      }
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const bf16x8 pb = acc_to_b(s, hf), sb = acc_to_b(dp, hf);
#pragma unroll
        for (int t = 0; t < C::DT; ++t) {
          adv[t] = mfma32x32x16(frag_tr<DH>(ds, 32 * mt + 16 * hf, 32 * t, lane), pb, adv[t]);
          adk[t] = mfma32x32x16(frag_tr<DH>(qs, 32 * mt + 16 * hf, 32 * t, lane), sb, adk[t]);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  };

  // Phases, each a loop over one tile body (uniform over the workgroup, so every
  // barrier is reached by all waves): the ragged last query tile (masked), the tiles
  // every key of the workgroup fully sees (unmasked), and the tiles that straddle the
  // workgroup's keys (masked); a wave skips the arithmetic of tiles entirely before
  // its keys.
  const bool ragged = ntiles > 0 && qstart + 64 * (ntiles - 1) + 63 >= S;
  const int it_a = ragged ? 1 : 0;
  const int it_b = k0 + C::KEYS > S ? it_a : std::max(it_a, ntiles - n_diag);
  auto step = [&](int it) {
    if (it + 2 < ntiles) wait_vmcnt<2 * C::DPS>();
    else if (it + 1 < ntiles) wait_vmcnt<C::DPS>();
    else wait_vmcnt<0>();
    __syncthreads();                  // stage it visible; every wave is done with stage it-1
    if (it + C::NS - 1 < ntiles) issue(it + C::NS - 1);  // into the slot of stage it-1
  };
  auto visible = [&](int it) { return !(a.causal && qstart + 64 * (ntiles - 1 - it) + 63 < kw); };
#pragma unroll
  for (int st = 0; st < C::NS - 1; ++st)
    if (st < ntiles) issue(st);
  int it = 0;
  for (; it < it_a; ++it) {
    step(it);
    if (visible(it)) tile(it, std::true_type{});
  }
  for (; it < it_b; ++it) {
    step(it);
    tile(it, std::false_type{});
  }
  for (; it < ntiles; ++it) {
    step(it);
    if (visible(it)) tile(it, std::true_type{});
  }

  if (key < a.Sp) {
    const int64_t col = (int64_t)b * a.Sp + key;
    bf16* dKt = (bf16*)a.dkt + (int64_t)h * DH * a.ld_dt + col;
    bf16* dVt = (bf16*)a.dvt + (int64_t)h * DH * a.ld_dt + col;
#pragma unroll
    for (int t = 0; t < C::DT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t d = 32 * t + acc_row(r, lane);
        dKt[d * a.ld_dt] = (bf16)(adk[t][r] * LN2);
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
  const float* ndelta = a.ndelta + ((int64_t)b * a.H + h) * a.Sp;
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
      dls[tid] = q < S ? ndelta[q] : 0.0f;
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
      const float ds = p * (dpv + dls[i]);
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
    const int64_t nblk = (a.S + DkvCfg<DH>::KEYS - 1) / DkvCfg<DH>::KEYS;
    hipLaunchKernelGGL(k, dim3((unsigned)(nblk * a.H * a.B)), dim3(64 * DkvCfg<DH>::NW), DkvCfg<DH>::LDS, s, a);
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

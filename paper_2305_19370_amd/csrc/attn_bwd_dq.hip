// Attention backward, query-outer dQ kernel (bf16 MFMA and fp32 VALU variants).
#include <algorithm>

#include "attn_common.h"

namespace bpt {

// ====================================================================== backward dQ, bf16
// Query-outer: 8 waves (two per SIMD, so one wave's VALU work overlaps the other's
// MFMAs) of 32 queries each, 256 per workgroup, loop over key tiles of 64:
// S^T = K Q^T, dP^T = V dO^T, dS^T = P^T (dP^T - Delta), dQ^T += K^T dS^T. K^T
// fragments come from the K tile by transposing LDS reads. Q carries log2(e)/sqrt(dh),
// and the score MFMAs start from minus the base-2 log-sum-exp of the lane's query, so
// exp2 of the accumulator is P.
template <int DH>
struct DqCfg {
  static constexpr int KSTEPS = DH / 16, DT = DH / 32;
  static constexpr int NW = 8;                      // waves per workgroup
  static constexpr int QROWS = 32 * NW;             // queries per workgroup
  static constexpr int TB = RmTile<DH>::BYTES;
  static constexpr int STAGE = 2 * TB;              // K and V tiles of 64 keys
  static constexpr int NS = 4;                      // stages in the ring
  static constexpr int LDS = NS * STAGE;
  static constexpr int DPS = Ring2<DH, NW>::DPW;    // copies per wave per stage
};

template <int DH>
__global__ __launch_bounds__(512, 1) void attn_bwd_dq_bf16_kernel(AttnArgs a) {
  using C = DqCfg<DH>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int S = (int)a.S;
  const int nblk = (S + C::QROWS - 1) / C::QROWS;
  int hh, blk;
  xcd_map_heads((int)blockIdx.x, a.H * a.B, nblk, hh, blk);
  const int h = hh % a.H, b = hh / a.H;
  const int qt = a.causal ? nblk - 1 - blk : blk;   // causal: the blocks with the most keys first
  const int q0 = qt * C::QROWS;
  const int qw = q0 + 32 * wave;
  const int qrow = qw + (lane & 31);
  const float scale = rsqrtf((float)DH);

  const bf16* Qb = (const bf16*)a.q + (int64_t)b * a.S * a.ld_q + h * DH;
  const bf16* Kb = (const bf16*)a.k + (int64_t)b * a.S * a.ld_k + h * DH;
  const bf16* Vb = (const bf16*)a.v + (int64_t)b * a.S * a.ld_v + h * DH;
  const bf16* dOb = (const bf16*)a.dout + (int64_t)b * a.S * a.ld_do + h * DH;

  bf16x8 qf[C::KSTEPS], dof[C::KSTEPS];
  const bool qok = qrow < S;
  const int qr = qok ? qrow : S - 1;
#pragma unroll
  for (int kk = 0; kk < C::KSTEPS; ++kk) {
    qf[kk] = __builtin_bit_cast(bf16x8, ld16(Qb + (int64_t)qr * a.ld_q + 16 * kk + 8 * (lane >> 5)));
    dof[kk] = __builtin_bit_cast(bf16x8, ld16(dOb + (int64_t)qr * a.ld_do + 16 * kk + 8 * (lane >> 5)));
    settle(qf[kk]);
    settle(dof[kk]);
  }
  const int64_t sidx = ((int64_t)b * a.H + h) * a.Sp + qr;
  const float nlse2 = qok ? a.nlse2[sidx] : 0.0f;
  const float ndl = qok ? a.ndelta[sidx] : 0.0f;   // -Delta
  settle(nlse2);
  settle(ndl);
  const int kv_last = !qok ? -1 : (a.causal ? qrow : S - 1);   // last key this query may see

  const int kv_end = a.causal ? (q0 + C::QROWS < S ? q0 + C::QROWS : S) : S;
  const int ntiles = (kv_end + 63) / 64;
  const RingOff<DH, C::NW> roff = ring_offsets<DH, C::NW>((int)a.ld_k, (int)a.ld_v, wave, lane);
  auto issue = [&](int j) {
    char* st = smem + (j % C::NS) * C::STAGE;
    if (64 * j + 63 < S) ring_issue_full<DH, C::NW>(st, Kb, (int)a.ld_k, 64 * j, Vb, (int)a.ld_v, 64 * j, roff, wave);
    else ring_issue<DH, C::NW>(st, Kb, (int)a.ld_k, 64 * j, Vb, (int)a.ld_v, 64 * j, S - 1, wave, lane);
  };

  f32x16 acc[C::DT];                                // dQ^T of the wave's queries
#pragma unroll
  for (int t = 0; t < C::DT; ++t) acc[t] = f32x16{};

  auto tile = [&](int j, auto MASK) {
    const int kv0 = 64 * j;
    const char* kt = smem + (j % C::NS) * C::STAGE;
    const char* vt = kt + C::TB;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      f32x16 s, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] = nlse2;                                // the MFMAs leave the exponent of P
        dp[r] = ndl;                                 // and dP^T - Delta
      }
#pragma unroll
      for (int kk = 0; kk < C::KSTEPS; ++kk) {
        s = mfma32x32x16(frag_rows<DH>(kt, 32 * mt, 2 * kk, lane), qf[kk], s);
        dp = mfma32x32x16(frag_rows<DH>(vt, 32 * mt, 2 * kk, lane), dof[kk], dp);
      }
      // key offset of register r: acc_row(r, lane); the lane part moves into the limit
      // so that every comparison is against a constant
      const int lim = kv_last - kv0 - 32 * mt - 4 * (lane >> 5);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = fast_exp2(s[r]);
        if constexpr (decltype(MASK)::value) p = (8 * (r >> 2) + (r & 3) <= lim) ? p : 0.0f;
        s[r] = p * dp[r];                           // dS^T
      }
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const bf16x8 sb = acc_to_b(s, hf);
#pragma unroll
        for (int t = 0; t < C::DT; ++t)
          acc[t] = mfma32x32x16(frag_tr<DH>(kt, 32 * mt + 16 * hf, 32 * t, lane), sb, acc[t]);
      }
    }
  };

  // Key tiles every query of the workgroup fully sees take the unmasked body; the
  // diagonal and ragged tiles (and every tile of a block with queries past the end)
  // take the masked one. Every barrier is reached by all waves; a wave skips the
  // arithmetic of tiles entirely after its queries.
  int n_full = a.causal ? std::min(ntiles, (q0 + 1) / 64) : ntiles;
  n_full = std::min(n_full, S / 64);
  if (q0 + C::QROWS > S) n_full = 0;
#pragma unroll
  for (int st = 0; st < C::NS - 1; ++st)
    if (st < ntiles) issue(st);
  auto step = [&](int j) {
    // stage j has landed once at most the stages issued after it are pending
    if (j + 2 < ntiles) wait_vmcnt<2 * C::DPS>();
    else if (j + 1 < ntiles) wait_vmcnt<C::DPS>();
    else wait_vmcnt<0>();
    __syncthreads();                  // stage j visible; every wave is done with stage j-1
    if (j + C::NS - 1 < ntiles) issue(j + C::NS - 1);   // into the slot of stage j-1
  };
  int j = 0;
  for (; j < n_full; ++j) {
    step(j);
    tile(j, std::false_type{});
  }
  for (; j < ntiles; ++j) {
    step(j);
    if (!(a.causal && 64 * j > qw + 31)) tile(j, std::true_type{});
  }

  if (qrow < a.Sp) {
    bf16* dQt = (bf16*)a.dqt + (int64_t)h * DH * a.ld_dt + (int64_t)b * a.Sp + qrow;
#pragma unroll
    for (int t = 0; t < C::DT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int d = 32 * t + acc_row(r, lane);
        dQt[(int64_t)d * a.ld_dt] = (bf16)(qok ? acc[t][r] * scale : 0.0f);
      }
  }
}

template <int DH>
__global__ __launch_bounds__(64) void attn_bwd_dq_f32_kernel(AttnArgs a) {
  extern __shared__ float fsm[];
  float* Qown = fsm;                       // [DH][65]
  float* dOown = Qown + DH * 65;           // [DH][65]
  float* Ks = dOown + DH * 65;             // [16][DH]
  float* Vs = Ks + 16 * DH;                // [16][DH]
  const int tid = threadIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int64_t S = a.S, q0 = (int64_t)blockIdx.x * 64, q = q0 + tid;
  const float scale = rsqrtf((float)DH);
  const float* Qp = (const float*)a.q + (int64_t)h * DH;
  const float* Kp = (const float*)a.k + (int64_t)h * DH;
  const float* Vp = (const float*)a.v + (int64_t)h * DH;
  const float* dOp = (const float*)a.dout + (int64_t)h * DH;
  const int64_t sidx = ((int64_t)b * a.H + h) * a.Sp + q;
  const float lq = q < S ? a.lse[sidx] : 0.0f;
  const float ndl = q < S ? a.ndelta[sidx] : 0.0f;
  for (int d = 0; d < DH; ++d) {
    Qown[d * 65 + tid] = q < S ? Qp[(b * S + q) * a.ld_q + d] : 0.0f;
    dOown[d * 65 + tid] = q < S ? dOp[(b * S + q) * a.ld_do + d] : 0.0f;
  }
  float dq[DH];
#pragma unroll
  for (int d = 0; d < DH; ++d) dq[d] = 0.0f;
  const int64_t kv_end = a.causal ? (q0 + 64 < S ? q0 + 64 : S) : S;
  for (int64_t kv0 = 0; kv0 < kv_end; kv0 += 16) {
    __syncthreads();
    for (int i = tid; i < 16 * DH; i += 64) {
      const int r = i / DH, d = i % DH;
      const int64_t kv = kv0 + r;
      Ks[i] = kv < S ? Kp[(b * S + kv) * a.ld_k + d] : 0.0f;
      Vs[i] = kv < S ? Vp[(b * S + kv) * a.ld_v + d] : 0.0f;
    }
    __syncthreads();
    for (int jj = 0; jj < 16; ++jj) {
      const int64_t kv = kv0 + jj;
      float sv = 0.0f, dpv = 0.0f;
#pragma unroll
      for (int d = 0; d < DH; ++d) {
        sv = fmaf(Qown[d * 65 + tid], Ks[jj * DH + d], sv);
        dpv = fmaf(dOown[d * 65 + tid], Vs[jj * DH + d], dpv);
      }
      const bool ok = q < S && kv < S && !(a.causal && kv > q);
      const float p = ok ? __expf(sv * scale - lq) : 0.0f;
      const float ds = p * (dpv + ndl);
#pragma unroll
      for (int d = 0; d < DH; ++d) dq[d] = fmaf(ds, Ks[jj * DH + d], dq[d]);
    }
  }
  if (q < a.Sp) {
    float* dQt = (float*)a.dqt + (int64_t)h * DH * a.ld_dt + (int64_t)b * a.Sp + q;
    const bool real = q < S;
#pragma unroll
    for (int d = 0; d < DH; ++d) dQt[(int64_t)d * a.ld_dt] = real ? dq[d] * scale : 0.0f;
  }
}


template <int DH>
static hipError_t dq_launch(Dt dt, const AttnArgs& a, hipStream_t s) {
  if (a.S <= 0 || a.B <= 0) return hipSuccess;
  if (dt == BF16) {
    auto k = attn_bwd_dq_bf16_kernel<DH>;
    hipError_t e = set_lds(k, DqCfg<DH>::LDS);
    if (e != hipSuccess) return e;
    const int64_t nblk = (a.S + DqCfg<DH>::QROWS - 1) / DqCfg<DH>::QROWS;
    hipLaunchKernelGGL(k, dim3((unsigned)(nblk * a.H * a.B)), dim3(64 * DqCfg<DH>::NW), DqCfg<DH>::LDS, s, a);
  } else {
    const int lds = (2 * DH * 65 + 2 * 16 * DH) * 4;
    hipError_t e = set_lds(attn_bwd_dq_f32_kernel<DH>, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_bwd_dq_f32_kernel<DH>, dim3((unsigned)(a.Sp / 64), a.H, a.B), dim3(64), lds, s, a);
  }
  return hipGetLastError();
}

hipError_t attn_bwd_dq(Dt dt, const AttnArgs& a, hipStream_t s) {
  if (a.dh == 64) return dq_launch<64>(dt, a, s);
  if (a.dh == 128) return dq_launch<128>(dt, a, s);
  return hipErrorInvalidValue;
}

}  // namespace bpt

// Blockwise attention for the BPT layer (paper, Section 3, eq. 3): for each query
// tile, iterate over key/value tiles keeping a running row maximum and row sum,
// rescale the running numerator by exp(old_max - new_max), and normalise once at
// the end. The backward rebuilds each probability tile from the saved
// log-sum-exp, P = exp(s - lse), so no S x S matrix is ever stored.
//
// bf16 kernels (gfx950 MFMA 32x32x16, fp32 accumulation, wave64):
//  * scores are computed transposed, S^T[kv, q] = K Q^T, so that each lane owns a
//    single query column: the row max / row sum of the softmax reduce over the
//    lane's own accumulator registers plus one exchange with lane ^ 32;
//  * the accumulator of S^T is, after exp and bf16 rounding, directly the B
//    operand of O^T[d, q] += V^T[d, kv] P^T[kv, q] (the K index order inside one
//    MFMA is permuted consistently on the A side), so P never touches LDS;
//  * K and V tiles of 64 keys (token-major, as the projections write them) stream
//    through a 4-stage LDS ring filled by direct global->LDS copies; V^T fragments
//    come from the V tile by transposing LDS reads;
//  * 8 waves of 32 queries share each stage; two waves per SIMD let one wave's
//    softmax run while the other's MFMAs do;
//  * Q arrives multiplied by log2(e)/sqrt(dh) (the projection's epilogue applies it),
//    so scores are base-2 logits, and the score MFMAs start from minus the row's
//    reference maximum: exp2 of the accumulator is the weight, and the backward
//    kernels start them from minus the base-2 log-sum-exp in the same way.
// fp32 kernels: one query (or key) row per thread with VALU FMAs; used by the
// fp32 parity workload.
#include <algorithm>

#include "attn_common.h"

namespace bpt {

// ====================================================================== forward, bf16
// 8 waves (two per SIMD, so that one wave's softmax overlaps the other's MFMAs), 32
// queries per wave, 256 per workgroup; all waves share the K/V stages of the ring.
template <int DH>
struct FwdCfg {
  static constexpr int KSTEPS = DH / 16, DT = DH / 32;
  static constexpr int NW = 8;                      // waves per workgroup
  static constexpr int QROWS = 32 * NW;             // queries per workgroup
  static constexpr int TB = RmTile<DH>::BYTES;
  static constexpr int STAGE = 2 * TB;              // K and V tiles of 64 keys
  static constexpr int NS = 4;                      // stages in the ring
  static constexpr int LDS = NS * STAGE;
  static constexpr int DPS = Ring2<DH, NW>::DPW;    // copies per wave per stage
};

// Largest exponent growth (base 2) tolerated before the running numerator is
// rescaled: exp-weights stay <= 2^8, and the final division uses the same
// reference maximum, so the result is unchanged.
static constexpr float RESCALE_LOG2 = 8.0f;
// Largest per-lane sum of one tile's exp-weights (32 keys) accepted without computing
// the tile's maximum.
static constexpr float SUM_MAX = 65536.0f;

template <int DH>
__global__ __launch_bounds__(512, 1) void attn_fwd_bf16_kernel(AttnArgs a) {
  using C = FwdCfg<DH>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int S = (int)a.S;
  const int nblk = (int)((a.q_end - a.q_begin + C::QROWS - 1) / C::QROWS);
  int hh, blk;
  xcd_map((int)blockIdx.x, a.H * a.nb, hh, blk);
  const int h = hh % a.H, b = a.b_begin + hh / a.H;
  const int qt = a.causal ? nblk - 1 - blk : blk;   // causal: the blocks with the most keys first
  const int q0 = (int)a.q_begin + qt * C::QROWS;
  const int qw = q0 + 32 * wave;                    // first query of this wave
  const int qrow = qw + (lane & 31);

  const bf16* Qb = (const bf16*)a.q + (int64_t)b * a.S * a.ld_q + h * DH;
  const bf16* Kb = (const bf16*)a.k + (int64_t)b * a.S * a.ld_k + h * DH;
  const bf16* Vb = (const bf16*)a.v + (int64_t)b * a.S * a.ld_v + h * DH;

  // the wave's 32 queries (one per lane column) as B operands
  bf16x8 qf[C::KSTEPS];
  const int qr = qrow < S ? qrow : S - 1;
#pragma unroll
  for (int kk = 0; kk < C::KSTEPS; ++kk) {
    qf[kk] = __builtin_bit_cast(bf16x8, ld16(Qb + (int64_t)qr * a.ld_q + 16 * kk + 8 * (lane >> 5)));
    settle(qf[kk]);
  }
  const int kv_last = a.causal ? qr : S - 1;       // last key this lane's query may see

  const int kv_end = a.causal ? (q0 + C::QROWS < S ? q0 + C::QROWS : S) : S;
  const int ntiles = (kv_end + 63) / 64;
  const RingOff<DH, C::NW> roff = ring_offsets<DH, C::NW>((int)a.ld_k, (int)a.ld_v, wave, lane);
  auto issue = [&](int j) {
    char* st = smem + (j % C::NS) * C::STAGE;
    if (64 * j + 63 < S) ring_issue_full<DH, C::NW>(st, Kb, (int)a.ld_k, 64 * j, Vb, (int)a.ld_v, 64 * j, roff, wave);
    else ring_issue<DH, C::NW>(st, Kb, (int)a.ld_k, 64 * j, Vb, (int)a.ld_v, 64 * j, S - 1, wave, lane);
  };

  f32x16 acc[C::DT];                                // O^T of the wave's queries
#pragma unroll
  for (int t = 0; t < C::DT; ++t) acc[t] = f32x16{};
  // Q carries log2(e)/sqrt(dh), so the scores are base-2 logits. ref is the row's
  // reference maximum (base 2); the score MFMAs start from -ref, so that they leave
  // score - ref, the exponent of the weight, with no VALU work per score.
  float ref = 0.0f, l_run = 0.0f;
  f32x16 sinit = f32x16{};

  // Weights exp2(t - d) of the tile's exponents t = score - ref, with d = 0 or d the
  // lane's maximum of t (shared with lane ^ 32); their sum over the lane's 32 keys.
  auto weights = [&](const f32x16 (&t)[2], float d, f32x16 (&p)[2]) {
    float rs = 0.0f;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        p[mt][r] = fast_exp2(t[mt][r] - d);
        rs += p[mt][r];
      }
    return rs;
  };
  auto tile_max = [&](const f32x16 (&t)[2]) {
    float mx = NEG_INF;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, t[mt][r]);
    return max_halves(mx);
  };
  // Move the reference up by d (per lane) and rescale numerator and sum to it.
  auto move_ref = [&](float d) {
    if (__ballot(d != 0.0f)) {
      asm volatile("" ::: "memory");                       // keep the rescale behind the branch
      const float corr = fast_exp2(-d);
      l_run *= corr;
#pragma unroll
      for (int t = 0; t < C::DT; ++t) acc[t] *= corr;
      ref += d;
#pragma unroll
      for (int r = 0; r < 16; ++r) sinit[r] = -ref;
    }
  };

  // EXACT: the tile sets the reference to its row maximum (the first tile of every
  // wave: it holds key 0, which every query sees, so every reference ends up finite).
  // Otherwise the weights are taken against the current reference directly, and the
  // tile maximum is only computed when a lane's sum of weights exceeds SUM_MAX (a
  // score above the reference by more than about log2(SUM_MAX / 32)); the reference
  // then moves when the maximum is above it by more than RESCALE_LOG2. Every weight
  // stays <= SUM_MAX, and no row sum can vanish, the first tile having left a weight
  // of 1 at its maximum.
  auto tile = [&](int j, auto MASK, auto EXACT) {
    const int kv0 = 64 * j;
    const char* kt = smem + (j % C::NS) * C::STAGE;
    const char* vt = kt + C::TB;
    // K fragments of the whole tile, read at once so that only the first MFMA waits
    bf16x8 kf[C::KSTEPS][2];
#pragma unroll
    for (int kk = 0; kk < C::KSTEPS; ++kk)
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) kf[kk][mt] = frag_rows<DH>(kt, 32 * mt, 2 * kk, lane);
    __builtin_amdgcn_sched_barrier(0);
    // T^T[key, query] = K Q^T - ref
    f32x16 t[2] = {sinit, sinit};
#pragma unroll
    for (int kk = 0; kk < C::KSTEPS; ++kk)
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) t[mt] = mfma32x32x16(kf[kk][mt], qf[kk], t[mt]);
    if constexpr (decltype(MASK)::value) {
      // key offset of register r: 32 mt + acc_row(r, lane); the lane part moves into the
      // limit so that every comparison is against a constant
      const int lim = kv_last - kv0 - 4 * (lane >> 5);
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) t[mt][r] = (32 * mt + 8 * (r >> 2) + (r & 3) <= lim) ? t[mt][r] : NEG_INF;
    }
    f32x16 p[2];
    float rs;
    if constexpr (decltype(EXACT)::value) {
      const float mx = tile_max(t);                        // finite: key 0 is in this tile
      ref += mx;
#pragma unroll
      for (int r = 0; r < 16; ++r) sinit[r] = -ref;
      rs = weights(t, mx, p);
    } else {
      rs = weights(t, 0.0f, p);
      if (__ballot(!(rs <= SUM_MAX))) {
        asm volatile("" ::: "memory");
        const float mx = tile_max(t);
        const float d = mx > RESCALE_LOG2 ? mx : 0.0f;
        move_ref(d);
        rs = weights(t, d, p);
      }
    }
    l_run += rs;
    // O^T[d, query] += V^T P^T, V^T fragments by transposing reads of the V tile
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const bf16x8 pb = acc_to_b(p[mt], hf);
#pragma unroll
        for (int t2 = 0; t2 < C::DT; ++t2)
          acc[t2] = mfma32x32x16(frag_tr<DH>(vt, 32 * mt + 16 * hf, 32 * t2, lane), pb, acc[t2]);
      }
  };

  // Key tiles every query of the workgroup fully sees take the unmasked body; the
  // diagonal and ragged tiles take the masked one. Every barrier is reached by all
  // waves; a wave skips the arithmetic of tiles entirely after its queries.
  int n_full = a.causal ? std::min(ntiles, (q0 + 1) / 64) : ntiles;
  n_full = std::min(n_full, S / 64);
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
  constexpr std::true_type Y{};
  constexpr std::false_type N{};
  int j = 0;
  if (ntiles > 0) {                   // tile 0 holds key 0, which every query sees
    step(0);
    if (n_full > 0) tile(0, N, Y);
    else tile(0, Y, Y);
    j = 1;
  }
  for (; j < n_full; ++j) {
    step(j);
    tile(j, N, N);
  }
  for (; j < ntiles; ++j) {
    step(j);
    if (!(a.causal && 64 * j > qw + 31)) tile(j, Y, N);
  }

  const float l_tot = sum_halves(l_run);
  if (qrow < (int)a.q_end && qrow < S) {
    const float inv = 1.0f / l_tot;
    bf16* Op = (bf16*)a.o + ((int64_t)b * a.S + qrow) * a.ld_o + h * DH;
#pragma unroll
    for (int t = 0; t < C::DT; ++t)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        bf16x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (bf16)(acc[t][4 * rg + e] * inv);
        *(bf16x4*)(Op + 32 * t + 8 * rg + 4 * (lane >> 5)) = v;
      }
    if (lane < 32) a.lse[((int64_t)b * a.H + h) * a.Sp + qrow] = (ref + log2f(l_tot)) * LN2;
  }
}

// ====================================================================== fp32 kernels
template <int DH>
__global__ __launch_bounds__(64) void attn_fwd_f32_kernel(AttnArgs a) {
  __shared__ float Ks[32][DH + 1], Vs[32][DH + 1];
  const int tid = threadIdx.x, h = blockIdx.y, b = a.b_begin + blockIdx.z;
  const int64_t S = a.S;
  const int64_t q0 = a.q_begin + (int64_t)blockIdx.x * 64, q = q0 + tid;
  const float scale = rsqrtf((float)DH), c = scale * LOG2E;
  const float* Qp = (const float*)a.q + (int64_t)h * DH;
  const float* Kp = (const float*)a.k + (int64_t)h * DH;
  const float* Vp = (const float*)a.v + (int64_t)h * DH;
  float qr[DH], acc[DH];
#pragma unroll
  for (int d = 0; d < DH; ++d) {
    qr[d] = q < S ? Qp[(b * S + q) * a.ld_q + d] : 0.0f;
    acc[d] = 0.0f;
  }
  float m_run = NEG_INF, l_run = 0.0f;
  const int64_t kv_end = a.causal ? (q0 + 64 < S ? q0 + 64 : S) : S;
  for (int64_t kv0 = 0; kv0 < kv_end; kv0 += 32) {
    for (int i = tid; i < 32 * DH; i += 64) {
      const int r = i / DH, d = i % DH;
      const int64_t kv = kv0 + r;
      Ks[r][d] = kv < S ? Kp[(b * S + kv) * a.ld_k + d] : 0.0f;
      Vs[r][d] = kv < S ? Vp[(b * S + kv) * a.ld_v + d] : 0.0f;
    }
    __syncthreads();
    float sc[32];
    float mx = NEG_INF;
#pragma unroll
    for (int jj = 0; jj < 32; ++jj) {
      float sv = 0.0f;
#pragma unroll
      for (int d = 0; d < DH; ++d) sv = fmaf(qr[d], Ks[jj][d], sv);
      const int64_t kv = kv0 + jj;
      if (kv >= S || (a.causal && kv > q)) sv = NEG_INF;
      sc[jj] = sv;
      mx = fmaxf(mx, sv);
    }
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == NEG_INF) ? 0.0f : m_new;
    const float corr = exp2f((m_run - m_use) * c);
    l_run *= corr;
#pragma unroll
    for (int d = 0; d < DH; ++d) acc[d] *= corr;
#pragma unroll
    for (int jj = 0; jj < 32; ++jj) {
      const float p = exp2f((sc[jj] - m_use) * c);
      l_run += p;
#pragma unroll
      for (int d = 0; d < DH; ++d) acc[d] = fmaf(p, Vs[jj][d], acc[d]);
    }
    m_run = m_new;
    __syncthreads();
  }
  if (q < a.q_end && q < S) {
    float* Op = (float*)a.o + (b * S + q) * a.ld_o + (int64_t)h * DH;
    const float inv = 1.0f / l_run;
#pragma unroll
    for (int d = 0; d < DH; ++d) Op[d] = acc[d] * inv;
    a.lse[((int64_t)b * a.H + h) * a.Sp + q] = m_run * scale + logf(l_run);
  }
}


template <int DH>
static hipError_t fwd_launch(Dt dt, const AttnArgs& a, hipStream_t s) {
  const int64_t nq = a.q_end - a.q_begin;
  if (nq <= 0 || a.nb <= 0) return hipSuccess;
  if (dt == BF16) {
    auto kern = attn_fwd_bf16_kernel<DH>;
    hipError_t e = set_lds(kern, FwdCfg<DH>::LDS);
    if (e != hipSuccess) return e;
    const int64_t nblk = (nq + FwdCfg<DH>::QROWS - 1) / FwdCfg<DH>::QROWS;
    hipLaunchKernelGGL(kern, dim3((unsigned)(nblk * a.H * a.nb)), dim3(64 * FwdCfg<DH>::NW), FwdCfg<DH>::LDS, s, a);
  } else {
    hipLaunchKernelGGL(attn_fwd_f32_kernel<DH>, dim3((unsigned)((nq + 63) / 64), a.H, a.nb),
                       dim3(64), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t attn_fwd(Dt dt, const AttnArgs& a, hipStream_t s) {
  if (a.dh == 64) return fwd_launch<64>(dt, a, s);
  if (a.dh == 128) return fwd_launch<128>(dt, a, s);
  return hipErrorInvalidValue;
}

}  // namespace bpt

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
//  * K and V^T tiles of 64 keys are staged in double-buffered LDS with a 16-byte
//    chunk XOR swizzle; scores use exp2 with log2(e)/sqrt(dh) folded in one FMA.
// fp32 kernels: one query (or key) row per thread with VALU FMAs; used by the
// fp32 parity workload.
#include "common.h"
#include "internal.h"

namespace bpt {

static constexpr float LOG2E = 1.4426950408889634f;
static constexpr float LN2 = 0.6931471805599453f;
static constexpr float NEG_INF = -__builtin_inff();

// Row-major tile with rows of DH bf16 (DH/8 chunks of 16 bytes).
template <int DH>
BPT_DEV int rm_addr(int row, int kc) { return row * (DH * 2) + ((kc ^ (row & 7)) << 4); }
// Feature-major tile [DH][64]: 64 tokens = 8 chunks per row.
BPT_DEV int fm_addr(int row, int tok) { return row * 128 + (((tok >> 3) ^ (row & 7)) << 4) + ((tok & 7) << 1); }

BPT_DEV u32x4 ld16(const void* p) { return *(const u32x4*)p; }

// A-operand fragment for a contraction over 16 tokens starting at `tok0` of a
// feature-major LDS tile: lane l supplies row (row0 + l%32) at tokens
// tok0 + 4*(l/32) + {0..3} and tok0 + 8 + 4*(l/32) + {0..3}, matching the order in
// which an MFMA accumulator hands its rows to the next MFMA as a B operand.
BPT_DEV bf16x8 fm_frag(const char* tile, int row, int tok0, int lane) {
  const int t = tok0 + 4 * (lane >> 5);
  const u32x2 lo = *(const u32x2*)(tile + fm_addr(row, t));
  const u32x2 hi = *(const u32x2*)(tile + fm_addr(row, t + 8));
  u32x4 v = {lo[0], lo[1], hi[0], hi[1]};
  return __builtin_bit_cast(bf16x8, v);
}

// Registers 8*hf .. 8*hf+7 of an accumulator as a bf16 B operand.
BPT_DEV bf16x8 acc_to_b(const f32x16& s, int hf) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (bf16)s[8 * hf + i];
  return r;
}

// ====================================================================== forward, bf16
template <int DH>
struct FwdCfg {
  static constexpr int KC = DH / 8, KSTEPS = DH / 16, DT = DH / 32;
  static constexpr int KBYTES = 64 * DH * 2, VBYTES = DH * 64 * 2;
  static constexpr int STAGE = KBYTES + VBYTES;
  static constexpr int LDS = 2 * STAGE;
  static constexpr int CK = 64 * KC / 256, CV = DH * 8 / 256;   // 16-byte chunks per thread
};

template <int DH>
__global__ __launch_bounds__(256, 2) void attn_fwd_bf16_kernel(AttnArgs a) {
  using C = FwdCfg<DH>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = blockIdx.y, b = a.b_begin + blockIdx.z;
  const int64_t S = a.S;
  const int64_t q0 = a.q_begin + (int64_t)blockIdx.x * 128;
  const int64_t qw = q0 + 32 * wave;
  const int64_t qrow = qw + (lane & 31);
  const float scale = rsqrtf((float)DH);
  const float c = scale * LOG2E;

  const bf16* Qp = (const bf16*)a.q + (int64_t)h * DH;
  const bf16* Kp = (const bf16*)a.k + (int64_t)h * DH;
  const bf16* Vt = (const bf16*)a.vt + (int64_t)h * DH * a.ld_vt + (int64_t)b * a.Sp;

  bf16x8 qf[C::KSTEPS];
#pragma unroll
  for (int kk = 0; kk < C::KSTEPS; ++kk) {
    u32x4 v = {0, 0, 0, 0};
    if (qrow < S) v = ld16(Qp + (b * S + qrow) * a.ld_q + 16 * kk + 8 * (lane >> 5));
    qf[kk] = __builtin_bit_cast(bf16x8, v);
  }

  const int64_t kv_end = a.causal ? (q0 + 128 < S ? q0 + 128 : S) : S;
  const int ntiles = (int)((kv_end + 63) / 64);

  u32x4 rk[C::CK], rv[C::CV];
  auto gload = [&](int j) {
    const int64_t kv0 = (int64_t)j * 64;
#pragma unroll
    for (int i = 0; i < C::CK; ++i) {
      const int cc = tid + 256 * i, row = cc / C::KC, kc = cc % C::KC;
      const int64_t kv = kv0 + row;
      rk[i] = kv < S ? ld16(Kp + (b * S + kv) * a.ld_k + kc * 8) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int i = 0; i < C::CV; ++i) {
      const int cc = tid + 256 * i, d = cc >> 3, ch = cc & 7;
      rv[i] = ld16(Vt + (int64_t)d * a.ld_vt + kv0 + ch * 8);   // kv0 + 64 <= Sp; pad is zero
    }
  };
  auto lstore = [&](int buf) {
    char* kt = smem + buf * C::STAGE;
    char* vt = kt + C::KBYTES;
#pragma unroll
    for (int i = 0; i < C::CK; ++i) {
      const int cc = tid + 256 * i;
      *(u32x4*)(kt + rm_addr<DH>(cc / C::KC, cc % C::KC)) = rk[i];
    }
#pragma unroll
    for (int i = 0; i < C::CV; ++i) {
      const int cc = tid + 256 * i, d = cc >> 3, ch = cc & 7;
      *(u32x4*)(vt + d * 128 + ((ch ^ (d & 7)) << 4)) = rv[i];
    }
  };

  f32x16 acc[C::DT];
#pragma unroll
  for (int t = 0; t < C::DT; ++t) acc[t] = f32x16{};
  float m_run = NEG_INF, l_run = 0.0f;

  if (ntiles > 0) {
    gload(0);
    lstore(0);
  }
  __syncthreads();
  for (int j = 0; j < ntiles; ++j) {
    const int buf = j & 1;
    if (j + 1 < ntiles) gload(j + 1);
    const int64_t kv0 = (int64_t)j * 64;
    const bool skip = a.causal && kv0 > qw + 31;
    if (!skip) {
      const char* kt = smem + buf * C::STAGE;
      const char* vt = kt + C::KBYTES;
      f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int kk = 0; kk < C::KSTEPS; ++kk) {
        const int kc = 2 * kk + (lane >> 5);
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
          const bf16x8 af = *(const bf16x8*)(kt + rm_addr<DH>(32 * mt + (lane & 31), kc));
          s[mt] = mfma32x32x16(af, qf[kk], s[mt]);
        }
      }
      const bool need_mask = (a.causal && kv0 + 63 > qw) || (kv0 + 64 > S);
      if (need_mask) {
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int64_t kv = kv0 + 32 * mt + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (kv >= S || (a.causal && kv > qrow)) s[mt][r] = NEG_INF;
          }
      }
      float mx = NEG_INF;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[mt][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx);
      const float m_use = (m_new == NEG_INF) ? 0.0f : m_new;
      const float corr = exp2f((m_run - m_use) * c);
      const float mc = m_use * c;
      float rs = 0.0f;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = exp2f(fmaf(s[mt][r], c, -mc));
          s[mt][r] = p;
          rs += p;
        }
      l_run = l_run * corr + rs;
      m_run = m_new;
#pragma unroll
      for (int t = 0; t < C::DT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][r] *= corr;
      bf16x8 pb[2][2];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) pb[mt][hf] = acc_to_b(s[mt], hf);
#pragma unroll
      for (int t = 0; t < C::DT; ++t)
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int hf = 0; hf < 2; ++hf) {
            const bf16x8 af = fm_frag(vt, 32 * t + (lane & 31), 32 * mt + 16 * hf, lane);
            acc[t] = mfma32x32x16(af, pb[mt][hf], acc[t]);
          }
    }
    if (j + 1 < ntiles) lstore(buf ^ 1);
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (qrow < a.q_end && qrow < S) {
    const float inv = 1.0f / l_tot;
    bf16* Op = (bf16*)a.o + (b * S + qrow) * a.ld_o + (int64_t)h * DH;
#pragma unroll
    for (int t = 0; t < C::DT; ++t)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        bf16x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (bf16)(acc[t][4 * rg + e] * inv);
        *(bf16x4*)(Op + 32 * t + 8 * rg + 4 * (lane >> 5)) = v;
      }
    if (lane < 32) a.lse[((int64_t)b * a.H + h) * a.Sp + qrow] = m_run * scale + logf(l_tot);
  }
}

// ====================================================================== backward dQ, bf16
// Query-outer: per query tile, loop over key tiles; S^T = K Q^T, dP^T = V dO^T,
// dS^T = P^T (dP^T - Delta), dQ^T += K^T dS^T.
template <int DH>
struct DqCfg {
  static constexpr int KC = DH / 8, KSTEPS = DH / 16, DT = DH / 32;
  static constexpr int RBYTES = 64 * DH * 2;
  static constexpr int STAGE = 3 * RBYTES;            // K, V row-major; K^T feature-major
  static constexpr int LDS = 2 * STAGE;
  static constexpr int CR = 64 * KC / 256, CT = DH * 8 / 256;
};

template <int DH>
__global__ __launch_bounds__(256, 1) void attn_bwd_dq_bf16_kernel(AttnArgs a) {
  using C = DqCfg<DH>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t S = a.S;
  const int64_t q0 = (int64_t)blockIdx.x * 128;
  const int64_t qw = q0 + 32 * wave;
  const int64_t qrow = qw + (lane & 31);
  const float scale = rsqrtf((float)DH);
  const float c = scale * LOG2E;

  const bf16* Qp = (const bf16*)a.q + (int64_t)h * DH;
  const bf16* Kp = (const bf16*)a.k + (int64_t)h * DH;
  const bf16* Vp = (const bf16*)a.v + (int64_t)h * DH;
  const bf16* dOp = (const bf16*)a.dout + (int64_t)h * DH;
  const bf16* Kt = (const bf16*)a.kt + (int64_t)h * DH * a.ld_kt + (int64_t)b * a.Sp;

  bf16x8 qf[C::KSTEPS], dof[C::KSTEPS];
#pragma unroll
  for (int kk = 0; kk < C::KSTEPS; ++kk) {
    u32x4 v = {0, 0, 0, 0}, w = {0, 0, 0, 0};
    if (qrow < S) {
      v = ld16(Qp + (b * S + qrow) * a.ld_q + 16 * kk + 8 * (lane >> 5));
      w = ld16(dOp + (b * S + qrow) * a.ld_do + 16 * kk + 8 * (lane >> 5));
    }
    qf[kk] = __builtin_bit_cast(bf16x8, v);
    dof[kk] = __builtin_bit_cast(bf16x8, w);
  }
  const int64_t sidx = ((int64_t)b * a.H + h) * a.Sp + qrow;
  const float lse2 = qrow < S ? a.lse[sidx] * LOG2E : 0.0f;
  const float dl = qrow < S ? a.delta[sidx] : 0.0f;

  const int64_t kv_end = a.causal ? (q0 + 128 < S ? q0 + 128 : S) : S;
  const int ntiles = (int)((kv_end + 63) / 64);

  u32x4 rk[C::CR], rvv[C::CR], rt[C::CT];
  auto gload = [&](int j) {
    const int64_t kv0 = (int64_t)j * 64;
#pragma unroll
    for (int i = 0; i < C::CR; ++i) {
      const int cc = tid + 256 * i, row = cc / C::KC, kc = cc % C::KC;
      const int64_t kv = kv0 + row;
      rk[i] = kv < S ? ld16(Kp + (b * S + kv) * a.ld_k + kc * 8) : u32x4{0, 0, 0, 0};
      rvv[i] = kv < S ? ld16(Vp + (b * S + kv) * a.ld_v + kc * 8) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int i = 0; i < C::CT; ++i) {
      const int cc = tid + 256 * i, d = cc >> 3, ch = cc & 7;
      rt[i] = ld16(Kt + (int64_t)d * a.ld_kt + kv0 + ch * 8);
    }
  };
  auto lstore = [&](int buf) {
    char* ks = smem + buf * C::STAGE;
    char* vs = ks + C::RBYTES;
    char* kts = vs + C::RBYTES;
#pragma unroll
    for (int i = 0; i < C::CR; ++i) {
      const int cc = tid + 256 * i;
      *(u32x4*)(ks + rm_addr<DH>(cc / C::KC, cc % C::KC)) = rk[i];
      *(u32x4*)(vs + rm_addr<DH>(cc / C::KC, cc % C::KC)) = rvv[i];
    }
#pragma unroll
    for (int i = 0; i < C::CT; ++i) {
      const int cc = tid + 256 * i, d = cc >> 3, ch = cc & 7;
      *(u32x4*)(kts + d * 128 + ((ch ^ (d & 7)) << 4)) = rt[i];
    }
  };

  f32x16 acc[C::DT];
#pragma unroll
  for (int t = 0; t < C::DT; ++t) acc[t] = f32x16{};

  if (ntiles > 0) {
    gload(0);
    lstore(0);
  }
  __syncthreads();
  for (int j = 0; j < ntiles; ++j) {
    const int buf = j & 1;
    if (j + 1 < ntiles) gload(j + 1);
    const int64_t kv0 = (int64_t)j * 64;
    const bool skip = a.causal && kv0 > qw + 31;
    if (!skip) {
      const char* ks = smem + buf * C::STAGE;
      const char* vs = ks + C::RBYTES;
      const char* kts = vs + C::RBYTES;
      f32x16 s[2] = {f32x16{}, f32x16{}}, dp[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int kk = 0; kk < C::KSTEPS; ++kk) {
        const int kc = 2 * kk + (lane >> 5);
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
          const bf16x8 ak = *(const bf16x8*)(ks + rm_addr<DH>(32 * mt + (lane & 31), kc));
          s[mt] = mfma32x32x16(ak, qf[kk], s[mt]);
          const bf16x8 av = *(const bf16x8*)(vs + rm_addr<DH>(32 * mt + (lane & 31), kc));
          dp[mt] = mfma32x32x16(av, dof[kk], dp[mt]);
        }
      }
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t kv = kv0 + 32 * mt + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          const bool ok = qrow < S && kv < S && !(a.causal && kv > qrow);
          const float p = ok ? exp2f(fmaf(s[mt][r], c, -lse2)) : 0.0f;
          s[mt][r] = p * (dp[mt][r] - dl);          // dS^T
        }
#pragma unroll
      for (int t = 0; t < C::DT; ++t)
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int hf = 0; hf < 2; ++hf) {
            const bf16x8 af = fm_frag(kts, 32 * t + (lane & 31), 32 * mt + 16 * hf, lane);
            acc[t] = mfma32x32x16(af, acc_to_b(s[mt], hf), acc[t]);
          }
    }
    if (j + 1 < ntiles) lstore(buf ^ 1);
    __syncthreads();
  }

  if (qrow < a.Sp) {
    bf16* dQt = (bf16*)a.dqt + (int64_t)h * DH * a.ld_dt + (int64_t)b * a.Sp + qrow;
    const bool real = qrow < S;
#pragma unroll
    for (int t = 0; t < C::DT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int d = 32 * t + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        dQt[(int64_t)d * a.ld_dt] = (bf16)(real ? acc[t][r] * scale : 0.0f);
      }
  }
}

// ====================================================================== backward dK dV, bf16
// Key-outer: each wave owns 32 keys; loop over query tiles of 64. S = Q K^T and
// dP = dO V^T have the key on the lane axis, so P and dS feed dV^T += dO^T P and
// dK^T += Q^T dS directly as B operands.
template <int DH>
struct DkvCfg {
  static constexpr int KC = DH / 8, KSTEPS = DH / 16, DT = DH / 32;
  static constexpr int RBYTES = 64 * DH * 2;
  static constexpr int STAGE = 4 * RBYTES + 2 * 64 * 4;   // Q, dO, Q^T, dO^T, lse, delta
  static constexpr int LDS = 2 * STAGE;
  static constexpr int CR = 64 * KC / 256, CT = DH * 8 / 256;
};

template <int DH>
__global__ __launch_bounds__(256, 1) void attn_bwd_dkdv_bf16_kernel(AttnArgs a) {
  using C = DkvCfg<DH>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t S = a.S;
  const int64_t k0 = (int64_t)blockIdx.x * 128;
  const int64_t kw = k0 + 32 * wave;
  const int64_t kvrow = kw + (lane & 31);
  const float scale = rsqrtf((float)DH);
  const float c = scale * LOG2E;

  const bf16* Qp = (const bf16*)a.q + (int64_t)h * DH;
  const bf16* Kp = (const bf16*)a.k + (int64_t)h * DH;
  const bf16* Vp = (const bf16*)a.v + (int64_t)h * DH;
  const bf16* dOp = (const bf16*)a.dout + (int64_t)h * DH;
  const bf16* Qt = (const bf16*)a.qt + (int64_t)h * DH * a.ld_qt + (int64_t)b * a.Sp;
  const bf16* dOt = (const bf16*)a.dot + (int64_t)h * DH * a.ld_dot + (int64_t)b * a.Sp;
  const float* lse = a.lse + ((int64_t)b * a.H + h) * a.Sp;
  const float* delta = a.delta + ((int64_t)b * a.H + h) * a.Sp;

  bf16x8 kf[C::KSTEPS], vf[C::KSTEPS];
#pragma unroll
  for (int kk = 0; kk < C::KSTEPS; ++kk) {
    u32x4 v = {0, 0, 0, 0}, w = {0, 0, 0, 0};
    if (kvrow < S) {
      v = ld16(Kp + (b * S + kvrow) * a.ld_k + 16 * kk + 8 * (lane >> 5));
      w = ld16(Vp + (b * S + kvrow) * a.ld_v + 16 * kk + 8 * (lane >> 5));
    }
    kf[kk] = __builtin_bit_cast(bf16x8, v);
    vf[kk] = __builtin_bit_cast(bf16x8, w);
  }

  const int64_t qstart = a.causal ? (k0 / 64) * 64 : 0;
  const int ntiles = qstart < S ? (int)((S - qstart + 63) / 64) : 0;

  u32x4 rq[C::CR], rd[C::CR], rqt[C::CT], rdt[C::CT];
  float rl = 0.0f, rdl = 0.0f;
  auto gload = [&](int j) {
    const int64_t qt0 = qstart + (int64_t)j * 64;
#pragma unroll
    for (int i = 0; i < C::CR; ++i) {
      const int cc = tid + 256 * i, row = cc / C::KC, kc = cc % C::KC;
      const int64_t q = qt0 + row;
      rq[i] = q < S ? ld16(Qp + (b * S + q) * a.ld_q + kc * 8) : u32x4{0, 0, 0, 0};
      rd[i] = q < S ? ld16(dOp + (b * S + q) * a.ld_do + kc * 8) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int i = 0; i < C::CT; ++i) {
      const int cc = tid + 256 * i, d = cc >> 3, ch = cc & 7;
      rqt[i] = ld16(Qt + (int64_t)d * a.ld_qt + qt0 + ch * 8);
      rdt[i] = ld16(dOt + (int64_t)d * a.ld_dot + qt0 + ch * 8);
    }
    if (tid < 64) {
      const int64_t q = qt0 + tid;
      rl = q < S ? lse[q] * LOG2E : 0.0f;
      rdl = q < S ? delta[q] : 0.0f;
    }
  };
  auto lstore = [&](int buf) {
    char* qs = smem + buf * C::STAGE;
    char* ds = qs + C::RBYTES;
    char* qts = ds + C::RBYTES;
    char* dts = qts + C::RBYTES;
    float* ls = (float*)(dts + C::RBYTES);
#pragma unroll
    for (int i = 0; i < C::CR; ++i) {
      const int cc = tid + 256 * i;
      *(u32x4*)(qs + rm_addr<DH>(cc / C::KC, cc % C::KC)) = rq[i];
      *(u32x4*)(ds + rm_addr<DH>(cc / C::KC, cc % C::KC)) = rd[i];
    }
#pragma unroll
    for (int i = 0; i < C::CT; ++i) {
      const int cc = tid + 256 * i, d = cc >> 3, ch = cc & 7;
      *(u32x4*)(qts + d * 128 + ((ch ^ (d & 7)) << 4)) = rqt[i];
      *(u32x4*)(dts + d * 128 + ((ch ^ (d & 7)) << 4)) = rdt[i];
    }
    if (tid < 64) {
      ls[tid] = rl;
      ls[64 + tid] = rdl;
    }
  };

  f32x16 adv[C::DT], adk[C::DT];
#pragma unroll
  for (int t = 0; t < C::DT; ++t) {
    adv[t] = f32x16{};
    adk[t] = f32x16{};
  }

  if (ntiles > 0) {
    gload(0);
    lstore(0);
  }
  __syncthreads();
  for (int j = 0; j < ntiles; ++j) {
    const int buf = j & 1;
    if (j + 1 < ntiles) gload(j + 1);
    const int64_t qt0 = qstart + (int64_t)j * 64;
    const bool skip = a.causal && qt0 + 63 < kw;
    if (!skip) {
      const char* qs = smem + buf * C::STAGE;
      const char* ds = qs + C::RBYTES;
      const char* qts = ds + C::RBYTES;
      const char* dts = qts + C::RBYTES;
      const float* ls = (const float*)(dts + C::RBYTES);
      f32x16 s[2] = {f32x16{}, f32x16{}}, dp[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int kk = 0; kk < C::KSTEPS; ++kk) {
        const int kc = 2 * kk + (lane >> 5);
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
          const bf16x8 aq = *(const bf16x8*)(qs + rm_addr<DH>(32 * mt + (lane & 31), kc));
          s[mt] = mfma32x32x16(aq, kf[kk], s[mt]);
          const bf16x8 ad = *(const bf16x8*)(ds + rm_addr<DH>(32 * mt + (lane & 31), kc));
          dp[mt] = mfma32x32x16(ad, vf[kk], dp[mt]);
        }
      }
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int qi = 32 * mt + 8 * rg + 4 * (lane >> 5);
          const f32x4 l4 = *(const f32x4*)(ls + qi);
          const f32x4 d4 = *(const f32x4*)(ls + 64 + qi);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int r = 4 * rg + e;
            const int64_t q = qt0 + qi + e;
            const bool ok = q < S && kvrow < S && !(a.causal && kvrow > q);
            const float p = ok ? exp2f(fmaf(s[mt][r], c, -l4[e])) : 0.0f;
            s[mt][r] = p;
            dp[mt][r] = p * (dp[mt][r] - d4[e]);     // dS
          }
        }
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const bf16x8 pb = acc_to_b(s[mt], hf);
          const bf16x8 sb = acc_to_b(dp[mt], hf);
#pragma unroll
          for (int t = 0; t < C::DT; ++t) {
            const bf16x8 ado = fm_frag(dts, 32 * t + (lane & 31), 32 * mt + 16 * hf, lane);
            adv[t] = mfma32x32x16(ado, pb, adv[t]);
            const bf16x8 aqt = fm_frag(qts, 32 * t + (lane & 31), 32 * mt + 16 * hf, lane);
            adk[t] = mfma32x32x16(aqt, sb, adk[t]);
          }
        }
    }
    if (j + 1 < ntiles) lstore(buf ^ 1);
    __syncthreads();
  }

  if (kvrow < a.Sp) {
    const int64_t col = (int64_t)b * a.Sp + kvrow;
    bf16* dKt = (bf16*)a.dkt + (int64_t)h * DH * a.ld_dt + col;
    bf16* dVt = (bf16*)a.dvt + (int64_t)h * DH * a.ld_dt + col;
#pragma unroll
    for (int t = 0; t < C::DT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t d = 32 * t + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        dKt[d * a.ld_dt] = (bf16)(adk[t][r] * scale);
        dVt[d * a.ld_dt] = (bf16)adv[t][r];
      }
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
  const float* Vt = (const float*)a.vt + (int64_t)h * DH * a.ld_vt + (int64_t)b * a.Sp;
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
      const int d2 = i / 32, r2 = i % 32;
      Vs[r2][d2] = (kv0 + r2 < S) ? Vt[(int64_t)d2 * a.ld_vt + kv0 + r2] : 0.0f;
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
  const float dl = q < S ? a.delta[sidx] : 0.0f;
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
      const float ds = p * (dpv - dl);
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

// ====================================================================== launchers
template <typename K>
static hipError_t set_lds(K kern, int bytes) {
  return hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

template <int DH>
static hipError_t fwd_launch(Dt dt, const AttnArgs& a, hipStream_t s) {
  const int64_t nq = a.q_end - a.q_begin;
  if (nq <= 0 || a.nb <= 0) return hipSuccess;
  if (dt == BF16) {
    auto kern = attn_fwd_bf16_kernel<DH>;
    hipError_t e = set_lds(kern, FwdCfg<DH>::LDS);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)((nq + 127) / 128), a.H, a.nb), dim3(256),
                       FwdCfg<DH>::LDS, s, a);
  } else {
    hipLaunchKernelGGL(attn_fwd_f32_kernel<DH>, dim3((unsigned)((nq + 63) / 64), a.H, a.nb),
                       dim3(64), 0, s, a);
  }
  return hipGetLastError();
}

// part 0: dK, dV (key-outer); part 1: dQ (query-outer).
template <int DH>
static hipError_t bwd_launch(Dt dt, int part, const AttnArgs& a, hipStream_t s) {
  if (a.S <= 0 || a.B <= 0) return hipSuccess;
  if (dt == BF16) {
    const unsigned tiles = (unsigned)((a.Sp + 127) / 128);
    if (part == 0) {
      auto k = attn_bwd_dkdv_bf16_kernel<DH>;
      hipError_t e = set_lds(k, DkvCfg<DH>::LDS);
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(k, dim3(tiles, a.H, a.B), dim3(256), DkvCfg<DH>::LDS, s, a);
    } else {
      auto k = attn_bwd_dq_bf16_kernel<DH>;
      hipError_t e = set_lds(k, DqCfg<DH>::LDS);
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(k, dim3(tiles, a.H, a.B), dim3(256), DqCfg<DH>::LDS, s, a);
    }
  } else {
    const unsigned tiles = (unsigned)(a.Sp / 64);
    if (part == 0) {
      const int lds = (2 * DH * 65 + 2 * 16 * DH + 32) * 4;
      hipError_t e = set_lds(attn_bwd_dkdv_f32_kernel<DH>, lds);
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(attn_bwd_dkdv_f32_kernel<DH>, dim3(tiles, a.H, a.B), dim3(64), lds, s, a);
    } else {
      const int lds = (2 * DH * 65 + 2 * 16 * DH) * 4;
      hipError_t e = set_lds(attn_bwd_dq_f32_kernel<DH>, lds);
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(attn_bwd_dq_f32_kernel<DH>, dim3(tiles, a.H, a.B), dim3(64), lds, s, a);
    }
  }
  return hipGetLastError();
}

hipError_t attn_fwd(Dt dt, const AttnArgs& a, hipStream_t s) {
  if (a.dh == 64) return fwd_launch<64>(dt, a, s);
  if (a.dh == 128) return fwd_launch<128>(dt, a, s);
  return hipErrorInvalidValue;
}

hipError_t attn_bwd(Dt dt, int part, const AttnArgs& a, hipStream_t s) {
  if (a.dh == 64) return bwd_launch<64>(dt, part, a, s);
  if (a.dh == 128) return bwd_launch<128>(dt, part, a, s);
  return hipErrorInvalidValue;
}

}  // namespace bpt

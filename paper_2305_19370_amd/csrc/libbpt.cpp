// libbpt host side: argument validation, buffer layout and the launch sequence of
// one Blockwise Parallel Transformer layer (Algorithm 1 of the paper) forward and
// backward. Allocates nothing on the device; every launch goes to the caller's
// stream and nothing synchronises.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "libbpt.h"
#include "internal.h"

using namespace bpt;

namespace {

thread_local std::string g_err;

bpt_status fail(bpt_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

constexpr int64_t kAlign = 256;
// Automatic FFN group: at least 16384 rows, and for a narrow FFN as many rows as keep the
// [., F] intermediate at 2^27 elements (256 MiB in bf16), so that the group's GEMMs are
// tall enough to fill the chip and few enough that their per-launch costs stay small.
constexpr int64_t kDefaultGroupRows = 16384;
constexpr int64_t kGroupElems = int64_t(1) << 27;
int64_t auto_group_rows(int64_t F) { return std::max(kDefaultGroupRows, kGroupElems / std::max<int64_t>(F, 1)); }

int64_t rup(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
size_t esize(int32_t dt) { return dt == BPT_BF16 ? 2 : 4; }

struct Dims {
  int64_t B, S, D, H, F, dh, T, Sp, Tp, R, Rp;
  int64_t nbg, Rs;       // FFN group: nbg whole sequences (Rs = S), or Rs rows of one (nbg = 1)
  size_t E;
  bool drop;             // residual-branch dropout on (rate > 0)
};

Dims dims_of(const bpt_config& c) {
  Dims d;
  d.B = c.B; d.S = c.S; d.D = c.D; d.H = c.H; d.F = c.F;
  d.dh = c.D / c.H;
  d.T = c.B * c.S;
  d.drop = c.dropout > 0.0f;
  d.Sp = rup(c.S, 64);
  d.Tp = c.B * d.Sp;
  const int64_t g = c.group_blocks > 0 ? c.group_blocks
                                      : std::max<int64_t>(1, (auto_group_rows(c.F) + c.Bq - 1) / c.Bq);
  // A group holds up to g * Bq rows: a run of Rs rows of one sequence or, when at least two
  // whole sequences fit, nbg whole sequences (their tokens are contiguous), so that short
  // sequences still give the FFN GEMMs their full height.
  const int64_t rows = g * c.Bq;
  if (c.B > 1 && rows >= 2 * c.S) {
    d.nbg = std::min<int64_t>(c.B, rows / c.S);
    d.Rs = c.S;
  } else {
    d.nbg = 1;
    d.Rs = std::min<int64_t>(rows, c.S);
  }
  d.R = d.nbg * d.Rs;
  d.Rp = rup(d.R, 64);
  d.E = esize(c.dtype);
  return d;
}

bpt_status check(const bpt_config* c) {
  if (!c) return fail(BPT_ERR_INVALID_ARG, "config is NULL");
  if (c->B < 1 || c->S < 1 || c->D < 1 || c->H < 1 || c->F < 1)
    return fail(BPT_ERR_INVALID_ARG, "B, S, D, H, F must be >= 1 (got %lld %lld %lld %lld %lld)",
                (long long)c->B, (long long)c->S, (long long)c->D, (long long)c->H, (long long)c->F);
  if (c->D % c->H != 0)
    return fail(BPT_ERR_INVALID_ARG, "D=%lld is not divisible by H=%lld", (long long)c->D, (long long)c->H);
  if (c->Bq < 1 || c->Bq > c->S || c->Bkv < 1 || c->Bkv > c->S)
    return fail(BPT_ERR_INVALID_ARG, "block lengths must satisfy 1 <= Bq, Bkv <= S (got %lld, %lld, S=%lld)",
                (long long)c->Bq, (long long)c->Bkv, (long long)c->S);
  if (c->causal != 0 && c->causal != 1) return fail(BPT_ERR_INVALID_ARG, "causal must be 0 or 1");
  if ((c->dtype != BPT_F32 && c->dtype != BPT_BF16) || (c->out_dtype != BPT_F32 && c->out_dtype != BPT_BF16))
    return fail(BPT_ERR_INVALID_ARG, "dtype / out_dtype must be BPT_F32 or BPT_BF16");
  if (c->group_blocks < 0) return fail(BPT_ERR_INVALID_ARG, "group_blocks must be >= 0");
  if (!(c->ln_eps > 0.0f)) return fail(BPT_ERR_INVALID_ARG, "ln_eps must be > 0");
  if (c->activation != BPT_GELU && c->activation != BPT_RELU)
    return fail(BPT_ERR_INVALID_ARG, "activation must be BPT_GELU or BPT_RELU");
  if (!(c->dropout >= 0.0f && c->dropout < 1.0f))
    return fail(BPT_ERR_INVALID_ARG, "dropout rate must lie in [0, 1)");
  const int64_t dh = c->D / c->H;
  if (dh != 64 && dh != 128)
    return fail(BPT_ERR_UNSUPPORTED, "head dim D/H=%lld unsupported (64 or 128)", (long long)dh);
  if (c->D % 64 != 0 || c->F % 64 != 0)
    return fail(BPT_ERR_UNSUPPORTED, "D and F must be multiples of 64 (got %lld, %lld)", (long long)c->D,
                (long long)c->F);
  // element indices are 64-bit everywhere; grid dimensions are 32-bit
  if (c->B > 65535 || c->H > 65535) return fail(BPT_ERR_UNSUPPORTED, "B and H must be <= 65535");
  if (c->B * rup(c->S, 64) > (int64_t)1 << 40) return fail(BPT_ERR_UNSUPPORTED, "B*S too large");
  return BPT_OK;
}

// Bump allocator over a caller-provided region. With a zero base the returned
// "pointers" are the byte offsets, which is how the sizes and layouts are computed.
struct Bump {
  uintptr_t base;
  int64_t off = 0;
  explicit Bump(void* b) : base((uintptr_t)b) {}
  void* take(int64_t bytes) {
    off = rup(off, kAlign);
    void* p = (void*)(base + (uintptr_t)off);
    off += bytes;
    return p;
  }
};

struct SavedPtrs {
  void *qkv, *o;
  float *lse, *h, *mu1, *rstd1, *mu2, *rstd2;
};

SavedPtrs saved_layout(const Dims& d, void* base, int64_t* total) {
  Bump bp(base);
  SavedPtrs s;
  s.qkv = bp.take(d.T * 3 * d.D * d.E);
  s.o = bp.take(d.T * d.D * d.E);
  s.lse = (float*)bp.take(d.B * d.H * d.Sp * 4);
  s.h = (float*)bp.take(d.T * d.D * 4);
  s.mu1 = (float*)bp.take(d.T * 4);
  s.rstd1 = (float*)bp.take(d.T * 4);
  s.mu2 = (float*)bp.take(d.T * 4);
  s.rstd2 = (float*)bp.take(d.T * 4);
  *total = rup(bp.off, kAlign);
  return s;
}

struct FwdWs {
  void *u, *vg, *gg;
  float* acc;            // FFN output of a group before its dropout (null: no dropout)
};

FwdWs fwd_ws(const Dims& d, void* base, int64_t* total) {
  Bump bp(base);
  FwdWs w;
  w.u = bp.take(d.T * d.D * d.E);
  w.vg = bp.take(d.R * d.D * d.E);
  w.gg = bp.take(d.R * d.F * d.E);
  w.acc = d.drop ? (float*)bp.take(d.R * d.D * 4) : nullptr;
  *total = rup(bp.off, kAlign);
  return w;
}

struct BwdWs {
  void *wcat;
  void *vg, *gT, *dzT;
  void* gpT;             // GELU'(Z^T): fp32 on the fp32 path, fp16 on the bf16 path
  float *dv, *dh, *dU, *ndelta, *nlse2, *partial, *scratch;
  void *dhe, *dhT, *dO, *dqkvT, *u;
  float* kpart;          // K-slice partials of the D x D weight gradients (null: no split)
  float* fpart;          // K-slice partials of dW1 / dW2 (null: no split)
  void* dYm;             // dY through the FFN branch's dropout (null: no dropout)
};

// Slices of K for an M x N weight-gradient GEMM (fp32 C, plain store) over K tokens whose
// 256 x 256 tile grid would leave most of the 256 CUs idle (a narrow layer: D < 4096, or
// D x F < 256 tiles): the slices run as batch entries into fp32 partials that sum_slices
// adds into C in a fixed order. Every slice is a multiple of 64 tokens.
constexpr int kMaxKSplit = 16;
int ksplit_cap(int64_t M, int64_t N) {   // the most slices the tile grid allows
  const int64_t tiles = ((M + 255) / 256) * ((N + 255) / 256);
  int z = 1;
  while (z < kMaxKSplit && tiles * 2 * z <= 256) z *= 2;
  return z;
}
int ksplit(int64_t M, int64_t N, int64_t K) {
  if (K % 64 != 0) return 1;
  const int cap = ksplit_cap(M, N);
  int z = 1;
  while (z < cap && K % (64 * 2 * z) == 0) z *= 2;
  return z;
}

BwdWs bwd_ws(const Dims& d, void* base, int64_t* total) {
  Bump bp(base);
  BwdWs w;
  w.wcat = bp.take(3 * d.D * d.D * d.E);
  w.vg = bp.take(d.R * d.D * d.E);
  w.gT = bp.take(d.F * d.Rp * d.E);
  w.gpT = bp.take(d.F * d.Rp * (d.E == 2 ? 2 : 4));   // fp16 on the bf16 path, else fp32
  w.dzT = bp.take(d.F * d.Rp * d.E);
  w.dv = (float*)bp.take(d.T * d.D * 4);
  w.dh = (float*)bp.take(d.T * d.D * 4);
  w.dhe = bp.take(d.T * d.D * d.E);
  w.dhT = bp.take(d.D * d.Tp * d.E);
  w.dO = bp.take(d.T * d.D * d.E);
  w.ndelta = (float*)bp.take(d.B * d.H * d.Sp * 4);
  w.nlse2 = (float*)bp.take(d.B * d.H * d.Sp * 4);
  w.dqkvT = bp.take(3 * d.D * d.Tp * d.E);
  w.u = bp.take(d.T * d.D * d.E);
  w.dU = (float*)bp.take(d.T * d.D * 4);
  w.partial = (float*)bp.take((int64_t)layer_norm_param_grad_ws(std::max(d.D, d.F)) * 4);
  w.scratch = (float*)bp.take(2 * std::max(d.D, d.F) * 4);
  const int kz = d.S % 64 == 0 ? ksplit(d.D, d.D, d.T) : 1;   // the whole-batch GEMMs below
  w.kpart = kz > 1 ? (float*)bp.take(kz * d.D * d.D * 4) : nullptr;
  const int fz = ksplit_cap(d.D, d.F);                      // dW1 and dW2 per FFN group
  w.fpart = fz > 1 ? (float*)bp.take(fz * d.D * d.F * 4) : nullptr;
  w.dYm = d.drop ? bp.take(d.T * d.D * d.E) : nullptr;
  *total = rup(bp.off, kAlign);
  return w;
}

// the dropout masks' generator key, threshold and scale for branch `site`
DropArgs drop_args(const bpt_config& c, uint32_t site, int64_t row0) {
  DropArgs a;
  a.k0 = (uint32_t)(c.dropout_seed & 0xFFFFFFFFu);
  a.k1 = (uint32_t)(c.dropout_seed >> 32);
  a.site = site;
  const double th = std::floor((double)c.dropout * 4294967296.0);
  a.threshold = (uint32_t)std::min(th, 4294967295.0);
  a.scale = (float)(1.0 / (1.0 - (double)c.dropout));
  a.row0 = row0;
  return a;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

#define HIPCHK(expr)                                                                   \
  do {                                                                                 \
    hipError_t _e = (expr);                                                            \
    if (_e != hipSuccess) return fail(BPT_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(_e)); \
  } while (0)

char* off(const void* p, int64_t bytes) { return (char*)p + bytes; }


// ---------------------------------------------------------------- launch profiler
// Off by default. When on, every launch of bpt_layer_fwd / bpt_layer_bwd is
// bracketed by two HIP events recorded on the launch stream, tagged with the
// call site's name and its algorithmic flops / HBM bytes.
struct ProfRec {
  std::string name;
  double flops, bytes;
  hipEvent_t a, b;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<ProfRec> g_prof;
std::vector<hipEvent_t> g_pool;
size_t g_pool_used = 0;

hipEvent_t pool_event() {
  if (g_pool_used == g_pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    g_pool.push_back(e);
  }
  return g_pool[g_pool_used++];
}

// set while a call that must not allocate runs: its launches bypass the profiler, whose
// first use creates HIP events
thread_local bool t_noalloc = false;

template <class Fn>
hipError_t launch(const char* name, double flops, double bytes, hipStream_t s, Fn&& fn) {
  if (!g_prof_on || t_noalloc) return fn();
  std::lock_guard<std::mutex> lk(g_prof_mu);
  hipEvent_t a = pool_event(), b = pool_event();
  if (!a || !b || hipEventRecord(a, s) != hipSuccess) return fn();
  hipError_t e = fn();
  if (hipEventRecord(b, s) == hipSuccess) g_prof.push_back({name, flops, bytes, a, b});
  return e;
}

#define RUN(name, flops, bytes, expr)                                                        \
  do {                                                                                       \
    hipError_t _e = launch(name, (double)(flops), (double)(bytes), s, [&] { return (expr); }); \
    if (_e != hipSuccess) return fail(BPT_ERR_HIP, "%s: %s", name, hipGetErrorString(_e));  \
  } while (0)

double gemm_flops(const GemmArgs& g) { return 2.0 * g.M * g.N * g.K * g.batch; }
double gemm_bytes(const GemmArgs& g, size_t eab, size_t ec) {
  const double ncols = (double)std::max(g.N, g.Nstore);
  return ((double)g.M * g.K + (double)g.N * g.K) * eab * g.batch + (double)g.M * ncols * ec * g.batch;
}
// visible (query, key) pairs of query rows [q0, q1) of one sequence of length S
double attn_pairs(int64_t q0, int64_t q1, int64_t S, int causal) {
  if (!causal) return (double)(q1 - q0) * S;
  return 0.5 * ((double)q1 * (q1 + 1) - (double)q0 * (q0 + 1));
}


// ---------------------------------------------------------------- cross-entropy of an LM head
constexpr int64_t kDefaultXentRows = 8192;     // tokens whose logits are live at once

bpt_status xent_check(const bpt_xent_config* c) {
  if (!c) return fail(BPT_ERR_INVALID_ARG, "config is NULL");
  if (c->T < 1 || c->D < 1 || c->V < 1)
    return fail(BPT_ERR_INVALID_ARG, "T, D, V must be >= 1 (got %lld %lld %lld)", (long long)c->T,
                (long long)c->D, (long long)c->V);
  if (c->ldw < c->V) return fail(BPT_ERR_INVALID_ARG, "ldw=%lld < V=%lld", (long long)c->ldw, (long long)c->V);
  if (c->block_rows < 0) return fail(BPT_ERR_INVALID_ARG, "block_rows must be >= 0");
  if (c->dtype != BPT_F32 && c->dtype != BPT_BF16) return fail(BPT_ERR_INVALID_ARG, "dtype must be BPT_F32 or BPT_BF16");
  if (c->reserved != 0) return fail(BPT_ERR_INVALID_ARG, "reserved must be 0");
  if (c->ldw % 64 != 0 || c->D % 64 != 0)
    return fail(BPT_ERR_UNSUPPORTED, "ldw and D must be multiples of 64 (got %lld, %lld)", (long long)c->ldw,
                (long long)c->D);
  if (c->T > ((int64_t)1 << 31) - 1) return fail(BPT_ERR_UNSUPPORTED, "T too large");
  return BPT_OK;
}

struct XentDims {
  int64_t T, D, V, ldw, R, Rp;   // R: rows per block; Rp: R rounded up to 64
  size_t E;
};

XentDims xent_dims(const bpt_xent_config& c) {
  XentDims d;
  d.T = c.T; d.D = c.D; d.V = c.V; d.ldw = c.ldw;
  d.R = std::min(c.block_rows > 0 ? c.block_rows : kDefaultXentRows, c.T);
  d.Rp = rup(d.R, 64);
  d.E = esize(c.dtype);
  return d;
}

struct XentWs {
  float* logits;   // forward: [R, ldw] fp32
  float* tok;      // forward: [T] token losses
  void* g;         // backward: [ldw, Rp] in dtype, the logits' gradient of one block, transposed
};

XentWs xent_ws(const XentDims& d, void* base, int backward, int64_t* total) {
  Bump bp(base);
  XentWs w{};
  if (backward) {
    w.g = bp.take(d.Rp * d.ldw * (int64_t)d.E);
  } else {
    w.logits = (float*)bp.take(d.R * d.ldw * 4);
    w.tok = (float*)bp.take(d.T * 4);
  }
  *total = rup(bp.off, kAlign);
  return w;
}

}  // namespace

// Workspace of bpt_layer_fwd_noalloc: the library's own device memory, one copy per GPU,
// held until the process ends. In host code `scratch` is a stand-in for the symbol, not a
// device address: kernels get the address hipGetSymbolAddress returns on each device.
static constexpr size_t kScratchBytes = BPT_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {
std::mutex g_scratch_mu;
std::vector<void*> g_scratch_dev;   // scratch's address on device i (null until first use there)

// scratch's address on the current device, looked up once per device
bpt_status scratch_ptr(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(BPT_ERR_HIP, "hipGetDevice failed: %s", hipGetErrorString(e));
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if ((size_t)dev >= g_scratch_dev.size()) g_scratch_dev.resize((size_t)dev + 1, nullptr);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(BPT_ERR_HIP, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return BPT_OK;
}
}  // namespace

extern "C" {

bpt_status bpt_validate(const bpt_config* cfg) { return check(cfg); }

int64_t bpt_group_rows(const bpt_config* cfg) {
  if (check(cfg) != BPT_OK) return -1;
  return dims_of(*cfg).R;
}

size_t bpt_saved_bytes(const bpt_config* cfg) {
  if (check(cfg) != BPT_OK) return 0;
  int64_t total;
  saved_layout(dims_of(*cfg), nullptr, &total);
  return (size_t)total;
}

bpt_status bpt_saved_layout_of(const bpt_config* cfg, bpt_saved_layout* out) {
  bpt_status st = check(cfg);
  if (st != BPT_OK) return st;
  if (!out) return fail(BPT_ERR_INVALID_ARG, "out is NULL");
  int64_t total;
  SavedPtrs s = saved_layout(dims_of(*cfg), nullptr, &total);   // zero base: pointers are offsets
  out->qkv = (size_t)(uintptr_t)s.qkv;
  out->o = (size_t)(uintptr_t)s.o;
  out->lse = (size_t)(uintptr_t)s.lse;
  out->h = (size_t)(uintptr_t)s.h;
  out->mu1 = (size_t)(uintptr_t)s.mu1;
  out->rstd1 = (size_t)(uintptr_t)s.rstd1;
  out->mu2 = (size_t)(uintptr_t)s.mu2;
  out->rstd2 = (size_t)(uintptr_t)s.rstd2;
  out->total = (size_t)total;
  return BPT_OK;
}

size_t bpt_workspace_bytes(const bpt_config* cfg, int backward) {
  if (check(cfg) != BPT_OK) return 0;
  int64_t total;
  const Dims d = dims_of(*cfg);
  if (backward) bwd_ws(d, nullptr, &total);
  else fwd_ws(d, nullptr, &total);
  return (size_t)total;
}

bpt_status bpt_bwd_qkv_grad_offset(const bpt_config* cfg, size_t* offset) {
  bpt_status st = check(cfg);
  if (st != BPT_OK) return st;
  if (!offset) return fail(BPT_ERR_INVALID_ARG, "offset is NULL");
  int64_t total;
  BwdWs w = bwd_ws(dims_of(*cfg), nullptr, &total);   // zero base: pointers are offsets
  *offset = (size_t)(uintptr_t)w.dqkvT;
  return BPT_OK;
}

const char* bpt_status_string(int st) {
  switch (st) {
    case BPT_OK: return "BPT_OK";
    case BPT_ERR_INVALID_ARG: return "BPT_ERR_INVALID_ARG";
    case BPT_ERR_UNSUPPORTED: return "BPT_ERR_UNSUPPORTED";
    case BPT_ERR_WORKSPACE: return "BPT_ERR_WORKSPACE";
    case BPT_ERR_HIP: return "BPT_ERR_HIP";
  }
  return "BPT_ERR_UNKNOWN";
}

const char* bpt_last_error(void) { return g_err.c_str(); }

size_t bpt_describe(const bpt_config* cfg, char* buf, size_t n) {
  if (!buf || n == 0) return 0;
  if (check(cfg) != BPT_OK) {
    buf[0] = 0;
    return 0;
  }
  const Dims d = dims_of(*cfg);
  const bool bf = cfg->dtype == BPT_BF16;
  int w = snprintf(buf, n,
                   "dtype=%s attention: q-tile=%d kv-step=%d (%s); backward dK/dV kv-tile=%d q-step=%d, "
                   "dQ q-tile=%d kv-step=%d; gemm: %s; ffn %s, group rows=%lld (%lld sequence(s) x %lld rows; "
                   "query blocks of %lld)",
                   bf ? "bf16" : "f32", bf ? 256 : 64, bf ? 64 : 32,
                   bf ? "MFMA 32x32x16 bf16, fp32 accumulate, 32 rows per wave" : "fp32 VALU",
                   bf ? 256 : 64, bf ? 64 : 16, bf ? 256 : 64, bf ? 64 : 16,
                   bf ? "MFMA bf16 256x256 (8 waves) or 128x128 (4 waves) tiles, K-step 32"
                      : "fp32 VALU 64x64 tiles",
                   cfg->activation == BPT_RELU ? "relu" : "gelu", (long long)d.R, (long long)d.nbg, (long long)d.Rs,
                   (long long)cfg->Bq);
  return w < 0 ? 0 : std::min((size_t)w, n - 1);
}

bpt_status bpt_profile_enable(int on) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (on) {             // start a new record; turning off keeps it for bpt_profile_report
    g_prof.clear();
    g_pool_used = 0;
  }
  g_prof_on = on != 0;
  return BPT_OK;
}

size_t bpt_profile_report(char* buf, size_t n) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  struct Agg { int count = 0; double ms = 0, flops = 0, bytes = 0; };
  std::map<std::string, Agg> agg;
  for (const ProfRec& r : g_prof) {
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) ms = -1.0f;
    Agg& a = agg[r.name];
    a.count += 1;
    a.ms += ms;
    a.flops += r.flops;
    a.bytes += r.bytes;
  }
  std::string out = "{";
  bool first = true;
  for (auto& kv : agg) {
    char line[512];
    snprintf(line, sizeof line, "%s\"%s\": {\"count\": %d, \"ms\": %.6f, \"flops\": %.6e, \"bytes\": %.6e}",
             first ? "" : ", ", kv.first.c_str(), kv.second.count, kv.second.ms, kv.second.flops,
             kv.second.bytes);
    out += line;
    first = false;
  }
  out += "}";
  if (buf && n > 0) {
    const size_t k = std::min(out.size(), n - 1);
    memcpy(buf, out.data(), k);
    buf[k] = 0;
  }
  return out.size();
}

bpt_status bpt_layer_fwd_noalloc(const bpt_config* cfg, const void* X, const bpt_params* p, void* Y, void* saved,
                                 void* stream) {
  bpt_status st = check(cfg);
  if (st != BPT_OK) return st;
  int64_t need;
  fwd_ws(dims_of(*cfg), nullptr, &need);
  if ((size_t)need > kScratchBytes)
    return fail(BPT_ERR_WORKSPACE, "this configuration needs %lld workspace bytes, more than the %zu of the "
                "static scratch of bpt_layer_fwd_noalloc (use bpt_layer_fwd with a workspace)",
                (long long)need, kScratchBytes);
  void* ws = nullptr;
  if ((st = scratch_ptr(&ws)) != BPT_OK) return st;
  struct NoAlloc {
    NoAlloc() { t_noalloc = true; }
    ~NoAlloc() { t_noalloc = false; }
  } guard;
  return bpt_layer_fwd(cfg, X, p, Y, saved, ws, kScratchBytes, stream);
}

bpt_status bpt_layer_fwd(const bpt_config* cfg, const void* X, const bpt_params* p, void* Y, void* saved,
                         void* ws, size_t ws_bytes, void* stream) {
  bpt_status st = check(cfg);
  if (st != BPT_OK) return st;
  if (!X || !p || !Y || !saved || !ws) return fail(BPT_ERR_INVALID_ARG, "NULL X, params, Y, saved or workspace");
  if (!p->Wq || !p->Wk || !p->Wv || !p->Wo || !p->W1 || !p->W2)
    return fail(BPT_ERR_INVALID_ARG, "NULL weight pointer");
  if (X == Y) return fail(BPT_ERR_INVALID_ARG, "Y must not alias X");
  const void* ptrs[] = {X, Y, saved, ws, p->Wq, p->Wk, p->Wv, p->Wo, p->W1, p->W2,
                        p->ln1_g, p->ln1_b, p->ln2_g, p->ln2_b, p->b1, p->b2};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return fail(BPT_ERR_INVALID_ARG, "pointer %p is not 16-byte aligned", q);
  const Dims d = dims_of(*cfg);
  const Epi act = cfg->activation == BPT_RELU ? EPI_RELU : EPI_GELU;   // FFN epilogue of eq. (2)
  int64_t need, stotal;
  FwdWs w = fwd_ws(d, ws, &need);
  if ((int64_t)ws_bytes < need)
    return fail(BPT_ERR_WORKSPACE, "workspace %zu bytes < required %lld", ws_bytes, (long long)need);
  SavedPtrs sv = saved_layout(d, saved, &stotal);
  hipStream_t s = (hipStream_t)stream;
  const Dt E = cfg->dtype == BPT_BF16 ? BF16 : F32;
  const Dt OUT = cfg->out_dtype == BPT_BF16 ? BF16 : F32;
  const int64_t D = d.D, F = d.F, T = d.T, E_ = (int64_t)d.E;
  const size_t EO = esize(cfg->out_dtype);

  // U = LN1(X); [Q | K | V] = U [Wq | Wk | Wv]  (Algorithm 1: project the input)
  RUN("layernorm.fwd", 0, 2.0 * T * D * E_,
      layer_norm(E, E, X, D, p->ln1_g, p->ln1_b, w.u, D, sv.mu1, sv.rstd1, T, D, cfg->ln_eps, 0, s));
  // the weights [D_in, D_out] are read as they are: B operands stored K-major
  const void* wqkv[3] = {p->Wq, p->Wk, p->Wv};
  for (int i = 0; i < 3; ++i) {
    GemmArgs g;
    g.A = w.u; g.lda = D; g.B = wqkv[i]; g.ldb = D; g.trans_b = 1;
    // bf16 attention takes Q multiplied by log2(e)/sqrt(dh): scores in base-2 units
    if (i == 0 && E == BF16) g.alpha = (float)(1.4426950408889634 / std::sqrt((double)d.dh));
    g.C = off(sv.qkv, i * D * E_); g.ldc = 3 * D; g.M = T; g.N = D; g.K = D;
    RUN("gemm.qkv", gemm_flops(g), gemm_bytes(g, E_, E_), gemm(E, EPI_STORE, E, F32, g, s));
  }

  // Outer loop over groups of query blocks: attention for the group, then the
  // output projection, LN2, FFN and both residuals for the same rows.
  for (int64_t b = 0; b < d.B; b += d.nbg) {
    const int64_t nb = std::min(d.nbg, d.B - b);   // sequences in this group (several only if whole)
    for (int64_t s0 = 0; s0 < d.S; s0 += d.Rs) {
      const int64_t rs = std::min(d.Rs, d.S - s0), r = nb * rs;
      const int64_t t0 = b * d.S + s0;
      AttnArgs a;
      a.q = sv.qkv; a.ld_q = 3 * D;
      a.k = off(sv.qkv, D * E_); a.ld_k = 3 * D;
      a.v = off(sv.qkv, 2 * D * E_); a.ld_v = 3 * D;
      a.o = sv.o; a.ld_o = D;
      a.lse = sv.lse;
      a.S = d.S; a.Sp = d.Sp; a.B = (int)d.B; a.H = (int)d.H; a.dh = (int)d.dh; a.causal = cfg->causal;
      a.q_begin = s0; a.q_end = s0 + rs; a.b_begin = (int)b; a.nb = (int)nb;
      const double pairs = attn_pairs(s0, s0 + rs, d.S, cfg->causal) * d.H * nb;
      RUN("attn.fwd", 4.0 * d.dh * pairs, (3.0 * rs + 2.0 * (s0 + rs)) * nb * D * E_, attn_fwd(E, a, s));

      GemmArgs go;     // h = X + O Wo
      go.A = off(sv.o, t0 * D * E_); go.lda = D; go.B = p->Wo; go.ldb = D; go.trans_b = 1;
      go.C = sv.h + t0 * D; go.ldc = D; go.R = off(X, t0 * D * E_); go.ldr = D;
      go.M = r; go.N = D; go.K = D;
      if (!d.drop) {
        RUN("gemm.wo", gemm_flops(go), gemm_bytes(go, E_, 4) + (double)r * D * E_,
            gemm(E, EPI_RESID, F32, E, go, s));
      } else {   // O Wo into h, then h = X + drop(h) in place
        go.R = nullptr;
        RUN("gemm.wo", gemm_flops(go), gemm_bytes(go, E_, 4), gemm(E, EPI_STORE, F32, F32, go, s));
        RUN("dropout.fwd", 0, (double)r * D * (8 + E_),
            dropout_add(sv.h + t0 * D, E, off(X, t0 * D * E_), nullptr, F32, sv.h + t0 * D, r, D,
                        drop_args(*cfg, 0, t0), s));
      }

      RUN("layernorm.fwd", 0, (double)r * D * (4 + E_),
          layer_norm(F32, E, sv.h + t0 * D, D, p->ln2_g, p->ln2_b, w.vg, D, sv.mu2 + t0, sv.rstd2 + t0, r,
                     D, cfg->ln_eps, 0, s));

      GemmArgs g1;     // G = GELU(LN2(h) W1 + b1)
      g1.A = w.vg; g1.lda = D; g1.B = p->W1; g1.ldb = F; g1.trans_b = 1; g1.C = w.gg; g1.ldc = F;
      g1.bias = p->b1; g1.M = r; g1.N = F; g1.K = D;
      RUN("gemm.ffn1", gemm_flops(g1), gemm_bytes(g1, E_, E_), gemm(E, act, E, F32, g1, s));

      GemmArgs g2;     // Y = h + G W2 + b2
      g2.A = w.gg; g2.lda = F; g2.B = p->W2; g2.ldb = D; g2.trans_b = 1; g2.C = off(Y, t0 * D * EO);
      g2.ldc = D; g2.R = sv.h + t0 * D; g2.ldr = D; g2.bias = p->b2; g2.M = r; g2.N = D; g2.K = F;
      if (!d.drop) {
        RUN("gemm.ffn2", gemm_flops(g2), gemm_bytes(g2, E_, EO) + 4.0 * r * D, gemm(E, EPI_RESID, OUT, F32, g2, s));
      } else {   // G W2 into fp32 workspace, then Y = h + drop(. + b2)
        g2.C = w.acc; g2.R = nullptr; g2.bias = nullptr;
        RUN("gemm.ffn2", gemm_flops(g2), gemm_bytes(g2, E_, 4), gemm(E, EPI_STORE, F32, F32, g2, s));
        RUN("dropout.fwd", 0, (double)r * D * (8 + EO),
            dropout_add(w.acc, F32, sv.h + t0 * D, p->b2, OUT, off(Y, t0 * D * EO), r, D, drop_args(*cfg, 1, t0), s));
      }
    }
  }
  return BPT_OK;
}

bpt_status bpt_layer_bwd(const bpt_config* cfg, const void* X, const bpt_params* p, const void* saved,
                         const void* dY, void* dX, const bpt_grads* gr, void* ws, size_t ws_bytes,
                         void* stream) {
  bpt_status st = check(cfg);
  if (st != BPT_OK) return st;
  if (!X || !p || !saved || !dY || !dX || !ws)
    return fail(BPT_ERR_INVALID_ARG, "NULL X, params, saved, dY, dX or workspace");
  if (!p->Wq || !p->Wk || !p->Wv || !p->Wo || !p->W1 || !p->W2)
    return fail(BPT_ERR_INVALID_ARG, "NULL weight pointer");
  if (dX == dY || dX == X) return fail(BPT_ERR_INVALID_ARG, "dX must not alias dY or X");
  bpt_grads G = {};
  if (gr) G = *gr;
  const void* ptrs[] = {X, saved, dY, dX, ws, p->Wq, p->Wk, p->Wv, p->Wo, p->W1, p->W2, p->ln1_g, p->ln1_b,
                        p->ln2_g, p->ln2_b, p->b1, p->b2, G.dln1_g, G.dln1_b, G.dWq, G.dWk, G.dWv, G.dWo,
                        G.dln2_g, G.dln2_b, G.dW1, G.db1, G.dW2, G.db2};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return fail(BPT_ERR_INVALID_ARG, "pointer %p is not 16-byte aligned", q);
  const Dims d = dims_of(*cfg);
  const Epi act = cfg->activation == BPT_RELU ? EPI_RELU : EPI_GELU;   // FFN epilogue of eq. (2)
  int64_t need, stotal;
  BwdWs w = bwd_ws(d, ws, &need);
  if ((int64_t)ws_bytes < need)
    return fail(BPT_ERR_WORKSPACE, "workspace %zu bytes < required %lld", ws_bytes, (long long)need);
  SavedPtrs sv = saved_layout(d, (void*)saved, &stotal);
  hipStream_t s = (hipStream_t)stream;
  const Dt E = cfg->dtype == BPT_BF16 ? BF16 : F32;
  const Dt OUT = cfg->out_dtype == BPT_BF16 ? BF16 : F32;
  const int64_t D = d.D, F = d.F, T = d.T, Tp = d.Tp, Sp = d.Sp, S = d.S, E_ = (int64_t)d.E;
  const size_t EO = esize(cfg->out_dtype);
  const int B = (int)d.B;
  const double tb = 2.0 * E_;   // bytes per element of a transpose / copy (read + write)
  // GELU'(Z) between the FFN recompute and dZ: fp16 on the bf16 path (its rounding,
  // 2^-11 relative, is far below the bf16 rounding of the dZ operand that follows)
  const Dt GP = E == BF16 ? F16 : F32;
  const int64_t GP_ = GP == F16 ? 2 : 4;

  RUN("copy.weights", 0, tb * D * D, copy2d(E, p->Wq, D, w.wcat, 3 * D, D, D, s));
  RUN("copy.weights", 0, tb * D * D, copy2d(E, p->Wk, D, off(w.wcat, D * E_), 3 * D, D, D, s));
  RUN("copy.weights", 0, tb * D * D, copy2d(E, p->Wv, D, off(w.wcat, 2 * D * E_), 3 * D, D, D, s));

  // ---- FFN and LN2 backward, per group of query blocks, recomputing the FFN intermediate
  bool first = true;
  // the FFN branch sees dY through its dropout; the residual path sees dY itself
  const void* dYf = dY;
  if (d.drop) {
    RUN("dropout.bwd", 0, (double)T * D * 2 * E_, dropout_scale(E, dY, E, w.dYm, T, D, drop_args(*cfg, 1, 0), s));
    dYf = w.dYm;
  }
  for (int64_t b = 0; b < d.B; b += d.nbg) {
    const int64_t nb = std::min(d.nbg, d.B - b);
    for (int64_t s0 = 0; s0 < S; s0 += d.Rs) {
      const int64_t r = nb * std::min(d.Rs, S - s0), rp = rup(r, 64), t0 = b * S + s0;
      const void* dYg = off(dYf, t0 * D * E_);
      RUN("layernorm.fwd", 0, (double)r * D * (4 + E_),
          layer_norm(F32, E, sv.h + t0 * D, D, p->ln2_g, p->ln2_b, w.vg, D, sv.mu2 + t0, sv.rstd2 + t0, r, D,
                     cfg->ln_eps, 1, s));
      {   // Z^T = W1^T v^T: G^T = GELU(Z^T + b1), GELU'(Z^T)
        GemmArgs g;
        g.A = p->W1; g.lda = F; g.trans_a = 1; g.B = w.vg; g.ldb = D;
        g.C = w.gT; g.ldc = d.Rp; g.C2 = w.gpT; g.ldc2 = d.Rp; g.c2t = GP;
        g.bias = p->b1; g.bias_on_m = 1; g.M = F; g.N = r; g.Nstore = rp; g.K = D;
        RUN("gemm.bwd_ffn1_recompute", gemm_flops(g), gemm_bytes(g, E_, E_ + GP_), gemm(E, act, E, F32, g, s));
      }
      {   // dZ^T = (W2 dY^T) * GELU'(Z^T)
        GemmArgs g;
        g.A = p->W2; g.lda = D; g.B = dYg; g.ldb = D; g.C = w.dzT; g.ldc = d.Rp; g.R = w.gpT; g.ldr = d.Rp;
        g.M = F; g.N = r; g.Nstore = rp; g.K = D;
        RUN("gemm.bwd_dz", gemm_flops(g), gemm_bytes(g, E_, E_ + GP_), gemm(E, EPI_MUL, E, GP, g, s));
      }
      if (G.db1) RUN("reduce.bias", 0, (double)F * r * E_, row_sum(E, w.dzT, d.Rp, F, r, G.db1, first ? 0 : 1, s));
      // K slices of the FFN weight gradients for a group of whole 64-row blocks (every slice
      // inside the group's rows, so no clamped rows)
      const int fz = w.fpart && r % 64 == 0 ? ksplit(D, F, r) : 1;
      if (G.dW2) {   // dW2 = G^T dY, dY read token-major (G^T is zero past the group's rows)
        GemmArgs g;
        g.A = w.gT; g.lda = d.Rp; g.B = dYg; g.ldb = D; g.trans_b = 1; g.b_rows = r;
        g.C = G.dW2; g.ldc = D; g.M = F; g.N = D; g.K = rp; g.accumulate = first ? 0 : 1;
        if (fz > 1) {
          g.b_rows = 0; g.batch = fz; g.K = r / fz; g.sA = g.K; g.sB = g.K * D;
          g.C = w.fpart; g.sC = F * D; g.accumulate = 0;
        }
        RUN("gemm.bwd_dw2", gemm_flops(g), gemm_bytes(g, E_, 4), gemm(E, EPI_STORE, F32, F32, g, s));
        if (fz > 1)
          RUN("reduce.ksplit", 0, (double)(fz + 1) * F * D * 4, sum_slices(w.fpart, fz, F * D, G.dW2, first ? 0 : 1, s));
      }
      {   // dv = dZ W1^T, dZ read from its feature-major copy
        GemmArgs g;
        g.A = w.dzT; g.lda = d.Rp; g.trans_a = 1; g.a_cols = d.Rp;
        g.B = p->W1; g.ldb = F; g.C = w.dv + t0 * D; g.ldc = D;
        g.M = r; g.N = D; g.K = F;
        RUN("gemm.bwd_dv", gemm_flops(g), gemm_bytes(g, E_, 4), gemm(E, EPI_STORE, F32, F32, g, s));
      }
      if (G.dW1) {   // dW1 = v^T dZ, v read token-major (dZ^T is zero past the group's rows)
        GemmArgs g;
        g.A = w.vg; g.lda = D; g.trans_a = 1; g.a_rows = r;
        g.B = w.dzT; g.ldb = d.Rp; g.C = G.dW1; g.ldc = F;
        g.M = D; g.N = F; g.K = rp; g.accumulate = first ? 0 : 1;
        if (fz > 1) {
          g.a_rows = 0; g.batch = fz; g.K = r / fz; g.sA = g.K * D; g.sB = g.K;
          g.C = w.fpart; g.sC = D * F; g.accumulate = 0;
        }
        RUN("gemm.bwd_dw1", gemm_flops(g), gemm_bytes(g, E_, 4), gemm(E, EPI_STORE, F32, F32, g, s));
        if (fz > 1)
          RUN("reduce.ksplit", 0, (double)(fz + 1) * D * F * 4, sum_slices(w.fpart, fz, D * F, G.dW1, first ? 0 : 1, s));
      }
      first = false;
    }
  }
  // dh = dY + LN2^T(dv)
  RUN("layernorm.bwd", 0, (double)T * D * (4 + 4 + E_ + 4 + E_),
      layer_norm_bwd(F32, sv.h, sv.mu2, sv.rstd2, p->ln2_g, w.dv, E, dY, F32, w.dh, E, w.dhe, T, D, s));
  if (G.dln2_g || G.dln2_b)
    RUN("reduce.layernorm", 0, (double)T * D * 8,
        layer_norm_param_grad(F32, sv.h, sv.mu2, sv.rstd2, w.dv, G.dln2_g ? G.dln2_g : w.scratch,
                              G.dln2_b ? G.dln2_b : w.scratch + D, w.partial, T, D, s));
  if (G.db2) RUN("reduce.bias", 0, (double)T * D * E_, col_sum(E, dYf, D, T, D, G.db2, 0, w.partial, s));
  if (d.drop)   // the output projection sees dh through its dropout
    RUN("dropout.bwd", 0, (double)T * D * (4 + E_), dropout_scale(F32, w.dh, E, w.dhe, T, D, drop_args(*cfg, 0, 0), s));

  // ---- output projection backward: dO = dh Wo^T, dWo = O^T dh
  {
    GemmArgs g;
    g.A = w.dhe; g.lda = D; g.B = p->Wo; g.ldb = D; g.C = w.dO; g.ldc = D; g.M = T; g.N = D; g.K = D;
    RUN("gemm.bwd_do", gemm_flops(g), gemm_bytes(g, E_, E_), gemm(E, EPI_STORE, E, F32, g, s));
  }
  // With S % 64 == 0 every sequence is whole 64-token rows (Sp == S): O, dh and u are
  // token-major and the feature-major dQ^T, dK^T, dV^T unpadded over the whole batch, so
  // each D x D weight gradient is one GEMM with K = T (split along K when D < 4096).
  const bool whole = S % 64 == 0;
  const int kz = whole && w.kpart ? ksplit(D, D, T) : 1;
  auto wgrad = [&](const char* name, GemmArgs g, float* out, int64_t sa, int64_t sb) -> bpt_status {
    if (kz > 1) {   // K slices of T / kz tokens; A and B step by sa and sb elements per slice
      g.batch = kz; g.K = T / kz; g.sA = sa * g.K; g.sB = sb * g.K; g.C = w.kpart; g.sC = D * D;
    }
    RUN(name, gemm_flops(g), gemm_bytes(g, E_, 4), gemm(E, EPI_STORE, F32, F32, g, s));
    if (kz > 1) RUN("reduce.ksplit", 0, (double)(kz + 1) * D * D * 4, sum_slices(w.kpart, kz, D * D, out, 0, s));
    return BPT_OK;
  };
  if (G.dWo && whole) {
    GemmArgs g;
    g.A = sv.o; g.lda = D; g.trans_a = 1; g.B = w.dhe; g.ldb = D; g.trans_b = 1; g.C = G.dWo; g.ldc = D;
    g.M = D; g.N = D; g.K = T;
    if ((st = wgrad("gemm.bwd_dwo", g, G.dWo, D, D)) != BPT_OK) return st;
  } else if (G.dWo && S % 32 == 0) {   // per sequence: O and dh both read token-major (K = S exactly)
    for (int b = 0; b < B; ++b) {
      GemmArgs g;
      g.A = off(sv.o, b * S * D * E_); g.lda = D; g.trans_a = 1;
      g.B = off(w.dhe, b * S * D * E_); g.ldb = D; g.trans_b = 1; g.C = G.dWo; g.ldc = D;
      g.M = D; g.N = D; g.K = S; g.accumulate = b > 0;
      RUN("gemm.bwd_dwo", gemm_flops(g), gemm_bytes(g, E_, 4), gemm(E, EPI_STORE, F32, F32, g, s));
    }
  } else if (G.dWo) {   // O read token-major, dh from its zero-padded feature-major copy
    RUN("transpose.act", 0, tb * T * D, transpose(E, w.dhe, D, S * D, w.dhT, Tp, Sp, S, D, Sp, B, s));
    for (int b = 0; b < B; ++b) {
      GemmArgs g;
      g.A = off(sv.o, b * S * D * E_); g.lda = D; g.trans_a = 1; g.a_rows = S;
      g.B = off(w.dhT, b * Sp * E_); g.ldb = Tp; g.C = G.dWo; g.ldc = D;
      g.M = D; g.N = D; g.K = Sp; g.accumulate = b > 0;
      RUN("gemm.bwd_dwo", gemm_flops(g), gemm_bytes(g, E_, 4), gemm(E, EPI_STORE, F32, F32, g, s));
    }
  }

  // ---- attention backward, probabilities rebuilt from the saved log-sum-exp
  RUN("attn.delta", 0, 2.0 * T * D * E_, attn_delta(E, w.dO, sv.o, D, sv.lse, w.ndelta, w.nlse2, B, S, Sp, (int)d.H, (int)d.dh, s));
  {
    AttnArgs a;
    a.q = sv.qkv; a.ld_q = 3 * D;
    a.k = off(sv.qkv, D * E_); a.ld_k = 3 * D;
    a.v = off(sv.qkv, 2 * D * E_); a.ld_v = 3 * D;
    a.dout = w.dO; a.ld_do = D;
    a.dqt = w.dqkvT; a.dkt = off(w.dqkvT, D * Tp * E_); a.dvt = off(w.dqkvT, 2 * D * Tp * E_); a.ld_dt = Tp;
    a.lse = sv.lse; a.ndelta = w.ndelta; a.nlse2 = w.nlse2;
    a.S = S; a.Sp = Sp; a.B = B; a.H = (int)d.H; a.dh = (int)d.dh; a.causal = cfg->causal;
    const double pairs = attn_pairs(0, S, S, cfg->causal) * d.H * B;
    // key-outer: S = Q K^T, dP = dO V^T, dV += P^T dO, dK += dS^T Q (4 contractions)
    RUN("attn.bwd_dkdv", 8.0 * d.dh * pairs, 8.0 * T * D * E_, attn_bwd_dkdv(E, a, s));
    // query-outer: S^T, dP^T, dQ += dS K (3 contractions)
    RUN("attn.bwd_dq", 6.0 * d.dh * pairs, 6.0 * T * D * E_, attn_bwd_dq(E, a, s));
  }

  // ---- QKV projection and LN1 backward
  if (G.dWq || G.dWk || G.dWv) {
    RUN("layernorm.fwd", 0, 2.0 * T * D * E_,
        layer_norm(E, E, X, D, p->ln1_g, p->ln1_b, w.u, D, sv.mu1, sv.rstd1, T, D, cfg->ln_eps, 1, s));
    // per sequence: u read token-major; dQ^T, dK^T, dV^T are zero past the sequence end
    float* outs[3] = {G.dWq, G.dWk, G.dWv};
    for (int i = 0; i < 3; ++i) {
      if (!outs[i]) continue;
      if (whole) {   // u rows and dQ^T / dK^T / dV^T columns contiguous over the batch
        GemmArgs g;
        g.A = w.u; g.lda = D; g.trans_a = 1;
        g.B = off(w.dqkvT, i * D * Tp * E_); g.ldb = Tp; g.C = outs[i]; g.ldc = D;
        g.M = D; g.N = D; g.K = T;
        if ((st = wgrad("gemm.bwd_dwqkv", g, outs[i], D, 1)) != BPT_OK) return st;
        continue;
      }
      for (int b = 0; b < B; ++b) {
        GemmArgs g;
        g.A = off(w.u, b * S * D * E_); g.lda = D; g.trans_a = 1; g.a_rows = S;
        g.B = off(w.dqkvT, (i * D * Tp + b * Sp) * E_); g.ldb = Tp; g.C = outs[i]; g.ldc = D;
        g.M = D; g.N = D; g.K = Sp; g.accumulate = b > 0;
        RUN("gemm.bwd_dwqkv", gemm_flops(g), gemm_bytes(g, E_, 4), gemm(E, EPI_STORE, F32, F32, g, s));
      }
    }
  }
  // dU = [dQ dK dV] [Wq Wk Wv]^T, [dQ dK dV] read feature-major: one GEMM over the batch
  // when its columns are contiguous (S % 64 == 0), else one per sequence
  for (int b = 0; b < (whole ? 1 : B); ++b) {
    GemmArgs g;
    g.A = off(w.dqkvT, b * Sp * E_); g.lda = Tp; g.trans_a = 1; g.a_cols = Tp - b * Sp;
    g.B = w.wcat; g.ldb = 3 * D; g.C = w.dU + b * S * D; g.ldc = D; g.M = whole ? T : S; g.N = D; g.K = 3 * D;
    RUN("gemm.bwd_du", gemm_flops(g), gemm_bytes(g, E_, 4), gemm(E, EPI_STORE, F32, F32, g, s));
  }
  RUN("layernorm.bwd", 0, (double)T * D * (E_ + 4 + 4 + EO),
      layer_norm_bwd(E, X, sv.mu1, sv.rstd1, p->ln1_g, w.dU, F32, w.dh, OUT, dX, OUT, nullptr, T, D, s));
  if (G.dln1_g || G.dln1_b)
    RUN("reduce.layernorm", 0, (double)T * D * (E_ + 4),
        layer_norm_param_grad(E, X, sv.mu1, sv.rstd1, w.dU, G.dln1_g ? G.dln1_g : w.scratch,
                              G.dln1_b ? G.dln1_b : w.scratch + D, w.partial, T, D, s));
  return BPT_OK;
}

// ---------------------------------------------------------------- cross-entropy of an LM head
bpt_status bpt_xent_validate(const bpt_xent_config* cfg) { return xent_check(cfg); }

size_t bpt_xent_workspace_bytes(const bpt_xent_config* cfg, int backward) {
  if (xent_check(cfg) != BPT_OK) return 0;
  int64_t total;
  xent_ws(xent_dims(*cfg), nullptr, backward, &total);
  return (size_t)total;
}

bpt_status bpt_xent_fwd(const bpt_xent_config* cfg, const void* h, const void* W, const int32_t* targets,
                        float* loss, float* lse, void* ws, size_t ws_bytes, void* stream) {
  bpt_status st = xent_check(cfg);
  if (st != BPT_OK) return st;
  const void* ptrs[] = {h, W, targets, loss, lse, ws};
  for (const void* q : ptrs) {
    if (!q) return fail(BPT_ERR_INVALID_ARG, "h, W, targets, loss, lse and workspace must not be NULL");
    if (!aligned16(q)) return fail(BPT_ERR_INVALID_ARG, "pointer %p is not 16-byte aligned", q);
  }
  const XentDims d = xent_dims(*cfg);
  int64_t need;
  XentWs w = xent_ws(d, ws, 0, &need);
  if ((int64_t)ws_bytes < need)
    return fail(BPT_ERR_WORKSPACE, "workspace %zu bytes < required %lld", ws_bytes, (long long)need);
  hipStream_t s = (hipStream_t)stream;
  const Dt E = cfg->dtype == BPT_BF16 ? BF16 : F32;
  const int64_t E_ = (int64_t)d.E;
  for (int64_t t0 = 0; t0 < d.T; t0 += d.R) {
    const int64_t r = std::min(d.R, d.T - t0);
    GemmArgs g;   // logits of the block: h W, W read as it is stored (B operand K-major)
    g.A = (const char*)h + t0 * d.D * E_; g.lda = d.D;
    g.B = W; g.ldb = d.ldw; g.trans_b = 1;
    g.C = w.logits; g.ldc = d.ldw; g.M = r; g.N = d.ldw; g.K = d.D;
    RUN("xent.logits", gemm_flops(g), gemm_bytes(g, E_, 4), gemm(E, EPI_STORE, F32, F32, g, s));
    RUN("xent.rows", 0, (double)r * d.ldw * 4,
        xent_rows(w.logits, d.ldw, r, d.V, targets + t0, lse + t0, w.tok + t0, s));
  }
  RUN("xent.mean", 0, (double)d.T * 4, mean_of(w.tok, d.T, loss, s));
  return BPT_OK;
}

bpt_status bpt_xent_bwd(const bpt_xent_config* cfg, const void* h, const void* W, const int32_t* targets,
                        const float* lse, float dloss, void* dh, float* dW, void* ws, size_t ws_bytes,
                        void* stream) {
  bpt_status st = xent_check(cfg);
  if (st != BPT_OK) return st;
  const void* ptrs[] = {h, W, targets, lse, dh, ws};
  for (const void* q : ptrs) {
    if (!q) return fail(BPT_ERR_INVALID_ARG, "h, W, targets, lse, dh and workspace must not be NULL");
    if (!aligned16(q)) return fail(BPT_ERR_INVALID_ARG, "pointer %p is not 16-byte aligned", q);
  }
  if (dW && !aligned16(dW)) return fail(BPT_ERR_INVALID_ARG, "pointer %p is not 16-byte aligned", (void*)dW);
  const XentDims d = xent_dims(*cfg);
  int64_t need;
  XentWs w = xent_ws(d, ws, 1, &need);
  if ((int64_t)ws_bytes < need)
    return fail(BPT_ERR_WORKSPACE, "workspace %zu bytes < required %lld", ws_bytes, (long long)need);
  hipStream_t s = (hipStream_t)stream;
  const Dt E = cfg->dtype == BPT_BF16 ? BF16 : F32;
  const int64_t E_ = (int64_t)d.E;
  for (int64_t t0 = 0; t0 < d.T; t0 += d.R) {
    const int64_t r = std::min(d.R, d.T - t0), rp = rup(r, 64);
    const char* hb = (const char*)h + t0 * d.D * E_;
    {   // G^T [ldw, rp] = (dloss / T)(softmax - onehot) of the block's logits, recomputed
        // transposed (W read as stored is the K-major A operand, h the contiguous B);
        // columns past r and rows past V are written as zeros
      GemmArgs g;
      g.A = W; g.lda = d.ldw; g.trans_a = 1; g.B = hb; g.ldb = d.D;
      g.C = w.g; g.ldc = d.Rp; g.M = d.ldw; g.N = r; g.Nstore = rp; g.K = d.D;
      g.alpha = dloss / (float)d.T; g.rowv = lse + t0; g.tgt = targets + t0; g.nvalid = d.V;
      RUN("xent.grad_logits", gemm_flops(g), gemm_bytes(g, E_, E_), gemm(E, EPI_XENT_T, E, F32, g, s));
    }
    {   // dh = G W^T: G read from its transposed copy (K-major A), W rows contiguous along
        // the vocabulary
      GemmArgs g;
      g.A = w.g; g.lda = d.Rp; g.trans_a = 1; g.a_cols = d.Rp; g.B = W; g.ldb = d.ldw;
      g.C = (char*)dh + t0 * d.D * E_; g.ldc = d.D; g.M = r; g.N = d.D; g.K = d.ldw;
      RUN("xent.dh", gemm_flops(g), gemm_bytes(g, E_, E_), gemm(E, EPI_STORE, E, F32, g, s));
    }
    if (dW) {   // dW = h^T G: h read token-major (K-major A), G^T rows contiguous along the
                // tokens (zero past row r)
      GemmArgs g;
      g.A = hb; g.lda = d.D; g.trans_a = 1; g.a_rows = r;
      g.B = w.g; g.ldb = d.Rp;
      g.C = dW; g.ldc = d.ldw; g.M = d.D; g.N = d.ldw; g.K = rp; g.accumulate = t0 > 0;
      RUN("xent.dW", gemm_flops(g), gemm_bytes(g, E_, 4), gemm(E, EPI_STORE, F32, F32, g, s));
    }
  }
  return BPT_OK;
}

// ---------------------------------------------------------------- GPT training step pieces
static bpt_status dtype_ok(int32_t t, const char* what) {
  if (t != BPT_F32 && t != BPT_BF16) return fail(BPT_ERR_INVALID_ARG, "%s %d is not a bpt_dtype", what, (int)t);
  return BPT_OK;
}
static Dt dt_of(int32_t t) { return t == BPT_BF16 ? BF16 : F32; }

static bpt_status embed_check(const bpt_embed_config* c) {
  if (!c) return fail(BPT_ERR_INVALID_ARG, "NULL config");
  if (c->B < 1 || c->S < 1 || c->D < 1 || c->V < 1)
    return fail(BPT_ERR_INVALID_ARG, "B, S, D, V must be >= 1");
  if (c->D % 8) return fail(BPT_ERR_UNSUPPORTED, "D = %lld is not a multiple of 8", (long long)c->D);
  if (c->B * c->S > INT32_MAX / 4 || c->V > INT32_MAX)
    return fail(BPT_ERR_UNSUPPORTED, "B*S or V too large");
  bpt_status st = dtype_ok(c->dtype, "dtype");
  return st != BPT_OK ? st : dtype_ok(c->grad_dtype, "grad_dtype");
}

bpt_status bpt_embed_fwd(const bpt_embed_config* cfg, const int32_t* tokens, const void* Wte, const void* Wpe,
                         void* X, void* stream) {
  bpt_status st = embed_check(cfg);
  if (st != BPT_OK) return st;
  if (!tokens || !Wte || !X) return fail(BPT_ERR_INVALID_ARG, "NULL tokens, Wte or X");
  const void* ptrs[] = {tokens, Wte, Wpe, X};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return fail(BPT_ERR_INVALID_ARG, "pointer %p is not 16-byte aligned", q);
  hipStream_t s = (hipStream_t)stream;
  const int64_t T = cfg->B * cfg->S, E_ = cfg->dtype == BPT_BF16 ? 2 : 4;
  RUN("gpt.embed", 0, (double)T * 4 + (double)T * cfg->D * E_ * (Wpe ? 3 : 2),
      embed_fwd(dt_of(cfg->dtype), tokens, Wte, Wpe, X, T, cfg->S, cfg->D, cfg->V, s));
  return BPT_OK;
}

bpt_status bpt_embed_bwd(const bpt_embed_config* cfg, const int32_t* tokens, const void* dX, float* dWte,
                         float* dWpe, void* stream) {
  bpt_status st = embed_check(cfg);
  if (st != BPT_OK) return st;
  if (!tokens || !dX) return fail(BPT_ERR_INVALID_ARG, "NULL tokens or dX");
  const void* ptrs[] = {tokens, dX, dWte, dWpe};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return fail(BPT_ERR_INVALID_ARG, "pointer %p is not 16-byte aligned", q);
  hipStream_t s = (hipStream_t)stream;
  const int64_t T = cfg->B * cfg->S, G_ = cfg->grad_dtype == BPT_BF16 ? 2 : 4;
  const Dt GT = dt_of(cfg->grad_dtype);
  if (dWte)
    RUN("gpt.embed_dWte", 0, (double)cfg->V * cfg->D * 4 + (double)T * cfg->D * (G_ + 4),
        embed_dwte(GT, tokens, dX, dWte, T, cfg->D, cfg->V, s));
  if (dWpe)
    RUN("gpt.embed_dWpe", 0, (double)T * cfg->D * G_ + (double)cfg->S * cfg->D * 4,
        embed_dwpe(GT, dX, dWpe, cfg->B, cfg->S, cfg->D, s));
  return BPT_OK;
}

static bpt_status ln_check(const bpt_ln_config* c) {
  if (!c) return fail(BPT_ERR_INVALID_ARG, "NULL config");
  if (c->rows < 1 || c->D < 1) return fail(BPT_ERR_INVALID_ARG, "rows and D must be >= 1");
  if (c->D % 8) return fail(BPT_ERR_UNSUPPORTED, "D = %lld is not a multiple of 8", (long long)c->D);
  if (!(c->eps >= 0.0f)) return fail(BPT_ERR_INVALID_ARG, "eps must be >= 0");
  if (c->rows > INT32_MAX) return fail(BPT_ERR_UNSUPPORTED, "rows too large");
  bpt_status st = dtype_ok(c->in_dtype, "in_dtype");
  return st != BPT_OK ? st : dtype_ok(c->out_dtype, "out_dtype");
}

// workspace of bpt_ln_bwd: column-sum partials, then (bf16 dY) an fp32 copy of dY
static int64_t ln_ws_parts(const bpt_ln_config& c, int64_t* dy_off) {
  const int64_t part = rup((int64_t)layer_norm_param_grad_ws(c.D) * 4, kAlign);
  *dy_off = part;
  return part + (c.out_dtype == BPT_BF16 ? rup(c.rows * c.D * 4, kAlign) : 0);
}

size_t bpt_ln_workspace_bytes(const bpt_ln_config* cfg) {
  if (ln_check(cfg) != BPT_OK) return 0;
  int64_t o;
  return (size_t)ln_ws_parts(*cfg, &o);
}

bpt_status bpt_ln_fwd(const bpt_ln_config* cfg, const void* X, const float* g, const float* b, void* Y,
                      float* mean, float* rstd, void* stream) {
  bpt_status st = ln_check(cfg);
  if (st != BPT_OK) return st;
  if (!X || !Y || !mean || !rstd) return fail(BPT_ERR_INVALID_ARG, "NULL X, Y, mean or rstd");
  if (X == Y) return fail(BPT_ERR_INVALID_ARG, "Y must not alias X");
  const void* ptrs[] = {X, g, b, Y, mean, rstd};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return fail(BPT_ERR_INVALID_ARG, "pointer %p is not 16-byte aligned", q);
  hipStream_t s = (hipStream_t)stream;
  const int64_t R = cfg->rows, D = cfg->D;
  const double io = (double)R * D * ((cfg->in_dtype == BPT_BF16 ? 2 : 4) + (cfg->out_dtype == BPT_BF16 ? 2 : 4));
  RUN("gpt.ln_f", 0, io + (double)R * 8,
      layer_norm(dt_of(cfg->in_dtype), dt_of(cfg->out_dtype), X, D, g, b, Y, D, mean, rstd, R, D, cfg->eps, 0, s));
  return BPT_OK;
}

bpt_status bpt_ln_bwd(const bpt_ln_config* cfg, const void* X, const float* g, const float* mean,
                      const float* rstd, const void* dY, void* dX, float* dg, float* db, void* ws,
                      size_t ws_bytes, void* stream) {
  bpt_status st = ln_check(cfg);
  if (st != BPT_OK) return st;
  if (!X || !mean || !rstd || !dY || !dX || !ws)
    return fail(BPT_ERR_INVALID_ARG, "NULL X, mean, rstd, dY, dX or workspace");
  if (dX == dY || dX == X) return fail(BPT_ERR_INVALID_ARG, "dX must not alias dY or X");
  if ((dg == nullptr) != (db == nullptr))
    return fail(BPT_ERR_INVALID_ARG, "dg and db must both be given or both be NULL");
  const void* ptrs[] = {X, g, mean, rstd, dY, dX, dg, db, ws};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return fail(BPT_ERR_INVALID_ARG, "pointer %p is not 16-byte aligned", q);
  int64_t dy_off;
  const int64_t need = ln_ws_parts(*cfg, &dy_off);
  if ((int64_t)ws_bytes < need)
    return fail(BPT_ERR_WORKSPACE, "workspace %zu bytes < required %lld", ws_bytes, (long long)need);
  hipStream_t s = (hipStream_t)stream;
  const int64_t R = cfg->rows, D = cfg->D;
  const Dt TI = dt_of(cfg->in_dtype);
  const int64_t I_ = cfg->in_dtype == BPT_BF16 ? 2 : 4;
  float* partial = (float*)ws;
  const float* dy32 = (const float*)dY;
  if (cfg->out_dtype == BPT_BF16) {
    float* c = (float*)off(ws, dy_off);
    RUN("gpt.ln_f_dy32", 0, (double)R * D * 6, bf16_to_f32(dY, c, R * D, s));
    dy32 = c;
  }
  RUN("gpt.ln_f_bwd", 0, (double)R * D * (2 * I_ + 4) + (double)R * 8,
      layer_norm_bwd(TI, X, mean, rstd, g, dy32, F32, nullptr, TI, dX, TI, nullptr, R, D, s));
  if (dg) {
    RUN("gpt.ln_f_params", 0, (double)R * D * (I_ + 4),
        layer_norm_param_grad(TI, X, mean, rstd, dy32, dg, db, partial, R, D, s));
  }
  return BPT_OK;
}

bpt_status bpt_adamw_step(const bpt_adamw_config* cfg, int64_t n, float* p, const float* g, float* m, float* v,
                          void* p_lowp, void* stream) {
  if (!cfg) return fail(BPT_ERR_INVALID_ARG, "NULL config");
  if (n < 0) return fail(BPT_ERR_INVALID_ARG, "n must be >= 0");
  if (cfg->step < 1) return fail(BPT_ERR_INVALID_ARG, "step must be >= 1");
  if (!(cfg->beta1 >= 0.0f && cfg->beta1 < 1.0f && cfg->beta2 >= 0.0f && cfg->beta2 < 1.0f))
    return fail(BPT_ERR_INVALID_ARG, "beta1 and beta2 must lie in [0, 1)");
  if (!(cfg->eps > 0.0f) || !(cfg->lr >= 0.0f) || !(cfg->weight_decay >= 0.0f))
    return fail(BPT_ERR_INVALID_ARG, "eps must be > 0, lr and weight_decay >= 0");
  if (p_lowp) {
    bpt_status st = dtype_ok(cfg->lowp_dtype, "lowp_dtype");
    if (st != BPT_OK) return st;
  }
  if (n == 0) return BPT_OK;
  if (!p || !g || !m || !v) return fail(BPT_ERR_INVALID_ARG, "NULL p, g, m or v");
  const void* ptrs[] = {p, g, m, v, p_lowp};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return fail(BPT_ERR_INVALID_ARG, "pointer %p is not 16-byte aligned", q);
  hipStream_t s = (hipStream_t)stream;
  const double c1 = 1.0 / (1.0 - std::pow((double)cfg->beta1, (double)cfg->step));
  const double c2 = 1.0 / (1.0 - std::pow((double)cfg->beta2, (double)cfg->step));
  const int64_t L_ = p_lowp ? (cfg->lowp_dtype == BPT_BF16 ? 2 : 4) : 0;
  RUN("gpt.adamw", 0, (double)n * (28 + L_),
      adamw(dt_of(cfg->lowp_dtype), p, g, m, v, p_lowp, n, cfg->lr, cfg->beta1, cfg->beta2, cfg->eps,
            cfg->weight_decay, (float)c1, (float)c2, s));
  return BPT_OK;
}

}  // extern "C"

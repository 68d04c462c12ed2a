// C ABI of librft: argument validation, workspace layout and the launch
// sequence of every entry point declared in rft.h.  Every call enqueues on the
// caller's stream and returns without synchronising.
#include <stdarg.h>
#include <stdio.h>

#include <cmath>
#include <algorithm>
#include <limits>
#include <mutex>
#include <string>

#include "rft_internal.h"

using namespace rft;

namespace {

thread_local std::string g_err;

rft_status fail(rft_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

rft_status hip_fail(hipError_t e, const char* where) {
  return fail(RFT_E_HIP, "%s: HIP error %d (%s)", where, (int)e, hipGetErrorString(e));
}

#define RFT_HIP(call, where)                        \
  do {                                              \
    hipError_t e_ = (call);                         \
    if (e_ != hipSuccess) return hip_fail(e_, where); \
  } while (0)

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

rft_status check_tokens(const rft_tokens* tok, const char* fn) {
  if (!tok) return fail(RFT_E_NULL, "%s: tokens is NULL", fn);
  if (tok->T < 0 || tok->n_seq < 0)
    return fail(RFT_E_SHAPE, "%s: T=%lld n_seq=%lld must be >= 0", fn, (long long)tok->T,
                (long long)tok->n_seq);
  if (tok->T > (int64_t)std::numeric_limits<int32_t>::max() / 2)
    return fail(RFT_E_SHAPE, "%s: T=%lld exceeds the supported 2^30 rows", fn, (long long)tok->T);
  if (tok->n_seq == 0 && tok->T != 0)
    return fail(RFT_E_SHAPE, "%s: T=%lld rows but n_seq = 0", fn, (long long)tok->T);
  if (!tok->seq_start) return fail(RFT_E_NULL, "%s: tokens.seq_start is NULL", fn);
  if (tok->T > 0 && (!tok->mask || !tok->token_ids))
    return fail(RFT_E_NULL, "%s: tokens.mask / tokens.token_ids is NULL", fn);
  return RFT_OK;
}

rft_status check_hw(const char* fn, int64_t T, const void* hidden, const void* weight, int dtype,
                    int64_t d, int64_t V) {
  if (dtype != RFT_F32 && dtype != RFT_BF16) return fail(RFT_E_DTYPE, "%s: dtype %d unknown", fn, dtype);
  if (d < 1 || V < 1) return fail(RFT_E_SHAPE, "%s: d=%lld V=%lld must be >= 1", fn, (long long)d, (long long)V);
  if (V > (int64_t)std::numeric_limits<int32_t>::max() / 2 || d > (1 << 20))
    return fail(RFT_E_SHAPE, "%s: d=%lld V=%lld too large", fn, (long long)d, (long long)V);
  if (!weight || (T > 0 && !hidden)) return fail(RFT_E_NULL, "%s: hidden / weight is NULL", fn);
  if (dtype == RFT_BF16) {
    if (d % 8) return fail(RFT_E_SHAPE, "%s: bf16 needs d %% 8 == 0 (d=%lld)", fn, (long long)d);
    // a 256-row tile of dZ [rows, Vpad] is one buffer descriptor (< 2^31 bytes)
    if (round_up(V, 256) * 2 * 256 >= ((int64_t)1 << 31))
      return fail(RFT_E_SHAPE, "%s: bf16 supports V <= %lld (V=%lld)", fn,
                  (long long)(((int64_t)1 << 22) - 256), (long long)V);
    if ((hidden && !aligned16(hidden)) || !aligned16(weight))
      return fail(RFT_E_SHAPE, "%s: bf16 hidden / weight must be 16-byte aligned", fn);
  }
  return RFT_OK;
}

rft_status check_params(const rft_ppo_params* p, const char* fn) {
  if (!p) return fail(RFT_E_NULL, "%s: params is NULL", fn);
  if (!(p->eps_low >= 0.f && p->eps_low <= 1.f))
    return fail(RFT_E_PARAM, "%s: eps_low=%g must be in [0, 1]", fn, (double)p->eps_low);
  if (!(p->eps_high >= 0.f)) return fail(RFT_E_PARAM, "%s: eps_high=%g must be >= 0", fn, (double)p->eps_high);
  if (!(p->kl_coef >= 0.f) || !std::isfinite(p->kl_coef))
    return fail(RFT_E_PARAM, "%s: kl_coef=%g must be finite and >= 0", fn, (double)p->kl_coef);
  if (p->agg != RFT_AGG_SEQ_MEAN_TOKEN_MEAN && p->agg != RFT_AGG_TOKEN_MEAN)
    return fail(RFT_E_PARAM, "%s: agg=%d unknown", fn, p->agg);
  if (!(p->denom_override >= 0.0) || !std::isfinite(p->denom_override))
    return fail(RFT_E_PARAM, "%s: denom_override=%g must be finite and >= 0", fn, p->denom_override);
  if (!(p->mix_mu >= 0.f && p->mix_mu <= 1.f))
    return fail(RFT_E_PARAM, "%s: mix_mu=%g must be in [0, 1]", fn, (double)p->mix_mu);
  if (!(p->entropy_coef >= 0.f) || !std::isfinite(p->entropy_coef))
    return fail(RFT_E_PARAM, "%s: entropy_coef=%g must be finite and >= 0", fn,
                (double)p->entropy_coef);
  return RFT_OK;
}

LossConst loss_const(const rft_ppo_params* p, int64_t V) {
  LossConst c;
  c.eps_low = p->eps_low;
  c.eps_high = p->eps_high;
  c.beta = p->kl_coef;
  c.agg = p->agg;
  c.denom = p->denom_override;
  c.V = V;
  c.thr_lo = p->eps_low < 1.f ? (float)std::log(1.0 - (double)p->eps_low)
                              : -std::numeric_limits<float>::infinity();
  c.thr_hi = std::isfinite(p->eps_high) ? (float)std::log1p((double)p->eps_high)
                                        : std::numeric_limits<float>::infinity();
  c.is_expert = nullptr;
  c.mix = 0;
  c.mu = p->mix_mu;
  c.ent_coef = p->entropy_coef;
  return c;
}

LossConst loss_const(const rft_ppo_params* p, int64_t V, const rft_tokens& tok) {
  LossConst c = loss_const(p, V);
  c.is_expert = tok.is_expert;
  c.mix = tok.is_expert ? 1 : 0;
  return c;
}

rft_status check_ws(const char* fn, void* ws, size_t have, size_t need) {
  if (need == 0) return RFT_OK;
  if (!ws) return fail(RFT_E_WORKSPACE, "%s: workspace is NULL (%zu bytes needed)", fn, need);
  if (!aligned16(ws)) return fail(RFT_E_WORKSPACE, "%s: workspace must be 16-byte aligned", fn);
  if (have < need) return fail(RFT_E_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, have, need);
  return RFT_OK;
}

// ---------------------------------------------------- workspace layouts --
struct FwdWs {
  TokMeta m;
  uint16_t* hc;  // compacted hidden rows (bf16 path): row-major, or tile-blocked
  uint16_t* wb;  // tile-blocked copy of W [Vpad, d] (blocked bf16 path only)
  float *pm, *ps, *pu, *zy;
  int ntiles;
  int64_t ldp;
  size_t bytes;
};
bool fwd_blocked_ok(int dtype, int64_t d) { return dtype == RFT_BF16 && mfma_fwd_blk_ok(d); }
// blocked: the bf16 forward from tile-blocked copies of the compacted rows
// [round_up(T, 256), d] and of W [Vpad, d] (d a multiple of 64), for the
// 384 x 256 GEMM tile; the copy of W adds Vpad d 2 bytes.
FwdWs carve_fwd(void* base, const rft_tokens& tok, int64_t d, int64_t V, int dtype,
                bool blocked = false) {
  Carver c(base);
  FwdWs w;
  w.m = carve_tokmeta(c, tok.T, tok.n_seq);
  const int64_t hrows = blocked ? round_up(tok.T > 0 ? tok.T : 1, 256) : (tok.T > 0 ? tok.T : 1);
  w.hc = dtype == RFT_BF16 ? c.take<uint16_t>((size_t)hrows * d) : nullptr;
  w.wb = blocked ? c.take<uint16_t>((size_t)round_up(V, 256) * d) : nullptr;
  int tn = dtype == RFT_BF16 ? kMfmaTileN : kSimtTileN;
  w.ntiles = (int)((V + tn - 1) / tn);
  w.ldp = tok.T > 0 ? tok.T : 1;
  w.pm = c.take<float>((size_t)w.ntiles * w.ldp);
  w.ps = c.take<float>((size_t)w.ntiles * w.ldp);
  w.pu = c.take<float>((size_t)w.ntiles * w.ldp);
  w.zy = c.take<float>((size_t)w.ldp);
  w.bytes = c.bytes();
  return w;
}

struct LossWs {
  TokMeta m;
  LossPartial* parts;
  LossPartial* parts2;  // per_row: the partials of 256-row blocks (nullptr otherwise)
  size_t bytes;
};
LossWs carve_loss(void* base, const rft_tokens& tok, bool per_row) {
  Carver c(base);
  LossWs w;
  w.m = carve_tokmeta(c, tok.T, tok.n_seq);
  int64_t np = per_row ? tok.T : (tok.T + 255) / 256;
  w.parts = c.take<LossPartial>(np > 0 ? np : 1);
  w.parts2 = per_row ? c.take<LossPartial>((size_t)((np + 255) / 256 > 0 ? (np + 255) / 256 : 1))
                     : nullptr;
  w.bytes = c.bytes();
  return w;
}

struct DpoCarve {
  TokMeta m;
  DpoWs d;
  size_t bytes;
};
DpoCarve carve_dpo(void* base, const rft_tokens& tok) {
  Carver c(base);
  DpoCarve w;
  w.m = carve_tokmeta(c, tok.T, tok.n_seq);
  const size_t n = (size_t)(tok.n_seq > 0 ? tok.n_seq : 1);
  w.d.pi = c.take<double>(n);
  w.d.rho = c.take<double>(n);
  w.d.bad = c.take<int32_t>(n);
  w.d.coef = c.take<float>(n);
  w.bytes = c.bytes();
  return w;
}

struct BwdWs {
  TokMeta m;
  uint16_t *hc, *wt, *dz, *dzt, *hct;  // bf16 path: wt, dz, dZ^T, Hc^T tile-blocked
  float* dz32;                         // fp32 path
  int64_t Tc, Vpad, dpad;
  size_t bytes;
};
constexpr int64_t kBf16Align = 256;   // row chunk / vocabulary padding of the bf16 path
constexpr int64_t kF32Align = 64;
constexpr int64_t kRecommendTc = 131072;

BwdWs carve_bwd(void* base, const rft_tokens& tok, int64_t d, int64_t V, int dtype, int64_t Tc) {
  Carver c(base);
  BwdWs w = {};
  w.m = carve_tokmeta(c, tok.T, tok.n_seq);
  w.Tc = Tc;
  if (dtype == RFT_BF16) {
    w.Vpad = round_up(V, kBf16Align);
    w.dpad = round_up(d, kBf16Align);
    w.hc = c.take<uint16_t>((size_t)(tok.T > 0 ? tok.T : 1) * d);
    w.wt = c.take<uint16_t>((size_t)w.dpad * w.Vpad);
    w.dz = c.take<uint16_t>((size_t)Tc * w.Vpad);
    w.dzt = c.take<uint16_t>((size_t)w.Vpad * Tc);
    w.hct = c.take<uint16_t>((size_t)w.dpad * Tc);
  } else {
    w.Vpad = round_up(V, kF32Align);
    w.dz32 = c.take<float>((size_t)Tc * w.Vpad);
  }
  w.bytes = c.bytes();
  return w;
}

int64_t bwd_align(int dtype) { return dtype == RFT_BF16 ? kBf16Align : kF32Align; }

// Upper bound of a row chunk: the dW GEMM reads 256-row panels of the
// tile-blocked transposed chunk buffers (256 Tc bf16 values) through one
// buffer descriptor with 32-bit offsets, so 256 Tc 2 bytes must stay below
// 2^31.  2^21 rows is below that bound for both dtypes.
constexpr int64_t kMaxTc = (int64_t)1 << 21;
static_assert(256 * kMaxTc * 2 < ((int64_t)1 << 31), "chunk panel must fit a descriptor");

int64_t bwd_tc_max(const rft_tokens& tok, int dtype) {
  int64_t a = bwd_align(dtype);
  int64_t t = round_up(tok.T > 0 ? tok.T : 1, a);
  return t < kMaxTc ? t : kMaxTc;
}

// largest row chunk (a multiple of the alignment) whose workspace fits, 0 if none
int64_t bwd_tc_for(const rft_tokens& tok, int64_t d, int64_t V, int dtype, size_t ws_bytes) {
  int64_t a = bwd_align(dtype);
  int64_t kmax = bwd_tc_max(tok, dtype) / a;
  if (carve_bwd(nullptr, tok, d, V, dtype, a).bytes > ws_bytes) return 0;
  int64_t lo = 1, hi = kmax;  // invariant: chunk lo*a fits
  while (lo < hi) {
    int64_t mid = (lo + hi + 1) / 2;
    if (carve_bwd(nullptr, tok, d, V, dtype, mid * a).bytes <= ws_bytes) lo = mid; else hi = mid - 1;
  }
  return lo * a;
}

// Fused step (bf16): compacted hidden rows, transposed weight, per-chunk
// log-sum-exp partials, the sampled logits, the loss partials, the chunk
// buffer (fp16 y, then bf16 dZ, in dz) and the chunk's dZ^T [Vpad, Tc] and
// hidden rows transposed [dpad, Tc] (the weight gradient's K-contiguous
// operands).  W^T, dz, dZ^T and Hc^T are tile-blocked (blk_index): every
// k-step of the backward GEMMs reads contiguous 32 KiB blocks.
struct StepWs {
  TokMeta m;
  uint16_t *hc, *wb, *wt, *dz, *dzt, *hct;  // hc [Tpad, Kp], wb [Vpad, Kp] blocked (forward)
  float *pm, *ps, *pu, *zy;
  float *ce, *cmu;  // per chunk row: entropy-bonus coefficient and softmax mean
  LossPartial* parts;
  int ntiles;
  int64_t Tc, Vpad, dpad, Kp;
  size_t bytes;
};
StepWs carve_step(void* base, const rft_tokens& tok, int64_t d, int64_t V, int64_t Tc) {
  Carver c(base);
  StepWs w = {};
  const int64_t T1 = tok.T > 0 ? tok.T : 1;
  w.m = carve_tokmeta(c, tok.T, tok.n_seq);
  w.Tc = Tc;
  w.Vpad = round_up(V, kBf16Align);
  w.ntiles = (int)(w.Vpad / kMfmaTileN);
  w.dpad = round_up(d, kBf16Align);
  w.Kp = round_up(d, 64);
  w.hc = c.take<uint16_t>((size_t)round_up(T1, kBf16Align) * w.Kp);
  w.wb = c.take<uint16_t>((size_t)w.Vpad * w.Kp);
  w.wt = c.take<uint16_t>((size_t)w.dpad * w.Vpad);
  w.pm = c.take<float>((size_t)w.ntiles * Tc);
  w.ps = c.take<float>((size_t)w.ntiles * Tc);
  w.pu = c.take<float>((size_t)w.ntiles * Tc);
  w.zy = c.take<float>((size_t)T1);
  w.ce = c.take<float>((size_t)Tc);
  w.cmu = c.take<float>((size_t)Tc);
  w.parts = c.take<LossPartial>((size_t)((T1 + 255) / 256));
  w.dz = c.take<uint16_t>((size_t)Tc * w.Vpad);
  w.dzt = c.take<uint16_t>((size_t)w.Vpad * Tc);
  w.hct = c.take<uint16_t>((size_t)w.dpad * Tc);
  w.bytes = c.bytes();
  return w;
}

// largest row chunk (a multiple of 256) whose step workspace fits, 0 if none
int64_t step_tc_for(const rft_tokens& tok, int64_t d, int64_t V, size_t ws_bytes) {
  const int64_t a = kBf16Align;
  const int64_t kmax = bwd_tc_max(tok, RFT_BF16) / a;
  if (carve_step(nullptr, tok, d, V, a).bytes > ws_bytes) return 0;
  int64_t lo = 1, hi = kmax;
  while (lo < hi) {
    int64_t mid = (lo + hi + 1) / 2;
    if (carve_step(nullptr, tok, d, V, mid * a).bytes <= ws_bytes) lo = mid; else hi = mid - 1;
  }
  return lo * a;
}

// fp32 step: the three calls share the front of the workspace; the entropy
// bonus coefficients [T] follow it.
size_t step_f32_front(const rft_tokens& tok, int64_t d, int64_t V, int64_t Tc) {
  size_t a = carve_fwd(nullptr, tok, d, V, RFT_F32).bytes;
  size_t b = carve_loss(nullptr, tok, false).bytes;
  size_t c = carve_bwd(nullptr, tok, d, V, RFT_F32, Tc).bytes;
  return (size_t)round_up((int64_t)std::max(a, std::max(b, c)), 256);
}
size_t step_f32_bytes(const rft_tokens& tok, int64_t d, int64_t V, int64_t Tc) {
  return step_f32_front(tok, d, V, Tc) + (size_t)round_up((tok.T > 0 ? tok.T : 1) * 4, 256);
}

rft_status check_fused_logits(const char* fn, const rft_tokens* tok, const float* logits, int64_t V,
                              const float* old_logp, const float* ref_logp, const float* adv,
                              const rft_ppo_params* params, const float* logp,
                              const float* d_logits, const rft_ppo_stats* stats) {
  rft_status st = check_tokens(tok, fn);
  if (st) return st;
  if ((st = check_params(params, fn))) return st;
  if (V < 1 || V > (int64_t)std::numeric_limits<int32_t>::max() / 2)
    return fail(RFT_E_SHAPE, "%s: V=%lld", fn, (long long)V);
  if (!stats) return fail(RFT_E_NULL, "%s: stats is NULL", fn);
  if (tok->T > 0 && (!logits || !old_logp || !adv || !logp || !d_logits))
    return fail(RFT_E_NULL, "%s: logits / old_logp / adv / logp / d_logits is NULL", fn);
  if (tok->T > 0 && params->kl_coef > 0.f && !ref_logp)
    return fail(RFT_E_NULL, "%s: ref_logp is NULL with kl_coef > 0", fn);
  return RFT_OK;
}

// Scratch of the entry point that allocates nothing
// (rft_ppo_clip_fused_logits_noalloc): the workspace of the loss-only call
// (token bookkeeping and one loss partial per row) in a file-scope device
// array.  Each GPU holds its own copy for the life of the process; in host
// code `scratch` only names the symbol, so kernels get the device address
// looked up once per device (scratch_ptr).
constexpr size_t kNoAllocScratchBytes = (size_t)16 << 20;
constexpr int kNoAllocMaxDevices = 64;
__attribute__((used)) static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kNoAllocMaxDevices] = {};

// Device address of this device's scratch array (looked up on the first call
// on each device, with that device current); nullptr and *e set on failure.
void* scratch_ptr(hipError_t* e) {
  int dev = -1;
  *e = hipGetDevice(&dev);
  if (*e != hipSuccess) return nullptr;
  if (dev < 0 || dev >= kNoAllocMaxDevices) {
    *e = hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    *e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (*e != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

// ================================================================== ABI ==
extern "C" {

int rft_abi_version(void) { return RFT_ABI_VERSION; }

const char* rft_status_str(int s) {
  switch (s) {
    case RFT_OK: return "ok";
    case RFT_E_NULL: return "null pointer";
    case RFT_E_SHAPE: return "invalid shape";
    case RFT_E_DTYPE: return "invalid dtype";
    case RFT_E_PARAM: return "invalid parameter";
    case RFT_E_WORKSPACE: return "workspace too small";
    case RFT_E_UNSUPPORTED: return "unsupported";
    case RFT_E_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* rft_last_error(void) { return g_err.c_str(); }

size_t rft_workspace_bytes(int op, const rft_tokens* tok, int64_t d, int64_t V, int dtype) {
  if (!tok || tok->T < 0 || tok->n_seq < 0 || V < 1) return 0;
  switch (op) {
    case RFT_OP_TOKEN_LOGPROBS:
      if (dtype != RFT_F32 && dtype != RFT_BF16) return 0;
      return carve_fwd(nullptr, *tok, d, V, dtype, fwd_blocked_ok(dtype, d)).bytes;
    case RFT_OP_TOKEN_LOGPROBS_FROM_LOGITS:
    case RFT_OP_PPO_BWD_LOGITS:
      return 0;
    case RFT_OP_PPO_FWD:
    case RFT_OP_SFT_FWD:
      return carve_loss(nullptr, *tok, false).bytes;
    case RFT_OP_DPO_FWD:
      return carve_dpo(nullptr, *tok).bytes;
    case RFT_OP_PPO_FUSED_LOGITS:
      return carve_loss(nullptr, *tok, true).bytes;
    case RFT_OP_PPO_BWD: {
      if ((dtype != RFT_F32 && dtype != RFT_BF16) || d < 1) return 0;
      int64_t tc = bwd_tc_max(*tok, dtype);
      if (tc > kRecommendTc) tc = kRecommendTc;
      return carve_bwd(nullptr, *tok, d, V, dtype, tc).bytes;
    }
    case RFT_OP_PPO_STEP: {
      if ((dtype != RFT_F32 && dtype != RFT_BF16) || d < 1) return 0;
      int64_t tc = bwd_tc_max(*tok, dtype);
      if (tc > kRecommendTc) tc = kRecommendTc;
      return dtype == RFT_BF16 ? carve_step(nullptr, *tok, d, V, tc).bytes
                               : step_f32_bytes(*tok, d, V, tc);
    }
    default:
      return 0;
  }
}

size_t rft_workspace_min_bytes(int op, const rft_tokens* tok, int64_t d, int64_t V, int dtype) {
  if (op == RFT_OP_PPO_BWD || op == RFT_OP_PPO_STEP) {
    if (!tok || tok->T < 0 || tok->n_seq < 0 || V < 1 || d < 1) return 0;
    if (dtype != RFT_F32 && dtype != RFT_BF16) return 0;
    if (op == RFT_OP_PPO_STEP)
      return dtype == RFT_BF16 ? carve_step(nullptr, *tok, d, V, kBf16Align).bytes
                               : step_f32_bytes(*tok, d, V, bwd_align(dtype));
    return carve_bwd(nullptr, *tok, d, V, dtype, bwd_align(dtype)).bytes;
  }
  if (op == RFT_OP_TOKEN_LOGPROBS) {
    if (!tok || tok->T < 0 || tok->n_seq < 0 || V < 1) return 0;
    if (dtype != RFT_F32 && dtype != RFT_BF16) return 0;
    return carve_fwd(nullptr, *tok, d, V, dtype).bytes;
  }
  return rft_workspace_bytes(op, tok, d, V, dtype);
}

size_t rft_workspace_bytes_rows(int op, const rft_tokens* tok, int64_t d, int64_t V, int dtype,
                                int64_t chunk_rows) {
  if (op != RFT_OP_PPO_BWD && op != RFT_OP_PPO_STEP) return 0;
  if (!tok || tok->T < 0 || tok->n_seq < 0 || V < 1 || d < 1 || chunk_rows < 1) return 0;
  if (dtype != RFT_F32 && dtype != RFT_BF16) return 0;
  int64_t tc = round_up(chunk_rows, bwd_align(dtype));
  const int64_t tmax = bwd_tc_max(*tok, dtype);
  if (tc > tmax) tc = tmax;
  if (op == RFT_OP_PPO_STEP)
    return dtype == RFT_BF16 ? carve_step(nullptr, *tok, d, V, tc).bytes
                             : step_f32_bytes(*tok, d, V, tc);
  return carve_bwd(nullptr, *tok, d, V, dtype, tc).bytes;
}

int64_t rft_chunk_rows(int op, const rft_tokens* tok, int64_t d, int64_t V, int dtype,
                       size_t ws_bytes) {
  if (!tok || tok->T < 0 || tok->n_seq < 0 || V < 1 || d < 1) return 0;
  if (dtype != RFT_F32 && dtype != RFT_BF16) return 0;
  if (op == RFT_OP_PPO_BWD) return bwd_tc_for(*tok, d, V, dtype, ws_bytes);
  if (op == RFT_OP_PPO_STEP) {
    if (dtype == RFT_BF16) return step_tc_for(*tok, d, V, ws_bytes);
    // fp32: the separate backward runs in the front of the workspace
    const int64_t tail = round_up((tok->T > 0 ? tok->T : 1) * 4, 256);
    if ((int64_t)ws_bytes < tail + 256) return 0;
    const size_t front = (size_t)(((int64_t)ws_bytes - tail) / 256 * 256);
    if (front < step_f32_front(*tok, d, V, bwd_align(dtype))) return 0;
    return bwd_tc_for(*tok, d, V, dtype, front);
  }
  return 0;
}

rft_status rft_group_advantages(const float* rewards, int64_t n_groups, int32_t group_size,
                                float eps, int32_t unbiased, float* adv, void* stream) {
  const char* fn = "rft_group_advantages";
  if (n_groups < 0 || group_size < 1)
    return fail(RFT_E_SHAPE, "%s: n_groups=%lld group_size=%d", fn, (long long)n_groups, group_size);
  if (n_groups > 0 && (!rewards || !adv)) return fail(RFT_E_NULL, "%s: rewards / adv is NULL", fn);
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(RFT_E_PARAM, "%s: eps=%g", fn, (double)eps);
  if (n_groups > 0 && rewards == adv) return fail(RFT_E_PARAM, "%s: adv may not alias rewards", fn);
  RFT_HIP(launch_group_adv(rewards, n_groups, group_size, eps, unbiased ? 1 : 0, adv,
                           (hipStream_t)stream),
          fn);
  return RFT_OK;
}

size_t rft_group_advantages_ids_workspace_bytes(int64_t n, int64_t n_groups) {
  if (n < 0 || n_groups < 0 || n > (int64_t)std::numeric_limits<int32_t>::max() ||
      n_groups > (int64_t)std::numeric_limits<int32_t>::max())
    return 0;
  Carver c(nullptr);
  carve_adv_ids(c, n, n_groups);
  return c.bytes();
}

rft_status rft_group_advantages_ids(const float* rewards, const int32_t* group_id, int64_t n,
                                    int64_t n_groups, int32_t mode, float eps, int32_t unbiased,
                                    float* adv, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "rft_group_advantages_ids";
  if (n < 0 || n_groups < 0 || n > (int64_t)std::numeric_limits<int32_t>::max() ||
      n_groups > (int64_t)std::numeric_limits<int32_t>::max())
    return fail(RFT_E_SHAPE, "%s: n=%lld n_groups=%lld", fn, (long long)n, (long long)n_groups);
  if (n > 0 && (!rewards || !group_id || !adv))
    return fail(RFT_E_NULL, "%s: rewards / group_id / adv is NULL", fn);
  if (mode != RFT_ADV_GRPO && mode != RFT_ADV_MEAN_CENTER && mode != RFT_ADV_LEAVE_ONE_OUT)
    return fail(RFT_E_PARAM, "%s: mode=%d unknown", fn, mode);
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(RFT_E_PARAM, "%s: eps=%g", fn, (double)eps);
  if (n > 0 && rewards == adv) return fail(RFT_E_PARAM, "%s: adv may not alias rewards", fn);
  if (n == 0) return RFT_OK;
  rft_status st;
  if ((st = check_ws(fn, ws, ws_bytes, rft_group_advantages_ids_workspace_bytes(n, n_groups))))
    return st;
  Carver c(ws);
  const AdvIdsWs w = carve_adv_ids(c, n, n_groups);
  RFT_HIP(launch_group_adv_ids(rewards, group_id, n, n_groups, mode, eps, unbiased ? 1 : 0, adv, w,
                               (hipStream_t)stream),
          fn);
  return RFT_OK;
}

rft_status rft_token_logprobs(const rft_tokens* tok, const void* hidden, const void* weight,
                              int dtype, int64_t d, int64_t V, float* logp, float* entropy,
                              float* lse, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "rft_token_logprobs";
  rft_status st = check_tokens(tok, fn);
  if (st) return st;
  if ((st = check_hw(fn, tok->T, hidden, weight, dtype, d, V))) return st;
  if (tok->T > 0 && (!logp || !lse)) return fail(RFT_E_NULL, "%s: logp / lse is NULL", fn);
  FwdWs w = carve_fwd(nullptr, *tok, d, V, dtype);
  if ((st = check_ws(fn, ws, ws_bytes, w.bytes))) return st;
  // a workspace that also holds the tile-blocked copies selects that path
  const bool blocked = fwd_blocked_ok(dtype, d) &&
                       ws_bytes >= carve_fwd(nullptr, *tok, d, V, dtype, true).bytes;
  w = carve_fwd(ws, *tok, d, V, dtype, blocked);
  hipStream_t s = (hipStream_t)stream;
  if (tok->T == 0) return RFT_OK;
  RFT_HIP(launch_tokmeta(*tok, w.m, s), fn);
  if (blocked) {
    const uint16_t* W = (const uint16_t*)weight;
    RFT_HIP(launch_rows_to_blk((const uint16_t*)hidden, d, w.m.rows, w.m.meta, tok->T, d, w.hc, s),
            fn);
    RFT_HIP(launch_rows_to_blk(W, d, nullptr, nullptr, V, d, w.wb, s), fn);
    RFT_HIP(mfma_fwd_stats_blk(w.hc, d, w.wb, V, w.m.rows, tok->token_ids, w.m.meta, tok->T,
                               w.pm, w.ps, w.pu, w.ldp, w.zy, s),
            fn);
  } else if (dtype == RFT_BF16) {
    RFT_HIP(launch_gather_rows16((const uint16_t*)hidden, d, w.m.rows, w.m.meta, tok->T, w.hc, s),
            fn);
    RFT_HIP(mfma_fwd_stats(w.hc, d, (const uint16_t*)weight, V, w.m.rows,
                           tok->token_ids, w.m.meta, 0, tok->T, w.pm, w.ps, w.pu, w.ldp, w.zy, s),
            fn);
  } else {
    RFT_HIP(simt_fwd_stats((const float*)hidden, d, (const float*)weight, V, w.m.rows,
                           tok->token_ids, w.m.meta, tok->T, w.pm, w.ps, w.pu, w.ldp, w.zy, s),
            fn);
  }
  RFT_HIP(launch_merge_rows(*tok, w.m, V, w.pm, w.ps, w.pu, w.ntiles, w.ldp, w.zy, logp, entropy,
                            lse, s),
          fn);
  return RFT_OK;
}

rft_status rft_token_logprobs_from_logits(const rft_tokens* tok, const float* logits, int64_t V,
                                          float* logp, float* entropy, float* lse,
                                          float* gathered, void* ws, size_t ws_bytes,
                                          void* stream) {
  const char* fn = "rft_token_logprobs_from_logits";
  (void)ws;
  (void)ws_bytes;
  rft_status st = check_tokens(tok, fn);
  if (st) return st;
  if (V < 1 || V > (int64_t)std::numeric_limits<int32_t>::max() / 2)
    return fail(RFT_E_SHAPE, "%s: V=%lld", fn, (long long)V);
  if (tok->T > 0 && (!logits || !logp || !lse)) return fail(RFT_E_NULL, "%s: logits / logp / lse is NULL", fn);
  RFT_HIP(launch_logits_stats(logits, *tok, V, logp, entropy, lse, gathered, (hipStream_t)stream), fn);
  return RFT_OK;
}

rft_status rft_ppo_clip_loss_fwd(const rft_tokens* tok, int64_t V, const float* logp,
                                 const float* old_logp, const float* ref_logp, const float* adv,
                                 const float* entropy, const rft_ppo_params* params,
                                 float* grad_logp, float* grad_entropy, rft_ppo_stats* stats,
                                 void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "rft_ppo_clip_loss_fwd";
  rft_status st = check_tokens(tok, fn);
  if (st) return st;
  if ((st = check_params(params, fn))) return st;
  if (V < 1) return fail(RFT_E_SHAPE, "%s: V=%lld", fn, (long long)V);
  if (!stats) return fail(RFT_E_NULL, "%s: stats is NULL", fn);
  if (tok->T > 0 && (!logp || !old_logp || !adv || !grad_logp))
    return fail(RFT_E_NULL, "%s: logp / old_logp / adv / grad_logp is NULL", fn);
  if (tok->T > 0 && params->kl_coef > 0.f && !ref_logp)
    return fail(RFT_E_NULL, "%s: ref_logp is NULL with kl_coef > 0", fn);
  if (tok->T > 0 && params->entropy_coef > 0.f && !entropy)
    return fail(RFT_E_NULL, "%s: entropy is NULL with entropy_coef > 0", fn);
  LossWs w = carve_loss(nullptr, *tok, false);
  if ((st = check_ws(fn, ws, ws_bytes, w.bytes))) return st;
  w = carve_loss(ws, *tok, false);
  hipStream_t s = (hipStream_t)stream;
  RFT_HIP(launch_tokmeta(*tok, w.m, s), fn);
  LossConst c = loss_const(params, V, *tok);
  RFT_HIP(launch_loss_fwd(*tok, w.m, logp, old_logp, ref_logp,
                          adv, entropy, c, grad_logp, grad_entropy, w.parts, stats, s),
          fn);
  return RFT_OK;
}

rft_status rft_ppo_clip_loss_bwd(const rft_tokens* tok, const void* hidden, const void* weight,
                                 int dtype, int64_t d, int64_t V, const float* lse,
                                 const float* grad_logp, const float* grad_entropy,
                                 const float* entropy, float* d_hidden, float* d_weight,
                                 int32_t accumulate_dw, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "rft_ppo_clip_loss_bwd";
  rft_status st = check_tokens(tok, fn);
  if (st) return st;
  if ((st = check_hw(fn, tok->T, hidden, weight, dtype, d, V))) return st;
  if (!d_weight) return fail(RFT_E_NULL, "%s: d_weight is NULL", fn);
  if (tok->T > 0 && (!lse || !grad_logp || !d_hidden))
    return fail(RFT_E_NULL, "%s: lse / grad_logp / d_hidden is NULL", fn);
  if (tok->T > 0 && (!grad_entropy != !entropy))
    return fail(RFT_E_NULL, "%s: grad_entropy and entropy must be both given or both NULL", fn);
  size_t need = carve_bwd(nullptr, *tok, d, V, dtype, bwd_align(dtype)).bytes;
  if ((st = check_ws(fn, ws, ws_bytes, need))) return st;
  int64_t Tc = bwd_tc_for(*tok, d, V, dtype, ws_bytes);
  if (Tc <= 0) return fail(RFT_E_WORKSPACE, "%s: workspace too small", fn);
  BwdWs w = carve_bwd(ws, *tok, d, V, dtype, Tc);
  hipStream_t s = (hipStream_t)stream;
  const int64_t T = tok->T;
  RFT_HIP(launch_tokmeta(*tok, w.m, s), fn);
  if (T > 0) {
    RFT_HIP(launch_zero_masked_rows(tok->mask, T, d, d_hidden, s), fn);
  }
  int64_t nchunks = T > 0 ? (T + Tc - 1) / Tc : 0;
  const int32_t* cnt = w.m.meta;
  if (dtype == RFT_BF16) {
    const uint16_t* H = (const uint16_t*)hidden;
    const uint16_t* W = (const uint16_t*)weight;
    if (nchunks > 0) {
      RFT_HIP(launch_gather_rows16(H, d, w.m.rows, cnt, T, w.hc, s), fn);
      RFT_HIP(launch_transpose_blk(W, d, nullptr, 0, V, w.Vpad, w.dpad, w.wt, s), fn);
    }
    for (int64_t ci = 0; ci < nchunks; ++ci) {
      int64_t c0 = ci * Tc;
      RFT_HIP(mfma_dz(w.hc, d, W, V, w.Vpad, w.m.rows, tok->token_ids, lse, grad_logp,
                      grad_entropy, entropy, cnt, c0, Tc, w.dz, w.dzt, Tc, s),
              fn);
      RFT_HIP(launch_transpose_blk(w.hc, d, cnt, c0, Tc, Tc, w.dpad, w.hct, s), fn);
      // dH rows of this chunk: dZ [count, Vpad] . Wt[d, Vpad]^T, scattered to token rows
      RFT_HIP(mfma_gemm_store(w.dz, w.Vpad, w.wt, w.Vpad, Tc, d, w.Vpad, cnt, c0, Tc, 1, 0,
                              d_hidden, d, w.m.rows, c0, 0, s, 1, 1),
              fn);
      // dW += dZ^T . Hc over the chunk's rows, both operands K-contiguous (K = rows)
      RFT_HIP(mfma_gemm_store(w.dzt, Tc, w.hct, Tc, V, d, Tc, cnt, c0, Tc, 0, 1, d_weight, d,
                              nullptr, 0, (ci > 0 || accumulate_dw) ? 1 : 0, s, 1, 1),
              fn);
    }
    if (nchunks == 0 && !accumulate_dw) RFT_HIP(launch_fill_zero(d_weight, V * d, s), fn);
  } else {
    const float* H = (const float*)hidden;
    const float* W = (const float*)weight;
    for (int64_t ci = 0; ci < nchunks; ++ci) {
      int64_t c0 = ci * Tc;
      RFT_HIP(simt_dz(H, d, W, V, w.Vpad, w.m.rows, tok->token_ids, lse, grad_logp,
                      grad_entropy, entropy, cnt, c0, Tc, w.dz32, s),
              fn);
      // dH[m, j] = sum_v dZ[m, v] W[v, j]
      RFT_HIP(simt_gemm_store(w.dz32, w.Vpad, 1, W, 1, d, nullptr, 0, Tc, d, V, cnt, c0, Tc, 1, 0,
                              d_hidden, d, w.m.rows, c0, 0, s),
              fn);
      // dW[v, j] = sum_t dZ[t, v] H[rows[c0 + t], j]
      RFT_HIP(simt_gemm_store(w.dz32, 1, w.Vpad, H, 1, d, w.m.rows, c0, V, d, Tc, cnt, c0, Tc, 0, 1,
                              d_weight, d, nullptr, 0, (ci > 0 || accumulate_dw) ? 1 : 0, s),
              fn);
    }
    if (nchunks == 0 && !accumulate_dw) RFT_HIP(launch_fill_zero(d_weight, V * d, s), fn);
  }
  return RFT_OK;
}

rft_status rft_ppo_clip_loss_bwd_logits(const rft_tokens* tok, const float* logits, int64_t V,
                                        const float* lse, const float* grad_logp,
                                        const float* grad_entropy, const float* entropy,
                                        float* d_logits, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "rft_ppo_clip_loss_bwd_logits";
  (void)ws;
  (void)ws_bytes;
  rft_status st = check_tokens(tok, fn);
  if (st) return st;
  if (V < 1 || V > (int64_t)std::numeric_limits<int32_t>::max() / 2)
    return fail(RFT_E_SHAPE, "%s: V=%lld", fn, (long long)V);
  if (tok->T > 0 && (!logits || !lse || !grad_logp || !d_logits))
    return fail(RFT_E_NULL, "%s: logits / lse / grad_logp / d_logits is NULL", fn);
  if (tok->T > 0 && (!grad_entropy != !entropy))
    return fail(RFT_E_NULL, "%s: grad_entropy and entropy must be both given or both NULL", fn);
  RFT_HIP(launch_logits_bwd(logits, *tok, V, lse, grad_logp, grad_entropy, entropy, d_logits,
                            (hipStream_t)stream),
          fn);
  return RFT_OK;
}

rft_status rft_ppo_clip_fused_logits(const rft_tokens* tok, const float* logits, int64_t V,
                                     const float* old_logp, const float* ref_logp,
                                     const float* adv, const rft_ppo_params* params, float* logp,
                                     float* entropy, float* lse, float* grad_logp,
                                     float* d_logits, rft_ppo_stats* stats, void* ws,
                                     size_t ws_bytes, void* stream) {
  const char* fn = "rft_ppo_clip_fused_logits";
  rft_status st = check_fused_logits(fn, tok, logits, V, old_logp, ref_logp, adv, params, logp,
                                     d_logits, stats);
  if (st) return st;
  LossWs w = carve_loss(nullptr, *tok, true);
  if ((st = check_ws(fn, ws, ws_bytes, w.bytes))) return st;
  w = carve_loss(ws, *tok, true);
  hipStream_t s = (hipStream_t)stream;
  RFT_HIP(launch_tokmeta(*tok, w.m, s), fn);
  LossConst c = loss_const(params, V, *tok);
  RFT_HIP(launch_logits_fused(logits, *tok, w.m, V, old_logp,
                              ref_logp, adv, c, logp, entropy,
                              lse, grad_logp, d_logits, w.parts, w.parts2, stats, s),
          fn);
  return RFT_OK;
}

size_t rft_noalloc_scratch_bytes(void) { return kNoAllocScratchBytes; }

rft_status rft_ppo_clip_fused_logits_noalloc(const rft_tokens* tok, const float* logits, int64_t V,
                                             const float* old_logp, const float* ref_logp,
                                             const float* adv, const rft_ppo_params* params,
                                             float* logp, float* entropy, float* lse,
                                             float* grad_logp, float* d_logits,
                                             rft_ppo_stats* stats, void* stream) {
  const char* fn = "rft_ppo_clip_fused_logits_noalloc";
  rft_status st = check_fused_logits(fn, tok, logits, V, old_logp, ref_logp, adv, params, logp,
                                     d_logits, stats);
  if (st) return st;
  const size_t need = carve_loss(nullptr, *tok, true).bytes;
  if (need > kNoAllocScratchBytes)
    return fail(RFT_E_WORKSPACE,
                "%s: T=%lld rows and n_seq=%lld rollouts need %zu bytes of scratch, more than "
                "the %zu the library holds; use rft_ppo_clip_fused_logits with a workspace",
                fn, (long long)tok->T, (long long)tok->n_seq, need, kNoAllocScratchBytes);
  hipError_t e = hipSuccess;
  void* ws = scratch_ptr(&e);
  if (!ws) return hip_fail(e, fn);
  // every byte of the scratch that the call reads it writes first (the
  // bookkeeping kernels fill their arrays, every row writes its partial), so
  // the previous call's contents need no clearing
  return rft_ppo_clip_fused_logits(tok, logits, V, old_logp, ref_logp, adv, params, logp, entropy,
                                   lse, grad_logp, d_logits, stats, ws, kNoAllocScratchBytes,
                                   stream);
}

rft_status rft_ppo_clip_step(const rft_tokens* tok, const void* hidden, const void* weight,
                             int dtype, int64_t d, int64_t V, const float* old_logp,
                             const float* ref_logp, const float* adv,
                             const rft_ppo_params* params, float* logp, float* entropy,
                             float* lse, float* grad_logp, float* d_hidden, float* d_weight,
                             int32_t accumulate_dw, rft_ppo_stats* stats, void* ws,
                             size_t ws_bytes, void* stream) {
  const char* fn = "rft_ppo_clip_step";
  rft_status st = check_tokens(tok, fn);
  if (st) return st;
  if ((st = check_hw(fn, tok->T, hidden, weight, dtype, d, V))) return st;
  if ((st = check_params(params, fn))) return st;
  if (!stats || !d_weight) return fail(RFT_E_NULL, "%s: stats / d_weight is NULL", fn);
  if (tok->T > 0 && (!old_logp || !adv || !logp || !lse || !grad_logp || !d_hidden))
    return fail(RFT_E_NULL, "%s: old_logp / adv / logp / lse / grad_logp / d_hidden is NULL", fn);
  if (tok->T > 0 && params->kl_coef > 0.f && !ref_logp)
    return fail(RFT_E_NULL, "%s: ref_logp is NULL with kl_coef > 0", fn);
  if (tok->T > 0 && params->entropy_coef > 0.f && !entropy)
    return fail(RFT_E_NULL, "%s: entropy is NULL with entropy_coef > 0", fn);
  const float* ref = ref_logp;
  const bool bonus = params->entropy_coef > 0.f;
  if (dtype == RFT_F32) {
    if ((st = check_ws(fn, ws, ws_bytes, step_f32_bytes(*tok, d, V, bwd_align(dtype))))) return st;
    // the three calls share the front; the largest chunk that fits leaves room for egrad
    int64_t front = (int64_t)ws_bytes - round_up((tok->T > 0 ? tok->T : 1) * 4, 256);
    front = front / 256 * 256;
    float* egrad = bonus ? (float*)((char*)ws + front) : nullptr;
    if ((st = rft_token_logprobs(tok, hidden, weight, dtype, d, V, logp, entropy, lse, ws,
                                 (size_t)front, stream)))
      return st;
    if ((st = rft_ppo_clip_loss_fwd(tok, V, logp, old_logp, ref, adv, entropy, params, grad_logp,
                                    egrad, stats, ws, (size_t)front, stream)))
      return st;
    return rft_ppo_clip_loss_bwd(tok, hidden, weight, dtype, d, V, lse, grad_logp, egrad,
                                 bonus ? entropy : nullptr, d_hidden, d_weight, accumulate_dw, ws,
                                 (size_t)front, stream);
  }
  if ((st = check_ws(fn, ws, ws_bytes, carve_step(nullptr, *tok, d, V, kBf16Align).bytes)))
    return st;
  const int64_t Tc = step_tc_for(*tok, d, V, ws_bytes);
  if (Tc <= 0) return fail(RFT_E_WORKSPACE, "%s: workspace too small", fn);
  StepWs w = carve_step(ws, *tok, d, V, Tc);
  hipStream_t s = (hipStream_t)stream;
  const int64_t T = tok->T;
  const LossConst c = loss_const(params, V, *tok);
  const uint16_t* H = (const uint16_t*)hidden;
  const uint16_t* W = (const uint16_t*)weight;
  const int64_t nchunks = T > 0 ? (T + Tc - 1) / Tc : 0;
  const int32_t* cnt = w.m.meta;
  RFT_HIP(launch_tokmeta(*tok, w.m, s), fn);
  if (T > 0) {
    RFT_HIP(launch_zero_masked_rows(tok->mask, T, d, d_hidden, s), fn);
    // masked rows of the per-token outputs are 0; the chunks fill the valid rows
    RFT_HIP(launch_fill_zero(logp, T, s), fn);
    RFT_HIP(launch_fill_zero(lse, T, s), fn);
    if (entropy) RFT_HIP(launch_fill_zero(entropy, T, s), fn);
    RFT_HIP(launch_rows_to_blk(H, d, w.m.rows, cnt, T, w.Kp, w.hc, s), fn);
    RFT_HIP(launch_rows_to_blk(W, d, nullptr, nullptr, V, w.Kp, w.wb, s), fn);
    RFT_HIP(launch_transpose_blk(W, d, nullptr, 0, V, w.Vpad, w.dpad, w.wt, s), fn);
  }
  for (int64_t ci = 0; ci < nchunks; ++ci) {
    const int64_t c0 = ci * Tc;
    RFT_HIP(mfma_fwd_stats_y(w.hc, d, w.wb, V, w.Vpad, w.m.rows, tok->token_ids, cnt, c0, Tc, w.pm,
                             w.ps, w.pu, w.zy, w.dz, s),
            fn);
    RFT_HIP(launch_step_rows(w.m, tok->token_ids, V, c0, Tc, w.pm, w.ps, w.pu, w.ntiles, w.zy,
                             old_logp, ref, adv, c, logp, entropy, lse, grad_logp,
                             bonus ? w.ce : nullptr, w.cmu, s),
            fn);
    RFT_HIP(launch_dz_from_y_blk(w.dz, w.Vpad, Tc, V, w.m.rows, tok->token_ids, cnt, c0, w.pm,
                                 lse, grad_logp, bonus ? w.ce : nullptr, w.cmu, w.dzt, s),
            fn);
    RFT_HIP(launch_transpose_blk(w.hc, d, cnt, c0, Tc, Tc, w.dpad, w.hct, s, w.Kp), fn);
    RFT_HIP(mfma_gemm_store(w.dz, w.Vpad, w.wt, w.Vpad, Tc, d, w.Vpad, cnt, c0, Tc, 1, 0,
                            d_hidden, d, w.m.rows, c0, 0, s, 1, 1),
            fn);
    // dW = dZ^T . Hc with both operands K-contiguous (K = the chunk's rows)
    RFT_HIP(mfma_gemm_store(w.dzt, Tc, w.hct, Tc, V, d, Tc, cnt, c0, Tc, 0, 1, d_weight, d,
                            nullptr, 0, (ci > 0 || accumulate_dw) ? 1 : 0, s, 1, 1),
            fn);
  }
  if (nchunks == 0 && !accumulate_dw) RFT_HIP(launch_fill_zero(d_weight, V * d, s), fn);
  // loss and metrics over every row (rewrites grad_logp with the same values
  // and 0 on masked rows)
  RFT_HIP(launch_loss_fwd(*tok, w.m, logp, old_logp, ref, adv, entropy, c, grad_logp, nullptr,
                          w.parts, stats, s),
          fn);
  return RFT_OK;
}

rft_status rft_sft_loss_fwd(const rft_tokens* tok, int64_t V, const float* logp, int32_t agg,
                            double denom_override, float* grad_logp, rft_ppo_stats* stats,
                            void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "rft_sft_loss_fwd";
  rft_status st = check_tokens(tok, fn);
  if (st) return st;
  if (V < 1) return fail(RFT_E_SHAPE, "%s: V=%lld", fn, (long long)V);
  if (agg != RFT_AGG_SEQ_MEAN_TOKEN_MEAN && agg != RFT_AGG_TOKEN_MEAN)
    return fail(RFT_E_PARAM, "%s: agg=%d unknown", fn, agg);
  if (!(denom_override >= 0.0) || !std::isfinite(denom_override))
    return fail(RFT_E_PARAM, "%s: denom_override=%g must be finite and >= 0", fn, denom_override);
  if (!stats) return fail(RFT_E_NULL, "%s: stats is NULL", fn);
  if (tok->T > 0 && (!logp || !grad_logp))
    return fail(RFT_E_NULL, "%s: logp / grad_logp is NULL", fn);
  LossWs w = carve_loss(nullptr, *tok, false);
  if ((st = check_ws(fn, ws, ws_bytes, w.bytes))) return st;
  w = carve_loss(ws, *tok, false);
  hipStream_t s = (hipStream_t)stream;
  rft_tokens t2 = *tok;
  t2.is_expert = nullptr;
  RFT_HIP(launch_tokmeta(t2, w.m, s), fn);
  RFT_HIP(launch_sft_fwd(t2, w.m, V, logp, agg, denom_override, grad_logp, w.parts, stats, s), fn);
  return RFT_OK;
}

rft_status rft_dpo_loss_fwd(const rft_tokens* tok, int64_t V, const float* logp,
                            const float* ref_logp, float beta, float label_smoothing,
                            float* grad_logp, float* seq_logp, rft_dpo_stats* stats, void* ws,
                            size_t ws_bytes, void* stream) {
  const char* fn = "rft_dpo_loss_fwd";
  rft_status st = check_tokens(tok, fn);
  if (st) return st;
  if (V < 1) return fail(RFT_E_SHAPE, "%s: V=%lld", fn, (long long)V);
  if (tok->n_seq % 2)
    return fail(RFT_E_SHAPE, "%s: n_seq=%lld must be even (chosen, rejected pairs)", fn,
                (long long)tok->n_seq);
  if (!(beta > 0.f) || !std::isfinite(beta))
    return fail(RFT_E_PARAM, "%s: beta=%g must be finite and > 0", fn, (double)beta);
  if (!(label_smoothing >= 0.f && label_smoothing <= 0.5f))
    return fail(RFT_E_PARAM, "%s: label_smoothing=%g must be in [0, 0.5]", fn,
                (double)label_smoothing);
  if (!stats) return fail(RFT_E_NULL, "%s: stats is NULL", fn);
  if (tok->T > 0 && (!logp || !ref_logp || !grad_logp))
    return fail(RFT_E_NULL, "%s: logp / ref_logp / grad_logp is NULL", fn);
  DpoCarve w = carve_dpo(nullptr, *tok);
  if ((st = check_ws(fn, ws, ws_bytes, w.bytes))) return st;
  w = carve_dpo(ws, *tok);
  hipStream_t s = (hipStream_t)stream;
  rft_tokens t2 = *tok;
  t2.is_expert = nullptr;
  RFT_HIP(launch_tokmeta(t2, w.m, s), fn);
  RFT_HIP(launch_dpo(t2, w.m, V, logp, ref_logp, beta, label_smoothing, w.d, grad_logp, seq_logp,
                     stats, s),
          fn);
  return RFT_OK;
}

}  // extern "C"

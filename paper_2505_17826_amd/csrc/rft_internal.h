// Internal declarations shared by the HIP sources of librft (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <float.h>
#include <math.h>

#include "rft.h"

namespace rft {

// ------------------------------------------------------------------ types --
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}
// Round-to-nearest-even float -> bf16 bits (NaN stays a quiet NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// ------------------------------------------------------- wave reductions --
// DPP move within a row of 16 lanes.  The patterns used here are
// permutations within the row (every lane has a source), so bound_ctrl
// changes no value; setting it lets the compiler fold the move into the add
// or max that uses it.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}

// Reductions over the 16 lanes of each DPP row (four butterfly steps), over N
// independent values at a time; every lane of the row ends with the result.
template <int N>
__device__ __forceinline__ void row16_max_n(float (&v)[N]) {
#pragma unroll
  for (int e = 0; e < N; ++e) v[e] = fmaxf(v[e], dpp_f<0xB1>(v[e]));
#pragma unroll
  for (int e = 0; e < N; ++e) v[e] = fmaxf(v[e], dpp_f<0x4E>(v[e]));
#pragma unroll
  for (int e = 0; e < N; ++e) v[e] = fmaxf(v[e], dpp_f<0x141>(v[e]));
#pragma unroll
  for (int e = 0; e < N; ++e) v[e] = fmaxf(v[e], dpp_f<0x140>(v[e]));
}
template <int N>
__device__ __forceinline__ void row16_sum_n(float (&v)[N]) {
#pragma unroll
  for (int e = 0; e < N; ++e) v[e] += dpp_f<0xB1>(v[e]);
#pragma unroll
  for (int e = 0; e < N; ++e) v[e] += dpp_f<0x4E>(v[e]);
#pragma unroll
  for (int e = 0; e < N; ++e) v[e] += dpp_f<0x141>(v[e]);
#pragma unroll
  for (int e = 0; e < N; ++e) v[e] += dpp_f<0x140>(v[e]);
}

// Whole-wave (64 lanes) reductions via cross-lane shuffles.
__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_sum_f(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max_f(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_min_f(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ long long wave_sum_ll(long long v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Merge of two online log-sum-exp partials (m: max, s: sum exp(z - m),
// u: sum exp(z - m) z).  A partial with s == 0 is empty.
__device__ __forceinline__ void lse_merge(float& m, float& s, float& u, float m2, float s2,
                                          float u2) {
  if (s2 == 0.f) return;
  if (s == 0.f) { m = m2; s = s2; u = u2; return; }
  float M = fmaxf(m, m2);
  float a = exp2f((m - M) * kLog2e), b = exp2f((m2 - M) * kLog2e);
  s = s * a + s2 * b;
  u = u * a + u2 * b;
  m = M;
}

// ----------------------------------------------------- token bookkeeping --
// Compacted view of the masked rows, built on the device by the first kernels
// of every call (the workspace holds it).
struct TokMeta {
  int32_t* rows;     // [T]  k-th valid row (k < N)
  int32_t* row_seq;  // [T]  rollout of the k-th valid row
  int32_t* kidx;     // [T]  compacted index of row t, -1 if masked
  int32_t* n_i;      // [n_seq] valid tokens per rollout
  int32_t* blk;      // [nblk] per-block counts, then offsets
  int32_t* meta;     // [4]  N, S, expert tokens, expert rollouts with tokens
};

struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base((char*)b) {}
  template <class T>
  T* take(size_t count) {
    off = (off + 255) & ~size_t(255);
    T* p = base ? (T*)(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
  size_t bytes() const { return (off + 255) & ~size_t(255); }
};

constexpr int kK0Rows = 2048;  // rows per block of the compaction kernels

TokMeta carve_tokmeta(Carver& c, int64_t T, int64_t n_seq);
hipError_t launch_tokmeta(const rft_tokens& tok, const TokMeta& m, hipStream_t s);

// ------------------------------------------------------------------ loss --
struct LossConst {
  float thr_lo, thr_hi;   // fp32 log(1 - eps_low), log(1 + eps_high)
  float eps_low, eps_high, beta;
  int agg;
  double denom;           // 0 = use S or N
  int64_t V;
  int mix;                // 1: expert flags given (MIX loss)
  float mu;               // SFT weight of the MIX loss
  const uint8_t* is_expert;  // [n_seq] device flags, or nullptr
  float ent_coef;         // entropy bonus coefficient
};

// Per-token PPO-clip + k3 KL terms.  Returns false for an out-of-range id.
struct TokLoss {
  double w;     // aggregation weight
  float pg, kl, rho, g;
  bool clipped;
};

// Aggregation weight w_t of a valid token of a rollout with n_seq_i valid
// tokens, among N valid tokens in S rollouts (or the override denominator).
__device__ __forceinline__ double agg_weight(int agg, double denom, int n_seq_i, int N, int S) {
  double den;
  if (agg == RFT_AGG_SEQ_MEAN_TOKEN_MEAN) {
    double Sd = denom > 0 ? denom : (double)S;
    den = Sd * (double)n_seq_i;
  } else {
    den = denom > 0 ? denom : (double)N;
  }
  return den > 0 ? 1.0 / den : 0.0;
}

__device__ __forceinline__ TokLoss token_loss(float lp, float old, float ref, float A, int n_seq_i,
                                              int N, int S, const LossConst& c) {
  TokLoss r;
  r.w = agg_weight(c.agg, c.denom, n_seq_i, N, S);
  float delta = lp - old;
  r.rho = expf(delta);
  float lo = 1.f - c.eps_low, hi = 1.f + c.eps_high;
  float rb = fminf(fmaxf(r.rho, lo), hi);
  r.pg = fmaxf(-A * r.rho, -A * rb);
  r.clipped = (A > 0.f && delta > c.thr_hi) || (A < 0.f && delta < c.thr_lo);
  float dk = ref - lp;
  float em1 = expm1f(dk);
  r.kl = em1 - dk;
  // with beta = 0 the KL term is off: kl stays a metric and adds nothing
  // (not even a NaN from 0 * inf) to the loss or the gradient
  r.g = (r.clipped ? 0.f : -A * r.rho) - (c.beta > 0.f ? c.beta * em1 : 0.f);
  return r;
}

// Partial sums of one block of tokens, reduced in a fixed order.
struct LossPartial {
  double loss, pg, klw, kl, ent, ratio, sft, entw;
  long long clipped, bad, expert;
};

// Loss terms of one valid row whose id is in range: adds its terms to p and
// returns c_t = d loss / d logp; *e gets the coefficient of the entropy
// bonus (-d loss / d H_t).  meta = {N, S, expert tokens, expert rollouts with
// tokens}; the on-policy (GRPO) part uses the counts without the expert
// rollouts, scaled by 1 - mu under MIX, and carries the entropy bonus
// -ent_coef * w_t * H_t; an expert row contributes mu * (-logp) / (expert
// tokens) (the SFT term of the MIX loss).
__device__ __forceinline__ float row_loss(float lp, float old, float ref, float A, int n_seq_i,
                                          bool expert, const int32_t* meta, double ent,
                                          const LossConst& c, LossPartial& p, float* e) {
  p.ent = ent;
  *e = 0.f;
  if (c.mix && expert) {
    const int Ne = meta[2];
    const double inv = Ne > 0 ? 1.0 / (double)Ne : 0.0;
    p.sft = -(double)lp;
    p.loss = (double)c.mu * p.sft * inv;
    p.expert = 1;
    return (float)(-(double)c.mu * inv);
  }
  const int Ng = meta[0] - meta[2], Sg = meta[1] - meta[3];
  TokLoss L = token_loss(lp, old, ref, A, n_seq_i, Ng, Sg, c);
  const double scale = c.mix ? 1.0 - (double)c.mu : 1.0;
  const double bkl = c.beta > 0.f ? (double)c.beta * (double)L.kl : 0.0;
  p.loss = scale * (L.w * ((double)L.pg + bkl));
  p.pg = L.w * (double)L.pg;
  p.klw = L.w * bkl;
  p.kl = (double)L.kl;
  p.ratio = (double)L.rho;
  p.clipped = L.clipped ? 1 : 0;
  p.entw = L.w * ent;
  if (c.ent_coef > 0.f) {
    p.loss -= scale * (double)c.ent_coef * p.entw;
    *e = (float)(scale * (double)c.ent_coef * L.w);
  }
  return (float)(scale * L.w * (double)L.g);
}

// d loss / d z_j of one row: c (onehot - p_j) + e p_j (z_j - mu), with p_j the
// softmax probability, c = d loss / d logp, e the entropy-bonus coefficient
// and mu = lse - H the softmax mean of z (d H / d z_j = -p_j (z_j - mu)).
// The entropy term is taken as 0 where p = 0 (its value for any finite z, and
// its limit for a masked vocabulary entry z = -inf, where 0 * (z - mu) would
// be NaN).
__device__ __forceinline__ float dlogit(float c, float e, float mu, float p, float z, bool hot) {
  const float t = e * p * (z - mu);
  return c * ((hot ? 1.f : 0.f) - p) + (p > 0.f ? t : 0.f);
}

#define RFT_ZERO_PARTIAL LossPartial{0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0}

hipError_t launch_loss_final(const LossPartial* parts, int nparts, const int32_t* meta,
                             rft_ppo_stats* stats, hipStream_t s, int sft_only = 0);
// out[b] = the fixed-order sum of parts[256 b .. 256 b + 255] (n parts)
hipError_t launch_loss_reduce256(const LossPartial* parts, int64_t n, LossPartial* out,
                                 hipStream_t s);
hipError_t launch_sft_fwd(const rft_tokens& tok, const TokMeta& m, int64_t V, const float* logp,
                          int agg, double denom, float* grad, LossPartial* parts,
                          rft_ppo_stats* st, hipStream_t s);
struct DpoWs {
  double *pi, *rho;  // [n_seq] sums of policy / reference log-probs
  int32_t* bad;      // [n_seq] bad ids
  float* coef;       // [n_seq] d loss / d pi_s
};
hipError_t launch_dpo(const rft_tokens& tok, const TokMeta& m, int64_t V, const float* logp,
                      const float* ref, float beta, float ls, const DpoWs& w, float* grad,
                      float* seq_logp, rft_dpo_stats* st, hipStream_t s);

// ------------------------------------------------------------ launchers --
hipError_t launch_group_adv(const float* r, int64_t n_groups, int G, float eps, int unbiased,
                            float* adv, hipStream_t s);
struct AdvIdsWs {
  int32_t *cnt, *cur;  // [n_groups] members per group, scatter cursors
  int32_t* off;        // [n_groups + 1] start of each group's members in mem
  int32_t* tot;        // [ceil(n_groups / 1024)] block totals of the scan
  int32_t* mem;        // [n] rollout indices grouped by group id
};
AdvIdsWs carve_adv_ids(Carver& c, int64_t n, int64_t n_groups);
hipError_t launch_group_adv_ids(const float* r, const int32_t* gid, int64_t n, int64_t n_groups,
                                int mode, float eps, int unbiased, float* adv, const AdvIdsWs& w,
                                hipStream_t s);
hipError_t launch_loss_fwd(const rft_tokens& tok, const TokMeta& m, const float* logp,
                           const float* old, const float* ref, const float* adv, const float* ent,
                           const LossConst& c, float* grad, float* egrad, LossPartial* parts,
                           rft_ppo_stats* st, hipStream_t s);
hipError_t launch_merge_rows(const rft_tokens& tok, const TokMeta& m, int64_t V, const float* pm,
                             const float* ps, const float* pu, int ntiles, int64_t ld,
                             const float* zy, float* logp, float* ent, float* lse, hipStream_t s);
hipError_t mfma_fwd_stats(const uint16_t* H, int64_t d, const uint16_t* W, int64_t V,
                          const int32_t* rows, const int32_t* ids, const int32_t* cnt,
                          int64_t rows_off, int64_t cap, float* pm, float* ps, float* pu,
                          int64_t ldp, float* zy, hipStream_t s);
hipError_t mfma_fwd_stats_blk(const uint16_t* Hb, int64_t d, const uint16_t* Wb, int64_t V,
                              const int32_t* rows, const int32_t* ids, const int32_t* cnt,
                              int64_t cap, float* pm, float* ps, float* pu, int64_t ldp, float* zy,
                              hipStream_t s);
bool mfma_fwd_blk_ok(int64_t d);
hipError_t mfma_fwd_stats_y(const uint16_t* Hc, int64_t d, const uint16_t* W, int64_t V,
                            int64_t Vpad, const int32_t* rows, const int32_t* ids,
                            const int32_t* cnt, int64_t c0, int64_t Tc, float* pm, float* ps,
                            float* pu, float* zy, uint16_t* y, hipStream_t s);
hipError_t launch_step_rows(const TokMeta& m, const int32_t* ids, int64_t V, int64_t c0,
                            int64_t Tc, const float* pm, const float* ps, const float* pu,
                            int ntiles, const float* zy, const float* old, const float* ref,
                            const float* adv, const LossConst& c, float* logp, float* ent,
                            float* lse, float* grad, float* ce, float* cmu, hipStream_t s);
hipError_t launch_dz_from_y_blk(uint16_t* yz, int64_t Vpad, int64_t Tc, int64_t V,
                                const int32_t* rows, const int32_t* ids, const int32_t* meta,
                                int64_t c0, const float* pm, const float* lse, const float* grad,
                                const float* ce, const float* cmu, uint16_t* dzt, hipStream_t s);
hipError_t launch_transpose_blk(const uint16_t* src, int64_t ncols, const int32_t* meta,
                                int64_t r0, int64_t nrows, int64_t Kp, int64_t ncols_pad,
                                uint16_t* dst, hipStream_t s, int64_t src_kp = 0);
hipError_t launch_rows_to_blk(const uint16_t* src, int64_t d, const int32_t* rows,
                              const int32_t* meta, int64_t cap, int64_t Kp, uint16_t* dst,
                              hipStream_t s);
hipError_t mfma_dz(const uint16_t* H, int64_t d, const uint16_t* W, int64_t V, int64_t Vpad,
                   const int32_t* rows, const int32_t* ids, const float* lse, const float* cgrad,
                   const float* egrad, const float* ent, const int32_t* cnt, int64_t c0,
                   int64_t Tc, uint16_t* dz, uint16_t* dzt, int64_t ldzt, hipStream_t s);
hipError_t mfma_gemm_store(const uint16_t* A, int64_t lda, const uint16_t* B, int64_t ldb,
                           int64_t M, int64_t N, int64_t K, const int32_t* cnt, int64_t cnt_off,
                           int64_t cnt_cap, int m_from_cnt, int k_from_cnt, float* C, int64_t ldc,
                           const int32_t* rows, int64_t rows_off, int accumulate, hipStream_t s,
                           int a_blk = 0, int b_blk = 0);
hipError_t simt_fwd_stats(const float* H, int64_t d, const float* W, int64_t V, const int32_t* rows,
                          const int32_t* ids, const int32_t* cnt, int64_t cap, float* pm, float* ps,
                          float* pu, int64_t ldp, float* zy, hipStream_t s);
hipError_t simt_dz(const float* H, int64_t d, const float* W, int64_t V, int64_t Vpad,
                   const int32_t* rows, const int32_t* ids, const float* lse, const float* cgrad,
                   const float* egrad, const float* ent, const int32_t* cnt, int64_t c0,
                   int64_t Tc, float* dz, hipStream_t s);
hipError_t simt_gemm_store(const float* A, int64_t sam, int64_t sak, const float* B, int64_t sbn,
                           int64_t sbk, const int32_t* b_map, int64_t b_koff, int64_t M, int64_t N,
                           int64_t K, const int32_t* cnt, int64_t cnt_off, int64_t cnt_cap,
                           int m_from_cnt, int k_from_cnt, float* C, int64_t ldc,
                           const int32_t* rows, int64_t rows_off, int accumulate, hipStream_t s);
hipError_t launch_gather_rows16(const uint16_t* H, int64_t d, const int32_t* rows,
                                const int32_t* cnt, int64_t cap, uint16_t* Hc, hipStream_t s);
hipError_t launch_fill_zero(float* out, int64_t n, hipStream_t s);
hipError_t launch_zero_masked_rows(const uint8_t* mask, int64_t T, int64_t width, float* out,
                                   hipStream_t s);
hipError_t launch_logits_stats(const float* logits, const rft_tokens& tok, int64_t V, float* logp,
                               float* ent, float* lse, float* gathered, hipStream_t s);
hipError_t launch_logits_bwd(const float* logits, const rft_tokens& tok, int64_t V,
                             const float* lse, const float* grad, const float* egrad,
                             const float* ent, float* dl, hipStream_t s);
hipError_t launch_logits_fused(const float* logits, const rft_tokens& tok, const TokMeta& m,
                               int64_t V, const float* old, const float* ref, const float* adv,
                               const LossConst& c, float* logp, float* ent, float* lse,
                               float* grad, float* dl, LossPartial* parts, LossPartial* parts2,
                               rft_ppo_stats* st, hipStream_t s);

constexpr int kMfmaTileN = 256;  // vocabulary columns per forward tile (bf16 path)

// Tile-blocked layout of a bf16 GEMM operand X [R, K] (K-contiguous; R padded
// to a multiple of 256, K to a multiple of 64 = Kp): 256-row panels, each
// Kp / 64 consecutive blocks of 256 rows x 64 values, row-major in a block.
// A k-step of a 256-row GEMM tile reads one contiguous 32 KiB block.
__host__ __device__ constexpr int64_t blk_index(int64_t r, int64_t k, int64_t Kp) {
  return (((r >> 8) * (Kp >> 6) + (k >> 6)) << 14) + ((r & 255) << 6) + (k & 63);
}
constexpr int kSimtTileN = 64;   // (fp32 path)

}  // namespace rft

// Loss-only path from given fp32 logits [T, V]: one workgroup per row.
//   pass 1: stream the row (16-byte loads) keeping per-thread online
//           (max, sum exp, sum exp*z), reduce over the workgroup;
//   row terms: lse, entropy, logp = z_y - lse, the PPO-clip/KL loss terms
//           and c_t = d loss / d logp;
//   pass 2: re-read the row and write d_logits = c_t (onehot - exp(z - lse))
//           with non-temporal stores.
// One workgroup per CU (the kernel reserves most of the LDS) keeps the rows in
// flight small enough that the pass-2 re-read is served by the cache.
#include "rft_internal.h"

namespace rft {
namespace lg {

constexpr int NT = 1024;
constexpr int UNROLL = 4;

struct RowStats {
  float m, s, u;
};

__device__ __forceinline__ void acc4(RowStats& r, float4 q) {
  float mq = fmaxf(fmaxf(q.x, q.y), fmaxf(q.z, q.w));
  if (mq > r.m) {  // rescale to the new running max
    float sc = exp2f((r.m - mq) * kLog2e);
    r.s *= sc;
    r.u *= sc;
    r.m = mq;
  }
  float mk = r.m * kLog2e;
  float e0 = exp2f(fmaf(q.x, kLog2e, -mk)), e1 = exp2f(fmaf(q.y, kLog2e, -mk));
  float e2 = exp2f(fmaf(q.z, kLog2e, -mk)), e3 = exp2f(fmaf(q.w, kLog2e, -mk));
  r.s += (e0 + e1) + (e2 + e3);
  r.u += (e0 * q.x + e1 * q.y) + (e2 * q.z + e3 * q.w);
}

__device__ __forceinline__ void acc1(RowStats& r, float z) {
  if (z > r.m) {
    float sc = exp2f((r.m - z) * kLog2e);
    r.s *= sc;
    r.u *= sc;
    r.m = z;
  }
  float e = exp2f((z - r.m) * kLog2e);
  r.s += e;
  r.u += e * z;
}

// Workgroup reduction of the per-thread online partials, in a fixed order.
__device__ RowStats block_stats(RowStats r, RowStats* sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  float M = wave_max_f(r.m);
  float sc = (r.s > 0.f) ? exp2f((r.m - M) * kLog2e) : 0.f;
  float s = wave_sum_f(r.s * sc), u = wave_sum_f(r.u * sc);
  if (lane == 0) sh[w] = RowStats{M, s, u};
  __syncthreads();
  if (threadIdx.x == 0) {
    float m = -INFINITY, ss = 0.f, uu = 0.f;
    for (int i = 0; i < NT / 64; ++i) lse_merge(m, ss, uu, sh[i].m, sh[i].s, sh[i].u);
    sh[NT / 64] = RowStats{m, ss, uu};
  }
  __syncthreads();
  RowStats out = sh[NT / 64];
  __syncthreads();
  return out;
}

template <bool VEC>
__device__ RowStats row_pass1(const float* __restrict__ z, int64_t V, RowStats* sh) {
  RowStats r = {-INFINITY, 0.f, 0.f};
  if (VEC) {
    const float4* z4 = (const float4*)z;
    int64_t n4 = V >> 2;
    int64_t j = threadIdx.x;
    for (; j + (UNROLL - 1) * NT < n4; j += UNROLL * NT) {
      float4 q[UNROLL];
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) q[u] = z4[j + u * NT];
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) acc4(r, q[u]);
    }
    for (; j < n4; j += NT) acc4(r, z4[j]);
  } else {
    for (int64_t j = threadIdx.x; j < V; j += NT) acc1(r, z[j]);
  }
  return block_stats(r, sh);
}

template <bool VEC>
__device__ void row_pass2(const float* __restrict__ z, int64_t V, float lse, float c, int y,
                          float* __restrict__ out) {
  const float lk = lse * kLog2e;
  if (VEC) {
    const float4* z4 = (const float4*)z;
    floatx4* o4 = (floatx4*)out;
    int64_t n4 = V >> 2;
    for (int64_t j = threadIdx.x; j < n4; j += NT) {
      float4 q = z4[j];
      floatx4 d;
      d[0] = -c * exp2f(fmaf(q.x, kLog2e, -lk));
      d[1] = -c * exp2f(fmaf(q.y, kLog2e, -lk));
      d[2] = -c * exp2f(fmaf(q.z, kLog2e, -lk));
      d[3] = -c * exp2f(fmaf(q.w, kLog2e, -lk));
      if ((y >> 2) == j) d[y & 3] += c;
      __builtin_nontemporal_store(d, o4 + j);
    }
  } else {
    for (int64_t j = threadIdx.x; j < V; j += NT) {
      float d = -c * exp2f(fmaf(z[j], kLog2e, -lk));
      if (j == y) d += c;
      out[j] = d;
    }
  }
}

template <bool VEC>
__device__ void zero_row(float* __restrict__ out, int64_t V) {
  if (VEC) {
    floatx4* o4 = (floatx4*)out;
    floatx4 zz = {0.f, 0.f, 0.f, 0.f};
    for (int64_t j = threadIdx.x; j < (V >> 2); j += NT) __builtin_nontemporal_store(zz, o4 + j);
  } else {
    for (int64_t j = threadIdx.x; j < V; j += NT) out[j] = 0.f;
  }
}

// ---- statistics only (rft_token_logprobs_from_logits)
template <bool VEC>
__global__ void __launch_bounds__(NT) k_logits_stats(const float* __restrict__ logits, int64_t T,
                                                      int64_t V, const uint8_t* __restrict__ mask,
                                                      const int32_t* __restrict__ ids,
                                                      float* __restrict__ logp,
                                                      float* __restrict__ ent,
                                                      float* __restrict__ lse,
                                                      float* __restrict__ gathered) {
  __shared__ RowStats sh[NT / 64 + 1];
  int64_t t = blockIdx.x;
  if (!mask[t]) {
    if (threadIdx.x == 0) {
      logp[t] = 0.f;
      if (ent) ent[t] = 0.f;
      lse[t] = 0.f;
      if (gathered) gathered[t] = 0.f;
    }
    return;
  }
  const float* z = logits + t * V;
  RowStats r = row_pass1<VEC>(z, V, sh);
  if (threadIdx.x == 0) {
    float L = r.m + logf(r.s);
    int y = ids[t];
    bool ok = y >= 0 && (int64_t)y < V;
    float zy = ok ? z[y] : __int_as_float(0x7fc00000);
    lse[t] = L;
    if (ent) ent[t] = L - r.u / r.s;
    logp[t] = zy - L;
    if (gathered) gathered[t] = zy;
  }
}

// ---- d_logits only (rft_ppo_clip_loss_bwd_logits)
template <bool VEC>
__global__ void __launch_bounds__(NT) k_logits_bwd(const float* __restrict__ logits, int64_t T,
                                                    int64_t V, const uint8_t* __restrict__ mask,
                                                    const int32_t* __restrict__ ids,
                                                    const float* __restrict__ lse,
                                                    const float* __restrict__ grad,
                                                    float* __restrict__ dl) {
  int64_t t = blockIdx.x;
  float* out = dl + t * V;
  if (!mask[t]) {
    zero_row<VEC>(out, V);
    return;
  }
  int y = ids[t];
  row_pass2<VEC>(logits + t * V, V, lse[t], grad[t], (y >= 0 && (int64_t)y < V) ? y : -1, out);
}

// ---- fused: statistics, loss terms and d_logits (rft_ppo_clip_fused_logits)
template <bool VEC>
__global__ void __launch_bounds__(NT) k_logits_fused(
    const float* __restrict__ logits, int64_t T, int64_t V, const uint8_t* __restrict__ mask,
    const int32_t* __restrict__ ids, const int32_t* __restrict__ kidx,
    const int32_t* __restrict__ row_seq, const int32_t* __restrict__ n_i,
    const int32_t* __restrict__ meta, const float* __restrict__ old, const float* __restrict__ ref,
    const float* __restrict__ adv, LossConst cst, float* __restrict__ logp,
    float* __restrict__ ent, float* __restrict__ lse_out, float* __restrict__ grad_out,
    float* __restrict__ dl, LossPartial* __restrict__ parts) {
  // (the launch also reserves dynamic LDS it does not use, to keep one
  //  workgroup per CU)
  __shared__ RowStats sh[NT / 64 + 1];
  __shared__ float row_c;
  int64_t t = blockIdx.x;
  float* out = dl + t * V;
  int k = kidx[t];
  if (k < 0) {
    zero_row<VEC>(out, V);
    if (threadIdx.x == 0) {
      logp[t] = 0.f;
      if (ent) ent[t] = 0.f;
      if (lse_out) lse_out[t] = 0.f;
      if (grad_out) grad_out[t] = 0.f;
      parts[t] = LossPartial{0, 0, 0, 0, 0, 0, 0, 0};
    }
    return;
  }
  const float* z = logits + t * V;
  RowStats r = row_pass1<VEC>(z, V, sh);
  if (threadIdx.x == 0) {
    float L = r.m + logf(r.s);
    float H = L - r.u / r.s;
    int y = ids[t];
    bool ok = y >= 0 && (int64_t)y < V;
    float lp = ok ? z[y] - L : __int_as_float(0x7fc00000);
    logp[t] = lp;
    if (ent) ent[t] = H;
    if (lse_out) lse_out[t] = L;
    LossPartial p = {0, 0, 0, 0, 0, 0, 0, 0};
    float c = 0.f;
    if (!ok) {
      p.bad = 1;
    } else {
      int i = row_seq[k];
      float rf = ref ? ref[t] : lp;
      TokLoss Lt = token_loss(lp, old[t], rf, adv[i], n_i[i], meta[0], meta[1], cst);
      p.loss = Lt.w * ((double)Lt.pg + (double)cst.beta * (double)Lt.kl);
      p.pg = Lt.w * (double)Lt.pg;
      p.klw = Lt.w * (double)cst.beta * (double)Lt.kl;
      p.kl = (double)Lt.kl;
      p.ratio = (double)Lt.rho;
      p.ent = (double)H;
      p.clipped = Lt.clipped ? 1 : 0;
      c = (float)(Lt.w * (double)Lt.g);
    }
    if (grad_out) grad_out[t] = c;
    parts[t] = p;
    row_c = c;
    sh[NT / 64].m = L;
  }
  __syncthreads();
  float c = row_c, L = sh[NT / 64].m;
  int y = ids[t];
  row_pass2<VEC>(z, V, L, c, (y >= 0 && (int64_t)y < V) ? y : -1, out);
}

}  // namespace lg

static bool vec_ok(const void* p, int64_t V) {
  return (V % 4 == 0) && (((uintptr_t)p & 15) == 0);
}

hipError_t launch_logits_stats(const float* logits, const rft_tokens& tok, int64_t V, float* logp,
                               float* ent, float* lse, float* gathered, hipStream_t s) {
  if (tok.T <= 0) return hipSuccess;
  if (vec_ok(logits, V))
    lg::k_logits_stats<true><<<(unsigned)tok.T, lg::NT, 0, s>>>(logits, tok.T, V, tok.mask,
                                                                 tok.token_ids, logp, ent, lse, gathered);
  else
    lg::k_logits_stats<false><<<(unsigned)tok.T, lg::NT, 0, s>>>(logits, tok.T, V, tok.mask,
                                                                  tok.token_ids, logp, ent, lse, gathered);
  return hipGetLastError();
}

hipError_t launch_logits_bwd(const float* logits, const rft_tokens& tok, int64_t V,
                             const float* lse, const float* grad, float* dl, hipStream_t s) {
  if (tok.T <= 0) return hipSuccess;
  if (vec_ok(logits, V) && vec_ok(dl, V))
    lg::k_logits_bwd<true><<<(unsigned)tok.T, lg::NT, 0, s>>>(logits, tok.T, V, tok.mask,
                                                               tok.token_ids, lse, grad, dl);
  else
    lg::k_logits_bwd<false><<<(unsigned)tok.T, lg::NT, 0, s>>>(logits, tok.T, V, tok.mask,
                                                                tok.token_ids, lse, grad, dl);
  return hipGetLastError();
}

constexpr size_t kFusedReserve = 96 * 1024;  // bytes of LDS reserved per workgroup

hipError_t launch_logits_fused(const float* logits, const rft_tokens& tok, const TokMeta& m,
                               int64_t V, const float* old, const float* ref, const float* adv,
                               const LossConst& c, float* logp, float* ent, float* lse,
                               float* grad, float* dl, LossPartial* parts, rft_ppo_stats* st,
                               hipStream_t s) {
  if (tok.T > 0) {
    if (vec_ok(logits, V) && vec_ok(dl, V)) {
      hipError_t e = hipFuncSetAttribute((const void*)lg::k_logits_fused<true>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)kFusedReserve);
      if (e != hipSuccess) return e;
      lg::k_logits_fused<true><<<(unsigned)tok.T, lg::NT, kFusedReserve, s>>>(
          logits, tok.T, V, tok.mask, tok.token_ids, m.kidx, m.row_seq, m.n_i, m.meta, old, ref,
          adv, c, logp, ent, lse, grad, dl, parts);
    } else {
      hipError_t e = hipFuncSetAttribute((const void*)lg::k_logits_fused<false>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)kFusedReserve);
      if (e != hipSuccess) return e;
      lg::k_logits_fused<false><<<(unsigned)tok.T, lg::NT, kFusedReserve, s>>>(
          logits, tok.T, V, tok.mask, tok.token_ids, m.kidx, m.row_seq, m.n_i, m.meta, old, ref,
          adv, c, logp, ent, lse, grad, dl, parts);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_loss_final(parts, (int)tok.T, m.meta, st, s);
}

}  // namespace rft

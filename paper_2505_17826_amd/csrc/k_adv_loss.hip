// GRPO group advantages, the per-token PPO-clip/KL loss and the SFT loss with
// their fixed-order fp64 reduction, and the merge of the per-tile
// log-sum-exp partials into per-token log-prob / entropy / lse.
#include "rft_internal.h"

namespace rft {

// ---------------------------------------------------------- advantages ----
// GRPO (Sec. 3.2, Listing 4, advantage_fn "grpo"): one wavefront per group;
// mean and sample (or population) std by wavefront shuffles, computed in fp64.
__global__ void __launch_bounds__(256) k_group_adv(const float* __restrict__ r, int64_t n_groups,
                                                   int G, float eps, int unbiased,
                                                   float* __restrict__ adv) {
  int lane = threadIdx.x & 63;
  int64_t g = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (g >= n_groups) return;
  const float* rg = r + g * G;
  double s = 0.0;
  float mn = INFINITY, mx = -INFINITY;
  for (int j = lane; j < G; j += 64) {
    float v = rg[j];
    s += (double)v;
    mn = fminf(mn, v);
    mx = fmaxf(mx, v);
  }
  s = wave_sum_d(s);
  mn = wave_min_f(mn);
  mx = wave_max_f(mx);
  double mu = s / (double)G;
  double q = 0.0;
  for (int j = lane; j < G; j += 64) {
    double dv = (double)rg[j] - mu;
    q += dv * dv;
  }
  q = wave_sum_d(q);
  bool degenerate = (G < 2) || (mn == mx);
  double sd = degenerate ? 0.0 : sqrt(q / (double)(unbiased ? G - 1 : G));
  for (int j = lane; j < G; j += 64)
    adv[g * G + j] = degenerate ? 0.f : (float)(((double)rg[j] - mu) / (sd + (double)eps));
}

hipError_t launch_group_adv(const float* r, int64_t n_groups, int G, float eps, int unbiased,
                            float* adv, hipStream_t s) {
  if (n_groups > 0)
    k_group_adv<<<(unsigned)((n_groups + 3) / 4), 256, 0, s>>>(r, n_groups, G, eps, unbiased, adv);
  return hipGetLastError();
}

// ------------------------------------------- advantages over group ids ----
// Explicit, variable-size groups: one workgroup per group id scans the ids
// (members in index order, fp64 sums reduced in a fixed order) and writes the
// advantages of its members; rollouts whose id is outside [0, n_groups) get 0
// from k_adv_left_out.  Modes as rft_adv_mode.
template <typename Tv>
__device__ Tv block_sum256(Tv v, Tv* sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  return sh[0] + sh[1] + sh[2] + sh[3];
}

__global__ void __launch_bounds__(256) k_adv_left_out(const int32_t* __restrict__ gid, int64_t n,
                                                      int64_t n_groups, float* __restrict__ adv) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n && (gid[i] < 0 || (int64_t)gid[i] >= n_groups)) adv[i] = 0.f;
}

__global__ void __launch_bounds__(256) k_adv_groups(const float* __restrict__ r,
                                                    const int32_t* __restrict__ gid, int64_t n,
                                                    int mode, float eps, int unbiased,
                                                    float* __restrict__ adv) {
  __shared__ double shd[4];
  __shared__ int shi[4];
  __shared__ float shf[4];
  const int g = (int)blockIdx.x;
  double s = 0.0;
  int cnt = 0;
  float mn = INFINITY, mx = -INFINITY;
  for (int64_t i = threadIdx.x; i < n; i += 256) {
    if (gid[i] != g) continue;
    const float v = r[i];
    s += (double)v;
    ++cnt;
    mn = fminf(mn, v);
    mx = fmaxf(mx, v);
  }
  s = block_sum256(s, shd);
  cnt = block_sum256(cnt, shi);
  mn = wave_min_f(mn);
  mx = wave_max_f(mx);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) shf[threadIdx.x >> 6] = mn;
  __syncthreads();
  mn = fminf(fminf(shf[0], shf[1]), fminf(shf[2], shf[3]));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) shf[threadIdx.x >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(shf[0], shf[1]), fmaxf(shf[2], shf[3]));
  const double G = (double)cnt, mu = cnt > 0 ? s / G : 0.0;
  double sd = 0.0;
  if (mode == RFT_ADV_GRPO) {
    double q = 0.0;
    for (int64_t i = threadIdx.x; i < n; i += 256) {
      if (gid[i] != g) continue;
      const double dv = (double)r[i] - mu;
      q += dv * dv;
    }
    q = block_sum256(q, shd);
    sd = cnt > 1 ? sqrt(q / (unbiased ? G - 1.0 : G)) : 0.0;
  }
  const bool degenerate = cnt < 2 || (mode == RFT_ADV_GRPO && mn == mx);
  for (int64_t i = threadIdx.x; i < n; i += 256) {
    if (gid[i] != g) continue;
    const double v = (double)r[i];
    double a = 0.0;
    if (!degenerate) {
      if (mode == RFT_ADV_GRPO) a = (v - mu) / (sd + (double)eps);
      else if (mode == RFT_ADV_MEAN_CENTER) a = v - mu;
      else a = v - (s - v) / (G - 1.0);
    }
    adv[i] = (float)a;
  }
}

hipError_t launch_group_adv_ids(const float* r, const int32_t* gid, int64_t n, int64_t n_groups,
                                int mode, float eps, int unbiased, float* adv, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_adv_left_out<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(gid, n, n_groups, adv);
  if (n_groups > 0)
    k_adv_groups<<<(unsigned)n_groups, 256, 0, s>>>(r, gid, n, mode, eps, unbiased, adv);
  return hipGetLastError();
}

// -------------------------------------------------------- loss reduction ----
__device__ void block_reduce_partial(LossPartial& p, LossPartial* out) {
  __shared__ LossPartial sh[16];
  int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  p.loss = wave_sum_d(p.loss);
  p.pg = wave_sum_d(p.pg);
  p.klw = wave_sum_d(p.klw);
  p.kl = wave_sum_d(p.kl);
  p.ent = wave_sum_d(p.ent);
  p.ratio = wave_sum_d(p.ratio);
  p.sft = wave_sum_d(p.sft);
  p.entw = wave_sum_d(p.entw);
  p.clipped = wave_sum_ll(p.clipped);
  p.bad = wave_sum_ll(p.bad);
  p.expert = wave_sum_ll(p.expert);
  if (lane == 0) sh[w] = p;
  __syncthreads();
  if (threadIdx.x == 0) {
    LossPartial t = sh[0];
    for (int i = 1; i < (int)(blockDim.x >> 6); ++i) {
      t.loss += sh[i].loss; t.pg += sh[i].pg; t.klw += sh[i].klw; t.kl += sh[i].kl;
      t.ent += sh[i].ent; t.ratio += sh[i].ratio; t.sft += sh[i].sft; t.entw += sh[i].entw;
      t.clipped += sh[i].clipped; t.bad += sh[i].bad; t.expert += sh[i].expert;
    }
    *out = t;
  }
}

// Per-token loss over rows [0, T): grid of 256-row blocks.
__global__ void __launch_bounds__(256) k_loss_fwd(
    const uint8_t* __restrict__ mask, const int32_t* __restrict__ ids, const int32_t* __restrict__ kidx,
    const int32_t* __restrict__ row_seq, const int32_t* __restrict__ n_i, const int32_t* __restrict__ meta,
    int64_t T, const float* __restrict__ logp,
    const float* __restrict__ old, const float* __restrict__ ref, const float* __restrict__ adv,
    const float* __restrict__ ent, LossConst c, float* __restrict__ grad,
    float* __restrict__ egrad, LossPartial* __restrict__ parts) {
  int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  LossPartial p = RFT_ZERO_PARTIAL;
  if (t < T) {
    int k = kidx[t];
    float gout = 0.f, eout = 0.f;
    if (k >= 0) {
      int i = row_seq[k];
      int y = ids[t];
      if (y < 0 || (int64_t)y >= c.V) {
        p.bad = 1;
      } else {
        float lp = logp[t];
        float rf = ref ? ref[t] : lp;
        const bool ex = c.is_expert && c.is_expert[i];
        gout = row_loss(lp, old[t], rf, adv[i], n_i[i], ex, meta, ent ? (double)ent[t] : 0.0, c,
                        p, &eout);
      }
    }
    grad[t] = gout;
    if (egrad) egrad[t] = eout;
  }
  block_reduce_partial(p, parts + blockIdx.x);
}

// One block: fixed-order sum of the block partials into the stats struct.
__global__ void __launch_bounds__(1024) k_loss_final(const LossPartial* __restrict__ parts, int n,
                                                     const int32_t* __restrict__ meta,
                                                     rft_ppo_stats* __restrict__ st, int sft_only) {
  LossPartial p = RFT_ZERO_PARTIAL;
  // each thread sums a contiguous run, in order
  int per = (n + 1023) / 1024;
  int a = threadIdx.x * per, b = min(n, a + per);
  for (int i = a; i < b; ++i) {
    p.loss += parts[i].loss; p.pg += parts[i].pg; p.klw += parts[i].klw; p.kl += parts[i].kl;
    p.ent += parts[i].ent; p.ratio += parts[i].ratio; p.sft += parts[i].sft;
    p.entw += parts[i].entw;
    p.clipped += parts[i].clipped; p.bad += parts[i].bad; p.expert += parts[i].expert;
  }
  __shared__ LossPartial out;
  block_reduce_partial(p, &out);
  __syncthreads();
  if (threadIdx.x == 0) {
    const int N = meta[0], S = meta[1], Ne = meta[2], Ng = N - Ne;
    const double inv = N > 0 ? 1.0 / (double)N : 0.0;
    const double invg = Ng > 0 ? 1.0 / (double)Ng : 0.0;
    st->loss = N > 0 ? out.loss : 0.0;
    st->pg_loss = N > 0 ? out.pg : 0.0;
    st->kl_loss = N > 0 ? out.klw : 0.0;
    st->kl_mean = out.kl * invg;
    st->entropy_mean = out.ent * inv;
    st->ratio_mean = out.ratio * invg;
    st->clipfrac = (double)out.clipped * invg;
    st->n_valid = N;
    st->n_seq_valid = S;
    st->n_clipped = out.clipped;
    st->n_bad_ids = out.bad;
    st->sft_loss = sft_only ? st->loss : (Ne > 0 ? out.sft / (double)Ne : 0.0);
    st->n_expert = Ne;
    st->entropy_loss = N > 0 ? out.entw : 0.0;
  }
}

hipError_t launch_loss_final(const LossPartial* parts, int nparts, const int32_t* meta,
                             rft_ppo_stats* stats, hipStream_t s, int sft_only) {
  k_loss_final<<<1, 1024, 0, s>>>(parts, nparts, meta, stats, sft_only);
  return hipGetLastError();
}

// SFT loss of the train-only mode: sum_t w_t (-logp_t) over the valid rows
// whose id is in range, w_t the aggregation weight; grad = -w_t.
__global__ void __launch_bounds__(256) k_sft_fwd(
    const uint8_t* __restrict__ mask, const int32_t* __restrict__ ids,
    const int32_t* __restrict__ kidx, const int32_t* __restrict__ row_seq,
    const int32_t* __restrict__ n_i, const int32_t* __restrict__ meta, int64_t T, int64_t V,
    const float* __restrict__ logp, int agg, double denom, float* __restrict__ grad,
    LossPartial* __restrict__ parts) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  LossPartial p = RFT_ZERO_PARTIAL;
  if (t < T) {
    const int k = kidx[t];
    float g = 0.f;
    if (k >= 0) {
      const int y = ids[t];
      if (y < 0 || (int64_t)y >= V) {
        p.bad = 1;
      } else {
        const double w = agg_weight(agg, denom, n_i[row_seq[k]], meta[0], meta[1]);
        p.loss = w * -(double)logp[t];
        g = (float)-w;
      }
    }
    grad[t] = g;
  }
  block_reduce_partial(p, parts + blockIdx.x);
}

hipError_t launch_sft_fwd(const rft_tokens& tok, const TokMeta& m, int64_t V, const float* logp,
                          int agg, double denom, float* grad, LossPartial* parts,
                          rft_ppo_stats* st, hipStream_t s) {
  const int nb = (int)((tok.T + 255) / 256);
  if (nb > 0)
    k_sft_fwd<<<nb, 256, 0, s>>>(tok.mask, tok.token_ids, m.kidx, m.row_seq, m.n_i, m.meta, tok.T,
                                 V, logp, agg, denom, grad, parts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_loss_final(parts, nb, m.meta, st, s, 1);
}

hipError_t launch_loss_fwd(const rft_tokens& tok, const TokMeta& m, const float* logp,
                           const float* old, const float* ref, const float* adv, const float* ent,
                           const LossConst& c, float* grad, float* egrad, LossPartial* parts,
                           rft_ppo_stats* st, hipStream_t s) {
  int nb = (int)((tok.T + 255) / 256);
  if (nb > 0)
    k_loss_fwd<<<nb, 256, 0, s>>>(tok.mask, tok.token_ids, m.kidx, m.row_seq, m.n_i, m.meta,
                                  tok.T, logp, old, ref, adv, ent, c, grad, egrad, parts);
  return launch_loss_final(parts, nb, m.meta, st, s);
}

// -------------------------------------------------------- lse partials ----
// Merge the per-vocabulary-tile partials (m, s, u) of each valid row into
// lse, entropy = lse - u/s and logp = z_y - lse; masked rows get 0.
// parts are [ntiles][ld] with the compacted row index as the inner index.
__global__ void __launch_bounds__(256) k_merge_rows(
    const int32_t* __restrict__ kidx, const int32_t* __restrict__ ids, int64_t T, int64_t V,
    const float* __restrict__ pm, const float* __restrict__ ps, const float* __restrict__ pu,
    int ntiles, int64_t ld, const float* __restrict__ zy, float* __restrict__ logp,
    float* __restrict__ ent, float* __restrict__ lse) {
  int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= T) return;
  int k = kidx[t];
  if (k < 0) {
    logp[t] = 0.f;
    if (ent) ent[t] = 0.f;
    lse[t] = 0.f;
    return;
  }
  float m = -INFINITY, sm = 0.f, u = 0.f;
  for (int j = 0; j < ntiles; ++j) {
    int64_t o = (int64_t)j * ld + k;
    lse_merge(m, sm, u, pm[o], ps[o], pu[o]);
  }
  float L = m + logf(sm);
  lse[t] = L;
  if (ent) ent[t] = L - u / sm;
  int y = ids[t];
  logp[t] = (y >= 0 && (int64_t)y < V) ? zy[k] - L : __int_as_float(0x7fc00000);
}

hipError_t launch_merge_rows(const rft_tokens& tok, const TokMeta& m, int64_t V, const float* pm,
                             const float* ps, const float* pu, int ntiles, int64_t ld,
                             const float* zy, float* logp, float* ent, float* lse, hipStream_t s) {
  int nb = (int)((tok.T + 255) / 256);
  if (nb > 0)
    k_merge_rows<<<nb, 256, 0, s>>>(m.kidx, tok.token_ids, tok.T, V, pm, ps, pu, ntiles, ld, zy,
                                    logp, ent, lse);
  return hipGetLastError();
}

}  // namespace rft

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
// Explicit, variable-size groups (modes as rft_adv_mode), in work linear in
// the number of rollouts:
//   k_adv_count    count each group's rollouts (integer atomics: exact), and
//                  give 0 to rollouts whose id is outside [0, n_groups);
//   k_adv_scan_*   exclusive scan of the counts: group g's members go to
//                  mem[off[g] .. off[g + 1]);
//   k_adv_scatter  place each rollout index in its group's range (the order
//                  inside a range depends on the atomics);
//   k_adv_member_groups  one workgroup per group: sort the member indices
//                  (bitonic, in LDS), so the members are in index order
//                  whatever the scatter did, then fp64 sums over them in a
//                  fixed order and the advantages.  A group with more members
//                  than the LDS sort holds scans every id instead (members
//                  in index order as well), which only such large groups pay.
// Results are deterministic run to run.
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

__device__ float block_min256(float v, float* sh) {
  v = wave_min_f(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  return fminf(fminf(sh[0], sh[1]), fminf(sh[2], sh[3]));
}

__device__ float block_max256(float v, float* sh) {
  v = wave_max_f(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  return fmaxf(fmaxf(sh[0], sh[1]), fmaxf(sh[2], sh[3]));
}

constexpr int kAdvScanBlock = 1024;  // counts per block of the scan (4 per thread)
constexpr int kAdvSortSmall = 256;   // members the small-group kernel sorts (1 KiB of LDS)
constexpr int kAdvSortCap = 16384;   // members the large-group kernel sorts (64 KiB)

__global__ void __launch_bounds__(256) k_adv_zero2(int32_t* __restrict__ a, int32_t* __restrict__ b,
                                                   int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) {
    a[i] = 0;
    b[i] = 0;
  }
}

__global__ void __launch_bounds__(256) k_adv_count(const int32_t* __restrict__ gid, int64_t n,
                                                   int64_t n_groups, int32_t* __restrict__ cnt,
                                                   float* __restrict__ adv) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int g = gid[i];
  if (g < 0 || (int64_t)g >= n_groups) adv[i] = 0.f;
  else atomicAdd(cnt + g, 1);
}

// Per block of kAdvScanBlock counts: the block's total.
__global__ void __launch_bounds__(256) k_adv_scan_totals(const int32_t* __restrict__ cnt,
                                                         int64_t ng, int32_t* __restrict__ tot) {
  __shared__ int shi[4];
  const int64_t b0 = (int64_t)blockIdx.x * kAdvScanBlock;
  int v = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t g = b0 + threadIdx.x * 4 + k;
    v += g < ng ? cnt[g] : 0;
  }
  v = block_sum256(v, shi);
  if (threadIdx.x == 0) tot[blockIdx.x] = v;
}

// Exclusive scan of one int per thread over the 256 threads of a block.
__device__ int block_excl_scan256(int v, int* sh) {
  sh[threadIdx.x] = v;
  __syncthreads();
  for (int o = 1; o < 256; o <<= 1) {
    const int add = threadIdx.x >= (unsigned)o ? sh[threadIdx.x - o] : 0;
    __syncthreads();
    sh[threadIdx.x] += add;
    __syncthreads();
  }
  const int incl = sh[threadIdx.x];
  __syncthreads();
  return incl - v;
}

// One block: exclusive scan of the block totals, in place.
__global__ void __launch_bounds__(256) k_adv_scan_top(int32_t* __restrict__ tot, int64_t nb) {
  __shared__ int sh[256];
  int carry = 0;
  for (int64_t b0 = 0; b0 < nb; b0 += 256) {
    const int64_t b = b0 + threadIdx.x;
    const int v = b < nb ? tot[b] : 0;
    const int ex = block_excl_scan256(v, sh);
    if (b < nb) tot[b] = carry + ex;
    // the block's total: the last thread's exclusive value plus its own
    if (threadIdx.x == 255) sh[0] = ex + v;
    __syncthreads();
    carry += sh[0];
    __syncthreads();
  }
}

// off[g] = exclusive prefix of the counts; off[ng] = the total.
__global__ void __launch_bounds__(256) k_adv_scan_apply(const int32_t* __restrict__ cnt,
                                                        int64_t ng, const int32_t* __restrict__ tot,
                                                        int32_t* __restrict__ off) {
  __shared__ int sh[256];
  const int64_t b0 = (int64_t)blockIdx.x * kAdvScanBlock;
  int c[4], v = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t g = b0 + threadIdx.x * 4 + k;
    c[k] = g < ng ? cnt[g] : 0;
    v += c[k];
  }
  int run = tot[blockIdx.x] + block_excl_scan256(v, sh);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t g = b0 + threadIdx.x * 4 + k;
    if (g < ng) off[g] = run;
    run += c[k];
    if (g == ng - 1) off[ng] = run;
  }
}

__global__ void __launch_bounds__(256) k_adv_scatter(const int32_t* __restrict__ gid, int64_t n,
                                                     int64_t n_groups,
                                                     const int32_t* __restrict__ off,
                                                     int32_t* __restrict__ cur,
                                                     int32_t* __restrict__ mem) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int g = gid[i];
  if (g < 0 || (int64_t)g >= n_groups) return;
  mem[off[g] + atomicAdd(cur + g, 1)] = (int32_t)i;
}

// Advantage of reward v in a group with sum s, mean mu, std sd and G members.
__device__ __forceinline__ float adv_value(int mode, bool degenerate, double v, double s,
                                           double mu, double sd, double G, float eps) {
  if (degenerate) return 0.f;
  double a;
  if (mode == RFT_ADV_GRPO) a = (v - mu) / (sd + (double)eps);
  else if (mode == RFT_ADV_MEAN_CENTER) a = v - mu;
  else a = v - (s - v) / (G - 1.0);
  return (float)a;
}

// Groups with LO < G <= CAP members sort them in LDS; with CAP = kAdvSortCap
// the kernel also takes the groups beyond it (by scanning the ids).  Two
// instantiations split the groups so that the many small ones run with little
// LDS per workgroup.
template <int LO, int CAP>
__global__ void __launch_bounds__(256) k_adv_member_groups(
    const float* __restrict__ r, const int32_t* __restrict__ gid, int64_t n,
    const int32_t* __restrict__ off, const int32_t* __restrict__ mem, int mode, float eps,
    int unbiased, float* __restrict__ adv) {
  __shared__ int32_t key[CAP];
  __shared__ double shd[4];
  __shared__ float shf[4];
  const int g = (int)blockIdx.x;
  const int64_t a0 = off[g];
  const int G = off[g + 1] - (int32_t)a0;
  if (G <= LO || (CAP < kAdvSortCap && G > CAP)) return;
  const int tid = threadIdx.x;
  double s = 0.0, q = 0.0;
  float mn = INFINITY, mx = -INFINITY;
  if (G <= CAP) {
    int P = 1;
    while (P < G) P <<= 1;
    for (int k = tid; k < P; k += 256) key[k] = k < G ? mem[a0 + k] : 0x7fffffff;
    __syncthreads();
    // bitonic sort of key[0, P) ascending
    for (int size = 2; size <= P; size <<= 1) {
      for (int stride = size >> 1; stride > 0; stride >>= 1) {
        for (int k = tid; k < P / 2; k += 256) {
          const int lo = 2 * k - (k & (stride - 1));
          const int hi = lo + stride;
          const bool up = (lo & size) == 0;
          const int x = key[lo], y = key[hi];
          if ((x > y) == up) {
            key[lo] = y;
            key[hi] = x;
          }
        }
        __syncthreads();
      }
    }
    for (int k = tid; k < G; k += 256) {
      const float v = r[key[k]];
      s += (double)v;
      mn = fminf(mn, v);
      mx = fmaxf(mx, v);
    }
  } else {
    for (int64_t i = tid; i < n; i += 256) {
      if (gid[i] != g) continue;
      const float v = r[i];
      s += (double)v;
      mn = fminf(mn, v);
      mx = fmaxf(mx, v);
    }
  }
  s = block_sum256(s, shd);
  mn = block_min256(mn, shf);
  mx = block_max256(mx, shf);
  const double Gd = (double)G, mu = s / Gd;
  const bool degenerate = G < 2 || (mode == RFT_ADV_GRPO && mn == mx);
  double sd = 0.0;
  if (mode == RFT_ADV_GRPO && !degenerate) {
    if (G <= CAP) {
      for (int k = tid; k < G; k += 256) {
        const double dv = (double)r[key[k]] - mu;
        q += dv * dv;
      }
    } else {
      for (int64_t i = tid; i < n; i += 256) {
        if (gid[i] != g) continue;
        const double dv = (double)r[i] - mu;
        q += dv * dv;
      }
    }
    q = block_sum256(q, shd);
    sd = sqrt(q / (unbiased ? Gd - 1.0 : Gd));
  }
  if (G <= CAP) {
    for (int k = tid; k < G; k += 256) {
      const int i = key[k];
      adv[i] = adv_value(mode, degenerate, (double)r[i], s, mu, sd, Gd, eps);
    }
  } else {
    for (int64_t i = tid; i < n; i += 256)
      if (gid[i] == g) adv[i] = adv_value(mode, degenerate, (double)r[i], s, mu, sd, Gd, eps);
  }
}

AdvIdsWs carve_adv_ids(Carver& c, int64_t n, int64_t n_groups) {
  AdvIdsWs w;
  const int64_t ng = n_groups > 0 ? n_groups : 1;
  w.cnt = c.take<int32_t>((size_t)ng);
  w.cur = c.take<int32_t>((size_t)ng);
  w.off = c.take<int32_t>((size_t)ng + 1);
  w.tot = c.take<int32_t>((size_t)((ng + kAdvScanBlock - 1) / kAdvScanBlock));
  w.mem = c.take<int32_t>((size_t)(n > 0 ? n : 1));
  return w;
}

hipError_t launch_group_adv_ids(const float* r, const int32_t* gid, int64_t n, int64_t n_groups,
                                int mode, float eps, int unbiased, float* adv, const AdvIdsWs& w,
                                hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const unsigned nbn = (unsigned)((n + 255) / 256);
  if (n_groups > 0)
    k_adv_zero2<<<(unsigned)((n_groups + 255) / 256), 256, 0, s>>>(w.cnt, w.cur, n_groups);
  k_adv_count<<<nbn, 256, 0, s>>>(gid, n, n_groups, w.cnt, adv);
  if (n_groups == 0) return hipGetLastError();
  const int64_t nbs = (n_groups + kAdvScanBlock - 1) / kAdvScanBlock;
  k_adv_scan_totals<<<(unsigned)nbs, 256, 0, s>>>(w.cnt, n_groups, w.tot);
  k_adv_scan_top<<<1, 256, 0, s>>>(w.tot, nbs);
  k_adv_scan_apply<<<(unsigned)nbs, 256, 0, s>>>(w.cnt, n_groups, w.tot, w.off);
  k_adv_scatter<<<nbn, 256, 0, s>>>(gid, n, n_groups, w.off, w.cur, w.mem);
  k_adv_member_groups<0, kAdvSortSmall><<<(unsigned)n_groups, 256, 0, s>>>(
      r, gid, n, w.off, w.mem, mode, eps, unbiased, adv);
  k_adv_member_groups<kAdvSortSmall, kAdvSortCap><<<(unsigned)n_groups, 256, 0, s>>>(
      r, gid, n, w.off, w.mem, mode, eps, unbiased, adv);
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

__global__ void __launch_bounds__(256) k_loss_reduce256(const LossPartial* __restrict__ parts,
                                                        int64_t n, LossPartial* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  LossPartial p = i < n ? parts[i] : RFT_ZERO_PARTIAL;
  block_reduce_partial(p, out + blockIdx.x);
}

hipError_t launch_loss_reduce256(const LossPartial* parts, int64_t n, LossPartial* out,
                                 hipStream_t s) {
  if (n > 0) k_loss_reduce256<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(parts, n, out);
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
  // eight tiles' partials loaded ahead, merged in tile order
  int j = 0;
  for (; j + 8 <= ntiles; j += 8) {
    float a[8], b[8], c[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int64_t o = (int64_t)(j + q) * ld + k;
      a[q] = pm[o];
      b[q] = ps[o];
      c[q] = pu[o];
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) lse_merge(m, sm, u, a[q], b[q], c[q]);
  }
  for (; j < ntiles; ++j) {
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

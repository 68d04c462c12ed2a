// DPO loss over preference pairs (the train-only mode's preference-pair
// data, Sec. 2.1.1 and Sec. 2.3.1), rollouts 2k (chosen) and 2k+1 (rejected):
//   k_dpo_seq    one workgroup per rollout: pi_s and rho_s, the fp64 sums of
//                the policy and reference log-probs over its valid rows with
//                an in-range id, in a fixed order;
//   k_dpo_pairs  one workgroup: counts the pairs whose two rollouts both have
//                a valid row (P), then per pair u = beta ((pi_c - rho_c) -
//                (pi_r - rho_r)), the loss -(1 - ls) log sigmoid(u)
//                - ls log sigmoid(-u), its derivative, d loss / d pi_s for both
//                rollouts, and the statistics, reduced in a fixed order;
//   k_dpo_grad   grad_logp[t] = d loss / d pi_s of the row's rollout (0 on
//                masked rows and rows with an out-of-range id).
#include "rft_internal.h"

namespace rft {

constexpr int kPrefT = 256;

template <typename Tv>
__device__ Tv block_sum(Tv v, Tv* sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  __syncthreads();  // sh may still be read from a previous call
  if (lane == 0) sh[w] = v;
  __syncthreads();
  Tv t = sh[0];
  for (int i = 1; i < (int)(blockDim.x >> 6); ++i) t += sh[i];
  return t;
}

__global__ void __launch_bounds__(kPrefT) k_dpo_seq(
    const int32_t* __restrict__ seq_start, const uint8_t* __restrict__ mask,
    const int32_t* __restrict__ ids, int64_t T, int64_t V, const float* __restrict__ logp,
    const float* __restrict__ ref, double* __restrict__ pi, double* __restrict__ rho,
    int32_t* __restrict__ bad, float* __restrict__ seq_logp) {
  __shared__ double shd[kPrefT / 64];
  __shared__ int shi[kPrefT / 64];
  const int64_t s = blockIdx.x;
  int64_t a = seq_start[s], b = seq_start[s + 1];
  a = a < 0 ? 0 : (a > T ? T : a);
  b = b < a ? a : (b > T ? T : b);
  double sp = 0.0, sr = 0.0;
  int nb = 0;
  for (int64_t t = a + threadIdx.x; t < b; t += kPrefT) {
    if (!mask[t]) continue;
    const int y = ids[t];
    if (y < 0 || (int64_t)y >= V) {
      ++nb;
      continue;
    }
    sp += (double)logp[t];
    sr += (double)ref[t];
  }
  sp = block_sum(sp, shd);
  sr = block_sum(sr, shd);
  nb = block_sum(nb, shi);
  if (threadIdx.x == 0) {
    pi[s] = sp;
    rho[s] = sr;
    bad[s] = nb;
    if (seq_logp) seq_logp[s] = (float)sp;
  }
}

__device__ __forceinline__ double log_sigmoid(double x) {
  return -(fmax(-x, 0.0) + log1p(exp(-fabs(x))));
}

__global__ void __launch_bounds__(1024) k_dpo_pairs(
    int64_t n_pairs, const int32_t* __restrict__ n_i, const int32_t* __restrict__ meta,
    const double* __restrict__ pi, const double* __restrict__ rho,
    const int32_t* __restrict__ bad, double beta, double ls, float* __restrict__ coef,
    rft_dpo_stats* __restrict__ st) {
  __shared__ double shd[16];
  __shared__ long long shl[16];
  // each thread takes a contiguous run of pairs, in order
  const int64_t per = (n_pairs + 1023) / 1024;
  const int64_t k0 = (int64_t)threadIdx.x * per;
  const int64_t k1 = k0 + per < n_pairs ? k0 + per : n_pairs;
  long long cnt = 0, nbad = 0;
  for (int64_t k = k0; k < k1; ++k) {
    cnt += (n_i[2 * k] > 0 && n_i[2 * k + 1] > 0) ? 1 : 0;
    nbad += bad[2 * k] + bad[2 * k + 1];
  }
  const long long P = block_sum(cnt, shl);
  nbad = block_sum(nbad, shl);
  double sl = 0.0, sc = 0.0, sj = 0.0, su = 0.0;
  long long acc = 0;
  for (int64_t k = k0; k < k1; ++k) {
    float cc = 0.f;
    if (n_i[2 * k] > 0 && n_i[2 * k + 1] > 0) {
      const double rc = beta * (pi[2 * k] - rho[2 * k]);
      const double rj = beta * (pi[2 * k + 1] - rho[2 * k + 1]);
      const double u = rc - rj;
      sl += -(1.0 - ls) * log_sigmoid(u) - ls * log_sigmoid(-u);
      sc += rc;
      sj += rj;
      su += u;
      acc += u > 0.0 ? 1 : 0;
      // d loss_k / d u = -(1 - ls) sigmoid(-u) + ls sigmoid(u)
      const double dldu = -(1.0 - ls) * exp(log_sigmoid(-u)) + ls * exp(log_sigmoid(u));
      cc = (float)(beta * dldu / (double)P);
    }
    coef[2 * k] = cc;
    coef[2 * k + 1] = -cc;
  }
  sl = block_sum(sl, shd);
  sc = block_sum(sc, shd);
  sj = block_sum(sj, shd);
  su = block_sum(su, shd);
  acc = block_sum(acc, shl);
  if (threadIdx.x == 0) {
    const double inv = P > 0 ? 1.0 / (double)P : 0.0;
    st->loss = sl * inv;
    st->chosen_reward = sc * inv;
    st->rejected_reward = sj * inv;
    st->reward_acc = (double)acc * inv;
    st->margin_mean = su * inv;
    st->n_pairs = P;
    st->n_valid = meta[0];
    st->n_bad_ids = nbad;
  }
}

__global__ void __launch_bounds__(256) k_dpo_grad(const int32_t* __restrict__ kidx,
                                                  const int32_t* __restrict__ row_seq,
                                                  const int32_t* __restrict__ ids, int64_t T,
                                                  int64_t V, const float* __restrict__ coef,
                                                  float* __restrict__ grad) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= T) return;
  const int k = kidx[t];
  float g = 0.f;
  if (k >= 0) {
    const int y = ids[t];
    if (y >= 0 && (int64_t)y < V) g = coef[row_seq[k]];
  }
  grad[t] = g;
}

hipError_t launch_dpo(const rft_tokens& tok, const TokMeta& m, int64_t V, const float* logp,
                      const float* ref, float beta, float ls, const DpoWs& w, float* grad,
                      float* seq_logp, rft_dpo_stats* st, hipStream_t s) {
  if (tok.n_seq > 0)
    k_dpo_seq<<<(unsigned)tok.n_seq, kPrefT, 0, s>>>(tok.seq_start, tok.mask, tok.token_ids,
                                                     tok.T, V, logp, ref, w.pi, w.rho, w.bad,
                                                     seq_logp);
  k_dpo_pairs<<<1, 1024, 0, s>>>(tok.n_seq / 2, m.n_i, m.meta, w.pi, w.rho, w.bad, (double)beta,
                                 (double)ls, w.coef, st);
  if (tok.T > 0)
    k_dpo_grad<<<(unsigned)((tok.T + 255) / 256), 256, 0, s>>>(m.kidx, m.row_seq, tok.token_ids,
                                                               tok.T, V, w.coef, grad);
  return hipGetLastError();
}

}  // namespace rft

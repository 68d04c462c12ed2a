// Loss-only path from given fp32 logits [T, V]: one workgroup per row.
//   pass 1: stream the row (16-byte loads) keeping per-thread online
//           (max, sum exp, sum exp*z), reduce over the workgroup in a fixed
//           order;
//   row terms: lse, entropy, logp = z_y - lse, the PPO-clip/KL loss terms
//           and c_t = d loss / d logp;
//   pass 2: d_logits = c_t (onehot - p) + e_t p (z - mu_t) (p the softmax,
//           e_t the entropy-bonus coefficient, mu_t = lse - entropy) with
//           non-temporal stores.
// The fused kernel keeps the row on chip between the passes (registers, then
// LDS) so that a row of up to about 600 KB is read from HBM once.  Every kernel
// here gives each thread the same chunks of the row in the same order, so the
// statistics-only, d_logits-only and fused kernels agree bit for bit.
#include "rft_internal.h"

namespace rft {
namespace lg {

constexpr int NT = 512;
constexpr int UNROLL = 4;

struct RowStats {
  float m, s, u;
};

// Online (max, sum exp, sum exp * z) over a thread's logits.  Every exponent
// argument is <= 0 (hardware exp2; results below 2^-126 flush to 0).  Logits
// of -inf (masked entries) add nothing: while the running max is still -inf
// the exponents are taken against 0, and z is clamped to the finite range in
// the product exp * z (0 * z stays 0).
__device__ __forceinline__ float zfin(float z) { return fmaxf(z, -FLT_MAX); }

__device__ __forceinline__ void acc4(RowStats& r, float4 q) {
  float mq = fmaxf(fmaxf(q.x, q.y), fmaxf(q.z, q.w));
  if (mq > r.m) {  // rescale to the new running max
    float sc = __builtin_amdgcn_exp2f((r.m - mq) * kLog2e);
    r.s *= sc;
    r.u *= sc;
    r.m = mq;
  }
  float mk = r.m == -INFINITY ? 0.f : r.m * kLog2e;
  float e0 = __builtin_amdgcn_exp2f(fmaf(q.x, kLog2e, -mk));
  float e1 = __builtin_amdgcn_exp2f(fmaf(q.y, kLog2e, -mk));
  float e2 = __builtin_amdgcn_exp2f(fmaf(q.z, kLog2e, -mk));
  float e3 = __builtin_amdgcn_exp2f(fmaf(q.w, kLog2e, -mk));
  r.s += (e0 + e1) + (e2 + e3);
  r.u += (e0 * zfin(q.x) + e1 * zfin(q.y)) + (e2 * zfin(q.z) + e3 * zfin(q.w));
}

__device__ __forceinline__ void acc1(RowStats& r, float z) {
  if (z > r.m) {
    float sc = __builtin_amdgcn_exp2f((r.m - z) * kLog2e);
    r.s *= sc;
    r.u *= sc;
    r.m = z;
  }
  float e = __builtin_amdgcn_exp2f(fmaf(z, kLog2e, r.m == -INFINITY ? 0.f : -r.m * kLog2e));
  r.s += e;
  r.u += e * zfin(z);
}

// Workgroup reduction of the per-thread online partials, in a fixed order.
template <int NTH = NT>
__device__ RowStats block_stats(RowStats r, RowStats* sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  float M = wave_max_f(r.m);
  float sc = (r.s > 0.f) ? __builtin_amdgcn_exp2f((r.m - M) * kLog2e) : 0.f;
  float s = wave_sum_f(r.s * sc), u = wave_sum_f(r.u * sc);
  if (lane == 0) sh[w] = RowStats{M, s, u};
  __syncthreads();
  if (threadIdx.x == 0) {
    float m = -INFINITY, ss = 0.f, uu = 0.f;
    for (int i = 0; i < NTH / 64; ++i) lse_merge(m, ss, uu, sh[i].m, sh[i].s, sh[i].u);
    sh[NTH / 64] = RowStats{m, ss, uu};
  }
  __syncthreads();
  RowStats out = sh[NTH / 64];
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

// d_logits of one row: c (onehot - p) + e p (z - mu) (dlogit), 16-byte stores.
template <bool VEC>
__device__ void row_pass2(const float* __restrict__ z, int64_t V, float lse, float c, float e,
                          float mu, int y, float* __restrict__ out) {
  const float lk = lse * kLog2e;
  if (VEC) {
    const float4* z4 = (const float4*)z;
    floatx4* o4 = (floatx4*)out;
    int64_t n4 = V >> 2;
    for (int64_t j = threadIdx.x; j < n4; j += NT) {
      float4 q = z4[j];
      const int hot = (y >> 2) == j ? (y & 3) : -1;
      floatx4 d;
      d[0] = dlogit(c, e, mu, __builtin_amdgcn_exp2f(fmaf(q.x, kLog2e, -lk)), q.x, hot == 0);
      d[1] = dlogit(c, e, mu, __builtin_amdgcn_exp2f(fmaf(q.y, kLog2e, -lk)), q.y, hot == 1);
      d[2] = dlogit(c, e, mu, __builtin_amdgcn_exp2f(fmaf(q.z, kLog2e, -lk)), q.z, hot == 2);
      d[3] = dlogit(c, e, mu, __builtin_amdgcn_exp2f(fmaf(q.w, kLog2e, -lk)), q.w, hot == 3);
      __builtin_nontemporal_store(d, o4 + j);
    }
  } else {
    for (int64_t j = threadIdx.x; j < V; j += NT)
      out[j] = dlogit(c, e, mu, __builtin_amdgcn_exp2f(fmaf(z[j], kLog2e, -lk)), z[j], j == y);
  }
}

template <bool VEC, int NTH = NT>
__device__ void zero_row(float* __restrict__ out, int64_t V) {
  if (VEC) {
    floatx4* o4 = (floatx4*)out;
    floatx4 zz = {0.f, 0.f, 0.f, 0.f};
    for (int64_t j = threadIdx.x; j < (V >> 2); j += NTH) __builtin_nontemporal_store(zz, o4 + j);
  } else {
    for (int64_t j = threadIdx.x; j < V; j += NTH) out[j] = 0.f;
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
                                                    const float* __restrict__ egrad,
                                                    const float* __restrict__ ent,
                                                    float* __restrict__ dl) {
  int64_t t = blockIdx.x;
  float* out = dl + t * V;
  if (!mask[t]) {
    zero_row<VEC>(out, V);
    return;
  }
  int y = ids[t];
  const float L = lse[t];
  const float e = egrad ? egrad[t] : 0.f, mu = egrad ? L - ent[t] : 0.f;
  row_pass2<VEC>(logits + t * V, V, L, grad[t], e, mu, (y >= 0 && (int64_t)y < V) ? y : -1, out);
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
  __shared__ float row_c, row_e, row_mu;
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
      parts[t] = RFT_ZERO_PARTIAL;
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
    LossPartial p = RFT_ZERO_PARTIAL;
    float c = 0.f, e = 0.f;
    if (!ok) {
      p.bad = 1;
    } else {
      int i = row_seq[k];
      float rf = ref ? ref[t] : lp;
      const bool ex = cst.is_expert && cst.is_expert[i];
      c = row_loss(lp, old[t], rf, adv[i], n_i[i], ex, meta, (double)H, cst, p, &e);
    }
    if (grad_out) grad_out[t] = c;
    parts[t] = p;
    row_c = c;
    row_e = e;
    row_mu = L - H;
    sh[NT / 64].m = L;
  }
  __syncthreads();
  float c = row_c, L = sh[NT / 64].m;
  int y = ids[t];
  row_pass2<VEC>(z, V, L, c, row_e, row_mu, (y >= 0 && (int64_t)y < V) ? y : -1, out);
}

// ---- fused, with the row kept on chip: the first REG*NTC float4 of the row
// stay in registers and the next LCAP float4 in LDS between the two passes;
// only the remainder is read twice.
typedef int v4i __attribute__((ext_vector_type(4)));
constexpr int NTC = NT;                  // 2 waves per SIMD
constexpr int REG = 56;                  // float4 per thread held in registers
constexpr int REG_ENT = 54;              // the same with the entropy-bonus term (no spills)
// float4 held in LDS (152 KiB): with the registers, rows of up to 153600
// fp32 logits stay on chip (both vocabularies of the workloads)
constexpr int LCAP = 19 * NTC;
constexpr size_t kCachedLds = (size_t)LCAP * 16;
static_assert(LCAP % NTC == 0, "every thread fills the same number of LDS slots");

// d_logits of four logits; ENT adds the entropy-bonus term e p (z - mu)
template <bool ENT>
__device__ __forceinline__ floatx4 dlogit4(floatx4 q, float lk, float c, float e, float mu,
                                           int64_t j, int y) {
  const int hot = (y >> 2) == j ? (y & 3) : -1;
  floatx4 d;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float p = __builtin_amdgcn_exp2f(fmaf(q[i], kLog2e, -lk));
    d[i] = ENT ? dlogit(c, e, mu, p, q[i], hot == i) : c * ((hot == i ? 1.f : 0.f) - p);
  }
  return d;
}

__device__ __forceinline__ void acc4v(RowStats& r, floatx4 q) {
  acc4(r, make_float4(q[0], q[1], q[2], q[3]));
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void* p, int64_t bytes) {
  uint64_t a = (uint64_t)p;
  uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  int nr = __builtin_amdgcn_readfirstlane((int)bytes);
  return __builtin_amdgcn_make_buffer_rsrc((void*)(((uint64_t)hi << 32) | lo), 0, nr, 0x00020000);
}

template <bool ENT, int REGS>
__global__ void __launch_bounds__(NTC) k_logits_fused_cached(
    const float* __restrict__ logits, int64_t T, int64_t V, const uint8_t* __restrict__ mask,
    const int32_t* __restrict__ ids, const int32_t* __restrict__ kidx,
    const int32_t* __restrict__ row_seq, const int32_t* __restrict__ n_i,
    const int32_t* __restrict__ meta, const float* __restrict__ old, const float* __restrict__ ref,
    const float* __restrict__ adv, LossConst cst, float* __restrict__ logp,
    float* __restrict__ ent, float* __restrict__ lse_out, float* __restrict__ grad_out,
    float* __restrict__ dl, LossPartial* __restrict__ parts) {
  extern __shared__ floatx4 row_lds[];  // LCAP float4
  __shared__ RowStats sh[NTC / 64 + 1];
  __shared__ float row_c, row_e, row_mu;
  const int tid = threadIdx.x;
  const int64_t t = blockIdx.x;
  float* out = dl + t * V;
  const int k = kidx[t];
  // one row is V * 4 bytes (at most 1 GiB, checked by the launcher)
  const __amdgpu_buffer_rsrc_t rin = row_rsrc(logits + t * V, V * 4);
  const __amdgpu_buffer_rsrc_t rout = row_rsrc(out, V * 4);
  const uint32_t vo = (uint32_t)tid * 16u;
  constexpr uint32_t SU = (uint32_t)NTC * 16u;  // bytes between a thread's chunks
  const int64_t n4 = V >> 2;
  if (k < 0) {
    const floatx4 zz = {0.f, 0.f, 0.f, 0.f};
    for (int64_t j = tid, o = vo; j < n4; j += NTC, o += SU)
      __builtin_amdgcn_raw_buffer_store_b128((v4i)zz, rout, (uint32_t)o, 0, 2);
    if (tid == 0) {
      logp[t] = 0.f;
      if (ent) ent[t] = 0.f;
      if (lse_out) lse_out[t] = 0.f;
      if (grad_out) grad_out[t] = 0.f;
      parts[t] = RFT_ZERO_PARTIAL;
    }
    return;
  }
  // The row's scalars for the loss terms (uniform over the workgroup: scalar
  // loads), issued now so that they have arrived when pass 1 ends.
  const int y0 = ids[t];
  const bool ok = y0 >= 0 && (int64_t)y0 < V;
  const float zy = ok ? logits[t * V + y0] : 0.f;
  const int i_seq = row_seq[k];
  const float old_t = old[t], ref_t = ref ? ref[t] : 0.f, adv_i = adv[i_seq];
  const int n_seq_i = n_i[i_seq];
  const int32_t meta4[4] = {meta[0], meta[1], meta[2], meta[3]};

  // pass 1.  The LDS part of the row goes straight from HBM into LDS
  // (buffer_load ... lds, all of a lane's chunks in flight at once: lane l of
  // wave w fills slot s = c NTC + 64 w + l with chunk j_lds + s, the slot the
  // same thread reads back), then the register part, then the rest; chunks
  // past the row read as 0 and are left out of the statistics.
  const int64_t j_lds = (int64_t)REGS * NTC, j_rest = j_lds + LCAP;
  {
    const int w = tid >> 6;
#pragma unroll
    for (int c = 0; c < LCAP / NTC; ++c) {
      const int64_t j = j_lds + (int64_t)c * NTC + tid;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rin, (__attribute__((address_space(3))) void*)(row_lds + c * NTC + w * 64), 16,
          j < n4 ? (uint32_t)(j * 16) : 0x80000000u, 0, 0, 2);
    }
  }
  const int u_full = (int)min((int64_t)REGS, n4 / NTC);  // chunks complete for every thread
  // a lane whose chunk lies past the row takes a vector offset of 2^31, out of
  // range for the descriptor whether or not the scalar offset is counted
  const int nv = (int)min((int64_t)REGS, (n4 - tid + NTC - 1) / NTC);  // this lane's chunks
  floatx4 regs[REGS];
#pragma unroll
  for (int u = 0; u < REGS; ++u)
    regs[u] = (floatx4)__builtin_amdgcn_raw_buffer_load_b128(rin, u < nv ? vo : 0x80000000u,
                                                             (uint32_t)u * SU, 2);
  RowStats r = {-INFINITY, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < REGS; ++u) {
    if (u < u_full || (u == u_full && tid + (int64_t)u * NTC < n4)) acc4v(r, regs[u]);
  }
  // the direct-to-LDS loads have landed: this wave's loads are all back
  // (vmcnt 0), then the barrier (each thread reads back only its own slots)
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  __syncthreads();
  for (int64_t j = j_lds + tid, s_ = tid; j < n4 && s_ < LCAP; j += NTC, s_ += NTC)
    acc4v(r, row_lds[s_]);
  for (int64_t j = j_rest + tid; j < n4; j += NTC)
    acc4v(r, (floatx4)__builtin_amdgcn_raw_buffer_load_b128(rin, (uint32_t)(j * 16), 0, 0));
  r = block_stats<NTC>(r, sh);
  if (tid == 0) {
    float L = r.m + logf(r.s);
    float H = L - r.u / r.s;
    float lp = ok ? zy - L : __int_as_float(0x7fc00000);
    logp[t] = lp;
    if (ent) ent[t] = H;
    if (lse_out) lse_out[t] = L;
    LossPartial p = RFT_ZERO_PARTIAL;
    float c = 0.f, e = 0.f;
    if (!ok) {
      p.bad = 1;
    } else {
      float rf = ref ? ref_t : lp;
      const bool ex = cst.is_expert && cst.is_expert[i_seq];  // MIX only
      LossConst cc = cst;
      if (!ENT) cc.ent_coef = 0.f;  // the launcher picks ENT = (ent_coef > 0)
      c = row_loss(lp, old_t, rf, adv_i, n_seq_i, ex, meta4, (double)H, cc, p, &e);
    }
    if (grad_out) grad_out[t] = c;
    parts[t] = p;
    row_c = c;
    row_e = e;
    row_mu = L - H;
    sh[NTC / 64].m = L;
  }
  __syncthreads();
  const float c = row_c, lk = sh[NTC / 64].m * kLog2e, e = row_e, mu = row_mu;
  const int y = ok ? y0 : -1;
  // pass 2: same three regions; stores past the row are dropped by the descriptor
  uint32_t vo2 = vo;
  int nv2 = nv;
  asm volatile("" : "+v"(vo2), "+v"(nv2));  // recomputed here, not held through pass 1
#pragma unroll
  for (int u = 0; u < REGS; ++u)
    __builtin_amdgcn_raw_buffer_store_b128(
        (v4i)dlogit4<ENT>(regs[u], lk, c, e, mu, tid + (int64_t)u * NTC, y), rout,
        u < nv2 ? vo2 + (uint32_t)u * SU : 0x80000000u, 0, 2);
  for (int64_t j = j_lds + tid, s_ = tid; j < n4 && s_ < LCAP; j += NTC, s_ += NTC)
    __builtin_amdgcn_raw_buffer_store_b128((v4i)dlogit4<ENT>(row_lds[s_], lk, c, e, mu, j, y), rout,
                                           (uint32_t)(j * 16), 0, 2);
  for (int64_t j = j_rest + tid; j < n4; j += NTC)
    __builtin_amdgcn_raw_buffer_store_b128(
        (v4i)dlogit4<ENT>((floatx4)__builtin_amdgcn_raw_buffer_load_b128(rin, (uint32_t)(j * 16), 0, 0),
                     lk, c, e, mu, j, y),
        rout, (uint32_t)(j * 16), 0, 2);
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
                             const float* lse, const float* grad, const float* egrad,
                             const float* ent, float* dl, hipStream_t s) {
  if (tok.T <= 0) return hipSuccess;
  if (vec_ok(logits, V) && vec_ok(dl, V))
    lg::k_logits_bwd<true><<<(unsigned)tok.T, lg::NT, 0, s>>>(logits, tok.T, V, tok.mask,
                                                               tok.token_ids, lse, grad, egrad,
                                                               ent, dl);
  else
    lg::k_logits_bwd<false><<<(unsigned)tok.T, lg::NT, 0, s>>>(logits, tok.T, V, tok.mask,
                                                                tok.token_ids, lse, grad, egrad,
                                                                ent, dl);
  return hipGetLastError();
}

constexpr size_t kFusedReserve = 96 * 1024;  // bytes of LDS reserved per workgroup

hipError_t launch_logits_fused(const float* logits, const rft_tokens& tok, const TokMeta& m,
                               int64_t V, const float* old, const float* ref, const float* adv,
                               const LossConst& c, float* logp, float* ent, float* lse,
                               float* grad, float* dl, LossPartial* parts, LossPartial* parts2,
                               rft_ppo_stats* st, hipStream_t s) {
  if (tok.T > 0) {
    // buffer descriptors span one row: 32-bit byte offsets
    if (vec_ok(logits, V) && vec_ok(dl, V) && V <= ((int64_t)1 << 28)) {
      const void* fn = c.ent_coef > 0.f ? (const void*)lg::k_logits_fused_cached<true, lg::REG_ENT>
                                        : (const void*)lg::k_logits_fused_cached<false, lg::REG>;
      hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)lg::kCachedLds);
      if (e != hipSuccess) return e;
      if (c.ent_coef > 0.f)
        lg::k_logits_fused_cached<true, lg::REG_ENT><<<(unsigned)tok.T, lg::NTC, lg::kCachedLds, s>>>(
            logits, tok.T, V, tok.mask, tok.token_ids, m.kidx, m.row_seq, m.n_i, m.meta, old, ref,
            adv, c, logp, ent, lse, grad, dl, parts);
      else
        lg::k_logits_fused_cached<false, lg::REG><<<(unsigned)tok.T, lg::NTC, lg::kCachedLds, s>>>(
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
  // one partial per row: first reduced per 256-row block (fixed order), so
  // that the final single-workgroup sum reads T / 256 partials
  if ((e = launch_loss_reduce256(parts, tok.T, parts2, s)) != hipSuccess) return e;
  return launch_loss_final(parts2, (int)((tok.T + 255) / 256), m.meta, st, s);
}

}  // namespace rft

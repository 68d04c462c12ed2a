// Kernels of the fused trainer step (rft_ppo_clip_step), per chunk of
// compacted rows [c0, c0 + Tc):
//   k_step_rows   merge the chunk's log-sum-exp partials into lse, entropy and
//                 logp, and form the per-token loss gradient c_t = dL/dlogp
//                 (PPO-clip surrogate with the k3 KL term, Sec. 3 of the paper,
//                 and the on-policy / expert split of the MIX loss), and, with
//                 an entropy bonus, its coefficient e_t and the softmax mean
//                 mu_t = lse_t - H_t of the row;
//   k_dz_from_y   dZ = c_t (onehot(y_t) - p) + e_t p (z - mu_t) from the fp16
//                 y = z - (row maximum over the 256-column tile) that the
//                 forward GEMM stored, written in place as bf16 [Tc, Vpad]
//                 (the dH GEMM's operand) and transposed, [Vpad, Tc] (the dW
//                 GEMM's, K-contiguous);
//   k_transpose_hc  the chunk's compacted hidden rows transposed, [d, Tc]
//                 (the dW GEMM's other operand).
// The arithmetic of k_step_rows is that of k_merge_rows and k_loss_fwd (same
// merge order, same per-token formula), so the step and the separate calls
// give the same log-probs and gradients bit for bit.
#include "rft_internal.h"

namespace rft {

__global__ void __launch_bounds__(256) k_step_rows(
    const int32_t* __restrict__ rows, const int32_t* __restrict__ row_seq,
    const int32_t* __restrict__ n_i, const int32_t* __restrict__ meta,
    const int32_t* __restrict__ ids, int64_t V, int64_t c0, int64_t Tc,
    const float* __restrict__ pm, const float* __restrict__ ps, const float* __restrict__ pu,
    int ntiles, const float* __restrict__ zy, const float* __restrict__ old,
    const float* __restrict__ ref, const float* __restrict__ adv, LossConst c,
    float* __restrict__ logp, float* __restrict__ ent, float* __restrict__ lse,
    float* __restrict__ grad, float* __restrict__ ce, float* __restrict__ cmu) {
  const int64_t kl = (int64_t)blockIdx.x * 256 + threadIdx.x;  // row within the chunk
  const int64_t k = c0 + kl;                                    // compacted row
  if (kl >= Tc || k >= (int64_t)meta[0]) return;
  const int t = rows[k];
  float m = -INFINITY, sm = 0.f, u = 0.f;
  for (int j = 0; j < ntiles; ++j) {
    const int64_t o = (int64_t)j * Tc + kl;
    lse_merge(m, sm, u, pm[o], ps[o], pu[o]);
  }
  const float L = m + logf(sm);
  const float H = L - u / sm;
  lse[t] = L;
  if (ent) ent[t] = H;
  const int y = ids[t];
  const bool ok = y >= 0 && (int64_t)y < V;
  const float lp = ok ? zy[k] - L : __int_as_float(0x7fc00000);
  logp[t] = lp;
  float gout = 0.f, eout = 0.f;
  if (ok) {
    const int i = row_seq[k];
    const float rf = ref ? ref[t] : lp;
    const bool ex = c.is_expert && c.is_expert[i];
    LossPartial p = RFT_ZERO_PARTIAL;
    gout = row_loss(lp, old[t], rf, adv[i], n_i[i], ex, meta, 0.0, c, p, &eout);
  }
  grad[t] = gout;
  if (ce) {
    ce[kl] = eout;
    cmu[kl] = L - H;
  }
}

// One 512-thread workgroup per 128 x 256 tile of the chunk (64 KiB of LDS, so
// two workgroups share a CU and one's loads overlap the other's stores).
// Thread tid owns the 8 x 8 block (row block rb = tid / 32, column block
// cb = tid % 32): it issues its eight 16-byte row pieces at once (a wave reads
// two 512-byte rows per instruction) and writes dZ back in place.  The
// transposed copy is staged in LDS (column c of the tile as a 256-byte row,
// its 16-byte chunk j at chunk j ^ ((c >> 3) & 15): the 32 lanes writing one
// column position of 32 blocks hit 16 distinct bank groups) and leaves as
// 16-byte stores, a wave writing four 256-byte rows of dZ^T per instruction.
// Rows of the last tile past the count are written as 0 in both layouts (the
// dW GEMM reads K up to the next multiple of 64).  Tiles wholly past the
// chunk's count are skipped (the backward GEMMs read rows only up to the count).
constexpr int kDzT = 512;
constexpr int kDzRows = 128;  // rows per tile

__device__ __forceinline__ uint32_t bf16_bits(float f) { return (uint32_t)f32_to_bf16(f); }

__global__ void __launch_bounds__(kDzT) k_dz_from_y(
    uint16_t* __restrict__ yz, int64_t Vpad, int64_t Tc, int64_t V,
    const int32_t* __restrict__ rows, const int32_t* __restrict__ ids,
    const int32_t* __restrict__ meta, int64_t c0, const float* __restrict__ pm,
    const float* __restrict__ lse, const float* __restrict__ grad, const float* __restrict__ ce,
    const float* __restrict__ cmu, int ntc, uint16_t* __restrict__ dzt, int64_t ldt) {
  __shared__ float rL[kDzRows], rC[kDzRows], rM[kDzRows], rE[kDzRows], rD[kDzRows];
  __shared__ int rY[kDzRows];
  __shared__ __attribute__((aligned(16))) uint16_t stT[256 * kDzRows];  // [tile column][tile row]
  const int tid = threadIdx.x;
  const int nt = (int)(blockIdx.x % ntc), mt = (int)(blockIdx.x / ntc);
  int64_t count = (int64_t)meta[0] - c0;
  count = count < 0 ? 0 : (count > Tc ? Tc : count);
  const int64_t r0 = (int64_t)mt * kDzRows;
  if (r0 >= count) return;
  const int64_t n0 = (int64_t)nt * 256;
  const int cb = tid & 31, rb = tid >> 5;
  uint16_t* src = yz + (r0 + rb * 8) * Vpad + n0 + cb * 8;
  // this thread's eight row pieces, all in flight before the row parameters
  uint4 in[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) in[r] = *(const uint4*)(src + r * Vpad);
  if (tid < kDzRows) {
    const int64_t r = r0 + tid;
    float L_ = 0.f, C_ = 0.f, M_ = 0.f, E_ = 0.f, D_ = 0.f;
    int Y_ = -1;
    if (r < count) {
      const int t = rows[c0 + r];
      L_ = lse[t];
      C_ = grad[t];
      Y_ = ids[t];
      M_ = pm[(int64_t)nt * Tc + r];
      if (ce) {
        E_ = ce[r];
        D_ = M_ - cmu[r];  // z - mu = y + (tile maximum - mu)
      }
    }
    rL[tid] = L_ * kLog2e;
    rC[tid] = C_;
    rM[tid] = M_ * kLog2e;
    rE[tid] = E_;
    rD[tid] = D_;
    rY[tid] = Y_;
  }
  __syncthreads();
  uint32_t tcol[8][4];  // column q of the block: its 8 rows as bf16 pairs
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int rl = rb * 8 + r;
    const float Lk = rL[rl], Ck = rC[rl], Mk = rM[rl], Ek = rE[rl], Dk = rD[rl];
    const int Yk = rY[rl];
    const bool rv = r0 + rl < count;
    const uint32_t w[4] = {in[r].x, in[r].y, in[r].z, in[r].w};
    uint32_t o[4];
#pragma unroll
    for (int q2 = 0; q2 < 4; ++q2) {
      uint32_t pair = 0;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int q = 2 * q2 + hh;
        const int64_t col = n0 + cb * 8 + q;
        const uint16_t hb = (uint16_t)(w[q2] >> (hh * 16));
        const float yv = (float)__builtin_bit_cast(_Float16, hb);
        const float p = exp2f(fmaf(yv, kLog2e, Mk - Lk));
        float d = dlogit(Ck, Ek, -Dk, p, yv, col == (int64_t)Yk);
        d = (rv && col < V) ? d : 0.f;
        const uint32_t b = bf16_bits(d);
        pair |= b << (hh * 16);
        if (r & 1) tcol[q][r >> 1] |= b << 16;
        else tcol[q][r >> 1] = b;
      }
      o[q2] = pair;
    }
    *(uint4*)(src + r * Vpad) = make_uint4(o[0], o[1], o[2], o[3]);
  }
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const int c = cb * 8 + q;
    *(uint4*)(stT + c * kDzRows + ((rb ^ (cb & 15)) << 3)) =
        make_uint4(tcol[q][0], tcol[q][1], tcol[q][2], tcol[q][3]);
  }
  __syncthreads();
  // dZ^T rows n0 .. n0 + 255, columns r0 .. r0 + 127: 16 chunks per row
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int i = it * kDzT + tid, c = i >> 4, j = i & 15;
    const uint4 v = *(const uint4*)(stT + c * kDzRows + ((j ^ ((c >> 3) & 15)) << 3));
    *(uint4*)(dzt + (n0 + c) * ldt + r0 + j * 8) = v;
  }
}

// Hc^T [d, ldt] of the chunk's compacted hidden rows [c0, c0 + count): 64 x 64
// tiles through LDS; columns count .. (next multiple of 256) are written as 0.
__global__ void __launch_bounds__(256) k_transpose_hc(const uint16_t* __restrict__ hc, int64_t d,
                                                      const int32_t* __restrict__ meta, int64_t c0,
                                                      int64_t Tc, uint16_t* __restrict__ hct,
                                                      int64_t ldt) {
  __shared__ uint16_t t[64][66];
  int64_t count = (int64_t)meta[0] - c0;
  count = count < 0 ? 0 : (count > Tc ? Tc : count);
  const int64_t kend = (count + 255) / 256 * 256;
  const int64_t k0 = (int64_t)blockIdx.x * 64, j0 = (int64_t)blockIdx.y * 64;
  if (k0 >= kend) return;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int r = ty; r < 64; r += 4) {
    const int64_t k = k0 + r, j = j0 + tx;
    t[r][tx] = (k < count && j < d) ? hc[(c0 + k) * d + j] : (uint16_t)0;
  }
  __syncthreads();
  for (int r = ty; r < 64; r += 4) {
    const int64_t j = j0 + r, k = k0 + tx;
    if (j < d) hct[j * ldt + k] = t[tx][r];
  }
}

hipError_t launch_step_rows(const TokMeta& m, const int32_t* ids, int64_t V, int64_t c0,
                            int64_t Tc, const float* pm, const float* ps, const float* pu,
                            int ntiles, const float* zy, const float* old, const float* ref,
                            const float* adv, const LossConst& c, float* logp, float* ent,
                            float* lse, float* grad, float* ce, float* cmu, hipStream_t s) {
  const int nb = (int)((Tc + 255) / 256);
  k_step_rows<<<nb, 256, 0, s>>>(m.rows, m.row_seq, m.n_i, m.meta, ids, V, c0, Tc, pm, ps, pu,
                                 ntiles, zy, old, ref, adv, c, logp, ent, lse, grad, ce, cmu);
  return hipGetLastError();
}

hipError_t launch_dz_from_y(uint16_t* yz, int64_t Vpad, int64_t Tc, int64_t V,
                            const int32_t* rows, const int32_t* ids, const int32_t* meta,
                            int64_t c0, const float* pm, const float* lse, const float* grad,
                            const float* ce, const float* cmu, uint16_t* dzt, int64_t ldt,
                            hipStream_t s) {
  const int ntc = (int)(Vpad / 256);
  const int64_t nb = (Tc / kDzRows) * ntc;
  k_dz_from_y<<<(unsigned)nb, kDzT, 0, s>>>(yz, Vpad, Tc, V, rows, ids, meta, c0, pm, lse, grad,
                                            ce, cmu, ntc, dzt, ldt);
  return hipGetLastError();
}

hipError_t launch_transpose_hc(const uint16_t* hc, int64_t d, const int32_t* meta, int64_t c0,
                               int64_t Tc, uint16_t* hct, int64_t ldt, hipStream_t s) {
  const dim3 grid((unsigned)(Tc / 64), (unsigned)((d + 63) / 64));
  k_transpose_hc<<<grid, 256, 0, s>>>(hc, d, meta, c0, Tc, hct, ldt);
  return hipGetLastError();
}

}  // namespace rft

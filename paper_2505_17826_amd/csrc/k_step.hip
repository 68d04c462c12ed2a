// Kernels of the fused trainer step (rft_ppo_clip_step), per chunk of
// compacted rows [c0, c0 + Tc):
//   k_step_rows   merge the chunk's log-sum-exp partials into lse, entropy and
//                 logp, and form the per-token loss gradient c_t = dL/dlogp
//                 (PPO-clip surrogate with the k3 KL term, Sec. 3 of the paper,
//                 and the on-policy / expert split of the MIX loss), and, with
//                 an entropy bonus, its coefficient e_t and the softmax mean
//                 mu_t = lse_t - H_t of the row;
//   k_dz_from_y_blk  dZ = c_t (onehot(y_t) - p) + e_t p (z - mu_t) from the
//                 fp16 y = z - (row maximum over the 256-column tile) that the
//                 forward GEMM stored, written in place as bf16 [Tc, Vpad]
//                 (the dH GEMM's operand) and transposed, [Vpad, Tc] (the dW
//                 GEMM's, K-contiguous), both tile-blocked;
//   k_transpose_blk  the chunk's compacted hidden rows transposed, [dpad, Tc],
//                 and the weight transposed, [dpad, Vpad], tile-blocked (the
//                 dW and dH GEMMs' other operands).
// The separate backward (rft_ppo_clip_loss_bwd) uses the same blocked
// transposes.
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
  // eight tiles' partials loaded ahead, merged in tile order
  int j = 0;
  for (; j + 8 <= ntiles; j += 8) {
    float a[8], b[8], c[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int64_t o = (int64_t)(j + q) * Tc + kl;
      a[q] = pm[o];
      b[q] = ps[o];
      c[q] = pu[o];
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) lse_merge(m, sm, u, a[q], b[q], c[q]);
  }
  for (; j < ntiles; ++j) {
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

// Tile-blocked variant (the layout the step's backward GEMMs read, blk_index):
// dZ is [Tc, Vpad] blocked, in the place of y, whose 256 x 256 tiles the
// forward stored column-major in the same 128 KiB (the forward then stages
// a tile in LDS with one 8-byte write per four rows of a column); dZ^T is
// [Vpad, Tc] blocked.  One 256-thread workgroup per (256-row panel,
// 256-column vocabulary tile).  Thread tid owns the 8 x 8 piece (rows
// rb * 8 .., columns cb * 8 ..) of each 256 x 64 block: y's block i is the
// same 32 KiB as dZ's block i, read as eight 16-byte column pieces; the next
// block's pieces are in flight while a block is converted, and every thread
// has read a block before any thread writes dZ over it (168 registers
// without the entropy bonus: three workgroups per CU).  The
// conversion has no branches (the hardware exp2 and packed bf16 conversion,
// 32-bit indices, column masks only in the last vocabulary tile); the pass
// is bound by HBM (5.3 TB/s on its 153 GB at the 7B shape).  dZ goes back in place, and
// column q of a piece (eight consecutive chunk rows of dZ^T row v) is 16
// contiguous bytes of dZ^T, so the transposed copy needs no LDS: the 8 lanes
// with one cb fill a whole 128-byte row piece of a dZ^T block.  Rows of the
// panel past the count and columns past V are written as 0 in both layouts
// (the dW GEMM reads K up to the next multiple of 64); panels wholly past the
// count are skipped (the backward GEMMs read rows only up to the count).
constexpr int kDzbT = 256;

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
// Two fp32 values to a packed bf16 pair (a in the low half), rounded to
// nearest even by the hardware conversion.
__device__ __forceinline__ uint32_t pk_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

// dZ of one thread's 8 x 8 piece of a block (cur[q]: the piece's column q,
// rows rb * 8 .. rb * 8 + 7 of y; zrow: its first row in the dZ block; zcol:
// its first row of the transposed piece in the dZ^T block; columns colb ..):
// p = 2^(y log2 e + (tile maximum - lse) log2 e) with the hardware exp2 (its
// argument is <= 0), dZ = c (onehot - p) (+ e p (z - mu) with the entropy
// bonus); rows at or past nvalid give 0, and with MASKCOL columns at or past V.
// Two rows at a time: the row pairs of a row and the column pairs of the
// transposed piece are each one packed conversion.
template <bool BONUS, bool MASKCOL>
__device__ __forceinline__ void dz_piece(const uint4 (&cur)[8], int rb, int colb, int V,
                                         const float* rL, const float* rC, const float* rE,
                                         const float* rD, const int* rY, int nvalid,
                                         uint16_t* zrow, uint16_t* zcol) {
  uint32_t tcol[8][4];  // column q of the piece: its 8 rows as bf16 pairs
#pragma unroll
  for (int r = 0; r < 8; r += 2) {
    float d[2][8];
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
      const int rl = rb * 8 + r + rr;
      const float Lk = rL[rl], Ck = rC[rl];
      const float Ek = BONUS ? rE[rl] : 0.f, Dk = BONUS ? rD[rl] : 0.f;
      const int Yk = rY[rl];
      const bool rv = rl < nvalid;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int col = colb + q;
        const int rp = r + rr;  // row of the piece: half rp & 1 of word rp >> 1 of column q
        const uint32_t w = rp < 2 ? cur[q].x : rp < 4 ? cur[q].y : rp < 6 ? cur[q].z : cur[q].w;
        const uint16_t hb = (uint16_t)(w >> ((rp & 1) * 16));
        const float yv = (float)__builtin_bit_cast(_Float16, hb);
        const float p = __builtin_amdgcn_exp2f(fmaf(yv, kLog2e, Lk));
        float v = BONUS ? dlogit(Ck, Ek, -Dk, p, yv, col == Yk)
                        : Ck * ((col == Yk ? 1.f : 0.f) - p);
        if (MASKCOL) v = col < V ? v : 0.f;
        d[rr][q] = rv ? v : 0.f;
      }
    }
#pragma unroll
    for (int rr = 0; rr < 2; ++rr)
      *(uint4*)(zrow + (r + rr) * 64) =
          make_uint4(pk_bf16(d[rr][0], d[rr][1]), pk_bf16(d[rr][2], d[rr][3]),
                     pk_bf16(d[rr][4], d[rr][5]), pk_bf16(d[rr][6], d[rr][7]));
#pragma unroll
    for (int q = 0; q < 8; ++q) tcol[q][r >> 1] = pk_bf16(d[0][q], d[1][q]);
  }
#pragma unroll
  for (int q = 0; q < 8; ++q)
    *(uint4*)(zcol + (q << 6)) = make_uint4(tcol[q][0], tcol[q][1], tcol[q][2], tcol[q][3]);
}

template <bool BONUS>
__global__ void __launch_bounds__(kDzbT, BONUS ? 2 : 3) k_dz_from_y_blk(
    uint16_t* __restrict__ yz, int64_t Vpad, int64_t Tc, int64_t V,
    const int32_t* __restrict__ rows, const int32_t* __restrict__ ids,
    const int32_t* __restrict__ meta, int64_t c0, const float* __restrict__ pm,
    const float* __restrict__ lse, const float* __restrict__ grad, const float* __restrict__ ce,
    const float* __restrict__ cmu, uint16_t* __restrict__ dzt) {
  __shared__ float rL[256], rC[256], rE[256], rD[256];
  __shared__ int rY[256];
  const int tid = threadIdx.x;
  constexpr int NB = 4;                  // blocks of 64 columns per workgroup
  const int ng = (int)(Vpad / 64) / NB;  // workgroups per panel
  const int g = (int)(blockIdx.x % ng), pn = (int)(blockIdx.x / ng);
  const int kb0 = g * NB;                // first block of the panel
  const int nt = kb0 >> 2;               // its 256-column vocabulary tile
  int64_t count = (int64_t)meta[0] - c0;
  count = count < 0 ? 0 : (count > Tc ? Tc : count);
  const int64_t r0 = (int64_t)pn * 256;
  if (r0 >= count) return;
  const int cb = tid & 7, rb = tid >> 3;
  uint16_t* const tile = yz + (((int64_t)pn * (Vpad >> 6) + kb0) << 14);
  uint16_t* const blk = tile + rb * 512 + cb * 8;         // dZ: row rb * 8 of the block, column cb * 8
  const uint16_t* const ycol = tile + cb * 8 * 256 + rb * 8;  // y: column cb * 8, row rb * 8
  uint4 cur[8], nxt[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) cur[q] = *(const uint4*)(ycol + q * 256);
  {
    const int64_t r = r0 + tid;
    float L_ = 0.f, C_ = 0.f, M_ = 0.f, E_ = 0.f, D_ = 0.f;
    int Y_ = -1;
    if (r < count) {
      const int t = rows[c0 + r];
      L_ = lse[t];
      C_ = grad[t];
      Y_ = ids[t];
      M_ = pm[(int64_t)nt * Tc + r];
      if (BONUS) {
        E_ = ce[r];
        D_ = M_ - cmu[r];  // z - mu = y + (tile maximum - mu)
      }
    }
    rL[tid] = (M_ - L_) * kLog2e;  // p = 2^(y log2 e + (tile maximum - lse) log2 e)
    rC[tid] = C_;
    rE[tid] = E_;
    rD[tid] = D_;
    rY[tid] = Y_;
  }
  __syncthreads();
  uint16_t* const tb = dzt + (((int64_t)nt * (Tc >> 6) + (r0 >> 6) + (rb >> 3)) << 14) + ((rb & 7) << 3);
  const bool colfull = (int64_t)(nt + 1) * 256 <= V;  // every column of the tile is < V
  const int nvalid = (int)(count - r0 < 256 ? count - r0 : 256);
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    // the next block's loads come after the previous block's stores, so that
    // the count of outstanding accesses below covers exactly those loads
    asm volatile("" ::: "memory");
    if (i + 1 < NB) {
#pragma unroll
      for (int q = 0; q < 8; ++q) nxt[q] = *(const uint4*)(ycol + (i + 1) * 16384 + q * 256);
    }
    // every thread has its piece of block i (its loads before the eight just
    // issued are complete) before any thread writes dZ over the block; the
    // empty asm statements keep the compiler from moving memory accesses
    // across the wait and the barrier
    asm volatile("" ::: "memory");
    if (i + 1 < NB)
      __builtin_amdgcn_s_waitcnt(0x0F78);  // vmcnt(8)
    else
      __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    const int kb = (kb0 & 3) + i;  // block within the vocabulary tile
    uint16_t* const zrow = blk + i * 16384;
    uint16_t* const zcol = tb + ((kb * 64 + cb * 8) << 6);
    const int colb = nt * 256 + kb * 64 + cb * 8;
    if (colfull)
      dz_piece<BONUS, false>(cur, rb, colb, (int)V, rL, rC, rE, rD, rY, nvalid, zrow, zcol);
    else
      dz_piece<BONUS, true>(cur, rb, colb, (int)V, rL, rC, rE, rD, rY, nvalid, zrow, zcol);
    if (i + 1 < NB) {
#pragma unroll
      for (int r = 0; r < 8; ++r) cur[r] = nxt[r];
    }
  }
}

// Rows of a row-major src [*, d] (bf16) into a tile-blocked dst [npad, Kp]
// (Kp = d rounded up to 64): dst row k = src row rows[k] (rows = nullptr: row
// k) for k < n, n = cap or the device count clamped to [0, cap]; rows k in
// [n, next multiple of 256) and columns d .. Kp - 1 are written as 0.  One
// workgroup per row at a time, 16 bytes per thread: 8 lanes fill a 128-byte
// row piece of a block.  The fused step's compacted hidden rows (the forward
// GEMM's A) and its copy of the weight (B) are made this way.
__global__ void __launch_bounds__(256) k_rows_to_blk(const uint16_t* __restrict__ src, int64_t d,
                                                     const int32_t* __restrict__ rows,
                                                     const int32_t* __restrict__ meta,
                                                     int64_t cap, int64_t Kp,
                                                     uint16_t* __restrict__ dst) {
  int64_t n = cap;
  if (meta) {
    n = meta[0];
    n = n < 0 ? 0 : (n > cap ? cap : n);
  }
  const int64_t kend = (n + 255) / 256 * 256;
  const int64_t nch = Kp >> 3;
  for (int64_t k = blockIdx.x; k < kend; k += gridDim.x) {
    const bool valid = k < n;
    const int64_t sr = valid ? (rows ? (int64_t)rows[k] : k) : 0;
    for (int64_t c = threadIdx.x; c < nch; c += 256) {
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (valid && c * 8 < d) v = *(const uint4*)(src + sr * d + c * 8);
      *(uint4*)(dst + blk_index(k, c * 8, Kp)) = v;
    }
  }
}

// Row-major src [rows, ncols] (bf16; tile-blocked with Kp = src_kp when
// src_kp > 0) to the tile-blocked transpose dst
// [ncols_pad, Kp]: dst(j, t) = src[r0 + t][j] for the rows t < n (n = nrows,
// or the device count minus r0 clamped to [0, nrows] when meta is given);
// rows t in [n, next multiple of 256) and columns j in [ncols, ncols_pad) are
// written as 0.  A 64 x 64 tile per workgroup through LDS; the output piece
// (64 rows j of 64 consecutive t) is 8 contiguous KiB of one block.
__global__ void __launch_bounds__(256) k_transpose_blk(const uint16_t* __restrict__ src,
                                                       int64_t ncols,
                                                       const int32_t* __restrict__ meta,
                                                       int64_t r0, int64_t nrows, int64_t Kp,
                                                       int64_t src_kp, uint16_t* __restrict__ dst) {
  __shared__ uint16_t t[64][66];
  int64_t n = nrows;
  if (meta) {
    n = (int64_t)meta[0] - r0;
    n = n < 0 ? 0 : (n > nrows ? nrows : n);
  }
  const int64_t kend = (n + 255) / 256 * 256;
  const int64_t t0 = (int64_t)blockIdx.x * 64, j0 = (int64_t)blockIdx.y * 64;
  if (t0 >= kend) return;
  const int tid = threadIdx.x;
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int c = it * 256 + tid, row = c >> 3, ch = c & 7;
    const int64_t tt = t0 + row, j = j0 + ch * 8;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (tt < n && j < ncols)
      v = *(const uint4*)(src + (src_kp ? blk_index(r0 + tt, j, src_kp) : (r0 + tt) * ncols + j));
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) t[row][ch * 8 + e] = (uint16_t)(w[e >> 1] >> ((e & 1) * 16));
  }
  __syncthreads();
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int c = it * 256 + tid, jr = c >> 3, tc = c & 7;
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      o[e] = (uint32_t)t[tc * 8 + 2 * e][jr] | ((uint32_t)t[tc * 8 + 2 * e + 1][jr] << 16);
    *(uint4*)(dst + blk_index(j0 + jr, t0 + tc * 8, Kp)) = make_uint4(o[0], o[1], o[2], o[3]);
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

hipError_t launch_dz_from_y_blk(uint16_t* yz, int64_t Vpad, int64_t Tc, int64_t V,
                                const int32_t* rows, const int32_t* ids, const int32_t* meta,
                                int64_t c0, const float* pm, const float* lse, const float* grad,
                                const float* ce, const float* cmu, uint16_t* dzt, hipStream_t s) {
  const int64_t nb = (Tc / 256) * (Vpad / 256);
  if (nb > 0 && ce)
    k_dz_from_y_blk<true><<<(unsigned)nb, kDzbT, 0, s>>>(yz, Vpad, Tc, V, rows, ids, meta, c0, pm,
                                                         lse, grad, ce, cmu, dzt);
  else if (nb > 0)
    k_dz_from_y_blk<false><<<(unsigned)nb, kDzbT, 0, s>>>(yz, Vpad, Tc, V, rows, ids, meta, c0,
                                                          pm, lse, grad, ce, cmu, dzt);
  return hipGetLastError();
}

hipError_t launch_transpose_blk(const uint16_t* src, int64_t ncols, const int32_t* meta,
                                int64_t r0, int64_t nrows, int64_t Kp, int64_t ncols_pad,
                                uint16_t* dst, hipStream_t s, int64_t src_kp) {
  const dim3 grid((unsigned)(Kp / 64), (unsigned)(ncols_pad / 64));
  if (Kp > 0 && ncols_pad > 0)
    k_transpose_blk<<<grid, 256, 0, s>>>(src, ncols, meta, r0, nrows, Kp, src_kp, dst);
  return hipGetLastError();
}

hipError_t launch_rows_to_blk(const uint16_t* src, int64_t d, const int32_t* rows,
                              const int32_t* meta, int64_t cap, int64_t Kp, uint16_t* dst,
                              hipStream_t s) {
  const int64_t nb = (cap + 255) / 256 * 256;
  if (nb > 0)
    k_rows_to_blk<<<(unsigned)(nb < 16384 ? nb : 16384), 256, 0, s>>>(src, d, rows, meta, cap,
                                                                       Kp, dst);
  return hipGetLastError();
}

}  // namespace rft

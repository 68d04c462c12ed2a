// Token bookkeeping: compaction of the masked rows (the "unpadding" a
// training engine does before the model, Sec. 2.1.2) and per-rollout counts of
// the tokens that enter the objective (action mask, Sec. 2.2 / Sec. 3.1.2).
// Integer work, bit-exact and deterministic: block counts, one scan, scatter.
#include "rft_internal.h"

namespace rft {

namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = kK0Rows / kThreads;  // 8 consecutive rows per thread

__device__ int block_sum_int(int v, int* red) {
  int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  v = wave_sum_i(v);
  if (lane == 0) red[w] = v;
  __syncthreads();
  int t = 0;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) t += red[i];
  __syncthreads();
  return t;
}

// Exclusive scan of one int per thread over a block of kThreads threads.
__device__ int block_excl_scan(int v, int* sh) {
  sh[threadIdx.x] = v;
  __syncthreads();
  for (int o = 1; o < kThreads; o <<= 1) {
    int add = threadIdx.x >= (unsigned)o ? sh[threadIdx.x - o] : 0;
    __syncthreads();
    sh[threadIdx.x] += add;
    __syncthreads();
  }
  int incl = sh[threadIdx.x];
  __syncthreads();
  return incl - v;
}

__global__ void __launch_bounds__(kThreads) k_block_count(const uint8_t* __restrict__ mask,
                                                          int64_t T, int32_t* __restrict__ blk) {
  __shared__ int red[4];
  int64_t r0 = (int64_t)blockIdx.x * kK0Rows;
  int c = 0;
  for (int j = threadIdx.x; j < kK0Rows; j += kThreads) {
    int64_t t = r0 + j;
    if (t < T && mask[t]) ++c;
  }
  c = block_sum_int(c, red);
  if (threadIdx.x == 0) blk[blockIdx.x] = c;
}

__global__ void __launch_bounds__(kThreads) k_seq_count(const uint8_t* __restrict__ mask,
                                                        const int32_t* __restrict__ ss,
                                                        int64_t n_seq, int64_t T,
                                                        int32_t* __restrict__ n_i) {
  __shared__ int red[4];
  int64_t i = blockIdx.x;
  int64_t a = ss[i], b = ss[i + 1];
  a = a < 0 ? 0 : (a > T ? T : a);
  b = b < a ? a : (b > T ? T : b);
  int c = 0;
  for (int64_t t = a + threadIdx.x; t < b; t += kThreads) c += mask[t] ? 1 : 0;
  c = block_sum_int(c, red);
  if (threadIdx.x == 0) n_i[i] = c;
}

// One block: block counts -> exclusive offsets (in place), N and S.
__global__ void __launch_bounds__(kThreads) k_scan(int32_t* __restrict__ blk, int nblk,
                                                   const int32_t* __restrict__ n_i, int64_t n_seq,
                                                   const uint8_t* __restrict__ is_expert,
                                                   int32_t* __restrict__ meta) {
  __shared__ int sh[kThreads];
  __shared__ int red[4];
  int carry = 0;
  for (int b0 = 0; b0 < nblk; b0 += kThreads) {
    int b = b0 + threadIdx.x;
    int v = b < nblk ? blk[b] : 0;
    int ex = block_excl_scan(v, sh);
    if (b < nblk) blk[b] = carry + ex;
    carry += block_sum_int(v, red);
  }
  int s = 0, ne = 0, se = 0;
  for (int64_t i = threadIdx.x; i < n_seq; i += kThreads) {
    s += n_i[i] > 0 ? 1 : 0;
    if (is_expert && is_expert[i]) {
      ne += n_i[i];
      se += n_i[i] > 0 ? 1 : 0;
    }
  }
  s = block_sum_int(s, red);
  ne = block_sum_int(ne, red);
  se = block_sum_int(se, red);
  if (threadIdx.x == 0) {
    meta[0] = carry;
    meta[1] = s;
    meta[2] = ne;
    meta[3] = se;
  }
}

__device__ __forceinline__ int seq_of(const int32_t* __restrict__ ss, int64_t n_seq, int64_t t) {
  // largest i in [0, n_seq-1] with ss[i] <= t (clamped, always in bounds)
  int lo = 0, hi = (int)n_seq - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if ((int64_t)ss[mid] <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__global__ void __launch_bounds__(kThreads) k_scatter(const uint8_t* __restrict__ mask,
                                                      const int32_t* __restrict__ ss, int64_t n_seq,
                                                      int64_t T, const int32_t* __restrict__ blk,
                                                      int32_t* __restrict__ rows,
                                                      int32_t* __restrict__ row_seq,
                                                      int32_t* __restrict__ kidx) {
  __shared__ int sh[kThreads];
  int64_t r0 = (int64_t)blockIdx.x * kK0Rows + (int64_t)threadIdx.x * kPerThread;
  uint8_t f[kPerThread];
  int c = 0;
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    int64_t t = r0 + j;
    f[j] = (t < T && mask[t]) ? 1 : 0;
    c += f[j];
  }
  int off = blk[blockIdx.x] + block_excl_scan(c, sh);
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    int64_t t = r0 + j;
    if (t >= T) break;
    if (f[j]) {
      rows[off] = (int32_t)t;
      row_seq[off] = seq_of(ss, n_seq, t);
      kidx[t] = off;
      ++off;
    } else {
      kidx[t] = -1;
    }
  }
}

}  // namespace

TokMeta carve_tokmeta(Carver& c, int64_t T, int64_t n_seq) {
  TokMeta m;
  int64_t nblk = (T + kK0Rows - 1) / kK0Rows;
  m.rows = c.take<int32_t>(T > 0 ? T : 1);
  m.row_seq = c.take<int32_t>(T > 0 ? T : 1);
  m.kidx = c.take<int32_t>(T > 0 ? T : 1);
  m.n_i = c.take<int32_t>(n_seq > 0 ? n_seq : 1);
  m.blk = c.take<int32_t>(nblk > 0 ? nblk : 1);
  m.meta = c.take<int32_t>(4);
  return m;
}

hipError_t launch_tokmeta(const rft_tokens& tok, const TokMeta& m, hipStream_t s) {
  int64_t T = tok.T, n_seq = tok.n_seq;
  int nblk = (int)((T + kK0Rows - 1) / kK0Rows);
  if (nblk > 0) k_block_count<<<nblk, kThreads, 0, s>>>(tok.mask, T, m.blk);
  if (n_seq > 0) k_seq_count<<<(unsigned)n_seq, kThreads, 0, s>>>(tok.mask, tok.seq_start, n_seq, T, m.n_i);
  k_scan<<<1, kThreads, 0, s>>>(m.blk, nblk, m.n_i, n_seq, tok.is_expert, m.meta);
  if (nblk > 0 && n_seq > 0)
    k_scatter<<<nblk, kThreads, 0, s>>>(tok.mask, tok.seq_start, n_seq, T, m.blk, m.rows,
                                        m.row_seq, m.kidx);
  return hipGetLastError();
}

}  // namespace rft

// fp32 path of the policy head (hidden/weight given in fp32) and the small
// layout kernels (hidden-row compaction, weight transpose,
// masked-row zero fill).
//
// The fp32 GEMM is a plain SIMT tile (64x64, K step 16, 4x4 outputs per
// thread) with general operand strides, so the forward, the recompute, dH and
// dW all use one kernel:
//   C[m, n] = sum_k A(m, k) B(n, k)
//   A(m, k) = A[rowA(m) * sam + k * sak],  rowA(m) = a_map ? a_map[a_moff + m] : m
//   B(n, k) = B[n * sbn + rowB(k) * sbk],  rowB(k) = b_map ? b_map[b_koff + k] : k
#include "rft_internal.h"

namespace rft {
namespace sm {

constexpr int BM = 64, BN = 64, BK = 16, NT = 256;
enum { EPI_STATS = 0, EPI_DZ = 1, EPI_STORE = 2 };

struct Args {
  const float* A; int64_t sam, sak; const int32_t* a_map; int64_t a_moff;
  const float* B; int64_t sbn, sbk; const int32_t* b_map; int64_t b_koff;
  int M, N, K;
  int NB;  // rows of B that exist (B(n, k) is read only for n < NB; 0 = N)
  const int32_t* cnt; int64_t cnt_off, cnt_cap; int m_from_cnt, k_from_cnt;
  const int32_t* rows; int64_t rows_off;
  const int32_t* ids; const float* lse; const float* cgrad;
  const float* egrad; const float* ent;  // EPI_DZ entropy bonus (egrad nullptr = none)
  float* pm; float* ps; float* pu; int64_t ldp; float* zy;
  float* dz; int64_t ldz; int64_t Vvalid;
  float* C; int64_t ldc; int accumulate; int c_scatter;
};

__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_f<0xB1>(v));
  v = fmaxf(v, dpp_f<0x4E>(v));
  v = fmaxf(v, dpp_f<0x141>(v));
  v = fmaxf(v, dpp_f<0x140>(v));
  return v;
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_f<0xB1>(v);
  v += dpp_f<0x4E>(v);
  v += dpp_f<0x141>(v);
  v += dpp_f<0x140>(v);
  return v;
}

template <int EPI>
__global__ void __launch_bounds__(NT) k_gemm32(const Args g) {
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[BK][BN + 4];
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  int M = g.M, K = g.K;
  if (g.cnt) {
    int64_t c = (int64_t)g.cnt[0] - g.cnt_off;
    c = c < 0 ? 0 : (c > g.cnt_cap ? g.cnt_cap : c);
    if (g.m_from_cnt) M = (int)c;
    if (g.k_from_cnt) K = (int)c;
  }
  const int N = g.N;
  const int NB = g.NB > 0 ? g.NB : N;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  if (m0 >= M) return;
  if (EPI == EPI_STORE && g.k_from_cnt && K == 0 && g.accumulate) return;

  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += BK) {
    // each thread loads 4 elements of each operand tile
    for (int e = tid; e < BM * BK; e += NT) {
      int kk = e / BM, mm = e % BM;
      int m = m0 + mm, k = k0 + kk;
      float va = 0.f;
      if (m < M && k < K) {
        int64_t r = g.a_map ? (int64_t)g.a_map[g.a_moff + m] : (int64_t)m;
        va = g.A[r * g.sam + (int64_t)k * g.sak];
      }
      As[kk][mm] = va;
      int n = n0 + mm;
      float vb = 0.f;
      if (n < NB && k < K) {
        int64_t rk = g.b_map ? (int64_t)g.b_map[g.b_koff + k] : (int64_t)k;
        vb = g.B[(int64_t)n * g.sbn + rk * g.sbk];
      }
      Bs[kk][mm] = vb;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }

  // thread (ty, tx) holds rows m0 + ty + 16 i, cols n0 + tx + 16 j
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty + 16 * i;
    const bool rv = m < M;
    if (EPI == EPI_STATS) {
      int y = -1;
      if (rv) y = g.ids[g.rows[g.rows_off + m]];
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (n0 + tx + 16 * j < N) mx = fmaxf(mx, acc[i][j]);
      mx = row16_max(mx);
      float s = 0.f, u = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int n = n0 + tx + 16 * j;
        if (n < N) {
          float p = expf(acc[i][j] - mx);
          s += p;
          u += p * acc[i][j];
        }
        if (rv && n == y) g.zy[g.rows_off + m] = acc[i][j];
      }
      s = row16_sum(s);
      u = row16_sum(u);
      if (rv && tx == 0) {
        int64_t o = (int64_t)blockIdx.x * g.ldp + g.rows_off + m;
        g.pm[o] = mx;
        g.ps[o] = s;
        g.pu[o] = u;
      }
    } else if (EPI == EPI_DZ) {
      int y = -1;
      float L = 0.f, c = 0.f, e = 0.f, mu = 0.f;
      if (rv) {
        int t = g.rows[g.rows_off + m];
        y = g.ids[t];
        L = g.lse[t];
        c = g.cgrad[t];
        if (g.egrad) {
          e = g.egrad[t];
          mu = L - g.ent[t];
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int n = n0 + tx + 16 * j;
        if (n < N) {
          float d = 0.f;
          if (rv && n < g.Vvalid) d = dlogit(c, e, mu, expf(acc[i][j] - L), acc[i][j], n == y);
          g.dz[(int64_t)m * g.ldz + n] = d;
        }
      }
    } else {
      if (!rv) continue;
      int64_t dst = (g.c_scatter ? (int64_t)g.rows[g.rows_off + m] : (int64_t)m) * g.ldc;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int n = n0 + tx + 16 * j;
        if (n < N) {
          float v = acc[i][j];
          if (g.accumulate) v += g.C[dst + n];
          g.C[dst + n] = v;
        }
      }
    }
  }
}

}  // namespace sm

static dim3 grid32(int64_t M, int64_t N) {
  return dim3((unsigned)((N + sm::BN - 1) / sm::BN), (unsigned)((M + sm::BM - 1) / sm::BM));
}

hipError_t simt_fwd_stats(const float* H, int64_t d, const float* W, int64_t V, const int32_t* rows,
                          const int32_t* ids, const int32_t* cnt, int64_t cap, float* pm, float* ps,
                          float* pu, int64_t ldp, float* zy, hipStream_t s) {
  if (cap <= 0) return hipSuccess;
  sm::Args a = {};
  a.A = H; a.sam = d; a.sak = 1; a.a_map = rows; a.a_moff = 0;
  a.B = W; a.sbn = d; a.sbk = 1;
  a.M = (int)cap; a.N = (int)V; a.K = (int)d;
  a.cnt = cnt; a.cnt_off = 0; a.cnt_cap = cap; a.m_from_cnt = 1;
  a.rows = rows; a.rows_off = 0; a.ids = ids;
  a.pm = pm; a.ps = ps; a.pu = pu; a.ldp = ldp; a.zy = zy;
  sm::k_gemm32<sm::EPI_STATS><<<grid32(cap, V), sm::NT, 0, s>>>(a);
  return hipGetLastError();
}

// dZ (fp32) of compacted rows [c0, c0 + Tc) into dz [Tc, ldz]; columns >= V are 0.
hipError_t simt_dz(const float* H, int64_t d, const float* W, int64_t V, int64_t Vpad,
                   const int32_t* rows, const int32_t* ids, const float* lse, const float* cgrad,
                   const float* egrad, const float* ent, const int32_t* cnt, int64_t c0,
                   int64_t Tc, float* dz, hipStream_t s) {
  sm::Args a = {};
  a.A = H; a.sam = d; a.sak = 1; a.a_map = rows; a.a_moff = c0;
  a.B = W; a.sbn = d; a.sbk = 1;
  a.M = (int)Tc; a.N = (int)Vpad; a.K = (int)d;
  a.cnt = cnt; a.cnt_off = c0; a.cnt_cap = Tc; a.m_from_cnt = 1;
  a.rows = rows; a.rows_off = c0; a.ids = ids; a.lse = lse; a.cgrad = cgrad;
  a.egrad = egrad; a.ent = ent;
  a.dz = dz; a.ldz = Vpad; a.Vvalid = V;
  a.NB = (int)V;  // W has V rows; columns V..Vpad-1 are written as 0
  sm::k_gemm32<sm::EPI_DZ><<<grid32(Tc, Vpad), sm::NT, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t simt_gemm_store(const float* A, int64_t sam, int64_t sak, const float* B, int64_t sbn,
                           int64_t sbk, const int32_t* b_map, int64_t b_koff, int64_t M, int64_t N,
                           int64_t K, const int32_t* cnt, int64_t cnt_off, int64_t cnt_cap,
                           int m_from_cnt, int k_from_cnt, float* C, int64_t ldc,
                           const int32_t* rows, int64_t rows_off, int accumulate, hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  sm::Args a = {};
  a.A = A; a.sam = sam; a.sak = sak;
  a.B = B; a.sbn = sbn; a.sbk = sbk; a.b_map = b_map; a.b_koff = b_koff;
  a.M = (int)M; a.N = (int)N; a.K = (int)K;
  a.cnt = cnt; a.cnt_off = cnt_off; a.cnt_cap = cnt_cap; a.m_from_cnt = m_from_cnt;
  a.k_from_cnt = k_from_cnt;
  a.C = C; a.ldc = ldc; a.rows = rows; a.rows_off = rows_off; a.c_scatter = rows != nullptr;
  a.accumulate = accumulate;
  sm::k_gemm32<sm::EPI_STORE><<<grid32(M, N), sm::NT, 0, s>>>(a);
  return hipGetLastError();
}

// ------------------------------------------------------- layout helpers ----
// Hc[k, :] = H[rows[k], :] for the valid rows k < count (bf16, 16-byte copies):
// the compacted hidden states every GEMM of the bf16 path reads.
__global__ void __launch_bounds__(256) k_gather_rows16(const uint16_t* __restrict__ H, int64_t d,
                                                       const int32_t* __restrict__ rows,
                                                       const int32_t* __restrict__ cnt,
                                                       int64_t cap, uint16_t* __restrict__ Hc) {
  int64_t n = cnt[0];
  n = n < 0 ? 0 : (n > cap ? cap : n);
  const int64_t d8 = d >> 3;
  for (int64_t k = blockIdx.x; k < n; k += gridDim.x) {
    const uint4* src = (const uint4*)(H + (int64_t)rows[k] * d);
    uint4* dst = (uint4*)(Hc + k * d);
    for (int64_t j = threadIdx.x; j < d8; j += 256) dst[j] = src[j];
  }
}

// Zero the rows of out[T, width] whose mask is 0.
__global__ void __launch_bounds__(256) k_zero_masked_rows(const uint8_t* __restrict__ mask,
                                                          int64_t T, int64_t width,
                                                          float* __restrict__ out) {
  for (int64_t t = blockIdx.x; t < T; t += gridDim.x) {
    if (mask[t]) continue;
    for (int64_t j = threadIdx.x; j < width; j += 256) out[t * width + j] = 0.f;
  }
}

__global__ void __launch_bounds__(256) k_fill_zero(float* __restrict__ out, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    out[i] = 0.f;
}

hipError_t launch_fill_zero(float* out, int64_t n, hipStream_t s) {
  if (n > 0) {
    int64_t b = (n + 255) / 256;
    k_fill_zero<<<(unsigned)(b < 8192 ? b : 8192), 256, 0, s>>>(out, n);
  }
  return hipGetLastError();
}

hipError_t launch_gather_rows16(const uint16_t* H, int64_t d, const int32_t* rows,
                                const int32_t* cnt, int64_t cap, uint16_t* Hc, hipStream_t s) {
  if (cap > 0) k_gather_rows16<<<(unsigned)(cap < 16384 ? cap : 16384), 256, 0, s>>>(H, d, rows, cnt, cap, Hc);
  return hipGetLastError();
}

hipError_t launch_zero_masked_rows(const uint8_t* mask, int64_t T, int64_t width, float* out,
                                   hipStream_t s) {
  if (T > 0) k_zero_masked_rows<<<(unsigned)(T < 4096 ? T : 4096), 256, 0, s>>>(mask, T, width, out);
  return hipGetLastError();
}

}  // namespace rft

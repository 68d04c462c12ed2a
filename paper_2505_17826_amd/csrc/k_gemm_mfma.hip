// bf16 MFMA "NT" GEMM core for gfx950 with the trainer-step epilogues:
//   C[m, n] = sum_k A[m, k] * B[n, k]   (both operands K-contiguous, bf16)
// 256x256 workgroup tile, BK = 64, eight wavefronts (two per SIMD, so one
// wave's LDS and barrier waits overlap the other's MFMAs), each owning 64x128
// of C as 4x8 v_mfma_f32_16x16x32_bf16 tiles (fp32 accumulators).  Operands go
// straight from HBM/L2 into LDS with buffer_load_dwordx4 ... lds (no staging
// registers), issued by four of the eight waves; the buffer descriptor covers only the tile's valid rows, so rows
// past the end and the K tail read as zeros without branches.  LDS holds
// 16-byte chunks XOR-swizzled by row pair (conflict-free ds_read_b128 of MFMA
// fragments in the 64-bank LDS) in two stages.  Workgroups map to tiles so
// that the ones resident on one XCD work on neighbouring tiles (shared L2)
// and all XCDs sweep the same B columns together (shared last-level cache).
// The number of rows can come from a device counter, so the host never waits
// for the count of valid tokens.
//
// Operand layouts: row-major with leading dimension ld, or tile-blocked (the
// layout the fused step keeps its backward operands in): 256-row panels, each
// 256 x Kp (Kp = ld, a multiple of 64) stored as Kp / 64 consecutive blocks of
// 256 rows x 64 values, row-major inside a block (blk_index in rft_internal.h).
// A k-step of a tile then reads one contiguous 32 KiB block per operand instead
// of 256 pieces of 128 bytes a row pitch apart; with row pitches of hundreds of
// KiB (dZ, W^T, dZ^T, Hc^T) the scattered pieces cost 10-15% of the GEMM.
//
// Epilogues:
//   EPI_STATS  forward of the policy head: per row and 256-column vocabulary
//              tile, online log-sum-exp partials (max, sum exp, sum exp*z) and
//              the logit of the sampled token.  Logits are never stored.
//   EPI_STATS_Y  EPI_STATS, and also z minus the row's maximum over the
//              tile, rounded to fp16, each 256 x 256 tile column-major in the
//              128 KiB that the tile-blocked [rows, Vpad] layout gives it (the
//              backward then forms dZ from it instead of recomputing z).
//   EPI_DZ     backward recompute: dZ = c (onehot(y) - p) + e p (z - mu) in bf16,
//              written tile-blocked [rows, Vpad] (the dH operand) and
//              transposed, [Vpad, ldzt] (the dW operand, K-contiguous).
//   EPI_STORE  fp32 result, optionally scattered to rows through a map and
//              optionally added to the existing values.  On tile-blocked
//              operands (dH, dW of the step) k_gemm384 does this on a
//              384 x 256 tile (fewer operand bytes per flop).
#include <atomic>
#include <cstdlib>

#include "rft_internal.h"

namespace rft {
namespace mf {

constexpr int BM = 256, BN = 256, BK = 64, NT = 512;
constexpr int A_BYTES = BM * BK * 2;
constexpr int B_BYTES = BN * BK * 2;
constexpr int STAGE = A_BYTES + B_BYTES;  // 64 KiB
constexpr int ROWP = BM * 20;             // per-row epilogue parameters (five words)
// dZ epilogue: one 256x256 bf16 tile staged in LDS, rows padded to 528 bytes
// (conflict-free 2- and 8-byte writes, contiguous 16-byte reads); the
// transposed tile (dZ^T, and the forward's y, staged column by column) uses
// rows of 544 bytes (a lane's 8-byte write of four consecutive rows of one
// column: the 16 columns of a lane group 8 banks apart, the 4 row groups 2
// banks apart, so a wave's 64 writes cover every bank twice)
constexpr int STG_PITCH = 528;
constexpr int STG_PITCH_T = 544;
constexpr int STG_BYTES = 256 * STG_PITCH_T;
constexpr int LDS_MAIN = 2 * STAGE + ROWP > STG_BYTES ? 2 * STAGE + ROWP : STG_BYTES;
// statistics epilogue: exchange between the two column halves of a tile,
// outside the staging tile (partials [256][3], half maxima [2][256])
constexpr int XCH_BYTES = 256 * 3 * 4 + 2 * 256 * 4;
constexpr int LDS_TOTAL = LDS_MAIN + XCH_BYTES;

enum { EPI_STATS = 0, EPI_DZ = 1, EPI_STORE = 2, EPI_STATS_Y = 3 };

typedef __attribute__((address_space(3))) void* lds_ptr;

// wait for this wave's outstanding vector-memory loads (including the
// loads that write LDS directly)
__device__ __forceinline__ void wait_vm() { __builtin_amdgcn_s_waitcnt(0x0F70); }

struct Args {
  const uint16_t* A;  // [M, lda]
  int64_t lda;
  const uint16_t* B;  // [NB, ldb]
  int64_t ldb;
  int M, N, K;        // host values (M, K are caps when taken from the device counter)
  int NB;             // rows of B that exist (read only for n < NB; 0 = N)
  int a_blk, b_blk;   // operand tile-blocked (ld = Kp; whole 256-row panels are read)
  const int32_t* cnt; // device counter: c = clamp(*cnt - cnt_off, 0, cnt_cap) (nullptr = none)
  int64_t cnt_off;
  int64_t cnt_cap;
  int m_from_cnt;     // M = c
  int k_from_cnt;     // K = round_up(c, BK)
  // epilogue data
  const int32_t* rows;  // compacted row -> token row (index rows_off + m)
  int64_t rows_off;
  const int32_t* ids;
  const float* lse;
  const float* cgrad;
  const float* egrad;  // EPI_DZ entropy-bonus coefficients (nullptr = none)
  const float* ent;    //   and entropies, read only with egrad
  float* pm; float* ps; float* pu; int64_t ldp; float* zy;  // EPI_STATS: partials at p_off + m,
  int64_t p_off;                                            //   zy at rows_off + m
  uint16_t* y; int64_t ldy;                                 // EPI_STATS_Y: fp16 z - tile max, the
                                                            //   tiles of a blocked [rows, ldy]
                                                            //   buffer, each column-major
  uint16_t* dz; int64_t ldz; int64_t Vvalid;                  // EPI_DZ, tile-blocked (Kp = ldz)
  uint16_t* dzt; int64_t ldzt;                                //   and dZ^T [Vpad, ldzt] blocked (nullptr = none)
  float* C; int64_t ldc; int accumulate; int c_scatter;  // EPI_STORE
  int sel;            // EPI_STORE with both tile sizes launched: 1 = the 384-row kernel runs
  int ncu;            //   only if prefer384(M, N, ncu), 2 = the 256-row kernel only if not
};

// fp32-store GEMM on tile-blocked operands: whether the 384 x 256 tile beats
// the 256 x 256 one for an M x N result on ncu compute units.  Tiles run in
// rounds of ncu (one workgroup per CU), so the time is about ceil(tiles / ncu)
// tile times; a 384-row tile takes 1.43 times a 256-row one (1.5 times the
// work at ~5% more flops per cycle, measured on the 7B shapes).  E.g. d_hidden
// of 131072 rows and d = 3584: 19 rounds of 384 (27.2) against 28 of 256;
// with d = 1536: 9 (12.9) against 12; 36901 rows, d = 3584: 6 (8.6) against 8.
__host__ __device__ inline bool prefer384(int64_t M, int64_t N, int64_t ncu) {
  const int64_t tn = (N + 255) / 256;
  const int64_t r4 = ((M + 383) / 384 * tn + ncu - 1) / ncu;
  const int64_t r2 = ((M + 255) / 256 * tn + ncu - 1) / ncu;
  return r4 * 143 < r2 * 100;
}

// Raw buffer descriptor (wave-uniform) over `bytes` bytes from p.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, int64_t bytes) {
  uint64_t a = (uint64_t)p;
  uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  int nr = __builtin_amdgcn_readfirstlane((int)bytes);
  return __builtin_amdgcn_make_buffer_rsrc((void*)(((uint64_t)hi << 32) | lo), 0, nr, 0x00020000);
}

// LDS layout of a stage: rows of BK bf16 (128 B), 16-byte chunk c of row r
// stored at chunk c ^ ((r >> 1) & 7).  The LDS serves 256 B per clock in 64
// banks, i.e. two 128-byte rows; a ds_read_b128 of an MFMA fragment (32 rows,
// one logical chunk) then touches 16 distinct 16-byte bank groups in every
// group of 16 lanes, so fragment reads are conflict free.
//
// Stage loader: waves 0 .. NLOAD-1 issue the loads (NLOAD = 4: wave w fills
// rows [w*64, w*64+64) of the A tile and then of the B tile with 8 + 8
// instructions of 8 rows each; NLOAD = 2: 128 rows with 16 + 16); the other
// waves only compute.  (Measured on gfx950: four loader waves issuing A
// and B in two separate runs keep the L2 round trip of the direct-to-LDS
// loads markedly shorter than eight waves or interleaved A/B loads.)  Lane l
// writes LDS slot l of an instruction (row p*8 + l/8 of the wave's rows,
// physical chunk l%8), so it loads logical chunk
// (l%8) ^ (((p*8 + l/8) >> 1) & 7) = (l%8) ^ (l/16) ^ 4*(p&1); the two
// parities of p take the offsets vA[0|1], vB[0|1].  Chunks at or past K are
// read from outside the descriptor (0).
// Loader waves per epilogue: two for the GEMMs on tile-blocked operands (dH
// and dW: 1-1.7% faster than four; the fused step's forward: 3% faster than
// four, one 15% slower), four for the forward on row-major operands.
template <int EPI> constexpr int kNLoad = (EPI == EPI_STORE || EPI == EPI_STATS_Y) ? 2 : 4;
struct LoadGeom {
  uint32_t vA[2], vB[2];  // per-lane byte offsets for even / odd p (k0 = 0)
  int kc[2];              // logical chunk * 8 (first element) for even / odd p
  uint32_t sA, sB;        // bytes between instructions (8 rows)
  uint32_t kA, kB;        // bytes per element of k0 (2 row-major, 512 blocked)
};

template <int NLOAD>
__device__ __forceinline__ void load_stage(__amdgpu_buffer_rsrc_t rA, __amdgpu_buffer_rsrc_t rB,
                                           char* dst, int k0, int K, const LoadGeom& lg) {
  constexpr int NI = 32 / NLOAD;  // instructions per operand per loader wave
#pragma unroll
  for (int p = 0; p < NI; ++p) {
    const int q = p & 1;
    const uint32_t va = k0 + lg.kc[q] < K ? lg.vA[q] + (uint32_t)k0 * lg.kA : 0x80000000u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (lds_ptr)(dst + p * 1024), 16,
                                             va + (uint32_t)p * lg.sA, 0, 0, 0);
  }
#pragma unroll
  for (int p = 0; p < NI; ++p) {
    const int q = p & 1;
    const uint32_t vb = k0 + lg.kc[q] < K ? lg.vB[q] + (uint32_t)k0 * lg.kB : 0x80000000u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rB, (lds_ptr)(dst + A_BYTES + p * 1024), 16,
                                             vb + (uint32_t)p * lg.sB, 0, 0, 0);
  }
}

// Tile order.  Workgroup b runs on XCD x = b % 8 as the j = b / 8-th
// workgroup dispatched there.  M-tiles are taken in super-groups of 8 SG: XCD
// x owns M-tiles [8 SG s + SG x, 8 SG s + SG x + SG) of super-group s and
// walks them SG at a time along N, so with SG = 8 the 32 workgroups resident
// on one XCD cover 8 M-tiles x 4 N-tiles (A and B slabs shared in that XCD's
// L2) and all XCDs read the same B columns at the same time (shared in the
// last-level cache).  M-tiles past the last full super-group are dealt
// round-robin over the XCDs.  Returns false for workgroups with no tile.
// SG = 8 for the forward GEMMs (N = the vocabulary); SG = 4 (4 x 8 tiles per
// XCD) for the fp32-store GEMMs, whose N is the hidden size and whose big
// operand streams from HBM: dH and dW 1.2% faster, the forward 2% slower.
template <int EPI> constexpr int kSG = EPI == EPI_STORE ? 4 : 8;
template <int SG>
__device__ __forceinline__ bool tile_of(int b, int nTm, int nTn, int& mt, int& nt) {
  const int x = b & 7, j = b >> 3;
  const int full = nTm / (8 * SG);
  const int per = SG * nTn;  // tiles per XCD per super-group
  if (j < full * per) {
    const int s_ = j / per, r = j - s_ * per;
    mt = s_ * 8 * SG + x * SG + r % SG;
    nt = r / SG;
    return true;
  }
  const int R = nTm - full * 8 * SG;
  const int t = (j - full * per) * 8 + x;
  if (t >= R * nTn) return false;
  mt = full * 8 * SG + t % R;
  nt = t / R;
  return true;
}

// Workgroups needed for nTm x nTn tiles in that order (non-decreasing in
// nTm, so a grid sized for the largest M covers every smaller M).
template <int SG>
inline int64_t grid_tiles(int64_t nTm, int64_t nTn) {
  const int64_t full = nTm / (8 * SG);
  const int64_t R = nTm - full * 8 * SG;
  return 8 * (full * SG * nTn + (R * nTn + 7) / 8);
}

// Workgroup barrier without the implicit wait for outstanding loads; the
// empty asm statements keep the compiler from moving LDS accesses across it.
__device__ __forceinline__ void barrier_lds() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Copy a staged 256 x 256 tile of 16-bit values to the tile-blocked layout:
// the 256 x 256 tile is four
// consecutive 256 x 64 blocks (dst = the first), 128 contiguous KiB.  Reads
// are those of stage_copy_out (16 lanes take 256 contiguous bytes of one LDS
// row, rows PITCH bytes apart); every 128-byte row piece of a block is
// written whole, with non-temporal stores (the forward's y is read back only
// after the whole forward of the chunk: 4 ms less per 7B step than cached
// stores).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
template <int PITCH>
__device__ __forceinline__ void stage_copy_out_blk(const char* st, uint16_t* dst, int tid) {
#pragma unroll 4
  for (int it = 0; it < 16; ++it) {
    const int c = it * NT + tid, row = c >> 5, ch = c & 31;
    const uint4 v = *(const uint4*)(st + row * PITCH + ch * 16);
    __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v),
                                (u32x4*)(dst + (ch >> 3) * (BM * BK) + row * BK + (ch & 7) * 8));
  }
}

// Copy a 256 x 256 tile of 16-bit values staged column by column (column c
// at c * PITCH bytes) to dst as 256 columns of 512 contiguous bytes (the
// tile column-major, 128 contiguous KiB): 32 lanes take one column, with
// non-temporal stores (the forward's y is read back only after the whole
// forward of the chunk).
template <int PITCH>
__device__ __forceinline__ void stage_copy_out_cm(const char* st, uint16_t* dst, int tid) {
#pragma unroll 4
  for (int it = 0; it < 16; ++it) {
    const int c = it * NT + tid, col = c >> 5, ch = c & 31;
    const uint4 v = *(const uint4*)(st + col * PITCH + ch * 16);
    __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v), (u32x4*)(dst + col * 256 + ch * 8));
  }
}

// Write four 16-bit values (rows r..r+3 of one column, packed in v) into the
// row-major staging tile.
__device__ __forceinline__ void stage_col4(char* q0, uint2 v) {
  *(uint16_t*)(q0) = (uint16_t)v.x;
  *(uint16_t*)(q0 + STG_PITCH) = (uint16_t)(v.x >> 16);
  *(uint16_t*)(q0 + 2 * STG_PITCH) = (uint16_t)v.y;
  *(uint16_t*)(q0 + 3 * STG_PITCH) = (uint16_t)(v.y >> 16);
}

// Two fp32 values to a packed fp16 pair (a in the low half), rounded to
// nearest even (one v_cvt_pk_f16_f32).
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pk_f16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, f16x2_t));
}

template <int EPI>
__global__ void __launch_bounds__(NT, 1) k_gemm(const Args g) {
  constexpr bool kStats = EPI == EPI_STATS || EPI == EPI_STATS_Y;
  __shared__ __attribute__((aligned(16))) char lds[LDS_TOTAL];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 1, wn = wid & 1;  // 4 x 2 waves, wave tile 64 x 128

  int M = g.M, K = g.K;
  if (g.cnt) {
    int64_t c = (int64_t)g.cnt[0] - g.cnt_off;
    c = c < 0 ? 0 : (c > g.cnt_cap ? g.cnt_cap : c);
    if (g.m_from_cnt) M = (int)c;
    if (g.k_from_cnt) K = (int)((c + BK - 1) / BK * BK);
  }
  const int N = g.N;
  const int NB = g.NB > 0 ? g.NB : N;
  if (EPI == EPI_STORE && g.k_from_cnt && K == 0 && g.accumulate) return;  // nothing to add
  if (EPI == EPI_STORE && g.sel == 2 && prefer384(M, N, g.ncu)) return;  // the 384-row kernel's
  const int nTm = (M + BM - 1) / BM, nTn = (N + BN - 1) / BN;
  // The grid is sized for the largest possible M; workgroups without a tile
  // for the device count exit at once.
  int mt, nt;
  if (!tile_of<kSG<EPI>>((int)blockIdx.x, nTm, nTn, mt, nt)) return;
  const int nk = (K + BK - 1) / BK;

  // per-lane load geometry (see load_stage): row w*64 + p*8 + (lane>>3)
  constexpr int NLOAD = kNLoad<EPI>;
  const bool loader = wid < NLOAD;
  LoadGeom lg;
  {
    const int ld_row = (wid % NLOAD) * (256 / NLOAD) + (lane >> 3);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int ch = (lane & 7) ^ (lane >> 4) ^ (q * 4);
      lg.kc[q] = ch * 8;
      lg.vA[q] = (uint32_t)(ld_row * (g.a_blk ? 64 : g.lda) * 2 + ch * 16);
      lg.vB[q] = (uint32_t)(ld_row * (g.b_blk ? 64 : g.ldb) * 2 + ch * 16);
    }
    lg.sA = (uint32_t)(8 * (g.a_blk ? 64 : g.lda) * 2);
    lg.sB = (uint32_t)(8 * (g.b_blk ? 64 : g.ldb) * 2);
    lg.kA = g.a_blk ? 512u : 2u;
    lg.kB = g.b_blk ? 512u : 2u;
  }
  // MFMA tiles: v_mfma_f32_16x16x32_bf16, 4 x 8 tiles of 16 x 16 per wave
  // (measured 3-4% faster than 4 x 2 tiles of 32x32x16 on the same main loop,
  // and the forward's row reductions stay inside one 16-lane DPP row).
  // Element q of tile (i, j) is row wm*64 + i*16 + q4*4 + q and column
  // wn*128 + j*16 + r16 of the workgroup tile.
  const int r16 = lane & 15, q4 = lane >> 4;

  int32_t* rp_i = (int32_t*)(lds + 2 * STAGE);
  float* rp_a = (float*)(lds + 2 * STAGE + BM * 4);
  float* rp_b = (float*)(lds + 2 * STAGE + BM * 8);
  float* rp_e = (float*)(lds + 2 * STAGE + BM * 12);
  float* rp_u = (float*)(lds + 2 * STAGE + BM * 16);

  {
    const int m0 = mt * BM, n0 = nt * BN;

    // buffer descriptors over the tile's valid rows: everything else reads 0
    // (a blocked operand interleaves the rows of its panel, so the descriptor
    // spans the whole panel and the panel's rows past the end hold zeros)
    const int rowsA = g.a_blk ? BM : min(BM, M - m0);
    const int rowsB = NB > n0 ? (g.b_blk ? BN : min(BN, NB - n0)) : 0;
    const int nb0 = rowsB > 0 ? n0 : 0;
    const __amdgpu_buffer_rsrc_t rA = make_rsrc(g.A + (int64_t)m0 * g.lda, rowsA * g.lda * 2);
    const __amdgpu_buffer_rsrc_t rB = make_rsrc(g.B + (int64_t)nb0 * g.ldb, rowsB * g.ldb * 2);

    // per-row epilogue parameters for this tile (threads 0..255, one row each)
    if (tid < BM) {
      int m = m0 + tid;
      bool v = m < M;
      if (kStats) {
        int y = -1;
        if (v) y = g.ids[g.rows[g.rows_off + m]];
        rp_i[tid] = y;
      } else if (EPI == EPI_DZ) {
        int y = -1;
        float L_ = 0.f, c_ = 0.f, e_ = 0.f, u_ = 0.f;
        if (v) {
          int t = g.rows[g.rows_off + m];
          y = g.ids[t];
          L_ = g.lse[t];
          c_ = g.cgrad[t];
          if (g.egrad) {
            e_ = g.egrad[t];
            u_ = L_ - g.ent[t];
          }
        }
        rp_i[tid] = y;
        rp_a[tid] = L_;
        rp_b[tid] = c_;
        rp_e[tid] = e_;
        rp_u[tid] = u_;
      } else {
        rp_i[tid] = (v && g.c_scatter) ? g.rows[g.rows_off + m] : m;
      }
    }

    floatx4 acc4[4][8];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc4[i][j] = (floatx4){0.f, 0.f, 0.f, 0.f};

    char* const ldsw = lds + (wid % NLOAD) * ((256 / NLOAD) * 128);
    if (nk > 0 && loader) load_stage<NLOAD>(rA, rB, ldsw, 0, K, lg);
    __syncthreads();  // first stage and the per-row parameters are visible to every wave
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + 1 < nk && loader)
        load_stage<NLOAD>(rA, rB, ldsw + ((kt + 1) & 1) * STAGE, (kt + 1) * BK, K, lg);
      const char* As = lds + (kt & 1) * STAGE;
      const char* Bs = As + A_BYTES;
      {
        // lane l holds row (l & 15) of a fragment and K-chunk ks * 4 + (l >> 4)
        // of the stage's eight 16-byte chunks
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          bf16x8 a[4], b[8];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int row = wm * 64 + i * 16 + r16;
            a[i] = *(const bf16x8*)(As + row * 128 + (((ks * 4 + q4) ^ ((row >> 1) & 7)) << 4));
          }
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int row = wn * 128 + j * 16 + r16;
            b[j] = *(const bf16x8*)(Bs + row * 128 + (((ks * 4 + q4) ^ ((row >> 1) & 7)) << 4));
          }
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 8; ++j)
              acc4[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc4[i][j], 0, 0, 0);
        }
      }
      // Before the barrier: this wave's loads of the next stage have landed
      // and its fragment reads of this stage are complete, so after the
      // barrier no wave still reads the buffer that the next loads overwrite.
      wait_vm();
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
      barrier_lds();
    }

    // ------------------------------------------------------------ epilogue
    if constexpr (kStats) {
      // A lane holds 16 rows (e = 4 i + q) of its 16-lane group, 8 columns
      // each; a row's 128 columns of this wave lie in the 16 lanes of one DPP row.
      float* xm = (float*)(lds + LDS_MAIN);            // partials of the wn = 1 half [256][3]
      float* xmax = (float*)(lds + LDS_MAIN + 3072);   // half maxima [2][256] (STATS_Y)
      const int colb16 = n0 + wn * 128 + r16;
      bool cv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) cv[j] = colb16 + j * 16 < N;
      // tiles wholly inside N (all but at most the last column of tiles) skip
      // the column masks; the exponent is the hardware exp2 (arguments <= 0,
      // results below 2^-126 flush to 0)
      const bool full = n0 + BN <= N;
      __builtin_amdgcn_sched_barrier(0);
      float mx[16], sm[16], um[16];
      if (full) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const floatx4* t = acc4[e >> 2];
          const int q = e & 3;
          mx[e] = fmaxf(fmaxf(fmaxf(t[0][q], t[1][q]), fmaxf(t[2][q], t[3][q])),
                        fmaxf(fmaxf(t[4][q], t[5][q]), fmaxf(t[6][q], t[7][q])));
        }
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          float v = -INFINITY;
#pragma unroll
          for (int j = 0; j < 8; ++j) v = cv[j] ? fmaxf(v, acc4[e >> 2][j][e & 3]) : v;
          mx[e] = v;
        }
      }
      row16_max_n(mx);
      // logit of the sampled token, picked with selects outside the store's
      // branch (a dynamic index there makes the compiler copy the tiles); a
      // row's token lies in a given 128-column half tile with probability
      // 128 / V, so the wave skips the picking unless one of its rows has it
      {
        int yl[16];
        bool here = false;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int rl = wm * 64 + (e >> 2) * 16 + q4 * 4 + (e & 3);
          yl[e] = rp_i[rl] - (n0 + wn * 128);
          here = here || (unsigned)yl[e] < 128u;
        }
        if (__builtin_amdgcn_ballot_w64(here)) {
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int rl = wm * 64 + (e >> 2) * 16 + q4 * 4 + (e & 3);
            const int jj = yl[e] >> 4;
            float z = acc4[e >> 2][0][e & 3];
#pragma unroll
            for (int j = 1; j < 8; ++j) z = jj == j ? acc4[e >> 2][j][e & 3] : z;
            if ((unsigned)yl[e] < 128u && (yl[e] & 15) == r16) g.zy[g.rows_off + m0 + rl] = z;
          }
        }
      }
      // lane r16 of group q4 owns row e = r16 of that group
      const int rl = wm * 64 + (r16 >> 2) * 16 + q4 * 4 + (r16 & 3);
      if (EPI == EPI_STATS_Y) {
        // y = z - (row maximum over the tile) <= 0, rounded to fp16, stored
        // before the exponent sums so that the stores drain while those run
        // (the sums and the merge below are the statistics-only forward's
        // arithmetic); rows past M and columns past N hold values the
        // backward never uses
        float hm = mx[0];
#pragma unroll
        for (int e = 1; e < 16; ++e) hm = r16 == e ? mx[e] : hm;
        xmax[wn * 256 + rl] = hm;
        __syncthreads();  // also: every row parameter read before the staging tile covers them
        uint2 hv[4][8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int rl0 = wm * 64 + i * 16 + q4 * 4;
          float mr[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) mr[q] = fmaxf(mx[i * 4 + q], xmax[(1 - wn) * 256 + rl0 + q]);
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            hv[i][j].x = pk_f16(acc4[i][j][0] - mr[0], acc4[i][j][1] - mr[1]);
            hv[i][j].y = pk_f16(acc4[i][j][2] - mr[2], acc4[i][j][3] - mr[3]);
          }
        }
        // staged column by column: a lane's four rows of a column in one
        // 8-byte write
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 8; ++j)
            *(uint2*)(lds + (wn * 128 + j * 16 + r16) * STG_PITCH_T + (wm * 64 + i * 16 + q4 * 4) * 2) =
                hv[i][j];
        __syncthreads();
        // y: the tile's 128 KiB of the tile-blocked [Tc, Vpad] buffer (panel
        // m0, from block n0 / 64), holding the tile column-major
        stage_copy_out_cm<STG_PITCH_T>(lds, g.y + (int64_t)m0 * g.ldy + (int64_t)n0 * BM, tid);
      }
      if (full) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          float s0 = 0.f, u0 = 0.f;
          const float mk = mx[e] * kLog2e;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float z = acc4[e >> 2][j][e & 3];
            const float p = __builtin_amdgcn_exp2f(fmaf(z, kLog2e, -mk));
            s0 += p;
            u0 = fmaf(p, z, u0);
          }
          sm[e] = s0;
          um[e] = u0;
        }
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          float s0 = 0.f, u0 = 0.f;
          const float mk = mx[e] == -INFINITY ? 0.f : mx[e] * kLog2e;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float z = acc4[e >> 2][j][e & 3];
            const float p = cv[j] ? __builtin_amdgcn_exp2f(fmaf(z, kLog2e, -mk)) : 0.f;
            s0 += p;
            u0 = cv[j] ? fmaf(p, z, u0) : u0;
          }
          sm[e] = s0;
          um[e] = u0;
        }
      }
      row16_sum_n(sm);
      row16_sum_n(um);
      float om = mx[0], os = sm[0], ou = um[0];
#pragma unroll
      for (int e = 1; e < 16; ++e) {
        const bool sel = r16 == e;
        om = sel ? mx[e] : om;
        os = sel ? sm[e] : os;
        ou = sel ? um[e] : ou;
      }
      if (wn == 1) {
        xm[rl * 3 + 0] = om;
        xm[rl * 3 + 1] = os;
        xm[rl * 3 + 2] = ou;
      }
      __syncthreads();
      if (wn == 0) {
        const int m = m0 + rl;
        if (m < M) {
          lse_merge(om, os, ou, xm[rl * 3 + 0], xm[rl * 3 + 1], xm[rl * 3 + 2]);
          const int64_t o = (int64_t)nt * g.ldp + g.p_off + m;
          g.pm[o] = om;
          g.ps[o] = os;
          g.pu[o] = ou;
        }
      }
    } else if (EPI == EPI_DZ) {
      // d = c (onehot - p) + e p (z - mu) in bf16, packed per lane as four
      // consecutive rows of one column
      uint2 hv[4][8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        __builtin_amdgcn_sched_barrier(0);
        const int rl0 = wm * 64 + i * 16 + q4 * 4;
        float Lr[4], cr[4], er[4], ur[4];
        int yr[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          yr[q] = rp_i[rl0 + q];
          Lr[q] = rp_a[rl0 + q] * kLog2e;
          cr[q] = rp_b[rl0 + q];
          er[q] = rp_e[rl0 + q];
          ur[q] = rp_u[rl0 + q];
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int col = n0 + wn * 128 + j * 16 + r16;
          const bool cvalid = col < g.Vvalid;
          uint32_t hb[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float z = acc4[i][j][q];
            const float p = __builtin_amdgcn_exp2f(fmaf(z, kLog2e, -Lr[q]));
            const float d = dlogit(cr[q], er[q], ur[q], p, z, col == yr[q]);
            hb[q] = f32_to_bf16(cvalid ? d : 0.f);
          }
          hv[i][j].x = hb[0] | (hb[1] << 16);
          hv[i][j].y = hb[2] | (hb[3] << 16);
        }
      }
      // Stage the tile through LDS and write it with 16-byte stores that
      // cover whole lines: a wave writes two 512-byte rows per instruction.
      char* const st = lds;
      __syncthreads();  // every wave is done with the stages and the row parameters
      // dZ [rows, Vpad]: element (row, col) at byte row * pitch + col * 2
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j)
          stage_col4(st + (wm * 64 + i * 16 + q4 * 4) * STG_PITCH + (wn * 128 + j * 16 + r16) * 2,
                     hv[i][j]);
      __syncthreads();
      // dZ and dZ^T are tile-blocked: the tile is four consecutive blocks of
      // each (dZ panel m0, blocks from column n0; dZ^T panel n0, blocks from m0)
      stage_copy_out_blk<STG_PITCH>(st, g.dz + (int64_t)m0 * g.ldz + (int64_t)n0 * BM, tid);
      if (g.dzt) {
        // dZ^T: tile column c (vocabulary) as a 512-byte row of the 256 chunk rows
        __syncthreads();  // the row-major copy has left the staging tile
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 8; ++j)
            *(uint2*)(st + (wn * 128 + j * 16 + r16) * STG_PITCH_T +
                      (wm * 64 + i * 16 + q4 * 4) * 2) = hv[i][j];
        __syncthreads();
        stage_copy_out_blk<STG_PITCH_T>(st, g.dzt + (int64_t)n0 * g.ldzt + (int64_t)m0 * BM, tid);
      }
    } else {  // EPI_STORE
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int rl = wm * 64 + i * 16 + q4 * 4 + q;
          const int m = m0 + rl;
          if (m >= M) continue;
          const int64_t dst = (int64_t)rp_i[rl] * g.ldc;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int col = n0 + wn * 128 + j * 16 + r16;
            if (col < N) {
              float v = acc4[i][j][q];
              if (g.accumulate) v += g.C[dst + col];
              g.C[dst + col] = v;
            }
          }
        }
      }
    }
  }
}


// The GEMM on a 384 x 256 workgroup tile for tile-blocked operands: the
// fp32 store of the step's dH and dW (EPI_STORE), the fused step's forward
// (EPI_STATS_Y) and the forward of rft_token_logprobs given the workspace for
// blocked operands (EPI_STATS).  Eight waves of 96 x 128 (6 x 8 tiles of 16x16x32, 192
// accumulator registers), two 80 KiB stages (all of the LDS), two loader
// waves.  17% fewer operand bytes and 22% fewer LDS fragment bytes per flop
// than the 256 x 256 tile; the per-element k order is the same, so the results
// are bit-identical to k_gemm's.  A 384-row tile starts at row 0 or 128 of a
// 256-row panel P0 of A and continues into P1 = P0 + 1; one descriptor covers
// both (adjacent in memory), P1 only if it holds rows < M (otherwise the tile's
// rows there load the same rows of P0, which reach only rows of C that are not
// stored).  K must be a multiple of 64 (or come from the counter): there is no
// per-lane K tail, and each load takes its lane part of the offset from one of
// two registers and its instruction's part as a scalar offset (the
// per-instruction offsets held in registers across the loop spilled).  The LDS
// layout, swizzle and fragment reads are those of k_gemm; rows 16 i + r16 of a
// wave's fragments share the swizzle (r16 >> 1) & 7.
constexpr int BM4 = 384;
constexpr int A_BYTES4 = BM4 * BK * 2;      // 48 KiB
constexpr int STAGE4 = A_BYTES4 + B_BYTES;  // 80 KiB
template <int EPI> constexpr int kSG4 = EPI == EPI_STORE ? 4 : 8;
template <int EPI> constexpr int kNLoad4 = 2;
// forward epilogue's LDS after the main loop: the y staging tile, the two
// column halves' row maxima [2][384], the wn = 1 half's partials [384][3] and
// the rows' token ids [384]
constexpr int X4_MAX = STG_BYTES, X4_PART = X4_MAX + 2 * BM4 * 4, X4_IDS = X4_PART + 3 * BM4 * 4;
static_assert(X4_IDS + BM4 * 4 <= 2 * STAGE4, "forward epilogue exceeds the LDS");

template <int EPI>
__global__ void __launch_bounds__(NT, 1) k_gemm384(const Args g) {
  static_assert(EPI == EPI_STORE || EPI == EPI_STATS || EPI == EPI_STATS_Y,
                "384-row tile: store or forward");
  constexpr bool kStats = EPI != EPI_STORE;
  __shared__ __attribute__((aligned(16))) char lds[2 * STAGE4];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 1, wn = wid & 1;  // 4 x 2 waves, wave tile 96 x 128
  int M = g.M, K = g.K;
  if (g.cnt) {
    int64_t c = (int64_t)g.cnt[0] - g.cnt_off;
    c = c < 0 ? 0 : (c > g.cnt_cap ? g.cnt_cap : c);
    if (g.m_from_cnt) M = (int)c;
    if (g.k_from_cnt) K = (int)((c + BK - 1) / BK * BK);
  }
  const int N = g.N;
  if (EPI == EPI_STORE && g.k_from_cnt && K == 0 && g.accumulate) return;  // nothing to add
  if (EPI == EPI_STORE && g.sel == 1 && !prefer384(M, N, g.ncu)) return;  // the 256-row kernel's
  const int nTm = (M + BM4 - 1) / BM4, nTn = (N + BN - 1) / BN;
  int mt, nt;
  if (!tile_of<kSG4<EPI>>((int)blockIdx.x, nTm, nTn, mt, nt)) return;
  const int nk = (K + BK - 1) / BK;
  constexpr int NLOAD = kNLoad4<EPI>;
  constexpr int RA = BM4 / NLOAD, RB = BN / NLOAD;  // rows of A and of B per loader wave
  static_assert(RA % 16 == 0 && RB % 16 == 0, "offset parity follows the row-pair swizzle");
  const bool loader = wid < NLOAD;
  const int lw = wid % NLOAD;
  const int m0 = mt * BM4, n0 = nt * BN;
  const int P0 = m0 >> 8, base0 = m0 & 255;
  const int64_t pa = (int64_t)256 * g.lda;  // elements per panel of A
  const bool p1ok = (P0 + 1) * 256 < M;
  const __amdgpu_buffer_rsrc_t rA = make_rsrc(g.A + P0 * pa, (p1ok ? 2 : 1) * pa * 2);
  const uint32_t pbytes = p1ok ? (uint32_t)(pa * 2) : 0u;
  const int64_t pb = (int64_t)256 * g.ldb;
  const __amdgpu_buffer_rsrc_t rB = make_rsrc(g.B + (int64_t)nt * pb, pb * 2);
  // forward: the sampled token of each row (threads 0..383, -1 past M), held
  // in a register through the main loop (the stages fill the LDS)
  int tok = -1;
  if (kStats && tid < BM4 && m0 + tid < M) tok = g.ids[g.rows[g.rows_off + m0 + tid]];
  // lane part of the offsets for even / odd instructions (see load_stage)
  uint32_t vq[2];
#pragma unroll
  for (int q = 0; q < 2; ++q)
    vq[q] = (uint32_t)((lane >> 3) * 128 + (((lane & 7) ^ (lane >> 4) ^ (q * 4)) << 4));
  auto load = [&](char* dst, int k0) {
    const uint32_t kofs = (uint32_t)k0 * 512u;  // a 64-column block is 32 KiB
#pragma unroll
    for (int p = 0; p < RA / 8; ++p) {  // A: rows lw * RA + 8 p ..
      const int R0 = lw * RA + 8 * p;
      const int pr = base0 + R0;  // row from the start of P0 (>= 256: in P1)
      const uint32_t so = __builtin_amdgcn_readfirstlane(
          kofs + (uint32_t)((pr & 255) * 128) + (uint32_t)(pr >> 8) * pbytes);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (lds_ptr)(dst + R0 * 128), 16, vq[p & 1], so,
                                               0, 0);
    }
#pragma unroll
    for (int p = 0; p < RB / 8; ++p) {  // B: rows lw * RB + 8 p ..
      const int R0 = lw * RB + 8 * p;
      const uint32_t so = __builtin_amdgcn_readfirstlane(kofs + (uint32_t)(R0 * 128));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rB, (lds_ptr)(dst + A_BYTES4 + R0 * 128), 16,
                                               vq[p & 1], so, 0, 0);
    }
  };
  const int r16 = lane & 15, q4 = lane >> 4;
  floatx4 acc4[6][8];
#pragma unroll
  for (int i = 0; i < 6; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc4[i][j] = (floatx4){0.f, 0.f, 0.f, 0.f};
  if (nk > 0 && loader) load(lds, 0);
  __syncthreads();  // first stage visible to every wave
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk && loader) load(lds + ((kt + 1) & 1) * STAGE4, (kt + 1) * BK);
    const char* As = lds + (kt & 1) * STAGE4;
    const char* Al = As + (wm * 96 + r16) * 128;
    const char* Bl = As + A_BYTES4 + (wn * 128 + r16) * 128;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int cho = ((ks * 4 + q4) ^ ((r16 >> 1) & 7)) << 4;
      bf16x8 a[6];
#pragma unroll
      for (int i = 0; i < 6; ++i) a[i] = *(const bf16x8*)(Al + i * 2048 + cho);
#pragma unroll
      for (int jh = 0; jh < 4; ++jh) {
        bf16x8 b[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) b[j] = *(const bf16x8*)(Bl + (jh * 2 + j) * 2048 + cho);
#pragma unroll
        for (int i = 0; i < 6; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc4[i][jh * 2 + j] =
                __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc4[i][jh * 2 + j], 0, 0, 0);
      }
    }
    // this wave's loads of the next stage have landed and its reads of this
    // stage are complete before the barrier
    wait_vm();
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    barrier_lds();
  }
  // element q of tile (i, j) is row wm*96 + i*16 + q4*4 + q and column
  // wn*128 + j*16 + r16 of the workgroup tile
  if constexpr (EPI == EPI_STORE) {
#pragma unroll
    for (int i = 0; i < 6; ++i) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int m = m0 + wm * 96 + i * 16 + q4 * 4 + q;
        if (m >= M) continue;
        const int64_t dst = (int64_t)(g.c_scatter ? g.rows[g.rows_off + m] : m) * g.ldc;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int col = n0 + wn * 128 + j * 16 + r16;
          if (col < N) {
            float v = acc4[i][j][q];
            if (g.accumulate) v += g.C[dst + col];
            g.C[dst + col] = v;
          }
        }
      }
    }
  } else {
    // Forward: k_gemm's EPI_STATS(_Y) arithmetic per row and 256-column tile
    // (the same maxima, exponent sums in the same order, the same merge of
    // the two column halves), on 24 rows per lane: row e (0..23) of lane
    // group q4 is tile row wm*96 + (e/4)*16 + q4*4 + e%4.  After the
    // reductions lane r16 owns rows e = r16 and, for r16 < 8, e = 16 + r16.
    // The last k-step's barrier has passed: the stages are free.
    float* const xmax = (float*)(lds + X4_MAX);
    float* const xm = (float*)(lds + X4_PART);
    int32_t* const rp_i = (int32_t*)(lds + X4_IDS);
    auto rl_of = [&](int e) { return wm * 96 + (e >> 2) * 16 + q4 * 4 + (e & 3); };
    if (tid < BM4) rp_i[tid] = tok;
    const int colb16 = n0 + wn * 128 + r16;
    bool cv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) cv[j] = colb16 + j * 16 < N;
    const bool full = n0 + BN <= N;
    __builtin_amdgcn_sched_barrier(0);
    float mx[24];
    if (full) {
#pragma unroll
      for (int e = 0; e < 24; ++e) {
        const floatx4* t = acc4[e >> 2];
        const int q = e & 3;
        mx[e] = fmaxf(fmaxf(fmaxf(t[0][q], t[1][q]), fmaxf(t[2][q], t[3][q])),
                      fmaxf(fmaxf(t[4][q], t[5][q]), fmaxf(t[6][q], t[7][q])));
      }
    } else {
#pragma unroll
      for (int e = 0; e < 24; ++e) {
        float v = -INFINITY;
#pragma unroll
        for (int j = 0; j < 8; ++j) v = cv[j] ? fmaxf(v, acc4[e >> 2][j][e & 3]) : v;
        mx[e] = v;
      }
    }
    row16_max_n(mx);
    {
      float h0 = mx[0], h1 = mx[16];
#pragma unroll
      for (int e = 1; e < 16; ++e) h0 = r16 == e ? mx[e] : h0;
#pragma unroll
      for (int e = 17; e < 24; ++e) h1 = r16 == e - 16 ? mx[e] : h1;
      xmax[wn * BM4 + rl_of(r16)] = h0;
      if (r16 < 8) xmax[wn * BM4 + rl_of(16 + r16)] = h1;
    }
    __syncthreads();  // token ids and half maxima visible
    // logit of the sampled token (as in k_gemm: selects, and only in waves
    // where one of the rows has its token in this half tile)
    {
      const int nw = n0 + wn * 128;
      bool here = false;
#pragma unroll
      for (int e = 0; e < 24; ++e) here |= (unsigned)(rp_i[rl_of(e)] - nw) < 128u;
      if (__builtin_amdgcn_ballot_w64(here)) {
        // branch-free stores: a lane whose column is not the row's token
        // stores past the end of a descriptor over the tile's 384 entries of
        // zy, which the hardware drops
        const __amdgpu_buffer_rsrc_t rZ = make_rsrc(g.zy + g.rows_off + m0, (int64_t)BM4 * 4);
#pragma unroll
        for (int e = 0; e < 24; ++e) {
          const int yl = rp_i[rl_of(e)] - nw;
          const int jj = yl >> 4;
          float z = acc4[e >> 2][0][e & 3];
#pragma unroll
          for (int j = 1; j < 8; ++j) z = jj == j ? acc4[e >> 2][j][e & 3] : z;
          const bool mine = (unsigned)yl < 128u && (yl & 15) == r16;
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(z), rZ,
                                                mine ? (uint32_t)rl_of(e) * 4u : 0x80000000u, 0, 0);
        }
      }
    }
    // y = z - (row maximum over the tile) in fp16, staged column by column and
    // copied out once per 256-row panel that the tile touches: panel P0 gets
    // tile rows [0, 256 - base0) at its rows [base0, 256), panel P1 (only if it
    // holds rows < M) tile rows [256 - base0, 384) at its rows [0, base0 + 128).
    // Each panel's 256 x 256 tile is column-major in the 128 KiB that the
    // tile-blocked [rows, Vpad] layout gives it; the two row halves of a panel
    // that two 384-row tiles share are disjoint 256-byte pieces of every column.
#pragma unroll
    for (int p = 0; p < (EPI == EPI_STATS_Y ? 2 : 0); ++p) {
      if (p == 1 && !p1ok) break;
      const int tlo = p == 0 ? 0 : 256 - base0;
      const int thi = p == 0 ? 256 - base0 : BM4;
#pragma unroll
      for (int i = 0; i < 6; ++i) {
        const int gr = wm * 96 + i * 16;  // a 16-row group lies in one panel
        if (gr < tlo || gr >= thi) continue;
        const int pr = (base0 + gr + q4 * 4) & 255;  // panel row of the lane's first row
        float mr[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) mr[q] = fmaxf(mx[i * 4 + q], xmax[(1 - wn) * BM4 + gr + q4 * 4 + q]);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          uint2 hv;
          hv.x = pk_f16(acc4[i][j][0] - mr[0], acc4[i][j][1] - mr[1]);
          hv.y = pk_f16(acc4[i][j][2] - mr[2], acc4[i][j][3] - mr[3]);
          *(uint2*)(lds + (wn * 128 + j * 16 + r16) * STG_PITCH_T + pr * 2) = hv;
        }
      }
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's staging writes done
      barrier_lds();
      const int plo = p == 0 ? base0 : 0;
      const int sh = (p == 0 ? 256 - base0 : base0 + 128) == 256 ? 5 : 4;  // log2 chunks per column
      uint16_t* const dst = g.y + (int64_t)(P0 + p) * 256 * g.ldy + (int64_t)n0 * 256 + plo;
      const char* const src = lds + plo * 2;
      for (int c = tid; c < (256 << sh); c += NT) {
        const int col = c >> sh, ch = c & ((1 << sh) - 1);
        const uint4 v = *(const uint4*)(src + col * STG_PITCH_T + ch * 16);
        __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v),
                                    (u32x4*)(dst + col * 256 + ch * 8));
      }
      // every staged value is read (its store issued) before the next panel's
      // staging overwrites it
      barrier_lds();
    }
    // exponent sums in two batches of 12 rows (registers), each reduced and
    // picked into the lane's own rows before the next
    float om0 = mx[0], os0 = 0.f, ou0 = 0.f, om1 = mx[16], os1 = 0.f, ou1 = 0.f;
#pragma unroll
    for (int e = 1; e < 16; ++e) om0 = r16 == e ? mx[e] : om0;
#pragma unroll
    for (int e = 17; e < 24; ++e) om1 = r16 == e - 16 ? mx[e] : om1;
#pragma unroll
    for (int bt = 0; bt < 2; ++bt) {
      float sm[12], um[12];
#pragma unroll
      for (int k = 0; k < 12; ++k) {
        const int e = bt * 12 + k;
        float s0 = 0.f, u0 = 0.f;
        if (full) {
          const float mk = mx[e] * kLog2e;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float z = acc4[e >> 2][j][e & 3];
            const float pe = __builtin_amdgcn_exp2f(fmaf(z, kLog2e, -mk));
            s0 += pe;
            u0 = fmaf(pe, z, u0);
          }
        } else {
          const float mk = mx[e] == -INFINITY ? 0.f : mx[e] * kLog2e;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float z = acc4[e >> 2][j][e & 3];
            const float pe = cv[j] ? __builtin_amdgcn_exp2f(fmaf(z, kLog2e, -mk)) : 0.f;
            s0 += pe;
            u0 = cv[j] ? fmaf(pe, z, u0) : u0;
          }
        }
        sm[k] = s0;
        um[k] = u0;
      }
      row16_sum_n(sm);
      row16_sum_n(um);
#pragma unroll
      for (int k = 0; k < 12; ++k) {
        const int e = bt * 12 + k;
        if (e < 16) {
          os0 = r16 == e ? sm[k] : os0;
          ou0 = r16 == e ? um[k] : ou0;
        } else {
          os1 = r16 == e - 16 ? sm[k] : os1;
          ou1 = r16 == e - 16 ? um[k] : ou1;
        }
      }
    }
    const int rl0 = rl_of(r16), rl1 = rl_of(16 + r16);  // rl1: lanes r16 < 8
    if (wn == 1) {
      xm[rl0 * 3 + 0] = om0;
      xm[rl0 * 3 + 1] = os0;
      xm[rl0 * 3 + 2] = ou0;
      if (r16 < 8) {
        xm[rl1 * 3 + 0] = om1;
        xm[rl1 * 3 + 1] = os1;
        xm[rl1 * 3 + 2] = ou1;
      }
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    barrier_lds();  // no wait for the y stores still in flight
    if (wn == 0) {
      if (m0 + rl0 < M) {
        lse_merge(om0, os0, ou0, xm[rl0 * 3 + 0], xm[rl0 * 3 + 1], xm[rl0 * 3 + 2]);
        const int64_t o = (int64_t)nt * g.ldp + g.p_off + m0 + rl0;
        g.pm[o] = om0;
        g.ps[o] = os0;
        g.pu[o] = ou0;
      }
      if (r16 < 8 && m0 + rl1 < M) {
        lse_merge(om1, os1, ou1, xm[rl1 * 3 + 0], xm[rl1 * 3 + 1], xm[rl1 * 3 + 2]);
        const int64_t o = (int64_t)nt * g.ldp + g.p_off + m0 + rl1;
        g.pm[o] = om1;
        g.ps[o] = os1;
        g.pu[o] = ou1;
      }
    }
  }
}

}  // namespace mf

// ------------------------------------------------------------ launchers ----
template <int EPI>
static unsigned grid_for(int64_t M_cap, int64_t N) {
  return (unsigned)mf::grid_tiles<mf::kSG<EPI>>((M_cap + mf::BM - 1) / mf::BM,
                                                (N + mf::BN - 1) / mf::BN);
}
template <int EPI>
static unsigned grid_for384(int64_t M_cap, int64_t N) {
  return (unsigned)mf::grid_tiles<mf::kSG4<EPI>>((M_cap + mf::BM4 - 1) / mf::BM4,
                                                 (N + mf::BN - 1) / mf::BN);
}
// RFT_GEMM_STORE_TILE: 256 or 384 fixes the tile of the fp32-store GEMM on
// tile-blocked operands, anything else (or unset) leaves it to prefer384.
static int store_tile_env() {
  const char* v = std::getenv("RFT_GEMM_STORE_TILE");
  if (!v) return 0;
  const int t = std::atoi(v);
  return t == 256 || t == 384 ? t : 0;
}

// Compute units of the current device (cached per device; host threads may
// call concurrently, so the cache entries are atomic).
static hipError_t cu_count(int* n) {
  static std::atomic<int> cache[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < 64) {
    const int c = cache[dev].load(std::memory_order_relaxed);
    if (c > 0) {
      *n = c;
      return hipSuccess;
    }
  }
  e = hipDeviceGetAttribute(n, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  if (*n < 1) *n = 1;
  if (dev >= 0 && dev < 64) cache[dev].store(*n, std::memory_order_relaxed);
  return hipSuccess;
}

// The 384-row tile takes tile-blocked operands whose two-panel descriptor and
// scalar offsets fit 32 bits and whose K needs no tail.
static bool fits384(int64_t lda, int64_t ldb, int64_t K, int k_from_cnt) {
  return lda < ((int64_t)1 << 21) && ldb < ((int64_t)1 << 22) && (k_from_cnt || K % mf::BK == 0);
}

// Forward of the policy head over the compacted hidden rows Hc [rows_off, rows_off + cap):
// online-LSE partials [ntiles][ldp] and the sampled-token logit zy.
hipError_t mfma_fwd_stats(const uint16_t* Hc, int64_t d, const uint16_t* W, int64_t V,
                          const int32_t* rows, const int32_t* ids, const int32_t* cnt,
                          int64_t rows_off, int64_t cap, float* pm, float* ps, float* pu,
                          int64_t ldp, float* zy, hipStream_t s) {
  mf::Args a = {};
  a.A = Hc + rows_off * d; a.lda = d;
  a.B = W; a.ldb = d;
  a.M = (int)cap; a.N = (int)V; a.K = (int)d;
  a.cnt = cnt; a.cnt_off = rows_off; a.cnt_cap = cap; a.m_from_cnt = 1;
  a.rows = rows; a.rows_off = rows_off; a.ids = ids;
  a.pm = pm; a.ps = ps; a.pu = pu; a.ldp = ldp; a.zy = zy; a.p_off = rows_off;
  mf::k_gemm<mf::EPI_STATS><<<grid_for<mf::EPI_STATS>(cap, V), mf::NT, 0, s>>>(a);
  return hipGetLastError();
}

// Whether the forward from tile-blocked copies takes this d.
bool mfma_fwd_blk_ok(int64_t d) { return d % mf::BK == 0 && fits384(d, d, d, 0); }

// The same forward from tile-blocked copies: Hb [round_up(cap, 256), Kp] of the
// compacted rows and Wb [Vpad, Kp] (Kp = d, a multiple of 64, below 2^21).
hipError_t mfma_fwd_stats_blk(const uint16_t* Hb, int64_t d, const uint16_t* Wb, int64_t V,
                              const int32_t* rows, const int32_t* ids, const int32_t* cnt,
                              int64_t cap, float* pm, float* ps, float* pu, int64_t ldp, float* zy,
                              hipStream_t s) {
  if (!fits384(d, d, d, 0)) return hipErrorInvalidValue;
  mf::Args a = {};
  a.A = Hb; a.lda = d; a.a_blk = 1;
  a.B = Wb; a.ldb = d; a.b_blk = 1;
  a.M = (int)cap; a.N = (int)V; a.K = (int)d;
  a.cnt = cnt; a.cnt_off = 0; a.cnt_cap = cap; a.m_from_cnt = 1;
  a.rows = rows; a.rows_off = 0; a.ids = ids;
  a.pm = pm; a.ps = ps; a.pu = pu; a.ldp = ldp; a.zy = zy; a.p_off = 0;
  mf::k_gemm384<mf::EPI_STATS><<<grid_for384<mf::EPI_STATS>(cap, V), mf::NT, 0, s>>>(a);
  return hipGetLastError();
}

// Forward of one chunk of compacted rows [c0, c0 + Tc) for the fused step:
// Hc and W tile-blocked with Kp = d rounded up to 64 (c0 and Tc multiples of
// 256); partials [ntiles][Tc] indexed by the chunk row, zy by the compacted
// row, and y = z - (row maximum over the tile) in fp16 into y [Tc, Vpad]:
// each 256 x 256 tile in the 128 KiB the tile-blocked layout gives it,
// column-major.
hipError_t mfma_fwd_stats_y(const uint16_t* Hc, int64_t d, const uint16_t* W, int64_t V,
                            int64_t Vpad, const int32_t* rows, const int32_t* ids,
                            const int32_t* cnt, int64_t c0, int64_t Tc, float* pm, float* ps,
                            float* pu, float* zy, uint16_t* y, hipStream_t s) {
  const int64_t Kp = (d + 63) / 64 * 64;
  mf::Args a = {};
  a.A = Hc + c0 * Kp; a.lda = Kp; a.a_blk = 1;
  a.B = W; a.ldb = Kp; a.b_blk = 1;
  a.M = (int)Tc; a.N = (int)V; a.K = (int)d;
  a.cnt = cnt; a.cnt_off = c0; a.cnt_cap = Tc; a.m_from_cnt = 1;
  a.rows = rows; a.rows_off = c0; a.ids = ids;
  a.pm = pm; a.ps = ps; a.pu = pu; a.ldp = Tc; a.zy = zy; a.p_off = 0;
  a.y = y; a.ldy = Vpad;
  if (fits384(Kp, Kp, d, 0)) {
    mf::k_gemm384<mf::EPI_STATS_Y><<<grid_for384<mf::EPI_STATS_Y>(Tc, V), mf::NT, 0, s>>>(a);
    return hipGetLastError();
  }
  mf::k_gemm<mf::EPI_STATS_Y><<<grid_for<mf::EPI_STATS_Y>(Tc, V), mf::NT, 0, s>>>(a);
  return hipGetLastError();
}

// Backward recompute of one chunk of compacted rows [c0, c0 + Tc): dZ (bf16)
// into dz [Tc, Vpad] and dZ^T into dzt [Vpad, ldzt], both tile-blocked
// (Tc a multiple of 256, ldzt = Tc).
hipError_t mfma_dz(const uint16_t* Hc, int64_t d, const uint16_t* W, int64_t V, int64_t Vpad,
                   const int32_t* rows, const int32_t* ids, const float* lse, const float* cgrad,
                   const float* egrad, const float* ent, const int32_t* cnt, int64_t c0,
                   int64_t Tc, uint16_t* dz, uint16_t* dzt, int64_t ldzt, hipStream_t s) {
  mf::Args a = {};
  a.A = Hc + c0 * d; a.lda = d;
  a.B = W; a.ldb = d;
  a.M = (int)Tc; a.N = (int)Vpad; a.K = (int)d;
  a.cnt = cnt; a.cnt_off = c0; a.cnt_cap = Tc; a.m_from_cnt = 1;
  a.rows = rows; a.rows_off = c0; a.ids = ids; a.lse = lse; a.cgrad = cgrad;
  a.egrad = egrad; a.ent = ent;
  a.dz = dz; a.ldz = Vpad; a.Vvalid = V;
  a.dzt = dzt; a.ldzt = ldzt;
  a.NB = (int)V;  // W has V rows; columns V..Vpad-1 of dZ are written as 0
  // dz rows are indexed by the chunk-local m (m0 + row)
  mf::k_gemm<mf::EPI_DZ><<<grid_for<mf::EPI_DZ>(Tc, Vpad), mf::NT, 0, s>>>(a);
  return hipGetLastError();
}

// C[M, N] (+)= A[M, K] . B[N, K]^T with fp32 output; optional row scatter of C
// through rows[rows_off + m]; M or K can come from the device counter.  A
// blocked operand (a_blk / b_blk) has ld = Kp and whole 256-row panels whose
// rows past M (N) and columns past K hold zeros.
hipError_t mfma_gemm_store(const uint16_t* A, int64_t lda, const uint16_t* B, int64_t ldb,
                           int64_t M, int64_t N, int64_t K, const int32_t* cnt, int64_t cnt_off,
                           int64_t cnt_cap, int m_from_cnt, int k_from_cnt, float* C, int64_t ldc,
                           const int32_t* rows, int64_t rows_off, int accumulate, hipStream_t s,
                           int a_blk, int b_blk) {
  mf::Args a = {};
  a.A = A; a.lda = lda; a.B = B; a.ldb = ldb;
  a.a_blk = a_blk; a.b_blk = b_blk;
  a.M = (int)M; a.N = (int)N; a.K = (int)K;
  a.cnt = cnt; a.cnt_off = cnt_off; a.cnt_cap = cnt_cap; a.m_from_cnt = m_from_cnt;
  a.k_from_cnt = k_from_cnt;
  a.C = C; a.ldc = ldc; a.rows = rows; a.rows_off = rows_off; a.c_scatter = rows != nullptr;
  a.accumulate = accumulate;
  // tile-blocked operands: the 384 x 256 tile where its one descriptor over
  // two panels of A and its scalar offsets fit 32 bits, K needs no tail and
  // it takes fewer rounds of tiles (prefer384).  With the rows on the device
  // both kernels are launched with the same test there: the other one's
  // workgroups return at once (a few microseconds).  RFT_GEMM_STORE_TILE=256
  // or 384 in the environment fixes the choice (the results are the same bit
  // for bit).
  const int force = store_tile_env();
  if (a_blk && b_blk && fits384(lda, ldb, K, k_from_cnt) && force != 256) {
    int ncu = 0;
    hipError_t e = cu_count(&ncu);
    if (e != hipSuccess) return e;
    if (force == 384) {
      mf::k_gemm384<mf::EPI_STORE><<<grid_for384<mf::EPI_STORE>(M, N), mf::NT, 0, s>>>(a);
      return hipGetLastError();
    }
    if (!m_from_cnt) {
      if (mf::prefer384(M, N, ncu)) {
        mf::k_gemm384<mf::EPI_STORE><<<grid_for384<mf::EPI_STORE>(M, N), mf::NT, 0, s>>>(a);
        return hipGetLastError();
      }
    } else {
      a.ncu = ncu;
      a.sel = 1;
      mf::k_gemm384<mf::EPI_STORE><<<grid_for384<mf::EPI_STORE>(M, N), mf::NT, 0, s>>>(a);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      a.sel = 2;
    }
  }
  mf::k_gemm<mf::EPI_STORE><<<grid_for<mf::EPI_STORE>(M, N), mf::NT, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace rft

// GEMM C = epi(A B^T) on MFMA for gfx950.
//
// Both operands are K-contiguous (nn.Linear layout), which is exactly the
// per-lane layout the MFMA operands want: every lane feeds a 16-byte run of
// consecutive k.  Workgroup tile 256 x 256, k-tile 128 bytes per row (64
// bf16 / 32 f32), 8 waves arranged 2 (M) x 4 (N), each owning a 128 x 64
// block = 4 x 2 MFMA 32x32 tiles.  Operand tiles are staged through LDS,
// double-buffered (2 x 64 KB of the 160 KB LDS), with the 16-byte chunks of
// each row XOR-swizzled by (row & 7) so both the row-contiguous stores and
// the 32-row fragment reads are bank-conflict free.  Ragged M and N are
// handled by clamping the load rows and predicating the stores; K must be a
// multiple of the k-tile (the plan pads pruned widths to 64).
#include "common.h"
#include "kernels.h"

namespace dif {

constexpr int G_BM = 256, G_BN = 256;
constexpr int G_THREADS = 512;
constexpr int G_CH = 8;  // 16-byte chunks per k-tile row (128 bytes)

template <typename T, typename OutT>
struct GemmParams {
  const T* A;
  const T* B;
  OutT* C;
  int64_t lda, ldb, ldc;
  int M, N, K;
  const float* bias;
  const float* gate0;
  const float* gate1;
};

template <typename T, typename OutT, int EPI>
__global__ __launch_bounds__(G_THREADS) void gemm_nt_kernel(GemmParams<T, OutT> p) {
  __shared__ u32x4 smem[2][G_BM + G_BN][G_CH];
  constexpr int VEC = Chunk<T>::VEC;
  constexpr int BK = G_CH * VEC;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int g = lane >> 5, col = lane & 31;

  // logical tile: XCD-contiguous ranges, then groups of GM row-tiles that
  // walk the N tiles together (operand reuse in L2)
  const int nbm = (p.M + G_BM - 1) / G_BM, nbn = (p.N + G_BN - 1) / G_BN;
  const int bid = xcd_remap(blockIdx.x, nbm * nbn);
  constexpr int GM = 8;
  const int group = bid / (GM * nbn);
  const int first_m = group * GM;
  const int gsize = min(nbm - first_m, GM);
  const int in_group = bid - group * GM * nbn;
  const int m0 = (first_m + in_group % gsize) * G_BM;
  const int n0 = (in_group / gsize) * G_BN;

  // global -> LDS staging: thread loads chunk lc of rows lr + 64 i
  const int lc = tid & 7, lr = tid >> 3;
  const T* a_src[4];
  const T* b_src[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ra = min(m0 + lr + 64 * i, p.M - 1);
    const int rb = min(n0 + lr + 64 * i, p.N - 1);
    a_src[i] = p.A + (int64_t)ra * p.lda + lc * VEC;
    b_src[i] = p.B + (int64_t)rb * p.ldb + lc * VEC;
  }
  u32x4 ra_reg[4], rb_reg[4];
  const int nk = p.K / BK;

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  if (nk > 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra_reg[i] = *reinterpret_cast<const u32x4*>(a_src[i]);
      rb_reg[i] = *reinterpret_cast<const u32x4*>(b_src[i]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = lr + 64 * i;
      smem[0][row][lc ^ (row & 7)] = ra_reg[i];
      smem[0][G_BM + row][lc ^ (row & 7)] = rb_reg[i];
    }
  }
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      const int64_t off = (int64_t)(kt + 1) * BK;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ra_reg[i] = *reinterpret_cast<const u32x4*>(a_src[i] + off);
        rb_reg[i] = *reinterpret_cast<const u32x4*>(b_src[i] + off);
      }
    }
#pragma unroll
    for (int ks = 0; ks < G_CH / 2; ++ks) {
      const int c = (2 * ks + g) ^ (col & 7);
      u32x4 af[4], bfr[2];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = smem[buf][wm * 128 + i * 32 + col][c];
#pragma unroll
      for (int j = 0; j < 2; ++j) bfr[j] = smem[buf][G_BM + wn * 64 + j * 32 + col][c];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) Mma<T>::step(acc[i][j], af[i], bfr[j]);
    }
    if (more) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = lr + 64 * i;
        smem[buf ^ 1][row][lc ^ (row & 7)] = ra_reg[i];
        smem[buf ^ 1][G_BM + row][lc ^ (row & 7)] = rb_reg[i];
      }
    }
    __syncthreads();
  }

  // epilogue: lane holds column n of each tile, 16 rows
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = n0 + wn * 64 + j * 32 + col;
    if (n >= p.N) continue;
    const float bias = p.bias ? p.bias[n] : 0.f;
    float gate = 1.f;
    if (EPI == EPI_RESIDUAL && p.gate0) gate = p.gate0[n] + (p.gate1 ? p.gate1[n] : 0.f);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * 128 + i * 32 + acc_row(r, g);
        if (m < p.M) {
          OutT* dst = p.C + (int64_t)m * p.ldc + n;
          const float v = acc[i][j][r] + bias;
          if (EPI == EPI_STORE) {
            *dst = from_f32<OutT>(v);
          } else if (EPI == EPI_GELU) {
            *dst = from_f32<OutT>(gelu_tanh(v));
          } else {
            *dst = from_f32<OutT>(to_f32(*dst) + gate * v);
          }
        }
      }
    }
  }
}

template <typename T, typename OutT>
hipError_t launch_gemm(const T* A, int64_t lda, const T* B, int64_t ldb, OutT* C, int64_t ldc,
                       int M, int N, int K, int epi, const float* bias, const float* gate0,
                       const float* gate1, hipStream_t stream) {
  if (M <= 0 || N <= 0) return hipSuccess;
  GemmParams<T, OutT> p{A, B, C, lda, ldb, ldc, M, N, K, bias, gate0, gate1};
  const int tiles = ((M + G_BM - 1) / G_BM) * ((N + G_BN - 1) / G_BN);
  dim3 grid(tiles), block(G_THREADS);
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((gemm_nt_kernel<T, OutT, EPI_STORE>), grid, block, 0, stream, p); break;
    case EPI_GELU: hipLaunchKernelGGL((gemm_nt_kernel<T, OutT, EPI_GELU>), grid, block, 0, stream, p); break;
    default: hipLaunchKernelGGL((gemm_nt_kernel<T, OutT, EPI_RESIDUAL>), grid, block, 0, stream, p); break;
  }
  return hipGetLastError();
}

template hipError_t launch_gemm<bf16, bf16>(const bf16*, int64_t, const bf16*, int64_t, bf16*, int64_t,
                                            int, int, int, int, const float*, const float*,
                                            const float*, hipStream_t);
template hipError_t launch_gemm<bf16, float>(const bf16*, int64_t, const bf16*, int64_t, float*, int64_t,
                                             int, int, int, int, const float*, const float*,
                                             const float*, hipStream_t);
template hipError_t launch_gemm<float, float>(const float*, int64_t, const float*, int64_t, float*,
                                              int64_t, int, int, int, int, const float*,
                                              const float*, const float*, hipStream_t);

}  // namespace dif

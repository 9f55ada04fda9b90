// HBM-bound row kernels for gfx950: LayerNorm + AdaLN modulation,
// QK RMSNorm + 3D RoPE, V transpose, plan-time gather, timestep GEMV and
// small elementwise steps.  Rows are read once with 16-byte vector loads,
// kept in registers between the statistics and the apply pass, and written
// once; statistics are fp32 whatever the storage type.
#include <algorithm>

#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace dif {

constexpr int R_THREADS = 256;
constexpr int R_WAVES = R_THREADS / kWave;
constexpr int R_MAXC = 16;   // 16-byte chunks per lane per row (D <= 1024 * VEC)
constexpr int R_RPW = 8;     // rows per wave
constexpr int R_ROWS = R_WAVES * R_RPW;

// ---------------------------------------------------------------------------
// LayerNorm (biased variance, eps) + AdaLN modulation or affine.
// The workgroup first folds the per-column vectors into LDS (shift and
// 1 + scale, or weight and bias); each wave then normalises R_RPW rows, one
// row at a time: one statistics pass (sum and sum of squares of the row
// shifted by its first element) with the row kept packed in registers, then
// the apply pass.  Reductions are wave-local.
// ---------------------------------------------------------------------------
// The row kernels that stage per-column vectors in LDS run 16 waves per
// workgroup, so the staging is shared by 128 rows (measured: 4.6 TB/s vs 3.3
// TB/s with 4 waves on [32760, 5120] bf16).
constexpr int NORM_WAVES = 16;
constexpr int NORM_RPW = 8;

// 16-byte chunks each lane holds for a row of D elements, rounded up to one
// of the instantiated register budgets (4, 8, 12, 16); 0 if D is too wide.
template <typename T>
inline int chunks_per_lane(int D) {
  const int c = (D / Chunk<T>::VEC + kWave - 1) / kWave;
  return c <= 4 ? 4 : c <= 8 ? 8 : c <= 12 ? 12 : c <= R_MAXC ? R_MAXC : 0;
}
template <typename T, int MAXC>
__global__ __launch_bounds__(64 * NORM_WAVES) void norm_kernel(const T* __restrict__ x, T* __restrict__ y,
                                                         int M, int D, int mode, const float* p0,
                                                         const float* p1, const float* p2,
                                                         const float* p3, float eps) {
  constexpr int VEC = Chunk<T>::VEC;
  extern __shared__ float vec_lds[];  // [2][D]: multiplier, addend
  float* mul = vec_lds;
  float* add = vec_lds + D;
  for (int n = threadIdx.x; n < D; n += 64 * NORM_WAVES) {
    if (mode == 0) {
      mul[n] = 1.f + p2[n] + (p3 ? p3[n] : 0.f);
      add[n] = p0[n] + (p1 ? p1[n] : 0.f);
    } else {
      mul[n] = p0[n];
      add[n] = p1[n];
    }
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int nch = D / VEC;
  const float inv_d = 1.f / (float)D;
  for (int rr = 0; rr < NORM_RPW; ++rr) {
    const int64_t row = (int64_t)blockIdx.x * (NORM_WAVES * NORM_RPW) + (threadIdx.x >> 6) * NORM_RPW + rr;
    if (row >= M) break;
    const T* xr = x + row * D;
    u32x4 raw[MAXC];
    // one pass over shifted data: sum and sum of squares of (x - x0), where
    // x0 is the row's first element, keep the variance free of cancellation
    const float x0 = to_f32(xr[0]);
    float s = 0.f, ss = 0.f;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int c = lane + kWave * i;
      if (c < nch) {
        raw[i] = *reinterpret_cast<const u32x4*>(xr + c * VEC);
        float v[VEC];
        Chunk<T>::unpack(raw[i], v);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const float d = v[e] - x0;
          s += d;
          ss += d * d;
        }
      }
    }
    const float ms = wave_sum(s) * inv_d;
    const float mean = x0 + ms;
    const float var = fmaxf(wave_sum(ss) * inv_d - ms * ms, 0.f);
    const float rstd = rsqrtf(var + eps);
    T* yr = y + row * D;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int c = lane + kWave * i;
      if (c < nch) {
        float v[VEC], out[VEC];
        Chunk<T>::unpack(raw[i], v);
        const f32x4* m4 = reinterpret_cast<const f32x4*>(mul + c * VEC);
        const f32x4* a4 = reinterpret_cast<const f32x4*>(add + c * VEC);
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q) {
          const f32x4 mu = m4[q], ad = a4[q];
#pragma unroll
          for (int e = 0; e < 4; ++e) out[4 * q + e] = (v[4 * q + e] - mean) * rstd * mu[e] + ad[e];
        }
        *reinterpret_cast<u32x4*>(yr + c * VEC) = Chunk<T>::pack(out);
      }
      __builtin_amdgcn_sched_barrier(0);  // bound the LDS reads kept in flight
    }
  }
}

template <typename T>
hipError_t launch_norm(const T* x, T* y, int M, int D, int mode, const float* p0, const float* p1,
                       const float* p2, const float* p3, float eps, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  const dim3 grid((M + NORM_WAVES * NORM_RPW - 1) / (NORM_WAVES * NORM_RPW));
  const size_t lds = 2 * D * sizeof(float);
  switch (chunks_per_lane<T>(D)) {
    case 4: hipLaunchKernelGGL((norm_kernel<T, 4>), grid, dim3(64 * NORM_WAVES), lds, stream, x, y, M,
                               D, mode, p0, p1, p2, p3, eps); break;
    case 8: hipLaunchKernelGGL((norm_kernel<T, 8>), grid, dim3(64 * NORM_WAVES), lds, stream, x, y, M,
                               D, mode, p0, p1, p2, p3, eps); break;
    case 12: hipLaunchKernelGGL((norm_kernel<T, 12>), grid, dim3(64 * NORM_WAVES), lds, stream, x, y,
                                M, D, mode, p0, p1, p2, p3, eps); break;
    case 16: hipLaunchKernelGGL((norm_kernel<T, 16>), grid, dim3(64 * NORM_WAVES), lds, stream, x, y,
                                M, D, mode, p0, p1, p2, p3, eps); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// QK RMSNorm over the full model width (pruned channels count as zeros, so
// the sum of squares of the kept channels is divided by D) + 3D RoPE.
// Gains are staged in LDS once per workgroup.  Lane l always covers the
// same head-local pairs (64 * VEC is a multiple of head_dim), so its
// rotation factors are fetched once per row.  A wave issues the loads of
// both segments (q and k) of its row before the first reduction waits on
// them, with the rotation-table reads in their shadow.
// ---------------------------------------------------------------------------
constexpr int QK_WAVES = 8;    // 16 KB of loads in flight per wave; registers for both segments
// Rows per wave.  One segment: 4, so 32760 video tokens make 1024 workgroups,
// several per CU, with more rows' loads in flight (5.3 TB/s; 16 rows per
// wave, one workgroup per CU, reached 4.2).  Two segments (q and k, twice the
// loads per row): 16 (5.4-5.5 TB/s against 5.3 with 4).
template <int NSEG>
constexpr int qk_rpw() { return NSEG == 2 ? 16 : 4; }
template <typename T, int MAXC, int NSEG>
__global__ __launch_bounds__(64 * QK_WAVES) void qk_norm_kernel(T* buf, int64_t ld, int rows, int a,
                                                            int nseg, int off0, int off1,
                                                            const float* g0, const float* g1,
                                                            const int32_t* gidx, float scale0,
                                                            float inv_dim, float eps, RopeDesc rope) {
  constexpr int VEC = Chunk<T>::VEC;
  constexpr int NP = VEC / 2;  // pairs per chunk
  extern __shared__ float gain_lds[];  // [nseg][a]
  for (int n = threadIdx.x; n < a; n += 64 * QK_WAVES) {
    const int gn = gidx ? gidx[n] : n;
    gain_lds[n] = g0[gn] * scale0;
    if (nseg > 1) gain_lds[a + n] = g1[gn];
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int nch = a / VEC;
  const int jb = ((lane * VEC) % rope.head_dim) / 2;  // first head-local pair of this lane
  constexpr int RPW = qk_rpw<NSEG>();
  for (int rr = 0; rr < RPW; ++rr) {
    const int64_t row = (int64_t)blockIdx.x * (QK_WAVES * RPW) + (threadIdx.x >> 6) * RPW + rr;
    if (row >= rows) break;
    // both segments' loads go out before anything waits on them
    u32x4 raw[NSEG][MAXC];
#pragma unroll
    for (int sg = 0; sg < NSEG; ++sg) {
      const T* xr = buf + row * ld + (sg == 0 ? off0 : off1);
#pragma unroll
      for (int i = 0; i < MAXC; ++i) {
        const int c = lane + kWave * i;
        if (c < nch) raw[sg][i] = *reinterpret_cast<const u32x4*>(xr + c * VEC);
      }
    }
    // rotation factors of this lane's pairs (table reads overlap the loads)
    float cs[NP], sn[NP];
    if (rope.table) {
      const int n = (int)(row % rope.L);
      const int pw = n % rope.gw, pr = (n / rope.gw) % rope.gh, pf = n / (rope.gw * rope.gh);
#pragma unroll
      for (int k = 0; k < NP; ++k) {
        const int j = jb + k;
        int idx;
        if (j < rope.jt) {
          idx = pf * rope.jt + j;
        } else if (j < rope.jt + rope.jh) {
          idx = rope.gf * rope.jt + pr * rope.jh + (j - rope.jt);
        } else {
          idx = rope.gf * rope.jt + rope.gh * rope.jh + pw * rope.jw + (j - rope.jt - rope.jh);
        }
        cs[k] = rope.table[2 * idx];
        sn[k] = rope.table[2 * idx + 1];
      }
    }
    float rstd[NSEG];
#pragma unroll
    for (int sg = 0; sg < NSEG; ++sg) {
      float ss = 0.f;
#pragma unroll
      for (int i = 0; i < MAXC; ++i) {
        const int c = lane + kWave * i;
        if (c < nch) {
          float v[VEC];
          Chunk<T>::unpack(raw[sg][i], v);
#pragma unroll
          for (int e = 0; e < VEC; ++e) ss += v[e] * v[e];
        }
      }
      rstd[sg] = rsqrtf(wave_sum(ss) * inv_dim + eps);
    }
#pragma unroll
    for (int sg = 0; sg < NSEG; ++sg) {
      T* xr = buf + row * ld + (sg == 0 ? off0 : off1);
      const float* gain = gain_lds + sg * a;
#pragma unroll
      for (int i = 0; i < MAXC; ++i) {
        const int c = lane + kWave * i;
        if (c < nch) {
          float out[VEC];
          Chunk<T>::unpack(raw[sg][i], out);
          const f32x4* g4 = reinterpret_cast<const f32x4*>(gain + c * VEC);
#pragma unroll
          for (int q = 0; q < VEC / 4; ++q) {
            const f32x4 gg = g4[q];
#pragma unroll
            for (int e = 0; e < 4; ++e) out[4 * q + e] *= rstd[sg] * gg[e];
          }
          if (rope.table) {
#pragma unroll
            for (int k = 0; k < NP; ++k) {
              const float x0 = out[2 * k], x1 = out[2 * k + 1];
              out[2 * k] = x0 * cs[k] - x1 * sn[k];
              out[2 * k + 1] = x0 * sn[k] + x1 * cs[k];
            }
          }
          *reinterpret_cast<u32x4*>(xr + c * VEC) = Chunk<T>::pack(out);
        }
      }
    }
  }
}

template <typename T>
hipError_t launch_qk_norm(T* buf, int64_t ld, int rows, int a, int nseg, int off0, int off1,
                          const float* g0, const float* g1, float inv_norm_dim, float eps,
                          const RopeDesc* rope, hipStream_t stream, const int32_t* gain_idx,
                          float scale0) {
  if (rows <= 0 || a <= 0) return hipSuccess;
  RopeDesc rd{};
  if (rope) rd = *rope;
  if (rd.head_dim <= 0) rd.head_dim = 64;   // no rotation: any width dividing 64 * VEC
  constexpr int VEC = Chunk<T>::VEC;
  if ((64 * VEC) % rd.head_dim != 0) return hipErrorInvalidValue;
  // q and k in one launch while both fit the registers (up to 8 chunks per
  // lane), else one launch per segment
  auto launch = [&](auto c_tag, auto nseg_tag, int off_a, int off_b, const float* ga,
                    const float* gb, float sa) {
    constexpr int C = decltype(c_tag)::value, NS = decltype(nseg_tag)::value;
    constexpr int rows_per_wg = QK_WAVES * qk_rpw<NS>();
    const dim3 grid((rows + rows_per_wg - 1) / rows_per_wg);
    hipLaunchKernelGGL((qk_norm_kernel<T, C, NS>), grid, dim3(64 * QK_WAVES), NS * a * sizeof(float),
                       stream, buf, ld, rows, a, NS, off_a, off_b, ga, gb, gain_idx, sa,
                       inv_norm_dim, eps, rd);
  };
  auto by_chunks = [&](auto c_tag) {
    constexpr int C = decltype(c_tag)::value;
    using One = std::integral_constant<int, 1>;
    using Two = std::integral_constant<int, 2>;
    if (nseg == 1) {
      launch(c_tag, One{}, off0, 0, g0, nullptr, scale0);
      return;
    }
    if constexpr (C <= 8) {
      launch(c_tag, Two{}, off0, off1, g0, g1, scale0);
    } else {
      launch(c_tag, One{}, off0, 0, g0, nullptr, scale0);
      launch(c_tag, One{}, off1, 0, g1, nullptr, 1.f);
    }
  };
  switch (chunks_per_lane<T>(a)) {
    case 4: by_chunks(std::integral_constant<int, 4>{}); break;
    case 8: by_chunks(std::integral_constant<int, 8>{}); break;
    case 12: by_chunks(std::integral_constant<int, 12>{}); break;
    case 16: by_chunks(std::integral_constant<int, 16>{}); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// V -> V^T per sample, 64 x 64 tiles through LDS, zero-filled key padding
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(R_THREADS) void transpose_vt_kernel(const T* __restrict__ src,
                                                                 int64_t lds, int a, int Lk,
                                                                 T* __restrict__ vt, int64_t ldvt) {
  __shared__ float tile[64][65];
  const int j0 = blockIdx.x * 64, c0 = blockIdx.y * 64, b = blockIdx.z;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int jj = ty; jj < 64; jj += R_WAVES) {
    const int j = j0 + jj, c = c0 + tx;
    float v = 0.f;
    if (j < Lk && c < a) v = to_f32(src[((int64_t)b * Lk + j) * lds + c]);
    tile[jj][tx] = v;
  }
  __syncthreads();
  for (int cc = ty; cc < 64; cc += R_WAVES) {
    const int c = c0 + cc, j = j0 + tx;
    if (c < a && j < ldvt) vt[((int64_t)b * a + c) * ldvt + j] = from_f32<T>(tile[tx][cc]);
  }
}

// bf16: a lane moves an 8-token x 8-channel block: eight 16-byte loads of
// token rows, a register transpose (v_perm_b32 pairs 16-bit halves of two
// token rows; the rest is register renaming) and eight 16-byte stores of
// channel rows.  Lanes (cx, ty) of a wave: 8 lanes read 128 contiguous
// bytes of a token row and 8 lanes write 128 contiguous bytes of a V^T row.
// Tokens past Lk are written as zeros up to ldvt (a multiple of 8).
__global__ __launch_bounds__(R_THREADS) void transpose_vt8_kernel(const bf16* __restrict__ src,
                                                                  int64_t lds, int a, int Lk,
                                                                  bf16* __restrict__ vt,
                                                                  int64_t ldvt) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int cx = lane & 7, ty = lane >> 3;
  const int c0 = blockIdx.y * 64 + cx * 8;                        // first channel
  const int64_t t0 = ((int64_t)blockIdx.x * R_WAVES + wave) * 64 + ty * 8;   // first token
  const int b = blockIdx.z;
  if (t0 >= ldvt || c0 >= a) return;
  uint32_t in[8][4];
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (t0 + r < Lk) v = *reinterpret_cast<const u32x4*>(src + ((int64_t)b * Lk + t0 + r) * lds + c0);
#pragma unroll
    for (int d = 0; d < 4; ++d) in[r][d] = v[d];
  }
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int d = c >> 1;
    const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;    // high or low halves
    u32x4 o;
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] = __builtin_amdgcn_perm(in[2 * k + 1][d], in[2 * k][d], sel);
    *reinterpret_cast<u32x4*>(vt + ((int64_t)b * a + c0 + c) * ldvt + t0) = o;
  }
}

template <typename T>
hipError_t launch_transpose_vt(const T* src, int64_t lds, int a, int B, int Lk, T* Vt,
                               int64_t ldvt, hipStream_t stream) {
  if (a <= 0 || B <= 0) return hipSuccess;
  if constexpr (sizeof(T) == 2) {
    if (a % 64 == 0 && ldvt % 8 == 0 && lds % 8 == 0 &&
        reinterpret_cast<uintptr_t>(src) % 16 == 0 && reinterpret_cast<uintptr_t>(Vt) % 16 == 0) {
      dim3 grid((unsigned)((ldvt + 64 * R_WAVES - 1) / (64 * R_WAVES)), (unsigned)(a / 64), (unsigned)B);
      hipLaunchKernelGGL(transpose_vt8_kernel, grid, dim3(R_THREADS), 0, stream, src, lds, a, Lk, Vt,
                         ldvt);
      return hipGetLastError();
    }
  }
  dim3 grid((unsigned)((ldvt + 63) / 64), (unsigned)((a + 63) / 64), (unsigned)B);
  hipLaunchKernelGGL((transpose_vt_kernel<T>), grid, dim3(R_THREADS), 0, stream, src, lds, a, Lk,
                     Vt, ldvt);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// plan-time gather of kept rows / columns
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(R_THREADS) void gather_kernel(const T* __restrict__ src, int64_t lds,
                                                           T* __restrict__ dst, int64_t ldd,
                                                           int cols, const int32_t* ridx,
                                                           const int32_t* cidx) {
  const int64_t r = blockIdx.x;
  const int sr = ridx ? ridx[r] : (int)r;
  for (int c = threadIdx.x; c < cols; c += R_THREADS) {
    const int sc = cidx ? cidx[c] : c;
    T v = from_f32<T>(0.f);
    if (sr >= 0 && sc >= 0) v = src[(int64_t)sr * lds + sc];
    dst[r * ldd + c] = v;
  }
}

template <typename T>
hipError_t launch_gather(const T* src, int64_t lds, T* dst, int64_t ldd, int rows, int cols,
                         const int32_t* ridx, const int32_t* cidx, hipStream_t stream) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  hipLaunchKernelGGL((gather_kernel<T>), dim3(rows), dim3(R_THREADS), 0, stream, src, lds, dst, ldd,
                     cols, ridx, cidx);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Kept heads of the cached text projections, 16 bytes per lane.  A kept head
// is head_dim consecutive channels starting at a multiple of head_dim, so
// every aligned group of V = 16 / sizeof(T) table entries is one contiguous,
// aligned 16-byte vector of the source.
//   cols: dst[r, j] = src[r, idx[j]]              (r < rows, j < cols)
//   rows: dst[b, r, :] = src[b, idx[r], :]        (r < rows, n per row)
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(R_THREADS) void gather_cols16_kernel(const T* __restrict__ src,
                                                                  int64_t lds, T* __restrict__ dst,
                                                                  int64_t ldd, int64_t total, int nvec,
                                                                  const int32_t* __restrict__ idx) {
  constexpr int V = 16 / sizeof(T);
  const int64_t i = (int64_t)blockIdx.x * R_THREADS + threadIdx.x;
  if (i >= total) return;
  const int64_t r = i / nvec;
  const int q = (int)(i - r * nvec);
  const int sc = idx[q * V];
  *reinterpret_cast<u32x4*>(dst + r * ldd + (int64_t)q * V) =
      *reinterpret_cast<const u32x4*>(src + r * lds + sc);
}

template <typename T>
__global__ __launch_bounds__(R_THREADS) void gather_rows16_kernel(const T* __restrict__ src,
                                                                  int64_t src_bs, T* __restrict__ dst,
                                                                  int64_t dst_bs, int64_t ld, int rows,
                                                                  const int32_t* __restrict__ idx) {
  constexpr int V = 16 / sizeof(T);
  const int64_t nvec = ld / V;
  const int64_t i = (int64_t)blockIdx.x * R_THREADS + threadIdx.x;
  if (i >= (int64_t)rows * nvec) return;
  const int64_t r = i / nvec, q = i - r * nvec;
  const int64_t b = blockIdx.y;
  *reinterpret_cast<u32x4*>(dst + b * dst_bs + r * ld + q * V) =
      *reinterpret_cast<const u32x4*>(src + b * src_bs + (int64_t)idx[r] * ld + q * V);
}

template <typename T>
hipError_t launch_gather_cols16(const T* src, int64_t lds, T* dst, int64_t ldd, int rows, int cols,
                                const int32_t* idx, hipStream_t stream) {
  constexpr int V = 16 / sizeof(T);
  if (rows <= 0 || cols <= 0) return hipSuccess;
  if (cols % V || lds % V || ldd % V || reinterpret_cast<uintptr_t>(src) % 16 ||
      reinterpret_cast<uintptr_t>(dst) % 16)
    return hipErrorInvalidValue;
  const int64_t total = (int64_t)rows * (cols / V);
  hipLaunchKernelGGL((gather_cols16_kernel<T>), dim3((unsigned)((total + R_THREADS - 1) / R_THREADS)),
                     dim3(R_THREADS), 0, stream, src, lds, dst, ldd, total, cols / V, idx);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_gather_rows16(const T* src, int64_t src_bs, T* dst, int64_t dst_bs, int64_t ld,
                                int rows, int batches, const int32_t* idx, hipStream_t stream) {
  constexpr int V = 16 / sizeof(T);
  if (rows <= 0 || batches <= 0 || ld <= 0) return hipSuccess;
  if (ld % V || src_bs % V || dst_bs % V || reinterpret_cast<uintptr_t>(src) % 16 ||
      reinterpret_cast<uintptr_t>(dst) % 16)
    return hipErrorInvalidValue;
  const int64_t total = (int64_t)rows * (ld / V);
  hipLaunchKernelGGL((gather_rows16_kernel<T>),
                     dim3((unsigned)((total + R_THREADS - 1) / R_THREADS), (unsigned)batches),
                     dim3(R_THREADS), 0, stream, src, src_bs, dst, dst_bs, ld, rows, idx);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// FFN channel norms: sqrt(|W1[j, :]|^2 + b1[j]^2 + |W2[:, j]|^2), in double
// (one-time preprocessing; a thread per channel, W2 reads coalesced over j)
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(R_THREADS) void ffn_norms_kernel(const T* __restrict__ w1,
                                                              const float* __restrict__ b1,
                                                              const T* __restrict__ w2, int D, int F,
                                                              double* __restrict__ out) {
  const int j = blockIdx.x * R_THREADS + threadIdx.x;
  if (j >= F) return;
  double acc = (double)b1[j] * (double)b1[j];
  for (int d = 0; d < D; ++d) {
    const double v = (double)to_f32(w1[(int64_t)j * D + d]);
    const double u = (double)to_f32(w2[(int64_t)d * F + j]);
    acc += v * v + u * u;
  }
  out[j] = sqrt(acc);
}

template <typename T>
hipError_t launch_ffn_norms(const T* w1, const float* b1, const T* w2, int D, int F, double* out,
                            hipStream_t stream) {
  if (F <= 0) return hipSuccess;
  hipLaunchKernelGGL((ffn_norms_kernel<T>), dim3((F + R_THREADS - 1) / R_THREADS), dim3(R_THREADS), 0,
                     stream, w1, b1, w2, D, F, out);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// timestep embedding pieces
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(R_THREADS) void gemv_kernel(const T* __restrict__ W,
                                                         const float* __restrict__ x,
                                                         const float* __restrict__ bias,
                                                         float* __restrict__ out, int N, int K) {
  constexpr int VEC = Chunk<T>::VEC;
  const int n = blockIdx.x * R_WAVES + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (n >= N) return;
  const T* wr = W + (int64_t)n * K;
  float acc = 0.f;
  for (int k = lane * VEC; k < K; k += kWave * VEC) {
    float w[VEC];
    Chunk<T>::unpack(*reinterpret_cast<const u32x4*>(wr + k), w);
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc += w[e] * x[k + e];
  }
  acc = wave_sum(acc);
  if (lane == 0) out[n] = acc + (bias ? bias[n] : 0.f);
}

template <typename T>
hipError_t launch_gemv(const T* W, const float* x, const float* bias, float* out, int N, int K,
                       hipStream_t stream) {
  if (N <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemv_kernel<T>), dim3((N + R_WAVES - 1) / R_WAVES), dim3(R_THREADS), 0, stream,
                     W, x, bias, out, N, K);
  return hipGetLastError();
}

// [cos(t w_j), sin(t w_j)], w_j = 10000^(-j/half), in double precision:
// t w_j reaches ~1e3 rad, where a float argument already loses 1e-4.
__global__ void sinusoid_kernel(float t, int half, float* out) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= half) return;
  const double arg = (double)t * pow(10000.0, -(double)j / (double)half);
  out[j] = (float)cos(arg);
  out[half + j] = (float)sin(arg);
}

hipError_t launch_sinusoid(float t, int dim, float* out, hipStream_t stream) {
  const int half = dim / 2;
  hipLaunchKernelGGL(sinusoid_kernel, dim3((half + 255) / 256), dim3(256), 0, stream, t, half, out);
  return hipGetLastError();
}

__global__ void silu_kernel(const float* x, float* y, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] = x[i] / (1.f + expf(-x[i]));
}

hipError_t launch_silu(const float* x, float* y, int n, hipStream_t stream) {
  hipLaunchKernelGGL(silu_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, x, y, n);
  return hipGetLastError();
}

__global__ void euler_kernel(float* z, const float* v, float dsig, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    z[i] = fmaf(dsig, v[i], z[i]);
}

hipError_t launch_euler(float* z, const float* v, float dsig, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 65536);
  hipLaunchKernelGGL(euler_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, z, v, dsig, n);
  return hipGetLastError();
}

// z = (1 - st) * (z - sf * v) + st * eps   (eps unused when st == 0)
__global__ void renoise_kernel(float* z, const float* v, float sf, float st, const float* eps,
                               int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const float x = fmaf(-sf, v[i], z[i]);
    z[i] = eps ? fmaf(st, eps[i], (1.f - st) * x) : x;
  }
}

hipError_t launch_renoise(float* z, const float* v, float sigma_from, float sigma_to,
                          const float* eps, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 65536);
  hipLaunchKernelGGL(renoise_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, z, v, sigma_from,
                     sigma_to, eps, n);
  return hipGetLastError();
}

template <typename T>
__global__ void cast_kernel(const float* src, T* dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = from_f32<T>(src[i]);
}

template <typename T>
hipError_t launch_cast(const float* src, T* dst, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 65536);
  hipLaunchKernelGGL((cast_kernel<T>), dim3((unsigned)blocks), dim3(256), 0, stream, src, dst, n);
  return hipGetLastError();
}

#define INST(T)                                                                                \
  template hipError_t launch_norm<T>(const T*, T*, int, int, int, const float*, const float*,  \
                                     const float*, const float*, float, hipStream_t);          \
  template hipError_t launch_qk_norm<T>(T*, int64_t, int, int, int, int, int, const float*,    \
                                        const float*, float, float, const RopeDesc*,           \
                                        hipStream_t, const int32_t*, float);                   \
  template hipError_t launch_transpose_vt<T>(const T*, int64_t, int, int, int, T*, int64_t,    \
                                             hipStream_t);                                     \
  template hipError_t launch_gather<T>(const T*, int64_t, T*, int64_t, int, int,               \
                                       const int32_t*, const int32_t*, hipStream_t);           \
  template hipError_t launch_gather_cols16<T>(const T*, int64_t, T*, int64_t, int, int,        \
                                              const int32_t*, hipStream_t);                    \
  template hipError_t launch_gather_rows16<T>(const T*, int64_t, T*, int64_t, int64_t, int, int,\
                                              const int32_t*, hipStream_t);                    \
  template hipError_t launch_gemv<T>(const T*, const float*, const float*, float*, int, int,   \
                                     hipStream_t);                                             \
  template hipError_t launch_cast<T>(const float*, T*, int64_t, hipStream_t);                  \
  template hipError_t launch_ffn_norms<T>(const T*, const float*, const T*, int, int, double*,  \
                                          hipStream_t);
INST(float)
INST(bf16)
#undef INST

}  // namespace dif

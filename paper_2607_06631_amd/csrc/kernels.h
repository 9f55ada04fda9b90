// Host-side launchers of the gfx950 kernels (internal to libdif).
// Every launcher enqueues on `stream` and returns hipGetLastError().
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dif {

typedef __bf16 bf16;

enum Epi { EPI_STORE = 0, EPI_GELU = 1, EPI_RESIDUAL = 2 };

// Optional index-table gather of the B operand from a union weight matrix.
//   rows:    B row of each of the N output columns (-1: zero row, zero bias);
//            b_rows = rows of the union matrix.  Epilogues STORE and GELU.
//   kchunks: for each 16-byte chunk c of the K extent, the chunk of every B
//            row it is read from (-1: zeros); at most 8192 chunks.  Epilogue
//            RESIDUAL.  A operand columns are compacted as K.
//   nseg > 1: B (and bias) of segments 1.. come from seg_b / seg_bias; the
//            segments share A and the row table, segment s writes C columns
//            [s*N, (s+1)*N).  Epilogues STORE and GELU.
struct GemmGather {
  const int32_t* rows;
  const int32_t* kchunks;
  int b_rows;
  int nseg = 1;
  const void* seg_b[2] = {nullptr, nullptr};
  const float* seg_bias[2] = {nullptr, nullptr};
};

// Transposed output for the columns of a store-epilogue GEMM from output
// column col0 on (col0 on a 256-column tile boundary, or the first column of
// a segment): column col0 + d of row m = b * L + j goes to
// vt[(b * dims + d) * ldvt + j].  Used to write V^T straight from the QKV
// projection.
struct GemmVt {
  void* vt;
  int64_t ldvt;
  int col0, dims, L;
};

// C[M,N] = epi(A[M,K] * B[N,K]^T); T in {float, __bf16}; OutT in {T, float}.
template <typename T, typename OutT>
hipError_t launch_gemm(const T* A, int64_t lda, const T* B, int64_t ldb, OutT* C, int64_t ldc,
                       int M, int N, int K, int epi, const float* bias, const float* gate0,
                       const float* gate1, hipStream_t stream, const GemmGather* gather = nullptr,
                       const GemmVt* vt = nullptr);

// Flash attention; V given transposed (see dif_attention in dif.h).
// q_scaled: Q already multiplied by log2(e)/sqrt(head_dim).  With a scratch
// region split_part of attention_split_bytes(head_dim) bytes and the device's
// CU count, a final round of workgroups that would run at most half full is
// split along the keys and merged by a second launch.
template <typename T>
hipError_t launch_attention(int head_dim, const T* Q, int64_t ldq, const T* K, int64_t ldk,
                            const T* Vt, int64_t ldvt, T* O, int64_t ldo, int B, int Lq, int Lk,
                            int H, hipStream_t stream, bool q_scaled = false,
                            float* split_part = nullptr, int ncu = 0);
size_t attention_split_bytes(int head_dim);
// The library's static split workspace on the current device (resolved once
// per device): its device address and size.
hipError_t attention_static_scratch(float** ptr, size_t* bytes);
constexpr int kAttnLongKeys = 4096;   // from this key count on, bf16 attention runs 8 waves

// Row LayerNorm of x [M, D] then
//   mode 0: y = xhat * (1 + p2 + p3) + (p0 + p1)      (AdaLN; p1/p3 may be null)
//   mode 1: y = xhat * p0 + p1                          (affine)
template <typename T>
hipError_t launch_norm(const T* x, T* y, int M, int D, int mode, const float* p0,
                       const float* p1, const float* p2, const float* p3, float eps,
                       hipStream_t stream);

// In place on rows of buf (stride ld): for each of nseg segments of width a
// at column offset off[s]: y = x / sqrt(sum(x^2) * inv_norm_dim + eps) * gain[s][idx[c]]
// (idx null: identity), times scale0 on segment 0,
// then (rope != null) rotate consecutive pairs of each head_dim-wide head by
// the token's 3D angles.
struct RopeDesc {
  const float* table;  // float2 (cos, sin) entries, see rope_table_size
  int L;               // tokens per sample (row % L = token)
  int gf, gh, gw;      // token grid
  int jt, jh, jw;      // pairs per axis
  int head_dim;
};
template <typename T>
hipError_t launch_qk_norm(T* buf, int64_t ld, int rows, int a, int nseg, int off0, int off1,
                          const float* g0, const float* g1, float inv_norm_dim, float eps,
                          const RopeDesc* rope, hipStream_t stream,
                          const int32_t* gain_idx = nullptr, float scale0 = 1.f);

// Vt[(b*a + c)*ldvt + j] = src[(b*Lk + j)*lds + c] for j < Lk, 0 for Lk <= j < ldvt.
template <typename T>
hipError_t launch_transpose_vt(const T* src, int64_t lds, int a, int B, int Lk, T* Vt,
                               int64_t ldvt, hipStream_t stream);

// dst[r][c] = src[ridx[r]][cidx[c]] (identity when an index table is null,
// zero when an index is negative).
template <typename T>
hipError_t launch_gather(const T* src, int64_t lds, T* dst, int64_t ldd, int rows, int cols,
                         const int32_t* ridx, const int32_t* cidx, hipStream_t stream);

// 16-byte gathers of whole kept heads (idx groups of 16 / sizeof(T) entries
// are aligned runs of consecutive channels):
//   cols: dst[r][j] = src[r][idx[j]]                      r < rows, j < cols
//   rows: dst[b*dst_bs + r*ld + :] = src[b*src_bs + idx[r]*ld + :]   r < rows, b < batches
// hipErrorInvalidValue when a width / stride is not a whole number of vectors
// or a base pointer is not 16-byte aligned.
template <typename T>
hipError_t launch_gather_cols16(const T* src, int64_t lds, T* dst, int64_t ldd, int rows, int cols,
                                const int32_t* idx, hipStream_t stream);
template <typename T>
hipError_t launch_gather_rows16(const T* src, int64_t src_bs, T* dst, int64_t dst_bs, int64_t ld,
                                int rows, int batches, const int32_t* idx, hipStream_t stream);

// out[n] = act_out(sum_k W[n,k] * x[k] + bias[n]); W [N, K] row-major.
template <typename T>
hipError_t launch_gemv(const T* W, const float* x, const float* bias, float* out, int N, int K,
                       hipStream_t stream);

hipError_t launch_sinusoid(float t, int dim, float* out, hipStream_t stream);
// Sustained-MFMA-rate probe (shape 0: 32x32x16, 1: 16x16x32 bf16): 2
// workgroups per CU; *flops = FLOPs of the launch.
hipError_t launch_mfma_probe(int shape, int iters, float* sink, int ncu, hipStream_t stream,
                             double* flops);
hipError_t launch_silu(const float* x, float* y, int n, hipStream_t stream);
hipError_t launch_euler(float* z, const float* v, float dsig, int64_t n, hipStream_t stream);

// out[j] = sqrt(|W1[j, :]|^2 + b1[j]^2 + |W2[:, j]|^2) (double), W1 [F, D], W2 [D, F].
template <typename T>
hipError_t launch_ffn_norms(const T* w1, const float* b1, const T* w2, int D, int F, double* out,
                            hipStream_t stream);
// z = (1 - sigma_to) (z - sigma_from v) + sigma_to eps; eps null means sigma_to = 0.
hipError_t launch_renoise(float* z, const float* v, float sigma_from, float sigma_to,
                          const float* eps, int64_t n, hipStream_t stream);
template <typename T>
hipError_t launch_cast(const float* src, T* dst, int64_t n, hipStream_t stream);

}  // namespace dif

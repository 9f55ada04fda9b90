// Host stand-ins for the HIP runtime calls and kernel launchers that libdif's
// host runtime (csrc/api.cpp) makes, so that the runtime's validation, plan
// layout, workspace carving and error paths run on the CPU under
// AddressSanitizer and UndefinedBehaviorSanitizer.
//
// "Device" memory is host memory here.  Every launcher stand-in computes
// nothing; it reads the first and last element of each operand region the
// real kernel reads, writes those of each region it writes, and checks every
// index table entry against the matrix it indexes, so that a carving or
// table mistake in the host runtime becomes an out-of-bounds access that the
// sanitizer reports.  Test infrastructure only.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "../../paper_2607_06631_amd/csrc/kernels.h"

extern "C" long g_stub_launches = 0;   // kernel launches seen (read by the harness)

namespace {

volatile unsigned char g_sink;

void rd(const void* p, size_t bytes) {
  if (bytes == 0) return;
  if (!p) {
    std::fprintf(stderr, "stub: read of %zu bytes through a null pointer\n", bytes);
    std::abort();
  }
  const unsigned char* c = static_cast<const unsigned char*>(p);
  g_sink = c[0];
  g_sink = c[bytes - 1];
}

void wr(void* p, size_t bytes) {
  if (bytes == 0) return;
  if (!p) {
    std::fprintf(stderr, "stub: write of %zu bytes through a null pointer\n", bytes);
    std::abort();
  }
  unsigned char* c = static_cast<unsigned char*>(p);
  c[0] = c[0];
  c[bytes - 1] = c[bytes - 1];
}

void check(bool ok, const char* what) {
  if (!ok) {
    std::fprintf(stderr, "stub: %s\n", what);
    std::abort();
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// HIP runtime
// ---------------------------------------------------------------------------
struct StubEvent {
  int recorded;
};

hipError_t hipGetDevice(int* id) {
  *id = 0;
  return hipSuccess;
}

hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t attr, int) {
  *v = attr == hipDeviceAttributeMultiprocessorCount ? 256 : 0;
  return hipSuccess;
}

hipError_t hipGetDevicePropertiesR0600(hipDeviceProp_tR0600* prop, int) {
  std::memset(prop, 0, sizeof(*prop));
  std::strcpy(prop->gcnArchName, "gfx950:sramecc+:xnack-");
  prop->multiProcessorCount = 256;
  return hipSuccess;
}

const char* hipGetErrorString(hipError_t e) { return e == hipSuccess ? "no error" : "stub error"; }

hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind, hipStream_t) {
  rd(src, n);
  wr(dst, n);
  std::memcpy(dst, src, n);
  return hipSuccess;
}

hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }

// The library keeps its timing events for the life of the process, so the
// stand-ins come from static storage rather than the heap.
StubEvent g_events[1 << 16];
int g_nevents = 0;

hipError_t hipEventCreate(hipEvent_t* e) {
  if (g_nevents == (int)(sizeof(g_events) / sizeof(g_events[0]))) return hipErrorOutOfMemory;
  StubEvent* ev = &g_events[g_nevents++];
  ev->recorded = 0;
  *e = reinterpret_cast<hipEvent_t>(ev);
  return hipSuccess;
}

hipError_t hipEventRecord(hipEvent_t e, hipStream_t) {
  reinterpret_cast<StubEvent*>(e)->recorded = 1;
  return hipSuccess;
}

hipError_t hipEventSynchronize(hipEvent_t e) {
  return reinterpret_cast<StubEvent*>(e)->recorded ? hipSuccess : hipErrorInvalidValue;
}

hipError_t hipEventElapsedTime(float* ms, hipEvent_t a, hipEvent_t b) {
  check(reinterpret_cast<StubEvent*>(a)->recorded && reinterpret_cast<StubEvent*>(b)->recorded,
        "elapsed time of an unrecorded event");
  *ms = 0.25f;
  return hipSuccess;
}

// ---------------------------------------------------------------------------
// kernel launchers
// ---------------------------------------------------------------------------
namespace dif {

template <typename T, typename OutT>
hipError_t launch_gemm(const T* A, int64_t lda, const T* B, int64_t ldb, OutT* C, int64_t ldc,
                       int M, int N, int K, int epi, const float* bias, const float* gate0,
                       const float* gate1, hipStream_t, const GemmGather* gather,
                       const GemmVt* vt) {
  ++g_stub_launches;
  if (M <= 0 || N <= 0) return hipSuccess;
  // (a K-chunk table reads chunks of the union rows: ldb bounds the table's
  // entries, not the compacted reduction extent K)
  const bool kch = gather && gather->kchunks;
  if (!(lda >= K && (kch || ldb >= K) && ldc >= N)) {
    std::fprintf(stderr, "stub: gemm M=%d N=%d K=%d lda=%lld ldb=%lld ldc=%lld\n", M, N, K,
                 (long long)lda, (long long)ldb, (long long)ldc);
    check(false, "gemm: leading dimension below the extent");
  }
  const int nseg = gather ? gather->nseg : 1;
  if (K > 0) rd(A, ((size_t)(M - 1) * lda + K) * sizeof(T));
  const T* bs[3] = {B, gather ? (const T*)gather->seg_b[0] : nullptr,
                    gather ? (const T*)gather->seg_b[1] : nullptr};
  const float* biases[3] = {bias, gather ? gather->seg_bias[0] : nullptr,
                            gather ? gather->seg_bias[1] : nullptr};
  constexpr int VEC = 16 / sizeof(T);
  for (int s = 0; s < nseg; ++s) {
    if (gather && gather->rows) {
      for (int n = 0; n < N; ++n) {
        const int r = gather->rows[n];
        check(r >= -1 && r < gather->b_rows, "gemm: row table entry out of range");
        if (r >= 0 && K > 0) rd(bs[s] + (size_t)r * ldb, (size_t)K * sizeof(T));
        if (r >= 0 && biases[s]) rd(biases[s] + r, sizeof(float));
      }
    } else if (gather && gather->kchunks) {
      for (int c = 0; c < K / VEC; ++c) {
        const int u = gather->kchunks[c];
        check(u >= -1 && (int64_t)u * VEC + VEC <= ldb, "gemm: K-chunk table entry out of range");
        if (u >= 0) rd(bs[s] + (size_t)(N - 1) * ldb + (size_t)u * VEC, 16);
      }
      if (biases[s]) rd(biases[s], (size_t)N * sizeof(float));
    } else {
      if (K > 0) rd(bs[s], ((size_t)(N - 1) * ldb + K) * sizeof(T));
      if (biases[s]) rd(biases[s], (size_t)N * sizeof(float));
    }
  }
  if (epi == EPI_RESIDUAL) {
    if (gate0) rd(gate0, (size_t)N * sizeof(float));
    if (gate1) rd(gate1, (size_t)N * sizeof(float));
  }
  int ccols = nseg * N;
  if (vt) {
    check(vt->col0 >= 0 && vt->col0 + vt->dims <= nseg * N && M % vt->L == 0,
          "gemm: transposed output outside the columns");
    ccols = vt->col0;
    const size_t batches = (size_t)M / vt->L;
    wr(vt->vt, ((batches * vt->dims - 1) * vt->ldvt + vt->L) * sizeof(OutT));
  }
  if (ccols > 0) {
    check(ccols <= ldc, "gemm: output columns beyond ldc");
    if (epi == EPI_RESIDUAL) rd(C, ((size_t)(M - 1) * ldc + ccols) * sizeof(OutT));
    wr(C, ((size_t)(M - 1) * ldc + ccols) * sizeof(OutT));
  }
  return hipSuccess;
}

template <typename T>
hipError_t launch_attention(int dh, const T* Q, int64_t ldq, const T* K, int64_t ldk, const T* Vt,
                            int64_t ldvt, T* O, int64_t ldo, int B, int Lq, int Lk, int H,
                            hipStream_t, bool, float* split_part, int) {
  ++g_stub_launches;
  if (B <= 0 || Lq <= 0 || H <= 0) return hipSuccess;
  const size_t w = (size_t)H * dh;
  rd(Q, ((size_t)(B * (size_t)Lq - 1) * ldq + w) * sizeof(T));
  rd(K, ((size_t)(B * (size_t)Lk - 1) * ldk + w) * sizeof(T));
  rd(Vt, (((size_t)B * H * dh - 1) * ldvt + Lk) * sizeof(T));
  wr(O, ((size_t)(B * (size_t)Lq - 1) * ldo + w) * sizeof(T));
  if (split_part) wr(split_part, attention_split_bytes(dh));
  return hipSuccess;
}

size_t attention_split_bytes(int head_dim) {
  return (size_t)2 * 128 * 256 * (head_dim + 2) * sizeof(float);
}

hipError_t attention_static_scratch(float** ptr, size_t* bytes) {
  alignas(256) static float buf[2 * 128 * 256 * 130];
  *ptr = buf;
  *bytes = sizeof(buf);
  return hipSuccess;
}

template <typename T>
hipError_t launch_norm(const T* x, T* y, int M, int D, int mode, const float* p0, const float* p1,
                       const float* p2, const float* p3, float, hipStream_t) {
  ++g_stub_launches;
  rd(x, (size_t)M * D * sizeof(T));
  wr(y, (size_t)M * D * sizeof(T));
  rd(p0, D * sizeof(float));
  if (p1) rd(p1, D * sizeof(float));
  if (mode == 0 && p2) rd(p2, D * sizeof(float));
  if (mode == 0 && p3) rd(p3, D * sizeof(float));
  return hipSuccess;
}

template <typename T>
hipError_t launch_qk_norm(T* buf, int64_t ld, int rows, int a, int nseg, int off0, int off1,
                          const float* g0, const float* g1, float, float, const RopeDesc* rope,
                          hipStream_t, const int32_t* gain_idx, float) {
  ++g_stub_launches;
  const int off = nseg > 1 ? (off0 > off1 ? off0 : off1) : off0;
  rd(buf, ((size_t)(rows - 1) * ld + off + a) * sizeof(T));
  wr(buf, ((size_t)(rows - 1) * ld + off + a) * sizeof(T));
  const float* g[2] = {g0, g1};
  for (int s = 0; s < nseg; ++s) {
    if (gain_idx) {
      for (int c = 0; c < a; ++c) {
        check(gain_idx[c] >= 0, "qk_norm: negative gain index");
        rd(g[s] + gain_idx[c], sizeof(float));
      }
    } else {
      rd(g[s], (size_t)a * sizeof(float));
    }
  }
  if (rope) {
    const size_t n = (size_t)rope->gf * rope->jt + (size_t)rope->gh * rope->jh + (size_t)rope->gw * rope->jw;
    rd(rope->table, n * 2 * sizeof(float));
    check(rope->jt + rope->jh + rope->jw == rope->head_dim / 2, "qk_norm: RoPE pairs != head_dim / 2");
  }
  return hipSuccess;
}

template <typename T>
hipError_t launch_transpose_vt(const T* src, int64_t lds, int a, int B, int Lk, T* Vt, int64_t ldvt,
                               hipStream_t) {
  ++g_stub_launches;
  rd(src, (((size_t)B * Lk - 1) * lds + a) * sizeof(T));
  wr(Vt, ((size_t)B * a * ldvt) * sizeof(T));
  return hipSuccess;
}

template <typename T>
hipError_t launch_gather(const T* src, int64_t lds, T* dst, int64_t ldd, int rows, int cols,
                         const int32_t* ridx, const int32_t* cidx, hipStream_t) {
  ++g_stub_launches;
  if (rows <= 0 || cols <= 0) return hipSuccess;
  wr(dst, ((size_t)(rows - 1) * ldd + cols) * sizeof(T));
  for (int r = 0; r < rows; ++r) {
    const int sr = ridx ? ridx[r] : r;
    if (sr < 0) continue;
    for (int c = 0; c < cols; ++c) {
      const int sc = cidx ? cidx[c] : c;
      if (sc < 0) continue;
      check(sc < lds || lds == 1, "gather: column index beyond the source row");
      rd(src + (size_t)sr * lds + sc, sizeof(T));
    }
  }
  return hipSuccess;
}

template <typename T>
hipError_t launch_gather_cols16(const T* src, int64_t lds, T* dst, int64_t ldd, int rows, int cols,
                                const int32_t* idx, hipStream_t) {
  ++g_stub_launches;
  wr(dst, ((size_t)(rows - 1) * ldd + cols) * sizeof(T));
  for (int j = 0; j < cols; ++j) {
    check(idx[j] >= 0 && idx[j] < lds, "gather_cols16: index beyond the row");
    rd(src + (size_t)(rows - 1) * lds + idx[j], sizeof(T));
  }
  return hipSuccess;
}

template <typename T>
hipError_t launch_gather_rows16(const T* src, int64_t src_bs, T* dst, int64_t dst_bs, int64_t ld,
                                int rows, int batches, const int32_t* idx, hipStream_t) {
  ++g_stub_launches;
  for (int b = 0; b < batches; ++b) {
    wr(dst + (size_t)b * dst_bs, (size_t)rows * ld * sizeof(T));
    for (int r = 0; r < rows; ++r) {
      check(idx[r] >= 0, "gather_rows16: negative index");
      rd(src + (size_t)b * src_bs + (size_t)idx[r] * ld, (size_t)ld * sizeof(T));
    }
  }
  return hipSuccess;
}

template <typename T>
hipError_t launch_gemv(const T* W, const float* x, const float* bias, float* out, int N, int K,
                       hipStream_t) {
  ++g_stub_launches;
  rd(W, (size_t)N * K * sizeof(T));
  rd(x, (size_t)K * sizeof(float));
  rd(bias, (size_t)N * sizeof(float));
  wr(out, (size_t)N * sizeof(float));
  return hipSuccess;
}

hipError_t launch_sinusoid(float, int dim, float* out, hipStream_t) {
  ++g_stub_launches;
  wr(out, (size_t)dim * sizeof(float));
  return hipSuccess;
}

hipError_t launch_mfma_probe(int shape, int iters, float* sink, int ncu, hipStream_t, double* flops) {
  ++g_stub_launches;
  check(shape >= 0 && shape <= 2 && iters >= 1 && ncu >= 1, "mfma_probe: bad launch");
  wr(sink, sizeof(float));
  *flops = 2.0 * ncu * 4 * (4.0 * ((iters + 3) / 4)) * 8 * (2.0 * 32 * 32 * 16);
  return hipSuccess;
}

hipError_t launch_silu(const float* x, float* y, int n, hipStream_t) {
  ++g_stub_launches;
  rd(x, (size_t)n * sizeof(float));
  wr(y, (size_t)n * sizeof(float));
  return hipSuccess;
}

hipError_t launch_euler(float* z, const float* v, float, int64_t n, hipStream_t) {
  ++g_stub_launches;
  rd(v, (size_t)n * sizeof(float));
  wr(z, (size_t)n * sizeof(float));
  return hipSuccess;
}

template <typename T>
hipError_t launch_ffn_norms(const T* w1, const float* b1, const T* w2, int D, int F, double* out,
                            hipStream_t) {
  ++g_stub_launches;
  rd(w1, (size_t)F * D * sizeof(T));
  rd(b1, (size_t)F * sizeof(float));
  rd(w2, (size_t)D * F * sizeof(T));
  // a known order for the harness: channel j gets norm (j * 7) % F
  for (int j = 0; j < F; ++j) out[j] = (double)((j * 7) % F);
  return hipSuccess;
}

hipError_t launch_renoise(float* z, const float* v, float, float, const float* eps, int64_t n,
                          hipStream_t) {
  ++g_stub_launches;
  rd(v, (size_t)n * sizeof(float));
  if (eps) rd(eps, (size_t)n * sizeof(float));
  wr(z, (size_t)n * sizeof(float));
  return hipSuccess;
}

template <typename T>
hipError_t launch_cast(const float* src, T* dst, int64_t n, hipStream_t) {
  ++g_stub_launches;
  rd(src, (size_t)n * sizeof(float));
  wr(dst, (size_t)n * sizeof(T));
  return hipSuccess;
}

#define GEMM_INST(T, OutT)                                                                    \
  template hipError_t launch_gemm<T, OutT>(const T*, int64_t, const T*, int64_t, OutT*, int64_t, \
                                           int, int, int, int, const float*, const float*,    \
                                           const float*, hipStream_t, const GemmGather*,      \
                                           const GemmVt*);
GEMM_INST(bf16, bf16)
GEMM_INST(bf16, float)
GEMM_INST(float, float)
#undef GEMM_INST

#define INST(T)                                                                                  \
  template hipError_t launch_attention<T>(int, const T*, int64_t, const T*, int64_t, const T*,   \
                                          int64_t, T*, int64_t, int, int, int, int, hipStream_t, \
                                          bool, float*, int);                                    \
  template hipError_t launch_norm<T>(const T*, T*, int, int, int, const float*, const float*,   \
                                     const float*, const float*, float, hipStream_t);           \
  template hipError_t launch_qk_norm<T>(T*, int64_t, int, int, int, int, int, const float*,      \
                                        const float*, float, float, const RopeDesc*,            \
                                        hipStream_t, const int32_t*, float);                    \
  template hipError_t launch_transpose_vt<T>(const T*, int64_t, int, int, int, T*, int64_t,      \
                                             hipStream_t);                                      \
  template hipError_t launch_gather<T>(const T*, int64_t, T*, int64_t, int, int, const int32_t*, \
                                       const int32_t*, hipStream_t);                            \
  template hipError_t launch_gather_cols16<T>(const T*, int64_t, T*, int64_t, int, int,          \
                                              const int32_t*, hipStream_t);                     \
  template hipError_t launch_gather_rows16<T>(const T*, int64_t, T*, int64_t, int64_t, int, int, \
                                              const int32_t*, hipStream_t);                     \
  template hipError_t launch_gemv<T>(const T*, const float*, const float*, float*, int, int,     \
                                     hipStream_t);                                              \
  template hipError_t launch_ffn_norms<T>(const T*, const float*, const T*, int, int, double*,   \
                                          hipStream_t);                                         \
  template hipError_t launch_cast<T>(const float*, T*, int64_t, hipStream_t);
INST(bf16)
INST(float)
#undef INST

}  // namespace dif

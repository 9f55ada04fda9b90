// Bidirectional flash attention on MFMA for gfx950.
//
// Work split: one workgroup = 4 waves = 128 queries of one (sample, head);
// a wave owns 32 queries and walks all keys in tiles of 64.
//
// The scores are computed transposed, S^T = K Q^T, with MFMA 32x32 tiles:
// the A operand is the K tile (rows = keys, from LDS), the B operand is
// Q^T (columns = queries), held in registers for the whole key loop.  A lane
// then owns one query column and 16 keys of each 32-key tile, so the
// softmax row statistics are lane-local plus one exchange with lane^32.
// The K rows are placed in LDS in a permuted order (key_slot) chosen so that
// accumulator register r of lane group g holds key 16*g + r: each lane group's 16 probabilities are consecutive keys, which
// makes them directly the B operand (P^T) of O^T += V^T P^T, and makes the
// matching V^T operand one contiguous 16-byte LDS read.  V is consumed
// transposed (Vt, [head_dim rows][keys]) so that read is row-contiguous.
//
// Online softmax in base 2 (scores pre-multiplied by log2(e)/sqrt(dh))
// with a lazy rescale: the exponent base only moves (and O^T, l are
// rescaled) when a query's running max exceeds it by more than kSlack.
// Key tails are masked to -inf; V^T chunks past the last key are zero-filled.
// At most 256 registers per lane, so two waves share each SIMD and one
// wave's softmax overlaps the other's MFMA work.
#include "common.h"
#include "kernels.h"

namespace dif {

constexpr int AT_THREADS = 256;
constexpr int AT_BM = 128;  // queries per workgroup
constexpr int AT_BN = 64;   // keys per tile
constexpr float kSlack = 8.f;  // log2 headroom of the lazy softmax rescale

template <typename T>
struct AttnParams {
  const T* Q;
  const T* K;
  const T* Vt;
  T* O;
  int64_t ldq, ldk, ldvt, ldo;
  int B, Lq, Lk, H;
  float c;  // log2(e) / sqrt(head_dim)
};

// LDS row of key kappa (0..31) inside a 32-key sub-tile.
__device__ __forceinline__ int key_slot(int kappa) {
  const int gq = kappa >> 4, k = (kappa & 15) >> 2, j = kappa & 3;
  return 8 * k + 4 * gq + j;
}

template <typename T, int DH>
__global__ __launch_bounds__(AT_THREADS, 2) void flash_attn_kernel(AttnParams<T> p) {
  constexpr int VEC = Chunk<T>::VEC;
  constexpr int KCH = DH * (int)sizeof(T) / 16;     // chunks per K row
  constexpr int VCH = AT_BN * (int)sizeof(T) / 16;  // chunks per V^T row
  constexpr int NQS = DH / Mma<T>::KS;              // MMA steps over head_dim
  constexpr int NPC = 16 / VEC;                     // P chunks per 32-key sub-tile
  constexpr int K_PER_T = AT_BN * KCH / AT_THREADS;
  constexpr int V_PER_T = DH * VCH / AT_THREADS;
  static_assert(K_PER_T * AT_THREADS == AT_BN * KCH, "K tile split");
  static_assert(V_PER_T * AT_THREADS == DH * VCH, "V tile split");
  __shared__ u32x4 ks_[2][AT_BN][KCH];
  __shared__ u32x4 vs_[2][DH][VCH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, col = lane & 31;

  const int nqb = (p.Lq + AT_BM - 1) / AT_BM;
  const int bid = xcd_remap(blockIdx.x, nqb * p.H * p.B);
  const int qb = bid % nqb, hb = bid / nqb;
  const int h = hb % p.H, b = hb / p.H;

  const int q = qb * AT_BM + wave * 32 + col;
  const int64_t qrow = (int64_t)b * p.Lq + min(q, p.Lq - 1);

  // Q^T fragments: chunk (2s + g) of this query's head slice
  u32x4 qf[NQS];
#pragma unroll
  for (int s = 0; s < NQS; ++s)
    qf[s] = *reinterpret_cast<const u32x4*>(p.Q + qrow * p.ldq + h * DH + (2 * s + g) * VEC);

  const T* kbase = p.K + (int64_t)b * p.Lk * p.ldk + h * DH;
  const T* vbase = p.Vt + ((int64_t)b * p.H + h) * DH * p.ldvt;
  const int ntiles = (p.Lk + AT_BN - 1) / AT_BN;

  u32x4 kreg[K_PER_T], vreg[V_PER_T];
  auto gload = [&](int kt) {
    const int key0 = kt * AT_BN;
#pragma unroll
    for (int i = 0; i < K_PER_T; ++i) {
      const int id = tid + AT_THREADS * i;
      const int key = min(key0 + id / KCH, p.Lk - 1);
      kreg[i] = *reinterpret_cast<const u32x4*>(kbase + (int64_t)key * p.ldk + (id % KCH) * VEC);
    }
#pragma unroll
    for (int i = 0; i < V_PER_T; ++i) {
      const int id = tid + AT_THREADS * i;
      const int d = id / VCH, k0 = key0 + (id % VCH) * VEC;
      if (k0 + VEC <= p.Lk) {
        vreg[i] = *reinterpret_cast<const u32x4*>(vbase + (int64_t)d * p.ldvt + k0);
      } else if (k0 < p.Lk) {
        float tmp[VEC];
        Chunk<T>::unpack(*reinterpret_cast<const u32x4*>(vbase + (int64_t)d * p.ldvt + k0), tmp);
#pragma unroll
        for (int e = 0; e < VEC; ++e)
          if (k0 + e >= p.Lk) tmp[e] = 0.f;
        vreg[i] = Chunk<T>::pack(tmp);
      } else {
        vreg[i] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < K_PER_T; ++i) {
      const int id = tid + AT_THREADS * i;
      const int kl = id / KCH, c = id % KCH;
      const int row = (kl & ~31) + key_slot(kl & 31);
      ks_[buf][row][swz<KCH>(row, c)] = kreg[i];
    }
#pragma unroll
    for (int i = 0; i < V_PER_T; ++i) {
      const int id = tid + AT_THREADS * i;
      const int d = id / VCH, c = id % VCH;
      vs_[buf][d][swz<VCH>(d, c)] = vreg[i];
    }
  };

  f32x16 o[DH / 32];
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[dt][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  gload(0);
  sstore(0);
  __syncthreads();

  for (int kt = 0; kt < ntiles; ++kt) {
    const int buf = kt & 1;
    const bool more = kt + 1 < ntiles;
    if (more) gload(kt + 1);

    // S^T for two 32-key sub-tiles
    f32x16 s[2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kk][r] = 0.f;
#pragma unroll
      for (int st = 0; st < NQS; ++st) {
        const u32x4 a = ks_[buf][kk * 32 + col][swz<KCH>(col, 2 * st + g)];
        Mma<T>::step(s[kk], a, qf[st]);
      }
    }
    const int key0 = kt * AT_BN;
    if (key0 + AT_BN > p.Lk) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (key0 + kk * 32 + 16 * g + r >= p.Lk) s[kk][r] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kk][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32)) * p.c;
    // Lazy rescale: the exponent base m_run only moves when some query's
    // max exceeds it by more than kSlack (probabilities stay <= 2^kSlack,
    // far from float overflow); numerator and denominator share the base,
    // so the normalised result is unchanged.
    if (__any(mx > m_run + kSlack)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
      m_run = m_new;
    }
    float rs = 0.f;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = __builtin_amdgcn_exp2f(fmaf(s[kk][r], p.c, -m_run));
        s[kk][r] = e;
        rs += e;
      }
    rs += __shfl_xor(rs, 32);
    l_run += rs;

    // O^T += V^T P^T
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int u = 0; u < NPC; ++u) {
        float pv[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) pv[e] = s[kk][u * VEC + e];
        const u32x4 pc = Chunk<T>::pack(pv);
        const int vc = (kk * 32 + 16 * g) / VEC + u;
#pragma unroll
        for (int dt = 0; dt < DH / 32; ++dt) {
          const u32x4 a = vs_[buf][dt * 32 + col][swz<VCH>(col, vc)];
          Mma<T>::step(o[dt], a, pc);
        }
      }
    }

    if (more) sstore(buf ^ 1);
    __syncthreads();
  }

  if (q < p.Lq) {
    const float inv = 1.f / l_run;
    T* dst = p.O + ((int64_t)b * p.Lq + q) * p.ldo + h * DH;
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int d = dt * 32 + 8 * rr + 4 * g;
        if constexpr (sizeof(T) == 4) {
          f32x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = o[dt][4 * rr + e] * inv;
          *reinterpret_cast<f32x4*>(dst + d) = v;
        } else {
          bf16x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = (bf16)(o[dt][4 * rr + e] * inv);
          *reinterpret_cast<bf16x4*>(dst + d) = v;
        }
      }
  }
}

template <typename T>
hipError_t launch_attention(int head_dim, const T* Q, int64_t ldq, const T* K, int64_t ldk,
                            const T* Vt, int64_t ldvt, T* O, int64_t ldo, int B, int Lq, int Lk,
                            int H, hipStream_t stream) {
  if (B <= 0 || Lq <= 0 || H <= 0) return hipSuccess;
  AttnParams<T> p{Q, K, Vt, O, ldq, ldk, ldvt, ldo, B, Lq, Lk, H,
                  1.4426950408889634f / sqrtf((float)head_dim)};
  const int blocks = ((Lq + AT_BM - 1) / AT_BM) * H * B;
  dim3 grid(blocks), block(AT_THREADS);
  if (head_dim == 128) {
    hipLaunchKernelGGL((flash_attn_kernel<T, 128>), grid, block, 0, stream, p);
  } else if (head_dim == 64) {
    hipLaunchKernelGGL((flash_attn_kernel<T, 64>), grid, block, 0, stream, p);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template hipError_t launch_attention<bf16>(int, const bf16*, int64_t, const bf16*, int64_t,
                                           const bf16*, int64_t, bf16*, int64_t, int, int, int,
                                           int, hipStream_t);
template hipError_t launch_attention<float>(int, const float*, int64_t, const float*, int64_t,
                                            const float*, int64_t, float*, int64_t, int, int,
                                            int, int, hipStream_t);

}  // namespace dif

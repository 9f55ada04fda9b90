// Bidirectional flash attention on MFMA for gfx950.
//
// Work split: one workgroup = 8 waves of one (sample, head); a wave owns 32
// queries and walks all keys in tiles of 64, as two 32-key halves.  Eight
// waves share each K / V^T tile copied into LDS, which halves those copies
// per flop against four waves (measured +4%); one workgroup fills a CU.
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
// Online softmax in base 2 with a lazy rescale: the exponent base m only
// moves (and O^T, l are rescaled) when a 32-key half's probabilities for a
// query sum to more than 2^kSlack, so the common path has no row maximum
// (measured +1.5% against a per-half maximum test).  The base enters through the MFMA accumulator: the first
// MFMA of a half adds C = -m (sixteen registers that change only with m), so
// with queries pre-scaled by log2(e)/sqrt(dh) (done by the QK-norm kernel
// before its bf16 rounding) the MFMA output is already the exponent and the
// VALU does no per-score scale or subtraction.  Unscaled queries (the plain
// operator) take one multiply per score instead.
// Key tails are masked to -inf; V^T chunks past the last key are zero-filled.
// The MFMA blocks run at raised wave priority, so when both waves of a SIMD
// are ready the one issuing MFMAs wins and the other's softmax VALU work
// fills the gaps (measured +2%).
// The kernel fits in 256 registers per lane (two waves per SIMD).
#include <mutex>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace dif {

// waves per workgroup: 8 when the keys are long (bf16), 4 for short key
// sequences (the text tokens), where eight waves leave too few workgroups and
// too few key tiles to amortise each workgroup's prologue
constexpr int kLongKeys = kAttnLongKeys;
constexpr int kMaxSplitItems = 128;   // split items one workspace region holds
constexpr int AT_BN = 64;        // keys per tile
constexpr float kSlack = 8.f;    // log2 headroom of the lazy softmax rescale

template <typename T>
struct AttnParams {
  const T* Q;
  const T* K;
  const T* Vt;
  T* O;
  int64_t ldq, ldk, ldvt, ldo;
  int B, Lq, Lk, H;
  float c;  // log2(e) / sqrt(head_dim)
  // Work items (query block, head, sample) [0, nreg) run whole; items from
  // nreg on are split along the keys at tile split_tile, each half writing
  // its unnormalised output and (m, l) to part for attn_merge_kernel.
  int nreg, split_tile;
  float* part;
};

// Partial-result layout of a split item s and key half k (0, 1), for BMQ
// queries: [s][k][BMQ][DH] output sums, then [s][k][BMQ][2] (m, l).
template <int DH>
__host__ __device__ inline size_t part_o_off(int s, int k, int q, int bmq) {
  return ((size_t)(2 * s + k) * bmq + q) * DH;
}
template <int DH>
__host__ __device__ inline size_t part_ml_off(int nsplit, int s, int k, int q, int bmq) {
  return (size_t)2 * nsplit * bmq * DH + ((size_t)(2 * s + k) * bmq + q) * 2;
}

// LDS row of key kappa (0..31) inside a 32-key sub-tile.
__device__ __forceinline__ int key_slot(int kappa) {
  const int gq = kappa >> 4, k = (kappa & 15) >> 2, j = kappa & 3;
  return 8 * k + 4 * gq + j;
}

// SC: queries arrive pre-multiplied by log2(e)/sqrt(dh); AT_WAVES waves per
// workgroup (4 or 8: two waves per SIMD either way).
template <typename T, int DH, bool SC, int AT_WAVES>
__global__ __launch_bounds__(64 * AT_WAVES, 8 / AT_WAVES) void flash_attn_kernel(AttnParams<T> p) {
  constexpr int AT_THREADS = 64 * AT_WAVES;
  constexpr int VEC = Chunk<T>::VEC;
  constexpr int KCH = DH * (int)sizeof(T) / 16;     // chunks per K row
  constexpr int VCH = AT_BN * (int)sizeof(T) / 16;  // chunks per V^T row
  constexpr int NQS = DH / Mma<T>::KS;              // MMA steps over head_dim
  constexpr int NPC = 16 / VEC;                     // P chunks per 32-key sub-tile
  constexpr int K_PER_T = AT_BN * KCH / AT_THREADS;
  constexpr int V_PER_T = DH * VCH / AT_THREADS;
  constexpr int BMQ = AT_WAVES * 32;                // queries per workgroup
  static_assert(K_PER_T * AT_THREADS == AT_BN * KCH, "K tile split");
  static_assert(V_PER_T * AT_THREADS == DH * VCH, "V tile split");
  __shared__ u32x4 ks_[2][AT_BN][KCH];
  __shared__ u32x4 vs_[2][DH][VCH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, col = lane & 31;

  const int nqb = (p.Lq + BMQ - 1) / BMQ;
  const int ntiles = (p.Lk + AT_BN - 1) / AT_BN;
  // this workgroup's item and key-tile range [t0, t1)
  int bid, split = -1, t0 = 0, t1 = ntiles;
  if ((int)blockIdx.x < p.nreg) {
    bid = xcd_remap(blockIdx.x, p.nreg);
  } else {
    const int sidx = (int)blockIdx.x - p.nreg;   // dispatched last: the final round
    bid = p.nreg + (sidx >> 1);
    split = sidx;
    if (sidx & 1) t0 = p.split_tile;
    else t1 = p.split_tile;
  }
  const int qb = bid % nqb, hb = bid / nqb;
  const int h = hb % p.H, b = hb / p.H;

  // Q^T fragments: chunk (2s + g) of this lane's query
  u32x4 qf[NQS];
  {
    const int q = qb * BMQ + wave * 32 + col;
    const int64_t qrow = (int64_t)b * p.Lq + min(q, p.Lq - 1);
#pragma unroll
    for (int s = 0; s < NQS; ++s)
      qf[s] = *reinterpret_cast<const u32x4*>(p.Q + qrow * p.ldq + h * DH + (2 * s + g) * VEC);
  }

  const T* kbase = p.K + (int64_t)b * p.Lk * p.ldk + h * DH;
  const T* vbase = p.Vt + ((int64_t)b * p.H + h) * DH * p.ldvt;

  // Full tiles are copied straight into LDS with buffer loads (no staging
  // registers): each wave instruction fills 1 KB of LDS, lane l writing
  // bytes [16 l, 16 l + 16), so every lane fetches the element that the
  // permuted / swizzled layout puts in its slot.  Per-tile descriptors are
  // built in SGPRs and lane offsets are tile-invariant.  K rows at or past
  // Lk fall outside the K descriptor and read as zero (their scores are
  // masked).  The last tile, if it ends past Lk, goes through registers and
  // zero-fills V^T beyond Lk element by element.
  constexpr uint32_t kRsrcWord3 = 0x00020000u;
  constexpr int ES = (int)sizeof(T);
  constexpr int KRPI = 64 / KCH;                  // K rows per wave instruction
  constexpr int VRPI = 64 / VCH;                  // V^T rows per wave instruction
  constexpr int KI = AT_BN / (KRPI * AT_WAVES);   // K instructions per wave
  constexpr int VI = DH / (VRPI * AT_WAVES);      // V^T instructions per wave
  static_assert(KI * KRPI * AT_WAVES == AT_BN && VI * VRPI * AT_WAVES == DH, "direct tile split");
  uint32_t kd_off[KI], vd_off[VI];
#pragma unroll
  for (int j = 0; j < KI; ++j) {
    const int row = (j * AT_WAVES + wave) * KRPI + lane / KCH;  // LDS row
    const int kk = row >> 5, i = row & 31;
    const int key = kk * 32 + 16 * ((i >> 2) & 1) + 4 * (i >> 3) + (i & 3);  // inverse of key_slot
    kd_off[j] = (uint32_t)((key * p.ldk + swz<KCH>(row, lane % KCH) * VEC) * ES);
  }
#pragma unroll
  for (int j = 0; j < VI; ++j) {
    const int d = (j * AT_WAVES + wave) * VRPI + lane / VCH;
    vd_off[j] = (uint32_t)((d * p.ldvt + swz<VCH>(d, lane % VCH) * VEC) * ES);
  }
  const int64_t v_bytes = (int64_t)DH * p.ldvt * ES;
  auto k_rsrc = [&](int key0) {
    const int64_t kb = (int64_t)(p.Lk - key0) * p.ldk * ES;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(kbase + (int64_t)key0 * p.ldk), (short)0,
                                             (uint32_t)(kb < 0xffffffffll ? kb : 0xffffffffll),
                                             kRsrcWord3);
  };
  auto load_direct = [&](int kt, int buf) {
#if defined(__HIP_DEVICE_COMPILE__)
    typedef __attribute__((address_space(3))) void lds_t;
    const int key0 = kt * AT_BN;
    const __amdgpu_buffer_rsrc_t kr = k_rsrc(key0);
    const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<T*>(vbase + key0), (short)0, (uint32_t)(v_bytes - (int64_t)key0 * ES), kRsrcWord3);
#pragma unroll
    for (int j = 0; j < KI; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (lds_t*)&ks_[buf][(j * AT_WAVES + wave) * KRPI][0], 16,
                                               kd_off[j], 0, 0, 0);
#pragma unroll
    for (int j = 0; j < VI; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_t*)&vs_[buf][(j * AT_WAVES + wave) * VRPI][0], 16,
                                               vd_off[j], 0, 0, 0);
#endif
  };
  // tail tile: through registers, V^T zero-filled past Lk
  auto load_tail = [&](int kt, int buf) {
    const int key0 = kt * AT_BN;
    const __amdgpu_buffer_rsrc_t kr = k_rsrc(key0);
#pragma unroll
    for (int i = 0; i < K_PER_T; ++i) {
      const int id = tid + AT_THREADS * i;
      const int kl = id / KCH, c = id % KCH;
      const u32x4 v = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(kr, (uint32_t)((kl * p.ldk + c * VEC) * ES), 0, 0));
      const int row = (kl & ~31) + key_slot(kl & 31);
      ks_[buf][row][swz<KCH>(row, c)] = v;
    }
#pragma unroll
    for (int i = 0; i < V_PER_T; ++i) {
      const int id = tid + AT_THREADS * i;
      const int d = id / VCH, c = id % VCH, k0 = key0 + c * VEC;
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (k0 < p.Lk) {
        float tmp[VEC];
        Chunk<T>::unpack(*reinterpret_cast<const u32x4*>(vbase + (int64_t)d * p.ldvt + k0), tmp);
#pragma unroll
        for (int e = 0; e < VEC; ++e)
          if (k0 + e >= p.Lk) tmp[e] = 0.f;
        v = Chunk<T>::pack(tmp);
      }
      vs_[buf][d][swz<VCH>(d, c)] = v;
    }
  };
  auto load_tile = [&](int kt, int buf) {
    if ((kt + 1) * AT_BN <= p.Lk) load_direct(kt, buf);
    else load_tail(kt, buf);
  };

  f32x16 o[DH / 32];
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[dt][r] = 0.f;
  float l_run = 0.f;
  const float uscale = SC ? 1.f : p.c;   // MFMA output units -> log2 units

  // S^T of half kk of the tile in buffer buf, plus c0 (an accumulator
  // initialiser); K fragments are read in batches of KB ahead of their MFMAs.
  auto scores = [&](int buf, int kk, const f32x16& c0) {
    constexpr int KB = NQS >= 8 ? NQS / 2 : NQS;
    f32x16 s = c0;
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int s0 = 0; s0 < NQS; s0 += KB) {
      u32x4 kf[KB];
#pragma unroll
      for (int st = 0; st < KB; ++st) kf[st] = ks_[buf][kk * 32 + col][swz<KCH>(col, 2 * (s0 + st) + g)];
#pragma unroll
      for (int st = 0; st < KB; ++st) Mma<T>::step(s, kf[st], qf[s0 + st]);
    }
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(0);
    return s;
  };
  auto mask = [&](f32x16& s, int key) {   // keys >= Lk -> -inf
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (key + 16 * g + r >= p.Lk) s[r] = -INFINITY;
  };

  load_tile(t0, 0);
  wait_vmcnt<0>();   // this wave's direct-to-LDS loads have landed
  __syncthreads();   // ... and every other wave's

  // Initial base: the max of each query's first 32 scores of the range (its
  // first key exists, so it is finite).  negm holds -m in MFMA output units.
  float m_run;
  f32x16 negm;
  {
    f32x16 z;
#pragma unroll
    for (int r = 0; r < 16; ++r) z[r] = 0.f;
    f32x16 s0 = scores(0, 0, z);
    if (t0 * AT_BN + 32 > p.Lk) mask(s0, t0 * AT_BN);
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s0[r]);
    m_run = fmaxf(mx, __shfl_xor(mx, 32)) * uscale;
#pragma unroll
    for (int r = 0; r < 16; ++r) negm[r] = -m_run / uscale;
  }

  // One key tile.  The LDS buffer and whether the tile needs the key-tail
  // masks are compile-time, so fragment addresses are lane constants plus
  // immediate offsets and full tiles carry no masking code.
  auto tile = [&](int kt, auto buf_c, auto masked_c) {
    constexpr int buf = decltype(buf_c)::value;
    constexpr bool MASKED = decltype(masked_c)::value;
    // buffer buf^1 was last read before the previous barrier
    if (kt + 1 < t1) load_tile(kt + 1, buf ^ 1);

    const int key0 = kt * AT_BN;
    // the two 32-key halves of the tile in turn: S^T, softmax, O^T += V^T P^T
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      __builtin_amdgcn_sched_barrier(0);   // halves are not interleaved (register budget)
      f32x16 s = scores(buf, kk, negm);   // (scores - m) in MFMA output units
      // (the tail tile masks before its V^T reads: fewer registers live
      // across the branch)
      if (MASKED && key0 + kk * 32 + 32 > p.Lk) mask(s, key0 + kk * 32);
      // V^T fragments of this half, in flight during the softmax
      u32x4 vf[NPC][DH / 32];
#pragma unroll
      for (int u = 0; u < NPC; ++u)
#pragma unroll
        for (int dt = 0; dt < DH / 32; ++dt)
          vf[u][dt] = vs_[buf][dt * 32 + col][swz<VCH>(col, (kk * 32 + 16 * g) / VEC + u)];
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (!SC) {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] *= uscale;
      }
      // probabilities against the current base, packed as the B operand of
      // O^T += V^T P^T, and this half's lane-partial row sum
      u32x4 pc[NPC];
      float lh = 0.f;
      auto probs = [&]() {
#pragma unroll
        for (int u = 0; u < NPC; ++u) {
          float pv[VEC];
#pragma unroll
          for (int e = 0; e < VEC; ++e) pv[e] = __builtin_amdgcn_exp2f(s[u * VEC + e]);
          pc[u] = Chunk<T>::pack(pv);
          float t[VEC];
#pragma unroll
          for (int e = 0; e < VEC; ++e) t[e] = pv[e];
#pragma unroll
          for (int w = VEC / 2; w > 0; w /= 2)
#pragma unroll
            for (int e = 0; e < w; ++e) t[e] += t[e + w];
          lh = u == 0 ? t[0] : lh + t[0];
        }
      };
      probs();
      // Lazy rescale, triggered by the half's row sum: while no probability
      // of the half sums above 2^kSlack, every one is at most that, and the
      // base stays.  Otherwise (a score moved far above the base, or
      // overflowed) the base moves up to the half's maximum, O^T and l are
      // rescaled and the probabilities recomputed.  Numerator and
      // denominator share the base, so the normalised result is unchanged.
      // A fully masked half sums to 0 and never moves the base.
      if (__any(!(lh <= (float)(1 << (int)kSlack)))) {
        float mx = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[r]);
        const float d = fmaxf(fmaxf(mx, __shfl_xor(mx, 32)), 0.f);
        const float alpha = __builtin_amdgcn_exp2f(-d);
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s[r] -= d;
          negm[r] -= d / uscale;
        }
        m_run += d;
        probs();
      }
      l_run += lh;
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int u = 0; u < NPC; ++u)
#pragma unroll
        for (int dt = 0; dt < DH / 32; ++dt) Mma<T>::step(o[dt], vf[u][dt], pc[u]);
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(0);
    }

    wait_vmcnt<0>();   // tile kt+1 (direct-to-LDS) has landed for this wave
    __syncthreads();
  };
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  const int nfull = min(p.Lk / AT_BN, t1);   // tiles of 64 valid keys in the range
  int kt = t0;   // (t0 is even: buffer 0 holds tile t0)
  for (; kt + 2 <= nfull; kt += 2) {
    tile(kt, B0{}, std::false_type{});
    tile(kt + 1, B1{}, std::false_type{});
  }
  if (kt < nfull) tile(kt++, B0{}, std::false_type{});
  if (kt < t1) {   // the partial last tile
    if ((kt - t0) & 1) tile(kt, B1{}, std::true_type{});
    else tile(kt, B0{}, std::true_type{});
  }

  const int q = qb * BMQ + wave * 32 + col;
  const float l = l_run + __shfl_xor(l_run, 32);
  if (split >= 0) {
    // unnormalised sums and this half's (m, l), combined by attn_merge_kernel
    const int nsplit = (int)(gridDim.x - p.nreg) / 2;
    const int ql = wave * 32 + col;
    float* po = p.part + part_o_off<DH>(split >> 1, split & 1, ql, BMQ);
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        f32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = o[dt][4 * rr + e];
        *reinterpret_cast<f32x4*>(po + dt * 32 + 8 * rr + 4 * g) = v;
      }
    if (g == 0) {
      float* pml = p.part + part_ml_off<DH>(nsplit, split >> 1, split & 1, ql, BMQ);
      pml[0] = m_run;
      pml[1] = l;
    }
    return;
  }
  if (q >= p.Lq) return;
  const float inv = 1.f / l;
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

// Combines the two key halves of each split item: with m = max(m0, m1) and
// a_k = 2^(m_k - m), O = (a0 O0 + a1 O1) / (a0 l0 + a1 l1).  One workgroup
// per split item, a thread per four output dims of a query.
template <typename T, int DH, int BMQ>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnParams<T> p, int nsplit) {
  const int sidx = blockIdx.x;
  const int nqb = (p.Lq + BMQ - 1) / BMQ;
  const int item = p.nreg + sidx;
  const int qb = item % nqb, hb = item / nqb;
  const int h = hb % p.H, b = hb / p.H;
  for (int idx = threadIdx.x; idx < BMQ * DH / 4; idx += 256) {
    const int ql = idx / (DH / 4), d = (idx % (DH / 4)) * 4;
    const int q = qb * BMQ + ql;
    if (q >= p.Lq) continue;
    const float* ml0 = p.part + part_ml_off<DH>(nsplit, sidx, 0, ql, BMQ);
    const float* ml1 = p.part + part_ml_off<DH>(nsplit, sidx, 1, ql, BMQ);
    const float m = fmaxf(ml0[0], ml1[0]);
    const float a0 = __builtin_amdgcn_exp2f(ml0[0] - m), a1 = __builtin_amdgcn_exp2f(ml1[0] - m);
    const float inv = 1.f / (a0 * ml0[1] + a1 * ml1[1]);
    const f32x4 o0 = *reinterpret_cast<const f32x4*>(p.part + part_o_off<DH>(sidx, 0, ql, BMQ) + d);
    const f32x4 o1 = *reinterpret_cast<const f32x4*>(p.part + part_o_off<DH>(sidx, 1, ql, BMQ) + d);
    T* dst = p.O + ((int64_t)b * p.Lq + q) * p.ldo + h * DH + d;
#pragma unroll
    for (int e = 0; e < 4; ++e) dst[e] = from_f32<T>((a0 * o0[e] + a1 * o1[e]) * inv);
  }
}

template <typename T, int DH, int W>
void launch_w(AttnParams<T> p, bool q_scaled, hipStream_t stream, int ncu) {
  constexpr int BMQ = W * 32;
  const int items = ((p.Lq + BMQ - 1) / BMQ) * p.H * p.B;
  // Workgroups fill a CU (W = 8) or half of one (W = 4).  When the last
  // round of workgroups would be at most half full, its items are split
  // along the keys into two halves each, so the round is full and half as
  // long; a merge pass combines the halves.
  const int slots = ncu * (W == 8 ? 1 : 2);
  const int rem = slots > 0 ? items % slots : 0;
  const int nfull = p.Lk / AT_BN;
  int nsplit = 0;
  if (p.part && rem > 0 && 2 * rem <= slots && rem <= kMaxSplitItems && nfull >= 4 && BMQ <= 256)
    nsplit = rem;
  p.nreg = items - nsplit;
  p.split_tile = (nfull / 2) & ~1;
  const int blocks = p.nreg + 2 * nsplit;
  if (q_scaled)
    hipLaunchKernelGGL((flash_attn_kernel<T, DH, true, W>), dim3(blocks), dim3(64 * W), 0, stream, p);
  else
    hipLaunchKernelGGL((flash_attn_kernel<T, DH, false, W>), dim3(blocks), dim3(64 * W), 0, stream, p);
  if (nsplit > 0)
    hipLaunchKernelGGL((attn_merge_kernel<T, DH, BMQ>), dim3(nsplit), dim3(256), 0, stream, p, nsplit);
}

template <typename T, int DH>
void launch_dh(const AttnParams<T>& p, bool q_scaled, hipStream_t stream, int ncu) {
  // (float32 keeps four waves: its head-128 kernel needs one wave per SIMD)
  if constexpr (sizeof(T) == 2) {
    if (p.Lk >= kLongKeys) {
      launch_w<T, DH, 8>(p, q_scaled, stream, ncu);
      return;
    }
  }
  launch_w<T, DH, 4>(p, q_scaled, stream, ncu);
}

size_t attention_split_bytes(int head_dim) {
  return (size_t)2 * kMaxSplitItems * 256 * (head_dim + 2) * sizeof(float);
}

// Key-split partial sums for callers that cannot allocate: one buffer in
// static device memory, which every device the library runs on holds until
// the process ends.  Sized for head_dim 128 (the largest split workspace;
// it does not grow with the problem, the split is capped at kMaxSplitItems
// items).  Host code reaches it only through the address
// hipGetSymbolAddress returns on each device.
constexpr size_t kStaticSplitBytes = (size_t)2 * kMaxSplitItems * 256 * (128 + 2) * sizeof(float);
static __device__ __align__(256) float scratch[kStaticSplitBytes / sizeof(float)];

hipError_t attention_static_scratch(float** out, size_t* bytes) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static float* ptrs[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(mu);
  if (!ptrs[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    ptrs[dev] = static_cast<float*>(p);
  }
  *out = ptrs[dev];
  *bytes = kStaticSplitBytes;
  return hipSuccess;
}

template <typename T>
hipError_t launch_attention(int head_dim, const T* Q, int64_t ldq, const T* K, int64_t ldk,
                            const T* Vt, int64_t ldvt, T* O, int64_t ldo, int B, int Lq, int Lk,
                            int H, hipStream_t stream, bool q_scaled, float* split_part,
                            int ncu) {
  if (B <= 0 || Lq <= 0 || H <= 0) return hipSuccess;
  AttnParams<T> p{Q, K, Vt, O, ldq, ldk, ldvt, ldo, B, Lq, Lk, H,
                  1.4426950408889634f / sqrtf((float)head_dim), 0, 0, split_part};
  if (head_dim == 128) {
    launch_dh<T, 128>(p, q_scaled, stream, ncu);
  } else if (head_dim == 64) {
    launch_dh<T, 64>(p, q_scaled, stream, ncu);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template hipError_t launch_attention<bf16>(int, const bf16*, int64_t, const bf16*, int64_t,
                                           const bf16*, int64_t, bf16*, int64_t, int, int, int,
                                           int, hipStream_t, bool, float*, int);
template hipError_t launch_attention<float>(int, const float*, int64_t, const float*, int64_t,
                                            const float*, int64_t, float*, int64_t, int, int,
                                            int, int, hipStream_t, bool, float*, int);

}  // namespace dif

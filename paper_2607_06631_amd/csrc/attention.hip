// Bidirectional flash attention on MFMA for gfx950.
//
// Three kernels share one arithmetic: bf16 with head_dim 128 on long key
// sequences (the blocks' self-attention) runs flash_attn_g2_kernel, four
// waves of two 32-query groups each (below); the other long-key cases run
// the eight-wave flash_attn_kernel, short key sequences (text tokens) and
// float32 the four-wave one.
//
// Work split of flash_attn_kernel: one workgroup = 8 waves of one (sample,
// head); a wave owns 32 queries and walks all keys in tiles of 64, as two
// 32-key halves.  Eight waves share each K / V^T tile copied into LDS,
// which halves those copies per flop against four waves (measured +4%);
// one workgroup fills a CU.
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
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
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

// Writes the 32 output rows a wave holds (query lane % 32; accumulator
// o[dt], register 4 rr + e, holds dim 32 dt + 8 rr + 4 g + e with
// g = lane / 32), times inv and converted to T, to dst (row stride ld;
// rows >= nrows are skipped) through the wave's own LDS region of
// 32 * DH * sizeof(T) bytes, which must be free.  Direct stores would put
// 32 rows into every store instruction; staged, each instruction writes
// whole rows.  The staging swizzles a row's 16-byte chunks by the row
// (and, for 2-byte T, the two 8-byte halves of a chunk by the next row
// bit), so the 8-byte column writes and the row reads are free of bank
// conflicts at head_dim 128.  A wave's LDS instructions execute in order:
// between its writes and reads a wavefront-scope fence (no barrier) keeps
// the compiler from reordering them.
template <typename T, int DH>
__device__ __forceinline__ void store_rows_staged(const f32x16 (&o)[DH / 32], float inv, char* stage,
                                                  T* dst, int64_t ld, int nrows, int lane) {
  constexpr int ES = (int)sizeof(T);
  constexpr int RB = DH * ES;     // bytes per row
  constexpr int CPR = RB / 16;    // 16-byte chunks per row
  constexpr int RPI = 64 / CPR;   // rows per read-back instruction
  static_assert(RPI * CPR == 64 && 32 % RPI == 0, "row staging split");
  // (opaque, so no address arithmetic of this epilogue is merged with, and
  // kept live from, the key loop's)
  asm volatile("" : "+v"(lane));
  const int col = lane & 31, g = lane >> 5;
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int byte = (dt * 32 + 8 * rr + 4 * g) * ES;
      if constexpr (ES == 4) {
        f32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = o[dt][4 * rr + e] * inv;
        *reinterpret_cast<f32x4*>(stage + col * RB + 16 * ((byte / 16) ^ (col % CPR))) = v;
      } else {
        bf16x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (bf16)(o[dt][4 * rr + e] * inv);
        const int half = ((byte / 8) & 1) ^ ((col / CPR) & 1);
        *reinterpret_cast<bf16x4*>(stage + col * RB + 16 * ((byte / 16) ^ (col % CPR)) + 8 * half) = v;
      }
    }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
  for (int i = 0; i < 32 / RPI; ++i) {
    const int row = i * RPI + lane / CPR, c = lane % CPR;
    u32x4 v = *reinterpret_cast<const u32x4*>(stage + row * RB + 16 * (c ^ (row % CPR)));
    if constexpr (ES == 2) {
      if (((i * RPI) / CPR) & 1) v = u32x4{v[2], v[3], v[0], v[1]};   // (uniform per instruction)
    }
    if (row < nrows) *reinterpret_cast<u32x4*>(reinterpret_cast<char*>(dst + row * ld) + 16 * c) = v;
  }
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
  // Output rows through LDS (free since the last tile's barrier).  A lane
  // holds four consecutive dims of its query per register group, so direct
  // stores would put 32 rows in every store instruction; staged, each
  // instruction writes whole rows (full 128-byte lines).
  const float inv = 1.f / l;
  store_rows_staged<T, DH>(o, inv, wave < 4 ? reinterpret_cast<char*>(&ks_[0][0][0]) + wave * 32 * DH * (int)sizeof(T)
                                             : reinterpret_cast<char*>(&vs_[0][0][0]) + (wave - 4) * 32 * DH * (int)sizeof(T),
                           p.O + ((int64_t)b * p.Lq + qb * BMQ + wave * 32) * p.ldo + h * DH, p.ldo,
                           min(32, p.Lq - (qb * BMQ + wave * 32)), lane);
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

// Long bf16 key sequences, head_dim 128: two 32-query groups per wave.
//
// One workgroup = 4 waves, one per SIMD, each owning 64 queries as two
// groups of 32 (g0, g1); 256 queries per workgroup as in the eight-wave
// kernel.  Every K and V^T fragment read from LDS feeds the MFMAs of both
// groups, so LDS fragment reads per flop are half the eight-wave kernel's.
// The score, softmax and output arithmetic is the eight-wave kernel's, in
// the same order per query (same K layout, transposed scores with -m in
// the accumulator, the same lazy-rescale test on the same 32 queries), so
// the two kernels give bit-identical results.
//
// With one wave per SIMD the wave hides its own softmax: the key loop is a
// software pipeline of blocks of 16 MFMAs, each carrying the softmax of one
// group's 32-key half:
//   X(t,h): S(t,h,g1) = K Q1^T and O1 += V^T P(prev,g1);  softmax S(t,h,g0)
//   Y(t,h): S(next,g0) = K Q0^T and O0 += V^T P(t,h,g0);  softmax S(t,h,g1)
// Score and output MFMAs alternate, so no MFMA waits for the one before
// it.  The softmax of a half is spread over its block: its 16
// exponentials in the first ten MFMA slots, each bf16 pair and row-sum add
// one slot after its inputs, so the half's sum is ready by the 14th MFMA;
// the lazy-rescale test and its (rare, out-of-line) branch then come
// before the block's last MFMA, which belongs to the other group and so is
// untouched by a rescale (+3.0 % against the test after the last MFMA,
// +2.5 % of that from not waiting on a chain of adds; +1.5 % more with the
// rescale block laid out off the straight path).  K fragments of the next half are
// read behind the score MFMAs that consume the current ones, V^T fragments
// behind the output MFMAs, so every read has a block of MFMAs to land.
//
// K / V^T tiles sit in a ring of three LDS buffers with one workgroup
// barrier per tile, after the first MFMA of X(t,1) (which reads no LDS):
// it publishes tile t+1 (each wave waited for its own direct-to-LDS loads)
// and frees the buffer of tile t-1, into which tile t+2 is then loaded,
// one load instruction behind each score MFMA.  Each ring slot is its own
// LDS variable, which is what lets the compiler see that those loads
// cannot alias the reads of the other slots (otherwise it waits for them
// before every read).  (A four-slot ring, two tiles in flight, measured
// 0.4 % slower.)
//
// The MFMAs are inline assembly so that the Q^T fragments and the O^T
// accumulators stay in AGPRs (the 512 registers of a lone wave hold both
// groups only with them there) while scores and fragments stay in VGPRs.
// The compiler does not see inline MFMAs as MFMAs, so the code keeps the
// hardware's dependency distances itself: an MFMA result is read by the
// VALU only after at least two further MFMAs and a dozen instructions, an
// explicit wait precedes the first output MFMA of a block (two wait states
// after the VALU writes its operand), and the rare rescale path and the
// epilogue wait out the MFMA pipeline before touching the accumulators.
// Plain VALU code may still be scheduled across those waits, and a register
// an MFMA reads may be reused right after it, so values the VALU writes for
// an MFMA (-m, recomputed probabilities) are pinned by empty register
// constraints ahead of each wait, -m stays live to the end of the kernel
// (an MFMA reads its accumulator input during its passes), and the first
// k-step of the prologue takes a zero accumulator as an inline constant.
// tests/test_mfma_hazards.py scans the compiled kernel for all three
// hazard patterns.
// The tile loads' buffer descriptors span exactly one full tile (a
// multiply-add of scalars per tile instead of a 64-bit bound clamp, +1.3 %).
// Measured against the eight-wave kernel on the blocks' launch (32760
// tokens, 24-40 heads): +11 to +12 % (1.28 -> 1.42-1.44 PFLOP/s).
namespace g2 {
__device__ __forceinline__ void mma_sc(f32x16& d, const u32x4& a, const u32x4& b, const f32x16& c) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %3" : "=&v"(d) : "v"(a), "a"(b), "v"(c));
}
// the first k-step with a zero accumulator (an inline constant: no registers)
__device__ __forceinline__ void mma_s0(f32x16& d, const u32x4& a, const u32x4& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(d) : "v"(a), "a"(b));
}
__device__ __forceinline__ void mma_s(f32x16& d, const u32x4& a, const u32x4& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(d) : "v"(a), "a"(b));
}
__device__ __forceinline__ void mma_o(f32x16& d, const u32x4& a, const u32x4& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(d) : "v"(a), "v"(b));
}
__device__ __forceinline__ void mma_o_first(f32x16& d, const u32x4& a, const u32x4& b) {
  asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(d) : "v"(a), "v"(b));
}
// wait out the MFMA pipeline before the VALU reads an MFMA result
__device__ __forceinline__ void mfma_drain() { asm volatile("s_nop 15\n\ts_nop 15" ::); }
// two wait states after the VALU wrote an MFMA operand
__device__ __forceinline__ void valu_to_mfma() { asm volatile("s_nop 4" ::); }
template <typename X>
__device__ __forceinline__ void pin(X& x) { asm volatile("" : "+v"(x)); }
template <typename X>
__device__ __forceinline__ void pin_a(X& x) { asm volatile("" : "+a"(x)); }
// a volatile LDS read, kept in program order among the inline MFMAs
__device__ __forceinline__ u32x4 lds_read(const u32x4* ptr) {
  typedef __attribute__((address_space(3))) const volatile u32x4 lds_u32x4;
  return *(lds_u32x4*)ptr;
}
}  // namespace g2

template <bool SC>
__global__ __launch_bounds__(256, 1) void flash_attn_g2_kernel(AttnParams<bf16> p) {
  using T = bf16;
  constexpr int NBUF = 3;   // LDS ring slots
  constexpr int DH = 128, W = 4, THREADS = 256, VEC = 8;
  constexpr int KCH = DH * 2 / 16;       // 16 chunks per K row
  constexpr int VCH = AT_BN * 2 / 16;    // 8 chunks per V^T row
  constexpr int NQS = DH / 16;           // 8 MMA steps over head_dim
  constexpr int BMQ = 256;
  constexpr int K_PER_T = AT_BN * KCH / THREADS;
  constexpr int V_PER_T = DH * VCH / THREADS;
  static_assert(K_PER_T * THREADS == AT_BN * KCH && V_PER_T * THREADS == DH * VCH, "tile split");
  // one LDS variable per ring slot: the compiler tells direct-to-LDS loads
  // into one slot from reads of another only across distinct variables
  __shared__ u32x4 ks0_[AT_BN][KCH], ks1_[AT_BN][KCH], ks2_[AT_BN][KCH];
  __shared__ u32x4 vs0_[DH][VCH], vs1_[DH][VCH], vs2_[DH][VCH];
  auto kbuf = [&](int b) __attribute__((always_inline)) -> u32x4(*)[KCH] {
    return b == 0 ? ks0_ : b == 1 ? ks1_ : ks2_;
  };
  auto vbuf = [&](int b) __attribute__((always_inline)) -> u32x4(*)[VCH] {
    return b == 0 ? vs0_ : b == 1 ? vs1_ : vs2_;
  };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, col = lane & 31;

  const int nqb = (p.Lq + BMQ - 1) / BMQ;
  const int ntiles = (p.Lk + AT_BN - 1) / AT_BN;
  int bid, split = -1, t0 = 0, t1 = ntiles;
  if ((int)blockIdx.x < p.nreg) {
    bid = xcd_remap(blockIdx.x, p.nreg);
  } else {
    const int sidx = (int)blockIdx.x - p.nreg;
    bid = p.nreg + (sidx >> 1);
    split = sidx;
    if (sidx & 1) t0 = p.split_tile;
    else t1 = p.split_tile;
  }
  const int qb = bid % nqb, hb = bid / nqb;
  const int h = hb % p.H, b = hb / p.H;

  u32x4 qf[2][NQS];
#pragma unroll
  for (int gr = 0; gr < 2; ++gr) {
    const int q = qb * BMQ + wave * 64 + gr * 32 + col;
    const int64_t qrow = (int64_t)b * p.Lq + min(q, p.Lq - 1);
#pragma unroll
    for (int s = 0; s < NQS; ++s)
      qf[gr][s] = *reinterpret_cast<const u32x4*>(p.Q + qrow * p.ldq + h * DH + (2 * s + g) * VEC);
  }
#pragma unroll
  for (int gr = 0; gr < 2; ++gr)
#pragma unroll
    for (int s = 0; s < NQS; ++s) g2::pin_a(qf[gr][s]);   // AGPRs from here on

  const T* kbase = p.K + (int64_t)b * p.Lk * p.ldk + h * DH;
  const T* vbase = p.Vt + ((int64_t)b * p.H + h) * DH * p.ldvt;

  // direct-to-LDS tile copies, as in the eight-wave kernel
  constexpr uint32_t kRsrcWord3 = 0x00020000u;
  constexpr int ES = 2;
  constexpr int KRPI = 64 / KCH;
  constexpr int VRPI = 64 / VCH;
  constexpr int KI = AT_BN / (KRPI * W);
  constexpr int VI = DH / (VRPI * W);
  static_assert(KI * KRPI * W == AT_BN && VI * VRPI * W == DH, "direct tile split");
  uint32_t kd_off[KI], vd_off[VI];
#pragma unroll
  for (int j = 0; j < KI; ++j) {
    const int row = (j * W + wave) * KRPI + lane / KCH;
    const int kk = row >> 5, i = row & 31;
    const int key = kk * 32 + 16 * ((i >> 2) & 1) + 4 * (i >> 3) + (i & 3);
    kd_off[j] = (uint32_t)((key * p.ldk + swz<KCH>(row, lane % KCH) * VEC) * ES);
  }
#pragma unroll
  for (int j = 0; j < VI; ++j) {
    const int d = (j * W + wave) * VRPI + lane / VCH;
    vd_off[j] = (uint32_t)((d * p.ldvt + swz<VCH>(d, lane % VCH) * VEC) * ES);
  }
  const int64_t v_bytes = (int64_t)DH * p.ldvt * ES;
  auto k_rsrc = [&](int key0) {
    const int64_t kb = (int64_t)(p.Lk - key0) * p.ldk * ES;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(kbase + (int64_t)key0 * p.ldk), (short)0,
                                             (uint32_t)(kb < 0xffffffffll ? kb : 0xffffffffll),
                                             kRsrcWord3);
  };
  auto load_direct = [&](int kt, auto buf_c) {
#if defined(__HIP_DEVICE_COMPILE__)
    const int buf = (int)buf_c;
    typedef __attribute__((address_space(3))) void lds_t;
    const int key0 = kt * AT_BN;
    const __amdgpu_buffer_rsrc_t kr = k_rsrc(key0);
    const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<T*>(vbase + key0), (short)0, (uint32_t)(v_bytes - (int64_t)key0 * ES), kRsrcWord3);
#pragma unroll
    for (int j = 0; j < KI; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (lds_t*)&kbuf(buf)[(j * W + wave) * KRPI][0], 16,
                                               kd_off[j], 0, 0, 0);
#pragma unroll
    for (int j = 0; j < VI; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_t*)&vbuf(buf)[(j * W + wave) * VRPI][0], 16,
                                               vd_off[j], 0, 0, 0);
#endif
  };
  // one direct-to-LDS instruction j of tile kt (j < KI: K rows, else V^T
  // rows), LDS address from the wave index in an SGPR
  [[maybe_unused]] const int wave_s = __builtin_amdgcn_readfirstlane(wave) & (W - 1);   // (known range 0..W-1)
  // (full tiles only -- the key-tail tile goes through registers -- so the
  // descriptors span exactly the tile: every access is inside it)
  const uint32_t k_tile_bytes = (uint32_t)(AT_BN * p.ldk * ES);
  const uint32_t v_tile_bytes = (uint32_t)(DH * p.ldvt * ES);
  auto load_one = [&](int kt, int buf, int j) __attribute__((always_inline)) {
#if defined(__HIP_DEVICE_COMPILE__)
    typedef __attribute__((address_space(3))) void lds_t;
    if (j < KI) {
      const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<T*>(kbase) + (uint64_t)(uint32_t)kt * (AT_BN * (uint64_t)p.ldk), (short)0, k_tile_bytes,
          kRsrcWord3);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (lds_t*)&kbuf(buf)[(j * W + wave_s) * KRPI][0], 16,
                                               kd_off[j], 0, 0, 0);
    } else {
      const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<T*>(vbase) + (uint32_t)kt * AT_BN, (short)0, v_tile_bytes, kRsrcWord3);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_t*)&vbuf(buf)[((j - KI) * W + wave_s) * VRPI][0], 16,
                                               vd_off[j - KI], 0, 0, 0);
    }
#endif
  };
  auto load_tail = [&](int kt, auto buf_c) {
    const int buf = (int)buf_c;
    const int key0 = kt * AT_BN;
    const __amdgpu_buffer_rsrc_t kr = k_rsrc(key0);
#pragma unroll
    for (int i = 0; i < K_PER_T; ++i) {
      const int id = tid + THREADS * i;
      const int kl = id / KCH, c = id % KCH;
      const u32x4 v = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(kr, (uint32_t)((kl * p.ldk + c * VEC) * ES), 0, 0));
      const int row = (kl & ~31) + key_slot(kl & 31);
      kbuf(buf)[row][swz<KCH>(row, c)] = v;
    }
#pragma unroll
    for (int i = 0; i < V_PER_T; ++i) {
      const int id = tid + THREADS * i;
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
      vbuf(buf)[d][swz<VCH>(d, c)] = v;
    }
  };
  auto load_tile = [&](int kt, auto buf_c) {
    if ((kt + 1) * AT_BN <= p.Lk) load_direct(kt, buf_c);
    else load_tail(kt, buf_c);
  };

  f32x16 o[2][DH / 32];
#pragma unroll
  for (int gr = 0; gr < 2; ++gr)
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[gr][dt][r] = 0.f;
#pragma unroll
  for (int gr = 0; gr < 2; ++gr)
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt) g2::pin_a(o[gr][dt]);
  float l_run[2] = {0.f, 0.f}, m_run[2];
  f32x16 negm[2], s[2];
  u32x4 kf[NQS], vf[8];
  u32x4 pc[2][2];
  const float uscale = SC ? 1.f : p.c;

  // (buf: a compile-time buffer, or a run-time one for the last tile)
  auto read_k = [&](auto buf_c, int kk, int i) __attribute__((always_inline)) {
    const int buf = (int)buf_c;
    kf[i] = g2::lds_read(&kbuf(buf)[kk * 32 + col][swz<KCH>(col, 2 * i + g)]);
  };
  // fragment i = 4 u + dt: head dims [32 dt, 32 dt + 32), keys 8 u.. of the lane group's 16
  auto read_v = [&](auto buf_c, int kk, int i) __attribute__((always_inline)) {
    const int buf = (int)buf_c;
    const int u = i >> 2, dt = i & 3;
    vf[i] = g2::lds_read(&vbuf(buf)[dt * 32 + col][swz<VCH>(col, (kk * 32 + 16 * g) / VEC + u)]);
  };
  auto mask = [&](f32x16& x, int key) {   // keys >= Lk -> -inf
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (key + 16 * g + r >= p.Lk) x[r] = -INFINITY;
  };
  // softmax pieces of group gr: exponential of score e, then per 8-key chunk
  // u the packed P^T operand and the chunk's probability sum
  float pe[2][16];
  float lsum[2][2];
  float ta[2][2][4], tb[2][2][2];   // the row-sum tree of each 8-key chunk
  float lh[2];                        // the half's probability sum
  // Group gr's softmax pieces issued after MFMA k (0..15) of a block: the
  // exponentials e0..e7 two per slot in slots 0-3 and e8..e15 one per slot
  // in 4-11; each bf16 pair of the P^T operand and each add of the chunk
  // sums ((e0+e4)+(e2+e6)) + ((e1+e5)+(e3+e7)) one slot after its last
  // input, so the half's sum is ready when the block ends (its test then
  // does not wait on a chain of adds) -- at most five VALU instructions
  // between two MFMAs.
  auto sm_slot = [&](int gr, int k) __attribute__((always_inline)) {
    auto es = [](int e) { return e < 12 ? e >> 1 : e - 6; };   // slot of exponential e
#pragma unroll
    for (int e = 0; e < 16; ++e)
      if (es(e) == k) {
        float x = s[gr][e];
        if constexpr (!SC) x *= uscale;
        pe[gr][e] = __builtin_amdgcn_exp2f(x);
        g2::pin(pe[gr][e]);
      }
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (es(2 * j + 1) + 1 == k) {
        bf16x2 v2 = {(bf16)pe[gr][2 * j], (bf16)pe[gr][2 * j + 1]};
        pc[gr][j >> 2][j & 3] = __builtin_bit_cast(uint32_t, v2);
        g2::pin(pc[gr][j >> 2]);
      }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (es(8 * u + q + 4) + 1 == k) {
          ta[gr][u][q] = pe[gr][8 * u + q] + pe[gr][8 * u + q + 4];
          g2::pin(ta[gr][u][q]);
        }
      const int b0 = es(8 * u + 6) + 2, b1 = es(8 * u + 7) + 2;
      if (b0 == k) {
        tb[gr][u][0] = ta[gr][u][0] + ta[gr][u][2];
        g2::pin(tb[gr][u][0]);
      }
      if (b1 == k) {
        tb[gr][u][1] = ta[gr][u][1] + ta[gr][u][3];
        g2::pin(tb[gr][u][1]);
      }
      if ((b0 > b1 ? b0 : b1) + 1 == k) {
        lsum[gr][u] = tb[gr][u][0] + tb[gr][u][1];
        g2::pin(lsum[gr][u]);
      }
    }
    if (k == 13) {
      lh[gr] = lsum[gr][0] + lsum[gr][1];
      g2::pin(lh[gr]);
    }
  };
  auto sm_exp = [&](int gr, int e) __attribute__((always_inline)) {
    float x = s[gr][e];
    if constexpr (!SC) x *= uscale;
    pe[gr][e] = __builtin_amdgcn_exp2f(x);
    g2::pin(pe[gr][e]);
  };
  auto sm_pack = [&](int gr, int u) __attribute__((always_inline)) {
    pc[gr][u] = Chunk<T>::pack(&pe[gr][8 * u]);
    float t[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) t[e] = pe[gr][8 * u + e];
#pragma unroll
    for (int w = VEC / 2; w > 0; w /= 2)
#pragma unroll
      for (int e = 0; e < w; ++e) t[e] += t[e + w];
    lsum[gr][u] = t[0];
    g2::pin(pc[gr][u]);
    g2::pin(lsum[gr][u]);
  };
  // Lazy rescale of group gr after its half's probabilities (see the
  // eight-wave kernel): rare; it reads and rewrites the AGPR accumulators.
  auto sm_check = [&](int gr) __attribute__((always_inline)) {
    if (__builtin_expect(__any(!(lh[gr] <= (float)(1 << (int)kSlack))), 0)) {
      g2::mfma_drain();
      float mx = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[gr][r]);
      const float d = fmaxf(fmaxf(mx, __shfl_xor(mx, 32)) * uscale, 0.f);
      const float alpha = __builtin_amdgcn_exp2f(-d);
      l_run[gr] *= alpha;
      // one accumulator at a time (16 registers through the VALU)
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt) {
        g2::pin_a(o[gr][dt]);   // its reads cannot move above this point
#pragma unroll
        for (int r = 0; r < 16; ++r) o[gr][dt][r] *= alpha;
        g2::pin_a(o[gr][dt]);
      }
      const float dm = d / uscale;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[gr][r] -= dm;
        negm[gr][r] -= dm;
      }
      m_run[gr] += d;
#pragma unroll
      for (int e = 0; e < 16; ++e) sm_exp(gr, e);
      sm_pack(gr, 0);
      sm_pack(gr, 1);
      lh[gr] = lsum[gr][0] + lsum[gr][1];
      g2::pin(negm[gr]);
      g2::pin(pc[gr][0]);
      g2::pin(pc[gr][1]);
      g2::valu_to_mfma();
    }
    l_run[gr] += lh[gr];
  };

  // ---- prologue: tiles t0 .. t0+NBUF-2 in flight, the base m of each group
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  load_tile(t0, I0{});
  load_tile(t0 + 1, I1{});
  wait_vmcnt<0>();
  __syncthreads();
  {
#pragma unroll
    for (int i = 0; i < NQS; ++i) read_k(I0{}, 0, i);
#pragma unroll
    for (int gr = 0; gr < 2; ++gr) {
      g2::mma_s0(s[gr], kf[0], qf[gr][0]);
#pragma unroll
      for (int i = 1; i < NQS; ++i) g2::mma_s(s[gr], kf[i], qf[gr][i]);
    }
    g2::mfma_drain();
#pragma unroll
    for (int gr = 0; gr < 2; ++gr) {
      if (t0 * AT_BN + 32 > p.Lk) mask(s[gr], t0 * AT_BN);
      float mx = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[gr][r]);
      m_run[gr] = fmaxf(mx, __shfl_xor(mx, 32)) * uscale;
#pragma unroll
      for (int r = 0; r < 16; ++r) negm[gr][r] = -m_run[gr] / uscale;
    }
    // (the pins keep the VALU writes of negm ahead of the wait states)
    g2::pin(negm[0]);
    g2::pin(negm[1]);
    g2::valu_to_mfma();
    // S(t0, 0, g0) against the base
    g2::mma_sc(s[0], kf[0], qf[0][0], negm[0]);
#pragma unroll
    for (int i = 1; i < NQS; ++i) g2::mma_s(s[0], kf[i], qf[0][i]);
  }

  // X(t, H): S(t,H,g1), then O1 += V^T P(prev, g1); softmax of S(t,H,g0).
  // NEXT: a next half exists (its K fragments are read here); FIRST: no
  // previous half (t = t0, H = 0).
  auto blockX = [&](int t, auto buf_c, auto h_c, auto next_c, auto first_c, auto masked_c) __attribute__((always_inline)) {
    constexpr bool MASKED = decltype(masked_c)::value;
    constexpr int H = decltype(h_c)::value;
    constexpr bool NEXT = decltype(next_c)::value;
    constexpr bool FIRST = decltype(first_c)::value;
    const auto Bc = buf_c;
    const int key0 = t * AT_BN + H * 32;
    // H = 1 with a next tile: the tile barrier, then tile t+NBUF-1 is loaded
    // into tile t-1's buffer.  With a compile-time buffer the eight loads go
    // one behind each score MFMA, unconditionally: past the range (or for
    // the key-tail tile, which is then rewritten through registers) they
    // load the last full tile into the free buffer.
    constexpr bool CT = !std::is_integral<decltype(buf_c)>::value;
    constexpr bool LOADS = H == 1 && NEXT;
    const int lt = t + NBUF - 1;
    const int lbuf = ((int)buf_c + NBUF - 1) % NBUF;
    const int nfull = p.Lk / AT_BN;
    if constexpr (FIRST) {
      // S(t0,0,g0) was just computed: wait out the MFMA pipeline
      g2::mfma_drain();
#pragma unroll
      for (int i = 0; i < 8; ++i) read_v(Bc, H, i);
    }
    if constexpr (MASKED) {
      if (key0 + 32 > p.Lk) mask(s[0], key0);
    }
    __builtin_amdgcn_sched_barrier(0);
    // score and output MFMAs alternate, so no MFMA waits on the one before it
#pragma unroll
    for (int i = 0; i < NQS; ++i) {
      if (i == 0) g2::mma_sc(s[1], kf[0], qf[1][0], negm[1]);
      else g2::mma_s(s[1], kf[i], qf[1][i]);
      if constexpr (LOADS) {
        if (i == 0) {
          // (the first score MFMA reads no LDS and runs under the barrier)
          // tile t+1 landed (own loads) and every read of tile t-1 done
          __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (0 << 8));   // vmcnt(0) lgkmcnt(0)
          asm volatile("" ::: "memory");
          __builtin_amdgcn_s_barrier();
          if constexpr (!CT) {
            if (lt < t1) load_tile(lt, lbuf);
          }
        }
      }
      if constexpr (NEXT) {
        if constexpr (H == 0) read_k(Bc, 1, i);
        else read_k(((int)buf_c + 1) % NBUF, 0, i);   // tile t+1's buffer
      }
      if constexpr (LOADS && CT) load_one(min(lt, nfull - 1), lbuf, i);
      sm_slot(0, 2 * i);
      // group 0's test, before the last MFMA (group 1's: a rescale of
      // group 0 leaves it alone)
      if (i == 7) sm_check(0);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (!FIRST) {
        if (i == 0) g2::mma_o_first(o[1][i & 3], vf[i], pc[1][i >> 2]);
        else g2::mma_o(o[1][i & 3], vf[i], pc[1][i >> 2]);
        read_v(Bc, H, i);
      }
      sm_slot(0, 2 * i + 1);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (LOADS && CT) {
      if (lt < t1 && (lt + 1) * AT_BN > p.Lk) {   // the key-tail tile, once
        wait_vmcnt<0>();
        load_tail(lt, lbuf);
      }
    }
    // (without output MFMAs behind them, the scores of g1 need the drain)
    if constexpr (FIRST) g2::mfma_drain();
  };
  // Y(t, H): S(next, g0), then O0 += V^T P(t,H,g0); softmax of S(t,H,g1).
  auto blockY = [&](int t, auto buf_c, auto h_c, auto next_c, auto masked_c) __attribute__((always_inline)) {
    constexpr bool MASKED = decltype(masked_c)::value;
    constexpr bool NEXT = decltype(next_c)::value;
    constexpr int H = decltype(h_c)::value;
    const int key0 = t * AT_BN + H * 32;
    if constexpr (MASKED) {
      if (key0 + 32 > p.Lk) mask(s[1], key0);
    }
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (NEXT) {
#pragma unroll
      for (int i = 0; i < NQS; ++i) {
        if (i == 0) g2::mma_sc(s[0], kf[0], qf[0][0], negm[0]);
        else g2::mma_s(s[0], kf[i], qf[0][i]);
        sm_slot(1, 2 * i);
        if (i == 7) sm_check(1);   // (the last MFMA is group 0's)
        __builtin_amdgcn_sched_barrier(0);
        if (i == 0) g2::mma_o_first(o[0][i & 3], vf[i], pc[0][i >> 2]);
        else g2::mma_o(o[0][i & 3], vf[i], pc[0][i >> 2]);
        sm_slot(1, 2 * i + 1);
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        if (i == 0) g2::mma_o_first(o[0][i & 3], vf[i], pc[0][i >> 2]);
        else g2::mma_o(o[0][i & 3], vf[i], pc[0][i >> 2]);
        sm_slot(1, 2 * i);
        sm_slot(1, 2 * i + 1);
        __builtin_amdgcn_sched_barrier(0);
      }
      sm_check(1);
    }
  };
  using TF = std::true_type;
  using FF = std::false_type;
  auto tile = [&](int t, auto buf_c, auto last_c) __attribute__((always_inline)) {
    constexpr bool LAST = decltype(last_c)::value;
    // only the last tile of the range can end past Lk
    blockX(t, buf_c, I0{}, TF{}, FF{}, last_c);
    blockY(t, buf_c, I0{}, TF{}, last_c);
    blockX(t, buf_c, I1{}, std::integral_constant<bool, !LAST>{}, FF{}, last_c);
    blockY(t, buf_c, I1{}, std::integral_constant<bool, !LAST>{}, last_c);
  };

  // first tile (its first block has no previous half)
  blockX(t0, I0{}, I0{}, TF{}, TF{}, FF{});
  blockY(t0, I0{}, I0{}, TF{}, FF{});
  blockX(t0, I0{}, I1{}, TF{}, FF{}, FF{});
  blockY(t0, I0{}, I1{}, TF{}, FF{});
  // middle tiles t0+1 .. t1-2 in ring order (buffers 1, 2, .., 0, 1, ..), in
  // groups of NBUF with compile-time buffers; the few left over and the last
  // tile take their buffer as a run-time value (there the compiler waits for
  // in-flight tile loads before each LDS read: a few tiles per workgroup)
  int t = t0 + 1;
  for (; t + NBUF < t1; t += NBUF) {
    tile(t, I1{}, FF{});
    tile(t + 1, I2{}, FF{});
    tile(t + 2, I0{}, FF{});
  }
  for (; t + 1 < t1; ++t) tile(t, (t - t0) % NBUF, FF{});
  tile(t, (t - t0) % NBUF, TF{});
  wait_vmcnt<0>();   // (loads past the range must land before the workgroup ends)
  // drain: O1 += V^T P(last half, g1)
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    if (i == 0) g2::mma_o_first(o[1][i & 3], vf[i], pc[1][i >> 2]);
    else g2::mma_o(o[1][i & 3], vf[i], pc[1][i >> 2]);
  }
  g2::mfma_drain();
  // negm is the accumulator input of the last score MFMAs: live until the
  // drain, so its registers are not rewritten while they may be read
  g2::pin(negm[0]);
  g2::pin(negm[1]);

  if (split >= 0) {
    const int nsplit = (int)(gridDim.x - p.nreg) / 2;
#pragma unroll
    for (int gr = 0; gr < 2; ++gr) {
      const int ql = wave * 64 + gr * 32 + col;
      const float l = l_run[gr] + __shfl_xor(l_run[gr], 32);
      float* po = p.part + part_o_off<DH>(split >> 1, split & 1, ql, BMQ);
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          f32x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = o[gr][dt][4 * rr + e];
          *reinterpret_cast<f32x4*>(po + dt * 32 + 8 * rr + 4 * g) = v;
        }
      if (g == 0) {
        float* pml = p.part + part_ml_off<DH>(nsplit, split >> 1, split & 1, ql, BMQ);
        pml[0] = m_run[gr];
        pml[1] = l;
      }
    }
    return;
  }
  // Output rows through LDS: once every wave is past its last fragment
  // reads, each wave stages its 64 rows in a 16 KB ring slot of its own.
  __syncthreads();
  char* stage = reinterpret_cast<char*>(wave == 0   ? &ks0_[0][0]
                                        : wave == 1 ? &ks1_[0][0]
                                        : wave == 2 ? &ks2_[0][0]
                                                    : &vs0_[0][0]);
#pragma unroll
  for (int gr = 0; gr < 2; ++gr) {
    const int q0 = qb * BMQ + wave * 64 + gr * 32;
    const float l = l_run[gr] + __shfl_xor(l_run[gr], 32);
    store_rows_staged<T, DH>(o[gr], 1.f / l, stage + gr * 32 * DH * (int)sizeof(T),
                             p.O + ((int64_t)b * p.Lq + q0) * p.ldo + h * DH, p.ldo,
                             min(32, p.Lq - q0), lane);
  }
}

template <bool SC>
void launch_g2(AttnParams<bf16> p, hipStream_t stream, int ncu) {
  constexpr int BMQ = 256;
  const int items = ((p.Lq + BMQ - 1) / BMQ) * p.H * p.B;
  const int rem = ncu > 0 ? items % ncu : 0;
  const int nfull = p.Lk / AT_BN;
  int nsplit = 0;
  if (p.part && rem > 0 && 2 * rem <= ncu && rem <= kMaxSplitItems && nfull >= 4) nsplit = rem;
  p.nreg = items - nsplit;
  p.split_tile = (nfull / 2) & ~1;
  hipLaunchKernelGGL((flash_attn_g2_kernel<SC>), dim3(p.nreg + 2 * nsplit), dim3(256), 0, stream, p);
  if (nsplit > 0)
    hipLaunchKernelGGL((attn_merge_kernel<bf16, 128, BMQ>), dim3(nsplit), dim3(256), 0, stream, p, nsplit);
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
      if constexpr (DH == 128) {
        if (q_scaled) launch_g2<true>(p, stream, ncu);
        else launch_g2<false>(p, stream, ncu);
      } else {
        launch_w<T, DH, 8>(p, q_scaled, stream, ncu);
      }
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

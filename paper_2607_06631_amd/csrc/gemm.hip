// GEMM C = epi(A B^T) on MFMA for gfx950.
//
// Both operands are K-contiguous (nn.Linear layout), which is exactly the
// per-lane layout the MFMA operands want: every lane feeds a 16-byte run of
// consecutive k. Workgroup tile 256 x 256 (128 x 128 for small problems),
// k-tile 128 bytes per row (64 bf16 / 32 f32), split over a grid of waves
// that each own a block of 32x32 output blocks (bf16: four 16x16x32 MFMA
// tiles each; f32: one 32x32x2 tile). Operand tiles are copied
// global -> LDS by buffer loads that write LDS directly (no staging
// registers, no LDS store instructions), double-buffered (2 x 64 KB of the
// 160 KB LDS at 256 x 256): tile kt+1 is requested while tile kt is
// computed. The 16-byte chunks of each row are XOR-swizzled (swz) so the
// 32-row fragment reads are bank-conflict free; each lane fetches the chunk
// that the swizzle places in the LDS slot its load writes. Ragged M and N:
// rows past the matrix read as zero through the descriptor bounds and
// stores are predicated; K must be a multiple of the k-tile (the plan pads
// pruned widths to 64).
//
// Index-table gather (the step's active parameters read in place from the
// union weight set, no compacted copy):
//   GA_ROWS  output column n uses B row rows[n] (-1: a zero row); the bias
//            is gathered the same way.  Used where whole heads or FFN
//            channels are dropped from the output width.
//   GA_KCH   16-byte K chunk c of every B row is read from chunk kch[c] of
//            that row (-1: zeros).  Used where dropped heads or FFN chunks
//            shorten the reduction.  The chunk table is staged in LDS once.
// Masked rows / chunks get an offset past the descriptor's range, which the
// buffer load returns as zero.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace dif {
// Fragment k of a k-step in the order its MFMAs first use them (MFMA i
// multiplies A row block i / TN by B column block i % TN): the value is a
// row block index (< TM) or TM + a column block index.  For 4 x 2 blocks:
// A0 B0 B1 A1 A2 A3.
// (a table built at compile time: indexing it with an unrolled loop's
// counter gives constants, so the fragment arrays stay in registers)
template <int TM, int TN>
struct FirstUse {
  int v[TM + TN];
};
template <int TM, int TN>
__host__ __device__ constexpr FirstUse<TM, TN> first_use_table() {
  FirstUse<TM, TN> t{};
  bool seen[TM + TN] = {};
  int n = 0;
  for (int i = 0; i < TM * TN; ++i) {
    const int a = i / TN, b = TM + i % TN;
    if (!seen[a]) {
      seen[a] = true;
      t.v[n++] = a;
    }
    if (!seen[b]) {
      seen[b] = true;
      t.v[n++] = b;
    }
  }
  return t;
}

constexpr int G_BKC = 8;    // 16-byte chunks per k-tile row (128 bytes)
constexpr int BN_MAX = 256; // largest workgroup tile width over the shapes below

enum { GA_NONE = 0, GA_ROWS = 1, GA_KCH = 2 };
constexpr uint32_t kMasked = 0x80000000u;  // buffer offset beyond any descriptor range

// Up to three B matrices ("segments", e.g. the q, k and v weights) share A
// and one launch; segment s writes output columns [s*N, (s+1)*N).
constexpr int kMaxSeg = 3;

template <typename T, typename OutT>
struct GemmParams {
  const T* A;
  const T* Bs[kMaxSeg];
  OutT* C;
  int64_t lda, ldb, ldc;
  int M, N, K;
  const float* biases[kMaxSeg];
  int nseg;
  const float* gate0;
  const float* gate1;
  const int32_t* rows;   // GA_ROWS
  const int32_t* kch;    // GA_KCH
  int b_rows;            // GA_ROWS: rows of the union B matrix
  int vec4;              // C rows allow aligned 4-element accesses
  // transposed output: columns from output column vt_col0 on go to
  // vt[(b * vt_dims + col - vt_col0) * ldvt + j] for row m = b * vt_L + j
  OutT* vt;
  int64_t ldvt;
  int vt_col0, vt_dims, vt_L;
  int vt_vec4;           // vt rows allow aligned 4-element stores and vt_L % 4 == 0
};

// four consecutive output elements: 8-byte (bf16) or 16-byte (f32) accesses
__device__ __forceinline__ void load4(const bf16* p, float* v) {
  const bf16x4 x = *reinterpret_cast<const bf16x4*>(p);
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = (float)x[e];
}
__device__ __forceinline__ void load4(const float* p, float* v) {
  const f32x4 x = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = x[e];
}
__device__ __forceinline__ void store4(bf16* p, const float* v) {
  bf16x4 x;
#pragma unroll
  for (int e = 0; e < 4; ++e) x[e] = (bf16)v[e];
  *reinterpret_cast<bf16x4*>(p) = x;
}
__device__ __forceinline__ void store4(float* p, const float* v) {
  f32x4 x;
#pragma unroll
  for (int e = 0; e < 4; ++e) x[e] = v[e];
  *reinterpret_cast<f32x4*>(p) = x;
}

// WGM x WGN waves; each wave owns TM x TN 32x32 output blocks; two LDS stages
// of BKC 16-byte chunks per operand row.
template <typename T, typename OutT, int EPI, int GA, int WGM, int WGN, int TM, int TN, int BKC>
__global__ __launch_bounds__(64 * WGM * WGN, 8 / (WGM * WGN)) void gemm_nt_kernel(GemmParams<T, OutT> p) {
  constexpr int NW = WGM * WGN;
  constexpr int NT = 64 * NW;
  constexpr int BM = WGM * TM * 32, BN = WGN * TN * 32;
  constexpr int VEC = Chunk<T>::VEC;
  constexpr int BK = BKC * VEC;
  constexpr int RPI = 64 / BKC;           // rows filled by one wave load instruction (1 KB)
  // Eight waves: waves 0..3, the older wave of each SIMD pair, issue all of
  // a tile's loads.  The older wave wins the SIMD's issue arbitration and
  // finishes its share of a k-tile first; the loads' issue time then comes
  // off the younger wave, which ends each k-tile (measured 4.7% on the
  // step's five projection shapes).
  constexpr int NLW = NW == 8 ? 4 : NW;   // loading waves
  constexpr int LA = BM / (RPI * NLW), LB = BN / (RPI * NLW);
  constexpr int LPT = LA + LB;            // loads per thread per k-tile
  static_assert(LA * RPI * NLW == BM && LB * RPI * NLW == BN, "staging split");
  __shared__ u32x4 smem[2][BM + BN][BKC];
  static_assert(sizeof(smem) >= (size_t)NW * 64 * 64 * sizeof(float), "epilogue staging");
  extern __shared__ uint32_t kch_lds[];   // GA_KCH: byte offset of each K chunk

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int g = lane >> 5, col = lane & 31;
  // bf16: each 32 x 32 block of the wave is four 16 x 16 MFMA tiles
  // (v_mfma_f32_16x16x32_bf16, k 32 per instruction): at the same operand
  // bytes per flop it draws less power than the 32 x 32 x 16 form, and the
  // chip holds a higher clock under it (2.03 against 1.75 PFLOP/s sustained
  // with every CU issuing nothing else; here 1.83-2.04 against 1.57-1.71
  // GHz, +1 % per step: the tile loads, not the matrix units, bound the
  // k-loop).  float32 keeps 32 x 32 x 2, and so does the row-gathered B
  // (its eight per-instruction row offsets would not fit beside the
  // 16 x 16 schedule's registers).
  constexpr bool M16 = std::is_same<T, bf16>::value && GA != GA_ROWS;

  // logical tile: XCD-contiguous ranges, then groups of GM row-tiles that
  // walk the N tiles of all segments together (operand reuse in L2)
  const int nbm = (p.M + BM - 1) / BM, nbn = (p.N + BN - 1) / BN;
  const int nbv = nbn * p.nseg;
  const int bid = xcd_remap(blockIdx.x, nbm * nbv);
  constexpr int GM = 8;
  const int group = bid / (GM * nbv);
  const int first_m = group * GM;
  const int gsize = min(nbm - first_m, GM);
  const int in_group = bid - group * GM * nbv;
  const int m0 = (first_m + in_group % gsize) * BM;
  const int nt = in_group / gsize;
  const int sg = nt / nbn;
  const int n0 = (nt - sg * nbn) * BN;
  const T* Bsg = p.Bs[sg];
  const float* bias_sg = p.biases[sg];
  OutT* Csg = p.C + (int64_t)sg * p.N;

  // global -> LDS staging with buffer loads against block-local
  // descriptors; rows past M / N fall outside the descriptor and read as
  // zero.
  constexpr uint32_t kRsrcWord3 = 0x00020000u;
  const uint32_t a_bytes = (uint32_t)(min(BM, p.M - m0) * p.lda * (int64_t)sizeof(T));
  // GA_ROWS: one descriptor over the whole union matrix, rows picked per thread
  const uint32_t b_bytes =
      GA == GA_ROWS ? (uint32_t)((int64_t)p.b_rows * p.ldb * (int64_t)sizeof(T))
                    : (uint32_t)(min(BN, p.N - n0) * p.ldb * (int64_t)sizeof(T));
  const T* b_base = GA == GA_ROWS ? Bsg : Bsg + (int64_t)n0 * p.ldb;
  const __amdgpu_buffer_rsrc_t a_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<T*>(p.A + (int64_t)m0 * p.lda), (short)0, a_bytes, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t b_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(b_base), (short)0, b_bytes, kRsrcWord3);
  // lane offsets of load instruction i: the first one's plus i times a
  // row stride, added when the load issues (kept whole in the vector offset,
  // which the descriptor's range check covers), except for gathered B rows,
  // which need one per instruction
  constexpr int LBV = GA == GA_ROWS ? LB : 1;
  uint32_t a_off[1], b_off[LBV];
  const uint32_t a_step = (uint32_t)(NLW * RPI * p.lda * (int64_t)sizeof(T));
  const uint32_t b_step = (uint32_t)(NLW * RPI * p.ldb * (int64_t)sizeof(T));
  // direct-to-LDS: instruction i of loading wave lw fills LDS rows
  // (i*NLW + lw)*RPI .. +RPI (1 KB); lane l writes 16 bytes at 16*l, i.e. row
  // +l/BKC, physical chunk l%BKC, and fetches the logical chunk the swizzle
  // places there.  The swizzle depends on row bits 0..3 only, which are
  // l/BKC's (RPI = 16) or l/BKC's and lw's parity (RPI = 8): one logical
  // chunk for all i.
  static_assert(RPI == 16 || (RPI == 8 && NLW % 2 == 0), "direct staging layout");
  const int lw = wave % NLW;
  const bool loader = wave < NLW;
  auto drow = [&](int i) { return (i * NLW + lw) * RPI + lane / BKC; };
  const int dchunk = swz<BKC>(drow(0), lane % BKC);
  a_off[0] = (uint32_t)((drow(0) * p.lda + dchunk * VEC) * (int64_t)sizeof(T));
#pragma unroll
  for (int i = 0; i < LBV; ++i) {
    if constexpr (GA == GA_ROWS) {
      const int n = n0 + drow(i);
      const int r = n < p.N ? p.rows[n] : -1;
      b_off[i] = r >= 0 ? (uint32_t)((r * p.ldb + dchunk * VEC) * (int64_t)sizeof(T)) : kMasked;
    } else if constexpr (GA == GA_KCH) {
      b_off[i] = (uint32_t)(drow(i) * p.ldb * (int64_t)sizeof(T));
    } else {
      b_off[i] = (uint32_t)((drow(i) * p.ldb + dchunk * VEC) * (int64_t)sizeof(T));
    }
  }
  const int nk = p.K / BK;
  if constexpr (GA == GA_KCH) {
    for (int c = tid; c < p.K / VEC; c += NT) {
      const int u = p.kch[c];
      kch_lds[c] = u >= 0 ? (uint32_t)u * 16u : kMasked;
    }
    __syncthreads();
  }

  uint32_t kb = 0;   // GA_KCH: byte offset of this lane's chunk in the next tile to issue
  auto kb_fetch = [&](int kt) {
    if constexpr (GA == GA_KCH) {
      if (kt < nk) kb = kch_lds[kt * BKC + dchunk];
    }
  };
  typedef __attribute__((address_space(3))) void lds_t;
  // load u (0 .. LPT-1) of this loading wave's share of tile kt into stage
  // st: A rows, then B rows (LDS destinations from a scalar wave index)
  const int lw_s = __builtin_amdgcn_readfirstlane(lw);
  auto issue_one = [&](int kt, int u, auto st_c) {
#if defined(__HIP_DEVICE_COMPILE__)
    constexpr int st = decltype(st_c)::value;
    const int koff = kt * BK * (int)sizeof(T);
    // (opaque copies: the per-instruction offsets are formed here, not
    // hoisted out of the k-loop into registers of their own)
    uint32_t a0 = a_off[0], b0 = b_off[0];
    asm volatile("" : "+v"(a0), "+v"(b0));
    if (u < LA) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(a_rsrc, (lds_t*)&smem[st][(u * NLW + lw_s) * RPI][0],
                                               16, a0 + u * a_step, koff, 0, 0);
    } else {
      const int i = u - LA;
      lds_t* dst = (lds_t*)&smem[st][BM + (i * NLW + lw_s) * RPI][0];
      if constexpr (GA == GA_KCH)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(b_rsrc, dst, 16, b0 + i * b_step + kb, 0, 0, 0);
      else if constexpr (GA == GA_ROWS)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(b_rsrc, dst, 16, b_off[i], koff, 0, 0);
      else
        __builtin_amdgcn_raw_ptr_buffer_load_lds(b_rsrc, dst, 16, b0 + i * b_step, koff, 0, 0);
    }
#endif
  };
  auto issue = [&](int kt) {
#pragma unroll
    for (int u = 0; u < LPT; ++u)
      if (loader) issue_one(kt, u, std::integral_constant<int, 0>{});
  };

  // accumulators: 32 x 32 blocks (float32) or 16 x 16 tiles (bf16), the same
  // 16 registers per 32 x 32 block either way
  constexpr int AM = M16 ? 2 * TM : TM, AN = M16 ? 2 * TN : TN;
  typedef typename std::conditional<M16, f32x4, f32x16>::type AccT;
  constexpr int AR = M16 ? 4 : 16;
  AccT acc[AM][AN];
#pragma unroll
  for (int i = 0; i < AM; ++i)
#pragma unroll
    for (int j = 0; j < AN; ++j)
#pragma unroll
      for (int r = 0; r < AR; ++r) acc[i][j][r] = 0.f;

  // MFMA operand fragments, double-buffered in registers: the fragments of
  // k-step ks+1 are read while the MFMAs of k-step ks issue, one read after
  // each MFMA, in the order k-step ks+1's MFMAs first use them.  Scheduling
  // barriers keep that order (left alone, the compiler sinks every read next
  // to its first use).
  // k-steps per k-tile: 16 k (32 x 32 x 16) or 32 k (16 x 16 x 32) each
  constexpr int KSN = M16 ? BKC / 4 : BKC / 2;
  static_assert(KSN % 2 == 0, "fragment slots alternate");
  // fragments: rows of 32 (lane % 32, chunk 2 ks + lane / 32) or of 16
  // (lane % 16, chunk 4 ks + lane / 16)
  constexpr int FR = M16 ? 16 : 32;
  u32x4 fa[M16 ? 1 : 2][AM], fb[M16 ? 1 : 2][AN];
  const int frow = M16 ? (lane & 15) : col;
  constexpr FirstUse<AM, AN> fu = first_use_table<AM, AN>();
  // fragment read r (first_use order) of k-step ks of stage st into slot
  auto frag_one = [&](int st, int ks, int slot, int r) {
    const int c = M16 ? swz<BKC>(frow, 4 * ks + (lane >> 4)) : swz<BKC>(col, 2 * ks + g);
    // (rows are frow + multiples of 16, so the swizzle sees frow's bits)
    if (r < AM) fa[slot][r] = smem[st][wm * TM * 32 + r * FR + frow][c];
    else fb[slot][r - AM] = smem[st][BM + wn * TN * 32 + (r - AM) * FR + frow][c];
  };
  // One k-tile (stage st is compile-time, so fragment and load addresses are
  // constants plus immediate offsets): wait for this wave's loads of tile kt,
  // barrier (everyone's have landed and everyone is done with tile kt-1's
  // stage), compute tile kt while requesting tile kt+1 into that stage.  Half
  // of the loads go out before the first k-step and half after its MFMAs:
  // issued in one burst, or spread over the k-steps, they measured slower.
  if (nk > 0) {
    kb_fetch(0);
    issue(0);
    kb_fetch(1);
  }
  auto ktile = [&](int kt, auto st_c) {
    constexpr int st = decltype(st_c)::value;
    using NS = std::integral_constant<int, st ^ 1>;
    const bool more = kt + 1 < nk;
    wait_vmcnt<0>();
    __syncthreads();
    if (more && loader) {
#pragma unroll
      for (int u = 0; u < LPT / 2; ++u) issue_one(kt + 1, u, NS{});
    }
#pragma unroll
    for (int r = 0; r < AM + AN; ++r) frag_one(st, 0, 0, fu.v[r]);
#pragma unroll
    for (int ks = 0; ks < KSN; ++ks) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < AM * AN; ++i) {
        if constexpr (M16) {
          // Two halves over the B fragments (B 0..AN/2-1, then the rest),
          // each running through every A fragment, so every fragment is
          // read for the next k-step into its own registers right after its
          // last MFMA here (one register slot per fragment): the first
          // half's B after MFMA AM * AN / 2 - 1, A fragment a after its
          // second-half use, the second half's B after the last MFMA
          constexpr int HB = AN / 2;
          const int h = i / (AM * HB), a = (i % (AM * HB)) / HB, b = h * HB + i % HB;
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, fa[0][a]),
                                                              __builtin_bit_cast(bf16x8, fb[0][b]),
                                                              acc[a][b], 0, 0, 0);
          if (ks + 1 < KSN) {
            if (i == AM * HB - 1) {
#pragma unroll
              for (int bb = 0; bb < HB; ++bb) frag_one(st, ks + 1, 0, AM + bb);
            }
            if (h == 1 && i % HB == HB - 1) frag_one(st, ks + 1, 0, a);
            if (i == AM * AN - 1) {
#pragma unroll
              for (int bb = HB; bb < AN; ++bb) frag_one(st, ks + 1, 0, AM + bb);
            }
          }
        } else {
          Mma<T>::step(acc[i / AN][i % AN], fa[ks & 1][i / AN], fb[ks & 1][i % AN]);
          if (ks + 1 < KSN && i < AM + AN) frag_one(st, ks + 1, (ks + 1) & 1, fu.v[i]);
        }
        // the tile's second half of loads: after the first k-step's MFMAs
        // (32 x 32 x 16), or after its first eight (16 x 16 x 32: its k-steps
        // are half as many and the loads want the time to land; after the
        // whole k-step 3 % slower, all at the barrier 0.8 %)
        if (M16 && ks == 0 && i == 7 && more && loader) {
#pragma unroll
          for (int u = LPT / 2; u < LPT; ++u) issue_one(kt + 1, u, NS{});
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      if (!M16 && ks == 0 && more && loader) {
#pragma unroll
        for (int u = LPT / 2; u < LPT; ++u) issue_one(kt + 1, u, NS{});
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    kb_fetch(kt + 2);
  };
  {
    int kt = 0;
    for (; kt + 2 <= nk; kt += 2) {
      ktile(kt, std::integral_constant<int, 0>{});
      ktile(kt + 1, std::integral_constant<int, 1>{});
    }
    if (kt < nk) ktile(kt, std::integral_constant<int, 0>{});
  }
  __syncthreads();

  // Epilogue through LDS (the operand buffers are free after the last
  // barrier).  A lane holds one column of each 32x32 tile, so direct stores
  // would move two bytes per lane; instead each wave stages its block in
  // passes of 64 x 64 as float32 (bias added, GELU or the column gate
  // applied) in its own 16 KB of LDS, then moves rows of four consecutive
  // elements per lane: 16 lanes cover a 64-column row, so loads of the
  // residual and the stores are whole 128-byte (bf16) row segments.  The
  // staging layout flips column bit 5 every four rows, which keeps both the
  // column writes and the row reads free of bank conflicts.
  // A wave only reads back what it staged itself, and a wave's LDS
  // instructions execute in order, so between its writes and reads the
  // staging needs no workgroup barrier, only a wavefront-scope fence that
  // keeps the compiler from reordering them (and, unlike a barrier, does not
  // wait for the wave's outstanding residual loads).
  static_assert(TM % 2 == 0 && TN % 2 == 0, "epilogue passes of 64 x 64 per wave");
  float* stage = reinterpret_cast<float*>(&smem[0][0][0]) + wave * (64 * 64);
  auto wave_sync = [] {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };
  // Register r (0..15) of this lane's 32 x 32 block (i, j): its value and
  // its row and column inside the block.  32 x 32 x 16 layout: column
  // lane % 32, rows acc_row(r, lane / 32).  16 x 16 tiles (M16): tile
  // (r / 8, r / 4 % 2) of the block, row 4 (lane / 16) + r % 4 of it,
  // column lane % 16.  Registers 4q .. 4q+3 are four consecutive rows of
  // one column in both layouts.
  auto av = [&](int i, int j, int r) -> float {
    if constexpr (M16) return acc[2 * i + (r >> 3)][2 * j + ((r >> 2) & 1)][r & 3];
    else return acc[i][j][r];
  };
  auto arow = [&](int r) { return M16 ? 16 * (r >> 3) + 4 * (lane >> 4) + (r & 3) : acc_row(r, g); };
  auto acol = [&](int r) { return M16 ? 16 * ((r >> 2) & 1) + (lane & 15) : col; };
  // staging column flips: bit 5 every four rows (32 x 32: a lane group's
  // rows are 8 apart) or bits 4..5 by row bits 2..3 (16 x 16: the four lane
  // groups write rows 4 apart); both leave the row reads conflict-free
  auto sidx = [](int r, int c) {
    return M16 ? r * 64 + (c ^ (((r >> 2) & 3) << 4)) : r * 64 + (c ^ (((r >> 2) & 1) << 5));
  };
  // per-column bias and gate of the lane's columns: one per 32-column block,
  // or two (the two 16-column tiles) in the M16 layout
  constexpr int CS = M16 ? 2 : 1;
  float colv[TN][CS], gatev[TN][CS];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int cs = 0; cs < CS; ++cs) {
      const int n = n0 + wn * TN * 32 + j * 32 + acol(4 * cs);
      colv[j][cs] = 0.f;
      gatev[j][cs] = 1.f;
      if (n < p.N) {
        if constexpr (GA == GA_ROWS) {
          const int r = p.rows[n];
          if (bias_sg && r >= 0) colv[j][cs] = bias_sg[r];
        } else {
          if (bias_sg) colv[j][cs] = bias_sg[n];
        }
        if (EPI == EPI_RESIDUAL && p.gate0) gatev[j][cs] = p.gate0[n] + (p.gate1 ? p.gate1[n] : 0.f);
      }
    }
  // (register r's column set: r / 4 % 2 for M16)
  auto csel = [](int r) { return M16 ? ((r >> 2) & 1) : 0; };
  constexpr int NPASS = (TM / 2) * (TN / 2);
  // A tile whose columns start at or past vt_col0 stores transposed (the
  // host keeps vt_col0 on a tile or segment boundary, so this is uniform).
  if constexpr (EPI == EPI_STORE) {
    if (p.vt && sg * p.N + n0 >= p.vt_col0) {
      // staging [dim][token]: token bits 2.. are XORed with dim bits 0..3, so
      // each lane's 16-byte writes of four consecutive tokens of one dim and
      // the 16-byte reads of four consecutive tokens are both free of bank
      // conflicts
      auto tidx = [](int d, int t) { return d * 64 + (t ^ ((d & 15) << 2)); };
#pragma unroll
      for (int ps = 0; ps < NPASS; ++ps) {
        const int rb = ps / (TN / 2), ch = ps % (TN / 2);
#pragma unroll
        for (int ii = 0; ii < 2; ++ii)
#pragma unroll
          for (int jj = 0; jj < 2; ++jj) {
            const int i = 2 * rb + ii, j = 2 * ch + jj;
            // registers 4q .. 4q+3 hold four consecutive tokens of one dim:
            // one 16-byte write each
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              f32x4 v;
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = av(i, j, 4 * q + e) + colv[j][csel(4 * q)];
              *reinterpret_cast<f32x4*>(&stage[tidx(jj * 32 + acol(4 * q), ii * 32 + arow(4 * q))]) = v;
            }
          }
        wave_sync();
        const int q4 = lane & 15;                                    // 4-token group
        const int m = m0 + wm * TM * 32 + rb * 64 + 4 * q4;          // its first token
        const int bb = m / p.vt_L, jt = m - bb * p.vt_L;
        const bool full4 = p.vt_vec4 && m + 4 <= p.M;                // same sample, aligned
#pragma unroll
        for (int t = 0; t < 16; ++t) {
          const int dl = t * 4 + (lane >> 4);                        // dim within the pass
          const int n = n0 + wn * TN * 32 + ch * 64 + dl;
          const f32x4 sv = *reinterpret_cast<const f32x4*>(&stage[tidx(dl, 4 * q4)]);
          if (n >= p.N || m >= p.M) continue;
          const int dim = sg * p.N + n - p.vt_col0;
          float v[4] = {sv[0], sv[1], sv[2], sv[3]};
          if (full4) {
            store4(p.vt + ((int64_t)bb * p.vt_dims + dim) * p.ldvt + jt, v);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int me = m + e;
              if (me >= p.M) break;
              const int be = me / p.vt_L, je = me - be * p.vt_L;
              p.vt[((int64_t)be * p.vt_dims + dim) * p.ldvt + je] = from_f32<OutT>(v[e]);
            }
          }
        }
        if (ps + 1 < NPASS) wave_sync();
      }
      return;
    }
  }
  // Residual rows are requested ahead of the staging, every pass's rows up
  // front for bf16 output (in flight through all of the staging), pass by
  // pass for float output (whose rows would not fit in the registers left).
  // Loaded row by row next to the stores, each load would wait for the
  // previous row's store (the compiler cannot rule out that they overlap):
  // one memory round trip per row.
  typedef typename std::conditional<std::is_same<OutT, float>::value, f32x4, bf16x4>::type Out4;
  constexpr bool RES = EPI == EPI_RESIDUAL;
  constexpr int RES_AHEAD = RES && sizeof(Out4) == 8 ? NPASS : 1;
  Out4 xres[RES_AHEAD][RES ? 16 : 1];
  const __amdgpu_buffer_rsrc_t c_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      Csg + (int64_t)m0 * p.ldc, (short)0,
      (uint32_t)((int64_t)min(BM, p.M - m0) * p.ldc * (int64_t)sizeof(OutT)), kRsrcWord3);
  // unconditional buffer loads (an exact count of loads in flight lets the
  // staging wait only for the bias and gate): rows past M fall outside the
  // descriptor and lanes of the ragged path get an offset past it, both
  // reading zero
  auto load_res = [&](int ps, Out4* dst) {
    const int rb = ps / (TN / 2), ch = ps % (TN / 2);
    const int nb = n0 + wn * TN * 32 + ch * 64 + (lane & 15) * 4;
    const bool full4 = p.vec4 && nb + 4 <= p.N;
    // (a select, not a branch per load; kMasked plus a row offset inside the
    // tile stays past the descriptor, which the host keeps below kMasked)
    const uint32_t base = full4 ? (uint32_t)nb * (uint32_t)sizeof(OutT) : kMasked;
    const uint32_t row_bytes = (uint32_t)p.ldc * (uint32_t)sizeof(OutT);
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const int rt = wm * TM * 32 + rb * 64 + t * 4 + (lane >> 4);   // row within the tile
      const uint32_t off = base + (uint32_t)rt * row_bytes;
      if constexpr (sizeof(Out4) == 8)
        dst[t] = __builtin_bit_cast(Out4, __builtin_amdgcn_raw_buffer_load_b64(c_rsrc, off, 0, 0));
      else
        dst[t] = __builtin_bit_cast(Out4, __builtin_amdgcn_raw_buffer_load_b128(c_rsrc, off, 0, 0));
    }
  };
  if constexpr (RES && RES_AHEAD == NPASS) {
#pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) load_res(ps, xres[ps]);
  }
#pragma unroll
  for (int ps = 0; ps < NPASS; ++ps) {
    const int rb = ps / (TN / 2), ch = ps % (TN / 2);   // 64-row block, 64-column half
    const int cq = lane & 15;                          // 4-column chunk of the row
    const int nb = n0 + wn * TN * 32 + ch * 64 + cq * 4;
    const bool full4 = p.vec4 && nb + 4 <= p.N;
    if constexpr (RES && RES_AHEAD == 1) load_res(ps, xres[0]);
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int i = 2 * rb + ii, j = 2 * ch + jj;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float v = av(i, j, r) + colv[j][csel(r)];
          if (EPI == EPI_GELU) v = gelu_tanh(v);
          if (EPI == EPI_RESIDUAL) v *= gatev[j][csel(r)];
          stage[sidx(ii * 32 + arow(r), jj * 32 + acol(r))] = v;
        }
      }
    wave_sync();
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const int rl = t * 4 + (lane >> 4);              // row within the pass
      const int m = m0 + wm * TM * 32 + rb * 64 + rl;
      const f32x4 sv = *reinterpret_cast<const f32x4*>(&stage[sidx(rl, cq * 4)]);
      float v[4] = {sv[0], sv[1], sv[2], sv[3]};
      if (m >= p.M || nb >= p.N) continue;
      OutT* dst = Csg + (int64_t)m * p.ldc + nb;
      if (full4) {
        if constexpr (EPI == EPI_RESIDUAL) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] += (float)xres[RES_AHEAD == 1 ? 0 : ps][t][e];
        }
        store4(dst, v);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (nb + e < p.N) {
            if (EPI == EPI_RESIDUAL) v[e] += to_f32(dst[e]);
            dst[e] = from_f32<OutT>(v[e]);
          }
      }
    }
    if (ps + 1 < NPASS) wave_sync();   // reads done before the next pass overwrites
  }
}

// LDS left beside the two operand stages (2 x 512 rows x 128 B) for the
// K-chunk table
constexpr int kMaxKChunks = (160 * 1024 - 2 * 512 * G_BKC * 16) / 4;

// 256 x 256 workgroup tile as 8 waves (2 x 4) of 128 x 64.
constexpr int G_WGM = 2, G_WGN = 4, G_TM = 4, G_TN = 2;
// Store-epilogue problems with fewer 256 x 256 tiles than half the CUs (the
// 512 text tokens' K / V projection) take 128 x 128 tiles of 4 waves of
// 64 x 64 instead, two workgroups per CU: four times the workgroups.
constexpr int kSmallProblemTiles = 128;
template <typename T, typename OutT, int EPI, int GA, int WGM, int WGN, int TM, int TN>
void launch_cfg(const GemmParams<T, OutT>& p, hipStream_t stream) {
  constexpr int BM = WGM * TM * 32, BN = WGN * TN * 32;
  const int tiles = ((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN) * p.nseg;
  const size_t dyn = GA == GA_KCH ? (size_t)(p.K / Chunk<T>::VEC) * sizeof(uint32_t) : 0;
  hipLaunchKernelGGL((gemm_nt_kernel<T, OutT, EPI, GA, WGM, WGN, TM, TN, G_BKC>),
                     dim3(tiles), dim3(64 * WGM * WGN), dyn, stream, p);
}
template <typename T, typename OutT, int EPI, int GA>
void launch_tile(const GemmParams<T, OutT>& p, hipStream_t stream) {
  if constexpr (EPI == EPI_STORE) {
    const int big = ((p.M + 255) / 256) * ((p.N + 255) / 256) * p.nseg;
    if (big < kSmallProblemTiles) {
      launch_cfg<T, OutT, EPI, GA, 2, 2, 2, 2>(p, stream);
      return;
    }
  }
  launch_cfg<T, OutT, EPI, GA, G_WGM, G_WGN, G_TM, G_TN>(p, stream);
}

template <typename T, typename OutT>
hipError_t launch_gemm(const T* A, int64_t lda, const T* B, int64_t ldb, OutT* C, int64_t ldc,
                       int M, int N, int K, int epi, const float* bias, const float* gate0,
                       const float* gate1, hipStream_t stream, const GemmGather* gather,
                       const GemmVt* vt) {
  if (M <= 0 || N <= 0) return hipSuccess;
  // 256-row blocks of A, B and C are addressed through 32-bit buffer
  // descriptors whose offsets from kMasked on read as zero
  if ((int64_t)BN_MAX * lda * (int64_t)sizeof(T) >= (int64_t)kMasked ||
      (int64_t)BN_MAX * ldb * (int64_t)sizeof(T) >= (int64_t)kMasked ||
      (int64_t)BN_MAX * ldc * (int64_t)sizeof(OutT) >= (int64_t)kMasked)
    return hipErrorInvalidValue;
  GemmParams<T, OutT> p{};
  p.A = A;
  p.Bs[0] = B;
  p.C = C;
  p.lda = lda;
  p.ldb = ldb;
  p.ldc = ldc;
  p.M = M;
  p.N = N;
  p.K = K;
  p.biases[0] = bias;
  p.nseg = 1;
  p.gate0 = gate0;
  p.gate1 = gate1;
  p.vec4 = (ldc % 4 == 0) && (reinterpret_cast<uintptr_t>(C) % (4 * sizeof(OutT)) == 0);
  if (vt) {
    // the transposed columns must start on a tile boundary (one B matrix) or
    // at a segment, so every tile is wholly transposed or not
    const int nseg = gather ? gather->nseg : 1;
    const bool aligned = nseg > 1 ? vt->col0 % N == 0 : vt->col0 % BN_MAX == 0;
    if (epi != EPI_STORE || !vt->vt || vt->L <= 0 || vt->dims <= 0 || vt->ldvt < vt->L || !aligned ||
        vt->col0 < 0 || vt->col0 + vt->dims > nseg * N || M % vt->L != 0)
      return hipErrorInvalidValue;
    p.vt = static_cast<OutT*>(vt->vt);
    p.ldvt = vt->ldvt;
    p.vt_col0 = vt->col0;
    p.vt_dims = vt->dims;
    p.vt_L = vt->L;
    p.vt_vec4 = vt->L % 4 == 0 && vt->ldvt % 4 == 0 &&
                reinterpret_cast<uintptr_t>(vt->vt) % (4 * sizeof(OutT)) == 0;
  }
  if (gather && gather->nseg > 1) {
    if (gather->nseg > kMaxSeg || epi == EPI_RESIDUAL) return hipErrorInvalidValue;
    p.nseg = gather->nseg;
    for (int sg = 1; sg < p.nseg; ++sg) {
      p.Bs[sg] = static_cast<const T*>(gather->seg_b[sg - 1]);
      p.biases[sg] = gather->seg_bias[sg - 1];
    }
  }
  if (!gather || (!gather->rows && !gather->kchunks)) {  // (segments allowed)
    switch (epi) {
      case EPI_STORE: launch_tile<T, OutT, EPI_STORE, GA_NONE>(p, stream); break;
      case EPI_GELU: launch_tile<T, OutT, EPI_GELU, GA_NONE>(p, stream); break;
      default: launch_tile<T, OutT, EPI_RESIDUAL, GA_NONE>(p, stream); break;
    }
  } else if (gather->rows && !gather->kchunks) {
    // the whole union matrix must stay addressable below the masked offset
    if (gather->b_rows <= 0 || (int64_t)gather->b_rows * ldb * (int64_t)sizeof(T) >= (int64_t)kMasked)
      return hipErrorInvalidValue;
    p.rows = gather->rows;
    p.b_rows = gather->b_rows;
    switch (epi) {
      case EPI_STORE: launch_tile<T, OutT, EPI_STORE, GA_ROWS>(p, stream); break;
      case EPI_GELU: launch_tile<T, OutT, EPI_GELU, GA_ROWS>(p, stream); break;
      default: return hipErrorInvalidValue;
    }
  } else if (gather->kchunks && !gather->rows) {
    if (epi != EPI_RESIDUAL || K / Chunk<T>::VEC > kMaxKChunks ||
        (int64_t)BN_MAX * ldb * (int64_t)sizeof(T) >= (int64_t)kMasked)
      return hipErrorInvalidValue;
    p.kch = gather->kchunks;
    launch_tile<T, OutT, EPI_RESIDUAL, GA_KCH>(p, stream);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// The chip's sustained MFMA rate with nothing else running: every CU holds
// two workgroups of four waves, each wave issuing independent bf16 MFMAs
// (32 x 32 x 16 on eight accumulators, or 16 x 16 x 32 on sixteen, the
// same FLOPs per iteration) on operands from a hash of the thread
// (random-looking bf16 of magnitude ~1, rotated between iterations), no
// memory traffic.  The result only decides whether a never-taken store
// happens, so the work cannot be optimised away.  The rate it reaches is
// the ceiling the power limit leaves for MFMA-bound kernels of that shape
// (the clock drops below its 2.4 GHz maximum under this load, and by how
// much depends on the shape).
template <bool M16>
__global__ __launch_bounds__(256, 2) void mfma_probe_kernel(int iters4, float* sink) {
  const uint32_t t = blockIdx.x * 256u + threadIdx.x;
  bf16x8 a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint32_t h = (t * 8u + (uint32_t)(i * 8 + e)) * 2654435761u;
      h ^= h >> 15;
      h *= 2246822519u;
      h ^= h >> 13;
      a[i][e] = (bf16)(((float)(h & 0xffff) - 32768.f) / 32768.f);
      b[i][e] = (bf16)(((float)(h >> 16) - 32768.f) / 32768.f);
    }
  typedef typename std::conditional<M16, f32x4, f32x16>::type AccT;
  constexpr int NACC = M16 ? 16 : 8, NR = M16 ? 4 : 16;   // 262144 FLOPs per u step either way
  AccT c[NACC];
#pragma unroll
  for (int j = 0; j < NACC; ++j)
#pragma unroll
    for (int r = 0; r < NR; ++r) c[j][r] = 0.f;
  for (int it = 0; it < iters4; ++it) {
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int j = 0; j < NACC; ++j) {
        if constexpr (M16)
          c[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[(j + u) & 3], b[(j >> 2) & 3], c[j], 0, 0, 0);
        else
          c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(j + u) & 3], b[j & 3], c[j], 0, 0, 0);
      }
  }
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < NACC; ++j)
#pragma unroll
    for (int r = 0; r < NR; ++r) sum += c[j][r];
  if (sum == 1234567.f) *sink = sum;
}

// The same for the softmax's exponential (v_exp_f32, the instruction the
// attention kernels evaluate 2^x with): every lane runs sixteen independent
// chains x <- 2^(-x), which stay in [0.5, 1] (the negation is a free source
// modifier, so the loop is nothing but exponentials).  Eight workgroups of
// four waves per CU (eight waves per SIMD) hide the instruction's latency.
__global__ __launch_bounds__(256) void exp_probe_kernel(int iters4, float* sink) {
  const uint32_t t = blockIdx.x * 256u + threadIdx.x;
  float x[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) x[j] = 0.5f + (float)((t * 16u + (uint32_t)j) & 1023u) / 2048.f;
  for (int it = 0; it < iters4; ++it) {
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int j = 0; j < 16; ++j) x[j] = __builtin_amdgcn_exp2f(-x[j]);
  }
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < 16; ++j) sum += x[j];
  if (sum == 1234567.f) *sink = sum;
}

hipError_t launch_mfma_probe(int shape, int iters, float* sink, int ncu, hipStream_t stream,
                             double* flops) {
  const int iters4 = (iters + 3) / 4;
  if (shape == 2) {
    // per lane and iteration: 16 exponentials
    const int eblocks = 8 * ncu;
    *flops = (double)eblocks * 256 * (4.0 * iters4) * 16;
    hipLaunchKernelGGL(exp_probe_kernel, dim3(eblocks), dim3(256), 0, stream, iters4, sink);
    return hipGetLastError();
  }
  const int blocks = 2 * ncu;
  // per wave and iteration: 8 MFMAs of 32 x 32 x 16 or 16 of 16 x 16 x 32
  *flops = (double)blocks * 4 * (4.0 * iters4) * 8 * (2.0 * 32 * 32 * 16);
  if (shape == 0)
    hipLaunchKernelGGL(mfma_probe_kernel<false>, dim3(blocks), dim3(256), 0, stream, iters4, sink);
  else
    hipLaunchKernelGGL(mfma_probe_kernel<true>, dim3(blocks), dim3(256), 0, stream, iters4, sink);
  return hipGetLastError();
}

#define INST(T, OutT)                                                                         \
  template hipError_t launch_gemm<T, OutT>(const T*, int64_t, const T*, int64_t, OutT*, int64_t, \
                                           int, int, int, int, const float*, const float*,    \
                                           const float*, hipStream_t, const GemmGather*,      \
                                           const GemmVt*);
INST(bf16, bf16)
INST(bf16, float)
INST(float, float)
#undef INST

}  // namespace dif

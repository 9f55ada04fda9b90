// Device-side building blocks shared by the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dif {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kXcds = 8;   // MI355X: 8 XCDs, workgroups dispatched round-robin

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }

// A 16-byte chunk holds VEC elements of T.
template <typename T> struct Chunk {
  static constexpr int VEC = 16 / sizeof(T);
  __device__ static void unpack(const u32x4& c, float* out) {
    if constexpr (sizeof(T) == 4) {
      f32x4 v = __builtin_bit_cast(f32x4, c);
#pragma unroll
      for (int e = 0; e < 4; ++e) out[e] = v[e];
    } else {
      bf16x8 v = __builtin_bit_cast(bf16x8, c);
#pragma unroll
      for (int e = 0; e < 8; ++e) out[e] = (float)v[e];
    }
  }
  __device__ static u32x4 pack(const float* in) {
    if constexpr (sizeof(T) == 4) {
      f32x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = in[e];
      return __builtin_bit_cast(u32x4, v);
    } else {
      bf16x8 v;
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = (bf16)in[e];
      return __builtin_bit_cast(u32x4, v);
    }
  }
};

// One MFMA "k-step" on 32x32 tiles: every lane contributes one 16-byte
// chunk of A (row lane%32) and of B (column lane%32); lane group lane/32
// covers the second half of the k extent.
//   bf16: v_mfma_f32_32x32x16_bf16, k extent 16
//   f32 : 4 x v_mfma_f32_32x32x2_f32, k extent 8 (element e of both groups)
template <typename T> struct Mma;
template <> struct Mma<bf16> {
  static constexpr int KS = 16;
  __device__ __forceinline__ static void step(f32x16& acc, const u32x4& a, const u32x4& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
  }
};
template <> struct Mma<float> {
  static constexpr int KS = 8;
  __device__ __forceinline__ static void step(f32x16& acc, const u32x4& a, const u32x4& b) {
    f32x4 fa = __builtin_bit_cast(f32x4, a), fb = __builtin_bit_cast(f32x4, b);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[0], fb[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[1], fb[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[2], fb[2], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[3], fb[3], acc, 0, 0, 0);
  }
};

// Row of accumulator register r for lane group g in a 32x32 MFMA tile
// (column is lane % 32).
__device__ __forceinline__ int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

// Workgroup `bid` runs on XCD bid % 8.  Return a logical tile index such
// that each XCD receives one contiguous range of logical tiles, so tiles
// that share operands share that XCD's L2.
__device__ __forceinline__ int xcd_remap(int bid, int total) {
  const int q = total / kXcds, r = total % kXcds;
  const int x = bid % kXcds, local = bid / kXcds;
  return (x < r) ? x * (q + 1) + local : r * (q + 1) + (x - r) * q + local;
}

// LDS position of 16-byte chunk c in row `row` of a tile whose rows hold CH
// chunks.  A wave's 16-byte LDS accesses are served in groups of lanes
// that read consecutive rows at the same logical chunk; the XOR makes
// every group of 8 lanes (128-byte window) and of 16 lanes (256-byte
// window) hit distinct banks, for row-contiguous writes as well.
template <int CH>
__device__ __forceinline__ int swz(int row, int c) {
  static_assert(CH == 8 || CH >= 16, "LDS rows of 8 or >= 16 chunks");
  if constexpr (CH == 8) {
    return c ^ ((row & 7) ^ ((row >> 3) & 1));
  } else {
    return c ^ (row & 15);
  }
}

// s_waitcnt vmcnt(n) with the other counters left alone.  Buffer loads
// that write LDS directly are counted by vmcnt, and a workgroup barrier
// does not wait for them on its own.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Sum over the 64 lanes of a wave, returned to every lane.  DPP steps:
// pairs and quads (quad_perm), 8 lanes (row_half_mirror), 16 lanes
// (row_mirror), then row 0 into row 1 and row 2 into row 3 (row_bcast:15,
// rows 1 and 3 only) and rows 0-1 into rows 2-3 (row_bcast:31, rows 2 and 3
// only); lane 63 then holds the total, which is read back as a scalar.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_add(float v) {
  const int t = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROW_MASK, 0xf, false);
  return v + __builtin_bit_cast(float, t);
}
__device__ __forceinline__ float wave_sum(float v) {
  v = dpp_add<0xb1, 0xf>(v);    // quad_perm [1,0,3,2]
  v = dpp_add<0x4e, 0xf>(v);    // quad_perm [2,3,0,1]
  v = dpp_add<0x141, 0xf>(v);   // row_half_mirror
  v = dpp_add<0x140, 0xf>(v);   // row_mirror
  v = dpp_add<0x142, 0xa>(v);   // row_bcast:15
  v = dpp_add<0x143, 0xc>(v);   // row_bcast:31
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// GELU with the tanh approximation, 0.5 x (1 + tanh(u)), u = sqrt(2/pi)(x +
// 0.044715 x^3), evaluated as x / (1 + exp(-2u)) (the identity
// 0.5 (1 + tanh u) = 1 / (1 + e^{-2u})) with the hardware exp2 and
// reciprocal; saturates correctly (exp2 -> inf gives 0, -> 0 gives x).
__device__ __forceinline__ float gelu_tanh(float x) {
  constexpr float k = -2.f * 0.7978845608028654f * 1.4426950408889634f;  // -2 sqrt(2/pi) log2(e)
  const float t = x * fmaf(0.044715f * x, x, 1.f);                        // x + 0.044715 x^3
  return x * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(k * t));
}

}  // namespace dif

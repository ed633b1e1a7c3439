// Device helpers shared by the gfx950 kernels: storage types, rounding,
// 16-byte fragments, MFMA on one k-block, and wave64 reductions.
//
// Every kernel is compiled with -ffp-contract=off: the arithmetic of a row
// never depends on how many rows a launch carries or on which template
// instance runs it, so a tree pass and a one-token pass produce identical
// bits for the same logical inputs.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

#define CH_INF __builtin_inff()

__device__ __forceinline__ float bf2f(bf16_t v) { return __uint_as_float(((uint32_t)v) << 16); }

// float -> bf16, round to nearest, ties to even (NaN -> quiet NaN): gfx950's
// v_cvt_pk_bf16_f32, with denormals preserved (the kernels' float mode).
__device__ __forceinline__ bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

// Storage-type traits.  A "fragment" is the 16 bytes one lane feeds into a
// 16x16 MFMA k-block: VEC consecutive elements along the reduction axis.
template <typename T> struct ET;
template <> struct ET<float> {
  static constexpr int VEC = 4;
  __device__ static float to_f(float v) { return v; }
  __device__ static float from_f(float v) { return v; }
};
template <> struct ET<bf16_t> {
  static constexpr int VEC = 8;
  __device__ static float to_f(bf16_t v) { return bf2f(v); }
  __device__ static bf16_t from_f(float v) { return f2bf(v); }
};

__device__ __forceinline__ int4 ld16(const void* p) { return *reinterpret_cast<const int4*>(p); }
__device__ __forceinline__ void st16(void* p, int4 v) { *reinterpret_cast<int4*>(p) = v; }

// acc += A_frag x B_frag over one k-block of 4*VEC reduction indices.
// Lane l supplies row/column (l & 15) and reduction indices (l >> 4)*VEC ..
// +VEC-1 of the block.  bf16: one v_mfma_f32_16x16x32_bf16.  f32: four
// v_mfma_f32_16x16x4_f32, the i-th consuming element i of every lane.
template <typename T> __device__ __forceinline__ f32x4 mfma_kb(int4 a, int4 b, f32x4 acc);
template <> __device__ __forceinline__ f32x4 mfma_kb<bf16_t>(int4 a, int4 b, f32x4 acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), acc,
                                                 0, 0, 0);
}
template <> __device__ __forceinline__ f32x4 mfma_kb<float>(int4 a, int4 b, f32x4 acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__int_as_float(a.x), __int_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__int_as_float(a.y), __int_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__int_as_float(a.z), __int_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__int_as_float(a.w), __int_as_float(b.w), acc, 0, 0, 0);
  return acc;
}

// Butterfly all-reductions over the 64 lanes of a wave.  Each stage adds a
// lane's value to its partner's in commutative pairs, so every lane ends
// with bit-identical results.
// Cross-lane combination on the VALU (DPP inside a 16-lane row, gfx950 lane
// swaps across rows); every lane ends with the same value, combined in a
// fixed order.  Each step adds a lane's value to its partner's, and the two
// partners add the same two operands, so they agree bit for bit.
enum { DPP_XOR1 = 0xB1, DPP_XOR2 = 0x4E, DPP_MIRROR8 = 0x141, DPP_MIRROR16 = 0x140, DPP_ROR8 = 0x128 };
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
// (even row's value, odd row's value) of each pair of 16-lane rows, and
// (value in lanes 0-31, value in lanes 32-63), both on every lane
__device__ __forceinline__ float2 row_pair(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return float2{__uint_as_float(r[0]), __uint_as_float(r[1])};
}
__device__ __forceinline__ float2 half_pair(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return float2{__uint_as_float(r[0]), __uint_as_float(r[1])};
}
// over lanes l, l ^ 16, l ^ 32, l ^ 48 (the same position in the four rows)
__device__ __forceinline__ float rows_sum(float v) {
  float2 p = row_pair(v);
  p = half_pair(p.x + p.y);
  return p.x + p.y;
}
__device__ __forceinline__ float rows_max(float v) {
  float2 p = row_pair(v);
  p = half_pair(fmaxf(p.x, p.y));
  return fmaxf(p.x, p.y);
}
// over the 16 lanes of a row
__device__ __forceinline__ float row16_sum(float v) {
  v = v + dpp_mov<DPP_XOR1>(v);
  v = v + dpp_mov<DPP_XOR2>(v);
  v = v + dpp_mov<DPP_MIRROR8>(v);
  return v + dpp_mov<DPP_MIRROR16>(v);
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_mov<DPP_XOR1>(v));
  v = fmaxf(v, dpp_mov<DPP_XOR2>(v));
  v = fmaxf(v, dpp_mov<DPP_MIRROR8>(v));
  return fmaxf(v, dpp_mov<DPP_MIRROR16>(v));
}
// over all 64 lanes (call with every lane active)
__device__ __forceinline__ float wave_sum(float v) { return rows_sum(row16_sum(v)); }
__device__ __forceinline__ float wave_max(float v) { return rows_max(row16_max(v)); }

__device__ __forceinline__ float silu_f(float x) { return x / (1.0f + expf(-x)); }

// exp(a - b) for the online softmax, with exp(-inf - x) = 0.
__device__ __forceinline__ float exp_diff(float a, float b) { return (a == -CH_INF) ? 0.0f : expf(a - b); }

// Activations that feed a GEMM are stored in MFMA fragment order: element
// (row, col) of a matrix with `mtiles` 16-row tiles lives in tile
// (col / KB, row / 16) at lane ((col % KB) / VEC) * 16 + row % 16, element
// col % VEC, so that one fragment load is a contiguous 1 KiB.
template <typename T>
__device__ __forceinline__ int64_t tiled_index(int mtiles, int row, int col) {
  constexpr int VEC = ET<T>::VEC, KB = 4 * VEC;
  const int kb = col / KB, w = col % KB;
  const int lane = (w / VEC) * 16 + (row & 15);
  return (((int64_t)kb * mtiles + (row >> 4)) * 64 + lane) * VEC + (w % VEC);
}
template <typename T>
__device__ __forceinline__ void store_tiled(T* base, int mtiles, int row, int col, float v) {
  base[tiled_index<T>(mtiles, row, col)] = ET<T>::from_f(v);
}
template <typename T>
__device__ __forceinline__ void copy_tiled(T* base, int mtiles, int row, int col, T v) {
  base[tiled_index<T>(mtiles, row, col)] = v;
}

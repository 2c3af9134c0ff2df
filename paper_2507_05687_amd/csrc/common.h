// Shared device/host definitions of libgrpo (internal; not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

namespace grpo {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Workspace header (first 256 bytes of every workspace). Each error kind has
// its own word so that kernels can raise it with a plain store.
struct WsHeader {
  int32_t err_token;     // nonzero: some valid row had a token id outside [0, V)
  int32_t err_seqlens;   // nonzero: cu_seqlens was not monotone from 0 to N
  int32_t num_valid;     // number of valid rows after packing
  int32_t err_capacity;  // nonzero: more valid rows than the workspace was sized for
  int32_t pad_[60];
};

constexpr int kTile = 256;  // GEMM tile edge (rows and columns)
constexpr int kBK = 32;     // GEMM K step = column width of a tiled-layout block
// Tiled layout of a GEMM operand with R rows and K columns: blocks of 256 rows
// x 32 columns (16 KiB of bf16, rows of 64 bytes), block (rb, kb) at
// (rb * ceil(K/32) + kb) * kTileElems elements; padding rows and columns are 0.
constexpr int kTileElems = kTile * kBK;

__host__ __device__ inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
__host__ __device__ inline int64_t ceil_div(int64_t x, int64_t m) { return (x + m - 1) / m; }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// fp32 -> bf16, round to nearest even, with gfx950's packed conversion
// instruction: two values -> one 32-bit word (first value in the low half).
__device__ __forceinline__ uint32_t bf16_pack2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{a, b}), bf16x2_t));
}
__device__ __forceinline__ uint16_t bf16_bits(float a) {
  return __builtin_bit_cast(uint16_t, (__bf16)a);
}
__device__ inline float bf16_bits_to_f32(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

constexpr float kLog2e = 1.4426950408889634f;


// Calls f(std::integral_constant<int, i>) for i = 0..N-1, unrolled at compile
// time, so that register arrays indexed by i are never demoted to memory.
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

}  // namespace grpo

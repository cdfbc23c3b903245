// Internal device helpers shared by the library's kernels (not part of the public ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vc {

constexpr int D = 128;    // head dimension
constexpr int BLK = 128;  // rows per quantization block / attention tile

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v2f __attribute__((ext_vector_type(2)));
typedef unsigned int u4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// fp32 -> bf16 bits, round to nearest even (gfx950 converts in hardware with RNE).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  __bf16 b = (__bf16)f;
  return __builtin_bit_cast(uint16_t, b);
}

// Byte offset inside one 128x128 int8 block of Q or K codes, tiled for the INT8 matrix
// instruction: [rb 4][dc 4][dh 2][r 32][e 16].
__host__ __device__ __forceinline__ int qk_tile_offset(int row, int ch) {
  return (((row >> 5) * 4 + (ch >> 5)) * 2 + ((ch >> 4) & 1)) * 512 + (row & 31) * 16 + (ch & 15);
}

// Byte offset inside one 128x128 block of E4M3 V residual codes: [kc 2][db 4][kh 2][sh 2][c 32][t 16].
__host__ __device__ __forceinline__ int v_tile_offset(int key, int ch) {
  const int kb = key >> 5, w = key & 31;
  const int kc = kb >> 1, sh = kb & 1, kh = (w >> 2) & 1, t = 4 * (w >> 3) + (w & 3);
  return ((((kc * 4 + (ch >> 5)) * 2 + kh) * 2 + sh) * 32 + (ch & 31)) * 16 + t;
}

// Rotary pair i (0..63) rotates with frames (0..21), rows (22..42) or columns (43..63).
__device__ __forceinline__ int rope_axis(int pair) { return pair < 22 ? 0 : (pair < 43 ? 1 : 2); }

__device__ __forceinline__ int clamp_index(int v, int n) { return v < 0 ? 0 : (v >= n ? n - 1 : v); }

}  // namespace vc

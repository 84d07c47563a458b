// Shared definitions of the gfx950 kernels of the LoPA verify step.
//
// Fragment-packed bf16 layout (used for every GEMM operand):
//   a matrix X with R rows and K columns (R % 16 == 0, K % 32 == 0) is stored as
//   1 KiB fragments of 16 rows x 32 columns. Inside a fragment, lane
//   l = (r % 16) + 16 * ((c % 32) / 8) holds the 8 consecutive columns
//   c = 8 * (l / 16) .. +7 of row r % 16, i.e. exactly the per-lane operand of
//   v_mfma_f32_16x16x32_bf16 (A: lane -> row, B: lane -> column of W^T).
//   A wave reads one fragment as 64 lanes x 16 contiguous bytes.
//
// Activations ("A" operands, R = padded rows Mp):   fragment (rb, kb) at
//   ((kb * (Mp/16)) + rb) * 512 elements.
// Weights (W [N, K] in [out, in] order, "B" operand): blocks of 16 output
//   features, grouped in tiles of nb consecutive blocks (nb fixed per weight);
//   each block's 64-column chunk kc is two fragments (kk = 0, 1: columns
//   32 kk .. +31), fragment (tile t, kc, block j of the tile, kk) at
//   (((t * (K / 64) + kc) * nb + j) * 2 + kk) * 512. One GEMM iteration of a
//   tile streams one contiguous nb x 2 KiB chunk.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x8 __attribute__((ext_vector_type(8)));

// fp32 -> bf16 bits, round to nearest even (gfx950 converts in hardware:
// v_cvt_pk_bf16_f32; NaN stays NaN)
__device__ __forceinline__ uint16_t f2bf_bits(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}
__device__ __forceinline__ float bf2f_bits(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma16(const uint4& a, const uint4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// KV tile layout (cache and staging). A head's K region and its V region each
// hold tiles of KV_TILE = 32 positions, d x 32 elements per tile, stored in
// the order the attention's MFMAs take them, so that every 1 KiB operand
// fragment is one contiguous run:
//   K: fragment (kb, kk) of a tile (kb < 2, kk < d / 32) at elements
//      ((kb d/32 + kk) 64 + lane) 8; lane = c16 + 16 g holds position
//      8 (c16 / 4) + 4 kb + c16 % 4 of the tile, dimensions 32 kk + 8 g .. + 7
//      (an S^T = K Q^T tile then gives lane (c16, g) positions 8 g .. 8 g + 7);
//   V: fragment db (< d / 16) at elements (db 64 + lane) 8; lane = c16 + 16 g
//      holds dimension 16 db + c16, positions 8 g .. 8 g + 7.
constexpr int KV_TILE = 32;
__host__ __device__ __forceinline__ int64_t kv_k_off(int p, int e, int d) {
  const int p32 = p & 31, kb = (p32 >> 2) & 1, c16 = 4 * (p32 >> 3) + (p32 & 3);
  return (int64_t)(p >> 5) * 32 * d +
         ((((kb * (d >> 5) + (e >> 5)) * 64 + c16 + 16 * ((e >> 3) & 3)) << 3) | (e & 7));
}
__host__ __device__ __forceinline__ int64_t kv_v_off(int p, int e, int d) {
  const int p32 = p & 31;
  return (int64_t)(p >> 5) * 32 * d + ((((e >> 4) * 64 + (e & 15) + 16 * (p32 >> 3)) << 3) | (p32 & 7));
}

// element offset of (row r, column c) in an activation matrix packed with Mp rows
__device__ __forceinline__ int64_t packA_off(int r, int c, int Mp) {
  int rb = r >> 4, kb = c >> 5;
  int lane = (r & 15) + 16 * ((c & 31) >> 3);
  return ((int64_t)(kb * (Mp >> 4) + rb) * 64 + lane) * 8 + (c & 7);
}

// Workgroup barrier that orders LDS accesses only. __syncthreads() also orders
// global memory, which makes the compiler drain every outstanding global load
// (vmcnt(0)) at the barrier and so destroys any load pipelining across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

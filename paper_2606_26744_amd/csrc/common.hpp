// Device helpers shared by the gfx950 kernels of libhdf.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hdf {

typedef uint16_t bf16_t;  // raw bf16 bits
typedef short bf16x8_t __attribute__((ext_vector_type(8)));   // MFMA bf16 operand (8 values)
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));   // one 16-byte access

constexpr int kWave = 64;

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// fp32 -> bf16, round to nearest, ties to even (inputs finite).
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return bf16_t(u >> 16);
}

// Two packed bf16 (low half = element 0) -> floats.
__device__ __forceinline__ float lo_bf(uint32_t p) { return __uint_as_float(p << 16); }
__device__ __forceinline__ float hi_bf(uint32_t p) { return __uint_as_float(p & 0xFFFF0000u); }
__device__ __forceinline__ uint32_t pack_bf2(float a, float b) {
  return uint32_t(f2bf(a)) | (uint32_t(f2bf(b)) << 16);
}

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), acc, false);
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

template <typename T>
__device__ __forceinline__ T wave_max(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Workgroup barrier for LDS hand-off only: waits for this wave's LDS traffic and
// meets the other waves, without draining outstanding global loads (prefetches
// stay in flight across it).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ u32x4 ld16(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ u32x4 ld_nt16(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ __forceinline__ void st_nt16(void* p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

// KV cache layout.  Rows (positions) of one head are grouped in tiles of 64, each
// tile 64*hd contiguous elements in the order in which the attention kernel's 64
// lanes take their matrix-core operands, so every operand load is one contiguous
// 1 KB (bf16) access:
//   keys   (S^T = K.Q^T, K the A operand of v_mfma_f32_16x16x32_bf16): row r of the
//          tile is row ql = 4*((r%32)/8) + r%4 of 16-key sub-tile st = 2*(r/32) +
//          (r/4)%2; dim i is k-slice j = i/32, lane group g = (i/8)%4, element i%8;
//          offset ((st*(hd/32) + j)*64 + 16g + ql)*8 + i%8
//   values (O^T += V^T.P^T, V^T the A operand): dim i is row ql = i%16 of 16-dim
//          tile dt = i/16; row r is k-slice r/32, lane group (r/8)%4, element r%8;
//          offset (((r/32)*(hd/16) + dt)*64 + 16*((r/8)%4) + ql)*8 + r%8
__host__ __device__ __forceinline__ int64_t kc_offset(int r, int i, int hd) {
  const int rr = r & 31;
  const int st = 2 * (r >> 5) + ((rr >> 2) & 1);
  const int ql = 4 * (rr >> 3) + (rr & 3);
  return ((int64_t(st) * (hd >> 5) + (i >> 5)) * 64 + ((i >> 3) & 3) * 16 + ql) * 8 + (i & 7);
}
__host__ __device__ __forceinline__ int64_t vc_offset(int r, int i, int hd) {
  return ((int64_t(r >> 5) * (hd >> 4) + (i >> 4)) * 64 + ((r >> 3) & 3) * 16 + (i & 15)) * 8 +
         (r & 7);
}
// Element offset of (row, dim) in one head's keys / values (cap rows, cap % 64 == 0).
__host__ __device__ __forceinline__ int64_t kc_index(int64_t row, int i, int hd) {
  return (row >> 6) * 64 * hd + kc_offset(int(row & 63), i, hd);
}
__host__ __device__ __forceinline__ int64_t vc_index(int64_t row, int i, int hd) {
  return (row >> 6) * 64 * hd + vc_offset(int(row & 63), i, hd);
}

// SiLU(g) * u, the gated MLP activation.
__device__ __forceinline__ float silu_mul(float g, float u) { return g / (1.f + __expf(-g)) * u; }

// Rotate-half RoPE of the pair (x1, x2) = (x[i], x[i + hd/2]) by the angle with
// cosine c and sine s.
__device__ __forceinline__ void rope_rotate(float& x1, float& x2, float c, float s) {
  const float u1 = x1, u2 = x2;
  x1 = u1 * c - u2 * s;
  x2 = u2 * c + u1 * s;
}

// Order-preserving map of a finite fp32 to uint32 (larger float -> larger key).
__device__ __forceinline__ uint32_t f32_order_key(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float f32_from_order_key(uint32_t k) {
  uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
  return __uint_as_float(u);
}

// A row's packed argmax key (order key of the maximum << 32 | ~column): its column and,
// when max_logit is given, the maximum.
__device__ __forceinline__ void decode_argmax_key(unsigned long long k, int32_t* argmax,
                                                  float* max_logit) {
  *argmax = int32_t(0xFFFFFFFFu - uint32_t(k & 0xFFFFFFFFull));
  if (max_logit != nullptr) *max_logit = f32_from_order_key(uint32_t(k >> 32));
}

}  // namespace hdf

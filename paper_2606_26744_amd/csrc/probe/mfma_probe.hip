// Matrix-core probe for the bench (libhdf_probe.so, not part of libhdf's ABI): the rate
// at which the chip retires v_mfma_f32_32x32x16_bf16 (the instruction every bf16 GEMM of
// the library issues) when nothing else limits it, to measure what the matrix-core
// bound kernels can reach.
//
// Every wave keeps four independent accumulator chains in registers and issues `iters`
// rounds of four MFMAs; no memory is touched inside the loop.  The operands are bf16
// values with random signs and mantissas (magnitudes in [1/8, 1/2)), different in every
// lane and for every chain, like the data of a GEMM: the sustained rate depends on the operand data (with near-constant operands the
// chip holds a higher clock), and random data is what the library's GEMMs see.  Launch:
// `blocks` workgroups of four waves (four workgroups per CU fill every SIMD with four
// waves).  The sums of the accumulators go to `sink` only in a case that never happens,
// so that the work is not optimised away.  FLOPs per launch = blocks * 4 waves * 4 chains
// * iters * 32768.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ __bf16 rnd_bf16(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352dU;
  x ^= x >> 15;
  x *= 0x846ca68bU;
  x ^= x >> 16;
  // random sign, exponent field 124 or 125 (|v| in [1/8, 1/2)), 7 random mantissa bits
  const uint16_t h = uint16_t((x & 0x8000u) | ((0x7Cu + ((x >> 7) & 1u)) << 7) | (x & 0x7Fu));
  return __builtin_bit_cast(__bf16, h);
}

__global__ void __launch_bounds__(256)
mfma_probe_kernel(float* __restrict__ sink, int iters) {
  const uint32_t seed = (blockIdx.x * 256u + threadIdx.x) * 64u;
  bf16x8_t a[4], b[4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a[c][i] = rnd_bf16(seed + c * 16 + i);
      b[c][i] = rnd_bf16(seed + c * 16 + 8 + i + 0x9e3779b9u);
    }
  f32x16_t acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int c = 0; c < 4; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[c], b[c], acc[c], 0, 0, 0);
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  if (s == 1.2345f) sink[blockIdx.x] = s;   // never true; keeps the work
}

}  // namespace

// Returns 0, or the HIP error of the launch.  blocks > 0, iters > 0; sink: device memory
// of at least `blocks` floats.
extern "C" int hdf_probe_mfma(int blocks, int iters, void* sink, void* stream) {
  if (blocks <= 0 || iters <= 0 || sink == nullptr) return int(hipErrorInvalidValue);
  hipLaunchKernelGGL(mfma_probe_kernel, dim3(blocks), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<float*>(sink), iters);
  return int(hipGetLastError());
}

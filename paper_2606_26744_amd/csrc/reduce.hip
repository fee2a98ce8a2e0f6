// Gated residual reducer -- Eq. (1), Sec. 2.2 (the target's hc_head collapse form).
//
// Per token t (independently): x = vec(H_t) (path-major), r = 1/sqrt(mean(x^2)+eps),
// z_j = gate_scale * r * (W_g[j] . x) + b_j, alpha_j = sigmoid(z_j) + gate_offset,
// Y_t = sum_j alpha_j P_j with P_j = H_t[j] (or H_t[j] RMS-normalised over d).
//
// Bandwidth-bound: every token's m*d inputs are read from HBM exactly once.
// One workgroup per CU walks a strided list of tokens.  Each thread owns one
// 16-byte column slice (8 bf16 or 4 fp32 columns) of every path, so the weighted
// sum needs no data exchange; the only exchange is the workgroup reduction of
// 2m partials (m per-path sums of squares + m gate dots), one LDS barrier per
// token.  The thread's slice of W_g (m gates x m paths x slice) stays in registers
// for the whole token loop when it fits (m <= 4), so W_g is read once per
// workgroup.  The next token's inputs are prefetched into registers before the
// current token's reduction.
#include "common.hpp"
#include "kernels.hpp"

namespace hdf {

template <typename T>
struct Vec16;
template <>
struct Vec16<bf16_t> {
  static constexpr int N = 8;
  u32x4 v;
  __device__ __forceinline__ float get(int i) const {
    uint32_t w = v[i >> 1];
    return (i & 1) ? hi_bf(w) : lo_bf(w);
  }
};
template <>
struct Vec16<float> {
  static constexpr int N = 4;
  u32x4 v;
  __device__ __forceinline__ float get(int i) const { return __uint_as_float(v[i]); }
};

template <typename T>
__device__ __forceinline__ u32x4 pack_out(const float* y);
template <>
__device__ __forceinline__ u32x4 pack_out<bf16_t>(const float* y) {
  return u32x4{pack_bf2(y[0], y[1]), pack_bf2(y[2], y[3]), pack_bf2(y[4], y[5]),
               pack_bf2(y[6], y[7])};
}
template <>
__device__ __forceinline__ u32x4 pack_out<float>(const float* y) {
  return u32x4{__float_as_uint(y[0]), __float_as_uint(y[1]), __float_as_uint(y[2]),
               __float_as_uint(y[3])};
}

// Dot of one 16-byte slice of W with one 16-byte slice of x, accumulated.
template <typename T>
__device__ __forceinline__ float slice_dot(const u32x4& w, const u32x4& x, float acc);
template <>
__device__ __forceinline__ float slice_dot<bf16_t>(const u32x4& w, const u32x4& x, float acc) {
  acc = dot2_bf16(w.x, x.x, acc);
  acc = dot2_bf16(w.y, x.y, acc);
  acc = dot2_bf16(w.z, x.z, acc);
  acc = dot2_bf16(w.w, x.w, acc);
  return acc;
}
template <>
__device__ __forceinline__ float slice_dot<float>(const u32x4& w, const u32x4& x, float acc) {
  acc = fmaf(__uint_as_float(w.x), __uint_as_float(x.x), acc);
  acc = fmaf(__uint_as_float(w.y), __uint_as_float(x.y), acc);
  acc = fmaf(__uint_as_float(w.z), __uint_as_float(x.z), acc);
  acc = fmaf(__uint_as_float(w.w), __uint_as_float(x.w), acc);
  return acc;
}

constexpr int kReduceMaxThreads = 512;

// SLOTS: 16-byte column slices per thread per path (1 or 2): 1 while a token of width
// d needs at most 256 threads, else 2 (at most 512 threads).  With at most 8 waves a
// workgroup may use up to 256 VGPRs per lane, enough for the resident W_g slice
// (m*m*SLOTS slices) and one prefetched token.
template <typename T, int MP, int SLOTS>
__global__ void __launch_bounds__(kReduceMaxThreads)
hc_reduce_kernel(const T* __restrict__ H, const T* __restrict__ Wg, const float* __restrict__ bg,
                 int64_t n_tok, int d, ReduceScalars sc, T* __restrict__ Y,
                 float* __restrict__ alpha) {
  constexpr int VEC = Vec16<T>::N;
  constexpr bool W_REG = (MP * SLOTS <= 4) || (MP <= 4 && SLOTS <= 2);
  constexpr bool PREFETCH = W_REG;
  constexpr int NP = 2 * MP;  // partials per token: MP sums of squares, MP gate dots
  constexpr int NX = MP * SLOTS;
  __shared__ float part[2][kReduceMaxThreads / kWave][NP];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wid = tid >> 6;
  const int nwaves = blockDim.x >> 6;
  const int nthr = blockDim.x;
  const int64_t row = int64_t(MP) * d;  // elements of one token
  // Slice k of this thread covers columns col(k) .. col(k)+VEC-1.
  bool act[SLOTS];
  int col[SLOTS];
#pragma unroll
  for (int k = 0; k < SLOTS; ++k) {
    col[k] = (k * nthr + tid) * VEC;
    act[k] = col[k] < d;
  }

  // Resident W_g slices: w[g][j*SLOTS+k] covers slice k of path j for gate g.
  u32x4 w[W_REG ? MP : 1][W_REG ? NX : 1];
  if constexpr (W_REG) {
#pragma unroll
    for (int g = 0; g < MP; ++g)
#pragma unroll
      for (int j = 0; j < MP; ++j)
#pragma unroll
        for (int k = 0; k < SLOTS; ++k)
          w[g][j * SLOTS + k] = act[k] ? ld16(Wg + int64_t(g) * row + int64_t(j) * d + col[k])
                                       : u32x4{0, 0, 0, 0};
  }
  float bias[MP];
#pragma unroll
  for (int g = 0; g < MP; ++g) bias[g] = bg[g];

  // Loads are never predicated: a token index past the end is clamped to the last
  // token (its data is never used) and idle lanes read a valid column and zero it
  // with a select.  Unpredicated loads keep the compiler's outstanding-load count
  // exact, so the next token's loads stay in flight across the reduction.
  int colc[SLOTS];
#pragma unroll
  for (int k = 0; k < SLOTS; ++k) colc[k] = act[k] ? col[k] : 0;
  auto load_token = [&](int64_t tt, u32x4* dst) {
    const int64_t tc = tt < n_tok ? tt : n_tok - 1;
#pragma unroll
    for (int j = 0; j < MP; ++j)
#pragma unroll
      for (int k = 0; k < SLOTS; ++k) {
        const u32x4 v = ld_nt16(H + tc * row + int64_t(j) * d + colc[k]);
        dst[j * SLOTS + k] = act[k] ? v : u32x4{0, 0, 0, 0};
      }
  };

  int64_t t = blockIdx.x;
  u32x4 x[NX];
  load_token(t, x);
  int buf = 0;
  for (; t < n_tok; t += gridDim.x) {
    u32x4 xn[PREFETCH ? NX : 1];
    if constexpr (PREFETCH) load_token(t + gridDim.x, xn);  // next token of this workgroup

    float p[NP];
#pragma unroll
    for (int j = 0; j < MP; ++j) {
      float acc = 0.f;
#pragma unroll
      for (int k = 0; k < SLOTS; ++k) acc = slice_dot<T>(x[j * SLOTS + k], x[j * SLOTS + k], acc);
      p[j] = acc;
    }
    if constexpr (W_REG) {
#pragma unroll
      for (int g = 0; g < MP; ++g) {
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < NX; ++i) acc = slice_dot<T>(w[g][i], x[i], acc);
        p[MP + g] = acc;
      }
    } else {
      // W_g slices come from the cache, one gate at a time (bounded registers).
#pragma unroll 1
      for (int g = 0; g < MP; ++g) {
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < MP; ++j) {
#pragma unroll
          for (int k = 0; k < SLOTS; ++k) {
            const u32x4 wv = act[k] ? ld16(Wg + int64_t(g) * row + int64_t(j) * d + col[k])
                                    : u32x4{0, 0, 0, 0};
            acc = slice_dot<T>(wv, x[j * SLOTS + k], acc);
          }
        }
#pragma unroll
        for (int gg = 0; gg < MP; ++gg)
          if (gg == g) p[MP + gg] = acc;
      }
    }
#pragma unroll
    for (int i = 0; i < NP; ++i) p[i] = wave_sum(p[i]);
    if (lane == 0) {
#pragma unroll
      for (int i = 0; i < NP; ++i) part[buf][wid][i] = p[i];
    }
    lds_barrier();
    float tot[NP];
#pragma unroll
    for (int i = 0; i < NP; ++i) tot[i] = 0.f;
    for (int q = 0; q < nwaves; ++q) {
#pragma unroll
      for (int i = 0; i < NP; ++i) tot[i] += part[buf][q][i];
    }
    buf ^= 1;

    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < MP; ++j) ss += tot[j];
    const float r = rsqrtf(ss / float(row) + sc.eps);
    float a[MP];
#pragma unroll
    for (int g = 0; g < MP; ++g) {
      const float z = sc.gate_scale * r * tot[MP + g] + bias[g];
      a[g] = 1.f / (1.f + __expf(-z)) + sc.gate_offset;
    }
    float coef[MP];
#pragma unroll
    for (int j = 0; j < MP; ++j)
      coef[j] = sc.per_path_norm ? a[j] * rsqrtf(tot[j] / float(d) + sc.eps) : a[j];

#pragma unroll
    for (int k = 0; k < SLOTS; ++k) {
      if (act[k]) {
        float y[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
          float acc = coef[0] * Vec16<T>{x[k]}.get(i);
#pragma unroll
          for (int j = 1; j < MP; ++j) acc = fmaf(coef[j], Vec16<T>{x[j * SLOTS + k]}.get(i), acc);
          y[i] = acc;
        }
        st_nt16(Y + t * d + col[k], pack_out<T>(y));
      }
    }
    if (alpha != nullptr && tid < MP) {
#pragma unroll
      for (int g = 0; g < MP; ++g)
        if (g == tid) alpha[t * MP + g] = a[g];
    }
    if constexpr (PREFETCH) {
#pragma unroll
      for (int i = 0; i < NX; ++i) x[i] = xn[i];
    } else {
      load_token(t + gridDim.x, x);
    }
  }
}

template <typename T, int MP, int SLOTS>
static hipError_t launch_reduce_t(const void* H, const void* Wg, const float* bg, int64_t n_tok,
                                  int d, const ReduceScalars& sc, void* Y, float* alpha,
                                  hipStream_t s) {
  constexpr int VEC = Vec16<T>::N;
  const int slices = d / VEC;                                // 16-byte slices per path
  const int per_thread = (slices + SLOTS - 1) / SLOTS;      // threads needed
  const int threads = ((per_thread + kWave - 1) / kWave) * kWave;
  auto kern = hc_reduce_kernel<T, MP, SLOTS>;
  int per_cu = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, threads, 0);
  if (e != hipSuccess) return e;
  if (per_cu < 1) per_cu = 1;
  const int64_t want = int64_t(per_cu) * device_cu_count();
  const int grid = int(n_tok < want ? n_tok : want);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(threads), 0, s, static_cast<const T*>(H),
                     static_cast<const T*>(Wg), bg, n_tok, d, sc, static_cast<T*>(Y), alpha);
  return hipGetLastError();
}

template <typename T, int MP>
static hipError_t launch_reduce_s(const void* H, const void* Wg, const float* bg, int64_t n_tok,
                                  int d, const ReduceScalars& sc, void* Y, float* alpha,
                                  hipStream_t s) {
  constexpr int VEC = Vec16<T>::N;
  // Two slices per thread from 256 slices up: smaller workgroups, two of them per CU, so
  // more tokens in flight (16384 x 4 x 4096: 184 -> 121 us).
  if (d <= VEC * 256)
    return launch_reduce_t<T, MP, 1>(H, Wg, bg, n_tok, d, sc, Y, alpha, s);
  return launch_reduce_t<T, MP, 2>(H, Wg, bg, n_tok, d, sc, Y, alpha, s);
}

template <typename T>
static hipError_t launch_reduce_m(int m, const void* H, const void* Wg, const float* bg,
                                  int64_t n_tok, int d, const ReduceScalars& sc, void* Y,
                                  float* alpha, hipStream_t s) {
  switch (m) {
    case 1: return launch_reduce_s<T, 1>(H, Wg, bg, n_tok, d, sc, Y, alpha, s);
    case 2: return launch_reduce_s<T, 2>(H, Wg, bg, n_tok, d, sc, Y, alpha, s);
    case 3: return launch_reduce_s<T, 3>(H, Wg, bg, n_tok, d, sc, Y, alpha, s);
    case 4: return launch_reduce_s<T, 4>(H, Wg, bg, n_tok, d, sc, Y, alpha, s);
    case 5: return launch_reduce_s<T, 5>(H, Wg, bg, n_tok, d, sc, Y, alpha, s);
    case 6: return launch_reduce_s<T, 6>(H, Wg, bg, n_tok, d, sc, Y, alpha, s);
    case 7: return launch_reduce_s<T, 7>(H, Wg, bg, n_tok, d, sc, Y, alpha, s);
    case 8: return launch_reduce_s<T, 8>(H, Wg, bg, n_tok, d, sc, Y, alpha, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_hc_reduce(bool bf16, int m, const void* H, const void* Wg, const float* bg,
                            int64_t n_tok, int d, const ReduceScalars& sc, void* Y, float* alpha,
                            hipStream_t s) {
  return bf16 ? launch_reduce_m<bf16_t>(m, H, Wg, bg, n_tok, d, sc, Y, alpha, s)
              : launch_reduce_m<float>(m, H, Wg, bg, n_tok, d, sc, Y, alpha, s);
}

}  // namespace hdf

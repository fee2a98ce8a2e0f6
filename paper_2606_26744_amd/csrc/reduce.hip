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
// current token's reduction; for wide bf16 tokens a ring of register sets keeps two
// tokens in flight (hc_reduce_ring_kernel).
#include <type_traits>

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

// Ring form for wide bf16 tokens (m <= 4): PF tokens of a workgroup are in flight while
// it reduces the current one.  The ring holds PF + 1 register sets indexed statically
// (the token loop is unrolled by PF + 1), so no register ever moves: a load is waited
// for only when its token comes up, PF tokens after it was issued.  (Copying a
// prefetched set into the working set at the end of each token, as the kernel above
// does, waits for the newest load there, so one token is in flight at a time and every
// token costs a full memory latency.)  Gates [0, WL) take their W_g slices from LDS,
// gates [WL, MP) from registers, which keeps the ring within the register budget of
// one workgroup per CU.
template <int MP, int SLOTS, int PF, int WL, int THREADS>
__global__ void __launch_bounds__(THREADS)
hc_reduce_ring_kernel(const bf16_t* __restrict__ H, const bf16_t* __restrict__ Wg,
                      const float* __restrict__ bg, int64_t n_tok, int d, ReduceScalars sc,
                      bf16_t* __restrict__ Y, float* __restrict__ alpha) {
  constexpr int VEC = 8;
  constexpr int NP = 2 * MP;
  constexpr int NX = MP * SLOTS;
  constexpr int NWR = MP - WL;            // gates with register-resident W_g slices
  static_assert(WL >= 0 && WL <= MP, "WL");
  extern __shared__ __attribute__((aligned(16))) unsigned char ring_smem[];
  __shared__ float part[2][THREADS / kWave][NP];
  bf16_t* wl = reinterpret_cast<bf16_t*>(ring_smem);   // [WL][MP * d]

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wid = tid >> 6;
  const int nwaves = blockDim.x >> 6;
  const int nthr = blockDim.x;
  const int64_t row = int64_t(MP) * d;
  bool act[SLOTS];
  int col[SLOTS], colc[SLOTS];
#pragma unroll
  for (int k = 0; k < SLOTS; ++k) {
    col[k] = (k * nthr + tid) * VEC;
    act[k] = col[k] < d;
    colc[k] = act[k] ? col[k] : 0;
  }
  // W_g: gates >= WL in registers, gates < WL copied into LDS (each thread its own slices).
  u32x4 w[NWR > 0 ? NWR : 1][NX];
#pragma unroll
  for (int g = 0; g < MP; ++g)
#pragma unroll
    for (int j = 0; j < MP; ++j)
#pragma unroll
      for (int k = 0; k < SLOTS; ++k) {
        const u32x4 v = act[k] ? ld16(Wg + int64_t(g) * row + int64_t(j) * d + col[k])
                               : u32x4{0, 0, 0, 0};
        if (g >= WL) {
          w[g - WL][j * SLOTS + k] = v;
        } else if (act[k]) {
          *reinterpret_cast<u32x4*>(wl + int64_t(g) * row + int64_t(j) * d + col[k]) = v;
        }
      }
  float bias[MP];
#pragma unroll
  for (int g = 0; g < MP; ++g) bias[g] = bg[g];

  // Unpredicated loads (tokens past the end clamped to the last one, idle lanes on a
  // valid column, zeroed by a select) keep the compiler's outstanding-load counts exact.
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
  int buf = 0;
  auto process = [&](int64_t t, const u32x4* x) {
    float p[NP];
#pragma unroll
    for (int j = 0; j < MP; ++j) {
      float acc = 0.f;
#pragma unroll
      for (int k = 0; k < SLOTS; ++k) acc = slice_dot<bf16_t>(x[j * SLOTS + k], x[j * SLOTS + k], acc);
      p[j] = acc;
    }
#pragma unroll
    for (int g = 0; g < MP; ++g) {
      float acc = 0.f;
#pragma unroll
      for (int j = 0; j < MP; ++j)
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
          u32x4 wv;
          if (g >= WL)
            wv = w[g >= WL ? g - WL : 0][j * SLOTS + k];
          else
            wv = *reinterpret_cast<const u32x4*>(wl + int64_t(g) * row + int64_t(j) * d + colc[k]);
          acc = slice_dot<bf16_t>(wv, x[j * SLOTS + k], acc);
        }
      p[MP + g] = acc;
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
          float acc = coef[0] * Vec16<bf16_t>{x[k]}.get(i);
#pragma unroll
          for (int j = 1; j < MP; ++j)
            acc = fmaf(coef[j], Vec16<bf16_t>{x[j * SLOTS + k]}.get(i), acc);
          y[i] = acc;
        }
        st_nt16(Y + t * d + col[k], pack_out<bf16_t>(y));
      }
    }
    if (alpha != nullptr && tid < MP) {
#pragma unroll
      for (int g = 0; g < MP; ++g)
        if (g == tid) alpha[t * MP + g] = a[g];
    }
  };

  if constexpr (WL > 0) __syncthreads();   // the LDS copy of W_g is complete
  const int64_t G = gridDim.x;
  u32x4 xs[PF + 1][NX];
#pragma unroll
  for (int u = 0; u < PF; ++u) load_token(blockIdx.x + u * G, xs[u]);
  for (int64_t t = blockIdx.x; t < n_tok; t += (PF + 1) * G) {
#pragma unroll
    for (int u = 0; u <= PF; ++u) {
      const int64_t tt = t + u * G;
      load_token(tt + PF * G, xs[(u + PF) % (PF + 1)]);
      if (tt < n_tok) process(tt, xs[u]);
    }
  }
}

template <int MP, int SLOTS, int PF, int WL, int THREADS>
static hipError_t launch_reduce_ring(const void* H, const void* Wg, const float* bg, int64_t n_tok,
                                     int d, const ReduceScalars& sc, void* Y, float* alpha,
                                     hipStream_t s) {
  auto kern = hc_reduce_ring_kernel<MP, SLOTS, PF, WL, THREADS>;
  const int per_thread = (d / 8 + SLOTS - 1) / SLOTS;   // 16-byte slices per path, rounded up
  const int threads = ((per_thread + kWave - 1) / kWave) * kWave;
  const size_t lds = size_t(WL) * MP * d * sizeof(bf16_t);
  hipError_t e = hipSuccess;
  if (lds > 0) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                            hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
  }
  int per_cu = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, threads, lds);
  if (e != hipSuccess) return e;
  if (per_cu < 1) per_cu = 1;
  const int64_t want = int64_t(per_cu) * device_cu_count();
  const int grid = int(n_tok < want ? n_tok : want);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(threads), lds, s, static_cast<const bf16_t*>(H),
                     static_cast<const bf16_t*>(Wg), bg, n_tok, d, sc, static_cast<bf16_t*>(Y),
                     alpha);
  return hipGetLastError();
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
  // Tokens wider than 4096 (two slices per thread, one workgroup per CU): the ring form
  // with two tokens in flight.  65536 x 4 x 7168: 902 -> 824 us (5.7 TB/s), against 818 us
  // for a load/store probe with exactly this traffic and no arithmetic.  For m = 4 one
  // gate's W_g slices go to LDS to make room for the ring (two gates in LDS: 846 us; three
  // tokens in flight: 850 us; 512 threads, so every SIMD has two waves: 861 us).
  if constexpr (std::is_same<T, bf16_t>::value && MP <= 4) {
    if (d > 8 * 512 && d <= 8 * 1024)
      return launch_reduce_ring<MP, 2, 2, (MP == 4 ? 1 : 0), 512>(H, Wg, bg, n_tok, d, sc, Y,
                                                                    alpha, s);
  }
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

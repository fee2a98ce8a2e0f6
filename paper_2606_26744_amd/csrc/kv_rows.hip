// Copies between row-major keys/values ([n][n_heads*head_dim], one row per position) and
// the KV cache's tile layout (kc_offset / vc_offset in common.hpp), in both directions.
// A caller that computes keys and values itself (its own prefill, a cache restored from
// elsewhere) fills the cache with these, and tests read it back, without knowing the
// layout.
//
// Keys: every eight consecutive dims of one row are eight consecutive elements of the
// key tile, so an item is (row, head, octet): one 16-byte (bf16) load and store.
// Values: eight consecutive rows of one dim are eight consecutive elements of the value
// tile when the rows are eight consecutive cache rows starting at a multiple of 8; an
// item is (group of 8 input rows, head, dim): consecutive threads take consecutive dims,
// so the row-major side is coalesced, and the cache side is one 16-byte access for such
// a run, eight single elements otherwise.
#include "common.hpp"
#include "kernels.hpp"

namespace hdf {

namespace {

constexpr int kKvThreads = 256;

template <typename T>
struct alignas(16) Oct {
  T v[8];
};

template <typename T>
__device__ __forceinline__ Oct<T> ld8(const T* p) {
  return *reinterpret_cast<const Oct<T>*>(p);
}
template <typename T>
__device__ __forceinline__ void st8(T* p, const Oct<T>& o) {
  *reinterpret_cast<Oct<T>*>(p) = o;
}

__device__ __forceinline__ int64_t cache_row(const int32_t* rows, int64_t row0, int64_t i) {
  return rows != nullptr ? int64_t(rows[i]) : row0 + i;
}

// WRITE: row-major -> cache; otherwise cache -> row-major.  Rows outside [0, cap) are
// skipped on writes and read as zeros.
template <typename T, bool WRITE>
__global__ void __launch_bounds__(kKvThreads)
kv_keys_kernel(T* __restrict__ kc, int64_t cap, T* __restrict__ krows, int64_t n,
               const int32_t* __restrict__ rows, int64_t row0, int nh, int hd) {
  const int d = nh * hd;
  const int oct = hd >> 3;
  const int64_t items = n * nh * oct;
  for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < items;
       e += int64_t(gridDim.x) * blockDim.x) {
    const int64_t i = e / (nh * oct);
    const int rem = int(e - i * (nh * oct));
    const int h = rem / oct, i0 = (rem - h * oct) * 8;
    const int64_t r = cache_row(rows, row0, i);
    const bool in = r >= 0 && r < cap;
    T* rm = krows + i * d + h * hd + i0;
    T* tc = kc + int64_t(h) * cap * hd + (in ? kc_index(r, i0, hd) : 0);
    if constexpr (WRITE) {
      if (in) st8(tc, ld8(rm));
    } else {
      Oct<T> o;
      if (in) {
        o = ld8(tc);
      } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) o.v[k] = T(0);
      }
      st8(rm, o);
    }
  }
}

template <typename T, bool WRITE>
__global__ void __launch_bounds__(kKvThreads)
kv_values_kernel(T* __restrict__ vc, int64_t cap, T* __restrict__ vrows, int64_t n,
                 const int32_t* __restrict__ rows, int64_t row0, int nh, int hd) {
  const int d = nh * hd;
  const int64_t groups = (n + 7) >> 3;
  const int64_t items = groups * d;
  for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < items;
       e += int64_t(gridDim.x) * blockDim.x) {
    const int64_t g = e / d;
    const int col = int(e - g * d);
    const int h = col / hd, i = col - h * hd;
    const int64_t i0 = 8 * g;
    const int cnt = int(n - i0 < 8 ? n - i0 : 8);
    T* head = vc + int64_t(h) * cap * hd;
    const int64_t r0 = cache_row(rows, row0, i0);
    bool run = cnt == 8 && r0 >= 0 && r0 + 8 <= cap && (r0 & 7) == 0;
    if (run && rows != nullptr) {
#pragma unroll
      for (int k = 1; k < 8; ++k) run = run && int64_t(rows[i0 + k]) == r0 + k;
    }
    if (run) {
      T* tc = head + vc_index(r0, i, hd);
      if constexpr (WRITE) {
        Oct<T> o;
#pragma unroll
        for (int k = 0; k < 8; ++k) o.v[k] = vrows[(i0 + k) * d + col];
        st8(tc, o);
      } else {
        const Oct<T> o = ld8(tc);
#pragma unroll
        for (int k = 0; k < 8; ++k) vrows[(i0 + k) * d + col] = o.v[k];
      }
    } else {
      for (int k = 0; k < cnt; ++k) {
        const int64_t r = cache_row(rows, row0, i0 + k);
        const bool in = r >= 0 && r < cap;
        if constexpr (WRITE) {
          if (in) head[vc_index(r, i, hd)] = vrows[(i0 + k) * d + col];
        } else {
          vrows[(i0 + k) * d + col] = in ? head[vc_index(r, i, hd)] : T(0);
        }
      }
    }
  }
}

unsigned grid_for(int64_t items) {
  int64_t b = (items + kKvThreads - 1) / kKvThreads;
  if (b > 65536) b = 65536;
  return unsigned(b < 1 ? 1 : b);
}

template <typename T, bool WRITE>
hipError_t kv_rows_t(void* kc, void* vc, int64_t cap, void* krows, void* vrows, int64_t n,
                     const int32_t* rows, int64_t row0, int nh, int hd, hipStream_t s) {
  if (kc != nullptr && krows != nullptr)
    hipLaunchKernelGGL((kv_keys_kernel<T, WRITE>), dim3(grid_for(n * nh * (hd / 8))),
                       dim3(kKvThreads), 0, s, static_cast<T*>(kc), cap, static_cast<T*>(krows),
                       n, rows, row0, nh, hd);
  if (vc != nullptr && vrows != nullptr)
    hipLaunchKernelGGL((kv_values_kernel<T, WRITE>), dim3(grid_for(((n + 7) / 8) * nh * hd)),
                       dim3(kKvThreads), 0, s, static_cast<T*>(vc), cap, static_cast<T*>(vrows),
                       n, rows, row0, nh, hd);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_kv_rows(bool bf16, bool write, void* kc, void* vc, int64_t cap, void* krows,
                          void* vrows, int64_t n, const int32_t* rows, int64_t row0, int nh,
                          int hd, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (bf16)
    return write ? kv_rows_t<bf16_t, true>(kc, vc, cap, krows, vrows, n, rows, row0, nh, hd, s)
                 : kv_rows_t<bf16_t, false>(kc, vc, cap, krows, vrows, n, rows, row0, nh, hd, s);
  return write ? kv_rows_t<float, true>(kc, vc, cap, krows, vrows, n, rows, row0, nh, hd, s)
               : kv_rows_t<float, false>(kc, vc, cap, krows, vrows, n, rows, row0, nh, hd, s);
}

}  // namespace hdf

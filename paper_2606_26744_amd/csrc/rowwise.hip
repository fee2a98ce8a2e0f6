// Row-wise kernels of the block drafter: RMSNorms, the token-embedding gather,
// split-K reduction fused with the residual update and the next RMSNorm, the
// projection epilogues (RoPE + scatter into the attention layouts, SiLU gate)
// and the per-row plan of the context rows projected in this step.
//
// All are HBM/L2-bound elementwise passes over rows of width d: one 256-thread
// workgroup per row (norm kernels) with 16-byte or 8-byte accesses, fp32
// arithmetic, one rounding to the working dtype at every stored tensor.
#include "common.hpp"
#include "kernels.hpp"

namespace hdf {

constexpr int kRowThreads = 256;

template <typename T>
__device__ __forceinline__ void load4(const T* p, float* v);
template <>
__device__ __forceinline__ void load4<bf16_t>(const bf16_t* p, float* v) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  v[0] = lo_bf(u.x); v[1] = hi_bf(u.x); v[2] = lo_bf(u.y); v[3] = hi_bf(u.y);
}
template <>
__device__ __forceinline__ void load4<float>(const float* p, float* v) {
  const float4 u = *reinterpret_cast<const float4*>(p);
  v[0] = u.x; v[1] = u.y; v[2] = u.z; v[3] = u.w;
}
template <typename T>
__device__ __forceinline__ void store4(T* p, const float* v);
template <>
__device__ __forceinline__ void store4<bf16_t>(bf16_t* p, const float* v) {
  *reinterpret_cast<uint2*>(p) = make_uint2(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]));
}
template <>
__device__ __forceinline__ void store4<float>(float* p, const float* v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
template <typename T>
__device__ __forceinline__ void store1(T* p, float v);
template <>
__device__ __forceinline__ void store1<bf16_t>(bf16_t* p, float v) { *p = f2bf(v); }
template <>
__device__ __forceinline__ void store1<float>(float* p, float v) { *p = v; }

__device__ __forceinline__ float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  if (lane == 0) sh[wid] = v;
  __syncthreads();
  float t = 0.f;
  for (int w = 0; w < int(blockDim.x >> 6); ++w) t += sh[w];
  __syncthreads();
  return t;
}

// Rows are at most 8192 wide: 8 groups of 4 per thread at 256 threads.
constexpr int kMaxGroups = 8;

template <typename T>
__global__ void __launch_bounds__(kRowThreads)
row_norm_kernel(const T* __restrict__ in, const float* __restrict__ gamma, float eps, int d,
                T* __restrict__ out) {
  __shared__ float sh[kRowThreads / 64];
  const int64_t r = blockIdx.x;
  const T* x = in + r * d;
  float v[kMaxGroups][4];
  float ss = 0.f;
#pragma unroll
  for (int g = 0; g < kMaxGroups; ++g) {
    const int c = (g * kRowThreads + threadIdx.x) * 4;
    if (c < d) {
      load4<T>(x + c, v[g]);
#pragma unroll
      for (int j = 0; j < 4; ++j) ss = fmaf(v[g][j], v[g][j], ss);
    }
  }
  ss = block_sum(ss, sh);
  const float rs = rsqrtf(ss / float(d) + eps);
#pragma unroll
  for (int g = 0; g < kMaxGroups; ++g) {
    const int c = (g * kRowThreads + threadIdx.x) * 4;
    if (c < d) {
      float o[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = v[g][j] * rs * (gamma ? gamma[c + j] : 1.f);
      store4<T>(out + r * d + c, o);
    }
  }
}

template <typename T>
__global__ void __launch_bounds__(kRowThreads)
embed_norm_kernel(const int32_t* __restrict__ tokens, const T* __restrict__ emb,
                  const float* __restrict__ gamma, float eps, int d, float* __restrict__ h,
                  T* __restrict__ u) {
  __shared__ float sh[kRowThreads / 64];
  const int64_t r = blockIdx.x;
  const T* x = emb + int64_t(tokens[r]) * d;
  float v[kMaxGroups][4];
  float ss = 0.f;
#pragma unroll
  for (int g = 0; g < kMaxGroups; ++g) {
    const int c = (g * kRowThreads + threadIdx.x) * 4;
    if (c < d) {
      load4<T>(x + c, v[g]);
      *reinterpret_cast<float4*>(h + r * d + c) = make_float4(v[g][0], v[g][1], v[g][2], v[g][3]);
#pragma unroll
      for (int j = 0; j < 4; ++j) ss = fmaf(v[g][j], v[g][j], ss);
    }
  }
  ss = block_sum(ss, sh);
  const float rs = rsqrtf(ss / float(d) + eps);
#pragma unroll
  for (int g = 0; g < kMaxGroups; ++g) {
    const int c = (g * kRowThreads + threadIdx.x) * 4;
    if (c < d) {
      float o[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = v[g][j] * rs * (gamma ? gamma[c + j] : 1.f);
      store4<T>(u + r * d + c, o);
    }
  }
}

template <typename T>
__global__ void __launch_bounds__(kRowThreads)
residual_norm_kernel(const float* __restrict__ parts, int S, int64_t M,
                     const float* __restrict__ gamma, float eps, int d, float* __restrict__ h,
                     T* __restrict__ u) {
  __shared__ float sh[kRowThreads / 64];
  const int64_t r = blockIdx.x;
  float v[kMaxGroups][4];
  float ss = 0.f;
#pragma unroll
  for (int g = 0; g < kMaxGroups; ++g) {
    const int c = (g * kRowThreads + threadIdx.x) * 4;
    if (c < d) {
      float4 acc = *reinterpret_cast<const float4*>(parts + r * d + c);
      for (int z = 1; z < S; ++z) {
        const float4 t = *reinterpret_cast<const float4*>(parts + (int64_t(z) * M + r) * d + c);
        acc.x += t.x; acc.y += t.y; acc.z += t.z; acc.w += t.w;
      }
      float4 hv = *reinterpret_cast<const float4*>(h + r * d + c);
      hv.x += acc.x; hv.y += acc.y; hv.z += acc.z; hv.w += acc.w;
      *reinterpret_cast<float4*>(h + r * d + c) = hv;
      v[g][0] = hv.x; v[g][1] = hv.y; v[g][2] = hv.z; v[g][3] = hv.w;
#pragma unroll
      for (int j = 0; j < 4; ++j) ss = fmaf(v[g][j], v[g][j], ss);
    }
  }
  ss = block_sum(ss, sh);
  const float rs = rsqrtf(ss / float(d) + eps);
#pragma unroll
  for (int g = 0; g < kMaxGroups; ++g) {
    const int c = (g * kRowThreads + threadIdx.x) * 4;
    if (c < d) {
      float o[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = v[g][j] * rs * (gamma ? gamma[c + j] : 1.f);
      store4<T>(u + r * d + c, o);
    }
  }
}

// Rows of y_new -> (position, cache row): sequence s owns rows new_offsets[s] ..
// new_offsets[s+1]-1, which are its last n_s context positions.
__global__ void plan_rows_kernel(const int32_t* __restrict__ ctx_len,
                                 const int32_t* __restrict__ new_offsets,
                                 const int32_t* __restrict__ kv_offsets, int n_seq, int64_t n_new,
                                 int32_t* __restrict__ plan_pos, int32_t* __restrict__ plan_row) {
  const int64_t r = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (r >= n_new) return;
  int lo = 0, hi = n_seq - 1;  // last s with new_offsets[s] <= r
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (new_offsets[mid] <= r) lo = mid; else hi = mid - 1;
  }
  const int s = lo;
  const int ns = new_offsets[s + 1] - new_offsets[s];
  const int pos = ctx_len[s] - ns + int(r - new_offsets[s]);
  plan_pos[r] = pos;
  plan_row[r] = kv_offsets[s] + pos;
}

__device__ __forceinline__ void row_dest(const QkvEpiArgs& a, int r, int& pos, int64_t& drow,
                                         int& s, int& kslot) {
  if (a.first_part == 0) {
    s = r / a.B;
    kslot = r - s * a.B;
    pos = a.ctx_len[s] + kslot;
    drow = int64_t(s) * 64 + kslot;
  } else {
    s = 0;
    kslot = 0;
    pos = a.plan_pos[r];
    drow = a.plan_row[r];
  }
}

// Q and K columns: sum the split-K partials, rotate pairs (i, i+hd/2), store.
// grid (M, number of rotated parts), one pair per thread iteration.
template <typename T>
__global__ void __launch_bounds__(kRowThreads)
qk_rope_kernel(QkvEpiArgs a) {
  const int r = blockIdx.x;
  const int part = a.first_part + blockIdx.y;  // 0 = Q, 1 = K
  const int ncol = (3 - a.first_part) * a.d;
  const int half = a.hd / 2;
  int pos, s, kslot;
  int64_t drow;
  row_dest(a, r, pos, drow, s, kslot);
  const int64_t base = int64_t(r) * ncol + int64_t(part - a.first_part) * a.d;
  for (int j = threadIdx.x; j < a.d / 2; j += kRowThreads) {
    const int hh = j / half, i = j - hh * half;
    const int64_t c1 = base + int64_t(hh) * a.hd + i;
    float x1 = 0.f, x2 = 0.f;
    for (int z = 0; z < a.S; ++z) {
      const int64_t off = int64_t(z) * a.M * ncol;
      x1 += a.parts[off + c1];
      x2 += a.parts[off + c1 + half];
    }
    float y1 = x1, y2 = x2;
    if (a.rope_cs != nullptr) {
      const float2 cs = *reinterpret_cast<const float2*>(a.rope_cs + (int64_t(pos) * half + i) * 2);
      y1 = x1 * cs.x - x2 * cs.y;
      y2 = x2 * cs.x + x1 * cs.y;
    }
    T* dst;
    if (part == 0)
      dst = static_cast<T*>(a.q) + ((int64_t(s) * a.nh + hh) * a.B + kslot) * a.hd;
    else
      dst = static_cast<T*>(a.k) + (int64_t(hh) * a.cap + drow) * a.hd;
    store1<T>(dst + i, y1);
    store1<T>(dst + i + half, y2);
  }
}

// V columns: sum partials and write transposed (positions fastest) through an LDS
// tile of 64 rows x 64 columns.
template <typename T>
__global__ void __launch_bounds__(kRowThreads)
v_transpose_kernel(QkvEpiArgs a) {
  __shared__ float tile[64][65];
  const int r0 = blockIdx.x * 64;
  const int c0 = blockIdx.y * 64;
  const int ncol = (3 - a.first_part) * a.d;
  const int64_t vcol = int64_t(2 - a.first_part) * a.d;
  for (int e = threadIdx.x; e < 64 * 64; e += kRowThreads) {
    const int rr = e >> 6, cc = e & 63;
    float x = 0.f;
    if (r0 + rr < a.M) {
      for (int z = 0; z < a.S; ++z)
        x += a.parts[(int64_t(z) * a.M + r0 + rr) * ncol + vcol + c0 + cc];
    }
    tile[rr][cc] = x;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 64 * 64; e += kRowThreads) {
    const int cc = e >> 6, rr = e & 63;
    const int r = r0 + rr;
    if (r >= a.M) continue;
    int pos, s, kslot;
    int64_t drow;
    row_dest(a, r, pos, drow, s, kslot);
    const int col = c0 + cc;
    const int hh = col / a.hd, i = col - hh * a.hd;
    T* dst = static_cast<T*>(a.vt) + (int64_t(hh) * a.hd + i) * a.cap + drow;
    store1<T>(dst, tile[rr][cc]);
  }
}

template <typename T>
__global__ void __launch_bounds__(kRowThreads)
silu_kernel(const float* __restrict__ parts, int S, int64_t M, int F, T* __restrict__ act) {
  const int64_t n4 = M * F / 4;
  for (int64_t e = int64_t(blockIdx.x) * kRowThreads + threadIdx.x; e < n4;
       e += int64_t(gridDim.x) * kRowThreads) {
    const int64_t idx = e * 4;
    const int64_t r = idx / F;
    const int c = int(idx - r * F);
    float g[4] = {0, 0, 0, 0}, u[4] = {0, 0, 0, 0};
    for (int z = 0; z < S; ++z) {
      const float* row = parts + (int64_t(z) * M + r) * (2 * int64_t(F));
      const float4 gv = *reinterpret_cast<const float4*>(row + c);
      const float4 uv = *reinterpret_cast<const float4*>(row + F + c);
      g[0] += gv.x; g[1] += gv.y; g[2] += gv.z; g[3] += gv.w;
      u[0] += uv.x; u[1] += uv.y; u[2] += uv.z; u[3] += uv.w;
    }
    float o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = g[j] / (1.f + __expf(-g[j])) * u[j];
    store4<T>(act + idx, o);
  }
}

// ---------------------------------------------------------------------------- host side

hipError_t launch_plan_rows(const int32_t* ctx_len, const int32_t* new_offsets,
                            const int32_t* kv_offsets, int n_seq, int64_t n_new, int32_t* plan_pos,
                            int32_t* plan_row, hipStream_t s) {
  if (n_new <= 0) return hipSuccess;
  hipLaunchKernelGGL(plan_rows_kernel, dim3(unsigned((n_new + 255) / 256)), dim3(256), 0, s,
                     ctx_len, new_offsets, kv_offsets, n_seq, n_new, plan_pos, plan_row);
  return hipGetLastError();
}

hipError_t launch_row_norm(bool bf16, const void* in, const float* gamma, float eps, int64_t rows,
                           int d, void* out, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(row_norm_kernel<bf16_t>, dim3(unsigned(rows)), dim3(kRowThreads), 0, s,
                       static_cast<const bf16_t*>(in), gamma, eps, d, static_cast<bf16_t*>(out));
  else
    hipLaunchKernelGGL(row_norm_kernel<float>, dim3(unsigned(rows)), dim3(kRowThreads), 0, s,
                       static_cast<const float*>(in), gamma, eps, d, static_cast<float*>(out));
  return hipGetLastError();
}

hipError_t launch_embed_norm(bool bf16, const int32_t* tokens, const void* emb, const float* gamma,
                             float eps, int64_t rows, int d, float* h, void* u, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(embed_norm_kernel<bf16_t>, dim3(unsigned(rows)), dim3(kRowThreads), 0, s,
                       tokens, static_cast<const bf16_t*>(emb), gamma, eps, d, h,
                       static_cast<bf16_t*>(u));
  else
    hipLaunchKernelGGL(embed_norm_kernel<float>, dim3(unsigned(rows)), dim3(kRowThreads), 0, s,
                       tokens, static_cast<const float*>(emb), gamma, eps, d, h,
                       static_cast<float*>(u));
  return hipGetLastError();
}

hipError_t launch_residual_norm(bool bf16, const float* parts, int S, const float* gamma, float eps,
                                int64_t rows, int d, float* h, void* u, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(residual_norm_kernel<bf16_t>, dim3(unsigned(rows)), dim3(kRowThreads), 0, s,
                       parts, S, rows, gamma, eps, d, h, static_cast<bf16_t*>(u));
  else
    hipLaunchKernelGGL(residual_norm_kernel<float>, dim3(unsigned(rows)), dim3(kRowThreads), 0, s,
                       parts, S, rows, gamma, eps, d, h, static_cast<float*>(u));
  return hipGetLastError();
}

hipError_t launch_qkv_epilogue(bool bf16, const QkvEpiArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  const dim3 g1(unsigned(a.M), unsigned(2 - a.first_part));
  const dim3 g2(unsigned((a.M + 63) / 64), unsigned(a.d / 64));
  if (bf16) {
    hipLaunchKernelGGL(qk_rope_kernel<bf16_t>, g1, dim3(kRowThreads), 0, s, a);
    hipLaunchKernelGGL(v_transpose_kernel<bf16_t>, g2, dim3(kRowThreads), 0, s, a);
  } else {
    hipLaunchKernelGGL(qk_rope_kernel<float>, g1, dim3(kRowThreads), 0, s, a);
    hipLaunchKernelGGL(v_transpose_kernel<float>, g2, dim3(kRowThreads), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_silu_epilogue(bool bf16, const float* parts, int S, int64_t M, int F, void* act,
                                hipStream_t s) {
  if (M <= 0) return hipSuccess;
  const int64_t n4 = M * F / 4;
  int64_t blocks = (n4 + kRowThreads - 1) / kRowThreads;
  if (blocks > 65536) blocks = 65536;
  if (bf16)
    hipLaunchKernelGGL(silu_kernel<bf16_t>, dim3(unsigned(blocks)), dim3(kRowThreads), 0, s, parts,
                       S, M, F, static_cast<bf16_t*>(act));
  else
    hipLaunchKernelGGL(silu_kernel<float>, dim3(unsigned(blocks)), dim3(kRowThreads), 0, s, parts, S,
                       M, F, static_cast<float*>(act));
  return hipGetLastError();
}

}  // namespace hdf

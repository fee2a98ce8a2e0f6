// Row-wise kernels of the block drafter: the call's first kernel (per-row plan of
// the context rows projected in this call, their RMSNorm, the token-embedding
// gather and the block's first RMSNorm), split-K reduction fused with the residual
// update and the next RMSNorm, and the projection epilogues (RoPE + scatter into
// the attention layouts, SiLU gate).
//
// All are HBM/L2-bound elementwise passes over rows of width d: one 256-thread
// workgroup per row (norm kernels) with 16-byte or 8-byte accesses, fp32
// arithmetic, one rounding to the working dtype at every stored tensor.
#include "common.hpp"
#include "kernels.hpp"
#include "qkv_epi.hpp"

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

// First kernel of a drafter call, one 256-thread workgroup per row:
//   context rows: (position, cache row) of the row, c = RMSNorm(y) * ctx_norm; a row past
//                 its sequence's new rows (new_counts, or past new_offsets[n_seq]) or
//                 outside the cached range gets position and cache row -1 and is not
//                 stored by the epilogue;
//   block rows:   h = float(emb[token]), u = RMSNorm(h) * attn_norm[0].
template <typename T>
__device__ __forceinline__ void load8(const T* p, float* v);
template <>
__device__ __forceinline__ void load8<bf16_t>(const bf16_t* p, float* v) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  v[0] = lo_bf(u.x); v[1] = hi_bf(u.x); v[2] = lo_bf(u.y); v[3] = hi_bf(u.y);
  v[4] = lo_bf(u.z); v[5] = hi_bf(u.z); v[6] = lo_bf(u.w); v[7] = hi_bf(u.w);
}
template <>
__device__ __forceinline__ void load8<float>(const float* p, float* v) {
  load4<float>(p, v);
  load4<float>(p + 4, v + 4);
}
template <typename T>
__device__ __forceinline__ void store8(T* p, const float* v);
template <>
__device__ __forceinline__ void store8<bf16_t>(bf16_t* p, const float* v) {
  *reinterpret_cast<uint4*>(p) = make_uint4(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]),
                                            pack_bf2(v[4], v[5]), pack_bf2(v[6], v[7]));
}
template <>
__device__ __forceinline__ void store8<float>(float* p, const float* v) {
  store4<float>(p, v);
  store4<float>(p + 4, v + 4);
}

// Eight consecutive elements per thread and group: rows up to 4 x 8 x 256 = 8192 wide.
constexpr int kMaxGroups8 = 4;

template <typename T>
__global__ void __launch_bounds__(kRowThreads)
prep_kernel(PrepArgs a) {
  __shared__ float sh[kRowThreads / 64];
  const int b = blockIdx.x;
  const bool ctx = b < a.n_ctx;
  const int64_t r = ctx ? a.r0 + b : int64_t(b - a.n_ctx);
  const T* x = ctx ? static_cast<const T*>(a.y) + r * a.d
                   : static_cast<const T*>(a.emb) + int64_t(a.tokens[r]) * a.d;
  // The row's loads first, so that the plan's dependent loads below overlap them.
  float v[kMaxGroups8][8];
#pragma unroll
  for (int g = 0; g < kMaxGroups8; ++g) {
    const int c = (g * kRowThreads + threadIdx.x) * 8;
    if (c < a.d) load8<T>(x + c, v[g]);
  }
  if (ctx && threadIdx.x == 0) {
    int lo = 0, hi = a.n_seq - 1;   // last s with new_offsets[s] <= r
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (a.new_offsets[mid] <= r) lo = mid; else hi = mid - 1;
    }
    int ns = a.new_offsets[lo + 1] - a.new_offsets[lo];
    if (a.new_counts != nullptr) ns = min(ns, max(a.new_counts[lo], 0));
    const int j = int(r - a.new_offsets[lo]);
    const int pos = a.ctx_len[lo] - ns + j;
    const bool valid = r < a.new_offsets[a.n_seq] && j < ns && pos >= 0 &&
                       (a.page_table == nullptr || (pos >> 6) < a.max_pages);
    a.plan_pos[r] = valid ? pos : -1;
    a.plan_row[r] = !valid ? -1
                    : a.page_table != nullptr
                        ? a.page_table[int64_t(lo) * a.max_pages + (pos >> 6)] * 64 + (pos & 63)
                        : a.kv_offsets[lo] + pos;
  }
  float* hrow = ctx ? nullptr : a.h + r * a.d;
  const float* gamma = ctx ? a.ctx_gamma : a.attn_gamma;
  T* out = ctx ? static_cast<T*>(a.c) + int64_t(b) * a.d : static_cast<T*>(a.u) + r * a.d;
  float ss = 0.f;
#pragma unroll
  for (int g = 0; g < kMaxGroups8; ++g) {
    const int c = (g * kRowThreads + threadIdx.x) * 8;
    if (c < a.d) {
      if (hrow != nullptr) store8<float>(hrow + c, v[g]);
#pragma unroll
      for (int j = 0; j < 8; ++j) ss = fmaf(v[g][j], v[g][j], ss);
    }
  }
  ss = block_sum(ss, sh);
  const float rs = rsqrtf(ss / float(a.d) + a.eps);
#pragma unroll
  for (int g = 0; g < kMaxGroups8; ++g) {
    const int c = (g * kRowThreads + threadIdx.x) * 8;
    if (c < a.d) {
      float gm[8];
      if (gamma != nullptr) {
        load8<float>(gamma + c, gm);
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) gm[j] = 1.f;
      }
      float o[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] = v[g][j] * rs * gm[j];
      store8<T>(out + c, o);
    }
  }
}

// One 1024-thread workgroup per row: every thread owns at most two float4 groups, so
// all split-K partial loads of a row are in flight together.
constexpr int kResThreads = 1024;

template <typename T>
__global__ void __launch_bounds__(kResThreads)
residual_norm_kernel(const float* __restrict__ parts, int S, int64_t M,
                     const float* __restrict__ gamma, float eps, int d, float* __restrict__ h,
                     T* __restrict__ u) {
  __shared__ float sh[kResThreads / 64];
  const int64_t r = blockIdx.x;
  float v[2][4];
  float ss = 0.f;
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    const int c = (g * kResThreads + threadIdx.x) * 4;
    if (c < d) {
      float4 acc = *reinterpret_cast<const float4*>(h + r * d + c);
      float4 p = *reinterpret_cast<const float4*>(parts + r * d + c);
#pragma unroll 4
      for (int z = 1; z < S; ++z) {
        const float4 t = *reinterpret_cast<const float4*>(parts + (int64_t(z) * M + r) * d + c);
        p.x += t.x; p.y += t.y; p.z += t.z; p.w += t.w;
      }
      acc.x += p.x; acc.y += p.y; acc.z += p.z; acc.w += p.w;
      *reinterpret_cast<float4*>(h + r * d + c) = acc;
      v[g][0] = acc.x; v[g][1] = acc.y; v[g][2] = acc.z; v[g][3] = acc.w;
#pragma unroll
      for (int j = 0; j < 4; ++j) ss = fmaf(v[g][j], v[g][j], ss);
    }
  }
  ss = block_sum(ss, sh);
  const float rs = rsqrtf(ss / float(d) + eps);
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    const int c = (g * kResThreads + threadIdx.x) * 4;
    if (c < d) {
      float o[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = v[g][j] * rs * (gamma ? gamma[c + j] : 1.f);
      store4<T>(u + r * d + c, o);
    }
  }
}

// Projection epilogue: one workgroup per tile of kQkvRows rows x one head (qkv_epi.hpp);
// the tiles of the first set of rows, then those of the optional second one.
template <typename T, int HD>
__global__ void __launch_bounds__(kQkvThreads)
qkv_epilogue_kernel(QkvEpiArgs a0, QkvEpiArgs a1, int nb0) {
  __shared__ QkvEpiSmem<HD> sm;
  const bool second = int(blockIdx.x) >= nb0;
  const QkvEpiArgs a = second ? a1 : a0;
  const int r0 = (second ? int(blockIdx.x) - nb0 : int(blockIdx.x)) * kQkvRows;
  qkv_epi_tile<T, HD>(a, r0, min(kQkvRows, a.M - r0), int(blockIdx.y), int(threadIdx.x), sm);
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
    for (int j = 0; j < 4; ++j) o[j] = silu_mul(g[j], u[j]);
    store4<T>(act + idx, o);
  }
}

// out = sum_z parts[z] (+ bias per column), rounded to the working dtype; rows of N
// columns (N % 4 == 0), four consecutive columns per item.
template <typename T>
__global__ void __launch_bounds__(kRowThreads)
split_sum_store_kernel(const float* __restrict__ parts, int S, int64_t M, int N,
                       const float* __restrict__ bias, T* __restrict__ out) {
  const int64_t n4 = M * N / 4;
  const int64_t zs = M * N;
  for (int64_t e = int64_t(blockIdx.x) * kRowThreads + threadIdx.x; e < n4;
       e += int64_t(gridDim.x) * kRowThreads) {
    const int64_t idx = e * 4;
    const int c = int(idx % N);
    float4 x = *reinterpret_cast<const float4*>(parts + idx);
    for (int z = 1; z < S; ++z) {
      const float4 t = *reinterpret_cast<const float4*>(parts + z * zs + idx);
      x.x += t.x; x.y += t.y; x.z += t.z; x.w += t.w;
    }
    float o[4] = {x.x, x.y, x.z, x.w};
    if (bias != nullptr) {
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] += bias[c + j];
    }
    store4<T>(out + idx, o);
  }
}

// ---------------------------------------------------------------------------- host side

hipError_t launch_prep(bool bf16, const PrepArgs& a, hipStream_t s) {
  const int64_t wgs = int64_t(a.n_ctx) + a.n_blk;
  if (wgs <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(prep_kernel<bf16_t>, dim3(unsigned(wgs)), dim3(kRowThreads), 0, s, a);
  else
    hipLaunchKernelGGL(prep_kernel<float>, dim3(unsigned(wgs)), dim3(kRowThreads), 0, s, a);
  return hipGetLastError();
}

// After a verification round: sequence s committed accept_len[s] + 1 positions (its
// accepted drafts and the target's token after them), which become its newest context
// rows for the next round; that token is the next block's anchor (slot 0).
__global__ void advance_context_kernel(int n_seq, const int32_t* __restrict__ accept_len,
                                       int32_t* __restrict__ ctx_len, int32_t* __restrict__ new_counts,
                                       const int32_t* __restrict__ next_anchor,
                                       int32_t* __restrict__ block_tokens, int B) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= n_seq) return;
  const int n = accept_len[s] + 1;
  ctx_len[s] += n;
  if (new_counts != nullptr) new_counts[s] = n;
  if (block_tokens != nullptr) block_tokens[int64_t(s) * B] = next_anchor[s];
}

hipError_t launch_advance_context(int n_seq, const int32_t* accept_len, int32_t* ctx_len,
                                  int32_t* new_counts, const int32_t* next_anchor,
                                  int32_t* block_tokens, int B, hipStream_t s) {
  if (n_seq <= 0) return hipSuccess;
  hipLaunchKernelGGL(advance_context_kernel, dim3(unsigned((n_seq + 255) / 256)), dim3(256), 0, s,
                     n_seq, accept_len, ctx_len, new_counts, next_anchor, block_tokens, B);
  return hipGetLastError();
}

hipError_t launch_residual_norm(bool bf16, const float* parts, int S, const float* gamma, float eps,
                                int64_t rows, int d, float* h, void* u, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(residual_norm_kernel<bf16_t>, dim3(unsigned(rows)), dim3(kResThreads), 0, s,
                       parts, S, rows, gamma, eps, d, h, static_cast<bf16_t*>(u));
  else
    hipLaunchKernelGGL(residual_norm_kernel<float>, dim3(unsigned(rows)), dim3(kResThreads), 0, s,
                       parts, S, rows, gamma, eps, d, h, static_cast<float*>(u));
  return hipGetLastError();
}

hipError_t launch_qkv_epilogue2(bool bf16, const QkvEpiArgs& a, const QkvEpiArgs& b,
                                hipStream_t s) {
  const int nb0 = a.M > 0 ? (a.M + kQkvRows - 1) / kQkvRows : 0;
  const int nb1 = b.M > 0 ? (b.M + kQkvRows - 1) / kQkvRows : 0;
  if (nb0 + nb1 == 0) return hipSuccess;
  const int nh = nb0 > 0 ? a.nh : b.nh, hd = nb0 > 0 ? a.hd : b.hd;
  const dim3 grid(unsigned(nb0 + nb1), unsigned(nh));
  if (bf16) {
    if (hd == 128)
      hipLaunchKernelGGL((qkv_epilogue_kernel<bf16_t, 128>), grid, dim3(kQkvThreads), 0, s, a, b, nb0);
    else
      hipLaunchKernelGGL((qkv_epilogue_kernel<bf16_t, 64>), grid, dim3(kQkvThreads), 0, s, a, b, nb0);
  } else {
    if (hd == 128)
      hipLaunchKernelGGL((qkv_epilogue_kernel<float, 128>), grid, dim3(kQkvThreads), 0, s, a, b, nb0);
    else
      hipLaunchKernelGGL((qkv_epilogue_kernel<float, 64>), grid, dim3(kQkvThreads), 0, s, a, b, nb0);
  }
  return hipGetLastError();
}

hipError_t launch_qkv_epilogue(bool bf16, const QkvEpiArgs& a, hipStream_t s) {
  QkvEpiArgs none = a;
  none.M = 0;
  return launch_qkv_epilogue2(bf16, a, none, s);
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

hipError_t launch_split_sum_store(bool bf16, const float* parts, int S, int64_t M, int N,
                                  const float* bias, void* out, hipStream_t s) {
  const int64_t n4 = M * N / 4;
  if (n4 <= 0) return hipSuccess;
  int64_t blocks = (n4 + kRowThreads - 1) / kRowThreads;
  if (blocks > 65536) blocks = 65536;
  if (bf16)
    hipLaunchKernelGGL(split_sum_store_kernel<bf16_t>, dim3(unsigned(blocks)), dim3(kRowThreads), 0,
                       s, parts, S, M, N, bias, static_cast<bf16_t*>(out));
  else
    hipLaunchKernelGGL(split_sum_store_kernel<float>, dim3(unsigned(blocks)), dim3(kRowThreads), 0,
                       s, parts, S, M, N, bias, static_cast<float*>(out));
  return hipGetLastError();
}

}  // namespace hdf

// LM-head KL distillation forward (Sec. 2.4): for the first P draft positions of every
// block, KL(softmax(t/T) || softmax(z/T)) between the teacher logits t = LMHead of the
// path-mean target state at position a+k-1 and the draft logits z of slot k, the
// cross entropy of the draft logits against the ground truth, and
//     L_KL = T^2 / P * mean_blocks sum_k KL,   L = L_CE + alpha * L_KL.
// The teacher's projection is the LM-head GEMM of gemm.hip (logits kept); the KL of a
// row pair is one split pass over the vocabulary with online log-sum-exps.
#include "common.hpp"
#include "kernels.hpp"

namespace hdf {

constexpr int kKlThreads = 256;

__device__ __forceinline__ float to_f32(bf16_t x) { return bf2f(x); }
__device__ __forceinline__ float to_f32(float x) { return x; }
template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) { return f2bf(x); }
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }

// Teacher state: mean over the m paths, RMSNorm, * gamma, rounded to T.
template <typename T>
__global__ void __launch_bounds__(kKlThreads)
pool_norm_kernel(const T* __restrict__ H, int m, int d, const float* __restrict__ gamma, float eps,
                 T* __restrict__ out) {
  __shared__ float sh[kKlThreads / 64];
  __shared__ float row[8192];
  const int64_t r = blockIdx.x;
  const T* h = H + r * int64_t(m) * d;
  float ss = 0.f;
  for (int c = threadIdx.x; c < d; c += kKlThreads) {
    float acc = 0.f;
    for (int j = 0; j < m; ++j) acc += to_f32(h[int64_t(j) * d + c]);
    const float x = acc / float(m);
    row[c] = x;
    ss = fmaf(x, x, ss);
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
  for (int w = 0; w < kKlThreads / 64; ++w) tot += sh[w];
  const float rs = rsqrtf(tot / float(d) + eps);
  for (int c = threadIdx.x; c < d; c += kKlThreads)
    out[r * d + c] = from_f32<T>(row[c] * rs * (gamma ? gamma[c] : 1.f));
}

// Online state of one part of a (teacher, student) row pair at temperature T:
// teacher log-sum-exp (mt, st), a = sum_v exp(t_v/T - mt) * (t_v - z_v)/T, and the
// student log-sum-exp (mz, sz).
struct KlState {
  float mt, st, a, mz, sz;
};

__device__ __forceinline__ void kl_merge(KlState& x, const KlState& y) {
  if (y.st > 0.f) {
    if (x.st == 0.f) {
      x.mt = y.mt; x.st = y.st; x.a = y.a;
    } else if (y.mt > x.mt) {
      const float f = __expf(x.mt - y.mt);
      x.st = x.st * f + y.st; x.a = x.a * f + y.a; x.mt = y.mt;
    } else {
      const float f = __expf(y.mt - x.mt);
      x.st += y.st * f; x.a += y.a * f;
    }
  }
  if (y.sz > 0.f) {
    if (x.sz == 0.f) {
      x.mz = y.mz; x.sz = y.sz;
    } else if (y.mz > x.mz) {
      x.sz = x.sz * __expf(x.mz - y.mz) + y.sz; x.mz = y.mz;
    } else {
      x.sz += y.sz * __expf(y.mz - x.mz);
    }
  }
}

// Row pair i = s*P + (k-1): teacher row i of tl [n*P][V]; student row s*B + k of zl (ld).
__global__ void __launch_bounds__(kKlThreads)
kl_pass_kernel(const float* __restrict__ tl, const float* __restrict__ zl, int64_t ld, int B, int P,
               int V, int chunk, int n_parts, float inv_t, KlState* __restrict__ part) {
  __shared__ KlState sh[kKlThreads / 64];
  const int64_t i = blockIdx.x;
  const int j = blockIdx.y;
  const int64_t s = i / P, k = i - s * P + 1;
  const float* t = tl + i * int64_t(V);
  const float* z = zl + (s * B + k) * ld;
  const int c0 = j * chunk, c1 = min(V, c0 + chunk);
  KlState st{-INFINITY, 0.f, 0.f, -INFINITY, 0.f};
  for (int v = c0 + threadIdx.x; v < c1; v += kKlThreads) {
    const float tt = t[v] * inv_t, zz = z[v] * inv_t;
    KlState one{tt, 1.f, tt - zz, zz, 1.f};
    kl_merge(st, one);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    KlState y{__shfl_xor(st.mt, o, kWave), __shfl_xor(st.st, o, kWave), __shfl_xor(st.a, o, kWave),
              __shfl_xor(st.mz, o, kWave), __shfl_xor(st.sz, o, kWave)};
    kl_merge(st, y);
  }
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = st;
  __syncthreads();
  if (threadIdx.x == 0) {
    KlState x = sh[0];
    for (int w = 1; w < kKlThreads / 64; ++w) kl_merge(x, sh[w]);
    part[i * n_parts + j] = x;
  }
}

// kl[i] = a/st - (mt + log st) + (mz + log sz); ce from the student log-sum-exps; losses.
__global__ void __launch_bounds__(kKlThreads)
kl_finish_kernel(const KlState* __restrict__ part, int n_parts, int n_seq, int P, int B,
                 const float* __restrict__ zl, int64_t ld, const float* __restrict__ zlse,
                 const int32_t* __restrict__ labels, float T, float alpha,
                 float* __restrict__ kl, float* __restrict__ ce, float* __restrict__ loss) {
  __shared__ float sh[2][kKlThreads / 64];
  float skl = 0.f, sce = 0.f;
  for (int i = threadIdx.x; i < n_seq * P; i += kKlThreads) {
    KlState x = part[int64_t(i) * n_parts];
    for (int j = 1; j < n_parts; ++j) kl_merge(x, part[int64_t(i) * n_parts + j]);
    const float v = x.a / x.st - (x.mt + logf(x.st)) + (x.mz + logf(x.sz));
    kl[i] = v;
    skl += v;
  }
  const int K = B - 1;
  if (labels != nullptr) {
    for (int i = threadIdx.x; i < n_seq * K; i += kKlThreads) {
      const int64_t s = i / K, k = i - s * K + 1;
      const int64_t r = s * B + k;
      const float v = zlse[r] - zl[r * ld + labels[i]];
      if (ce != nullptr) ce[i] = v;
      sce += v;
    }
  }
  skl = wave_sum(skl);
  sce = wave_sum(sce);
  if ((threadIdx.x & 63) == 0) {
    sh[0][threadIdx.x >> 6] = skl;
    sh[1][threadIdx.x >> 6] = sce;
  }
  __syncthreads();
  if (threadIdx.x == 0 && loss != nullptr) {
    float a = 0.f, c = 0.f;
    for (int w = 0; w < kKlThreads / 64; ++w) {
      a += sh[0][w];
      c += sh[1][w];
    }
    const float l_kl = T * T / float(P) * a / float(n_seq);
    const float l_ce = labels != nullptr ? c / float(n_seq * K) : 0.f;
    loss[0] = l_kl;
    loss[1] = l_ce;
    loss[2] = l_ce + alpha * l_kl;
  }
}

__global__ void fill_u64_kernel(unsigned long long* p, int64_t n) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0ull;
}

static int kl_parts(int64_t rows, int V, int& chunk) {
  const int64_t want = (4 * int64_t(device_cu_count()) + rows - 1) / (rows > 0 ? rows : 1);
  const int max_parts = (V + 2047) / 2048;
  int np = int(want < 1 ? 1 : (want > max_parts ? max_parts : want));
  chunk = (V + np - 1) / np;
  return (V + chunk - 1) / chunk;
}

static size_t al256(size_t x) { return (x + 255) / 256 * 256; }

size_t kl_ws_bytes(int n_seq, int B, int P, int d, int V, bool bf16) {
  const size_t R = size_t(n_seq) * P, M = size_t(n_seq) * B;
  int ch;
  const int np = kl_parts(int64_t(R), V, ch);
  return al256(R * d * (bf16 ? 2 : 4)) + al256(R * 8) + al256(R * 4) + al256(R * size_t(V) * 4) +
         al256(R * np * sizeof(KlState)) + al256(M * 4) + al256(sample_parts_bytes(int64_t(M), V));
}

hipError_t launch_kl_forward(bool bf16, const void* H_pos, int m, const float* gamma, float eps,
                             const void* W_lm, int d, int V, const float* zl, int64_t ld, int B,
                             const int32_t* labels, int n_seq, int P, float T, float alpha,
                             float* kl, float* ce, float* loss, void* ws, hipStream_t s) {
  const int64_t R = int64_t(n_seq) * P, M = int64_t(n_seq) * B;
  char* p = static_cast<char*>(ws);
  void* th = p;                       p += al256(size_t(R) * d * (bf16 ? 2 : 4));
  auto* keys = reinterpret_cast<unsigned long long*>(p); p += al256(size_t(R) * 8);
  auto* am = reinterpret_cast<int32_t*>(p);             p += al256(size_t(R) * 4);
  auto* tl = reinterpret_cast<float*>(p);               p += al256(size_t(R) * V * 4);
  int ch;
  const int np = kl_parts(R, V, ch);
  auto* part = reinterpret_cast<KlState*>(p);           p += al256(size_t(R) * np * sizeof(KlState));
  auto* zlse = reinterpret_cast<float*>(p);             p += al256(size_t(M) * 4);
  void* rs_ws = p;
  if (bf16)
    hipLaunchKernelGGL(pool_norm_kernel<bf16_t>, dim3(unsigned(R)), dim3(kKlThreads), 0, s,
                       static_cast<const bf16_t*>(H_pos), m, d, gamma, eps, static_cast<bf16_t*>(th));
  else
    hipLaunchKernelGGL(pool_norm_kernel<float>, dim3(unsigned(R)), dim3(kKlThreads), 0, s,
                       static_cast<const float*>(H_pos), m, d, gamma, eps, static_cast<float*>(th));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(fill_u64_kernel, dim3(unsigned((R + 255) / 256)), dim3(256), 0, s, keys, R);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_lm_head(bf16, th, W_lm, R, d, V, keys, am, nullptr, tl, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kl_pass_kernel, dim3(unsigned(R), unsigned(np)), dim3(kKlThreads), 0, s, tl,
                     zl, ld, B, P, V, ch, np, 1.f / T, part);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (labels != nullptr) {
    e = launch_row_softmax(zl, M, V, ld, 1.f, false, 0, 0, nullptr, zlse, rs_ws, s);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kl_finish_kernel, dim3(1), dim3(kKlThreads), 0, s, part, np, n_seq, P, B, zl,
                     ld, zlse, labels, T, alpha, kl, ce, loss);
  return hipGetLastError();
}

}  // namespace hdf

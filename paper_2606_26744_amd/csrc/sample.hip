// Temperature sampling of draft tokens and speculative-sampling verification (the
// temperature-1 results of the paper's tables; the rule itself is the standard one of
// speculative decoding, which the paper does not restate: accept draft x_i with
// probability min(1, p_i(x_i) / q_i(x_i)), at the first rejection draw from
// max(0, p - q) renormalised, after K acceptances draw the bonus from p_K).
//
// Random numbers: Philox4x64-10 (Salmon et al., SC'11), key (seed, stream), counter
// (row, v/8, purpose, 0); word (v%8)/2 of the block gives two uniforms, from its high
// 32 bits for even v and its low 32 bits for odd v: u = (top 24 bits + 1/2) * 2^-24.  A draw from
// softmax(s) is argmax_v (s_v - log(-log u_v)) (Gumbel-max), so no probability vector
// is ever materialised: a pass over the logits keeps a running log-sum-exp and the
// best perturbed score.
#include "common.hpp"
#include "kernels.hpp"

namespace hdf {

constexpr int kSampleThreads = 256;
constexpr int kPurposeDraft = 0, kPurposeAccept = 1, kPurposeResample = 2;

__device__ __forceinline__ void philox4x64_10(uint64_t c[4], uint64_t k0, uint64_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B97F4A7C15ull;
      k1 += 0xBB67AE8584CAA73Bull;
    }
    const uint64_t hi0 = __umul64hi(0xD2E7470EE14C6C93ull, c[0]);
    const uint64_t lo0 = 0xD2E7470EE14C6C93ull * c[0];
    const uint64_t hi1 = __umul64hi(0xCA5A826395121157ull, c[2]);
    const uint64_t lo1 = 0xCA5A826395121157ull * c[2];
    const uint64_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
  }
}

// Uniforms of the eight entries 8*g .. 8*g+7 of one row.
__device__ __forceinline__ void uniforms8(uint64_t seed, uint64_t stream, uint64_t row, uint64_t g,
                                          int purpose, float u[8]) {
  uint64_t c[4] = {row, g, uint64_t(purpose), 0ull};
  philox4x64_10(c, seed, stream);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    u[2 * j] = (float(uint32_t(c[j] >> 40)) + 0.5f) * 5.9604644775390625e-8f;
    u[2 * j + 1] = (float(uint32_t(c[j] & 0xFFFFFFFFull) >> 8) + 0.5f) * 5.9604644775390625e-8f;
  }
}

constexpr int kGroupsPerPass = 4;   // 8-entry groups each thread loads before computing

__device__ __forceinline__ float gumbel(float u) { return -logf(-logf(u)); }

__device__ __forceinline__ unsigned long long sample_key(float score, int v) {
  return (static_cast<unsigned long long>(f32_order_key(score)) << 32) |
         static_cast<unsigned long long>(0xFFFFFFFFu - static_cast<uint32_t>(v));
}

// Running state of one thread over part of a row: log-sum-exp (m, s) of the scaled
// logits and the best perturbed score (ties to the lowest index).
struct RowState {
  float m, s, best;
  int idx;
};

__device__ __forceinline__ void lse_add(RowState& st, float x) {
  if (x > st.m) {
    st.s = st.s * __expf(st.m - x) + 1.f;
    st.m = x;
  } else {
    st.s += __expf(x - st.m);
  }
}

__device__ __forceinline__ void best_add(RowState& st, float score, int v) {
  if (score > st.best || (score == st.best && v < st.idx)) {
    st.best = score;
    st.idx = v;
  }
}

__device__ __forceinline__ void merge(RowState& a, const RowState& b) {
  if (b.s > 0.f) {
    if (a.s == 0.f) {
      a.m = b.m;
      a.s = b.s;
    } else if (b.m > a.m) {
      a.s = a.s * __expf(a.m - b.m) + b.s;
      a.m = b.m;
    } else {
      a.s += b.s * __expf(b.m - a.m);
    }
  }
  if (b.best > a.best || (b.best == a.best && b.idx < a.idx)) {
    a.best = b.best;
    a.idx = b.idx;
  }
}

// Workgroup reduction of RowState (all threads get the result).
__device__ RowState block_merge(RowState st, RowState* sh) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    RowState b;
    b.m = __shfl_xor(st.m, o, kWave);
    b.s = __shfl_xor(st.s, o, kWave);
    b.best = __shfl_xor(st.best, o, kWave);
    b.idx = __shfl_xor(st.idx, o, kWave);
    merge(st, b);
  }
  if (lane == 0) sh[wid] = st;
  __syncthreads();
  RowState t = sh[0];
  for (int w = 1; w < int(blockDim.x >> 6); ++w) merge(t, sh[w]);
  __syncthreads();
  return t;
}

// Pass over logits row `row`, columns [c0, c1) (c0 % 8 == 0): partial log-sum-exp of
// logits * inv_t and, with SAMPLE, the Gumbel-max draw.  Partial j of the row goes to
// part[row * n_parts + j].  Each thread loads kGroupsPerPass groups of eight logits
// (two 16-byte loads each when the row is 16-byte aligned) before it computes, so that
// the loads of a pass are in flight together.
template <bool SAMPLE>
__global__ void __launch_bounds__(kSampleThreads)
row_pass_kernel(const float* __restrict__ logits, int64_t ld, int V, int n_parts, int chunk,
                float inv_t, uint64_t seed, uint64_t stream, RowState* __restrict__ part) {
  __shared__ RowState sh[kSampleThreads / 64];
  const int64_t row = blockIdx.x;
  const int j = blockIdx.y;
  const int c0 = j * chunk, c1 = min(V, c0 + chunk);
  const float* z = logits + row * ld;
  const bool vec = (reinterpret_cast<uintptr_t>(z) & 15u) == 0;
  RowState st{-INFINITY, 0.f, -INFINITY, 0x7FFFFFFF};
  for (int g0 = c0 / 8 + threadIdx.x; 8 * g0 < c1; g0 += kSampleThreads * kGroupsPerPass) {
    float x[kGroupsPerPass][8];
#pragma unroll
    for (int q = 0; q < kGroupsPerPass; ++q) {
      const int v0 = 8 * (g0 + q * kSampleThreads);
      if (vec && v0 + 8 <= c1) {
        const float4 a = *reinterpret_cast<const float4*>(z + v0);
        const float4 b = *reinterpret_cast<const float4*>(z + v0 + 4);
        x[q][0] = a.x; x[q][1] = a.y; x[q][2] = a.z; x[q][3] = a.w;
        x[q][4] = b.x; x[q][5] = b.y; x[q][6] = b.z; x[q][7] = b.w;
      } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) x[q][k] = (v0 + k < c1) ? z[v0 + k] : 0.f;
      }
    }
#pragma unroll
    for (int q = 0; q < kGroupsPerPass; ++q) {
      const int g = g0 + q * kSampleThreads;
      if (8 * g >= c1) continue;
      const int nv = min(8, c1 - 8 * g);   // valid entries of the group (8 but at the end)
      float xs[8];
      float gm = -INFINITY;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        xs[k] = k < nv ? x[q][k] * inv_t : -INFINITY;
        gm = fmaxf(gm, xs[k]);
      }
      // One rescale per group: s <- s e^(m - m') + sum_k e^(x_k - m'), m' = max(m, max_k x_k).
      const float mn = fmaxf(st.m, gm);
      float add = 0.f;
#pragma unroll
      for (int k = 0; k < 8; ++k) add += __expf(xs[k] - mn);
      st.s = st.s * __expf(st.m - mn) + add;
      st.m = mn;
      if constexpr (SAMPLE) {
        float u[8];
        uniforms8(seed, stream, uint64_t(row), uint64_t(g), kPurposeDraft, u);
        // The group's best perturbed score, lowest index first; groups come in increasing
        // order, so a tie with the running best keeps the running (lower) index.
        float gb = -INFINITY;
        int gk = 0;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const float sc = k < nv ? xs[k] - __logf(-logf(u[k])) : -INFINITY;
          if (sc > gb) {
            gb = sc;
            gk = k;
          }
        }
        if (gb > st.best) {
          st.best = gb;
          st.idx = 8 * g + gk;
        }
      }
    }
  }
  st = block_merge(st, sh);
  if (threadIdx.x == 0) part[row * n_parts + j] = st;
}

// Combines the partials of every row: lse[row] = m + log(s); token[row] = best index.
__global__ void row_finish_kernel(const RowState* __restrict__ part, int64_t rows, int n_parts,
                                  float* __restrict__ lse, int32_t* __restrict__ tokens) {
  const int64_t row = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (row >= rows) return;
  RowState a = part[row * n_parts];
  for (int j = 1; j < n_parts; ++j) merge(a, part[row * n_parts + j]);
  if (lse != nullptr) lse[row] = a.m + logf(a.s);
  if (tokens != nullptr) tokens[row] = a.idx;
}

static void row_split(int64_t rows, int V, int& n_parts, int& chunk) {
  // Enough workgroups for four per CU, each at least 2048 columns wide; chunks are
  // whole 8-entry groups.
  const int64_t want = (4 * int64_t(device_cu_count()) + rows - 1) / (rows > 0 ? rows : 1);
  const int max_parts = (V + 2047) / 2048;
  n_parts = int(want < 1 ? 1 : (want > max_parts ? max_parts : want));
  chunk = ((V + n_parts - 1) / n_parts + 7) / 8 * 8;
  n_parts = (V + chunk - 1) / chunk;
}

size_t sample_parts_bytes(int64_t rows, int V) {
  int np, ch;
  row_split(rows, V, np, ch);
  return size_t(rows) * size_t(np) * sizeof(RowState);
}

hipError_t launch_row_softmax(const float* logits, int64_t rows, int V, int64_t ld, float inv_t,
                              bool sample, uint64_t seed, uint64_t stream, int32_t* tokens,
                              float* lse, void* part_ws, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  int np, ch;
  row_split(rows, V, np, ch);
  RowState* part = static_cast<RowState*>(part_ws);
  const dim3 grid(static_cast<unsigned>(rows), static_cast<unsigned>(np));
  if (sample)
    hipLaunchKernelGGL(row_pass_kernel<true>, grid, dim3(kSampleThreads), 0, s, logits, ld, V, np, ch,
                       inv_t, seed, stream, part);
  else
    hipLaunchKernelGGL(row_pass_kernel<false>, grid, dim3(kSampleThreads), 0, s, logits, ld, V, np,
                       ch, inv_t, seed, stream, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(row_finish_kernel, dim3(unsigned((rows + 255) / 256)), dim3(256), 0, s, part,
                     rows, np, lse, tokens);
  return hipGetLastError();
}

// Decisions of one sequence per wave: lane i tests slot i (u q < p); n = first
// rejection or K.  Writes n, the verified-token row prefix (drafts 0..n-1) and clears
// the sequence's two draw keys.
__global__ void __launch_bounds__(64)
accept_decide_kernel(const int32_t* __restrict__ draft, int draft_stride,
                     const float* __restrict__ draft_logits, const float* __restrict__ draft_lse,
                     int64_t ld, const float* __restrict__ target_logits,
                     const float* __restrict__ target_lse, int K, int V, float inv_t,
                     uint64_t seed, uint64_t stream, int32_t* __restrict__ n_out,
                     int32_t* __restrict__ tgt, unsigned long long* __restrict__ keys) {
  const int s = blockIdx.x;
  const int lane = threadIdx.x;
  int n = K;
  for (int c0 = 0; c0 < K; c0 += 64) {
    const int i = c0 + lane;
    bool reject = false;
    if (i < K) {
      const int64_t dr = int64_t(s) * draft_stride + i;
      const int x = draft[dr];
      const float q = __expf(draft_logits[dr * ld + x] * inv_t - draft_lse[dr]);
      const int64_t tr = int64_t(s) * (K + 1) + i;
      const float p = __expf(target_logits[tr * V + x] * inv_t - target_lse[tr]);
      float u[8];
      uniforms8(seed, stream, uint64_t(s), uint64_t(i >> 3), kPurposeAccept, u);
      reject = !(u[i & 7] * q < p);
    }
    const unsigned long long m = __ballot(reject);
    if (m != 0ull) {
      n = c0 + __ffsll(static_cast<long long>(m)) - 1;
      break;
    }
  }
  for (int i = lane; i <= K; i += 64) {
    tgt[int64_t(s) * (K + 1) + i] = i < n ? draft[int64_t(s) * draft_stride + i] : -1;
  }
  if (lane == 0) {
    n_out[s] = n;
    keys[2 * s] = 0ull;
    keys[2 * s + 1] = 0ull;
  }
}

// The draw after the decisions, split over the vocabulary: workgroup (s, j) scans
// columns [j*chunk, ...) of row n of sequence s.  Key 0: max(0, p_n - q_n) after a
// rejection, log p_K after K acceptances; key 1: log p_n (used only if the residual
// has no positive entry).
__global__ void __launch_bounds__(kSampleThreads)
accept_draw_kernel(const float* __restrict__ draft_logits, const float* __restrict__ draft_lse,
                   int64_t ld, int draft_stride, const float* __restrict__ target_logits,
                   const float* __restrict__ target_lse, int K, int V, int chunk, float inv_t,
                   uint64_t seed, uint64_t stream, const int32_t* __restrict__ n_in,
                   unsigned long long* __restrict__ keys) {
  __shared__ RowState sh[kSampleThreads / 64];
  const int s = blockIdx.x, j = blockIdx.y;
  const int n = n_in[s];
  const int64_t tr = int64_t(s) * (K + 1) + n;
  const float* zt = target_logits + tr * V;
  const float lt = target_lse[tr];
  const bool resid = n < K;
  const int64_t dr = int64_t(s) * draft_stride + (resid ? n : 0);
  const float* zd = draft_logits + dr * ld;
  const float ld_ = resid ? draft_lse[dr] : 0.f;
  const int c0 = j * chunk, c1 = min(V, c0 + chunk);
  RowState a{-INFINITY, 0.f, -INFINITY, 0x7FFFFFFF};   // residual / bonus
  RowState b{-INFINITY, 0.f, -INFINITY, 0x7FFFFFFF};   // log p_n fallback
  for (int g = c0 / 8 + threadIdx.x; 8 * g < c1; g += kSampleThreads) {
    float u[8];
    uniforms8(seed, stream, uint64_t(s), uint64_t(g), kPurposeResample, u);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int v = 8 * g + k;
      if (v < c1) {
        const float gm = gumbel(u[k]);
        const float lp = zt[v] * inv_t - lt;
        if (resid) {
          const float w = __expf(lp) - __expf(zd[v] * inv_t - ld_);
          if (w > 0.f) best_add(a, logf(w) + gm, v);
          best_add(b, lp + gm, v);
        } else {
          best_add(a, lp + gm, v);
        }
      }
    }
  }
  a = block_merge(a, sh);
  b = block_merge(b, sh);
  if (threadIdx.x == 0) {
    if (a.idx != 0x7FFFFFFF) atomicMax(keys + 2 * s, sample_key(a.best, a.idx));
    if (b.idx != 0x7FFFFFFF) atomicMax(keys + 2 * s + 1, sample_key(b.best, b.idx));
  }
}

__global__ void accept_finish_kernel(int n_seq, int K, const int32_t* __restrict__ n_in,
                                     const unsigned long long* __restrict__ keys,
                                     int32_t* __restrict__ tgt) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= n_seq) return;
  const unsigned long long k = keys[2 * s] != 0ull ? keys[2 * s] : keys[2 * s + 1];
  tgt[int64_t(s) * (K + 1) + n_in[s]] = int32_t(0xFFFFFFFFu - uint32_t(k & 0xFFFFFFFFull));
}

size_t accept_sample_ws_bytes(int n_seq, int K, int V) {
  const size_t rows = size_t(n_seq) * (K + 1);
  auto al = [](size_t x) { return (x + 255) / 256 * 256; };
  return al(rows * 4) + al(size_t(n_seq) * 4) + al(size_t(n_seq) * 16) + al(rows * 4) +
         al(sample_parts_bytes(int64_t(rows), V));
}

hipError_t launch_accept_sample(const int32_t* draft, int draft_stride, const float* draft_logits,
                                const float* draft_lse, int64_t ld, const float* target_logits,
                                int n_seq, int K, int V, float inv_t, uint64_t seed,
                                uint64_t stream, int32_t* acc, int32_t* anchor, int32_t* offs,
                                int32_t* toks, void* ws, hipStream_t s) {
  const int64_t rows = int64_t(n_seq) * (K + 1);
  auto al = [](size_t x) { return (x + 255) / 256 * 256; };
  char* p = static_cast<char*>(ws);
  float* tlse = reinterpret_cast<float*>(p);
  p += al(size_t(rows) * 4);
  int32_t* n_buf = reinterpret_cast<int32_t*>(p);
  p += al(size_t(n_seq) * 4);
  unsigned long long* keys = reinterpret_cast<unsigned long long*>(p);
  p += al(size_t(n_seq) * 16);
  int32_t* tgt = reinterpret_cast<int32_t*>(p);
  p += al(size_t(rows) * 4);
  hipError_t e = launch_row_softmax(target_logits, rows, V, V, inv_t, false, 0, 0, nullptr, tlse,
                                    p, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(accept_decide_kernel, dim3(n_seq), dim3(64), 0, s, draft, draft_stride,
                     draft_logits, draft_lse, ld, target_logits, tlse, K, V, inv_t, seed, stream,
                     n_buf, tgt, keys);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  int np, ch;
  row_split(n_seq, V, np, ch);
  hipLaunchKernelGGL(accept_draw_kernel, dim3(n_seq, np), dim3(kSampleThreads), 0, s, draft_logits,
                     draft_lse, ld, draft_stride, target_logits, tlse, K, V, ch, inv_t, seed, stream,
                     n_buf, keys);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(accept_finish_kernel, dim3((n_seq + 255) / 256), dim3(256), 0, s, n_seq, K,
                     n_buf, keys, tgt);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // The verified tokens of sequence s now read drafts 0..n-1 then the draw, which differs
  // from draft n (a rejected draft has p < q, so its residual weight is 0): greedy
  // acceptance against this row yields n, the draw as next anchor and the commits.
  return launch_accept(draft, draft_stride, tgt, n_seq, K, acc, anchor, offs, toks, s);
}

}  // namespace hdf

// Greedy acceptance (Sec. 1: the target keeps the longest agreeing draft prefix;
// Sec. 3.4: tau, the accepted length per round).
//
// One workgroup: each thread scans one sequence's drafts for the first mismatch,
// then a workgroup prefix sum over (n_s + 1) gives the packed commit offsets, and
// each thread copies its committed target tokens.  Sequences beyond the
// workgroup size are handled in successive passes with a running carry.
#include "common.hpp"
#include "kernels.hpp"

namespace hdf {

constexpr int kAcceptThreads = 1024;

__global__ void __launch_bounds__(kAcceptThreads)
accept_kernel(const int32_t* __restrict__ draft, int stride, const int32_t* __restrict__ target,
              int n_seq, int K, int32_t* __restrict__ acc, int32_t* __restrict__ anchor,
              int32_t* __restrict__ offs, int32_t* __restrict__ toks) {
  __shared__ int scan[kAcceptThreads];
  const int tid = threadIdx.x;
  int carry = 0;
  for (int base = 0; base < n_seq; base += kAcceptThreads) {
    const int s = base + tid;
    int n = 0;
    if (s < n_seq) {
      const int32_t* dr = draft + int64_t(s) * stride;
      const int32_t* tg = target + int64_t(s) * (K + 1);
      while (n < K && dr[n] == tg[n]) ++n;
      acc[s] = n;
      anchor[s] = tg[n];
    }
    const int v = (s < n_seq) ? n + 1 : 0;
    scan[tid] = v;
    __syncthreads();
    // Hillis-Steele inclusive scan.
    for (int o = 1; o < kAcceptThreads; o <<= 1) {
      const int add = (tid >= o) ? scan[tid - o] : 0;
      __syncthreads();
      scan[tid] += add;
      __syncthreads();
    }
    const int excl = carry + scan[tid] - v;
    if (s < n_seq) {
      if (offs != nullptr) offs[s] = excl;
      if (toks != nullptr) {
        const int32_t* tg = target + int64_t(s) * (K + 1);
        for (int i = 0; i <= n; ++i) toks[excl + i] = tg[i];
      }
    }
    carry += scan[kAcceptThreads - 1];
    __syncthreads();
  }
  if (offs != nullptr && tid == 0) offs[n_seq] = carry;
}

hipError_t launch_accept(const int32_t* draft, int stride, const int32_t* target, int n_seq,
                         int K, int32_t* acc, int32_t* anchor, int32_t* offs, int32_t* toks,
                         hipStream_t s) {
  hipLaunchKernelGGL(accept_kernel, dim3(1), dim3(kAcceptThreads), 0, s, draft, stride, target,
                     n_seq, K, acc, anchor, offs, toks);
  return hipGetLastError();
}

}  // namespace hdf

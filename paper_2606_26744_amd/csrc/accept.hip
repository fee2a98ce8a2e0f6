// Greedy acceptance (Sec. 1: the target keeps the longest agreeing draft prefix;
// Sec. 3.4: tau, the accepted length per round), optionally preceded by the LM head's
// argmax finalisation (hdf_accept_keys).
//
// One workgroup of 16 waves, sequences in chunks of 1024:
//   1. one wave per sequence: its lanes compare 64 draft positions at once (ballot of
//      the mismatches, with a sentinel at position K), so n_s costs one round of loads;
//   2. an exclusive prefix sum over the chunk's (n_s + 1) (wave scans, then the wave
//      totals) gives the packed commit offsets, continued across chunks by a carry;
//   3. one wave per sequence copies its n_s + 1 committed target tokens.
#include "common.hpp"
#include "kernels.hpp"

namespace hdf {

constexpr int kAcceptThreads = 1024;
constexpr int kAcceptWaves = kAcceptThreads / kWave;

// keys != NULL: the workgroup first turns the LM head's packed argmax keys of rows
// 0 .. M-1 into argmax (and max_logit) and clears them, then reads its drafts from the
// argmax it has just written (draft points into it); the workgroup barrier with the fence
// before it makes those stores visible to every wave.
__global__ void __launch_bounds__(kAcceptThreads)
accept_kernel(const int32_t* draft, int stride, const int32_t* __restrict__ target,
              int n_seq, int K, int32_t* __restrict__ acc, int32_t* __restrict__ anchor,
              int32_t* __restrict__ offs, int32_t* __restrict__ toks,
              unsigned long long* __restrict__ keys, int64_t M, int32_t* argmax,
              float* __restrict__ max_logit) {
  __shared__ int len[kAcceptThreads];     // n_s + 1, then the exclusive offsets
  __shared__ int nacc[kAcceptThreads];    // n_s
  __shared__ int wsum[kAcceptWaves];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wid = tid >> 6;
  if (keys != nullptr) {
    for (int64_t i = tid; i < M; i += kAcceptThreads) {
      decode_argmax_key(keys[i], argmax + i, max_logit != nullptr ? max_logit + i : nullptr);
      keys[i] = 0ull;   // the workspace is handed back zeroed
    }
    __threadfence_block();
    __syncthreads();
  }
  int carry = 0;
  for (int base = 0; base < n_seq; base += kAcceptThreads) {
    const int cnt = min(kAcceptThreads, n_seq - base);
    for (int j = wid; j < cnt; j += kAcceptWaves) {
      const int64_t s = base + j;
      const int32_t* dr = draft + s * stride;
      const int32_t* tg = target + s * (K + 1);
      int n = K, an = 0;
      for (int c0 = 0; c0 <= K; c0 += kWave) {
        const int i = c0 + lane;
        const int32_t dv = i < K ? dr[i] : 0;
        const int32_t tv = i <= K ? tg[i] : 0;
        unsigned long long miss = __ballot(i < K && dv != tv);
        if (K - c0 < kWave) miss |= 1ull << (K - c0);    // position K ends every scan
        if (miss != 0ull) {
          const int f = __ffsll(static_cast<long long>(miss)) - 1;
          n = c0 + f;
          an = __shfl(tv, f, kWave);
          break;
        }
      }
      if (lane == 0) {
        acc[s] = n;
        anchor[s] = an;
        len[j] = n + 1;
        nacc[j] = n;
      }
    }
    __syncthreads();
    // Exclusive scan of len[0 .. cnt): inclusive scan inside each wave, then the totals.
    int v = tid < cnt ? len[tid] : 0;
    int incl = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int t = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += t;
    }
    if (lane == kWave - 1) wsum[wid] = incl;
    __syncthreads();
    int before = 0, total = 0;
    for (int w = 0; w < kAcceptWaves; ++w) {
      const int ws = wsum[w];
      if (w < wid) before += ws;
      total += ws;
    }
    const int excl = carry + before + incl - v;
    if (tid < cnt) {
      len[tid] = excl;
      if (offs != nullptr) offs[base + tid] = excl;
    }
    __syncthreads();
    if (toks != nullptr) {
      for (int j = wid; j < cnt; j += kAcceptWaves) {
        const int64_t s = base + j;
        const int n = nacc[j];
        const int o = len[j];
        const int32_t* tg = target + s * (K + 1);
        for (int i = lane; i <= n; i += kWave) toks[o + i] = tg[i];
      }
    }
    carry += total;
    __syncthreads();
  }
  if (offs != nullptr && tid == 0) offs[n_seq] = carry;
}

hipError_t launch_accept(const int32_t* draft, int stride, const int32_t* target, int n_seq,
                         int K, int32_t* acc, int32_t* anchor, int32_t* offs, int32_t* toks,
                         hipStream_t s) {
  hipLaunchKernelGGL(accept_kernel, dim3(1), dim3(kAcceptThreads), 0, s, draft, stride, target,
                     n_seq, K, acc, anchor, offs, toks, nullptr, int64_t(0), nullptr, nullptr);
  return hipGetLastError();
}

hipError_t launch_accept_keys(unsigned long long* keys, int64_t M, int32_t* argmax,
                              float* max_logit, int draft_off, int stride,
                              const int32_t* target, int n_seq, int K, int32_t* acc,
                              int32_t* anchor, int32_t* offs, int32_t* toks, hipStream_t s) {
  hipLaunchKernelGGL(accept_kernel, dim3(1), dim3(kAcceptThreads), 0, s, argmax + draft_off,
                     stride, target, n_seq, K, acc, anchor, offs, toks, keys, M, argmax,
                     max_logit);
  return hipGetLastError();
}

}  // namespace hdf

// Dense contractions of the drafter step: C[M][N] = A[M][K] . B[N][K]^T with
// fp32 accumulation.  Both operands are K-contiguous (the [out][in] layout of
// every projection and of the LM head), which is the natural operand layout of
// the CDNA matrix cores.
//
// bf16: v_mfma_f32_32x32x16_bf16 on 128x128 (or 64x128) tiles, BK = 64, four
// waves of 64 lanes in a 2x2 grid.  Global->LDS staging goes through registers
// with STAGES K-tiles in flight per workgroup (the weight stream of the skinny
// GEMMs is HBM-bound, so bytes in flight per CU set the speed); the LDS tiles are
// double-buffered and padded by 16 bytes per row so the 16-byte operand reads of
// 32 consecutive rows hit distinct banks.  Split-K runs over gridDim.z.
// Tiles are handed out so that workgroups sharing a B tile (the weights) run on
// the same XCD back to back and meet in that XCD's L2.
//
// Epilogues:
//   PARTIAL  fp32 C (or split-K partial z at C + z*M*N) straight from registers
//   ARGMAX   LM head: the tile is staged in LDS, each row's (max, lowest index)
//            is folded into a packed 64-bit key with one atomicMax per row and
//            tile; the logits are stored only when asked for
//
// fp32 (small correctness-size workloads): a plain LDS-tiled VALU kernel with
// the same epilogues.
#include <atomic>

#include "common.hpp"
#include "kernels.hpp"

namespace hdf {

constexpr int kGemmThreads = 256;
constexpr int kBK = 64;        // K granularity of every GEMM (K % kBK == 0)

__device__ __forceinline__ int remap_tile(int bid, int total) {
  // XCD-aware order: dispatch sends consecutive workgroups round-robin over the 8
  // XCDs; give each XCD a contiguous run of tile ids (tiles of one B column block
  // are consecutive ids).
  const int per = total >> 3;
  if (bid < (per << 3)) return (bid & 7) * per + (bid >> 3);
  return bid;
}

// Row-wise (max, lowest index) of an fp32 tile staged in LDS, folded into keys[].
template <int BM, int BN, int LDC>
__device__ __forceinline__ void argmax_epilogue(const float* Cs, int m0, int n0, int M, int N,
                                                unsigned long long* keys, float* logits) {
  constexpr int TPR = kGemmThreads / BM;  // threads per row (2 or 4)
  constexpr int CPT = BN / TPR;           // columns per thread
  const int tid = threadIdx.x;
  const int r = tid / TPR;
  const int part = tid % TPR;
  const int row = m0 + r;
  float best = -INFINITY;
  int bcol = 0x7FFFFFFF;
  if (row < M) {
    const int c0 = part * CPT;
#pragma unroll 4
    for (int c = 0; c < CPT; ++c) {
      const int col = n0 + c0 + c;
      const float v = Cs[r * LDC + c0 + c];
      if (col < N && v > best) {
        best = v;
        bcol = col;
      }
    }
  }
#pragma unroll
  for (int o = 1; o < TPR; o <<= 1) {
    const float ov = __shfl_xor(best, o, kWave);
    const int oc = __shfl_xor(bcol, o, kWave);
    if (ov > best || (ov == best && oc < bcol)) {
      best = ov;
      bcol = oc;
    }
  }
  if (part == 0 && row < M && bcol != 0x7FFFFFFF) {
    const unsigned long long key =
        (static_cast<unsigned long long>(f32_order_key(best)) << 32) |
        static_cast<unsigned long long>(0xFFFFFFFFu - static_cast<uint32_t>(bcol));
    atomicMax(keys + row, key);
  }
  if (logits != nullptr) {
    // Coalesced copy of the tile: each thread moves 4 consecutive columns.
    for (int i = tid * 4; i < BM * BN; i += kGemmThreads * 4) {
      const int rr = i / BN, cc = i % BN;
      const int grow = m0 + rr, gcol = n0 + cc;
      if (grow >= M) continue;
      float* dst = logits + int64_t(grow) * N + gcol;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (gcol + j < N) dst[j] = Cs[rr * LDC + cc + j];
    }
  }
}

template <int BM, int BN, int BK, int STAGES, int EPI>
__global__ void __launch_bounds__(kGemmThreads)
gemm_bf16_kernel(GemmArgs p) {
  constexpr int WM = 2, WN = 2;
  constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
  constexpr int kLDK = BK + 8;                       // padded LDS row (bf16 elements)
  constexpr int CPR = BK / 8;                        // 16-byte chunks per row of a K-tile
  constexpr int A_CH = BM * BK / 8 / kGemmThreads;  // 16-byte chunks per thread per K-tile
  constexpr int B_CH = BN * BK / 8 / kGemmThreads;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  bf16_t* As = reinterpret_cast<bf16_t*>(smem);          // [2][BM][kLDK]
  bf16_t* Bs = As + 2 * BM * kLDK;                        // [2][BN][kLDK]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int wm = wid / WN, wn = wid % WN;

  const int mt = (p.M + BM - 1) / BM;
  const int nt = (p.N + BN - 1) / BN;
  const int tile = remap_tile(blockIdx.x, mt * nt);
  const int n_tile = tile / mt, m_tile = tile % mt;
  const int m0 = m_tile * BM, n0 = n_tile * BN;

  const int nk_all = p.K / BK;
  const int z = blockIdx.z;
  const int kt_begin = (nk_all * z) / gridDim.z;
  const int kt_end = (nk_all * (z + 1)) / gridDim.z;
  const int nk = kt_end - kt_begin;

  const bf16_t* A = static_cast<const bf16_t*>(p.A);
  const bf16_t* B = static_cast<const bf16_t*>(p.B);

  u32x4 ra[STAGES][A_CH], rb[STAGES][B_CH];

  // Rows past M (or N) are clamped to the last valid row rather than predicated: they
  // only feed accumulator rows/columns that are never stored, and unpredicated loads
  // keep the compiler's outstanding-load counting exact, so the prefetched stages stay
  // in flight across iterations.
  // A wave instruction covers 64 / CPR rows x CPR*16 contiguous bytes of each row.
  auto gload = [&](int kt, u32x4* da, u32x4* db) {
    const int64_t k = int64_t(kt_begin + kt) * BK;
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
      const int c = tid + i * kGemmThreads;
      const int row = min(m0 + c / CPR, p.M - 1), col = (c % CPR) * 8;
      da[i] = ld16(A + int64_t(row) * p.lda + k + col);
    }
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
      const int c = tid + i * kGemmThreads;
      const int row = min(n0 + c / CPR, p.N - 1), col = (c % CPR) * 8;
      db[i] = ld16(B + int64_t(row) * p.ldb + k + col);
    }
  };
  auto sstore = [&](const u32x4* da, const u32x4* db, int buf) {
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
      const int c = tid + i * kGemmThreads;
      const int row = c / CPR, col = (c % CPR) * 8;
      *reinterpret_cast<u32x4*>(As + (buf * BM + row) * kLDK + col) = da[i];
    }
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
      const int c = tid + i * kGemmThreads;
      const int row = c / CPR, col = (c % CPR) * 8;
      *reinterpret_cast<u32x4*>(Bs + (buf * BN + row) * kLDK + col) = db[i];
    }
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  if (nk > 0) {
    const int arow = wm * (BM / WM) + (lane & 31);
    const int brow = wn * (BN / WN) + (lane & 31);
    const int kof = 8 * (lane >> 5);
    auto compute = [&](int buf) {
      const bf16_t* as = As + buf * BM * kLDK;
      const bf16_t* bs = Bs + buf * BN * kLDK;
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        bf16x8_t af[TM], bfr[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          af[i] = *reinterpret_cast<const bf16x8_t*>(as + (arow + i * 32) * kLDK + ks * 16 + kof);
#pragma unroll
        for (int j = 0; j < TN; ++j)
          bfr[j] = *reinterpret_cast<const bf16x8_t*>(bs + (brow + j * 32) * kLDK + ks * 16 + kof);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
      }
    };
    // One K-tile step with ring slot u (a compile-time constant after unrolling):
    // refill slot u with tile t+STAGES (tile t is already in LDS), compute tile t,
    // move tile t+1 from its slot into the other LDS buffer, barrier.  Tile indices
    // past the end are clamped to the last tile (an L2 hit, never used), so every
    // load and store is unconditional.
    auto step = [&](int t, int u) {
      gload(min(t + STAGES, nk - 1), ra[u], rb[u]);
      compute(t & 1);
      sstore(ra[(u + 1) % STAGES], rb[(u + 1) % STAGES], (t + 1) & 1);
      __syncthreads();
    };
#pragma unroll
    for (int st = 0; st < STAGES; ++st) gload(min(st, nk - 1), ra[st], rb[st]);
    sstore(ra[0], rb[0], 0);
    __syncthreads();
    int kt = 0;
    for (; kt + STAGES <= nk; kt += STAGES) {
#pragma unroll
      for (int u = 0; u < STAGES; ++u) step(kt + u, u);
    }
#pragma unroll
    for (int u = 0; u < STAGES; ++u)
      if (kt + u < nk) step(kt + u, u);
  }

  if constexpr (EPI == kEpiPartial) {
    float* C = p.C + int64_t(z) * p.M * p.N;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = n0 + wn * (BN / WN) + j * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + wm * (BM / WM) + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (row < p.M && col < p.N) C[int64_t(row) * p.N + col] = acc[i][j][r];
        }
      }
  } else {
    constexpr int LDC = BN + 4;
    float* Cs = reinterpret_cast<float*>(smem);
    // The last loop iteration ended with a barrier, so LDS is free.
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = wn * (BN / WN) + j * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wm * (BM / WM) + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          Cs[row * LDC + col] = acc[i][j][r];
        }
      }
    __syncthreads();
    argmax_epilogue<BM, BN, LDC>(Cs, m0, n0, p.M, p.N, p.keys, p.C);
  }
}

// fp32 operands: 64x64 tiles, BK = 16, each thread owns a 4x4 block of C.
template <int EPI>
__global__ void __launch_bounds__(kGemmThreads)
gemm_f32_kernel(GemmArgs p) {
  constexpr int BM = 64, BN = 64, BKF = 16;
  __shared__ float As[BKF][BM + 4];
  __shared__ float Bs[BKF][BN + 4];
  __shared__ float Cs[BM * (BN + 4)];
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;
  const int mt = (p.M + BM - 1) / BM;
  const int nt = (p.N + BN - 1) / BN;
  const int tile = remap_tile(blockIdx.x, mt * nt);
  const int m0 = (tile % mt) * BM, n0 = (tile / mt) * BN;
  const int nk_all = p.K / BKF;
  const int z = blockIdx.z;
  const int kt_begin = (nk_all * z) / gridDim.z;
  const int kt_end = (nk_all * (z + 1)) / gridDim.z;
  const float* A = static_cast<const float*>(p.A);
  const float* B = static_cast<const float*>(p.B);
  float c[4][4] = {};
  for (int kt = kt_begin; kt < kt_end; ++kt) {
    const int64_t k0 = int64_t(kt) * BKF;
    for (int i = tid; i < BM * BKF; i += kGemmThreads) {
      const int r = i / BKF, kk = i % BKF;
      As[kk][r] = (m0 + r < p.M) ? A[int64_t(m0 + r) * p.lda + k0 + kk] : 0.f;
      Bs[kk][r] = (n0 + r < p.N) ? B[int64_t(n0 + r) * p.ldb + k0 + kk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BKF; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) c[i][j] = fmaf(a[i], b[j], c[i][j]);
    }
    __syncthreads();
  }
  if constexpr (EPI == kEpiPartial) {
    float* C = p.C + int64_t(z) * p.M * p.N;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = m0 + ty * 4 + i, col = n0 + tx * 4 + j;
        if (row < p.M && col < p.N) C[int64_t(row) * p.N + col] = c[i][j];
      }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) Cs[(ty * 4 + i) * (BN + 4) + tx * 4 + j] = c[i][j];
    __syncthreads();
    argmax_epilogue<BM, BN, BN + 4>(Cs, m0, n0, p.M, p.N, p.keys, p.C);
  }
}

__global__ void argmax_init_kernel(unsigned long long* keys, int64_t M) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < M) keys[i] = 0ull;
}

__global__ void argmax_finalize_kernel(const unsigned long long* keys, int64_t M, int32_t* argmax,
                                       float* max_logit) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= M) return;
  const unsigned long long k = keys[i];
  argmax[i] = int32_t(0xFFFFFFFFu - uint32_t(k & 0xFFFFFFFFull));
  if (max_logit != nullptr) max_logit[i] = f32_from_order_key(uint32_t(k >> 32));
}

// ---------------------------------------------------------------------------- host side

template <typename K>
static hipError_t set_lds(K kern, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  // Once per kernel instantiation (the attribute is per function, not per device).
  static std::atomic<bool> done{false};
  if (done.load(std::memory_order_acquire)) return hipSuccess;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(bytes));
  if (e == hipSuccess) done.store(true, std::memory_order_release);
  return e;
}

template <int BM, int EPI>
static hipError_t launch_bf16(const GemmArgs& a, int splits, hipStream_t s) {
  constexpr int BN = 128, BK = kBK, STAGES = 3;
  auto kern = gemm_bf16_kernel<BM, BN, BK, STAGES, EPI>;
  const size_t main_lds = size_t(2) * (BM + BN) * (BK + 8) * sizeof(bf16_t);
  const size_t epi_lds = (EPI == kEpiPartial) ? 0 : size_t(BM) * (BN + 4) * sizeof(float);
  const size_t lds = main_lds > epi_lds ? main_lds : epi_lds;
  hipError_t e = set_lds(kern, lds);
  if (e != hipSuccess) return e;
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  hipLaunchKernelGGL(kern, dim3(tiles, 1, splits), dim3(kGemmThreads), lds, s, a);
  return hipGetLastError();
}

static hipError_t launch_gemm_any(bool bf16, int epi, const GemmArgs& a, int splits,
                                  hipStream_t s) {
  if (bf16) {
    if (a.M <= 64)
      return epi == kEpiPartial ? launch_bf16<64, kEpiPartial>(a, splits, s)
                                : launch_bf16<64, kEpiArgmax>(a, splits, s);
    return epi == kEpiPartial ? launch_bf16<128, kEpiPartial>(a, splits, s)
                              : launch_bf16<128, kEpiArgmax>(a, splits, s);
  }
  const int tiles = ((a.M + 63) / 64) * ((a.N + 63) / 64);
  if (epi == kEpiPartial)
    hipLaunchKernelGGL(gemm_f32_kernel<kEpiPartial>, dim3(tiles, 1, splits), dim3(kGemmThreads), 0,
                       s, a);
  else
    hipLaunchKernelGGL(gemm_f32_kernel<kEpiArgmax>, dim3(tiles, 1, splits), dim3(kGemmThreads), 0,
                       s, a);
  return hipGetLastError();
}

int gemm_k_align(bool bf16) { return bf16 ? kBK : 16; }

int gemm_pick_splits(bool bf16, int M, int N, int K) {
  const int BM = bf16 ? (M <= 64 ? 64 : 128) : 64;
  const int BN = bf16 ? 128 : 64;
  const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  const int nk = K / gemm_k_align(bf16);
  // One wave of workgroups over the CUs; every split keeps at least 8 K-tiles and the
  // fp32 partials (S * M * N * 4 bytes, read back once) stay small next to the weights.
  const int target = device_cu_count();
  int s = (target + tiles - 1) / tiles;
  const int max_s = nk / 8 > 1 ? nk / 8 : 1;
  if (s > max_s) s = max_s;
  if (s > 8) s = 8;
  return s < 1 ? 1 : s;
}

hipError_t launch_gemm_partial(bool bf16, const void* A, int64_t lda, const void* B, int64_t ldb,
                               int M, int N, int K, int splits, float* C, hipStream_t s) {
  GemmArgs a{};
  a.A = A; a.lda = lda; a.B = B; a.ldb = ldb;
  a.M = M; a.N = N; a.K = K; a.C = C; a.keys = nullptr;
  return launch_gemm_any(bf16, kEpiPartial, a, splits, s);
}

hipError_t launch_lm_head(bool bf16, const void* hidden, const void* W, int64_t M, int d, int V,
                          unsigned long long* keys, int32_t* argmax, float* max_logit,
                          float* logits, hipStream_t s) {
  const int threads = 256;
  const unsigned blocks = unsigned((M + threads - 1) / threads);
  hipLaunchKernelGGL(argmax_init_kernel, dim3(blocks), dim3(threads), 0, s, keys, M);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // Rows are processed in chunks that keep the int32 tile arithmetic in range.
  const int64_t chunk = 1 << 20;
  for (int64_t r0 = 0; r0 < M; r0 += chunk) {
    const int rows = int(M - r0 < chunk ? M - r0 : chunk);
    GemmArgs a{};
    const size_t el = bf16 ? 2 : 4;
    a.A = static_cast<const char*>(hidden) + r0 * d * el;
    a.lda = d; a.B = W; a.ldb = d;
    a.M = rows; a.N = V; a.K = d;
    a.C = logits != nullptr ? logits + r0 * V : nullptr;
    a.keys = keys + r0;
    e = launch_gemm_any(bf16, kEpiArgmax, a, 1, s);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(argmax_finalize_kernel, dim3(blocks), dim3(threads), 0, s, keys, M, argmax,
                     max_logit);
  return hipGetLastError();
}

}  // namespace hdf

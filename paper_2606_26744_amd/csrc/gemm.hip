// Dense contractions of the drafter step: C[M][N] = A[M][K] . W[N][K]^T with fp32
// accumulation.  A (activations) is row-major; W (weights) is stored in the
// MFMA-packed layout of hdf_pack_weight:
//   element (n, k) at (((n/128)*(K/16) + k/16)*4 + (n%128)/32)*512
//                     + ((n%32) + 32*((k%16)/8))*8 + k%8
// i.e. every block of 32 rows x 16 k is 512 elements laid out in exactly the order
// the 64 lanes of a wave hold the B operand of v_mfma_f32_32x32x16_bf16 (lane l: row
// l%32, k 8*(l/32)..+7), and the four 32-row blocks of a 128-row group sit side by
// side for every 16 k.  A wave streams its weights straight from HBM into registers
// with one contiguous 1 KB load per instruction, the four waves of a workgroup read
// one contiguous 16 KB run per 64-k step, and no weight byte passes through LDS.
//
// bf16 kernel: NW waves (4, 6 or 8), each owning TN 32-column blocks (1; 2 for the LM
// head's 128-row weight stream; 4 for the matrix-core bound shapes) and all BM rows
// (BM = 128, or 64 when M <= 64) of a 32*NW*TN-column tile.  The activation slice
// (BM x 64) is shared through a double-buffered, padded LDS tile.  A ring of STAGES
// K-steps of weights is in flight per wave; activations are fetched one step further
// ahead than weights because memory counters complete in issue order.  The matrix-core
// bound tiles (128 x 512, 4 waves of 4 x 4 blocks, one wave per SIMD) run the deep K loop
// described at its code.
// Split-K runs over gridDim.z; tiles are ordered so that the M-tiles of one weight
// column block run on the same XCD back to back (its L2 serves the re-reads); in tall
// matrix-core bound problems an XCD's concurrent tiles form 8 x 4 blocks of row and column
// tiles instead.
//
// Epilogues:
//   PARTIAL  fp32 C (or split-K partial z at C + z*M*N) straight from registers
//   ARGMAX   LM head: the transposed product, so that per row (max, lowest index) is
//            taken over a lane's registers, then across the two lane halves and the
//            waves in LDS, and folded into a packed 64-bit key with one atomicMax per
//            row and tile; the logits are stored only when asked for
//
// fp32 (small correctness-size workloads): a plain LDS-tiled VALU kernel reading the
// same packed weight layout, with the same epilogues.
#include <initializer_list>

#include "common.hpp"
#include "kernels.hpp"

namespace hdf {

constexpr int kGemmThreads = 256;
constexpr int kBK = 64;        // K granularity of the bf16 kernel (K % kBK == 0)
constexpr int kGroupRows = 8;  // row tiles per group in the tile order of tall problems

__host__ __device__ __forceinline__ int64_t packed_index(int64_t n, int64_t k, int64_t K) {
  return (((n >> 7) * (K >> 4) + (k >> 4)) * 4 + ((n >> 5) & 3)) * 512 +
         ((n & 31) + 32 * ((k & 15) >> 3)) * 8 + (k & 7);
}

__device__ __forceinline__ int remap_tile(int bid, int total) {
  // XCD-aware order: dispatch sends consecutive workgroups round-robin over the 8
  // XCDs; give each XCD a contiguous run of tile ids (the M-tiles of one weight
  // column block are consecutive ids).
  const int per = total >> 3;
  if (bid < (per << 3)) return (bid & 7) * per + (bid >> 3);
  return bid;
}

__device__ __forceinline__ unsigned long long argmax_key(float v, int col) {
  return (static_cast<unsigned long long>(f32_order_key(v)) << 32) |
         static_cast<unsigned long long>(0xFFFFFFFFu - static_cast<uint32_t>(col));
}

// Activation unit of the deep K loop in LDS: row r's four 16-byte chunks (8 of K each)
// sit at chunk positions c ^ unit_swizzle(r), so that the row-wise stores (four threads
// a row) and the fragment reads (32 rows, one chunk each) meet distinct banks.
__device__ __forceinline__ int unit_swizzle(int r) { return ((r >> 1) ^ (r >> 2)) & 3; }

// TN: 32-column weight blocks per wave (1, 2 or 4).  Each activation fragment read from
// LDS feeds TN matrix-core operations, so wider waves cut the LDS traffic per MFMA; the
// compute-bound shapes (a few hundred rows and more) need it, the weight streams of
// 128 rows prefer more waves per CU instead.
// NT: fetch the weights with non-temporal loads (they stream past the caches).  Right
// when one row tile reads every weight byte once; with several row tiles the others
// re-read the weights from L2, so they are fetched through the caches.
// PP: the ping-pong K loop (128 x 512 tiles, 8 waves of two blocks): the two waves of a
// SIMD alternate between a memory phase and a compute phase.  The K/V and argmax
// epilogues of the matrix-core bound shapes run on it.
// DEEP: the K loop of the matrix-core bound partial-sum tiles (128 x 512, 4 waves of 4 x 4
// blocks, one wave per SIMD, a STAGES-unit weight ring in registers).
template <int BM, int NW, int STAGES, int EPI, int TN = 1, bool NT = (TN == 1), bool PP = false,
          bool DEEP = false>
__global__ void __launch_bounds__(NW * 64)
gemm_bf16_kernel(GemmArgs p) {
  constexpr int THREADS = NW * 64;
  constexpr int TM = BM / 32;
  constexpr int NB = NW * TN;                     // 32-column blocks of a tile
  constexpr int BN = 32 * NB;
  constexpr int LDA = kBK + 8;                    // padded LDS row (bf16 elements)
  constexpr int A_CHUNKS = BM * kBK / 8;           // 16-byte chunks of an activation step
  constexpr int A_CH = (A_CHUNKS + THREADS - 1) / THREADS;
  constexpr int LDC = 33;                         // padded row of a wave's 32 columns
  static_assert(EPI == kEpiPartial || NB % 4 == 0, "argmax and K/V tiles are whole 128-column slabs");
  // LDS: the activation buffers, reused after the K loop by the K/V epilogue and the
  // ARGMAX epilogue's logits to stage the fp32 tile 128 columns at a time ([block][row]
  // [32 columns]), and by the ARGMAX epilogue's per-wave row maxima.
  constexpr size_t kMainLds = PP     ? size_t(4) * BM * (32 + 8) * sizeof(bf16_t)   // NBUF units
                              : DEEP ? size_t(2) * BM * 32 * sizeof(bf16_t)          // two K units
                                     : size_t(2) * BM * LDA * sizeof(bf16_t);
  constexpr size_t kEpiLds = (EPI != kEpiPartial)
      ? size_t(4) * BM * LDC * sizeof(float) + (EPI == kEpiKV ? size_t(2) * BM * sizeof(int) : 0)
      : 0;
  __shared__ __attribute__((aligned(16))) unsigned char smem[kMainLds > kEpiLds ? kMainLds : kEpiLds];
  typedef bf16_t ATile[BM][LDA];
  ATile* As = reinterpret_cast<ATile*>(smem);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;

  // Tiles of the first problem, then those of the optional second one.
  const int tiles1 = ((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
  int tile = remap_tile(blockIdx.x, gridDim.x);
  const bool second = tile >= tiles1;
  if (second) {
    tile -= tiles1;
    p.A = p.A2;
    p.lda = p.lda2;
    p.B = p.B2;
    p.M = p.M2;
    p.N = p.N2;
    p.C = p.C2;
  }
  const int mt = (p.M + BM - 1) / BM;
  int n_tile = tile / mt, m_tile = tile % mt;
  if ((PP || DEEP) && mt > kGroupRows) {
    // Tall problems (the cold context projection): consecutive tile ids walk a group of
    // kGroupRows row tiles, then the next column block, so the 32 tiles an XCD runs at
    // once are 8 row tiles x 4 column blocks and share their activation and weight slices
    // in its L2 (with row tiles of one column block only, every activation slice missed):
    // 16384 x 4096 x 8192 with the K/V epilogue 1.58 -> 1.55 ms per cold step, the
    // 540K-row cold ragged step 46.5 -> 44.3 ms.
    const int nt = (p.N + BN - 1) / BN;
    const int in_group = kGroupRows * nt;
    const int g = tile / in_group, first = g * kGroupRows;
    const int gm = min(mt - first, kGroupRows);
    const int r = tile - g * in_group;
    m_tile = first + r % gm;
    n_tile = r / gm;
  }
  const int m0 = m_tile * BM, n0 = n_tile * BN;

  const int nk_all = p.K / kBK;
  const int z = blockIdx.z;
  const int kt_begin = (nk_all * z) / gridDim.z;
  const int kt_end = (nk_all * (z + 1)) / gridDim.z;
  const int nk = kt_end - kt_begin;

  const bf16_t* A = static_cast<const bf16_t*>(p.A);
  // This wave's 32-row weight blocks: block b = n_tile*NB + wid*TN + tn is sub-block
  // b%4 of 128-row group b/4 (rows past N are zero padding of the packed layout; a
  // group past the last one is clamped to it, and the columns it computes are never
  // stored).
  const int n_groups = (p.N + 127) >> 7;
  const bf16_t* Bw[TN];
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) {
    const int blk = n_tile * NB + wid * TN + tn;
    const int grp = min(blk >> 2, n_groups - 1);
    Bw[tn] = static_cast<const bf16_t*>(p.B) +
             (int64_t(grp) * (p.K >> 4) * 4 + (blk & 3)) * 512 + lane * 8;
  }

  // Argmax tiles compute the transposed product (the weights as the A operand): a lane
  // then holds 16 columns of one row per 32-column block, and the row maxima are taken
  // in registers.  Every other tile holds C = A.W^T (a lane: one column, 16 rows).
  auto mma = [](bf16x8_t act, bf16x8_t w, f32x16_t c) {
    if constexpr (EPI == kEpiArgmax)
      return __builtin_amdgcn_mfma_f32_32x32x16_bf16(w, act, c, 0, 0, 0);
    else
      return __builtin_amdgcn_mfma_f32_32x32x16_bf16(act, w, c, 0, 0, 0);
  };
  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][tn][r] = 0.f;

  if constexpr (PP) {
    // Waves 4-7 (group 1) run one phase behind waves 0-3 (group 0); the two waves of a
    // SIMD come one from each group.  In its memory phase a wave reads the activation
    // fragments of its next unit (32 of K) from LDS, stores its share of a later unit's
    // activations into LDS and issues the weight loads of the unit D ahead; in its
    // compute phase it runs the unit's 16 MFMAs from registers only.  A workgroup
    // barrier ends every phase, so while one wave of a SIMD computes, the other loads.
    static_assert(BM == 128 && NW == 8 && TN == 2, "ping-pong tiles are 128 x 512, 8 waves");
    constexpr int UK = 32;                   // K of one unit (two MFMA sub-steps)
    constexpr int LDU = UK + 8;              // padded LDS row of a unit (bf16 elements)
    constexpr int NBUF = 4;                  // LDS buffers of activation units
    constexpr int D = 2;                     // weight units in flight ahead of their use
    constexpr int NR = D + 1;
    static_assert(size_t(NBUF) * BM * LDU * sizeof(bf16_t) <= sizeof(smem), "LDS");
    typedef bf16_t UTile[BM][LDU];
    UTile* Au = reinterpret_cast<UTile*>(smem);
    const int nu = nk * (kBK / UK);
    const int64_t ku0 = int64_t(kt_begin) * (kBK / UK);
    const int grp = wid >> 2;
    // Activation staging: thread tid moves row tid/4, 16-byte chunk tid%4 of each unit
    // (512 threads x 16 B = one 128 x 32 unit).  Rows past M are clamped, units past the
    // end re-read the last one; neither is ever used.
    const bf16_t* a_src = A + int64_t(min(m0 + (tid >> 2), p.M - 1)) * p.lda + (tid & 3) * 8;
    auto a_load = [&](int u) { return ld16(a_src + (ku0 + min(u, nu - 1)) * UK); };
    auto a_store = [&](const u32x4& v, int u) {
      *reinterpret_cast<u32x4*>(&Au[u % NBUF][tid >> 2][(tid & 3) * 8]) = v;
    };
    // Units past the end are never used: their loads read the activations' first 16
    // bytes (in L2) instead of the weights again (see load_b below).
    auto b_load = [&](int u, u32x4* dst) {
      const bool live = u < nu;
      const int64_t kb = (ku0 + (live ? u : 0)) * (UK / 16);
#pragma unroll
      for (int ss = 0; ss < 2; ++ss)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
          dst[ss * TN + tn] = ld16(live ? Bw[tn] + (kb + ss) * 4 * 512 : A);
    };
    const int arow = lane & 31;
    const int kof = 8 * (lane >> 5);
    if (nu > 0) {
      u32x4 rb[NR][2 * TN];
      u32x4 areg = a_load(0);
      a_store(areg, 0);
      areg = a_load(1);
      a_store(areg, 1);
      areg = a_load(2);
#pragma unroll
      for (int j = 0; j < D; ++j) b_load(j, rb[j]);
      __syncthreads();
      if (grp == 1) __syncthreads();   // group 1 starts one phase behind
      // Unit u: buffer u % NBUF holds its activations (written during the memory phases
      // of unit u-2 by both groups); rb[slot] its weights (loaded D units earlier).
      auto unit = [&](int u, int slot) {
        bf16x8_t af[2][TM];
#pragma unroll
        for (int ss = 0; ss < 2; ++ss)
#pragma unroll
          for (int i = 0; i < TM; ++i)
            af[ss][i] = *reinterpret_cast<const bf16x8_t*>(
                &Au[u % NBUF][arow + 32 * i][ss * 16 + kof]);
        a_store(areg, u + 2);
        areg = a_load(u + 3);
        b_load(u + D, rb[(slot + D) % NR]);
        __syncthreads();
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ss = 0; ss < 2; ++ss)
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int tn = 0; tn < TN; ++tn)
              acc[i][tn] = mma(af[ss][i], __builtin_bit_cast(bf16x8_t, rb[slot][ss * TN + tn]),
                               acc[i][tn]);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
      };
      int u = 0;
      for (; u + NR <= nu; u += NR) {
#pragma unroll
        for (int j = 0; j < NR; ++j) unit(u + j, j);
      }
#pragma unroll
      for (int j = 0; j < NR; ++j)
        if (u + j < nu) unit(u + j, j);
      if (grp == 0) __syncthreads();   // group 0 ends one phase later
    }
  } else if constexpr (DEEP) {
    // One wave per SIMD.  Each wave owns all 128 rows and one 128-row weight group (4 x 4
    // blocks of 32 x 32), so every activation fragment read from LDS feeds four MFMAs and
    // the 512 accumulators fill the accumulation registers.  A unit is 32 of K (two MFMA
    // sub-steps).  The weights of a unit (8 KB a wave, 1 KB per load) go straight into a
    // ring of R register slots, issued D = R - 1 units before their MFMAs.  The
    // activations come through two swizzled LDS unit buffers: a thread stores its share
    // of unit u+1 in the first half of unit u, one workgroup barrier follows, and the
    // fragments of unit u+1's first sub-step are read during the second half, those of its
    // second sub-step during the first half of unit u+1.  Loads are issued in the order
    // they are waited for (the activations of unit u+D+1, then the weights of unit u+D),
    // so the in-order load counter never makes one wait for the other.
    static_assert(BM == 128 && NW == 4 && TN == 4, "deep tiles are 128 x 512, 4 waves of 4 x 4 blocks");
    constexpr int UK = 32;
    constexpr int R = STAGES;
    constexpr int D = R - 1;
    typedef bf16_t UTile[BM * UK];
    UTile* Au = reinterpret_cast<UTile*>(smem);
    const int nu = nk * (kBK / UK);
    const int64_t ku0 = int64_t(kt_begin) * (kBK / UK);
    // Activation staging: 512 chunks of 16 bytes per unit, thread tid moves chunks tid and
    // tid + 256 (row q/4, chunk q%4).  Rows past M are clamped, units past the end re-read
    // the last one; neither is ever used.
    const bf16_t* a_src[2];
    int a_lds[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int q = tid + 256 * j, row = q >> 2, c = q & 3;
      a_src[j] = A + int64_t(min(m0 + row, p.M - 1)) * p.lda + c * 8;
      a_lds[j] = row * UK + ((c ^ unit_swizzle(row)) * 8);
    }
    // Fragment of sub-step ss, row block i: lane l reads row 32i + l%32, chunk 2ss + l/32.
    const int fr = lane & 31;
    int f_off[2];
#pragma unroll
    for (int ss = 0; ss < 2; ++ss) f_off[ss] = fr * UK + (((2 * ss + (lane >> 5)) ^ unit_swizzle(fr)) * 8);
    auto a_load = [&](int u, u32x4* dst) {
      const int64_t k = (ku0 + min(u, nu - 1)) * UK;
      dst[0] = ld16(a_src[0] + k);
      dst[1] = ld16(a_src[1] + k);
    };
    auto a_store = [&](const u32x4* src, int buf) {
      *reinterpret_cast<u32x4*>(&Au[buf][a_lds[0]]) = src[0];
      *reinterpret_cast<u32x4*>(&Au[buf][a_lds[1]]) = src[1];
    };
    // Units past the end are never used: their loads read the activations' first 16
    // bytes (in L2) instead of the weights.
    auto b_load = [&](int u, u32x4 (*dst)[TN]) {
      const bool live = u < nu;
      const int64_t kb = (ku0 + (live ? u : 0)) * (UK / 16);
#pragma unroll
      for (int ss = 0; ss < 2; ++ss)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
          dst[ss][tn] = ld16(live ? Bw[tn] + (kb + ss) * 4 * 512 : A);
    };
    auto frag = [&](int buf, int ss, int i) {
      return *reinterpret_cast<const bf16x8_t*>(&Au[buf][f_off[ss] + 32 * i * UK]);
    };
    if (nu > 0) {
      u32x4 rb[R][2][TN];
      u32x4 ra[R][2];
      a_load(0, ra[0]);
#pragma unroll
      for (int x = 0; x < D; ++x) {
        a_load(x + 1, ra[(x + 1) % R]);
        b_load(x, rb[x]);
      }
      a_store(ra[0], 0);
      lds_barrier();
      bf16x8_t f0[TM], f1[TM];
#pragma unroll
      for (int i = 0; i < TM; ++i) f0[i] = frag(0, 0, i);
      // Unit u in ring slot s = u % R.
      auto unit = [&](int u, int s) {
#pragma unroll
        for (int i = 0; i < TM; ++i) f1[i] = frag(u & 1, 1, i);
        a_store(ra[(u + 1) % R], (u + 1) & 1);
        a_load(u + D + 1, ra[(u + D + 1) % R]);
        b_load(u + D, rb[(s + D) % R]);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int tn = 0; tn < TN; ++tn)
            acc[i][tn] = mma(f0[i], __builtin_bit_cast(bf16x8_t, rb[s][0][tn]), acc[i][tn]);
        lds_barrier();
#pragma unroll
        for (int i = 0; i < TM; ++i) f0[i] = frag((u + 1) & 1, 0, i);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int tn = 0; tn < TN; ++tn)
            acc[i][tn] = mma(f1[i], __builtin_bit_cast(bf16x8_t, rb[s][1][tn]), acc[i][tn]);
      };
      int u = 0;
      for (; u + R <= nu; u += R) {
#pragma unroll
        for (int j = 0; j < R; ++j) unit(u + j, j);
      }
#pragma unroll
      for (int j = 0; j < R; ++j)
        if (u + j < nu) unit(u + j, j);
    }
    lds_barrier();   // the epilogues reuse LDS
  } else if (nk > 0) {
    u32x4 ra[STAGES][A_CH];
    u32x4 rb[STAGES][TN * 4];
    // Activation chunk c of a K-step: row c/8, 16-byte column c%8.  Rows past M are
    // clamped (their products are never stored); loads stay unpredicated so the
    // compiler's outstanding-load counting is exact.
    auto load_a = [&](int kt, u32x4* dst) {
      const int64_t k = int64_t(kt_begin + min(kt, nk - 1)) * kBK;
#pragma unroll
      for (int i = 0; i < A_CH; ++i) {
        const int c = min(tid + i * THREADS, A_CHUNKS - 1);   // spare threads repeat the last
        const int row = min(m0 + (c >> 3), p.M - 1);
        dst[i] = ld16(A + int64_t(row) * p.lda + k + (c & 7) * 8);
      }
    };
    // The ring issues STAGES steps past the last one; those are never used.  Their loads
    // read the activations' first 16 bytes (one line, in L2) rather than the last weight
    // step again: a re-read of the weights would come from HBM (the non-temporal streams
    // do not keep them in L2), STAGES of the nk steps extra (O/down: 2 of 8).  The loads
    // are still issued, so the compiler's outstanding-load counting stays exact.
    auto load_b = [&](int kt, u32x4* dst) {
      const bool live = kt < nk;
      const int64_t kb = int64_t(kt_begin + (live ? kt : 0)) * (kBK / 16);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          const bf16_t* src = live ? Bw[tn] + (kb + q) * 4 * 512 : A;
          dst[q * TN + tn] = NT ? ld_nt16(src) : ld16(src);
        }
    };
    auto store_a = [&](const u32x4* src, int buf) {
#pragma unroll
      for (int i = 0; i < A_CH; ++i) {
        const int c = min(tid + i * THREADS, A_CHUNKS - 1);
        *reinterpret_cast<u32x4*>(&As[buf][c >> 3][(c & 7) * 8]) = src[i];
      }
    };
    const int arow = lane & 31;
    const int kof = 8 * (lane >> 5);
    auto compute = [&](int buf, const u32x4* bq) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const bf16x8_t af =
              *reinterpret_cast<const bf16x8_t*>(&As[buf][arow + 32 * i][q * 16 + kof]);
#pragma unroll
          for (int tn = 0; tn < TN; ++tn)
            acc[i][tn] = mma(af, __builtin_bit_cast(bf16x8_t, bq[q * TN + tn]), acc[i][tn]);
        }
      }
    };
    // Prologue.  The weights do not depend on the previous kernel, so B(0) is issued first
    // and its HBM latency overlaps the activations' L2 latency (issued after A(0) it came
    // one L2 round trip later).  Then A(1..STAGES-1) and B(1..STAGES-1) in the order they
    // are consumed, A(0) into LDS (loads complete in issue order: this waits for B(0) and
    // A(0) only), and A(STAGES) into the register slot A(0) leaves.
    load_b(0, rb[0]);
    load_a(0, ra[0]);
#pragma unroll
    for (int st = 1; st < STAGES; ++st) {
      load_a(st, ra[st]);
      load_b(st, rb[st]);
    }
    store_a(ra[0], 0);
    load_a(STAGES, ra[0]);
    __syncthreads();
    // Step t (ring slot u = t % STAGES): compute with A(t) in LDS and B(t) in rb[u];
    // move A(t+1) into the other LDS buffer; refill the freed slots with A(t+1+STAGES)
    // and B(t+STAGES); barrier.
    auto step = [&](int t, int u) {
      compute(t & 1, rb[u]);
      store_a(ra[(u + 1) % STAGES], (t + 1) & 1);
      load_a(t + 1 + STAGES, ra[(u + 1) % STAGES]);
      load_b(t + STAGES, rb[u]);
      __syncthreads();
    };
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
    for (int tn = 0; tn < TN; ++tn) {
      const int col = n0 + 32 * (wid * TN + tn) + (lane & 31);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (row < p.M && col < p.N) C[int64_t(row) * p.N + col] = acc[i][tn][r];
        }
    }
  } else if constexpr (EPI == kEpiKV) {
    // Context K/V rows straight into the cache, one 128-column slab (whole heads) of the
    // tile at a time through LDS ([block][row][column of the block]): K columns get RoPE
    // at the row's position (pairs i, i + hd/2 of a head) and go to the key tile layout,
    // four consecutive dims per store; V columns go to the transposed value layout with
    // consecutive threads on consecutive rows of one dim.  The same fp32 values and the
    // same rounding as the partial-sum path and its epilogue kernel.
    float* Cs = reinterpret_cast<float*>(smem);
    // The tile's row table: cache row (-1: not stored) and position of every row, read
    // once here so that no store below waits on a dependent global load.
    int* rtab = reinterpret_cast<int*>(Cs + 4 * BM * LDC);
    int* ptab = rtab + BM;
    const bool is_v = n0 >= p.kv_d;
    const int HD = p.hd, HALF = HD >> 1;
    if (tid < BM) {
      const int row = m0 + tid;
      const int dr = row < p.M ? p.plan_row[row] : -1;
      rtab[tid] = dr;
      ptab[tid] = dr >= 0 ? p.plan_pos[row] : 0;
    }
    auto at = [&](int rr, int cc) { return Cs[((cc >> 5) * BM + rr) * LDC + (cc & 31)]; };
    // K items (row, octet of eight rotated pairs): 8 octets per row of a slab, each stored
    // as two 16-byte runs (dims i0..i0+7 and i0+hd/2..i0+hd/2+7 are contiguous in the key
    // tile layout).  A thread's items are rows rr, rr + THREADS/8, ... of one octet, the
    // same rows and dims in every slab, so their rotation-table entries are fetched once
    // per tile, before the first slab (rows without a cache row fetch entry 0 and are
    // skipped).  The barriers below order LDS traffic only, so the stores of one slab
    // stay in flight while the next one is staged.
    constexpr int KI = BM * 8 / THREADS;
    static_assert(KI * THREADS == BM * 8, "whole items per thread");
    const int oc = tid & 7;
    const int kj = (8 * oc) / HALF;           // head inside the slab
    const int i0 = 8 * oc - kj * HALF;
    float4 cs[KI][4];
    lds_barrier();                             // the row table
    if (!is_v && p.rope_cs != nullptr) {
#pragma unroll
      for (int it = 0; it < KI; ++it) {
        const float* c = p.rope_cs + (int64_t(ptab[(tid >> 3) + it * (THREADS / 8)]) * HALF + i0) * 2;
#pragma unroll
        for (int q = 0; q < 4; ++q) cs[it][q] = *reinterpret_cast<const float4*>(c + 4 * q);
      }
    }
#pragma unroll 1
    for (int slab = 0; slab < NB / 4; ++slab) {
      if (slab > 0) lds_barrier();
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int b = wid * TN + tn;
        if ((b >> 2) == slab) {
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int rr = 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
              Cs[((b & 3) * BM + rr) * LDC + (lane & 31)] = acc[i][tn][r];
            }
        }
      }
      lds_barrier();
      const int c0 = n0 + 128 * slab - (is_v ? p.kv_d : 0);   // slab start inside K or V
      if (c0 >= p.kv_d) continue;                             // columns past N
      if (!is_v) {
        const int j = kj;
#pragma unroll
        for (int it = 0; it < KI; ++it) {
          const int rr = (tid >> 3) + it * (THREADS / 8);
          const int drow = rtab[rr];
          if (drow < 0) continue;
          float y1[8], y2[8];
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            y1[k] = at(rr, j * HD + i0 + k);
            y2[k] = at(rr, j * HD + HALF + i0 + k);
          }
          if (p.rope_cs != nullptr) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              rope_rotate(y1[2 * q], y2[2 * q], cs[it][q].x, cs[it][q].y);
              rope_rotate(y1[2 * q + 1], y2[2 * q + 1], cs[it][q].z, cs[it][q].w);
            }
          }
          bf16_t* kh = static_cast<bf16_t*>(p.kc) + int64_t(c0 / HD + j) * p.cap * HD;
          *reinterpret_cast<uint4*>(kh + kc_index(drow, i0, HD)) =
              make_uint4(pack_bf2(y1[0], y1[1]), pack_bf2(y1[2], y1[3]), pack_bf2(y1[4], y1[5]),
                         pack_bf2(y1[6], y1[7]));
          *reinterpret_cast<uint4*>(kh + kc_index(drow, i0 + HALF, HD)) =
              make_uint4(pack_bf2(y2[0], y2[1]), pack_bf2(y2[2], y2[3]), pack_bf2(y2[4], y2[5]),
                         pack_bf2(y2[6], y2[7]));
        }
      } else {
        // Items (group of 8 rows, dim): consecutive threads on consecutive dims; a group
        // whose 8 rows are 8 consecutive cache rows starting at a multiple of 8 is one
        // 16-byte run of the value tile layout, any other group is stored element-wise.
        for (int e = tid; e < (BM / 8) * 128; e += THREADS) {
          const int cc = e & 127, rg = e >> 7;
          const int row0 = m0 + 8 * rg;
          if (row0 >= p.M) continue;
          const int col = c0 + cc;
          bf16_t* vh = static_cast<bf16_t*>(p.vtc) + int64_t(col / HD) * p.cap * HD;
          const int i = col % HD;
          const int d0 = rtab[8 * rg];
          bool run = row0 + 8 <= p.M && d0 >= 0 && (d0 & 7) == 0;
#pragma unroll
          for (int k = 1; k < 8; ++k) run = run && rtab[8 * rg + k] == d0 + k;
          if (run) {
            float v[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) v[k] = at(8 * rg + k, cc);
            *reinterpret_cast<uint4*>(vh + vc_index(d0, i, HD)) =
                make_uint4(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]),
                           pack_bf2(v[6], v[7]));
          } else {
            for (int k = 0; k < 8 && row0 + k < p.M; ++k) {
              const int dr = rtab[8 * rg + k];
              if (dr >= 0) vh[vc_index(dr, i, HD)] = f2bf(at(8 * rg + k, cc));
            }
          }
        }
      }
    }
  } else {
    // Transposed tile: lane l holds row 32i + l%32 and, of 32-column block b, columns
    // 32b + 8(r/4) + 4(l/32) + r%4 (r = 0..15).  Each lane scans its columns in increasing
    // order (lowest column on ties), the two lane halves of a row meet by a shuffle, the
    // waves' (max, column) pairs meet in LDS, and one atomic per row folds the tile's pair
    // into the row's packed key.  The K loop ended with a barrier, so LDS is free.
    float* Cs = reinterpret_cast<float*>(smem);
    const int tok = lane & 31;
    float best[TM];
    int bcol[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      best[i] = -INFINITY;
      bcol[i] = 0x7FFFFFFF;
    }
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int cb = n0 + 32 * (wid * TN + tn) + 4 * (lane >> 5);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int col = cb + 8 * (r >> 2) + (r & 3);
        const bool in = col < p.N;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          // selects, not branches: one compare and two conditional moves per value
          const float v = acc[i][tn][r];
          const bool take = in & (v > best[i]);
          best[i] = take ? v : best[i];
          bcol[i] = take ? col : bcol[i];
        }
      }
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const float ov = __shfl_xor(best[i], 32, kWave);
      const int oc = __shfl_xor(bcol[i], 32, kWave);
      if (ov > best[i] || (ov == best[i] && oc < bcol[i])) {
        best[i] = ov;
        bcol[i] = oc;
      }
    }
    if (p.C != nullptr) {
      // Logits (tests, sampling): the tile goes through LDS four waves (128 columns) at a
      // time ([block][row][column of the block]) and leaves as coalesced rows.
#pragma unroll
      for (int slab = 0; slab < NB / 4; ++slab) {
        if (slab > 0) __syncthreads();
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          const int b = wid * TN + tn;
          if ((b >> 2) == slab) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
              for (int r = 0; r < 16; ++r)
                Cs[((b & 3) * BM + 32 * i + tok) * LDC + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)] =
                    acc[i][tn][r];
          }
        }
        __syncthreads();
        const int cs0 = n0 + 128 * slab;
        for (int e = tid; e < BM * 128; e += THREADS) {
          const int rr = e >> 7, cc = e & 127;
          if (m0 + rr < p.M && cs0 + cc < p.N)
            p.C[int64_t(m0 + rr) * p.N + cs0 + cc] = Cs[((cc >> 5) * BM + rr) * LDC + (cc & 31)];
        }
      }
      __syncthreads();
    }
    float* rv = Cs;                                          // [wave][row] maxima
    int* rc = reinterpret_cast<int*>(Cs + NW * BM);          // [wave][row] columns
    if (lane < 32) {
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        rv[wid * BM + 32 * i + tok] = best[i];
        rc[wid * BM + 32 * i + tok] = bcol[i];
      }
    }
    __syncthreads();
    if (tid < BM && m0 + tid < p.M) {
      float bv = rv[tid];
      int bc = rc[tid];
#pragma unroll
      for (int w = 1; w < NW; ++w) {
        const float ov = rv[w * BM + tid];
        const int oc = rc[w * BM + tid];
        if (ov > bv || (ov == bv && oc < bc)) {
          bv = ov;
          bc = oc;
        }
      }
      if (bc != 0x7FFFFFFF) atomicMax(p.keys + m0 + tid, argmax_key(bv, bc));
    }
  }
}

// fp32 operands: 64x64 tiles, BK = 16, each thread owns a 4x4 block of C; the
// weights are read through the packed index.
template <int EPI>
__global__ void __launch_bounds__(kGemmThreads)
gemm_f32_kernel(GemmArgs p) {
  constexpr int BM = 64, BN = 64, BKF = 16;
  __shared__ float As[BKF][BM + 4];
  __shared__ float Bs[BKF][BN + 4];
  __shared__ float Cs[BM][BN + 4];
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
      Bs[kk][r] = (n0 + r < p.N) ? B[packed_index(n0 + r, k0 + kk, p.K)] : 0.f;
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
      for (int j = 0; j < 4; ++j) Cs[ty * 4 + i][tx * 4 + j] = c[i][j];
    __syncthreads();
    // Four threads per row, 16 columns each, lowest column on ties.
    const int r = tid >> 2, part = tid & 3;
    float best = -INFINITY;
    int bcol = 0x7FFFFFFF;
    if (m0 + r < p.M) {
      for (int cc = part * 16; cc < part * 16 + 16; ++cc) {
        const int gcol = n0 + cc;
        if (gcol < p.N) {
          const float v = Cs[r][cc];
          if (p.C != nullptr) p.C[int64_t(m0 + r) * p.N + gcol] = v;
          if (v > best) {
            best = v;
            bcol = gcol;
          }
        }
      }
    }
#pragma unroll
    for (int o = 1; o < 4; o <<= 1) {
      const float ov = __shfl_xor(best, o, kWave);
      const int oc = __shfl_xor(bcol, o, kWave);
      if (ov > best || (ov == best && oc < bcol)) {
        best = ov;
        bcol = oc;
      }
    }
    if (part == 0 && m0 + r < p.M && bcol != 0x7FFFFFFF)
      atomicMax(p.keys + m0 + r, argmax_key(best, bcol));
  }
}

__global__ void argmax_finalize_kernel(unsigned long long* keys, int64_t M, int32_t* argmax,
                                       float* max_logit) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= M) return;
  decode_argmax_key(keys[i], argmax + i, max_logit != nullptr ? max_logit + i : nullptr);
  keys[i] = 0ull;   // the workspace is handed back zeroed
}

// Row-major [N][K] -> packed layout, one 16-byte (bf16) or 32-byte (fp32) lane chunk
// of 8 elements per thread; rows N..ceil(N/128)*128-1 are written as zeros.
template <typename T>
__global__ void pack_weight_kernel(const T* __restrict__ src, T* __restrict__ dst, int N, int K) {
  const int64_t chunks = int64_t((N + 127) / 128) * (K / 16) * 4 * 64;
  for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < chunks;
       e += int64_t(gridDim.x) * blockDim.x) {
    const int lane = int(e & 63);
    const int64_t blk = e >> 6;                 // ((group * (K/16)) + kb) * 4 + sub
    const int sub = int(blk & 3);
    const int64_t kb = (blk >> 2) % (K / 16), grp = (blk >> 2) / (K / 16);
    const int64_t n = grp * 128 + sub * 32 + (lane & 31);
    const int64_t k = kb * 16 + 8 * (lane >> 5);
    T* d = dst + e * 8;
#pragma unroll
    for (int j = 0; j < 8; ++j) d[j] = (n < N) ? src[n * K + k + j] : T(0);
  }
}

// ---------------------------------------------------------------------------- host side

// Matrix-core bound tiles: 128 x 512 in the deep K loop, 4 waves of 4 x 4 blocks with a
// 4-unit weight ring (3 or 4 units measured the same; the register file holds no more).
constexpr int kDeepWaves = 4, kDeepBlocks = 4, kDeepRing = 4;

template <int EPI>
static void launch_bf16_deep(const GemmArgs& a, int splits, hipStream_t s) {
  constexpr int BN = 32 * kDeepWaves * kDeepBlocks;
  const int tiles = ((a.M + 127) / 128) * ((a.N + BN - 1) / BN) +
                    ((a.M2 + 127) / 128) * ((a.N2 + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_bf16_kernel<128, kDeepWaves, kDeepRing, EPI, kDeepBlocks, false, false, true>),
                     dim3(tiles, 1, splits), dim3(kDeepWaves * 64), 0, s, a);
}

template <int NW, int TN, int STAGES = 4, bool NT = (TN == 1)>
static void launch_bf16_partial(const GemmArgs& a, int splits, hipStream_t s) {
  const int BM = (a.M <= 64 && a.M2 <= 64) ? 64 : 128;
  constexpr int BN = 32 * NW * TN;
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN) +
                    ((a.M2 + BM - 1) / BM) * ((a.N2 + BN - 1) / BN);
  const dim3 grid(tiles, 1, splits), block(NW * 64);
  if (BM == 64)
    hipLaunchKernelGGL((gemm_bf16_kernel<64, NW, STAGES, kEpiPartial, TN, NT>), grid, block, 0, s,
                       a);
  else
    hipLaunchKernelGGL((gemm_bf16_kernel<128, NW, STAGES, kEpiPartial, TN, NT>), grid, block, 0, s,
                       a);
}

// One pass for 128 < M <= 256 rows: every row in one tile (192 or 256 rows), 8 waves of
// one 32-column block, the weights streamed once (non-temporal).  Two 128-row tiles
// re-streamed the weights through L2 instead (M = 192: 277 -> 211 us, M = 256: 289 -> 262
// us).  One column block per wave reads a 1 KB activation fragment per MFMA, which at 256
// rows is the LDS bandwidth of the CU.
template <int BM>
static void launch_bf16_argmax_tall(const GemmArgs& a, hipStream_t s) {
  constexpr int BN = 32 * 8;
  const dim3 grid((a.N + BN - 1) / BN, 1, 1), block(8 * 64);
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, 8, 2, kEpiArgmax, 1, true>), grid, block, 0, s, a);
}

template <int NW, int TN, int STAGES>
static void launch_bf16_argmax(const GemmArgs& a, hipStream_t s) {
  if (a.M > 128 && a.M <= 192) return launch_bf16_argmax_tall<192>(a, s);
  if (a.M > 192 && a.M <= 256) return launch_bf16_argmax_tall<256>(a, s);
  const int BM = a.M <= 64 ? 64 : 128;
  constexpr int BN = 32 * NW * TN;
  const int mt = (a.M + BM - 1) / BM;
  const int tiles = mt * ((a.N + BN - 1) / BN);
  const dim3 grid(tiles, 1, 1), block(NW * 64);
  // One row tile: every weight byte is read once, so the weights stream past the caches.
  if (BM == 64)
    hipLaunchKernelGGL((gemm_bf16_kernel<64, NW, STAGES, kEpiArgmax, TN, true>), grid, block, 0,
                       s, a);
  else if (mt == 1)
    hipLaunchKernelGGL((gemm_bf16_kernel<128, NW, STAGES, kEpiArgmax, TN, true>), grid, block, 0,
                       s, a);
  else
    hipLaunchKernelGGL((gemm_bf16_kernel<128, NW, STAGES, kEpiArgmax, TN, (TN == 1), (TN == 2)>),
                       grid, block, 0, s, a);
}

static hipError_t launch_gemm_any(bool bf16, int epi, const GemmArgs& a, GemmPlan plan,
                                  hipStream_t s) {
  if (bf16) {
    if (epi == kEpiPartial) {
      if (plan.tn == kDeepBlocks) {
        launch_bf16_deep<kEpiPartial>(a, plan.splits, s);
      } else if (!plan.nt) {
        launch_bf16_partial<8, 1, 4, false>(a, plan.splits, s);
      } else if (plan.nw == 8) {
        launch_bf16_partial<8, 1>(a, plan.splits, s);
      } else if (plan.nw == 6) {
        launch_bf16_partial<6, 1, 3>(a, plan.splits, s);
      } else {
        launch_bf16_partial<4, 1, 2>(a, plan.splits, s);
      }
    } else {
      launch_bf16_argmax<8, 2, 2>(a, s);
    }
    return hipGetLastError();
  }
  const int tiles = ((a.M + 63) / 64) * ((a.N + 63) / 64);
  if (epi == kEpiPartial)
    hipLaunchKernelGGL(gemm_f32_kernel<kEpiPartial>, dim3(tiles, 1, plan.splits),
                       dim3(kGemmThreads), 0, s, a);
  else
    hipLaunchKernelGGL(gemm_f32_kernel<kEpiArgmax>, dim3(tiles, 1, 1), dim3(kGemmThreads), 0, s,
                       a);
  return hipGetLastError();
}

int gemm_k_align(bool bf16) { return bf16 ? kBK : 16; }

GemmPlan gemm_plan(bool bf16, int M, int N, int K) { return gemm_plan2(bf16, M, N, 0, 0, K); }

static GemmPlan plan_stream(int BM, int M, int N, int M2, int N2, int nk, int ncu,
                            std::initializer_list<int> waves);

GemmPlan gemm_plan2(bool bf16, int M, int N, int M2, int N2, int K) {
  const int ncu = device_cu_count();
  const int nk = K / gemm_k_align(bf16);
  if (!bf16) {
    const int tiles = ((M + 63) / 64) * ((N + 63) / 64);
    int s = (ncu + tiles - 1) / tiles;
    const int max_s = nk / 8 > 1 ? nk / 8 : 1;
    s = s > max_s ? max_s : (s > 8 ? 8 : s);
    return GemmPlan{4, s < 1 ? 1 : s};
  }
  // One workgroup per CU works best for these weight streams: a CU holding two
  // workgroups while others hold one doubles the kernel's critical path.  Pick the
  // tile width (4, 6 or 8 waves of 32 columns) and K split whose workgroup count fills
  // the CUs best without exceeding them; ties go to fewer splits (less partial
  // traffic) and then to more waves (more bytes in flight per CU).  Every split keeps
  // at least 8 K-steps.
  // Above 128 rows the products are matrix-core bound: waves then own two column blocks
  // each, which halves the LDS traffic per MFMA, and fetch the weights through the caches
  // so that the other row tiles find them in L2 (measured at M = 1024: down 90 -> 71 us,
  // the cold context projection 1182 -> 800 us).
  const int BM = (M <= 64 && M2 <= 64) ? 64 : 128;
  const bool mfma_bound = M > 128 || M2 > 128;
  if (mfma_bound) {
    // Matrix-core bound: the deep 128 x 512 tiles.  The time is about the
    // number of rounds of workgroups over the CUs times the K range of one workgroup,
    // plus the fp32 partials of every extra split (charged 15% each): pick the split
    // that minimises rounds / splits * (1 + 0.15 (splits - 1)).  At 1024 rows: gate/up
    // 2 splits (197 -> 185 us), down 4 (86 -> 71 us), QKV 1.
    const int tiles = ((M + BM - 1) / BM) * ((N + 511) / 512) +
                      ((M2 + BM - 1) / BM) * ((N2 + 511) / 512);
    int best_s = 1;
    double best_t = 1e30;
    for (int sp = 1; sp <= 8; ++sp) {
      if (sp > 1 && nk / sp < 8) break;
      const double t = double((tiles * sp + ncu - 1) / ncu) / sp * (1.0 + 0.15 * (sp - 1));
      if (t < best_t - 1e-9) {
        best_t = t;
        best_s = sp;
      }
    }
    return GemmPlan{kDeepWaves, best_s, kDeepBlocks};
  }
  return plan_stream(BM, M, N, M2, N2, nk, ncu, {4, 6, 8});
}

GemmPlan gemm_plan_shared(int M, int N, int M2, int N2, int K) {
  // The row tiles of the first problem (at most two) read the same weight columns at
  // about the same time on one XCD: 8-wave tiles with the weights fetched through L2.
  GemmPlan p = plan_stream(128, M, N, M2, N2, K / kBK, device_cu_count(), {8});
  p.nt = false;
  return p;
}

static GemmPlan plan_stream(int BM, int M, int N, int M2, int N2, int nk, int ncu,
                            std::initializer_list<int> waves) {
  const int tn = 1;
  GemmPlan best{4, 1, tn};
  double best_fill = -1.0;
  for (int nw : waves) {
    const int bn = 32 * nw * tn;
    const int tiles = ((M + BM - 1) / BM) * ((N + bn - 1) / bn) +
                      ((M2 + BM - 1) / BM) * ((N2 + bn - 1) / bn);
    for (int s = 1; s <= 16; ++s) {
      if (s > 1 && nk / s < 8) break;
      const int wgs = tiles * s;
      const int rounds = (wgs + ncu - 1) / ncu;
      const double fill = double(wgs) / double(rounds * ncu);   // busy fraction of CU-rounds
      // Prefer a single round; more rounds only when they are nearly full.
      const double score = fill / rounds + (rounds == 1 ? 1.0 : 0.0);
      const bool tie = score > best_fill - 1e-9 && score < best_fill + 1e-9;
      if (score > best_fill + 1e-9 ||
          (tie && (s < best.splits || (s == best.splits && nw > best.nw)))) {
        best_fill = score;
        best = GemmPlan{nw, s, tn};
      }
    }
  }
  return best;
}

size_t packed_weight_elems(int N, int K) { return size_t((N + 127) / 128) * 128 * size_t(K); }

hipError_t launch_pack_weight(bool bf16, const void* src, void* dst, int N, int K, hipStream_t s) {
  const int64_t chunks = int64_t((N + 127) / 128) * (K / 16) * 4 * 64;
  int64_t blocks = (chunks + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(pack_weight_kernel<bf16_t>, dim3(unsigned(blocks)), dim3(256), 0, s,
                       static_cast<const bf16_t*>(src), static_cast<bf16_t*>(dst), N, K);
  else
    hipLaunchKernelGGL(pack_weight_kernel<float>, dim3(unsigned(blocks)), dim3(256), 0, s,
                       static_cast<const float*>(src), static_cast<float*>(dst), N, K);
  return hipGetLastError();
}

hipError_t launch_gemm_partial(bool bf16, const void* A, int64_t lda, const void* B, int M, int N,
                               int K, GemmPlan plan, float* C, hipStream_t s) {
  GemmArgs a{};
  a.A = A; a.lda = lda; a.B = B;
  a.M = M; a.N = N; a.K = K; a.C = C; a.keys = nullptr;
  return launch_gemm_any(bf16, kEpiPartial, a, plan, s);
}

hipError_t launch_gemm_partial2(const void* A, int64_t lda, const void* B, int M, int N,
                                float* C, const void* A2, int64_t lda2, const void* B2, int M2,
                                int N2, float* C2, int K, GemmPlan plan, hipStream_t s) {
  GemmArgs a{};
  a.A = A; a.lda = lda; a.B = B;
  a.M = M; a.N = N; a.K = K; a.C = C; a.keys = nullptr;
  a.A2 = A2; a.lda2 = lda2; a.B2 = B2; a.M2 = M2; a.N2 = N2; a.C2 = C2;
  return launch_gemm_any(true, kEpiPartial, a, plan, s);
}

hipError_t launch_gemm_kv(const void* A, int64_t lda, const void* B, int M, int d, int hd,
                          GemmPlan plan, const int32_t* plan_pos, const int32_t* plan_row,
                          const float* rope_cs, void* kc, void* vtc, int64_t cap, hipStream_t s) {
  // 512-column tiles lie wholly in K or in V when d % 512 == 0.
  // The matrix-core bound plan with one K split; the K/V epilogue runs on the ping-pong
  // tiles of the same 512 columns.
  if (plan.tn != kDeepBlocks || plan.nw != kDeepWaves || plan.splits != 1 || (hd != 64 && hd != 128) ||
      d % 512 != 0)
    return hipErrorInvalidValue;
  if (M <= 0) return hipSuccess;
  GemmArgs a{};
  a.A = A; a.lda = lda; a.B = B;
  a.M = M; a.N = 2 * d; a.K = d;
  a.plan_pos = plan_pos; a.plan_row = plan_row; a.rope_cs = rope_cs;
  a.kc = kc; a.vtc = vtc; a.cap = cap; a.kv_d = d; a.hd = hd;
  const int tiles = ((M + 127) / 128) * ((2 * d + 511) / 512);
  hipLaunchKernelGGL((gemm_bf16_kernel<128, 8, 2, kEpiKV, 2, false, true>), dim3(tiles), dim3(512),
                     0, s, a);
  return hipGetLastError();
}

GemmPlan lm_head_plan(int64_t) {
  // 8 waves of two 32-column blocks each (512-column tiles).  Above 128 rows the product
  // is matrix-core bound and two blocks per wave halve the LDS traffic per MFMA (M = 1024:
  // 914 -> 848 us); at 128 rows and fewer it is a weight stream, and the wider tile halves
  // the activation bytes each CU reads per weight byte (M = 128: 173 -> 166 us).
  return GemmPlan{8, 1, 2};
}

hipError_t launch_lm_head_keys(bool bf16, const void* hidden, const void* W, int64_t M, int d,
                               int V, unsigned long long* keys, float* logits, hipStream_t s) {
  // keys are zero on entry (the workspace contract); the GEMM folds every row's maximum
  // into them.  Rows are processed in chunks that keep the int32 tile arithmetic in range.
  const int64_t chunk = 1 << 20;
  for (int64_t r0 = 0; r0 < M; r0 += chunk) {
    const int rows = int(M - r0 < chunk ? M - r0 : chunk);
    GemmArgs a{};
    const size_t el = bf16 ? 2 : 4;
    a.A = static_cast<const char*>(hidden) + r0 * d * el;
    a.lda = d; a.B = W;
    a.M = rows; a.N = V; a.K = d;
    a.C = logits != nullptr ? logits + r0 * V : nullptr;
    a.keys = keys + r0;
    const hipError_t e = launch_gemm_any(bf16, kEpiArgmax, a, lm_head_plan(M), s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_lm_head(bool bf16, const void* hidden, const void* W, int64_t M, int d, int V,
                          unsigned long long* keys, int32_t* argmax, float* max_logit,
                          float* logits, hipStream_t s) {
  const hipError_t e = launch_lm_head_keys(bf16, hidden, W, M, d, V, keys, logits, s);
  if (e != hipSuccess) return e;
  // The finalize pass turns the keys into outputs and clears them.
  const int threads = 256;
  const unsigned blocks = unsigned((M + threads - 1) / threads);
  hipLaunchKernelGGL(argmax_finalize_kernel, dim3(blocks), dim3(threads), 0, s, keys, M, argmax,
                     max_logit);
  return hipGetLastError();
}

}  // namespace hdf

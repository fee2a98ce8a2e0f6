// Block attention of the one-pass drafter: every block query of a sequence attends
// to all of that sequence's cached context keys and to all B block keys, with no
// mask (bidirectional within the block; block slots are predicted jointly from
// the anchor and the context, Sec. 1 and Sec. 2.1).  Softmax scale 1/sqrt(hd),
// fp32 softmax with online rescaling.
//
// Layouts (one layer): keys and values of a head in 64-row tiles, each tile in the
// operand order of the MFMA instructions below (kc_offset / vc_offset), so a 64-key
// tile of one head is 16 KB of contiguous keys plus 16 KB of contiguous values and
// every operand load is a contiguous 1 KB per wave.  The context of sequence s starts
// at cache row kv_offsets[s] (a multiple of 64), or, in a paged cache, its tile j is
// page page_table[s][j]; its block keys sit in 64-row slot s of separate block buffers
// of the same layout.
//
// bf16 kernel: grid (chunk, head, sequence x 16-query group), 8 waves.
// With one chunk (n_chunks == 1) a workgroup takes all of its sequence's context
// tiles and the block's tile and writes the normalised output rows.  Otherwise
// chunks 0 .. n_chunks-1 take chunk_len context keys each and chunk n_chunks the
// block's tile, every one writes a partial (O, m, l), and a combine kernel merges
// them (log-sum-exp rescaling).  Wave w takes tiles w, w + NW, ...  A wave keeps its 16
// queries' state in registers:
//   S^T (keys x queries) = K . Q^T     v_mfma_f32_16x16x32_bf16, Q as the B operand
//   O^T (hd x queries)  += V^T . P^T   same instruction, V^T as the A operand, P^T
//                                      as a bf16 hi + lo pair
// Keys inside each 32-key step are ordered so that the S^T accumulator a lane
// holds (4 keys of one query per 16-key sub-tile) is exactly the 8 keys of one
// query the P^T operand needs, so P never leaves registers.  The key loop reads no
// LDS and issues no dependent global loads (the chunk's cache tiles are looked up
// once, into LDS, before it); the two waves of a SIMD overlap one's loads with the
// other's products.  The waves of a workgroup merge through LDS at the end.
//
// When one workgroup owns a (sequence, head) and the projections left split-K partials,
// the workgroup first runs the projection epilogue of its head (qkv_epi.hpp): the
// sequence's new context rows into the cache, its block rows' Q into the Q buffer and K,
// V into the block buffers, all read back only by this workgroup; that saves the
// epilogue's own launch.
#include "common.hpp"
#include "kernels.hpp"
#include "qkv_epi.hpp"

namespace hdf {

constexpr int kCombineThreads = 256;
constexpr int kKeyTile = 64;
constexpr int kMaxChunkTiles = kAttnMaxChunk / kKeyTile;
constexpr int kAttnSortSeqs = 1024;   // longest-context-first dispatch up to this many sequences

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Context chunks of a sequence of T cached positions.
__device__ __forceinline__ int attn_ctx_chunks(const AttnArgs& a, int T) {
  return min(a.n_chunks, (T + a.chunk_len - 1) / a.chunk_len);
}

constexpr int kAttnWaves = 8;
constexpr int kAttnThreads = 64 * kAttnWaves;

// Two waves per SIMD (one workgroup per CU): 256 VGPRs per wave at most.
// FUSE: the workgroup first runs the projection epilogue of its (sequence, head) (AttnArgs
// fuse_epi; only with one workgroup per (sequence, head)).
template <int HD, bool FUSE>
__global__ void __launch_bounds__(kAttnThreads) __attribute__((amdgpu_waves_per_eu(2)))
attn_bf16_kernel(AttnArgs a, bf16_t* __restrict__ out) {
  constexpr int NJ = HD / 32;   // MFMA steps over the head dimension for S
  constexpr int NDT = HD / 16;  // 16-row tiles of O^T
  __shared__ float red_o[kAttnWaves][16][HD + 1];
  __shared__ float red_m[kAttnWaves][16];
  __shared__ float red_l[kAttnWaves][16];
  __shared__ int64_t ctile[kMaxChunkTiles];   // cache tile of each context tile of the chunk

  // Grid (head, sequence slot x query group, chunk): every sequence's first chunk is
  // dispatched before any second chunk, and the blocks' own workgroups (a few keys each)
  // come last, so the long chunks do not trail the launch (ragged 64-sequence step 3.03 ->
  // 3.01 ms against chunk-fastest order).  When the launch is more than two rounds of
  // workgroups, sequence slot j takes the sequence with the j-th longest context (ties by
  // index), so that the dispatch runs longest first and the launch ends on short
  // workgroups: the workgroup ranks the lengths itself (ragged step 3.035 -> 2.991 ms,
  // four alternating runs of 40 steps each).
  const int chunk = blockIdx.z;
  const int h = blockIdx.x;
  const int nqg = (a.B + 15) / 16;
  int s = blockIdx.y / nqg;
  const int qg = blockIdx.y - s * nqg;
  if (!FUSE && a.n_seq > 1 && a.n_seq <= kAttnSortSeqs &&
      uint64_t(gridDim.x) * gridDim.y * gridDim.z > 2ull * uint64_t(a.n_cus)) {
    __shared__ int lens[kAttnSortSeqs];
    __shared__ int pick;
    for (int t = threadIdx.x; t < a.n_seq; t += kAttnThreads) lens[t] = a.ctx_len[t];
    __syncthreads();
    // The ranks are a permutation of 0 .. n_seq-1, so exactly one thread finds slot s.
    for (int t = threadIdx.x; t < a.n_seq; t += kAttnThreads) {
      const int tt = lens[t];
      int rank = 0;
      for (int u = 0; u < a.n_seq; ++u) {
        const int tu = lens[u];
        rank += (tu > tt) || (tu == tt && u < t);
      }
      if (rank == s) pick = t;
    }
    __syncthreads();
    s = pick;
  }
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int g = lane >> 4;       // lane group 0..3
  const int ql = lane & 15;      // query within the group / row within a sub-tile
  const int T = a.ctx_len[s];
  const bool direct = a.n_chunks == 1;
  const bool blk_chunk = chunk == a.n_chunks;   // the block's own workgroup
  if (!direct && !blk_chunk && chunk >= attn_ctx_chunks(a, T)) return;  // past the context

  if constexpr (FUSE) {
    // Head h of this sequence's projected rows, 16 rows a round: threads 0-255 its
    // context rows (new_offsets[s] .. new_offsets[s+1]-1 of epi_ctx), threads 256-511
    // its B block rows (epi_blk).  The keys and values land in the cache and the block
    // buffers and Q in the Q buffer, where the code below reads them; nobody else reads
    // them before the next kernel.  Both halves run every round (the tile function holds
    // workgroup barriers); an empty tile stores nothing and reads row 0.
    static_assert(kAttnThreads == 2 * kQkvThreads, "two epilogue tiles per round");
    __shared__ QkvEpiSmem<HD> esm[2];
    const int half = threadIdx.x / kQkvThreads, et = threadIdx.x % kQkvThreads;
    // The sequence's context rows, clamped to the rows the epilogue holds (offsets past
    // them have no plan entries and no partials; the stand-alone epilogue stops there too).
    const int c1 = min(max(a.new_offsets[s + 1], 0), a.epi_ctx.M);
    const int c0 = min(max(a.new_offsets[s], 0), c1);
    const int rounds = max((c1 - c0 + kQkvRows - 1) / kQkvRows, (a.B + kQkvRows - 1) / kQkvRows);
    for (int it = 0; it < rounds; ++it) {
      if (half == 0) {
        const int r0 = c0 + it * kQkvRows;
        const int rows = max(0, min(kQkvRows, c1 - r0));
        qkv_epi_tile<bf16_t, HD>(a.epi_ctx, rows > 0 ? r0 : 0, rows, h, et, esm[0]);
      } else {
        const int rows = max(0, min(kQkvRows, a.B - it * kQkvRows));
        qkv_epi_tile<bf16_t, HD>(a.epi_blk, rows > 0 ? s * a.B + it * kQkvRows : 0, rows, h, et,
                                 esm[1]);
      }
    }
    __threadfence_block();
    __syncthreads();
  }

  // Context keys [k_lo, k_hi) of the chunk in 64-row tiles (the sequence's tile t is
  // cache tile kv_offsets[s]/64 + t, or page page_table[s][t] of a paged cache); the
  // block's tile (B keys, slot s of the block buffers) follows them.
  const int k_lo = blk_chunk ? 0 : min(T, chunk * a.chunk_len);
  const int k_hi = blk_chunk ? 0 : min(T, k_lo + a.chunk_len);
  const int nct = (k_hi - k_lo + kKeyTile - 1) / kKeyTile;
  const int ntiles = nct + ((direct || blk_chunk) ? 1 : 0);
  const bf16_t* kch = static_cast<const bf16_t*>(a.kc) + int64_t(h) * a.cap * HD;
  const bf16_t* vch = static_cast<const bf16_t*>(a.vtc) + int64_t(h) * a.cap * HD;
  const bf16_t* kbh = static_cast<const bf16_t*>(a.kb) + int64_t(h) * a.capb * HD + lane * 8;
  const bf16_t* vbh = static_cast<const bf16_t*>(a.vtb) + int64_t(h) * a.capb * HD + lane * 8;
  // The chunk's cache tiles go to LDS first, so the key loop has no dependent global
  // loads (each would make a wave wait for all of its outstanding tile loads).
  if (a.page_table != nullptr) {
    const int32_t* pt = a.page_table + int64_t(s) * a.max_pages + (k_lo >> 6);
    for (int j = threadIdx.x; j < nct; j += kAttnThreads) ctile[j] = pt[j];
  } else {
    const int64_t t0 = (a.kv_offsets[s] >> 6) + (k_lo >> 6);
    for (int j = threadIdx.x; j < nct; j += kAttnThreads) ctile[j] = t0 + j;
  }
  __syncthreads();
  // Tile i's first operand (plus this lane's 16 bytes) and its number of valid keys.
  auto k_src = [&](int i) -> const bf16_t* {
    return i >= nct ? kbh + int64_t(s) * 64 * HD : kch + ctile[i] * 64 * HD + lane * 8;
  };
  auto v_src = [&](int i) -> const bf16_t* {
    return i >= nct ? vbh + int64_t(s) * 64 * HD : vch + ctile[i] * 64 * HD + lane * 8;
  };
  auto valid_of = [&](int i) { return i >= nct ? a.B : min(kKeyTile, k_hi - k_lo - i * kKeyTile); };

  // Q^T operand: lane holds Q[query ql][32j + 8g .. +7].
  const int q = qg * 16 + ql;
  bf16x8_t qf[NJ];
  {
    const bf16_t* qrow = static_cast<const bf16_t*>(a.q) + ((int64_t(s) * a.nh + h) * a.B + q) * HD;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      u32x4 v = (q < a.B) ? ld16(qrow + 32 * j + 8 * g) : u32x4{0, 0, 0, 0};
      qf[j] = __builtin_bit_cast(bf16x8_t, v);
    }
  }

  f32x4_t oacc[NDT];
#pragma unroll
  for (int i = 0; i < NDT; ++i) oacc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;
  float l_run = 0.f;

  // K operands of the four 16-key sub-tiles: sub-tile st = 2*ks + p, row r -> key
  // 32ks + 8(r/4) + 4p + r%4 of the tile (the order of the cache tile layout); each
  // operand is 64 lanes x 16 contiguous bytes.  V^T operands: lane holds
  // V^T[16dt + ql][32ks + 8g .. +7].  Each key and value is read once a call: the loads are
  // non-temporal (measured: 8 x 2048 positions 54 -> 49 us, the ragged step's 1533 ->
  // 1438 us).
  bf16x8_t kf[4][NJ];
  u32x4 vf[2][NDT];
  auto load_k = [&](int i) {
    const bf16_t* kt = k_src(i);
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        kf[st][j] = __builtin_bit_cast(bf16x8_t, ld_nt16(kt + (st * NJ + j) * 512));
  };
  auto load_v = [&](int i) {
    const bf16_t* vt = v_src(i);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) vf[ks][dt] = ld_nt16(vt + (ks * NDT + dt) * 512);
  };
  for (int i = wid; i < ntiles; i += kAttnWaves) {
    load_k(i);
    load_v(i);
    const int nval = valid_of(i);
    float sv[4][4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[st][j], qf[j], acc, 0, 0, 0);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = 32 * (st >> 1) + 8 * g + 4 * (st & 1) + e;
        sv[st][e] = (key < nval) ? acc[e] * a.scale_log2 : -INFINITY;
      }
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int e = 0; e < 4; ++e) tmax = fmaxf(tmax, sv[st][e]);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, kWave));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, kWave));
    const float m_new = fmaxf(m_run, tmax);   // finite: every tile has a valid key
    const float alpha = fast_exp2(m_run - m_new);
    m_run = m_new;
    float psum = 0.f;
    float pv[4][4];
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        pv[st][e] = fast_exp2(sv[st][e] - m_new);
        psum += pv[st][e];
      }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int e = 0; e < 4; ++e) oacc[dt][e] *= alpha;

    // Keys past the valid ones carry P = 0; zero their V too (the slot padding is never
    // written and may hold anything).  Only a segment's last tile is partial; its V
    // operands are masked in place (lane keys 32ks + 8g .. +7).
    if (nval < kKeyTile) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int nvalid = nval - (32 * ks + 8 * g);
        uint32_t keep[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          keep[e] = ((2 * e < nvalid) ? 0x0000FFFFu : 0u) | ((2 * e + 1 < nvalid) ? 0xFFFF0000u : 0u);
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int e = 0; e < 4; ++e) vf[ks][dt][e] &= keep[e];
      }
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      // P^T operand: keys 32ks + 8g + 0..7 of query ql, as a bf16 pair hi + lo
      // (P carries ~16 significant bits into the fp32 accumulation; the key loop is
      // HBM-bound, so the second MFMA is free).
      uint32_t hw[4], lw[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = pv[2 * ks + (e >> 1)][2 * (e & 1)];
        const float p1 = pv[2 * ks + (e >> 1)][2 * (e & 1) + 1];
        const bf16_t h0 = f2bf(p0), h1 = f2bf(p1);
        hw[e] = uint32_t(h0) | (uint32_t(h1) << 16);
        lw[e] = pack_bf2(p0 - bf2f(h0), p1 - bf2f(h1));
      }
      const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, u32x4{hw[0], hw[1], hw[2], hw[3]});
      const bf16x8_t pf_lo = __builtin_bit_cast(bf16x8_t, u32x4{lw[0], lw[1], lw[2], lw[3]});
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const bf16x8_t vop = __builtin_bit_cast(bf16x8_t, vf[ks][dt]);
        oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pf, oacc[dt], 0, 0, 0);
        oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pf_lo, oacc[dt], 0, 0, 0);
      }
    }
  }

  // Wave -> LDS: lane (g, ql) holds O^T[16dt + 4g + i][ql].
  l_run += __shfl_xor(l_run, 16, kWave);
  l_run += __shfl_xor(l_run, 32, kWave);
  if (g == 0) {
    red_m[wid][ql] = m_run;
    red_l[wid][ql] = l_run;
  }
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int e = 0; e < 4; ++e) red_o[wid][ql][16 * dt + 4 * g + e] = oacc[dt][e];
  __syncthreads();

  // Merge of the waves: thread -> (query qq, two consecutive dims).
  const int64_t pidx = ((int64_t(s) * a.nh + h) * (a.n_chunks + 1) + chunk) * a.QB + qg * 16;
  for (int e = threadIdx.x; e < 16 * (HD / 2); e += kAttnThreads) {
    const int qq = e / (HD / 2), dim = 2 * (e - qq * (HD / 2));
    float mm = red_m[0][qq];
#pragma unroll
    for (int w = 1; w < kAttnWaves; ++w) mm = fmaxf(mm, red_m[w][qq]);
    float o0 = 0.f, o1 = 0.f, l = 0.f;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) {
      const float f = (red_m[w][qq] == -INFINITY) ? 0.f : fast_exp2(red_m[w][qq] - mm);
      o0 += f * red_o[w][qq][dim];
      o1 += f * red_o[w][qq][dim + 1];
      l += f * red_l[w][qq];
    }
    if (direct) {
      const int qo = qg * 16 + qq;
      if (qo < a.B) {
        const float inv = 1.f / l;
        *reinterpret_cast<uint32_t*>(out + (int64_t(s) * a.B + qo) * (a.nh * HD) +
                                     int64_t(h) * HD + dim) = pack_bf2(o0 * inv, o1 * inv);
      }
    } else {
      *reinterpret_cast<float2*>(a.part_o + (pidx + qq) * HD + dim) = make_float2(o0, o1);
      if (dim == 0) {
        a.part_ml[(pidx + qq) * 2 + 0] = mm;
        a.part_ml[(pidx + qq) * 2 + 1] = l;
      }
    }
  }
}

// Merge the chunk partials of one (sequence, head, 16-query group) -> O rows.
// Phase 1 reads every chunk's (m, l), phase 2 turns them into per-chunk weights
// exp2(m_c - M) / L, phase 3 forms each output quad from independent loads.
template <typename T>
__global__ void __launch_bounds__(kCombineThreads)
attn_combine_kernel(AttnArgs a, T* __restrict__ out) {
  extern __shared__ float cw[];  // [16][n_chunks + 1] weights, then [16][n_chunks + 1] m
  const int h = blockIdx.y;
  const int nqg = (a.B + 15) / 16;
  const int s = blockIdx.x / nqg;
  const int qg = blockIdx.x - s * nqg;
  const int nc = attn_ctx_chunks(a, a.ctx_len[s]) + 1;   // context chunks + the block's
  const int NC = a.n_chunks + 1;
  float* cm = cw + 16 * NC;
  const int d = a.nh * a.hd;
  const int64_t base = (int64_t(s) * a.nh + h) * NC;
  // Phase 1: (m, l) of every chunk of the sequence (the block's is chunk n_chunks).
  for (int e = threadIdx.x; e < 16 * nc; e += kCombineThreads) {
    const int qq = e / nc;
    const int c = e - qq * nc;
    const int cc = (c == nc - 1) ? a.n_chunks : c;
    const int64_t pi = (base + cc) * a.QB + qg * 16 + qq;
    cm[qq * NC + c] = a.part_ml[pi * 2];
    cw[qq * NC + c] = a.part_ml[pi * 2 + 1];
  }
  __syncthreads();
  // Phase 2: per-query weights.
  if (threadIdx.x < 16) {
    const int qq = threadIdx.x;
    float mm = -INFINITY;
    for (int c = 0; c < nc; ++c) mm = fmaxf(mm, cm[qq * NC + c]);
    float l = 0.f;
    for (int c = 0; c < nc; ++c) {
      const float f = (cm[qq * NC + c] == -INFINITY) ? 0.f : fast_exp2(cm[qq * NC + c] - mm);
      cm[qq * NC + c] = f;
      l += f * cw[qq * NC + c];
    }
    const float inv = 1.f / l;
    for (int c = 0; c < nc; ++c) cw[qq * NC + c] = cm[qq * NC + c] * inv;
  }
  __syncthreads();
  // Phase 3: outputs, four consecutive dims per item.
  const int quads = a.hd / 4;
  for (int e = threadIdx.x; e < 16 * quads; e += kCombineThreads) {
    const int qq = e / quads;
    const int q = qg * 16 + qq;
    if (q >= a.B) continue;
    const int i0 = (e - qq * quads) * 4;
    float o[4] = {0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < nc; ++c) {
      const float wgt = cw[qq * NC + c];
      const int cc = (c == nc - 1) ? a.n_chunks : c;
      const float4 v = *reinterpret_cast<const float4*>(
          a.part_o + ((base + cc) * a.QB + q) * a.hd + i0);
      o[0] = fmaf(wgt, v.x, o[0]);
      o[1] = fmaf(wgt, v.y, o[1]);
      o[2] = fmaf(wgt, v.z, o[2]);
      o[3] = fmaf(wgt, v.w, o[3]);
    }
    T* dst = out + (int64_t(s) * a.B + q) * d + int64_t(h) * a.hd + i0;
    if constexpr (sizeof(T) == 2) {
      *reinterpret_cast<uint2*>(dst) = make_uint2(pack_bf2(o[0], o[1]), pack_bf2(o[2], o[3]));
    } else {
      *reinterpret_cast<float4*>(dst) = make_float4(o[0], o[1], o[2], o[3]);
    }
  }
}

// fp32 path (small correctness-size workloads): one thread per query, keys streamed
// from the same layouts, exact expf softmax with online rescaling.
template <int HD>
__global__ void attn_f32_kernel(AttnArgs a, float* __restrict__ out) {
  const int s = blockIdx.x, h = blockIdx.y;
  const int q = threadIdx.x;
  if (q >= a.B) return;
  constexpr int hd = HD;
  const int d = a.nh * hd;
  const float* Q = static_cast<const float*>(a.q) + ((int64_t(s) * a.nh + h) * a.B + q) * hd;
  const float scale = rsqrtf(float(hd));
  float o[HD];
#pragma unroll
  for (int i = 0; i < hd; ++i) o[i] = 0.f;
  float m = -INFINITY, l = 0.f;
  for (int seg = 0; seg < 2; ++seg) {
    const float* K;    // this head's keys and values
    const float* Vt;
    const int32_t* pt = nullptr;
    int64_t row0 = 0;  // cache row of the segment's first key (contiguous layouts)
    int n;
    if (seg == 0) {
      K = static_cast<const float*>(a.kc) + int64_t(h) * a.cap * hd;
      Vt = static_cast<const float*>(a.vtc) + int64_t(h) * a.cap * hd;
      if (a.page_table != nullptr)
        pt = a.page_table + int64_t(s) * a.max_pages;
      else
        row0 = a.kv_offsets[s];
      n = a.ctx_len[s];
    } else {
      K = static_cast<const float*>(a.kb) + int64_t(h) * a.capb * hd;
      Vt = static_cast<const float*>(a.vtb) + int64_t(h) * a.capb * hd;
      row0 = int64_t(s) * 64;
      n = a.B;
    }
    for (int j = 0; j < n; ++j) {
      const int64_t row = pt != nullptr ? int64_t(pt[j >> 6]) * 64 + (j & 63) : row0 + j;
      float sc = 0.f;
      for (int i = 0; i < hd; ++i) sc = fmaf(Q[i], K[kc_index(row, i, hd)], sc);
      sc *= scale;
      const float mn = fmaxf(m, sc);
      const float al = expf(m - mn);
      const float p = expf(sc - mn);
      l = l * al + p;
#pragma unroll
      for (int i = 0; i < hd; ++i)
        o[i] = o[i] * al + p * Vt[vc_index(row, i, hd)];
      m = mn;
    }
  }
  float* dst = out + (int64_t(s) * a.B + q) * d + int64_t(h) * hd;
#pragma unroll
  for (int i = 0; i < hd; ++i) dst[i] = o[i] / l;
}

hipError_t launch_attention(bool bf16, const AttnArgs& args, void* out, hipStream_t s) {
  AttnArgs a = args;
  a.n_cus = device_cu_count();
  if (a.n_seq <= 0) return hipSuccess;
  if (!bf16) {
    if (a.hd == 128)
      hipLaunchKernelGGL(attn_f32_kernel<128>, dim3(a.n_seq, a.nh), dim3(64), 0, s, a,
                         static_cast<float*>(out));
    else
      hipLaunchKernelGGL(attn_f32_kernel<64>, dim3(a.n_seq, a.nh), dim3(64), 0, s, a,
                         static_cast<float*>(out));
    return hipGetLastError();
  }
  if (a.n_chunks < 1 || a.chunk_len % kKeyTile != 0 || a.chunk_len > kAttnMaxChunk)
    return hipErrorInvalidValue;
  const int nqg = (a.B + 15) / 16;
  const dim3 grid(a.nh, a.n_seq * nqg, a.n_chunks == 1 ? 1 : a.n_chunks + 1);
  bf16_t* o = static_cast<bf16_t*>(out);
  if (a.fuse_epi) {
    // The projection epilogue runs in the attention workgroups: one per (sequence, head).
    if (a.n_chunks != 1 || nqg != 1 || a.new_offsets == nullptr) return hipErrorInvalidValue;
    if (a.hd == 128)
      hipLaunchKernelGGL((attn_bf16_kernel<128, true>), grid, dim3(kAttnThreads), 0, s, a, o);
    else
      hipLaunchKernelGGL((attn_bf16_kernel<64, true>), grid, dim3(kAttnThreads), 0, s, a, o);
    return hipGetLastError();
  }
  if (a.hd == 128)
    hipLaunchKernelGGL((attn_bf16_kernel<128, false>), grid, dim3(kAttnThreads), 0, s, a, o);
  else
    hipLaunchKernelGGL((attn_bf16_kernel<64, false>), grid, dim3(kAttnThreads), 0, s, a, o);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_chunks == 1) return e;
  const size_t lds = size_t(2) * 16 * (a.n_chunks + 1) * sizeof(float);
  hipLaunchKernelGGL(attn_combine_kernel<bf16_t>, dim3(a.n_seq * nqg, a.nh), dim3(kCombineThreads),
                     lds, s, a, o);
  return hipGetLastError();
}

}  // namespace hdf

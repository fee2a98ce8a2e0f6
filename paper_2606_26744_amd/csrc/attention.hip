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
// bf16 kernel: grid (context chunk + 1 block chunk, head, sequence x 16-query
// group), 4 waves.  A wave streams 64-key tiles and keeps its 16 queries' state
// in registers:
//   S^T (keys x queries) = K . Q^T     v_mfma_f32_16x16x32_bf16, Q as the B operand
//   O^T (hd x queries)  += V^T . P^T   same instruction, V^T as the A operand, P^T
//                                      as a bf16 hi + lo pair
// Keys inside each 32-key step are ordered so that the S^T accumulator a lane
// holds (4 keys of one query per 16-key sub-tile) is exactly the 8 keys of one
// query the P^T operand needs, so P never leaves registers.  No LDS in the key loop.  The four
// waves of a workgroup merge through LDS at the end; chunks merge in a combine
// kernel (log-sum-exp rescaling).
#include "common.hpp"
#include "kernels.hpp"

namespace hdf {

constexpr int kAttnThreads = 256;
constexpr int kAttnWaves = 4;
constexpr int kKeyTile = 64;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int HD>
__global__ void __launch_bounds__(kAttnThreads)
attn_bf16_kernel(AttnArgs a) {
  constexpr int NJ = HD / 32;   // MFMA steps over the head dimension for S
  constexpr int NDT = HD / 16;  // 16-row tiles of O^T
  __shared__ float red_o[kAttnWaves][16][HD + 1];
  __shared__ float red_m[kAttnWaves][16];
  __shared__ float red_l[kAttnWaves][16];

  const int chunk = blockIdx.x;
  const int h = blockIdx.y;
  const int nqg = (a.B + 15) / 16;
  const int s = blockIdx.z / nqg;
  const int qg = blockIdx.z - s * nqg;
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int g = lane >> 4;       // lane group 0..3
  const int ql = lane & 15;      // query within the group / row within a sub-tile
  const int T = a.ctx_len[s];

  // 64-row tiles of this head's keys (values): tile j of the segment is tile
  // tile0 + j, or page pt[j] of a paged cache.
  const bf16_t* khead;
  const bf16_t* vhead;
  const int32_t* pt = nullptr;
  int64_t tile0 = 0;
  int k_lo, k_hi;
  if (chunk < a.n_chunks) {
    k_lo = chunk * a.chunk_len;
    if (k_lo >= T) return;  // nothing of this sequence in this chunk
    k_hi = min(T, k_lo + a.chunk_len);
    khead = static_cast<const bf16_t*>(a.kc) + int64_t(h) * a.cap * HD;
    vhead = static_cast<const bf16_t*>(a.vtc) + int64_t(h) * a.cap * HD;
    if (a.page_table != nullptr)
      pt = a.page_table + int64_t(s) * a.max_pages;
    else
      tile0 = a.kv_offsets[s] >> 6;
  } else {
    k_lo = 0;
    k_hi = a.B;
    khead = static_cast<const bf16_t*>(a.kb) + int64_t(h) * a.capb * HD;
    vhead = static_cast<const bf16_t*>(a.vtb) + int64_t(h) * a.capb * HD;
    tile0 = s;
  }
  auto tile_of = [&](int t) -> int64_t { return pt != nullptr ? int64_t(pt[t >> 6]) : tile0 + (t >> 6); };

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

  // The tile of the next iteration is looked up one iteration ahead.
  int64_t tile = (k_lo + wid * kKeyTile < k_hi) ? tile_of(k_lo + wid * kKeyTile) : 0;
  for (int t0 = k_lo + wid * kKeyTile; t0 < k_hi; t0 += kAttnWaves * kKeyTile) {
    const int tn = t0 + kAttnWaves * kKeyTile;
    const int64_t tile_next = tn < k_hi ? tile_of(tn) : 0;
    // K operands of the four 16-key sub-tiles: sub-tile st = 2*ks + p, row r -> key
    // t0 + 32ks + 8(r/4) + 4p + r%4 (the order of the cache tile layout).
    // In the cache tile layout each operand is 64 lanes x 16 contiguous bytes.
    const bf16_t* ktile = khead + tile * 64 * HD + lane * 8;
    bf16x8_t kf[4][NJ];
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        kf[st][j] = __builtin_bit_cast(bf16x8_t, ld16(ktile + (st * NJ + j) * 512));
    // V^T operands: lane holds V^T[16dt + ql][t0 + 32ks + 8g .. +7].
    const bf16_t* vtile = vhead + tile * 64 * HD + lane * 8;
    u32x4 vf[2][NDT];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) vf[ks][dt] = ld16(vtile + (ks * NDT + dt) * 512);

    float sv[4][4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[st][j], qf[j], acc, 0, 0, 0);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = t0 + 32 * (st >> 1) + 8 * g + 4 * (st & 1) + i;
        sv[st][i] = (key < k_hi) ? acc[i] * a.scale_log2 : -INFINITY;
      }
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int i = 0; i < 4; ++i) tmax = fmaxf(tmax, sv[st][i]);
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
      for (int i = 0; i < 4; ++i) {
        pv[st][i] = fast_exp2(sv[st][i] - m_new);
        psum += pv[st][i];
      }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) oacc[dt][i] *= alpha;

#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      // P^T operand: keys 32ks + 8g + 0..7 of query ql, as a bf16 pair hi + lo
      // (P carries ~16 significant bits into the fp32 accumulation; the key loop is
      // HBM-bound, so the second MFMA is free).
      float pk[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pk[i] = pv[2 * ks][i];
        pk[4 + i] = pv[2 * ks + 1][i];
      }
      uint32_t hw[4], lw[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bf16_t h0 = f2bf(pk[2 * e]), h1 = f2bf(pk[2 * e + 1]);
        hw[e] = uint32_t(h0) | (uint32_t(h1) << 16);
        lw[e] = pack_bf2(pk[2 * e] - bf2f(h0), pk[2 * e + 1] - bf2f(h1));
      }
      const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, u32x4{hw[0], hw[1], hw[2], hw[3]});
      const bf16x8_t pf_lo = __builtin_bit_cast(bf16x8_t, u32x4{lw[0], lw[1], lw[2], lw[3]});
      // Keys past the segment end carry P = 0; zero their V too (the slot padding
      // is never written and may hold anything).
      const int kfirst = t0 + 32 * ks + 8 * g;
      const int nvalid = k_hi - kfirst;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        u32x4 v = vf[ks][dt];
        if (nvalid < 8) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t keep_lo = (2 * e < nvalid) ? 0x0000FFFFu : 0u;
            const uint32_t keep_hi = (2 * e + 1 < nvalid) ? 0xFFFF0000u : 0u;
            v[e] &= (keep_lo | keep_hi);
          }
        }
        const bf16x8_t vop = __builtin_bit_cast(bf16x8_t, v);
        oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pf, oacc[dt], 0, 0, 0);
        oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pf_lo, oacc[dt], 0, 0, 0);
      }
    }
    tile = tile_next;
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
    for (int i = 0; i < 4; ++i) red_o[wid][ql][16 * dt + 4 * g + i] = oacc[dt][i];
  __syncthreads();

  const int64_t pidx = ((int64_t(s) * a.nh + h) * (a.n_chunks + 1) + chunk) * a.QB + qg * 16;
  for (int e = threadIdx.x; e < 16 * HD; e += kAttnThreads) {
    const int qq = e / HD, dim = e - qq * HD;
    float mm = red_m[0][qq];
#pragma unroll
    for (int w = 1; w < kAttnWaves; ++w) mm = fmaxf(mm, red_m[w][qq]);
    float o = 0.f, l = 0.f;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) {
      const float f = (red_m[w][qq] == -INFINITY) ? 0.f : fast_exp2(red_m[w][qq] - mm);
      o += f * red_o[w][qq][dim];
      l += f * red_l[w][qq];
    }
    a.part_o[(pidx + qq) * HD + dim] = o;
    if (dim == 0) {
      a.part_ml[(pidx + qq) * 2 + 0] = mm;
      a.part_ml[(pidx + qq) * 2 + 1] = l;
    }
  }
}

// Merge the chunk partials of one (sequence, head, 16-query group) -> O rows.
// Phase 1 reads every chunk's (m, l), phase 2 turns them into per-chunk weights
// exp2(m_c - M) / L, phase 3 forms each output quad from independent loads.
template <typename T>
__global__ void __launch_bounds__(kAttnThreads)
attn_combine_kernel(AttnArgs a, T* __restrict__ out) {
  extern __shared__ float cw[];  // [16][n_chunks + 1] weights, then [16][n_chunks + 1] m
  const int h = blockIdx.y;
  const int nqg = (a.B + 15) / 16;
  const int s = blockIdx.x / nqg;
  const int qg = blockIdx.x - s * nqg;
  const int T_s = a.ctx_len[s];
  const int nc = min(a.n_chunks, (T_s + a.chunk_len - 1) / a.chunk_len);
  const int NC = a.n_chunks + 1;
  float* cm = cw + 16 * NC;
  const int d = a.nh * a.hd;
  const int64_t base = (int64_t(s) * a.nh + h) * NC;
  // Phase 1: (m, l) of every used chunk (nc context chunks, then the block chunk).
  for (int e = threadIdx.x; e < 16 * (nc + 1); e += kAttnThreads) {
    const int qq = e / (nc + 1);
    const int c = e - qq * (nc + 1);
    const int cc = (c == nc) ? a.n_chunks : c;
    const int64_t pi = (base + cc) * a.QB + qg * 16 + qq;
    cm[qq * NC + c] = a.part_ml[pi * 2];
    cw[qq * NC + c] = a.part_ml[pi * 2 + 1];
  }
  __syncthreads();
  // Phase 2: per-query weights.
  if (threadIdx.x < 16) {
    const int qq = threadIdx.x;
    float mm = -INFINITY;
    for (int c = 0; c <= nc; ++c) mm = fmaxf(mm, cm[qq * NC + c]);
    float l = 0.f;
    for (int c = 0; c <= nc; ++c) {
      const float f = (cm[qq * NC + c] == -INFINITY) ? 0.f : fast_exp2(cm[qq * NC + c] - mm);
      cm[qq * NC + c] = f;
      l += f * cw[qq * NC + c];
    }
    const float inv = 1.f / l;
    for (int c = 0; c <= nc; ++c) cw[qq * NC + c] = cm[qq * NC + c] * inv;
  }
  __syncthreads();
  // Phase 3: outputs, four consecutive dims per item.
  const int quads = a.hd / 4;
  for (int e = threadIdx.x; e < 16 * quads; e += kAttnThreads) {
    const int qq = e / quads;
    const int q = qg * 16 + qq;
    if (q >= a.B) continue;
    const int i0 = (e - qq * quads) * 4;
    float o[4] = {0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c <= nc; ++c) {
      const int cc = (c == nc) ? a.n_chunks : c;
      const float wgt = cw[qq * NC + c];
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

hipError_t launch_attention(bool bf16, const AttnArgs& a, void* out, hipStream_t s) {
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
  const int nqg = (a.B + 15) / 16;
  const dim3 grid(a.n_chunks + 1, a.nh, a.n_seq * nqg);
  if (a.hd == 128)
    hipLaunchKernelGGL(attn_bf16_kernel<128>, grid, dim3(kAttnThreads), 0, s, a);
  else
    hipLaunchKernelGGL(attn_bf16_kernel<64>, grid, dim3(kAttnThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t lds = size_t(2) * 16 * (a.n_chunks + 1) * sizeof(float);
  hipLaunchKernelGGL(attn_combine_kernel<bf16_t>, dim3(a.n_seq * nqg, a.nh), dim3(kAttnThreads),
                     lds, s, a, static_cast<bf16_t*>(out));
  return hipGetLastError();
}

}  // namespace hdf

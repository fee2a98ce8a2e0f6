// Projection epilogue of one tile of up to kQkvRows rows x one head, shared by the
// stand-alone epilogue kernel (rowwise.hip) and the attention kernel that runs it as its
// prologue (attention.hip): sums the split-K partials, rotates (i, i+hd/2) pairs of Q and
// K at each row's position (RoPE) and stores Q row-major ([n_seq][nh][B][hd]) and K in the
// cache's tile layout; V goes through LDS so that eight consecutive positions of one dim
// leave as one store.  Every thread owns one item of eight dims (a rotated octet of Q or K,
// or eight dims of V) and issues the loads of up to kQkvSplitBatch splits (and its RoPE
// table entries) before the first add; the sums run in split order, as one split at a time
// would.
//
// Rows r0 .. r0 + rows - 1 of the argument set; rows may be 0 (the call then stores
// nothing), in which case row r0 must still be a row of the partial buffers, since the
// loads are issued unpredicated.  kQkvThreads threads take part (tid 0 .. kQkvThreads - 1);
// the function holds three workgroup barriers, which every thread of the workgroup must
// reach the same number of times.  The first one lets back-to-back calls on the same
// `sm` follow each other: the row table of a call is written only after every thread has
// finished reading the previous call's.  The barriers order LDS traffic only: the
// global stores of a call may still be in flight when it returns.
#pragma once

#include "common.hpp"
#include "kernels.hpp"

namespace hdf {

constexpr int kQkvRows = 16;
constexpr int kQkvThreads = 256;
constexpr int kQkvSplitBatch = 4;

template <int HD>
struct QkvEpiSmem {
  float vt_tile[kQkvRows][HD + 1];
  int pos[kQkvRows], seq[kQkvRows], slot[kQkvRows];
  int64_t drow[kQkvRows];
};

template <typename T>
__device__ __forceinline__ void epi_store8(T* p, const float* v);
template <>
__device__ __forceinline__ void epi_store8<bf16_t>(bf16_t* p, const float* v) {
  *reinterpret_cast<uint4*>(p) = make_uint4(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]),
                                            pack_bf2(v[4], v[5]), pack_bf2(v[6], v[7]));
}
template <>
__device__ __forceinline__ void epi_store8<float>(float* p, const float* v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
template <typename T>
__device__ __forceinline__ void epi_store1(T* p, float v);
template <>
__device__ __forceinline__ void epi_store1<bf16_t>(bf16_t* p, float v) { *p = f2bf(v); }
template <>
__device__ __forceinline__ void epi_store1<float>(float* p, float v) { *p = v; }

// Position and destination row of projected row r: block rows (first_part 0) are slot
// r % B of sequence r / B at position ctx_len[s] + slot, stored in row s * 64 + slot of the
// block buffers; context rows take the plan's position and cache row (-1: not a new row).
__device__ __forceinline__ void qkv_row_dest(const QkvEpiArgs& a, int r, int& pos,
                                             int64_t& drow, int& s, int& kslot) {
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

__device__ __forceinline__ void epi_add4(float4& x, const float4 t) {
  x.x += t.x; x.y += t.y; x.z += t.z; x.w += t.w;
}

template <typename T, int HD>
__device__ __forceinline__ void qkv_epi_tile(const QkvEpiArgs& a, int r0, int rows, int h,
                                             int tid, QkvEpiSmem<HD>& sm) {
  constexpr int HALF = HD / 2;
  constexpr int OCT = HALF / 8;          // rotated octets per row and part
  constexpr int VOCT = HD / 8;           // octets of V per row
  static_assert(kQkvRows * 2 * OCT <= kQkvThreads && kQkvRows * VOCT <= kQkvThreads &&
                    (kQkvRows / 8) * HD <= kQkvThreads,
                "one item of each kind per thread");
  lds_barrier();
  if (tid < rows) {
    int pos, s, k;
    int64_t drow;
    qkv_row_dest(a, r0 + tid, pos, drow, s, k);
    sm.pos[tid] = pos;
    sm.seq[tid] = s;
    sm.slot[tid] = k;
    sm.drow[tid] = drow;
  }
  lds_barrier();
  const int nrot = 2 - a.first_part;  // Q and K, or K only

  // This thread's rotated item (row rr, part, octet o: dims i0..i0+7 and i0+HALF..) and
  // V item (row rv, dims 8*ov..8*ov+7).  A context row that is not new has nothing to
  // store.  A thread without an item of a kind loads row 0 of the tile in its place
  // (results unused), so that the loads carry no per-thread branch.
  const int rr = tid / (nrot * OCT);
  const int pp = (tid / OCT) % nrot;
  const int i0 = (tid % OCT) * 8;
  const bool has_r = rr < rows && sm.drow[rr] >= 0;
  const int part = a.first_part + pp;
  const float* rsrc = part == 0 ? a.pq : a.pkv;
  const int64_t rzs = part == 0 ? a.zs_q : a.zs_kv;
  const float* rp = rsrc + int64_t(r0 + (has_r ? rr : 0)) * (part == 0 ? a.ld_q : a.ld_kv) +
                    int64_t(h) * HD + i0;
  const int rv = tid / VOCT, ov = tid % VOCT;
  const bool has_v = rv < rows;
  const float* vp = a.pkv + a.d + int64_t(r0 + (has_v ? rv : 0)) * a.ld_kv + int64_t(h) * HD + 8 * ov;

  float4 cs[4];
  if (has_r && a.rope_cs != nullptr) {
    const float* c = a.rope_cs + (int64_t(sm.pos[rr]) * HALF + i0) * 2;
#pragma unroll
    for (int j = 0; j < 4; ++j) cs[j] = *reinterpret_cast<const float4*>(c + 4 * j);
  }
  // Accumulators start at -0, so adding split 0 gives exactly split 0.
  const float4 nz = make_float4(-0.f, -0.f, -0.f, -0.f);
  float4 xr[4] = {nz, nz, nz, nz};   // dims i0..+3, i0+4..+7, i0+HALF..+3, i0+HALF+4..+7
  float4 xv[2] = {nz, nz};
  for (int z0 = 0; z0 < a.S; z0 += kQkvSplitBatch) {
    float4 tr[kQkvSplitBatch][4], tv[kQkvSplitBatch][2];
#pragma unroll
    for (int j = 0; j < kQkvSplitBatch; ++j) {
      if (z0 + j < a.S) {   // uniform: no per-thread branch between the loads
        const float* q = rp + (z0 + j) * rzs;
        tr[j][0] = *reinterpret_cast<const float4*>(q);
        tr[j][1] = *reinterpret_cast<const float4*>(q + 4);
        tr[j][2] = *reinterpret_cast<const float4*>(q + HALF);
        tr[j][3] = *reinterpret_cast<const float4*>(q + HALF + 4);
        const float* w = vp + (z0 + j) * a.zs_kv;
        tv[j][0] = *reinterpret_cast<const float4*>(w);
        tv[j][1] = *reinterpret_cast<const float4*>(w + 4);
      }
    }
#pragma unroll
    for (int j = 0; j < kQkvSplitBatch; ++j) {
      if (z0 + j < a.S) {
#pragma unroll
        for (int g = 0; g < 4; ++g) epi_add4(xr[g], tr[j][g]);
        epi_add4(xv[0], tv[j][0]);
        epi_add4(xv[1], tv[j][1]);
      }
    }
  }

  if (has_r) {
    float y1[8] = {xr[0].x, xr[0].y, xr[0].z, xr[0].w, xr[1].x, xr[1].y, xr[1].z, xr[1].w};
    float y2[8] = {xr[2].x, xr[2].y, xr[2].z, xr[2].w, xr[3].x, xr[3].y, xr[3].z, xr[3].w};
    if (a.rope_cs != nullptr) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        rope_rotate(y1[2 * j], y2[2 * j], cs[j].x, cs[j].y);
        rope_rotate(y1[2 * j + 1], y2[2 * j + 1], cs[j].z, cs[j].w);
      }
    }
    if (part == 0) {
      T* dst = static_cast<T*>(a.q) + ((int64_t(sm.seq[rr]) * a.nh + h) * a.B + sm.slot[rr]) * HD;
      epi_store8<T>(dst + i0, y1);
      epi_store8<T>(dst + i0 + HALF, y2);
    } else {
      // Eight consecutive dims (i0 % 8 == 0) are contiguous in the cache tile layout.
      T* kh = static_cast<T*>(a.k) + int64_t(h) * a.cap * HD;
      epi_store8<T>(kh + kc_index(sm.drow[rr], i0, HD), y1);
      epi_store8<T>(kh + kc_index(sm.drow[rr], i0 + HALF, HD), y2);
    }
  }
  if (has_v) {
    float* t = &sm.vt_tile[rv][8 * ov];
    t[0] = xv[0].x; t[1] = xv[0].y; t[2] = xv[0].z; t[3] = xv[0].w;
    t[4] = xv[1].x; t[5] = xv[1].y; t[6] = xv[1].z; t[7] = xv[1].w;
  }
  lds_barrier();
  // V out: item (dim i, group of eight rows).  Eight new rows at eight consecutive cache
  // rows starting at a multiple of 8 are one contiguous run of the value tile layout.
  const int i = tid % HD, g = tid / HD;
  const int gr0 = 8 * g;
  if (gr0 < rows) {
    T* vt = static_cast<T*>(a.vt) + int64_t(h) * a.cap * HD;
    const int64_t d0 = sm.drow[gr0];
    bool run = gr0 + 8 <= rows && d0 >= 0 && (d0 & 7) == 0;
#pragma unroll
    for (int k = 1; k < 8; ++k) run = run && sm.drow[gr0 + k] == d0 + k;
    if (run) {
      float v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = sm.vt_tile[gr0 + k][i];
      epi_store8<T>(vt + vc_index(d0, i, HD), v);
    } else {
      for (int k = 0; k < 8 && gr0 + k < rows; ++k)
        if (sm.drow[gr0 + k] >= 0)
          epi_store1<T>(vt + vc_index(sm.drow[gr0 + k], i, HD), sm.vt_tile[gr0 + k][i]);
    }
  }
}

}  // namespace hdf

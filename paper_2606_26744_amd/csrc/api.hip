// C ABI of libhdf: argument validation, workspace planning and kernel dispatch.
// Every check runs on the host before the first HIP call, so a rejected call
// touches neither the device nor any output.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <initializer_list>
#include <mutex>

#include "../../include/hdf.h"
#include "kernels.hpp"

namespace {

thread_local char g_err[512];

hdf_status fail(hdf_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

hdf_status ok() {
  g_err[0] = '\0';
  return HDF_OK;
}

hdf_status hip_fail(hipError_t e, const char* where) {
  return fail(HDF_E_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

namespace hdf {

int device_cu_count() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v > 0) return v;
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = 256;
  cache[dev].store(n, std::memory_order_relaxed);
  return n;
}

}  // namespace hdf


// ---------------------------------------------------------------- drafter planning
namespace {

constexpr int64_t kCtxChunk = 16384;  // context rows projected per GEMM launch
// Context rows that share one launch with the block's Q/K/V.  More rows keep the matrix
// cores busy on their own, and the block's tiles would only add a partial round
// (8 x 2048 cold rows: 9 rounds of workgroups instead of 8, 1032 -> 927 us).
constexpr int64_t kGroupRows = 2048;

// Up to 128 context rows and 128 block rows: one problem takes both row sets over the
// K/V columns (two row tiles streaming the same weights through L2), the other the block
// rows over the Q columns, so the K/V weights are fetched once per layer, not twice.
bool kv_shared(bool bf, int64_t n_new, size_t M) {
  return bf && n_new > 0 && n_new <= 128 && M <= 128;
}

hdf_status validate_drafter(const hdf_drafter* w) {
  if (w == nullptr) return fail(HDF_E_INVALID, "drafter: null");
  if (w->dtype != HDF_F32 && w->dtype != HDF_BF16) return fail(HDF_E_INVALID, "drafter: bad dtype");
  if (w->n_layers < 1) return fail(HDF_E_INVALID, "drafter: n_layers < 1");
  if (w->d <= 0 || w->n_heads <= 0 || w->head_dim <= 0 || w->d_ff <= 0 || w->vocab <= 0)
    return fail(HDF_E_INVALID, "drafter: non-positive size");
  if (int64_t(w->n_heads) * w->head_dim != w->d)
    return fail(HDF_E_INVALID, "drafter: n_heads * head_dim != d");
  if (w->head_dim != 64 && w->head_dim != 128)
    return fail(HDF_E_UNSUPPORTED, "drafter: head_dim %d not in {64, 128}", w->head_dim);
  if (w->d % 128 != 0 || w->d > 8192)
    return fail(HDF_E_UNSUPPORTED, "drafter: d=%d must be a multiple of 128 up to 8192", w->d);
  if (w->d_ff % 64 != 0) return fail(HDF_E_UNSUPPORTED, "drafter: d_ff %% 64 != 0");
  if (!(w->eps > 0.f)) return fail(HDF_E_INVALID, "drafter: eps must be > 0");
  if (w->tok_emb == nullptr || w->w_qkv == nullptr || w->w_o == nullptr ||
      w->w_gate_up == nullptr || w->w_down == nullptr || w->attn_norm == nullptr ||
      w->mlp_norm == nullptr)
    return fail(HDF_E_INVALID, "drafter: null weight pointer");
  for (int l = 0; l < w->n_layers; ++l)
    if (w->w_qkv[l] == nullptr || w->w_o[l] == nullptr || w->w_gate_up[l] == nullptr ||
        w->w_down[l] == nullptr)
      return fail(HDF_E_INVALID, "drafter: null weight of layer %d", l);
  if (w->rope_cs != nullptr && w->rope_max_pos < 1)
    return fail(HDF_E_INVALID, "drafter: rope_max_pos < 1 with a RoPE table");
  return HDF_OK;
}

struct DraftPlan {
  size_t plan_pos, plan_row, c, h, u, q, kb, vtb, parts, part_o, part_ml, attn, act, total;
  int chunk_len;
};

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

DraftPlan plan_workspace(const hdf_drafter& w, int n_seq, int B, int64_t n_new, int max_ctx) {
  DraftPlan P{};
  const bool bf = w.dtype == HDF_BF16;
  const size_t el = bf ? 2 : 4;
  const size_t d = w.d, F = w.d_ff;
  const size_t M = size_t(n_seq) * B;
  const size_t QB = size_t((B + 15) / 16) * 16;
  const int64_t crow = n_new < kCtxChunk ? n_new : kCtxChunk;
  // Attention split (8-wave workgroups, one per CU).  When one round of them covers every
  // (sequence, head) pair, a chunk is the longest power of two from 512 up that still
  // gives every CU a workgroup (at most 16384): 8 x 2048 positions take one chunk of
  // 2048 keys and need no merge.  Otherwise chunks are the longest power of two in
  // [512, 16384] that still gives four workgroups per CU (each chunk costs a partial
  // output and a merge): one chunk of 16384 keys for 64 sequences of up to 16K positions
  // (ragged step 3.82 -> 3.27 ms from 512 to 4096 keys with 4-wave workgroups, 3.22 ->
  // 3.17 ms from those to 8-wave workgroups of 8192 keys, 3.01 -> 2.97 ms from 8192 keys
  // and a merge to one chunk).
  {
    const int64_t pairs = int64_t(n_seq) * w.n_heads * ((B + 15) / 16);
    const int64_t cus = hdf::device_cu_count();
    int64_t c = 512;
    while (c < hdf::kAttnMaxChunk && c < max_ctx &&
           pairs * ((max_ctx + 2 * c - 1) / (2 * c)) >= cus)
      c *= 2;
    if (pairs * std::max<int64_t>(1, (max_ctx + c - 1) / c) > cus) {
      const int64_t per_wg = int64_t(n_seq) * max_ctx * w.n_heads / (int64_t(4) * cus);
      c = 512;
      while (c < hdf::kAttnMaxChunk && 2 * c <= per_wg) c *= 2;
    }
    P.chunk_len = int(c);
  }
  const size_t n_chunks = size_t(std::max(1, (max_ctx + P.chunk_len - 1) / P.chunk_len));
  size_t parts = 0;
  auto upd = [&](int64_t rows, int N, int K) {
    if (rows <= 0) return;
    const size_t sp = size_t(hdf::gemm_plan(bf, int(rows), N, K).splits);
    const size_t b = sp * size_t(rows) * size_t(N) * 4;
    if (b > parts) parts = b;
  };
  upd(crow, 2 * w.d, w.d);
  upd(n_new % kCtxChunk, 2 * w.d, w.d);  // a shorter last chunk may split further
  if (kv_shared(bf, n_new, M)) {
    // [context rows; block rows] x K/V and block rows x Q in one launch.
    const int rows1 = int(n_new + M);
    const size_t sp = size_t(hdf::gemm_plan_shared(rows1, 2 * w.d, int(M), w.d, w.d).splits);
    const size_t b = sp * (size_t(rows1) * 2 * w.d + M * w.d) * 4;
    if (b > parts) parts = b;
  } else if (bf && n_new > 0 && n_new <= kGroupRows) {
    // Context K/V and block QKV in one launch: both problems' partials.
    const size_t sp = size_t(hdf::gemm_plan2(bf, int(n_new), 2 * w.d, int(M), 3 * w.d, w.d).splits);
    const size_t b = sp * (size_t(n_new) * 2 * w.d + M * 3 * w.d) * 4;
    if (b > parts) parts = b;
  }
  upd(int64_t(M), 3 * w.d, w.d);
  upd(int64_t(M), w.d, w.d);
  upd(int64_t(M), 2 * w.d_ff, w.d);
  upd(int64_t(M), w.d, w.d_ff);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  P.plan_pos = take(size_t(n_new) * 4);
  P.plan_row = take(size_t(n_new) * 4);
  // The block rows' normed states u follow the context rows' c, so that one GEMM
  // problem can take both row sets.
  P.c = take((size_t(crow) + M) * d * el);
  P.u = P.c + size_t(crow) * d * el;
  P.h = take(M * d * 4);
  P.q = take(M * d * el);
  P.kb = take(size_t(w.n_heads) * size_t(n_seq) * 64 * w.head_dim * el);
  P.vtb = take(size_t(w.n_heads) * size_t(n_seq) * 64 * w.head_dim * el);
  P.parts = take(parts);
  const size_t pslots = size_t(n_seq) * w.n_heads * (n_chunks + 1) * QB;
  P.part_o = take(pslots * w.head_dim * 4);
  P.part_ml = take(pslots * 2 * 4);
  P.attn = take(M * d * el);
  P.act = take(M * F * el);
  P.total = off;
  return P;
}

}  // namespace

extern "C" {

const char* hdf_last_error(void) { return g_err; }

int hdf_version(void) { return 100; }

hdf_status hdf_hc_reduce(const void* H, const void* W_g, const float* b_g, int64_t n_tok, int m,
                         int d, hdf_dtype dtype, const hdf_reduce_params* params, void* Y,
                         float* alpha, hdf_stream_t stream) {
  if (dtype != HDF_F32 && dtype != HDF_BF16) return fail(HDF_E_INVALID, "hc_reduce: bad dtype");
  if (n_tok < 0) return fail(HDF_E_INVALID, "hc_reduce: n_tok < 0");
  if (m < 1 || m > 8) return fail(HDF_E_INVALID, "hc_reduce: m=%d outside [1, 8]", m);
  if (d <= 0) return fail(HDF_E_INVALID, "hc_reduce: d=%d", d);
  const bool bf = dtype == HDF_BF16;
  const int vec = bf ? 8 : 4;
  if (d % vec != 0) return fail(HDF_E_INVALID, "hc_reduce: d=%d not a multiple of %d", d, vec);
  if (d / vec > 1024)
    return fail(HDF_E_UNSUPPORTED, "hc_reduce: d=%d above %d for this dtype", d, 1024 * vec);
  hdf_reduce_params p = {1e-6f, 1.0f, 0.0f, 0};
  if (params != nullptr) p = *params;
  if (!(p.eps > 0.f)) return fail(HDF_E_INVALID, "hc_reduce: eps must be > 0");
  if (p.per_path_norm != 0 && p.per_path_norm != 1)
    return fail(HDF_E_INVALID, "hc_reduce: per_path_norm must be 0 or 1");
  if (n_tok == 0) return ok();
  if (H == nullptr || W_g == nullptr || b_g == nullptr || Y == nullptr)
    return fail(HDF_E_INVALID, "hc_reduce: null pointer");
  if (!aligned16(H) || !aligned16(W_g) || !aligned16(Y))
    return fail(HDF_E_INVALID, "hc_reduce: H, W_g and Y must be 16-byte aligned");
  if (int64_t(m) * d * n_tok / n_tok != int64_t(m) * d)
    return fail(HDF_E_INVALID, "hc_reduce: size overflow");
  hdf::ReduceScalars sc{p.eps, p.gate_scale, p.gate_offset, p.per_path_norm};
  hipError_t e = hdf::launch_hc_reduce(bf, m, H, W_g, b_g, n_tok, d, sc, Y, alpha,
                                       reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "hc_reduce launch");
  return ok();
}

// Generic fc reducer: rows are projected kFcChunk at a time, each chunk's split-K
// partials summed (+ bias) and rounded by one row-wise pass.
static constexpr int64_t kFcChunk = 16384;

static bool fc_shape_ok(int m, int d, hdf_dtype dtype) {
  if (dtype != HDF_F32 && dtype != HDF_BF16) return false;
  if (m < 1 || m > 8 || d < 4 || d % 4 != 0) return false;
  return (int64_t(m) * d) % hdf::gemm_k_align(dtype == HDF_BF16) == 0;
}

static size_t fc_parts_bytes(int64_t n_tok, int m, int d, hdf_dtype dtype) {
  const int64_t rows = n_tok < kFcChunk ? n_tok : kFcChunk;
  if (rows <= 0) return 0;
  const hdf::GemmPlan pl = hdf::gemm_plan(dtype == HDF_BF16, int(rows), d, m * d);
  return size_t(pl.splits) * size_t(rows) * size_t(d) * 4;
}

size_t hdf_fc_reduce_workspace(int64_t n_tok, int m, int d, hdf_dtype dtype) {
  if (n_tok < 0 || !fc_shape_ok(m, d, dtype)) return 0;
  return (fc_parts_bytes(n_tok, m, d, dtype) + 255) / 256 * 256;
}

hdf_status hdf_fc_reduce(const void* H, const void* W_fc, const float* b_fc, int64_t n_tok, int m,
                         int d, hdf_dtype dtype, void* Y, void* ws, size_t ws_bytes,
                         hdf_stream_t stream) {
  if (dtype != HDF_F32 && dtype != HDF_BF16) return fail(HDF_E_INVALID, "fc_reduce: bad dtype");
  if (n_tok < 0) return fail(HDF_E_INVALID, "fc_reduce: n_tok < 0");
  if (m < 1 || m > 8) return fail(HDF_E_INVALID, "fc_reduce: m=%d outside [1, 8]", m);
  if (!fc_shape_ok(m, d, dtype))
    return fail(HDF_E_INVALID, "fc_reduce: d=%d (need d %% 4 == 0 and m*d a multiple of %d)", d,
                hdf::gemm_k_align(dtype == HDF_BF16));
  if (n_tok > INT32_MAX) return fail(HDF_E_UNSUPPORTED, "fc_reduce: n_tok beyond 2^31 - 1");
  if (n_tok == 0) return ok();
  if (H == nullptr || W_fc == nullptr || Y == nullptr)
    return fail(HDF_E_INVALID, "fc_reduce: null pointer");
  if (!aligned16(H) || !aligned16(W_fc) || !aligned16(Y))
    return fail(HDF_E_INVALID, "fc_reduce: H, W_fc and Y must be 16-byte aligned");
  const size_t need = fc_parts_bytes(n_tok, m, d, dtype);
  if (ws == nullptr || ws_bytes < need)
    return fail(HDF_E_WORKSPACE, "fc_reduce: workspace of %zu bytes needed, %zu given", need,
                ws_bytes);
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0)
    return fail(HDF_E_INVALID, "fc_reduce: workspace must be 256-byte aligned");
  const bool bf = dtype == HDF_BF16;
  const size_t el = bf ? 2 : 4;
  const int K = m * d;
  const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  float* parts = static_cast<float*>(ws);
  for (int64_t r0 = 0; r0 < n_tok; r0 += kFcChunk) {
    const int rows = int(n_tok - r0 < kFcChunk ? n_tok - r0 : kFcChunk);
    const hdf::GemmPlan pl = hdf::gemm_plan(bf, rows, d, K);
    hipError_t e = hdf::launch_gemm_partial(bf, static_cast<const char*>(H) + r0 * K * el, K, W_fc,
                                            rows, d, K, pl, parts, s);
    if (e != hipSuccess) return hip_fail(e, "fc_reduce gemm");
    e = hdf::launch_split_sum_store(bf, parts, pl.splits, rows, d, b_fc,
                                    static_cast<char*>(Y) + r0 * d * el, s);
    if (e != hipSuccess) return hip_fail(e, "fc_reduce store");
  }
  return ok();
}

size_t hdf_sample_workspace(int64_t rows, int vocab) {
  if (rows < 0 || vocab < 1) return 0;
  return (hdf::sample_parts_bytes(rows, vocab) + 255) / 256 * 256;
}

hdf_status hdf_sample_tokens(const float* logits, int64_t rows, int vocab, int64_t ld,
                             float temperature, uint64_t seed, uint64_t stream_id, int32_t* tokens,
                             float* lse, void* ws, size_t ws_bytes, hdf_stream_t stream) {
  if (rows < 0 || vocab < 1) return fail(HDF_E_INVALID, "sample_tokens: rows=%lld vocab=%d",
                                          static_cast<long long>(rows), vocab);
  if (ld < vocab) return fail(HDF_E_INVALID, "sample_tokens: ld < vocab");
  if (!(temperature > 0.f) || !(temperature < INFINITY))
    return fail(HDF_E_INVALID, "sample_tokens: temperature must be positive and finite");
  if (rows > 65535) return fail(HDF_E_UNSUPPORTED, "sample_tokens: more than 65535 rows");
  if (rows == 0) return ok();
  if (logits == nullptr || (tokens == nullptr && lse == nullptr))
    return fail(HDF_E_INVALID, "sample_tokens: null pointer");
  const size_t need = hdf_sample_workspace(rows, vocab);
  if (ws == nullptr || ws_bytes < need)
    return fail(HDF_E_WORKSPACE, "sample_tokens: workspace of %zu bytes needed, %zu given", need,
                ws_bytes);
  hipError_t e = hdf::launch_row_softmax(logits, rows, vocab, ld, 1.f / temperature,
                                         tokens != nullptr, seed, stream_id, tokens, lse, ws,
                                         reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "sample_tokens launch");
  return ok();
}

size_t hdf_accept_sample_workspace(int n_seq, int K, int vocab) {
  if (n_seq < 0 || K < 0 || vocab < 1) return 0;
  return hdf::accept_sample_ws_bytes(n_seq, K, vocab);
}

hdf_status hdf_accept_sample(const int32_t* draft, int draft_stride, const float* draft_logits,
                             const float* draft_lse, int64_t ld, const float* target_logits,
                             int n_seq, int K, int vocab, float temperature, uint64_t seed,
                             uint64_t stream_id, int32_t* accept_len, int32_t* next_anchor,
                             int32_t* commit_offsets, int32_t* commit_tokens, void* ws,
                             size_t ws_bytes, hdf_stream_t stream) {
  if (n_seq < 0) return fail(HDF_E_INVALID, "accept_sample: n_seq < 0");
  if (K < 0 || K > 1024) return fail(HDF_E_INVALID, "accept_sample: K=%d outside [0, 1024]", K);
  if (vocab < 1) return fail(HDF_E_INVALID, "accept_sample: vocab < 1");
  if (draft_stride < K) return fail(HDF_E_INVALID, "accept_sample: draft_stride < K");
  if (K > 0 && ld < vocab) return fail(HDF_E_INVALID, "accept_sample: ld < vocab");
  if (!(temperature > 0.f) || !(temperature < INFINITY))
    return fail(HDF_E_INVALID, "accept_sample: temperature must be positive and finite");
  if (n_seq > 65535 || int64_t(n_seq) * (K + 1) > 65535)
    return fail(HDF_E_UNSUPPORTED, "accept_sample: more than 65535 target rows");
  if (n_seq == 0) return ok();
  if ((K > 0 && (draft == nullptr || draft_logits == nullptr || draft_lse == nullptr)) ||
      target_logits == nullptr || accept_len == nullptr || next_anchor == nullptr)
    return fail(HDF_E_INVALID, "accept_sample: null pointer");
  const size_t need = hdf::accept_sample_ws_bytes(n_seq, K, vocab);
  if (ws == nullptr || ws_bytes < need)
    return fail(HDF_E_WORKSPACE, "accept_sample: workspace of %zu bytes needed, %zu given", need,
                ws_bytes);
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0)
    return fail(HDF_E_INVALID, "accept_sample: workspace must be 256-byte aligned");
  hipError_t e = hdf::launch_accept_sample(draft, draft_stride, draft_logits, draft_lse, ld,
                                           target_logits, n_seq, K, vocab, 1.f / temperature, seed,
                                           stream_id, accept_len, next_anchor, commit_offsets,
                                           commit_tokens, ws, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "accept_sample launch");
  return ok();
}

size_t hdf_kl_forward_workspace(int n_seq, int B, int P, int d, int vocab, hdf_dtype dtype) {
  if (n_seq < 0 || B < 2 || P < 1 || P > B - 1 || d < 64 || vocab < 1 ||
      (dtype != HDF_F32 && dtype != HDF_BF16))
    return 0;
  return hdf::kl_ws_bytes(n_seq, B, P, d, vocab, dtype == HDF_BF16);
}

hdf_status hdf_kl_forward(const void* H_pos, int m, const float* gamma, float eps, const void* W_lm,
                          int d, int vocab, hdf_dtype dtype, const float* student_logits,
                          int64_t ld, int B, const int32_t* labels, int n_seq, int P,
                          float temperature, float alpha, float* kl, float* ce, float* loss,
                          void* ws, size_t ws_bytes, hdf_stream_t stream) {
  if (dtype != HDF_F32 && dtype != HDF_BF16) return fail(HDF_E_INVALID, "kl_forward: bad dtype");
  if (n_seq < 0) return fail(HDF_E_INVALID, "kl_forward: n_seq < 0");
  if (m < 1 || m > 8) return fail(HDF_E_INVALID, "kl_forward: m=%d outside [1, 8]", m);
  if (B < 2 || B > 64) return fail(HDF_E_INVALID, "kl_forward: B=%d outside [2, 64]", B);
  if (P < 1 || P > B - 1) return fail(HDF_E_INVALID, "kl_forward: P=%d outside [1, B-1]", P);
  if (d % 64 != 0 || d < 64 || d > 8192)
    return fail(HDF_E_INVALID, "kl_forward: d=%d must be a multiple of 64 up to 8192", d);
  if (vocab < 1 || ld < vocab) return fail(HDF_E_INVALID, "kl_forward: vocab/ld");
  if (!(eps > 0.f)) return fail(HDF_E_INVALID, "kl_forward: eps must be > 0");
  if (!(temperature > 0.f) || !(temperature < INFINITY))
    return fail(HDF_E_INVALID, "kl_forward: temperature must be positive and finite");
  if (int64_t(n_seq) * B > 65535)
    return fail(HDF_E_UNSUPPORTED, "kl_forward: more than 65535 draft rows");
  if (n_seq == 0) return ok();
  if (H_pos == nullptr || W_lm == nullptr || student_logits == nullptr || kl == nullptr)
    return fail(HDF_E_INVALID, "kl_forward: null pointer");
  const size_t need = hdf::kl_ws_bytes(n_seq, B, P, d, vocab, dtype == HDF_BF16);
  if (ws == nullptr || ws_bytes < need)
    return fail(HDF_E_WORKSPACE, "kl_forward: workspace of %zu bytes needed, %zu given", need,
                ws_bytes);
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0)
    return fail(HDF_E_INVALID, "kl_forward: workspace must be 256-byte aligned");
  hipError_t e = hdf::launch_kl_forward(dtype == HDF_BF16, H_pos, m, gamma, eps, W_lm, d, vocab,
                                        student_logits, ld, B, labels, n_seq, P, temperature, alpha,
                                        kl, ce, loss, ws, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "kl_forward launch");
  return ok();
}

hdf_status hdf_accept(const int32_t* draft, int draft_stride, const int32_t* target, int n_seq,
                      int K, int32_t* accept_len, int32_t* next_anchor, int32_t* commit_offsets,
                      int32_t* commit_tokens, hdf_stream_t stream) {
  if (n_seq < 0) return fail(HDF_E_INVALID, "accept: n_seq < 0");
  if (K < 0 || K > 1024) return fail(HDF_E_INVALID, "accept: K=%d outside [0, 1024]", K);
  if (draft_stride < K) return fail(HDF_E_INVALID, "accept: draft_stride < K");
  if (n_seq == 0) return ok();
  if ((K > 0 && draft == nullptr) || target == nullptr || accept_len == nullptr ||
      next_anchor == nullptr)
    return fail(HDF_E_INVALID, "accept: null pointer");
  if (int64_t(n_seq) * (K + 1) > INT32_MAX)
    return fail(HDF_E_UNSUPPORTED, "accept: n_seq*(K+1) exceeds int32 offsets");
  hipError_t e = hdf::launch_accept(draft, draft_stride, target, n_seq, K, accept_len, next_anchor,
                                    commit_offsets, commit_tokens,
                                    reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "accept launch");
  return ok();
}

hdf_status hdf_rope_table(float* out_host, int n_pos, int head_dim, double theta) {
  if (out_host == nullptr) return fail(HDF_E_INVALID, "rope_table: null pointer");
  if (n_pos < 0 || head_dim <= 0 || head_dim % 2 != 0)
    return fail(HDF_E_INVALID, "rope_table: bad sizes");
  if (!(theta > 0.0)) return fail(HDF_E_INVALID, "rope_table: theta must be > 0");
  const int half = head_dim / 2;
  for (int p = 0; p < n_pos; ++p) {
    for (int i = 0; i < half; ++i) {
      const double inv = pow(theta, -2.0 * double(i) / double(head_dim));
      const double a = double(p) * inv;
      out_host[(int64_t(p) * half + i) * 2 + 0] = float(cos(a));
      out_host[(int64_t(p) * half + i) * 2 + 1] = float(sin(a));
    }
  }
  return ok();
}

size_t hdf_kv_cache_bytes(const hdf_drafter* w, int64_t kv_cap) {
  if (w == nullptr || kv_cap < 0) return 0;
  const size_t el = w->dtype == HDF_BF16 ? 2 : 4;
  return size_t(w->n_layers) * size_t(w->d) * size_t(kv_cap) * el;
}

static hdf_status kv_rows_check(const char* fn, const void* kc, const void* vc, int64_t kv_cap,
                                int layer, int n_heads, int head_dim, hdf_dtype dtype,
                                const int32_t* rows, int64_t row0, int64_t n_rows,
                                const void* krows, const void* vrows) {
  if (dtype != HDF_F32 && dtype != HDF_BF16) return fail(HDF_E_INVALID, "%s: bad dtype", fn);
  if (n_rows < 0 || row0 < 0 || layer < 0 || n_heads < 1)
    return fail(HDF_E_INVALID, "%s: negative size, row or layer", fn);
  if (head_dim != 64 && head_dim != 128)
    return fail(HDF_E_UNSUPPORTED, "%s: head_dim %d not in {64, 128}", fn, head_dim);
  if (kv_cap <= 0 || kv_cap % 64 != 0)
    return fail(HDF_E_INVALID, "%s: kv_cap must be a positive multiple of 64", fn);
  if (kv_cap > INT32_MAX || n_rows > INT32_MAX)
    return fail(HDF_E_UNSUPPORTED, "%s: rows beyond 2^31 - 1", fn);
  if (rows == nullptr && row0 + n_rows > kv_cap)
    return fail(HDF_E_INVALID, "%s: rows row0..row0+n_rows-1 leave the cache (kv_cap %lld)", fn,
                static_cast<long long>(kv_cap));
  if (n_rows == 0) return HDF_OK;
  const bool kp = kc != nullptr && krows != nullptr, vp = vc != nullptr && vrows != nullptr;
  if (!kp && !vp) return fail(HDF_E_INVALID, "%s: neither a key nor a value pair given", fn);
  if ((kc == nullptr) != (krows == nullptr) || (vc == nullptr) != (vrows == nullptr))
    return fail(HDF_E_INVALID, "%s: a cache array without its rows (or the reverse)", fn);
  for (const void* p : {kc, vc, krows, vrows})
    if (p != nullptr && !aligned16(p))
      return fail(HDF_E_INVALID, "%s: tensors must be 16-byte aligned", fn);
  return HDF_OK;
}

hdf_status hdf_kv_write_rows(const void* k_rows, const void* v_rows, int64_t n_rows,
                             const int32_t* rows, int64_t row0, int layer, int n_heads,
                             int head_dim, hdf_dtype dtype, void* kv_k, void* kv_vt,
                             int64_t kv_cap, hdf_stream_t stream) {
  const hdf_status st = kv_rows_check("kv_write_rows", kv_k, kv_vt, kv_cap, layer, n_heads,
                                      head_dim, dtype, rows, row0, n_rows, k_rows, v_rows);
  if (st != HDF_OK || n_rows == 0) return st == HDF_OK ? ok() : st;
  const size_t el = dtype == HDF_BF16 ? 2 : 4;
  const size_t layer_bytes = size_t(n_heads) * size_t(kv_cap) * head_dim * el;
  char* kc = kv_k ? static_cast<char*>(kv_k) + size_t(layer) * layer_bytes : nullptr;
  char* vc = kv_vt ? static_cast<char*>(kv_vt) + size_t(layer) * layer_bytes : nullptr;
  const hipError_t e = hdf::launch_kv_rows(dtype == HDF_BF16, true, kc, vc, kv_cap,
                                           const_cast<void*>(k_rows), const_cast<void*>(v_rows),
                                           n_rows, rows, row0, n_heads, head_dim,
                                           reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "kv_write_rows launch");
  return ok();
}

hdf_status hdf_kv_read_rows(const void* kv_k, const void* kv_vt, int64_t kv_cap, int layer,
                            int n_heads, int head_dim, hdf_dtype dtype, const int32_t* rows,
                            int64_t row0, int64_t n_rows, void* k_rows, void* v_rows,
                            hdf_stream_t stream) {
  const hdf_status st = kv_rows_check("kv_read_rows", kv_k, kv_vt, kv_cap, layer, n_heads,
                                      head_dim, dtype, rows, row0, n_rows, k_rows, v_rows);
  if (st != HDF_OK || n_rows == 0) return st == HDF_OK ? ok() : st;
  const size_t el = dtype == HDF_BF16 ? 2 : 4;
  const size_t layer_bytes = size_t(n_heads) * size_t(kv_cap) * head_dim * el;
  const char* kc = kv_k ? static_cast<const char*>(kv_k) + size_t(layer) * layer_bytes : nullptr;
  const char* vc = kv_vt ? static_cast<const char*>(kv_vt) + size_t(layer) * layer_bytes : nullptr;
  const hipError_t e = hdf::launch_kv_rows(dtype == HDF_BF16, false, const_cast<char*>(kc),
                                           const_cast<char*>(vc), kv_cap, k_rows, v_rows, n_rows,
                                           rows, row0, n_heads, head_dim,
                                           reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "kv_read_rows launch");
  return ok();
}

size_t hdf_draft_block_workspace(const hdf_drafter* w, int n_seq, int B, int64_t n_new,
                                 int max_ctx) {
  if (validate_drafter(w) != HDF_OK || n_seq < 0 || B < 1 || B > 64 || n_new < 0 || max_ctx < 0)
    return 0;
  return plan_workspace(*w, n_seq, B, n_new, max_ctx).total;
}

// Both cache forms: kv_offsets (contiguous slots) or page_table (pages of 64 rows; the
// cache then holds kv_cap / 64 pages).
static hdf_status draft_block_impl(const hdf_drafter* w, int n_seq, int B, const int32_t* ctx_len,
                                   int max_ctx, const void* y_new, const int32_t* new_offsets,
                                   const int32_t* new_counts, int64_t n_new,
                                   const int32_t* kv_offsets,
                                   const int32_t* page_table, int max_pages, void* kv_k,
                                   void* kv_vt, int64_t kv_cap, const int32_t* tokens,
                                   void* hidden, void* ws, size_t ws_bytes,
                                   hdf_stream_t stream) {
  hdf_status st = validate_drafter(w);
  if (st != HDF_OK) return st;
  if (n_seq < 0) return fail(HDF_E_INVALID, "draft_block: n_seq < 0");
  if (B < 1 || B > 64) return fail(HDF_E_INVALID, "draft_block: B=%d outside [1, 64]", B);
  if (max_ctx < 0 || n_new < 0) return fail(HDF_E_INVALID, "draft_block: negative size");
  if (kv_cap < 0 || kv_cap % 64 != 0)
    return fail(HDF_E_INVALID, "draft_block: kv_cap must be a non-negative multiple of 64");
  if (kv_cap > INT32_MAX)
    return fail(HDF_E_UNSUPPORTED, "draft_block: cache rows beyond 2^31 - 1");
  if (page_table != nullptr && int64_t(max_pages) * 64 < max_ctx)
    return fail(HDF_E_INVALID, "draft_block: max_pages=%d cannot hold max_ctx=%d", max_pages,
                max_ctx);
  if (w->rope_cs != nullptr && int64_t(max_ctx) + B > w->rope_max_pos)
    return fail(HDF_E_INVALID, "draft_block: max_ctx + B exceeds the RoPE table (%d)",
                w->rope_max_pos);
  if (n_seq == 0) return ok();
  if (ctx_len == nullptr || (kv_offsets == nullptr && page_table == nullptr) ||
      tokens == nullptr || hidden == nullptr)
    return fail(HDF_E_INVALID, "draft_block: null pointer");
  if (n_new > 0 && (y_new == nullptr || new_offsets == nullptr))
    return fail(HDF_E_INVALID, "draft_block: null y_new/new_offsets with n_new > 0");
  if ((n_new > 0 || max_ctx > 0) && (kv_k == nullptr || kv_vt == nullptr || kv_cap == 0))
    return fail(HDF_E_INVALID, "draft_block: a context needs a KV cache");
  if (!aligned16(hidden) || (y_new && !aligned16(y_new)) || (kv_k && !aligned16(kv_k)) ||
      (kv_vt && !aligned16(kv_vt)))
    return fail(HDF_E_INVALID, "draft_block: tensors must be 16-byte aligned");
  const DraftPlan P = plan_workspace(*w, n_seq, B, n_new, max_ctx);
  if (ws == nullptr || ws_bytes < P.total)
    return fail(HDF_E_WORKSPACE, "draft_block: workspace of %zu bytes needed, %zu given", P.total,
                ws_bytes);
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0)
    return fail(HDF_E_INVALID, "draft_block: workspace must be 256-byte aligned");

  const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const bool bf = w->dtype == HDF_BF16;
  const int d = w->d, nh = w->n_heads, hd = w->head_dim, F = w->d_ff, L = w->n_layers;
  const int M = n_seq * B;
  const size_t el = bf ? 2 : 4;
  char* base = static_cast<char*>(ws);
  int32_t* plan_pos = reinterpret_cast<int32_t*>(base + P.plan_pos);
  int32_t* plan_row = reinterpret_cast<int32_t*>(base + P.plan_row);
  void* cbuf = base + P.c;
  float* h = reinterpret_cast<float*>(base + P.h);
  void* u = base + P.u;
  void* q = base + P.q;
  void* kb = base + P.kb;
  void* vtb = base + P.vtb;
  float* parts = reinterpret_cast<float*>(base + P.parts);
  float* part_o = reinterpret_cast<float*>(base + P.part_o);
  float* part_ml = reinterpret_cast<float*>(base + P.part_ml);
  void* attn = base + P.attn;
  void* act = base + P.act;
  const int64_t capb = int64_t(n_seq) * 64;
  const size_t layer_kv = size_t(nh) * size_t(kv_cap) * hd * el;  // bytes of one layer's k
  hipError_t e;
#define HDF_TRY(x)                                  \
  do {                                              \
    e = (x);                                        \
    if (e != hipSuccess) return hip_fail(e, #x);    \
  } while (0)

  // First kernel: context rows r0.. (position, cache row; RMSNorm(y) * ctx_norm) and,
  // with the first chunk, the block rows (h = emb[tokens]; u = RMSNorm(h) * attn_norm[0]).
  auto prep = [&](int64_t r0, int rows, bool block) {
    hdf::PrepArgs pa{};
    pa.y = y_new; pa.r0 = r0; pa.n_ctx = rows; pa.ctx_gamma = w->ctx_norm; pa.c = cbuf;
    pa.ctx_len = ctx_len; pa.new_offsets = new_offsets; pa.new_counts = new_counts;
    pa.kv_offsets = kv_offsets;
    pa.page_table = page_table; pa.max_pages = max_pages;
    pa.n_seq = n_seq; pa.plan_pos = plan_pos; pa.plan_row = plan_row;
    pa.n_blk = block ? M : 0; pa.tokens = tokens; pa.emb = w->tok_emb;
    pa.attn_gamma = w->attn_norm[0]; pa.h = h; pa.u = u;
    pa.d = d; pa.eps = w->eps;
    return hdf::launch_prep(bf, pa, s);
  };
  auto ctx_epi = [&](int l, int64_t r0, int rows, int S, const float* pp) {
    hdf::QkvEpiArgs ea{};
    ea.pkv = pp; ea.ld_kv = 2 * int64_t(d); ea.zs_kv = int64_t(rows) * 2 * d;
    ea.S = S; ea.M = rows; ea.first_part = 1;
    ea.d = d; ea.nh = nh; ea.hd = hd; ea.B = B;
    ea.ctx_len = ctx_len; ea.plan_pos = plan_pos + r0; ea.plan_row = plan_row + r0;
    ea.rope_cs = w->rope_cs;
    ea.q = nullptr;
    ea.k = static_cast<char*>(kv_k) + l * layer_kv;
    ea.vt = static_cast<char*>(kv_vt) + l * layer_kv;
    ea.cap = kv_cap;
    return ea;
  };
  auto blk_epi = [&](int S, const float* pp) {
    hdf::QkvEpiArgs ea{};
    ea.pq = pp; ea.ld_q = 3 * int64_t(d); ea.zs_q = int64_t(M) * 3 * d;
    ea.pkv = pp + d; ea.ld_kv = ea.ld_q; ea.zs_kv = ea.zs_q;
    ea.S = S; ea.M = M; ea.first_part = 0;
    ea.d = d; ea.nh = nh; ea.hd = hd; ea.B = B;
    ea.ctx_len = ctx_len; ea.rope_cs = w->rope_cs;
    ea.q = q; ea.k = kb; ea.vt = vtb; ea.cap = capb;
    return ea;
  };
  // Context rows projected in this call: with a bf16 drafter and at most kGroupRows of
  // them, each layer's context K/V share one GEMM launch and one epilogue launch with
  // the block's Q/K/V (below); otherwise K/V of every layer go into the cache here, in
  // chunks of kCtxChunk rows.
  const bool grouped = bf && n_new > 0 && n_new <= kGroupRows;
  const bool shared = kv_shared(bf, n_new, size_t(M));
  if (n_new == 0) HDF_TRY(prep(0, 0, true));
  if (grouped) HDF_TRY(prep(0, int(n_new), true));
  for (int64_t r0 = 0; !grouped && r0 < n_new; r0 += kCtxChunk) {
    const int rows = int(n_new - r0 < kCtxChunk ? n_new - r0 : kCtxChunk);
    HDF_TRY(prep(r0, rows, r0 == 0));
    for (int l = 0; l < L; ++l) {
      // Rows d..3d-1 (W_k; W_v) of the packed W_qkv: d/128 whole row groups in.
      const char* wkv = static_cast<const char*>(w->w_qkv[l]) + size_t(d) * d * el;
      const hdf::GemmPlan Sp = hdf::gemm_plan(bf, rows, 2 * d, d);
      if (bf && Sp.tn == 4 && Sp.nw == 4 && Sp.splits == 1 && (hd == 64 || hd == 128) &&
          d % 512 == 0) {
        // One K split: RoPE and the cache stores happen in the GEMM's epilogue, so the
        // fp32 rows never go through memory.
        HDF_TRY(hdf::launch_gemm_kv(cbuf, d, wkv, rows, d, hd, Sp, plan_pos + r0, plan_row + r0,
                                    w->rope_cs, static_cast<char*>(kv_k) + l * layer_kv,
                                    static_cast<char*>(kv_vt) + l * layer_kv, kv_cap, s));
      } else {
        HDF_TRY(hdf::launch_gemm_partial(bf, cbuf, d, wkv, rows, 2 * d, d, Sp, parts, s));
        HDF_TRY(hdf::launch_qkv_epilogue(bf, ctx_epi(l, r0, rows, Sp.splits, parts), s));
      }
    }
  }

  const int n_chunks = std::max(1, (max_ctx + P.chunk_len - 1) / P.chunk_len);
  // With one attention workgroup per (sequence, head), the projection epilogue of the
  // shared launch runs inside the attention kernel (no launch of its own).
  const bool fuse_epi = shared && n_chunks == 1 && B <= 16 && (hd == 64 || hd == 128);
  for (int l = 0; l < L; ++l) {
    hdf::QkvEpiArgs fused_ctx{}, fused_blk{};
    // Q, K_b, V_b with RoPE at T_s + k (and the context rows' K/V when grouped).
    if (shared) {
      const char* wkv = static_cast<const char*>(w->w_qkv[l]) + size_t(d) * d * el;
      const int rows1 = int(n_new) + M;
      const hdf::GemmPlan Sg = hdf::gemm_plan_shared(rows1, 2 * d, M, d, d);
      float* parts_kv = parts;                                       // [S][rows1][2d]
      float* parts_q = parts + size_t(Sg.splits) * rows1 * 2 * d;    // [S][M][d]
      HDF_TRY(hdf::launch_gemm_partial2(cbuf, d, wkv, rows1, 2 * d, parts_kv, u, d, w->w_qkv[l],
                                        M, d, parts_q, d, Sg, s));
      hdf::QkvEpiArgs ce = ctx_epi(l, 0, int(n_new), Sg.splits, parts_kv);
      ce.zs_kv = int64_t(rows1) * 2 * d;
      hdf::QkvEpiArgs be = blk_epi(Sg.splits, parts_q);
      be.pq = parts_q; be.ld_q = d; be.zs_q = int64_t(M) * d;
      be.pkv = parts_kv + size_t(n_new) * 2 * d; be.ld_kv = 2 * int64_t(d);
      be.zs_kv = ce.zs_kv;
      if (fuse_epi) {
        fused_ctx = ce;
        fused_blk = be;
      } else {
        HDF_TRY(hdf::launch_qkv_epilogue2(bf, ce, be, s));
      }
    } else if (grouped) {
      const char* wkv = static_cast<const char*>(w->w_qkv[l]) + size_t(d) * d * el;
      const int rows = int(n_new);
      const hdf::GemmPlan Sg = hdf::gemm_plan2(bf, rows, 2 * d, M, 3 * d, d);
      float* parts_blk = parts + size_t(Sg.splits) * rows * 2 * d;
      HDF_TRY(hdf::launch_gemm_partial2(cbuf, d, wkv, rows, 2 * d, parts, u, d, w->w_qkv[l], M,
                                        3 * d, parts_blk, d, Sg, s));
      HDF_TRY(hdf::launch_qkv_epilogue2(bf, ctx_epi(l, 0, rows, Sg.splits, parts),
                                        blk_epi(Sg.splits, parts_blk), s));
    } else {
      const hdf::GemmPlan Sqp = hdf::gemm_plan(bf, M, 3 * d, d);
      HDF_TRY(hdf::launch_gemm_partial(bf, u, d, w->w_qkv[l], M, 3 * d, d, Sqp, parts, s));
      HDF_TRY(hdf::launch_qkv_epilogue(bf, blk_epi(Sqp.splits, parts), s));
    }

    hdf::AttnArgs aa{};
    aa.q = q;
    aa.kc = static_cast<char*>(kv_k) + l * layer_kv;
    aa.vtc = static_cast<char*>(kv_vt) + l * layer_kv;
    aa.cap = kv_cap; aa.kv_offsets = kv_offsets; aa.ctx_len = ctx_len;
    aa.page_table = page_table; aa.max_pages = max_pages;
    aa.kb = kb; aa.vtb = vtb; aa.capb = capb;
    aa.n_seq = n_seq; aa.nh = nh; aa.hd = hd; aa.B = B; aa.QB = ((B + 15) / 16) * 16;
    aa.n_chunks = n_chunks; aa.chunk_len = P.chunk_len;
    aa.scale_log2 = float(1.4426950408889634 / sqrt(double(hd)));
    aa.part_o = part_o; aa.part_ml = part_ml;
    aa.fuse_epi = fuse_epi ? 1 : 0;
    aa.new_offsets = new_offsets;
    aa.epi_ctx = fused_ctx;
    aa.epi_blk = fused_blk;
    HDF_TRY(hdf::launch_attention(bf, aa, attn, s));

    // h += O Wo^T; u = RMSNorm(h) * mlp_norm.
    const hdf::GemmPlan Sop = hdf::gemm_plan(bf, M, d, d);
    const int So = Sop.splits;
    HDF_TRY(hdf::launch_gemm_partial(bf, attn, d, w->w_o[l], M, d, d, Sop, parts, s));
    HDF_TRY(hdf::launch_residual_norm(bf, parts, So, w->mlp_norm[l], w->eps, M, d, h, u, s));

    // act = SiLU(u Wg^T) * (u Wu^T); h += act Wd^T; next norm.
    const hdf::GemmPlan Sgp = hdf::gemm_plan(bf, M, 2 * F, d);
    const int Sg = Sgp.splits;
    HDF_TRY(hdf::launch_gemm_partial(bf, u, d, w->w_gate_up[l], M, 2 * F, d, Sgp, parts, s));
    HDF_TRY(hdf::launch_silu_epilogue(bf, parts, Sg, M, F, act, s));
    const hdf::GemmPlan Sdp = hdf::gemm_plan(bf, M, d, F);
    const int Sd = Sdp.splits;
    HDF_TRY(hdf::launch_gemm_partial(bf, act, F, w->w_down[l], M, d, F, Sdp, parts, s));
    const bool last = (l + 1 == L);
    HDF_TRY(hdf::launch_residual_norm(bf, parts, Sd, last ? w->final_norm : w->attn_norm[l + 1],
                                      w->eps, M, d, h, last ? hidden : u, s));
  }
#undef HDF_TRY
  return ok();
}

hdf_status hdf_draft_block(const hdf_drafter* w, int n_seq, int B, const int32_t* ctx_len,
                           int max_ctx, const void* y_new, const int32_t* new_offsets,
                           int64_t n_new, const int32_t* kv_offsets, void* kv_k, void* kv_vt,
                           int64_t kv_cap, const int32_t* tokens, void* hidden, void* ws,
                           size_t ws_bytes, hdf_stream_t stream) {
  if (n_seq > 0 && kv_offsets == nullptr) return fail(HDF_E_INVALID, "draft_block: null kv_offsets");
  return draft_block_impl(w, n_seq, B, ctx_len, max_ctx, y_new, new_offsets, nullptr, n_new,
                          kv_offsets, nullptr, 0, kv_k, kv_vt, kv_cap, tokens, hidden, ws,
                          ws_bytes, stream);
}

hdf_status hdf_draft_block_paged(const hdf_drafter* w, int n_seq, int B, const int32_t* ctx_len,
                                 int max_ctx, const void* y_new, const int32_t* new_offsets,
                                 const int32_t* new_counts, int64_t n_new,
                                 const int32_t* page_table, int max_pages,
                                 void* kv_k, void* kv_vt, int64_t kv_pages,
                                 const int32_t* tokens, void* hidden, void* ws, size_t ws_bytes,
                                 hdf_stream_t stream) {
  if (n_seq > 0 && page_table == nullptr)
    return fail(HDF_E_INVALID, "draft_block_paged: null page_table");
  if (max_pages < 0) return fail(HDF_E_INVALID, "draft_block_paged: max_pages < 0");
  if (kv_pages < 0 || kv_pages > INT32_MAX / 64)
    return fail(HDF_E_INVALID, "draft_block_paged: kv_pages=%lld outside [0, 2^25)",
                static_cast<long long>(kv_pages));
  return draft_block_impl(w, n_seq, B, ctx_len, max_ctx, y_new, new_offsets, new_counts, n_new,
                          nullptr, page_table, max_pages, kv_k, kv_vt, kv_pages * 64, tokens,
                          hidden, ws, ws_bytes, stream);
}

hdf_status hdf_advance_context(int n_seq, const int32_t* accept_len, int32_t* ctx_len,
                               int32_t* new_counts, const int32_t* next_anchor,
                               int32_t* block_tokens, int B, hdf_stream_t stream) {
  if (n_seq < 0) return fail(HDF_E_INVALID, "advance_context: n_seq < 0");
  if (n_seq > 0 && (accept_len == nullptr || ctx_len == nullptr))
    return fail(HDF_E_INVALID, "advance_context: null accept_len/ctx_len");
  if (block_tokens != nullptr) {
    if (next_anchor == nullptr)
      return fail(HDF_E_INVALID, "advance_context: block_tokens given without next_anchor");
    if (B < 1 || B > 1025) return fail(HDF_E_INVALID, "advance_context: B=%d outside [1, 1025]", B);
    if (int64_t(n_seq) * B > INT32_MAX)
      return fail(HDF_E_UNSUPPORTED, "advance_context: n_seq*B exceeds int32 offsets");
  }
  const hipError_t e = hdf::launch_advance_context(n_seq, accept_len, ctx_len, new_counts,
                                                   next_anchor, block_tokens, B,
                                                   reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "advance_context launch");
  return ok();
}

size_t hdf_packed_weight_bytes(int N, int K, hdf_dtype dtype) {
  if (N < 1 || K < 16 || K % 16 != 0 || (dtype != HDF_F32 && dtype != HDF_BF16)) return 0;
  return hdf::packed_weight_elems(N, K) * (dtype == HDF_BF16 ? 2 : 4);
}

hdf_status hdf_pack_weight(const void* W, void* W_packed, int N, int K, hdf_dtype dtype,
                           hdf_stream_t stream) {
  if (dtype != HDF_F32 && dtype != HDF_BF16) return fail(HDF_E_INVALID, "pack_weight: bad dtype");
  if (N < 1 || K < 16 || K % 16 != 0)
    return fail(HDF_E_INVALID, "pack_weight: N=%d K=%d (need N >= 1, K a positive multiple of 16)",
                N, K);
  if (W == nullptr || W_packed == nullptr) return fail(HDF_E_INVALID, "pack_weight: null pointer");
  if (W == W_packed) return fail(HDF_E_INVALID, "pack_weight: in-place packing is not supported");
  hipError_t e = hdf::launch_pack_weight(dtype == HDF_BF16, W, W_packed, N, K,
                                         reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "pack_weight launch");
  return ok();
}

size_t hdf_lm_head_workspace(int64_t M, int vocab) {
  if (M < 0 || vocab < 1) return 0;
  return size_t((M * 8 + 255) / 256 * 256);
}

hdf_status hdf_lm_head_argmax(const void* hidden, const void* W_lm, int64_t M, int d, int vocab,
                              hdf_dtype dtype, int32_t* argmax, float* max_logit, float* logits,
                              void* ws, size_t ws_bytes, hdf_stream_t stream) {
  if (dtype != HDF_F32 && dtype != HDF_BF16) return fail(HDF_E_INVALID, "lm_head: bad dtype");
  if (M < 0) return fail(HDF_E_INVALID, "lm_head: M < 0");
  if (d <= 0 || d % 64 != 0) return fail(HDF_E_INVALID, "lm_head: d=%d not a positive multiple of 64", d);
  if (vocab < 1) return fail(HDF_E_INVALID, "lm_head: vocab < 1");
  if (M == 0) return ok();
  if (hidden == nullptr || W_lm == nullptr || argmax == nullptr)
    return fail(HDF_E_INVALID, "lm_head: null pointer");
  if (!aligned16(hidden) || !aligned16(W_lm))
    return fail(HDF_E_INVALID, "lm_head: hidden and W_lm must be 16-byte aligned");
  const size_t need = hdf_lm_head_workspace(M, vocab);
  if (ws == nullptr || ws_bytes < need)
    return fail(HDF_E_WORKSPACE, "lm_head: workspace of %zu bytes needed, %zu given", need, ws_bytes);
  if ((reinterpret_cast<uintptr_t>(ws) & 7u) != 0)
    return fail(HDF_E_INVALID, "lm_head: workspace must be 8-byte aligned");
  hipError_t e = hdf::launch_lm_head(dtype == HDF_BF16, hidden, W_lm, M, d, vocab,
                                     static_cast<unsigned long long*>(ws), argmax, max_logit,
                                     logits, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "lm_head launch");
  return ok();
}

hdf_status hdf_lm_head_argmax_keys(const void* hidden, const void* W_lm, int64_t M, int d,
                                   int vocab, hdf_dtype dtype, void* ws, size_t ws_bytes,
                                   hdf_stream_t stream) {
  if (dtype != HDF_F32 && dtype != HDF_BF16) return fail(HDF_E_INVALID, "lm_head_keys: bad dtype");
  if (M < 0) return fail(HDF_E_INVALID, "lm_head_keys: M < 0");
  if (d <= 0 || d % 64 != 0)
    return fail(HDF_E_INVALID, "lm_head_keys: d=%d not a positive multiple of 64", d);
  if (vocab < 1) return fail(HDF_E_INVALID, "lm_head_keys: vocab < 1");
  if (M == 0) return ok();
  if (hidden == nullptr || W_lm == nullptr) return fail(HDF_E_INVALID, "lm_head_keys: null pointer");
  if (!aligned16(hidden) || !aligned16(W_lm))
    return fail(HDF_E_INVALID, "lm_head_keys: hidden and W_lm must be 16-byte aligned");
  const size_t need = hdf_lm_head_workspace(M, vocab);
  if (ws == nullptr || ws_bytes < need)
    return fail(HDF_E_WORKSPACE, "lm_head_keys: workspace of %zu bytes needed, %zu given", need,
                ws_bytes);
  if ((reinterpret_cast<uintptr_t>(ws) & 7u) != 0)
    return fail(HDF_E_INVALID, "lm_head_keys: workspace must be 8-byte aligned");
  hipError_t e = hdf::launch_lm_head_keys(dtype == HDF_BF16, hidden, W_lm, M, d, vocab,
                                          static_cast<unsigned long long*>(ws), nullptr,
                                          reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "lm_head_keys launch");
  return ok();
}

hdf_status hdf_accept_keys(void* ws, int n_seq, int B, int32_t* argmax, float* max_logit,
                           const int32_t* target, int32_t* accept_len, int32_t* next_anchor,
                           int32_t* commit_offsets, int32_t* commit_tokens, hdf_stream_t stream) {
  if (n_seq < 0) return fail(HDF_E_INVALID, "accept_keys: n_seq < 0");
  if (B < 1 || B > 1025) return fail(HDF_E_INVALID, "accept_keys: B=%d outside [1, 1025]", B);
  if (n_seq == 0) return ok();
  if (ws == nullptr || argmax == nullptr || target == nullptr || accept_len == nullptr ||
      next_anchor == nullptr)
    return fail(HDF_E_INVALID, "accept_keys: null pointer");
  if ((reinterpret_cast<uintptr_t>(ws) & 7u) != 0)
    return fail(HDF_E_INVALID, "accept_keys: workspace must be 8-byte aligned");
  const int64_t M = int64_t(n_seq) * B;
  if (M > INT32_MAX) return fail(HDF_E_UNSUPPORTED, "accept_keys: n_seq*B exceeds int32 offsets");
  hipError_t e = hdf::launch_accept_keys(static_cast<unsigned long long*>(ws), M, argmax,
                                         max_logit, 1, B, target, n_seq, B - 1, accept_len,
                                         next_anchor, commit_offsets, commit_tokens,
                                         reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "accept_keys launch");
  return ok();
}

// ---------------------------------------------------------- LM head without a workspace
// For callers that cannot allocate: the per-row argmax keys live in this file-scope device
// array (one copy per GPU, held until the process ends) instead of a workspace.  In host
// code `scratch` names a host-side stand-in, never the device memory: its device address
// is looked up once per device (hipGetSymbolAddress) and only that address is used.
}  // extern "C"

namespace {

constexpr int64_t kNoAllocRows = 65536;   // rows of one call; 512 KiB of keys
static __device__ __align__(256) unsigned long long scratch[kNoAllocRows];

__global__ void zero_keys_kernel(unsigned long long* keys, int64_t n) {
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * blockDim.x)
    keys[i] = 0ull;
}

std::mutex g_noalloc_mu;
unsigned long long* g_noalloc_keys[64];   // device address of `scratch` per device (set up)

// Device address of this device's `scratch`, set up on first use: address lookup, one
// clearing pass on `s` and a wait for it, so that every later call (on any stream) finds
// the keys zero, as the LM-head kernels require.
hdf_status noalloc_keys(hipStream_t s, unsigned long long** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "lm_head_argmax_noalloc: hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(HDF_E_UNSUPPORTED, "lm_head_argmax_noalloc: device %d", dev);
  std::lock_guard<std::mutex> lock(g_noalloc_mu);
  if (g_noalloc_keys[dev] == nullptr) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    e = hipStreamIsCapturing(s, &cs);
    if (e != hipSuccess) return hip_fail(e, "lm_head_argmax_noalloc: hipStreamIsCapturing");
    if (cs != hipStreamCaptureStatusNone)
      return fail(HDF_E_INVALID,
                  "lm_head_argmax_noalloc: the first call on a device sets up its key array "
                  "and must not be captured");
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol,
                      "lm_head_argmax_noalloc: hipGetSymbolAddress");
    unsigned long long* keys = static_cast<unsigned long long*>(p);
    hipLaunchKernelGGL(zero_keys_kernel, dim3(256), dim3(256), 0, s, keys, kNoAllocRows);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "lm_head_argmax_noalloc: clearing the keys");
    g_noalloc_keys[dev] = keys;
  }
  *out = g_noalloc_keys[dev];
  return HDF_OK;
}

}  // namespace

extern "C" {

hdf_status hdf_lm_head_argmax_noalloc(const void* hidden, const void* W_lm, int64_t M, int d,
                                      int vocab, hdf_dtype dtype, int32_t* argmax,
                                      float* max_logit, float* logits, hdf_stream_t stream) {
  if (dtype != HDF_F32 && dtype != HDF_BF16)
    return fail(HDF_E_INVALID, "lm_head_argmax_noalloc: bad dtype");
  if (M < 0) return fail(HDF_E_INVALID, "lm_head_argmax_noalloc: M < 0");
  if (d <= 0 || d % 64 != 0)
    return fail(HDF_E_INVALID, "lm_head_argmax_noalloc: d=%d not a positive multiple of 64", d);
  if (vocab < 1) return fail(HDF_E_INVALID, "lm_head_argmax_noalloc: vocab < 1");
  if (M > kNoAllocRows)
    return fail(HDF_E_UNSUPPORTED, "lm_head_argmax_noalloc: M=%lld above %lld rows",
                static_cast<long long>(M), static_cast<long long>(kNoAllocRows));
  if (M == 0) return ok();
  if (hidden == nullptr || W_lm == nullptr || argmax == nullptr)
    return fail(HDF_E_INVALID, "lm_head_argmax_noalloc: null pointer");
  if (!aligned16(hidden) || !aligned16(W_lm))
    return fail(HDF_E_INVALID, "lm_head_argmax_noalloc: hidden and W_lm must be 16-byte aligned");
  const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  unsigned long long* keys = nullptr;
  const hdf_status st = noalloc_keys(s, &keys);
  if (st != HDF_OK) return st;
  // The same kernels as hdf_lm_head_argmax; its finalize pass hands the keys back zeroed.
  hipError_t e = hdf::launch_lm_head(dtype == HDF_BF16, hidden, W_lm, M, d, vocab, keys, argmax,
                                     max_logit, logits, s);
  if (e != hipSuccess) return hip_fail(e, "lm_head_argmax_noalloc launch");
  return ok();
}

}  // extern "C"

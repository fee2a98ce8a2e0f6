// C ABI of libhdf: argument validation, workspace planning and kernel dispatch.
// Every check runs on the host before the first HIP call, so a rejected call
// touches neither the device nor any output.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
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

size_t hdf_draft_block_workspace(const hdf_drafter* w, int n_seq, int B, int64_t n_new,
                                 int max_ctx) {
  (void)w; (void)n_seq; (void)B; (void)n_new; (void)max_ctx;
  return 0;
}

hdf_status hdf_draft_block(const hdf_drafter* w, int n_seq, int B, const int32_t* ctx_len,
                           int max_ctx, const void* y_new, const int32_t* new_offsets,
                           int64_t n_new, const int32_t* kv_offsets, void* kv_k, void* kv_vt,
                           int64_t kv_cap, const int32_t* tokens, void* hidden, void* ws,
                           size_t ws_bytes, hdf_stream_t stream) {
  return fail(HDF_E_UNSUPPORTED, "draft_block: not built yet");
}

size_t hdf_lm_head_workspace(int64_t M, int vocab) { return 0; }

hdf_status hdf_lm_head_argmax(const void* hidden, const void* W_lm, int64_t M, int d, int vocab,
                              hdf_dtype dtype, int32_t* argmax, float* max_logit, float* logits,
                              void* ws, size_t ws_bytes, hdf_stream_t stream) {
  return fail(HDF_E_UNSUPPORTED, "lm_head_argmax: not built yet");
}

}  // extern "C"

// Internal launchers of libhdf (not exported).  Each returns the first HIP error
// it meets; argument checking is done by the C-ABI layer before any launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hdf {

// Compute units of the current device (cached per device).
int device_cu_count();

struct ReduceScalars {
  float eps, gate_scale, gate_offset;
  int per_path_norm;
};

hipError_t launch_hc_reduce(bool bf16, int m, const void* H, const void* Wg, const float* bg,
                            int64_t n_tok, int d, const ReduceScalars& sc, void* Y, float* alpha,
                            hipStream_t s);

hipError_t launch_accept(const int32_t* draft, int stride, const int32_t* target, int n_seq,
                         int K, int32_t* acc, int32_t* anchor, int32_t* offs, int32_t* toks,
                         hipStream_t s);
// The LM head's argmax finalisation and the acceptance in one workgroup: rows 0 .. M-1 of
// keys -> argmax (and max_logit, may be NULL), keys cleared; then launch_accept's work
// with draft = argmax + draft_off.
hipError_t launch_accept_keys(unsigned long long* keys, int64_t M, int32_t* argmax,
                              float* max_logit, int draft_off, int stride,
                              const int32_t* target, int n_seq, int K, int32_t* acc,
                              int32_t* anchor, int32_t* offs, int32_t* toks, hipStream_t s);

// ---------------------------------------------------------------- GEMM (gemm.hip)
constexpr int kEpiPartial = 0;  // fp32 C / split-K partials
constexpr int kEpiArgmax = 1;   // LM head: fused row argmax (+ optional fp32 logits in C)
constexpr int kEpiKV = 2;       // context K/V rows: RoPE on K, stored into the cache layouts

struct GemmArgs {
  const void* A;   // [M][lda] row-major activations
  int64_t lda;
  const void* B;   // [N][K] weights in the packed layout (hdf_pack_weight)
  int M, N, K;
  float* C;
  unsigned long long* keys;
  // Optional second problem of the same K in the same launch (partial GEMMs only):
  // its tiles follow the first problem's; C2[z][M2][N2].
  const void* A2;
  int64_t lda2;
  const void* B2;
  int M2, N2;
  float* C2;
  // kEpiKV: columns [0, kv_d) are K, [kv_d, 2 kv_d) V, in heads of hd; row r goes to
  // cache row plan_row[r] (-1: not stored) at position plan_pos[r].
  const int32_t* plan_pos;
  const int32_t* plan_row;
  const float* rope_cs;   // [pos][hd/2][2] or NULL
  void* kc;               // [nh][cap][hd] key tiles of the layer
  void* vtc;              // [nh][hd][cap] value tiles of the layer
  int64_t cap;
  int kv_d, hd;
};

int gemm_k_align(bool bf16);                       // K must be a multiple of this
// Launch shape of a partial-sum GEMM: waves per workgroup (32 columns each; bf16:
// 4, 6 or 8) and the number of K splits.
struct GemmPlan {
  int nw, splits;
  int tn = 1;       // 32-column blocks per wave (4 for the matrix-core bound shapes)
  bool nt = true;   // one-block waves: weights streamed past the caches
};
GemmPlan gemm_plan(bool bf16, int M, int N, int K);
// Plan of two problems of the same K launched together (M2 = 0: one problem).
GemmPlan gemm_plan2(bool bf16, int M, int N, int M2, int N2, int K);
// Two problems of the same K in one launch where the first one's row tiles (up to 256
// rows) share weight columns: weights fetched through L2 (8 waves of one block).
GemmPlan gemm_plan_shared(int M, int N, int M2, int N2, int K);
size_t packed_weight_elems(int N, int K);          // rows rounded up to 128
hipError_t launch_pack_weight(bool bf16, const void* src, void* dst, int N, int K, hipStream_t s);
// C[z][M][N] (fp32) = A[M][K] . W[N][K]^T over the z-th of `splits` K ranges; W packed.
hipError_t launch_gemm_partial(bool bf16, const void* A, int64_t lda, const void* B, int M, int N,
                               int K, GemmPlan plan, float* C, hipStream_t s);
// Two bf16 problems of the same K in one launch (one wave of workgroups for both).
hipError_t launch_gemm_partial2(const void* A, int64_t lda, const void* B, int M, int N,
                                float* C, const void* A2, int64_t lda2, const void* B2, int M2,
                                int N2, float* C2, int K, GemmPlan plan, hipStream_t s);
// Context K/V projection straight into the cache: A [M][d] normed context rows (bf16),
// B the packed W_k; W_v rows (2d x d), RoPE on K at plan_pos, stores at plan_row.  Only
// for plans of one K split and two-block waves and d % 512 == 0 (returns
// hipErrorInvalidValue otherwise).
hipError_t launch_gemm_kv(const void* A, int64_t lda, const void* B, int M, int d, int hd,
                          GemmPlan plan, const int32_t* plan_pos, const int32_t* plan_row,
                          const float* rope_cs, void* kc, void* vtc, int64_t cap, hipStream_t s);
// keys: M 64-bit scratch words.  logits may be NULL.
hipError_t launch_lm_head(bool bf16, const void* hidden, const void* W, int64_t M, int d, int V,
                          unsigned long long* keys, int32_t* argmax, float* max_logit,
                          float* logits, hipStream_t s);
// The GEMM of launch_lm_head only: the keys are left folded, not finalised or cleared.
hipError_t launch_lm_head_keys(bool bf16, const void* hidden, const void* W, int64_t M, int d,
                               int V, unsigned long long* keys, float* logits, hipStream_t s);
// Tile shape of the LM head's bf16 kernel for M rows (waves, blocks per wave).
GemmPlan lm_head_plan(int64_t M);

// ---------------------------------------------------------------- row-wise (rowwise.hip)
struct QkvEpiArgs {
  // Split-K partials of the rows' projections: split z of row r, column j of Q at
  // pq[z*zs_q + r*ld_q + j], of K at pkv[z*zs_kv + r*ld_kv + j], of V at the same + d.
  const float* pq;
  int64_t ld_q, zs_q;
  const float* pkv;
  int64_t ld_kv, zs_kv;
  int S, M;
  int first_part;        // 0: Q, K, V (block rows); 1: K, V only (context rows)
  int d, nh, hd, B;
  const int32_t* ctx_len;   // block rows: position = ctx_len[s] + k
  const int32_t* plan_pos;  // context rows: position and cache row per row (-1: not a new row)
  const int32_t* plan_row;
  const float* rope_cs;     // [pos][hd/2][2] or NULL
  void* q;                  // block rows: [n_seq][nh][B][hd]
  void* k;                  // [nh][cap][hd]
  void* vt;                 // [nh][hd][cap]
  int64_t cap;
};

struct PrepArgs {
  // context rows r0 .. r0+n_ctx-1 of y_new: plan_pos/plan_row[r] and c[r - r0]
  const void* y;
  int64_t r0;
  int n_ctx;
  const float* ctx_gamma;
  void* c;
  const int32_t* ctx_len;
  const int32_t* new_offsets;
  const int32_t* new_counts;   // [n_seq] rows of each sequence that are new, or NULL (all)
  const int32_t* kv_offsets;
  const int32_t* page_table;   // paged cache: [n_seq][max_pages] page of each 64-row tile, or NULL
  int max_pages;
  int n_seq;
  int32_t* plan_pos;
  int32_t* plan_row;
  // block rows (n_blk of them, or none): h = float(emb[tokens]), u = RMSNorm(h) * attn_gamma
  int n_blk;
  const int32_t* tokens;
  const void* emb;
  const float* attn_gamma;
  float* h;
  void* u;
  int d;
  float eps;
};
hipError_t launch_prep(bool bf16, const PrepArgs& a, hipStream_t s);
// ctx_len[s] += accept_len[s] + 1; new_counts[s] = accept_len[s] + 1 (new_counts may be NULL)
hipError_t launch_advance_context(int n_seq, const int32_t* accept_len, int32_t* ctx_len,
                                  int32_t* new_counts, const int32_t* next_anchor,
                                  int32_t* block_tokens, int B, hipStream_t s);
// h += sum_z parts[z]; u = RMSNorm(h) * gamma
hipError_t launch_residual_norm(bool bf16, const float* parts, int S, const float* gamma, float eps,
                                int64_t rows, int d, float* h, void* u, hipStream_t s);
hipError_t launch_qkv_epilogue(bool bf16, const QkvEpiArgs& a, hipStream_t s);
// Two epilogues (context rows, block rows) in one launch.
hipError_t launch_qkv_epilogue2(bool bf16, const QkvEpiArgs& a, const QkvEpiArgs& b,
                                hipStream_t s);
// out[M][N] = sum_z parts[z][M][N] (+ bias[N], may be NULL), rounded to the dtype; N % 4 == 0
hipError_t launch_split_sum_store(bool bf16, const float* parts, int S, int64_t M, int N,
                                  const float* bias, void* out, hipStream_t s);
// act = SiLU(gate) * up from parts [S][M][2F] (gate columns first)
hipError_t launch_silu_epilogue(bool bf16, const float* parts, int S, int64_t M, int F, void* act,
                                hipStream_t s);

// ---------------------------------------------------------------- sampling (sample.hip)
// Workspace bytes of launch_row_softmax for `rows` rows of V columns.
size_t sample_parts_bytes(int64_t rows, int V);
// Per row of logits [rows][ld]: lse = logsumexp(logits * inv_t) and, with `sample`, a
// token drawn from softmax(logits * inv_t) (Philox4x64-10 Gumbel noise); tokens/lse may
// be NULL.
hipError_t launch_row_softmax(const float* logits, int64_t rows, int V, int64_t ld, float inv_t,
                              bool sample, uint64_t seed, uint64_t stream, int32_t* tokens,
                              float* lse, void* part_ws, hipStream_t s);
size_t accept_sample_ws_bytes(int n_seq, int K, int V);
hipError_t launch_accept_sample(const int32_t* draft, int draft_stride, const float* draft_logits,
                                const float* draft_lse, int64_t ld, const float* target_logits,
                                int n_seq, int K, int V, float inv_t, uint64_t seed,
                                uint64_t stream, int32_t* acc, int32_t* anchor, int32_t* offs,
                                int32_t* toks, void* ws, hipStream_t s);

// ---------------------------------------------------------------- KL forward (kl.hip)
size_t kl_ws_bytes(int n_seq, int B, int P, int d, int V, bool bf16);
hipError_t launch_kl_forward(bool bf16, const void* H_pos, int m, const float* gamma, float eps,
                             const void* W_lm, int d, int V, const float* zl, int64_t ld, int B,
                             const int32_t* labels, int n_seq, int P, float T, float alpha,
                             float* kl, float* ce, float* loss, void* ws, hipStream_t s);

// ---------------------------------------------------------------- cache rows (kv_rows.hip)
// write: k/v rows [n][nh*hd] -> cache tiles of one layer (kc, vc); otherwise the reverse.
// Cache row of input row i: rows[i], or row0 + i when rows is NULL; rows outside [0, cap)
// are skipped (write) or read as zeros.  A NULL pair (kc/krows or vc/vrows) is skipped.
hipError_t launch_kv_rows(bool bf16, bool write, void* kc, void* vc, int64_t cap, void* krows,
                          void* vrows, int64_t n, const int32_t* rows, int64_t row0, int nh,
                          int hd, hipStream_t s);

// ---------------------------------------------------------------- attention (attention.hip)
struct AttnArgs {
  const void* q;             // [n_seq][nh][B][hd]
  const void* kc;            // layer's context keys   [nh][cap][hd]
  const void* vtc;           // layer's context values [nh][hd][cap]
  int64_t cap;
  const int32_t* kv_offsets; // [n_seq+1] cache slot of each sequence (contiguous cache)
  const int32_t* page_table; // [n_seq][max_pages] page of each 64-row tile (paged cache), or NULL
  int max_pages;
  const int32_t* ctx_len;    // [n_seq]
  const void* kb;            // block keys   [nh][capb][hd], slot s at row 64*s
  const void* vtb;           // block values [nh][hd][capb]
  int64_t capb;
  int n_seq, nh, hd, B, QB;  // QB = B rounded up to 16
  int n_chunks, chunk_len;   // context chunks of the grid (chunk_len % 64 == 0)
  float scale_log2;          // log2(e) / sqrt(hd)
  float* part_o;             // [n_seq][nh][n_chunks+1][QB][hd]
  float* part_ml;            // [n_seq][nh][n_chunks+1][QB][2]
  // Projection epilogue run by the attention kernel itself (bf16, one workgroup per
  // (sequence, head): n_chunks == 1, B <= 16): the workgroup of (s, h) first finishes head
  // h of the context rows new_offsets[s] .. new_offsets[s+1]-1 of epi_ctx and of the block
  // rows of s (epi_blk), then attends.  fuse_epi = 0: the epilogue ran before.
  int fuse_epi;
  const int32_t* new_offsets;  // [n_seq+1]
  QkvEpiArgs epi_ctx, epi_blk;
  int n_cus;                   // set by launch_attention (the dispatch order uses it)
};

// Longest context chunk of one bf16 attention workgroup.
constexpr int kAttnMaxChunk = 16384;

// out: [n_seq*B][nh*hd] attention output rows in the working dtype.
hipError_t launch_attention(bool bf16, const AttnArgs& a, void* out, hipStream_t s);

}  // namespace hdf

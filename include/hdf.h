/*
 * hdf.h -- C ABI of the HyperDFlash drafter-step library (libhdf.so), MI355X / gfx950.
 *
 * One decode round of HyperDFlash drafting (arxiv 2606.26744):
 *   1. hdf_hc_reduce       gated residual reducer, Eq. (1) of Sec. 2.2
 *      (hdf_fc_reduce      the generic dense fc reducer, the fallback of Sec. 2.2)
 *   2. hdf_draft_block     one-pass DFlash block drafter over the reduced context
 *                          (Sec. 1, Sec. 2.1; slot alignment of Sec. 2.3)
 *   3. hdf_lm_head_argmax  draft logits z_k and greedy draft tokens (Sec. 2.3)
 *   4. hdf_accept          greedy verification: longest agreeing prefix (Sec. 1, Sec. 3.4)
 *      (hdf_sample_tokens, hdf_accept_sample: the same at temperature T > 0;
 *       hdf_advance_context: the committed positions become the next round's context)
 *
 * Conventions shared by every call:
 *   - Tensor arguments are DEVICE pointers unless marked "host".  Tensors are dense,
 *     row-major, caller-allocated and caller-owned.  The library never allocates or
 *     frees device memory; scratch space comes in through a caller-supplied workspace
 *     whose size the matching *_workspace query returns.
 *   - Calls are asynchronous: they validate, enqueue kernels on `stream` and return.
 *     Outputs are valid once the stream has been synchronised.
 *   - Errors are status codes; nothing throws across the ABI.  Argument errors are
 *     detected on the host before anything is enqueued (HDF_E_INVALID,
 *     HDF_E_UNSUPPORTED, HDF_E_WORKSPACE) and leave every output untouched.  A HIP
 *     launch failure returns HDF_E_HIP.  hdf_last_error() describes the last failure
 *     of the calling thread.
 *   - Values that live in device memory (offsets, lengths, token ids) are
 *     preconditions, not checked: offsets monotone, lengths within the stated
 *     bounds, token ids in [0, vocab).
 *   - Outputs never alias inputs.  Calls on different streams are independent;
 *     the library keeps no state between calls.
 *   - bf16 data is IEEE binary32 truncated to its upper 16 bits (1-8-7); conversions
 *     to bf16 round to nearest, ties to even.  Inputs must be finite.
 */
#ifndef HDF_H_
#define HDF_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* hdf_stream_t; /* a hipStream_t; NULL = the null stream */

typedef enum {
  HDF_OK = 0,
  HDF_E_INVALID = 1,     /* null pointer, negative size, inconsistent shapes        */
  HDF_E_UNSUPPORTED = 2, /* a valid request outside what the kernels implement      */
  HDF_E_WORKSPACE = 3,   /* workspace missing or smaller than the *_workspace size  */
  HDF_E_HIP = 4          /* a HIP runtime call or kernel launch failed               */
} hdf_status;

typedef enum { HDF_F32 = 0, HDF_BF16 = 1 } hdf_dtype;

/* Text of the last failure on the calling thread ("" if none).  Valid until the
 * thread's next hdf_* call. */
const char* hdf_last_error(void);
/* Library ABI version: major * 10000 + minor * 100 + patch. */
int hdf_version(void);

/* ------------------------------------------------------------------------------
 * 1. Gated residual reducer -- Eq. (1), Sec. 2.2.
 *
 * For every token t of an m-path Hyper-Connection residual H_t (m rows of width d):
 *     x      = vec(H_t)                         path-major: x[j*d + c] = H[t][j][c]
 *     r      = 1 / sqrt(mean(x^2) + eps)        mean over all m*d entries
 *     z_j    = gate_scale * r * (W_g[j] . x) + b_g[j]     (= W_g RMSNorm(x) + b)
 *     alpha_j= sigmoid(z_j) + gate_offset       independent per-path gates
 *     P_j    = H_t[j], or H_t[j] / sqrt(mean_c(H_t[j][c]^2) + eps) if per_path_norm
 *     Y_t    = sum_j alpha_j P_j                summed in ascending j
 * The paper's W_f (m x m*d) is W_g here, one contiguous row per gate.  gate_scale,
 * gate_offset stand for the scale factor and small offset of the target's hc_head
 * implementation (Sec. 2.2), which Eq. (1) abstracts away; per_path_norm is the
 * drafter-side per-path RMSNorm Sec. 2.2 mentions.
 *
 * Arithmetic is fp32; Y is written in `dtype` (rounded once).
 * ----------------------------------------------------------------------------*/
typedef struct {
  float eps;          /* RMSNorm epsilon (> 0); default 1e-6        */
  float gate_scale;   /* default 1                                   */
  float gate_offset;  /* default 0                                   */
  int per_path_norm;  /* 0 (default) or 1                            */
} hdf_reduce_params;

/* H     [n_tok][m][d]  dtype
 * W_g   [m][m*d]       dtype
 * b_g   [m]            fp32
 * params  host pointer or NULL for the defaults
 * Y     [n_tok][d]     dtype (out)
 * alpha [n_tok][m]     fp32 (out, may be NULL)
 * Limits: 1 <= m <= 8; d % 8 == 0 (bf16) or d % 4 == 0 (fp32); d <= 8192 (bf16) or
 * d <= 4096 (fp32); n_tok >= 0 (0 is a no-op).  Pointers 16-byte aligned. */
hdf_status hdf_hc_reduce(const void* H, const void* W_g, const float* b_g, int64_t n_tok,
                         int m, int d, hdf_dtype dtype, const hdf_reduce_params* params,
                         void* Y, float* alpha, hdf_stream_t stream);

/* ------------------------------------------------------------------------------
 * 1b. Generic fc reducer, the fallback path collapse (Sec. 2.2, Table 1): a static
 * dense projection of the flattened multi-path residual,
 *     y_t = W_fc vec(H_t) (+ b_fc),   vec path-major (index j*d + c),
 * with no normalisation (about 67M parameters at m = 4, d = 4096, against the gated
 * reducer's 65K).  Accumulation in fp32, Y rounded to `dtype`.
 * ----------------------------------------------------------------------------*/
/* Workspace bytes of hdf_fc_reduce (0 on invalid arguments). */
size_t hdf_fc_reduce_workspace(int64_t n_tok, int m, int d, hdf_dtype dtype);
/* H     [n_tok][m][d] dtype
 * W_fc  [d][m*d] dtype, packed (hdf_pack_weight with N = d, K = m*d)
 * b_fc  [d] fp32 or NULL (no bias)
 * Y     [n_tok][d] dtype (out)
 * ws, ws_bytes  at least hdf_fc_reduce_workspace(...) bytes, 256-byte aligned; its
 *       contents on entry do not matter.
 * Limits: 1 <= m <= 8; d % 4 == 0; m*d a multiple of 64 (bf16) or 16 (fp32);
 *         0 <= n_tok < 2^31 (0 is a no-op).  H, W_fc, Y 16-byte aligned. */
hdf_status hdf_fc_reduce(const void* H, const void* W_fc, const float* b_fc, int64_t n_tok, int m,
                         int d, hdf_dtype dtype, void* Y, void* ws, size_t ws_bytes,
                         hdf_stream_t stream);

/* ------------------------------------------------------------------------------
 * Weight layout of every projection and of the LM head.
 *
 * A weight W[N][K] (N outputs, K inputs; PyTorch's [out][in]) is passed in the
 * MFMA-packed layout: element (n, k) sits at
 *     (((n/128) * (K/16) + k/16) * 4 + (n%128)/32) * 512
 *       + ((n%32) + 32*((k%16)/8)) * 8  +  k%8
 * so each block of 32 rows x 16 columns is 512 contiguous elements in the order the
 * 64 lanes of a wave hold a matrix-core operand, the four 32-row blocks of a 128-row
 * group sit side by side for every 16 columns, and the groups follow each other
 * along K.  Rows are padded with zeros to a multiple of 128.  Pack once when the
 * weights are loaded.  Sub-matrices of whole 128-row groups are plain offsets into a
 * packed matrix (rows r..r+n of W start at element r*K when r%128 == 0).
 * ----------------------------------------------------------------------------*/
/* Bytes of the packed copy of an N x K weight (0 on invalid arguments). */
size_t hdf_packed_weight_bytes(int N, int K, hdf_dtype dtype);
/* W [N][K] row-major (device) -> W_packed (device, hdf_packed_weight_bytes bytes).
 * Limits: N >= 1, K a positive multiple of 16; W_packed must not overlap W. */
hdf_status hdf_pack_weight(const void* W, void* W_packed, int N, int K, hdf_dtype dtype,
                           hdf_stream_t stream);

/* ------------------------------------------------------------------------------
 * 2. One-pass block drafter (Sec. 1, Sec. 2.1, Sec. 2.3).
 *
 * Each sequence s has a context of T_s positions whose reduced states were
 * produced by the reducer.  The drafter block holds B slots at positions
 * T_s .. T_s+B-1: slot 0 is the accepted anchor token, slots 1..B-1 hold mask
 * tokens (the anchor-plus-mask block input format, Sec. 2.1); slot k's final
 * state predicts the token at position T_s + k (Sec. 2.3).
 *
 * Layer reading (the paper fixes the interface, not the layers): pre-norm
 * transformer layers, multi-head attention with n_heads * head_dim = d, a
 * SiLU-gated MLP of width d_ff, no biases, RMSNorms with fp32 weights.
 *   context row i:  c = RMSNorm(y_i) * ctx_norm
 *                   per layer K_i = RoPE(c Wk^T, pos i), V_i = c Wv^T   -> KV cache
 *   block:          h = tok_emb[tokens]                      (fp32 residual stream)
 *   per layer:      u = RMSNorm(h) * attn_norm
 *                   Q,Kb,Vb = u Wq^T, u Wk^T, u Wv^T; RoPE on Q, Kb at T_s + k
 *                   every block query attends to all T_s context keys and all B
 *                   block keys, no mask (bidirectional in the block), softmax scale
 *                   1/sqrt(head_dim)
 *                   h += O Wo^T;  v = RMSNorm(h) * mlp_norm
 *                   h += (SiLU(v Wgate^T) * (v Wup^T)) Wdown^T
 *   output:         hidden = RMSNorm(h) * final_norm
 * RoPE is rotate-half over the whole head: pair (i, i + head_dim/2) turns by
 * pos * theta^(-2i/head_dim), with cos/sin taken from `rope_cs`.
 * Stored intermediates (c, K, V, u, Q, attention output, v, SiLU*up, hidden) are
 * rounded to `dtype`; h and all accumulations are fp32.
 * ----------------------------------------------------------------------------*/
typedef struct {
  int n_layers, d, n_heads, head_dim, d_ff, vocab;
  hdf_dtype dtype;
  float eps;                     /* RMSNorm epsilon for every norm (> 0)                */
  const void* tok_emb;           /* [vocab][d] row-major (rows are gathered by token id) */
  const float* ctx_norm;         /* [d] or NULL (all ones)                              */
  const float* const* attn_norm; /* host array [n_layers] of device [d] (entries NULL = ones) */
  /* Projection weights, each packed (hdf_pack_weight):                                */
  const void* const* w_qkv;      /* host array [n_layers] of device [3d][d]: Wq;Wk;Wv rows */
  const void* const* w_o;        /* host array [n_layers] of device [d][d]              */
  const float* const* mlp_norm;  /* host array [n_layers] of device [d] (NULL = ones)   */
  const void* const* w_gate_up;  /* host array [n_layers] of device [2*d_ff][d]: gate;up */
  const void* const* w_down;     /* host array [n_layers] of device [d][d_ff]           */
  const float* final_norm;       /* [d] or NULL                                         */
  const float* rope_cs;          /* [rope_max_pos][head_dim/2][2] (cos, sin) fp32, or
                                    NULL for no rotary embedding; see hdf_rope_table    */
  int rope_max_pos;              /* positions 0 .. rope_max_pos-1 are tabulated         */
} hdf_drafter;

/* Fills a HOST buffer out[n_pos][head_dim/2][2] with cos and sin of
 * pos * theta^(-2i/head_dim), evaluated in double precision and rounded to fp32.
 * The caller copies it to the device once and passes it as hdf_drafter.rope_cs. */
hdf_status hdf_rope_table(float* out_host, int n_pos, int head_dim, double theta);

/* KV cache, caller-owned, `dtype` elements, keys and values in two arrays of the same
 * shape [n_layers][n_heads][kv_cap/64][64*head_dim]: the rows (positions) of one head
 * are grouped in tiles of 64, and each tile holds its 64 x head_dim keys (values) in
 * the order in which the attention kernel's 64 lanes take their matrix-core operands,
 * so that every operand fetch is one contiguous 1 KB access.  With r the row inside
 * the tile and i the dim:
 *   keys:   ((st*(head_dim/32) + i/32)*64 + 16*((i/8)%4) + ql)*8 + i%8,
 *           st = 2*(r/32) + (r/4)%2,  ql = 4*((r%32)/8) + r%4
 *   values: (((r/32)*(head_dim/16) + i/16)*64 + 16*((r/8)%4) + i%16)*8 + r%8
 * Keys are stored after RoPE.  Context position i of sequence s lives at cache row
 * kv_offsets[s] + i.  Every kv_offsets[s] must be a multiple of 64 and
 * kv_offsets[s+1] - kv_offsets[s] >= T_s rounded up to a multiple of 64 (so 64-row
 * tiles never leave a sequence's slot); kv_cap is a multiple of 64 and
 * >= kv_offsets[n_seq].  Rows past T_s inside a slot are never used. */
size_t hdf_kv_cache_bytes(const hdf_drafter* w, int64_t kv_cap); /* bytes of k (= of vt) */

/* Row-major keys and values to and from the cache layout above, one layer at a time:
 * row i of k_rows / v_rows ([n_rows][n_heads*head_dim], keys after RoPE, head h in
 * columns h*head_dim ..) is cache row rows[i] (device int32 [n_rows]), or row0 + i when
 * rows is NULL.  With a paged cache (hdf_draft_block_paged) position p of a sequence is
 * row page_table[s][p/64]*64 + p%64.  These let a caller that holds keys and values in
 * row-major form (its own prefill, a cache saved elsewhere) fill or inspect a cache
 * without reproducing the tile layout, which is this library's own (the attention
 * kernel's operand order, not a layout the paper prescribes).
 * kv_k, kv_vt  the whole cache [n_layers][n_heads][kv_cap/64][64*head_dim]; `layer`
 *              selects the layer (0 <= layer < n_layers, not checked against the cache)
 * Either pair (kv_k with k_rows, kv_vt with v_rows) may be NULL to skip keys or values,
 * not both.  Writes touch only the cache rows named; reads of a row outside [0, kv_cap)
 * (from `rows`) return zeros and writes to one are skipped.
 * Limits: head_dim in {64, 128}; kv_cap a positive multiple of 64 below 2^31;
 *         0 <= n_rows < 2^31 (0 is a no-op); without `rows`, row0 + n_rows <= kv_cap;
 *         the tensors 16-byte aligned.  Rows named twice in one write: either wins. */
hdf_status hdf_kv_write_rows(const void* k_rows, const void* v_rows, int64_t n_rows,
                             const int32_t* rows, int64_t row0, int layer, int n_heads,
                             int head_dim, hdf_dtype dtype, void* kv_k, void* kv_vt,
                             int64_t kv_cap, hdf_stream_t stream);
hdf_status hdf_kv_read_rows(const void* kv_k, const void* kv_vt, int64_t kv_cap, int layer,
                            int n_heads, int head_dim, hdf_dtype dtype, const int32_t* rows,
                            int64_t row0, int64_t n_rows, void* k_rows, void* v_rows,
                            hdf_stream_t stream);

/* Workspace bytes hdf_draft_block needs for these sizes (0 on invalid arguments). */
size_t hdf_draft_block_workspace(const hdf_drafter* w, int n_seq, int B, int64_t n_new,
                                 int max_ctx);

/* n_seq       sequences (0 is a no-op), B block slots (1..64)
 * ctx_len     [n_seq] int32: T_s, the context length of sequence s (1..max_ctx)
 * max_ctx     host: an upper bound on every T_s (sizes the attention grid)
 * y_new       [n_new][d] dtype: reduced states of the context rows projected in this
 *             call, packed by sequence
 * new_offsets [n_seq+1] int32: rows new_offsets[s] .. new_offsets[s+1]-1 of y_new
 *             belong to sequence s and are its LAST context positions
 *             (T_s - n_s .. T_s - 1 with n_s = new_offsets[s+1] - new_offsets[s]);
 *             new_offsets[0] = 0, new_offsets[n_seq] = n_new.  A cold step passes the
 *             whole context (n_s = T_s); a warm step only the newest rows, the
 *             earlier rows' keys/values being already in the cache.
 * n_new       host: total new rows (>= 0)
 * kv_offsets  [n_seq+1] int32: cache slot of each sequence (see above)
 * kv_k, kv_vt, kv_cap  the KV cache; rows of the new positions are written
 * tokens      [n_seq][B] int32: anchor then mask ids
 * hidden      [n_seq*B][d] dtype (out): final-normed block states, row s*B + k
 * ws, ws_bytes  workspace of at least hdf_draft_block_workspace(...) bytes, 256-byte
 *             aligned; its contents on entry do not matter.
 * Limits: head_dim in {64, 128}; n_heads * head_dim == d; d % 128 == 0;
 *         d_ff % 64 == 0; max_ctx + B <= rope_max_pos when rope_cs is given. */
hdf_status hdf_draft_block(const hdf_drafter* w, int n_seq, int B, const int32_t* ctx_len,
                           int max_ctx, const void* y_new, const int32_t* new_offsets,
                           int64_t n_new, const int32_t* kv_offsets, void* kv_k, void* kv_vt,
                           int64_t kv_cap, const int32_t* tokens, void* hidden, void* ws,
                           size_t ws_bytes, hdf_stream_t stream);

/* Paged KV cache: the same drafter step over a cache whose rows are a pool of
 * kv_pages pages of 64 rows, [n_layers][n_heads][kv_pages][64*head_dim] with the tile
 * layout above (one page = one tile).  Context position i of sequence s lives in row
 * i%64 of page page_table[s*max_pages + i/64], so a sequence grows by taking any free
 * page and no sequence needs a contiguous slot (the serving loop that appends the
 * n_s + 1 accepted positions of every round, Sec. 1).
 * page_table  [n_seq][max_pages] int32 (device): pages 0 .. ceil(T_s/64)-1 of every
 *             sequence must be valid page indices in [0, kv_pages) and no page may be
 *             listed twice among the pages written by this call (new rows), nor be a
 *             page of another sequence (pages shared between sequences, such as a common
 *             prefix, are read-only); entries past a sequence's last page are not read.
 *             Not checked on the device.
 * max_pages   host: row stride of page_table; max_pages * 64 >= max_ctx
 * kv_pages    host: pages in the pool (kv_pages * 64 < 2^31)
 * new_counts  [n_seq] int32 (device) or NULL.  NULL: every row new_offsets[s] ..
 *             new_offsets[s+1]-1 is new, as in hdf_draft_block.  Given: only the first
 *             min(new_counts[s], new_offsets[s+1] - new_offsets[s]) rows of sequence s are
 *             new, its positions T_s - n_s .. T_s - 1 with that n_s; its other rows are
 *             read but neither projected into the cache nor used.  This lets a chained
 *             decode loop size the call for an upper bound (B rows per sequence, every
 *             sequence committing at most B positions a round) while the counts come
 *             from the device (hdf_advance_context after hdf_accept), so the host never
 *             waits for the accepted lengths.  A row whose position would fall outside
 *             [0, max_pages * 64) is skipped likewise.
 * Every other argument and limit is that of hdf_draft_block. */
hdf_status hdf_draft_block_paged(const hdf_drafter* w, int n_seq, int B, const int32_t* ctx_len,
                                 int max_ctx, const void* y_new, const int32_t* new_offsets,
                                 const int32_t* new_counts, int64_t n_new,
                                 const int32_t* page_table, int max_pages,
                                 void* kv_k, void* kv_vt, int64_t kv_pages,
                                 const int32_t* tokens, void* hidden, void* ws, size_t ws_bytes,
                                 hdf_stream_t stream);

/* ------------------------------------------------------------------------------
 * 3. LM head with fused greedy argmax (Sec. 2.3: z_k are the draft logits).
 *
 * logits[r][v] = sum_c hidden[r][c] * W_lm[v][c]   (fp32 accumulation)
 * argmax[r]    = the smallest v with logits[r][v] == max_v logits[r][v]
 * The full logits matrix is never stored unless `logits` is given.
 * ----------------------------------------------------------------------------*/
size_t hdf_lm_head_workspace(int64_t M, int vocab);

/* hidden    [M][d] dtype; W_lm [vocab][d] dtype, packed (hdf_pack_weight)
 * argmax    [M] int32 (out)
 * max_logit [M] fp32 (out, may be NULL)
 * logits    [M][vocab] fp32 (out, may be NULL; for tests)
 * ws, ws_bytes  at least hdf_lm_head_workspace(M, vocab) bytes, 8-byte aligned,
 *           holding zeros before its first use (allocate it zero-filled); every call
 *           hands it back zeroed (it holds the per-row argmax keys the kernels fold
 *           into), so it can be reused as is.  Calls sharing a workspace must not run
 *           concurrently.
 * Limits: d % 64 == 0; 1 <= vocab < 2^31; M >= 0. */
hdf_status hdf_lm_head_argmax(const void* hidden, const void* W_lm, int64_t M, int d, int vocab,
                              hdf_dtype dtype, int32_t* argmax, float* max_logit, float* logits,
                              void* ws, size_t ws_bytes, hdf_stream_t stream);

/* The GEMM of hdf_lm_head_argmax alone (Sec. 2.3), for the greedy step that hands its
 * argmax straight to the acceptance (hdf_accept_keys): every row's (maximum, lowest
 * column) is folded into the workspace as a packed 64-bit key and left there; nothing is
 * written to argmax or max_logit and the workspace is not cleared.  The next call on the
 * same workspace must be hdf_accept_keys over the same rows (M = n_seq * B), which turns
 * the keys into argmax / max_logit and hands the workspace back zeroed.
 * hidden, W_lm, M, d, vocab, dtype, ws, ws_bytes and limits: as hdf_lm_head_argmax. */
hdf_status hdf_lm_head_argmax_keys(const void* hidden, const void* W_lm, int64_t M, int d,
                                   int vocab, hdf_dtype dtype, void* ws, size_t ws_bytes,
                                   hdf_stream_t stream);

/* hdf_lm_head_argmax for callers that cannot allocate device memory (code under HIP
 * graph capture, serving loops or harnesses that forbid allocation): the same kernels and
 * results, with no workspace argument.  The per-row argmax keys live in a library-owned
 * device array of 65536 64-bit words (512 KiB), one per GPU, held until the process
 * ends; the call allocates nothing.
 * Every call on one GPU shares that array and hands it back zeroed: calls that overlap on
 * one GPU (other streams, other threads) race and must be serialised by the caller.  The
 * first call on each GPU sets the array up (finds its address, clears it and waits for the
 * clear on `stream`), so it must not be made while `stream` is being captured
 * (HDF_E_INVALID).
 * Arguments, outputs and limits as hdf_lm_head_argmax, and M <= 65536
 * (HDF_E_UNSUPPORTED above). */
hdf_status hdf_lm_head_argmax_noalloc(const void* hidden, const void* W_lm, int64_t M, int d,
                                      int vocab, hdf_dtype dtype, int32_t* argmax,
                                      float* max_logit, float* logits, hdf_stream_t stream);

/* ------------------------------------------------------------------------------
 * 4. Greedy acceptance (Sec. 1: the target keeps the longest draft prefix that
 * agrees with its own tokens; Sec. 3.4: tau, the mean accepted length).
 *
 * For sequence s with drafts d_i = draft[s*draft_stride + i] (i = 0..K-1) and target
 * tokens t_i = target[s*(K+1) + i] (i = 0..K):
 *     n_s = max { j <= K : d_i == t_i for all i < j }
 *     accept_len[s]  = n_s                 (tau of this round is n_s + 1)
 *     next_anchor[s] = t_{n_s}             (the target's own next token)
 *     commit_offsets = exclusive prefix sum of (n_s + 1), n_seq+1 entries
 *     commit_tokens[commit_offsets[s] + i] = t_i for i = 0..n_s
 * With the LM head's argmax array of a block (row s*B + k is slot k), the drafts
 * are slots 1..B-1: draft = argmax + 1, draft_stride = B, K = B - 1.
 * ----------------------------------------------------------------------------*/
/* draft   int32, row s at draft + s*draft_stride, K entries (draft_stride >= K)
 * target  [n_seq][K+1] int32
 * accept_len, next_anchor  [n_seq] int32 (out)
 * commit_offsets [n_seq+1] int32 (out, may be NULL)
 * commit_tokens  [n_seq*(K+1)] int32 capacity (out, may be NULL)
 * Limits: n_seq >= 0, 0 <= K <= 1024. */
hdf_status hdf_accept(const int32_t* draft, int draft_stride, const int32_t* target, int n_seq,
                      int K, int32_t* accept_len, int32_t* next_anchor, int32_t* commit_offsets,
                      int32_t* commit_tokens, hdf_stream_t stream);

/* The finalisation of hdf_lm_head_argmax_keys and hdf_accept on the blocks' drafts in one
 * launch (Sec. 2.3 argmax; Sec. 1 and Sec. 3.4 acceptance).  The workspace holds the
 * packed keys of the M = n_seq * B block rows (row s*B + k is slot k of sequence s) that
 * hdf_lm_head_argmax_keys left in it.  Writes argmax [M] int32 and max_logit [M] fp32 (may
 * be NULL) exactly as hdf_lm_head_argmax would, clears the keys (the workspace is handed
 * back zeroed), then runs hdf_accept with draft = argmax + 1, draft_stride = B and K = B - 1
 * (the drafts are slots 1 .. B-1).
 * ws        the workspace of the hdf_lm_head_argmax_keys call (8-byte aligned)
 * target, accept_len, next_anchor, commit_offsets, commit_tokens: as hdf_accept
 * Limits: n_seq >= 0, 1 <= B <= 1025, n_seq * B < 2^31. */
hdf_status hdf_accept_keys(void* ws, int n_seq, int B, int32_t* argmax, float* max_logit,
                           const int32_t* target, int32_t* accept_len, int32_t* next_anchor,
                           int32_t* commit_offsets, int32_t* commit_tokens, hdf_stream_t stream);

/* Context growth after a round (Sec. 1: the n_s accepted drafts and the target's token
 * after them join the context, and that token anchors the next block; Sec. 3.4:
 * tau = n_s + 1): for every s,
 *   ctx_len[s]        += accept_len[s] + 1
 *   new_counts[s]      = accept_len[s] + 1      (skipped when new_counts is NULL)
 *   block_tokens[s*B]  = next_anchor[s]         (skipped when block_tokens is NULL)
 * accept_len   [n_seq] int32 (device): hdf_accept's output
 * ctx_len      [n_seq] int32 (device, in/out); new_counts [n_seq] int32 (device, out)
 * next_anchor  [n_seq] int32 (device): hdf_accept's output; required with block_tokens
 * block_tokens [n_seq][B] int32 (device, in/out): the next round's block tokens; only
 *              slot 0 of each row is written (the mask slots stay)
 * B            the block size, 1 <= B <= 1025, when block_tokens is given (else ignored)
 * The next round's hdf_draft_block_paged takes ctx_len, new_counts and block_tokens as
 * they are, with no host read in between.  The caller keeps max_ctx and the page table
 * ahead of the growth (at most B positions a round with B = K + 1).
 * Errors: HDF_E_INVALID for n_seq < 0, null accept_len / ctx_len, block_tokens without
 * next_anchor or B outside [1, 1025]; HDF_E_UNSUPPORTED when n_seq * B >= 2^31. */
hdf_status hdf_advance_context(int n_seq, const int32_t* accept_len, int32_t* ctx_len,
                               int32_t* new_counts, const int32_t* next_anchor,
                               int32_t* block_tokens, int B, hdf_stream_t stream);

/* ------------------------------------------------------------------------------
 * 5. Temperature sampling and speculative-sampling verification (the temperature-1
 * results of Tables 2 and 3).  The paper does not restate the verification rule;
 * this is the standard one of speculative decoding: with p_i the target's and q_i
 * the drafter's softmax(logits / T) at the position of draft i,
 *     draft x_i is accepted with probability min(1, p_i(x_i) / q_i(x_i)), in order;
 *     at the first rejection n the next token is drawn from max(0, p_n - q_n)
 *     renormalised; after K acceptances it is drawn from p_K (the bonus token).
 * Random numbers come from Philox4x64-10 (Salmon et al., SC'11) with key
 * (seed, stream_id) and counter (row, v/8, purpose, 0); word (v%8)/2 of the block gives
 * two uniforms, from its high 32 bits for even v and its low 32 bits for odd v:
 * u = (top 24 bits of the half + 1/2) / 2^24.  Purpose 0: the noise of hdf_sample_tokens
 * (row = logits row, v = token); 1: the acceptance uniform of draft i of sequence s
 * (row = s, v = i); 2: the noise of the final draw of sequence s (row = s, v = token).
 * Draws from softmax(x) are argmax_v (x_v - log(-log u_v)) (Gumbel-max).
 * ----------------------------------------------------------------------------*/
/* Workspace bytes of hdf_sample_tokens for `rows` rows (0 on invalid arguments). */
size_t hdf_sample_workspace(int64_t rows, int vocab);
/* logits  rows x vocab fp32, row r at logits + r*ld (e.g. the LM head's logits output)
 * tokens  [rows] int32 (out, may be NULL): a draw from softmax(logits[r] / temperature)
 * lse     [rows] fp32 (out, may be NULL): logsumexp(logits[r] / temperature)
 * Limits: 0 <= rows <= 65535, vocab >= 1, ld >= vocab, 0 < temperature < inf; at least
 * one of tokens and lse. */
hdf_status hdf_sample_tokens(const float* logits, int64_t rows, int vocab, int64_t ld,
                             float temperature, uint64_t seed, uint64_t stream_id, int32_t* tokens,
                             float* lse, void* ws, size_t ws_bytes, hdf_stream_t stream);
/* Workspace bytes of hdf_accept_sample (0 on invalid arguments). */
size_t hdf_accept_sample_workspace(int n_seq, int K, int vocab);
/* draft          int32, draft i of sequence s at draft[s*draft_stride + i] (drawn from
 *                the draft distributions, e.g. hdf_sample_tokens on the LM head logits)
 * draft_logits   fp32, the logits of draft i of sequence s at row s*draft_stride + i of
 *                a matrix with row stride ld (the rows the drafts were drawn from)
 * draft_lse      fp32 [same rows]: logsumexp(draft logits / temperature) (hdf_sample_tokens)
 * target_logits  [n_seq][K+1][vocab] fp32: row i of sequence s holds the target's logits
 *                for the token at draft position i (i = K: the token after the drafts)
 * accept_len, next_anchor, commit_offsets, commit_tokens  as for hdf_accept; the
 *                committed tokens of s are its accepted drafts followed by the drawn token
 * With the LM head's logits of a block (row s*B + k is slot k): draft = tokens + 1,
 * draft_logits = logits + vocab, draft_lse = lse + 1, draft_stride = B, ld = vocab,
 * K = B - 1.
 * ws, ws_bytes   at least hdf_accept_sample_workspace(n_seq, K, vocab) bytes, 256-byte
 *                aligned; its contents on entry do not matter.
 * Limits: n_seq >= 0, 0 <= K <= 1024, n_seq * (K + 1) <= 65535, 0 < temperature < inf. */
hdf_status hdf_accept_sample(const int32_t* draft, int draft_stride, const float* draft_logits,
                             const float* draft_lse, int64_t ld, const float* target_logits,
                             int n_seq, int K, int vocab, float temperature, uint64_t seed,
                             uint64_t stream_id, int32_t* accept_len, int32_t* next_anchor,
                             int32_t* commit_offsets, int32_t* commit_tokens, void* ws,
                             size_t ws_bytes, hdf_stream_t stream);

/* ------------------------------------------------------------------------------
 * 6. LM-head KL distillation forward (Sec. 2.4, a training-side objective).
 *
 * Block s with its anchor at index a: slot k = 1..P targets token index a+k and is
 * supervised by the teacher t_k = LMHead(h_{a+k-1}), h the mean of the target's m
 * residual paths at that position and LMHead(h) = (RMSNorm(h) * gamma) W_lm^T:
 *     kl[s][k-1] = KL(softmax(t_k / T) || softmax(z_k / T)),  z_k the draft logits of slot k
 *     ce[s][k-1] = -log softmax(z_k)[labels[s][k-1]]          (k = 1..B-1)
 *     loss = { L_KL = T^2/P * mean_s sum_k kl[s][k-1],  L_CE = mean ce,  L_CE + alpha L_KL }
 * The pooled, normed teacher state is rounded to `dtype` before the projection.
 * ----------------------------------------------------------------------------*/
size_t hdf_kl_forward_workspace(int n_seq, int B, int P, int d, int vocab, hdf_dtype dtype);
/* H_pos           [n_seq][P][m][d] dtype: target residual paths at positions a .. a+P-1
 * gamma           [d] fp32 or NULL (ones); eps > 0
 * W_lm            [vocab][d] dtype, packed (hdf_pack_weight)
 * student_logits  fp32, slot k of block s at row s*B + k, row stride ld (the LM head's
 *                 logits of the drafted blocks)
 * labels          [n_seq][B-1] int32 ground-truth tokens of slots 1..B-1, or NULL (no CE)
 * kl              [n_seq][P] fp32 (out); ce [n_seq][B-1] fp32 (out, may be NULL);
 * loss            [3] fp32 (out, may be NULL): L_KL, L_CE (0 without labels), L
 * Limits: 1 <= m <= 8; 2 <= B <= 64; 1 <= P <= B-1; d % 64 == 0, d <= 8192;
 *         n_seq * B <= 65535; 0 < temperature < inf. */
hdf_status hdf_kl_forward(const void* H_pos, int m, const float* gamma, float eps, const void* W_lm,
                          int d, int vocab, hdf_dtype dtype, const float* student_logits,
                          int64_t ld, int B, const int32_t* labels, int n_seq, int P,
                          float temperature, float alpha, float* kl, float* ce, float* loss,
                          void* ws, size_t ws_bytes, hdf_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HDF_H_ */

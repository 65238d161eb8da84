/*
 * tk_attn.h - thin-key attention on AMD Instinct MI355X (gfx950).
 *
 * Fused attention forward O = softmax(scale * Q K^T) V in which queries and
 * keys are "thin" (r entries per head) while values and outputs keep the full
 * head width d_v: the asymmetric attention of "Thin Keys, Full Values"
 * (arXiv 2603.04427), Sec. 2.1, Eq. 1-4. Because the attention weights are
 * scalars, no projection is needed between the r-wide selection and the
 * d_v-wide value sum (the remark after Eq. 4). Thin keys come either from
 * training with a small d_select or from factoring a pretrained key projection
 * (Sec. 2.3, Eq. 6-7, with the factor absorbed into the query projection); both
 * hand the kernels the same r-wide Q and K.
 *
 * Conventions shared by all entry points
 *  - Every tensor pointer is a DEVICE pointer owned by the caller; the library
 *    never allocates, frees or synchronises, and keeps no state between calls,
 *    except for the fixed per-GPU scratch array behind tk_attn_decode_noalloc.
 *  - Layouts are dense and head-major (innermost dimension last), in elements.
 *  - Query head h reads KV head g = h / (H_q / H_kv) (grouped-query attention;
 *    the Mistral-7B setting of Sec. 3, Exp. 8 has 32 query heads over 8 KV heads).
 *  - scale <= 0 or NaN selects 1/sqrt(r), the 1/sqrt(d_head^QK) of Eq. 4.
 *  - Accumulation is fp32; bf16 outputs are rounded to nearest-even once.
 *  - Calls are asynchronous on `stream` (NULL = the null stream). Argument
 *    checks run on the host before any HIP call and return an error without
 *    launching anything; device faults surface on the stream as usual.
 *  - No exception crosses this interface.
 */
#ifndef TK_ATTN_H
#define TK_ATTN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TK_OK = 0,
    TK_ERR_INVALID_ARG = 1,  /* null pointer, bad dimension, inconsistent shapes */
    TK_ERR_UNSUPPORTED = 2,  /* valid arguments that no kernel here implements   */
    TK_ERR_WORKSPACE = 3,    /* decode workspace missing or smaller than needed   */
    TK_ERR_HIP = 4           /* the HIP runtime reported an error at launch       */
} tk_status;

typedef enum {
    TK_F32 = 0,
    TK_BF16 = 1,
    TK_FP8_E4M3 = 2, /* OCP E4M3FN codes (bias 7, no infinities, max 448) */
    TK_INT4 = 3      /* 4-bit integer key codes -7 .. 7, stored excess-8 (nibble c + 8),
                        two per byte, the even entry in the low nibble */
} tk_dtype;

/*
 * Causal (or full) prefill attention over a whole sequence: the attention core
 * of Eq. 4 for every query row at once. Prefill is compute-bound (the paper's
 * prefill roofline appendix); thin keys cut the Q K^T work by r / d_head.
 *
 *   Q [batch, H_q,  seq_q, r]     K [batch, H_kv, seq_k, r]
 *   V [batch, H_kv, seq_k, d_v]   O [batch, H_q,  seq_q, d_v]   (written)
 *   all of `dtype`: TK_BF16 (bf16 matrix cores, fp32 accumulation) or TK_F32
 *   (fp32 matrix cores).
 *
 * causal != 0: query row i sees keys 0 .. i + (seq_k - seq_q) (bottom-right
 * alignment, so a chunk of new queries sees the whole cached prefix); requires
 * seq_q <= seq_k. causal == 0: every row sees all seq_k keys.
 * Supported: r in {16, 32, 64, 128}; d_v in {64, 128}; H_q % H_kv == 0.
 * seq_q == 0 or batch == 0 is a no-op; seq_k == 0 with seq_q > 0 is invalid.
 */
tk_status tk_attn_prefill(const void* Q, const void* K, const void* V, void* O,
                          int batch, int H_q, int H_kv, int seq_q, int seq_k, int r, int d_v,
                          int causal, float scale, tk_dtype dtype, hipStream_t stream);

/*
 * Training forward: tk_attn_prefill for bf16 that also writes each query row's
 * log-sum-exp, the statistic the backward pass recomputes the attention weights
 * from (the weights of Eq. 4 are exp(scale q.k - lse)).
 *
 *   Q, K, V, O, shapes, causal, scale: as tk_attn_prefill, bf16 only.
 *   lse [batch, H_q, seq_q] fp32 (written): natural log of the sum over the
 *       row's visible keys of exp(scale * q.k), with the attention weights rounded
 *       to bf16 as the kernel forms them (so it matches the normalisation of O).
 * O is bitwise the output of tk_attn_prefill for the same arguments.
 * Errors as tk_attn_prefill; lse == NULL is invalid; TK_F32 is unsupported.
 */
tk_status tk_attn_prefill_lse(const void* Q, const void* K, const void* V, void* O, float* lse,
                              int batch, int H_q, int H_kv, int seq_q, int seq_k, int r, int d_v,
                              int causal, float scale, hipStream_t stream);

/*
 * Bytes of device workspace tk_attn_prefill_backward needs: two fp32 per query
 * row (D = rowsum(dO * O) and the row's log-sum-exp in log2 units), rounded up
 * to 256 (at least 256). Returns 0 for invalid shapes.
 */
size_t tk_attn_prefill_backward_workspace_bytes(int batch, int H_q, int seq_q);

/*
 * Backward pass of the thin-key prefill: the gradients of the attention core of
 * Eq. 4 with respect to the r-wide Q and K and the d_v-wide V, needed to train
 * thin-key models from scratch (Sec. 3, Exp. 7 and 7b, whose shorter wall-clock
 * comes from the smaller Q K^T work in both passes). With P the attention
 * weights and D = rowsum(dO * O):
 *     dV = P^T dO,   dS = P * (dO V^T - D),   dQ = scale dS K,   dK = scale dS^T Q
 * where dK and dV sum over the H_q / H_kv query heads of each KV head.
 *
 *   Q [batch, H_q, seq_q, r]   K [batch, H_kv, seq_k, r]   V [batch, H_kv, seq_k, d_v]
 *   O, dO [batch, H_q, seq_q, d_v]: the forward output and the loss gradient
 *   lse [batch, H_q, seq_q] fp32: from tk_attn_prefill_lse with the same arguments
 *   dQ [batch, H_q, seq_q, r], dK [batch, H_kv, seq_k, r],
 *   dV [batch, H_kv, seq_k, d_v]: written (overwritten, not accumulated)
 *   all tensors bf16 except lse; accumulation in fp32, one rounding per output.
 *   workspace: device memory of at least
 *       tk_attn_prefill_backward_workspace_bytes(batch, H_q, seq_q) bytes,
 *       4-byte aligned, no initial contents required; calls sharing it must
 *       not run concurrently.
 * causal and scale as tk_attn_prefill. No atomics: results are bitwise
 * reproducible. Keys that no row sees get zero gradients; seq_q == 0 with
 * seq_k > 0 writes zero dK and dV; batch == 0 is a no-op.
 * Supported: r in {32, 64, 128}; d_v in {64, 128}; H_q % H_kv == 0.
 * Errors: TK_ERR_INVALID_ARG for null or misaligned (16 bytes) tensors or
 * inconsistent shapes, TK_ERR_WORKSPACE for a missing or small workspace,
 * TK_ERR_UNSUPPORTED for other r or d_v.
 */
tk_status tk_attn_prefill_backward(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                                   const float* lse, void* dQ, void* dK, void* dV,
                                   int batch, int H_q, int H_kv, int seq_q, int seq_k, int r, int d_v,
                                   int causal, float scale, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/*
 * Bytes of device workspace tk_attn_decode needs for these shapes (split-K
 * partial results). A pure function of its arguments: no device query.
 * Returns 0 for invalid shapes.
 */
size_t tk_attn_decode_workspace_bytes(int batch, int H_q, int H_kv, int max_ctx, int d_v);

/*
 * Single-token decode against a thin-key / full-value cache (Sec. 2.4, Eq. 9:
 * keys occupy r / d_v of the value footprint), with grouped-query sharing, an
 * optional paged layout and optional fp8 keys (the composition with
 * quantisation proposed in Sec. 6). Decode is memory-bound (Sec. 4.2, Eq. 10):
 * every cached K and V byte is read exactly once per call.
 *
 *   Q [batch, H_q, r] bf16            O [batch, H_q, d_v] bf16 (written)
 *   ctx_lens [batch] int32 (device): sequence b attends to its first
 *       ctx_lens[b] cached tokens (the current token already appended).
 *       Values are clamped to [0, max_ctx]; 0 writes a zero output row.
 *   max_ctx (host): an upper bound on ctx_lens; sizes the launch.
 *   contiguous cache (block_table == NULL):
 *       K_cache [batch, H_kv, max_ctx, r]   V_cache [batch, H_kv, max_ctx, d_v]
 *       k_scale [batch, H_kv, max_ctx]
 *   paged cache (block_table != NULL):
 *       K_cache [num_blocks, H_kv, block_size, r]
 *       V_cache [num_blocks, H_kv, block_size, d_v]
 *       k_scale [num_blocks, H_kv, block_size]
 *       block_table [batch, max_blocks_per_seq] int32 (device): token t of
 *       sequence b is slot t % block_size of block block_table[b][t / block_size].
 *       block_size must be a power of two >= 64 and
 *       max_ctx <= block_size * max_blocks_per_seq. A table entry outside
 *       [0, num_blocks) is never dereferenced: that sequence's output is NaN.
 *   k_dtype: TK_BF16 keys; TK_FP8_E4M3 key codes (r bytes per row); or TK_INT4
 *       4-bit key codes (r/2 bytes per row, so K_cache rows are r/2 bytes wide).
 *       Quantised keys come with one fp32 scale per (token, KV head) in k_scale
 *       (the key row is code * scale); k_scale must be NULL for bf16 keys.
 *   V_cache is always bf16.
 *   workspace: device memory of at least
 *       tk_attn_decode_workspace_bytes(batch, H_q, H_kv, max_ctx, d_v) bytes,
 *       256-byte aligned. It holds per-split partial results and a small
 *       leading region of arrival counters: the buffer must be all zero before
 *       its first use (allocate it zeroed); every completed call leaves the
 *       counters zero again, so it can be reused without clearing. Calls that
 *       share one workspace must not run concurrently.
 * Supported: r in {16, 32, 64, 128}; d_v in {64, 128}; H_q % H_kv == 0.
 * The split of the context depends only on the shapes, so results are bitwise
 * reproducible from run to run.
 */
tk_status tk_attn_decode(const void* Q, const void* K_cache, const void* V_cache, void* O,
                         int batch, int H_q, int H_kv, const int32_t* ctx_lens, int max_ctx,
                         int r, int d_v, float scale,
                         tk_dtype k_dtype, const float* k_scale,
                         const int32_t* block_table, int block_size, int max_blocks_per_seq,
                         int num_blocks,
                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * tk_attn_decode without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation). Arguments, layouts, results and errors are
 * those of tk_attn_decode, and the same kernels run with the same split, so
 * outputs are bitwise equal to tk_attn_decode's.
 *
 * Instead of a caller's workspace the call uses a fixed device array inside the
 * library: 4 MiB per GPU, held from the first call on that GPU until the process
 * ends. Every supported shape fits (a split context has fewer than 4096
 * (sequence, head, split) partial rows); a call that would need more returns
 * TK_ERR_WORKSPACE before touching the GPU. On the first call on a device (the
 * current device, which must be the stream's device, else TK_ERR_INVALID_ARG)
 * the library looks up that device's copy and clears its counters with a small
 * kernel on `stream`; every completed call leaves them zero again.
 * The call allocates nothing and makes no hipMalloc or hipFree. All calls on one
 * GPU share the array: calls that may overlap on one GPU (different streams,
 * host threads or processes) race and must be serialised by the caller.
 */
tk_status tk_attn_decode_noalloc(const void* Q, const void* K_cache, const void* V_cache, void* O,
                                 int batch, int H_q, int H_kv, const int32_t* ctx_lens, int max_ctx,
                                 int r, int d_v, float scale,
                                 tk_dtype k_dtype, const float* k_scale,
                                 const int32_t* block_table, int block_size, int max_blocks_per_seq,
                                 int num_blocks, hipStream_t stream);

/*
 * Append n_new tokens per sequence to a thin-key / full-value cache: the write
 * that precedes decode (the thin-K / full-V cache of Sec. 2.4, Eq. 9). Token t
 * of sequence b and KV head g is stored at cache position positions[b] + t.
 *
 *   K_new [batch, H_kv, n_new, r] bf16      V_new [batch, H_kv, n_new, d_v] bf16
 *   positions [batch] int32 (device): first position written for sequence b.
 *   K_cache, V_cache, k_scale, block_table, block_size, max_blocks_per_seq,
 *       num_blocks, k_dtype: the cache layouts of tk_attn_decode. A contiguous
 *       cache holds max_ctx positions per sequence; a paged one
 *       block_size * max_blocks_per_seq (max_ctx is then not used); block_size
 *       must be a power of two.
 *   k_dtype TK_BF16 copies the key rows. TK_FP8_E4M3 quantises each key row on
 *       the way in (the composition with quantisation of Sec. 6): its scale is
 *       max|k| / 448 over the row's r entries (1.0 for an all-zero row), stored in
 *       k_scale, and each entry becomes the OCP E4M3 code of k / scale rounded to
 *       nearest-even; both steps in fp32 with IEEE division. TK_INT4 does the same
 *       with scale max|k| / 7 and code k / scale rounded half-to-even and clipped
 *       to [-7, 7], stored excess-8 (see tk_dtype).
 * A token whose position is negative or not below the capacity, or whose block
 * table entry lies outside [0, num_blocks), is not written (nothing else is
 * touched). Tokens of one call must land on distinct positions. V_cache rows and
 * bf16 key rows are bit-exact copies.
 * Supported: r in {16, 32, 64, 128}; d_v in {64, 128}; batch * H_kv <= 65535.
 * batch == 0 or n_new == 0 is a no-op. Pointers to bf16 data and the caches must
 * be 16-byte aligned.
 */
tk_status tk_cache_append(const void* K_new, const void* V_new, int batch, int H_kv, int n_new, int r, int d_v,
                          const int32_t* positions, void* K_cache, void* V_cache, int max_ctx,
                          tk_dtype k_dtype, float* k_scale,
                          const int32_t* block_table, int block_size, int max_blocks_per_seq,
                          int num_blocks, hipStream_t stream);

/*
 * One projection of a layer converted to thin keys (Sec. 2.3, Eq. 6-7), written
 * head-major for the attention calls above:
 *
 *     Y[b, h, s, :] = X[b, s, :] W[:, h * width .. (h + 1) * width - 1]
 *
 * After the key projection of every KV head is factored as W_K ~= A B (a
 * truncated SVD) and B is absorbed into the query projection, a layer needs
 * the absorbed queries q' = x W_Q' and the thin keys k' = x A (width r each),
 * and its unchanged values v = x W_V (width d_v): three calls of this function.
 *
 *   X  [batch, seq, d_model] bf16: the layer's input rows (hidden states)
 *   Wt [n_heads * width, d_model] bf16: W transposed (row n is column n of W)
 *   Y  [batch, n_heads, seq, width] bf16 (the Q / K / V layout of
 *       tk_attn_prefill and the K_new / V_new layout of tk_cache_append)
 * Products on the bf16 matrix cores, fp32 accumulation, one round-to-nearest-
 * even to bf16. Supported: d_model % 32 == 0 and d_model <= 2^22, width % 4 == 0;
 * pointers 16-byte aligned. batch == 0 or seq == 0 is a no-op.
 */
tk_status tk_project_heads(const void* X, const void* Wt, void* Y, int batch, int seq, int d_model,
                           int n_heads, int width, hipStream_t stream);

/* A static, human-readable name for a status code. Never NULL. */
const char* tk_status_str(tk_status status);

/* Library version, major * 10000 + minor * 100 + patch. */
int tk_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TK_ATTN_H */

/*
 * topk_attn.h -- C ABI of the MI355X (gfx950) top-k attention library.
 *
 * The library computes top-k attention (arXiv 2106.06899, Section 2.2, Eq. 4):
 *
 *     out = activation( top-k( Q K^T ) ) V
 *
 * row by row: each query keeps the k keys with the largest raw scores q.k_j,
 * an activation runs over those k survivors only, and the k matching value rows
 * are summed with the resulting weights. Queries are processed in chunks of
 * `chunk` rows (Section 2.2, "Query chunking"); the chunk size bounds the
 * working memory and never changes the result. The feed-forward layer written
 * as attention (Eq. 3: keys W1, values W2, ReLU) has calls of its own (topk_ffn*).
 *
 * Entry points: the forward calls (topk_attn, topk_ffn); their *_with_cache
 * variants, which also write each row's selection for training; the backward
 * calls (topk_attn_backward, topk_ffn_backward), which recompute from that cache
 * and the inputs only (Section 2.2, "Input checkpointing"); workspace queries and
 * registration; two process-wide settings (topk_set_memory_budget,
 * topk_set_backward_lists); and debug and test hooks.
 *
 * Conventions shared by every call:
 *  - Every tensor pointer is a caller-owned DEVICE pointer to contiguous row-major
 *    data, 16-byte aligned. The library never frees caller memory.
 *  - dtype is TOPK_F32 or TOPK_BF16 for all of a call's tensors; scores are
 *    accumulated in fp32; outputs are stored in the input dtype (bf16 is rounded
 *    to nearest-even).
 *  - Calls validate their arguments synchronously; on any error they return a
 *    negative status, launch nothing and leave `out` untouched. On success all
 *    work is enqueued on `hip_stream` (a hipStream_t; NULL = the null stream) and
 *    the call returns without waiting.
 *  - Selection order: (score desc, key index asc); among equal scores the lower
 *    key index is kept. Inputs are assumed finite.
 *  - Working memory: either the buffer registered with topk_set_workspace() on
 *    the calling thread, or (when none is registered) stream-ordered memory the
 *    library allocates and frees on `hip_stream`.
 *  - Calls on different streams are safe if they use different workspaces.
 *    Each call reads the process-wide settings once, when it is made; a change
 *    applies to the calls made after it (and changes what the workspace queries
 *    return).
 */
#ifndef TOPK_ATTN_H
#define TOPK_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* element types */
#define TOPK_F32 0
#define TOPK_BF16 1

/* status codes */
#define TOPK_OK 0
#define TOPK_E_INVAL -1       /* a size, k, chunk, scale, flag or dtype is out of range */
#define TOPK_E_NULL -2        /* a required pointer is NULL */
#define TOPK_E_ALIGN -3       /* a tensor pointer is not 16-byte aligned */
#define TOPK_E_UNSUPPORTED -4 /* valid arguments outside what the library implements */
#define TOPK_E_NOMEM -5       /* the registered workspace is too small / allocation failed */
#define TOPK_E_HIP -6         /* a HIP runtime call or kernel launch failed */

/*
 * topk_attn -- top-k attention (Eq. 4 with softmax; temperature of Eq. 1; causal
 * mask of Eq. 2), for B*H independent heads (Section 2.1, multi-head attention).
 *
 *   Q   [B, H, Lq, d]   queries
 *   K   [B, H, Lk, d]   keys
 *   V   [B, H, Lk, d]   values
 *   out [B, H, Lq, d]   written: out[i] = sum_{j in S_i} w_ij V[j], with S_i the
 *                       k_eff = min(k, #valid keys) keys of largest q_i.k_j and
 *                       w_ij = exp(scale*(s_ij - max_S s)) / sum_S exp(...)
 *   k       1 <= k <= Lk
 *   chunk   query chunk size C >= 1 (0 = library default); result-neutral
 *   causal  0 or 1; with 1, key j is valid for query i iff j <= i (0-based)
 *   scale   1/lambda of Eq. 1, finite and > 0; used only inside the softmax
 *           (selection uses the raw score, which is invariant to scale > 0)
 *   dtype   TOPK_F32 or TOPK_BF16; d must be a multiple of 8 and <= 1024
 */
int topk_attn(const void* Q, const void* K, const void* V, void* out,
              int64_t B, int64_t H, int64_t Lq, int64_t Lk, int64_t d,
              int64_t k, int64_t chunk, int causal, float scale,
              int dtype, void* hip_stream);

/*
 * topk_attn_dense -- query chunking with the top-k disabled, the comparison
 * baseline of Section 2.2 ("Query chunking") and Section 3: every valid key of a
 * query contributes, out[i] = sum_j softmax_j(scale * q_i.k_j) V[j] (Eq. 1, with
 * the causal mask of Eq. 2); the same result as topk_attn with k = Lk. Arguments
 * as topk_attn without k. Computed by a streaming softmax over key tiles (no score
 * tile is stored, no workspace is used); chunk only sets how queries are grouped.
 * Supports bf16 inputs with d = 64 or 128 (else TOPK_E_UNSUPPORTED). topk_attn
 * itself calls this for k = Lk above the select's limit of 2048 keys.
 */
int topk_attn_dense(const void* Q, const void* K, const void* V, void* out,
                    int64_t B, int64_t H, int64_t Lq, int64_t Lk, int64_t d,
                    int64_t chunk, int causal, float scale, int dtype, void* hip_stream);

/*
 * topk_ffn -- the feed-forward layer recast as attention (Eq. 3) with the top-k
 * of Eq. 4 and a ReLU activation: out[i] = sum_{j in S_i} max(x_i.W1[j], 0) W2[j],
 * where S_i holds the k largest scores x_i.W1[j]. No bias, no temperature; ReLU
 * applies after selection, so negative survivors are selected with weight 0.
 *
 *   X   [N, d_model]      token inputs (the queries)
 *   W1  [d_ff, d_model]   keys: row j is key j
 *   W2  [d_ff, d_model]   values: row j is value j
 *   out [N, d_model]      written
 *   k       1 <= k <= d_ff;  chunk: token chunk size (0 = default), result-neutral
 *   dtype   TOPK_F32 or TOPK_BF16; d_model must be a multiple of 8 and <= 1024
 */
int topk_ffn(const void* X, const void* W1, const void* W2, void* out,
             int64_t N, int64_t d_model, int64_t d_ff, int64_t k,
             int64_t chunk, int dtype, void* hip_stream);

/*
 * Debug / parity variants: the same computation, plus, when non-NULL,
 *   idx_out   int32 [rows, k]: the selected key indices of each query row in the
 *             order (score desc, index asc); -1 pads rows with k_eff < k
 *   score_out fp32  [rows, k]: their raw (unscaled) fp32 scores; -inf pads
 * where rows = B*H*Lq (attention) or N (FFN), in the row order of `out`.
 */
int topk_attn_debug(const void* Q, const void* K, const void* V, void* out,
                    int64_t B, int64_t H, int64_t Lq, int64_t Lk, int64_t d,
                    int64_t k, int64_t chunk, int causal, float scale,
                    int dtype, void* hip_stream, int32_t* idx_out, float* score_out);
int topk_ffn_debug(const void* X, const void* W1, const void* W2, void* out,
                   int64_t N, int64_t d_model, int64_t d_ff, int64_t k,
                   int64_t chunk, int dtype, void* hip_stream,
                   int32_t* idx_out, float* score_out);

/*
 * Forward pass for training with input checkpointing (Section 2.2, "Input
 * checkpointing"): the same computation as topk_attn / topk_ffn, also writing the
 * cache the backward calls take: top_idx int32 [rows, k] and top_dots fp32
 * [rows, k], laid out as idx_out / score_out above (both required, 4-byte aligned,
 * caller-owned device memory). Unlike the debug variants these calls do not read
 * anything back: they only enqueue on hip_stream. Errors as topk_attn, and
 * TOPK_E_NULL when top_idx or top_dots is NULL.
 */
int topk_attn_with_cache(const void* Q, const void* K, const void* V, void* out,
                         int64_t B, int64_t H, int64_t Lq, int64_t Lk, int64_t d,
                         int64_t k, int64_t chunk, int causal, float scale,
                         int dtype, void* hip_stream, int32_t* top_idx, float* top_dots);
int topk_ffn_with_cache(const void* X, const void* W1, const void* W2, void* out,
                        int64_t N, int64_t d_model, int64_t d_ff, int64_t k,
                        int64_t chunk, int dtype, void* hip_stream,
                        int32_t* top_idx, float* top_dots);

/*
 * Workspace (bytes) a call with these arguments uses under the memory budget;
 * 0 when the arguments are invalid. Register at least this much with
 * topk_set_workspace() to run without library allocations. The budget caps the
 * number of query chunks in flight, so the figure is O(chunk) per chunk and
 * never exceeds the budget plus a fixed remainder (at least one chunk runs per
 * pass whatever the budget).
 */
size_t topk_attn_workspace_bytes(int64_t B, int64_t H, int64_t Lq, int64_t Lk, int64_t d,
                                 int64_t k, int64_t chunk, int causal, int dtype);
size_t topk_ffn_workspace_bytes(int64_t N, int64_t d_model, int64_t d_ff, int64_t k,
                                int64_t chunk, int dtype);

/*
 * Register (dev_ptr, bytes) as the calling thread's workspace for later calls;
 * (NULL, 0) unregisters it. The caller owns the memory and must keep it alive
 * until the enqueued work has finished. A call whose schedule does not fit the
 * registered size first shrinks the number of chunks in flight and returns
 * TOPK_E_NOMEM only if one chunk does not fit. Returns TOPK_OK, or TOPK_E_NULL
 * for a NULL pointer with bytes > 0, or TOPK_E_ALIGN for a pointer that is not
 * 256-byte aligned.
 */
int topk_set_workspace(void* dev_ptr, size_t bytes);

/*
 * topk_attn_noalloc -- for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same arguments, computation and result as topk_attn, with the whole workspace
 * inside a fixed scratch array of TOPK_NOALLOC_SCRATCH_BYTES that the library
 * keeps on every GPU it runs on until the process ends. The call makes no
 * hipMalloc, hipFree or other allocating call and ignores any workspace registered
 * with topk_set_workspace; the caller still owns Q, K, V and out. Its query-chunk
 * passes are fitted into the scratch; when a single chunk needs more, it returns
 * TOPK_E_NOMEM before launching anything. Every call on one GPU uses that GPU's
 * scratch, which keeps the last call's contents (each call initialises what it
 * reads): calls of one process that overlap in time on the same GPU (other
 * streams, other threads) race, and the caller must order them. Errors as
 * topk_attn, plus TOPK_E_HIP when there is no current device or the scratch
 * address cannot be obtained.
 */
#define TOPK_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
int topk_attn_noalloc(const void* Q, const void* K, const void* V, void* out,
                      int64_t B, int64_t H, int64_t Lq, int64_t Lk, int64_t d,
                      int64_t k, int64_t chunk, int causal, float scale,
                      int dtype, void* hip_stream);
size_t topk_noalloc_scratch_bytes(void);  /* TOPK_NOALLOC_SCRATCH_BYTES */

/*
 * The forward calls' memory budget, process-wide: the most workspace a call sizes
 * for itself (the chunks of a call run in passes of as many chunks as fit; a
 * budget below one chunk's needs runs one chunk per pass, the paper's sequential
 * query chunking of Section 2.2). 0 restores the default of 8 GiB. A registered
 * workspace (topk_set_workspace) takes the place of the budget. Returns TOPK_OK.
 */
int topk_set_memory_budget(size_t bytes);

/* Message describing the calling thread's last non-OK return ("" if none). */
const char* topk_last_error(void);

/*
 * Which implementation the arguments select: 1 = fused score+filter path
 * (bf16 MFMA score tiles, candidates filtered on chip), 2 = chunk-tile path
 * (the chunk's score tile in workspace, then a row-wise select), 3 = both, by rows
 * (causal masks on the fused path: the first 1024 R rows of every head, whose few
 * valid keys give the fused threshold sample too few blocks, run on the chunk-tile
 * path; R = 3, 6, 12 for k <= 32, 64, 128), 4 = filtered chunk-tile path (bf16,
 * d % 32 == 0, k <= 512, 2048 < Lk <= 65536: every 16th key is scored first, each
 * row's threshold comes from those samples, and only the scores reaching it are kept
 * as candidates, by the fused path's score kernel at d = 128 and by the chunk-tile
 * GEMM otherwise; the rest as the fused path), or a negative status for invalid
 * arguments. For tests and reports.
 */
int topk_attn_path(int64_t B, int64_t H, int64_t Lq, int64_t Lk, int64_t d,
                   int64_t k, int64_t chunk, int causal, int dtype);
int topk_ffn_path(int64_t N, int64_t d_model, int64_t d_ff, int64_t k,
                  int64_t chunk, int dtype);

/*
 * Stage timing, for benchmarks. After topk_profile_begin(), every call made on
 * the calling thread records a pair of HIP events on its own stream around each
 * launch group: stage 0 = score tiles (fused scan, or chunk-tile scores),
 * 1 = row select, 2 = fallback recomputation (fused and filtered paths), 3 = activation
 * and gather, 4 = a backward call. topk_profile_end() waits for those events, writes the summed
 * milliseconds and the number of timed launches of the first n_stages stages
 * into stage_ms / stage_launches (host arrays, either may be NULL) and stops
 * recording. Returns TOPK_OK or TOPK_E_HIP.
 */
int topk_profile_begin(void);
int topk_profile_end(double* stage_ms, int64_t* stage_launches, int n_stages);

/*
 * Backward pass of top-k attention with input checkpointing (Section 2.2, "Input
 * checkpointing", and the backward pseudo-code that follows it). The forward pass
 * caches only its inputs and each row's selection: top_idx (int32 [B, H, Lq, k],
 * -1 pads) and top_dots (float [B, H, Lq, k], the raw fp32 scores q . k of the
 * selected keys), exactly what topk_attn_debug writes as idx_out / score_out.
 * Given d_out = dLoss/d(out) ([B, H, Lq, d]), this recomputes the softmax with
 * temperature `scale` over the k survivors from the cached scores, backpropagates
 * through it, and writes
 *   d_Q [B, H, Lq, d] = sum_m d_top_dots[m] K[j_m]             (per query row),
 *   d_K [B, H, Lk, d] = sum over the rows that selected key j of d_top_dots * Q[row],
 *   d_V [B, H, Lk, d] = sum over the rows that selected key j of weight * d_out[row],
 * keys selected by no row get zeros. All tensors are caller-owned device memory,
 * contiguous, in `dtype` (fp32 accumulation; bf16 results rounded to nearest even);
 * every output element is written. Entries of top_idx outside [0, Lk) are padding.
 * The sums over a key's rows run in increasing (row, slot) order, so results do
 * not depend on scheduling (with atomic lists, see topk_set_backward_lists, only
 * for keys that at most 1024 rows selected). Workspace:
 * topk_attn_backward_workspace_bytes() bytes, O(B*H*(Lq*k + Lk)) (the registered
 * workspace, or one allocated on the stream). Errors as topk_attn; additionally
 * TOPK_E_UNSUPPORTED when B*H*Lq*k or B*H*Lk reaches 2^31.
 */
int topk_attn_backward(const void* Q, const void* K, const void* V, const int32_t* top_idx, const float* top_dots,
                       const void* d_out, void* d_Q, void* d_K, void* d_V, int64_t B, int64_t H, int64_t Lq,
                       int64_t Lk, int64_t d, int64_t k, float scale, int dtype, void* hip_stream);

/*
 * Backward pass of the top-k feed-forward layer (Eq. 3 as top-k attention: keys
 * W1, values W2, ReLU, no temperature), with the same cache (top_idx, top_dots:
 * [N, k], as topk_ffn_debug writes them) and d_out [N, d_model]. Writes
 * d_X [N, d_model], d_W1 [d_ff, d_model], d_W2 [d_ff, d_model]; the ReLU gradient is
 * zero where the cached score is <= 0. Same conventions as topk_attn_backward.
 */
int topk_ffn_backward(const void* X, const void* W1, const void* W2, const int32_t* top_idx, const float* top_dots,
                      const void* d_out, void* d_X, void* d_W1, void* d_W2, int64_t N, int64_t d_model, int64_t d_ff,
                      int64_t k, int dtype, void* hip_stream);

/*
 * How the backward calls group the selected (row, key) pairs by key, process-wide:
 * TOPK_LISTS_AUTO (default) takes the bucket sort for heads of up to 2^19 keys
 * and atomic counters beyond; TOPK_LISTS_BUCKET asks for the bucket sort (a
 * backward call on a larger head then fails with TOPK_E_UNSUPPORTED);
 * TOPK_LISTS_ATOMIC asks for the atomic counters. The bucket sort (a two-level
 * stable counting sort in LDS) writes every list in increasing pair order; atomic
 * counters fill lists in arbitrary order and sort lists of up to 1024 pairs before
 * summing. Both give the same gradients, bit for bit, where the atomic lists are
 * sorted. The workspace size depends on the setting. Returns TOPK_OK, or
 * TOPK_E_INVAL for another mode.
 */
#define TOPK_LISTS_AUTO 0
#define TOPK_LISTS_BUCKET 1
#define TOPK_LISTS_ATOMIC 2
int topk_set_backward_lists(int mode);

/* Workspace the backward calls need (0 for invalid arguments). */
size_t topk_attn_backward_workspace_bytes(int64_t B, int64_t H, int64_t Lq, int64_t Lk, int64_t d, int64_t k,
                                          int dtype);
size_t topk_ffn_backward_workspace_bytes(int64_t N, int64_t d_model, int64_t d_ff, int64_t k, int dtype);

/*
 * Test hook: the number of query rows that the last topk_attn_debug /
 * topk_ffn_debug call on the calling thread selected through a fallback path
 * (rows whose sampled threshold or candidate buffers could not prove the
 * candidate set complete, and were selected from all their keys instead). Debug
 * calls read this count back from the device, so they wait for their stream.
 * Returns -1 when the thread's last debug call failed or none was made.
 */
int64_t topk_last_fallback_rows(void);

/*
 * Test hook: run one wave of the bf16 MFMA used by the fused path on inputs that
 * tag each operand element with its row or column, and write, for every lane l
 * and accumulator register v, the output row (key) into rows_out[l*16+v] and
 * column (query) into cols_out[l*16+v]. Both are int32 device buffers of 1024
 * entries. Lets a GPU test confirm the lane layout the fused kernel assumes.
 */
int topk_selftest_mfma_layout(int32_t* rows_out, int32_t* cols_out, void* hip_stream);

/*
 * Debug hook. The library also builds as libtopk_check.so (compiled with
 * TOPK_CHECK_INDICES): there every forward call waits for its stream and returns
 * TOPK_E_HIP for an error its kernels raised while running, and the finalize counts
 * selected indices outside the value matrix (which it clamps in every build, so that
 * no read leaves the matrix). This returns that count since the last call and resets
 * it (waits for the device), or -1 in the normal build.
 */
int64_t topk_debug_bad_indices(void);

/*
 * Measurement hook: run only the fused path's score kernel (its sampled threshold
 * phase and scan) of a topk_attn call on bf16 Q, K [B, H, L, 64] with 32 < k <= 64,
 * as many passes as the call would run; with score_only = 1 the scan's score-core
 * ablation runs instead (the same K tile pipeline, MFMAs and block maxima, no
 * filter and no candidate output). Nothing useful is written; the kernels' time is
 * read with topk_profile_begin / topk_profile_end (stage "score"). Allocates its
 * workspace. TOPK_E_UNSUPPORTED for other shapes or paths.
 */
int topk_scan_ablation(const void* Q, const void* K, int64_t B, int64_t H, int64_t Lq, int64_t Lk,
                       int64_t d, int64_t k, int64_t chunk, int score_only, void* hip_stream);

/*
 * Measurement hook: the sustained rate of v_mfma_f32_32x32x16_bf16 on the current
 * device (a register-only stream of independent MFMAs, two waves per SIMD on every
 * CU, timed with HIP events), in TFLOP/s, and the shader clock those MFMAs ran at
 * (shader clock counter over the constant 100 MHz counter), in MHz. Waits for the
 * stream. Returns TOPK_OK, TOPK_E_NULL, TOPK_E_NOMEM or TOPK_E_HIP.
 */
int topk_probe_mfma(double* tflops, double* clock_mhz, void* hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* TOPK_ATTN_H */

/*
 * sparstar.h -- C ABI of the SparSTAR hot path on AMD Instinct MI355X (gfx950).
 *
 * SparSTAR (arXiv 2608.10519) sparsifies the late-scale attention of a
 * next-scale video generator.  For every (batch, head) it
 *   1. cuts Q and K, in their original order, into contiguous blocks of
 *      `block_size` tokens and mean-pools each block over the nominal block
 *      length (Section 5.1);
 *   2. scores every selectable key block against every query block with
 *      S_ij = D^-1/2 * qbar_i . kbar_j (Eq. 2);
 *   3. keeps the forced blocks dense (the blocks touching any forced token
 *      range: the text, plus the reference for the first clip; Eq. 3) and
 *      takes the top k = min(n_sel, max(1, ceil(rho * n_sel))) of the others
 *      (Eq. 4-6);
 *   4. runs forward-only attention over the selected key blocks (Eq. 7,
 *      Section 5.3), writing O and the log-sum-exp.
 *
 * Conventions shared by every call
 *   - Tensors are dense, row-major, in device memory (HBM):
 *       Q [B, H, Lq, D] bf16, K and V [B, H, Lk, D] bf16, O [B, H, Lq, D] bf16,
 *       lse [B, H, Lq] fp32, kv_num_blocks [B, H, n_q] int32,
 *       kv_indices [B, H, n_q, kv_stride] int32,
 *     with n_q = ceil(Lq / block_size) and n_k = ceil(Lk / block_size).
 *     bf16 buffers are passed as `const void*` (16-bit patterns), 16-byte aligned.
 *   - The caller owns every buffer.  The library allocates no device memory,
 *     copies nothing between host and device and never synchronises: each call
 *     validates its arguments on the host, enqueues its kernels on `stream`
 *     (a hipStream_t passed as void*, so that this header needs no HIP
 *     include; NULL is the default stream) and returns.
 *   - Return value: SPARSTAR_OK, or a negative code.  Argument errors are
 *     detected on the host before any HIP call (nothing is launched, outputs are
 *     untouched); a failed launch returns SPARSTAR_ERR_HIP.  Faults inside a
 *     kernel surface at the caller's next synchronisation, as for any HIP
 *     work.  sparstar_last_error() describes the last non-OK return on the
 *     calling thread.
 *   - The library holds no state besides that thread-local message and the
 *     per-GPU scratch array of sparstar_score_blocks_static; calls on
 *     different streams may run concurrently, except that calls of
 *     sparstar_score_blocks_static on one GPU share that array.
 */
#ifndef SPARSTAR_H
#define SPARSTAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* A half-open token range [begin, end) of the key sequence. */
typedef struct {
  int64_t begin;
  int64_t end;
} sparstar_range;

enum {
  SPARSTAR_OK = 0,
  SPARSTAR_ERR_INVALID_ARG = -1, /* a null pointer, a bad size or value      */
  SPARSTAR_ERR_UNSUPPORTED = -2, /* a head_dim / block_size not built        */
  SPARSTAR_ERR_WORKSPACE = -3,   /* workspace missing or too small           */
  SPARSTAR_ERR_HIP = -4          /* a HIP launch or runtime call failed      */
};

/* Upper bound on forced ranges and heads the selector accepts. */
#define SPARSTAR_MAX_KEEP_RANGES 8
#define SPARSTAR_MAX_HEADS 256

/*
 * Bytes of device scratch sparstar_score_blocks needs for these sizes: the
 * pooled blocks qbar [B,H,n_q,D] and kbar [B,H,n_k,D] (4 bytes per element:
 * each block is kept as a power-of-two scale times a pair of fp16 parts), the
 * blocks' scales (int32, [B,H,n_q] and [B,H,n_k]) and the fp32 score matrix
 * S [B,H,n_q,n_k] with its rows padded to a multiple of 32 floats, each region
 * 256-byte aligned.  Returns 0 for invalid sizes.
 */
size_t sparstar_score_workspace_bytes(int B, int H, int64_t Lq, int64_t Lk, int D, int block_size);

/*
 * The smallest valid kv_stride for sparstar_score_blocks with these arguments:
 * |J_keep| + max_h k_h (Eq. 3-5).  Arguments as for sparstar_score_blocks (Lq,
 * B and D do not matter).  Returns a negative SPARSTAR_ERR_* code on invalid
 * arguments.  Host-only; touches no device.
 */
int64_t sparstar_kv_stride(int H, int64_t Lk, int block_size, const double* budget, int n_budget,
                           const sparstar_range* keep, int n_keep);

/*
 * The selector: block pooling (Section 5.1), block scores (Eq. 2), keep and
 * selectable sets (Eq. 3-4), budget (Eq. 5) and the retained supports
 * A_i (Eq. 6), written as the forward-only block mask of Section 5.3.
 *
 *   q, k            device bf16 Q [B,H,Lq,D] and K [B,H,Lk,D].
 *   B, H, Lq, Lk    sizes; B, H >= 1 (H <= SPARSTAR_MAX_HEADS), Lq >= 0, Lk >= 1.
 *   D               head dim, 64 or 128.
 *   block_size      b, 64 or 128 (the same b for queries and keys).
 *   budget          host array of densities rho in [0, 1]: n_budget == 1 (all
 *                   heads) or n_budget == H (one per head).  The budget of head h
 *                   is k_h = min(n_sel, max(1, ceil(rho_h * n_sel))), where a
 *                   product within 1e-9 * max(1, n_sel) of an integer counts as
 *                   that integer.
 *   keep, n_keep    host array of forced token ranges, 0 <= begin <= end <= Lk,
 *                   n_keep <= SPARSTAR_MAX_KEEP_RANGES (keep may be NULL when
 *                   n_keep == 0).  J_keep = { j : block j meets some range }.
 *   kv_num_blocks   device out [B,H,n_q]: |J_keep| + k_h for every row.
 *   kv_indices      device out [B,H,n_q,kv_stride]: the first kv_num_blocks
 *                   entries of each row are A_i in ascending block order (the
 *                   forced blocks included); later entries are left untouched.
 *   kv_stride       row stride of kv_indices; must be >= |J_keep| + max_h k_h.
 *   scores          optional device out [B,H,n_q,n_k] fp32: S_ij for selectable
 *                   j; entries of forced columns are unspecified.  NULL to keep
 *                   S in the workspace only.
 *   workspace       device scratch of >= sparstar_score_workspace_bytes(...)
 *                   bytes, 256-byte aligned; its contents need no initialisation
 *                   and are garbage afterwards.
 *
 * Ties in S are broken toward the lower block index.  The call is deterministic.
 * Lq == 0 is a no-op.
 */
int sparstar_score_blocks(const void* q, const void* k, int B, int H, int64_t Lq, int64_t Lk, int D,
                          int block_size, const double* budget, int n_budget, const sparstar_range* keep,
                          int n_keep, int32_t* kv_num_blocks, int32_t* kv_indices, int kv_stride, float* scores,
                          void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of device scratch the library holds per GPU for sparstar_score_blocks_static (64 MiB). */
#define SPARSTAR_STATIC_SCRATCH_BYTES ((size_t)64 << 20)

/*
 * sparstar_score_blocks for callers that cannot allocate device memory, not
 * even a workspace: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation.  Same arguments, results and errors as
 * sparstar_score_blocks, without the workspace: its scratch (the pooled blocks
 * qbar and kbar, and S when `scores` is NULL) lives in a device array of
 * SPARSTAR_STATIC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends.  With `scores` given, S goes there and only
 * qbar + kbar and their scales use the scratch (41.9 MB at 24 heads, 72,000
 * queries and 144,512 keys in 64-token blocks); sizes that need more than the scratch
 * return SPARSTAR_ERR_WORKSPACE before any HIP call.
 *   - The call allocates nothing: no hipMalloc, hipFree or allocating library
 *     routine.  The first call on a device looks up the array's device address
 *     there (hipGetSymbolAddress) and keeps it.
 *   - Every call on one GPU shares that GPU's array, which keeps the contents
 *     of the last call; nothing in it needs to start at zero.  Calls that
 *     overlap on one GPU (concurrent streams, or host threads) race on it: the
 *     caller must order them.
 *   - Devices 0..63 are served; others return SPARSTAR_ERR_UNSUPPORTED.
 */
int sparstar_score_blocks_static(const void* q, const void* k, int B, int H, int64_t Lq, int64_t Lk, int D,
                                 int block_size, const double* budget, int n_budget, const sparstar_range* keep,
                                 int n_keep, int32_t* kv_num_blocks, int32_t* kv_indices, int kv_stride,
                                 float* scores, void* stream);

/* Most key blocks per row that sparstar_score_blocks_fused accepts. */
#define SPARSTAR_FUSED_MAX_BLOCKS 2304

/*
 * The selector of sparstar_score_blocks with the scores and the selection in
 * one kernel: S of 16 query blocks of one head is computed into LDS and each
 * row is selected from there, so S never reaches memory (the fusion that
 * Section 5.3's mask construction suggests).  Same arguments, results and
 * errors as sparstar_score_blocks with scores == NULL, except that rows of more
 * than SPARSTAR_FUSED_MAX_BLOCKS key blocks return SPARSTAR_ERR_UNSUPPORTED.
 * The scores are summed in another order than the separate score kernel's, so
 * a row whose k-th and (k+1)-th scores are within fp32 rounding may select
 * differently.  At the 720p shape (2258 key blocks) the separate kernels are
 * faster: one such work-group fills a CU's LDS, so its score and selection
 * phases cannot overlap those of another.
 */
int sparstar_score_blocks_fused(const void* q, const void* k, int B, int H, int64_t Lq, int64_t Lk, int D,
                                int block_size, const double* budget, int n_budget, const sparstar_range* keep,
                                int n_keep, int32_t* kv_num_blocks, int32_t* kv_indices, int kv_stride,
                                void* workspace, size_t workspace_bytes, void* stream);

/*
 * Bytes of device workspace that lets the attention calls below split the key
 * blocks of every query block into contiguous ranges and merge the partial
 * results.  Lists that can hold >= 24,576 keys (kv_stride x block_size; for
 * the dense call, every key block of the row) take 16 ranges (two per XCD of
 * the MI355X, taken one after the other, so that each XCD's L2 streams about
 * one sixteenth of a head's K/V at a time); shorter lists take 8, one per XCD,
 * where the fixed cost of each range outweighs the locality.  So the dense call
 * and a sparse call whose lists name every block, in order, give the same bits.
 * The workspace is sized for 16: per
 * (batch, head, query block, range, query row) the range's unnormalised
 * partial P V in fp16, scaled by a power of two chosen per row so that its
 * largest magnitude lies in [0.5, 1) ([.., D]; any finite bf16 range of V keeps
 * fp16's relative precision), and four fp32 values (running max, the row sums
 * of the bf16-rounded and of the unrounded softmax numerators, the row's
 * scale exponent).  0 when the key sequence has fewer than 16 blocks (no
 * split), and for invalid sizes.
 */
size_t sparstar_attn_workspace_bytes(int B, int H, int64_t Lq, int64_t Lk, int D, int block_size);

/*
 * Block-sparse attention forward over the lists of sparstar_score_blocks
 * (Eq. 7): query token t of block i attends to the key tokens u < Lk of the
 * blocks kv_indices[b,h,i,0 .. kv_num_blocks[b,h,i]).
 *   O_t   = sum_u softmax_u(s * q_t . k_u) v_u   (bf16 out, fp32 accumulation)
 *   lse_t = ln sum_u exp(s * q_t . k_u)          (fp32, natural log)
 * with s = softmax_scale, or D^-1/2 when softmax_scale <= 0.  A row whose list is
 * empty gets O = 0 and lse = -inf.  The softmax weights applied to V are
 * rounded to bf16 and O is normalised by their sum, so they sum to one exactly
 * (V = 1 gives O = 1); lse is taken from the sum of the unrounded fp32
 * weights.  Rows t >= Lq of a partial last query block are never written.
 *
 *   q, k, v         device bf16 Q [B,H,Lq,D], K and V [B,H,Lk,D].
 *   D, block_size   as for sparstar_score_blocks.
 *   kv_num_blocks, kv_indices, kv_stride   device, as written by
 *                   sparstar_score_blocks: each list ascending and
 *                   duplicate-free.  Defensively, a count is clamped to
 *                   [0, kv_stride] and an entry outside [0, n_k) is skipped, so
 *                   a malformed list gives unspecified values but never an
 *                   out-of-range access.
 *   o               device bf16 out [B,H,Lq,D].
 *   lse             device fp32 out [B,H,Lq], or NULL.
 *   workspace       NULL for a single pass, or device scratch of at least
 *                   sparstar_attn_workspace_bytes(...) bytes (256-byte aligned,
 *                   no initialisation needed, garbage afterwards) for the
 *                   key-range split.  The two paths round P relative to
 *                   different running maxima, so O agrees to the bf16 rounding
 *                   of P and O and lse to fp32 rounding.
 */
int sparstar_sparse_attn_fwd(const void* q, const void* k, const void* v, int B, int H, int64_t Lq, int64_t Lk,
                             int D, int block_size, const int32_t* kv_num_blocks, const int32_t* kv_indices,
                             int kv_stride, float softmax_scale, void* o, float* lse, void* workspace,
                             size_t workspace_bytes, void* stream);

/*
 * Dense attention forward with the same tile engine: every query attends to
 * all Lk keys (the FlashAttention-2 comparison of Section 6, and the dense
 * early scales).  Arguments as for sparstar_sparse_attn_fwd; the key tiles are
 * `block_size` tokens.
 */
int sparstar_dense_attn_fwd(const void* q, const void* k, const void* v, int B, int H, int64_t Lq, int64_t Lk, int D,
                            int block_size, float softmax_scale, void* o, float* lse, void* workspace,
                            size_t workspace_bytes, void* stream);

/*
 * Forced token ranges of Eq. 3 for clip `clip` (1-based; Section 5.2,
 * "Clip-Dependent Retained and Selectable Blocks"): clip 1 keeps the text and
 * the final image-pyramid reference dense, a clip c >= 2 keeps only the text
 * (its preceding-clip reference blocks are ranked jointly with the current
 * ones).  Host only; the result feeds the `keep` argument of
 * sparstar_score_blocks and sparstar_kv_stride.
 *   text, ref   token ranges [begin, end) of the two segments in the key
 *               sequence (0 <= begin <= end)
 *   out, cap    receive the ranges, text first; cap >= 2 always suffices
 * Returns the number of ranges written (1 or 2), or SPARSTAR_ERR_INVALID_ARG
 * for clip < 1, a malformed range, a NULL `out` or a `cap` below the count.
 */
int sparstar_clip_keep_ranges(int clip, sparstar_range text, sparstar_range ref, sparstar_range* out, int cap);

/*
 * Scale-wise density schedule (Section 5.2, Eq. 5, and the supplement's
 * "Sparsity Schedule and Later-Clip Policy"): the n_finest finest scales of a
 * clip group, in order of increasing token count, get the densities
 * finest_rho, and the lookup is by query length, so any scale with the token
 * count of a sparsified scale shares its density; all other scales stay dense.
 * The paper's 720p setting sparsifies the four finest scales with
 * (0.625, 0.1875, 0.1875, 0.09375) (native scales s26-s29 of clip 1; s38-s41 of
 * clip 2 in the ten-second evaluation, whose clip 1 is dense).  Host only.
 *   scale_lq     [n_scales] query length of every scale of the clip group, in
 *                generation order
 *   finest_rho   [n_finest] densities in [0, 1] of the last n_finest scales
 *   rho_out      [n_scales] receives rho of each scale, or -1.0 for a dense scale
 * Returns SPARSTAR_OK, or SPARSTAR_ERR_INVALID_ARG for n_finest > n_scales,
 * negative counts, NULL arrays with positive counts, a density outside [0, 1]
 * or two sparsified scales with equal token counts and different densities.
 */
int sparstar_scale_densities(const int64_t* scale_lq, int n_scales, const double* finest_rho, int n_finest,
                             double* rho_out);

/*
 * Retained attention mass (Section 4, the analysis of how much dense softmax
 * mass a selection keeps): for every query t,
 *   mass_t = sum over the selected keys u of softmax_u(s * q_t . k_u)
 *          = exp(lse_sel_t - lse_all_t),
 * where lse_sel is the log-sum-exp written by sparstar_sparse_attn_fwd and
 * lse_all the one written by sparstar_dense_attn_fwd on the same Q, K and
 * softmax scale.  A row with lse_sel = -inf (an empty list) gets 0.
 *   lse_sel, lse_all   device fp32 [n], 4-byte aligned
 *   mass               device fp32 out [n]; may be the same buffer as lse_sel
 * Returns SPARSTAR_OK, or SPARSTAR_ERR_INVALID_ARG for n < 0 or a NULL pointer
 * with n > 0.
 */
int sparstar_retained_mass(const float* lse_sel, const float* lse_all, int64_t n, float* mass, void* stream);

/* Upper bound on the sampled query rows of sparstar_token_topk_mass. */
#define SPARSTAR_MAX_MASS_ROWS 16

/*
 * Bytes of device scratch sparstar_token_topk_mass needs: the fp32 logits of
 * the sampled rows against every key, [B, H, n_rows, Lk].  0 for invalid sizes.
 */
size_t sparstar_token_topk_workspace_bytes(int B, int H, int64_t Lk, int n_rows);

/*
 * Token-wise upper bound of the retained mass (Section 4): for each (b, h) and
 * each sampled query position t = rows[r], the largest dense softmax mass any
 * n = n_tokens[b,h,r] keys can hold, i.e. the sum of the n largest weights
 *   exp(s * q_t . k_u - lse_all[b,h,t])   over u in [0, Lk).
 * The logits are recomputed in fp32 from the bf16 inputs; equal logits at the
 * n-th place fill the remaining places one weight each.
 *   q, k, B, H, Lq, Lk, D, softmax_scale   as for sparstar_dense_attn_fwd
 *                   (Lq >= 1, B * H <= 65535)
 *   rows, n_rows    HOST int64 [n_rows], 1 <= n_rows <= SPARSTAR_MAX_MASS_ROWS:
 *                   query positions in [0, Lq), the same for every (b, h)
 *   n_tokens        device int32 [B, H, n_rows]; each value is clamped to [0, Lk]
 *   lse_all         device fp32 [B, H, Lq], the dense log-sum-exp on the same
 *                   inputs and scale (sparstar_dense_attn_fwd)
 *   mass            device fp32 out [B, H, n_rows]
 *   workspace       device scratch of >= sparstar_token_topk_workspace_bytes(...)
 *                   bytes, 4-byte aligned, garbage afterwards
 * Returns SPARSTAR_OK or a negative code as for the other calls.
 */
int sparstar_token_topk_mass(const void* q, const void* k, int B, int H, int64_t Lq, int64_t Lk, int D,
                             const int64_t* rows, int n_rows, const int32_t* n_tokens, const float* lse_all,
                             float softmax_scale, float* mass, void* workspace, size_t workspace_bytes,
                             void* stream);

/* Message for the last non-OK return on this thread ("" if none). */
const char* sparstar_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SPARSTAR_H */

/*
 * hd.h -- C ABI of libhd.so: the Hidden Decoding hot path on AMD MI355X (gfx950).
 *
 * Paper: "Hidden Decoding at Scale: Latent Computation Scaling for Large Language
 * Models".  Notation used below (0-based, token-major interleave):
 *   L tokens, n streams, N = n*L expanded positions, expanded row p = t*n + s
 *   (eq. (expansion) places stream k of token i at physical position (i-1)n + k;
 *   eq. (indices) recovers token and stream from the position).
 *
 * Conventions shared by every entry point:
 *   - All tensor pointers are DEVICE pointers owned by the caller, 16-byte aligned,
 *     dense and row-major in the layouts stated per function.
 *   - The library never allocates, frees or synchronises device memory (the one
 *     device array it owns, the scratch of hd_sfa_decode_noalloc, is part of its code
 *     object).  Work is enqueued on `stream` (0 = the null stream) and the call returns
 *     after enqueue.
 *     Outputs are overwritten, never accumulated into (hd_embed_grad_scatter_add, whose
 *     purpose is to add into a dense gradient, is the one exception).
 *   - Arguments are validated on the host before anything is enqueued.  On a
 *     non-HD_OK return nothing has been enqueued, except for HD_ERR_HIP, which
 *     reports a launch failure; hd_last_error() then holds a readable detail.
 *   - Per-batch slices of the attention tensors (q, k, v, o, dO, dq, dk, dv and the
 *     decode caches) must stay below 2^31 bytes (32-bit offsets inside the kernels);
 *     larger inputs are rejected with HD_ERR_INVALID_ARG.  The expansion, its
 *     gradient and the final-stream gather state their own limits.
 *   - Calls are thread-safe with respect to each other; calls that write the same
 *     output buffers on overlapping streams race, as with any kernel.
 */
#ifndef HD_H
#define HD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t *hd_stream_t; /* a hipStream_t */

typedef enum {
    HD_OK = 0,
    HD_ERR_INVALID_ARG = 1, /* null pointer, bad size, misalignment, short workspace */
    HD_ERR_UNSUPPORTED = 2, /* valid request this build does not implement (e.g. D) */
    HD_ERR_HIP = 3          /* the HIP runtime reported an error at launch */
} hd_status_t;

/*
 * Attention mask of one Stream-Factorized Attention layer (Sec. "Stream-Factorized
 * Attention").  With t = p / n and s = p % n:
 *   HD_SFA_INTRA -- eq. (mask_intra): query p sees key p' iff s' == s and t' <= t
 *                   (intra-stream layer, Fig. "masks" panel (c)).
 *   HD_SFA_MIX   -- full cross-stream layer, Fig. "masks" panel (a): the standard
 *                   causal mask over the expanded sequence, i.e. t' < t, or t' == t
 *                   and s' <= s (p' <= p).
 *   HD_SFA_LOCAL -- local cross-stream layer, Fig. "masks" panel (b): the causal mask
 *                   of HD_SFA_MIX restricted to a sliding window of w expanded
 *                   positions, p - w < p' <= p.  The paper gives no w, so it is an
 *                   explicit argument of the *_local entry points below.
 */
typedef enum { HD_SFA_INTRA = 0, HD_SFA_MIX = 1, HD_SFA_LOCAL = 2 } hd_sfa_mode_t;

typedef enum { HD_DTYPE_BF16 = 0, HD_DTYPE_F32 = 1 } hd_dtype_t;

/*
 * hd_expand_embed -- multi-stream token expansion, eq. (expansion):
 *   out[b][t*n + s][:] = tables[s][ids[b][t]][:]     (tables[0] is the paper's E_1)
 *
 * ids          device int32 [B][L], token ids.
 * tables       device [n][V][Dm] of `dtype` (bf16 or f32), the n per-stream tables.
 * out          device [B][n*L][Dm] of `dtype`, overwritten.
 * bad_id_count device int32 (nullable).  For each id outside [0, V) the n rows of that
 *              token are written as zeros and *bad_id_count is incremented once (so
 *              the caller zeroes it first to obtain a count).
 * Errors: INVALID_ARG for null ids/tables/out, B, L, n, Dm <= 0, V <= 0,
 *         V > INT32_MAX, B*L >= 2^31, n*Dm*element size >= 2^31 bytes (one token's
 *         expanded rows), or unaligned pointers.
 */
hd_status_t hd_expand_embed(const int32_t *ids, const void *tables, void *out, int B, int L,
                            int n, int64_t V, int Dm, hd_dtype_t dtype,
                            int32_t *bad_id_count, hd_stream_t stream);

/*
 * hd_expand_embed_bwd -- gradient of eq. (expansion) with respect to the n tables.
 * The expansion is a gather, so for an upstream gradient dout of its output
 *   dtables[s][x][:] = sum over tokens (b, t) with ids[b][t] == x of dout[b][t*n + s][:]
 * (tokens whose id lies outside [0, V) contribute nothing).  The result is returned
 * sparse, for the distinct in-range ids of the batch only:
 *
 * ids        device int32 [B][L], the ids the forward expanded.
 * dout       device [B][n*L][Dm] of `dtype` (bf16 or f32).
 * uniq_ids   device int32 [B*L]: entries 0 .. *num_uniq-1 receive the distinct ids in
 *            ascending order; later entries are not written.
 * drows      device float [n][B*L][Dm]: drows[s][u][:] = dtables[s][uniq_ids[u]][:] for
 *            u < *num_uniq, summed in fp32 over the id's tokens in ascending (b, t)
 *            order (deterministic: no atomics); rows u >= *num_uniq are not written.
 * num_uniq   device int32, receives the number of distinct in-range ids.
 * workspace  device, 256-byte aligned, at least hd_expand_embed_bwd_workspace_bytes(B, L)
 *            bytes; contents on entry ignored, on exit unspecified.
 * Errors: INVALID_ARG for null pointers, sizes <= 0, V > INT32_MAX, B*L > 4194304,
 *         misaligned pointers (dout, drows 16 bytes; ids, uniq_ids, num_uniq 4 bytes) or
 *         a missing or short workspace.
 */
size_t hd_expand_embed_bwd_workspace_bytes(int B, int L);
hd_status_t hd_expand_embed_bwd(const int32_t *ids, const void *dout, int B, int L, int n,
                                int64_t V, int Dm, hd_dtype_t dtype, int32_t *uniq_ids,
                                float *drows, int32_t *num_uniq, void *workspace,
                                size_t workspace_bytes, hd_stream_t stream);

/*
 * hd_embed_grad_scatter_add -- adds the sparse table gradient of hd_expand_embed_bwd
 * into a dense one:  dtables[s][uniq_ids[u]][:] += drows[s][u][:]  for u < *num_uniq.
 * This entry point ACCUMULATES into dtables (the exception to the overwrite rule):
 * gradients of several batches add up before an optimizer step.  The ids are distinct,
 * so every destination row has one writer and the result is deterministic.
 *
 * uniq_ids, drows, num_uniq  as written by hd_expand_embed_bwd; max_rows is the row
 *            capacity B*L that drows was laid out with ([n][max_rows][Dm]).
 * dtables    device float [n][V][Dm].
 * Errors: INVALID_ARG for null pointers, sizes <= 0, V > INT32_MAX or pointers that are
 *         not 4-byte aligned.
 */
hd_status_t hd_embed_grad_scatter_add(const int32_t *uniq_ids, const float *drows,
                                      const int32_t *num_uniq, int max_rows, int n, int64_t V,
                                      int Dm, float *dtables, hd_stream_t stream);

/*
 * hd_cyclic_replicate -- Cyclic Replication Initialization, eq. (cyclic_init) (Sec.
 * "Progressive Expansion"): growing the expansion factor from n to m, a multiple of n,
 * the m tables become dst[s] = src[s mod n] (for m = 2n: E_{n+k} <- E_k; n = 2 -> 4
 * gives (E1, E2, E1, E2)).
 *
 * src  device [n][V][Dm] of `dtype`;  dst  device [m][V][Dm] of `dtype`, overwritten.
 * dst may be the same buffer as src (growth in place: src then has room for m tables
 * and only tables n .. m-1 are written); any other overlap is rejected.
 * Errors: INVALID_ARG for null or unaligned (16-byte) pointers, n <= 0, m not a
 *         multiple of n or above 65535, V or Dm <= 0, or overlapping buffers.
 */
hd_status_t hd_cyclic_replicate(const void *src, void *dst, int n, int m, int64_t V, int Dm,
                                hd_dtype_t dtype, hd_stream_t stream);

/*
 * hd_final_stream_gather -- the input of the training loss, eq. (hd_loss) (Sec. "Training
 * objective"): only the final stream of each token is supervised, so the loss reads token
 * i's hidden state at expanded position i*n + n - 1 (the paper's t = i n, 1-based):
 *   out[b][i][:] = h[b][i*n + n - 1][:]
 *
 * h    device [B][n*L][Dm] of `dtype` (bf16 or f32), the last layer's hidden states.
 * out  device [B][L][Dm] of `dtype`, overwritten; must not overlap h.
 * Errors: INVALID_ARG for null or unaligned (16-byte) pointers, B, L, n, Dm <= 0,
 *         B*n*L > INT32_MAX, an output of 2^31 copy words or more (16-byte words when
 *         Dm*esize is a multiple of 16, else 4- or 2-byte words), or overlapping buffers.
 */
hd_status_t hd_final_stream_gather(const void *h, void *out, int B, int L, int n, int Dm,
                                   hd_dtype_t dtype, hd_stream_t stream);

/*
 * hd_final_stream_gather_bwd -- its adjoint: the gradient with respect to h of a loss on
 * the gathered rows,
 *   dh[b][i*n + n - 1][:] = dout[b][i][:],   dh[b][i*n + s][:] = 0 for s < n - 1
 * (the first n - 1 streams of a token receive no direct loss).
 *
 * dout device [B][L][Dm] of `dtype`;  dh  device [B][n*L][Dm] of `dtype`, overwritten in
 *      full; must not overlap dout.
 * Errors: as hd_final_stream_gather (the size limit applies to dh).
 */
hd_status_t hd_final_stream_gather_bwd(const void *dout, void *dh, int B, int L, int n, int Dm,
                                       hd_dtype_t dtype, hd_stream_t stream);

/*
 * hd_sfa_fwd -- Stream-Factorized Attention forward over the expanded sequence.
 *   O_p = sum_{p' visible from p} softmax_p'(scale * q_p . k_p') v_p'
 *   lse_p = log sum_{p' visible} exp(scale * q_p . k_p')       (natural log)
 * with the visibility of `mode` (eq. (mask_intra) or the full causal mask).
 *
 * q, o   device [B][N][Hq][D]  of `dtype`.
 * k, v   device [B][N][Hkv][D] of `dtype`; query head h uses key/value head
 *        h / (Hq / Hkv) (grouped-query attention, contiguous groups).
 * lse    device float [B][Hq][N].
 * scale  softmax scale, finite and > 0 (typically 1/sqrt(D)), used exactly as given.
 * Every row sees at least its own key, so no row is empty and no output is NaN for
 * finite inputs.  INTRA reads only the keys of the query's own stream.
 * Errors: INVALID_ARG for null pointers, any size <= 0, Hq % Hkv != 0, bad scale,
 *         misalignment or oversize tensors, or mode HD_SFA_LOCAL (which needs a window:
 *         hd_sfa_fwd_local); UNSUPPORTED for D not in {32, 64, 128}.
 */
hd_status_t hd_sfa_fwd(const void *q, const void *k, const void *v, void *o, float *lse,
                       int B, int L, int n, int Hq, int Hkv, int D, hd_sfa_mode_t mode,
                       float scale, hd_dtype_t dtype, hd_stream_t stream);

/*
 * hd_sfa_fwd_local -- hd_sfa_fwd for a local cross-stream layer (Fig. "masks" panel
 * (b)): query p sees keys p' with p - window < p' <= p, so every row sees its own key
 * and at most `window` keys in all.  window >= N gives the HD_SFA_MIX result.  Only the
 * key tiles that meet a query tile's window are read, so the cost is O(N * window).
 * Arguments, layouts and errors as hd_sfa_fwd, plus INVALID_ARG for window < 1.
 */
hd_status_t hd_sfa_fwd_local(const void *q, const void *k, const void *v, void *o, float *lse,
                             int B, int L, int n, int Hq, int Hkv, int D, int window,
                             float scale, hd_dtype_t dtype, hd_stream_t stream);

/*
 * hd_sfa_bwd_workspace_bytes -- device workspace hd_sfa_bwd needs for these sizes:
 * two fp32 statistics per query row ([B][Hq][N] each), and for bf16 the tiles of
 * dS = P (dP - Delta) in bf16, 16 KB per 64 query rows x 128 keys that hold a visible
 * pair (about B*Hq*N*N bytes for HD_SFA_MIX, B*Hq*n*L*L for HD_SFA_INTRA).  For
 * HD_SFA_LOCAL it returns the HD_SFA_MIX size, which is enough for every window;
 * hd_sfa_bwd_local_workspace_bytes gives the (smaller) size for one window.
 * Returns 0 for arguments hd_sfa_bwd would reject.
 */
size_t hd_sfa_bwd_workspace_bytes(int B, int L, int n, int Hq, int Hkv, int D,
                                  hd_sfa_mode_t mode, hd_dtype_t dtype);

/*
 * hd_sfa_bwd_min_workspace_bytes -- the smallest workspace hd_sfa_bwd accepts for these
 * sizes.  For bf16 a workspace below hd_sfa_bwd_workspace_bytes(...) runs the backward
 * in query bands: the query rows are taken in bands of whole 256-row units, and each
 * band's dK/dV pass stores only that band's dS tiles, which its dQ pass then reads; dK
 * and dV are carried from band to band as fp32 partials.  The smallest workspace holds
 * the two row statistics, those partials (2 * B*N*Hkv*D fp32) and the dS tiles of the
 * largest 256-row unit (about 2*B*Hq*256*N bytes for HD_SFA_MIX), so it grows linearly
 * in N.  Bands take whatever room the workspace leaves, so more workspace means fewer
 * and larger bands; results agree with the one-pass run to fp32 summation order (the
 * band partials are added in a fixed order, so every run is deterministic).  For fp32
 * (no dS tiles) it equals hd_sfa_bwd_workspace_bytes.  For HD_SFA_LOCAL it returns the
 * HD_SFA_MIX size.  Returns 0 for arguments hd_sfa_bwd would reject.
 */
size_t hd_sfa_bwd_min_workspace_bytes(int B, int L, int n, int Hq, int Hkv, int D,
                                      hd_sfa_mode_t mode, hd_dtype_t dtype);

/*
 * hd_sfa_bwd_local_workspace_bytes -- workspace hd_sfa_bwd_local needs for a local
 * cross-stream layer of the given window (for bf16 about 2*B*Hq*N*window bytes of dS
 * tiles when the window is well below N).  Returns 0 for arguments hd_sfa_bwd_local would reject.
 */
size_t hd_sfa_bwd_local_workspace_bytes(int B, int L, int n, int Hq, int Hkv, int D, int window,
                                        hd_dtype_t dtype);
/* hd_sfa_bwd_local_min_workspace_bytes -- the smallest workspace hd_sfa_bwd_local accepts
 * for this window (query bands as for hd_sfa_bwd_min_workspace_bytes).  Returns 0 for
 * arguments hd_sfa_bwd_local would reject. */
size_t hd_sfa_bwd_local_min_workspace_bytes(int B, int L, int n, int Hq, int Hkv, int D,
                                            int window, hd_dtype_t dtype);

/*
 * hd_sfa_bwd -- gradients of the forward above, recomputing the attention
 * probabilities from q, k and the forward's lse:
 *   P = exp(scale q k^T - lse), dP = dO v^T, Delta = rowsum(dO * O),
 *   dS = P * (dP - Delta), dq = scale dS k, dk = scale dS^T q, dv = P^T dO,
 * dk/dv summed over the query heads of each key/value group.
 *
 * q, o, dO, dq  device [B][N][Hq][D] of `dtype`;  k, v, dk, dv  device [B][N][Hkv][D].
 * lse           device float [B][Hq][N] exactly as written by hd_sfa_fwd.
 * workspace     device, 256-byte aligned, at least hd_sfa_bwd_min_workspace_bytes(...)
 *               bytes (workspace_bytes gives its size); contents on entry are ignored
 *               and on exit unspecified.  The bf16 path stores dS there in its dK/dV
 *               pass and its dQ pass reads it back, so dQ costs one product instead of
 *               a recomputation of S and dP.  With hd_sfa_bwd_workspace_bytes(...) or
 *               more this is one pass over all query rows (the fastest); with less, a
 *               sequence of query bands (see hd_sfa_bwd_min_workspace_bytes).
 * Errors: as hd_sfa_fwd, plus INVALID_ARG for a missing workspace or one below
 *         hd_sfa_bwd_min_workspace_bytes(...).
 */
hd_status_t hd_sfa_bwd(const void *q, const void *k, const void *v, const void *o,
                       const float *lse, const void *dO, void *dq, void *dk, void *dv, int B,
                       int L, int n, int Hq, int Hkv, int D, hd_sfa_mode_t mode, float scale,
                       hd_dtype_t dtype, void *workspace, size_t workspace_bytes,
                       hd_stream_t stream);

/*
 * hd_sfa_bwd_local -- hd_sfa_bwd for a local cross-stream layer (Fig. "masks" panel
 * (b)) of the given window; lse as written by hd_sfa_fwd_local with the same window,
 * workspace of at least hd_sfa_bwd_local_min_workspace_bytes(..., window, dtype) bytes
 * (one pass from hd_sfa_bwd_local_workspace_bytes(..., window, dtype) bytes up).
 * Arguments, layouts and errors as hd_sfa_bwd, plus INVALID_ARG for window < 1.
 */
hd_status_t hd_sfa_bwd_local(const void *q, const void *k, const void *v, const void *o,
                             const float *lse, const void *dO, void *dq, void *dk, void *dv,
                             int B, int L, int n, int Hq, int Hkv, int D, int window,
                             float scale, hd_dtype_t dtype, void *workspace,
                             size_t workspace_bytes, hd_stream_t stream);

/*
 * Final-stream layers (Sec. "Training Cost", KV-mirror): in the mirrored layers only the
 * final stream of each token is run, while keys and values cover all n streams (they
 * come from an earlier layer).  Query row t of these layers sits at expanded position
 * t*n + n - 1 and sees, with window == 0, every key p' <= t*n + n - 1 (the full
 * cross-stream mask of HD_SFA_MIX), or with window >= 1 the keys
 * t*n + n - 1 - window < p' <= t*n + n - 1 (the local mask of HD_SFA_LOCAL).  An
 * intra-stream mirrored layer needs no entry point of its own: it is plain causal
 * attention over the final-stream rows.
 *
 * hd_sfa_fwd_final
 *   q, o   device [B][L][Hq][D] bf16 (final-stream rows only).
 *   k, v   device [B][n*L][Hkv][D] bf16, all expanded rows.
 *   lse    device float [B][Hq][L], natural log.
 * hd_sfa_bwd_final
 *   dO, dq device [B][L][Hq][D];  dk, dv  device [B][n*L][Hkv][D] (summed over the query
 *   heads of each group; keys that no final-stream query sees get zero);
 *   workspace of at least hd_sfa_bwd_final_min_workspace_bytes(...) bytes;
 *   hd_sfa_bwd_final_workspace_bytes(...) (the two row statistics per query row and the
 *   bf16 dS tiles: 16 KB per 64 query rows x 128 keys of a key band, about
 *   2*B*Hq*L*n*L bytes without a window) or more runs it in one pass, less in query
 *   bands.
 * Other arguments, conventions and errors as hd_sfa_fwd / hd_sfa_bwd, plus INVALID_ARG
 * for window < 0 and UNSUPPORTED for dtype HD_DTYPE_F32 or n > 63.
 */
hd_status_t hd_sfa_fwd_final(const void *q, const void *k, const void *v, void *o, float *lse,
                             int B, int L, int n, int Hq, int Hkv, int D, int window,
                             float scale, hd_dtype_t dtype, hd_stream_t stream);
size_t hd_sfa_bwd_final_workspace_bytes(int B, int L, int n, int Hq, int Hkv, int D, int window,
                                        hd_dtype_t dtype);
/* the smallest workspace hd_sfa_bwd_final accepts (query bands as for hd_sfa_bwd) */
size_t hd_sfa_bwd_final_min_workspace_bytes(int B, int L, int n, int Hq, int Hkv, int D,
                                            int window, hd_dtype_t dtype);
hd_status_t hd_sfa_bwd_final(const void *q, const void *k, const void *v, const void *o,
                             const float *lse, const void *dO, void *dq, void *dk, void *dv,
                             int B, int L, int n, int Hq, int Hkv, int D, int window,
                             float scale, hd_dtype_t dtype, void *workspace,
                             size_t workspace_bytes, hd_stream_t stream);

/*
 * hd_sfa_decode -- parallel-stream decode (Sec. "Inference Cost": at a decode step the
 * n streams of a sequence's new token are processed together in one pass).  For every sequence b with
 * ctx_tokens[b] = c tokens before the new one, query row s (stream s of the new token,
 * expanded position c*n + s) attends under `mode`'s mask to the sequence's cached rows:
 *   HD_SFA_INTRA: rows t*n + s for t <= c (its own stream: 1/n of the cache);
 *   HD_SFA_MIX  : rows p' <= c*n + s;
 *   HD_SFA_LOCAL: rows c*n + s - window < p' <= c*n + s.
 * The new token's own keys and values must already be in the cache (rows c*n .. c*n+n-1);
 * rows past c*n + n - 1 are never read.  Forward only.
 *
 * q               device bf16 [B][n][Hq][D], the new token's n query rows per sequence.
 * k_cache,v_cache device bf16 [B][n*Lcap][Hkv][D], expanded rows p = t*n + s (grouped
 *                 heads as in hd_sfa_fwd).
 * ctx_tokens      device int32 [B], each in [0, max_ctx_tokens].
 * max_ctx_tokens  host bound on ctx_tokens (sizes the launch and the workspace), < Lcap.
 * o               device bf16 [B][n][Hq][D];  lse  device float [B][Hq][n] (natural log).
 * window          the local window (HD_SFA_LOCAL, >= 1); ignored by the other modes.
 * workspace       device, 256-byte aligned, hd_sfa_decode_workspace_bytes(...) bytes:
 *                 fp32 partial results per 256 cached rows.
 * Errors: INVALID_ARG for null or misaligned pointers, sizes <= 0, Hq % Hkv != 0, a bad
 *         mode, window or scale, max_ctx_tokens outside [0, Lcap), oversize tensors or a
 *         short workspace; UNSUPPORTED for fp32 or D not in {32, 64, 128}.
 */
size_t hd_sfa_decode_workspace_bytes(int B, int Lcap, int n, int Hq, int Hkv, int D,
                                     hd_sfa_mode_t mode, int window, int max_ctx_tokens);
hd_status_t hd_sfa_decode(const void *q, const void *k_cache, const void *v_cache,
                          const int32_t *ctx_tokens, int max_ctx_tokens, void *o, float *lse,
                          int B, int Lcap, int n, int Hq, int Hkv, int D, hd_sfa_mode_t mode,
                          int window, float scale, hd_dtype_t dtype, void *workspace,
                          size_t workspace_bytes, hd_stream_t stream);

/*
 * hd_sfa_decode_noalloc -- hd_sfa_decode for callers that cannot allocate device memory
 * (code under HIP graph capture, serving loops that must not call the allocator): the
 * same computation, arguments and results, with the fp32 partials kept in a scratch
 * array that the library holds on each GPU it runs on, from the first such call on that
 * GPU until the process ends.  The call allocates nothing.
 *
 * Limit: the partials of one call, hd_sfa_decode_workspace_bytes(...) for the same
 * arguments, must fit the scratch, hd_sfa_decode_noalloc_max_bytes() = 128 MiB
 * (for example 16 sequences of 4096 tokens at n=4, 32 query / 8 key-value heads of
 * width 128, in any mode); larger requests return HD_ERR_INVALID_ARG with nothing
 * enqueued.
 * Every call on a GPU uses that GPU's one scratch array: calls that can run at the same
 * time on one GPU (different streams, or different host threads without ordering)
 * race and corrupt each other's results; calls on one stream are ordered.  The first
 * call on a GPU looks the array's address up (hipGetSymbolAddress) and may therefore
 * return HD_ERR_HIP if the runtime fails.
 * Errors: as hd_sfa_decode (without the workspace ones), plus INVALID_ARG for sizes
 * beyond the limit.
 */
hd_status_t hd_sfa_decode_noalloc(const void *q, const void *k_cache, const void *v_cache,
                                  const int32_t *ctx_tokens, int max_ctx_tokens, void *o,
                                  float *lse, int B, int Lcap, int n, int Hq, int Hkv, int D,
                                  hd_sfa_mode_t mode, int window, float scale, hd_dtype_t dtype,
                                  hd_stream_t stream);
size_t hd_sfa_decode_noalloc_max_bytes(void);

/* Static name of a status code ("HD_OK", ...). */
const char *hd_status_str(hd_status_t s);

/* Detail of the last non-OK return on the calling thread ("" if none). */
const char *hd_last_error(void);

/*
 * Per-kernel timing (diagnostics, not needed for normal use).  While enabled, every
 * kernel the library launches is bracketed by a pair of HIP events recorded on the
 * launch stream (event objects are created on first use and reused).
 * hd_timing_filter restricts this to kernels whose timing name starts with `prefix`
 * (NULL or "" restores all; the string is copied), so that a measurement can bracket
 * one kernel without adding events around the others.
 * hd_timing_collect waits for the recorded events, writes up to `max` entries of
 * accumulated (kernel name, launch count, total milliseconds) and clears the record.
 * Returns the number of entries written, or -1 on a HIP error.
 */
typedef struct {
    char name[64];
    int launches;
    double total_ms;
} hd_kernel_time_t;

hd_status_t hd_timing_enable(int enable);
hd_status_t hd_timing_filter(const char *prefix);
int hd_timing_collect(hd_kernel_time_t *out, int max);

#ifdef __cplusplus
}
#endif

#endif /* HD_H */

/*
 * h2o.h - C ABI of libh2o.so, the MI355X (gfx950) H2O chunk step.
 *
 * One chunk step of sparse attention with the heavy-hitter-oracle (H2O) cache
 * policy, as stated in "Learning how to Forget: Fine-tuning for Long-Context
 * Sparse Attention":
 *
 *   1. h2o_sdpa_chunk: scaled dot-product attention of the chunk's T queries
 *      over [M cache slots || the chunk's T keys] (Eq. main-sdpa,
 *      Eq. main-sdpa-comp), causal inside the chunk (the token-position mask of
 *      Sec. "Discussion: SDPA Kernels for Sparse Attention"; every cache token
 *      precedes the chunk), returning the output, the per-row log-sum-exp and
 *      the summed attention weights sum_i m_{i,j} per key column (Sec.
 *      "Variants of Heavy-Hitter Oracle", Sec. "Computing Summed Attention
 *      Weights in SDPA"), summed over the query heads of each GQA group.
 *   2. h2o_accumulate_scores: the running H2O score phi += sum_i m_{i,j}
 *      (Eq. h2o-score) for the M cache slots.
 *   3. h2o_evict_insert: per (batch, KV head) overwrite the k slots with the
 *      smallest score (Sec. "Variants of Heavy-Hitter Oracle") by the chunk's
 *      keys and values - the scatter of Sec. "Fine-Tuning for Sparse
 *      Attention" along the slot axis (Sec. "Buffer Read/Write Access by
 *      torch.scatter, torch.gather").
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers are device pointers (HIP global memory) unless stated. All
 *    tensors are dense, C-contiguous, 16-byte aligned, and owned by the
 *    caller; the library never keeps a pointer after the call returns.
 *  - Shapes (row-major):
 *        q, out            [B, Hq,  T, d]       dtype
 *        k_cache, v_cache  [B, Hkv, M, d]       dtype
 *        k_new, v_new      [B, Hkv, T, d]       dtype
 *        lse               [B, Hq,  T]          float32
 *        wsum              [B, Hkv, M + T]      float32
 *        scores            [B, Hkv, M]          float32
 *        token_pos         [B, Hkv, M]          int32
 *        evict_idx         [B, Hkv, k]          int32
 *    Query head hq belongs to KV head hq / (Hq / Hkv) (contiguous groups).
 *    Key column j < M is cache slot j; column M + t is chunk key t.
 *  - dtype: H2O_F32 (float32) or H2O_BF16 (bfloat16). lse, wsum and scores
 *    are float32 in both modes.
 *  - stream: a hipStream_t passed as void* (NULL = the null stream). Work is
 *    only enqueued; nothing synchronises. A device fault surfaces at the
 *    caller's next synchronisation.
 *  - Errors: every function returns an h2o_status. Arguments are validated
 *    on the host before anything is enqueued, so on error no buffer is
 *    touched. h2o_last_error() returns a message for the calling thread's
 *    last non-OK status.
 *  - Calls that share buffers must be ordered by the caller (same stream).
 */
#ifndef H2O_H
#define H2O_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  H2O_OK = 0,
  H2O_EINVAL = 1,      /* null pointer, k != T, T < 1, M < k, bad scale     */
  H2O_ESHAPE = 2,      /* Hq % Hkv != 0, d not in {64,128}, sizes <= 0, or
                          (M+T)*d or (Hq/Hkv)*T*d >= 2^30 elements per head   */
  H2O_EDTYPE = 3,      /* dtype not H2O_F32 / H2O_BF16                        */
  H2O_EALIGN = 4,      /* a tensor pointer is not 16-byte aligned             */
  H2O_EWORKSPACE = 5,  /* workspace smaller than h2o_workspace_bytes()        */
  H2O_ENODEVICE = 6,   /* no usable gfx950 device                             */
  H2O_ELAUNCH = 7      /* a kernel launch failed                              */
} h2o_status;

typedef enum { H2O_F32 = 0, H2O_BF16 = 1 } h2o_dtype;

/* The ranking the eviction uses (Sec. "Variants of Heavy-Hitter Oracle"):
 *   H2O_POLICY_H2O   the accumulated score phi itself, per (b, KV head)
 *   H2O_POLICY_NORM  h2o_norm: phi divided by the slot's age t - token_pos,
 *                    t = pos0 + T (the tokens processed, this chunk
 *                    included); one correctly rounded float32 division per
 *                    slot; every age must lie in [1, 2^24) (not checked:
 *                    it is device data)
 *   H2O_POLICY_ORIG  h2o_orig: phi summed over the batch (float32 additions
 *                    in increasing b), one slot set per KV head shared by
 *                    every batch entry */
typedef enum {
  H2O_POLICY_H2O = 0,
  H2O_POLICY_NORM = 1,
  H2O_POLICY_ORIG = 2
} h2o_policy;

/* Bytes of device scratch h2o_sdpa_chunk needs for this shape (0 on invalid
 * arguments). The workspace holds partial row statistics and per-row-tile
 * partial column sums; its contents on entry are ignored. */
size_t h2o_workspace_bytes(int B, int Hq, int Hkv, int T, int M, int d,
                           int dtype);

/* SDPA of the chunk over [cache || chunk] plus summed attention weights.
 *
 *   out[b,hq,i,:] = sum_j m_{i,j} V_j,  m_{i,j} = exp(s_{i,j} - lse[b,hq,i])
 *   s_{i,j} = scale * <q[b,hq,i], K_j>  for visible (i,j), where
 *            K_j = k_cache[b,h,j] (j < M, always visible) or
 *                  k_new[b,h,j-M] (visible iff j-M <= i), h = hq / (Hq/Hkv)
 *   lse[b,hq,i]  = log sum_{visible j} exp(s_{i,j})        (natural log)
 *   wsum[b,h,j]  = sum_{hq in group h} sum_i m_{i,j}         (written, not
 *                  accumulated; invisible pairs contribute 0)
 *
 * scale is usually 1/sqrt(d) and must be finite and > 0. T >= 1, M >= 0.
 * With dtype H2O_BF16 the products run on bf16 MFMA with float32
 * accumulation, the softmax and all sums are float32 and out is rounded to
 * bf16 (nearest even). out must not alias any input. */
int h2o_sdpa_chunk(const void* q, const void* k_cache, const void* v_cache,
                   const void* k_new, const void* v_new, void* out, float* lse,
                   float* wsum, void* workspace, size_t workspace_bytes, int B,
                   int Hq, int Hkv, int T, int M, int d, float scale,
                   int dtype, void* stream);

/* scores[b,h,j] += wsum[b,h,j] for j < M: one IEEE float32 addition per slot
 * (Eq. h2o-score as a running sum over chunks). wsum has M + T columns; only
 * the first M are read. scores and wsum must not overlap. */
int h2o_accumulate_scores(float* scores, const float* wsum, int B, int Hkv,
                          int M, int T, void* stream);

/* Eviction and insert for one chunk (k == T: every chunk key is inserted).
 * Per (b,h): E = the k slots j < M with the smallest (scores[j], j) in
 * lexicographic order (score first, lower slot wins ties, -0.0 == +0.0;
 * scores must not be NaN), written to evict_idx in ascending slot order.
 * Then for i < k, with slot = E[i]:
 *   k_cache[b,h,slot,:] = k_new[b,h,i,:],  v_cache[b,h,slot,:] = v_new[b,h,i,:]
 *   scores[b,h,slot]    = wsum[b,h,M+i]    (the new key's own summed weight)
 *   token_pos[b,h,slot] = pos0 + i         (skipped when token_pos is NULL)
 * All other slots are unchanged. Inputs k_new/v_new/wsum must not overlap
 * the buffers written. */
int h2o_evict_insert(void* k_cache, void* v_cache, float* scores,
                     int32_t* token_pos, const void* k_new, const void* v_new,
                     const float* wsum, int32_t* evict_idx, int B, int Hkv,
                     int M, int T, int d, int k, int32_t pos0, int dtype,
                     void* stream);

/* h2o_chunk_step in two calls with the same arguments, for callers that
 * overlap the cache maintenance of one layer with the attention of the next
 * (the eviction of a layer is not needed by the next layer's queries):
 *   h2o_chunk_step_attend  writes out and lse (and, except on the T == 1
 *                          bf16 path, wsum);
 *   h2o_chunk_step_evict   completes wsum, accumulates the scores, picks the
 *                          slots and inserts the chunk.
 * The evict call reads what the attend call left in the workspace: it must
 * run after the attend call (same stream, or an event between streams), and
 * nothing may use the workspace, scores, cache or token_pos of this state in
 * between. Together they give the bits of h2o_chunk_step. */
int h2o_chunk_step_attend(const void* q, void* k_cache, void* v_cache,
                          float* scores, int32_t* token_pos, const void* k_new,
                          const void* v_new, void* out, float* lse, float* wsum,
                          int32_t* evict_idx, void* workspace,
                          size_t workspace_bytes, int B, int Hq, int Hkv, int T,
                          int M, int d, float scale, int32_t pos0, int dtype,
                          void* stream);
int h2o_chunk_step_evict(const void* q, void* k_cache, void* v_cache,
                         float* scores, int32_t* token_pos, const void* k_new,
                         const void* v_new, void* out, float* lse, float* wsum,
                         int32_t* evict_idx, void* workspace,
                         size_t workspace_bytes, int B, int Hq, int Hkv, int T,
                         int M, int d, float scale, int32_t pos0, int dtype,
                         void* stream);

/* Bytes of device scratch h2o_evict_insert_policy needs (0 for
 * H2O_POLICY_H2O and on invalid arguments): the ranked keys (NORM: B*Hkv*M
 * floats; ORIG: Hkv*M floats plus Hkv*k indices). */
size_t h2o_evict_workspace_bytes(int B, int Hkv, int M, int k, int policy);

/* h2o_evict_insert with the ranking of `policy` (an h2o_policy). E is the k
 * slots with the smallest (key, slot) where key is the policy's value for
 * the slot; for H2O_POLICY_ORIG the E of KV head h is the same for every b.
 * The insert is that of h2o_evict_insert: the new slots take the new key's
 * own summed weight wsum[b,h,M+i] as their (unnormalised) score and pos0 + i
 * as their position. H2O_POLICY_NORM needs token_pos (the ages); the
 * others accept NULL. workspace holds at least h2o_evict_workspace_bytes()
 * (H2O_EWORKSPACE otherwise; NULL is fine when that is 0), its contents on
 * entry are ignored. With H2O_POLICY_H2O the result is that of
 * h2o_evict_insert, bit for bit. */
int h2o_evict_insert_policy(void* k_cache, void* v_cache, float* scores,
                            int32_t* token_pos, const void* k_new,
                            const void* v_new, const float* wsum,
                            int32_t* evict_idx, int B, int Hkv, int M, int T,
                            int d, int k, int32_t pos0, int dtype, int policy,
                            void* workspace, size_t workspace_bytes,
                            void* stream);

/* The three calls above in one: h2o_sdpa_chunk, then h2o_accumulate_scores,
 * then h2o_evict_insert with k = T (the step of Sec. "Fine-Tuning for Sparse
 * Attention": attend over cache and chunk, add the summed weights to the H2O
 * scores of Eq. h2o-score, overwrite the T lowest-scored slots with the
 * chunk). Arguments and results are those of the three calls (same bits);
 * every buffer they read or write is an argument here, the workspace is the
 * one h2o_workspace_bytes() sizes, and M >= T. For T == 1 in bf16 the step
 * is two kernel launches: the split attention kernel, then one block per KV
 * head that merges the splits, accumulates the scores, picks the slot and
 * inserts; other shapes run the kernels of the three calls in order. */
int h2o_chunk_step(const void* q, void* k_cache, void* v_cache, float* scores,
                   int32_t* token_pos, const void* k_new, const void* v_new,
                   void* out, float* lse, float* wsum, int32_t* evict_idx,
                   void* workspace, size_t workspace_bytes, int B, int Hq,
                   int Hkv, int T, int M, int d, float scale, int32_t pos0,
                   int dtype, void* stream);

/* h2o_chunk_step without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation). Arguments, results and errors are those
 * of h2o_chunk_step (same kernels, same bits), with the scratch taken from a
 * fixed array of h2o_noalloc_scratch_bytes() bytes (32 MiB) inside the
 * library instead: one array per GPU the library runs on, held until the
 * process ends. No call allocates or frees memory. A shape whose
 * h2o_workspace_bytes() exceeds the array returns H2O_EWORKSPACE before
 * anything is enqueued (the decode shape B8 Hq32 Hkv8 d64 M4096 needs about
 * 8 MiB). Every call on one GPU shares that GPU's array, and the array keeps
 * what the last call left there (no kernel reads it before writing it), so
 * calls that can overlap on one GPU - different streams, host threads -
 * race and must be ordered by the caller. */
size_t h2o_noalloc_scratch_bytes(void);
int h2o_chunk_step_noalloc(const void* q, void* k_cache, void* v_cache, float* scores,
                           int32_t* token_pos, const void* k_new, const void* v_new, void* out,
                           float* lse, float* wsum, int32_t* evict_idx, int B, int Hq, int Hkv,
                           int T, int M, int d, float scale, int32_t pos0, int dtype,
                           void* stream);

/* ---- The paper's order of a chunk step: insert, then attend (Sec.
 * "Discussion: SDPA Kernels for Sparse Attention"). The chunk is written into
 * the cache first and the attention masks each slot by its token position:
 * slot j is visible to chunk query i iff token_pos[b,h,j] <= pos0 + i (the
 * causal mask of sparse attention, -inf * 1{P + i < t(b,h,j)} with P = pos0),
 * for any int32 positions, monotone or not. */

/* Bytes of device scratch for h2o_sdpa_cache (policy H2O_POLICY_H2O) or for
 * h2o_chunk_step_insert_first with `policy` (0 on invalid arguments). */
size_t h2o_cache_workspace_bytes(int B, int Hq, int Hkv, int T, int M, int d,
                                 int dtype, int policy);

/* Attention of T queries (token positions pos0 .. pos0+T-1) over the M >= 1
 * cache slots alone, masked by token_pos [B,Hkv,M] (int32, read only):
 *   out[b,hq,i,:] = sum_j m_{i,j} v_cache[b,h,j,:] over visible slots j,
 *   lse[b,hq,i]   = log sum_{visible j} exp(s_{i,j}),
 *   wsum[b,h,j]   = sum_{hq in group h} sum_i m_{i,j}   ([B,Hkv,M], written)
 * with s_{i,j} as in h2o_sdpa_chunk. A query that sees no slot gets out 0
 * and lse -inf and adds nothing to wsum. Other arguments, precision and
 * errors as for h2o_sdpa_chunk; workspace of h2o_cache_workspace_bytes(...,
 * H2O_POLICY_H2O). */
int h2o_sdpa_cache(const void* q, const void* k_cache, const void* v_cache,
                   const int32_t* token_pos, void* out, float* lse, float* wsum,
                   void* workspace, size_t workspace_bytes, int B, int Hq, int Hkv,
                   int T, int M, int d, float scale, int32_t pos0, int dtype,
                   void* stream);

/* One chunk step in the paper's order (Sec. "Sparse Attention. Key-Value
 * Caching", the mask of Sec. "Discussion: SDPA Kernels for Sparse
 * Attention"), M >= T:
 *   1. E = the T slots ranked lowest by `policy` (an h2o_policy) on the
 *      scores after pos0 tokens (h2o_norm: ages pos0 - token_pos, which must
 *      lie in [1, 2^24)), in ascending slot order, into evict_idx [B,Hkv,T];
 *   2. chunk key/value i goes to slot E[i], with token_pos pos0 + i and
 *      score 0 (Eq. h2o-score sums from the slot's own position);
 *   3. h2o_sdpa_cache over the updated cache (out, lse, wsum [B,Hkv,M]);
 *   4. scores[b,h,j] += wsum[b,h,j] for all M slots (one float32 addition).
 * token_pos is required. Workspace of h2o_cache_workspace_bytes(..., policy);
 * its contents on entry are ignored. For T == 1 in bf16 with H2O_POLICY_H2O
 * the step is two kernel launches (the attention kernel picks the slot and
 * attends with the chunk's row already in place, then one kernel merges the
 * splits and accumulates), with the same results as steps 1-4 in turn. */
int h2o_chunk_step_insert_first(const void* q, void* k_cache, void* v_cache,
                                float* scores, int32_t* token_pos,
                                const void* k_new, const void* v_new, void* out,
                                float* lse, float* wsum, int32_t* evict_idx,
                                void* workspace, size_t workspace_bytes, int B,
                                int Hq, int Hkv, int T, int M, int d, float scale,
                                int32_t pos0, int dtype, int policy, void* stream);

/* ---- Fine-tuning (Sec. "Fine-Tuning for Sparse Attention"). */

/* Bytes of device scratch for h2o_sdpa_chunk_backward (0 on invalid
 * arguments): one float per packed query row for float32; for bf16 one per
 * row and key-range split, plus float32 partials of dq [splits,B,Hq,T,d] when
 * the shape has too few query rows to fill the GPU (e.g. 2 splits, 32 MiB at
 * B1 Hq32 T1024 d128). */
size_t h2o_backward_workspace_bytes(int B, int Hq, int Hkv, int T, int M, int d,
                                    int dtype);

/* Backward of h2o_sdpa_chunk (token_pos NULL: keys [cache || chunk], causal in
 * the chunk) or of h2o_sdpa_cache (token_pos non-NULL, positions pos0..: the
 * cache slots with the token-position mask; k_new, v_new, dk_new and dv_new
 * are not used and may be NULL). Given the forward's lse and the output
 * gradient dout [B,Hq,T,d], writes the gradients of the loss sum(dout * out):
 *   dq [B,Hq,T,d]; dk_cache, dv_cache [B,Hkv,M,d]; dk_new, dv_new [B,Hkv,T,d]
 * (written, not accumulated; a KV head's gradients sum over its GQA group).
 * With P = softmax(scale Q K^T) (masked, rebuilt from lse), dP = dout V^T
 * and D_r = sum_j P_rj dP_rj (from P and dP, not from a rounded output):
 *   dV = P^T dout,  dS = P * (dP - D),  dQ = scale dS K,  dK = scale dS^T Q.
 * The summed weights of the forward carry no gradient (they only steer the
 * discrete eviction). Float32 arithmetic for float32 data; bf16 data runs
 * on bf16 MFMA with float32 accumulation, P and dS (formed in float32 with
 * the row's D) rounded to bf16 as the operands of the dV, dK and dQ
 * products. Gradients are stored in dtype (bf16 nearest-even). Workspace of
 * h2o_backward_workspace_bytes(). */
int h2o_sdpa_chunk_backward(const void* q, const void* k_cache,
                            const void* v_cache, const void* k_new,
                            const void* v_new, const int32_t* token_pos,
                            const float* lse, const void* dout,
                            void* dq, void* dk_cache, void* dv_cache, void* dk_new,
                            void* dv_new, void* workspace, size_t workspace_bytes,
                            int B, int Hq, int Hkv, int T, int M, int d,
                            float scale, int32_t pos0, int dtype, void* stream);

/* Delta encoding of the KV recurrence (Eq. recurrence-reverse, Sec. "Buffer
 * Read/Write Access by torch.scatter, torch.gather"): with idx [B,Hkv,k]
 * (int32 slots, out-of-range entries skipped),
 *   h2o_kv_gather:   delta[b,h,i,:] = cache[b,h,idx[b,h,i],:]
 *   h2o_kv_scatter:  cache[b,h,idx[b,h,i],:] = src[b,h,i,:]
 * cache [B,Hkv,M,d], delta/src [B,Hkv,k,d], in dtype. The gather of the slots
 * a chunk is about to overwrite, scattered back after the insert, restores
 * the cache bit for bit. Slots in one row of idx must be distinct for the
 * scatter. */
int h2o_kv_gather(const void* cache, const int32_t* idx, void* delta, int B,
                  int Hkv, int M, int k, int d, int dtype, void* stream);
int h2o_kv_scatter(void* cache, const int32_t* idx, const void* src, int B,
                   int Hkv, int M, int k, int d, int dtype, void* stream);

/* The selection of h2o_evict_insert alone: for each of `rows` rows of M
 * float32 scores, the k smallest by (score, index), ascending indices, into
 * idx_out [rows, k]. 0 <= k <= M. */
int h2o_bottomk(const float* scores, int rows, int M, int k, int32_t* idx_out,
                void* stream);

/* Message for the calling thread's last non-OK status ("" if none). The
 * pointer stays valid until the thread's next call into the library. */
const char* h2o_last_error(void);

/* Testing hook, not needed in normal use: force the bf16 SDPA kernel path of
 * h2o_sdpa_chunk for every later call in the process (-1 automatic, 0 the
 * generic VALU kernels, 1 the MFMA prefill kernels, 2 the decode kernels,
 * which need T == 1). float32 always uses the generic kernels. 0 also puts
 * h2o_sdpa_chunk_backward on its VALU kernels. Returns H2O_EINVAL for other
 * values. */
int h2o_debug_force_path(int path);

/* Benchmark hook, not needed in normal use. h2o_debug_timing(1) makes every
 * kernel launch of the library go through hipExtLaunchKernel with a start and
 * a stop event, which the runtime stamps at the kernel's own begin and end
 * (do not use it under stream capture); h2o_debug_timing(0) stops it.
 * Either call clears the totals. h2o_debug_kernel_time(id, &ms, &n) waits for
 * the recorded events and returns the summed duration (milliseconds) and the
 * launch count of kernel `id` since the last h2o_debug_timing call. Ids:
 *   0 generic lse pass   1 generic main pass   2 MFMA lse pass
 *   3 MFMA main pass     4 split reduce        5 column-sum reduce
 *   6 accumulate         7 bottom-k            8 insert
 *   9 decode split      10 decode combine     11 argmin + insert (k == 1)
 *  12 decode finish (h2o_chunk_step, T == 1)
 *  13 score-variant keys and index broadcast (h2o_evict_insert_policy)
 *  14 backward dQ (VALU: and the rows' D)  15 backward dK/dV
 *  16 KV gather / scatter   17 backward rows' D (MFMA path)
 *  18 backward dQ split reduce (MFMA path)
 *  19 bottom-k and insert in one launch (h2o_chunk_step, 1 < T <= 4096) */
int h2o_debug_timing(int on);
int h2o_debug_kernel_time(int kernel_id, double* total_ms, long* count);

/* Library version string. */
const char* h2o_version(void);

#ifdef __cplusplus
}
#endif
#endif /* H2O_H */

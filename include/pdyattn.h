/*
 * pdyattn -- packed variable-length softmax attention, forward and backward,
 * for AMD Instinct MI355X (gfx950).
 *
 * The operation is scaled dot-product attention as written in Eq. (2) of the
 * problem formulation (section 3):  A = Softmax(Q K^T / sqrt(d)) V, applied per
 * head to a packed batch of dynamic-length sequences laid out as in the
 * tensor-layout specification (Table 2, section 4.2: activations b x s/p x h,
 * here packed to [T, H, d] with segment offsets).  The backward computes the
 * gradient of that expression, which the training workloads of section 5.1
 * need.  Readings of points the paper leaves open:
 *   - d is the head dimension (h/n of Table 4); the scale is an argument.
 *   - segments never attend to each other; with causal = 1 key j is visible
 *     to query i iff j <= i within the segment.
 *   - grouped heads: query head h reads key/value head h / (Hq / Hkv).
 *   - lse is the natural-log log-sum-exp of the scaled logits, [Hq, T].
 *
 * Conventions shared by every entry point:
 *   - All tensor pointers are DEVICE pointers owned by the caller; the library
 *     never allocates or frees device memory.  Dense, row-major, last dim
 *     contiguous, 16-byte aligned.  bf16 tensors are raw IEEE bfloat16 bits.
 *   - cu_seqlens is an int32 device array of num_seqs + 1 offsets with
 *     cu[0] = 0, cu[i] <= cu[i+1], cu[num_seqs] = total_tokens.  Zero-length
 *     segments are allowed.  Its contents are trusted (reading them on the
 *     host would force a synchronisation); attn_validate_cu_seqlens checks it.
 *   - max_seqlen must be >= every segment length (an upper bound suffices);
 *     with num_seqs = 1 it must equal total_tokens (the one segment is
 *     [0, T)), else the call returns PDY_ERR_INVALID_ARG.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = default stream) and
 *     the call returns without synchronising.  Outputs are fully overwritten.
 *   - Argument errors are reported before anything is launched.  A non-OK
 *     status leaves a thread-local message in pdy_last_error().
 *   - Scratch memory comes from the caller's `workspace` (16-byte aligned,
 *     at least the size the matching *_workspace_size query returns).
 *   - Calls on different streams with disjoint outputs and workspaces may run
 *     concurrently, except attn_bwd_noalloc calls on the same GPU (they share
 *     its static scratch array); the library holds no other global state
 *     besides per-thread error text, the optional per-thread kernel timing
 *     records and a one-time setup of kernel attributes.
 *   - Results are bitwise reproducible run to run (no atomics feed outputs).
 *   - Launches too small to fill the GPU (fewer than 512 work items, e.g. a
 *     single 8K-token sequence over 4 heads) split each item's work into
 *     parts (split-K) whose fp32 partial results are combined in a second
 *     kernel: 2 or 4 parts per item, or, for a causal single sequence whose
 *     parts fit one round on the GPU, more parts for the heavier items (at
 *     most 16); the choice depends only on the sizes and the causal flag
 *     (the workspace queries cover both values of the flag).  A segment's results
 *     therefore do not depend on the other segments of its batch, but a batch
 *     and the same segment alone may round differently when one of the two
 *     launches is split.
 */
#ifndef PDYATTN_H
#define PDYATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PDY_OK = 0,
  PDY_ERR_INVALID_ARG = -1, /* null/misaligned pointer, bad size or flag          */
  PDY_ERR_UNSUPPORTED = -2, /* head_dim not in {64, 128}                            */
  PDY_ERR_WORKSPACE = -3,   /* workspace smaller than the query function asks for */
  PDY_ERR_HIP = -4          /* a HIP runtime call failed (message has the detail) */
} pdy_status;

/* Bytes of workspace attn_fwd needs for these sizes (>= 256; for a split-K
 * launch it includes the parts' fp32 O and LSE, under 129 MiB).
 * Returns 0 when the sizes are invalid. */
size_t attn_fwd_workspace_size(int32_t total_tokens, int32_t num_seqs, int32_t max_seqlen,
                               int32_t num_heads_q, int32_t num_heads_kv, int32_t head_dim);

/* Bytes of workspace attn_bwd needs (it holds D = rowsum(dO * O), fp32
 * [Hq, T], the tile schedules and, for split-K launches, the parts' fp32
 * partial gradients, under 384 MiB).  Returns 0 when the sizes are
 * invalid. */
size_t attn_bwd_workspace_size(int32_t total_tokens, int32_t num_seqs, int32_t max_seqlen,
                               int32_t num_heads_q, int32_t num_heads_kv, int32_t head_dim);

/* Forward of Eq. (2) (section 3) over a packed batch.
 *   q   bf16 [T, Hq,  d]        k, v  bf16 [T, Hkv, d]
 *   o   bf16 [T, Hq,  d] (out)  lse   fp32 [Hq, T]    (out, natural log)
 *   num_heads_q % num_heads_kv == 0;  head_dim in {64, 128};  causal in {0, 1};
 *   scale finite and > 0 (usually 1/sqrt(head_dim)).
 * T = 0 is a no-op.  o and lse must not alias the inputs. */
pdy_status attn_fwd(const void* q, const void* k, const void* v, const int32_t* cu_seqlens,
                    int32_t num_seqs, int32_t total_tokens, int32_t max_seqlen,
                    int32_t num_heads_q, int32_t num_heads_kv, int32_t head_dim,
                    int32_t causal, float scale,
                    void* o, float* lse,
                    void* workspace, size_t workspace_bytes, void* stream);

/* Backward of Eq. (2) (section 3): gradients of sum(dout * o).
 *   q, o, dout bf16 [T, Hq, d];  k, v bf16 [T, Hkv, d];  lse fp32 [Hq, T] as
 *   written by attn_fwd for the same inputs.
 *   dq fp32 [T, Hq, d] (out);  dk, dv fp32 [T, Hkv, d] (out; with grouped
 *   heads each sums its query heads).  Gradients are fp32 so that large
 *   accumulated values keep their precision.
 * Same size/flag rules as attn_fwd. */
pdy_status attn_bwd(const void* q, const void* k, const void* v, const void* o, const float* lse,
                    const void* dout, const int32_t* cu_seqlens,
                    int32_t num_seqs, int32_t total_tokens, int32_t max_seqlen,
                    int32_t num_heads_q, int32_t num_heads_kv, int32_t head_dim,
                    int32_t causal, float scale,
                    float* dq, float* dk, float* dv,
                    void* workspace, size_t workspace_bytes, void* stream);

/* ---- One long sequence split into chunks (context parallelism) ----
 * Sequence-sharded strategies (section 2.2: Megatron-style context
 * parallelism, its ZeRO-3 variant, the fine-grained two-level ring) give a
 * device the queries of positions q_offset .. q_offset+tq-1 and, one chunk
 * at a time, the keys/values of positions k_offset .. k_offset+tk-1 of the
 * same sequence.  Eq. (2) restricted to one key chunk gives a partial output
 * and log-sum-exp; attn_merge combines partials of the same rows into the
 * result over the union of the chunks.  With causal = 1 a key is visible to
 * a query iff its position is <= the query's; a row that sees no key of the
 * chunk gets o = 0 and lse = -inf (the neutral element of attn_merge).
 * Sizes: tq, tk >= 0, offsets >= 0; tensors [tq, Hq, d] (q, o, dout, dq),
 * [tk, Hkv, d] (k, v, dk, dv), lse fp32 [Hq, tq].  Other rules as above. */
size_t attn_fwd_chunk_workspace_size(int32_t tq, int32_t tk, int32_t num_heads_q,
                                     int32_t num_heads_kv, int32_t head_dim);
size_t attn_bwd_chunk_workspace_size(int32_t tq, int32_t tk, int32_t num_heads_q,
                                     int32_t num_heads_kv, int32_t head_dim);

/* Partial forward of a query chunk over one key/value chunk:
 * o bf16 [tq, Hq, d] and lse fp32 [Hq, tq] (out).  tq = 0 is a no-op;
 * tk = 0 gives o = 0, lse = -inf (k and v may then be NULL). */
pdy_status attn_fwd_chunk(const void* q, const void* k, const void* v, int32_t tq, int32_t tk,
                          int32_t q_offset, int32_t k_offset,
                          int32_t num_heads_q, int32_t num_heads_kv, int32_t head_dim,
                          int32_t causal, float scale,
                          void* o, float* lse,
                          void* workspace, size_t workspace_bytes, void* stream);

/* Contribution of one (query chunk, key chunk) pair to the gradient of
 * sum(dout * O): o and lse are the FINAL output and log-sum-exp of the query
 * rows (merged over every key chunk), dout their upstream gradient.
 * Writes dq fp32 [tq, Hq, d] (this pair's part; the chunk's dQ is the sum
 * over its key chunks) and dk, dv fp32 [tk, Hkv, d] (this pair's part; a key
 * chunk's gradient is the sum over query chunks); with accumulate = 1 the
 * part is added to what dq, dk and dv hold.  Rows with lse = -inf
 * contribute nothing.  tq = 0 writes zero dk, dv (accumulate = 0) or leaves
 * them (accumulate = 1). */
pdy_status attn_bwd_chunk(const void* q, const void* k, const void* v, const void* o,
                          const float* lse, const void* dout, int32_t tq, int32_t tk,
                          int32_t q_offset, int32_t k_offset,
                          int32_t num_heads_q, int32_t num_heads_kv, int32_t head_dim,
                          int32_t causal, float scale,
                          float* dq, float* dk, float* dv, int32_t accumulate,
                          void* workspace, size_t workspace_bytes, void* stream);

/* Combine two partial results of the same T query rows:
 *   lse = log(exp(lse_a) + exp(lse_b)),  o = sum_x exp(lse_x - lse) o_x
 * (bf16 [T, Hq, d] and fp32 [Hq, T]).  o/lse may alias o_a/lse_a or
 * o_b/lse_b (in place).  Needs no workspace. */
pdy_status attn_merge(const void* o_a, const float* lse_a, const void* o_b, const float* lse_b,
                      int32_t total_tokens, int32_t num_heads_q, int32_t head_dim,
                      void* o, float* lse, void* stream);

/* Debug helper: copies cu_seqlens to the host (synchronising `stream`) and
 * checks cu[0] = 0, monotonicity and cu[num_seqs] = total_tokens.  On success
 * writes the longest segment length to *max_seqlen_out (may be NULL). */
pdy_status attn_validate_cu_seqlens(const int32_t* cu_seqlens, int32_t num_seqs,
                                    int32_t total_tokens, int32_t* max_seqlen_out,
                                    void* stream);

/* attn_bwd for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same computation, arguments and outputs as attn_bwd, without the
 * workspace.  Its scratch (the tile schedules, D and any split-K partial
 * gradients) is a static device array of 64 MiB per GPU, held from the
 * first call on that GPU until the process ends.  Sizes whose schedules and
 * D alone exceed 64 MiB (Hq * T beyond about 16.7 million (row, head)
 * pairs) return PDY_ERR_WORKSPACE before anything is launched.  A launch
 * small enough to split (see above) whose partial gradients would not fit
 * takes fewer parts; its results may then differ from attn_bwd's in
 * rounding (well inside the stated tolerance), otherwise they equal
 * attn_bwd's bit for bit.  The call allocates nothing (no hipMalloc, no
 * library allocation); on its first use on a device it looks up that
 * device's address of the array.  The array keeps the last call's contents,
 * none of which a call reads before writing it.  Every call on one GPU uses
 * the same array: calls that overlap on one GPU (other streams, other
 * threads) race and must be serialised by the caller. */
pdy_status attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o,
                            const float* lse, const void* dout, const int32_t* cu_seqlens,
                            int32_t num_seqs, int32_t total_tokens, int32_t max_seqlen,
                            int32_t num_heads_q, int32_t num_heads_kv, int32_t head_dim,
                            int32_t causal, float scale, float* dq, float* dk, float* dv,
                            void* stream);

/* Static text for a status code. */
const char* pdy_status_string(int32_t status);

/* Detail of the last non-OK status returned on this thread ("" if none). */
const char* pdy_last_error(void);

/* Kernel timing (measurement support for the per-length cost tables the
 * paper's hybrid cost models are fitted to, section 4.3).  Between
 * pdy_profile_start and pdy_profile_stop, every kernel this thread launches
 * is bracketed by two HIP events recorded on the launch's own stream.
 * pdy_profile_stop waits for those events and writes, for each kernel id
 * k < n, the number of launches and their summed duration in milliseconds
 * (arrays of n caller-owned host elements).  Kernel ids are
 * 0..pdy_kernel_count()-1, named by pdy_kernel_name. */
int32_t pdy_kernel_count(void);
const char* pdy_kernel_name(int32_t k);
pdy_status pdy_profile_start(void);
pdy_status pdy_profile_stop(int32_t* launches, double* total_ms, int32_t n);

#ifdef __cplusplus
}
#endif
#endif /* PDYATTN_H */

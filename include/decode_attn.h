/*
 * decode_attn.h -- C ABI of the MI355X (gfx950) decode-attention library.
 *
 * Single-query decode attention over a KV cache for MHA, GQA and MQA, and the
 * per-step KV-cache append, as derived in "MoA-Structured Decode Attention:
 * DNF Derivation, KV-Cache Accumulation, GQA/MQA, and OpenACC Kernel"
 * (Mullin and Hains, 2026).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.  Every array argument is a DEVICE pointer (memory of the current
 * HIP device) to contiguous row-major data, owned by the caller.  The library
 * allocates nothing and keeps no pointer after a call returns.  Layouts are the
 * row-major offsets of the paper's ONF section (element <l,j> of an <n,d_k>
 * slab at l*d_k + j), lifted over batch and heads:
 *     q     float [B][h_q][d_k]        query vector of every query head
 *     K     float [B][h_kv][n_max][d_k] key cache, one slab per KV head
 *     V     float [B][h_kv][n_max][d_v] value cache
 *     len   int32 [B]                   valid rows per sequence (device)
 *     out   float [B][h_q][d_v]         attention output
 *     k_new float [B][h_kv][d_k], v_new float [B][h_kv][d_v]  rows to append
 * n_max is the capacity (row stride of a slab).  Rows at or beyond len[b] may
 * hold anything, NaN included: they are never read.
 *
 * Head map.  Query head h uses KV head floor(h*h_kv/h_q) (the psi-selection
 * of eq. (10); h_kv must divide h_q), so the G = h_q/h_kv query heads of a
 * group share one KV slab, which the decode reads from HBM once per group.
 *
 * Execution.  Calls only validate their arguments on the host and enqueue
 * kernels on `stream` (a hipStream_t; NULL = the null stream); they return
 * before the work runs.  Results are valid once the stream has reached that
 * point.  Work enqueued on one stream runs in order, so an append followed by
 * a decode on the same stream sees the appended row; `len` never needs to
 * visit the host.
 *
 * Errors.  Every argument is checked before anything is enqueued; on a non-OK
 * status nothing was enqueued and no memory was touched.  DA_ERR_HIP reports
 * a launch failure from the HIP runtime.  No C++ exception crosses the ABI.
 *
 * Precision.  fp32 storage and arithmetic (the paper's 4-byte traffic model),
 * products accumulated in fp32 by the matrix cores, exponentials by the
 * hardware base-2 exponential.  Results agree with an exact evaluation within
 * 1e-5 absolute for N(0,1) inputs; the append is a bit-exact copy.
 */
#ifndef DECODE_ATTN_H
#define DECODE_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum da_status {
    DA_OK = 0,
    DA_ERR_NULL = 1,        /* a required pointer is NULL                          */
    DA_ERR_SHAPE = 2,       /* a size < 1 or too large, h_kv not dividing h_q
                               (or, tuning calls only, a bad chunk_rows)          */
    DA_ERR_UNSUPPORTED = 3, /* d_k or d_v not in {64, 128, 256} (decode), or not a
                               multiple of 4 (append)                              */
    DA_ERR_ALIGN = 4,       /* a float array not 16-byte aligned, len not 4-byte   */
    DA_ERR_SCALE = 5,       /* scale is NaN or infinite                            */
    DA_ERR_WORKSPACE = 6,   /* workspace NULL or smaller than required             */
    DA_ERR_HIP = 7          /* the HIP runtime reported an error at launch         */
} da_status;

/* Human-readable name of a status code (static string, never NULL; codes
 * outside the enumeration give "unknown da_status"). */
const char *da_status_string(da_status status);

/*
 * Workspace.  The decode keeps, per (b, query head), a few partial results
 * (a reference score, at most 8 base-2 units below the largest score seen,
 * the sum of exponentials against it, the unnormalised weighted sum of V
 * rows) plus a few counters per (b, KV head) that schedule the work.  The
 * counter region -- the first da_decode_workspace_counter_bytes() bytes --
 * must be zero before a decode starts; every completed decode leaves it zero
 * again, so a workspace can be reused call after call without clearing (and
 * a call can be captured in a HIP graph and replayed).  A da_decode_partial
 * that is not followed by its da_decode_merge (or a stream torn down between
 * the two) leaves counters set: the next decode on that workspace would then
 * skip rows, so such a workspace must be cleared first, with
 * da_decode_workspace_reset or by zeroing the counter region.  The rest of
 * the workspace needs no initialisation.  One workspace serves one decode at
 * a time: decodes that overlap in time (on different streams) need separate
 * workspaces.
 */

/*
 * Bytes of device workspace da_decode_attn, da_decode_step and the
 * da_decode_partial + da_decode_merge pair need for these shapes (the
 * library chooses its work decomposition; the size covers every device the
 * library runs on).  Returns 0 if the shapes are invalid.
 */
size_t da_decode_workspace_bytes(int B, int h_q, int h_kv, int n_max, int d_k,
                                 int d_v);

/*
 * Leading bytes of that workspace that hold the scheduling counters (the part
 * that must be zero when a decode starts).  Returns 0 if the shapes are
 * invalid.
 */
size_t da_decode_workspace_counter_bytes(int B, int h_q, int h_kv, int n_max,
                                         int d_k, int d_v);

/*
 * Clears the counter region of a workspace for decodes of these shapes (h_q
 * counts query rows: h_q*T for the T-row calls), with a kernel on `stream`
 * (no memset node, so it can sit inside a captured HIP graph).  For
 * recovering a workspace left by a partial without its merge; a workspace
 * that only ever saw complete decodes never needs it.
 * Errors: DA_ERR_NULL (workspace NULL), DA_ERR_SHAPE / DA_ERR_UNSUPPORTED
 * (shapes), DA_ERR_WORKSPACE (workspace_bytes below the counter region),
 * DA_ERR_ALIGN (workspace not 16-byte aligned), DA_ERR_HIP.
 */
da_status da_decode_workspace_reset(void *workspace, size_t workspace_bytes,
                                    int B, int h_q, int h_kv, int n_max,
                                    int d_k, int d_v, void *stream);

/*
 * Decode attention, eqs. (1)-(3) (Algorithm 1) for every batch b and query
 * head h, with the psi-selection head map of eq. (10):
 *     s[l]  = scale * sum_j q[b,h,j] * K[b,g,l,j],   g = floor(h*h_kv/h_q),
 *             for l < n_b = min(max(len[b], 0), n_max)
 *     a     = softmax(s)                (max-subtracted, eq. (2))
 *     out[b,h,d] = sum_l a[l] * V[b,g,l,d]
 * n_b = 0 gives out[b,h,:] = 0.  `scale` is applied once to the dot product
 * (the caller passes 1/sqrt(d_k) for standard attention).
 *
 * A resident set of workgroups shares the rows of all (b, KV head) slabs:
 * most of each slab in row ranges fixed in advance (proportional to the
 * lengths), the rest in small units handed out dynamically; a workgroup
 * folds everything it reads from one slab into one running softmax state
 * (the online form of eq. (2)) and leaves one partial per visit; a second
 * launch combines the partials exactly (a regrouping of eqs. (2)-(3) over
 * disjoint row sets).  Which workgroup takes which dynamic unit varies, so
 * the summation order varies from call to call within fp32 rounding.  Short
 * caches (n_max <= 4608, h_q / h_kv <= 16, d_k + d_v <= 256), and short
 * batches of such heads whatever their length (fewer than 16 * 256 units of
 * 192 rows over all slabs), are cut into row ranges only, run at two
 * workgroups per CU; so are other batches too short for the dynamic units
 * to move work (fewer than 32 units per workgroup), at one per CU.  When
 * every slab is a single segment (n_max <= 768, or at least 2048 (b, KV
 * head) slabs with n_max <= 4608, h_q / h_kv <= 16 and d_k + d_v <= 256) the
 * decode is a single launch that writes out directly.  Equivalent to
 * da_decode_partial followed by da_decode_merge.
 *
 * Supported: d_k, d_v in {64, 128, 256}; any B, h_q, h_kv >= 1 with h_kv | h_q.
 * workspace: see above; at least da_decode_workspace_bytes(...) bytes,
 * 16-byte aligned.  out must not overlap the inputs.
 * Errors, checked in this order: DA_ERR_NULL (q, K, V, len, out), DA_ERR_SHAPE,
 * DA_ERR_UNSUPPORTED, DA_ERR_ALIGN, DA_ERR_SCALE, DA_ERR_WORKSPACE, then
 * DA_ERR_HIP from the launch.
 */
da_status da_decode_attn(const float *q, const float *K, const float *V,
                         const int32_t *len, float scale, float *out, int B,
                         int h_q, int h_kv, int n_max, int d_k, int d_v,
                         void *workspace, size_t workspace_bytes, void *stream);

/*
 * Append and decode in one step: the effect of da_kv_append(K, V, k_new,
 * v_new, len, ...) followed by da_decode_attn(q, K, V, len, ...) -- eqs.
 * (6)-(7) then (1)-(3), the order of one autoregressive step of the paper's
 * multi-step cache -- in two kernel launches instead of three: the partial
 * launch reads the new row of each KV head straight from k_new / v_new (and
 * writes it into the cache meanwhile), and the merge advances len.  When
 * every slab is short (n_max within one segment), h_q / h_kv <= 16 and
 * d_k + d_v <= 256, the whole step is one launch: one workgroup per
 * (b, KV head, head group) writes its output rows, and the last workgroup of
 * each sequence to finish advances len[b].  Same results, same argument
 * rules as the two calls; k_new [B][h_kv][d_k] and v_new [B][h_kv][d_v] must
 * not overlap K / V.
 */
da_status da_decode_step(const float *q, float *K, float *V,
                         const float *k_new, const float *v_new, int32_t *len,
                         float scale, float *out, int B, int h_q, int h_kv,
                         int n_max, int d_k, int d_v, void *workspace,
                         size_t workspace_bytes, void *stream);

/*
 * First half of da_decode_attn / da_decode_step: scores of all G query heads
 * of each group over the slab's rows (K and V rows read from HBM once per
 * (b, KV head)), their reference scores, sums of exponentials and
 * unnormalised weighted sums of V rows, written to the workspace as per-visit
 * partials.  k_new and v_new are both NULL (plain decode; K and V are only
 * read) or both set (the fused append of da_decode_step: row len[b] of every
 * KV head is taken from them and written into K / V).  Must be followed by
 * da_decode_merge on the same workspace and stream, which also resets the
 * counters (see the workspace notes above for a partial left without it).
 */
da_status da_decode_partial(const float *q, float *K, float *V,
                            const float *k_new, const float *v_new,
                            const int32_t *len, float scale, int B, int h_q,
                            int h_kv, int n_max, int d_k, int d_v,
                            void *workspace, size_t workspace_bytes,
                            void *stream);

/*
 * Second half: combines the partials of every (b, query head) into
 * out[b,h,:] (largest reference, rescaled sums, one division) and resets the
 * workspace counters to zero.  The shapes must be those of the
 * da_decode_partial call that filled the workspace.  len is NULL after a
 * plain decode; after a partial with a fused append it is that call's len,
 * and every len[b] with 0 <= len[b] < n_max advances by one.
 */
da_status da_decode_merge(float *out, int32_t *len, int B, int h_q, int h_kv,
                          int n_max, int d_k, int d_v, void *workspace,
                          size_t workspace_bytes, void *stream);

/*
 * Decode with T query rows per query head (T >= 1): the rank-2 query of the
 * paper's training form, softmax(scale * Q (+.x Omega<2,2>) K)
 * (+.x Omega<2,2>) V, for a step that submits T consecutive positions at
 * once (speculative verification, chunked prefill), with causal visibility:
 * query row r of sequence b sits at cache position p = clamp(len[b], 0,
 * n_max) - T + r (the cache's last T positions) and attends rows 0..p; a row
 * with p < 0 gives 0.  T = 1 is da_decode_attn.
 *     q   float [B][h_q][T][d_k]      out float [B][h_q][T][d_v]
 * The T rows of every query head of a group are scored from the same K/V
 * reads (the kernels treat them as h_q*T query heads), so the workspace is
 * that of a single-row decode with h_q*T query heads:
 * da_decode_workspace_bytes(B, h_q*T, h_kv, ...) bytes, its counter region
 * da_decode_workspace_counter_bytes(B, h_q*T, h_kv, ...).  T <= 4096.  Other
 * rules as da_decode_attn.
 */
da_status da_decode_multi(const float *q, const float *K, const float *V,
                          const int32_t *len, float scale, float *out, int B,
                          int h_q, int h_kv, int n_max, int d_k, int d_v, int T,
                          void *workspace, size_t workspace_bytes, void *stream);

/*
 * T autoregressive steps in one: the effect of T successive da_decode_step
 * calls whose rows are given together -- row r of k_new [B][h_kv][T][d_k] /
 * v_new [B][h_kv][T][d_v] appended at len[b] + r while the cache has room
 * (da_kv_append_rows), and query row r of q [B][h_q][T][d_k] attending rows
 * 0 .. min(len[b] + r, n_max - 1) of the grown cache (len[b] the value on
 * entry; nothing if len[b] < 0).  Two launches (one under the conditions
 * da_decode_step names, with h_q*T / h_kv for h_q / h_kv); len advances by
 * the rows that fit.  Workspace as da_decode_multi.
 *
 * While every row fits (0 <= len[b] and len[b] + T <= n_max) this equals
 * da_kv_append_rows followed by da_decode_multi.  Near capacity the two
 * differ on purpose: here row r still attends the rows a single step r
 * would see (rows that did not fit are simply absent), whereas
 * da_decode_multi places its T rows at the cache's last T positions.  E.g.
 * len[b] = n_max - 2, T = 4: here rows 0..3 attend up to n_max-2, n_max-1,
 * n_max-1, n_max-1; after da_kv_append_rows, da_decode_multi's rows attend
 * up to n_max-4 .. n_max-1.
 */
da_status da_decode_multi_step(const float *q, float *K, float *V,
                               const float *k_new, const float *v_new,
                               int32_t *len, float scale, float *out, int B,
                               int h_q, int h_kv, int n_max, int d_k, int d_v,
                               int T, void *workspace, size_t workspace_bytes,
                               void *stream);

/*
 * KV-cache append, eqs. (6)-(7) (K_{t+1} = K_t # k_t, V_{t+1} = V_t # v_t,
 * Proposition 2): for every b with 0 <= t = len[b] < n_max and every KV head
 * g, copies k_new[b,g,:] to K[b,g,t,:] and v_new[b,g,:] to V[b,g,t,:] bit for
 * bit, then sets len[b] = t + 1.  No other cache row is touched.  A sequence
 * whose cache is full (len[b] >= n_max) or whose len[b] is negative is left
 * unchanged, len included.
 * Supported: d_k, d_v positive multiples of 4; 16-byte aligned float arrays.
 */
da_status da_kv_append(float *K, float *V, const float *k_new,
                       const float *v_new, int32_t *len, int B, int h_kv,
                       int n_max, int d_k, int d_v, void *stream);

/*
 * T rows at once: da_kv_append applied T times in order, row r of every
 * (b, g) taken from k_new [B][h_kv][T][d_k] / v_new [B][h_kv][T][d_v].  Rows
 * land at len[b] + r while the cache has room; len[b] advances by the rows
 * written.  1 <= T <= 4096; other rules as da_kv_append.
 */
da_status da_kv_append_rows(float *K, float *V, const float *k_new,
                            const float *v_new, int32_t *len, int B, int h_kv,
                            int n_max, int d_k, int d_v, int T, void *stream);

/*
 * da_decode_attn without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): same arguments minus the workspace,
 * same results, same validation.  The workspace is a fixed 64 MiB array in
 * device memory that the library holds on every GPU it is loaded on, until
 * the process ends; the call allocates nothing (no hipMalloc or allocating
 * library routine).  Shapes whose da_decode_workspace_bytes() exceeds 64 MiB
 * (67108864 bytes) are rejected with DA_ERR_WORKSPACE before anything is
 * enqueued.  Each call first clears the array's counter region with a
 * kernel.  All calls on one GPU share that GPU's array: calls that overlap
 * in time on one GPU (concurrent streams, or several host threads) race and
 * give wrong results; serialise them, or use da_decode_attn with separate
 * workspaces.  DA_ERR_HIP also reports a failed lookup of the array.
 */
da_status da_decode_attn_noalloc(const float *q, const float *K,
                                 const float *V, const int32_t *len,
                                 float scale, float *out, int B, int h_q,
                                 int h_kv, int n_max, int d_k, int d_v,
                                 void *stream);

/*
 * ---------------------------------------------------------------------------
 * Tuning and testing only.  The entry points above choose their own segment
 * size (the most rows a workgroup reads from its static range in one go,
 * and for caches scheduled without a static share also the unit handed out
 * dynamically).  These variants take it explicitly as chunk_rows, a positive
 * multiple of 768 (0 = the library's choice), for sweeps and for tests that
 * force a decomposition; results are the same decode within fp32 rounding.
 * Not a stable interface: the decomposition may change without notice.
 * A workspace sized by da_decode_workspace_bytes_ex for some chunk_rows
 * serves only calls with that chunk_rows.  DA_ERR_SHAPE also covers an
 * invalid chunk_rows.
 *
 * The environment variable DECODE_ATTN_DYNAMIC_MIN_UNITS (a non-negative
 * integer, read at every call; default 32) is the fewest scheduling units
 * per resident workgroup, counted at n_max rows per slab, for which a decode
 * keeps part of each slab for dynamic hand-out; below it every slab is
 * divided in advance.  0 keeps the dynamic part wherever the schedule has
 * one (tests use it to cover that path on small caches).  It changes neither
 * the workspace size nor the results beyond fp32 rounding.
 * ---------------------------------------------------------------------------
 */

/* Segment rows the entry points above pick for these shapes (a positive
 * multiple of 768; for the T-row calls pass h_q*T).  0 if the shapes are
 * invalid. */
int da_decode_chunk_rows(int B, int h_q, int h_kv, int n_max, int d_k, int d_v);

/* Workspace bytes for chunk_rows (0 = the library's choice, which gives
 * da_decode_workspace_bytes).  0 if the shapes or chunk_rows are invalid. */
size_t da_decode_workspace_bytes_ex(int B, int h_q, int h_kv, int n_max,
                                    int d_k, int d_v, int chunk_rows);

/* da_decode_multi (T = 1: da_decode_attn) with an explicit chunk_rows. */
da_status da_decode_multi_ex(const float *q, const float *K, const float *V,
                             const int32_t *len, float scale, float *out,
                             int B, int h_q, int h_kv, int n_max, int d_k,
                             int d_v, int T, int chunk_rows, void *workspace,
                             size_t workspace_bytes, void *stream);

/* da_decode_partial for T query rows per head (causal, as da_decode_multi;
 * with k_new / v_new the T-row append of da_decode_multi_step) with an
 * explicit chunk_rows. */
da_status da_decode_partial_ex(const float *q, float *K, float *V,
                               const float *k_new, const float *v_new,
                               const int32_t *len, float scale, int B,
                               int h_q, int h_kv, int n_max, int d_k, int d_v,
                               int T, int chunk_rows, void *workspace,
                               size_t workspace_bytes, void *stream);

/* da_decode_merge for T query rows per head with an explicit chunk_rows (the
 * T and chunk_rows of the partial that filled the workspace; len advances by
 * the rows that fit). */
da_status da_decode_merge_ex(float *out, int32_t *len, int B, int h_q,
                             int h_kv, int n_max, int d_k, int d_v, int T,
                             int chunk_rows, void *workspace,
                             size_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* DECODE_ATTN_H */

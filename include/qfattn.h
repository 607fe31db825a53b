/*
 * qfattn — split-KV grouped-query decode attention for AMD Instinct MI355X (gfx950).
 *
 * The operation is the cache-side sweep of the Q-First decode protocol (arXiv:2608.15473, §2):
 * the device is given the current query of every request and returns, for each query head, the
 * attention vector over the positions already in the KV cache together with its log-sum-exp.
 * The cache of a request may be cut into any number of position shards; each shard returns the
 * pair (O, ln Z) of §5,
 *
 *     s_i = scale * q . k_i,   Z = sum_i exp(s_i),   O = (sum_i exp(s_i) v_i) / Z,
 *
 * and the pairs of all shards merge into the result of one sweep over the whole cache (§5: any
 * partition, any order; an empty shard is ln Z = -inf with a vector that is never read).
 *
 * Entry points: the sweep and its merge (qf_attn_decode_split, qf_attn_combine, or both in one
 * launch: qf_attn_decode, and qf_attn_decode_noalloc for callers that cannot allocate;
 * qf_attn_decode_split_unfolded leaves sub-shard chunks as extra slots); the decode step
 * around them (qf_attn_combine_current folds in the current token, qf_kv_append writes it to the
 * cache, qf_attn_combine_current_append does both in one launch); the dense products of a decoder block (qf_linear) and the sweep sharing one launch with
 * one of them (qf_attn_decode_split_beside); and a host-side simulation of the layer-wise decode
 * schedule (qf_schedule_simulate).
 *
 * Conventions shared by every entry point
 *   - Every pointer argument except `stream` is a DEVICE pointer, owned by the caller, except
 *     where a declaration says HOST (qf_schedule_simulate, the `beside` struct of
 *     qf_attn_decode_split_beside).  The library allocates no memory, keeps no pointer after
 *     returning and holds no per-call state; the one exception is qf_attn_decode_noalloc, which
 *     works in a fixed device array of the library's own.
 *   - Every call is asynchronous: it validates its arguments on the host, enqueues its kernels on
 *     `stream` (a hipStream_t; NULL = the legacy default stream) and returns without waiting.
 *   - Return value: QF_OK (0) or a negative QF_E* code.  On error nothing has been enqueued, and
 *     qf_last_error() describes the problem.  No C++ exception crosses this boundary.
 *   - bf16 tensors are IEEE-754 binary32 truncated to the upper 16 bits (bfloat16), stored as
 *     uint16.  All index tensors are int32.
 *   - Device-resident contents (block-table entries, context lengths, shard counts) cannot be
 *     checked on the host without a synchronisation.  The kernels check them instead: a value out
 *     of range never causes an out-of-bounds access; the affected request's log-sum-exp outputs
 *     are set to NaN so the error is visible downstream.
 */
#ifndef QFATTN_H
#define QFATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define QF_VERSION 8

#define QF_OK 0
#define QF_EINVAL (-1)       /* null pointer, negative or inconsistent size, Hq % Hkv != 0   */
#define QF_EUNSUPPORTED (-2) /* head_dim != 128, page_size != 16, Hq/Hkv not in {1,2,4,8}     */
#define QF_EALIGN (-3)       /* a pointer is not aligned as documented below                 */
#define QF_EHIP (-4)         /* the HIP runtime refused a launch; message from hipGetErrorString */

/* Upper bound on the query heads Hq of every call (the merge kernels address one round of 16 slots
 * of a row with 32-bit offsets); larger values are rejected with QF_EINVAL. */
#define QF_MAX_Q_HEADS 4096

/* Shape of one decode step.  Every field is a host value. */
typedef struct qf_decode_desc {
  int32_t batch;             /* B  >= 0 requests (B == 0: the calls do nothing)               */
  int32_t n_q_heads;         /* Hq query heads, 1 <= Hq <= QF_MAX_Q_HEADS                     */
  int32_t n_kv_heads;        /* Hkv >= 1 KV heads; G = Hq / Hkv query heads share one KV head */
  int32_t head_dim;          /* D, must be 128                                                */
  int32_t page_size;         /* P, positions per cache page, must be 16                       */
  int32_t max_pages_per_seq; /* row length (stride) of the block table, >= 1                  */
  int32_t num_pages;         /* physical pages in the K and V pools, >= 1                     */
  int32_t max_shards;        /* S_max >= 1, the shard-slot dimension of the partial outputs   */
  float softmax_scale;       /* finite; logits are scale * q . k (1/sqrt(128) for Qwen3)      */
} qf_decode_desc;

/*
 * Bytes of device workspace qf_attn_decode_split needs for this shape (0 is possible).  The
 * workspace holds partial states of sub-shard chunks when a shape has fewer (request, KV head,
 * shard) units than the sweep keeps resident on the GPU at once; otherwise, when the shards are
 * long, 128+ pages each at full capacity (ceil(max_pages_per_seq / max_shards) >= 128), and
 * B * max_shards <= 8192, the sweep's dispatch order: ceil(B * max_shards * Hkv / 8) * 8 int32,
 * written by a small kernel enqueued just before the sweep (the (request, shard) pairs ranked by
 * length, longest first, their units dealt to the GPU's XCDs by their measured speeds).  The
 * order decides only when and where each unit is swept, never the results, which are the same
 * bits in any order.  Host call; depends on the
 * descriptor and on that resident count, which is queried from the current device once per
 * process (an MI355X is assumed when there is no device), so query and launch agree.
 * Returns QF_OK, or QF_EINVAL / QF_EUNSUPPORTED for a descriptor qf_attn_decode_split rejects.
 */
int qf_attn_decode_split_workspace_size(const qf_decode_desc* desc, size_t* bytes);

/*
 * The sweep, split into position shards (§2 protocol, §5 shard pairs).
 *
 *   q           bf16 [B, Hq, D], 16-byte aligned.  Query head h reads KV head h / G.
 *   k_cache     bf16 [num_pages, Hkv, P, D], 16-byte aligned: page p, KV head g, slot i holds the
 *   v_cache     key (value) of the position that the block table maps to (p, i).
 *   block_table int32 [B, max_pages_per_seq]; logical page j of request b is physical page
 *               block_table[b * max_pages_per_seq + j].  Entries past a request's last page are
 *               never read.  NULL means the identity map b * max_pages_per_seq + j, which needs
 *               num_pages >= B * max_pages_per_seq.
 *   ctx_lens    int32 [B], 0 <= n_b <= max_pages_per_seq * P: cached positions of request b
 *               (the current token is not included, §2).
 *   n_shards    int32 [B], 1 <= S_b <= max_shards: how many shards request b is cut into.
 *               Shard s takes logical pages [s*K, min((s+1)*K, pages_b)) with
 *               pages_b = ceil(n_b / P) and K = ceil(pages_b / S_b); the positions of the last
 *               page are clipped to n_b.  Shards past the end are empty.
 *   part_out    fp32 [B, max_shards, Hq, D], 16-byte aligned: O of shard s (normalised, §5).
 *               Not written for empty shards or for slots s >= S_b (§5: never read).
 *   part_lse    fp32 [B, max_shards, Hq], 4-byte aligned: natural-log ln Z of shard s; -inf for
 *               an empty shard and for every slot s >= S_b; NaN if request b's inputs were out
 *               of range (see above), and NaN (O too) where a NaN in q, K or V reaches the
 *               shard's scores (a NaN in V alone poisons only that dim of O).
 *   workspace   device buffer of at least qf_attn_decode_split_workspace_size() bytes, 16-byte
 *               aligned; may be NULL when that size is 0.  Its contents need no initialisation
 *               and are garbage afterwards.  Calls that may run at the same time (other streams)
 *               need workspaces of their own.
 *   stream      hipStream_t.
 */
int qf_attn_decode_split(const qf_decode_desc* desc, const void* q, const void* k_cache,
                         const void* v_cache, const int32_t* block_table,
                         const int32_t* ctx_lens, const int32_t* n_shards, float* part_out,
                         float* part_lse, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Sub-shard chunks per shard that the sweep uses for this shape (host call): C >= 1; C > 1 exactly
 * when the shape has fewer (request, KV head, shard) units than the sweep keeps resident on the
 * GPU at once (the workspace then holds the chunks' partial states): the pages of every shard are
 * cut into C consecutive ranges, so that the sweep fills the GPU once, each range keeping at
 * least 3 pages per wavefront.  Where a chunk would hold fewer than 128 pages at full capacity
 * (ceil(max_pages_per_seq / max_shards) / C < 128) the ranges are ceil(len / C) pages, len the
 * shard's page count, the last ones shorter or empty; otherwise their sizes alternate between two
 * weights (1080 : 920), because the chunks alternate between the even- and odd-numbered XCDs of
 * the device and the odd ones stream slower.  Any partition gives the same merged attention
 * (§5).  Like the workspace size, C depends on the device's resident workgroups.  Returns QF_OK,
 * QF_EINVAL or QF_EUNSUPPORTED.
 */
int qf_attn_decode_split_chunks(const qf_decode_desc* desc, int32_t* chunks);

/*
 * The sweep of qf_attn_decode_split without folding the sub-shard chunks into their shards: slot
 * s * C + c of request b receives the pair (O, ln Z) of chunk c of shard s, C =
 * qf_attn_decode_split_chunks() (with C == 1 the slots are the shards and the results are
 * qf_attn_decode_split's, bit for bit).  A chunk is itself a shard of a finer split of the same cache (§5: any
 * partition), so qf_attn_combine over the max_shards * C slots gives the result of the folded
 * sweep followed by the combine, up to the order of the fp32 sums, with one launch fewer and no
 * workspace: for callers that need only the merged attention, not per-shard partials.  Having no
 * workspace, it sweeps long shards in their plain order (shard index descending, never ranked
 * by length); with C == 1 qf_attn_decode_split is the faster call on long shards.
 *
 *   q ... n_shards   as for qf_attn_decode_split.
 *   slot_out    fp32 [B, n_slots, Hq, D], 16-byte aligned: O of every non-empty chunk.
 *   slot_lse    fp32 [B, n_slots, Hq], 4-byte aligned: ln Z of every chunk slot; -inf for an
 *               empty chunk and for every chunk of a slot s >= S_b; NaN as for part_lse.
 *   n_slots     the slot dimension of slot_out and slot_lse: must equal max_shards * C
 *               (QF_EINVAL otherwise, with nothing enqueued).
 *   stream      hipStream_t.
 */
int qf_attn_decode_split_unfolded(const qf_decode_desc* desc, const void* q, const void* k_cache,
                                  const void* v_cache, const int32_t* block_table,
                                  const int32_t* ctx_lens, const int32_t* n_shards,
                                  float* slot_out, float* slot_lse, int32_t n_slots,
                                  void* stream);

/*
 * The sweep and the merge in ONE launch: the result of qf_attn_decode_split followed by
 * qf_attn_combine on the same inputs, without materialising the per-shard outputs in caller
 * buffers.  Bitwise the same when the shape needs no sub-shard chunks
 * (qf_attn_decode_split_chunks() == 1) and max_shards <= 64; otherwise the slots are
 * grouped differently (the chunks of every shard merge in the same pass as the shards; more than
 * 64 slots are summed by 4 wavefronts instead of 8 or 16), which can move the last bits.  The last
 * workgroup to finish a (request, KV head) merges that group's slots (partial states stay in the
 * workspace), so the merge's launch and its wait for the sweep's tail disappear.  Being one
 * launch, it sweeps long shards in their plain order (no ranked dispatch order).
 *
 *   q ... n_shards   as for qf_attn_decode_split.
 *   out              bf16 [B, Hq, D], 4-byte aligned; lse fp32 [B, Hq] natural log, or NULL.
 *                    Values as for qf_attn_combine.
 *   workspace        device buffer of at least qf_attn_decode_workspace_size() bytes (the
 *                    partial states), 16-byte aligned; no initialisation needed.
 *   counters         int32 device array of n_counters >= B * Hkv entries, 4-byte aligned, one
 *                    per (request, KV head).  It must be ZERO-FILLED before its first use; every
 *                    call leaves the entries it used at zero again, so an array zero-filled once
 *                    serves any number of calls with any descriptor (as long as it is large
 *                    enough).  Calls that share a workspace or counters must not run
 *                    concurrently.
 * Returns the codes of qf_attn_decode_split; QF_EINVAL also for a NULL out, workspace or
 * counters, a workspace that is too small or too few counters.
 */
int qf_attn_decode_workspace_size(const qf_decode_desc* desc, size_t* bytes);
int qf_attn_decode(const qf_decode_desc* desc, const void* q, const void* k_cache,
                   const void* v_cache, const int32_t* block_table, const int32_t* ctx_lens,
                   const int32_t* n_shards, void* out, float* lse, void* workspace,
                   size_t workspace_bytes, int32_t* counters, int64_t n_counters,
                   void* stream);

/*
 * qf_attn_decode for callers that cannot allocate device memory or pass a workspace (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the same sweep and
 * merge in one launch, with the same results (bitwise) as qf_attn_decode on the same inputs, but
 * the partial states and the per-(request, KV head) counters live in a fixed device array of the
 * library's own, QF_NOALLOC_SCRATCH_BYTES (64 MiB) on every GPU the library runs on, held until the
 * process ends.  The call allocates nothing; it enqueues a small kernel that clears the counters
 * it will use, then the decode.
 *
 *   q ... n_shards, out, lse   as for qf_attn_decode.
 *   stream                     hipStream_t of the CURRENT device (the scratch used is the current
 *                              device's; its address is looked up on the first call there).
 * Limits: the shape's qf_attn_decode_workspace_size() must be at most QF_NOALLOC_STATE_BYTES and
 * batch * n_kv_heads at most QF_NOALLOC_MAX_GROUPS; otherwise QF_EINVAL, with nothing enqueued.
 * Every call on a GPU shares that GPU's array, whose contents are left from the last call: calls
 * that may overlap on one GPU (concurrent streams, or host threads) race and give wrong results;
 * serialise them (one stream), or use qf_attn_decode with a workspace and counters per stream.
 * Returns the codes of qf_attn_decode; QF_EHIP also when the array's address cannot be found.
 */
#define QF_NOALLOC_SCRATCH_BYTES (64u << 20)
#define QF_NOALLOC_STATE_BYTES ((64u << 20) - (256u << 10))
#define QF_NOALLOC_MAX_GROUPS 65536
int qf_attn_decode_noalloc(const qf_decode_desc* desc, const void* q, const void* k_cache,
                           const void* v_cache, const int32_t* block_table,
                           const int32_t* ctx_lens, const int32_t* n_shards, void* out,
                           float* lse, void* stream);

/*
 * The merge of §5 over every shard slot: for each request b and query head h,
 *
 *     m = max_s ln Z_s,  w_s = exp(ln Z_s - m) (w_s = 0, and O_s unread, where ln Z_s = -inf),
 *     out = sum_s w_s O_s / sum_s w_s,   lse = m + ln(sum_s w_s),
 *
 * the N-way form of the pairwise lerp/sigmoid/logaddexp merge; every weight is at most 1, so
 * nothing overflows however large the log partitions are.
 *
 *   part_out    fp32 [B, max_shards, Hq, D], 16-byte aligned (as written by the sweep).
 *   part_lse    fp32 [B, max_shards, Hq], 4-byte aligned.
 *   out         bf16 [B, Hq, D], 4-byte aligned; round-to-nearest-even.  All slots empty
 *               (n_b = 0): +0.  A NaN log-sum-exp among the slots: NaN.
 *   lse         fp32 [B, Hq] natural log, or NULL if not wanted.  All empty: -inf.
 *   head_dim must be 128; 1 <= n_q_heads <= QF_MAX_Q_HEADS.
 */
int qf_attn_combine(int32_t batch, int32_t n_q_heads, int32_t head_dim, int32_t max_shards,
                    const float* part_out, const float* part_lse, void* out, float* lse,
                    void* stream);

/*
 * The merge above followed by the current token (§2 protocol table and combine; Appendix A fold):
 * with (o_<j, lse_<j) the merge of the shard slots of request b and query head h,
 *
 *     s_jj = scale * q_j . k_j,   out = lerp(v_j, o_<j, sigma(lse_<j - s_jj)),
 *     lse  = logaddexp(lse_<j, s_jj),   sigma(x) = 1 / (1 + exp(-x)),
 *
 * i.e. attention over the cached positions plus the current one.  Correct for either sign of
 * s_jj - lse_<j (short caches, Appendix E) and for an empty cache (out = v_j, lse = s_jj).
 *
 *   q           bf16 [B, Hq, D] (the same query the sweep used), 4-byte aligned.
 *   k_cur,v_cur bf16 [B, Hkv, D]: the current token's key and value; query head h uses KV head
 *               h / G.  4-byte aligned.
 *   part_out, part_lse, out, lse as for qf_attn_combine.  head_dim must be 128;
 *   1 <= n_q_heads <= QF_MAX_Q_HEADS.
 */
int qf_attn_combine_current(int32_t batch, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                            int32_t max_shards, const float* part_out, const float* part_lse,
                            const void* q, const void* k_cur, const void* v_cur,
                            float softmax_scale, void* out, float* lse, void* stream);

/*
 * The cache write of §2: k_j and v_j of every request are stored at its position n_b = ctx_lens[b],
 * i.e. physical page block_table[b * max_pages_per_seq + n_b / P] (identity map when NULL), slot
 * n_b % P, for every KV head.  The page must already belong to the request.
 *
 *   desc        as for qf_attn_decode_split (batch, n_kv_heads, head_dim, page_size,
 *               max_pages_per_seq, num_pages are used).
 *   k_cache,
 *   v_cache     bf16 [num_pages, Hkv, P, D], written in place; 4-byte aligned.
 *   ctx_lens    int32 [B]; when advance != 0, ctx_lens[b] becomes n_b + 1 after the write.
 *   k_new,v_new bf16 [B, Hkv, D]; 4-byte aligned.
 *   status      optional int32 device word: set to 1 (never cleared) when a request's append is
 *               skipped because n_b is outside [0, max_pages_per_seq * P) or its page is outside
 *               the pool; such a request's cache and ctx_lens are left unchanged.
 */
int qf_kv_append(const qf_decode_desc* desc, void* k_cache, void* v_cache,
                 const int32_t* block_table, int32_t* ctx_lens, const void* k_new,
                 const void* v_new, int32_t advance, int32_t* status, void* stream);

/*
 * qf_attn_combine_current and qf_kv_append (advance = 1) of the same current token in one launch:
 * the merge with the current token answers the query (out, lse), and the current token's key and
 * value are written at position n_b = ctx_lens[b] of every request, whose ctx_lens then becomes
 * n_b + 1 (§2: the key and value follow the query into the cache once it has been answered).
 * Results, cache contents, ctx_lens and status are exactly those of the two calls in sequence.
 * The sweep that produced the partials must have been issued before (it never reads position n_b).
 *
 *   desc        batch, n_q_heads, n_kv_heads, head_dim, page_size, max_pages_per_seq, num_pages,
 *               max_shards (the partials' slot count) and softmax_scale are used.
 *   part_out, part_lse, q, out, lse       as for qf_attn_combine_current.
 *   k_cur, v_cur                          the current token, as for qf_attn_combine_current; also
 *                                         what is appended (k_new, v_new of qf_kv_append).
 *   k_cache, v_cache, block_table, ctx_lens, status   as for qf_kv_append.
 */
int qf_attn_combine_current_append(const qf_decode_desc* desc, const float* part_out,
                                   const float* part_lse, const void* q, const void* k_cur,
                                   const void* v_cur, void* out, float* lse, void* k_cache,
                                   void* v_cache, const int32_t* block_table, int32_t* ctx_lens,
                                   int32_t* status, void* stream);

/*
 * Host-side simulation of the layer-wise decode schedule (Appendix D, the wiring as a schedule).
 * Not a GPU call: every pointer here is a HOST pointer, and the call is synchronous.
 *
 * Request r arrives at arrival[r] and sweeps its cache for attn_time[r] at every layer.  Each
 * layer's feed-forward is a pool serving one departure at a time; a departure takes ffn_time,
 * carries every request then waiting, and leaves only with at least min_batch waiting, or when
 * the oldest has waited max_wait (INFINITY: never; the paper's rule, under which a request can be
 * stranded).
 *   QF_WIRING_QFIRST:   e_1 = arrival + a, e_l = max(e_{l-1} + a, ffn_{l-1}), finish = ffn_L: at
 *                       e_l the request joins pool l and starts the sweep of layer l+1.
 *   QF_WIRING_COMPOSED: the request joins pool l when sweep l ends and sweeps layer l+1 when that
 *                       feed-forward returns.
 * At each instant every completion is applied before any pool decides whether to depart.
 *
 *   finish       double [n_requests]: return time of the last feed-forward; NaN if stranded.
 *   sweep_start, sweep_end, ffn_depart, ffn_return
 *                double [n_requests, n_layers] or NULL; NaN for what never happened.
 * Returns QF_OK or QF_EINVAL (n_layers < 1, min_batch < 1, ffn_time <= 0, max_wait < 0 or NaN,
 * non-finite arrival / attention time, negative attention time, unknown wiring).
 */
#define QF_WIRING_QFIRST 0
#define QF_WIRING_COMPOSED 1
int qf_schedule_simulate(int32_t n_requests, const double* arrival, const double* attn_time,
                         int32_t n_layers, int32_t wiring, double ffn_time, int32_t min_batch,
                         double max_wait, double* finish, double* sweep_start, double* sweep_end,
                         double* ffn_depart, double* ffn_return);

/*
 * The dense products of a decoder block at decode (§2 protocol: q_j = W_q N1(u_j); the
 * feed-forward M(N2 u_j); k_j, v_j = W_k N1(z_j), W_v N1(z_j); and W_o), each fused with the
 * normalisation or activation that feeds it and the residual add that follows it:
 *   out[m, n] = sum_{i < k} W[n, i] * P(x)[m, i]  (+ residual[m, n]),   m < rows, n < n_out
 *   QF_LINEAR_PLAIN     P(x) = x                                   x: bf16 [rows, k]
 *   QF_LINEAR_RMS_NORM  P(x) = x / sqrt(mean_i x^2 + eps) * gain   x: bf16 [rows, k], gain [k]
 *   QF_LINEAR_SWIGLU    P(x) = silu(x[:, :k]) * x[:, k:2k],  silu(t) = t / (1 + exp(-t))
 *                                                                  x: bf16 [rows, 2k]
 * (The paper names N1, N2 only as normalisations and M only as the feed-forward; the RMS form and
 * the SwiGLU feed-forward are those of the Qwen3 blocks it converts.)
 * W: bf16 [n_out, k] row-major (torch's [out, in] layout).  Outputs n < n_split go to
 * out [rows, n_split], the rest to out_b [rows, n_out - n_split] (one product can fill k and v);
 * residual: bf16 [rows, n_out] or NULL.  fp32 arithmetic, one round-to-nearest-even per output;
 * out must not alias x or residual.  Device pointers, caller-owned; asynchronous on `stream`.
 * prologue | QF_LINEAR_GLU_OUT: the rows of W alternate the feed-forward's gate and up
 * projections (row 2i = W_gate row i, row 2i + 1 = W_up row i), and the output is the activation
 * itself, out[m, i] = silu(y[m, 2i]) * y[m, 2i + 1], bf16 [rows, n_out / 2] (computed once per
 * element, from the fp32 sums); n_out must be even, n_split == n_out, residual NULL, and the
 * prologue PLAIN or RMS_NORM.
 * Returns QF_OK; QF_EINVAL (rows < 0, n_out < 1, k < 8, unknown prologue, n_split outside
 * [1, n_out], eps < 0 or NaN with RMS_NORM, NULL x / w / out, NULL gain with RMS_NORM, NULL out_b
 * with n_split < n_out, a GLU output without its conditions); QF_EUNSUPPORTED (rows > 8, k not a
 * multiple of 8); QF_EALIGN (x, w, gain not 16-byte aligned, out, out_b, residual not 2-byte
 * aligned); QF_EHIP (launch failed).  rows == 0 is a no-op.
 */
#define QF_LINEAR_PLAIN 0
#define QF_LINEAR_RMS_NORM 1
#define QF_LINEAR_SWIGLU 2
#define QF_LINEAR_GLU_OUT 16
int qf_linear(int32_t rows, int32_t n_out, int32_t k, int32_t prologue, const void* x,
              const void* w, const void* gain, float eps, const void* residual, void* out,
              int32_t n_split, void* out_b, void* stream);

/* The arguments of one qf_linear call, as a struct (for qf_attn_decode_split_beside). */
typedef struct {
  int32_t rows, n_out, k, prologue;
  const void* x;
  const void* w;
  const void* gain;
  float eps;
  const void* residual;
  void* out;
  int32_t n_split;
  void* out_b;
} qf_linear_args;

/*
 * The sweep beside the feed-forward (§3: the sweep of one layer and the feed-forward of another
 * do not wait for each other's results, so they may run at once): exactly qf_attn_decode_split(desc, q, ..., workspace_size) and
 * qf_linear(*beside), issued as ONE launch whose workgroups take either role, so that on one GPU
 * the two share every CU instead of running one after the other (preceded by the small kernel
 * that writes the dispatch order, where qf_attn_decode_split has one).  Results are bitwise those of
 * the two separate calls.  The caller guarantees that neither call's outputs overlap the other's
 * inputs or outputs.  Arguments, errors and ownership are those of the two calls (checked before
 * anything is launched); `beside` is a HOST pointer, read during the call.  With batch == 0 or
 * beside->rows == 0 only the other call is issued.
 */
int qf_attn_decode_split_beside(const qf_decode_desc* desc, const void* q, const void* k_cache,
                                const void* v_cache, const int32_t* block_table,
                                const int32_t* ctx_lens, const int32_t* n_shards,
                                float* part_out, float* part_lse, void* workspace,
                                size_t workspace_size, const qf_linear_args* beside,
                                void* stream);

/* Message for the last error on the calling thread; "" if none.  Valid until the thread's next
 * call into the library. */
const char* qf_last_error(void);

/* QF_VERSION of the loaded library. */
int qf_version(void);

#ifdef __cplusplus
}
#endif

#endif /* QFATTN_H */

/*
 * kvr.h -- C ABI of the KV-Rescue candidate-decode hot path (arxiv 2608.15797)
 * on AMD Instinct MI355X (gfx950).
 *
 * The library computes, for a batch of candidate sequences decoding one token
 * each (Eq. (3): N base and N helper candidates are sampled per reasoning step
 * and decoded together):
 *   - grouped-query decode attention over a KV-evicted cache (Eq. (1), third
 *     line) or over a full-context cache made of a shared prefix plus a private
 *     suffix (the full-context helper of Sec. 3.1), with the new token's key
 *     and value appended in the same call;
 *   - the accumulated-attention importance score of Sec. 2.1, summed over an
 *     observation window, either streamed during decode or recomputed from the
 *     window's queries;
 *   - TopB selection with a protected recent window and in-place compaction of
 *     every KV head (Eq. (1), first two lines; eviction settings of Sec. 4.1
 *     and the implementation details);
 *   - the full-vocabulary token entropy of Eq. (4) with the moving-average
 *     degeneration detector of Sec. 3.2.
 *
 * Conventions shared by every entry point
 *   - All array pointers are DEVICE pointers owned by the caller. The library
 *     never allocates, frees or retains them, and keeps no global state (the
 *     one exception is the device scratch of kvr_logit_entropy_batch_noalloc):
 *     calls on different streams are independent when their buffers do not
 *     alias.
 *   - Arrays are row-major with the innermost index last. Element types are
 *     float32 (KVR_F32) or bfloat16 (KVR_BF16); arithmetic is float32.
 *   - bfloat16 arrays and float32 vector arrays must be 16-byte aligned.
 *   - Every call validates its arguments on the host and returns a status;
 *     on any error nothing is enqueued. Work is enqueued on `stream` (NULL =
 *     the default stream) and completes asynchronously; a device fault shows
 *     up at the caller's next synchronisation.
 *   - Live lengths (len[s]) are caller-owned device arrays the library only
 *     reads; the caller advances them (a decode driver knows every length in
 *     advance: +1 per token, B after an eviction).
 */
#ifndef KVR_H
#define KVR_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define KVR_OK 0
#define KVR_EINVAL (-1)        /* bad pointer, shape, alignment or policy     */
#define KVR_EUNSUPPORTED (-2)  /* valid but not implemented (dtype, D, G, LDS) */
#define KVR_EHIP (-3)          /* the HIP runtime refused a launch            */
#define KVR_EWORKSPACE (-4)    /* workspace missing or too small              */

/* Element types. */
#define KVR_F32 0
#define KVR_BF16 1

/* Static description of a per-sequence KV cache.
 *   k, v : [S][L][Hkv][cap][D] elements of `dtype`, device memory.
 *   pos  : [S][L][Hkv][cap] int32 original token position of each slot, or
 *          NULL when positions are not tracked. */
typedef struct kvr_cache {
    void *k;
    void *v;
    int32_t *pos;
    int32_t S, L, Hkv, cap, D;
    int32_t dtype;
} kvr_cache;

/* Full-context prefix shared by groups of candidates (Sec. 2.2: candidates of
 * one step share the committed context).
 *   k, v : [P][L][Hkv][plen][D] of the cache dtype. Sequence s reads prefix
 *          s / (S / P); S must be a multiple of P (P == S: private contexts). */
typedef struct kvr_prefix {
    const void *k;
    const void *v;
    int32_t P, plen;
} kvr_prefix;

/* Eviction policy (Eq. (1) TopB with a protected recent window).
 *   B      : entries kept after an eviction, including the window;
 *   W      : protected recent window, also the observation window whose
 *            attention mass forms the importance score; 0 < W < B;
 *   buffer : headroom; a sequence evicts when its live length exceeds
 *            B + buffer. buffer >= W - 1 so every window step follows the
 *            previous eviction. The cache needs cap >= B + buffer + 1. */
typedef struct kvr_policy {
    int32_t B, W, buffer;
} kvr_policy;

/* Entropy-detector state for R candidate rows (Eq. (4) moving average;
 * implementation details: tau = 7.0, guard 24, window 12).
 *   hist : [R][window] float32, last `window` entropies in push order mod window;
 *   cnt  : [R] int32, entropies pushed so far;
 *   flag : [R] uint8, sticky degeneration flag.
 * State starts zeroed. Each call pushes H[r], increments cnt[r] and, once
 * cnt[r] >= guard, sets flag[r] = 1 if the mean of the last min(cnt, window)
 * entropies exceeds tau. */
typedef struct kvr_detector {
    float *hist;
    int32_t *cnt;
    uint8_t *flag;
    int32_t window, guard;
    float tau;
} kvr_detector;

/* Token sampler fused with the entropy pass (Sec. 4.1 decoding setup:
 * temperature 0.8, top-p 0.95, top-k 20).
 *   temperature : > 0; probabilities are softmax(logits / temperature);
 *   top_k       : 1 .. 64 candidates by logit, ties to the lower token id;
 *   top_p       : (0, 1]; the shortest prefix of the top_k (by probability,
 *                 renormalised over them) whose cumulative mass reaches top_p;
 *   seed, step  : the draw for row r uses u = top 24 bits of the first word of
 *                 Philox4x64-10 with counter (step, r, 0, 0) and key (seed, 0),
 *                 divided by 2^24; the token is the first of the prefix whose
 *                 cumulative mass exceeds u times the prefix mass. */
typedef struct kvr_sampler {
    float temperature;
    int32_t top_k;
    float top_p;
    uint64_t seed;
    uint64_t step;
} kvr_sampler;

/* Message for a status code (static storage). */
const char *kvr_strerror(int status);

/* Human-readable detail of the last failing call on this host thread. */
const char *kvr_last_error(void);

/*
 * kvr_decode_attn -- one decode step of grouped-query attention for S
 * candidate sequences and all L layers (Eq. (1) third line; Eq. (3)).
 *
 *   cache   : the sequences' own caches (evicted base cache, or the helper's
 *             private suffix). Written only at slot len[s]-1 (append).
 *   prefix  : NULL, or the shared full-context prefix attended before the own
 *             cache (helper). Requires a workspace (see below).
 *   len     : [S] int32 device, live entries of sequence s INCLUDING the token
 *             appended by this call; 1 <= len[s] <= cap.
 *   q       : [S][L][Hq][D], Hq = G * Hkv, 1 <= G <= 16. Query head qh reads
 *             KV head qh / G.
 *   scale   : softmax scale applied to q.k (commonly 1/sqrt(D)).
 *   k_new, v_new : [S][L][Hkv][D] key/value of the new token, written to slot
 *             len[s]-1 before attending; NULL when the caller already stored
 *             them (then both must be NULL).
 *   new_pos : [S] int32 original position of the new token, stored into
 *             cache->pos when both are non-NULL.
 *   out     : [S][L][Hq][D] attention output, cache dtype.
 *   policy, scores : NULL/NULL for no scoring. Otherwise scores is
 *             [S][L][Hkv][cap] float32 and the call streams the importance
 *             score: a sequence whose len n satisfies n >= B + buffer + 2 - W
 *             is in its observation window; for such a sequence, with
 *             r_j = sum over the G query heads of KV head h of softmax
 *             probability of slot j, the call sets scores[j] = r_j when n is
 *             the first window length or j == n-1, and scores[j] += r_j
 *             otherwise, for j < n. Other sequences' scores are untouched.
 *             Scoring is not available together with a prefix.
 *   workspace, workspace_bytes : device scratch of at least
 *             kvr_decode_attn_workspace_size() bytes (no initialisation
 *             needed); may be NULL/0 when that size is 0.
 * Errors: KVR_EINVAL (shape, pointer, alignment, policy), KVR_EUNSUPPORTED
 * (D not 64/128, G > 16, dtype, LDS limit), KVR_EWORKSPACE, KVR_EHIP.
 */
int kvr_decode_attn(const kvr_cache *cache, const kvr_prefix *prefix, const int32_t *len,
                    const void *q, int32_t Hq, float scale, const void *k_new,
                    const void *v_new, const int32_t *new_pos, void *out,
                    const kvr_policy *policy, float *scores, void *workspace,
                    size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes kvr_decode_attn needs for this geometry (0 without prefix). */
size_t kvr_decode_attn_workspace_size(const kvr_cache *cache, const kvr_prefix *prefix,
                                      int32_t Hq);

/*
 * kvr_accumulate_scores -- importance score recomputed from the last nq
 * queries of every sequence (accumulated attention of Sec. 2.1 over an
 * observation window; used when a step's tokens are encoded in one pass, as
 * when a helper step is committed to the base, Sec. 3.1 and Alg. 1).
 *
 *   cache, len : as for kvr_decode_attn (len includes all nq window tokens,
 *             which must already be in the cache).
 *   q_win   : [S][L][Hq][nq][D] queries of the last nq tokens, oldest first.
 *             Window row r attends causally over len[s] - (nq-1-r) entries.
 *   scores  : [S][L][Hkv][cap] float32. For j < len[s]: scores[j] = sum over
 *             rows r and the G query heads of KV head h of the probability of
 *             slot j (0 where row r cannot see j). accumulate != 0 adds to the
 *             stored value instead of overwriting. Slots >= len[s] untouched.
 * Results are bitwise reproducible (the bf16 kernels sum the per-row-block
 * contributions in 64-bit fixed point, 2^-32 resolution). Errors: as
 * kvr_decode_attn, and KVR_EUNSUPPORTED when cap exceeds 8192 slots (bf16:
 * one 8-byte accumulator per slot in 64 KiB of LDS) or (D + 2 cap) floats
 * exceed 64 KiB (float32).
 */
int kvr_accumulate_scores(const kvr_cache *cache, const int32_t *len, const void *q_win,
                          int32_t nq, int32_t Hq, float scale, float *scores,
                          int32_t accumulate, hipStream_t stream);

/*
 * kvr_evict_topb -- TopB eviction with a protected recent window and in-place
 * compaction (Eq. (1) first two lines).
 *
 * For every sequence with n = len[s] > B + buffer, and every (layer, KV head)
 * independently: the W newest slots [n-W, n) are kept; of the slots [0, n-W)
 * the B-W with the largest scores are kept, ties going to the lower slot
 * (selected by a wavefront radix select on the scores' order-preserving
 * 32-bit keys). The kept rows of k, v (and pos) move to slots 0..B-1 in their
 * original order. Sequences with len[s] <= B + buffer are not touched.
 *
 *   len     : [S] int32 device, live lengths (read only).
 *   len_out : NULL, or [S] int32 device receiving the new live lengths: B for
 *             evicted sequences, len[s] for the others. Must not overlap len
 *             (KVR_EINVAL). Callers that track lengths themselves pass NULL.
 *   scores  : [S][L][Hkv][cap] float32 importance scores (read only).
 *   kept    : NULL or [S][L][Hkv][B] int32, receives the kept pre-eviction
 *             slot ids in ascending order for evicted sequences.
 * Errors: KVR_EINVAL (shape, pointer, policy, overlap), KVR_EUNSUPPORTED (D,
 * dtype, cap + B above 16384 slots of LDS), KVR_EHIP.
 */
int kvr_evict_topb(const kvr_cache *cache, const int32_t *len, int32_t *len_out, const float *scores,
                   const kvr_policy *policy, int32_t *kept, hipStream_t stream);

/*
 * kvr_redundancy_scores -- redundancy-aware eviction score: query-attention
 * importance mixed with key redundancy (cosine similarity) with weight lambda,
 * after pooling (App. C, KV eviction; App. D.3). The paper names these parts
 * but gives no formula; this is the reading implemented. For every sequence
 * with n = len[s] > B + buffer and every (layer, KV head), over the candidates
 * c < m = n - W:
 *   P_c   = max of importance over the candidates within pool/2 slots of c;
 *   R_c   = mean cosine similarity of key c to the other m - 1 candidate keys
 *           (a zero key has cosine 0 with every key);
 *   out_c = lam * P_c / sum_c' P_c' - (1 - lam) * softmax_c(R)
 *           (the importance term is 1/m when all P are 0).
 * Other slots and sequences are not written. Feed `out` to kvr_evict_topb.
 *
 *   importance : [S][L][Hkv][cap] float32, e.g. the window scores streamed by
 *                kvr_decode_attn; `out` may be the same array.
 *   lam        : in [0, 1]; the paper uses 0.1.  pool : >= 1 (7 is common).
 * Errors: KVR_EINVAL (pointer, policy, lambda, pool), KVR_EUNSUPPORTED (dtype,
 * D, LDS: 3 cap + 5 D + 4 floats must fit in 64 KiB), KVR_EHIP.
 */
int kvr_redundancy_scores(const kvr_cache *cache, const int32_t *len, const float *importance,
                          const kvr_policy *policy, float lam, int32_t pool, float *out,
                          hipStream_t stream);

/*
 * kvr_logit_entropy -- token entropy H = -sum_v p(v) log p(v) of
 * p = softmax(inv_temp * logits) for R rows (Eq. (4)), natural log.
 *
 *   logits : [R][ld] of `dtype`; the first V columns of each row are used.
 *            ld >= V; for 16-byte vector loads ld * element size should be a
 *            multiple of 16 (other ld values run a scalar path).
 *   H      : [R] float32 output.
 *   det    : NULL, or detector state updated with the new entropies.
 *   workspace : at least kvr_logit_entropy_workspace_size(R, V) bytes of
 *            device scratch for per-split partial sums (no initialisation
 *            needed). May be NULL/0 when that size is 0.
 *   inv_temp : positive and finite (KVR_EINVAL otherwise).
 * -inf logits are allowed (they contribute 0); a row of only -inf is invalid.
 */
int kvr_logit_entropy(const void *logits, int32_t dtype, int32_t R, int32_t V, int64_t ld,
                      float inv_temp, float *H, const kvr_detector *det, void *workspace,
                      size_t workspace_bytes, hipStream_t stream);

size_t kvr_logit_entropy_workspace_size(int32_t R, int32_t V);

/* One set of logit rows for kvr_logit_entropy_batch; the fields mean what the
 * arguments of kvr_logit_entropy of the same names mean. */
typedef struct kvr_logit_set {
    const void *logits;   /* [R][ld] of dtype */
    int32_t dtype;
    int32_t R, V;
    int64_t ld;
    float inv_temp;
    float *H;             /* [R] float32 output */
    const kvr_detector *det;  /* NULL or this set's own detector state */
} kvr_logit_set;

#define KVR_ENTROPY_MAX_SETS 4

/*
 * kvr_logit_entropy_batch -- kvr_logit_entropy over several sets of rows in
 * one pass: the token entropies of every model that decodes in a step (the
 * base and helper logits of Eq. (4), one launch for all candidates and both
 * vocabularies, Sec. 3.1 batching). Each set keeps its own vocabulary size,
 * row stride, temperature, output and detector.
 *
 *   sets      : nsets descriptors in host memory (read during the call only).
 *   nsets     : 1 .. KVR_ENTROPY_MAX_SETS; every set has the same dtype, and
 *               the total row count is at most 65535.
 *   workspace : at least kvr_logit_entropy_batch_workspace_size(sets, nsets)
 *               bytes, 16-byte aligned (no initialisation); may be NULL/0
 *               when that size is 0.
 * The H and detector arrays of different sets must not overlap.
 * Errors: KVR_EINVAL (a set's arguments as for kvr_logit_entropy, nsets out
 * of range, mixed dtypes, too many rows), KVR_EUNSUPPORTED (dtype),
 * KVR_EWORKSPACE, KVR_EHIP. Nothing is enqueued on error.
 */
int kvr_logit_entropy_batch(const kvr_logit_set *sets, int32_t nsets, void *workspace,
                            size_t workspace_bytes, hipStream_t stream);

/* Depends on the sets' dtype, R, V, ld and inv_temp only (their pointers
 * are not read); 0 when those are invalid. */
size_t kvr_logit_entropy_batch_workspace_size(const kvr_logit_set *sets, int32_t nsets);

/*
 * kvr_decode_attn_entropy -- kvr_decode_attn and kvr_logit_entropy_batch over
 * the step's logit sets in one launch: the detector's entropies are
 * by-products of the decode step (App. C: the signals add negligible cost),
 * so their rows are read while the attention waves stream their caches (Eq.
 * (1) third line; Sec. 3.1; Eq. (4)).
 *
 * Arguments, results and errors are those of kvr_decode_attn (cache, prefix,
 * ..., workspace) and of kvr_logit_entropy_batch (sets, nsets), with one more
 * requirement: every set's rows start 16-byte aligned (logits and ld *
 * element size), KVR_EINVAL otherwise. Each logit row is reduced whole by one
 * wavefront of the launch, so the rows need no workspace.
 *   Without a prefix the rows ride in the own-cache launch, and the attention
 *   outputs and scores are bit for bit those of kvr_decode_attn.
 *   With a prefix (bfloat16 cache) they ride in the context launch, whose
 *   split plan gives their wavefronts slots of their own (at most half of
 *   the chip's), so the context is cut at other points than kvr_decode_attn
 *   cuts it: the outputs agree with kvr_decode_attn's to the rounding of
 *   the split partials. The workspace size is kvr_decode_attn_workspace_size
 *   (cache, prefix, Hq), which covers this plan.
 * The entropies agree with kvr_logit_entropy_batch to float32 rounding
 * (different summation order). For a float32 cache the entropy rows run as
 * a second kernel on the same stream.
 */
int kvr_decode_attn_entropy(const kvr_cache *cache, const kvr_prefix *prefix, const int32_t *len, const void *q,
                            int32_t Hq, float scale, const void *k_new, const void *v_new, const int32_t *new_pos,
                            void *out, const kvr_policy *policy, float *scores, void *workspace,
                            size_t workspace_bytes, const kvr_logit_set *sets, int32_t nsets, hipStream_t stream);

/*
 * kvr_decode_attn_entropy_sample -- kvr_decode_attn_entropy, and the next
 * token of every logit row drawn in the same launch (the sampler of
 * kvr_logit_entropy_sample, Sec. 4.1 decoding setup: temperature, top-k,
 * top-p): the step's decode attention, entropies, detector update and token
 * draw in one pass over the cache and the logits.
 *
 *   sampler : the settings of kvr_sampler, applied to every set; required.
 *   tokens  : host array of nsets pointers, tokens[k] an [R_k] int32 device
 *             array receiving the sampled ids of set k (the draw for row r of
 *             a set uses counter (step, r, 0, 0), as kvr_logit_entropy_sample
 *             does for that set's rows alone).
 * Arguments, results and errors otherwise as kvr_decode_attn_entropy; the
 * tokens are those kvr_logit_entropy_sample draws from the same rows with the
 * same settings (both take the k largest logits, ties to the lower id, and
 * the same draw). Errors: KVR_EINVAL also for sampler settings out of range
 * or a NULL tokens array or entry. Each row wave keeps its candidates in
 * 2 KiB of its LDS.
 */
int kvr_decode_attn_entropy_sample(const kvr_cache *cache, const kvr_prefix *prefix, const int32_t *len,
                                   const void *q, int32_t Hq, float scale, const void *k_new, const void *v_new,
                                   const int32_t *new_pos, void *out, const kvr_policy *policy, float *scores,
                                   void *workspace, size_t workspace_bytes, const kvr_logit_set *sets,
                                   int32_t nsets, const kvr_sampler *sampler, int32_t *const *tokens,
                                   hipStream_t stream);

/* Bytes of device scratch the library holds per GPU for
 * kvr_logit_entropy_batch_noalloc (the largest workspace it accepts). */
#define KVR_ENTROPY_SCRATCH_BYTES ((size_t)1 << 20)

/*
 * kvr_logit_entropy_batch_noalloc -- kvr_logit_entropy_batch without a caller
 * workspace and without allocating anything: for callers that cannot call
 * hipMalloc or pass fresh device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation). Same sets, results and
 * errors as kvr_logit_entropy_batch.
 *
 * The split partials go to a device array of KVR_ENTROPY_SCRATCH_BYTES that
 * the library holds on each GPU until the process ends (its address on a
 * device is looked up on the first call made with that device current). A
 * call whose workspace size (kvr_logit_entropy_batch_workspace_size) exceeds
 * it fails with KVR_EUNSUPPORTED and enqueues nothing. Every call on one GPU
 * shares that array: calls that overlap in time on one GPU (other streams,
 * other host threads) race and may return wrong entropies; calls on one
 * stream are ordered and safe. `stream` must belong to the current device
 * (KVR_EINVAL otherwise). Nothing needs clearing between calls: every partial
 * a call reads was written earlier in the same call.
 */
int kvr_logit_entropy_batch_noalloc(const kvr_logit_set *sets, int32_t nsets, hipStream_t stream);

/*
 * kvr_logit_entropy_sample -- kvr_logit_entropy and the next token of every
 * row from the same single pass over the logits (Eq. (4) entropy and the
 * detector as there; sampling as described at kvr_sampler).
 *
 *   tokens    : [R] int32 output, the sampled token id of each row.
 *   workspace : at least kvr_logit_entropy_sample_workspace_size(R, V, top_k)
 *               bytes of device scratch, 16-byte aligned (no initialisation).
 * Rows must hold at least one finite logit; NaN logits are not supported.
 * Errors: as kvr_logit_entropy, plus KVR_EINVAL for sampler settings out of
 * range.
 */
int kvr_logit_entropy_sample(const void *logits, int32_t dtype, int32_t R, int32_t V, int64_t ld,
                             float inv_temp, float *H, const kvr_detector *det,
                             const kvr_sampler *sampler, int32_t *tokens, void *workspace,
                             size_t workspace_bytes, hipStream_t stream);

size_t kvr_logit_entropy_sample_workspace_size(int32_t R, int32_t V, int32_t top_k);

/*
 * kvr_fork -- batched copy of live KV slots between sequences: forking the N
 * base candidates of a step from the persistent trajectory state, and
 * retaining a selected base candidate as the new state (App. C, the fork-based
 * best-of-(N+N) engine; Sec. 3.1 and Alg. 1: the selected base fork becomes
 * the next base state).
 *
 *   src, dst : caches with equal L, Hkv, D and dtype; S and cap may differ.
 *              They may describe the same cache: a row that is a source must
 *              then be its own source (src_index[r] == r, a no-op), otherwise
 *              what such a row passes on is unspecified.
 *   src_index: [dst->S] int32 device: source sequence of each destination.
 *              Destinations with an index outside [0, src->S) are skipped.
 *   len      : [dst->S] int32 device: slots to copy, clamped to [0, min(src
 *              cap, dst cap)]. For every (layer, KV head), slots [0, len[s])
 *              of k, v (and pos when both caches track positions) move from
 *              the source; slots beyond are untouched.
 *   src_scores, dst_scores : NULL/NULL, or [S][L][Hkv][cap] float32 score rows
 *              of the two caches, copied alongside (streamed window sums that a
 *              fork inherits).
 * Consecutive destinations (groups of 8) that share a source are served by
 * workgroups that read each piece of the source once, so a source fanned out
 * to N consecutive candidates is read from HBM once per group.
 * Errors: KVR_EINVAL (shape or pointer mismatch, dst->pos without src->pos,
 * one of the score pointers NULL), KVR_EUNSUPPORTED (dtype, D, L * Hkv above
 * 32767 or dst->S above 524280), KVR_EHIP.
 */
int kvr_fork(const kvr_cache *src, const kvr_cache *dst, const int32_t *src_index,
             const int32_t *len, const float *src_scores, float *dst_scores,
             hipStream_t stream);

/*
 * kvr_append -- bulk append of T tokens to every sequence: the base model
 * encoding an accepted helper step in one forward pass (App. C; Alg. 1:
 * append s_t to the base cache, then evict), or a prompt compressed in one
 * shot. Score the appended window with kvr_accumulate_scores (nq = min(W, T))
 * and evict with kvr_evict_topb afterwards.
 *
 *   len     : [S] int32 device, live length BEFORE the append (read only).
 *   T       : tokens per sequence, T >= 0 (0: nothing is enqueued).
 *   k_new, v_new : [S][L][Hkv][T][D] of the cache dtype; token i of
 *             sequence s goes to slot len[s] + i of every (layer, KV head).
 *   pos_new : NULL, or [S][T] int32 original positions, written to every
 *             layer and head (needs cache->pos).
 * Slots at or beyond cap are not written; the caller keeps len[s] + T <= cap.
 * Errors: KVR_EINVAL (pointer, alignment, T < 0, pos_new without cache->pos),
 * KVR_EUNSUPPORTED (dtype, D), KVR_EHIP.
 */
int kvr_append(const kvr_cache *cache, const int32_t *len, int32_t T, const void *k_new,
               const void *v_new, const int32_t *pos_new, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* KVR_H */
